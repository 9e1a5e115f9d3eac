"""C-ABI checks that need no GPU: the library loads, exports every entry point
the header declares, and rejects bad arguments on the host before any HIP
call (so no compute is launched here)."""
import ctypes
import os
import re
import subprocess

import pytest

from paper_2506_03781_amd import uniquan as uq

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def L():
    if not os.path.exists(uq.LIB_PATH):
        pytest.fail("libuniquan.so is not built; run __graft_entry__.build()")
    return uq.lib()


def test_exports_every_declared_symbol(L):
    decl = uq.declared_symbols()
    assert len(decl) >= 12
    for name in decl:
        assert hasattr(L, name), name
    # and the binding wraps each compute entry point under the same name
    for name in decl:
        if name not in ("uniquan_abi_version", "uniquan_last_error"):
            assert hasattr(uq, name), name


def test_dynamic_symbol_table_matches_header(L):
    out = subprocess.run(["nm", "-D", "--defined-only", uq.LIB_PATH], capture_output=True, text=True).stdout
    exported = set(re.findall(r"\b(uniquan_[a-z0-9_]+)\b", out))
    assert set(uq.declared_symbols()) <= exported


def test_abi_version(L):
    hdr = open(uq.HEADER).read()
    ver = int(re.search(r"#define UNIQUAN_ABI_VERSION (\d+)", hdr).group(1))
    assert L.uniquan_abi_version() == ver


FAKE = 1 << 20          # 16-byte aligned non-null "device" address, never dereferenced
ODD = FAKE + 4          # misaligned for 16-byte arrays


def fwd(L, R=4, C=256, k=3, g=128, W=FAKE, wdt=uq.UQ_BF16, s=FAKE, alpha=FAKE, z_b=FAKE, mode=0,
        codes=FAKE, W_hat=FAKE, odt=uq.UQ_BF16, s_r=None, delta=None, z_u=None):
    return L.uniquan_fq_fwd(R, C, k, g, W, wdt, s, s_r, delta, z_u, alpha, z_b, mode, codes, W_hat, odt, None)


@pytest.mark.parametrize("kw,status,text", [
    (dict(k=0), uq.UQ_EINVAL, "k=0"),
    (dict(k=8), uq.UQ_EINVAL, "k=8"),
    (dict(g=96), uq.UQ_EUNSUPPORTED, "power of two"),
    (dict(g=4), uq.UQ_EINVAL, "multiple of 8"),
    (dict(g=1028, C=2056), uq.UQ_EINVAL, "multiple of 8"),
    (dict(g=1032, C=2048), uq.UQ_EINVAL, "divide"),
    (dict(C=192), uq.UQ_EINVAL, "divide"),
    (dict(R=0), uq.UQ_EINVAL, "R=0"),
    (dict(W=None), uq.UQ_EINVAL, "W must not be NULL"),
    (dict(s=ODD), uq.UQ_EINVAL, "s must be 16-byte aligned"),
    (dict(codes=None), uq.UQ_EINVAL, "codes"),
    (dict(mode=3), uq.UQ_EINVAL, "mode"),
    (dict(wdt=2), uq.UQ_EINVAL, "dtype"),
    (dict(s_r=FAKE + 2), uq.UQ_EINVAL, "s_r"),
])
def test_fq_fwd_validation(L, kw, status, text):
    assert fwd(L, **kw) == status
    assert text in uq.last_error()


def test_large_groups_accepted_where_supported(L):
    """Groups of more than 512 weights (any multiple of 8 dividing C, e.g. one
    row of 11008): the quantizer entry points take them, the unified
    initialisation up to 16384 weights per group, the fused gradient-GEMM
    backward not at all."""
    assert L.uniquan_init_unified(4, 16392, 3, 16392, FAKE, 1, 30, 15, 0, FAKE, FAKE, FAKE, FAKE, None, None,
                                  None, None, None) == uq.UQ_EUNSUPPORTED
    assert "up to 16384" in uq.last_error()
    assert L.uniquan_layer_grad_ste_sgd(64, 4, 4096, 3, 4096, FAKE, FAKE, FAKE, 1, FAKE, None, None, None, FAKE,
                                        FAKE, FAKE, 0.1, 0.1, None, None, None, None) == uq.UQ_EUNSUPPORTED


def test_fq_bwd_validation(L):
    args = [4, 256, 3, 128, FAKE, 1, FAKE, None, None, None, FAKE, FAKE, FAKE, FAKE, 1,
            FAKE, FAKE, FAKE, None, None, FAKE, None, None]
    assert L.uniquan_fq_bwd(*args) == uq.UQ_EINVAL          # grad_s_r without group_ws
    assert "group_ws" in uq.last_error()
    args2 = list(args)
    args2[15] = ODD
    args2[20] = None
    assert L.uniquan_fq_bwd(*args2) == uq.UQ_EINVAL
    assert "grad_s" in uq.last_error()


def test_recon_validation(L):
    ws = L.uniquan_recon_ws(64, 256, 256)
    assert ws >= 1
    assert L.uniquan_layer_recon(60, 256, 256, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, ws, FAKE, 1, None) \
        == uq.UQ_EINVAL
    assert "multiple of 8" in uq.last_error()
    assert L.uniquan_layer_recon(64, 256, 256, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, ws - 1, FAKE, 1, None) \
        == uq.UQ_EINVAL
    assert "partials_len" in uq.last_error()
    assert L.uniquan_layer_recon(64, 256, 256, FAKE, None, FAKE, FAKE, FAKE, FAKE, FAKE, ws, FAKE, 1, None) \
        == uq.UQ_EINVAL
    assert "Xt" in uq.last_error()
    assert L.uniquan_layer_target(64, 256, 250, FAKE, FAKE, FAKE, None) == uq.UQ_EINVAL


def test_other_validation(L):
    assert L.uniquan_fold_to_bcq(4, 256, 3, 128, FAKE, 1, FAKE, None, None, None, FAKE, FAKE, FAKE, FAKE,
                                 FAKE, 2, None) == uq.UQ_EINVAL
    assert L.uniquan_bcq_dequant(4, 256, 3, 128, FAKE, FAKE, FAKE, FAKE, 5, None) == uq.UQ_EINVAL
    assert L.uniquan_init_greedy(4, 256, 3, 100, FAKE, 1, FAKE, None, None, None, FAKE, FAKE, None) == uq.UQ_EINVAL
    assert L.uniquan_sgd(0, FAKE, FAKE, ctypes.c_float(0.1), None) == uq.UQ_EINVAL


def test_layer_grad_ste_sgd_validation(L):
    def call(T=64, k=3, g=128, codes=FAKE):
        return L.uniquan_layer_grad_ste_sgd(T, 64, 256, k, g, FAKE, FAKE, FAKE, 1, FAKE, None, None, None,
                                            FAKE, FAKE, codes, ctypes.c_float(0.1), ctypes.c_float(0.1),
                                            None, None, None, None)
    assert call(k=5) == uq.UQ_EUNSUPPORTED
    assert call(g=256) == uq.UQ_EUNSUPPORTED
    assert call(T=48) == uq.UQ_EUNSUPPORTED
    assert call(T=60) == uq.UQ_EINVAL
    assert call(codes=None) == uq.UQ_EINVAL


@pytest.mark.parametrize("kw,status,text", [
    (dict(k=5), uq.UQ_EUNSUPPORTED, "k = 5"),
    (dict(G=0), uq.UQ_EINVAL, "grid_G"),
    (dict(G=4097), uq.UQ_EINVAL, "grid_G"),
    (dict(T=-1), uq.UQ_EINVAL, "alt_T"),
    (dict(clip=3), uq.UQ_EINVAL, "clip"),
    (dict(g=100), uq.UQ_EINVAL, "g=100"),
    (dict(alpha=None), uq.UQ_EINVAL, "alpha"),
    (dict(codes=FAKE + 4), uq.UQ_EINVAL, "codes"),
    (dict(W=ODD), uq.UQ_EINVAL, "W"),
])
def test_init_unified_validation(L, kw, status, text):
    a = dict(k=3, g=128, G=30, T=15, clip=0, W=FAKE, alpha=FAKE, codes=None)
    a.update(kw)
    st = L.uniquan_init_unified(4, 256, a["k"], a["g"], a["W"], 1, a["G"], a["T"], a["clip"],
                                FAKE, FAKE, a["alpha"], FAKE, a["codes"], None, None, None, None)
    assert st == status
    assert text in uq.last_error()
    assert L.uniquan_transpose_bf16(12, 16, FAKE, FAKE, None) == uq.UQ_EINVAL


def bcq_mm(L, T=1, R=256, C=512, k=3, g=128, X=FAKE, planes=FAKE, a16=FAKE, z16=FAKE, Y=FAKE, ws=FAKE,
           ws_len=1 << 30):
    return L.uniquan_bcq_matmul(T, R, C, k, g, X, planes, a16, z16, Y, ws, ws_len, None)


@pytest.mark.parametrize("kw,status,text", [
    (dict(k=5), uq.UQ_EUNSUPPORTED, "k=5"),
    (dict(C=320), uq.UQ_EUNSUPPORTED, "multiple of 128"),
    (dict(C=(1 << 22) + 128, R=2), uq.UQ_EUNSUPPORTED, "2^22"),
    (dict(g=64), uq.UQ_EUNSUPPORTED, "g=64"),
    (dict(g=384), uq.UQ_EINVAL, "divide"),
    (dict(T=9), uq.UQ_EUNSUPPORTED, "T=9"),
    (dict(T=0), uq.UQ_EUNSUPPORTED, "T=0"),
    (dict(planes=ODD), uq.UQ_EINVAL, "planes"),
    (dict(X=None), uq.UQ_EINVAL, "X"),
    (dict(ws_len=3), uq.UQ_EINVAL, "partials_len"),
])
def test_bcq_matmul_validation(L, kw, status, text):
    assert bcq_mm(L, **kw) == status
    assert text in uq.last_error()


def test_bcq_pack_validation(L):
    assert L.uniquan_bcq_pack(4, 256, 5, 128, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, None) == uq.UQ_EUNSUPPORTED
    assert L.uniquan_bcq_pack(4, 200, 2, 128, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, None) == uq.UQ_EUNSUPPORTED
    assert L.uniquan_bcq_pack(4, 256, 2, 128, FAKE, FAKE, FAKE, ODD, FAKE, FAKE, None) == uq.UQ_EINVAL
    assert "planes" in uq.last_error()
    assert L.uniquan_bcq_pack(0, 256, 2, 128, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, None) == uq.UQ_EINVAL
    # workspace: one partial row set per column slab, none for a single slab
    assert uq.uniquan_bcq_matmul_ws(1, 4096, 4096) == 32 * 4096
    assert uq.uniquan_bcq_matmul_ws(2, 28672, 8192) == 16 * 2 * 28672
    assert uq.uniquan_bcq_matmul_ws(1, 100, 128) == 0


def test_block_entry_validation(L):
    F = uq.UQ_F32
    assert L.uniquan_gemm_nt(0, 8, 8, FAKE, FAKE, FAKE, F, 1.0, None) == uq.UQ_EINVAL
    assert L.uniquan_gemm_nt(4, 12, 8, FAKE, FAKE, FAKE, F, 1.0, None) == uq.UQ_EINVAL
    assert "N=12" in uq.last_error()
    assert L.uniquan_gemm_nt(4, 8, 20, FAKE, FAKE, FAKE, F, 1.0, None) == uq.UQ_EINVAL
    assert L.uniquan_gemm_nt(4, 1 << 26, 8, FAKE, FAKE, FAKE, F, 1.0, None) == uq.UQ_EUNSUPPORTED
    assert L.uniquan_gemm_nt(4, 8, 8, ODD, FAKE, FAKE, F, 1.0, None) == uq.UQ_EINVAL
    assert L.uniquan_gemm_nt(4, 8, 8, FAKE, FAKE, FAKE, 7, 1.0, None) == uq.UQ_EINVAL
    assert L.uniquan_rope_table(0, 128, FAKE, None) == uq.UQ_EINVAL
    assert L.uniquan_rope_table(16, 7, FAKE, None) == uq.UQ_EINVAL
    gh = L.uniquan_gemm_heads
    assert gh(512, 4, 48, FAKE, FAKE, 512, 1, 1, FAKE, FAKE, None) == uq.UQ_EINVAL   # K % 32
    assert gh(512, 4, 64, FAKE, FAKE, 300, 1, 1, FAKE, FAKE, None) == uq.UQ_EINVAL   # L divides T
    assert gh(512, 4, 64, FAKE, FAKE, 512, 3, 1, FAKE, FAKE, None) == uq.UQ_EINVAL   # group divides H
    assert gh(512, 4, 64, FAKE, FAKE, 512, 1, 1, None, FAKE, None) == uq.UQ_EINVAL   # rotation needs the table
    assert gh(512, 4, 64, FAKE, FAKE, 512, 1, -1, FAKE, FAKE, None) == uq.UQ_EINVAL  # n_rot >= 0
    assert gh(512, 4, 64, FAKE, FAKE, 512, 2, 2, FAKE, FAKE, None) == uq.UQ_EINVAL   # some heads only: group 1
    assert uq.uniquan_gemm_block_loss_ws(8192, 4096) == 512
    assert L.uniquan_gemm_block_loss(8, 12, 8, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 64, FAKE, None) == uq.UQ_EINVAL
    assert L.uniquan_gemm_block_loss(8192, 4096, 64, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 10, FAKE, None) == uq.UQ_EINVAL
    rg = L.uniquan_gemm_nt_residual
    assert rg(4, 12, 8, FAKE, FAKE, FAKE, FAKE, None) == uq.UQ_EINVAL     # N % 8
    assert rg(4, 8, 8, FAKE, FAKE, ODD, FAKE, None) == uq.UQ_EINVAL       # R alignment
    assert rg(4, 8, 8, FAKE, FAKE, FAKE, None, None) == uq.UQ_EINVAL      # out required
    sb = L.uniquan_gemm_silu_bwd
    assert sb(64, 36, 64, FAKE, FAKE, 2.0, FAKE, FAKE, FAKE, FAKE, 0, None) == uq.UQ_EINVAL     # I % 8
    assert sb(64, 64, 48, FAKE, FAKE, 2.0, FAKE, FAKE, FAKE, FAKE, 0, None) == uq.UQ_EINVAL     # K % 32
    assert sb(64, 64, 64, FAKE, FAKE, 2.0, FAKE, FAKE, FAKE, FAKE, 56, None) == uq.UQ_EINVAL    # ld_d >= I
    assert "ld_d=56" in uq.last_error()
    assert sb(64, 64, 64, FAKE, FAKE, 2.0, FAKE, FAKE, FAKE, FAKE, 130, None) == uq.UQ_EINVAL   # ld_d % 4
    assert sb(64, 64, 64, FAKE, FAKE, 2.0, FAKE, FAKE, FAKE, ODD, 128, None) == uq.UQ_EINVAL    # dU alignment
    g = L.uniquan_gemm
    assert g(8, 8, 32, FAKE, 2, FAKE, 0, FAKE, F, 1.0, None) == uq.UQ_EINVAL
    assert g(8, 8, 48, FAKE, 1, FAKE, 0, FAKE, F, 1.0, None) == uq.UQ_EINVAL   # K-slow needs K % 32 == 0
    assert "K=48" in uq.last_error()
    assert g(12, 8, 32, FAKE, 1, FAKE, 1, FAKE, F, 1.0, None) == uq.UQ_EINVAL  # K-slow A needs M % 8 == 0
    assert g(12, 8, 32, FAKE, 0, ODD, 1, FAKE, F, 1.0, None) == uq.UQ_EINVAL
    assert g(4, 12, 8, FAKE, 0, FAKE, 0, FAKE, F, 1.0, None) == uq.UQ_EINVAL   # neither: the NT rules
    assert "uniquan_gemm_nt" in uq.last_error()
    assert L.uniquan_silu_mul_fwd(12, FAKE, FAKE, FAKE, None) == uq.UQ_EINVAL
    assert L.uniquan_silu_mul_fwd(0, FAKE, FAKE, FAKE, None) == uq.UQ_EINVAL
    assert L.uniquan_silu_mul_fwd(16, FAKE, None, FAKE, None) == uq.UQ_EINVAL
    assert L.uniquan_silu_mul_bwd(16, FAKE, FAKE, FAKE, ODD, FAKE, None) == uq.UQ_EINVAL
    assert L.uniquan_silu_mul_bwd(20, FAKE, FAKE, FAKE, FAKE, FAKE, None) == uq.UQ_EINVAL


def test_error_text_is_thread_local(L):
    import threading
    fwd(L, k=0)
    seen = {}

    def other():
        seen["t"] = uq.last_error()
    t = threading.Thread(target=other)
    t.start()
    t.join()
    assert seen["t"] == ""
    assert "k=0" in uq.last_error()


def test_binding_refuses_host_tensors():
    import torch
    with pytest.raises(ValueError):
        uq._p(torch.zeros(4), 4, None, "x")


def test_product_never_imports_oracle():
    """The library's Python side and HIP sources stay independent of oracle/."""
    pkg = os.path.join(ROOT, "paper_2506_03781_amd")
    for dirpath, _, files in os.walk(pkg):
        for f in files:
            if f.endswith((".py", ".hip", ".h", ".cpp")):
                txt = open(os.path.join(dirpath, f)).read()
                assert not re.search(r"^\s*(from|import)\s+oracle", txt, re.M), f
                assert "oracle/" not in txt, f


def test_recorder_classifies_launches(L):
    launches = {n for n in uq._SIGS if uq._is_launch(n)}
    assert "uniquan_fq_fwd" in launches and "uniquan_gemm_nt" in launches and "uniquan_bcq_matmul" in launches
    others = {n for n in uq._SIGS if n not in launches}
    assert others == ({"uniquan_abi_version", "uniquan_last_error", "uniquan_probe_mfma_flops", "uniquan_recon_noalloc_max_partials"} | {n for n in uq._SIGS if n.endswith("_ws")})


def test_replay_raises_on_error_status(L):
    bad = uq.Launches([("launch", L.uniquan_sgd, (0, FAKE, FAKE, 0.1, None), None)])
    assert len(bad) == 1
    with pytest.raises(uq.UniquanError, match="n must be"):
        bad(stream=0)


def test_record_propagates_and_resets(L):
    def failing():
        uq._check(uq.lib().uniquan_sgd(0, FAKE, FAKE, 0.1, None))
    with pytest.raises(uq.UniquanError):
        uq.record(failing)
    assert uq._recorder is None and uq.lib() is uq._load()


def test_probe_entry_validation(L):
    assert L.uniquan_probe_mfma_flops(10) == 2.0 * 32 * 32 * 16 * 8 * 10 * 4096
    assert L.uniquan_probe_stream(3, 64, FAKE, FAKE, FAKE, 64, None) == uq.UQ_EINVAL
    assert L.uniquan_probe_stream(0, 24, FAKE, None, FAKE, 64, None) == uq.UQ_EINVAL
    assert L.uniquan_probe_stream(0, 64, None, None, FAKE, 64, None) == uq.UQ_EINVAL
    assert L.uniquan_probe_stream(1, 64, None, None, FAKE, 64, None) == uq.UQ_EINVAL
    assert L.uniquan_probe_stream(2, 64, FAKE, FAKE, FAKE, 0, None) == uq.UQ_EINVAL
    assert L.uniquan_probe_mfma(0, FAKE, None) == uq.UQ_EINVAL


def test_decoder_entry_validation(L):
    B, F = uq.UQ_BF16, uq.UQ_F32
    g = L.uniquan_gemm_nt_batched
    assert g(8, 8, 8, 0, FAKE, 64, FAKE, 64, FAKE, 64, F, 1.0, 0, None) == uq.UQ_EINVAL
    assert g(8, 8, 8, 70000, FAKE, 64, FAKE, 64, FAKE, 64, F, 1.0, 0, None) == uq.UQ_EINVAL
    assert g(8, 8, 8, 2, FAKE, 64, FAKE, 64, FAKE, 32, F, 1.0, 0, None) == uq.UQ_EINVAL
    assert "stride_out" in uq.last_error()
    assert g(8, 8, 8, 2, FAKE, 4, FAKE, 64, FAKE, 64, F, 1.0, 0, None) == uq.UQ_EINVAL
    assert g(8, 12, 8, 2, FAKE, 64, FAKE, 96, FAKE, 96, F, 1.0, 0, None) == uq.UQ_EINVAL
    assert g(8, 8, 8, 2, ODD, 64, FAKE, 64, FAKE, 64, F, 1.0, 0, None) == uq.UQ_EINVAL
    assert g(64, 64, 64, 2, FAKE, 4096, FAKE, 4096, FAKE, 4096, F, 1.0, 4, None) == uq.UQ_EINVAL
    assert g(64, 64, 40, 2, FAKE, 2560, FAKE, 2560, FAKE, 4096, F, 1.0, 1, None) == uq.UQ_EINVAL   # K % 32
    assert g(64, 32, 64, 2, FAKE, 4096, FAKE, 2048, FAKE, 2048, F, 1.0, 1, None) == uq.UQ_EINVAL   # M != N
    assert g(64, 32, 32, 2, FAKE, 2048, FAKE, 1024, FAKE, 2048, F, 1.0, 2, None) == uq.UQ_EINVAL   # M != K
    assert L.uniquan_add_rmsnorm(4, 12, FAKE, None, FAKE, None, FAKE, FAKE, None) == uq.UQ_EINVAL
    assert L.uniquan_add_rmsnorm(4, 16, FAKE, FAKE, FAKE, None, FAKE, FAKE, None) == uq.UQ_EINVAL
    assert "R must be given" in uq.last_error()
    assert L.uniquan_rmsnorm_bwd(4, 16, None, None, FAKE, FAKE, FAKE, None, 2.0, FAKE, None, None) == uq.UQ_EINVAL
    assert L.uniquan_rope_split(6, 2, 4, 4, 1, FAKE, F, 1, FAKE, None) == uq.UQ_EINVAL       # L does not divide T
    assert L.uniquan_rope_split(6, 2, 3, 3, 1, FAKE, F, 1, FAKE, None) == uq.UQ_EINVAL       # odd d
    assert L.uniquan_rope_split(6, 4, 4, 3, 3, FAKE, F, 1, FAKE, None) == uq.UQ_EINVAL       # group does not divide H
    assert L.uniquan_rope_merge(6, 2, 4, 3, 1, 1, FAKE, 9, 1, FAKE, 0, None) == uq.UQ_EINVAL    # bad dtype
    assert L.uniquan_rope_merge(6, 2, 4, 3, 1, 0, FAKE, F, 1, FAKE, 0, None) == uq.UQ_EINVAL    # nsum
    assert L.uniquan_rope_merge(6, 2, 4, 3, 1, 1, FAKE, F, 1, FAKE, 6, None) == uq.UQ_EINVAL    # ld_out < H d
    assert "ld_out=6" in uq.last_error()
    assert L.uniquan_softmax_causal(10, 4, FAKE, FAKE, None) == uq.UQ_EINVAL
    assert L.uniquan_softmax_causal_bwd(8, 4, FAKE, None, FAKE, None) == uq.UQ_EINVAL
    assert L.uniquan_transpose_bf16_batched(0, 4, 4, FAKE, FAKE, None) == uq.UQ_EINVAL
    ws = uq.uniquan_block_loss_ws()
    assert ws >= 1
    assert L.uniquan_block_loss(16, FAKE, FAKE, FAKE, FAKE, FAKE, ws - 1, FAKE, None) == uq.UQ_EINVAL
    assert L.uniquan_block_loss(0, FAKE, FAKE, FAKE, FAKE, FAKE, ws, FAKE, None) == uq.UQ_EINVAL


def test_bench_refuses_several_gpus():
    """bench.py measures one GPU: --gpus N > 1 exits (status 2) with a
    message, before touching a device."""
    import sys as _sys
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    r = subprocess.run([_sys.executable, os.path.join(root, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120, cwd=root)
    assert r.returncode == 2
    assert "one GPU only" in r.stderr and r.stdout == ""


def test_bench_step_bytes_follow_the_step_kernels():
    """The algorithmic bytes bench.py charges uniquan_fq_step: one pass (read
    dL/dWhat, W, s, code; write s, What, code) for g <= 512 and for bf16
    groups of 513 to 16384 weights, the two passes' sum otherwise."""
    import importlib.util
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    spec = importlib.util.spec_from_file_location("bench_mod", os.path.join(root, "bench.py"))
    b = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(b)
    k = 3
    for g in (128, 4096, 11008, 16384):
        rd, wr = b.fq_step_bytes_per_weight(k, g)
        assert abs(rd - (2 + 2 + 4 + 1 + (4 * k + 12) / g)) < 1e-12
        assert abs(wr - (4 + 2 + 1 + (4 * k + 4) / g)) < 1e-12
    for g, wb in ((16392, 2), (4096, 4)):
        assert b.fq_step_bytes_per_weight(k, g, wb) == b.fq_read_write_bytes(k, g, "local", wb)
