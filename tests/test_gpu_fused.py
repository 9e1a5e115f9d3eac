"""GPU parity of the weight-gradient GEMM with the fused straight-through
backward and SGD update (uniquan_layer_grad_ste_sgd) against the oracle.

Inputs are seeded: the error tile Et (bf16) and X come from the generator,
so the oracle forms dL/dWhat = 2 Et^T X in fp64 from the same numbers; codes
and masks come from the oracle's forward.  Bars: gradients 1e-2 normwise and
per element (as the unfused backward); the SGD steps s' - s, alpha' - alpha,
z_B' - z_B within 1e-2 of -lr times the oracle's gradients.
"""
import numpy as np
import pytest
import torch

import oracle.uniquan as O
from paper_2506_03781_amd import synth
from paper_2506_03781_amd import uniquan as uq

pytestmark = pytest.mark.gpu

F32 = np.float32
DEV = "cuda"


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    uq.lib()
    torch.cuda.set_device(0)
    yield
    torch.cuda.synchronize()


def dev(a, dtype=torch.float32):
    return torch.from_numpy(np.ascontiguousarray(a)).to(DEV).to(dtype).contiguous()


def host(t):
    if t.dtype == torch.bfloat16:
        t = t.float()
    return t.cpu().numpy()


def close(x, ref, tol=1e-2, what=""):
    x = np.asarray(x, np.float64)
    ref = np.asarray(ref, np.float64)
    nrm = np.linalg.norm(ref)
    assert np.linalg.norm(x - ref) <= tol * max(nrm, 1e-30), f"{what}: normwise {np.linalg.norm(x - ref) / max(nrm, 1e-30)}"
    rms = np.sqrt(np.mean(ref * ref)) if ref.size else 0.0
    bad = np.abs(x - ref) > tol * np.maximum(np.abs(ref), rms) + 1e-30
    assert not bad.any(), f"{what}: {bad.sum()} elements out of tolerance, e.g. {x[bad][:3]} vs {ref[bad][:3]}"


def case(R, C, T, k, g, seed, wdt=torch.bfloat16, forward_codes=True):
    spec = synth.scaled(synth.WORKLOADS["attn4096"].matrices[0], R=R, C=C, T=T)
    spec.dtype = "bf16" if wdt == torch.bfloat16 else "f32"
    m = synth.make_matrix(spec, seed)
    p = O.init_param_set_b(m.W, m.s, k, g)
    rs = np.random.default_rng(seed + 100)
    if forward_codes:
        codes = O.fq_fwd(m.W, m.s, p["alpha"], p["z_b"], k, g, p["s_r"], p["delta"], p["z_u"])["codes"]
    else:  # large cases: random codes with random mask bits
        codes = (synth.random_codes(R, C, k, seed) | (rs.integers(0, 2, (R, C)) << 7)).astype(np.uint8)
    # a reconstruction error of the size the forward leaves (bf16, as stored)
    Et = synth.round_to_bf16((rs.standard_normal((R, T)) * 0.05).astype(F32))
    return m, p, codes, Et


def run_fused(m, p, codes, Et, k, g, lr_f, lr_b, wdt=torch.bfloat16):
    R, C = m.W.shape
    T = Et.shape[1]
    Gn = R * C // g
    Xd = dev(m.X, torch.bfloat16)
    Xt = torch.empty(C, T, dtype=torch.bfloat16, device=DEV)
    uq.uniquan_transpose_bf16(T, C, Xd, Xt)
    s = dev(m.s)
    alpha = dev(p["alpha"].reshape(-1))
    z_b = dev(p["z_b"])
    gs, ga, gz = torch.empty(R * C, device=DEV), torch.empty(Gn * k, device=DEV), torch.empty(Gn, device=DEV)
    uq.uniquan_layer_grad_ste_sgd(T, R, C, k, g, dev(Et, torch.bfloat16), Xt, dev(m.W, wdt), s, dev(p["s_r"]),
                                  dev(p["delta"]), dev(p["z_u"]), alpha, z_b, dev(codes, torch.uint8).reshape(-1),
                                  lr_f, lr_b, gs, ga, gz)
    torch.cuda.synchronize()
    return dict(s=host(s).reshape(R, C), alpha=host(alpha).reshape(Gn, k), z_b=host(z_b),
                grad_s=host(gs).reshape(R, C), grad_alpha=host(ga).reshape(Gn, k), grad_z_b=host(gz))


def check(R, C, T, k, g, seed, wdt=torch.bfloat16):
    m, p, codes, Et = case(R, C, T, k, g, seed, wdt)
    lr_f, lr_b = 0.005, 0.0005
    got = run_fused(m, p, codes, Et, k, g, lr_f, lr_b, wdt)
    Xb = synth.round_to_bf16(m.X).astype(np.float64)
    G = 2.0 * Et.astype(np.float64) @ Xb
    bw = O.fq_bwd(m.W, m.s, p["alpha"], p["z_b"], codes, G, k, g, p["s_r"], p["delta"], p["z_u"])
    close(got["grad_s"], bw["grad_s"], what="grad_s")
    close(got["grad_alpha"], bw["grad_alpha"], what="grad_alpha")
    close(got["grad_z_b"], bw["grad_z_b"], what="grad_z_b")
    close(got["s"].astype(np.float64) - m.s.astype(np.float64), -lr_f * bw["grad_s"], what="s step")
    close(got["alpha"].astype(np.float64) - p["alpha"].astype(np.float64), -lr_b * bw["grad_alpha"],
          what="alpha step")
    close(got["z_b"].astype(np.float64) - p["z_b"].astype(np.float64), -lr_b * bw["grad_z_b"], what="z_b step")


@pytest.mark.parametrize("k", [1, 2, 3, 4])
def test_fused_bwd_bits(k):
    check(256, 256, 64, k, 128, 31)


@pytest.mark.parametrize("g", [32, 64, 128])
def test_fused_bwd_group_sizes(g):
    check(128, 512, 96, 3, g, 32)


def test_fused_bwd_ragged_and_fp32_weights():
    # 300 rows and 384 columns: partial tiles in both dimensions
    check(300, 384, 96, 4, 128, 33)
    check(200, 256, 32, 2, 64, 34, wdt=torch.float32)


def test_fused_bwd_rejects_unsupported():
    m, p, codes, Et = case(64, 256, 64, 3, 128, 35)
    for kw, status in ((dict(k=5), uq.UQ_EUNSUPPORTED), (dict(g=256), uq.UQ_EUNSUPPORTED),
                       (dict(T=48), uq.UQ_EUNSUPPORTED)):
        a = dict(k=3, g=128, T=64)
        a.update(kw)
        with pytest.raises(uq.UniquanError) as e:
            run_args = (a["T"], 64, 256, a["k"], a["g"])
            t = torch.zeros(64 * 256, device=DEV, dtype=torch.bfloat16)
            f = torch.zeros(64 * 256 * 8, device=DEV)
            uq.uniquan_layer_grad_ste_sgd(*run_args, t, t, t, f, None, None, None, f, f,
                                          torch.zeros(64 * 256, dtype=torch.uint8, device=DEV), 0.1, 0.1)
        assert e.value.status == status


def sampled_rows_check(R, C, T, k, g, seed, rows):
    m, p, codes, Et = case(R, C, T, k, g, seed, forward_codes=False)
    lr_f, lr_b = 0.005, 0.0005
    got = run_fused(m, p, codes, Et, k, g, lr_f, lr_b)
    gpr = C // g
    gidx = (rows[:, None] * gpr + np.arange(gpr)[None, :]).reshape(-1)
    Xb = synth.round_to_bf16(m.X).astype(np.float64)
    G = 2.0 * Et[rows].astype(np.float64) @ Xb
    bw = O.fq_bwd(m.W[rows], m.s[rows], p["alpha"][gidx], p["z_b"][gidx], codes[rows], G, k, g,
                  p["s_r"][rows], p["delta"][gidx], p["z_u"][gidx])
    close(got["grad_s"][rows], bw["grad_s"], what="grad_s rows")
    close(got["grad_alpha"][gidx], bw["grad_alpha"], what="grad_alpha rows")
    close(got["z_b"][gidx].astype(np.float64) - p["z_b"][gidx], -lr_b * bw["grad_z_b"], what="z_b step rows")
    close(got["s"][rows].astype(np.float64) - m.s[rows], -lr_f * bw["grad_s"], what="s step rows")


def test_fused_bwd_large_ragged():
    """4100 x 3968 weights (17 x 16 tiles of 256 x 256, the last row tile 4
    rows deep and the last column tile half wide): the eight-wavefront
    launch with partial tiles; sampled rows, including the last ones."""
    R, C = 4100, 3968
    rows = np.array([0, 1, 127, 128, 2049, 4095, 4096, 4099])
    sampled_rows_check(R, C, 256, 3, 128, 37, rows)


def test_fused_bwd_full_size_attn4096():
    """4096 x 4096 weights, 2048 tokens, k = 4: the launch the fused step
    uses; sampled rows against the oracle."""
    R = C = 4096
    T, k, g = 2048, 4, 128
    m, p, codes, Et = case(R, C, T, k, g, 36, forward_codes=False)
    lr_f, lr_b = 0.005, 0.0005
    got = run_fused(m, p, codes, Et, k, g, lr_f, lr_b)
    rows = np.sort(np.random.default_rng(7).choice(R, 8, replace=False))
    gpr = C // g
    gidx = (rows[:, None] * gpr + np.arange(gpr)[None, :]).reshape(-1)
    Xb = synth.round_to_bf16(m.X).astype(np.float64)
    G = 2.0 * Et[rows].astype(np.float64) @ Xb
    bw = O.fq_bwd(m.W[rows], m.s[rows], p["alpha"][gidx], p["z_b"][gidx], codes[rows], G, k, g,
                  p["s_r"][rows], p["delta"][gidx], p["z_u"][gidx])
    close(got["grad_s"][rows], bw["grad_s"], what="grad_s rows")
    close(got["grad_alpha"][gidx], bw["grad_alpha"], what="grad_alpha rows")
    close(got["z_b"][gidx].astype(np.float64) - p["z_b"][gidx], -lr_b * bw["grad_z_b"], what="z_b step rows")
