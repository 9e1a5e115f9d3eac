"""GPU parity of the deployment form (uniquan_bcq_pack) and the inference
product (uniquan_bcq_matmul) against oracle/bcq_deploy.py.

Inputs are seeded: codes from the generator, alpha*, z* drawn here in fp32,
activations rounded to bf16 as the kernel reads them.  Bars: the stored form
bit-exact (plane words and binary16 parameter bits); the product within 1e-4
normwise and 1e-2 per element (max(|y|, rms(y)) floor) of the fp64 oracle on
the same stored values -- fp32 accumulation of bf16 x binary16 products.
Full-size shapes are checked on sampled rows (rows are independent).
"""
import numpy as np
import pytest
import torch

import oracle.bcq_deploy as D
import oracle.uniquan as U
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


def dev(a, dtype):
    return torch.from_numpy(np.ascontiguousarray(a)).to(DEV).to(dtype).contiguous()


def inputs(T, R, C, k, g, seed):
    rs = np.random.default_rng(seed)
    Gn = R * C // g
    codes = synth.random_codes(R, C, k, seed)
    a = rs.uniform(0.001, 0.05, (Gn, k)).astype(F32)
    z = (rs.standard_normal(Gn) * 0.01).astype(F32)
    X = synth.round_to_bf16(rs.standard_normal((T, C)).astype(F32))
    return codes, a, z, X


def gpu_pack(codes, a, z, k, g):
    R, C = codes.shape
    Gn = R * C // g
    planes = torch.empty(R * C * k // 32, dtype=torch.int32, device=DEV)
    a16 = torch.empty(Gn * k, dtype=torch.float16, device=DEV)
    z16 = torch.empty(Gn, dtype=torch.float16, device=DEV)
    uq.uniquan_bcq_pack(R, C, k, g, dev(codes, torch.uint8).reshape(-1), dev(a.reshape(-1), torch.float32),
                        dev(z, torch.float32), planes, a16, z16)
    return planes, a16, z16


def gpu_matmul(T, R, C, k, g, X, st):
    Y = torch.full((T, R), float("nan"), device=DEV)
    ws_n = uq.uniquan_bcq_matmul_ws(T, R, C)
    ws = torch.full((max(ws_n, 1),), float("nan"), device=DEV)
    uq.uniquan_bcq_matmul(T, R, C, k, g, dev(X, torch.bfloat16), *st, Y, ws)
    torch.cuda.synchronize()
    return Y.cpu().numpy()


def close(y, ref, what=""):
    y = np.asarray(y, np.float64)
    ref = np.asarray(ref, np.float64)
    assert np.all(np.isfinite(y)), what
    nrm = np.linalg.norm(ref)
    assert np.linalg.norm(y - ref) <= 1e-4 * nrm, f"{what}: normwise {np.linalg.norm(y - ref) / nrm}"
    rms = np.sqrt(np.mean(ref * ref))
    bad = np.abs(y - ref) > 1e-2 * np.maximum(np.abs(ref), rms)
    assert not bad.any(), f"{what}: {bad.sum()} elements out of tolerance"


@pytest.mark.parametrize("R,C,k,g", [(4, 256, 1, 128), (37, 384, 3, 128), (300, 1024, 4, 256), (5, 640, 2, 640),
                                     (1024, 2048, 4, 128)])
def test_pack_bit_exact(R, C, k, g):
    codes, a, z, _ = inputs(1, R, C, k, g, R + C + k)
    codes = codes | (np.random.default_rng(1).integers(0, 2, (R, C)) << 7).astype(np.uint8)  # mask bits ignored
    planes, a16, z16 = gpu_pack(codes, a, z, k, g)
    torch.cuda.synchronize()
    rp, ra, rz = D.pack(codes, a, z, k, g)
    assert np.array_equal(planes.cpu().numpy().view(np.uint32), rp.reshape(-1))
    assert np.array_equal(a16.cpu().numpy().view(np.uint16), ra.reshape(-1).view(np.uint16))
    assert np.array_equal(z16.cpu().numpy().view(np.uint16), rz.reshape(-1).view(np.uint16))


# shapes: one slab (no partial sums), ragged rows (partial row blocks),
# groups of 256 and of a whole row, 1 to 8 batch rows (tables up to 3, MFMA from 4)
@pytest.mark.parametrize("T,R,C,k,g", [(1, 256, 512, 3, 128), (8, 300, 384, 4, 128), (3, 1000, 1280, 2, 256),
                                       (5, 64, 128, 1, 128), (2, 513, 2560, 4, 2560), (7, 4000, 1152, 3, 128),
                                       (4, 1000, 1280, 3, 256), (6, 513, 2560, 2, 2560)])
def test_matmul(T, R, C, k, g):
    codes, a, z, X = inputs(T, R, C, k, g, T + R + C)
    st = gpu_pack(codes, a, z, k, g)
    Y = gpu_matmul(T, R, C, k, g, X, st)
    ref = D.matmul_f64(X, *D.pack(codes, a, z, k, g), R, C, g)
    close(Y, ref, f"Y {T}x{R}x{C} k={k} g={g}")
    # deterministic: a second call gives the same bits
    assert np.array_equal(gpu_matmul(T, R, C, k, g, X, st).view(np.uint32), Y.view(np.uint32))


def sampled(T, R, C, k, g, seed, n_rows):
    codes, a, z, X = inputs(T, R, C, k, g, seed)
    Y = gpu_matmul(T, R, C, k, g, X, gpu_pack(codes, a, z, k, g))
    rows = np.sort(np.random.default_rng(seed).choice(R, n_rows, replace=False))
    gpr = C // g
    gidx = (rows[:, None] * gpr + np.arange(gpr)[None, :]).reshape(-1)
    ref = D.matmul_f64(X, *D.pack(codes[rows], a[gidx], z[gidx], k, g), n_rows, C, g)
    close(Y[:, rows], ref, f"sampled rows {R}x{C}")


def test_matmul_wide_tables():
    """8 batch rows and 4 quads per slab (the MFMA form)."""
    sampled(8, 8192, 8192, 4, 128, 21, 64)


@pytest.mark.parametrize("T", [3, 6])
def test_matmul_partial_last_slab(T):
    """33 column quads at 2 per slab: the last slab holds one quad (table
    form at 3 batch rows, MFMA form at 6)."""
    sampled(T, 8192, 4224, 3, 128, 25, 48)


def test_matmul_full_size_attn4096():
    sampled(1, 4096, 4096, 4, 128, 22, 64)


def test_matmul_full_size_mlp70b_gate():
    sampled(1, 28672, 8192, 3, 128, 23, 32)


def test_fold_pack_matmul_chain():
    """Device fold -> device pack -> device product against the oracle's own
    fold -> pack -> product on the same seeded training state."""
    m = synth.make_matrix(synth.scaled(synth.WORKLOADS["attn4096"].matrices[0], R=192, C=512, T=4), 24)
    k, g = 3, 128
    R, C = m.W.shape
    Gn = R * C // g
    p = U.init_param_set_b(m.W, m.s, k, g)
    a_st = torch.empty(Gn * k, device=DEV)
    z_st = torch.empty(Gn, device=DEV)
    cd = torch.empty(R * C, dtype=torch.uint8, device=DEV)
    uq.uniquan_fold_to_bcq(R, C, k, g, dev(m.W, torch.bfloat16), dev(m.s, torch.float32),
                           dev(p["s_r"], torch.float32), dev(p["delta"], torch.float32),
                           dev(p["z_u"], torch.float32), dev(p["alpha"].reshape(-1), torch.float32),
                           dev(p["z_b"], torch.float32), a_st, z_st, cd)
    planes = torch.empty(R * C * k // 32, dtype=torch.int32, device=DEV)
    a16 = torch.empty(Gn * k, dtype=torch.float16, device=DEV)
    z16 = torch.empty(Gn, dtype=torch.float16, device=DEV)
    uq.uniquan_bcq_pack(R, C, k, g, cd, a_st, z_st, planes, a16, z16)
    X = m.X[:4]
    Y = gpu_matmul(4, R, C, k, g, X, (planes, a16, z16))
    fo = U.fold(m.W, m.s, p["alpha"], p["z_b"], k, g, p["s_r"], p["delta"], p["z_u"])
    ref_st = D.pack(fo["codes"], fo["alpha_star"], fo["z_star"], k, g)
    assert np.array_equal(planes.cpu().numpy().view(np.uint32), ref_st[0].reshape(-1))
    close(Y, D.matmul_f64(X, *ref_st, R, C, g), "chain")


def test_rejects_bad_shapes():
    t = torch.zeros(1 << 16, dtype=torch.int32, device=DEV)
    h = torch.zeros(1 << 16, dtype=torch.float16, device=DEV)
    with pytest.raises(uq.UniquanError) as e:
        uq.uniquan_bcq_matmul(9, 64, 128, 2, 128, torch.zeros(9 * 128, dtype=torch.bfloat16, device=DEV),
                              t, h, h, torch.zeros(9 * 64, device=DEV))
    assert e.value.status == uq.UQ_EUNSUPPORTED
