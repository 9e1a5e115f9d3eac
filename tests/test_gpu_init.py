"""GPU parity of the unified initialisation (uniquan_init_unified) against the
CPU oracle's float32 decision mirror (oracle/unified_init.py).

Bar: everything bit-exact -- Delta, z_U, z_B, alpha, the kept candidate's
error and its codes.  Both sides evaluate the same stated fp32 order
(pairwise group sums, exact inverse of C^T C, first-minimum nearest level),
so any difference is a defect.  At the full 4096 x 4096 size the oracle
recomputes sampled groups (groups are independent).
"""
import numpy as np
import pytest
import torch

import oracle.unified_init as UI
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


def weights(R, C, seed, dtype="bf16"):
    spec = synth.scaled(synth.WORKLOADS["attn4096"].matrices[0], R=R, C=C, T=64)
    spec.dtype = dtype
    return synth.make_matrix(spec, seed).W


def run_gpu(W, k, g, G, T, clip, wdt=torch.bfloat16, fill=True):
    R, C = W.shape
    Gn = R * C // g
    out = dict(delta=torch.full((Gn,), -7.0, device=DEV), z_u=torch.full((Gn,), -7.0, device=DEV),
               alpha=torch.full((Gn * k,), -7.0, device=DEV), z_b=torch.full((Gn,), -7.0, device=DEV),
               codes=torch.full((R * C,), 0xEE, dtype=torch.uint8, device=DEV),
               err=torch.full((Gn,), -7.0, device=DEV))
    if fill:
        out["s"] = torch.zeros(R * C, device=DEV)
        out["s_r"] = torch.zeros(R, device=DEV)
    Wd = torch.from_numpy(np.ascontiguousarray(W, F32)).to(DEV).to(wdt).contiguous()
    uq.uniquan_init_unified(R, C, k, g, Wd, G, T, clip, out["delta"], out["z_u"], out["alpha"],
                            out["z_b"], out["codes"], out["err"], out.get("s"), out.get("s_r"))
    torch.cuda.synchronize()
    h = {n: t.cpu().numpy() for n, t in out.items()}
    h["alpha"] = h["alpha"].reshape(Gn, k)
    h["codes"] = h["codes"].reshape(R, C)
    return h


def check(W, k, g, G, T, clip, wdt=torch.bfloat16):
    got = run_gpu(W, k, g, G, T, clip, wdt)
    ref = UI.unified_init(W, k, g, G=G, T=T, clip=clip)
    for name in ("delta", "z_u", "z_b", "alpha", "err"):
        assert np.array_equal(got[name], ref[name]), \
            f"{name}: {np.sum(got[name] != ref[name])} differ, e.g. {got[name][got[name] != ref[name]][:3]} " \
            f"vs {ref[name][got[name] != ref[name]][:3]}"
    assert np.array_equal(got["codes"], ref["codes"]), f"codes: {np.sum(got['codes'] != ref['codes'])} differ"
    assert np.all(got["s"] == 1) and np.all(got["s_r"] == 1)
    return got, ref


@pytest.mark.parametrize("clip", [0, 1, 2])
@pytest.mark.parametrize("G,T", [(1, 0), (1, 15), (6, 4)])
def test_init_bit_exact(clip, G, T):
    W = weights(16, 256, 1)
    check(W, 3, 128, G, T, clip)


@pytest.mark.parametrize("k", [1, 2, 3, 4])
def test_init_bits(k):
    W = weights(8, 512, 2)
    check(W, k, 128, 4, 5, 0)


@pytest.mark.parametrize("g", [8, 16, 32, 64, 256, 512])
@pytest.mark.parametrize("k", [2, 4])
def test_init_group_sizes(g, k):
    W = weights(4, 1024, 3)
    check(W, k, g, 3, 4, 1)


def test_init_ragged_fp32():
    # 37 x 384 = 14208 weights: 27 full wavefronts of 512 and a partial one.
    W = (np.random.default_rng(4).standard_t(5, size=(37, 384)) * 0.02).astype(F32)
    check(W, 4, 128, 5, 6, 2, wdt=torch.float32)
    # 7 x 72 with g = 8: 504 weights, one partial wavefront.
    W = (np.random.default_rng(5).standard_normal((7, 72)) * 0.1).astype(F32)
    check(W, 3, 8, 2, 3, 0, wdt=torch.float32)


def test_init_degenerate_groups():
    rs = np.random.default_rng(6)
    W = (rs.standard_normal((6, 256)) * 0.05).astype(F32)
    W[0, :128] = 0.25          # constant group: Delta' = 1 for every gamma
    W[1, 128:] = 0.0           # all-zero group
    W[2, :128] = np.where(np.arange(128) % 2 == 0, -0.5, 0.5)   # two values
    W[3, :] = np.round(W[3] * 64) / 64                          # coarse grid: exact ties
    for G, T in ((1, 5), (4, 3)):
        check(W, 2, 128, G, T, 0, wdt=torch.float32)
        check(W, 4, 128, G, T, 2, wdt=torch.float32)


def test_init_uniform_levels_recovered():
    vals = (np.arange(8) * 0.5 - 1.75).astype(F32)
    W = np.tile(np.repeat(vals, 16), (4, 1)).astype(F32)
    for r in range(1, 4):
        W[r] = np.random.default_rng(r).permutation(W[r])
    got, _ = check(W, 3, 128, 6, 3, 0, wdt=torch.float32)
    assert np.all(got["err"] == 0)
    assert np.all(got["alpha"] == np.array([2, 1, 0.5], F32))


def test_init_optional_outputs_and_determinism():
    W = weights(8, 256, 7)
    R, C = W.shape
    k, g = 3, 64
    Gn = R * C // g
    ref = run_gpu(W, k, g, 5, 4, 1)
    outs = [torch.empty(n, device=DEV) for n in (Gn, Gn, Gn * k, Gn)]
    Wd = torch.from_numpy(W).to(DEV).to(torch.bfloat16)
    uq.uniquan_init_unified(R, C, k, g, Wd, 5, 4, 1, *outs)
    torch.cuda.synchronize()
    for t, name in zip(outs, ("delta", "z_u", "alpha", "z_b")):
        assert np.array_equal(t.cpu().numpy().reshape(ref[name].shape), ref[name])
    again = run_gpu(W, k, g, 5, 4, 1)
    for name in ref:
        assert np.array_equal(again[name], ref[name])


# ---------------------------------------------------------------------------
# Per-row groups (g = C, above 512): one workgroup per group, the pairwise
# tree over the row zero-padded to a power of two, the int64 adjugate.
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("R,C,k,G,T,clip", [
    (5, 1000, 3, 3, 4, 0),     # not a power of two: 128 lanes of 8, padded to 1024
    (4, 1024, 2, 1, 6, 2),     # 128 lanes of 8, G = 1 (z_B updated)
    (3, 4096, 4, 3, 3, 1),     # 256 lanes of 16
    (2, 11008, 3, 2, 4, 0),    # the 7B down projection's row: lanes of 64, padded to 16384
    (2, 14336, 2, 2, 3, 2),    # the 8B down projection's row
    (2, 6152, 4, 1, 5, 0),     # lanes of 32 with a partly padded lane
])
def test_init_per_row_groups(R, C, k, G, T, clip):
    W = weights(R, C, 40 + k)
    check(W, k, C, G, T, clip)


def test_init_per_row_fp32_degenerate():
    rs = np.random.default_rng(12)
    W = (rs.standard_normal((4, 2048)) * 0.05).astype(F32)
    W[0] = 0.125               # constant row: Delta' = 1
    W[1] = 0.0                 # all-zero row
    W[2] = np.where(np.arange(2048) % 2 == 0, -0.5, 0.5)   # two values
    check(W, 3, 2048, 2, 4, 0, wdt=torch.float32)
    check(W, 4, 2048, 1, 3, 2, wdt=torch.float32)


def test_init_rejects_bad_arguments():
    W = torch.zeros(4 * 128, device=DEV, dtype=torch.bfloat16)
    o = [torch.empty(4 * 8, device=DEV) for _ in range(4)]
    for kw, status in ((dict(k=5), uq.UQ_EUNSUPPORTED), (dict(G=0), uq.UQ_EINVAL),
                       (dict(T=-1), uq.UQ_EINVAL), (dict(clip=3), uq.UQ_EINVAL)):
        a = dict(k=3, G=2, T=1, clip=0)
        a.update(kw)
        with pytest.raises(uq.UniquanError) as e:
            uq.uniquan_init_unified(4, 128, a["k"], 128, W, a["G"], a["T"], a["clip"], *o)
        assert e.value.status == status


# ---------------------------------------------------------------------------
# Full size: a 4096 x 4096 bf16 projection with the paper's grid (G = 30,
# T = 15), checked on sampled groups.
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("clip,G", [(0, 30), (2, 1)])
def test_init_full_size_attn4096(clip, G):
    m = synth.make_matrix(synth.WORKLOADS["attn4096"].matrices[0], 0)
    R, C = m.W.shape
    k, g, T = 4, 128, 15
    got = run_gpu(m.W, k, g, G, T, clip, fill=False)
    Gn = R * C // g
    gidx = np.sort(np.random.default_rng(clip).choice(Gn, 48, replace=False))
    Wg = m.W.reshape(Gn, g)[gidx]
    ref = UI.unified_init(Wg, k, g, G=G, T=T, clip=clip)
    for name in ("delta", "z_u", "z_b", "alpha", "err"):
        assert np.array_equal(got[name][gidx], ref[name]), name
    assert np.array_equal(got["codes"].reshape(Gn, g)[gidx], ref["codes"])
    assert np.all(np.isfinite(got["err"])) and np.all(got["delta"] > 0)
