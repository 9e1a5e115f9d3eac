"""GPU parity of block-level reconstruction for the MLP module
(paper_2506_03781_amd/block.py) against oracle/block_mlp.py.

Inputs are seeded: W_g, W_u [I, C], W_d [C, I] and X [T, C] from the
generator (bf16), quantizer parameters from the oracle's fixed-minimum
clipping with a greedy start.  The oracle evaluates the module with the same
storage points the device uses (G, U, H, E, dH, dG, dU in bf16) and
everything else in fp64; it never sees device output.  Bars: codes
bit-exact per matrix; the loss 1e-2; dL/dWhat of every matrix and the
straight-through gradients 1e-2 normwise and per element (max(|x|, rms)
floor; for grad_s the floor carries G's own bar through dwhat/ds), the
latter from the oracle's gradient rounded to bf16 as stored.
"""
import numpy as np
import pytest
import torch

import oracle.block_mlp as B
import oracle.uniquan as O
from paper_2506_03781_amd import synth
from paper_2506_03781_amd import uniquan as uq
from paper_2506_03781_amd.block import MLPBlock, QuantMatrix

pytestmark = pytest.mark.gpu

F32 = np.float32


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    uq.lib()
    torch.cuda.set_device(0)
    yield
    torch.cuda.synchronize()


def host(t):
    if t.dtype == torch.bfloat16:
        t = t.float()
    return t.cpu().numpy()


def close(x, ref, tol=1e-2, what=""):
    x = np.asarray(x, np.float64)
    ref = np.asarray(ref, np.float64)
    nrm = np.linalg.norm(ref)
    assert np.linalg.norm(x - ref) <= tol * max(nrm, 1e-30), f"{what}: normwise {np.linalg.norm(x - ref) / max(nrm, 1e-30)}"
    rms = np.sqrt(np.mean(ref * ref))
    bad = np.abs(x - ref) > tol * np.maximum(np.abs(ref), rms) + 1e-30
    assert not bad.any(), f"{what}: {bad.sum()} of {bad.size} elements out of tolerance"


def make_block(T, C, I, k, g, seed):
    spec = synth.scaled(synth.WORKLOADS["mlp7b"].matrices[0], R=I, C=C, T=T)
    mg = synth.make_matrix(spec, seed)
    mu = synth.make_matrix(synth.scaled(synth.WORKLOADS["mlp7b"].matrices[1], R=I, C=C, T=T), seed)
    md = synth.make_matrix(synth.scaled(synth.WORKLOADS["mlp7b"].matrices[2], R=C, C=I, T=T), seed)
    mats = {}
    for name, m in (("gate", mg), ("up", mu), ("down", md)):
        p = O.init_param_set_b(m.W, m.s, k, g)
        mats[name] = (m.W, m.s, p)
    return mg.X, mats


def device_block(X, mats, k, g):
    qs = {n: QuantMatrix(W, s, k, g, p["delta"], p["z_u"], p["s_r"], p["z_b"], p["alpha"])
          for n, (W, s, p) in mats.items()}
    blk = MLPBlock(X, qs["gate"], qs["up"], qs["down"])
    blk.prepare()
    return blk, qs


def oracle_fwd(mats, k, g, mode=O.MAP_FULL, prev=None, state=None):
    out = {}
    for n, (W, s, p) in mats.items():
        st = state[n] if state else dict(s=s, alpha=p["alpha"], z_b=p["z_b"])
        out[n] = O.fq_fwd(W, st["s"], st["alpha"], st["z_b"], k, g, p["s_r"], p["delta"], p["z_u"], mode,
                          None if prev is None else prev[n])
    return out


@pytest.mark.parametrize("T,C,I,k", [(256, 256, 512, 3), (128, 384, 640, 4)])
def test_block_step(T, C, I, k):
    g = 128
    X, mats = make_block(T, C, I, k, g, T + C + I)
    blk, qs = device_block(X, mats, k, g)
    blk.forward_backward(uq.MAP_FULL)
    for q in qs.values():
        q.fq_bwd_sgd(0.005, 0.0005, keep_grads=True)
    torch.cuda.synchronize()

    f = oracle_fwd(mats, k, g)
    for n in mats:
        assert np.array_equal(host(qs[n].codes).reshape(mats[n][0].shape), f[n]["codes"]), f"{n} codes"
    Wg, Wu, Wd = (mats[n][0] for n in ("gate", "up", "down"))
    Y_ref = B.mlp_forward(X, Wg, Wu, Wd, store=O.bf16_rne)["Y"]
    st = B.block_step(X, Y_ref, f["gate"]["what_bf16"], f["up"]["what_bf16"], f["down"]["what_bf16"],
                      store=O.bf16_rne)
    loss = float(blk.loss.item())
    assert abs(loss - st["loss"]) <= 1e-2 * st["loss"], (loss, st["loss"])
    for n, key in (("gate", "dWg"), ("up", "dWu"), ("down", "dWd")):
        close(host(qs[n].G), st[key], what=f"dL/dWhat_{n}")
        W, s, p = mats[n]
        Gb = O.bf16_rne(np.asarray(st[key], F32)).astype(np.float64)   # as the device stores it
        bw = O.fq_bwd(W, s, p["alpha"], p["z_b"], f[n]["codes"], Gb, k, g, p["s_r"], p["delta"], p["z_u"])
        # grad_s is G * dwhat/ds element by element; the device's G carries the
        # per-element error bar checked above (1e-2 of max(|G|, rms G)), so the
        # per-element floor for grad_s is rms(G) |dwhat/ds|, the latter from the
        # oracle with a gradient of ones.
        ds = O.fq_bwd(W, s, p["alpha"], p["z_b"], f[n]["codes"], np.ones_like(Gb), k, g, p["s_r"], p["delta"],
                      p["z_u"])["grad_s"]
        gs, ref = host(qs[n].grad_s).astype(np.float64), np.asarray(bw["grad_s"], np.float64)
        assert np.linalg.norm(gs - ref) <= 1e-2 * np.linalg.norm(ref), f"grad_s {n} normwise"
        floor = np.maximum(np.abs(ref), np.sqrt(np.mean(Gb * Gb)) * np.abs(ds))
        assert np.all(np.abs(gs - ref) <= 1e-2 * floor + 1e-30), f"grad_s {n} per element"
        close(host(qs[n].grad_alpha).reshape(-1, k), bw["grad_alpha"], what=f"grad_alpha {n}")
        close(host(qs[n].grad_z_b), bw["grad_z_b"], what=f"grad_z_b {n}")


def test_block_two_steps():
    """A FULL step then a LOCAL step with the SGD updates in between; the
    oracle carries its own state (agreement bars as for chained layer steps)."""
    T, C, I, k, g = 256, 256, 512, 3, 128
    X, mats = make_block(T, C, I, k, g, 7)
    blk, qs = device_block(X, mats, k, g)
    Wg, Wu, Wd = (mats[n][0] for n in ("gate", "up", "down"))
    Y_ref = B.mlp_forward(X, Wg, Wu, Wd, store=O.bf16_rne)["Y"]
    state = {n: dict(s=mats[n][1].copy(), alpha=mats[n][2]["alpha"].copy(), z_b=mats[n][2]["z_b"].copy())
             for n in mats}
    prev = None
    for i, mode in enumerate((uq.MAP_FULL, uq.MAP_LOCAL)):
        blk.step(mode)
        torch.cuda.synchronize()
        f = oracle_fwd(mats, k, g, mode, prev, state)
        st = B.block_step(X, Y_ref, f["gate"]["what_bf16"], f["up"]["what_bf16"], f["down"]["what_bf16"],
                          store=O.bf16_rne)
        assert abs(float(blk.loss.item()) - st["loss"]) <= 1e-2 * st["loss"], i
        for n, key in (("gate", "dWg"), ("up", "dWu"), ("down", "dWd")):
            agree = np.mean(host(qs[n].codes).reshape(mats[n][0].shape) == f[n]["codes"])
            assert agree >= (1.0 if i == 0 else 0.999), (i, n, agree)
            W, s, p = mats[n]
            Gb = O.bf16_rne(np.asarray(st[key], F32)).astype(np.float64)
            bw = O.fq_bwd(W, state[n]["s"], state[n]["alpha"], state[n]["z_b"], f[n]["codes"], Gb, k, g,
                          p["s_r"], p["delta"], p["z_u"])
            for name, lr in (("s", 0.005), ("alpha", 0.0005), ("z_b", 0.0005)):
                grad = bw["grad_" + name]
                state[n][name] = (np.asarray(state[n][name], F32)
                                  - (F32(lr) * np.asarray(grad, np.float64).astype(F32)).astype(F32)).astype(F32)
        prev = {n: f[n]["codes"] for n in mats}


@pytest.mark.parametrize("n", [8, 8 * 257, 8 * 256 * 300 + 24])
def test_silu_mul_kernels(n):
    """H = silu(G) U and its backward against the oracle's fp64 silu and
    silu' on the same bf16 inputs; one rounding to bf16 (2^-8 relative) plus
    fp32 evaluation, with a floor of 2^-20 |dH U| where silu' crosses zero."""
    rs = np.random.default_rng(n)
    G, U, dH = (O.bf16_rne((rs.standard_normal(n) * sc).astype(F32)) for sc in (3.0, 1.0, 0.1))
    dev = [torch.from_numpy(np.asarray(a, F32)).to("cuda").to(torch.bfloat16) for a in (G, U, dH)]
    H, dG, dU = (torch.empty(n, dtype=torch.bfloat16, device="cuda") for _ in range(3))
    uq.uniquan_silu_mul_fwd(dev[0], dev[1], H)
    uq.uniquan_silu_mul_bwd(dev[2], dev[0], dev[1], dG, dU)
    torch.cuda.synchronize()
    g, u, dh = (np.asarray(a, np.float64) for a in (G, U, dH))
    for name, x, ref, floor in (("H", H, B.silu(g) * u, 0.0),
                                ("dG", dG, dh * u * B.dsilu(g), 2.0 ** -20 * np.abs(dh * u)),
                                ("dU", dU, dh * B.silu(g), 0.0)):
        err = np.abs(host(x).astype(np.float64) - ref)
        assert np.all(err <= 2.0 ** -8 * np.abs(ref) + floor + 1e-38), (name, np.max(err / (np.abs(ref) + 1e-30)))


# (4100, 2104, 512), (4100, 2104, 480) and (4100, 4104, 256): the ping-pong
# kernel's 256 x 128 tiles with 64-deep and 32-deep stages and its 256 x 256
# tiles, ragged in both dimensions
@pytest.mark.parametrize("M,N,K", [(1, 8, 8), (200, 264, 136), (512, 384, 1024), (1000, 2056, 72),
                                   (4100, 2104, 512), (4100, 2104, 480), (4100, 4104, 256)])
def test_gemm_nt(M, N, K):
    """out = scale A B^T against fp64 on the same bf16 operands: fp32 output
    within 1e-5 of the row's absolute sum (accumulation order), bf16 output
    within one rounding of that."""
    rs = np.random.default_rng(M * N + K)
    A = O.bf16_rne(rs.standard_normal((M, K)).astype(F32))
    Bm = O.bf16_rne(rs.standard_normal((N, K)).astype(F32))
    a, b = np.asarray(A, np.float64), np.asarray(Bm, np.float64)
    ref = 2.0 * a @ b.T
    mag = 2.0 * np.abs(a) @ np.abs(b).T
    da, db = (torch.from_numpy(np.asarray(x, F32)).to("cuda").to(torch.bfloat16) for x in (A, Bm))
    o32 = torch.empty(M, N, dtype=torch.float32, device="cuda")
    o16 = torch.empty(M, N, dtype=torch.bfloat16, device="cuda")
    uq.uniquan_gemm_nt(M, N, K, da, db, o32, 2.0)
    uq.uniquan_gemm_nt(M, N, K, da, db, o16, 2.0)
    torch.cuda.synchronize()
    assert np.all(np.abs(host(o32) - ref) <= 1e-5 * mag)
    assert np.all(np.abs(host(o16) - ref) <= 2.0 ** -8 * np.abs(ref) + 1e-5 * mag)
