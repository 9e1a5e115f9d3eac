"""Full-size parity: the step the bench times, at the shapes of every
workload, on sampled rows.

Every oracle input is the seeded generator's or computed here from it:
W, X, s come from ``synth``; the quantization parameters from the recipe in
``step_params`` (numpy, from W); the previous codes of the LOCAL mapping from
``synth.random_codes``.  They are uploaded to the device, so nothing the HIP
path produced feeds the oracle.  Per sampled row: codes and the bf16
residual What - W bit-exact; the error rows E and the gradient rows against
fp64; the straight-through gradients of the fused backward+SGD kernel within
1e-2, per element against the oracle fed the bf16 gradient the kernel reads
and normwise against the unrounded fp64 chain.  The loss is checked against
the sum of squares of the device's own Et (a property at any size) and, at
4096 x 4096, against the oracle's fp64 loss over every row.
"""
import numpy as np
import pytest
import torch

import oracle.uniquan as O
from paper_2506_03781_amd import synth
from paper_2506_03781_amd import uniquan as uq

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
    rms = np.sqrt(np.mean(ref * ref)) if ref.size else 0.0
    bad = np.abs(x - ref) > tol * np.maximum(np.abs(ref), rms) + 1e-30
    assert not bad.any(), f"{what}: {bad.sum()} elements out of tolerance, e.g. {x[bad][:3]} vs {ref[bad][:3]}"


def normwise(x, ref, tol=1e-2, what=""):
    x = np.asarray(x, np.float64)
    ref = np.asarray(ref, np.float64)
    err = np.linalg.norm(x - ref) / max(np.linalg.norm(ref), 1e-30)
    assert err <= tol, f"{what}: normwise {err}"


def step_params(W, k, g, seed):
    """Quantization parameters for a full-size step: the fixed-minimum
    clipping range at gamma = 1 (Delta = (w_M - w_m) / (2^k - 1), z_U =
    -w_m / Delta), z_B = (2^k - 1) / 2 and alpha_i = 2^(i-1) / 2 (the uniform
    grid as binary-coding levels), each alpha perturbed by up to 10% so the
    levels are not uniform.  Computed in numpy from W."""
    R, C = W.shape
    w = W.reshape(-1, g)
    Gn = w.shape[0]
    wm, wM = w.min(axis=1).astype(np.float64), w.max(axis=1).astype(np.float64)
    delta = np.maximum((wM - wm) / ((1 << k) - 1), 1e-8).astype(F32)
    z_u = (-wm / delta.astype(np.float64)).astype(F32)
    rs = np.random.default_rng(seed)
    base = 0.5 * 2.0 ** np.arange(k)
    alpha = (base[None, :] * (1 + 0.1 * rs.uniform(-1, 1, (Gn, k)))).astype(F32)
    z_b = np.full(Gn, ((1 << k) - 1) / 2.0, F32)
    return dict(delta=delta, z_u=z_u, alpha=alpha, z_b=z_b, s_r=np.ones(R, F32))


def run_step(spec, k, seed, n_rows=8):
    from paper_2506_03781_amd.layer import QuantLayer
    g = 128
    m = synth.make_matrix(spec, seed)
    R, C, T = m.R, m.C, m.T
    p = step_params(m.W, k, g, seed)
    prev = synth.random_codes(R, C, k, seed + 1)
    lay = QuantLayer(m.W, m.X, m.s, k, g, residual=True, delta=p["delta"], z_u=p["z_u"], s_r=p["s_r"],
                     z_b=p["z_b"])
    lay.alpha.copy_(torch.from_numpy(p["alpha"].reshape(-1)))
    lay.codes.copy_(torch.from_numpy(prev.reshape(-1)))
    lay.prepare()
    lay.fq_fwd(uq.MAP_LOCAL)
    lay.recon(backward=False)
    uq.uniquan_layer_grad(T, R, C, lay.Et, lay.Xt, lay.G)
    lay.fq_bwd_sgd(keep_grads=True)
    torch.cuda.synchronize()

    rows = np.sort(np.random.default_rng(seed + 2).choice(R, n_rows, replace=False))
    gpr = C // g
    gidx = (rows[:, None] * gpr + np.arange(gpr)[None, :]).reshape(-1)
    Wr, sr = m.W[rows], m.s[rows]
    ref = O.fq_fwd(Wr, sr, p["alpha"][gidx], p["z_b"][gidx], k, g, None, p["delta"][gidx], p["z_u"][gidx],
                   uq.MAP_LOCAL, prev[rows])
    assert np.array_equal(host(lay.codes).reshape(R, C)[rows], ref["codes"]), "codes"
    res_b = O.bf16_rne(O.residual_f32(ref["what32"], Wr))
    assert np.array_equal(host(lay.W_hat)[rows], res_b), "residual"
    Xb = m.X.astype(np.float64)
    E_rows = Xb @ res_b.astype(np.float64).T                        # [T, rows]
    Et = host(lay.Et)
    close(Et[rows], E_rows.T, what="E rows")
    G_rows = 2.0 * O.bf16_rne(E_rows.T.astype(F32)).astype(np.float64) @ Xb
    close(host(lay.G)[rows], G_rows, what="grad_W_hat rows")
    # the backward consumes dL/dWhat as stored (bf16): per element against the
    # oracle fed its own gradient rounded the same way, normwise against the
    # unrounded fp64 chain
    got = dict(grad_s=host(lay.grad_s).reshape(R, C)[rows], grad_alpha=host(lay.grad_alpha).reshape(-1, k)[gidx],
               grad_z_b=host(lay.grad_z_b)[gidx])
    for G_in, check in ((O.bf16_rne(G_rows.astype(F32)).astype(np.float64), close), (G_rows, normwise)):
        bw = O.fq_bwd(Wr, sr, p["alpha"][gidx], p["z_b"][gidx], ref["codes"], G_in, k, g, None,
                      p["delta"][gidx], p["z_u"][gidx])
        for n in got:
            check(got[n], bw[n], what=n + " rows")
    # the loss is the sum of squares of the error the kernel stored (bf16)
    loss = float(lay.loss.item())
    L_et = float(np.sum(Et.astype(np.float64) ** 2))
    assert abs(loss - L_et) <= 1e-2 * L_et, (loss, L_et)
    return m, p, prev, lay, loss


def test_full_size_attn4096_step():
    spec = synth.WORKLOADS["attn4096"].matrices[0]
    m, p, prev, lay, loss = run_step(spec, 4, 40)
    # whole-matrix loss against the oracle (every row), fp64
    ref = O.fq_fwd(m.W, m.s, p["alpha"], p["z_b"], 4, 128, None, p["delta"], p["z_u"], uq.MAP_LOCAL, prev)
    Rw = O.bf16_rne(O.residual_f32(ref["what32"], m.W)).astype(np.float64)
    E = m.X.astype(np.float64) @ Rw.T
    L = float(np.sum(E * E))
    assert abs(loss - L) <= 1e-2 * L, (loss, L)


@pytest.mark.parametrize("name", ["gate_proj", "down_proj"])
def test_full_size_mlp7b_step(name):
    spec = [s for s in synth.WORKLOADS["mlp7b"].matrices if s.name == name][0]
    run_step(spec, 3, 41)


def test_full_size_mlp70b_gate_step():
    spec = synth.WORKLOADS["mlp70b"].matrices[0]
    run_step(spec, 2, 42, n_rows=4)
