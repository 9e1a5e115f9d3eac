"""Several optimisation steps in a row (Algorithm 1's inner loop for one
linear layer, with the local and periodic mapping schedule: FULL first, then
LOCAL on even steps and FROZEN on odd ones, each followed by the fused SGD
update) on the device and in the oracle, side by side.

The oracle carries its own state from step to step (its codes, s, alpha,
z_B); nothing the device computed is fed back.  The first step's codes are
bit-exact.  Both sides store E and dL/dWhat in bf16 at the same points, but
their fp32 and fp64 sums can round a stored value to neighbouring bf16
numbers (2^-8 relative), and SGD feeds such differences back.  Bars:
at least 99.9% of the codes equal at every step, the loss within 1e-2, and
the accumulated update of s, alpha and z_B (parameter minus its initial
value) within 2e-2 normwise; per element (for weights, and groups, whose
codes agreed at every step) within 1e-6 of the parameter scale plus 2^-6 of
the accumulated rounding sensitivity: with Gm = |G| + 2 |Et|^T |X| the scale
by which a stored dL/dWhat element can move when a bf16 rounding flips,
lr |d grad_s / d G| Gm for s and lr Delta sum_j Gm_j for alpha and z_B.
"""
import numpy as np
import pytest
import torch

import oracle.uniquan as O
from paper_2506_03781_amd import synth
from paper_2506_03781_amd import uniquan as uq
from paper_2506_03781_amd.layer import QuantLayer

pytestmark = pytest.mark.gpu

F32 = np.float32
LR_F, LR_B = 0.005, 0.0005


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    uq.lib()
    torch.cuda.set_device(0)
    yield
    torch.cuda.synchronize()


def sgd32(theta, grad, lr):
    """theta - lr * grad in fp32 with one rounding per operation (the
    gradient rounded to fp32 first, as the device holds it)."""
    g32 = np.asarray(grad, np.float64).astype(F32)
    return (np.asarray(theta, F32) - (F32(lr) * g32).astype(F32)).astype(F32)


def oracle_step(W, X, st, p, k, g, mode):
    f = O.fq_fwd(W, st["s"], st["alpha"], st["z_b"], k, g, p["s_r"], p["delta"], p["z_u"], mode, st["codes"])
    Rw = O.bf16_rne(O.residual_f32(f["what32"], W))
    E = X.astype(np.float64) @ Rw.astype(np.float64).T                  # [T, R]
    loss = float(np.sum(E * E))
    Eb = O.bf16_rne(E.astype(F32)).astype(np.float64)                   # stored Et (bf16)
    G = O.bf16_rne((2.0 * Eb.T @ X.astype(np.float64)).astype(F32))     # stored dL/dWhat (bf16)
    bw = O.fq_bwd(W, st["s"], st["alpha"], st["z_b"], f["codes"], G.astype(np.float64), k, g, p["s_r"],
                  p["delta"], p["z_u"])
    # Scale of each step's rounding sensitivity.  A stored dL/dWhat element can
    # differ by 2^-8 of Gm = |G| + 2 |Et|^T |X| (its own bf16 rounding, and
    # the roundings of the E values it sums); grad_s is linear in G with
    # slope |d grad_s / d G| (the backward of a gradient of ones), alpha and
    # z_B sum Delta G over the group.
    Gm = np.abs(G.astype(np.float64)) + 2.0 * np.abs(Eb).T @ np.abs(X.astype(np.float64))
    ones = O.fq_bwd(W, st["s"], st["alpha"], st["z_b"], f["codes"], np.ones_like(Gm), k, g, p["s_r"],
                    p["delta"], p["z_u"])
    gabs = LR_B * p["delta"].astype(np.float64) * Gm.reshape(-1, g).sum(axis=1)
    mag = dict(s=LR_F * np.abs(ones["grad_s"]) * Gm, alpha=np.repeat(gabs[:, None], k, axis=1), z_b=gabs)
    return dict(codes=f["codes"], s=sgd32(st["s"], bw["grad_s"], LR_F),
                alpha=sgd32(st["alpha"], bw["grad_alpha"], LR_B), z_b=sgd32(st["z_b"], bw["grad_z_b"], LR_B)), \
        loss, mag


@pytest.mark.parametrize("k", [3, 4])
def test_paper_schedule_six_steps(k):
    g = 128
    spec = synth.scaled(synth.WORKLOADS["attn4096"].matrices[0], R=192, C=512, T=256)
    m = synth.make_matrix(spec, 50 + k)
    p = O.init_param_set_b(m.W, m.s, k, g)
    lay = QuantLayer(m.W, m.X, m.s, k, g, residual=True, delta=p["delta"], z_u=p["z_u"], s_r=p["s_r"],
                     z_b=p["z_b"])
    lay.alpha.copy_(torch.from_numpy(p["alpha"].reshape(-1)))
    lay.prepare()
    st = dict(codes=None, s=m.s.copy(), alpha=p["alpha"].copy(), z_b=p["z_b"].copy())
    init = {n: st[n].astype(np.float64) for n in ("s", "alpha", "z_b")}
    acc = {n: np.zeros_like(init[n]) for n in init}
    same_w = np.ones(m.W.shape, bool)
    modes = [uq.MAP_FULL] + [uq.MAP_LOCAL if i % 2 == 0 else uq.MAP_FROZEN for i in range(5)]
    for i, mode in enumerate(modes):
        lay.fq_fwd(mode)
        lay.recon(True)
        lay.fq_bwd_sgd(LR_F, LR_B)
        torch.cuda.synchronize()
        st, loss, mag = oracle_step(m.W, m.X, st, p, k, g, mode)
        codes = lay.codes.cpu().numpy().reshape(m.W.shape)
        agree = np.mean(codes == st["codes"])
        if i == 0:
            assert agree == 1.0, "first step: codes bit-exact"
        assert agree >= 0.999, (i, agree)
        same_w &= codes == st["codes"]
        same_g = same_w.reshape(-1, g).all(axis=1)
        assert abs(float(lay.loss.item()) - loss) <= 1e-2 * loss, (i, float(lay.loss.item()), loss)
        for name, dev in (("s", lay.s), ("alpha", lay.alpha), ("z_b", lay.z_b)):
            acc[name] += mag[name]
            got = dev.cpu().numpy().reshape(st[name].shape).astype(np.float64) - init[name]
            ref = st[name].astype(np.float64) - init[name]
            assert np.linalg.norm(got - ref) <= 2e-2 * np.linalg.norm(ref), \
                (i, name, np.linalg.norm(got - ref) / np.linalg.norm(ref))
            keep = same_w if name == "s" else (same_g[:, None] if name == "alpha" else same_g)
            keep = np.broadcast_to(keep, ref.shape)
            bar = 1e-6 * np.abs(init[name]).max() + 2.0 ** -6 * acc[name]
            bad = (np.abs(got - ref) > bar) & keep
            assert not bad.any(), (i, name, int(bad.sum()), float(np.max((np.abs(got - ref) / bar)[keep])))
