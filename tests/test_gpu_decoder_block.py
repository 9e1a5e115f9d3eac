"""GPU parity of block-level reconstruction for a whole Transformer block
(paper_2506_03781_amd/block.py DecoderBlock) against
oracle/block_decoder.py.

Seeded inputs: the seven matrices from the generator's 7B block recipe at a
small shape (C = 256 in 2 heads of 128, I = 384, two sequences of 64
tokens; grouped-query cases C = 512 in 4 query heads over 2 or 1 key/value
heads; two sequences of 512 tokens in the long cases), norm weights
1 + 0.1 N(0, 1), quantizer parameters from the oracle's fixed-minimum
clipping with a greedy start.  The oracle evaluates the block in fp64 with
the device's bf16 storage points and never sees device output; the target
Y_ref is the oracle's (checked against the device's own full-precision
forward to 2e-2, then given to the device so that both sides share it).

Bars: codes bit-exact per matrix; the loss within 1e-2; dL/dWhat of all
seven matrices within 1e-2 normwise and, per element, within 8 sigma plus
the largest single rounding flip of the product's own operands plus one
bf16 ulp of the value (the device stores dL/dWhat in bf16), where sigma is
the spread that bf16 rounding decisions taken the other way at the
storage points propagate to that element (tests/block_bounds.py: a variance
model in which a stored value whose inputs differ by s rounds to the other
bf16 neighbour with probability s / ulp).  Calibrated on the oracle against
itself with fp32-sized perturbations before every rounding, the largest
observed difference is 3 sigma; sigma is a small fraction of the value for
most elements and grows only where the result is genuinely sensitive (the
q and k gradients of rows whose attention has near-ties), so a misplaced,
transposed or mis-scaled gradient still fails both bars.  The chained test
gives the second block the first quantized block's output as its input
(Algorithm 1 run from the bottom block up), each side computing that input
itself, checked on the loss and normwise; block 2 is then checked per
element on inputs both sides share.
"""
import numpy as np
import pytest
import torch

import block_bounds as BB
import oracle.block_decoder as D
import oracle.uniquan as O
from paper_2506_03781_amd import synth
from paper_2506_03781_amd import uniquan as uq
from paper_2506_03781_amd.block import DecoderBlock, QuantMatrix

pytestmark = pytest.mark.gpu

F32 = np.float32
N_SEQ, L, C, H, I, K, G = 2, 64, 256, 2, 384, 3, 128
T = N_SEQ * L
SHAPES = {"q": (C, C), "k": (C, C), "v": (C, C), "o": (C, C), "g": (I, C), "u": (I, C), "d": (C, I)}


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    uq.lib()
    torch.cuda.set_device(0)


def host(t):
    return (t.float() if t.dtype == torch.bfloat16 else t).cpu().numpy().astype(np.float64)


def close(x, ref, tol=1e-2, elem=0.1, what=""):
    x, ref = np.asarray(x, np.float64), np.asarray(ref, np.float64)
    nrm = np.linalg.norm(ref)
    assert np.linalg.norm(x - ref) <= tol * max(nrm, 1e-30), f"{what}: normwise {np.linalg.norm(x - ref) / nrm}"
    rms = np.sqrt(np.mean(ref * ref))
    ratio = np.abs(x - ref) / np.maximum(np.abs(ref), rms)
    assert np.all(ratio <= elem), f"{what}: {(ratio > elem).sum()} of {ratio.size} elements, worst {ratio.max():.3g}"


K_SIGMA = 8.0


def share_target(blk, Y_ref):
    """The oracle's target, checked against the device's own and then given
    to the device (fp32, as it stores it); returns it as the oracle uses it."""
    Y32 = np.asarray(Y_ref, F32)
    assert np.allclose(host(blk.Yref), Y32, rtol=2e-2, atol=2e-2 * np.abs(Y32).max())
    blk.Yref.copy_(torch.from_numpy(Y32).to(blk.Yref.device))
    return Y32.astype(np.float64)


def check_step(blk, qs, Xhat, Y32, what, g1, g2, n_seq, H_, n_kv, what_for=""):
    """Loss within 1e-2; each dL/dWhat within 1e-2 normwise and, per element,
    within K_SIGMA sigma plus the largest single rounding flip of its operands
    plus one bf16 ulp of the value (the device stores dL/dWhat in bf16)."""
    st, sig, flip = BB.decoder_step_spread(Xhat, Y32, what, g1, g2, n_seq, H_, n_kv=n_kv)
    loss = float(blk.loss.item())
    assert abs(loss - st["loss"]) <= 1e-2 * st["loss"], (what_for, loss, st["loss"])
    for n in what:
        x, ref = host(qs[n].G), st["grads"][n]
        nrm = np.linalg.norm(ref)
        assert np.linalg.norm(x - ref) <= 1e-2 * nrm, f"{what_for} {n}: normwise {np.linalg.norm(x - ref) / nrm}"
        rms = np.sqrt(np.mean(ref * ref))
        bar = K_SIGMA * sig[n] + flip[n] + 2.0 ** -8 * np.abs(ref) + 1e-6 * rms  # dL/dWhat is stored in bf16
        ratio = np.abs(x - ref) / bar
        rel = bar / np.maximum(np.abs(ref), rms)
        print(f"{what_for} dL/dWhat_{n}: worst |x - ref| / bar {ratio.max():.3g}; bar / max(|ref|, rms) "
              f"median {np.median(rel):.2g} max {rel.max():.2g}")
        assert np.all(ratio <= 1.0), f"{what_for} {n}: {(ratio > 1).sum()} of {ratio.size} elements, worst {ratio.max():.3g}"
    return st


def shapes_for(C_, I_, n_kv_d):
    return {"q": (C_, C_), "k": (n_kv_d, C_), "v": (n_kv_d, C_), "o": (C_, C_), "g": (I_, C_), "u": (I_, C_),
            "d": (C_, I_)}


def make_block(seed, qk_scale=1.0, shapes=SHAPES, T_=T):
    specs = synth.WORKLOADS["block7b"].matrices
    mats, X = {}, None
    C = shapes["q"][1]
    for name, spec in zip(shapes, specs):
        R_, C_ = shapes[name]
        m = synth.make_matrix(synth.scaled(spec, R=R_, C=C_, T=T_), seed)
        if X is None:
            X = m.X.astype(F32)
        W = m.W
        if name in ("q", "k") and qk_scale != 1.0:       # sharper attention: scores of order 1-10
            W = O.bf16_rne((np.asarray(W, F32) * F32(qk_scale)).astype(F32))
        mats[name] = (W, m.s, O.init_param_set_b(W, m.s, K, G))
    rs = np.random.default_rng(seed + 1000)
    g1 = (1.0 + 0.1 * rs.standard_normal(C)).astype(F32)
    g2 = (1.0 + 0.1 * rs.standard_normal(C)).astype(F32)
    return X, mats, g1, g2


def device_block(mats, g1, g2, H_=H, n_kv=None, T_=T, n_seq=N_SEQ):
    qs = {n: QuantMatrix(W, s, K, G, p["delta"], p["z_u"], p["s_r"], p["z_b"], p["alpha"])
          for n, (W, s, p) in mats.items()}
    return DecoderBlock(qs, g1, g2, T_, n_seq, H_, n_kv=n_kv), qs


def oracle_what(mats, mode=O.MAP_FULL):
    out = {}
    for n, (W, s, p) in mats.items():
        out[n] = O.fq_fwd(W, s, p["alpha"], p["z_b"], K, G, p["s_r"], p["delta"], p["z_u"], mode, None)
    return out


def wfp(mats):
    return {n: np.asarray(W, np.float64) for n, (W, _, _) in mats.items()}


def run_and_check(seed, qk_scale=1.0, shapes=SHAPES, H_=H, n_kv=None, T_=T, n_seq=N_SEQ, what_for=""):
    """One FULL-mode step of a device block against the oracle on shared
    inputs and target: codes bit-exact, then check_step."""
    X, mats, g1, g2 = make_block(seed, qk_scale, shapes, T_=T_)
    blk, qs = device_block(mats, g1, g2, H_, n_kv, T_=T_, n_seq=n_seq)
    nk = H_ if n_kv is None else n_kv
    blk.prepare(X)
    Y_ref = D.decoder_forward(X, wfp(mats), g1, g2, n_seq, H_, store=O.bf16_rne, n_kv=nk)["Y"]
    Y32 = share_target(blk, Y_ref)
    blk.set_input(X)
    blk.forward_backward(uq.MAP_FULL)
    torch.cuda.synchronize()
    f = oracle_what(mats)
    for n in mats:
        assert np.array_equal(host(qs[n].codes).reshape(shapes[n]).astype(np.uint8), f[n]["codes"]), f"{n} codes"
    return check_step(blk, qs, X, Y32, {n: f[n]["what_bf16"] for n in mats}, g1, g2, n_seq, H_, nk, what_for)


@pytest.mark.parametrize("qk_scale", [1.0, 6.0])
def test_decoder_block_step(qk_scale):
    st = run_and_check(3, qk_scale, what_for=f"qk {qk_scale}")
    if qk_scale > 1.0:   # the attention is far from uniform
        assert np.mean(np.max(st["P"][..., 8:, :], axis=-1)) > 0.3


def test_decoder_blocks_chained():
    """Block 2 runs on the quantized block 1's output (Xhat) against the
    full-precision block 1's output (X), as in the bottom-up order.  The
    chained run (each side computing block 2's inputs itself) is checked on
    the loss and normwise; block 2's gradients are checked element by element
    on inputs both sides share (the oracle's block-1 outputs, uploaded), so
    that the per-element bar measures block 2 and not the 1e-3 difference
    between the two sides' block-1 outputs it would otherwise amplify."""
    X, m1, g1a, g2a = make_block(5)
    _, m2, g1b, g2b = make_block(6)
    b1, _ = device_block(m1, g1a, g2a)
    b1.prepare(X)
    b1.set_input(X)
    xhat2 = b1.output().clone()
    x2 = b1.Yref.clone()
    b2, q2 = device_block(m2, g1b, g2b)
    b2.prepare(x2)
    b2.set_input(xhat2)
    b2.forward_backward(uq.MAP_FULL)
    torch.cuda.synchronize()

    f1 = oracle_what(m1)
    x2_o = D.decoder_forward(X, wfp(m1), g1a, g2a, N_SEQ, H, store=O.bf16_rne)["Y"].astype(F32)
    xhat2_o = D.decoder_forward(X, {n: f1[n]["what_bf16"] for n in m1}, g1a, g2a, N_SEQ, H,
                                store=O.bf16_rne)["Y"].astype(F32)
    close(host(xhat2), xhat2_o, tol=1e-3, elem=2e-2, what="Xhat of block 2")
    assert not np.allclose(xhat2_o, x2_o)          # the quantized path's input differs from the full-precision one
    f2 = oracle_what(m2)
    what2 = {n: f2[n]["what_bf16"] for n in m2}
    Y2_ref = D.decoder_forward(x2_o, wfp(m2), g1b, g2b, N_SEQ, H, store=O.bf16_rne)["Y"]
    st = D.decoder_step(xhat2_o, Y2_ref, what2, g1b, g2b, N_SEQ, H, store=O.bf16_rne)
    # the chained run
    assert abs(float(b2.loss.item()) - st["loss"]) <= 1e-2 * st["loss"]
    for n in m2:
        close(host(q2[n].G), st["grads"][n], elem=np.inf, what=f"chained block 2 dL/dWhat_{n}")
    # block 2 on the oracle's block-1 outputs and target
    b2.prepare(x2_o)
    Y2_32 = share_target(b2, Y2_ref)
    b2.set_input(xhat2_o)
    b2.forward_backward(uq.MAP_FULL)
    torch.cuda.synchronize()
    check_step(b2, q2, xhat2_o, Y2_32, what2, g1b, g2b, N_SEQ, H, H, "block 2")


def test_decoder_block_step_updates():
    """A FULL step then LOCAL steps with the SGD update: the loss stays finite
    and the straight-through backward of every matrix ran (parameters moved)."""
    X, mats, g1, g2 = make_block(8)
    blk, qs = device_block(mats, g1, g2)
    blk.prepare(X)
    blk.set_input(X)
    s0 = {n: q.s.clone() for n, q in qs.items()}
    losses = []
    for i, mode in enumerate((uq.MAP_FULL, uq.MAP_LOCAL, uq.MAP_LOCAL)):
        blk.step(mode, 1e-4, 1e-5)
        losses.append(float(blk.loss.item()))
    torch.cuda.synchronize()
    assert all(np.isfinite(losses)) and losses[0] > 0
    for n, q in qs.items():
        assert not torch.equal(q.s, s0[n]), n


@pytest.mark.parametrize("n_kv,qk_scale", [(2, 1.0), (2, 6.0), (1, 1.0)])
def test_decoder_block_grouped_query(n_kv, qk_scale):
    """Grouped-query attention: 4 query heads over n_kv key/value heads; the
    gradients of the shared k and v matrices sum over each group."""
    Hq, Cq, Iq = 4, 512, 384
    run_and_check(11 + n_kv, qk_scale, shapes_for(Cq, Iq, n_kv * (Cq // Hq)), Hq, n_kv,
                  what_for=f"n_kv {n_kv} qk {qk_scale}")


@pytest.mark.parametrize("n_kv", [2, 1])
def test_decoder_block_step_long_sequences(n_kv):
    """Two sequences of 512 tokens (several query and key blocks of the fused
    attention per head, its pipelined tiles and the diagonal masking over a
    long causal range), multi-head and grouped-query."""
    Hq, Cq, Iq = 2, 256, 384
    run_and_check(21 + n_kv, 1.0, shapes_for(Cq, Iq, n_kv * (Cq // Hq)), Hq, n_kv, T_=2 * 512, n_seq=2,
                  what_for=f"L 512 n_kv {n_kv}")


@pytest.mark.parametrize("form", ["overlap", "sequential", "replay"])
def test_decoder_block_fused_step_form(form):
    """quantize, then step_fused twice equals step twice followed by quantize:
    every matrix's s, alpha, z_B, codes and What, and the losses, bit for bit;
    with the quantizer passes on a second stream (overlap), on one stream
    (sequential), and replayed from a recording of the first fused step (its
    second stream and waits included)."""
    X, mats, g1, g2 = make_block(31)
    blocks = []
    for _ in range(2):
        blk, qs = device_block(mats, g1, g2)
        blk.prepare(X)
        blk.set_input(X)
        blocks.append((blk, qs))
    (a, qa), (b, qb) = blocks
    lr_f, lr_b = 1e-4, 1e-5
    la, lb = [], []
    a.quantize(uq.MAP_FULL)
    rec = None
    for nxt in (uq.MAP_LOCAL, uq.MAP_LOCAL):
        if form == "replay" and rec is not None:
            rec()
        elif form == "replay":
            rec = uq.record(a.step_fused, nxt, lr_f, lr_b)
        else:
            a.step_fused(nxt, lr_f, lr_b, overlap=form == "overlap")
        la.append(a.loss.clone())
    for mode in (uq.MAP_FULL, uq.MAP_LOCAL):
        b.step(mode, lr_f, lr_b)
        lb.append(b.loss.clone())
    b.quantize(uq.MAP_LOCAL)
    torch.cuda.synchronize()
    for x, y in zip(la, lb):
        assert torch.equal(x, y)
    for n in qa:
        for attr in ("s", "alpha", "z_b", "codes", "W_hat"):
            assert torch.equal(getattr(qa[n], attr), getattr(qb[n], attr)), (n, attr)


def test_decoder_block_stacked_kv_projection():
    """Grouped-query block at a shape where the stacked key/value projection
    ([W_k; W_v] in one product, the key heads rotated) fills the GPU (8192
    tokens, 8 key/value heads of 128): its key/value heads, E and loss equal
    those of the two separate projections (What_k, What_v as unstacked
    copies), bit for bit."""
    T_, n_seq, H_, n_kv, C_, I_ = 8192, 4, 16, 8, 2048, 256
    rs = np.random.default_rng(11)
    qs = {}
    for n, (R_, Cc) in shapes_for(C_, I_, n_kv * 128).items():
        W = O.bf16_rne((0.02 * rs.standard_normal((R_, Cc))).astype(F32))
        q = QuantMatrix(W, np.ones((R_, Cc), F32), K, G)
        q.init_unified(grid_G=4, alt_T=2)
        qs[n] = q
    g = np.ones(C_, F32)
    blk = DecoderBlock(qs, g, g, T_, n_seq, H_, n_kv=n_kv)
    X = torch.randn(T_, C_, device="cuda")
    blk.prepare(X)
    blk.set_input(X)
    blk.quantize(uq.MAP_FULL)
    assert blk._stacked_kv({n: q.W_hat for n, q in qs.items()}) is not None
    blk.forward()
    kv1, e1, l1 = blk.KVh.clone(), blk.E.clone(), blk.loss.clone()
    W2 = {n: q.W_hat for n, q in qs.items()}
    W2["k"], W2["v"] = W2["k"].clone(), W2["v"].clone()
    assert blk._stacked_kv(W2) is None
    blk._forward(W2, blk.Xhat, loss=True)
    torch.cuda.synchronize()
    bits = lambda t: t.contiguous().view(torch.int16)
    assert torch.equal(bits(kv1), bits(blk.KVh)), "key/value heads"
    assert torch.equal(bits(e1), bits(blk.E)), "E"
    assert torch.equal(l1, blk.loss), "loss"
