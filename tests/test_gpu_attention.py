"""GPU parity of the fused causal attention (uniquan_attn_fwd / _bwd) against
the decoder oracle's definitions at the 7B block's sequence length.

Inputs: seeded bf16 Q, K, V, dO (scaled so that the attention is sharp in
some rows), generated here; the oracle evaluates S = Q K^T scale in fp64, P =
bf16(causal softmax(S)), O = bf16(P V), dP = dO V^T, delta = dO . O,
dS = bf16(P (dP - delta)), dQ = dS K scale, dK = dS^T Q scale, dV = P^T dO,
the key/value gradients per query head (their sum over the query heads
sharing a key/value head is the gradient of that head), and the base-2
log-sum-exp of each row of S scale.

Bars.  The device takes the same rounding points in fp32; a value it rounds
to bf16 can land on the neighbouring bf16 number (2^-8 relative) where the
fp32 and fp64 results straddle a rounding boundary.  Each output is
therefore compared per element against 2^-6 of its rounding sensitivity (4x
one flip of every rounded term it sums) and 1e-2 normwise:
  O:  sO = |P| |V| + |O|;       dV: |P|^T |dO|;
  dQ: (|P| (|dP| + e)) |K| scale;   dK: (|P| (|dP| + e))^T |Q| scale,
with e_i = |dO_i| . sO_i: the row term delta = dO . O inherits the rounding
of O, which can exceed |delta| by far when the sum cancels (sharp rows).
The forward's row log-sum-exp matches the fp64 one to 1e-5 relative, and
delta = dO . O the fp64 one within 2^-7 e_i (the flips of O it sums).
"""
import numpy as np
import pytest
import torch

import oracle.block_decoder as D
import oracle.uniquan as O
from paper_2506_03781_amd import uniquan as uq

pytestmark = pytest.mark.gpu
F32 = np.float32
d = 128


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    uq.lib()
    torch.cuda.set_device(0)


def bfr(a):
    return O.bf16_rne(np.asarray(a, F32)).astype(np.float64)


def dev(a, dtype=torch.bfloat16):
    return torch.from_numpy(np.ascontiguousarray(np.asarray(a, F32))).to("cuda").to(dtype).contiguous()


def host(t):
    return (t.float() if t.dtype == torch.bfloat16 else t).cpu().numpy().astype(np.float64)


def check(x, ref, sens, what):
    err = np.abs(x - ref)
    nrm = np.linalg.norm(ref)
    assert np.linalg.norm(x - ref) <= 1e-2 * nrm, f"{what}: normwise {np.linalg.norm(x - ref) / nrm}"
    bar = 2.0 ** -6 * sens + 1e-7 * np.abs(ref).max()
    bad = err > bar
    assert not bad.any(), f"{what}: {bad.sum()} of {bad.size} elements, worst ratio {np.max(err / bar):.3g}"


@pytest.mark.parametrize("L,batch,kv_batch,sharp", [(2048, 4, 4, 1.0), (2048, 4, 2, 3.0), (1024, 8, 2, 2.0),
                                                    (256, 16, 16, 1.0), (96, 6, 2, 3.0), (64, 4, 1, 1.0)])
def test_attention_fused(L, batch, kv_batch, sharp):
    rs = np.random.default_rng(L + batch + kv_batch)
    sc = 1.0 / np.sqrt(d)
    Q = bfr(rs.standard_normal((batch, L, d)) * sharp)
    K = bfr(rs.standard_normal((kv_batch, L, d)) * sharp)
    V = bfr(rs.standard_normal((kv_batch, L, d)))
    dO = bfr(rs.standard_normal((batch, L, d)))
    kv = np.arange(batch) % kv_batch          # query batch g kv_batch + c uses key/value batch c
    # device
    dq, dk, dv, ddo = dev(Q), dev(K), dev(V), dev(dO)
    Od = torch.empty(batch, L, d, dtype=torch.bfloat16, device="cuda")
    lse = torch.empty(batch, L, device="cuda")
    uq.uniquan_attn_fwd(batch, kv_batch, L, d, dq, dk, dv, sc, Od, lse)
    delta = torch.empty(batch, L, device="cuda")
    gQ = torch.empty(batch, L, d, device="cuda")
    gK = torch.empty(batch, L, d, device="cuda")
    gV = torch.empty(batch, L, d, device="cuda")
    uq.uniquan_attn_bwd(batch, kv_batch, L, d, dq, dk, dv, Od, ddo, lse, sc, delta, gQ, gK, gV)
    torch.cuda.synchronize()
    # oracle, one query batch at a time
    got = dict(O=host(Od), lse=host(lse), delta=host(delta), dQ=host(gQ), dK=host(gK), dV=host(gV))
    low = np.tril(np.ones((L, L), dtype=bool))
    for b in range(batch):
        Kb, Vb = K[kv[b]], V[kv[b]]
        S = Q[b] @ Kb.T * sc
        Sm = np.where(low, S, -np.inf)
        mx = Sm.max(axis=1)
        ls = np.exp(Sm - mx[:, None]).sum(axis=1)
        lse_ref = (mx + np.log(ls)) / np.log(2.0)
        assert np.allclose(got["lse"][b], lse_ref, rtol=1e-5, atol=1e-5), f"row log-sum-exp {b}"
        P = bfr(D.causal_softmax(S))
        Oref = bfr(P @ Vb)
        sO = np.abs(P) @ np.abs(Vb) + np.abs(Oref)
        check(got["O"][b], Oref, sO, f"O[{b}]")
        dP = dO[b] @ Vb.T
        dl = np.sum(dO[b] * Oref, axis=1, keepdims=True)
        e_row = np.sum(np.abs(dO[b]) * sO, axis=1)
        assert np.all(np.abs(got["delta"][b] - dl[:, 0]) <= 2.0 ** -7 * e_row + 1e-12), f"delta {b}"
        dS = bfr(P * (dP - dl))
        sens = np.abs(P) * (np.abs(dP) + e_row[:, None])
        check(got["dQ"][b], dS @ Kb * sc, sens @ np.abs(Kb) * sc, f"dQ[{b}]")
        check(got["dK"][b], dS.T @ Q[b] * sc, sens.T @ np.abs(Q[b]) * sc, f"dK[{b}]")
        check(got["dV"][b], P.T @ dO[b], np.abs(P).T @ np.abs(dO[b]), f"dV[{b}]")


@pytest.mark.parametrize("n_seq,H,Hkv,L", [(2, 4, 4, 256), (2, 8, 2, 128), (1, 2, 2, 96)])
def test_attention_token_major_io(n_seq, H, Hkv, L):
    """tok_seqs > 0 reads O and dO token-major and writes dQ (and dK, dV with
    one query head per key/value head) token-major bf16 after the inverse
    rotation: bit for bit the head-major kernels followed by the stand-alone
    split of dO and merges of O and the gradients (grouped slot order with
    2 key/value heads for 8 query heads)."""
    grp = H // Hkv
    T = n_seq * L
    B, Bkv = H * n_seq, Hkv * n_seq
    rs = np.random.default_rng(T + H + Hkv)
    sc = 1.0 / np.sqrt(d)
    Q = dev(bfr(rs.standard_normal((B, L, d)) * 2.0))
    K = dev(bfr(rs.standard_normal((Bkv, L, d)) * 2.0))
    V = dev(bfr(rs.standard_normal((Bkv, L, d))))
    dO_tok = dev(bfr(rs.standard_normal((T, H * d))))
    cs = torch.empty(L, d // 2, 2, device="cuda")
    uq.uniquan_rope_table(L, d, cs)
    # head-major reference path
    dOh = torch.empty(B, L, d, dtype=torch.bfloat16, device="cuda")
    uq.uniquan_rope_split(T, H, d, L, dO_tok, dOh, rotate=False, group=grp)
    Oh = torch.empty(B, L, d, dtype=torch.bfloat16, device="cuda")
    lse = torch.empty(B, L, device="cuda")
    uq.uniquan_attn_fwd(B, Bkv, L, d, Q, K, V, sc, Oh, lse)
    O_ref = torch.empty(T, H * d, dtype=torch.bfloat16, device="cuda")
    uq.uniquan_rope_merge(T, H, d, L, Oh, O_ref, rotate=False, group=grp)
    delta = torch.empty(B, L, device="cuda")
    f = lambda: torch.empty(B, L, d, device="cuda")
    dQr, dKp, dVp = f(), f(), f()
    uq.uniquan_attn_bwd(B, Bkv, L, d, Q, K, V, Oh, dOh, lse, sc, delta, dQr, dKp, dVp)
    tokb = lambda n: torch.empty(T, n * d, dtype=torch.bfloat16, device="cuda")
    dQ_ref, dK_ref, dV_ref = tokb(H), tokb(Hkv), tokb(Hkv)
    uq.uniquan_rope_merge(T, H, d, L, dQr, dQ_ref, rotate=True, group=grp)
    uq.uniquan_rope_merge(T, Hkv, d, L, dKp, dK_ref, rotate=True, nsum=grp)
    uq.uniquan_rope_merge(T, Hkv, d, L, dVp, dV_ref, rotate=False, nsum=grp)
    # token-major path
    O_tok = tokb(H)
    lse2, delta2 = torch.empty(B, L, device="cuda"), torch.empty(B, L, device="cuda")
    uq.uniquan_attn_fwd(B, Bkv, L, d, Q, K, V, sc, O_tok, lse2, tok_seqs=n_seq, group=grp)
    dQ_tok = tokb(H)
    if Hkv == H:
        dK_tok, dV_tok = tokb(H), tokb(H)
    else:
        dK_tok, dV_tok = f(), f()
    uq.uniquan_attn_bwd(B, Bkv, L, d, Q, K, V, O_tok, dO_tok, lse2, sc, delta2, dQ_tok, dK_tok, dV_tok,
                        tok_seqs=n_seq, group=grp, cs=cs)
    if Hkv != H:
        dKp2, dVp2 = dK_tok, dV_tok
        dK_tok, dV_tok = tokb(Hkv), tokb(Hkv)
        uq.uniquan_rope_merge(T, Hkv, d, L, dKp2, dK_tok, rotate=True, nsum=grp)
        uq.uniquan_rope_merge(T, Hkv, d, L, dVp2, dV_tok, rotate=False, nsum=grp)
    torch.cuda.synchronize()
    bits = lambda t: t.view(torch.int16)
    assert torch.equal(lse2, lse) and torch.equal(delta2, delta)
    assert torch.equal(bits(O_tok), bits(O_ref)), "O"
    assert torch.equal(bits(dQ_tok), bits(dQ_ref)), "dQ"
    assert torch.equal(bits(dK_tok), bits(dK_ref)), "dK"
    assert torch.equal(bits(dV_tok), bits(dV_ref)), "dV"
