"""GPU parity of the fused causal attention (uniquan_attn_fwd / _bwd) against
the decoder oracle's definitions at the 7B block's sequence length.

Inputs: seeded bf16 Q, K, V, dO (scaled so that the attention is sharp in
some rows), generated here; the oracle evaluates S = Q K^T scale in fp64, P =
bf16(causal softmax(S)), O = bf16(P V), dP = dO V^T, delta = dO . O,
dS = bf16(P (dP - delta)), dQ = dS K scale, dK = dS^T Q scale, dV = P^T dO,
with the key/value gradients summed over the query heads sharing a head.

Bars.  The device takes the same rounding points in fp32; a value it rounds
to bf16 can land on the neighbouring bf16 number (2^-8 relative) where the
fp32 and fp64 results straddle a rounding boundary.  Each output is
therefore compared per element against 2^-6 of its rounding sensitivity (4x
one flip of every rounded term it sums) and 1e-2 normwise:
  O:  sO = |P| |V| + |O|;       dV: |P|^T |dO|;
  dQ: (|P| (|dP| + e)) |K| scale;   dK: (|P| (|dP| + e))^T |Q| scale,
with e_i = |dO_i| . sO_i: the row term delta = dO . O inherits the rounding
of O, which can exceed |delta| by far when the sum cancels (sharp rows).
The row maxima and sums of the forward match the fp64 ones to 1e-5.
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


@pytest.mark.parametrize("L,batch,kv_batch,sharp", [(2048, 4, 4, 1.0), (2048, 4, 2, 3.0), (96, 6, 2, 3.0),
                                                    (64, 4, 1, 1.0)])
def test_attention_fused(L, batch, kv_batch, sharp):
    rs = np.random.default_rng(L + batch + kv_batch)
    grp = batch // kv_batch
    sc = 1.0 / np.sqrt(d)
    Q = bfr(rs.standard_normal((batch, L, d)) * sharp)
    K = bfr(rs.standard_normal((kv_batch, L, d)) * sharp)
    V = bfr(rs.standard_normal((kv_batch, L, d)))
    dO = bfr(rs.standard_normal((batch, L, d)))
    kv = np.arange(batch) % kv_batch          # query batch g kv_batch + c uses key/value batch c
    # device
    dq, dk, dv, ddo = dev(Q), dev(K), dev(V), dev(dO)
    Vt = dev(np.swapaxes(V, 1, 2))
    Kt = dev(np.swapaxes(K, 1, 2))
    Qt = dev(np.swapaxes(Q, 1, 2))
    dOt = dev(np.swapaxes(dO, 1, 2))
    Od = torch.empty(batch, L, d, dtype=torch.bfloat16, device="cuda")
    m = torch.empty(batch, L, device="cuda")
    lsum = torch.empty(batch, L, device="cuda")
    uq.uniquan_attn_fwd(batch, kv_batch, L, d, dq, dk, Vt, sc, Od, m, lsum)
    delta = torch.empty(batch, L, device="cuda")
    gQ = torch.empty(batch, L, d, device="cuda")
    gK = torch.empty(kv_batch, L, d, device="cuda")
    gV = torch.empty(kv_batch, L, d, device="cuda")
    uq.uniquan_attn_bwd(batch, kv_batch, L, d, dq, Qt, dk, Kt, dv, Od, ddo, dOt, m, lsum, sc, delta, gQ, gK, gV)
    torch.cuda.synchronize()
    # oracle, one query batch at a time
    got = dict(O=host(Od), m=host(m), l=host(lsum), dQ=host(gQ), dK=host(gK), dV=host(gV))
    dK_ref = np.zeros((kv_batch, L, d))
    dV_ref = np.zeros((kv_batch, L, d))
    sK = np.zeros((kv_batch, L, d))
    sV = np.zeros((kv_batch, L, d))
    low = np.tril(np.ones((L, L), dtype=bool))
    for b in range(batch):
        Kb, Vb = K[kv[b]], V[kv[b]]
        S = Q[b] @ Kb.T * sc
        Sm = np.where(low, S, -np.inf)
        mx = Sm.max(axis=1)
        ls = np.exp(Sm - mx[:, None]).sum(axis=1)
        assert np.allclose(got["m"][b], mx, rtol=1e-5, atol=1e-5), f"row max {b}"
        assert np.allclose(got["l"][b], ls, rtol=1e-5), f"row sum {b}"
        P = bfr(D.causal_softmax(S))
        Oref = bfr(P @ Vb)
        sO = np.abs(P) @ np.abs(Vb) + np.abs(Oref)
        check(got["O"][b], Oref, sO, f"O[{b}]")
        dP = dO[b] @ Vb.T
        dl = np.sum(dO[b] * Oref, axis=1, keepdims=True)
        dS = bfr(P * (dP - dl))
        sens = np.abs(P) * (np.abs(dP) + np.sum(np.abs(dO[b]) * sO, axis=1, keepdims=True))
        check(got["dQ"][b], dS @ Kb * sc, sens @ np.abs(Kb) * sc, f"dQ[{b}]")
        dK_ref[kv[b]] += dS.T @ Q[b] * sc
        dV_ref[kv[b]] += P.T @ dO[b]
        sK[kv[b]] += sens.T @ np.abs(Q[b]) * sc
        sV[kv[b]] += np.abs(P).T @ np.abs(dO[b])
    for c in range(kv_batch):
        check(got["dK"][c], dK_ref[c], sK[c], f"dK[{c}]")
        check(got["dV"][c], dV_ref[c], sV[c], f"dV[{c}]")
    if grp > 1:
        assert np.abs(dK_ref).max() > 0
