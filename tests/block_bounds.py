"""Per-element spreads of the decoder block step's weight gradients under
bf16 rounding, for the whole-block parity bars.

Two evaluations of the block step that take the same bf16 storage points
(the ``store`` points of oracle/block_decoder.py) differ where a stored value
rounds to the other of the two bf16 numbers around it.  The device and the
oracle differ so: the device accumulates in fp32 where the oracle is exact,
so a value lying within that accumulation error of a rounding boundary can
round the other way, and every later value carries the difference.  This
module propagates the variance of those differences through the block's
forward and backward, with the oracle's own intermediates:

  a stored value v whose inputs differ by sigma rounds the other way with
  probability min(1, sigma / ulp) (ulp <= 2^-7 |v|, the bf16 spacing), so
  it adds min(ulp^2, sigma ulp) to the variance;
  fp32 accumulation adds (2^-24 (|A| |B|))^2 to a product's, and the
  softmax probabilities (2^-18 P)^2 before their rounding: an fp32
  exponential of an argument of up to ~20 less a log-sum-exp whose sum of up
  to 2048 rounded terms is good to ~2^-19;
  products        V(A B) = V_A B^2 + A^2 V_B
  RMSNorm         V_y = g^2 (r^2 V_x + x^2 V_r),  V_r = r^6 sum(x^2 V_x) / C^2
  rotary          V_y1 = c^2 V_x1 + s^2 V_x2  (and symmetrically)
  softmax         V_P_j = P_j^2 ((1 - P_j)^2 V_S_j + sum_{k != j} P_k^2 V_S_k)
  dS = P (dP - delta), with dP_ij - delta_i = dO_i . (V_j - O_i) taken
                  as one difference (it nearly cancels where a row of P
                  is nearly one-hot)
  element-wise    through the squared derivatives,
treating the contributions as independent.  The result, sigma per element of
each weight gradient, is a typical difference, not a worst case; the tests
allow a multiple of it.  Because a rounding decision taken the other way is
a rare event of a whole ulp, an element whose difference comes from one such
event lies many sigma out; flip_allowance adds, per element of a weight
gradient A^T B, the largest single flip of its own two stored operands,
2^-7 max_t |A_ti| |B_tj| for each.  Test infrastructure only.
"""
import numpy as np

import oracle.block_decoder as D
import oracle.uniquan as O
from oracle.block_mlp import dsilu, silu

ULP = 2.0 ** -7     # bf16 spacing relative to |v| (at most)
ACC = 2.0 ** -24    # fp32 accumulation, relative to |A| |B|
EXP = 2.0 ** -18    # softmax probability from fp32 exponentials and log-sum-exp, relative


def _bf16(x):
    return O.bf16_rne(np.asarray(x, np.float32)).astype(np.float64)


def _store_v(V, v):
    """Variance after a bf16 storage point of value v."""
    u = ULP * np.abs(v)
    return V + np.minimum(u * u, np.sqrt(V) * u)


def _mm_v(A, VA, B, VB):
    """Variance of A @ B (fp32 accumulation)."""
    acc = ACC * (np.abs(A) @ np.abs(B))
    return VA @ (B * B) + (A * A) @ VB + acc * acc


def _t(x):
    return np.swapaxes(x, -1, -2)


def _rms_v(x, g, r, V_x):
    C = x.shape[-1]
    V_r = r ** 6 * np.sum(x * x * V_x, axis=-1, keepdims=True) / (C * C)
    return g * g * (r * r * V_x + x * x * V_r), V_r


def _rot_v(V, ang):
    h = V.shape[-1] // 2
    c2, s2 = np.cos(ang) ** 2, np.sin(ang) ** 2
    v1, v2 = V[..., :h], V[..., h:]
    return np.concatenate([c2 * v1 + s2 * v2, c2 * v2 + s2 * v1], axis=-1)


def _d2silu(x):
    sg = 1.0 / (1.0 + np.exp(-x))
    return sg * (1.0 - sg) * (2.0 + x * (1.0 - 2.0 * sg))


def decoder_step_spread(Xhat, Y_ref, W, g1, g2, n_seq, H, n_kv=None):
    """(oracle step with bf16 storage, sigma per element of each weight
    gradient).  Xhat, Y_ref and the weights are shared exactly."""
    st = D.decoder_step(Xhat, Y_ref, W, g1, g2, n_seq, H, store=_bf16, n_kv=n_kv)
    Wf = {n: np.asarray(w, np.float64) for n, w in W.items()}
    g2a = np.asarray(g2, np.float64)
    T, C = st["R"].shape
    d = C // H
    grp = H // st["n_kv"]
    ang = st["ang"]
    sq = np.sqrt(d)
    sh = lambda x, h: D.split_heads(x, n_seq, h)  # noqa: E731
    z = np.zeros
    # forward (X shared: Z1 differs only by its own rounding, from fp32 row sums)
    Z1 = st["Z1"]
    V_Z1 = _store_v((ACC * np.abs(Z1)) ** 2, Z1)
    V_Qh = _store_v(_rot_v(sh(_mm_v(Z1, V_Z1, Wf["q"].T, z(Wf["q"].T.shape)), H), ang), st["Qh"])
    V_Kh = _store_v(_rot_v(sh(_mm_v(Z1, V_Z1, Wf["k"].T, z(Wf["k"].T.shape)), st["n_kv"]), ang), st["Kh"])
    V_Vh = _store_v(sh(_mm_v(Z1, V_Z1, Wf["v"].T, z(Wf["v"].T.shape)), st["n_kv"]), st["Vh"])
    V_Kx, V_Vx = np.repeat(V_Kh, grp, axis=1), np.repeat(V_Vh, grp, axis=1)
    V_S = _mm_v(st["Qh"], V_Qh, _t(st["Kx"]), _t(V_Kx)) / d
    P = st["P"]
    mask = np.tril(np.ones(P.shape[-2:], dtype=bool))
    V_Sm = np.where(mask, V_S, 0.0)
    rowv = np.sum(P * P * V_Sm, axis=-1, keepdims=True)
    V_P = _store_v(P * P * ((1.0 - P) ** 2 * V_Sm + rowv - P * P * V_Sm) + (EXP * P) ** 2, P)
    V_O = _store_v(D.merge_heads(_mm_v(P, V_P, st["Vx"], V_Vx)), st["O"])
    V_R = _mm_v(st["O"], V_O, Wf["o"].T, z(Wf["o"].T.shape))
    V_Z2r, V_r2 = _rms_v(st["R"], g2a, st["r2"], V_R)
    Z2 = st["Z2"]
    V_Z2 = _store_v(V_Z2r, Z2)
    G, Uu, Hm = st["G"], st["U"], st["H"]
    V_G = _store_v(_mm_v(Z2, V_Z2, Wf["g"].T, z(Wf["g"].T.shape)), G)
    V_U = _store_v(_mm_v(Z2, V_Z2, Wf["u"].T, z(Wf["u"].T.shape)), Uu)
    V_H = _store_v((dsilu(G) * Uu) ** 2 * V_G + silu(G) ** 2 * V_U, Hm)
    V_Y = V_R + _mm_v(Hm, V_H, Wf["d"].T, z(Wf["d"].T.shape))
    E = st["E"]
    V_E = _store_v(V_Y, E)
    dY, V_dY = 2.0 * E, 4.0 * V_E
    # MLP backward
    V_gd = _mm_v(_t(dY), _t(V_dY), Hm, V_H)
    dHm = _bf16(dY @ Wf["d"])
    V_dH = _store_v(_mm_v(dY, V_dY, Wf["d"], z(Wf["d"].shape)), dHm)
    ds, s_, d2 = dsilu(G), silu(G), _d2silu(G)
    dG, dU = _bf16(dHm * Uu * ds), _bf16(dHm * s_)
    V_dG = _store_v((Uu * ds) ** 2 * V_dH + (dHm * ds) ** 2 * V_U + (dHm * Uu * d2) ** 2 * V_G, dG)
    V_dU = _store_v(s_ ** 2 * V_dH + (dHm * ds) ** 2 * V_G, dU)
    V_gg = _mm_v(_t(dG), _t(V_dG), Z2, V_Z2)
    V_gu = _mm_v(_t(dU), _t(V_dU), Z2, V_Z2)
    V_dZ2 = _mm_v(dG, V_dG, Wf["g"], z(Wf["g"].shape)) + _mm_v(dU, V_dU, Wf["u"], z(Wf["u"].shape))
    dZ2, R, r2 = st["dZ2"], st["R"], st["r2"]
    gdy = dZ2 * g2a
    ssum = np.sum(gdy * R, axis=-1, keepdims=True)
    V_gdy = V_dZ2 * g2a ** 2
    V_ssum = np.sum(V_gdy * R ** 2 + gdy ** 2 * V_R, axis=-1, keepdims=True)
    V_rb = (r2 ** 2 * V_gdy + gdy ** 2 * V_r2
            + (V_R * (r2 ** 3 * ssum) ** 2 + (R * 3 * r2 ** 2 * ssum) ** 2 * V_r2 + (R * r2 ** 3) ** 2 * V_ssum)
            / (C * C))
    V_dR = V_dY + V_rb
    dA = _bf16(st["dR"])
    V_dA = _store_v(V_dR, dA)
    V_go = _mm_v(_t(dA), _t(V_dA), st["O"], V_O)
    dO = _bf16(dA @ Wf["o"])
    V_dOh = sh(_store_v(_mm_v(dA, V_dA, Wf["o"], z(Wf["o"].shape)), dO), H)
    dOh = sh(dO, H)
    Oh, V_Oh = sh(st["O"], H), sh(V_O, H)
    delta = np.sum(dOh * Oh, axis=-1, keepdims=True)
    dP = dOh @ _t(st["Vx"])
    Vx = st["Vx"]
    # variance of dO_i . (V_j - O_i) over d, expanded into products
    V_diff = (V_dOh @ _t(Vx * Vx) - 2.0 * (V_dOh * Oh) @ _t(Vx) + np.sum(V_dOh * Oh * Oh, axis=-1, keepdims=True)
              + (dOh * dOh) @ _t(V_Vx) + np.sum(dOh * dOh * V_Oh, axis=-1, keepdims=True))
    V_diff = np.maximum(V_diff, 0.0)
    dS = st["dS"]
    V_dS = _store_v(V_P * (dP - delta) ** 2 + P * P * V_diff, dS)
    V_dQh = _mm_v(dS, V_dS, st["Kx"], V_Kx) / d

    def group_sum(x):
        n, Hq, L, dd = x.shape
        return x.reshape(n, Hq // grp, grp, L, dd).sum(axis=2)

    V_dKh = group_sum(_mm_v(_t(dS), _t(V_dS), st["Qh"], V_Qh)) / d
    V_dVh = group_sum(_mm_v(_t(P), _t(V_P), dOh, V_dOh))
    V_dQ = _store_v(D.merge_heads(_rot_v(V_dQh, ang)), st["dQ"])
    V_dK = _store_v(D.merge_heads(_rot_v(V_dKh, ang)), st["dK"])
    V_dV = _store_v(D.merge_heads(V_dVh), st["dV"])
    flips = dict(q=_maxprod(st["dQ"], Z1), k=_maxprod(st["dK"], Z1), v=_maxprod(st["dV"], Z1),
                 o=_maxprod(dA, st["O"]), g=_maxprod(dG, Z2), u=_maxprod(dU, Z2), d=_maxprod(dY, Hm))
    V = dict(q=_mm_v(_t(st["dQ"]), _t(V_dQ), Z1, V_Z1), k=_mm_v(_t(st["dK"]), _t(V_dK), Z1, V_Z1),
             v=_mm_v(_t(st["dV"]), _t(V_dV), Z1, V_Z1), o=V_go, g=V_gg, u=V_gu, d=V_gd)
    return st, {n: np.sqrt(v) for n, v in V.items()}, {n: 2.0 * ULP * f for n, f in flips.items()}


def _maxprod(A, B, chunk=64):
    """max_t |A_ti| |B_tj| for A [T, I], B [T, J]."""
    A, B = np.abs(A), np.abs(B)
    out = np.zeros((A.shape[1], B.shape[1]))
    for t0 in range(0, A.shape[0], chunk):
        a, b = A[t0:t0 + chunk], B[t0:t0 + chunk]
        out = np.maximum(out, np.max(a[:, :, None] * b[:, None, :], axis=0))
    return out
