"""CPU oracle for UniQuan_F's unified initialisation (arXiv 2506.03781).

TEST INFRASTRUCTURE, like the rest of ``oracle/``: only ``tests/``,
``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of ``bench.py`` may
import it; the HIP library and its binding never do.

What it computes (Sec. 3, "Unified initialization"; appendix algorithms
"Unified Initialization" and "General alternating update"; appendix "Details
of clipping strategies").  For every group of g weights, independently:

* s = 1, s_r = 1, z_B = (2^k - 1) / 2;
* for gamma = 1/G, 2/G, ..., 1: a candidate scale Delta' = gamma (w_M - w_m) /
  (2^k - 1) and zero point z'_U from the clipping strategy (fixed minimum,
  fixed maximum or balanced); wbar = T_F(w; Delta', z'_U, 1, 1) (Eq. (1));
  alpha', z'_B from the general alternating update on wbar; the candidate's
  quantization error ||w - Q*_{I_F}(w)||^2 (Eq. (3));
* the candidate with the smallest error is kept.

The general alternating update: a greedy start (alpha and C fixed one bit at a
time: c_i = sign(r), alpha_i = mean |r|, r <- r - alpha_i c_i, with
r = wbar - z_B at the start), then T rounds of
  alpha <- (C^T C)^{-1} C^T (wbar - z_B 1),
  C     <- the nearest level's code for every weight,
  z_B   <- mean(wbar - C alpha)      (only when G = 1).

Everything is a chain of integer decisions (codes, the kept candidate), so the
whole initialisation is evaluated as a float32 decision mirror with a fixed,
stated order of operations that the GPU follows too:

* every sum over a group uses pairwise summation with adjacent pairing
  (level by level, element j of the next level is fl(x[2j] + x[2j+1])),
  over the group zero-padded to the next power of two (a whole row of 4096,
  11008 or 14336 weights is one group in the per-row setting);
* C^T C is a matrix of integers, and its inverse is taken exactly: the
  adjugate and determinant are exact integers (cofactor expansion), so
  alpha_a = fl32( fl64(sum_b adj_ab v_b) / fl64(det) ) with v = C^T (wbar - z_B 1)
  from the pairwise sums, each product adj_ab v_b rounded to float64 and the
  products added in ascending b (for g <= 512 the adjugate stays below 2^27
  and every product is exact; above, |adj| <= g^3 < 2^53 is still exact and
  only the products and sums round); a singular C^T C (det = 0) leaves
  alpha unchanged;
* the nearest level is the fp32 argmin of |fl(wbar - q)| over the ascending
  level table, ties to the lower level (the same rule as the forward);
* a constant group (w_M = w_m) takes Delta' = 1;
* the first candidate is always taken, a later one only when its error is
  strictly smaller (the paper starts the running minimum at the largest
  number, which is the same whenever the errors are finite).

Restricted to 1 <= k <= 4 (the paper's bit widths); any g (the library takes
multiples of 8 that divide C: powers of two up to 512 and per-row groups up
to 16384).
"""
from __future__ import annotations

import numpy as np

from .uniquan import (CODE_BITS, F32, F64, MAP_FULL, code_signs, fq_fwd, group_view,
                      levels_f32, map_full, sort_levels, transform_f32)

CLIP_FIXED_MIN = 0
CLIP_FIXED_MAX = 1
CLIP_BALANCED = 2


# ----------------------------------------------------------------------------
# Sums over a group.
# ----------------------------------------------------------------------------
def tree_sum_f32(x: np.ndarray) -> np.ndarray:
    """Pairwise sum over the last axis, fp32:
    ((x0 + x1) + (x2 + x3)) + ((x4 + x5) + (x6 + x7)) + ...,
    the axis zero-padded to the next power of two."""
    x = np.asarray(x, F32)
    n = x.shape[-1]
    assert n >= 1
    p2 = 1 << (n - 1).bit_length()
    if p2 != n:
        pad = np.zeros(x.shape[:-1] + (p2 - n,), F32)
        x = np.concatenate([x, pad], axis=-1)
    while x.shape[-1] > 1:
        x = (x[..., 0::2] + x[..., 1::2]).astype(F32)
    return x[..., 0]


# ----------------------------------------------------------------------------
# Clipping strategies (appendix "Details of clipping strategies").
# ----------------------------------------------------------------------------
def grid_gamma(G: int) -> np.ndarray:
    """gamma = j / G for j = 1..G, each a correctly rounded fp32 division."""
    return (np.arange(1, G + 1, dtype=F32) / F32(G)).astype(F32)


def clip_candidate(wm, wM, gamma, k, clip):
    """Delta' = (gamma (w_M - w_m)) / (2^k - 1) and z'_U, per group (fp32).

    fixed minimum: T_F(w_m) = 0        ->  z'_U = -(w_m / Delta')
    fixed maximum: T_F(w_M) = 2^k - 1  ->  z'_U = (2^k - 1) - (w_M / Delta')
    balanced:      T_F(gamma w_m) = 0  ->  z'_U = -((gamma w_m) / Delta')
    """
    wm = np.asarray(wm, F32)
    wM = np.asarray(wM, F32)
    gamma = F32(gamma)
    L1 = F32((1 << k) - 1)
    rng = (wM - wm).astype(F32)
    delta = ((gamma * rng).astype(F32) / L1).astype(F32)
    delta = np.where(delta > 0, delta, F32(1)).astype(F32)
    if clip == CLIP_FIXED_MIN:
        z_u = (-(wm / delta).astype(F32)).astype(F32)
    elif clip == CLIP_FIXED_MAX:
        z_u = (L1 - (wM / delta).astype(F32)).astype(F32)
    elif clip == CLIP_BALANCED:
        z_u = (-((gamma * wm).astype(F32) / delta).astype(F32)).astype(F32)
    else:
        raise ValueError("clip must be 0 (fixed min), 1 (fixed max) or 2 (balanced)")
    return delta, z_u


# ----------------------------------------------------------------------------
# General alternating update (appendix algorithm of that name).
# ----------------------------------------------------------------------------
def greedy_f32(x: np.ndarray, k: int):
    """Greedy start on x = wbar - z_B [n, g]: for i = 1..k, c_i = sign(r) with
    sign(0) = +1, alpha_i = (pairwise sum of |r|) / g, r <- r - c_i alpha_i.
    Returns alpha [n, k] fp32 and codes [n, g] (bit i set iff c_{i+1} = +1)."""
    r = np.asarray(x, F32).copy()
    n, g = r.shape
    alpha = np.zeros((n, k), F32)
    code = np.zeros((n, g), np.int64)
    for i in range(k):
        plus = r >= 0
        a = (tree_sum_f32(np.abs(r)) / F32(g)).astype(F32)
        alpha[:, i] = a
        code |= plus.astype(np.int64) << i
        r = np.where(plus, r - a[:, None], r + a[:, None]).astype(F32)
    return alpha, code


def det_int(A: np.ndarray) -> np.ndarray:
    """Exact determinant of integer matrices A [n, m, m] (int64), by cofactor
    expansion along the first row."""
    m = A.shape[-1]
    if m == 0:
        return np.ones(A.shape[0], np.int64)
    if m == 1:
        return A[:, 0, 0].astype(np.int64)
    rest = A[:, 1:, :]
    total = np.zeros(A.shape[0], np.int64)
    for j in range(m):
        minor = np.delete(rest, j, axis=2)
        total += (-1) ** j * A[:, 0, j].astype(np.int64) * det_int(minor)
    return total


def adjugate_int(A: np.ndarray) -> np.ndarray:
    """adj(A)[a, b] = (-1)^(a+b) det(A without row b and column a), exact int64."""
    m = A.shape[-1]
    adj = np.zeros(A.shape, np.int64)
    for a in range(m):
        for b in range(m):
            minor = np.delete(np.delete(A, b, axis=1), a, axis=2)
            adj[:, a, b] = (-1) ** (a + b) * det_int(minor)
    return adj


def gram_int(code: np.ndarray, k: int) -> np.ndarray:
    """C^T C per group, [n, k, k] int64 (C is g x k with entries +-1)."""
    sg = code_signs(k)[code]                       # [n, g, k]
    return np.einsum("nga,ngb->nab", sg, sg)


def signed_sums_f32(x: np.ndarray, code: np.ndarray, k: int) -> np.ndarray:
    """v = C^T x per group, each component a pairwise fp32 sum.  [n, k]."""
    v = np.zeros((x.shape[0], k), F32)
    for b in range(k):
        plus = ((code >> b) & 1) == 1
        v[:, b] = tree_sum_f32(np.where(plus, x, -x).astype(F32))
    return v


def ls_alpha(x: np.ndarray, code: np.ndarray, k: int, alpha_prev: np.ndarray) -> np.ndarray:
    """alpha = (C^T C)^{-1} C^T x with the exact inverse adj / det; rows with a
    singular C^T C keep alpha_prev.  [n, k] fp32."""
    M = gram_int(code, k)
    det = det_int(M)
    adj = adjugate_int(M)
    v = signed_sums_f32(x, code, k).astype(F64)
    S = adj[:, :, 0].astype(F64) * v[:, 0:1]
    for b in range(1, k):
        S = S + adj[:, :, b].astype(F64) * v[:, b:b + 1]
    ok = det != 0
    with np.errstate(divide="ignore", invalid="ignore"):
        a_new = (S / np.where(ok, det, 1).astype(F64)[:, None]).astype(F32)
    return np.where(ok[:, None], a_new, np.asarray(alpha_prev, F32)).astype(F32)


def nearest_codes(wbar: np.ndarray, alpha: np.ndarray, z_b: np.ndarray) -> np.ndarray:
    """argmin over codes of (wbar - (C' alpha + z_B))^2 per weight: the code of
    the nearest level in the ascending table, ties to the lower level."""
    qs, code_of, _ = sort_levels(levels_f32(alpha, z_b))
    pos = map_full(np.asarray(wbar, F32), qs)
    return np.take_along_axis(code_of, pos, axis=1)


def z_b_update(wbar: np.ndarray, code: np.ndarray, alpha: np.ndarray) -> np.ndarray:
    """z_B = mean(wbar - C alpha), C alpha summed left to right from 0 (fp32),
    the mean a pairwise sum divided by g."""
    g = wbar.shape[1]
    ca = levels_f32(alpha, np.zeros(wbar.shape[0], F32))     # C' alpha per code
    d = (np.asarray(wbar, F32) - np.take_along_axis(ca, code, axis=1)).astype(F32)
    return (tree_sum_f32(d) / F32(g)).astype(F32)


def general_alternating(wbar: np.ndarray, z_b: np.ndarray, k: int, G: int, T: int):
    """alpha', z'_B (and the last codes) for wbar [n, g] starting from z_B [n]."""
    wbar = np.asarray(wbar, F32)
    z_b = np.asarray(z_b, F32).copy()
    x = (wbar - z_b[:, None]).astype(F32)
    alpha, code = greedy_f32(x, k)
    for _ in range(T):
        alpha = ls_alpha(x, code, k, alpha)
        code = nearest_codes(wbar, alpha, z_b)
        if G == 1:
            z_b = z_b_update(wbar, code, alpha)
            x = (wbar - z_b[:, None]).astype(F32)
    return alpha, z_b, code


# ----------------------------------------------------------------------------
# Unified initialisation (appendix algorithm "Unified Initialization").
# ----------------------------------------------------------------------------
def candidate_error(W, k, g, delta, z_u, alpha, z_b):
    """e' = ||w - Q*_{I_F}(w)||^2 per group with s = 1, s_r = 1: pairwise fp32
    sum of fl(d * d), d = fl(w - what), what the forward's fp32 output."""
    R, C = W.shape
    ones = np.ones((R, C), F32)
    out = fq_fwd(np.asarray(W, F32), ones, alpha, z_b, k, g, delta=delta, z_u=z_u,
                 mode=MAP_FULL)
    w = group_view(np.asarray(W, F32), g)
    d = (w - group_view(out["what32"], g)).astype(F32)
    return tree_sum_f32((d * d).astype(F32)), out["codes"] & CODE_BITS


def improves(err_new, err_best):
    """A later candidate replaces the kept one only with a strictly smaller error."""
    return err_new < err_best


def unified_init(W, k, g, G=30, T=15, clip=CLIP_FIXED_MIN, return_trace=False):
    """Initialised Theta_{I_F} per group: dict of fp32 arrays delta, z_u, z_b
    [Gn], alpha [Gn, k], err [Gn] (kept candidate's error), codes [R, C]
    (FULL mapping of the kept candidate, no mask bit), s [R, C] and s_r [R]
    (ones), gamma_index [Gn] (0-based j of the kept candidate).
    With return_trace, also the per-candidate errors [G, Gn]."""
    assert 1 <= k <= 4 and G >= 1 and T >= 0
    W = np.asarray(W, F32)
    R, C = W.shape
    w = group_view(W, g)
    Gn = w.shape[0]
    wm, wM = w.min(axis=1), w.max(axis=1)
    z_b0 = np.full(Gn, F32(((1 << k) - 1) / 2.0), F32)
    ones = np.ones((R, C), F32)

    best = None
    trace = []
    for j, gamma in enumerate(grid_gamma(G)):
        delta, z_u = clip_candidate(wm, wM, gamma, k, clip)
        wbar = transform_f32(W, ones, g, delta=delta, z_u=z_u)
        alpha, z_b, _ = general_alternating(wbar, z_b0, k, G, T)
        err, codes = candidate_error(W, k, g, delta, z_u, alpha, z_b)
        trace.append(err)
        if best is None:
            best = dict(delta=delta, z_u=z_u, alpha=alpha, z_b=z_b, err=err,
                        codes=group_view(codes, g).copy(),
                        gamma_index=np.zeros(Gn, np.int64))
            continue
        take = improves(err, best["err"])
        best["delta"] = np.where(take, delta, best["delta"]).astype(F32)
        best["z_u"] = np.where(take, z_u, best["z_u"]).astype(F32)
        best["alpha"] = np.where(take[:, None], alpha, best["alpha"]).astype(F32)
        best["z_b"] = np.where(take, z_b, best["z_b"]).astype(F32)
        best["err"] = np.where(take, err, best["err"]).astype(F32)
        best["codes"] = np.where(take[:, None], group_view(codes, g), best["codes"])
        best["gamma_index"] = np.where(take, j, best["gamma_index"])
    best["codes"] = best["codes"].reshape(R, C).astype(np.uint8)
    best["s"] = ones
    best["s_r"] = np.ones(R, F32)
    if return_trace:
        best["trace"] = np.stack(trace)
    return best
