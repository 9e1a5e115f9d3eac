"""CPU oracle for the UniQuan_F fake-quant step (arXiv 2506.03781).

TEST INFRASTRUCTURE.  This package is the plain, slow reference that the HIP
library is checked against.  Only ``tests/``, ``__graft_entry__.smoke()`` and
the ``cpu_baseline`` leg of ``bench.py`` may import it; the library and its
Python binding never do, and this package imports nothing from them.  The only
code both sides share is the seeded input generator
``paper_2506_03781_amd.synth`` (data only, no arithmetic of the method).

Two halves:

* Decision mirror, float32.  Every integer or bit the method produces (sorted
  level positions, binary codes, the gradient-filter mask) is decided here in
  IEEE binary32 with one correctly rounded numpy operation per arithmetic step,
  in a fixed order, so the GPU can be compared bit for bit.
* Value path, float64.  Given the mirror's codes and mask, the quantized
  weights, reconstruction loss and straight-through gradients are evaluated in
  float64 and the GPU is compared within tolerance.

Notation follows the paper: W (weights), g (group size), k (bits), Delta and
z_U (uniform scale and zero point), s (element-wise scale), s_r (row-wise
scale), alpha (k binary-coding scales per group), z_B (binary-coding shift),
C (binary code matrix), wbar / wtilde / what (transformed / mapped / quantized
weight).

Layout conventions (shared with the C-ABI, restated here so this file stands
alone): W is [R, C] row-major; a group is g contiguous weights of one row, so
group id = r * (C / g) + c // g and Gn = R * C / g; alpha is [Gn, k] with
alpha[:, i] = alpha_{i+1}; a code is an integer b in [0, 2^k) whose bit i is
set iff the binary code entry c_{i+1} = +1; bit 7 of a stored code byte carries
the gradient-filter mask.

Readings taken where the paper is silent (each restated in the design doc):
ties between equidistant levels go to the lower level (the first of the
candidate set, in ascending order); equal level values are ordered by code;
the persisted mapping state is the code, and the mapped value is recomputed
from the current alpha, z_B at every call; tau = min_i |alpha_i|; the filter
acts only on the straight-through path into wbar; loss = squared Frobenius
norm (a sum, not a mean); fp32 -> bf16 rounds to nearest even.
"""
from __future__ import annotations

import numpy as np

F32 = np.float32
F64 = np.float64

MAP_FULL = 0
MAP_LOCAL = 1
MAP_FROZEN = 2

MASK_BIT = np.uint8(0x80)
CODE_BITS = np.uint8(0x7F)


# ----------------------------------------------------------------------------
# Grouping (Sec. 2.1: a matrix is split into groups of g weights that share
# quantization parameters; groups run along the input dimension).
# ----------------------------------------------------------------------------
def group_view(a: np.ndarray, g: int) -> np.ndarray:
    """[R, C] -> [Gn, g] view, group id = r * (C // g) + c // g."""
    R, C = a.shape
    assert C % g == 0
    return a.reshape(R * (C // g), g)


def per_group_rows(R: int, C: int, g: int) -> np.ndarray:
    """Row index of every group: [Gn]."""
    return np.repeat(np.arange(R), C // g)


# ----------------------------------------------------------------------------
# Binary-coding levels (Sec. 2.3): the 2^k levels of a group are
# z_B + sum_i c_i * alpha_i over all sign vectors c in {-1,+1}^k.
# ----------------------------------------------------------------------------
def code_signs(k: int) -> np.ndarray:
    """[2^k, k] matrix of +-1: row b, column i = +1 iff bit i of b is set."""
    b = np.arange(1 << k)[:, None]
    return np.where((b >> np.arange(k)[None, :]) & 1, 1, -1).astype(np.int64)


def levels_f32(alpha: np.ndarray, z_b: np.ndarray) -> np.ndarray:
    """Unsorted fp32 levels q[gid, b] = z_B + (+-alpha_1) + ... + (+-alpha_k).

    Summed left to right starting from z_B, one fp32 rounding per addition.
    """
    alpha = np.asarray(alpha, F32)
    Gn, k = alpha.shape
    sg = code_signs(k)
    q = np.repeat(np.asarray(z_b, F32)[:, None], 1 << k, axis=1)
    for i in range(k):
        term = np.where(sg[None, :, i] > 0, alpha[:, i:i + 1], -alpha[:, i:i + 1]).astype(F32)
        q = (q + term).astype(F32)
    return q


def levels_f64(alpha: np.ndarray, z_b: np.ndarray) -> np.ndarray:
    """Exact-ish fp64 levels z_B + C' alpha for every code (value path)."""
    alpha = np.asarray(alpha, F64)
    k = alpha.shape[1]
    return np.asarray(z_b, F64)[:, None] + alpha @ code_signs(k).T.astype(F64)


def sort_levels(q: np.ndarray):
    """Ascending sort of each group's levels, equal values ordered by code.

    Returns (qs, code_of, pos_of): qs[gid, j] is the j-th smallest level,
    code_of[gid, j] its code, pos_of[gid, b] the sorted position of code b.
    The paper's local mapping speaks of neighbouring levels, which presumes
    this ascending order (Appendix algorithm "Local and periodic mapping").
    """
    order = np.argsort(q, axis=1, kind="stable")
    qs = np.take_along_axis(q, order, axis=1)
    pos_of = np.argsort(order, axis=1, kind="stable")
    return qs, order.astype(np.int64), pos_of.astype(np.int64)


# ----------------------------------------------------------------------------
# Flexible-mapping transform, Eq. (1): wbar = w / (Delta * s * s_r) + z_U.
# ----------------------------------------------------------------------------
def expand_params(R, C, g, s_r=None, delta=None, z_u=None):
    Gn = R * C // g
    s_r = np.ones(R, F32) if s_r is None else np.asarray(s_r, F32)
    delta = np.ones(Gn, F32) if delta is None else np.asarray(delta, F32)
    z_u = np.zeros(Gn, F32) if z_u is None else np.asarray(z_u, F32)
    return s_r, delta, z_u


def transform_f32(W, s, g, s_r=None, delta=None, z_u=None) -> np.ndarray:
    """wbar in fp32 with den = (Delta * s_r) * s, then wbar = (w / den) + z_U.

    Returns [Gn, g].
    """
    R, C = W.shape
    s_r, delta, z_u = expand_params(R, C, g, s_r, delta, z_u)
    rows = per_group_rows(R, C, g)
    w = group_view(np.asarray(W, F32), g)
    sg = group_view(np.asarray(s, F32), g)
    ds = (delta * s_r[rows]).astype(F32)                 # Delta * s_r   [Gn]
    den = (ds[:, None] * sg).astype(F32)                 # (Delta s_r) s [Gn, g]
    return ((w / den).astype(F32) + z_u[:, None]).astype(F32)


def transform_minus_zu_f64(W, s, g, s_r=None, delta=None):
    """wbar - z_U = w / (Delta s_r s) in fp64 (value path), [Gn, g]."""
    R, C = W.shape
    s_r, delta, _ = expand_params(R, C, g, s_r, delta, None)
    rows = per_group_rows(R, C, g)
    w = group_view(np.asarray(W, F64), g)
    sg = group_view(np.asarray(s, F64), g)
    return w / (delta.astype(F64)[:, None] * s_r.astype(F64)[rows][:, None] * sg)


# ----------------------------------------------------------------------------
# Nearest-level mapping (Sec. 2.3 argmin; Eq. (3) with the local and periodic
# mapping of the appendix algorithm).
# ----------------------------------------------------------------------------
def map_full(wbar: np.ndarray, qs: np.ndarray) -> np.ndarray:
    """Sorted position of the nearest level: first j minimising |fl(wbar - qs_j)|.

    np.argmin returns the first minimum, which is the ascending scan with a
    strict '<' and hence the lower level on a tie.
    """
    D = np.abs((wbar[:, :, None] - qs[:, None, :]).astype(F32))
    return np.argmin(D, axis=2)


def map_local(wbar: np.ndarray, qs: np.ndarray, pos_prev: np.ndarray) -> np.ndarray:
    """Among {max(d-1,0), d, min(d+1,L-1)}, in that ascending order, keep the first
    nearest (strict '<').  d is the previous sorted position."""
    L = qs.shape[1]
    cand = [np.maximum(pos_prev - 1, 0), pos_prev, np.minimum(pos_prev + 1, L - 1)]
    best = cand[0]
    best_d = np.abs((wbar - np.take_along_axis(qs, best, axis=1)).astype(F32))
    for c in cand[1:]:
        d = np.abs((wbar - np.take_along_axis(qs, c, axis=1)).astype(F32))
        take = d < best_d
        best = np.where(take, c, best)
        best_d = np.where(take, d, best_d)
    return best


def tau_f32(alpha: np.ndarray) -> np.ndarray:
    """Gradient-filter threshold tau = min_i |alpha_i| per group (fp32)."""
    return np.min(np.abs(np.asarray(alpha, F32)), axis=1).astype(F32)


def bf16_rne(x: np.ndarray) -> np.ndarray:
    """Round fp32 to the nearest bf16 value, ties to even; returned as fp32."""
    u = np.ascontiguousarray(x, F32).view(np.uint32).astype(np.uint64)
    keep = u >> np.uint64(16)
    rem = u & np.uint64(0xFFFF)
    up = (rem > 0x8000) | ((rem == 0x8000) & ((keep & np.uint64(1)) == 1))
    r = (keep + up.astype(np.uint64)) << np.uint64(16)
    return r.astype(np.uint32).view(F32)


def fq_fwd(W, s, alpha, z_b, k, g, s_r=None, delta=None, z_u=None,
           mode=MAP_FULL, codes_prev=None):
    """Q*_{I_F} forward, Eq. (3): D_R( M*_B( T_F(w) ) ).

    Returns a dict with
      codes  [R, C] uint8: code | (mask << 7)
      pos    [R, C] int64: sorted position of the chosen level
      what32 [R, C] fp32: Delta * (wtilde32 - z_U) in fp32 (two roundings)
      what_bf16 [R, C] fp32 holding bf16 values: RNE(what32)
      what64 [R, C] fp64: Delta * (z_B + sum sigma_i alpha_i - z_U)
      mask   [R, C] bool
      wbar   [R, C] fp32
    """
    W = np.asarray(W, F32)
    R, C = W.shape
    alpha = np.asarray(alpha, F32).reshape(-1, k)
    z_b = np.asarray(z_b, F32)
    s_r_, delta_, z_u_ = expand_params(R, C, g, s_r, delta, z_u)
    wbar = transform_f32(W, s, g, s_r_, delta_, z_u_)
    qs, code_of, pos_of = sort_levels(levels_f32(alpha, z_b))
    if mode == MAP_FULL:
        pos = map_full(wbar, qs)
    else:
        prev = group_view(np.asarray(codes_prev, np.uint8) & CODE_BITS, g).astype(np.int64)
        pos0 = np.take_along_axis(pos_of, prev, axis=1)
        pos = map_local(wbar, qs, pos0) if mode == MAP_LOCAL else pos0
    code = np.take_along_axis(code_of, pos, axis=1)
    wt32 = np.take_along_axis(qs, pos, axis=1)
    err = np.abs((wbar - wt32).astype(F32))
    mask = ~(err > tau_f32(alpha)[:, None])
    what32 = (delta_[:, None] * (wt32 - z_u_[:, None]).astype(F32)).astype(F32)
    wt64 = np.take_along_axis(levels_f64(alpha, z_b), code, axis=1)
    what64 = delta_.astype(F64)[:, None] * (wt64 - z_u_.astype(F64)[:, None])
    codes = (code.astype(np.uint8) | np.where(mask, MASK_BIT, np.uint8(0))).astype(np.uint8)
    shape = (R, C)
    return dict(codes=codes.reshape(shape), pos=pos.reshape(shape),
                what32=what32.reshape(shape), what_bf16=bf16_rne(what32).reshape(shape),
                what64=what64.reshape(shape), mask=mask.reshape(shape),
                wbar=wbar.reshape(shape))


# ----------------------------------------------------------------------------
# Straight-through backward with gradient filtering (Appendix "Implementation
# details": STE with the filter |wbar - wtilde| > tau, tau = min(alpha)).
# ----------------------------------------------------------------------------
def fq_bwd(W, s, alpha, z_b, codes, grad_what, k, g, s_r=None, delta=None, z_u=None):
    """Gradients of L through what = Delta * (wtilde - z_U), fp64.

    wtilde = z_B + sum_i sigma_i alpha_i with the code held fixed, and
    d wtilde / d wbar := m (the filtered straight-through estimate), with
    wbar = w / (Delta s_r s) + z_U.  Returns grad_s [R, C], grad_alpha [Gn, k],
    grad_z_b, grad_delta, grad_z_u [Gn], grad_s_r [R].
    """
    W = np.asarray(W, F64)
    R, C = W.shape
    s_r_, delta_, z_u_ = expand_params(R, C, g, s_r, delta, z_u)
    d = delta_.astype(F64)[:, None]
    zu = z_u_.astype(F64)[:, None]
    G = group_view(np.asarray(grad_what, F64), g)
    cb = group_view(np.asarray(codes, np.uint8), g)
    code = (cb & CODE_BITS).astype(np.int64)
    m = ((cb & MASK_BIT) != 0).astype(F64)
    sig = code_signs(k)[code]                                       # [Gn, g, k]
    wt = np.take_along_axis(levels_f64(np.asarray(alpha, F64).reshape(-1, k), z_b), code, axis=1)
    x = transform_minus_zu_f64(W, s, g, s_r_, delta_)              # wbar - z_U
    gt = d * G                                                      # dL/dwtilde
    grad_alpha = np.einsum("ng,ngk->nk", gt, sig.astype(F64))
    grad_z_b = gt.sum(axis=1)
    sg = group_view(np.asarray(s, F64), g)
    grad_s = -(m * gt * x / sg)
    grad_delta = (G * ((wt - zu) - m * x)).sum(axis=1)
    grad_z_u = -(delta_.astype(F64) * ((1.0 - m) * G).sum(axis=1))
    rows = per_group_rows(R, C, g)
    per_group_sr = -(m * gt * x).sum(axis=1)
    grad_s_r = np.zeros(R, F64)
    np.add.at(grad_s_r, rows, per_group_sr)
    grad_s_r /= s_r_.astype(F64)
    return dict(grad_s=grad_s.reshape(R, C), grad_alpha=grad_alpha, grad_z_b=grad_z_b,
                grad_delta=grad_delta, grad_z_u=grad_z_u, grad_s_r=grad_s_r)


# ----------------------------------------------------------------------------
# Layer reconstruction (Algorithm 1 loss ||f(X) - f(X_hat; Phi_hat)||_F^2 for a
# single linear layer with X_hat = X): E = X W_hat^T - Y, L = sum E^2,
# dL/dW_hat = 2 E^T X.
# ----------------------------------------------------------------------------
def layer_target(X, W) -> np.ndarray:
    """Y = X W^T in fp64 on the stored operands, [T, R]."""
    return np.asarray(X, F64) @ np.asarray(W, F64).T


def recon(X, W_hat, Y):
    """Returns (E [T, R], loss, grad_W_hat [R, C]) in fp64."""
    X = np.asarray(X, F64)
    E = X @ np.asarray(W_hat, F64).T - np.asarray(Y, F64)
    loss = float(np.sum(E * E))
    grad = 2.0 * (E.T @ X)
    return E, loss, grad


# ----------------------------------------------------------------------------
# Unification theorem (Theorem 1 and its proof) and the code search, Eq. (4).
# ----------------------------------------------------------------------------
def residual_f32(what32, W):
    """Reconstruction residual What - W in fp32 (one rounding), [R, C]."""
    return (np.asarray(what32, F32) - np.asarray(W, F32)).astype(F32)


def recon_residual(X, Rw):
    """Single-layer reconstruction from the residual Rw = What - W:
    E = X Rw^T (which equals X What^T - X W^T), loss = sum E^2,
    dL/dWhat = 2 E^T X; fp64.  Returns (E [T, R], loss, grad [R, C])."""
    X = np.asarray(X, F64)
    E = X @ np.asarray(Rw, F64).T
    return E, float(np.sum(E * E)), 2.0 * E.T @ X


def fold_params_f32(alpha, z_b, k, delta=None, z_u=None):
    """alpha* = Delta * alpha, z*_B = Delta * (z_B - z_U), each a fp32 product."""
    alpha = np.asarray(alpha, F32).reshape(-1, k)
    Gn = alpha.shape[0]
    delta = np.ones(Gn, F32) if delta is None else np.asarray(delta, F32)
    z_u = np.zeros(Gn, F32) if z_u is None else np.asarray(z_u, F32)
    a_star = (delta[:, None] * alpha).astype(F32)
    z_star = (delta * (np.asarray(z_b, F32) - z_u).astype(F32)).astype(F32)
    return a_star, z_star


def fold(W, s, alpha, z_b, k, g, s_r=None, delta=None, z_u=None, code_src=0):
    """Theorem 1 parameters plus the deployable codes (bit 7 clear).

    code_src = 0: nearest level of the transformed weight wbar (keeps flexible
    mapping; |wbar - q_j| = |w/(s s_r) - q*_j| / Delta for Delta > 0).
    code_src = 1: Eq. (4) literally, nearest folded level q* of the raw w.
    """
    W = np.asarray(W, F32)
    R, C = W.shape
    a_star, z_star = fold_params_f32(alpha, z_b, k, delta, z_u)
    if code_src == 0:
        r = fq_fwd(W, s, alpha, z_b, k, g, s_r, delta, z_u, MAP_FULL)
        codes = (r["codes"] & CODE_BITS).astype(np.uint8)
    else:
        qs, code_of, _ = sort_levels(levels_f32(a_star, z_star))
        pos = map_full(group_view(W, g), qs)
        codes = np.take_along_axis(code_of, pos, axis=1).astype(np.uint8).reshape(R, C)
    return dict(alpha_star=a_star, z_star=z_star, codes=codes)


def bcq_dequant_f64(codes, alpha_star, z_star, k, g):
    """R_B(C; Theta*) = C alpha* + z*_B 1_g in fp64, [R, C]."""
    codes = np.asarray(codes, np.uint8)
    R, C = codes.shape
    code = group_view(codes & CODE_BITS, g).astype(np.int64)
    lv = levels_f64(np.asarray(alpha_star, F64).reshape(-1, k), z_star)
    return np.take_along_axis(lv, code, axis=1).reshape(R, C)


# ----------------------------------------------------------------------------
# Greedy binary-coding start (appendix algorithm "General alternating update",
# its first step: alpha and C are fixed one bit at a time).
# ----------------------------------------------------------------------------
def greedy_bcq(wbar, z_b, k):
    """Per group (rows of wbar [Gn, g]): r = wbar - z_B; for i = 1..k:
    c_i = sign(r) with sign(0) = +1, alpha_i = mean |r|, r <- r - alpha_i c_i.

    mean|r| is the least-squares scale of r on sign(r).  fp64.
    Returns alpha [Gn, k], codes [Gn, g] (int, bit i set iff c_{i+1} = +1).
    """
    r = np.asarray(wbar, F64) - np.asarray(z_b, F64)[:, None]
    Gn, g = r.shape
    alpha = np.zeros((Gn, k), F64)
    code = np.zeros((Gn, g), np.int64)
    for i in range(k):
        c = np.where(r >= 0, 1.0, -1.0)
        a = np.abs(r).mean(axis=1)
        alpha[:, i] = a
        code |= (c > 0).astype(np.int64) << i
        r = r - a[:, None] * c
    return alpha, code


def init_param_set_a(W, s, k, g):
    """Identity uniform part (Delta = 1, z_U = 0, s_r = 1), z_B = 0, alpha from the
    greedy start on wbar = w / s.  Returns dict of fp32 arrays."""
    R, C = W.shape
    Gn = R * C // g
    wbar = transform_f32(W, s, g)
    z_b = np.zeros(Gn, F32)
    alpha, _ = greedy_bcq(wbar, z_b, k)
    return dict(delta=np.ones(Gn, F32), z_u=np.zeros(Gn, F32), s_r=np.ones(R, F32),
                z_b=z_b, alpha=alpha.astype(F32))


def init_param_set_b(W, s, k, g):
    """Fixed-minimum clipping at gamma = 1 (Appendix "Details of clipping
    strategies"): Delta = (w_M - w_m) / (2^k - 1), z_U = -w_m / Delta;
    z_B = (2^k - 1) / 2 (unified initialisation); alpha from the greedy start on
    wbar - z_B.  Delta is floored at 1e-10 for constant groups."""
    R, C = W.shape
    w = group_view(np.asarray(W, F64), g)
    wm, wM = w.min(axis=1), w.max(axis=1)
    delta = np.maximum((wM - wm) / ((1 << k) - 1), 1e-10).astype(F32)
    z_u = (-wm / delta.astype(F64)).astype(F32)
    z_b = np.full(w.shape[0], ((1 << k) - 1) / 2.0, F32)
    s_r = np.ones(R, F32)
    wbar = transform_f32(W, s, g, s_r, delta, z_u)
    alpha, _ = greedy_bcq(wbar, z_b, k)
    return dict(delta=delta, z_u=z_u, s_r=s_r, z_b=z_b, alpha=alpha.astype(F32))


def greedy_alpha_f64(W, s, z_b, k, g, s_r=None, delta=None, z_u=None):
    """alpha of the greedy start on wbar (fp32 transform) - z_B, fp64 [Gn, k]."""
    wbar = transform_f32(np.asarray(W, F32), s, g, s_r, delta, z_u)
    alpha, _ = greedy_bcq(wbar, z_b, k)
    return alpha


def sgd_step(theta, grad, lr):
    """theta - lr * grad (plain SGD, the optimiser the paper names), fp64."""
    return np.asarray(theta, F64) - lr * np.asarray(grad, F64)
