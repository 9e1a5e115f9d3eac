"""Pins of the unified-initialisation oracle (CPU only).

The oracle evaluates the initialisation as an fp32 decision mirror in a fixed
order.  These tests tie it to facts fixed elsewhere: hand-computed sums, the
defining equations of the clipping strategies, the closed-form one-bit
optimum, exact integer identities of the adjugate, numpy's least squares,
brute force over all codes, the monotone decrease of alternating
minimisation, exact recovery of a uniform level set, and an independent
float64 implementation written here from the appendix algorithms.  The last
test plants plausible mistakes in the oracle and checks that a pin fails for
each one.
"""
import math

import numpy as np
import pytest

import oracle.unified_init as UI
import oracle.uniquan as U

F32 = np.float32
F64 = np.float64


def _weights(rs, R, C, scale=0.02):
    return (rs.standard_t(5, size=(R, C)) * scale).astype(F32)


# --------------------------------------------------------------------------
# I1: group sums.
# --------------------------------------------------------------------------
def pin_tree_sum():
    # Pairing by hand: (1e8 + 1) + (-1e8 + 1) rounds each pair to +-1e8 in fp32
    # (the spacing there is 8), so the pairwise sum is 0; a running sum would
    # give 1 and pairing (x0 + x2) + (x1 + x3) would give 2.
    x = np.array([[1e8, 1.0, -1e8, 1.0]], F32)
    assert UI.tree_sum_f32(x)[0] == 0.0
    # Small integers add exactly in any order.
    rs = np.random.default_rng(1)
    ints = rs.integers(-1000, 1000, size=(5, 256)).astype(F32)
    assert np.array_equal(UI.tree_sum_f32(ints), ints.astype(F64).sum(axis=1).astype(F32))
    # Pairwise summation error bound: |S - exact| <= log2(n) u sum|x| (u = 2^-24).
    v = rs.standard_normal((8, 512)).astype(F32)
    got = UI.tree_sum_f32(v).astype(F64)
    for i in range(8):
        exact = math.fsum(float(t) for t in v[i])
        bound = 9 * 2.0 ** -24 * float(np.abs(v[i].astype(F64)).sum())
        assert abs(got[i] - exact) <= bound
    assert UI.tree_sum_f32(np.array([[3.5]], F32))[0] == F32(3.5)
    # Lengths that are not powers of two (per-row groups): the same pairing
    # over the zero-padded vector; exact on small integers, and within the
    # pairwise bound of the next power of two at a 7B down-projection row.
    assert UI.tree_sum_f32(np.array([[1e8, 1.0, -1e8, 1.0, 5.0]], F32))[0] == 5.0
    ints = rs.integers(-1000, 1000, size=(3, 1000)).astype(F32)
    assert np.array_equal(UI.tree_sum_f32(ints), ints.astype(F64).sum(axis=1).astype(F32))
    v = rs.standard_normal((2, 11008)).astype(F32)
    got = UI.tree_sum_f32(v).astype(F64)
    for i in range(2):
        exact = math.fsum(float(t) for t in v[i])
        assert abs(got[i] - exact) <= 14 * 2.0 ** -24 * float(np.abs(v[i].astype(F64)).sum())


def test_i1_tree_sum():
    pin_tree_sum()


# --------------------------------------------------------------------------
# I2: clipping strategies (appendix "Details of clipping strategies").
# --------------------------------------------------------------------------
def pin_clipping():
    rs = np.random.default_rng(2)
    wm = (-0.05 - 0.05 * rs.random(64)).astype(F32)
    wM = (0.03 + 0.05 * rs.random(64)).astype(F32)
    for k in (1, 2, 3, 4):
        L1 = (1 << k) - 1
        for gamma in UI.grid_gamma(7):
            d_min, z_min = UI.clip_candidate(wm, wM, gamma, k, UI.CLIP_FIXED_MIN)
            d_max, z_max = UI.clip_candidate(wm, wM, gamma, k, UI.CLIP_FIXED_MAX)
            d_bal, z_bal = UI.clip_candidate(wm, wM, gamma, k, UI.CLIP_BALANCED)
            # Delta' = gamma (w_M - w_m) / (2^k - 1) for every strategy.
            want = float(gamma) * (wM.astype(F64) - wm.astype(F64)) / L1
            for d in (d_min, d_max, d_bal):
                assert np.allclose(d, want, rtol=4e-7, atol=0)
            tf = lambda w, d, z: ((w / d).astype(F32) + z).astype(F32)
            # Fixed minimum: T_F(w_m) = 0 (exactly, z'_U = -fl(w_m / Delta')).
            assert np.all(tf(wm, d_min, z_min) == 0)
            # Fixed maximum: T_F(w_M) = 2^k - 1 (within the rounding of one add).
            assert np.allclose(tf(wM, d_max, z_max), L1, rtol=0, atol=4 * L1 * 2.0 ** -23)
            # Balanced: T_F(gamma w_m) = 0 and T_F(gamma w_M) = 2^k - 1.
            assert np.all(tf((F32(gamma) * wm).astype(F32), d_bal, z_bal) == 0)
            assert np.allclose(tf((F32(gamma) * wM).astype(F32), d_bal, z_bal), L1,
                               rtol=0, atol=1e-4 * L1)
        # At gamma = 1 the three strategies describe the same clipping range.
        d0, z0 = UI.clip_candidate(wm, wM, F32(1), k, UI.CLIP_FIXED_MIN)
        d1, z1 = UI.clip_candidate(wm, wM, F32(1), k, UI.CLIP_FIXED_MAX)
        d2, z2 = UI.clip_candidate(wm, wM, F32(1), k, UI.CLIP_BALANCED)
        assert np.array_equal(d0, d1) and np.array_equal(d0, d2)
        assert np.array_equal(z0, z2)
        assert np.allclose(z0, z1, rtol=0, atol=8 * L1 * 2.0 ** -23)
    # A constant group takes Delta' = 1.
    d, z = UI.clip_candidate(np.array([0.25], F32), np.array([0.25], F32), F32(1), 3,
                             UI.CLIP_FIXED_MIN)
    assert d[0] == 1.0 and z[0] == -0.25
    assert np.array_equal(UI.grid_gamma(4), np.array([0.25, 0.5, 0.75, 1.0], F32))


def test_i2_clipping():
    pin_clipping()


# --------------------------------------------------------------------------
# I3: greedy start (Xu et al.'s Eq. (4), used as the first step).
# --------------------------------------------------------------------------
def pin_greedy():
    rs = np.random.default_rng(3)
    x = rs.standard_normal((32, 128)).astype(F32)
    # One bit: the least-squares optimum of x ~ alpha c is c = sign(x),
    # alpha = mean |x|.
    a1, c1 = UI.greedy_f32(x, 1)
    assert np.array_equal(c1, (x >= 0).astype(np.int64))
    assert np.allclose(a1[:, 0], np.abs(x.astype(F64)).mean(axis=1), rtol=1e-6, atol=0)
    # k bits: agrees with the float64 greedy routine on continuous data.
    a3, c3 = UI.greedy_f32(x, 3)
    a64, c64 = U.greedy_bcq(x, np.zeros(32, F32), 3)
    assert np.array_equal(c3, c64)
    assert np.allclose(a3, a64, rtol=1e-5, atol=0)
    # Greedy scales shrink: alpha_1 >= alpha_2 >= alpha_3 (each is the mean of
    # a residual bounded by the previous scale).
    assert np.all(np.diff(a64, axis=1) <= 1e-12)


def test_i3_greedy():
    pin_greedy()


# --------------------------------------------------------------------------
# I4: exact inverse of C^T C.
# --------------------------------------------------------------------------
def pin_adjugate():
    rs = np.random.default_rng(4)
    for k in (1, 2, 3, 4):
        A = rs.integers(-40, 41, size=(50, k, k)).astype(np.int64)
        codes = rs.integers(0, 1 << k, size=(50, 64))
        A = np.concatenate([A, UI.gram_int(codes, k)])
        if k >= 2:
            sing = A[:5].copy()
            sing[:, :, 1] = 2 * sing[:, :, 0]          # dependent columns
            A = np.concatenate([A, sing])
        adj = UI.adjugate_int(A)
        det = UI.det_int(A)
        eye = np.eye(k, dtype=np.int64)
        assert np.array_equal(np.einsum("nab,nbc->nac", adj, A), det[:, None, None] * eye)
        assert np.array_equal(np.einsum("nab,nbc->nac", A, adj), det[:, None, None] * eye)
        assert np.array_equal(det, np.rint(np.linalg.det(A.astype(F64))).astype(np.int64))
        if k >= 2:
            assert np.all(det[-5:] == 0)
    # C^T C of +-1 columns: diagonal g, off-diagonal = agreements - disagreements.
    codes = np.array([[0b01, 0b10, 0b11, 0b11]])
    M = UI.gram_int(codes, 2)
    assert M[0].tolist() == [[4, 0], [0, 4]]


def test_i4_adjugate():
    pin_adjugate()


# --------------------------------------------------------------------------
# I5: the alpha step is the least-squares solution.
# --------------------------------------------------------------------------
def pin_ls_alpha():
    rs = np.random.default_rng(5)
    n, g = 40, 128
    for k in (1, 2, 3, 4):
        code = rs.integers(0, 1 << k, size=(n, g))
        x = (rs.standard_normal((n, g)) * 2).astype(F32)
        prev = np.full((n, k), 7.0, F32)
        got = UI.ls_alpha(x, code, k, prev).astype(F64)
        sg = U.code_signs(k)[code].astype(F64)
        for i in range(n):
            want = np.linalg.lstsq(sg[i], x[i].astype(F64), rcond=None)[0]
            assert np.allclose(got[i], want, rtol=0, atol=1e-5 * max(1.0, np.abs(want).max()))
        # Data that lie exactly on the span with dyadic scales are recovered exactly.
        a_true = np.array([0.75, -0.5, 0.25, 0.125][:k], F32)
        x_exact = (sg @ a_true.astype(F64)).astype(F32)
        assert np.array_equal(UI.ls_alpha(x_exact, code, k, prev), np.tile(a_true, (n, 1)))
    # Singular C^T C (two equal code columns) keeps the previous alpha.
    code = rs.integers(0, 2, size=(3, 16)) * 0b11
    prev = np.array([[1.0, 2.0]] * 3, F32)
    assert np.array_equal(UI.ls_alpha(rs.standard_normal((3, 16)).astype(F32), code, 2, prev), prev)


def test_i5_ls_alpha():
    pin_ls_alpha()


# --------------------------------------------------------------------------
# I6: code step = brute force over every code; z_B step = closed-form mean.
# --------------------------------------------------------------------------
def pin_code_and_zb_steps():
    rs = np.random.default_rng(6)
    n, g, k = 30, 64, 3
    alpha = rs.uniform(0.1, 1.0, (n, k)).astype(F32)
    z_b = rs.standard_normal(n).astype(F32)
    wbar = (rs.standard_normal((n, g)) * 2 + z_b[:, None]).astype(F32)
    code = UI.nearest_codes(wbar, alpha, z_b)
    q32 = U.levels_f32(alpha, z_b)
    for i in range(n):
        for j in range(g):
            d = np.abs((wbar[i, j] - q32[i]).astype(F32))
            best = d.min()
            cand = [b for b in range(1 << k) if d[b] == best]
            low = min(cand, key=lambda b: (q32[i, b], b))   # lower level, then lower code
            assert code[i, j] == low
    # Exact ties go to the lower level: levels -1.5, -0.5, 0.5, 1.5 (alpha = (1, 0.5));
    # 0 is halfway between codes 2 (-1 + 0.5) and 1 (+1 - 0.5), 1.0 between 1 and 3.
    tie = UI.nearest_codes(np.array([[0.0, 1.0, -1.0, 2.0]], F32), np.array([[1.0, 0.5]], F32),
                           np.zeros(1, F32))
    assert tie[0].tolist() == [2, 1, 0, 3]
    # z_B minimises sum (wbar - C alpha - z_B)^2: derivative zero.
    zb = UI.z_b_update(wbar, code, alpha).astype(F64)
    ca = (U.code_signs(k)[code].astype(F64) * alpha.astype(F64)[:, None, :]).sum(-1)
    want = (wbar.astype(F64) - ca).mean(axis=1)
    assert np.allclose(zb, want, rtol=0, atol=1e-6 * (1 + np.abs(want)))


def test_i6_code_and_zb_steps():
    pin_code_and_zb_steps()


# --------------------------------------------------------------------------
# I7: alternating minimisation never increases the error (exact arithmetic),
# checked in float64 on the mirror's iterates.
# --------------------------------------------------------------------------
def _err64(wbar, code, alpha, z_b, k):
    ca = (U.code_signs(k)[code].astype(F64) * np.asarray(alpha, F64)[:, None, :]).sum(-1)
    return ((np.asarray(wbar, F64) - ca - np.asarray(z_b, F64)[:, None]) ** 2).sum(axis=1)


def pin_alternating_descent():
    rs = np.random.default_rng(7)
    n, g = 24, 128
    for k, G in ((2, 1), (3, 1), (4, 1), (3, 5)):
        wbar = (rs.standard_t(4, size=(n, g)) * 2 + ((1 << k) - 1) / 2).astype(F32)
        z0 = np.full(n, ((1 << k) - 1) / 2.0, F32)
        prev = None
        for T in range(0, 7):
            alpha, z_b, code = UI.general_alternating(wbar, z0, k, G, T)
            e = _err64(wbar, code, alpha, z_b, k)
            if prev is not None:
                assert np.all(e <= prev * (1 + 1e-5) + 1e-9)
            prev = e
            if G > 1:
                assert np.array_equal(z_b, z0)      # z_B is searched by the grid instead


def test_i7_alternating_descent():
    pin_alternating_descent()


# --------------------------------------------------------------------------
# I8: exact recovery of a uniform level set, and the grid's selection rule.
# --------------------------------------------------------------------------
def pin_uniform_recovery_and_selection():
    # w takes each of 8 evenly spaced values 16 times: fixed-minimum clipping
    # at gamma = 1 maps them to 0..7, z_B = 3.5, and the greedy start finds
    # alpha = (2, 1, 0.5), whose levels are exactly 0..7.
    vals = (np.arange(8) * 0.5 - 1.75).astype(F32)
    W = np.tile(np.repeat(vals, 16), (2, 1)).astype(F32)
    rs = np.random.default_rng(8)
    W[1] = rs.permutation(W[1])
    for G, T in ((1, 0), (1, 4), (6, 3)):
        out = UI.unified_init(W, 3, 128, G=G, T=T, clip=UI.CLIP_FIXED_MIN, return_trace=True)
        assert np.all(out["err"] == 0)
        assert np.array_equal(out["alpha"], np.tile(np.array([2, 1, 0.5], F32), (2, 1)))
        assert np.all(out["delta"] == 0.5) and np.all(out["z_u"] == 3.5)
        assert np.all(out["z_b"] == 3.5)
        assert np.all(out["gamma_index"] == G - 1)
        # Level j = 3.5 + 2 c_1 + c_2 + 0.5 c_3 = 4 b_0 + 2 b_1 + b_2 with b_i the
        # code bits (bit i set <=> c_{i+1} = +1): the code is j bit-reversed.
        j = np.searchsorted(vals, W)
        want_codes = ((j >> 2) & 1) | (((j >> 1) & 1) << 1) | ((j & 1) << 2)
        assert np.array_equal(out["codes"], want_codes.astype(np.uint8))
    # The kept candidate is the first with the smallest error.
    W = _weights(rs, 8, 256)
    out = UI.unified_init(W, 3, 64, G=9, T=2, clip=UI.CLIP_BALANCED, return_trace=True)
    tr = out["trace"]
    assert np.array_equal(out["err"], tr.min(axis=0))
    assert np.array_equal(out["gamma_index"], np.argmin(tr, axis=0))
    assert np.all(out["s"] == 1) and np.all(out["s_r"] == 1)
    # Constant groups give the same candidate for every gamma (Delta' = 1): the
    # first one is kept.
    Wc = np.full((2, 128), 0.125, F32)
    Wc[1] = -0.5
    out = UI.unified_init(Wc, 2, 64, G=5, T=2, clip=UI.CLIP_FIXED_MIN, return_trace=True)
    assert np.all(out["trace"] == out["trace"][0:1])
    assert np.all(out["gamma_index"] == 0)
    assert np.all(out["delta"] == 1)


def test_i8_uniform_recovery_and_selection():
    pin_uniform_recovery_and_selection()


# --------------------------------------------------------------------------
# I9: an independent float64 implementation of the two appendix algorithms
# (own greedy loop, numpy least squares, brute-force codes, plain means).
# --------------------------------------------------------------------------
def _unified_init_f64(W, k, g, G, T, clip):
    w = np.asarray(W, F64).reshape(-1, g)
    n = w.shape[0]
    L1 = 2 ** k - 1
    signs = U.code_signs(k).astype(F64)                     # [2^k, k]
    best_err = np.full(n, np.inf)
    for j in range(1, G + 1):
        gamma = j / G
        for i in range(n):
            wm, wM = w[i].min(), w[i].max()
            delta = gamma * (wM - wm) / L1 if wM > wm else 1.0
            if clip == UI.CLIP_FIXED_MIN:
                z_u = -wm / delta
            elif clip == UI.CLIP_FIXED_MAX:
                z_u = L1 - wM / delta
            else:
                z_u = -gamma * wm / delta
            wbar = w[i] / delta + z_u
            z_b = L1 / 2.0
            r = wbar - z_b
            cols, alpha = [], []
            for _ in range(k):
                c = np.where(r >= 0, 1.0, -1.0)
                a = np.abs(r).mean()
                cols.append(c)
                alpha.append(a)
                r = r - a * c
            Cm = np.stack(cols, axis=1)
            alpha = np.array(alpha)
            for _ in range(T):
                if np.linalg.matrix_rank(Cm) == k:
                    alpha = np.linalg.lstsq(Cm, wbar - z_b, rcond=None)[0]
                lev = z_b + signs @ alpha
                Cm = signs[np.argmin(np.abs(wbar[:, None] - lev[None, :]), axis=1)]
                if G == 1:
                    z_b = np.mean(wbar - Cm @ alpha)
            lev = z_b + signs @ alpha
            q = lev[np.argmin(np.abs(wbar[:, None] - lev[None, :]), axis=1)]
            e = np.sum((w[i] - delta * (q - z_u)) ** 2)
            if e < best_err[i]:
                best_err[i] = e
    return best_err


def pin_against_f64():
    rs = np.random.default_rng(9)
    W = _weights(rs, 8, 256)
    for k, G, T, clip in ((3, 1, 6, UI.CLIP_FIXED_MIN), (2, 5, 4, UI.CLIP_FIXED_MAX),
                          (4, 4, 3, UI.CLIP_BALANCED)):
        got = UI.unified_init(W, k, 128, G=G, T=T, clip=clip)["err"].astype(F64)
        want = _unified_init_f64(W, k, 128, G, T, clip)
        rel = np.abs(got - want) / want
        assert np.median(rel) < 1e-4
        assert np.all(rel < 2e-2)
    # per-row groups: a power of two above 512 and a row length that is not one
    for C, k, G, T, clip in ((1024, 3, 3, 4, UI.CLIP_FIXED_MIN), (1000, 2, 1, 6, UI.CLIP_BALANCED),
                             (1000, 4, 2, 3, UI.CLIP_FIXED_MAX)):
        W = _weights(rs, 4, C)
        got = UI.unified_init(W, k, C, G=G, T=T, clip=clip)["err"].astype(F64)
        want = _unified_init_f64(W, k, C, G, T, clip)
        rel = np.abs(got - want) / want
        assert np.all(rel < 2e-2), (C, k, rel)
        assert np.median(rel) < 1e-3, (C, k, rel)


def test_i9_against_f64():
    pin_against_f64()


# --------------------------------------------------------------------------
# Planted mistakes: each must make at least one pin fail.
# --------------------------------------------------------------------------
def _mut_tree_sum(x):                        # running sum instead of pairwise
    x = np.asarray(x, F32)
    acc = np.zeros(x.shape[:-1], F32)
    for j in range(x.shape[-1]):
        acc = (acc + x[..., j]).astype(F32)
    return acc


def _mut_clip(wm, wM, gamma, k, clip):       # fixed maximum solved with the wrong sign
    d, z = UI._orig_clip_candidate(wm, wM, gamma, k, clip)
    if clip == UI.CLIP_FIXED_MAX:
        z = ((1 << k) - 1 + (np.asarray(wM, F32) / d)).astype(F32)
    return d, z


def _mut_clip_balanced(wm, wM, gamma, k, clip):   # balanced without gamma in z_U
    if clip == UI.CLIP_BALANCED:
        clip = UI.CLIP_FIXED_MIN
    return UI._orig_clip_candidate(wm, wM, gamma, k, clip)


def _mut_greedy(x, k):                       # mean(r) instead of mean|r|
    r = np.asarray(x, F32).copy()
    n, g = r.shape
    alpha = np.zeros((n, k), F32)
    code = np.zeros((n, g), np.int64)
    for i in range(k):
        plus = r >= 0
        a = (UI.tree_sum_f32(r) / F32(g)).astype(F32)
        alpha[:, i] = a
        code |= plus.astype(np.int64) << i
        r = np.where(plus, r - a[:, None], r + a[:, None]).astype(F32)
    return alpha, code


def _mut_det(A):                             # cofactor signs dropped
    m = A.shape[-1]
    if m <= 1:
        return UI._orig_det_int(A)
    rest = A[:, 1:, :]
    return sum(A[:, 0, j].astype(np.int64) * _mut_det(np.delete(rest, j, axis=2)) for j in range(m))


def _mut_ls(x, code, k, alpha_prev):         # C^T x without the signs
    M = UI.gram_int(code, k)
    det = UI.det_int(M)
    adj = UI.adjugate_int(M)
    v = np.stack([UI.tree_sum_f32(x)] * k, axis=1).astype(F64)
    S = np.einsum("nab,nb->na", adj.astype(F64), v)
    ok = det != 0
    a = (S / np.where(ok, det, 1)[:, None]).astype(F32)
    return np.where(ok[:, None], a, alpha_prev).astype(F32)


def _mut_codes(wbar, alpha, z_b):            # ties to the upper level
    qs, code_of, _ = U.sort_levels(U.levels_f32(alpha, z_b))
    D = np.abs((wbar[:, :, None] - qs[:, None, :]).astype(F32))
    L = qs.shape[1]
    pos = L - 1 - np.argmin(D[:, :, ::-1], axis=2)
    return np.take_along_axis(code_of, pos, axis=1)


def _mut_zb(wbar, code, alpha):              # mean of wbar, C alpha forgotten
    return (UI.tree_sum_f32(wbar) / F32(wbar.shape[1])).astype(F32)


def _mut_alternating(wbar, z_b, k, G, T):    # z_B also updated during the grid search
    return UI._orig_general_alternating(wbar, z_b, k, 1, T)


def _mut_improves(err_new, err_best):        # last minimum instead of first
    return err_new <= err_best


def _mut_error(W, k, g, delta, z_u, alpha, z_b):   # error measured in the transformed space
    e, codes = UI._orig_candidate_error(W, k, g, delta, z_u, alpha, z_b)
    return (e / (np.asarray(delta, F32) ** 2)).astype(F32), codes


MUTATIONS = [
    ("tree_sum_f32", _mut_tree_sum),
    ("clip_candidate", _mut_clip),
    ("clip_candidate", _mut_clip_balanced),
    ("greedy_f32", _mut_greedy),
    ("det_int", _mut_det),
    ("ls_alpha", _mut_ls),
    ("nearest_codes", _mut_codes),
    ("z_b_update", _mut_zb),
    ("general_alternating", _mut_alternating),
    ("improves", _mut_improves),
    ("candidate_error", _mut_error),
]

PINS = [pin_tree_sum, pin_clipping, pin_greedy, pin_adjugate, pin_ls_alpha,
        pin_code_and_zb_steps, pin_alternating_descent, pin_uniform_recovery_and_selection,
        pin_against_f64]


@pytest.mark.parametrize("name,fn", MUTATIONS, ids=[f"{m[0]}-{m[1].__name__}" for m in MUTATIONS])
def test_planted_mistake_is_caught(monkeypatch, name, fn):
    monkeypatch.setitem(UI.__dict__, "_orig_" + name, getattr(UI, name))
    monkeypatch.setattr(UI, name, fn)
    failed = []
    for pin in PINS:
        try:
            pin()
        except AssertionError:
            failed.append(pin.__name__)
        except Exception:  # a crash also counts as detection
            failed.append(pin.__name__ + "!")
    assert failed, f"planted mistake in {name} passed every pin"
