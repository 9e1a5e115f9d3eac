"""Pins of the CPU oracle to facts the paper and mathematics fix (CPU only).

Each test checks the oracle against something other than itself: the paper's
worked level set, the uniform-quantization special case (a textbook rounding
routine), brute force over all codes, the closed form of the unification
theorem, least squares, finite differences and explicit loops.  The mutation
test at the end plants plausible mistakes in the oracle and checks that these
pins catch every one of them.
"""
import itertools
import os

import numpy as np
import pytest

import oracle.uniquan as U
from paper_2506_03781_amd import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
F32 = np.float32


def _rand_params(rs, Gn, k, scale=1.0):
    alpha = (rs.uniform(0.05, 1.0, (Gn, k)) * scale).astype(F32)
    z_b = (rs.standard_normal(Gn) * scale * 0.3).astype(F32)
    return alpha, z_b


# --------------------------------------------------------------------------
# P1: the k = 2 worked level set of Sec. 2.3.
# --------------------------------------------------------------------------
def pin_k2_levels():
    rows = [ln.split() for ln in open(os.path.join(GOLDEN, "bcq_k2_levels.txt"))
            if ln.strip() and not ln.startswith("#")]
    assert len(rows) == 4
    rs = np.random.default_rng(0)
    alpha, z_b = _rand_params(rs, 7, 2)
    q = U.levels_f64(alpha, z_b)
    for gid in range(7):
        want = sorted(float(z_b[gid]) + (1 if a == "+" else -1) * float(alpha[gid, 0])
                      + (1 if b == "+" else -1) * float(alpha[gid, 1]) for a, b in rows)
        assert np.allclose(sorted(q[gid]), want, rtol=0, atol=1e-12)
        # Code convention: bit i of the code set <=> +alpha_{i+1}.
        for a, b in rows:
            code = (1 if a == "+" else 0) | ((1 if b == "+" else 0) << 1)
            v = float(z_b[gid]) + (1 if a == "+" else -1) * float(alpha[gid, 0]) \
                + (1 if b == "+" else -1) * float(alpha[gid, 1])
            assert abs(q[gid, code] - v) < 1e-12
            assert abs(float(U.levels_f32(alpha, z_b)[gid, code]) - v) < 1e-6


def test_p1_k2_worked_levels():
    pin_k2_levels()


# --------------------------------------------------------------------------
# P2: any uniform quantizer is a binary-coding one (Sec. 2.3).  With
# alpha_i = 2^(i-2) and z_B = (2^k - 1)/2 the level of code b is b itself, so
# the mapping must equal FlexRound's Clip(round(wbar), 0, 2^k - 1) bit for bit
# (ties to the lower level), and Q_{I_F} must equal Q_F.
# --------------------------------------------------------------------------
def pin_uq_special_case():
    rs = np.random.default_rng(1)
    for k in range(1, 6):
        L = 1 << k
        R, C, g = 4, 64, 32
        Gn = R * C // g
        alpha = np.tile(np.array([2.0 ** i for i in range(k)], F32) * F32(0.5), (Gn, 1)).astype(F32)
        z_b = np.full(Gn, (L - 1) / 2.0, F32)
        assert np.array_equal(U.levels_f32(alpha, z_b), np.tile(np.arange(L, dtype=F32), (Gn, 1)))
        W = (rs.uniform(-0.3, 0.3, (R, C))).astype(F32)
        W[0, :8] = np.array([0.0, 0.3, -0.3, 0.1, 0.25, -0.05, 0.02, 0.29], F32)
        s = (1 + 0.05 * rs.standard_normal((R, C))).astype(F32)
        delta = np.full(Gn, 0.6 / (L - 1), F32)
        z_u = (rs.uniform(0, L - 1, Gn)).astype(F32)
        s_r = (1 + 0.05 * rs.standard_normal(R)).astype(F32)
        out = U.fq_fwd(W, s, alpha, z_b, k, g, s_r, delta, z_u)
        # Textbook FlexRound: wbar via Eq. (1), then Clip(round-half-down, 0, 2^k-1).
        den = ((np.repeat(delta, g).reshape(R, C) * s_r[:, None]).astype(F32) * s).astype(F32)
        wbar = ((W / den).astype(F32) + np.repeat(z_u, g).reshape(R, C)).astype(F32)
        wt = np.clip(np.ceil(wbar.astype(np.float64) - 0.5), 0, L - 1)
        assert np.array_equal((out["codes"] & 0x7F).astype(np.int64), wt.astype(np.int64))
        what_flexround = np.repeat(delta, g).reshape(R, C).astype(np.float64) * (
            wt - np.repeat(z_u, g).reshape(R, C).astype(np.float64))
        assert np.allclose(out["what64"], what_flexround, rtol=0, atol=1e-12)
        # Exact half-integers tie and go to the lower level.
        half = np.array([[0.5, 1.5, 2.5, -7.0, 1e6] + [0.0] * (g - 5)], F32)
        pos = U.map_full(half, np.arange(L, dtype=F32)[None, :])
        assert list(pos[0, :5]) == [0, min(1, L - 1), min(2, L - 1), 0, L - 1]
        # General s: a uniform grid of spacing 2 s centred at z_B.
        sc = F32(0.125)
        a2 = np.tile(np.array([2.0 ** i for i in range(k)], F32) * sc, (1, 1)).astype(F32)
        lv = np.sort(U.levels_f64(a2, np.array([0.25], F32))[0])
        assert np.allclose(np.diff(lv), 2 * float(sc), rtol=0, atol=1e-15)
        assert abs(lv.mean() - 0.25) < 1e-15


def test_p2_uq_special_case():
    pin_uq_special_case()


# --------------------------------------------------------------------------
# P3: brute force over all 2^k codes (unsorted) in the same fp32 arithmetic,
# ties broken to the lower level value, then to the lower code.
# --------------------------------------------------------------------------
def brute_force_codes(wbar, alpha, z_b, k):
    Gn, g = wbar.shape
    out = np.zeros((Gn, g), np.int64)
    for gid in range(Gn):
        lv = []
        for b in range(1 << k):
            v = F32(z_b[gid])
            for i in range(k):
                v = F32(v + (alpha[gid, i] if (b >> i) & 1 else -alpha[gid, i]))
            lv.append(v)
        for j in range(g):
            best = None
            for b in range(1 << k):
                d = abs(F32(wbar[gid, j] - lv[b]))
                key = (d, lv[b], b)
                if best is None or key < best[0]:
                    best = (key, b)
            out[gid, j] = best[1]
    return out


def adversarial_case(k, seed):
    """Groups with midpoint ties, duplicate levels, zero alphas, far outliers."""
    rs = np.random.default_rng(seed)
    g = 16
    Gn = 6
    alpha, z_b = _rand_params(rs, Gn, k)
    alpha[1, :] = alpha[1, 0]               # many duplicate levels
    alpha[2, -1] = 0.0                       # alpha_k = 0: pairs of equal levels
    alpha[3, :] = F32(0.25)                  # dyadic, exact midpoints
    z_b[3] = F32(0.5)
    wbar = (rs.standard_normal((Gn, g)) * 1.5).astype(F32)
    lv3 = np.sort(U.levels_f32(alpha[3:4], z_b[3:4])[0])
    mids = ((lv3[:-1] + lv3[1:]) / 2).astype(F32)
    wbar[3, :len(mids)] = mids[:g]
    wbar[4, :4] = np.array([1e6, -1e6, 3e38, -3e38], F32)
    wbar[5, :] = z_b[5]
    return wbar, alpha, z_b


def pin_brute_force():
    rs = np.random.default_rng(2)
    for k in range(1, 6):
        Gn, g = 5, 24
        alpha, z_b = _rand_params(rs, Gn, k)
        wbar = (rs.standard_normal((Gn, g)) * 1.2).astype(F32)
        qs, code_of, _ = U.sort_levels(U.levels_f32(alpha, z_b))
        got = np.take_along_axis(code_of, U.map_full(wbar, qs), axis=1)
        assert np.array_equal(got, brute_force_codes(wbar, alpha, z_b, k))
        wbar, alpha, z_b = adversarial_case(k, 10 + k)
        qs, code_of, _ = U.sort_levels(U.levels_f32(alpha, z_b))
        got = np.take_along_axis(code_of, U.map_full(wbar, qs), axis=1)
        assert np.array_equal(got, brute_force_codes(wbar, alpha, z_b, k))
    # fp64 brute force agrees where wbar is not within 1e-5 spacing of a midpoint.
    k = 3
    alpha, z_b = _rand_params(rs, 64, k)
    wbar = (rs.standard_normal((64, 32))).astype(F32)
    lv = U.levels_f64(alpha, z_b)
    d = np.abs(wbar.astype(np.float64)[:, :, None] - lv[:, None, :])
    best = np.argmin(d, axis=2)
    ds = np.sort(d, axis=2)
    clear = (ds[:, :, 1] - ds[:, :, 0]) > 1e-5
    qs, code_of, _ = U.sort_levels(U.levels_f32(alpha, z_b))
    got = np.take_along_axis(code_of, U.map_full(wbar, qs), axis=1)
    assert clear.mean() > 0.99
    assert np.array_equal(got[clear], best[clear])


def test_p3_brute_force_mapping():
    pin_brute_force()


# --------------------------------------------------------------------------
# P4: unification theorem, R_B(C; Theta*) = D_R(R_B(C; Theta_B); Theta_R).
# --------------------------------------------------------------------------
def pin_unification():
    rs = np.random.default_rng(3)
    k, g, Gn = 3, 16, 40
    alpha, z_b = _rand_params(rs, Gn, k)
    delta = rs.uniform(0.001, 0.05, Gn).astype(F32)
    z_u = rs.uniform(-3, 10, Gn).astype(F32)
    C = rs.choice([-1.0, 1.0], size=(Gn, g, k))
    lhs_inner = np.einsum("ngk,nk->ng", C, alpha.astype(np.float64)) + z_b.astype(np.float64)[:, None]
    rhs = delta.astype(np.float64)[:, None] * (lhs_inner - z_u.astype(np.float64)[:, None])
    a_star, z_star = U.fold_params_f32(alpha, z_b, k, delta, z_u)
    a64 = delta.astype(np.float64)[:, None] * alpha.astype(np.float64)
    z64 = delta.astype(np.float64) * (z_b.astype(np.float64) - z_u.astype(np.float64))
    lhs = np.einsum("ngk,nk->ng", C, a64) + z64[:, None]
    assert np.max(np.abs(lhs - rhs) / np.maximum(np.abs(rhs).max(axis=1, keepdims=True), 1e-30)) < 1e-12
    lhs32 = np.einsum("ngk,nk->ng", C, a_star.astype(np.float64)) + z_star.astype(np.float64)[:, None]
    assert np.max(np.abs(lhs32 - rhs) / np.abs(rhs).max(axis=1, keepdims=True)) < 1e-6
    # The fold of the forward's own codes reproduces the forward's output.
    R, Cc = 8, 64
    W = (rs.standard_normal((R, Cc)) * 0.02).astype(F32)
    s = (1 + 0.01 * rs.standard_normal((R, Cc))).astype(F32)
    p = U.init_param_set_b(W, s, k, g)
    fw = U.fq_fwd(W, s, p["alpha"], p["z_b"], k, g, p["s_r"], p["delta"], p["z_u"])
    fo = U.fold(W, s, p["alpha"], p["z_b"], k, g, p["s_r"], p["delta"], p["z_u"])
    assert np.array_equal(fo["codes"], fw["codes"] & 0x7F)
    rec = U.bcq_dequant_f64(fo["codes"], fo["alpha_star"], fo["z_star"], k, g)
    scale = np.abs(fw["what64"]).reshape(-1, g).max(axis=1).repeat(g).reshape(R, Cc)
    assert np.max(np.abs(rec - fw["what64"]) / scale) < 1e-6
    assert np.max(np.abs(rec - fw["what32"]) / scale) < 1e-6


def test_p4_unification_theorem():
    pin_unification()


# --------------------------------------------------------------------------
# P5: greedy start.  For one bit, mean|r| with c = sign(r) is the least-squares
# optimum; for more bits the residual norm never grows.
# --------------------------------------------------------------------------
def pin_greedy():
    rs = np.random.default_rng(4)
    w = rs.standard_normal((30, 128))
    z = rs.standard_normal(30) * 0.1
    a1, code1 = U.greedy_bcq(w, z, 1)
    for gid in range(30):
        c = np.where(w[gid] - z[gid] >= 0, 1.0, -1.0)
        assert np.array_equal(np.where(code1[gid] & 1, 1.0, -1.0), c)
        ls = np.linalg.lstsq(c[:, None], w[gid] - z[gid], rcond=None)[0][0]
        assert abs(ls - a1[gid, 0]) < 1e-12
        # optimum over all 1-bit codes: brute force over scales for this code
        assert np.sum((w[gid] - z[gid] - ls * c) ** 2) <= np.sum((w[gid] - z[gid] - 1.01 * ls * c) ** 2)
    for k in (2, 3, 4):
        a, code = U.greedy_bcq(w, z, k)
        prev = np.sum((w - z[:, None]) ** 2, axis=1)
        for kk in range(1, k + 1):
            sg = U.code_signs(k)[code][:, :, :kk]
            rec = np.einsum("ngk,nk->ng", sg, a[:, :kk]) + z[:, None]
            res = np.sum((w - rec) ** 2, axis=1)
            assert np.all(res <= prev + 1e-12)
            prev = res
        assert np.all(a >= 0)


def test_p5_greedy_start():
    pin_greedy()


# --------------------------------------------------------------------------
# P6: straight-through gradients against central finite differences of the
# surrogate what(theta) = Delta (z_B + sum sigma_i alpha_i
#                                 + m (wbar(theta) - wbar(theta0)) - z_U)
# with codes and mask frozen at theta0; L = sum G * what.
# --------------------------------------------------------------------------
def pin_ste_gradients():
    rs = np.random.default_rng(5)
    R, C, g, k = 3, 32, 16, 3
    Gn = R * C // g
    W = rs.standard_normal((R, C)) * 0.02
    s = 1 + 0.05 * rs.standard_normal((R, C))
    s_r = 1 + 0.05 * rs.standard_normal(R)
    p = U.init_param_set_b(W.astype(F32), s.astype(F32), k, g)
    delta = p["delta"].astype(np.float64)
    z_u = p["z_u"].astype(np.float64)
    alpha = p["alpha"].astype(np.float64)
    z_b = p["z_b"].astype(np.float64)
    W = W.astype(F32).astype(np.float64)
    fw = U.fq_fwd(W, s.astype(F32), alpha.astype(F32), z_b.astype(F32), k, g,
                  s_r.astype(F32), delta.astype(F32), z_u.astype(F32))
    codes = fw["codes"].copy()
    codes.reshape(-1)[::5] &= 0x7F          # some filtered weights
    code = U.group_view(codes & 0x7F, g).astype(np.int64)
    m = U.group_view(((codes & 0x80) != 0).astype(np.float64), g)
    sig = U.code_signs(k)[code].astype(np.float64)
    G = rs.standard_normal((R, C))
    rows = U.per_group_rows(R, C, g)

    def wbar(delta_, z_u_, s_, s_r_):
        return U.group_view(W, g) / (delta_[:, None] * s_r_[rows][:, None] * U.group_view(s_, g)) + z_u_[:, None]

    wb0 = wbar(delta, z_u, s, s_r)

    def loss(delta_=delta, z_u_=z_u, s_=s, s_r_=s_r, alpha_=alpha, z_b_=z_b):
        wt = np.einsum("ngk,nk->ng", sig, alpha_) + z_b_[:, None] + m * (wbar(delta_, z_u_, s_, s_r_) - wb0)
        what = delta_[:, None] * (wt - z_u_[:, None])
        return float(np.sum(U.group_view(G, g) * what))

    got = U.fq_bwd(W, s, alpha, z_b, codes, G, k, g, s_r, delta, z_u)
    h = 1e-6

    def fd(name, arr, idx):
        a1 = arr.copy(); a1[idx] += h
        a2 = arr.copy(); a2[idx] -= h
        return (loss(**{name: a1}) - loss(**{name: a2})) / (2 * h)

    for idx in [(0, 0), (1, 5), (2, 31), (0, 17)]:
        assert abs(fd("s_", s, idx) - got["grad_s"][idx]) <= 1e-6 * max(1, abs(got["grad_s"][idx]))
    for gid in range(Gn):
        for i in range(k):
            assert abs(fd("alpha_", alpha, (gid, i)) - got["grad_alpha"][gid, i]) < 1e-6
        assert abs(fd("z_b_", z_b, gid) - got["grad_z_b"][gid]) < 1e-6
        assert abs(fd("z_u_", z_u, gid) - got["grad_z_u"][gid]) < 1e-6
        hd = 1e-9
        d1 = delta.copy(); d1[gid] += hd
        d2 = delta.copy(); d2[gid] -= hd
        fdd = (loss(delta_=d1) - loss(delta_=d2)) / (2 * hd)
        assert abs(fdd - got["grad_delta"][gid]) <= 1e-5 * max(1, abs(fdd))
    for r in range(R):
        assert abs(fd("s_r_", s_r, r) - got["grad_s_r"][r]) <= 1e-6 * max(1, abs(got["grad_s_r"][r]))
    # With nothing filtered, z_U has no net effect on what.
    nomask = codes | 0x80
    got2 = U.fq_bwd(W, s, alpha, z_b, nomask, G, k, g, s_r, delta, z_u)
    assert np.max(np.abs(got2["grad_z_u"])) < 1e-12


def test_p6_ste_gradients():
    pin_ste_gradients()


# --------------------------------------------------------------------------
# P7: idempotence and the reconstruction against explicit loops.
# --------------------------------------------------------------------------
def pin_idempotence_and_recon():
    rs = np.random.default_rng(6)
    R, C, g, k, T = 4, 32, 16, 3, 5
    Gn = R * C // g
    alpha = np.tile(np.array([0.5, 0.25, 0.125], F32), (Gn, 1))
    z_b = np.full(Gn, 0.5, F32)
    delta = np.full(Gn, 0.0625, F32)
    z_u = np.full(Gn, 2.0, F32)
    code = rs.integers(0, 1 << k, (Gn, g))
    lv = U.levels_f64(alpha, z_b)
    W = (delta[:, None] * (np.take_along_axis(lv, code, axis=1) - z_u[:, None])).reshape(R, C).astype(F32)
    s = np.ones((R, C), F32)
    out = U.fq_fwd(W, s, alpha, z_b, k, g, None, delta, z_u)
    assert np.array_equal((out["codes"] & 0x7F).reshape(Gn, g), code)
    assert np.array_equal(out["what32"], W)
    assert np.all(out["mask"])
    X = U.bf16_rne(rs.standard_normal((T, C)).astype(F32))
    Y = U.layer_target(X, W)
    E, L, Gr = U.recon(X, out["what_bf16"], Y)
    assert L == 0.0 and not np.any(Gr)
    # Loss and gradient against explicit loops on another W_hat.
    Wh = U.bf16_rne((W + 0.01 * rs.standard_normal((R, C))).astype(F32))
    E, L, Gr = U.recon(X, Wh, Y)
    Lr = 0.0
    Er = np.zeros((T, R))
    for t in range(T):
        for r in range(R):
            acc = 0.0
            for c in range(C):
                acc += float(X[t, c]) * float(Wh[r, c])
            Er[t, r] = acc - Y[t, r]
            Lr += Er[t, r] ** 2
    assert abs(L - Lr) <= 1e-12 * max(Lr, 1e-300)
    for r in range(R):
        for c in range(0, C, 7):
            gref = sum(2 * Er[t, r] * float(X[t, c]) for t in range(T))
            assert abs(Gr[r, c] - gref) < 1e-12
    # dL/dW_hat also matches a finite difference of L.
    h = 1e-4
    W1 = Wh.astype(np.float64).copy(); W1[1, 3] += h
    W2 = Wh.astype(np.float64).copy(); W2[1, 3] -= h
    fdv = (U.recon(X, W1, Y)[1] - U.recon(X, W2, Y)[1]) / (2 * h)
    assert abs(fdv - Gr[1, 3]) < 1e-6 * max(1, abs(fdv))
    # The residual form: X (What - W)^T is the same error, loss and gradient.
    Rw = U.residual_f32(Wh, W)
    assert np.array_equal(Rw.astype(np.float64), Wh.astype(np.float64) - W.astype(np.float64))  # exact here
    E2, L2, G2 = U.recon_residual(X, Rw)
    assert np.max(np.abs(E2 - E)) <= 1e-12 * max(1.0, np.abs(E).max())
    assert abs(L2 - L) <= 1e-9 * L
    assert np.max(np.abs(G2 - Gr)) <= 1e-12 * max(1.0, np.abs(Gr).max())
    assert not np.any(U.residual_f32(out["what32"], W))   # exactly quantizable W: zero residual


def test_p7_idempotence_and_recon():
    pin_idempotence_and_recon()


# --------------------------------------------------------------------------
# P8: local and periodic mapping.  If no weight moved more than one sorted
# position since the last full mapping, local = full; a two-level jump stops
# one level short; frozen keeps the code.
# --------------------------------------------------------------------------
def pin_local_mapping():
    rs = np.random.default_rng(7)
    R, C, g, k = 8, 64, 32, 3
    W = (rs.standard_normal((R, C)) * 0.02).astype(F32)
    s = np.ones((R, C), F32)
    p = U.init_param_set_a(W, s, k, g)
    f0 = U.fq_fwd(W, s, p["alpha"], p["z_b"], k, g)
    s1 = synth.perturb(s, 0.02, 0, 3)
    a1 = synth.perturb(p["alpha"], 0.01, 0, 4)
    full = U.fq_fwd(W, s1, a1, p["z_b"], k, g)
    loc = U.fq_fwd(W, s1, a1, p["z_b"], k, g, mode=U.MAP_LOCAL, codes_prev=f0["codes"])
    qs, code_of, pos_of = U.sort_levels(U.levels_f32(a1, p["z_b"]))
    prev_pos = np.take_along_axis(pos_of, U.group_view(f0["codes"] & 0x7F, g).astype(np.int64), axis=1)
    moved = np.abs(U.group_view(full["pos"], g) - prev_pos)
    assert moved.max() <= 1 and moved.max() >= 1
    assert np.array_equal(loc["codes"], full["codes"])
    frozen = U.fq_fwd(W, s1, a1, p["z_b"], k, g, mode=U.MAP_FROZEN, codes_prev=f0["codes"])
    assert np.array_equal(frozen["codes"] & 0x7F, f0["codes"] & 0x7F)
    # Two-level jump: levels 0..7 (UQ grid), previous position 2, wbar at 5.
    alpha = np.array([[0.5, 1.0, 2.0]], F32)
    z_b = np.array([3.5], F32)
    wb = np.array([[5.0, 0.2, 6.9, 2.4]], F32)
    qs, code_of, pos_of = U.sort_levels(U.levels_f32(alpha, z_b))
    assert list(U.map_local(wb, qs, np.array([[2, 2, 7, 2]]))[0]) == [3, 1, 7, 2]
    assert list(U.map_full(wb, qs)[0]) == [5, 0, 7, 2]


def test_p8_local_mapping():
    pin_local_mapping()


# --------------------------------------------------------------------------
# P9: the two readings of the code search coincide when every step is exact
# (dyadic parameters, s = s_r = 1) and differ once s varies.
# --------------------------------------------------------------------------
def pin_fold_readings():
    rs = np.random.default_rng(8)
    R, C, g, k = 4, 64, 32, 3
    Gn = R * C // g
    alpha = np.tile(np.array([0.75, 0.5, 0.25], F32), (Gn, 1))
    z_b = np.full(Gn, 3.5, F32)
    delta = np.full(Gn, 2.0 ** -6, F32)
    z_u = np.full(Gn, 3.0, F32)
    W = (np.round(rs.standard_normal((R, C)) * 128) / 2 ** 12).astype(F32)
    s = np.ones((R, C), F32)
    f0 = U.fold(W, s, alpha, z_b, k, g, None, delta, z_u, code_src=0)
    f1 = U.fold(W, s, alpha, z_b, k, g, None, delta, z_u, code_src=1)
    assert np.array_equal(f0["codes"], f1["codes"])
    s2 = (1 + 0.05 * rs.standard_normal((R, C))).astype(F32)
    f2 = U.fold(W, s2, alpha, z_b, k, g, None, delta, z_u, code_src=0)
    f3 = U.fold(W, s2, alpha, z_b, k, g, None, delta, z_u, code_src=1)
    assert 0 < np.mean(f2["codes"] != f3["codes"]) < 0.5


def test_p9_fold_readings():
    pin_fold_readings()


def pin_mask_rule():
    """Filter: gradient kept iff |wbar - wtilde| <= tau = min alpha (equality kept).
    Expected flags worked by hand from the levels listed below."""
    alpha = np.array([[1.0, 0.25]], F32)
    z_b = np.array([0.0], F32)
    # levels: -1.25, -0.75, 0.75, 1.25 ; tau = 0.25
    W = np.array([[1.5, 1.75, 1.4, -1.5, 0.0, -2.0, 0.75, 1.51]], F32)
    out = U.fq_fwd(W, np.ones_like(W), alpha, z_b, 2, 8)
    assert list(out["mask"][0]) == [True, False, True, True, False, False, True, False]


def test_mask_rule():
    pin_mask_rule()


def pin_bf16_rne():
    xs = np.array([1.0, 1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, 1.0 + 2 ** -9, -3.0e-3, 65504.0, 1e-40], F32)
    got = U.bf16_rne(xs)
    for x, y in zip(xs, got):
        # nearest bf16 by exhaustive neighbourhood search, ties to even mantissa
        u = int(np.array([x], F32).view(np.uint32)[0] >> 16)
        cands = [np.array([(u + d) << 16], np.uint32).view(F32)[0] for d in (-1, 0, 1) if 0 <= u + d < (1 << 16)]
        best = min(cands, key=lambda c: (abs(float(c) - float(x)),
                                         (np.array([c], F32).view(np.uint32)[0] >> 16) & 1))
        assert float(best) == float(y)


def test_bf16_rne_against_definition():
    pin_bf16_rne()


def test_synth_shapes_and_statistics():
    spec = synth.scaled(synth.WORKLOADS["attn4096"].matrices[0], R=256, C=1024, T=64)
    m = synth.make_matrix(spec, 0)
    assert m.W.shape == (256, 1024) and m.X.shape == (64, 1024)
    assert np.array_equal(synth.round_to_bf16(m.W), m.W)
    assert len(m.outlier_cols) == round(0.01 * 1024)
    inl = np.setdiff1d(np.arange(1024), m.outlier_cols)
    assert 0.015 < m.W[:, inl].std() < 0.025
    assert abs(m.s.mean() - 1) < 1e-3
    m2 = synth.make_matrix(spec, 0)
    assert np.array_equal(m.W, m2.W) and np.array_equal(m.X, m2.X)


# --------------------------------------------------------------------------
# Planted mistakes: each plausible error in the oracle must fail some pin.
# --------------------------------------------------------------------------
PINS = [pin_k2_levels, pin_uq_special_case, pin_brute_force, pin_unification, pin_greedy,
        pin_ste_gradients, pin_idempotence_and_recon, pin_local_mapping, pin_fold_readings,
        pin_mask_rule, pin_bf16_rne]


def _mut_levels_order(alpha, z_b):          # sign convention flipped
    q = U.__dict__["_orig_levels_f32"](alpha, z_b)
    return q[:, ::-1].copy()


def _mut_transform(W, s, g, s_r=None, delta=None, z_u=None):   # multiply instead of divide by s
    R, C = W.shape
    s_r, delta, z_u = U.expand_params(R, C, g, s_r, delta, z_u)
    rows = U.per_group_rows(R, C, g)
    w = U.group_view(np.asarray(W, F32), g)
    den = (delta * s_r[rows]).astype(F32)[:, None] / U.group_view(np.asarray(s, F32), g)
    return ((w / den).astype(F32) + z_u[:, None]).astype(F32)


def _mut_map_last_min(wbar, qs):            # ties to the upper level
    D = np.abs((wbar[:, :, None] - qs[:, None, :]).astype(F32))
    L = qs.shape[1]
    return L - 1 - np.argmin(D[:, :, ::-1], axis=2)


def _mut_tau(alpha):                        # max instead of min
    return np.max(np.abs(np.asarray(alpha, F32)), axis=1).astype(F32)


def _mut_map_local(wbar, qs, pos_prev):     # two-sided window of 2
    L = qs.shape[1]
    best = np.maximum(pos_prev - 2, 0)
    bd = np.abs((wbar - np.take_along_axis(qs, best, axis=1)).astype(F32))
    for c in [np.maximum(pos_prev - 1, 0), pos_prev, np.minimum(pos_prev + 1, L - 1), np.minimum(pos_prev + 2, L - 1)]:
        d = np.abs((wbar - np.take_along_axis(qs, c, axis=1)).astype(F32))
        best = np.where(d < bd, c, best)
        bd = np.minimum(d, bd)
    return best


def _mut_fold(alpha, z_b, k, delta=None, z_u=None):     # dropped z_U
    a, z = U.__dict__["_orig_fold_params_f32"](alpha, z_b, k, delta, None)
    return a, z


def _mut_greedy(wbar, z_b, k):              # residual never updated
    r = np.asarray(wbar, np.float64) - np.asarray(z_b, np.float64)[:, None]
    alpha = np.zeros((r.shape[0], k))
    code = np.zeros(r.shape, np.int64)
    for i in range(k):
        c = np.where(r >= 0, 1.0, -1.0)
        alpha[:, i] = np.abs(r).mean(axis=1)
        code |= (c > 0).astype(np.int64) << i
    return alpha, code


def _mut_greedy_signed(wbar, z_b, k):       # mean(r) instead of mean|r|
    r = np.asarray(wbar, np.float64) - np.asarray(z_b, np.float64)[:, None]
    alpha = np.zeros((r.shape[0], k))
    code = np.zeros(r.shape, np.int64)
    for i in range(k):
        c = np.where(r >= 0, 1.0, -1.0)
        alpha[:, i] = r.mean(axis=1)
        code |= (c > 0).astype(np.int64) << i
        r = r - alpha[:, i:i + 1] * c
    return alpha, code


def _mut_recon(X, W_hat, Y):                # missing factor 2 in the gradient
    E, L, Gr = U.__dict__["_orig_recon"](X, W_hat, Y)
    return E, L, Gr / 2


MUTATIONS = [
    ("levels_f32", _mut_levels_order),
    ("transform_f32", _mut_transform),
    ("map_full", _mut_map_last_min),
    ("tau_f32", _mut_tau),
    ("map_local", _mut_map_local),
    ("fold_params_f32", _mut_fold),
    ("greedy_bcq", _mut_greedy),
    ("greedy_bcq", _mut_greedy_signed),
    ("recon", _mut_recon),
]


def _mut_bwd_sign(*a, **kw):                # sign error in grad_s
    out = U.__dict__["_orig_fq_bwd"](*a, **kw)
    out["grad_s"] = -out["grad_s"]
    return out


MUTATIONS.append(("fq_bwd", _mut_bwd_sign))


def _mut_levels64(alpha, z_b):              # shift dropped in the value path
    return U.__dict__["_orig_levels_f64"](alpha, np.zeros_like(np.asarray(z_b)))


def _mut_bf16_trunc(x):                     # truncation instead of round-to-nearest-even
    u = np.ascontiguousarray(x, F32).view(np.uint32)
    return (u & np.uint32(0xFFFF0000)).view(F32)


MUTATIONS += [("levels_f64", _mut_levels64), ("bf16_rne", _mut_bf16_trunc)]


def _mut_residual(what32, W):               # sign of the residual flipped
    return (np.asarray(W, F32) - np.asarray(what32, F32)).astype(F32)


def _mut_recon_residual(X, Rw):             # missing factor 2 in the gradient
    E, L, G = U._orig_recon_residual(X, Rw)
    return E, L, 0.5 * G


MUTATIONS += [("residual_f32", _mut_residual), ("recon_residual", _mut_recon_residual)]


@pytest.mark.parametrize("name,fn", MUTATIONS, ids=[f"{m[0]}-{m[1].__name__}" for m in MUTATIONS])
def test_planted_mistake_is_caught(monkeypatch, name, fn):
    monkeypatch.setitem(U.__dict__, "_orig_" + name, getattr(U, name))
    monkeypatch.setattr(U, name, fn)
    failed = []
    for pin in PINS:
        try:
            pin()
        except AssertionError:
            failed.append(pin.__name__)
        except Exception:  # a crash also counts as detection
            failed.append(pin.__name__ + "!")
    assert failed, f"planted mistake in {name} passed every pin"
