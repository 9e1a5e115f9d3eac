"""Pins of the deployment oracle (oracle/bcq_deploy.py) to facts that do not
come from the oracle itself: the bit count the paper gives for a stored group
(appendix "Memory usage": g k + 16 (k + 1) bits), a brute-force reading of
every stored bit on a tiny matrix, round-to-nearest-even into binary16 at
hand-picked ties, the closed form of a uniform level set, the fold path of
the training oracle (Theorem 1), and an explicit per-group evaluation of the
product.  Planted mistakes at the end must each fail one of them.
"""
import numpy as np
import pytest

import oracle.bcq_deploy as D
import oracle.uniquan as U

F32 = np.float32


def rand_codes(R, C, k, seed):
    return np.random.default_rng(seed).integers(0, 1 << k, size=(R, C), dtype=np.uint8)


def dyadic_params(Gn, k, seed):
    """alpha*, z* that binary16 holds exactly (at most 11 significant bits)."""
    rs = np.random.default_rng(seed)
    a = (rs.integers(1, 2048, size=(Gn, k)) / 4096.0).astype(F32)
    z = (rs.integers(-2047, 2048, size=Gn) / 2048.0).astype(F32)
    return a, z


def pin_bit_layout_brute_force():
    """Every stored bit, read one at a time with plain loops."""
    R, C, k = 3, 256, 3
    codes = rand_codes(R, C, k, 1)
    planes = D.pack_planes(codes, k)
    assert planes.shape == (k, C // 128, R, 4) and planes.dtype == np.uint32
    for i in range(k):
        for q in range(C // 128):
            for r in range(R):
                for m in range(4):
                    word = int(planes[i, q, r, m])
                    for j in range(32):
                        c = 128 * q + 32 * m + j
                        assert (word >> j) & 1 == (int(codes[r, c]) >> i) & 1, (i, q, r, m, j)
    assert np.array_equal(D.unpack_planes(planes, R, C), codes)


def pin_round_trip():
    for (R, C, k) in ((5, 512, 4), (7, 384, 1), (2, 128, 2)):
        codes = rand_codes(R, C, k, R + C + k)
        assert np.array_equal(D.unpack_planes(D.pack_planes(codes, k), R, C), codes)


def pin_storage_bits():
    """g k + 16 (k + 1) bits per group (appendix "Memory usage")."""
    for (R, C, k, g) in ((4, 512, 3, 128), (2, 1024, 4, 256), (3, 768, 2, 768), (1, 128, 1, 128)):
        Gn = R * C // g
        a, z = dyadic_params(Gn, k, 2)
        st = D.pack(rand_codes(R, C, k, 3), a, z, k, g)
        assert D.storage_bits(*st) == Gn * (g * k + 16 * (k + 1))


def pin_fp16_rounding():
    """binary16 keeps 10 fraction bits: ties round to the even neighbour."""
    one = 1.0
    vals = np.array([one + 2.0 ** -11,            # halfway between 1 and 1 + 2^-10 -> 1
                     one + 3 * 2.0 ** -11,        # halfway between 1 + 2^-10 and 1 + 2^-9 -> 1 + 2^-9
                     one + 2.0 ** -11 + 2.0 ** -20,   # just above the first tie -> 1 + 2^-10
                     -(one + 2.0 ** -11)], F32)
    want = np.array([1.0, 1.0 + 2.0 ** -9, 1.0 + 2.0 ** -10, -1.0])
    a16, z16 = D.params_fp16(vals.reshape(1, 4), np.zeros(1, F32), 1, 128, 4, 128)
    assert np.array_equal(a16.reshape(-1).astype(np.float64), want)


def pin_dequant_matches_training_fold():
    """With binary16-exact parameters the stored form reproduces
    R_B(C; Theta*) of the training oracle exactly (a different code path:
    level tables and a gather)."""
    R, C, k, g = 6, 512, 3, 128
    Gn = R * C // g
    a, z = dyadic_params(Gn, k, 4)
    codes = rand_codes(R, C, k, 5)
    st = D.pack(codes, a, z, k, g)
    W = D.dequant_f64(*st, R, C, g)
    assert np.array_equal(W, U.bcq_dequant_f64(codes, a, z, k, g))


def pin_uniform_closed_form():
    """alpha*_i = s 2^(i-1): the levels are z + s (2 b - (2^k - 1)) for code b,
    so the product is X times that matrix (computed here directly)."""
    R, C, k, g = 4, 256, 4, 128
    Gn = R * C // g
    s = 2.0 ** -6
    a = np.tile((s * 2.0 ** np.arange(k)).astype(F32), (Gn, 1))
    z = np.linspace(-0.5, 0.5, Gn).astype(np.float16).astype(F32)
    codes = rand_codes(R, C, k, 6)
    W = np.repeat(z.reshape(R, C // g), g, axis=1).astype(np.float64) + s * (2.0 * codes - (2 ** k - 1))
    X = np.random.default_rng(7).standard_normal((3, C))
    st = D.pack(codes, a, z, k, g)
    Y = D.matmul_f64(X, *st, R, C, g)
    assert np.allclose(Y, X @ W.T, rtol=1e-13, atol=1e-13)


def pin_per_group_evaluation():
    """y[t, r] = sum over groups of z S + sum_i alpha_i (2 P_i - S), with S the
    group's activation sum and P_i the sum over weights whose bit i is set:
    evaluated with plain loops on a tiny case."""
    R, C, k, g = 2, 256, 2, 128
    Gn = R * C // g
    a, z = dyadic_params(Gn, k, 8)
    codes = rand_codes(R, C, k, 9)
    X = np.random.default_rng(10).standard_normal((2, C))
    st = D.pack(codes, a, z, k, g)
    Y = D.matmul_f64(X, *st, R, C, g)
    for t in range(2):
        for r in range(R):
            y = 0.0
            for j in range(C // g):
                gid = r * (C // g) + j
                cols = range(j * g, (j + 1) * g)
                S = sum(X[t, c] for c in cols)
                y += float(z[gid]) * S
                for i in range(k):
                    P = sum(X[t, c] for c in cols if (int(codes[r, c]) >> i) & 1)
                    y += float(a[gid, i]) * (2 * P - S)
            assert abs(Y[t, r] - y) <= 1e-12 * max(1.0, abs(y))


def pin_theorem1_end_to_end():
    """Training-side What (fq_fwd) vs the stored form built from the fold:
    equal up to the binary16 rounding of alpha*, z*."""
    rs = np.random.default_rng(11)
    R, C, k, g = 4, 256, 3, 128
    W = (rs.standard_normal((R, C)) * 0.02).astype(F32)
    s = (1 + 0.01 * rs.standard_normal((R, C))).astype(F32)
    p = U.init_param_set_b(W, s, k, g)
    fo = U.fold(W, s, p["alpha"], p["z_b"], k, g, p["s_r"], p["delta"], p["z_u"])
    st = D.pack(fo["codes"], fo["alpha_star"], fo["z_star"], k, g)
    Wd = D.dequant_f64(*st, R, C, g)
    ref = U.fq_fwd(W, s, p["alpha"], p["z_b"], k, g, p["s_r"], p["delta"], p["z_u"])["what32"]
    bound = (np.abs(fo["z_star"]) + np.abs(fo["alpha_star"]).sum(axis=1)) * 2.0 ** -10
    err = np.abs(Wd - ref).reshape(-1, g).max(axis=1)
    assert np.all(err <= bound + 1e-7), (err, bound)


def pin_layout_checks():
    with pytest.raises(ValueError):
        D.pack(rand_codes(2, 192, 2, 0), *dyadic_params(3, 2, 0), 2, 64)
    with pytest.raises(ValueError):
        D.pack(rand_codes(2, 256, 5, 0), *dyadic_params(4, 5, 0), 5, 128)


PINS = [pin_bit_layout_brute_force, pin_round_trip, pin_storage_bits, pin_fp16_rounding,
        pin_dequant_matches_training_fold, pin_uniform_closed_form, pin_per_group_evaluation,
        pin_theorem1_end_to_end, pin_layout_checks]


@pytest.mark.parametrize("pin", PINS, ids=[p.__name__ for p in PINS])
def test_pin(pin):
    pin()


# --------------------------------------------------------------------------
# Planted mistakes
# --------------------------------------------------------------------------
def _mut_bit_order(codes, k):                    # bit j stored as bit 31 - j
    p = D._orig_pack_planes(codes, k)
    out = np.zeros_like(p)
    for j in range(32):
        out |= ((p >> np.uint32(j)) & np.uint32(1)) << np.uint32(31 - j)
    return out


def _mut_plane_shift(codes, k):                  # plane i holds bit i + 1
    return D._orig_pack_planes(np.asarray(codes, np.uint8) >> np.uint8(1), k)


def _mut_row_major(codes, k):                    # rows outermost instead of column quads
    p = D._orig_pack_planes(codes, k)
    k_, nq, R, _ = p.shape
    return np.ascontiguousarray(p.transpose(0, 2, 1, 3)).reshape(k_, nq, R, 4)


def _mut_fp16_trunc(alpha_star, z_star, R, C, k, g):   # truncation instead of RNE
    a, z = D._orig_params_fp16(alpha_star, z_star, R, C, k, g)
    def trunc(x32, x16):
        b = np.asarray(x32, np.float32).view(np.uint32) & np.uint32(0xFFFFE000)
        return b.view(np.float32).astype(np.float16)
    gpr = C // g
    a32 = np.asarray(alpha_star, np.float32).reshape(R, gpr, k).transpose(2, 1, 0)
    z32 = np.asarray(z_star, np.float32).reshape(R, gpr).T
    return trunc(a32, a), trunc(z32, z)


def _mut_params_order(alpha_star, z_star, R, C, k, g):  # [k, R, C/g] read as [k, C/g, R]
    gpr = C // g
    a = np.asarray(alpha_star, np.float32).reshape(R, gpr, k).transpose(2, 0, 1)
    z = np.asarray(z_star, np.float32).reshape(R, gpr)
    return (np.ascontiguousarray(a).reshape(k, gpr, R).astype(np.float16),
            np.ascontiguousarray(z).reshape(gpr, R).astype(np.float16))


def _mut_sigma01(planes, alpha16, z16, R, C, g):        # sigma in {0, 1} instead of {-1, +1}
    W = D._orig_dequant_f64(planes, alpha16, z16, R, C, g)
    a = np.asarray(alpha16, np.float16).astype(np.float64)
    return W + np.repeat(a.sum(axis=0).T, g, axis=1)    # adds back sum alpha: bit-0 terms become 0


def _mut_no_shift(planes, alpha16, z16, R, C, g):       # z*_B dropped
    return D._orig_dequant_f64(planes, alpha16, np.zeros_like(z16), R, C, g)


MUTATIONS = [("pack_planes", _mut_bit_order), ("pack_planes", _mut_plane_shift),
             ("pack_planes", _mut_row_major), ("params_fp16", _mut_fp16_trunc),
             ("params_fp16", _mut_params_order), ("dequant_f64", _mut_sigma01),
             ("dequant_f64", _mut_no_shift)]


@pytest.mark.parametrize("name,fn", MUTATIONS, ids=[f"{m[0]}-{m[1].__name__}" for m in MUTATIONS])
def test_planted_mistake_is_caught(monkeypatch, name, fn):
    monkeypatch.setitem(D.__dict__, "_orig_" + name, getattr(D, name))
    monkeypatch.setattr(D, name, fn)
    failed = []
    for pin in PINS:
        try:
            pin()
        except AssertionError:
            failed.append(pin.__name__)
        except Exception:  # a crash also counts as detection
            failed.append(pin.__name__ + "!")
    assert failed, f"planted mistake in {name} passed every pin"
