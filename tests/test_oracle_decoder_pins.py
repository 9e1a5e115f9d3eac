"""Pins of the decoder-block oracle (oracle/block_decoder.py) to facts
outside it: RMSNorm's closed form and scale invariance, the rotary
embedding's rotation properties (identity at position 0, norms kept,
dependence of q.k on the position difference only, exact inverse), the
causal softmax's row sums and causality, an explicit loop evaluation of the
block, central finite differences of the block loss for all seven weight
matrices, the zero-loss fixed point, where the storage hook applies, and the
reduction to the MLP oracle when the attention output projection is zero.
Planted mistakes must each fail one of them.
"""
import numpy as np
import pytest

import oracle.block_decoder as D
import oracle.block_mlp as M
import oracle.uniquan as U

F64 = np.float64


def tiny(seed, n_seq=2, L=3, C=8, H=2, I=12, scale=0.6, n_kv=None):
    rs = np.random.default_rng(seed)
    T = n_seq * L
    Ckv = C // H * (H if n_kv is None else n_kv)
    X = rs.standard_normal((T, C))
    W = {n: rs.standard_normal(sh) * scale for n, sh in
         (("q", (C, C)), ("k", (Ckv, C)), ("v", (Ckv, C)), ("o", (C, C)), ("g", (I, C)), ("u", (I, C)), ("d", (C, I)))}
    g1 = 1.0 + 0.2 * rs.standard_normal(C)
    g2 = 1.0 + 0.2 * rs.standard_normal(C)
    Y_ref = rs.standard_normal((T, C))
    return X, W, g1, g2, Y_ref, n_seq, H


def pin_rmsnorm():
    x = np.array([[3.0, -4.0, 0.0, 0.0]])
    y, r = D.rmsnorm(x, np.ones(4), eps=0.0)
    assert np.allclose(r, 1.0 / np.sqrt(25.0 / 4.0)) and np.allclose(y, x / 2.5)
    rs = np.random.default_rng(0)
    x = rs.standard_normal((5, 16))
    g = rs.standard_normal(16)
    y1, _ = D.rmsnorm(x, g, eps=0.0)
    y2, _ = D.rmsnorm(7.5 * x, g, eps=0.0)
    assert np.allclose(y1, y2, rtol=1e-13)
    # backward against central differences of <w, rmsnorm(x)>
    wv = rs.standard_normal((5, 16))
    _, r = D.rmsnorm(x, g)
    ana = D.rmsnorm_bwd(wv, x, g, r)
    h = 1e-6
    num = np.zeros_like(x)
    for idx in np.ndindex(x.shape):
        xp, xm = x.copy(), x.copy()
        xp[idx] += h
        xm[idx] -= h
        num[idx] = (np.sum(wv * D.rmsnorm(xp, g)[0]) - np.sum(wv * D.rmsnorm(xm, g)[0])) / (2 * h)
    assert np.allclose(ana, num, rtol=1e-6, atol=1e-8)


def pin_rope():
    rs = np.random.default_rng(1)
    L, d = 9, 8
    ang = D.rope_angles(L, d)
    assert np.allclose(ang[0], 0.0) and np.isclose(ang[1, 0], 1.0) and np.isclose(ang[1, 1], 1e4 ** -0.25)
    x = rs.standard_normal((L, d))
    y = D.rope(x, ang)
    assert np.allclose(y[0], x[0])
    h = d // 2
    assert np.allclose(y[:, :h] ** 2 + y[:, h:] ** 2, x[:, :h] ** 2 + x[:, h:] ** 2)
    assert np.allclose(D.rope(y, ang, inverse=True), x, atol=1e-13)
    # as complex numbers (x_i + i x_{i+d/2}) e^{i angle}
    z = (x[:, :h] + 1j * x[:, h:]) * np.exp(1j * ang)
    assert np.allclose(y[:, :h], z.real) and np.allclose(y[:, h:], z.imag)
    # q.k depends on the position difference only
    q, k = rs.standard_normal(d), rs.standard_normal(d)
    Q, K = D.rope(np.tile(q, (L, 1)), ang), D.rope(np.tile(k, (L, 1)), ang)
    assert np.isclose(Q[5] @ K[2], Q[7] @ K[4]) and np.isclose(Q[3] @ K[3], q @ k)


def pin_causal_softmax():
    rs = np.random.default_rng(2)
    S = rs.standard_normal((3, 6, 6))
    P = D.causal_softmax(S)
    assert np.allclose(P.sum(-1), 1.0) and np.all(np.triu(P[0], 1) == 0.0)
    assert np.allclose(P[:, 0, 0], 1.0)
    S2 = S.copy()
    S2[:, 2, 3:] += 50.0  # future keys of query 2
    assert np.allclose(D.causal_softmax(S2), P)
    row = np.exp(S[1, 4, :5] - S[1, 4, :5].max())
    assert np.allclose(P[1, 4, :5], row / row.sum())


def _loop_forward(X, W, g1, g2, n_seq, H):
    T, C = X.shape
    L, d = T // n_seq, C // H

    def norm(v, g):
        r = 1.0 / np.sqrt(sum(t * t for t in v) / len(v) + D.EPS)
        return [v[c] * r * g[c] for c in range(len(v))]

    def lin(v, Wm):
        return [sum(Wm[o, c] * v[c] for c in range(len(v))) for o in range(Wm.shape[0])]

    def rot(v, p):
        out = list(v)
        for i in range(d // 2):
            a = p * 1e4 ** (-2.0 * i / d)
            out[i] = v[i] * np.cos(a) - v[i + d // 2] * np.sin(a)
            out[i + d // 2] = v[i + d // 2] * np.cos(a) + v[i] * np.sin(a)
        return out

    Y = np.zeros((T, C))
    for sq in range(n_seq):
        toks = range(sq * L, (sq + 1) * L)
        Z = {t: norm(list(X[t]), g1) for t in toks}
        Q = {t: lin(Z[t], W["q"]) for t in toks}
        K = {t: lin(Z[t], W["k"]) for t in toks}
        V = {t: lin(Z[t], W["v"]) for t in toks}
        for t in toks:
            o = [0.0] * C
            for h in range(H):
                sl = slice(h * d, (h + 1) * d)
                qt = rot(Q[t][sl], t - sq * L)
                sc = []
                for u in toks:
                    if u > t:
                        continue
                    ku = rot(K[u][sl], u - sq * L)
                    sc.append((u, sum(a * b for a, b in zip(qt, ku)) / np.sqrt(d)))
                m = max(s for _, s in sc)
                den = sum(np.exp(s - m) for _, s in sc)
                for u, s in sc:
                    for j in range(d):
                        o[h * d + j] += np.exp(s - m) / den * V[u][sl][j]
            R = [X[t, c] + v for c, v in enumerate(lin(o, W["o"]))]
            Z2 = norm(R, g2)
            G, Uv = lin(Z2, W["g"]), lin(Z2, W["u"])
            Hm = [g / (1.0 + np.exp(-g)) * u for g, u in zip(G, Uv)]
            Y[t] = [R[c] + v for c, v in enumerate(lin(Hm, W["d"]))]
    return Y


def pin_forward_loops():
    X, W, g1, g2, _, n_seq, H = tiny(3)
    f = D.decoder_forward(X, W, g1, g2, n_seq, H)
    assert np.allclose(f["Y"], _loop_forward(X, W, g1, g2, n_seq, H), rtol=1e-11, atol=1e-11)


def pin_gradients_finite_differences():
    # multi-head (2 heads) and grouped-query (4 query heads sharing 2 key/value heads)
    for kw in (dict(H=2), dict(H=4, n_kv=2)):
        X, W, g1, g2, Y_ref, n_seq, H = tiny(4, **kw)
        nkv = kw.get("n_kv")
        st = D.decoder_step(X, Y_ref, W, g1, g2, n_seq, H, n_kv=nkv)
        h = 1e-6
        for name in W:
            num = np.zeros_like(W[name])
            for idx in np.ndindex(W[name].shape):
                Wp = {n: w.copy() for n, w in W.items()}
                Wm = {n: w.copy() for n, w in W.items()}
                Wp[name][idx] += h
                Wm[name][idx] -= h
                num[idx] = (D.decoder_step(X, Y_ref, Wp, g1, g2, n_seq, H, n_kv=nkv)["loss"]
                            - D.decoder_step(X, Y_ref, Wm, g1, g2, n_seq, H, n_kv=nkv)["loss"]) / (2 * h)
            scale = max(1.0, np.max(np.abs(num)))
            assert np.allclose(st["grads"][name], num, rtol=1e-5, atol=1e-6 * scale), (kw, name)


def pin_zero_loss():
    X, W, g1, g2, _, n_seq, H = tiny(5)
    Y = D.decoder_forward(X, W, g1, g2, n_seq, H)["Y"]
    st = D.decoder_step(X, Y, W, g1, g2, n_seq, H)
    assert st["loss"] == 0.0
    for g in st["grads"].values():
        assert np.all(g == 0.0)


def pin_store_hook():
    X, W, g1, g2, Y_ref, n_seq, H = tiny(6, L=4, C=16, H=2, I=24)
    st = D.decoder_step(X, Y_ref, W, g1, g2, n_seq, H, store=U.bf16_rne)
    for k in ("Z1", "Qh", "Kh", "Vh", "P", "O", "Z2", "G", "U", "H", "E", "dS", "dQ", "dK"):
        v = np.asarray(st[k], F64)
        assert np.array_equal(v, U.bf16_rne(v.astype(np.float32)).astype(F64)), k
    plain = D.decoder_step(X, Y_ref, W, g1, g2, n_seq, H)
    assert abs(plain["loss"] - st["loss"]) <= 1e-2 * plain["loss"]


def pin_reduces_to_mlp():
    """With W_o = 0 the attention module adds nothing: Y = X + MLP(RMSNorm(X; g2))."""
    X, W, g1, g2, _, n_seq, H = tiny(7)
    W["o"] = np.zeros_like(W["o"])
    f = D.decoder_forward(X, W, g1, g2, n_seq, H)
    z, _ = D.rmsnorm(X, g2)
    assert np.allclose(f["Y"], X + M.mlp_forward(z, W["g"], W["u"], W["d"])["Y"], rtol=1e-13, atol=1e-13)


def pin_grouped_heads():
    """Grouped-query attention equals multi-head attention whose key/value
    projections repeat each shared head's rows for every query head of its
    group; with as many key/value heads as query heads it is multi-head."""
    X, W, g1, g2, Y_ref, n_seq, H = tiny(9, C=16, H=4, n_kv=2)
    d, G = 16 // 4, 2
    Wm = dict(W)
    for n in ("k", "v"):
        Wm[n] = np.concatenate([W[n][kv * d:(kv + 1) * d] for kv in range(2) for _ in range(G)], axis=0)
    a = D.decoder_forward(X, W, g1, g2, n_seq, H, n_kv=2)["Y"]
    b = D.decoder_forward(X, Wm, g1, g2, n_seq, H)["Y"]
    assert np.allclose(a, b, rtol=1e-12, atol=1e-12)
    st_g = D.decoder_step(X, Y_ref, W, g1, g2, n_seq, H, n_kv=2)
    st_m = D.decoder_step(X, Y_ref, Wm, g1, g2, n_seq, H)
    for n in ("k", "v"):   # the shared head's gradient is the sum over its group's copies
        summed = sum(st_m["grads"][n].reshape(2, G, d, 16)[:, g] for g in range(G)).reshape(2 * d, 16)
        assert np.allclose(st_g["grads"][n], summed, rtol=1e-10, atol=1e-12), n
    assert np.allclose(D.decoder_forward(X, Wm, g1, g2, n_seq, H, n_kv=4)["Y"], b)


def pin_softmax_row_term():
    """DB10: the softmax backward's row term.  Without storage rounding the
    step's delta_i = dO_i . O_i equals sum_j P_ij dP_ij (O = P V), and dS has
    zero row sums (the softmax Jacobian annihilates constants); with the bf16
    storage hook the two row terms differ only by the rounding of O."""
    rs = np.random.default_rng(21)
    n_seq, H, C, I = 2, 2, 16, 12
    T = 2 * 5
    X = rs.standard_normal((T, C))
    W = {n: 0.3 * rs.standard_normal(sh) for n, sh in
         (("q", (C, C)), ("k", (C, C)), ("v", (C, C)), ("o", (C, C)), ("g", (I, C)), ("u", (I, C)), ("d", (C, I)))}
    g1, g2 = 1 + 0.1 * rs.standard_normal(C), 1 + 0.1 * rs.standard_normal(C)
    Y_ref = rs.standard_normal((T, C))
    st = D.decoder_step(X, Y_ref, W, g1, g2, n_seq, H)
    dOh = D.split_heads(st["dR"] @ W["o"], n_seq, H)
    dP = dOh @ np.swapaxes(st["Vx"], -1, -2)
    delta_p = np.sum(st["P"] * dP, axis=-1)
    delta_o = np.sum(dOh * D.split_heads(st["O"], n_seq, H), axis=-1)
    assert np.allclose(delta_o, delta_p, rtol=1e-12, atol=1e-12)
    assert np.allclose(st["dS"].sum(-1), 0.0, atol=1e-12)
    # the step's dS is P (dP - delta) with that row term
    assert np.allclose(st["dS"], st["P"] * (dP - delta_p[..., None]), rtol=1e-12, atol=1e-12)


PINS = [pin_rmsnorm, pin_rope, pin_causal_softmax, pin_forward_loops, pin_gradients_finite_differences,
        pin_zero_loss, pin_store_hook, pin_reduces_to_mlp, pin_grouped_heads, pin_softmax_row_term]


@pytest.mark.parametrize("pin", PINS, ids=[p.__name__ for p in PINS])
def test_pin(pin):
    pin()


def _mut_rope_sign(x, ang, inverse=False):        # rotation in the opposite sense
    return D._orig_rope(x, ang, not inverse)


def _mut_rope_halves(x, ang, inverse=False):      # pairs (2i, 2i+1) taken as (i, i + d/2) of a permuted vector
    x = np.asarray(x, F64)
    return D._orig_rope(x[..., ::-1], ang, inverse)[..., ::-1]


def _mut_mask(S):                                 # the diagonal masked too (first key only for row 0)
    S = np.asarray(S, F64)
    L = S.shape[-1]
    mask = np.triu(np.ones((L, L), dtype=bool), 0)
    mask[0, 0] = False
    Sm = np.where(mask, -np.inf, S)
    e = np.exp(Sm - np.max(Sm, axis=-1, keepdims=True))
    return e / np.sum(e, axis=-1, keepdims=True)


def _mut_rms_bwd(dy, x, gamma, r):               # second term dropped
    return r * np.asarray(dy, F64) * np.asarray(gamma, F64)


def _mut_rmsnorm(x, gamma, eps=D.EPS):           # mean absolute value instead of root mean square
    x = np.asarray(x, F64)
    r = 1.0 / (np.mean(np.abs(x), axis=-1, keepdims=True) + eps)
    return x * r * np.asarray(gamma, F64), r


def _mut_step_softmax_bwd(Xhat, Y_ref, W, g1, g2, n_seq, H, store=D._ident):  # dS without the row-sum term
    st = D._orig_decoder_step(Xhat, Y_ref, W, g1, g2, n_seq, H, store)
    dOh = D.split_heads(st["dR"] @ np.asarray(W["o"], F64), n_seq, H)
    dP = dOh @ np.swapaxes(st["Vh"], -1, -2)
    d = st["R"].shape[1] // H
    dQ = D.merge_heads(D.rope((st["P"] * dP) @ st["Kh"] / np.sqrt(d), st["ang"], inverse=True))
    st["grads"]["q"] = dQ.T @ st["Z1"]
    return st


def _mut_forward_scale(X, W, g1, g2, n_seq, H, store=D._ident):  # scores without 1/sqrt(d)
    Wq = {n: np.asarray(w, F64) for n, w in W.items()}
    Wq["q"] = Wq["q"] * np.sqrt(X.shape[1] // H)
    return D._orig_decoder_forward(X, Wq, g1, g2, n_seq, H, store)


def _mut_forward_residual(X, W, g1, g2, n_seq, H, store=D._ident):  # second residual dropped
    f = D._orig_decoder_forward(X, W, g1, g2, n_seq, H, store)
    f["Y"] = f["Y"] - f["R"]
    return f


MUTATIONS = [("rope", _mut_rope_sign), ("rope", _mut_rope_halves), ("causal_softmax", _mut_mask),
             ("rmsnorm_bwd", _mut_rms_bwd), ("rmsnorm", _mut_rmsnorm), ("decoder_step", _mut_step_softmax_bwd),
             ("decoder_forward", _mut_forward_scale), ("decoder_forward", _mut_forward_residual)]


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
        except Exception:
            failed.append(pin.__name__ + "!")
    assert failed, f"planted mistake in {name} passed every pin"
