"""Pins of the block-level MLP oracle (oracle/block_mlp.py) to facts outside
it: silu's closed forms and numerical derivative, central finite
differences of the block loss for every weight gradient, an explicit
triple-loop evaluation of the module on a tiny case, the zero-loss fixed
point, and where the storage hook applies.  Planted mistakes must each fail
one of them.
"""
import numpy as np
import pytest

import oracle.block_mlp as B
import oracle.uniquan as U

F64 = np.float64


def tiny(seed, T=3, C=4, I=5):
    rs = np.random.default_rng(seed)
    X = rs.standard_normal((T, C))
    W = [rs.standard_normal((I, C)) * 0.7, rs.standard_normal((I, C)) * 0.7, rs.standard_normal((C, I)) * 0.7]
    Y_ref = rs.standard_normal((T, C))
    return X, W, Y_ref


def pin_silu():
    x = np.linspace(-30, 30, 601)
    assert B.silu(0.0) == 0.0
    assert np.allclose(B.silu(x), x / (1.0 + np.exp(-x)), rtol=1e-14, atol=1e-300)
    assert abs(B.silu(40.0) - 40.0) < 1e-12 and abs(B.silu(-40.0)) < 1e-12
    h = 1e-6
    num = (B.silu(x + h) - B.silu(x - h)) / (2 * h)
    assert np.allclose(B.dsilu(x), num, rtol=1e-7, atol=1e-9)
    assert abs(B.dsilu(0.0) - 0.5) < 1e-15


def pin_gradients_finite_differences():
    X, (Wg, Wu, Wd), Y_ref = tiny(1)
    st = B.block_step(X, Y_ref, Wg, Wu, Wd)
    h = 1e-6
    for name, W, grad in (("g", Wg, st["dWg"]), ("u", Wu, st["dWu"]), ("d", Wd, st["dWd"])):
        num = np.zeros_like(W)
        for idx in np.ndindex(W.shape):
            Wp, Wm = W.copy(), W.copy()
            Wp[idx] += h
            Wm[idx] -= h
            args_p = dict(g=(Wp, Wu, Wd), u=(Wg, Wp, Wd), d=(Wg, Wu, Wp))[name]
            args_m = dict(g=(Wm, Wu, Wd), u=(Wg, Wm, Wd), d=(Wg, Wu, Wm))[name]
            num[idx] = (B.block_step(X, Y_ref, *args_p)["loss"] - B.block_step(X, Y_ref, *args_m)["loss"]) / (2 * h)
        assert np.allclose(grad, num, rtol=1e-6, atol=1e-7), (name, np.max(np.abs(grad - num)))


def pin_forward_loops():
    X, (Wg, Wu, Wd), _ = tiny(2)
    T, C = X.shape
    I = Wg.shape[0]
    f = B.mlp_forward(X, Wg, Wu, Wd)
    for t in range(T):
        h = []
        for i in range(I):
            g = sum(X[t, c] * Wg[i, c] for c in range(C))
            u = sum(X[t, c] * Wu[i, c] for c in range(C))
            h.append(g / (1.0 + np.exp(-g)) * u)
        for c in range(C):
            y = sum(h[i] * Wd[c, i] for i in range(I))
            assert abs(f["Y"][t, c] - y) <= 1e-12 * max(1.0, abs(y))


def pin_zero_loss():
    X, (Wg, Wu, Wd), _ = tiny(3)
    Y = B.mlp_forward(X, Wg, Wu, Wd)["Y"]
    st = B.block_step(X, Y, Wg, Wu, Wd)
    assert st["loss"] == 0.0
    for k in ("dWg", "dWu", "dWd"):
        assert np.all(st[k] == 0.0)


def pin_store_hook():
    X, (Wg, Wu, Wd), Y_ref = tiny(4, T=8, C=16, I=24)
    st = B.block_step(X, Y_ref, Wg, Wu, Wd, store=U.bf16_rne)
    for k in ("G", "U", "H", "E", "dH", "dG", "dU"):
        v = np.asarray(st[k], F64)
        assert np.array_equal(v, U.bf16_rne(v.astype(np.float32)).astype(F64)), k
    # with the identity the same step is the plain definition
    plain = B.block_step(X, Y_ref, Wg, Wu, Wd)
    assert plain["loss"] == st["loss"] or abs(plain["loss"] - st["loss"]) <= 1e-2 * plain["loss"]


PINS = [pin_silu, pin_gradients_finite_differences, pin_forward_loops, pin_zero_loss, pin_store_hook]


@pytest.mark.parametrize("pin", PINS, ids=[p.__name__ for p in PINS])
def test_pin(pin):
    pin()


def _mut_dsilu(x):                       # the x (1 - sigma) term dropped
    return B.sigmoid(x)


def _mut_silu(x):                        # sigma instead of x sigma
    return B.sigmoid(x)


def _mut_sigmoid(x):                     # logistic of -x
    return B._orig_sigmoid(-np.asarray(x, F64))


def _mut_block(Xhat, Y_ref, Wg_hat, Wu_hat, Wd_hat, store=B._ident):   # dU with silu' instead of silu
    st = B._orig_block_step(Xhat, Y_ref, Wg_hat, Wu_hat, Wd_hat, store)
    dU = st["dH"] * B.dsilu(st["G"])
    st["dWu"] = dU.T @ np.asarray(Xhat, F64)
    return st


def _mut_block_factor(Xhat, Y_ref, Wg_hat, Wu_hat, Wd_hat, store=B._ident):  # dY = E (factor 2 lost)
    st = B._orig_block_step(Xhat, Y_ref, Wg_hat, Wu_hat, Wd_hat, store)
    for k in ("dWd", "dWg", "dWu"):
        st[k] = st[k] / 2.0
    return st


def _mut_forward(X, Wg, Wu, Wd, store=B._ident):   # gate and up swapped inside silu
    f = B._orig_mlp_forward(X, Wu, Wg, Wd, store)
    return f


MUTATIONS = [("dsilu", _mut_dsilu), ("silu", _mut_silu), ("sigmoid", _mut_sigmoid), ("block_step", _mut_block),
             ("block_step", _mut_block_factor), ("mlp_forward", _mut_forward)]


@pytest.mark.parametrize("name,fn", MUTATIONS, ids=[f"{m[0]}-{m[1].__name__}" for m in MUTATIONS])
def test_planted_mistake_is_caught(monkeypatch, name, fn):
    monkeypatch.setitem(B.__dict__, "_orig_" + name, getattr(B, name))
    monkeypatch.setattr(B, name, fn)
    failed = []
    for pin in PINS:
        try:
            pin()
        except AssertionError:
            failed.append(pin.__name__)
        except Exception:
            failed.append(pin.__name__ + "!")
    assert failed, f"planted mistake in {name} passed every pin"
