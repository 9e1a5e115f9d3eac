"""CPU oracle for block-level reconstruction of a whole Transformer block
(Algorithm 1; the block is one multi-head attention module and one MLP
module, appendix "Units in LLMs"; the loss is the squared Frobenius distance
between the outputs of the full-precision block on X and of the quantized
block on X_hat, appendix "Error Types").

TEST INFRASTRUCTURE, under the same rules as ``oracle.uniquan``: only
``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import it, and it imports nothing from the HIP library.

The paper quantizes Mistral / Llama blocks and does not write the block out.
This oracle takes the standard pre-norm form of those models (the readings
are listed with the design notes):

    Z1 = RMSNorm(X; g1)
    Q = RoPE(Z1 W_q^T)  (H heads of d = C / H),
    K = RoPE(Z1 W_k^T), V = Z1 W_v^T  (H_kv heads of d; query head h uses
    key/value head h // (H / H_kv): grouped-query attention, the form of
    the Mistral and Llama-3 blocks; H_kv = H is multi-head attention)
    P = causal softmax(Q_h K_kv(h)^T / sqrt(d)) per sequence and head
    O = concat_h(P V_h),  A = O W_o^T,  R = X + A
    Z2 = RMSNorm(R; g2),  Y = R + silu(Z2 W_g^T) * (Z2 W_u^T) W_d^T

with RMSNorm(x; g) = x / sqrt(mean(x^2) + eps) * g (eps = 1e-5) over the
hidden dimension, and the rotary embedding in its rotate-half form: for
position p (within its sequence) and i < d/2, angle p * theta^(-2i/d)
(theta = 1e4) rotates the pair (x_i, x_{i+d/2}).  The T tokens are n_seq
sequences of T / n_seq consecutive tokens; attention never crosses them.

Everything is float64.  ``store`` is applied where a device keeps a value in
bf16 (Z1, the rotated Q and K, V, P, O, Z2, G, U, H, E, and in the backward
dH, dG, dU, dA, dO, dS, dQ, dK, dV); fp32 intermediates are left exact.
"""
from __future__ import annotations

import numpy as np

from .block_mlp import dsilu, silu

F64 = np.float64
EPS = 1e-5
THETA = 1e4


def _ident(x):
    return np.asarray(x, F64)


def rmsnorm(x, gamma, eps=EPS):
    """(y, r) with y = x r gamma and r = 1 / sqrt(mean(x^2) + eps) per row."""
    x = np.asarray(x, F64)
    r = 1.0 / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps)
    return x * r * np.asarray(gamma, F64), r


def rmsnorm_bwd(dy, x, gamma, r):
    """dL/dx of y = x r gamma: r (gamma dy) - x r^3 sum(gamma dy x) / C."""
    x = np.asarray(x, F64)
    gdy = np.asarray(dy, F64) * np.asarray(gamma, F64)
    C = x.shape[-1]
    return r * gdy - x * r ** 3 * np.sum(gdy * x, axis=-1, keepdims=True) / C


def rope_angles(L, d, theta=THETA):
    """[L, d/2] angles p * theta^(-2i/d)."""
    inv = theta ** (-np.arange(0, d, 2, dtype=F64) / d)
    return np.outer(np.arange(L, dtype=F64), inv)


def rope(x, ang, inverse=False):
    """Rotate pairs (x_i, x_{i+d/2}) of x [..., L, d] by ang [L, d/2]
    (by -ang when inverse)."""
    x = np.asarray(x, F64)
    h = x.shape[-1] // 2
    c, s = np.cos(ang), np.sin(ang)
    if inverse:
        s = -s
    x1, x2 = x[..., :h], x[..., h:]
    return np.concatenate([x1 * c - x2 * s, x2 * c + x1 * s], axis=-1)


def split_heads(x, n_seq, H):
    """[T, C] -> [n_seq, H, L, d]."""
    x = np.asarray(x, F64)
    T, C = x.shape
    return x.reshape(n_seq, T // n_seq, H, C // H).transpose(0, 2, 1, 3)


def merge_heads(x):
    """[n_seq, H, L, d] -> [T, C]."""
    n, H, L, d = x.shape
    return np.asarray(x, F64).transpose(0, 2, 1, 3).reshape(n * L, H * d)


def causal_softmax(S):
    """Row softmax of S [..., L, L] over keys j <= i."""
    S = np.asarray(S, F64)
    L = S.shape[-1]
    mask = np.triu(np.ones((L, L), dtype=bool), 1)
    Sm = np.where(mask, -np.inf, S)
    Sm = Sm - np.max(Sm, axis=-1, keepdims=True)
    e = np.exp(Sm)
    return e / np.sum(e, axis=-1, keepdims=True)


def decoder_forward(X, W, g1, g2, n_seq, H, store=_ident, n_kv=None):
    """All intermediates of the block on input X [T, C] with weights
    W = dict(q, o [C, C], k, v [n_kv d, C], g, u [I, C], d [C, I])
    (n_kv key/value heads, H by default)."""
    X = np.asarray(X, F64)
    T, C = X.shape
    d = C // H
    n_kv = H if n_kv is None else n_kv
    grp = H // n_kv                      # query heads per key/value head
    ang = rope_angles(T // n_seq, d)
    Wf = {n: np.asarray(w, F64) for n, w in W.items()}
    Z1r, r1 = rmsnorm(X, g1)
    Z1 = store(Z1r)
    Qh = store(rope(split_heads(Z1 @ Wf["q"].T, n_seq, H), ang))
    Kh = store(rope(split_heads(Z1 @ Wf["k"].T, n_seq, n_kv), ang))
    Vh = store(split_heads(Z1 @ Wf["v"].T, n_seq, n_kv))
    Kx, Vx = np.repeat(Kh, grp, axis=1), np.repeat(Vh, grp, axis=1)   # head h reads key/value head h // grp
    S = Qh @ np.swapaxes(Kx, -1, -2) / np.sqrt(d)
    P = store(causal_softmax(S))
    O = store(merge_heads(P @ Vx))
    A = O @ Wf["o"].T
    R = X + A
    Z2r, r2 = rmsnorm(R, g2)
    Z2 = store(Z2r)
    G = store(Z2 @ Wf["g"].T)
    U = store(Z2 @ Wf["u"].T)
    Hm = store(silu(G) * U)
    Y = R + Hm @ Wf["d"].T
    return dict(Z1=Z1, r1=r1, Qh=Qh, Kh=Kh, Vh=Vh, Kx=Kx, Vx=Vx, S=S, P=P, O=O, A=A, R=R, Z2=Z2, r2=r2, G=G, U=U,
                H=Hm, Y=Y, ang=ang, n_kv=n_kv)


def decoder_step(Xhat, Y_ref, W, g1, g2, n_seq, H, store=_ident, n_kv=None):
    """Loss ||Y(Xhat; W) - Y_ref||_F^2 and its gradient for each of the seven
    matrices (Algorithm 1's backpropagation; the input and the norm weights
    are not trained)."""
    f = decoder_forward(Xhat, W, g1, g2, n_seq, H, store, n_kv)
    grp = H // f["n_kv"]
    Wf = {n: np.asarray(w, F64) for n, w in W.items()}
    T, C = f["R"].shape
    d = C // H
    Ef = f["Y"] - np.asarray(Y_ref, F64)
    loss = float(np.sum(Ef * Ef))
    E = store(Ef)
    dY = 2.0 * E
    # MLP module
    gd = dY.T @ f["H"]
    dHm = store(dY @ Wf["d"])
    dG = store(dHm * f["U"] * dsilu(f["G"]))
    dU = store(dHm * silu(f["G"]))
    gg = dG.T @ f["Z2"]
    gu = dU.T @ f["Z2"]
    dZ2 = dG @ Wf["g"] + dU @ Wf["u"]
    dR = dY + rmsnorm_bwd(dZ2, f["R"], g2, f["r2"])
    # attention module
    dA = store(dR)
    go = dA.T @ f["O"]
    dOh = split_heads(store(dA @ Wf["o"]), n_seq, H)
    dP = dOh @ np.swapaxes(f["Vx"], -1, -2)
    # softmax backward: dS = P (dP - delta) with the row term delta_i =
    # sum_j P_ij dP_ij written as dO_i . O_i (the same value in exact
    # arithmetic, O = P V), evaluated from the stored O
    delta = np.sum(dOh * split_heads(f["O"], n_seq, H), axis=-1, keepdims=True)
    dS = store(f["P"] * (dP - delta))
    dQh = dS @ f["Kx"] / np.sqrt(d)

    def group_sum(x):  # per query head -> per key/value head
        n, Hq, L, dd = x.shape
        return x.reshape(n, Hq // grp, grp, L, dd).sum(axis=2)
    dKh = group_sum(np.swapaxes(dS, -1, -2) @ f["Qh"] / np.sqrt(d))
    dVh = group_sum(np.swapaxes(f["P"], -1, -2) @ dOh)
    dQ = store(merge_heads(rope(dQh, f["ang"], inverse=True)))
    dK = store(merge_heads(rope(dKh, f["ang"], inverse=True)))
    dV = store(merge_heads(dVh))
    grads = dict(q=dQ.T @ f["Z1"], k=dK.T @ f["Z1"], v=dV.T @ f["Z1"], o=go, g=gg, u=gu, d=gd)
    return dict(loss=loss, E=E, grads=grads, dR=dR, dZ2=dZ2, dS=dS, dQ=dQ, dK=dK, dV=dV, **f)
