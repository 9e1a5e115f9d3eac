"""CPU oracle for block-level reconstruction of a Transformer block's MLP
module (Algorithm 1: the loss is the squared Frobenius distance between the
block's output with full-precision and with quantized weights, and
backpropagation reaches every quantized matrix of the block).

TEST INFRASTRUCTURE, under the same rules as ``oracle.uniquan``: only
``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import it, and it imports nothing from the HIP library.

The module is the SiLU-gated MLP of the Mistral / Llama blocks the paper
quantizes: with activations X [T, C] and weights W_g, W_u [I, C], W_d [C, I],

    G = X W_g^T,  U = X W_u^T,  H = silu(G) * U,  Y = H W_d^T,
    silu(x) = x / (1 + exp(-x)).

For the loss L = ||Y(X; W) - Y(Xhat; What)||_F^2 the gradients are, with
E = Yhat - Y and dY = 2 E,

    dL/dWhat_d = dY^T H,   dH = dY What_d,
    dG = dH * U * silu'(G),   dU = dH * silu(G),
    dL/dWhat_g = dG^T Xhat,   dL/dWhat_u = dU^T Xhat,
    silu'(x) = sigma(x) (1 + x (1 - sigma(x))).

Everything is float64.  ``store`` is applied to each intermediate the device
keeps in memory (G, U, H, E, dH, dG, dU); the identity gives the plain
definition, ``oracle.uniquan.bf16_rne`` mirrors a device that stores them
in bf16.
"""
from __future__ import annotations

import numpy as np

F64 = np.float64


def sigmoid(x):
    """1 / (1 + exp(-x)), evaluated without cancellation on either side."""
    x = np.asarray(x, F64)
    e = np.exp(-np.abs(x))
    return np.where(x >= 0, 1.0 / (1.0 + e), e / (1.0 + e))


def silu(x):
    x = np.asarray(x, F64)
    return x * sigmoid(x)


def dsilu(x):
    x = np.asarray(x, F64)
    s = sigmoid(x)
    return s * (1.0 + x * (1.0 - s))


def _ident(x):
    return np.asarray(x, F64)


def mlp_forward(X, Wg, Wu, Wd, store=_ident):
    """G, U, H, Y of the MLP module (store applied to G, U and H)."""
    X = np.asarray(X, F64)
    G = store(X @ np.asarray(Wg, F64).T)
    U = store(X @ np.asarray(Wu, F64).T)
    H = store(silu(G) * U)
    Y = H @ np.asarray(Wd, F64).T
    return dict(G=G, U=U, H=H, Y=Y)


def block_step(Xhat, Y_ref, Wg_hat, Wu_hat, Wd_hat, store=_ident):
    """Loss and weight gradients of one reconstruction step of the module on
    quantized weights against the target output Y_ref [T, C]."""
    Xhat = np.asarray(Xhat, F64)
    f = mlp_forward(Xhat, Wg_hat, Wu_hat, Wd_hat, store)
    E = store(f["Y"] - np.asarray(Y_ref, F64))
    loss = float(np.sum((f["Y"] - np.asarray(Y_ref, F64)) ** 2))
    dY = 2.0 * E
    dWd = dY.T @ f["H"]
    dH = store(dY @ np.asarray(Wd_hat, F64))
    dG = store(dH * f["U"] * dsilu(f["G"]))
    dU = store(dH * silu(f["G"]))
    return dict(loss=loss, E=E, dWd=dWd, dH=dH, dG=dG, dU=dU, dWg=dG.T @ Xhat, dWu=dU.T @ Xhat, **f)
