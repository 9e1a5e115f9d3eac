"""Block-level reconstruction of a Transformer block's MLP module on the
device (Algorithm 1 with f = the SiLU-gated MLP: G = X W_g^T, U = X W_u^T,
H = silu(G) * U, Y = H W_d^T; loss ||Y(X; W) - Y(X; What)||_F^2, with
backpropagation to all three quantized matrices).

Every arithmetic step runs in libuniquan.so; torch only allocates device
memory.  Activations are kept transposed ([I, T]: one row per hidden unit),
so every product is an NT contraction with K contiguous in both operands:

    Gt = What_g X^T, Ut = What_u X^T          (uniquan_gemm_nt)
    Ht = silu(Gt) * Ut                          (uniquan_silu_mul_fwd)
    H = Ht^T                                    (uniquan_transpose_bf16)
    Et = What_d H^T - Yt_ref, loss, dL/dWhat_d = 2 Et Ht^T   (uniquan_layer_recon)
    dHt = 2 What_d^T Et  (= 2 (What_d^T)(E^T)^T)          (uniquan_gemm_nt)
    dGt, dUt = silu backward                    (uniquan_silu_mul_bwd)
    dL/dWhat_g = dGt X, dL/dWhat_u = dUt X      (uniquan_gemm_nt with Xt)

then the straight-through backward with the SGD update per matrix.  The
target Yt_ref comes from the same kernels on the full-precision weights.
"""
from __future__ import annotations

import numpy as np
import torch

from . import uniquan as uq
from .layer import to_dev


class QuantMatrix:
    """Quantizer state of one weight matrix W [R, C]: Theta_{I_F}, codes,
    the quantized weights What (bf16) and dL/dWhat (bf16)."""

    def __init__(self, W, s, k, g, delta=None, z_u=None, s_r=None, z_b=None, alpha=None, device="cuda"):
        R, C = W.shape
        self.R, self.C, self.k, self.g = R, C, k, g
        Gn = R * C // g
        self.Gn = Gn
        self.W = to_dev(W, torch.bfloat16, device)
        self.s = to_dev(s, torch.float32, device)
        self.delta = to_dev(np.ones(Gn, np.float32) if delta is None else delta, torch.float32, device)
        self.z_u = to_dev(np.zeros(Gn, np.float32) if z_u is None else z_u, torch.float32, device)
        self.s_r = to_dev(np.ones(R, np.float32) if s_r is None else s_r, torch.float32, device)
        self.z_b = to_dev(np.zeros(Gn, np.float32) if z_b is None else z_b, torch.float32, device)
        self.alpha = (torch.zeros(Gn * k, dtype=torch.float32, device=device) if alpha is None
                      else to_dev(np.asarray(alpha).reshape(-1), torch.float32, device))
        self.codes = torch.zeros(R * C, dtype=torch.uint8, device=device)
        self.W_hat = torch.empty(R, C, dtype=torch.bfloat16, device=device)
        self.G = torch.empty(R, C, dtype=torch.bfloat16, device=device)
        self.grad_s = torch.empty(R, C, dtype=torch.float32, device=device)
        self.grad_alpha = torch.empty(Gn * k, dtype=torch.float32, device=device)
        self.grad_z_b = torch.empty(Gn, dtype=torch.float32, device=device)

    def init_unified(self, grid_G=30, alt_T=15, clip=0):
        uq.uniquan_init_unified(self.R, self.C, self.k, self.g, self.W, grid_G, alt_T, clip, self.delta,
                                self.z_u, self.alpha, self.z_b, self.codes, None, self.s, self.s_r)

    def fq_fwd(self, mode):
        uq.uniquan_fq_fwd(self.R, self.C, self.k, self.g, self.W, self.s, self.s_r, self.delta, self.z_u,
                          self.alpha, self.z_b, mode, self.codes, self.W_hat)

    def fq_bwd_sgd(self, lr_f, lr_b, keep_grads=False):
        gs, ga, gz = (self.grad_s, self.grad_alpha, self.grad_z_b) if keep_grads else (None, None, None)
        uq.uniquan_fq_bwd_sgd(self.R, self.C, self.k, self.g, self.W, self.s, self.s_r, self.delta, self.z_u,
                              self.alpha, self.z_b, self.codes, self.G, gs, ga, gz, lr_f, lr_b)


class MLPBlock:
    """The MLP module of one block: gate/up [I, C], down [C, I], activations
    X [T, C] (the block's input, the same for the full-precision and the
    quantized module in a single-block reconstruction)."""

    def __init__(self, X, gate: QuantMatrix, up: QuantMatrix, down: QuantMatrix, device="cuda"):
        T, C = X.shape
        I = gate.R
        assert gate.C == C and up.R == I and up.C == C and down.R == C and down.C == I
        self.T, self.C, self.I = T, C, I
        self.gate, self.up, self.down = gate, up, down
        bf = dict(dtype=torch.bfloat16, device=device)
        self.X = to_dev(X, torch.bfloat16, device)
        self.Xt = torch.empty(C, T, **bf)
        self.Gt, self.Ut, self.Ht = (torch.empty(I, T, **bf) for _ in range(3))
        self.H = torch.empty(T, I, **bf)
        self.Yt_ref = torch.empty(C, T, dtype=torch.float32, device=device)
        self.Et = torch.empty(C, T, **bf)
        self.E = torch.empty(T, C, **bf)
        self.WdT = torch.empty(I, C, **bf)
        self.dHt, self.dGt, self.dUt = (torch.empty(I, T, **bf) for _ in range(3))
        self.partials = torch.empty(max(1, uq.uniquan_recon_ws(T, C, I)), dtype=torch.float32, device=device)
        self.loss = torch.zeros(1, dtype=torch.float32, device=device)

    def _forward_h(self, Wg, Wu):
        T, C, I = self.T, self.C, self.I
        uq.uniquan_gemm_nt(I, T, C, Wg, self.X, self.Gt)
        uq.uniquan_gemm_nt(I, T, C, Wu, self.X, self.Ut)
        uq.uniquan_silu_mul_fwd(self.Gt, self.Ut, self.Ht)
        uq.uniquan_transpose_bf16(I, T, self.Ht, self.H)

    def prepare(self):
        """Xt and the full-precision module's output Yt_ref [C, T] (fp32),
        once per block."""
        uq.uniquan_transpose_bf16(self.T, self.C, self.X, self.Xt)
        self._forward_h(self.gate.W, self.up.W)
        uq.uniquan_layer_target(self.T, self.C, self.I, self.H, self.down.W, self.Yt_ref)

    def forward_backward(self, mode):
        """Quantize the three matrices, the module's forward on What, the loss
        and dL/dWhat for each matrix (left in each QuantMatrix.G)."""
        T, C, I = self.T, self.C, self.I
        for q in (self.gate, self.up, self.down):
            q.fq_fwd(mode)
        self._forward_h(self.gate.W_hat, self.up.W_hat)
        uq.uniquan_layer_recon(T, C, I, self.H, self.Ht, self.down.W_hat, self.Yt_ref, self.loss, self.Et,
                               self.partials, self.down.G)
        uq.uniquan_transpose_bf16(C, T, self.Et, self.E)
        uq.uniquan_transpose_bf16(C, I, self.down.W_hat, self.WdT)
        uq.uniquan_gemm_nt(I, T, C, self.WdT, self.E, self.dHt, 2.0)
        uq.uniquan_silu_mul_bwd(self.dHt, self.Gt, self.Ut, self.dGt, self.dUt)
        uq.uniquan_gemm_nt(I, C, T, self.dGt, self.Xt, self.gate.G)
        uq.uniquan_gemm_nt(I, C, T, self.dUt, self.Xt, self.up.G)

    def step(self, mode=uq.MAP_FULL, lr_f=0.005, lr_b=0.0005, keep_grads=False):
        self.forward_backward(mode)
        for q in (self.gate, self.up, self.down):
            q.fq_bwd_sgd(lr_f, lr_b, keep_grads)
