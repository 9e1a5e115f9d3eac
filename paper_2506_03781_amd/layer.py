"""One linear layer's UniQuan_F optimisation state on the device, stepped
through the C ABI (Algorithm 1, inner loop, for a single linear layer).

Every arithmetic step runs in libuniquan.so; torch only allocates device
memory and provides the stream.
"""
from __future__ import annotations

import numpy as np
import torch

from . import uniquan as uq


def to_dev(a: np.ndarray, dtype=torch.float32, device="cuda") -> torch.Tensor:
    t = torch.from_numpy(np.ascontiguousarray(a))
    return t.to(device=device, dtype=dtype).contiguous()


class QuantLayer:
    """Device tensors of one matrix: W [R, C], X [T, C] and Theta_{I_F}.

    Theta_{I_F} comes from ``init_unified`` (the paper's initialisation), or
    Delta, z_U, s_r, z_B are set by the caller and alpha comes from
    ``init_greedy``.
    """

    def __init__(self, W, X, s, k, g, w_dtype=torch.bfloat16, device="cuda",
                 delta=None, z_u=None, s_r=None, z_b=None, grad_dtype=torch.bfloat16, residual=False):
        R, C = W.shape
        T = X.shape[0]
        # residual: W_hat holds What - W and the loss needs no target (Yt unused)
        self.residual = residual
        self.R, self.C, self.T, self.k, self.g = R, C, T, k, g
        Gn = R * C // g
        self.Gn = Gn
        dev = device
        self.W = to_dev(W, w_dtype, dev)
        self.W_bf16 = self.W if w_dtype == torch.bfloat16 else self.W.to(torch.bfloat16)
        self.X = to_dev(X, torch.bfloat16, dev)
        self.s = to_dev(s, torch.float32, dev)
        self.delta = to_dev(np.ones(Gn, np.float32) if delta is None else delta, torch.float32, dev)
        self.z_u = to_dev(np.zeros(Gn, np.float32) if z_u is None else z_u, torch.float32, dev)
        self.s_r = to_dev(np.ones(R, np.float32) if s_r is None else s_r, torch.float32, dev)
        self.z_b = to_dev(np.zeros(Gn, np.float32) if z_b is None else z_b, torch.float32, dev)
        self.alpha = torch.zeros(Gn * k, dtype=torch.float32, device=dev)
        self.codes = torch.zeros(R * C, dtype=torch.uint8, device=dev)
        self.W_hat = torch.empty(R, C, dtype=torch.bfloat16, device=dev)
        self.Xt = torch.empty(C, T, dtype=torch.bfloat16, device=dev)
        self.Yt = None if residual else torch.empty(R, T, dtype=torch.float32, device=dev)
        self.Et = torch.empty(R, T, dtype=torch.bfloat16, device=dev)
        self.partials = torch.empty(max(1, uq.uniquan_recon_ws(T, R, C)), dtype=torch.float32, device=dev)
        self.loss = torch.zeros(1, dtype=torch.float32, device=dev)
        self.G = torch.empty(R, C, dtype=grad_dtype, device=dev)
        self.grad_s = torch.empty(R, C, dtype=torch.float32, device=dev)
        self.grad_alpha = torch.empty(Gn * k, dtype=torch.float32, device=dev)
        self.grad_z_b = torch.empty(Gn, dtype=torch.float32, device=dev)

    def init_unified(self, grid_G=30, alt_T=15, clip=0, err=None):
        """Unified initialisation of Delta, z_U, alpha, z_B (and s = 1, s_r = 1)
        from W; the codes of the kept candidate go to ``codes``."""
        uq.uniquan_init_unified(self.R, self.C, self.k, self.g, self.W, grid_G, alt_T, clip,
                                self.delta, self.z_u, self.alpha, self.z_b, self.codes, err,
                                self.s, self.s_r)

    def init_greedy(self):
        uq.uniquan_init_greedy(self.R, self.C, self.k, self.g, self.W, self.s, self.s_r, self.delta,
                               self.z_u, self.z_b, self.alpha)

    def prepare(self):
        """Xt and (without the residual form) the fixed target Yt = W X^T, once
        per layer."""
        if self.Yt is not None:
            uq.uniquan_layer_target(self.T, self.R, self.C, self.X, self.W_bf16, self.Yt)
        uq.uniquan_transpose_bf16(self.T, self.C, self.X, self.Xt)

    def fq_fwd(self, mode=uq.MAP_FULL):
        fn = uq.uniquan_fq_fwd_residual if self.residual else uq.uniquan_fq_fwd
        fn(self.R, self.C, self.k, self.g, self.W, self.s, self.s_r, self.delta, self.z_u,
           self.alpha, self.z_b, mode, self.codes, self.W_hat)

    def recon(self, backward=True):
        uq.uniquan_layer_recon(self.T, self.R, self.C, self.X, self.Xt, self.W_hat, self.Yt, self.loss,
                               self.Et, self.partials, self.G if backward else None)

    def fq_bwd(self):
        uq.uniquan_fq_bwd(self.R, self.C, self.k, self.g, self.W, self.s, self.s_r, self.delta, self.z_u,
                          self.alpha, self.z_b, self.codes, self.G, self.grad_s, self.grad_alpha,
                          self.grad_z_b)

    def grad_ste_sgd(self, lr_f=0.005, lr_b=0.0005):
        """Weight-gradient GEMM with the straight-through backward and the SGD
        update in its epilogue (dL/dWhat stays on chip); needs Et from recon."""
        uq.uniquan_layer_grad_ste_sgd(self.T, self.R, self.C, self.k, self.g, self.Et, self.Xt, self.W, self.s,
                                      self.s_r, self.delta, self.z_u, self.alpha, self.z_b, self.codes,
                                      lr_f, lr_b)

    def fq_bwd_sgd(self, lr_f=0.005, lr_b=0.0005, keep_grads=False):
        """Backward with the SGD update of s, alpha, z_B fused into the same pass
        (gradients stored only with keep_grads)."""
        gs, ga, gz = (self.grad_s, self.grad_alpha, self.grad_z_b) if keep_grads else (None, None, None)
        uq.uniquan_fq_bwd_sgd(self.R, self.C, self.k, self.g, self.W, self.s, self.s_r, self.delta,
                              self.z_u, self.alpha, self.z_b, self.codes, self.G, gs, ga, gz, lr_f, lr_b)

    def fq_step(self, lr_f=0.005, lr_b=0.0005, next_mode=uq.MAP_LOCAL):
        """End of this step and start of the next in one pass: the backward with
        the SGD update (dL/dWhat in G, mask bits in codes), then the forward with
        next_mode on the updated parameters (W_hat and codes for the next step)."""
        uq.uniquan_fq_step(self.R, self.C, self.k, self.g, self.W, self.s, self.s_r, self.delta, self.z_u,
                           self.alpha, self.z_b, self.codes, self.G, lr_f, lr_b, next_mode, self.W_hat,
                           residual=self.residual)

    def sgd(self, lr_f=0.005, lr_b=0.0005):
        """Plain SGD with the paper's learning rates (Theta_F: s; Theta_B: alpha, z_B)."""
        uq.uniquan_sgd(self.s, self.grad_s, lr_f)
        uq.uniquan_sgd(self.alpha, self.grad_alpha, lr_b)
        uq.uniquan_sgd(self.z_b, self.grad_z_b, lr_b)

    def step(self, mode=uq.MAP_FULL, update=True):
        self.fq_fwd(mode)
        self.recon(True)
        if update:
            self.fq_bwd_sgd()
        else:
            self.fq_bwd()

    def fold(self, code_src=0):
        a = torch.empty(self.Gn * self.k, dtype=torch.float32, device=self.W.device)
        z = torch.empty(self.Gn, dtype=torch.float32, device=self.W.device)
        c = torch.empty(self.R * self.C, dtype=torch.uint8, device=self.W.device)
        uq.uniquan_fold_to_bcq(self.R, self.C, self.k, self.g, self.W, self.s, self.s_r, self.delta, self.z_u,
                               self.alpha, self.z_b, a, z, c, code_src)
        return a, z, c
