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

    def fq_step(self, lr_f, lr_b, next_mode, stream=None):
        """The straight-through backward with the SGD update and the next
        step's forward (next_mode) in one pass: W_hat and codes for the next
        step."""
        uq.uniquan_fq_step(self.R, self.C, self.k, self.g, self.W, self.s, self.s_r, self.delta, self.z_u,
                           self.alpha, self.z_b, self.codes, self.G, lr_f, lr_b, next_mode, self.W_hat,
                           stream=stream)


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


class DecoderBlock:
    """One whole Transformer block (Algorithm 1 with f = one multi-head
    attention module and one MLP module): pre-norm, rotary causal attention
    over n_seq sequences of L = T / n_seq tokens with H query heads of
    d = C / H and n_kv key/value heads (grouped-query attention, each shared
    by H / n_kv query heads; n_kv = H by default), and the SiLU-gated MLP.
    The seven matrices are QuantMatrix objects (q, o [C, C]; k, v
    [n_kv d, C]; g, u [I, C]; d [C, I]); g1, g2 are the norms' weights (not
    trained).  The block re-seats the W_hat and G arrays of g and u as the
    two halves of stacked [2I, C] arrays (their values kept), so that the
    backpropagation reads and writes both in one product each; with
    grouped-query attention, the W_hat and G arrays of k and v likewise.

    ``prepare(X)`` computes the full-precision block's output on the
    full-precision input X (the target); ``set_input(Xhat)`` gives the
    quantized block its input (the output of the preceding quantized blocks;
    X itself for the first block).  ``step`` is one reconstruction step on
    the quantized block: fake-quant, forward on What, the loss, the
    backpropagation to all seven matrices, and the straight-through backward
    with the SGD update.  ``output()`` is the quantized block's output on
    its input, the next block's Xhat.
    """

    NAMES = ("q", "k", "v", "o", "g", "u", "d")

    def __init__(self, mats: dict, g1, g2, T, n_seq, H, n_kv=None, device="cuda"):
        q, gm = mats["q"], mats["g"]
        C, I = q.C, gm.R
        n_kv = H if n_kv is None else n_kv
        assert C % H == 0 and T % n_seq == 0 and H % n_kv == 0
        assert C // H == 128 and (T // n_seq) % 32 == 0, "the fused attention takes d = 128 and L % 32 == 0"
        self.mats, self.T, self.C, self.I, self.H, self.n_seq = mats, T, C, I, H, n_seq
        # backward: independent products in pairs on two streams.  Off: on the 7B
        # block the concurrent products slow each other down (11.5 against
        # 9.9-10.1 ms per step)
        self.pair_streams = False
        self.d, self.L = C // H, T // n_seq
        self.Hkv, self.grp = n_kv, H // n_kv
        self.Ckv = n_kv * self.d
        assert mats["k"].R == self.Ckv and mats["v"].R == self.Ckv
        self.B = H * n_seq
        self.Bkv = n_kv * n_seq
        T, L, d, B, Ckv, Bkv = self.T, self.L, self.d, self.B, self.Ckv, self.Bkv
        f32 = dict(dtype=torch.float32, device=device)
        b16 = dict(dtype=torch.bfloat16, device=device)
        e = torch.empty
        self.g1 = to_dev(g1, torch.float32, device)
        self.g2 = to_dev(g2, torch.float32, device)
        self.Xhat, self.Yref, self.R, self.M32, self.Yhat = (e(T, C, **f32) for _ in range(5))
        self.Qf, self.dZa = (e(T, C, **f32) for _ in range(2))
        self.Kf = e(T, Ckv, **f32)
        self.r1, self.r2 = e(T, **f32), e(T, **f32)
        (self.Z1, self.O, self.Z2, self.E, self.dA, self.dO, self.dQ) = (e(T, C, **b16) for _ in range(7))
        self.Vb = e(T, Ckv, **b16)
        if self.grp > 1:
            # grouped-query: the key and value gradients side by side in one
            # [T, 2 Ckv] array and What_k; What_v and dL/dWhat_k; dL/dWhat_v
            # stacked [2 Ckv, C], so that their projection and their weight
            # gradients are one product each that fills the GPU
            self.dKV = e(T, 2 * Ckv, **b16)
            self.dK, self.dV = self.dKV[:, :Ckv], self.dKV[:, Ckv:]
            self.What_kv = self._stack(mats["k"], mats["v"], "W_hat")
            self.G_kv = self._stack(mats["k"], mats["v"], "G")
        else:
            self.dK, self.dV = (e(T, Ckv, **b16) for _ in range(2))
        # query heads in grouped slot order (see uniquan_rope_split), key/value heads plain
        self.Qh = e(B, L, d, **b16)
        # key heads then value heads in one array: one stacked projection
        # [W_k; W_v] writes both (keys rotated) where it fills the GPU
        self.KVh = e(2 * Bkv, L, d, **b16)
        self.Kh, self.Vh = self.KVh[:Bkv], self.KVh[Bkv:]
        # attention rows: base-2 log-sum-exp of the scores, the softmax backward's row term
        self.lse, self.delta = e(B, L, **f32), e(B, L, **f32)
        # cos and sin of every rotary angle of a sequence, for the projections'
        # head split and the attention gradients' inverse rotation
        self.rope_cs = e(L, d // 2, 2, **f32)
        uq.uniquan_rope_table(L, d, self.rope_cs)
        # grouped-query: dK, dV contributions per query head (summed per key/value head)
        self.dKp, self.dVp = (e(B, L, d, **f32) for _ in range(2)) if self.grp > 1 else (None, None)
        # MLP activations, one row per token; the gradients of G and U side by
        # side in one [T, 2I] array, and W_g, W_u (their What and dL/dWhat)
        # stacked in [2I, C] arrays, so that dL/dW_g; dL/dW_u = [dG dU]^T Z2
        # and dZ2 = [dG dU] [W_g; W_u] are one product each (K = 2I for dZ2)
        self.Gm, self.Um, self.Hm = (e(T, I, **b16) for _ in range(3))
        self.dGU = e(T, 2 * I, **b16)
        self.dGm, self.dUm = self.dGU[:, :I], self.dGU[:, I:]
        self.What_gu = self._stack(mats["g"], mats["u"], "W_hat")
        self.G_gu = self._stack(mats["g"], mats["u"], "G")
        self.partials_out = e(max(1, uq.uniquan_gemm_block_loss_ws(T, C)), **f32)
        self.loss = torch.zeros(1, **f32)
        self._rinv_tmp = e(T, **f32)
        self._z_tmp = e(T, C, **b16)

    @staticmethod
    def _stack(a, b, attr):
        """One [Ra + Rb, C] array holding a.attr then b.attr (their current
        values); both matrices' attr become row views of it."""
        x, y = getattr(a, attr), getattr(b, attr)
        st = torch.empty(x.shape[0] + y.shape[0], x.shape[1], dtype=x.dtype, device=x.device)
        st[:x.shape[0]].copy_(x)
        st[x.shape[0]:].copy_(y)
        setattr(a, attr, st[:x.shape[0]])
        setattr(b, attr, st[x.shape[0]:])
        return st

    # ---- forward on weights W (dict of bf16 [R, C] tensors) and fp32 input X
    def _forward(self, W, X, loss=False):
        """The block on X with weights W; with loss, the output product forms E
        and the loss against Yref in its store (M is not written)."""
        T, C, I, H, d, L, B = self.T, self.C, self.I, self.H, self.d, self.L, self.B
        sc = 1.0 / float(d) ** 0.5
        uq.uniquan_add_rmsnorm(T, C, X, None, self.g1, None, self.Z1, self.r1)
        Hkv, Ckv, Bkv, grp = self.Hkv, self.Ckv, self.Bkv, self.grp
        self._project_heads(W["q"], H, self.Qh, grp, True, self.Qf)
        Wkv = self._stacked_kv(W)
        if Wkv is not None:
            uq.uniquan_gemm_heads(T, 2 * Hkv, C, self.Z1, Wkv, L, self.KVh, cs=self.rope_cs, n_rot=Hkv)
        else:
            self._project_heads(W["k"], Hkv, self.Kh, 1, True, self.Kf)
            self._project_heads(W["v"], Hkv, self.Vh, 1, False, self.Vb)
        # causal attention with the score tiles on chip (query batch g Bkv + c uses key/value batch c)
        # (O written token-major: the merge of the heads is in the kernel's store)
        uq.uniquan_attn_fwd(B, Bkv, L, d, self.Qh, self.Kh, self.Vh, sc, self.O, self.lse,
                            tok_seqs=self.n_seq, group=grp)
        # R = X + O W_o^T in the product's store, then the second norm of R
        uq.uniquan_gemm_nt_residual(T, C, C, self.O, W["o"], X, self.R)
        uq.uniquan_add_rmsnorm(T, C, self.R, None, self.g2, None, self.Z2, self.r2)
        uq.uniquan_gemm_swiglu(T, I, C, self.Z2, W["g"], W["u"], self.Gm, self.Um, self.Hm)
        if loss:
            uq.uniquan_gemm_block_loss(T, C, I, self.Hm, W["d"], self.R, self.Yref, self.E, self.partials_out,
                                       self.loss)
        else:
            uq.uniquan_gemm_nt(T, C, I, self.Hm, W["d"], self.M32)

    def _stacked_kv(self, W):
        """[W_k; W_v] as one [2 Ckv, C] array when W's key and value weights are
        the stacked What (grouped-query) and the stacked product fills the GPU
        with 256 x 256 tiles, else None (two products)."""
        if self.grp == 1 or ((self.T + 255) // 256) * ((2 * self.Ckv + 255) // 256) < 256:
            return None
        kv = self.What_kv
        if W["k"].data_ptr() != kv.data_ptr() or W["v"].data_ptr() != kv[self.Ckv].data_ptr():
            return None
        return kv

    def _project_heads(self, Wm, n_heads, out, group, rotate, tmp):
        """out [n_heads, T, d] = the head split (rotated when rotate) of Z1 Wm^T:
        in the product's store where the product fills the GPU with 256 x 256
        tiles, else a product into tmp followed by the stand-alone split (the
        same values)."""
        T, C, d, L = self.T, self.C, self.d, self.L
        N = n_heads * d
        if ((T + 255) // 256) * ((N + 255) // 256) >= 256:
            uq.uniquan_gemm_heads(T, n_heads, C, self.Z1, Wm, L, out, group=group, rotate=rotate, cs=self.rope_cs)
        else:
            uq.uniquan_gemm_nt(T, N, C, self.Z1, Wm, tmp)
            uq.uniquan_rope_split(T, n_heads, d, L, tmp, out, rotate=rotate, group=group)

    def _sum_out(self, out):
        """out = R + M (fp32), through the residual-add path of the norm kernel."""
        uq.uniquan_add_rmsnorm(self.T, self.C, self.R, self.M32, self.g2, out, self._z_tmp, self._rinv_tmp)

    def prepare(self, X):
        """Target: the full-precision block's output on the full-precision input X [T, C]."""
        Xd = X if isinstance(X, torch.Tensor) else to_dev(X, torch.float32)
        self._forward({n: m.W for n, m in self.mats.items()}, Xd.float().contiguous())
        self._sum_out(self.Yref)

    def set_input(self, Xhat):
        Xd = Xhat if isinstance(Xhat, torch.Tensor) else to_dev(Xhat, torch.float32)
        self.Xhat.copy_(Xd.float())

    def quantize(self, mode):
        for q in self.mats.values():
            q.fq_fwd(mode)

    def forward(self):
        """The quantized block on Xhat with the current What, and the loss: E and
        L = ||f(Xhat; What) - Yref||^2 come from the output product's store."""
        self._forward({n: q.W_hat for n, q in self.mats.items()}, self.Xhat, loss=True)

    def compute_loss(self):
        """The loss is formed by forward(); kept as a step phase (no work)."""

    def forward_backward(self, mode):
        """Quantize, forward, loss and dL/dWhat of all seven matrices (left
        in each QuantMatrix.G)."""
        self.quantize(mode)
        self.forward()
        self.compute_loss()
        self.backward()

    def backward(self, done=None):
        """Backpropagation from E to dL/dWhat of the seven matrices.  done(n),
        if given, is called as soon as matrix n's gradient is final and its
        What is read no more in this step."""
        T, C, I, H, d, L, B = self.T, self.C, self.I, self.H, self.d, self.L, self.B
        sc = 1.0 / float(d) ** 0.5
        m = self.mats
        Wh = {n: q.W_hat for n, q in m.items()}
        done = done or (lambda n: None)
        # Independent products run in pairs, one on a second stream, so that
        # the last partial round of tiles of one fills with the other's tiles.
        main = torch.cuda.current_stream()
        ps = None
        if self.pair_streams:
            if getattr(self, "_pair", None) is None:
                self._pair = torch.cuda.Stream()
            ps = self._pair

        def fork():
            if ps is not None:
                uq.wait_stream(ps, main)

        def join():
            if ps is not None:
                uq.wait_stream(main, ps)

        # MLP module (dY = 2 E).  Weight gradients dY^T X read dY and X as
        # stored (both K-slow, K = tokens); input gradients dY W read W as
        # stored (K-slow, K = the matrix's rows).
        fork()
        uq.uniquan_gemm(C, I, T, self.E, 1, self.Hm, 1, m["d"].G, 2.0)
        uq.uniquan_gemm_silu_bwd(T, I, C, self.E, Wh["d"], 2.0, self.Gm, self.Um, self.dGm, self.dUm, stream=ps,
                                 ld_d=2 * I)
        join()
        done("d")
        # gate and up together: [dG dU] is [T, 2I], What_g; What_u and their
        # gradients are stacked [2I, C]
        for n, off in (("g", 0), ("u", I)):
            assert m[n].W_hat.data_ptr() == self.What_gu[off].data_ptr() and \
                m[n].G.data_ptr() == self.G_gu[off].data_ptr(), "What / G of gate and up must stay stacked"
        uq.uniquan_gemm(2 * I, C, T, self.dGU, 1, self.Z2, 1, self.G_gu)
        uq.uniquan_gemm(T, C, 2 * I, self.dGU, 0, self.What_gu, 1, self.dZa)
        done("g")
        done("u")
        # second norm and residual: dR = 2 E + RMSNorm backward
        uq.uniquan_rmsnorm_bwd(T, C, self.dZa, None, self.R, self.g2, self.r2, self.E, 2.0, self.dA)
        # attention module
        fork()
        uq.uniquan_gemm(C, C, T, self.dA, 1, self.O, 1, m["o"].G)
        uq.uniquan_gemm(T, C, C, self.dA, 0, Wh["o"], 1, self.dO, stream=ps)
        join()
        done("o")
        Hkv, Ckv, Bkv, grp = self.Hkv, self.Ckv, self.Bkv, self.grp
        # O and dO token-major; dQ (and dK, dV with one query head per key/value
        # head) written token-major and inverse-rotated by the kernels' stores
        if grp == 1:
            uq.uniquan_attn_bwd(B, Bkv, L, d, self.Qh, self.Kh, self.Vh, self.O, self.dO, self.lse, sc, self.delta,
                                self.dQ, self.dK, self.dV, tok_seqs=self.n_seq, group=grp, cs=self.rope_cs)
        else:
            uq.uniquan_attn_bwd(B, Bkv, L, d, self.Qh, self.Kh, self.Vh, self.O, self.dO, self.lse, sc, self.delta,
                                self.dQ, self.dKp, self.dVp, tok_seqs=self.n_seq, group=grp, cs=self.rope_cs)
            uq.uniquan_rope_merge(T, Hkv, d, L, self.dKp, self.dK, rotate=True, nsum=grp, ld_out=2 * Ckv)
            uq.uniquan_rope_merge(T, Hkv, d, L, self.dVp, self.dV, rotate=False, nsum=grp, ld_out=2 * Ckv)
        uq.uniquan_gemm(C, C, T, self.dQ, 1, self.Z1, 1, m["q"].G)
        done("q")
        if grp > 1:
            for n, off in (("k", 0), ("v", Ckv)):
                assert m[n].G.data_ptr() == self.G_kv[off].data_ptr(), "dL/dWhat of k and v must stay stacked"
            uq.uniquan_gemm(2 * Ckv, C, T, self.dKV, 1, self.Z1, 1, self.G_kv)
        else:
            uq.uniquan_gemm(Ckv, C, T, self.dK, 1, self.Z1, 1, m["k"].G)
            uq.uniquan_gemm(Ckv, C, T, self.dV, 1, self.Z1, 1, m["v"].G)
        done("k")
        done("v")

    def update(self, lr_f=0.005, lr_b=0.0005, keep_grads=False):
        """Straight-through backward with the SGD update of every matrix."""
        for q in self.mats.values():
            q.fq_bwd_sgd(lr_f, lr_b, keep_grads)

    def step(self, mode=uq.MAP_FULL, lr_f=0.005, lr_b=0.0005, keep_grads=False):
        self.forward_backward(mode)
        self.update(lr_f, lr_b, keep_grads)

    def step_fused(self, next_mode=uq.MAP_LOCAL, lr_f=0.005, lr_b=0.0005, overlap=False):
        """One step in the fused form: the block's forward on the current
        What (left by quantize() or by the previous fused step), the loss,
        backpropagation, then per matrix the straight-through backward with
        SGD fused with the next step's forward (next_mode).  The same
        sequence of operations as step() across steps; each matrix's What is
        read once less and written once instead of twice.

        With overlap, each matrix's fused quantizer pass runs on a second
        stream as soon as its gradient is final and the backpropagation no
        longer reads its What; the current stream waits for them before the
        step returns, so the next step sees every What.  Off by default: on
        the 7B block the quantizer's workgroups take compute units that the
        products' next tiles wait for, and the step gets slower (11.9
        against 10.6 ms with 32 key/value heads, no change with 8)."""
        self.forward()
        self.compute_loss()
        if not overlap:
            self.backward()
            for q in self.mats.values():
                q.fq_step(lr_f, lr_b, next_mode)
            return
        main = torch.cuda.current_stream()
        if getattr(self, "_side", None) is None:
            self._side = torch.cuda.Stream()
        side = self._side

        def done(n):
            uq.wait_stream(side, main)
            self.mats[n].fq_step(lr_f, lr_b, next_mode, stream=side)

        self.backward(done)
        uq.wait_stream(main, side)

    def flops_per_step(self):
        """GEMM flops of one step: the seven projections forward and their
        weight gradients, the input gradients through the MLP and the output
        projection, and the attention products forward and backward (the
        causal half of each [L, L] product that is never computed is not
        counted)."""
        T, C, I, L, d, B = self.T, self.C, self.I, self.L, self.d, self.B
        lin = 2.0 * T * C * C * 2 + 2.0 * T * self.Ckv * C * 2 + 2.0 * T * C * I * 3
        attn = 2.0 * B * (L * (L + 1) / 2) * d
        return 2 * lin + 3 * (2.0 * T * C * I) + 2.0 * T * C * C + 6 * attn

    def output(self):
        """The quantized block's output on its input (fp32 [T, C]): the next
        block's Xhat.  The weights are the finished quantization's, i.e. the
        canonical FULL mapping with the current parameters (what the fold of
        Theorem 1 stores), so this ends the block's optimisation."""
        for q in self.mats.values():
            q.fq_fwd(uq.MAP_FULL)
        self._forward({n: q.W_hat for n, q in self.mats.items()}, self.Xhat)
        self._sum_out(self.Yhat)
        return self.Yhat
