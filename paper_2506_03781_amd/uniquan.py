"""Python binding of libuniquan.so (ctypes).

Argument marshalling only: every function passes torch tensors' device
pointers, sizes and the current HIP stream to the C entry point of the same
name and raises ``UniquanError`` on a non-OK status.  All arithmetic runs in
the library's HIP kernels; there is no fallback path.  The binding also
checks what the C ABI cannot: that each tensor is a contiguous device tensor
of the expected dtype with at least the number of elements the call touches.
"""
from __future__ import annotations

import ctypes
import os
import re

import torch

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libuniquan.so")
HEADER = os.path.join(os.path.dirname(HERE), "include", "uniquan.h")

UQ_OK, UQ_EINVAL, UQ_EUNSUPPORTED, UQ_EHIP = 0, 1, 2, 3
UQ_F32, UQ_BF16 = 0, 1
MAP_FULL, MAP_LOCAL, MAP_FROZEN = 0, 1, 2

_STATUS = {UQ_EINVAL: "EINVAL", UQ_EUNSUPPORTED: "EUNSUPPORTED", UQ_EHIP: "EHIP"}


class UniquanError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{_STATUS.get(status, status)}: {msg}")
        self.status = status


_i64, _i32, _vp, _f32 = ctypes.c_int64, ctypes.c_int, ctypes.c_void_p, ctypes.c_float
_SIGS = {
    "uniquan_abi_version": ([], _i32),
    "uniquan_last_error": ([], ctypes.c_char_p),
    "uniquan_fq_fwd": ([_i64, _i64, _i32, _i32, _vp, _i32, _vp, _vp, _vp, _vp, _vp, _vp, _i32, _vp, _vp, _i32, _vp], _i32),
    "uniquan_fq_fwd_residual": ([_i64, _i64, _i32, _i32, _vp, _i32, _vp, _vp, _vp, _vp, _vp, _vp, _i32, _vp, _vp, _i32,
                                 _vp], _i32),
    "uniquan_fq_bwd": ([_i64, _i64, _i32, _i32, _vp, _i32, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _i32,
                        _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp], _i32),
    "uniquan_fq_bwd_sgd": ([_i64, _i64, _i32, _i32, _vp, _i32, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _i32,
                            _vp, _vp, _vp, _f32, _f32, _vp], _i32),
    "uniquan_fq_step": ([_i64, _i64, _i32, _i32, _vp, _i32, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _i32, _f32, _f32,
                         _i32, _vp, _i32, _i32, _vp], _i32),
    "uniquan_layer_target": ([_i64, _i64, _i64, _vp, _vp, _vp, _vp], _i32),
    "uniquan_transpose_bf16": ([_i64, _i64, _vp, _vp, _vp], _i32),
    "uniquan_recon_ws": ([_i64, _i64, _i64], ctypes.c_size_t),
    "uniquan_layer_recon": ([_i64, _i64, _i64, _vp, _vp, _vp, _vp, _vp, _vp, _vp, ctypes.c_size_t, _vp, _i32, _vp], _i32),
    "uniquan_layer_recon_noalloc": ([_i64, _i64, _i64, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _i32, _vp], _i32),
    "uniquan_recon_noalloc_max_partials": ([], ctypes.c_size_t),
    "uniquan_layer_grad": ([_i64, _i64, _i64, _vp, _vp, _vp, _i32, _vp], _i32),
    "uniquan_layer_grad_ste_sgd": ([_i64, _i64, _i64, _i32, _i32, _vp, _vp, _vp, _i32, _vp, _vp, _vp, _vp, _vp, _vp,
                                    _vp, _f32, _f32, _vp, _vp, _vp, _vp], _i32),
    "uniquan_fold_to_bcq": ([_i64, _i64, _i32, _i32, _vp, _i32, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _i32, _vp], _i32),
    "uniquan_bcq_dequant": ([_i64, _i64, _i32, _i32, _vp, _vp, _vp, _vp, _i32, _vp], _i32),
    "uniquan_init_greedy": ([_i64, _i64, _i32, _i32, _vp, _i32, _vp, _vp, _vp, _vp, _vp, _vp, _vp], _i32),
    "uniquan_init_unified": ([_i64, _i64, _i32, _i32, _vp, _i32, _i32, _i32, _i32, _vp, _vp, _vp, _vp,
                              _vp, _vp, _vp, _vp, _vp], _i32),
    "uniquan_sgd": ([_i64, _vp, _vp, _f32, _vp], _i32),
    "uniquan_bcq_pack": ([_i64, _i64, _i32, _i32, _vp, _vp, _vp, _vp, _vp, _vp, _vp], _i32),
    "uniquan_gemm_nt": ([_i64, _i64, _i64, _vp, _vp, _vp, _i32, _f32, _vp], _i32),
    "uniquan_gemm": ([_i64, _i64, _i64, _vp, _i32, _vp, _i32, _vp, _i32, _f32, _vp], _i32),
    "uniquan_rope_table": ([_i32, _i32, _vp, _vp], _i32),
    "uniquan_gemm_swiglu": ([_i64, _i64, _i64, _vp, _vp, _vp, _vp, _vp, _vp, _vp], _i32),
    "uniquan_gemm_block_loss_ws": ([_i64, _i64], ctypes.c_size_t),
    "uniquan_gemm_block_loss": ([_i64, _i64, _i64, _vp, _vp, _vp, _vp, _vp, _vp, ctypes.c_size_t, _vp, _vp], _i32),
    "uniquan_gemm_nt_residual": ([_i64, _i64, _i64, _vp, _vp, _vp, _vp, _vp], _i32),
    "uniquan_gemm_silu_bwd": ([_i64, _i64, _i64, _vp, _vp, _f32, _vp, _vp, _vp, _vp, _i64, _vp], _i32),
    "uniquan_gemm_heads": ([_i64, _i32, _i64, _vp, _vp, _i32, _i32, _i32, _vp, _vp, _vp], _i32),
    "uniquan_silu_mul_fwd": ([_i64, _vp, _vp, _vp, _vp], _i32),
    "uniquan_silu_mul_bwd": ([_i64, _vp, _vp, _vp, _vp, _vp, _vp], _i32),
    "uniquan_gemm_nt_batched": ([_i64, _i64, _i64, _i64, _vp, _i64, _vp, _i64, _vp, _i64, _i32, _f32, _i32, _vp],
                                _i32),
    "uniquan_add_rmsnorm": ([_i64, _i64, _vp, _vp, _vp, _vp, _vp, _vp, _vp], _i32),
    "uniquan_rmsnorm_bwd": ([_i64, _i64, _vp, _vp, _vp, _vp, _vp, _vp, _f32, _vp, _vp, _vp], _i32),
    "uniquan_rope_split": ([_i64, _i32, _i32, _i32, _i32, _vp, _i32, _i32, _vp, _vp], _i32),
    "uniquan_rope_merge": ([_i64, _i32, _i32, _i32, _i32, _i32, _vp, _i32, _i32, _vp, _i64, _vp], _i32),
    "uniquan_softmax_causal": ([_i64, _i32, _vp, _vp, _vp], _i32),
    "uniquan_softmax_causal_bwd": ([_i64, _i32, _vp, _vp, _vp, _vp], _i32),
    "uniquan_transpose_bf16_batched": ([_i64, _i64, _i64, _vp, _vp, _vp], _i32),
    "uniquan_block_loss_ws": ([], ctypes.c_size_t),
    "uniquan_block_loss": ([_i64, _vp, _vp, _vp, _vp, _vp, ctypes.c_size_t, _vp, _vp], _i32),
    "uniquan_attn_fwd": ([_i64, _i64, _i32, _i32, _vp, _vp, _vp, _f32, _vp, _vp, _i32, _i32, _vp], _i32),
    "uniquan_attn_bwd": ([_i64, _i64, _i32, _i32, _vp, _vp, _vp, _vp, _vp, _vp, _f32, _vp, _vp, _vp, _vp, _i32, _i32,
                          _vp, _vp], _i32),
    "uniquan_probe_mfma_flops": ([_i32], ctypes.c_double),
    "uniquan_probe_stream": ([_i32, _i64, _vp, _vp, _vp, _i32, _vp], _i32),
    "uniquan_probe_mfma": ([_i32, _vp, _vp], _i32),
    "uniquan_bcq_matmul_ws": ([_i32, _i64, _i64], ctypes.c_size_t),
    "uniquan_bcq_matmul": ([_i32, _i64, _i64, _i32, _i32, _vp, _vp, _vp, _vp, _vp, _vp, ctypes.c_size_t, _vp],
                           _i32),
}

_lib = None
_recorder = None


def _load() -> ctypes.CDLL:
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with __graft_entry__.build() "
                               "(python paper_2506_03781_amd/build.py)")
        L = ctypes.CDLL(LIB_PATH)
        for name, (args, res) in _SIGS.items():
            fn = getattr(L, name)
            fn.argtypes = args
            fn.restype = res
        _lib = L
    return _lib


def lib() -> ctypes.CDLL:
    """The loaded library; raises if it has not been built."""
    L = _load()
    return L if _recorder is None else _recorder


def _is_launch(name: str) -> bool:
    """Entry points that enqueue work: status result, stream as last argument."""
    sig = _SIGS.get(name)
    return sig is not None and sig[1] is _i32 and len(sig[0]) > 0 and sig[0][-1] is _vp


def _stream_tag(ptr):
    """None for the stream current at recording (or the null stream), else
    the stream's handle."""
    if not ptr or not torch.cuda.is_available():
        return None
    return None if ptr == torch.cuda.current_stream().cuda_stream else ptr


class _Recorder:
    """Stands in for the library while ``record`` runs: every launch entry
    point is called as usual and its marshalled arguments are kept, with the
    stream it was enqueued on (the current one or another) and the waits
    between streams made through ``wait_stream``."""

    def __init__(self, real):
        self.real, self.calls = real, []

    def __getattr__(self, name):
        fn = getattr(self.real, name)
        if not _is_launch(name):
            return fn

        def call(*args):
            self.calls.append(("launch", fn, args, _stream_tag(args[-1])))
            return fn(*args)
        return call


def wait_stream(waiter, waitee):
    """waiter.wait_stream(waitee) (torch streams); kept by ``record`` so that
    a replay orders its streams the same way."""
    if _recorder is not None:
        _recorder.calls.append(("wait", _stream_tag(waiter.cuda_stream), _stream_tag(waitee.cuda_stream)))
    waiter.wait_stream(waitee)


class Launches:
    """Entry-point calls recorded once through the checked wrappers and
    replayed with the same marshalled arguments (pointers, sizes, scalars):
    calls made on the stream current at recording go to the stream given to
    the replay, calls made on other streams to streams of the replay's own
    (default priority), with the recorded waits between them.  The
    per-tensor checks run once, at recording.  The tensors behind the
    recorded pointers must stay alive and keep their storage; a status other
    than UQ_OK still raises."""

    def __init__(self, calls):
        self.calls = calls
        self._streams = {}

    def __len__(self):
        return sum(1 for c in self.calls if c[0] == "launch")

    def _side(self, tag):
        if tag not in self._streams:
            self._streams[tag] = torch.cuda.Stream()
        return self._streams[tag]

    def __call__(self, stream=None):
        main_ptr = _stream(stream)
        main = []  # the replay's stream as a torch stream, made only for waits

        def obj(tag):
            if tag is not None:
                return self._side(tag)
            if not main:
                main.append(stream if isinstance(stream, torch.cuda.Stream) else
                            torch.cuda.current_stream() if stream is None else torch.cuda.ExternalStream(main_ptr))
            return main[0]

        for c in self.calls:
            if c[0] == "wait":
                obj(c[1]).wait_stream(obj(c[2]))
                continue
            _, fn, args, tag = c
            status = fn(*args[:-1], main_ptr if tag is None else obj(tag).cuda_stream)
            if status != UQ_OK:
                raise UniquanError(status, last_error())


def record(fn, *args, **kwargs) -> Launches:
    """Run ``fn(*args, **kwargs)`` once (it executes normally) and return its
    launches for replay.  Not thread-safe: one recording at a time."""
    global _recorder
    if _recorder is not None:
        raise RuntimeError("record() does not nest")
    _recorder = _Recorder(_load())
    try:
        fn(*args, **kwargs)
        return Launches(_recorder.calls)
    finally:
        _recorder = None


def declared_symbols() -> list:
    """Entry points declared in include/uniquan.h."""
    txt = open(HEADER).read()
    return sorted(set(re.findall(r"\b(uniquan_[a-z0-9_]+)\s*\(", txt)))


def last_error() -> str:
    return lib().uniquan_last_error().decode()


def _check(status: int):
    if status != UQ_OK:
        raise UniquanError(status, last_error())


def _stream(stream):
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    return getattr(stream, "cuda_stream", stream)


def _dt(t: torch.Tensor) -> int:
    if t.dtype == torch.bfloat16:
        return UQ_BF16
    if t.dtype == torch.float32:
        return UQ_F32
    raise TypeError(f"unsupported dtype {t.dtype}")


def _p(t, n=None, dtypes=None, name="tensor"):
    """Device pointer of a contiguous tensor with >= n elements (None -> NULL)."""
    if t is None:
        return None
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if dtypes is not None and t.dtype not in dtypes:
        raise TypeError(f"{name} has dtype {t.dtype}, expected one of {dtypes}")
    if n is not None and t.numel() < n:
        raise ValueError(f"{name} has {t.numel()} elements, needs {n}")
    return t.data_ptr()


_F = (torch.float32,)
_W = (torch.float32, torch.bfloat16)
_B = (torch.bfloat16,)
_U8 = (torch.uint8,)
_H = (torch.float16,)
_U32 = (torch.int32, torch.uint32)  # bit-plane words (bits only)


def uniquan_fq_fwd(R, C, k, g, W, s, s_r, delta, z_u, alpha, z_b, mode, codes, W_hat, stream=None):
    N, Gn = R * C, R * C // g
    _check(lib().uniquan_fq_fwd(
        R, C, k, g, _p(W, N, _W, "W"), _dt(W), _p(s, N, _F, "s"), _p(s_r, R, _F, "s_r"),
        _p(delta, Gn, _F, "delta"), _p(z_u, Gn, _F, "z_u"), _p(alpha, Gn * k, _F, "alpha"),
        _p(z_b, Gn, _F, "z_b"), int(mode), _p(codes, N, _U8, "codes"), _p(W_hat, N, _W, "W_hat"),
        _dt(W_hat), _stream(stream)))


def uniquan_fq_fwd_residual(R, C, k, g, W, s, s_r, delta, z_u, alpha, z_b, mode, codes, R_out, stream=None):
    N, Gn = R * C, R * C // g
    _check(lib().uniquan_fq_fwd_residual(
        R, C, k, g, _p(W, N, _W, "W"), _dt(W), _p(s, N, _F, "s"), _p(s_r, R, _F, "s_r"),
        _p(delta, Gn, _F, "delta"), _p(z_u, Gn, _F, "z_u"), _p(alpha, Gn * k, _F, "alpha"),
        _p(z_b, Gn, _F, "z_b"), int(mode), _p(codes, N, _U8, "codes"), _p(R_out, N, _W, "R_out"),
        _dt(R_out), _stream(stream)))


def uniquan_fq_bwd(R, C, k, g, W, s, s_r, delta, z_u, alpha, z_b, codes, grad_W_hat,
                   grad_s, grad_alpha, grad_z_b, grad_delta=None, grad_z_u=None, grad_s_r=None,
                   group_ws=None, stream=None):
    N, Gn = R * C, R * C // g
    _check(lib().uniquan_fq_bwd(
        R, C, k, g, _p(W, N, _W, "W"), _dt(W), _p(s, N, _F, "s"), _p(s_r, R, _F, "s_r"),
        _p(delta, Gn, _F, "delta"), _p(z_u, Gn, _F, "z_u"), _p(alpha, Gn * k, _F, "alpha"),
        _p(z_b, Gn, _F, "z_b"), _p(codes, N, _U8, "codes"), _p(grad_W_hat, N, _W, "grad_W_hat"),
        _dt(grad_W_hat), _p(grad_s, N, _F, "grad_s"), _p(grad_alpha, Gn * k, _F, "grad_alpha"),
        _p(grad_z_b, Gn, _F, "grad_z_b"), _p(grad_delta, Gn, _F, "grad_delta"),
        _p(grad_z_u, Gn, _F, "grad_z_u"), _p(grad_s_r, R, _F, "grad_s_r"),
        _p(group_ws, Gn, _F, "group_ws"), _stream(stream)))


def uniquan_fq_bwd_sgd(R, C, k, g, W, s, s_r, delta, z_u, alpha, z_b, codes, grad_W_hat,
                       grad_s, grad_alpha, grad_z_b, lr_f, lr_b, stream=None):
    N, Gn = R * C, R * C // g
    _check(lib().uniquan_fq_bwd_sgd(
        R, C, k, g, _p(W, N, _W, "W"), _dt(W), _p(s, N, _F, "s"), _p(s_r, R, _F, "s_r"),
        _p(delta, Gn, _F, "delta"), _p(z_u, Gn, _F, "z_u"), _p(alpha, Gn * k, _F, "alpha"),
        _p(z_b, Gn, _F, "z_b"), _p(codes, N, _U8, "codes"), _p(grad_W_hat, N, _W, "grad_W_hat"),
        _dt(grad_W_hat), _p(grad_s, N, _F, "grad_s"), _p(grad_alpha, Gn * k, _F, "grad_alpha"),
        _p(grad_z_b, Gn, _F, "grad_z_b"), float(lr_f), float(lr_b), _stream(stream)))


def uniquan_fq_step(R, C, k, g, W, s, s_r, delta, z_u, alpha, z_b, codes, grad_W_hat, lr_f, lr_b, next_mode,
                    W_hat, residual=False, stream=None):
    """Backward + SGD of this step fused with the next step's forward (next_mode)."""
    N, Gn = R * C, R * C // g
    _check(lib().uniquan_fq_step(
        R, C, k, g, _p(W, N, _W, "W"), _dt(W), _p(s, N, _F, "s"), _p(s_r, R, _F, "s_r"),
        _p(delta, Gn, _F, "delta"), _p(z_u, Gn, _F, "z_u"), _p(alpha, Gn * k, _F, "alpha"),
        _p(z_b, Gn, _F, "z_b"), _p(codes, N, _U8, "codes"), _p(grad_W_hat, N, _W, "grad_W_hat"),
        _dt(grad_W_hat), float(lr_f), float(lr_b), int(next_mode), _p(W_hat, N, _W, "W_hat"), _dt(W_hat),
        int(bool(residual)), _stream(stream)))


def uniquan_layer_target(T, R, C, X, W, Yt, stream=None):
    _check(lib().uniquan_layer_target(T, R, C, _p(X, T * C, _B, "X"), _p(W, R * C, _B, "W"),
                                      _p(Yt, R * T, _F, "Yt"), _stream(stream)))


def uniquan_transpose_bf16(rows, cols, x, out, stream=None):
    _check(lib().uniquan_transpose_bf16(rows, cols, _p(x, rows * cols, _B, "in"),
                                        _p(out, rows * cols, _B, "out"), _stream(stream)))


def uniquan_recon_ws(T, R, C) -> int:
    return int(lib().uniquan_recon_ws(T, R, C))


def uniquan_layer_recon(T, R, C, X, Xt, W_hat, Yt, loss, Et_ws, partials_ws, grad_W_hat=None, stream=None):
    _check(lib().uniquan_layer_recon(
        T, R, C, _p(X, T * C, _B, "X"), _p(Xt, T * C, _B, "Xt"), _p(W_hat, R * C, _B, "W_hat"),
        _p(Yt, R * T, _F, "Yt"), _p(loss, 1, _F, "loss"), _p(Et_ws, R * T, _B, "Et_ws"),
        _p(partials_ws, uniquan_recon_ws(T, R, C), _F, "partials_ws"),
        partials_ws.numel() if partials_ws is not None else 0,
        _p(grad_W_hat, R * C, _W, "grad_W_hat"),
        _dt(grad_W_hat) if grad_W_hat is not None else UQ_BF16, _stream(stream)))


def uniquan_layer_recon_noalloc(T, R, C, X, Xt, W_hat, Yt, loss, Et, grad_W_hat=None, stream=None):
    """uniquan_layer_recon with the loss partials in the library's fixed scratch."""
    _check(lib().uniquan_layer_recon_noalloc(
        T, R, C, _p(X, T * C, _B, "X"), _p(Xt, T * C, _B, "Xt"), _p(W_hat, R * C, _B, "W_hat"),
        _p(Yt, R * T, _F, "Yt"), _p(loss, 1, _F, "loss"), _p(Et, R * T, _B, "Et"),
        _p(grad_W_hat, R * C, _W, "grad_W_hat"),
        _dt(grad_W_hat) if grad_W_hat is not None else UQ_BF16, _stream(stream)))


def uniquan_layer_grad(T, R, C, Et, Xt, grad_W_hat, stream=None):
    _check(lib().uniquan_layer_grad(T, R, C, _p(Et, R * T, _B, "Et"), _p(Xt, T * C, _B, "Xt"),
                                    _p(grad_W_hat, R * C, _W, "grad_W_hat"), _dt(grad_W_hat), _stream(stream)))


def uniquan_layer_grad_ste_sgd(T, R, C, k, g, Et, Xt, W, s, s_r, delta, z_u, alpha, z_b, codes, lr_f, lr_b,
                               grad_s=None, grad_alpha=None, grad_z_b=None, stream=None):
    N, Gn = R * C, R * C // g
    _check(lib().uniquan_layer_grad_ste_sgd(
        T, R, C, k, g, _p(Et, R * T, _B, "Et"), _p(Xt, T * C, _B, "Xt"), _p(W, N, _W, "W"), _dt(W),
        _p(s, N, _F, "s"), _p(s_r, R, _F, "s_r"), _p(delta, Gn, _F, "delta"), _p(z_u, Gn, _F, "z_u"),
        _p(alpha, Gn * k, _F, "alpha"), _p(z_b, Gn, _F, "z_b"), _p(codes, N, _U8, "codes"),
        float(lr_f), float(lr_b), _p(grad_s, N, _F, "grad_s"), _p(grad_alpha, Gn * k, _F, "grad_alpha"),
        _p(grad_z_b, Gn, _F, "grad_z_b"), _stream(stream)))


def uniquan_fold_to_bcq(R, C, k, g, W, s, s_r, delta, z_u, alpha, z_b, alpha_star, z_star,
                        codes_out=None, code_src=0, stream=None):
    N, Gn = R * C, R * C // g
    _check(lib().uniquan_fold_to_bcq(
        R, C, k, g, _p(W, N, _W, "W"), _dt(W) if W is not None else UQ_F32, _p(s, N, _F, "s"),
        _p(s_r, R, _F, "s_r"), _p(delta, Gn, _F, "delta"), _p(z_u, Gn, _F, "z_u"),
        _p(alpha, Gn * k, _F, "alpha"), _p(z_b, Gn, _F, "z_b"), _p(alpha_star, Gn * k, _F, "alpha_star"),
        _p(z_star, Gn, _F, "z_star"), _p(codes_out, N, _U8, "codes_out"), int(code_src), _stream(stream)))


def uniquan_bcq_dequant(R, C, k, g, codes, alpha, z_b, W_out, stream=None):
    N, Gn = R * C, R * C // g
    _check(lib().uniquan_bcq_dequant(R, C, k, g, _p(codes, N, _U8, "codes"), _p(alpha, Gn * k, _F, "alpha"),
                                     _p(z_b, Gn, _F, "z_b"), _p(W_out, N, _W, "W_out"), _dt(W_out),
                                     _stream(stream)))


def uniquan_init_greedy(R, C, k, g, W, s, s_r, delta, z_u, z_b, alpha, stream=None):
    N, Gn = R * C, R * C // g
    _check(lib().uniquan_init_greedy(
        R, C, k, g, _p(W, N, _W, "W"), _dt(W), _p(s, N, _F, "s"), _p(s_r, R, _F, "s_r"),
        _p(delta, Gn, _F, "delta"), _p(z_u, Gn, _F, "z_u"), _p(z_b, Gn, _F, "z_b"),
        _p(alpha, Gn * k, _F, "alpha"), _stream(stream)))


def uniquan_init_unified(R, C, k, g, W, grid_G, alt_T, clip, delta, z_u, alpha, z_b,
                         codes=None, err=None, s=None, s_r=None, stream=None):
    N, Gn = R * C, R * C // g
    _check(lib().uniquan_init_unified(
        R, C, k, g, _p(W, N, _W, "W"), _dt(W), int(grid_G), int(alt_T), int(clip),
        _p(delta, Gn, _F, "delta"), _p(z_u, Gn, _F, "z_u"), _p(alpha, Gn * k, _F, "alpha"),
        _p(z_b, Gn, _F, "z_b"), _p(codes, N, _U8, "codes"), _p(err, Gn, _F, "err"),
        _p(s, N, _F, "s"), _p(s_r, R, _F, "s_r"), _stream(stream)))


def uniquan_sgd(theta, grad, lr, stream=None):
    n = theta.numel()
    _check(lib().uniquan_sgd(n, _p(theta, n, _F, "theta"), _p(grad, n, _F, "grad"), float(lr), _stream(stream)))


def uniquan_bcq_pack(R, C, k, g, codes, alpha_star, z_star, planes, alpha16, z16, stream=None):
    """Stored form from the fold: planes (R*C*k/32 32-bit words), alpha16
    (Gn*k) and z16 (Gn) binary16 out."""
    N, Gn = R * C, R * C // g
    _check(lib().uniquan_bcq_pack(
        R, C, k, g, _p(codes, N, _U8, "codes"), _p(alpha_star, Gn * k, _F, "alpha_star"),
        _p(z_star, Gn, _F, "z_star"), _p(planes, N * k // 32, _U32, "planes"),
        _p(alpha16, Gn * k, _H, "alpha16"), _p(z16, Gn, _H, "z16"), _stream(stream)))


def uniquan_bcq_matmul_ws(T, R, C) -> int:
    return int(lib().uniquan_bcq_matmul_ws(T, R, C))


def uniquan_bcq_matmul(T, R, C, k, g, X, planes, alpha16, z16, Y, partials_ws=None, stream=None):
    """Y [T, R] fp32 = X [T, C] (bf16) times the stored layer's What^T."""
    N, Gn = R * C, R * C // g
    need = uniquan_bcq_matmul_ws(T, R, C)
    _check(lib().uniquan_bcq_matmul(
        T, R, C, k, g, _p(X, T * C, _B, "X"), _p(planes, N * k // 32, _U32, "planes"),
        _p(alpha16, Gn * k, _H, "alpha16"), _p(z16, Gn, _H, "z16"), _p(Y, T * R, _F, "Y"),
        _p(partials_ws, need, _F, "partials_ws") if need else _p(partials_ws, None, _F, "partials_ws"),
        partials_ws.numel() if partials_ws is not None else 0, _stream(stream)))


def uniquan_gemm_nt(M, N, K, A, B, out, scale=1.0, stream=None):
    """out [M, N] = scale * A [M, K] B [N, K]^T (bf16 operands; out bf16 or fp32)."""
    _check(lib().uniquan_gemm_nt(M, N, K, _p(A, M * K, _B, "A"), _p(B, N * K, _B, "B"),
                                 _p(out, M * N, _W, "out"), _dt(out), float(scale), _stream(stream)))


def uniquan_gemm(M, N, K, A, a_kslow, B, b_kslow, out, scale=1.0, stream=None):
    """out [M, N] = scale * sum_k A(m, k) B(n, k): A stored [M, K] or, with a_kslow, [K, M];
    B stored [N, K] or, with b_kslow, [K, N] (bf16 operands; out bf16 or fp32)."""
    _check(lib().uniquan_gemm(M, N, K, _p(A, M * K, _B, "A"), int(bool(a_kslow)), _p(B, N * K, _B, "B"),
                              int(bool(b_kslow)), _p(out, M * N, _W, "out"), _dt(out), float(scale), _stream(stream)))


def uniquan_rope_table(L, d, cs, stream=None):
    """cs [L, d/2, 2] fp32: cos and sin of every rotary angle (as uniquan_rope_split uses them)."""
    _check(lib().uniquan_rope_table(int(L), int(d), _p(cs, L * d, _F, "cs"), _stream(stream)))


def uniquan_gemm_heads(T, H, K, A, W, L, out, group=1, rotate=True, cs=None, stream=None, n_rot=None):
    """out [H, T, 128] bf16 = uniquan_rope_split(A [T, K] W [H 128, K]^T) (group, rotate as there);
    n_rot, if given, rotates only the heads h < n_rot."""
    N = H * 128
    nr = (H if rotate else 0) if n_rot is None else int(n_rot)
    _check(lib().uniquan_gemm_heads(T, H, K, _p(A, T * K, _B, "A"), _p(W, N * K, _B, "W"), int(L), int(group),
                                    nr, _p(cs, L * 128, _F, "cs") if nr else None,
                                    _p(out, T * N, _B, "out"), _stream(stream)))


def uniquan_gemm_swiglu(T, I, K, X, Wg, Wu, G, U, H, stream=None):
    """G = X Wg^T, U = X Wu^T (bf16 [T, I]) and H = silu(G) U in one product."""
    n = T * I
    _check(lib().uniquan_gemm_swiglu(T, I, K, _p(X, T * K, _B, "X"), _p(Wg, I * K, _B, "Wg"), _p(Wu, I * K, _B, "Wu"),
                                     _p(G, n, _B, "G"), _p(U, n, _B, "U"), _p(H, n, _B, "H"), _stream(stream)))


def uniquan_gemm_nt_residual(M, N, K, A, B, R, out, stream=None):
    """out = R + A B^T (fp32 [M, N]; A [M, K], B [N, K] bf16); out may be R."""
    _check(lib().uniquan_gemm_nt_residual(M, N, K, _p(A, M * K, _B, "A"), _p(B, N * K, _B, "B"),
                                          _p(R, M * N, _F, "R"), _p(out, M * N, _F, "out"), _stream(stream)))


def _p_rows(t, rows, cols, ld, dtypes, name):
    """Device pointer of a [rows, cols] tensor whose rows are ld elements apart
    (a contiguous tensor when ld == cols, else a column slice of a wider one)."""
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if t.dtype not in dtypes:
        raise TypeError(f"{name} has dtype {t.dtype}, expected one of {dtypes}")
    if tuple(t.shape) != (rows, cols) or (rows > 1 and t.stride(0) != ld) or t.stride(1) != 1:
        raise ValueError(f"{name} must be [{rows}, {cols}] with rows {ld} elements apart")
    return t.data_ptr()


def uniquan_gemm_silu_bwd(T, I, K, E, Wd, scale, G, U, dG, dU, stream=None, ld_d=0):
    """dG, dU of the SiLU product at dH = bf16(scale E Wd) (Wd stored [K, I]); dH is not written.
    With ld_d = 0, dG and dU are contiguous [T, I]; else [T, I] views whose rows
    are ld_d elements apart (dG = A[:, :I], dU = A[:, I:] of one [T, 2I] array A)."""
    n = T * I
    if ld_d:
        pg, pu = _p_rows(dG, T, I, ld_d, _B, "dG"), _p_rows(dU, T, I, ld_d, _B, "dU")
    else:
        pg, pu = _p(dG, n, _B, "dG"), _p(dU, n, _B, "dU")
    _check(lib().uniquan_gemm_silu_bwd(T, I, K, _p(E, T * K, _B, "E"), _p(Wd, K * I, _B, "Wd"), float(scale),
                                       _p(G, n, _B, "G"), _p(U, n, _B, "U"), pg, pu, int(ld_d), _stream(stream)))


def uniquan_gemm_block_loss_ws(T, C) -> int:
    return int(lib().uniquan_gemm_block_loss_ws(T, C))


def uniquan_gemm_block_loss(T, C, K, H, Wd, R, Yref, E, partials, loss, stream=None):
    """E = bf16((R + H Wd^T) - Yref) and loss = sum e^2 (partials: uniquan_gemm_block_loss_ws floats)."""
    n = T * C
    _check(lib().uniquan_gemm_block_loss(T, C, K, _p(H, T * K, _B, "H"), _p(Wd, C * K, _B, "Wd"), _p(R, n, _F, "R"),
                                         _p(Yref, n, _F, "Yref"), _p(E, n, _B, "E"),
                                         _p(partials, uniquan_gemm_block_loss_ws(T, C), _F, "partials"),
                                         partials.numel(), _p(loss, 1, _F, "loss"), _stream(stream)))


def uniquan_silu_mul_fwd(G, U, H, stream=None):
    n = G.numel()
    _check(lib().uniquan_silu_mul_fwd(n, _p(G, n, _B, "G"), _p(U, n, _B, "U"), _p(H, n, _B, "H"), _stream(stream)))


def uniquan_silu_mul_bwd(dH, G, U, dG, dU, stream=None):
    n = G.numel()
    _check(lib().uniquan_silu_mul_bwd(n, _p(dH, n, _B, "dH"), _p(G, n, _B, "G"), _p(U, n, _B, "U"),
                                      _p(dG, n, _B, "dG"), _p(dU, n, _B, "dU"), _stream(stream)))


def uniquan_gemm_nt_batched(M, N, K, batch, A, stride_a, B, stride_b, out, stride_out, scale=1.0, causal=0,
                            stream=None):
    """out_b = scale * A_b B_b^T for b < batch (strides in elements; 0 repeats an operand);
    causal 1/2/3 as declared in the header."""
    na = (batch - 1) * stride_a + M * K
    nb = (batch - 1) * stride_b + N * K
    no = (batch - 1) * stride_out + M * N
    _check(lib().uniquan_gemm_nt_batched(M, N, K, batch, _p(A, na, _B, "A"), stride_a, _p(B, nb, _B, "B"), stride_b,
                                         _p(out, no, _W, "out"), stride_out, _dt(out), float(scale), int(causal),
                                         _stream(stream)))


def uniquan_add_rmsnorm(T, C, X, A, gamma, R, Z, rinv, stream=None):
    n = T * C
    _check(lib().uniquan_add_rmsnorm(T, C, _p(X, n, _F, "X"), _p(A, n, _F, "A"), _p(gamma, C, _F, "gamma"),
                                     _p(R, n, _F, "R"), _p(Z, n, _B, "Z"), _p(rinv, T, _F, "rinv"), _stream(stream)))


def uniquan_rmsnorm_bwd(T, C, dZa, dZb, X, gamma, rinv, E, escale, dR, dRf=None, stream=None):
    n = T * C
    _check(lib().uniquan_rmsnorm_bwd(T, C, _p(dZa, n, _F, "dZa"), _p(dZb, n, _F, "dZb"), _p(X, n, _F, "X"),
                                     _p(gamma, C, _F, "gamma"), _p(rinv, T, _F, "rinv"), _p(E, n, _B, "E"),
                                     float(escale), _p(dR, n, _B, "dR"), _p(dRf, n, _F, "dRf"), _stream(stream)))


def uniquan_rope_split(T, H, d, L, x, out, rotate=True, group=1, stream=None):
    """Token-major x [T, H d] (fp32 or bf16) -> head-major bf16 out [H, T, d] (grouped slot order when group > 1)."""
    n = T * H * d
    _check(lib().uniquan_rope_split(T, H, d, L, int(group), _p(x, n, _W, "in"), _dt(x), int(bool(rotate)),
                                    _p(out, n, _B, "out"), _stream(stream)))


def uniquan_rope_merge(T, H, d, L, x, out, rotate=True, group=1, nsum=1, stream=None, ld_out=0):
    """Head-major x [nsum, H, T, d] (fp32 or bf16) -> token-major bf16 out [T, H d], partials summed;
    with ld_out, out is a [T, H d] view whose rows are ld_out elements apart."""
    n = T * H * d
    po = _p_rows(out, T, H * d, ld_out, _B, "out") if ld_out else _p(out, n, _B, "out")
    _check(lib().uniquan_rope_merge(T, H, d, L, int(group), int(nsum), _p(x, n * nsum, _W, "in"), _dt(x),
                                    int(bool(rotate)), po, int(ld_out), _stream(stream)))


def uniquan_softmax_causal(rows, L, S, P, stream=None):
    n = rows * L
    _check(lib().uniquan_softmax_causal(rows, L, _p(S, n, _F, "S"), _p(P, n, _B, "P"), _stream(stream)))


def uniquan_softmax_causal_bwd(rows, L, dP, P, dS, stream=None):
    n = rows * L
    _check(lib().uniquan_softmax_causal_bwd(rows, L, _p(dP, n, _F, "dP"), _p(P, n, _B, "P"), _p(dS, n, _B, "dS"),
                                            _stream(stream)))


def uniquan_attn_fwd(batch, kv_batch, L, d, Q, K, V, scale, O, row_lse, tok_seqs=0, group=1, stream=None):
    """Causal attention forward with on-chip score tiles (see the header); tok_seqs > 0 writes O
    token-major."""
    nq, nk = batch * L * d, kv_batch * L * d
    _check(lib().uniquan_attn_fwd(batch, kv_batch, L, d, _p(Q, nq, _B, "Q"), _p(K, nk, _B, "K"), _p(V, nk, _B, "V"),
                                  float(scale), _p(O, nq, _B, "O"), _p(row_lse, batch * L, _F, "row_lse"),
                                  int(tok_seqs), int(group), _stream(stream)))


def uniquan_attn_bwd(batch, kv_batch, L, d, Q, K, V, O, dO, row_lse, scale, delta, dQ, dK, dV, tok_seqs=0, group=1,
                     cs=None, stream=None):
    """Causal attention backward: dQ and dK, dV, and the row terms delta.  tok_seqs = 0: fp32 head-major
    gradients per query head; tok_seqs > 0: O, dO token-major, dQ token-major bf16 (inverse-rotated, cs from
    uniquan_rope_table), dK, dV token-major bf16 when kv_batch == batch, else fp32 per-query-head partials."""
    nq, nk, nr = batch * L * d, kv_batch * L * d, batch * L
    tq = _B if tok_seqs else _F
    tkv = _B if tok_seqs and kv_batch == batch else _F
    _check(lib().uniquan_attn_bwd(batch, kv_batch, L, d, _p(Q, nq, _B, "Q"), _p(K, nk, _B, "K"), _p(V, nk, _B, "V"),
                                  _p(O, nq, _B, "O"), _p(dO, nq, _B, "dO"), _p(row_lse, nr, _F, "row_lse"), float(scale),
                                  _p(delta, nr, _F, "delta"), _p(dQ, nq, tq, "dQ"), _p(dK, nq, tkv, "dK"),
                                  _p(dV, nq, tkv, "dV"), int(tok_seqs), int(group),
                                  _p(cs, L * d, _F, "cs") if tok_seqs else None, _stream(stream)))


def uniquan_transpose_bf16_batched(batch, R, C, x, out, stream=None):
    n = batch * R * C
    _check(lib().uniquan_transpose_bf16_batched(batch, R, C, _p(x, n, _B, "in"), _p(out, n, _B, "out"),
                                                _stream(stream)))


def uniquan_block_loss_ws():
    return int(lib().uniquan_block_loss_ws())


def uniquan_block_loss(n, R, M, Yref, E, partials, loss, stream=None):
    _check(lib().uniquan_block_loss(n, _p(R, n, _F, "R"), _p(M, n, _F, "M"), _p(Yref, n, _F, "Yref"),
                                    _p(E, n, _B, "E"), _p(partials, None, _F, "partials"), partials.numel(),
                                    _p(loss, 1, _F, "loss"), _stream(stream)))


def uniquan_probe_mfma_flops(iters) -> float:
    return float(lib().uniquan_probe_mfma_flops(int(iters)))


def uniquan_probe_stream(op, n_bytes, src, dst, sink, blocks=8192, stream=None):
    """Ceiling probe: op 0 reads src, 1 writes dst, 2 copies src -> dst (n_bytes each)."""
    for t, used, name in ((src, op != 1, "src"), (dst, op != 0, "dst")):
        if used and (t is None or t.numel() * t.element_size() < n_bytes):
            raise ValueError(f"{name} must hold {n_bytes} bytes")
    _check(lib().uniquan_probe_stream(int(op), int(n_bytes), _p(src, None, None, "src"), _p(dst, None, None, "dst"),
                                      _p(sink, 4, _F, "sink"), int(blocks), _stream(stream)))


def uniquan_probe_mfma(iters, sink, stream=None):
    _check(lib().uniquan_probe_mfma(int(iters), _p(sink, 4, _F, "sink"), _stream(stream)))


def uniquan_recon_noalloc_max_partials() -> int:
    return int(lib().uniquan_recon_noalloc_max_partials())
