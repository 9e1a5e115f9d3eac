"""Seeded synthetic inputs for the UniQuan_F fake-quant path.

This module is the only code shared by the HIP path's callers (tests, bench)
and the CPU oracle.  It draws data and nothing else: it holds none of the
method's arithmetic (no transform, level table, mapping, gradient or
initialisation).  Quantization parameters that the method itself derives
(alpha from the greedy binary-coding start, clipping-based Delta / z_U) are
computed by the callers, each side with its own code.

Workloads stand in for the paper's pretrained Mistral-7B / Llama-3 weights and
C4 / GSM8K calibration samples (Experimental setup; Appendix "Evaluation
Protocol": 128 sequences of 2048 tokens), which are not available: heavy-tailed
Student-t weights with outlier input channels, Gaussian or SiLU-gated Gaussian
activations, at the shapes of 7B / 70B attention and MLP projections.

Random streams: numpy ``Generator(PCG64(SeedSequence([seed, tag, sub, i])))``
with a fixed integer tag (and sub-tag) per tensor and i the index of a fixed
chunk of 2^22 elements, so every tensor is reproducible on its own and chunks
can be drawn in parallel.  Student-t(nu) samples are Z / sqrt(V / nu) with
Z ~ N(0, 1) and V ~ chi-square(nu) drawn as 2 Gamma(nu / 2).  Seeds 0, 1, 2
follow the paper's evaluation protocol.
"""
from __future__ import annotations

import zlib
from dataclasses import dataclass, field

import numpy as np

# Per-tensor stream tags.
TAG_W = 1
TAG_X = 2
TAG_S = 3
TAG_OUTLIER = 4
TAG_SILU_A = 5
TAG_SILU_B = 6
TAG_EXTRA = 7


def rng(seed: int, tag: int, sub: int = 0) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, tag, sub])))


def bf16_bits_from_f32(x: np.ndarray) -> np.ndarray:
    """Storage cast fp32 -> bf16 (round to nearest, ties to even), as uint16 bits."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    lsb = (u >> np.uint64(16)) & np.uint64(1)
    r = (u + np.uint64(0x7FFF) + lsb) >> np.uint64(16)
    return r.astype(np.uint16)


def f32_from_bf16_bits(b: np.ndarray) -> np.ndarray:
    return (np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def round_to_bf16(x: np.ndarray) -> np.ndarray:
    """fp32 values that are exactly representable in bf16 (RNE storage cast)."""
    return f32_from_bf16_bits(bf16_bits_from_f32(x))


@dataclass
class Matrix:
    """One weight matrix with its calibration input.

    W: [R, C] float32 (bf16-exact when ``dtype == 'bf16'``); X: [T, C] float32
    (bf16-exact when bf16); s: [R, C] float32 element-wise scales.
    """
    name: str
    R: int
    C: int
    T: int
    dtype: str
    W: np.ndarray
    X: np.ndarray
    s: np.ndarray
    outlier_cols: np.ndarray = field(default_factory=lambda: np.zeros(0, np.int64))


@dataclass
class MatrixSpec:
    name: str
    R: int
    C: int
    T: int
    dtype: str = "bf16"
    w_dist: str = "t"          # "normal" or "t"
    w_nu: float = 5.0
    w_std: float = 0.02
    w_outlier_frac: float = 0.0
    w_outlier_mult: float = 1.0
    x_dist: str = "normal"     # "normal" or "silu_gated"
    x_outlier_frac: float = 0.0
    x_outlier_mult: float = 1.0
    s_std: float = 0.01        # s = 1 + N(0, s_std^2); 0 => s = 1
    x_stream: int = 0          # matrices that share an input share this id


@dataclass
class Workload:
    name: str
    description: str
    ks: tuple
    group_size: int     # 0: one group per row (g = C of each matrix)
    matrices: list


def _name_tag(name: str) -> int:
    return zlib.crc32(name.encode())


# Large tensors are drawn in fixed chunks of CHUNK elements (row-major order),
# chunk i from its own stream rng(seed, tag, sub, i), so a tensor is the same
# whatever the number of threads that fill it.
CHUNK = 1 << 22
_POOL = None


def _pool():
    global _POOL
    if _POOL is None:
        import os
        from concurrent.futures import ThreadPoolExecutor
        n = max(1, min(16, len(os.sched_getaffinity(0))))
        _POOL = ThreadPoolExecutor(n)
    return _POOL


def _fill(shape, seed: int, tag: int, sub: int, draw) -> np.ndarray:
    """float32 array of `shape`; draw(generator, out) fills one flat chunk."""
    out = np.empty(shape, np.float32)
    flat = out.reshape(-1)
    n = flat.size
    starts = range(0, n, CHUNK)

    def one(i0):
        draw(np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, tag, sub, i0 // CHUNK]))),
             flat[i0:min(n, i0 + CHUNK)])

    list(_pool().map(one, starts))
    return out


def _student_t(nu: float, scale: float):
    """Student-t(nu) times scale: Z / sqrt(V / nu) with Z ~ N(0, 1) and
    V = 2 Gamma(nu / 2) ~ chi-square(nu), drawn in float64 and stored fp32."""
    def draw(g, out):
        z = g.standard_normal(out.size)
        v = g.standard_gamma(nu / 2.0, out.size) * (2.0 / nu)
        np.multiply(z / np.sqrt(v), scale, out=out, casting="same_kind")
    return draw


def _normal(scale: float = 1.0, shift: float = 0.0):
    def draw(g, out):
        g.standard_normal(out=out, dtype=np.float32)
        if scale != 1.0:
            out *= np.float32(scale)
        if shift != 0.0:
            out += np.float32(shift)
    return draw


def _weights(spec: MatrixSpec, seed: int, cols: np.ndarray) -> np.ndarray:
    sub = _name_tag(spec.name)
    if spec.w_dist == "normal":
        w = _fill((spec.R, spec.C), seed, TAG_W, sub, _normal(spec.w_std))
    else:
        nu = spec.w_nu
        w = _fill((spec.R, spec.C), seed, TAG_W, sub, _student_t(nu, spec.w_std / np.sqrt(nu / (nu - 2.0))))
    if cols.size and spec.w_outlier_mult != 1.0:
        w[:, cols] *= np.float32(spec.w_outlier_mult)
    return w


def _inputs(spec: MatrixSpec, seed: int, cols: np.ndarray) -> np.ndarray:
    if spec.x_dist == "normal":
        x = _fill((spec.T, spec.C), seed, TAG_X, spec.x_stream, _normal())
    else:
        a = _fill((spec.T, spec.C), seed, TAG_SILU_A, spec.x_stream, _normal())
        b = _fill((spec.T, spec.C), seed, TAG_SILU_B, spec.x_stream, _normal())
        x = (a / (np.float32(1.0) + np.exp(-a)) * b).astype(np.float32)
    if cols.size and spec.x_outlier_mult != 1.0:
        x[:, cols] *= np.float32(spec.x_outlier_mult)
    return x


def _round_bf16_inplace(x: np.ndarray) -> np.ndarray:
    """round_to_bf16 applied chunk by chunk in the thread pool."""
    flat = x.reshape(-1)

    def one(i0):
        c = flat[i0:i0 + CHUNK]
        c[...] = round_to_bf16(c)

    list(_pool().map(one, range(0, flat.size, CHUNK)))
    return x


def make_matrix(spec: MatrixSpec, seed: int = 0) -> Matrix:
    frac = max(spec.w_outlier_frac, spec.x_outlier_frac)
    n_out = int(round(frac * spec.C))
    cols = np.sort(rng(seed, TAG_OUTLIER, spec.C).choice(spec.C, n_out, replace=False)) if n_out else np.zeros(0, np.int64)
    w = _weights(spec, seed, cols if spec.w_outlier_frac > 0 else np.zeros(0, np.int64))
    x = _inputs(spec, seed, cols if spec.x_outlier_frac > 0 else np.zeros(0, np.int64))
    if spec.s_std > 0:
        s = _fill((spec.R, spec.C), seed, TAG_S, _name_tag(spec.name), _normal(spec.s_std, 1.0))
    else:
        s = np.ones((spec.R, spec.C), np.float32)
    if spec.dtype == "bf16":
        w = _round_bf16_inplace(w)
        x = _round_bf16_inplace(x)
    return Matrix(spec.name, spec.R, spec.C, spec.T, spec.dtype, w, x, s, cols)


# Heavy-tailed 7B-style distribution: Student-t(5) scaled to std 0.02 with 1% of
# input columns x20 in W and x10 in X.
def _spec7b(name, R, C, T, x_dist="normal", x_stream=0):
    return MatrixSpec(name, R, C, T, "bf16", "t", 5.0, 0.02, 0.01, 20.0,
                      x_dist, 0.01 if x_dist == "normal" else 0.0, 10.0, 0.01, x_stream)


def _spec70b(name, R, C, T, x_dist="normal"):
    return MatrixSpec(name, R, C, T, "bf16", "t", 4.0, 0.015, 0.0, 1.0,
                      x_dist, 0.005 if x_dist == "normal" else 0.0, 15.0, 0.01, 0)


WORKLOADS = {
    "layer256": Workload(
        "layer256", "single linear layer 256x256 fp32 N(0,0.02^2), X 64x256 N(0,1), k=3, g=128",
        (3,), 128,
        [MatrixSpec("w", 256, 256, 64, "f32", "normal", 0, 0.02, 0, 1, "normal", 0, 1, 0.0)]),
    "attn4096": Workload(
        "attn4096", "7B attention projection 4096x4096 bf16 t(5) outliers, X 2048x4096, k in {4,3}, g=128",
        (4, 3), 128, [_spec7b("q_proj", 4096, 4096, 2048)]),
    "mlp7b": Workload(
        "mlp7b", "7B MLP gate/up 11008x4096, down 4096x11008, X 4096 tokens, k=3, g=128",
        (3,), 128,
        [_spec7b("gate_proj", 11008, 4096, 4096), _spec7b("up_proj", 11008, 4096, 4096),
         _spec7b("down_proj", 4096, 11008, 4096, "silu_gated", 1)]),
    "block7b": Workload(
        "block7b", "7B decoder block, 7 matrices, X 8192 tokens, k=3, g=128",
        (3,), 128,
        [_spec7b("q_proj", 4096, 4096, 8192), _spec7b("k_proj", 4096, 4096, 8192),
         _spec7b("v_proj", 4096, 4096, 8192), _spec7b("o_proj", 4096, 4096, 8192, x_stream=2),
         _spec7b("gate_proj", 11008, 4096, 8192), _spec7b("up_proj", 11008, 4096, 8192),
         _spec7b("down_proj", 4096, 11008, 8192, "silu_gated", 1)]),
    "mlp7b_rows": Workload(
        "mlp7b_rows", "7B MLP gate/up 11008x4096, down 4096x11008, X 4096 tokens, k=3, one group per row "
        "(g = C: 4096 and 11008)",
        (3,), 0,
        [_spec7b("gate_proj", 11008, 4096, 4096), _spec7b("up_proj", 11008, 4096, 4096),
         _spec7b("down_proj", 4096, 11008, 4096, "silu_gated", 1)]),
    "mlp70b": Workload(
        "mlp70b", "70B MLP slice gate/up 28672x8192, down 8192x28672, X 4096 tokens, k in {2,3}, g=128",
        (2, 3), 128,
        [_spec70b("gate_proj", 28672, 8192, 4096), _spec70b("up_proj", 28672, 8192, 4096),
         _spec70b("down_proj", 8192, 28672, 4096, "silu_gated")]),
}


def scaled(spec: MatrixSpec, R: int | None = None, C: int | None = None, T: int | None = None) -> MatrixSpec:
    """Same distribution at another shape (small parity cases)."""
    d = dict(spec.__dict__)
    if R is not None:
        d["R"] = R
    if C is not None:
        d["C"] = C
    if T is not None:
        d["T"] = T
    return MatrixSpec(**d)


def random_codes(R: int, C: int, k: int, seed: int) -> np.ndarray:
    """Uniform random k-bit codes (uint8), e.g. previous mappings for LOCAL mode."""
    return rng(seed, TAG_EXTRA, 11).integers(0, 1 << k, size=(R, C), dtype=np.uint8)


def perturb(x: np.ndarray, rel: float, seed: int, sub: int) -> np.ndarray:
    """x * (1 + rel * N(0,1)) in fp32: a small optimiser-like move of parameters."""
    e = rng(seed, TAG_EXTRA, sub).standard_normal(x.shape).astype(np.float32)
    return (x * (np.float32(1.0) + np.float32(rel) * e)).astype(np.float32)
