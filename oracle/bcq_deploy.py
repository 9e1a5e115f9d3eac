"""CPU oracle for the deployment side of UniQuan_F (arXiv 2506.03781): the
stored form of a folded BCQ layer and its product with activations.

TEST INFRASTRUCTURE, under the same rules as ``oracle.uniquan``: only
``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import it, and it imports nothing from the HIP library.

What is stored (appendix "Memory usage"): per group of g weights, the binary
code matrix C in {-1, +1}^{g x k} at one bit per entry and the k + 1 real
parameters alpha*, z*_B of Theta*_B at 16 bits each, i.e. g k + 16 (k + 1)
bits per group.  The paper fixes the bit counts, not the arrangement; the
arrangement below is this library's (chosen so that 64 lanes working on 64
consecutive rows read contiguous memory) and is restated in the C header:

* planes: uint32 [k, C / 128, R, 4].  planes[i, q, r, m] holds columns
  128 q + 32 m .. 128 q + 32 m + 31 of row r for bit-plane i: its bit j is 1
  iff c_{i+1} = +1 for weight (r, 128 q + 32 m + j), i.e. bit i of the code.
* alpha16: float16 [k, C / g, R], alpha16[i, j, r] = RNE_fp16(alpha*_{i+1})
  of group (r, j); z16: float16 [C / g, R] likewise for z*_B.

The product (the inference step R_B(C; Theta*) applied to a batch of
activations, Table "schemes", last row) is defined in float64 from the stored
values: What[r, c] = z16 + sum_i alpha16_i sigma_i(r, c), Y = X What^T.
"""
from __future__ import annotations

import numpy as np

F64 = np.float64
QUAD = 128      # columns per 16-byte plane word group


def _check(R, C, k, g):
    if C % QUAD or C % g or g % QUAD:
        raise ValueError("need C % 128 == 0, C % g == 0 and g % 128 == 0")
    if not 1 <= k <= 4:
        raise ValueError("k in 1..4")


def pack_planes(codes: np.ndarray, k: int) -> np.ndarray:
    """Bit-planes of the codes (bits 0..k-1 of each code byte) in the layout
    above, uint32 [k, C/128, R, 4]."""
    codes = np.asarray(codes, np.uint8)
    R, C = codes.shape
    nq = C // QUAD
    out = np.zeros((k, nq, R, 4), np.uint32)
    # columns of word (q, m): 128 q + 32 m + j, j = 0..31
    cols = codes.reshape(R, nq, 4, 32).astype(np.uint32)
    weights = (np.uint32(1) << np.arange(32, dtype=np.uint32))
    for i in range(k):
        bits = (cols >> np.uint32(i)) & np.uint32(1)                 # [R, nq, 4, 32]
        words = (bits * weights).sum(axis=-1, dtype=np.uint64).astype(np.uint32)
        out[i] = words.transpose(1, 0, 2)                            # [nq, R, 4]
    return out


def unpack_planes(planes: np.ndarray, R: int, C: int) -> np.ndarray:
    """Codes [R, C] (uint8, bits 0..k-1) from the bit-planes."""
    planes = np.asarray(planes, np.uint32)
    k = planes.shape[0]
    codes = np.zeros((R, C), np.uint8)
    for i in range(k):
        w = planes[i].transpose(1, 0, 2)                             # [R, nq, 4]
        bits = (w[..., None] >> np.arange(32, dtype=np.uint32)) & np.uint32(1)
        codes |= (bits.reshape(R, C).astype(np.uint8) << np.uint8(i))
    return codes


def params_fp16(alpha_star: np.ndarray, z_star: np.ndarray, R: int, C: int, k: int, g: int):
    """alpha16 [k, C/g, R] and z16 [C/g, R]: the fp32 fold results rounded to
    IEEE binary16 (to nearest even), arranged row-fastest."""
    gpr = C // g
    a = np.asarray(alpha_star, np.float32).reshape(R, gpr, k)
    z = np.asarray(z_star, np.float32).reshape(R, gpr)
    return (np.ascontiguousarray(a.transpose(2, 1, 0)).astype(np.float16),
            np.ascontiguousarray(z.T).astype(np.float16))


def pack(codes, alpha_star, z_star, k, g):
    """The whole stored form: (planes, alpha16, z16)."""
    codes = np.asarray(codes, np.uint8)
    R, C = codes.shape
    _check(R, C, k, g)
    a16, z16 = params_fp16(alpha_star, z_star, R, C, k, g)
    return pack_planes(codes & np.uint8((1 << k) - 1), k), a16, z16


def storage_bits(planes, alpha16, z16) -> int:
    """Bits the stored form occupies."""
    return 8 * (np.asarray(planes).nbytes + np.asarray(alpha16).nbytes + np.asarray(z16).nbytes)


def dequant_f64(planes, alpha16, z16, R: int, C: int, g: int) -> np.ndarray:
    """What [R, C] = z16 + sum_i alpha16_i sigma_i in float64 (sigma = +1 for a
    set bit, -1 otherwise), from the stored form."""
    planes = np.asarray(planes, np.uint32)
    k = planes.shape[0]
    gpr = C // g
    codes = unpack_planes(planes, R, C).astype(np.int64)
    a = np.asarray(alpha16, np.float16).astype(F64)                  # [k, gpr, R]
    z = np.asarray(z16, np.float16).astype(F64)                      # [gpr, R]
    W = np.repeat(z.T, g, axis=1)                                    # [R, C]
    for i in range(k):
        sig = np.where((codes >> i) & 1, 1.0, -1.0)
        W = W + np.repeat(a[i].T, g, axis=1) * sig
    return W


def matmul_f64(X, planes, alpha16, z16, R: int, C: int, g: int) -> np.ndarray:
    """Y [T, R] = X What^T in float64 on the stored values (X as given)."""
    return np.asarray(X, F64) @ dequant_f64(planes, alpha16, z16, R, C, g).T
