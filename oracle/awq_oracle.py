"""CPU oracle for the fused weight-only quantized matmul (W4A16 / W8A16).

TEST INFRASTRUCTURE ONLY.  Only the test-suite, the smoke check and the
benchmark's CPU-baseline leg may import this module; the library never does.
It shares no code with the HIP path: plain numpy, float64 where arithmetic
happens, one step per function, in the order the paper describes them.

What is computed (the plain definition of the method's result; fusing the
steps changes where they run, not the mathematics -- Sections 1 and 4.1.1):

1. unpack   -- split packed storage into integer codes by mask and shift
               (Section 4.3, "GEMM microkernel" paragraph); the nibble order is
               the AWQ boundary format: nibble i of a 32-bit word holds column
               8j + i (4-bit) / one byte per code (8-bit).
2. group    -- code (k, n) uses the scale and zero-point of group g = floor(k/G)
               of column n: G consecutive weights of one column share them
               (Section 2.2; Section 4.2 metadata paragraph, G = 128).
3. dequant  -- w_hat = s_g * (q - z_g)                 (Section 2.2, Eq. 2);
               the symmetric form w_hat = s_g * q (Eq. 1) is the case z = 0.
               The paper's own W8A16 is symmetric, signed INT8, one scale per
               output channel (Section 2.2, last paragraph; Section 4.3):
               w_hat[k, n] = s[n] * q[k, n]  (dequant_sym).
4. matmul   -- C = A x B with A [M, K], B [K, N] the dequantized weights
               (Section 2.1 problem statement), accumulated in float64.
5. output   -- round-to-nearest-even to fp16 (the library's output dtype).

Pins (what fixes this oracle independently of itself) live in
``tests/test_oracle_pins.py``: hand-derived words of the boundary format, exact
rational arithmetic on tiny inputs, closed forms, an integer-matmul invariant,
one-hot probes of the group index and operand orientation, and planted
mistakes that the pins must catch.
"""
from __future__ import annotations

import numpy as np

__all__ = [
    "unpack_w4",
    "group_of",
    "dequant",
    "dequant_f16",
    "matmul",
    "to_f16",
    "w4a16",
    "w8a16",
    "dequant_sym",
    "w8a16_sym",
]


def unpack_w4(words: np.ndarray) -> np.ndarray:
    """Unpack AWQ int32 words ``[R, N/8]`` into uint8 codes ``[R, N]``.

    Section 4.3: extract each 4-bit field by shift and mask.  The word is
    reinterpreted as unsigned 32-bit first so that nibble 7 (which holds bit
    31, the sign bit of int32) shifts down without sign extension.
    """
    w = np.asarray(words).astype(np.int32).view(np.uint32)
    r, nw = w.shape
    out = np.empty((r, nw * 8), dtype=np.uint8)
    for i in range(8):
        out[:, i::8] = ((w >> np.uint32(4 * i)) & np.uint32(0xF)).astype(np.uint8)
    return out


def group_of(k: np.ndarray | int, group: int):
    """Group index of row ``k``: ``floor(k / G)`` (Section 2.2, G rows per group)."""
    return np.asarray(k) // group


def dequant(q: np.ndarray, z: np.ndarray, s: np.ndarray, group: int) -> np.ndarray:
    """Eq. 2 for every weight: ``w_hat[k, n] = s[g(k), n] * (q[k, n] - z[g(k), n])``.

    Computed in float64.  The product of an integer in [-255, 255] and an fp16
    scale needs at most 8 + 11 significant bits, so the result is also exactly
    representable in float32; the returned array is float64.
    """
    q = np.asarray(q)
    K, N = q.shape
    if K % group != 0:
        raise ValueError("K must be a multiple of the group size")
    g = group_of(np.arange(K), group)                 # [K]
    z_full = np.asarray(z).astype(np.float64)[g, :]   # [K, N]
    s_full = np.asarray(s).astype(np.float64)[g, :]   # [K, N]
    return s_full * (q.astype(np.float64) - z_full)


def dequant_f16(q: np.ndarray, z: np.ndarray, s: np.ndarray, group: int) -> np.ndarray:
    """The fp16 weight a matrix unit consumes: round-to-nearest-even of Eq. 2."""
    return dequant(q, z, s, group).astype(np.float16)


def matmul(x: np.ndarray, w: np.ndarray) -> np.ndarray:
    """``y[m, n] = sum_k x[m, k] * w[k, n]`` in float64 (Section 2.1, C = A x B).

    ``np.matmul`` on float64 operands is the library primitive for the sum.
    """
    return np.matmul(np.asarray(x).astype(np.float64), np.asarray(w).astype(np.float64))


def to_f16(y: np.ndarray) -> np.ndarray:
    """Round a float64 result to fp16, nearest-even, IEEE overflow to inf."""
    with np.errstate(over="ignore"):
        return np.asarray(y, dtype=np.float64).astype(np.float16)


def w4a16(x: np.ndarray, qweight: np.ndarray, qzeros: np.ndarray, scales: np.ndarray,
          group: int) -> np.ndarray:
    """Full W4A16 result in float64: unpack -> dequant (Eq. 2) -> matmul."""
    q = unpack_w4(qweight)
    z = unpack_w4(qzeros)
    return matmul(x, dequant(q, z, scales, group))


def w8a16(x: np.ndarray, qweight: np.ndarray, zeros: np.ndarray, scales: np.ndarray,
          group: int) -> np.ndarray:
    """Full W8A16 result in float64: the byte is the code -> dequant (Eq. 2) -> matmul."""
    return matmul(x, dequant(np.asarray(qweight, dtype=np.uint8),
                             np.asarray(zeros, dtype=np.uint8), scales, group))


def dequant_sym(q: np.ndarray, s: np.ndarray) -> np.ndarray:
    """Eq. 1 with one scale per output channel: ``w_hat[k, n] = s[n] * q[k, n]``.

    ``q`` is signed INT8 ``[K, N]``, ``s`` fp16 ``[N]`` (Section 2.2, W8A16 with
    per-channel symmetric quantization and no zero-points; Section 4.3, the
    INT8 value times the channel's scale).  float64; exact, as in ``dequant``.
    """
    q = np.asarray(q).astype(np.float64)
    s = np.asarray(s).astype(np.float64)
    return s[None, :] * q


def w8a16_sym(x: np.ndarray, qweight: np.ndarray, scales: np.ndarray) -> np.ndarray:
    """Full symmetric per-channel W8A16 result in float64: dequant (Eq. 1) -> matmul."""
    return matmul(x, dequant_sym(np.asarray(qweight, dtype=np.int8), scales))
