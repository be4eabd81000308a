"""CPU oracle for the BF16 form of the fused weight-only matmul.

TEST INFRASTRUCTURE ONLY.  Only the test-suite, the smoke check and the
benchmark's CPU-baseline leg may import this module; the library never does.
It shares no code with the HIP path: plain numpy, float64 where arithmetic
happens.

The paper's kernels take BF16 activations and BF16 scales (Section 2.2;
Section 4.2, the scales stored beside each weight tile; Section 4.3, the
dequantized weights written into a BF16 buffer before the multiply):

1. decode   -- a bfloat16 value is the upper 16 bits of an IEEE-754 binary32
               (sign, 8 exponent bits, 7 fraction bits); inputs travel as
               those 16-bit patterns.
2. unpack, group, Eq. 2 -- as in ``awq_oracle`` (exact in float64).
3. round    -- the dequantized weight is held in BF16 (Section 4.3): rounded
               to the nearest bfloat16, ties to an even last fraction bit.
4. matmul   -- C = A x B_bf16 in float64 (Section 2.1).
5. output   -- the library returns bfloat16, rounded the same way.

Pins live in ``tests/test_oracle_pins_bf16.py``.
"""
from __future__ import annotations

import numpy as np

from .awq_oracle import dequant, matmul, unpack_w4

__all__ = [
    "bf16_decode",
    "to_bf16",
    "bf16_encode",
    "dequant_bf16",
    "w4a16_bf16",
    "w8a16_bf16",
]

# bfloat16: 8 significant bits (1 implicit + 7 stored), exponent range of
# binary32: normal numbers from 2**-126, subnormals down to 2**-133, largest
# finite (2 - 2**-7) * 2**127.
_BF16_MANT_BITS = 8
_BF16_MIN_EXP = -126          # exponent of the smallest normal number
_BF16_MAX = (2.0 - 2.0 ** -7) * 2.0 ** 127


def bf16_decode(bits: np.ndarray) -> np.ndarray:
    """16-bit patterns -> float64 values: the pattern is the high half of a binary32."""
    b = np.asarray(bits).astype(np.uint16).astype(np.uint32) << np.uint32(16)
    return b.view(np.float32).astype(np.float64)


def to_bf16(v: np.ndarray) -> np.ndarray:
    """Round float64 values to the nearest bfloat16 value, ties to even.

    Written from the format's definition: a finite v = m * 2**e with
    0.5 <= |m| < 1 is rounded to a multiple of the quantum 2**(e - 8) (eight
    significant bits), or of 2**(-126 - 7) below the normal range; ``np.rint``
    rounds halves to the even integer.  Magnitudes that round past the largest
    finite value become inf, as does IEEE rounding.  Returns float64.
    """
    v = np.asarray(v, dtype=np.float64)
    out = np.array(v, dtype=np.float64, copy=True)
    fin = np.isfinite(v) & (v != 0)
    _, e = np.frexp(v[fin])
    qexp = np.maximum(e - _BF16_MANT_BITS, _BF16_MIN_EXP - (_BF16_MANT_BITS - 1))
    r = np.ldexp(np.rint(np.ldexp(v[fin], -qexp)), qexp)
    r = np.where(np.abs(r) > _BF16_MAX, np.copysign(np.inf, r), r)
    out[fin] = r
    return out


def bf16_encode(v: np.ndarray) -> np.ndarray:
    """16-bit patterns of values that are already bfloat16 (e.g. ``to_bf16`` output)."""
    f = np.asarray(v, dtype=np.float64).astype(np.float32)
    if not np.array_equal(f.astype(np.float64), np.asarray(v, dtype=np.float64), equal_nan=True):
        raise ValueError("values are not representable in binary32")
    u = f.view(np.uint32)
    if np.any(u & np.uint32(0xFFFF)):
        raise ValueError("values are not bfloat16 (low 16 bits set)")
    return (u >> np.uint32(16)).astype(np.uint16)


def dequant_bf16(q: np.ndarray, z: np.ndarray, s_bits: np.ndarray, group: int) -> np.ndarray:
    """The BF16 weight a matrix unit consumes: Eq. 2 with BF16 scales, rounded once.

    ``s_bits`` are the 16-bit patterns of the scales ``[K/G, N]``.  The exact
    product (at most 8 + 8 significant bits) is formed in float64, then
    rounded to the nearest bfloat16 (Section 4.3: the dequantized tile lives
    in a BF16 buffer).
    """
    return to_bf16(dequant(q, z, bf16_decode(s_bits), group))


def w4a16_bf16(x_bits: np.ndarray, qweight: np.ndarray, qzeros: np.ndarray,
               s_bits: np.ndarray, group: int) -> np.ndarray:
    """Full W4A16 result in float64 with BF16 activations and scales:
    unpack -> Eq. 2 -> round to BF16 -> matmul."""
    q = unpack_w4(qweight)
    z = unpack_w4(qzeros)
    return matmul(bf16_decode(x_bits), dequant_bf16(q, z, s_bits, group))


def w8a16_bf16(x_bits: np.ndarray, qweight: np.ndarray, zeros: np.ndarray,
               s_bits: np.ndarray, group: int) -> np.ndarray:
    """Full W8A16 result in float64 with BF16 activations and scales (the byte is the code)."""
    return matmul(bf16_decode(x_bits),
                  dequant_bf16(np.asarray(qweight, dtype=np.uint8),
                               np.asarray(zeros, dtype=np.uint8), s_bits, group))
