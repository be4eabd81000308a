"""Seeded synthetic inputs for the fused weight-only quantized matmul.

This module only draws random numbers and writes them in the AWQ boundary
format; it holds none of the method's arithmetic (no unpacking, no
dequantization, no contraction).  Both the CPU checker and the HIP path read
the arrays it returns.

Workload recipe (Section 2.2 defines the format; Section 5.1 and Table 1 the
shapes):

* activations ``x``: fp16 ``[M, K]``, ``x_std * N(0, 1)`` drawn in float64 then
  rounded to fp16;
* weight codes ``q``: uniform integers in ``[0, 2**bits - 1]``, ``[K, N]``;
* scales ``s``: uniform in ``[s_lo, s_hi]`` drawn in float64 then rounded to fp16,
  ``[K / G, N]`` (one per group of ``G`` consecutive ``k`` in one column);
* zero-points ``z``: uniform integers in ``[0, 2**bits - 1]``, ``[K / G, N]``.

Draw order is fixed as x -> q -> s -> z from one ``numpy.random.default_rng(seed)``.

Boundary encoding (the AWQ-style layout the library accepts):

* W4: ``qweight int32 [K, N/8]``; nibble ``i`` of word ``j`` (bits ``4i..4i+3``)
  holds column ``8j + i``.  ``qzeros int32 [K/G, N/8]`` packed the same way.
* W8: ``qweight uint8 [K, N]`` and ``zeros uint8 [K/G, N]`` stored as is.
* scales: fp16 ``[K/G, N]``.
"""
from __future__ import annotations

import numpy as np

__all__ = [
    "pack_nibbles",
    "make_inputs",
    "make_inputs_w8sym",
    "WORKLOADS",
    "make_inputs_bf16",
    "M_SWEEP",
    "M_SWEEP_SHAPES",
]


def pack_nibbles(codes: np.ndarray) -> np.ndarray:
    """Encode uint8 codes ``[R, N]`` (each in 0..15) as AWQ int32 words ``[R, N/8]``.

    Nibble ``i`` of word ``j`` (bits ``4i..4i+3``) holds column ``8j + i``.
    """
    codes = np.asarray(codes)
    if codes.ndim != 2 or codes.shape[1] % 8 != 0:
        raise ValueError("codes must be [R, N] with N a multiple of 8")
    if codes.size and (codes.min() < 0 or codes.max() > 15):
        raise ValueError("4-bit codes must lie in 0..15")
    r, n = codes.shape
    c = codes.astype(np.uint32).reshape(r, n // 8, 8)
    word = np.zeros((r, n // 8), dtype=np.uint32)
    for i in range(8):
        word |= c[:, :, i] << np.uint32(4 * i)
    return word.view(np.int32)


def make_inputs(bits: int, M: int, K: int, N: int, group: int = 128, seed: int = 0,
                x_std: float = 1.0, s_lo: float | None = None, s_hi: float | None = None,
                ) -> dict:
    """Draw one seeded workload.

    Returns a dict with the unpacked draws (``x``, ``q``, ``s``, ``z``) and the
    boundary tensors (``qweight``, ``qzeros`` for W4; ``qweight``, ``zeros`` for W8).
    """
    if bits not in (4, 8):
        raise ValueError("bits must be 4 or 8")
    if K % group != 0:
        raise ValueError("K must be a multiple of the group size")
    if bits == 4 and N % 8 != 0:
        raise ValueError("W4 needs N a multiple of 8")
    if s_lo is None:
        s_lo, s_hi = (0.005, 0.02) if bits == 4 else (0.0003, 0.001)
    qmax = (1 << bits) - 1
    rng = np.random.default_rng(seed)
    x = (x_std * rng.standard_normal((M, K))).astype(np.float16)
    q = rng.integers(0, qmax + 1, size=(K, N), dtype=np.uint8)
    s = rng.uniform(s_lo, s_hi, size=(K // group, N)).astype(np.float16)
    z = rng.integers(0, qmax + 1, size=(K // group, N), dtype=np.uint8)
    out = {"bits": bits, "M": M, "K": K, "N": N, "group": group,
           "x": x, "q": q, "s": s, "z": z}
    if bits == 4:
        out["qweight"] = pack_nibbles(q)
        out["qzeros"] = pack_nibbles(z)
    else:
        out["qweight"] = q
        out["zeros"] = z
    return out


def _bf16_bits(v: np.ndarray) -> np.ndarray:
    """float32 draws -> bfloat16 bit patterns by keeping the high 16 bits
    (truncation: the draw only has to be some bfloat16 value)."""
    return (np.asarray(v, dtype=np.float32).view(np.uint32) >> np.uint32(16)).astype(np.uint16)


def make_inputs_bf16(bits: int, M: int, K: int, N: int, group: int = 128, seed: int = 0,
                     x_std: float = 1.0, s_lo: float | None = None, s_hi: float | None = None,
                     ) -> dict:
    """Draw one seeded workload with BF16 activations and scales.

    Same draws and order as ``make_inputs`` (x -> q -> s -> z), except that x
    and s are drawn in float32 and handed over as bfloat16 bit patterns
    ``x_bits`` [M, K] and ``s_bits`` [K/G, N] (uint16).  The boundary tensors
    are as in ``make_inputs``.
    """
    if bits not in (4, 8):
        raise ValueError("bits must be 4 or 8")
    if K % group != 0:
        raise ValueError("K must be a multiple of the group size")
    if bits == 4 and N % 8 != 0:
        raise ValueError("W4 needs N a multiple of 8")
    if s_lo is None:
        s_lo, s_hi = (0.005, 0.02) if bits == 4 else (0.0003, 0.001)
    qmax = (1 << bits) - 1
    rng = np.random.default_rng(seed)
    x = _bf16_bits((x_std * rng.standard_normal((M, K))).astype(np.float32))
    q = rng.integers(0, qmax + 1, size=(K, N), dtype=np.uint8)
    s = _bf16_bits(rng.uniform(s_lo, s_hi, size=(K // group, N)).astype(np.float32))
    z = rng.integers(0, qmax + 1, size=(K // group, N), dtype=np.uint8)
    out = {"bits": bits, "M": M, "K": K, "N": N, "group": group,
           "x_bits": x, "q": q, "s_bits": s, "z": z}
    if bits == 4:
        out["qweight"] = pack_nibbles(q)
        out["qzeros"] = pack_nibbles(z)
    else:
        out["qweight"] = q
        out["zeros"] = z
    return out


def make_inputs_w8sym(M: int, K: int, N: int, seed: int = 0, x_std: float = 1.0,
                      s_lo: float = 0.0003, s_hi: float = 0.001) -> dict:
    """Draw one seeded per-channel symmetric INT8 workload (the paper's W8A16).

    Draw order x -> q -> s: ``x`` fp16 ``[M, K]`` as in ``make_inputs``; ``q``
    uniform signed integers in ``[-128, 127]``, int8 ``[K, N]``; ``s`` uniform in
    ``[s_lo, s_hi]`` drawn in float64 then rounded to fp16, one per column ``[N]``.
    """
    rng = np.random.default_rng(seed)
    x = (x_std * rng.standard_normal((M, K))).astype(np.float16)
    q = rng.integers(-128, 128, size=(K, N), dtype=np.int8)
    s = rng.uniform(s_lo, s_hi, size=(N,)).astype(np.float16)
    return {"M": M, "K": K, "N": N, "x": x, "q": q, "s": s, "qweight": q, "scales": s}


# The synthetic Llama-shaped workloads the library is measured and checked on.
# Each entry: name -> (bits, M values, K, N, x_std).  Scale ranges follow bits.
# The paper's GEMM sweep (Section 5: prompt lengths M from 256 to 8192 in steps
# of 256 at both Llama-3-8B MLP shapes, K and N swapped), W4A16, G = 128.
M_SWEEP = tuple(range(256, 8192 + 1, 256))
M_SWEEP_SHAPES = ((4096, 14336), (14336, 4096))

WORKLOADS = {
    "w4_gemm_m16_k2048_n2048": (4, (16,), 2048, 2048, 1.0),
    "w4_gemv_k4096_n14336": (4, (1, 4, 8), 4096, 14336, 1.0),
    "w8_k4096_n4096": (8, (1, 512), 4096, 4096, 1.0),
    "w4_gemm_m2048_k4096_n14336": (4, (2048,), 4096, 14336, 1.0),
    "w4_gemm_m2048_k14336_n4096": (4, (2048,), 14336, 4096, 1.0),
    "w4_gemm_m1024_k4096_n32768": (4, (1024,), 4096, 32768, 0.5),
    "w4_gemm_m1024_k32768_n8192": (4, (1024,), 32768, 8192, 0.5),
}
