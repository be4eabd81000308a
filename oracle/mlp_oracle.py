"""CPU oracle for a layer-level composite around the fused matmul: a
transformer MLP with a gated activation (the Llama-3-8B MLP shape the paper's
workloads come from; Section 5 evaluates the linear layers of such models).

TEST INFRASTRUCTURE ONLY: imported by the tests and the benchmark's CPU leg,
never by the library.  Plain numpy in float64; the composite keeps the fp16
rounding of every tensor the GPU path stores (the gate/up output and the
activated product), because those are part of what the composite defines.

    GU = x @ dequant([W_gate | W_up])          (one W4A16 GEMM, N = 2 I)
    H  = silu(GU[:, :I]) * GU[:, I:]           silu(g) = g / (1 + e^-g)
    Y  = H @ dequant(W_down)                   (one W4A16 GEMM, K = I)

The BF16 composite is the same with BF16 activations and scales, the stored
GU and H rounded to bfloat16 and each weight to BF16 (``bf16_oracle``).
"""
from __future__ import annotations

import numpy as np

from .awq_oracle import to_f16, w4a16
from .bf16_oracle import bf16_encode, to_bf16, w4a16_bf16

__all__ = ["silu", "silu_mul", "mlp_w4a16", "mlp_w4a16_bf16"]


def silu(g: np.ndarray) -> np.ndarray:
    """``g / (1 + exp(-g))`` in float64 (the sigmoid-weighted linear unit)."""
    g = np.asarray(g, dtype=np.float64)
    with np.errstate(over="ignore"):
        return g / (1.0 + np.exp(-g))


def silu_mul(gu: np.ndarray) -> np.ndarray:
    """``silu(gu[:, :N]) * gu[:, N:]`` in float64 for a ``[M, 2N]`` input."""
    gu = np.asarray(gu, dtype=np.float64)
    n = gu.shape[1] // 2
    return silu(gu[:, :n]) * gu[:, n:]


def mlp_w4a16(x, gu_qweight, gu_qzeros, gu_scales, d_qweight, d_qzeros, d_scales, group):
    """The composite: fp16 GU and H as stored between the steps, Y in float64."""
    gu = to_f16(w4a16(x, gu_qweight, gu_qzeros, gu_scales, group))
    h = to_f16(silu_mul(gu))
    return w4a16(h, d_qweight, d_qzeros, d_scales, group)


def mlp_w4a16_bf16(x_bits, gu_qweight, gu_qzeros, gu_s_bits, d_qweight, d_qzeros, d_s_bits, group):
    """The BF16 composite: bfloat16 GU and H as stored between the steps
    (inputs and scales as bfloat16 bit patterns), Y in float64."""
    gu = to_bf16(w4a16_bf16(x_bits, gu_qweight, gu_qzeros, gu_s_bits, group))
    h = to_bf16(silu_mul(gu))
    return w4a16_bf16(bf16_encode(h), d_qweight, d_qzeros, d_s_bits, group)
