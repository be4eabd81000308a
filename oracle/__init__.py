"""CPU oracle for the fused W4A16 / W8A16 matmul.

TEST INFRASTRUCTURE ONLY: imported by the tests, the smoke check and the
benchmark's CPU-baseline leg, never by the library.
"""
from .awq_oracle import (  # noqa: F401
    dequant,
    dequant_f16,
    dequant_sym,
    group_of,
    matmul,
    to_f16,
    unpack_w4,
    w4a16,
    w8a16,
    w8a16_sym,
)
from .mlp_oracle import mlp_w4a16, mlp_w4a16_bf16, silu, silu_mul  # noqa: F401
from .bf16_oracle import (  # noqa: F401
    bf16_decode,
    bf16_encode,
    dequant_bf16,
    to_bf16,
    w4a16_bf16,
    w8a16_bf16,
)
