"""Layer-level composite around the fused matmul (gate/up W4A16 GEMM ->
tf_silu_mul -> down W4A16 GEMM, the Llama-3-8B MLP) against the CPU oracle,
through the C ABI."""
from __future__ import annotations

import numpy as np
import pytest

import oracle
from paper_2606_11357_amd.synth import make_inputs

from test_gpu_parity import assert_parity, dev, pack, tf  # noqa: F401

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


def f16_ulps(a, b):
    """|a - b| in units in the last place of fp16 (finite values)."""
    ia = a.view(np.int16).astype(np.int32)
    ib = b.view(np.int16).astype(np.int32)
    ia = np.where(ia < 0, -32768 - ia, ia)
    ib = np.where(ib < 0, -32768 - ib, ib)
    return np.abs(ia - ib)


@pytest.mark.parametrize("M,N", [(1, 8), (7, 136), (64, 4096), (33, 14336)])
def test_silu_mul_vs_oracle(tf, M, N):
    """fp32 on the GPU against float64 on the host, both rounded to fp16 once:
    at most one ulp apart, almost always equal."""
    rng = np.random.default_rng(M * N)
    gu = (rng.standard_normal((M, 2 * N)) * 5.0).astype(np.float16)
    gu[0, :4] = np.array([0.0, 60000.0, -60000.0, -20.0], dtype=np.float16)
    got = tf.silu_mul(dev(gu)).cpu().numpy()
    want = oracle.to_f16(oracle.silu_mul(gu))
    ulps = f16_ulps(got, want)
    assert ulps.max() <= 1, (M, N, ulps.max())
    assert (ulps == 0).mean() >= 0.999


def _mlp_inputs(M, K, I, seed):
    gu = make_inputs(4, M, K, 2 * I, seed=seed)
    dn = make_inputs(4, 1, I, K, seed=seed + 1)
    return gu, dn


def _run_mlp(tf, gu, dn, K, I):
    pgu, pdn = pack(tf, gu), pack(tf, dn)
    x = dev(gu["x"])
    g = tf.w4a16_gemm(x, pgu, K, 2 * I, 128)
    h = tf.silu_mul(g)
    y = tf.w4a16_gemm(h, pdn, I, K, 128)
    torch.cuda.synchronize()
    return y.cpu().numpy()


@pytest.mark.parametrize("M,K,I", [(64, 512, 1024), (5, 1024, 512), (200, 256, 2048)])
def test_mlp_composite_parity(tf, M, K, I):
    gu, dn = _mlp_inputs(M, K, I, seed=M + I)
    got = _run_mlp(tf, gu, dn, K, I)
    want = oracle.mlp_w4a16(gu["x"], gu["qweight"], gu["qzeros"], gu["s"],
                            dn["qweight"], dn["qzeros"], dn["s"], 128)
    assert_parity(got, want, f"MLP composite {M}x{K}x{I}")


@pytest.mark.slow
def test_mlp_llama3_8b_full(tf):
    """Llama-3-8B MLP (hidden 4096, intermediate 14336) at M = 256: every
    element of Y against the oracle composite."""
    M, K, I = 256, 4096, 14336
    gu, dn = _mlp_inputs(M, K, I, seed=3)
    got = _run_mlp(tf, gu, dn, K, I)
    want = oracle.mlp_w4a16(gu["x"], gu["qweight"], gu["qzeros"], gu["s"],
                            dn["qweight"], dn["qzeros"], dn["s"], 128)
    assert_parity(got, want, "Llama-3-8B MLP, all of Y")


# ---------------------------------------------------------------------------
# the composite in BF16 (the paper's dtype)
# ---------------------------------------------------------------------------
def _bf16_dev(bits):
    return dev(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16)


def _bf16_bits(t):
    return t.view(torch.int16).cpu().numpy().view(np.uint16)


def bf16_ulps(a, b):
    """|a - b| in bfloat16 units in the last place (finite patterns)."""
    ia, ib = a.astype(np.int32), b.astype(np.int32)
    ia = np.where(ia >= 0x8000, 0x8000 - ia, ia)
    ib = np.where(ib >= 0x8000, 0x8000 - ib, ib)
    return np.abs(ia - ib)


@pytest.mark.parametrize("M,N", [(1, 8), (7, 136), (64, 4096), (33, 14336)])
def test_silu_mul_bf16_vs_oracle(tf, M, N):
    """fp32 on the GPU against float64 on the host, both rounded to bfloat16
    once: at most one ulp apart.  Gates stay above -88, where the fp32
    exponential of -g is finite (below, the GPU returns -0 for a product that
    is a bfloat16 subnormal at most)."""
    rng = np.random.default_rng(M * N + 1)
    v = (rng.standard_normal((M, 2 * N)) * 5.0).astype(np.float32)
    v[0, :4] = np.array([0.0, 1e30, -1e30, -20.0], dtype=np.float32)
    bits = (v.view(np.uint32) >> 16).astype(np.uint16)
    got = _bf16_bits(tf.silu_mul(_bf16_dev(bits)))
    want = oracle.bf16_encode(oracle.to_bf16(oracle.silu_mul(oracle.bf16_decode(bits))))
    ulps = bf16_ulps(got, want)
    assert ulps.max() <= 1, (M, N, ulps.max())


def _mlp_inputs_bf16(M, K, I, seed):
    from paper_2606_11357_amd.synth import make_inputs_bf16
    return make_inputs_bf16(4, M, K, 2 * I, seed=seed), make_inputs_bf16(4, 1, I, K, seed=seed + 1)


def _pack_bf16(tf, d):
    return tf.pack_w4(dev(d["qweight"]), dev(d["qzeros"]), dev(d["s_bits"].view(np.int16)),
                      d["K"], d["N"], d["group"])


@pytest.mark.parametrize("M,K,I", [(64, 512, 1024), (5, 1024, 512), (200, 256, 2048)])
def test_mlp_composite_bf16_parity(tf, M, K, I):
    """gate/up GEMM -> silu * up -> down GEMM in BF16 against the BF16 oracle
    composite, to the stated tolerance (a stored bfloat16 intermediate may
    round one ulp apart on the two sides, so no per-element bound)."""
    gu, dn = _mlp_inputs_bf16(M, K, I, seed=M + I + 7)
    x = _bf16_dev(gu["x_bits"])
    g = tf.w4a16_gemm(x, _pack_bf16(tf, gu), K, 2 * I, 128)
    h = tf.silu_mul(g)
    y = tf.w4a16_gemm(h, _pack_bf16(tf, dn), I, K, 128)
    torch.cuda.synchronize()
    got = oracle.bf16_decode(_bf16_bits(y))
    want = oracle.mlp_w4a16_bf16(gu["x_bits"], gu["qweight"], gu["qzeros"], gu["s_bits"],
                                 dn["qweight"], dn["qzeros"], dn["s_bits"], 128)
    scale = np.abs(want).max()
    err = np.abs(got - want).max()
    assert np.all(np.isfinite(got)) and err <= 1e-2 * scale, (M, K, I, err / scale)
