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
def test_mlp_llama3_8b_sampled(tf):
    """Llama-3-8B MLP (hidden 4096, intermediate 14336) at M = 256: sampled rows
    of Y against the oracle composite of those rows."""
    M, K, I = 256, 4096, 14336
    gu, dn = _mlp_inputs(M, K, I, seed=3)
    got = _run_mlp(tf, gu, dn, K, I)
    assert np.all(np.isfinite(got.astype(np.float64)))
    rows = np.array([0, 17, 100, 255])
    want = oracle.mlp_w4a16(gu["x"][rows], gu["qweight"], gu["qzeros"], gu["s"],
                            dn["qweight"], dn["qzeros"], dn["s"], 128)
    assert_parity(got[rows], want, "Llama-3-8B MLP sampled rows")
