"""GPU parity of the paper's own W8A16 form (signed INT8, one scale per
output channel, Eq. 1) through the C ABI: tf_pack_w8_sym, then the 8-bit
unpack / dequant / GEMV / GEMM entry points, against the CPU oracle."""
from __future__ import annotations

import numpy as np
import pytest

import oracle
from paper_2606_11357_amd.synth import make_inputs_w8sym

from test_gpu_parity import assert_parity, check_guard, dev, guarded_out, tf  # noqa: F401

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


def pack_sym(tf, d, group=128):
    return tf.pack_w8_sym(dev(d["qweight"]), dev(d["scales"]), d["K"], d["N"], group)


def run_sym(tf, kind, d, packed, group=128, x=None, workspace=None):
    x = d["x"] if x is None else x
    M, K, N = x.shape[0], d["K"], d["N"]
    buf, out = guarded_out(M, N)
    getattr(tf, f"w8a16_{kind}")(dev(x), packed, K, N, group, out=out, workspace=workspace)
    torch.cuda.synchronize()
    check_guard(buf)
    return out.cpu().numpy()


@pytest.mark.parametrize("K,N,group", [(256, 40, 128), (4096, 4096, 128), (512, 264, 64), (384, 104, 128)])
def test_pack_unpack_dequant_bitexact(tf, K, N, group):
    d = make_inputs_w8sym(1, K, N, seed=K + N)
    packed = pack_sym(tf, d, group)
    q, z = tf.unpack(8, packed, K, N, group)
    np.testing.assert_array_equal(q.cpu().numpy(), (d["q"].astype(np.int16) + 128).astype(np.uint8))
    assert np.all(z.cpu().numpy() == 128)
    want = oracle.dequant_sym(d["q"], d["s"])
    w32 = tf.dequant(8, packed, K, N, group, dtype=torch.float32).cpu().numpy()
    np.testing.assert_array_equal(w32.astype(np.float64), want)
    w16 = tf.dequant(8, packed, K, N, group, dtype=torch.float16).cpu().numpy()
    np.testing.assert_array_equal(w16.view(np.uint16), want.astype(np.float16).view(np.uint16))


@pytest.mark.parametrize("kind,M,K,N", [("gemv", 1, 4096, 4096), ("gemv", 4, 4096, 4096), ("gemv", 8, 2048, 520),
                                        ("gemm", 16, 4096, 4096), ("gemm", 100, 1024, 264),
                                        ("gemm", 512, 4096, 4096), ("gemm", 1030, 2048, 776)])
def test_matmul_parity(tf, kind, M, K, N):
    d = make_inputs_w8sym(M, K, N, seed=M * 3 + N)
    got = run_sym(tf, kind, d, pack_sym(tf, d))
    assert_parity(got, oracle.w8a16_sym(d["x"], d["qweight"], d["scales"]), f"w8 sym {kind} {M}x{K}x{N}")


@pytest.mark.parametrize("kind,M,K,N", [("gemv", 8, 4096, 512), ("gemm", 256, 4096, 512), ("gemm", 1024, 4096, 520)])
def test_integer_invariant_bitexact(tf, kind, M, K, N):
    """Unit scales and integer activations: every partial sum is an integer
    below 2**24, so the fp16 output must be the rounding of the exact integer
    result (|x| <= 3, |q| <= 128)."""
    rng = np.random.default_rng(7)
    d = make_inputs_w8sym(M, K, N, seed=11)
    d["scales"] = d["s"] = np.ones(N, dtype=np.float16)
    x = rng.integers(-3, 4, size=(M, K)).astype(np.float16)
    got = run_sym(tf, kind, d, pack_sym(tf, d), x=x)
    want = (x.astype(np.int64) @ d["q"].astype(np.int64)).astype(np.float64)
    np.testing.assert_array_equal(got.view(np.uint16), oracle.to_f16(want).view(np.uint16))
