"""tf_w4a16_gemv_noalloc (no workspace argument, no allocation: the
library's static per-device scratch) against tf_w4a16_gemv with a caller
workspace, through the C ABI: the same kernels and plan, so the outputs must
be identical bit for bit, and both within the stated tolerance of the oracle.
Several calls in a row, each smaller than the one before, so a later call
runs on the scratch an earlier, larger call left behind (its counters must
be back at zero); the last one does not split K at all."""
from __future__ import annotations

import numpy as np
import pytest

import oracle
from paper_2606_11357_amd.synth import make_inputs

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

TOL = 1e-2


@pytest.fixture(scope="module")
def tf():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2606_11357_amd import tilefuse
    tilefuse.load()
    return tilefuse


def _up(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


# (M, K, N): K split over many workgroups (few panels, long K), then smaller
# split shapes, then the decode shape that needs no split
CALLS = [(8, 14336, 4096), (3, 8192, 1024), (1, 14336, 2048), (2, 4096, 14336)]


def test_noalloc_matches_workspace_entry(tf):
    for i, (M, K, N) in enumerate(CALLS):
        print(f"noalloc call {i}: M={M} K={K} N={N}", flush=True)
        d = make_inputs(4, M, K, N, seed=40 + i)
        packed = tf.pack_w4(_up(d["qweight"]), _up(d["qzeros"]), _up(d["s"]), K, N)
        x = _up(d["x"])
        need = tf.workspace_bytes(4, M, K, N)
        ws = torch.zeros(max(need, 256), dtype=torch.uint8, device="cuda")
        want_ws = tf.w4a16_gemv(x, packed, K, N, workspace=ws)
        got = tf.w4a16_gemv_noalloc(x, packed, K, N)
        torch.cuda.synchronize()
        a, b = got.cpu().numpy(), want_ws.cpu().numpy()
        np.testing.assert_array_equal(a.view(np.uint16), b.view(np.uint16))
        ref = oracle.matmul(d["x"], oracle.dequant(d["q"], d["z"], d["s"], 128))
        err = np.abs(a.astype(np.float64) - ref).max() / np.abs(ref).max()
        assert err <= TOL, (M, K, N, err)
        # the same call again on the scratch it just used
        again = tf.w4a16_gemv_noalloc(x, packed, K, N)
        torch.cuda.synchronize()
        np.testing.assert_array_equal(again.cpu().numpy().view(np.uint16), a.view(np.uint16))


def test_noalloc_under_graph_capture(tf):
    """Captured into a HIP graph (the caller this entry point is for) and
    replayed several times, with eager calls in between: every replay equals
    the eager result bit for bit."""
    M, K, N = 4, 14336, 4096
    d = make_inputs(4, M, K, N, seed=77)
    packed = tf.pack_w4(_up(d["qweight"]), _up(d["qzeros"]), _up(d["s"]), K, N)
    x = _up(d["x"])
    eager = tf.w4a16_gemv_noalloc(x, packed, K, N)
    torch.cuda.synchronize()
    want = eager.cpu().numpy().view(np.uint16).copy()
    out = torch.empty((M, N), dtype=torch.float16, device="cuda")
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        tf.w4a16_gemv_noalloc(x, packed, K, N, out=out)
    for r in range(4):
        out.zero_()
        g.replay()
        torch.cuda.synchronize()
        np.testing.assert_array_equal(out.cpu().numpy().view(np.uint16), want, err_msg=f"replay {r}")
        tf.w4a16_gemv_noalloc(x, packed, K, N)
        torch.cuda.synchronize()
