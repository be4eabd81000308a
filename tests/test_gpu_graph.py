"""Matmul calls captured in a HIP graph and replayed: every replay must equal
the eager result bitwise (same kernels, same workspace, fixed summation
orders).  The K-split kernels leave their arrival counters at zero after each
call, which is what lets a captured call run again; eager work and
synchronizations run between the replays."""
from __future__ import annotations

import numpy as np
import pytest

from paper_2606_11357_amd.synth import make_inputs

from test_gpu_parity import dev, pack, tf  # noqa: F401

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

CASES = [("gemm", 4, 1100, 1024, 2320),   # 256-row tiles, stream-K
         ("gemm", 8, 300, 4096, 1024),    # 128-row tiles, split-K
         ("gemm", 4, 40, 4096, 1024),     # streaming matrix-core form, 64 row slots
         ("gemv", 4, 1, 14336, 4096),     # decode GEMV, K split
         ("gemv", 8, 5, 4096, 520)]


def test_graph_replays_match_eager(tf):
    ws = torch.zeros(max(tf.workspace_bytes(b, m, k, n) for _, b, m, k, n in CASES), dtype=torch.uint8,
                     device="cuda")
    calls = []
    for i, (kind, bits, M, K, N) in enumerate(CASES):
        d = make_inputs(bits, M, K, N, seed=300 + i)
        calls.append((getattr(tf, f"w{bits}a16_{kind}"), dev(d["x"]), pack(tf, d), K, N,
                      torch.empty((M, N), dtype=torch.float16, device="cuda")))

    def run_all():
        for fn, x, p, K, N, out in calls:
            fn(x, p, K, N, 128, out=out, workspace=ws)

    run_all()
    torch.cuda.synchronize()
    eager = [out.clone() for *_, out in calls]
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        run_all()
    torch.cuda.synchronize()
    for rep in range(3):
        for *_, out in calls:
            out.zero_()                       # eager work between replays
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for (kind, bits, M, K, N), e, (*_, out) in zip(CASES, eager, calls):
            np.testing.assert_array_equal(out.cpu().numpy().view(np.uint16), e.cpu().numpy().view(np.uint16),
                                          err_msg=f"replay {rep}: {kind} W{bits} {M}x{K}x{N}")
