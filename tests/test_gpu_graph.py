"""Matmul calls captured in a HIP graph and replayed: every replay must equal
the eager result bitwise (same kernels, same workspace, fixed summation
orders).  The kernels that count arrivals (the decode GEMV and the streaming
matrix-core form) leave their counters at zero after each call, and the tiled
GEMMs park K-split partials that a second launch sums, which is what lets a
captured call run again; eager work and synchronizations run between the
replays."""
from __future__ import annotations

import numpy as np
import pytest

from paper_2606_11357_amd.synth import make_inputs, make_inputs_bf16

from test_gpu_parity import dev, pack, tf  # noqa: F401

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

CASES = [("gemm", 4, 1100, 1024, 2320),   # 256-row tiles, stream-K
         ("gemm", 4, 200, 12288, 520),    # 128-row tiles, split-K
         ("gemm", 4, 200, 1024, 520),     # 64 x 128 tiles, K over the waves
         ("gemm", 4, 512, 512, 14336),    # 64 x 256 tiles, K over the waves
         ("gemm", 4, 40, 4096, 1024),     # streaming matrix-core form, 64 row slots
         ("gemm", 4, 20, 14336, 4096),    # streaming matrix-core form, factored, K split
         ("gemv", 4, 1, 14336, 4096),     # decode GEMV, K split
         ("gemv", 4, 1, 4096, 4096),      # decode GEMV, 4 column parts per panel
         ("gemv", 8, 5, 4096, 520)]       # ... 2 column parts, ragged panels


def _inputs(tf, dt, bits, M, K, N, seed):
    """x and the packed weight for fp16 or BF16 calls (BF16 scales packed as their bits)."""
    if dt == "f16":
        d = make_inputs(bits, M, K, N, seed=seed)
        return dev(d["x"]), pack(tf, d)
    d = make_inputs_bf16(bits, M, K, N, seed=seed)
    s = dev(d["s_bits"].view(np.int16))
    p = (tf.pack_w4(dev(d["qweight"]), dev(d["qzeros"]), s, K, N, 128) if bits == 4
         else tf.pack_w8(dev(d["qweight"]), dev(d["zeros"]), s, K, N, 128))
    return dev(d["x_bits"].view(np.int16)).view(torch.bfloat16), p


@pytest.mark.parametrize("dt", ["f16", "bf16"])
def test_graph_replays_match_eager(tf, dt):
    ws = torch.zeros(max(tf.workspace_bytes(b, m, k, n) for _, b, m, k, n in CASES), dtype=torch.uint8,
                     device="cuda")
    calls = []
    for i, (kind, bits, M, K, N) in enumerate(CASES):
        x, p = _inputs(tf, dt, bits, M, K, N, 300 + i)
        calls.append((getattr(tf, f"w{bits}a16_{kind}"), x, p, K, N,
                      torch.empty((M, N), dtype=x.dtype, device="cuda")))

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
            np.testing.assert_array_equal(out.view(torch.int16).cpu().numpy(), e.view(torch.int16).cpu().numpy(),
                                          err_msg=f"replay {rep}: {dt} {kind} W{bits} {M}x{K}x{N}")
