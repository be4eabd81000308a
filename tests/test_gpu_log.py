"""TF_LOG=1: each matmul call writes one line to stderr naming the kernel and
the plan the launcher chose (run in a child process, since the library reads
the variable once).  Without it the library prints nothing."""
from __future__ import annotations

import os
import subprocess
import sys

import pytest

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

SCRIPT = r"""
import numpy as np, torch
from paper_2606_11357_amd import tilefuse as tf
from paper_2606_11357_amd.synth import make_inputs
up = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()
for bits, M, K, N in ((4, 2048, 4096, 14336), (4, 2048, 14336, 4096), (8, 512, 4096, 4096),
                      (4, 1, 4096, 14336), (4, 16, 2048, 2048), (4, 1280, 4096, 14336)):
    d = make_inputs(bits, 1, K, N, seed=0)
    if bits == 4:
        p = tf.pack_w4(up(d["qweight"]), up(d["qzeros"]), up(d["s"]), K, N)
    else:
        p = tf.pack_w8(up(d["qweight"]), up(d["zeros"]), up(d["s"]), K, N)
    x = torch.zeros((M, K), dtype=torch.float16, device="cuda")
    (tf.w4a16_gemm if bits == 4 else tf.w8a16_gemm)(x, p, K, N)
# decode GEMV with few panels: two workgroups share each 32-column W8 panel
d = make_inputs(8, 1, 4096, 4096, seed=0)
p = tf.pack_w8(up(d["qweight"]), up(d["zeros"]), up(d["s"]), 4096, 4096)
tf.w8a16_gemv(torch.zeros((8, 4096), dtype=torch.float16, device="cuda"), p, 4096, 4096)
# prefill below 1024 rows: 64 x 256 tiles of the K-split GEMM
d = make_inputs(4, 1, 4096, 14336, seed=0)
p = tf.pack_w4(up(d["qweight"]), up(d["qzeros"]), up(d["s"]), 4096, 14336)
tf.w4a16_gemm(torch.zeros((512, 4096), dtype=torch.float16, device="cuda"), p, 4096, 14336)
torch.cuda.synchronize()
print("done")
"""


def _run(env_log):
    env = dict(os.environ)
    env.pop("TF_LOG", None)
    if env_log is not None:
        env["TF_LOG"] = env_log
    return subprocess.run([sys.executable, "-c", SCRIPT], cwd=ROOT, env=env, capture_output=True, text=True,
                          timeout=300)


def test_tf_log_names_each_plan():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    r = _run("1")
    assert r.returncode == 0 and "done" in r.stdout, r.stderr[-3000:]
    all_lines = [ln for ln in r.stderr.splitlines() if ln.startswith("[tilefuse] ")]
    lines = [ln for ln in all_lines if not ln.startswith("[tilefuse]   ")]
    assert len(lines) == 8, r.stderr
    assert "gemm256_kernel<4,1,f16> M=2048 K=4096 N=14336" in lines[0]
    assert "gemm256_kernel<4,1,f16> M=2048 K=14336 N=4096" in lines[1]
    assert "stream-K" in lines[1]
    assert "gemm_ks_kernel<8,1,f16,128>" in lines[2] and "M=512" in lines[2]
    assert "gemv_kernel<4,1," in lines[3] and "vector form" in lines[3]
    assert "gemv_kernel<4,16," in lines[4] and "matrix-core form" in lines[4]
    # 280 tiles of 256 x 256: one whole-tile round, the 24 after it on the K-split GEMM
    assert "gemm256_kernel<4,1,f16> M=1280 K=4096 N=14336" in lines[5]
    assert "K-split GEMM over the rest" in lines[5]
    rest = all_lines[all_lines.index(lines[5]) + 1]
    assert "gemm_ks_kernel<4,1,f16,128>" in rest and "tiles 256..279" in rest and "192 tiles of 64x128" in rest
    assert "gemv_kernel<8,8," in lines[6] and "128 panels x 2 column parts x 1 K slices" in lines[6]
    assert "gemm_ks_kernel<4,1,f16,256> M=512" in lines[7] and "8x56 tiles of 64x256" in lines[7]


def test_silent_without_tf_log():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    r = _run(None)
    assert r.returncode == 0 and "done" in r.stdout, r.stderr[-3000:]
    assert "[tilefuse]" not in r.stderr
