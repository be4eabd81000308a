"""GPU parity: the HIP path through the C ABI against the CPU oracle.

Bars:
  * unpack (codes, zero-points): bit-exact;
  * dequant: bit-exact, fp32 (exact Eq. 2) and fp16 (rounded once, RNE);
  * matmul: max|gpu - oracle| <= 1e-2 * max|oracle| per output matrix (the
    stated tolerance), and a stricter 1e-3 * max|oracle| regression bound that
    a dropped K term would already break;
  * integer invariant (s = 1, z = 0, integer activations): bit-exact against
    RNE_fp16 of the exact integer matmul;
  * bitwise reproducibility, and canaries around every output.
"""
from __future__ import annotations

import numpy as np
import pytest

import oracle
from paper_2606_11357_amd.synth import make_inputs, pack_nibbles

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

TOL = 1e-2          # stated tolerance, relative to max|oracle| per output matrix
STRICT = 1e-3       # internal regression bound
GUARD = 4096        # canary elements on each side of an output


@pytest.fixture(scope="module")
def tf():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2606_11357_amd import tilefuse
    tilefuse.load()
    return tilefuse


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def pack(tf, d):
    K, N, G = d["K"], d["N"], d["group"]
    if d["bits"] == 4:
        return tf.pack_w4(dev(d["qweight"]), dev(d["qzeros"]), dev(d["s"]), K, N, G)
    return tf.pack_w8(dev(d["qweight"]), dev(d["zeros"]), dev(d["s"]), K, N, G)


def guarded_out(M, N):
    buf = torch.full((M * N + 2 * GUARD,), -7.0, dtype=torch.float16, device="cuda")
    return buf, buf[GUARD:GUARD + M * N].view(M, N)


def check_guard(buf):
    g = torch.cat([buf[:GUARD], buf[-GUARD:]]).float().cpu().numpy()
    assert np.all(g == -7.0), "write outside the output"


def run(tf, kind, d, packed, x=None, workspace=None):
    K, N, G = d["K"], d["N"], d["group"]
    x = d["x"] if x is None else x
    M = x.shape[0]
    buf, out = guarded_out(M, N)
    fn = getattr(tf, f"w{d['bits']}a16_{kind}")
    fn(dev(x), packed, K, N, G, out=out, workspace=workspace)
    torch.cuda.synchronize()
    check_guard(buf)
    return out.cpu().numpy()


def ref(d, x=None, cols=None):
    x = d["x"] if x is None else x
    q, z, s = d["q"], d["z"], d["s"]
    if cols is not None:
        q, z, s = q[:, cols], z[:, cols], s[:, cols]
    return oracle.matmul(x, oracle.dequant(q, z, s, d["group"]))


def assert_parity(gpu, want, what=""):
    gpu = gpu.astype(np.float64)
    assert np.all(np.isfinite(gpu)), what
    scale = np.abs(want).max()
    err = np.abs(gpu - want).max()
    assert err <= TOL * scale, f"{what}: max err {err:.4g} > {TOL} * {scale:.4g}"
    assert err <= STRICT * scale, f"{what}: max err {err:.4g} > {STRICT} * {scale:.4g}"
    return err / scale


# ---------------------------------------------------------------------------
# unpack / dequant: bit-exact
# ---------------------------------------------------------------------------
SMALL = [(4, 256, 136, 128), (4, 128, 64, 32), (4, 2048, 2048, 128), (8, 256, 40, 128),
         (8, 192, 96, 64), (8, 4096, 4096, 128), (4, 96, 8, 32)]


@pytest.mark.parametrize("bits,K,N,G", SMALL)
def test_unpack_bitexact(tf, bits, K, N, G):
    d = make_inputs(bits, 1, K, N, group=G, seed=K + N)
    q, z = tf.unpack(bits, pack(tf, d), K, N, G)
    np.testing.assert_array_equal(q.cpu().numpy(), d["q"])
    np.testing.assert_array_equal(z.cpu().numpy(), d["z"])
    if bits == 4:   # the oracle's own unpack of the boundary words agrees
        np.testing.assert_array_equal(oracle.unpack_w4(d["qweight"]), d["q"])


@pytest.mark.parametrize("bits,K,N,G", SMALL)
def test_dequant_bitexact(tf, bits, K, N, G):
    d = make_inputs(bits, 1, K, N, group=G, seed=K * 3 + N)
    packed = pack(tf, d)
    w64 = oracle.dequant(d["q"], d["z"], d["s"], G)
    w32 = tf.dequant(bits, packed, K, N, G, dtype=torch.float32).cpu().numpy()
    np.testing.assert_array_equal(w32.view(np.uint32), w64.astype(np.float32).view(np.uint32))
    w16 = tf.dequant(bits, packed, K, N, G, dtype=torch.float16).cpu().numpy()
    np.testing.assert_array_equal(w16.view(np.uint16), oracle.dequant_f16(d["q"], d["z"], d["s"], G).view(np.uint16))


@pytest.mark.parametrize("bits", [4, 8])
def test_dequant_extreme_scales(tf, bits):
    """Scales from subnormal to the largest finite fp16, every code/zero pair."""
    qmax = (1 << bits) - 1
    K, G = 256 if bits == 8 else 32, 32
    N = 64
    rng = np.random.default_rng(99)
    q = np.tile(np.arange(K, dtype=np.int64)[:, None] % (qmax + 1), (1, N)).astype(np.uint8)
    z = rng.integers(0, qmax + 1, size=(K // G, N), dtype=np.uint8)
    sb = np.array([0x0001, 0x0002, 0x03FF, 0x0400, 0x1000, 0x2118, 0x3C00, 0x5000, 0x7BFF,
                   0x8001, 0xBC00, 0x0155, 0x1A2B, 0x2E66, 0x7800, 0x0010], dtype=np.uint16)
    s = np.tile(sb, (K // G, N // sb.size)).view(np.float16)
    d = {"bits": bits, "K": K, "N": N, "group": G, "q": q, "z": z, "s": s}
    if bits == 4:
        d["qweight"], d["qzeros"] = pack_nibbles(q), pack_nibbles(z)
    else:
        d["qweight"], d["zeros"] = q, z
    packed = pack(tf, d)
    with np.errstate(over="ignore"):
        want16 = oracle.dequant_f16(q, z, s, G)
    w16 = tf.dequant(bits, packed, K, N, G, dtype=torch.float16).cpu().numpy()
    np.testing.assert_array_equal(w16.view(np.uint16), want16.view(np.uint16))
    w32 = tf.dequant(bits, packed, K, N, G, dtype=torch.float32).cpu().numpy()
    np.testing.assert_array_equal(w32, oracle.dequant(q, z, s, G).astype(np.float32))


# ---------------------------------------------------------------------------
# matmul parity on small and ragged shapes (full comparison)
# ---------------------------------------------------------------------------
RAGGED = [(4, 1, 256, 136, 128), (4, 3, 128, 72, 32), (4, 8, 512, 200, 128),
          (8, 5, 256, 40, 128), (8, 8, 192, 104, 64), (4, 7, 96, 8, 32),
          (8, 2, 4096, 4096, 128), (4, 4, 2048, 2048, 128),
          (4, 6, 1024, 264, 128), (8, 6, 512, 104, 64), (8, 7, 2048, 136, 128),
          (4, 6, 4096, 1032, 32), (4, 2, 1024, 200, 64), (8, 4, 768, 72, 128)]


@pytest.mark.parametrize("bits,M,K,N,G", RAGGED)
def test_gemv_parity_small(tf, bits, M, K, N, G):
    d = make_inputs(bits, M, K, N, group=G, seed=M + K + N)
    assert_parity(run(tf, "gemv", d, pack(tf, d)), ref(d), f"gemv {bits} {M}x{K}x{N}")


@pytest.mark.parametrize("bits,M,K,N,G", [(4, 1, 4096, 200, 128), (4, 1, 4224, 200, 128),
                                           (8, 3, 4096, 104, 64), (8, 3, 4160, 104, 64),
                                           (4, 2, 4096, 72, 32), (4, 2, 4128, 72, 32)])
def test_gemv_one_round_boundary(tf, bits, M, K, N, G):
    """With 16 waves, K = 4096 gives each wave a run of 8 atoms, requested
    whole at the start (one round); one atom more per wave takes the
    refilled ring of two rounds.  Both sides of that boundary, with segments
    fixed at compile time (group 128) and known at run time."""
    d = make_inputs(bits, M, K, N, group=G, seed=7 * K + N)
    assert_parity(run(tf, "gemv", d, pack(tf, d), workspace=False), ref(d),
                  f"gemv {bits} {M}x{K}x{N} G={G}")


GEMM_SHAPES = [(4, 16, 2048, 2048, 128), (4, 17, 256, 136, 128), (4, 129, 512, 200, 64),
               (8, 33, 256, 40, 128), (8, 130, 384, 104, 128), (4, 9, 96, 8, 32),
               (4, 300, 1024, 520, 128), (8, 64, 128, 4096, 128), (4, 1, 256, 64, 128),
               (4, 200, 512, 328, 32), (8, 150, 512, 264, 64), (8, 140, 384, 72, 32),
               (4, 257, 768, 1000, 256), (8, 129, 1024, 200, 1024), (4, 96, 1152, 392, 96),
               (4, 600, 1024, 1040, 128), (8, 520, 512, 776, 64), (4, 513, 256, 2056, 32),
               (4, 1100, 512, 1040, 128), (8, 1030, 512, 776, 64), (4, 1280, 256, 520, 32),
               (8, 1025, 1024, 264, 1024), (4, 1024, 640, 2048, 64),
               (4, 12, 1024, 200, 64), (8, 16, 2048, 264, 128), (4, 13, 512, 1032, 32), (8, 10, 384, 40, 128),
               # 4..8 rows through the GEMM entry: the matrix-core streaming form
               (4, 4, 512, 136, 128), (8, 5, 384, 40, 32), (4, 8, 1024, 200, 64), (8, 7, 2048, 264, 128),
               (4, 6, 288, 72, 96), (4, 3, 256, 64, 128),
               # 17..64 rows: two or four row blocks of the streaming form
               (4, 24, 1024, 520, 128), (8, 31, 512, 72, 64), (4, 48, 2048, 264, 32), (8, 64, 1024, 2056, 128),
               (4, 40, 768, 136, 256),
               # 256..1023 rows with K >= 8192: the 256-row kernel (stream-K), partial row tiles
               (4, 300, 8192, 520, 128), (8, 600, 8192, 264, 64), (4, 257, 16384, 136, 32),
               # the 64 x 128 kernel with K split over the workgroup's waves: 8-bit with
               # 192..256 tiles (ragged N with a clamped last panel; 9 and 5 chunks split
               # unevenly over the four waves; groups of 64 and 32), 4-bit with 65 rows
               (8, 384, 1152, 4088, 64), (8, 420, 640, 3968, 32), (4, 65, 4096, 776, 128),
               # ... with 4-bit tiles of 64 x 256 (more than 1.5 rounds of 64 x 128 tiles): ragged
               # rows, columns (the last tile partly past N) and K (31 chunks), groups of 32 and 64
               (4, 1000, 3968, 4088, 32), (4, 300, 4096, 11008, 64), (4, 256, 4096, 14336, 128),
               # the 128-row GEMM: 4-bit beyond the 64 x 128 kernel's 1200 tiles, and
               # long K on few tiles (split-K)
               (4, 1000, 1024, 10000, 128), (4, 200, 12288, 520, 128), (8, 100, 16384, 264, 64),
               # 260 tiles of 256 x 256: one whole-tile round, the last 4 tiles (a partial
               # row tile, ragged N) by the 64 x 128 kernel, some of its parts wholly past C
               (4, 1100, 512, 13304, 64), (8, 1100, 1024, 13304, 128)]


@pytest.mark.parametrize("bits,M,K,N,G", GEMM_SHAPES)
def test_gemm_parity_small(tf, bits, M, K, N, G):
    d = make_inputs(bits, M, K, N, group=G, seed=M * 7 + K + N)
    assert_parity(run(tf, "gemm", d, pack(tf, d)), ref(d), f"gemm {bits} {M}x{K}x{N}")


@pytest.mark.parametrize("kind,bits,M,K,N", [("gemv", 4, 8, 4096, 1024), ("gemv", 8, 8, 4096, 512),
                                             ("gemm", 8, 256, 4096, 512), ("gemm", 4, 200, 8192, 256),
                                             ("gemv", 4, 1, 32768, 64), ("gemm", 4, 1030, 8192, 512),
                                             ("gemm", 8, 1024, 4096, 768), ("gemm", 4, 16, 4096, 1024),
                                             ("gemm", 8, 5, 8192, 512), ("gemm", 4, 64, 4096, 1024),
                                             ("gemm", 8, 33, 4096, 520), ("gemm", 4, 300, 8192, 520),
                                             ("gemm", 8, 384, 512, 4096), ("gemm", 4, 200, 1024, 520),
                                             ("gemm", 4, 1100, 512, 13304), ("gemm", 4, 512, 512, 14336)])
def test_integer_invariant_bitexact(tf, kind, bits, M, K, N):
    """s = 1, z = 0, integer x in [-3, 3]: every partial sum is an integer below
    2^24, so the fp16 output must be RNE of the exact integer matmul."""
    rng = np.random.default_rng(1234 + M)
    G = 128
    xi = rng.integers(-3, 4, size=(M, K))
    qi = rng.integers(0, 1 << bits, size=(K, N), dtype=np.uint8)
    if bits == 8:
        qi = (qi // 8).astype(np.uint8)      # keep |y| below the fp16 range limit
    z = np.zeros((K // G, N), dtype=np.uint8)
    d = {"bits": bits, "K": K, "N": N, "group": G, "q": qi, "z": z,
         "s": np.ones((K // G, N), dtype=np.float16), "x": xi.astype(np.float16)}
    if bits == 4:
        d["qweight"], d["qzeros"] = pack_nibbles(qi), pack_nibbles(z)
    else:
        d["qweight"], d["zeros"] = qi, z
    exact = xi.astype(np.int64) @ qi.astype(np.int64)
    assert np.abs(exact).max() < 65504
    got = run(tf, kind, d, pack(tf, d))
    np.testing.assert_array_equal(got.view(np.uint16), exact.astype(np.float64).astype(np.float16).view(np.uint16))


def test_closed_form(tf):
    """x = 1, q = 9, z = 2, s = 1/64 per column: y = K * 7 / 64 exactly."""
    K, N, G = 1024, 128, 128
    for bits in (4, 8):
        q = np.full((K, N), 9, dtype=np.uint8)
        z = np.full((K // G, N), 2, dtype=np.uint8)
        d = {"bits": bits, "K": K, "N": N, "group": G, "q": q, "z": z,
             "s": np.full((K // G, N), 1 / 64, dtype=np.float16)}
        if bits == 4:
            d["qweight"], d["qzeros"] = pack_nibbles(q), pack_nibbles(z)
        else:
            d["qweight"], d["zeros"] = q, z
        packed = pack(tf, d)
        for kind, M in (("gemv", 3), ("gemm", 40)):
            got = run(tf, kind, d, packed, x=np.ones((M, K), dtype=np.float16))
            np.testing.assert_array_equal(got, np.full((M, N), K * 7 / 64, dtype=np.float16))


@pytest.mark.parametrize("bits,M,K,N", [(4, 1, 4096, 14336), (4, 1, 14336, 4096), (8, 1, 14336, 4096),
                                        (4, 3, 8192, 1000), (8, 8, 8192, 520), (4, 5, 32768, 136),
                                        (4, 2, 256, 64), (8, 1, 4096, 4096), (8, 3, 14336, 2048),
                                        (4, 6, 14336, 1024), (8, 6, 8192, 520), (4, 7, 8192, 1000),
                                        (8, 7, 14336, 264), (4, 6, 4096, 14336), (8, 7, 4096, 4096)])
def test_gemv_workspace_modes(tf, bits, M, K, N):
    """Split-K (workspace) and single-pass (no workspace) kernels both meet the
    bar, and a workspace can be reused at once."""
    d = make_inputs(bits, M, K, N, seed=M * 11 + N)
    packed = pack(tf, d)
    want = ref(d)
    need = tf.workspace_bytes(bits, M, K, N)
    ws = torch.zeros(need + 256, dtype=torch.uint8, device="cuda") if need else False
    a = run(tf, "gemv", d, packed, workspace=ws)
    b = run(tf, "gemv", d, packed, workspace=ws)
    np.testing.assert_array_equal(a.view(np.uint16), b.view(np.uint16))
    c = run(tf, "gemv", d, packed, workspace=False)
    assert_parity(a, want, "gemv with workspace")
    assert_parity(c, want, "gemv without workspace")


def test_workspace_shared_across_shapes(tf):
    """One workspace serves a sequence of different problems (different M,
    bits, panel counts and K-splits) without clearing in between."""
    cases = [(8, 2, 14336, 4096), (4, 4, 8192, 2048), (4, 1, 14336, 4096), (8, 8, 8192, 520),
             (4, 7, 4096, 3000), (4, 1, 4096, 14336), (8, 1, 2048, 64), (4, 1, 14336, 4096)]
    need = max(tf.workspace_bytes(b, m, k, n) for b, m, k, n in cases)
    ws = torch.zeros(need, dtype=torch.uint8, device="cuda")
    for i, (bits, M, K, N) in enumerate(cases):
        d = make_inputs(bits, M, K, N, seed=100 + i)
        assert_parity(run(tf, "gemv", d, pack(tf, d), workspace=ws), ref(d),
                      f"shared workspace, case {i}: W{bits} {M}x{K}x{N}")


@pytest.mark.parametrize("bits,M,K,N,G", [(4, 16, 2048, 2048, 128), (8, 11, 4096, 520, 64),
                                           (4, 12, 16384, 512, 128), (8, 16, 14336, 1024, 128),
                                           (4, 1300, 2048, 1000, 128), (8, 1520, 1024, 776, 64),
                                           (4, 2048, 1024, 4096, 32), (4, 1100, 3072, 2320, 128),
                                           # 128-row tiles split along K (few tiles, long K)
                                           (4, 200, 12288, 1024, 128), (8, 100, 16384, 520, 64),
                                           (8, 40, 8192, 264, 32), (4, 64, 8192, 1024, 128),
                                           (8, 40, 4096, 4096, 128), (8, 256, 4096, 4096, 128),
                                           # 64 x 128 tiles with K over the waves (no workspace either way)
                                           (8, 512, 4096, 4096, 128), (4, 100, 4096, 3000, 128),
                                           (4, 300, 2048, 520, 64), (4, 700, 1536, 1000, 128),
                                           (4, 100, 4096, 9400, 128)])
def test_gemm_workspace_modes(tf, bits, M, K, N, G):
    """The K-split kernels (workspace: stream-K for 256-row tiles, split-K for
    128-row tiles) and the whole-tile kernels (no workspace) both meet the
    bar; a split result is bitwise repeatable and its workspace serves the
    next call at once."""
    d = make_inputs(bits, M, K, N, group=G, seed=M + N)
    packed = pack(tf, d)
    want = ref(d)
    need = tf.workspace_bytes(bits, M, K, N, G)
    ws = torch.zeros(need + 256, dtype=torch.uint8, device="cuda") if need else False
    a = run(tf, "gemm", d, packed, workspace=ws)
    b = run(tf, "gemm", d, packed, workspace=ws)
    np.testing.assert_array_equal(a.view(np.uint16), b.view(np.uint16))
    c = run(tf, "gemm", d, packed, workspace=False)
    assert_parity(a, want, f"gemm W{bits} {M}x{K}x{N} with workspace")
    assert_parity(c, want, f"gemm W{bits} {M}x{K}x{N} without workspace")


def test_workspace_shared_gemm_gemv(tf):
    """One workspace serves split-K GEMVs and stream-K GEMMs in turn."""
    cases = [("gemm", 4, 1300, 1024, 1000), ("gemv", 4, 1, 14336, 4096), ("gemm", 8, 1600, 2048, 520),
             ("gemv", 8, 3, 8192, 520), ("gemm", 4, 1300, 1024, 1000), ("gemm", 8, 300, 4096, 1024),
             ("gemm", 4, 12, 8192, 512), ("gemm", 4, 200, 2048, 2000)]
    need = max(tf.workspace_bytes(b, m, k, n) for _, b, m, k, n in cases)
    ws = torch.zeros(need, dtype=torch.uint8, device="cuda")
    for i, (kind, bits, M, K, N) in enumerate(cases):
        d = make_inputs(bits, M, K, N, seed=200 + i)
        assert_parity(run(tf, kind, d, pack(tf, d), workspace=ws), ref(d),
                      f"shared workspace, case {i}: {kind} W{bits} {M}x{K}x{N}")


@pytest.mark.parametrize("kind,M", [("gemv", 1), ("gemv", 8), ("gemm", 300), ("gemm", 1300)])
def test_bitwise_reproducible(tf, kind, M):
    d = make_inputs(4, M, 2048, 1024, seed=5)
    packed = pack(tf, d)
    a = run(tf, kind, d, packed)
    b = run(tf, kind, d, packed)
    np.testing.assert_array_equal(a.view(np.uint16), b.view(np.uint16))


# ---------------------------------------------------------------------------
# the Llama-shaped workloads at full size
# ---------------------------------------------------------------------------
def _sample_cols(N, rng, n=256):
    return np.sort(rng.choice(N, size=min(n, N), replace=False))


@pytest.mark.parametrize("M", [1, 4, 8])
def test_gemv_w4_k4096_n14336_full(tf, M):
    d = make_inputs(4, M, 4096, 14336, seed=0)
    assert_parity(run(tf, "gemv", d, pack(tf, d)), ref(d), f"W4 GEMV M={M}")


def test_w8_k4096_n4096_full(tf):
    d = make_inputs(8, 1, 4096, 4096, seed=0)
    assert_parity(run(tf, "gemv", d, pack(tf, d)), ref(d), "W8 GEMV M=1")
    d = make_inputs(8, 512, 4096, 4096, seed=0)
    assert_parity(run(tf, "gemm", d, pack(tf, d)), ref(d), "W8 GEMM M=512")


def test_gemm_w4_m16_k2048_n2048_full(tf):
    d = make_inputs(4, 16, 2048, 2048, seed=0)
    assert_parity(run(tf, "gemm", d, pack(tf, d)), ref(d), "W4 GEMM M=16")


def ref_blocked(d, x=None, block=2048):
    """The oracle over all of C, computed one block of output columns at a
    time (the float64 weight of a 32K-row shape would otherwise need
    gigabytes); each block is the same plain dequant + matmul as ``ref``."""
    x = d["x"] if x is None else x
    N = d["N"]
    out = np.empty((x.shape[0], N), dtype=np.float64)
    for c0 in range(0, N, block):
        cols = np.arange(c0, min(N, c0 + block))
        out[:, cols] = ref(d, x=x, cols=cols)
    return out


@pytest.mark.slow
@pytest.mark.parametrize("M,K,N,xstd", [(2048, 4096, 14336, 1.0), (2048, 14336, 4096, 1.0),
                                         (1024, 4096, 32768, 0.5), (1024, 32768, 8192, 0.5)])
def test_gemm_w4_large_full(tf, M, K, N, xstd):
    """The prefill workloads at full size (M = 2048 at both Llama-3-8B MLP
    shapes; M = 1024 at the 32K-dimension shapes) in the launch configuration
    the benchmark times (the default workspace), compared over every element
    of C against the oracle."""
    d = make_inputs(4, M, K, N, seed=0, x_std=xstd)
    got = run(tf, "gemm", d, pack(tf, d))
    assert_parity(got, ref_blocked(d), f"W4 GEMM {M}x{K}x{N} full")


@pytest.mark.slow
@pytest.mark.parametrize("M,K,N,xstd", [(2048, 4096, 14336, 1.0), (1024, 32768, 8192, 0.5)])
def test_gemm_w4_large_full_no_workspace(tf, M, K, N, xstd):
    """The same two workloads through the kernels that do not split K (no
    workspace): every element of C."""
    d = make_inputs(4, M, K, N, seed=1, x_std=xstd)
    got = run(tf, "gemm", d, pack(tf, d), workspace=False)
    assert_parity(got, ref_blocked(d), f"W4 GEMM {M}x{K}x{N} full, no workspace")


@pytest.mark.slow
def test_gemm_hybrid_one_chunk_per_block(tf):
    """264 tiles of 256 x 256 (M=2048, N=8448) at K=4096, 32 K chunks per tile,
    on 256 blocks: one whole wave of tiles, then the last 8 tiles split over
    all blocks, one K chunk each (32 segments per tile, summed by the
    reduction launch), the smallest remainder the hybrid schedule takes.  All
    of C against the oracle."""
    d = make_inputs(4, 2048, 4096, 8448, seed=5)
    assert_parity(run(tf, "gemm", d, pack(tf, d)), ref(d), "W4 GEMM hybrid, one K chunk per block")


@pytest.mark.slow
@pytest.mark.parametrize("M", [256, 1280, 4352, 8192])
@pytest.mark.parametrize("K,N", [(4096, 14336), (14336, 4096)])
def test_gemm_w4_msweep_sampled(tf, M, K, N):
    """Points of the paper's prompt-length sweep (M = 256..8192 step 256, both
    Llama-3-8B MLP shapes) at full size: sampled rows x columns against the
    oracle, all of C finite.  Covers the 64 x 128 kernel with K split over the
    workgroup's waves (M = 256, K = 4096), the 256-row kernel in whole-tile and
    stream-K forms and the largest M."""
    d = make_inputs(4, M, K, N, seed=M)
    got = run(tf, "gemm", d, pack(tf, d))
    assert np.all(np.isfinite(got.astype(np.float64)))
    rng = np.random.default_rng(M + K)
    rows = np.unique(np.concatenate([[0, M - 1], rng.choice(M, size=24, replace=False)]))
    cols = np.unique(np.concatenate([[0, N - 1], _sample_cols(N, rng, 254)]))
    want = ref(d, x=d["x"][rows], cols=cols)
    assert_parity(got[np.ix_(rows, cols)], want, f"W4 GEMM sweep {M}x{K}x{N} sampled")
