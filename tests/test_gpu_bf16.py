"""GPU parity of the BF16 entry points (BF16 activations and scales, the
paper's dtype) against the BF16 oracle, through the C ABI.

Bars:
  * dequant (tf_dequant, TF_BF16): bit-exact against RNE_bf16(s * (q - z)),
    zeros compared as values (the kernel forms s * q - z * s, whose exact zero
    is +0 where s * (q - z) with a negative scale gives -0);
  * matmul: max|gpu - oracle| <= 1e-2 * max|oracle| per output matrix (the
    stated tolerance) against the paper's arithmetic (each weight rounded to
    BF16), and, per element, |gpu - ref| <= 2^-8 |ref| + 1e-4 max|ref| (the
    output's own bfloat16 rounding is at most 2^-8 of the element; the fp32
    sums add far less than 1e-4 of the largest output, while one dropped K
    term is about max / sqrt(K)).  ref is the same oracle for the kernels
    that round each weight to BF16 before the multiply (tiled GEMMs, the
    64-slot streaming form, the GEMV from 5 rows); the factored forms (GEMV up
    to 4 rows, streaming matrix-core form up to 32 rows) apply the scale to a
    group's sums and never round a weight, so their ref is the exact
    contraction (Eq. 2 in float64 with the BF16 inputs);
  * integer invariant (s = 1, z = 0, integer activations): bit-exact against
    RNE_bf16 of the exact integer matmul;
  * canaries around every output.
Every kernel family runs: decode GEMV (M <= 8, both entry points for M <= 3),
the streaming matrix-core form (4 <= M <= 64), the 128-row GEMM (with and
without split-K, every metadata-per-chunk case and the generic kernel) and
the 256-row GEMM (whole tiles and stream-K).
"""
from __future__ import annotations

import numpy as np
import pytest

import oracle
from paper_2606_11357_amd.synth import make_inputs_bf16, pack_nibbles

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

TOL = 1e-2
REL_ELEM = 2.0 ** -8
ABS_ELEM = 1e-4
GUARD = 4096
CANARY = 0xC0E0            # bfloat16 -7.0


@pytest.fixture(scope="module")
def tf():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2606_11357_amd import tilefuse
    tilefuse.load()
    return tilefuse


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def dev_bf16(bits):
    """uint16 bfloat16 patterns -> a CUDA bfloat16 tensor with those bits."""
    return dev(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16)


def pack(tf, d):
    K, N, G = d["K"], d["N"], d["group"]
    s = dev(d["s_bits"].view(np.int16))           # the pack copies the 16-bit patterns
    if d["bits"] == 4:
        return tf.pack_w4(dev(d["qweight"]), dev(d["qzeros"]), s, K, N, G)
    return tf.pack_w8(dev(d["qweight"]), dev(d["zeros"]), s, K, N, G)


def run(tf, kind, d, packed, x_bits=None, workspace=None):
    K, N, G = d["K"], d["N"], d["group"]
    x_bits = d["x_bits"] if x_bits is None else x_bits
    M = x_bits.shape[0]
    buf = torch.full((M * N + 2 * GUARD,), int(np.uint16(CANARY).view(np.int16)), dtype=torch.int16,
                     device="cuda")
    out = buf[GUARD:GUARD + M * N].view(torch.bfloat16).view(M, N)
    fn = getattr(tf, f"w{d['bits']}a16_{kind}")
    fn(dev_bf16(x_bits), packed, K, N, G, out=out, workspace=workspace)
    torch.cuda.synchronize()
    b = buf.cpu().numpy().view(np.uint16)
    assert np.all(b[:GUARD] == CANARY) and np.all(b[-GUARD:] == CANARY), "write outside the output"
    return b[GUARD:GUARD + M * N].reshape(M, N)


def ref(d, x_bits=None, cols=None, exact=False):
    """The oracle: weights rounded to BF16 (the paper's arithmetic), or with
    exact=True the exact contraction of the same BF16 inputs."""
    x_bits = d["x_bits"] if x_bits is None else x_bits
    q, z, s = d["q"], d["z"], d["s_bits"]
    if cols is not None:
        q, z, s = q[:, cols], z[:, cols], s[:, cols]
    w = (oracle.dequant(q, z, oracle.bf16_decode(s), d["group"]) if exact
         else oracle.dequant_bf16(q, z, s, d["group"]))
    return oracle.matmul(oracle.bf16_decode(x_bits), w)


def factored(kind, M):
    """Whether the call runs a factored form that never rounds a weight: the
    decode GEMV up to 4 rows; through the GEMM entry, the GEMV (up to 3 rows)
    and the matrix-core streaming form with 16 or 32 row slots (up to 32)."""
    return M <= 4 if kind == "gemv" else M <= 32


def check(got, d, kind, what, cols=None):
    want = ref(d, cols=cols)
    path = ref(d, cols=cols, exact=True) if factored(kind, d["x_bits"].shape[0]) else want
    return assert_parity(got, want, what, path)


def assert_bf16_equal(got_bits, want_bits):
    """Equal values (so +0 == -0) and identical bits for every nonzero value."""
    gv, wv = oracle.bf16_decode(got_bits), oracle.bf16_decode(want_bits)
    np.testing.assert_array_equal(gv, wv)
    nz = wv != 0
    np.testing.assert_array_equal(got_bits[nz], want_bits[nz])


def assert_parity(gpu_bits, want, what="", path=None):
    gpu = oracle.bf16_decode(gpu_bits)
    assert np.all(np.isfinite(gpu)), what
    scale = np.abs(want).max()
    err = np.abs(gpu - want)
    assert err.max() <= TOL * scale, f"{what}: max err {err.max():.4g} > {TOL} * {scale:.4g}"
    path = want if path is None else path
    err = np.abs(gpu - path)
    bound = REL_ELEM * np.abs(path) + ABS_ELEM * np.abs(path).max()
    bad = np.argwhere(err > bound)
    assert bad.size == 0, f"{what}: {len(bad)} elements past the per-element bound, first {bad[0]}"
    return err.max() / scale


# ---------------------------------------------------------------------------
# dequant: bit-exact
# ---------------------------------------------------------------------------
SMALL = [(4, 256, 136, 128), (4, 128, 64, 32), (4, 2048, 2048, 128), (8, 256, 40, 128),
         (8, 192, 96, 64), (8, 4096, 4096, 128), (4, 96, 8, 32)]


@pytest.mark.parametrize("bits,K,N,G", SMALL)
def test_dequant_bf16_bitexact(tf, bits, K, N, G):
    d = make_inputs_bf16(bits, 1, K, N, group=G, seed=K * 5 + N)
    w = tf.dequant(bits, pack(tf, d), K, N, G, dtype=torch.bfloat16)
    got = w.view(torch.int16).cpu().numpy().view(np.uint16)
    want = oracle.bf16_encode(oracle.dequant_bf16(d["q"], d["z"], d["s_bits"], G))
    assert_bf16_equal(got, want)


@pytest.mark.parametrize("bits", [4, 8])
def test_dequant_bf16_extreme_scales(tf, bits):
    """Every code against random zero-points and scales from bfloat16
    subnormals to 2^97, both signs (the exact fp32 form needs z * s finite
    in fp32, i.e. |s| below about 2^119)."""
    qmax = (1 << bits) - 1
    K, G = 256 if bits == 8 else 32, 32
    N = 64
    rng = np.random.default_rng(98)
    q = np.tile(np.arange(K, dtype=np.int64)[:, None] % (qmax + 1), (1, N)).astype(np.uint8)
    z = rng.integers(0, qmax + 1, size=(K // G, N), dtype=np.uint8)
    sb = np.array([0x0001, 0x0002, 0x007F, 0x0080, 0x3F80, 0x3F81, 0x4300, 0x7000,
                   0x8001, 0xBF80, 0x0155, 0x1A2B, 0x2E66, 0x5000, 0x0010, 0xC37F], dtype=np.uint16)
    s_bits = np.tile(sb, (K // G, N // sb.size))
    d = {"bits": bits, "K": K, "N": N, "group": G, "q": q, "z": z, "s_bits": s_bits}
    if bits == 4:
        d["qweight"], d["qzeros"] = pack_nibbles(q), pack_nibbles(z)
    else:
        d["qweight"], d["zeros"] = q, z
    w = tf.dequant(bits, pack(tf, d), K, N, G, dtype=torch.bfloat16)
    got = w.view(torch.int16).cpu().numpy().view(np.uint16)
    assert_bf16_equal(got, oracle.bf16_encode(oracle.dequant_bf16(q, z, s_bits, G)))


# ---------------------------------------------------------------------------
# matmul parity, every kernel family
# ---------------------------------------------------------------------------
GEMM_CASES = [
    # bits, M, K, N, G
    (4, 1, 1024, 1024, 128), (4, 3, 2048, 520, 128),                   # GEMV through the GEMM entry
    (4, 4, 2048, 520, 128), (4, 16, 1024, 1024, 64), (4, 17, 1024, 1032, 128),
    (4, 33, 4096, 264, 128), (4, 64, 1024, 1024, 32),                  # streaming matrix-core form
    (4, 65, 1024, 1032, 128), (4, 300, 2048, 1024, 64), (4, 200, 1024, 1024, 32),
    (4, 777, 4096, 2056, 128),                                         # 64 x 128 GEMM, K over the waves
    (4, 1000, 3968, 4088, 32), (4, 512, 4096, 14336, 128),             # ... 64 x 256 tiles
    (4, 300, 4096, 11008, 64),
    (4, 200, 12288, 264, 128), (4, 130, 480, 264, 96),                 # 128-row GEMM, generic kernel
    (4, 1024, 1024, 2048, 128), (4, 2048, 2048, 4096, 128), (4, 1100, 1024, 1000, 128),
    (4, 4096, 1024, 4096, 128),                                        # 256-row GEMM
    (4, 300, 8192, 520, 128), (8, 600, 8192, 264, 64),                 # 256-row GEMM, 256 <= M < 1024, long K
    (8, 1, 1024, 1024, 128), (8, 8, 2048, 520, 128), (8, 33, 1024, 1024, 64),
    (8, 512, 4096, 4096, 128), (8, 129, 1024, 264, 32), (8, 1024, 1024, 4096, 128),
    (8, 2048, 2048, 2048, 64),
    (8, 384, 1152, 4088, 64), (8, 420, 640, 3968, 32),                 # 64 x 128 GEMM, 8-bit, ragged N / M
    (4, 1100, 512, 13304, 64),                                         # 256-row whole tiles + 64 x 128 rest
]


@pytest.mark.parametrize("ws", [True, False], ids=["ws", "nows"])
@pytest.mark.parametrize("bits,M,K,N,G", GEMM_CASES)
def test_gemm_bf16(tf, bits, M, K, N, G, ws):
    d = make_inputs_bf16(bits, M, K, N, group=G, seed=M * 7 + K + N + G)
    got = run(tf, "gemm", d, pack(tf, d), workspace=None if ws else False)
    check(got, d, "gemm", f"gemm bf16 w{bits} M={M} K={K} N={N} G={G} ws={ws}")


GEMV_CASES = [(4, 4096, 1032, 128), (8, 4096, 1032, 128), (4, 14336, 512, 128),
              (8, 14336, 512, 128), (4, 1024, 264, 64), (8, 2048, 136, 32), (4, 480, 264, 96)]


@pytest.mark.parametrize("M", [1, 2, 3, 4, 5, 6, 7, 8])
@pytest.mark.parametrize("bits,K,N,G", GEMV_CASES)
def test_gemv_bf16(tf, bits, M, K, N, G):
    d = make_inputs_bf16(bits, M, K, N, group=G, seed=M + K + N + G)
    packed = pack(tf, d)
    for ws in (None, False):
        got = run(tf, "gemv", d, packed, workspace=ws)
        check(got, d, "gemv", f"gemv bf16 w{bits} M={M} K={K} N={N} G={G} ws={ws is None}")


@pytest.mark.parametrize("bits,kind,M,K,N", [(4, "gemv", 1, 4096, 1032), (8, "gemv", 4, 4096, 520),
                                              (4, "gemm", 16, 4096, 1024), (8, "gemm", 64, 2048, 520),
                                              (4, "gemm", 512, 2048, 1024), (4, "gemm", 1024, 2048, 4096),
                                              (8, "gemm", 2048, 1024, 2048)])
def test_integer_invariant_bf16(tf, bits, kind, M, K, N):
    """s = 1, z = 0, integer activations: bit-exact RNE_bf16 of the integer matmul."""
    rng = np.random.default_rng(M + K)
    xi = rng.integers(-3, 4, size=(M, K))
    qi = rng.integers(0, 1 << bits, size=(K, N), dtype=np.uint8)
    G = 128
    x_bits = (xi.astype(np.float32).view(np.uint32) >> 16).astype(np.uint16)
    d = {"bits": bits, "K": K, "N": N, "group": G, "x_bits": x_bits,
         "s_bits": np.full((K // G, N), 0x3F80, dtype=np.uint16)}
    z = np.zeros((K // G, N), dtype=np.uint8)
    if bits == 4:
        d["qweight"], d["qzeros"] = pack_nibbles(qi), pack_nibbles(z)
    else:
        d["qweight"], d["zeros"] = qi, z
    got = run(tf, kind, d, pack(tf, d))
    exact = (xi.astype(np.int64) @ qi.astype(np.int64)).astype(np.float64)
    assert_bf16_equal(got, oracle.bf16_encode(oracle.to_bf16(exact)))


def check_blocked(got, d, kind, what, block=2048):
    """``check`` over all of C, the oracle computed one block of output
    columns at a time (bounded host memory at the 32K-dimension shapes); the
    stated tolerance is applied to the whole matrix, the per-element bound to
    every element."""
    N = d["N"]
    want = np.empty(got.shape, dtype=np.float64)
    path = np.empty(got.shape, dtype=np.float64) if factored(kind, d["x_bits"].shape[0]) else want
    for c0 in range(0, N, block):
        cols = np.arange(c0, min(N, c0 + block))
        want[:, cols] = ref(d, cols=cols)
        if path is not want:
            path[:, cols] = ref(d, cols=cols, exact=True)
    return assert_parity(got, want, what, path)


@pytest.mark.slow
@pytest.mark.parametrize("M,K,N,xstd", [(2048, 4096, 14336, 1.0), (2048, 14336, 4096, 1.0),
                                         (1024, 4096, 32768, 0.5), (1024, 32768, 8192, 0.5)])
def test_gemm_bf16_full_size(tf, M, K, N, xstd):
    """The Llama-3-8B MLP shapes at M = 2048 and the 32K-dimension shapes at
    M = 1024, in the benchmark's launch configuration (default workspace):
    every element of C."""
    G = 128
    d = make_inputs_bf16(4, M, K, N, group=G, seed=K + 2 * N, x_std=xstd)
    got = run(tf, "gemm", d, pack(tf, d))
    check_blocked(got, d, "gemm", f"gemm bf16 M={M} K={K} N={N} full")


def test_gemm_bf16_hybrid_one_chunk_per_block(tf):
    """264 tiles of 256 x 256 (M=2048, N=8448) at K=4096 on 256 blocks: one
    whole wave, then the last 8 tiles split over all blocks one K chunk each,
    summed by the reduction launch in its BF16 form.  All of C."""
    d = make_inputs_bf16(4, 2048, 4096, 8448, group=128, seed=11)
    check(run(tf, "gemm", d, pack(tf, d)), d, "gemm", "gemm bf16 hybrid, one K chunk per block")


def test_gemv_bf16_full_size(tf):
    """The decode GEMV at K = 4096, N = 14336 (M = 1), every output."""
    d = make_inputs_bf16(4, 1, 4096, 14336, group=128, seed=3)
    got = run(tf, "gemv", d, pack(tf, d))
    check(got, d, "gemv", "gemv bf16 M=1 K=4096 N=14336")


def test_bf16_and_fp16_agree_on_shared_values(tf):
    """Activations and scales representable in both formats (short mantissas,
    moderate exponents): the BF16 and fp16 entry points compute the same
    products; their outputs differ only by their own roundings."""
    from paper_2606_11357_amd.synth import make_inputs
    M, K, N, G = 64, 2048, 1024, 128
    d = make_inputs(4, M, K, N, group=G, seed=5)
    x16 = d["x"].astype(np.float32)
    x16 = (x16.view(np.uint32) & np.uint32(0xFFFF0000)).view(np.float32)          # 8 significant bits
    s16 = (d["s"].astype(np.float32).view(np.uint32) & np.uint32(0xFFFF0000)).view(np.float32)
    db = dict(d, x_bits=(x16.view(np.uint32) >> 16).astype(np.uint16),
              s_bits=(s16.view(np.uint32) >> 16).astype(np.uint16))
    got_bf = oracle.bf16_decode(run(tf, "gemm", db, pack(tf, db)))
    dh = dict(d, x=x16.astype(np.float16), s=s16.astype(np.float16))
    ph = tf.pack_w4(dev(dh["qweight"]), dev(dh["qzeros"]), dev(dh["s"]), K, N, G)
    got_h = tf.w4a16_gemm(dev(dh["x"]), ph, K, N, G).float().cpu().numpy().astype(np.float64)
    scale = np.abs(got_h).max()
    assert np.abs(got_bf - got_h).max() <= 2.0 ** -7 * scale
