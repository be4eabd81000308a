"""Pins for the CPU oracle: facts fixed by the paper's definitions and by
mathematics, independent of the oracle's own code.

Every ``check_*`` function takes a namespace with the oracle's steps
(``unpack_w4``, ``dequant``, ``matmul``, ``to_f16``) so that the same checks
also run against deliberately broken copies (planted on the CPU, bottom of this
file): each planted mistake must be caught by at least one check.

Citations: Eq. 1 / Eq. 2 (Section 2.2) for dequantization, Section 2.1 for the
C = A x B orientation, Section 4.3 for unpacking by mask and shift, Section 4.2
and Section 2.2 for the group of G = 128 weights of one column.
"""
from __future__ import annotations

import os
import types
from fractions import Fraction

import numpy as np
import pytest

import oracle
from paper_2606_11357_amd.synth import make_inputs, pack_nibbles

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")

REAL = types.SimpleNamespace(unpack_w4=oracle.unpack_w4, dequant=oracle.dequant,
                             matmul=oracle.matmul, to_f16=oracle.to_f16)


# --------------------------------------------------------------------------
# independent helpers (exact arithmetic, written from the number formats)
# --------------------------------------------------------------------------
def f16_value(bits: int) -> Fraction:
    """Exact value of an IEEE binary16 bit pattern (finite only)."""
    sign = -1 if bits & 0x8000 else 1
    e = (bits >> 10) & 0x1F
    f = bits & 0x3FF
    assert e != 0x1F, "non-finite"
    if e == 0:
        return sign * Fraction(f, 1 << 24)
    return sign * Fraction(1024 + f, 1024) * (Fraction(2) ** (e - 15))


def rne_f16_bits(v: Fraction) -> int:
    """Round an exact rational to binary16, nearest-even, overflow to inf."""
    sign = 0x8000 if v < 0 else 0
    a = abs(v)
    if a == 0:
        return sign
    e = 0
    while a >= Fraction(2) ** (e + 1):
        e += 1
    while a < Fraction(2) ** e:
        e -= 1
    e = max(e, -14)
    ulp = Fraction(2) ** (e - 10)
    m = a / ulp
    n = m.numerator // m.denominator
    rem = m - n
    if rem > Fraction(1, 2) or (rem == Fraction(1, 2) and n % 2 == 1):
        n += 1
    if n == 2048:
        n //= 2
        e += 1
    if e > 15:
        return sign | 0x7C00
    if n < 1024:                      # subnormal (e == -14)
        return sign | n
    return sign | ((e + 15) << 10) | (n - 1024)


def _f16_bits(a) -> np.ndarray:
    return np.asarray(a, dtype=np.float16).view(np.uint16)


def _y(ns, x, qw, qz, s, G, bits=4, zeros=None):
    if bits == 4:
        q, z = ns.unpack_w4(qw), ns.unpack_w4(qz)
    else:
        q, z = qw, zeros
    return ns.matmul(x, ns.dequant(q, z, s, G))


# --------------------------------------------------------------------------
# checks
# --------------------------------------------------------------------------
def check_unpack_golden(ns):
    """Hand-derived words of the boundary format (tests/golden/awq_words.txt)."""
    words, codes = [], []
    for line in open(os.path.join(GOLDEN, "awq_words.txt")):
        line = line.split("#", 1)[0].split()
        if not line:
            continue
        words.append(np.uint32(int(line[0], 16)))
        codes.append([int(c) for c in line[1:]])
    w = np.array(words, dtype=np.uint32).view(np.int32).reshape(-1, 1)
    got = ns.unpack_w4(w)
    assert got.shape == (len(codes), 8)
    np.testing.assert_array_equal(got, np.array(codes, dtype=np.uint8))
    # the same words laid out along a row: word j covers columns 8j..8j+7
    got_row = ns.unpack_w4(w.reshape(1, -1))
    np.testing.assert_array_equal(got_row.reshape(-1, 8), np.array(codes, dtype=np.uint8))


def check_unpack_roundtrip(ns):
    """Generator's packer (shift-or) -> oracle's unpacker returns the drawn codes."""
    rng = np.random.default_rng(123)
    for r, n in [(1, 8), (3, 64), (130, 136), (7, 2048)]:
        c = rng.integers(0, 16, size=(r, n), dtype=np.uint8)
        c[0, :8] = [15, 0, 15, 0, 0, 0, 0, 15]          # bit 31 set in word 0
        np.testing.assert_array_equal(ns.unpack_w4(pack_nibbles(c)), c)


def check_dequant_exact(ns):
    """Eq. 2 against exact rationals; its fp16 rounding against binary16 RNE."""
    rng = np.random.default_rng(7)
    scale_bits = np.concatenate([
        rng.integers(0x1800, 0x2600, size=96),        # ~0.0003 .. 0.02 (normal range)
        np.array([0x3C00, 0x0001, 0x03FF, 0x0400, 0x7BFF, 0xBC00, 0x2118, 0x251F]),
    ]).astype(np.uint16)
    G = 2
    for bits in (4, 8):
        qmax = (1 << bits) - 1
        qs = np.array([0, 1, 2, qmax // 2, qmax - 1, qmax], dtype=np.uint8)
        zs = np.array([0, 1, qmax // 2 + 1, qmax], dtype=np.uint8)
        # one column per scale; rows enumerate (q, z) pairs, two rows per group
        pairs = [(a, b) for a in qs for b in zs]
        K = 2 * len(pairs)
        q = np.zeros((K, scale_bits.size), dtype=np.uint8)
        z = np.zeros((K // G, scale_bits.size), dtype=np.uint8)
        for i, (a, b) in enumerate(pairs):
            q[2 * i, :] = a
            q[2 * i + 1, :] = b            # second row of the group: q == z -> exact 0
            z[i, :] = b
        s = np.tile(scale_bits.view(np.float16), (K // G, 1))
        w = ns.dequant(q, z, s, G)
        assert w.shape == (K, scale_bits.size)
        for i, (a, b) in enumerate(pairs):
            for c, sb in enumerate(scale_bits):
                exact = f16_value(int(sb)) * (int(a) - int(b))
                assert Fraction(float(w[2 * i, c])) == exact
                assert float(w[2 * i + 1, c]) == 0.0
                got = int(_f16_bits(ns.to_f16(w[2 * i:2 * i + 1, c]))[0])
                if exact == 0:          # IEEE sign of a zero product follows the scale
                    assert got & 0x7FFF == 0
                else:
                    assert got == rne_f16_bits(exact)
        # exact in float32 as well (the fp32 dequant of the library must equal it)
        np.testing.assert_array_equal(w.astype(np.float32).astype(np.float64), w)


def check_rounding_golden(ns):
    """Hand-derived binary16 roundings (tests/golden/fp16_rounding.txt)."""
    for line in open(os.path.join(GOLDEN, "fp16_rounding.txt")):
        line = line.split("#", 1)[0].split()
        if not line:
            continue
        v = Fraction(line[0])
        want = int(line[1], 16)
        assert rne_f16_bits(v) == want, line          # the helper agrees with the table
        got = int(_f16_bits(ns.to_f16(np.array([float(v)])))[0])
        assert got == want, (line, hex(got))


def check_special_cases(ns):
    """Eq. 1 as the z = 0 case; s = 1, z = 0 returns the code itself."""
    rng = np.random.default_rng(3)
    K, N, G = 64, 16, 32
    q = rng.integers(0, 256, size=(K, N), dtype=np.uint8)
    z0 = np.zeros((K // G, N), dtype=np.uint8)
    one = np.ones((K // G, N), dtype=np.float16)
    np.testing.assert_array_equal(ns.dequant(q, z0, one, G), q.astype(np.float64))
    s = rng.uniform(0.01, 0.02, size=(K // G, N)).astype(np.float16)
    sym = ns.dequant(q, z0, s, G)
    np.testing.assert_array_equal(sym, np.repeat(s.astype(np.float64), G, axis=0) * q)


def check_group_onehot(ns):
    """Weight (k0, n0) alone has q - z = 1: y[:, n0] = x[:, k0] * s[k0 // G, n0], rest 0.

    Fixes the group index (groups run along K inside one column), the
    orientation of C = A x B and the sign of q - z, without reusing the oracle.
    """
    rng = np.random.default_rng(11)
    M, K, N, G = 3, 256, 24, 64
    x = rng.standard_normal((M, K)).astype(np.float16)
    s = (2.0 ** rng.integers(-8, 2, size=(K // G, N))).astype(np.float16)
    zc = rng.integers(0, 15, size=(K // G, N), dtype=np.uint8)
    for k0, n0 in [(0, 0), (63, 5), (64, 5), (130, 17), (255, 23), (191, 8)]:
        q = np.repeat(zc, G, axis=0).copy()               # q == z everywhere
        q[k0, n0] += 1
        y = _y(ns, x, pack_nibbles(q), pack_nibbles(zc), s, G)
        want = np.zeros((M, N))
        want[:, n0] = x[:, k0].astype(np.float64) * float(s[k0 // G, n0])
        np.testing.assert_array_equal(y, want)


def check_matmul_bruteforce(ns):
    """Exact rational sums on tiny shapes, element by element in pure Python."""
    for (M, K, N, G, bits, seed) in [(1, 128, 8, 128, 4, 0), (3, 256, 16, 128, 4, 1),
                                     (3, 128, 8, 32, 4, 2), (2, 64, 8, 32, 8, 3),
                                     (1, 256, 16, 64, 8, 4)]:
        d = make_inputs(bits, M, K, N, group=G, seed=seed)
        y = _y(ns, d["x"], d["qweight"], d.get("qzeros"), d["s"], G, bits, d.get("zeros"))
        assert y.shape == (M, N)
        xs = [[Fraction(float(v)) for v in row] for row in d["x"]]
        ss = [[f16_value(int(b)) for b in row] for row in d["s"].view(np.uint16)]
        for m in range(M):
            for n in range(N):
                tot, absum = Fraction(0), Fraction(0)
                for k in range(K):
                    g = k // G
                    t = xs[m][k] * ss[g][n] * (int(d["q"][k, n]) - int(d["z"][g, n]))
                    tot += t
                    absum += abs(t)
                bound = K * 2.0 ** -52 * float(absum)
                assert abs(float(y[m, n]) - float(tot)) <= bound, (M, K, N, G, m, n)


def check_integer_invariant(ns):
    """s = 1, z = 0, integer activations: the result is an exact integer matmul."""
    rng = np.random.default_rng(5)
    for bits, K, N, G in [(8, 512, 64, 128), (4, 1024, 48, 128), (8, 4096, 16, 128)]:
        M = 4
        xi = rng.integers(-3, 4, size=(M, K))
        qi = rng.integers(0, 1 << bits, size=(K, N), dtype=np.uint8)
        x = xi.astype(np.float16)
        s = np.ones((K // G, N), dtype=np.float16)
        z = np.zeros((K // G, N), dtype=np.uint8)
        if bits == 4:
            y = _y(ns, x, pack_nibbles(qi), pack_nibbles(z), s, G)
        else:
            y = _y(ns, x, qi, None, s, G, 8, z)
        want = xi.astype(np.int64) @ qi.astype(np.int64)
        np.testing.assert_array_equal(y, want.astype(np.float64))


def check_closed_forms(ns):
    """x = 1, per-group constant q, z, s: y = sum_g G * (c_g - d_g) * s_g."""
    M, K, N, G = 2, 512, 16, 128
    ng = K // G
    c = np.array([15, 3, 0, 9], dtype=np.uint8)
    d = np.array([1, 3, 15, 0], dtype=np.uint8)
    sv = np.array([0.0078125, 0.5, 0.015625, 2.0], dtype=np.float16)
    x = np.ones((M, K), dtype=np.float16)
    q = np.repeat(np.repeat(c[:, None], N, axis=1), G, axis=0)
    z = np.repeat(d[:, None], N, axis=1)
    s = np.repeat(sv[:, None], N, axis=1)
    y = _y(ns, x, pack_nibbles(q), pack_nibbles(z), s, G)
    want = sum(G * (int(c[g]) - int(d[g])) * float(sv[g]) for g in range(ng))
    np.testing.assert_array_equal(y, np.full((M, N), want))
    # q == z everywhere gives exactly zero
    y0 = _y(ns, x, pack_nibbles(np.repeat(z, G, axis=0)), pack_nibbles(z), s, G)
    np.testing.assert_array_equal(y0, np.zeros((M, N)))


def check_linearity(ns):
    """Linear in x; scaling every scale by 2^e scales y by 2^e exactly."""
    d = make_inputs(4, 3, 256, 32, group=128, seed=9)
    y = _y(ns, d["x"], d["qweight"], d["qzeros"], d["s"], 128)
    x2 = make_inputs(4, 3, 256, 32, group=128, seed=10)["x"]
    y2 = _y(ns, x2, d["qweight"], d["qzeros"], d["s"], 128)
    ysum = _y(ns, d["x"].astype(np.float64) + x2.astype(np.float64), d["qweight"],
              d["qzeros"], d["s"], 128)
    np.testing.assert_allclose(ysum, y + y2, rtol=0, atol=1e-12 * np.abs(y).max())
    y4 = _y(ns, d["x"], d["qweight"], d["qzeros"], (d["s"] * np.float16(4)), 128)
    np.testing.assert_array_equal(y4, 4 * y)


CHECKS = [check_unpack_golden, check_unpack_roundtrip, check_dequant_exact,
          check_rounding_golden, check_special_cases, check_group_onehot,
          check_matmul_bruteforce, check_integer_invariant, check_closed_forms,
          check_linearity]


@pytest.mark.parametrize("check", CHECKS, ids=lambda f: f.__name__)
def test_oracle_pin(check):
    check(REAL)


def test_composed_entry_points_match_steps():
    """oracle.w4a16 / w8a16 are exactly unpack -> dequant -> matmul."""
    for bits in (4, 8):
        d = make_inputs(bits, 2, 256, 64, group=128, seed=21)
        if bits == 4:
            y = oracle.w4a16(d["x"], d["qweight"], d["qzeros"], d["s"], 128)
            y_steps = _y(REAL, d["x"], d["qweight"], d["qzeros"], d["s"], 128)
        else:
            y = oracle.w8a16(d["x"], d["qweight"], d["zeros"], d["s"], 128)
            y_steps = _y(REAL, d["x"], d["qweight"], None, d["s"], 128, 8, d["zeros"])
        np.testing.assert_array_equal(y, y_steps)


def test_generator_is_deterministic():
    a = make_inputs(4, 2, 256, 64, seed=0)
    b = make_inputs(4, 2, 256, 64, seed=0)
    c = make_inputs(4, 2, 256, 64, seed=1)
    for key in ("x", "q", "s", "z", "qweight", "qzeros"):
        np.testing.assert_array_equal(a[key], b[key])
    assert not np.array_equal(a["q"], c["q"])
    s = a["s"].astype(np.float64)
    assert s.min() >= 0.005 - 1e-5 and s.max() <= 0.02 + 1e-5
    assert a["q"].max() <= 15 and a["z"].max() <= 15


# --------------------------------------------------------------------------
# planted mistakes: every one must make at least one check fail
# --------------------------------------------------------------------------
def _mut_unpack_reversed(words):
    return oracle.unpack_w4(words).reshape(words.shape[0], -1, 8)[:, :, ::-1].reshape(
        words.shape[0], -1).copy()


def _mut_unpack_high_first(words):
    w = np.asarray(words).astype(np.int32).view(np.uint32)
    out = np.empty((w.shape[0], w.shape[1] * 8), dtype=np.uint8)
    for i in range(8):
        out[:, i::8] = ((w >> np.uint32(4 * ((i + 4) % 8))) & np.uint32(0xF)).astype(np.uint8)
    return out


def _mut_dequant_wrap_uint8(q, z, s, G):
    g = np.arange(q.shape[0]) // G
    return s.astype(np.float64)[g] * (q - np.asarray(z)[g]).astype(np.float64)   # uint8 wraps


def _mut_dequant_no_zero(q, z, s, G):
    g = np.arange(q.shape[0]) // G
    return s.astype(np.float64)[g] * q.astype(np.float64)


def _mut_dequant_sign(q, z, s, G):
    return -oracle.dequant(q, z, s, G)


def _mut_dequant_group_mod(q, z, s, G):
    K = q.shape[0]
    g = np.arange(K) % (K // G)
    return s.astype(np.float64)[g] * (q.astype(np.float64) - np.asarray(z).astype(np.float64)[g])


def _mut_dequant_scale_f16_product(q, z, s, G):
    # rounds the dequantized weight to fp16 before the sum (changes the exact value)
    return oracle.dequant(q, z, s, G).astype(np.float16).astype(np.float64)


def _mut_dequant_fma_form(q, z, s, G):
    g = np.arange(q.shape[0]) // G
    sf = s[g].astype(np.float16)
    zs = (np.asarray(z)[g].astype(np.float16) * sf).astype(np.float16)
    return (q.astype(np.float16) * sf - zs).astype(np.float16).astype(np.float64)


def _mut_matmul_drop_last(x, w):
    return oracle.matmul(np.asarray(x)[:, :-1], np.asarray(w)[:-1, :])


def _mut_matmul_f32(x, w):
    return np.matmul(np.asarray(x, dtype=np.float32), np.asarray(w, dtype=np.float32)).astype(np.float64)


def _mut_matmul_f16_acc(x, w):
    acc = np.zeros((np.asarray(x).shape[0], np.asarray(w).shape[1]), dtype=np.float16)
    for k in range(np.asarray(x).shape[1]):
        acc = (acc + np.outer(x[:, k], w[k, :]).astype(np.float16)).astype(np.float16)
    return acc.astype(np.float64)


def _mut_matmul_transposed_w(x, w):
    w = np.asarray(w)
    wt = w.reshape(w.shape[1], w.shape[0]).T            # row-major mis-read of [K, N]
    return oracle.matmul(x, wt)


def _mut_to_f16_truncate(y):
    y = np.asarray(y, dtype=np.float64)
    f = y.astype(np.float16)
    over = np.abs(f.astype(np.float64)) > np.abs(y)
    f[over] = np.nextafter(f[over], np.float16(0))
    return f


MUTANTS = {
    "unpack_reversed": dict(unpack_w4=_mut_unpack_reversed),
    "unpack_high_first": dict(unpack_w4=_mut_unpack_high_first),
    "dequant_wrap_uint8": dict(dequant=_mut_dequant_wrap_uint8),
    "dequant_no_zero": dict(dequant=_mut_dequant_no_zero),
    "dequant_sign": dict(dequant=_mut_dequant_sign),
    "dequant_group_mod": dict(dequant=_mut_dequant_group_mod),
    "dequant_f16_rounded": dict(dequant=_mut_dequant_scale_f16_product),
    "dequant_fma_form": dict(dequant=_mut_dequant_fma_form),
    "matmul_drop_last": dict(matmul=_mut_matmul_drop_last),
    "matmul_f32": dict(matmul=_mut_matmul_f32),
    "matmul_f16_acc": dict(matmul=_mut_matmul_f16_acc),
    "matmul_transposed_w": dict(matmul=_mut_matmul_transposed_w),
    "to_f16_truncate": dict(to_f16=_mut_to_f16_truncate),
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_planted_mistake_is_caught(name):
    ns = types.SimpleNamespace(**{**vars(REAL), **MUTANTS[name]})
    caught = []
    for check in CHECKS:
        try:
            check(ns)
        except Exception:  # any failure of a check flags the planted mistake
            caught.append(check.__name__)
    assert caught, f"planted mistake {name} passed every pin"
