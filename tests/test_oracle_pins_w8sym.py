"""Pins for the oracle of the paper's own W8A16 form: signed INT8 weights with
one scale per output channel and no zero-point (Section 2.2, Eq. 1 and the
W8A16 paragraph; Section 4.3: the INT8 value times the channel's scale).

As in ``test_oracle_pins.py`` every check takes a namespace with the oracle's
steps (``dequant_sym``, ``matmul``, ``to_f16``) so that planted mistakes can be
run through the same checks; each must be caught.
"""
from __future__ import annotations

import types
from fractions import Fraction

import numpy as np
import pytest

import oracle
from paper_2606_11357_amd.synth import make_inputs_w8sym

from test_oracle_pins import f16_value, rne_f16_bits

REAL = types.SimpleNamespace(dequant_sym=oracle.dequant_sym, matmul=oracle.matmul, to_f16=oracle.to_f16)


def _y(ns, x, q, s):
    return ns.matmul(x, ns.dequant_sym(q, s))


def check_dequant_exact(ns):
    """Every INT8 value times a sweep of fp16 scales: the product is exact (a
    rational computed with Fractions) and its fp16 rounding is the RNE of the
    exact value."""
    qs = np.arange(-128, 128, dtype=np.int8)
    sbits = np.array([0x0001, 0x03FF, 0x1000, 0x1234, 0x2000, 0x2A3B, 0x3C00, 0x3C01, 0x4000,
                      0x4A00, 0x57FF], dtype=np.uint16)
    q = np.repeat(qs[:, None], len(sbits), axis=1)
    s = sbits.view(np.float16)
    w = ns.dequant_sym(q, s)
    w16 = np.asarray(w).astype(np.float16).view(np.uint16)
    for i, qv in enumerate(qs):
        for j, sb in enumerate(sbits):
            exact = int(qv) * f16_value(int(sb))
            assert Fraction(float(w[i, j])) == exact, (int(qv), hex(int(sb)))
            want = rne_f16_bits(exact)
            if exact == 0:
                assert w16[i, j] & 0x7FFF == 0
            else:
                assert int(w16[i, j]) == want, (int(qv), hex(int(sb)))


def check_special_cases(ns):
    """q = 0 gives 0; s = 1 gives q; negating q negates the weight."""
    rng = np.random.default_rng(3)
    q = rng.integers(-127, 128, size=(64, 24), dtype=np.int8)
    s = rng.uniform(0.0003, 0.001, size=24).astype(np.float16)
    assert np.all(np.asarray(ns.dequant_sym(np.zeros_like(q), s)) == 0)
    np.testing.assert_array_equal(ns.dequant_sym(q, np.ones(24, dtype=np.float16)), q.astype(np.float64))
    np.testing.assert_array_equal(ns.dequant_sym(-q, s), -np.asarray(ns.dequant_sym(q, s)))


def check_channel_onehot(ns):
    """One nonzero scale, at column j, leaves only column j of the output
    nonzero: the scale belongs to an output channel n, not to a row k."""
    rng = np.random.default_rng(4)
    M, K, N = 3, 40, 16
    x = rng.standard_normal((M, K)).astype(np.float16)
    q = rng.integers(1, 128, size=(K, N), dtype=np.int8)
    for j in (0, 5, N - 1):
        s = np.zeros(N, dtype=np.float16)
        s[j] = 1
        y = np.asarray(_y(ns, x, q, s))
        assert np.all(y[:, np.arange(N) != j] == 0)
        want = [sum(Fraction(float(x[m, k])) * int(q[k, j]) for k in range(K)) for m in range(M)]
        assert [Fraction(float(v)) for v in y[:, j]] == want


def check_matmul_bruteforce(ns):
    """Exact rational sums on tiny shapes (every input is a dyadic rational)."""
    for (M, K, N, seed) in ((1, 32, 8, 0), (3, 64, 16, 1), (2, 96, 24, 2)):
        d = make_inputs_w8sym(M, K, N, seed=seed)
        y = np.asarray(_y(ns, d["x"], d["q"], d["s"]))
        for m in range(M):
            for n in range(N):
                terms = [Fraction(float(d["x"][m, k])) * int(d["q"][k, n]) * f16_value(int(d["s"].view(np.uint16)[n]))
                         for k in range(K)]
                exact = sum(terms)
                bound = K * Fraction(2) ** -52 * sum(abs(t) for t in terms)
                assert abs(Fraction(float(y[m, n])) - exact) <= bound, (M, K, N, m, n)


def check_integer_invariant(ns):
    """s = 1 and integer activations: the result is the integer matmul exactly."""
    rng = np.random.default_rng(5)
    M, K, N = 4, 256, 40
    x = rng.integers(-3, 4, size=(M, K)).astype(np.float16)
    q = rng.integers(-128, 128, size=(K, N), dtype=np.int8)
    y = np.asarray(_y(ns, x, q, np.ones(N, dtype=np.float16)))
    want = x.astype(np.int64) @ q.astype(np.int64)
    np.testing.assert_array_equal(y, want.astype(np.float64))


def check_closed_form(ns):
    """x = 1, q = c, s = sigma: every output is K * c * sigma."""
    M, K, N = 2, 128, 8
    for c, sb in ((-128, 0x1400), (127, 0x0C00), (-7, 0x3555)):
        s = np.full(N, sb, dtype=np.uint16).view(np.float16)
        y = np.asarray(_y(ns, np.ones((M, K), np.float16), np.full((K, N), c, np.int8), s))
        want = K * c * f16_value(sb)
        assert all(Fraction(float(v)) == want for v in y.ravel())


CHECKS = [check_dequant_exact, check_special_cases, check_channel_onehot, check_matmul_bruteforce,
          check_integer_invariant, check_closed_form]


@pytest.mark.parametrize("check", CHECKS, ids=lambda f: f.__name__)
def test_oracle_pin(check):
    check(REAL)


def test_composed_entry_point_matches_steps():
    d = make_inputs_w8sym(5, 256, 48, seed=9)
    np.testing.assert_array_equal(oracle.w8a16_sym(d["x"], d["qweight"], d["scales"]),
                                  oracle.matmul(d["x"], oracle.dequant_sym(d["q"], d["s"])))


def test_generator():
    a, b = make_inputs_w8sym(2, 64, 16, seed=1), make_inputs_w8sym(2, 64, 16, seed=1)
    for k in ("x", "q", "s"):
        np.testing.assert_array_equal(a[k], b[k])
    assert a["q"].dtype == np.int8 and a["q"].min() < 0 <= a["q"].max()
    assert a["s"].dtype == np.float16 and a["s"].shape == (16,)


# --------------------------------------------------------------------------
# planted mistakes (CPU only): each must fail at least one check
# --------------------------------------------------------------------------
def _mut_unsigned(q, s):          # INT8 read as unsigned bytes
    return np.asarray(s, np.float64)[None, :] * np.asarray(q).view(np.uint8).astype(np.float64)


def _mut_row_scale(q, s):         # scale indexed by row k instead of column n
    K = np.asarray(q).shape[0]
    sr = np.resize(np.asarray(s, np.float64), K)
    return sr[:, None] * np.asarray(q, np.float64)


def _mut_offset_zero(q, s):       # a stray zero-point of 128 (the asymmetric form)
    return np.asarray(s, np.float64)[None, :] * (np.asarray(q, np.float64) - 128)


def _mut_f16_product(q, s):       # the product rounded to fp16 before the matmul
    return (np.asarray(s, np.float16)[None, :] * np.asarray(q).astype(np.float16)).astype(np.float64)


def _mut_sign(q, s):
    return -np.asarray(s, np.float64)[None, :] * np.asarray(q, np.float64)


def _mut_matmul_drop_first(x, w):
    return np.matmul(np.asarray(x, np.float64)[:, 1:], np.asarray(w, np.float64)[1:, :])


MUTANTS = {
    "unsigned_int8": dict(dequant_sym=_mut_unsigned),
    "row_scale": dict(dequant_sym=_mut_row_scale),
    "stray_zero_point": dict(dequant_sym=_mut_offset_zero),
    "fp16_product": dict(dequant_sym=_mut_f16_product),
    "sign_flip": dict(dequant_sym=_mut_sign),
    "matmul_drops_first_term": dict(matmul=_mut_matmul_drop_first),
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_planted_mistake_is_caught(name):
    ns = types.SimpleNamespace(**{**vars(REAL), **MUTANTS[name]})
    caught = False
    for check in CHECKS:
        try:
            check(ns)
        except Exception:
            caught = True
            break
    assert caught, f"planted mistake {name} passed every check"
