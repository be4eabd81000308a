"""Pins for the MLP-composite oracle (not the paper's method: the layer around
it).  silu is pinned to a library sigmoid and to closed forms; the composite
to its definition on exact small cases.  Planted mistakes must be caught."""
from __future__ import annotations

import types

import numpy as np
import pytest
from scipy.special import expit

import oracle
from paper_2606_11357_amd.synth import pack_nibbles

REAL = types.SimpleNamespace(silu=oracle.silu, silu_mul=oracle.silu_mul)


def check_silu_library(ns):
    """silu(g) = g * expit(g) (scipy's logistic sigmoid) over a wide range."""
    g = np.linspace(-60, 60, 4001)
    np.testing.assert_allclose(ns.silu(g), g * expit(g), rtol=1e-14, atol=1e-300)


def check_silu_closed_forms(ns):
    """silu(0) = 0; silu(ln 3) = (3/4) ln 3; silu(-ln 3) = -(1/4) ln 3;
    silu(g) - silu(-g) = g (odd part is g / 2 times 2)."""
    ln3 = np.log(3.0)
    assert ns.silu(np.array([0.0]))[0] == 0.0
    np.testing.assert_allclose(ns.silu(np.array([ln3, -ln3])), [0.75 * ln3, -0.25 * ln3], rtol=1e-15)
    g = np.linspace(-20, 20, 401)
    np.testing.assert_allclose(ns.silu(g) - ns.silu(-g), g, rtol=1e-13, atol=1e-13)


def check_silu_mul_halves(ns):
    """The first N columns gate, the last N are multiplied: unit gate columns
    give silu(1) * u exactly where u is a power of two."""
    g = np.ones((2, 4))
    u = np.array([[1.0, 2.0, 4.0, 0.5], [-1.0, 8.0, 0.25, 16.0]])
    out = ns.silu_mul(np.concatenate([g, u], axis=1))
    np.testing.assert_array_equal(out, u * (1.0 / (1.0 + np.exp(-1.0))))
    out = ns.silu_mul(np.concatenate([u, np.ones((2, 4))], axis=1))
    np.testing.assert_allclose(out, u * expit(u), rtol=1e-15)


CHECKS = [check_silu_library, check_silu_closed_forms, check_silu_mul_halves]


@pytest.mark.parametrize("check", CHECKS, ids=lambda f: f.__name__)
def test_oracle_pin(check):
    check(REAL)


def test_composite_definition():
    """With unit scales and zero zero-points the composite is integer matmuls
    around the gate: checked against a hand-built float64 pipeline."""
    rng = np.random.default_rng(0)
    M, K, I, G = 3, 64, 32, 32
    x = rng.integers(-2, 3, size=(M, K)).astype(np.float16)
    qgu = rng.integers(0, 4, size=(K, 2 * I)).astype(np.uint8)
    qd = rng.integers(0, 4, size=(I, 8)).astype(np.uint8)
    z = lambda r, n: np.zeros((r, n), np.uint8)
    s = lambda r, n: np.ones((r, n), np.float16)
    y = oracle.mlp_w4a16(x, pack_nibbles(qgu), pack_nibbles(z(K // G, 2 * I)), s(K // G, 2 * I),
                         pack_nibbles(qd), pack_nibbles(z(I // G, 8)), s(I // G, 8), G)
    gu = (x.astype(np.int64) @ qgu.astype(np.int64)).astype(np.float64)
    gu = gu.astype(np.float16).astype(np.float64)
    h = (gu[:, :I] / (1.0 + np.exp(-gu[:, :I])) * gu[:, I:]).astype(np.float16).astype(np.float64)
    want = h @ qd.astype(np.float64)
    np.testing.assert_allclose(y, want, rtol=1e-12, atol=1e-9)


def test_composite_definition_bf16():
    """The BF16 composite with unit scales and zero zero-points: integer
    matmuls around the gate, GU and H rounded to bfloat16 by the exact
    rational rounding of the BF16 pins (not the oracle's own rounding)."""
    from fractions import Fraction
    from test_oracle_pins_bf16 import bf16_value, rne_bf16_bits
    rng = np.random.default_rng(1)
    M, K, I, G = 3, 64, 32, 32
    xi = rng.integers(-2, 3, size=(M, K))
    qgu = rng.integers(0, 4, size=(K, 2 * I)).astype(np.uint8)
    qd = rng.integers(0, 4, size=(I, 8)).astype(np.uint8)
    x_bits = (xi.astype(np.float32).view(np.uint32) >> 16).astype(np.uint16)
    z = lambda r, n: np.zeros((r, n), np.uint8)
    one = lambda r, n: np.full((r, n), 0x3F80, np.uint16)
    y = oracle.mlp_w4a16_bf16(x_bits, pack_nibbles(qgu), pack_nibbles(z(K // G, 2 * I)), one(K // G, 2 * I),
                              pack_nibbles(qd), pack_nibbles(z(I // G, 8)), one(I // G, 8), G)
    rnd = np.vectorize(lambda v: float(bf16_value(rne_bf16_bits(Fraction(float(v))))))
    gu = rnd((xi.astype(np.int64) @ qgu.astype(np.int64)).astype(np.float64))
    h = rnd(gu[:, :I] / (1.0 + np.exp(-gu[:, :I])) * gu[:, I:])
    want = h @ qd.astype(np.float64)
    np.testing.assert_allclose(y, want, rtol=1e-12, atol=1e-9)


def _mut_sigmoid_only(g):            # the gate without the factor g
    return 1.0 / (1.0 + np.exp(-np.asarray(g, np.float64)))


def _mut_wrong_sign(g):              # e^{+g}
    g = np.asarray(g, np.float64)
    return g / (1.0 + np.exp(g))


def _mut_swapped_halves(gu):         # gate taken from the second half
    gu = np.asarray(gu, np.float64)
    n = gu.shape[1] // 2
    return oracle.silu(gu[:, n:]) * gu[:, :n]


MUTANTS = {
    "sigmoid_only": dict(silu=_mut_sigmoid_only),
    "wrong_sign": dict(silu=_mut_wrong_sign),
    "swapped_halves": dict(silu_mul=_mut_swapped_halves),
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
