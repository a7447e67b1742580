"""Pins of the oracle's LM-head logits against exact arithmetic."""
import math
from fractions import Fraction

import numpy as np

import oracle


def test_logits_rows_exact_on_dyadic_inputs():
    rng = np.random.default_rng(0)
    h = rng.integers(-40, 41, (5, 96)) / 64.0
    w = rng.integers(-40, 41, (30, 96)) / 16.0
    got = oracle.lmhead.logits_rows(h, w)
    for a in range(5):
        for v in range(30):
            exact = sum(Fraction(float(h[a, k])) * Fraction(float(w[v, k])) for k in range(96))
            assert Fraction(float(got[a, v])) == exact


def test_logits_rows_match_correctly_rounded_sums():
    rng = np.random.default_rng(1)
    h = rng.standard_normal((3, 200)).astype(np.float32).astype(np.float64)
    w = rng.standard_normal((17, 200)).astype(np.float32).astype(np.float64)
    got = oracle.lmhead.logits_rows(h, w)
    for a in range(3):
        for v in range(17):
            ref = math.fsum(float(h[a, k]) * float(w[v, k]) for k in range(200))
            assert abs(got[a, v] - ref) <= 1e-12 * sum(abs(h[a] * w[v]))


def test_row_source_and_bound():
    rng = np.random.default_rng(2)
    h = rng.standard_normal((2, 3, 8))
    w = rng.standard_normal((5, 8))
    row = oracle.lmhead.row_source(h, w)
    assert np.allclose(row(1, 2), w @ h[1, 2])
    bnd = oracle.lmhead.accumulation_bound(h[0, 0], w, 2.0 ** -24)
    assert bnd == max(np.abs(w) @ np.abs(h[0, 0])) * 2.0 ** -24
    # a float32 evaluation stays within the bound's d-fold multiple
    l32 = (w.astype(np.float32) @ h[0, 0].astype(np.float32)).astype(np.float64)
    l64 = w.astype(np.float32).astype(np.float64) @ h[0, 0].astype(np.float32).astype(np.float64)
    assert np.all(np.abs(l32 - l64) <= 8 * oracle.lmhead.accumulation_bound(h[0, 0], w, 2.0 ** -24) + 1e-30)
