"""Pins of the oracle's per-position pass (greedy token, confidence, lse).

Each check pins the oracle to something other than itself: closed forms of
special rows, SciPy's logsumexp/softmax, and a 60-digit decimal brute force.
"""
import math
from decimal import Decimal, getcontext

import numpy as np
import pytest
import scipy.special

import oracle


def check_constant_row(fn=oracle.position_confidence):
    for V, x in [(1, 0.0), (7, 3.5), (126464, -2.25)]:
        t, c, eps, lse = fn(np.full(V, x))
        assert t == 0
        assert c == pytest.approx(1.0 / V, rel=1e-15)
        assert eps == pytest.approx((V - 1) / V, rel=1e-15)
        assert lse == pytest.approx(x + math.log(V), rel=1e-15, abs=1e-15)


def check_two_equal_maxima(fn=oracle.position_confidence):
    V = 1000
    r = np.full(V, -30.0)
    r[[417, 33]] = 5.0
    t, c, eps, lse = fn(r)
    assert t == 33                                # lowest index among the maxima
    s = 1.0 + (V - 2) * math.exp(-35.0)           # the other maximum contributes 1
    assert c == pytest.approx(1.0 / (1.0 + s), rel=1e-15)
    assert eps == pytest.approx(s / (1.0 + s), rel=1e-15)


def check_spike_closed_form(fn=oracle.position_confidence):
    V = 126464
    for h, k in [(0.5, 7), (12.0, 100000), (60.0, 5), (700.0, V - 1)]:
        r = np.zeros(V)
        r[k] = h
        t, c, eps, lse = fn(r)
        assert t == k
        s = (V - 1) * math.exp(-h)
        assert eps == pytest.approx(s / (1.0 + s), rel=1e-13)   # accurate even when c rounds to 1
        assert c == pytest.approx(1.0 / (1.0 + s), rel=1e-15)
        assert lse == pytest.approx(h + math.log1p(s), rel=1e-15)


def check_against_scipy(fn=oracle.position_confidence):
    rng = np.random.default_rng(7)
    for V in [2, 3, 64, 1000, 126464]:
        for scale in [0.5, 3.0, 20.0]:
            r = rng.standard_normal(V) * scale
            t, c, eps, lse = fn(r)
            p = scipy.special.softmax(r)
            assert t == int(np.argmax(p))
            assert c == pytest.approx(float(p.max()), rel=1e-13)
            assert eps == pytest.approx(1.0 - float(p.max()), rel=1e-10, abs=1e-15)
            assert lse == pytest.approx(float(scipy.special.logsumexp(r)), rel=1e-14)


def check_decimal_bruteforce(fn=oracle.position_confidence):
    """Tiny rows against a 60-digit softmax evaluated term by term."""
    getcontext().prec = 60
    rng = np.random.default_rng(11)
    for V in [1, 2, 5, 16]:
        for _ in range(20):
            r = np.round(rng.standard_normal(V) * 4, 3)
            if V > 1 and rng.random() < 0.3:
                r[rng.integers(V)] = r.max()             # plant a tie
            t, c, eps, lse = fn(r)
            d = [Decimal(float(v)) for v in r]
            M = max(d)
            first = d.index(M)
            z = sum((v - M).exp() for v in d)
            c_ref = Decimal(1) / z
            eps_ref = (z - 1) / z
            assert t == first
            assert c == pytest.approx(float(c_ref), rel=1e-15)
            assert eps == pytest.approx(float(eps_ref), rel=1e-14, abs=1e-300)
            assert lse == pytest.approx(float(M + z.ln()), rel=1e-15, abs=1e-15)


def test_constant_row():
    check_constant_row()


def test_two_equal_maxima_lowest_index():
    check_two_equal_maxima()


def test_spike_closed_form():
    check_spike_closed_form()


def test_against_scipy():
    check_against_scipy()


def test_decimal_bruteforce():
    check_decimal_bruteforce()


def test_bf16_and_fp32_inputs_are_exact():
    import torch
    r = torch.randn(5000, generator=torch.Generator().manual_seed(3)) * 4
    for dt in (torch.bfloat16, torch.float32):
        rr = r.to(dt)
        t, c, eps, lse = oracle.position_confidence(rr.to(torch.float64).numpy())
        ref = scipy.special.softmax(rr.to(torch.float64).numpy())
        assert t == int(np.argmax(ref))
        assert c == pytest.approx(float(ref.max()), rel=1e-13)


def test_nonfinite_and_empty_rejected():
    with pytest.raises(ValueError):
        oracle.position_confidence(np.array([0.0, np.nan]))
    with pytest.raises(ValueError):
        oracle.position_confidence(np.array([0.0, np.inf]))
    with pytest.raises(ValueError):
        oracle.position_confidence(np.array([]))


def test_batch_reads_only_candidates():
    B, L, V = 3, 6, 9
    rng = np.random.default_rng(1)
    data = rng.standard_normal((B, L, V))
    mask = np.array([[1, 0, 1, 1, 0, 1], [0, 0, 0, 0, 0, 0], [1, 1, 1, 1, 1, 1]], dtype=np.uint8)
    start, end = [1, 0, 2], [5, 6, 2]
    touched = []

    def row(b, i):
        touched.append((b, i))
        return data[b, i]

    tokens, conf, eps, lse = oracle.confidence(row, B, L, mask, start, end)
    assert sorted(touched) == [(0, 2), (0, 3)]
    for b in range(B):
        for i in range(L):
            if (b, i) in touched:
                t, c, e, s = oracle.position_confidence(data[b, i])
                assert (tokens[b, i], conf[b, i], eps[b, i], lse[b, i]) == (t, c, e, s)
            else:
                assert (tokens[b, i], conf[b, i], eps[b, i], lse[b, i]) == (-1, 0.0, 1.0, 0.0)
    with pytest.raises(ValueError):
        oracle.confidence(row, B, L, mask, [0, 0, 4], [1, 1, 3])
