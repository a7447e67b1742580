"""The vocabulary pass's float arithmetic, emulated on the CPU, at large
logit magnitudes.

The kernel keeps, per stretch of a row, a running maximum m, an integer
exponent reference K = exp_ref(m) and a double sum of terms
2^(x log2e - K), each term a float32 exp2 of a float32 argument formed by one
fused multiply-add.  This emulates that arithmetic exactly where it matters
(the fused multiply-add: a product of two floats is exact in double, and the
integer K is exact there too) and checks, for row maxima from 1e3 up to the
documented bound |logit| <= 1e7, that

  * the maximum's own argument lies in (-1, 0] (no overflow, no underflow);
  * the confidence and eps built from the emulated sums agree with the
    oracle on the same rows, eps to 1e-5 relative also when it is tiny (the
    greedy element's term never enters a sum).
"""
import math

import numpy as np
import pytest

import oracle

LOG2E_F = np.float32(1.44269504088896340736)
MAX_ABS_LOGIT = 1.0e7


def exp_ref(m: np.float32) -> np.float32:
    """Smallest integer >= m * log2e, from the exact double product, rounded
    up to a float when it is not one."""
    k = math.ceil(float(m) * float(LOG2E_F))
    kf = np.float32(k)
    if float(kf) < k:
        kf = np.nextafter(kf, np.float32(np.inf))
    return kf


def exp_ref_float_product(m: np.float32) -> np.float32:
    """The reference formed from the float32 product (the earlier form)."""
    return np.float32(math.ceil(float(np.float32(m * LOG2E_F))))


def arg(x, K) -> np.float32:
    """fma(x, log2e, -K) rounded once to float32."""
    return np.float32(float(x) * float(LOG2E_F) - float(K))


def emulate_row(row: np.ndarray, batch: int = 32):
    """(token, conf, eps) by the kernel's one-lane streaming scheme: the terms
    of every batch but the one where the running maximum first appeared go
    to acc; that batch is summed again at the end without one element equal
    to the maximum, so no sum ever holds the greedy term."""
    row = row.astype(np.float32)
    m, K, acc, pend, first, kept = -np.inf, np.float32(-3.0e38), 0.0, 0.0, -1, None
    for b0 in range(0, row.size, batch):
        xs = row[b0:b0 + batch]
        bm = xs.max()
        grows = bm > m
        Kn = max(exp_ref(max(m, bm)), np.float32(-3.0e38))
        shift = int(max(float(K) - float(Kn), -2000.0))
        acc, pend = math.ldexp(acc, shift), math.ldexp(pend, shift)
        m, K = max(m, bm), Kn
        bs = 0.0
        for x in xs:
            bs += float(np.float32(np.exp2(np.float64(arg(x, K)))))
        if grows:
            first = b0 + int(np.argmax(xs))
            kept = xs
            acc += pend
            pend = bs
        else:
            acc += bs
    left_out = False
    for x in kept:
        if not left_out and x == m:
            left_out = True
            continue
        acc += float(np.float32(np.exp2(np.float64(arg(x, K)))))
    eM = float(np.float32(np.exp2(np.float64(arg(m, exp_ref(np.float32(m)))))))
    sp = acc / eM
    return first, 1.0 / (1.0 + sp), sp / (1.0 + sp)


MAGNITUDES = [1e3, 1e4, 1e5, 1e6, 3e6, 9.99e6, MAX_ABS_LOGIT]


@pytest.mark.parametrize("M", MAGNITUDES + [-v for v in MAGNITUDES])
def test_maximum_argument_in_range(M):
    rng = np.random.default_rng(abs(int(M)) % 1000)
    ms = np.float32(M) + rng.uniform(-1.0, 1.0, 2000).astype(np.float32) * np.float32(min(abs(M), 64.0))
    for m in ms:
        m = np.float32(np.clip(m, -MAX_ABS_LOGIT, MAX_ABS_LOGIT))
        a = arg(m, exp_ref(m))
        assert -1.0 < a <= 0.0, (m, a)


def test_float_product_reference_was_not_exact():
    # with |m log2e| near 2^24 the float product rounds by up to 1/2, so its
    # ceiling can leave the maximum's argument above 0
    rng = np.random.default_rng(3)
    m = (np.float32(9.0e6) + rng.integers(0, 1 << 20, 20000).astype(np.float32)).astype(np.float32)
    assert max(arg(v, exp_ref_float_product(v)) for v in m) > 0.0
    assert max(arg(v, exp_ref(v)) for v in m) <= 0.0


@pytest.mark.parametrize("beyond", [1.5e9, 1e12, 1e20, -1e20, 2e38])
def test_no_overflow_beyond_the_bound(beyond):
    # outside the contract the argument still never exceeds 0
    m = np.float32(beyond)
    K = exp_ref(m)
    assert np.isfinite(K)
    assert arg(m, K) <= 0.0


@pytest.mark.parametrize("offset", [0.0, 1e3, -1e4, 1e5, -1e6, 1e7, -1e7])
def test_emulated_pass_matches_oracle(offset):
    rng = np.random.default_rng(11)
    V = 1500
    base = rng.normal(0.0, 1.0, V).astype(np.float32)
    base[rng.integers(0, V)] += 9.0
    base[rng.integers(0, V)] += 4.0
    row = (base + np.float32(offset)).astype(np.float32)   # rounded to the float grid at offset
    assert np.abs(row).max() <= MAX_ABS_LOGIT + 64
    row = np.clip(row, -MAX_ABS_LOGIT, MAX_ABS_LOGIT).astype(np.float32)
    t, c, e = emulate_row(row)
    ot, oc, oe, _ = oracle.position_confidence(row.astype(np.float64))
    assert t == ot
    assert abs(c - oc) <= 1e-5 * oc
    assert abs(e - oe) <= 1e-5 * oe


@pytest.mark.parametrize("spike", [22.0, 35.0, 50.0, 65.0, 80.0])
def test_emulated_eps_of_very_confident_rows(spike):
    # eps ~ V e^(1/2 - spike): from 1e-6 down to ~1e-31; the greedy term never
    # enters a sum, so eps keeps its relative accuracy
    rng = np.random.default_rng(int(spike))
    V = 4000
    row = rng.normal(0.0, 1.0, V).astype(np.float32)
    row[rng.integers(0, V)] = np.float32(spike)
    t, c, e = emulate_row(row)
    ot, oc, oe, _ = oracle.position_confidence(row.astype(np.float64))
    assert t == ot
    assert oe < 1e-5
    assert abs(e - oe) <= 1e-5 * oe, (e, oe)
