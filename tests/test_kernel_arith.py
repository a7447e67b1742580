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
    greedy element's term never enters a sum);
  * the merge of lanes and of a row's parts leaves out exactly one
    occurrence of the row maximum however the maximum is spread over them
    (ties within a lane, across lanes and across parts).
"""
import math

import numpy as np
import pytest

import oracle

LOG2E_F = np.float32(1.44269504088896340736)
MAX_ABS_LOGIT = 1.0e7


def exp_ref_exact(m: np.float32) -> np.float32:
    """The definition: the smallest integer >= m * log2e, from the exact
    double product (two floats' product fits a double's 53 bits), rounded up
    to a float when it is not one."""
    k = math.ceil(float(m) * float(LOG2E_F))
    kf = np.float32(k)
    if float(kf) < k:
        kf = np.nextafter(kf, np.float32(np.inf))
    return kf


def exp_ref(m: np.float32) -> np.float32:
    """The kernel's float formulation: p = fl(m log2e), the sign of the exact
    remainder m log2e - p (what fma(m, log2e, -p) returns), c = ceil(p); K =
    c + 1 when p is an integer below the exact product, else c; beyond 2^24
    the next float above c."""
    m = np.float32(m)
    p = np.float32(m * LOG2E_F)
    e = float(m) * float(LOG2E_F) - float(p)     # exact in double
    c = np.float32(np.ceil(p))
    if abs(c) < np.float32(16777216.0):
        return np.float32(c + np.float32(1.0)) if (c == p and e > 0.0) else c
    if np.isinf(c):
        return c
    return np.nextafter(c, np.float32(np.inf))


def exp_ref_float_product(m: np.float32) -> np.float32:
    """The reference formed from the float32 product (the earlier form)."""
    return np.float32(math.ceil(float(np.float32(m * LOG2E_F))))


def arg(x, K) -> np.float32:
    """fma(x, log2e, -K) rounded once to float32."""
    return np.float32(float(x) * float(LOG2E_F) - float(K))


def term(x, K) -> float:
    """The float32 exp2 of the fused argument, widened to double."""
    return float(np.float32(np.exp2(np.float64(arg(x, K)))))


def rescale(s: float, a, b) -> float:
    """s * 2^(a - b) for integer-valued a <= b (exact, as ldexp)."""
    return math.ldexp(s, int(max(float(a) - float(b), -2000.0)))


def ref_of(m) -> np.float32:
    """The reference with the floor a stretch of padding only keeps."""
    if m == -np.inf:
        return np.float32(-3.0e38)
    return max(exp_ref(np.float32(m)), np.float32(-3.0e38))


def emulate_stretch(xs: np.ndarray, idx: np.ndarray, batch: int):
    """(m, K, s, first) of one stretch by the kernel's one-lane streaming
    scheme: the terms of every batch but the one where the running maximum
    first appeared go to acc; that batch is summed again at the end without
    one element equal to the maximum, so s holds every term of the stretch
    but one occurrence of m."""
    m, K, acc, pend, first, kept = -np.inf, np.float32(-3.0e38), 0.0, 0.0, 0x7FFFFFFF, None
    for b0 in range(0, xs.size, batch):
        xb = xs[b0:b0 + batch]
        bm = xb.max()
        grows = bm > m
        Kn = ref_of(max(m, bm))
        acc, pend = rescale(acc, K, Kn), rescale(pend, K, Kn)
        m, K = max(m, bm), Kn
        bs = sum(term(x, K) for x in xb)
        if grows:
            first = int(idx[b0 + int(np.argmax(xb))])
            kept = xb
            acc += pend
            pend = bs
        else:
            acc += bs
    if kept is not None:
        left_out = False
        for x in kept:
            if not left_out and x == m:
                left_out = True
                continue
            acc += term(x, K)
    return m, K, acc, first


def combine(parts):
    """Stretches merged as the kernel merges lanes and a row's parts: the
    largest maximum M, every stretch but the lowest-index one holding M puts
    its own maximum's term back, then one sum."""
    M = max(p[0] for p in parts)
    K = ref_of(M)
    owner = next(i for i, p in enumerate(parts) if p[0] == M)
    total = 0.0
    for i, (m, Km, s, _) in enumerate(parts):
        total += rescale(s, Km, K)
        if i != owner:
            total += rescale(term(m, Km), Km, K)
    return M, K, total, min(p[3] for p in parts if p[0] == M)


def finish(M, K, S, first):
    """(token, conf, eps) from a row's (M, K, S): S / e_M is the sum of the
    other terms over the greedy one."""
    Kr = exp_ref(np.float32(M))
    sp = S / rescale(term(M, Kr), Kr, K)
    return first, 1.0 / (1.0 + sp), sp / (1.0 + sp)


def emulate_row(row: np.ndarray, E: int = 8, U: int = 4, lanes: int = 1, parts: int = 1):
    """(token, conf, eps) of one row the kernel's way: vectors of E elements,
    wave-load j of part w covering vectors (w + j parts) lanes + l for lanes
    l, each lane streaming batches of U vectors, lanes merged into a wave
    partial, the row's parts merged last."""
    row = row.astype(np.float32)
    nvec = (row.size + E - 1) // E
    waves = []
    for w in range(parts):
        lane_parts = []
        for lane in range(lanes):
            vecs = [v for v in range(w * lanes + lane, nvec, parts * lanes)]
            idx = np.array([v * E + e for v in vecs for e in range(E) if v * E + e < row.size],
                           dtype=np.int64)
            xs = row[idx] if idx.size else np.zeros(0, np.float32)
            lane_parts.append(emulate_stretch(xs, idx, U * E) if idx.size
                              else (-np.inf, np.float32(-3.0e38), 0.0, 0x7FFFFFFF))
        waves.append(combine(lane_parts))
    return finish(*combine(waves))


MAGNITUDES = [1e3, 1e4, 1e5, 1e6, 3e6, 9.99e6, MAX_ABS_LOGIT]


@pytest.mark.parametrize("M", MAGNITUDES + [-v for v in MAGNITUDES])
def test_maximum_argument_in_range(M):
    rng = np.random.default_rng(abs(int(M)) % 1000)
    ms = np.float32(M) + rng.uniform(-1.0, 1.0, 2000).astype(np.float32) * np.float32(min(abs(M), 64.0))
    for m in ms:
        m = np.float32(np.clip(m, -MAX_ABS_LOGIT, MAX_ABS_LOGIT))
        a = arg(m, exp_ref(m))
        assert -1.0 < a <= 0.0, (m, a)


def test_float_formulation_is_the_exact_ceiling_in_range():
    # the kernel forms K in float arithmetic; within |m| <= 1e7 it must equal
    # the ceiling of the exact product everywhere: random magnitudes, values
    # whose rounded product is an integer (the remainder's sign decides), and
    # the neighbours of those
    rng = np.random.default_rng(5)
    ms = [np.float32(v) for v in rng.uniform(-MAX_ABS_LOGIT, MAX_ABS_LOGIT, 20000)]
    ms += [np.float32(v) for v in rng.normal(0.0, 30.0, 20000)]
    hits = 0
    for k in rng.integers(-(1 << 23), 1 << 23, 20000):
        m0 = np.float32(float(k) / float(LOG2E_F))
        for m in (np.nextafter(m0, np.float32(-np.inf)), m0, np.nextafter(m0, np.float32(np.inf))):
            if abs(m) <= MAX_ABS_LOGIT:
                ms.append(m)
                hits += int(np.float32(m * LOG2E_F) == np.ceil(np.float32(m * LOG2E_F)))
    ms += [np.float32(0.0), np.float32(-0.0), np.float32(1e-45), np.float32(-1e-45),
           np.float32(MAX_ABS_LOGIT), np.float32(-MAX_ABS_LOGIT)]
    assert hits > 10000           # many rounded products are integers
    for m in ms:
        assert exp_ref(m) == exp_ref_exact(m), m


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


@pytest.mark.parametrize("lanes,parts", [(1, 1), (4, 1), (64, 1), (8, 4), (64, 16)])
@pytest.mark.parametrize("spike", [0.0, 30.0])
def test_emulated_split_rows_match_oracle(lanes, parts, spike):
    rng = np.random.default_rng(lanes * 100 + parts)
    V = 5003                       # ragged: the last vector is partial
    row = rng.normal(0.0, 1.0, V).astype(np.float32)
    if spike:
        row[rng.integers(0, V)] = np.float32(spike)
    t, c, e = emulate_row(row, lanes=lanes, parts=parts)
    ot, oc, oe, _ = oracle.position_confidence(row.astype(np.float64))
    assert t == ot
    assert abs(c - oc) <= 1e-5 * oc
    assert abs(e - oe) <= 1e-5 * oe, (e, oe)


@pytest.mark.parametrize("where", ["one_lane", "across_lanes", "across_parts", "everywhere"])
def test_emulated_tied_maxima(where):
    # k copies of the maximum: the greedy token is the lowest index and
    # s' counts the k - 1 other copies, so eps >= (k - 1) / k
    rng = np.random.default_rng(len(where))
    V, E, lanes, parts = 4096, 8, 8, 4
    row = rng.normal(0.0, 1.0, V).astype(np.float32)
    top = np.float32(12.0)
    if where == "one_lane":
        pos = [3, 5, 3 + E * lanes * parts]          # lane 0 of part 0, two batches
    elif where == "across_lanes":
        pos = [E * 1 + 2, E * 5, E * 7 + 7]         # lanes 1, 5, 7 of part 0
    elif where == "across_parts":
        pos = [E * lanes * 1, E * lanes * 2 + 9, E * lanes * 3 + 1]
    else:
        pos = list(rng.choice(V, 40, replace=False))
    row[pos] = top
    t, c, e = emulate_row(row, E=E, U=2, lanes=lanes, parts=parts)
    ot, oc, oe, _ = oracle.position_confidence(row.astype(np.float64))
    assert t == ot == min(pos)
    assert e >= (len(pos) - 1) / len(pos) * (1 - 1e-6)
    assert abs(c - oc) <= 1e-5 * oc
    assert abs(e - oe) <= 1e-5 * oe
