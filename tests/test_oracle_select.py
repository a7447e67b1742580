"""Pins of the oracle's selection rules.

Against: hand-derived worked examples (tests/golden/selection_examples.txt),
the paper's propositions checked exactly in rationals (equal-confidence
reduction, heterogeneity bonus, matched-factor dominance, adaptive factor),
brute-force enumeration of every candidate subset, and the probability
statements behind the rule (Frechet-Bonferroni bound and the greedy
equivalence theorem) on tiny joint distributions.
"""
import itertools
import os
from fractions import Fraction as Q

import numpy as np
import pytest

import oracle
from oracle import rules as osel

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "selection_examples.txt")


def load_golden():
    cases = []
    for line in open(GOLDEN):
        line = line.strip()
        if not line or line.startswith("#"):
            continue
        rule, param, confs, n_star, committed, flagged, note = [p.strip() for p in line.split("|")]
        parts = [q.strip() for q in confs.split(";")]
        c = [Q(v) for v in parts[0].split(",")]
        pos, eta = list(range(len(c))), None
        for extra in parts[1:]:
            key, val = extra.split("=")
            vals = val.split(",")
            if key == "pos":
                pos = [int(v) for v in vals]
            elif key == "eta":
                eta = [float(v) for v in vals] * (len(c) if len(vals) == 1 else 1)
        cases.append(dict(rule=rule, param=float(param), c=c, pos=pos, n_star=int(n_star),
                          committed=[int(v) for v in committed.split(",")],
                          flagged=bool(int(flagged)), note=note, eta=eta))
    return cases


def run_golden(select_block=oracle.select_block):
    cases = load_golden()
    assert len(cases) >= 25
    for cs in cases:
        eps = [float(1 - c) for c in cs["c"]]
        conf = [float(c) for c in cs["c"]]
        r = select_block(eps, conf, cs["pos"], cs["rule"], cs["param"], eta=cs["eta"])
        assert r.n_commit == cs["n_star"], cs
        assert r.committed == sorted(cs["committed"]), cs
        assert r.flagged == cs["flagged"], (cs, r.reasons)


def test_golden_examples():
    run_golden()


def random_profiles(rng, n_profiles, m_max=12, quantise=None):
    """Sorted eps profiles; `quantise` snaps values to multiples of 1/quantise."""
    out = []
    for _ in range(n_profiles):
        m = int(rng.integers(1, m_max + 1))
        kind = rng.integers(4)
        if kind == 0:
            eps = rng.uniform(0, 0.3, m)
        elif kind == 1:
            eps = rng.beta(0.5, 0.5, m)
        elif kind == 2:
            eps = np.concatenate([rng.uniform(0, 0.02, m // 2 + 1), rng.uniform(0.1, 0.6, m)])[:m]
        else:
            eps = np.full(m, rng.uniform(0, 0.5))
        if quantise:
            eps = np.round(eps * quantise) / quantise
        out.append(sorted(float(e) for e in eps))
    return out


def check_flat_reduction(profile_n_star=oracle.profile_n_star, factor_n_star=oracle.factor_n_star):
    """Equal-confidence corollary: Frechet(delta) == Factor(f = 1 - delta) on flat profiles."""
    rng = np.random.default_rng(3)
    for _ in range(400):
        m = int(rng.integers(1, 65))
        e = float(rng.choice([rng.uniform(0, 1), np.round(rng.uniform(0, 1) * 64) / 64]))
        eps = [e] * m
        for f in [0.0, 0.25, 0.5, 0.75, 1.0, float(rng.uniform(0, 1)), 1.5, 2.0, float(rng.uniform(1, 3))]:
            assert profile_n_star(eps, f) == factor_n_star(eps, f), (e, m, f)
        # also the closed form of the corollary: accept n iff c > 1 - f/(n+1)
        f = float(rng.uniform(0, 1))
        c = 1 - Q(e)
        acc = [n for n in range(1, m + 1) if c > 1 - Q(f) / (n + 1)]
        assert profile_n_star(eps, f) == (max(acc) if acc else 1)


def check_bonus_decomposition(frechet_quantities=oracle.frechet_quantities):
    """Heterogeneity bonus: G_n = F_n + B_n when L_n > 0; B_n >= 0; B_n = 0 iff flat."""
    rng = np.random.default_rng(5)
    hits = 0
    for eps in random_profiles(rng, 300, quantise=None) + random_profiles(rng, 200, quantise=16):
        qs = frechet_quantities(eps)
        c = [1 - Q(e) for e in eps]
        for q in qs:
            n = q["n"]
            assert q["B"] >= 0
            assert (q["B"] == 0) == all(c[j] == c[n - 1] for j in range(n))
            assert q["U"] == 1 - c[n - 1]
            assert q["L"] == max(Q(0), sum(c[:n], Q(0)) - (n - 1))
            if q["L"] > 0:
                hits += 1
                assert q["G"] == q["F"] + q["B"]
    assert hits > 500


def check_matched_dominance(profile_n_star=oracle.profile_n_star, factor_n_star=oracle.factor_n_star,
                            frechet_quantities=oracle.frechet_quantities):
    """Matched-factor dominance and the exact condition for strict separation (f <= 1)."""
    rng = np.random.default_rng(9)
    strict = 0
    for eps in random_profiles(rng, 300) + random_profiles(rng, 200, quantise=32):
        qs = frechet_quantities(eps)
        for f in [0.25, 0.5, 0.75, 1.0, float(rng.uniform(0, 1))]:
            delta = 1 - Q(f)
            for q in qs:
                n = q["n"]
                fac = (n + 1) * Q(eps[n - 1]) < Q(f)
                fre = q["G"] > delta
                if fac:
                    assert fre
                sep = fre and not fac
                assert sep == (q["F"] <= delta < q["F"] + q["B"])
                strict += sep
            assert profile_n_star(eps, f) >= factor_n_star(eps, f)
    assert strict > 50


def check_literal_equals_adaptive():
    """For f <= 1 the clipped literal G_n > delta and the adaptive-factor form agree."""
    rng = np.random.default_rng(13)
    for eps in random_profiles(rng, 500) + random_profiles(rng, 300, quantise=8):
        for f in [0.0, 0.25, 0.5, 0.75, 1.0, float(rng.uniform(0, 1))]:
            assert osel.profile_literal_n_star(eps, f) == osel.profile_adaptive_n_star(eps, f)


def test_flat_reduction():
    check_flat_reduction()


def test_bonus_decomposition():
    check_bonus_decomposition()


def test_matched_dominance():
    check_matched_dominance()


def test_literal_equals_adaptive_for_f_le_1():
    check_literal_equals_adaptive()


def test_literal_differs_for_f_gt_1():
    # the reading for f > 1: flat (0.5,0.5,0.5) at f = 2 (see golden file)
    assert osel.profile_literal_n_star([0.5] * 3, 2.0) == 3
    assert oracle.profile_n_star([0.5] * 3, 2.0) == 2


def subset_brute_force(c, positions, rule, f):
    """max |S| over all candidate subsets S whose own test passes, and one such S.

    profile: G(S) = max{0, sum_S c - (|S|-1)} - (1 - min_S c) > 1 - f
             (adaptive form without the clip when f > 1)
    factor : (|S|+1)(1 - min_S c) < f
    """
    best, best_sets = 0, []
    m = len(c)
    for k in range(1, m + 1):
        for S in itertools.combinations(range(m), k):
            cs = [c[i] for i in S]
            lo = min(cs)
            if rule == "factor":
                ok = (k + 1) * (1 - lo) < Q(f)
            else:
                raw = sum(cs, Q(0)) - (k - 1)
                Lb = raw if f > 1 else max(Q(0), raw)
                ok = Lb - (1 - lo) > 1 - Q(f)
            if ok:
                if k > best:
                    best, best_sets = k, []
                if k == best:
                    best_sets.append(sorted(positions[i] for i in S))
    return best, best_sets


def check_subset_bruteforce(select_block=oracle.select_block):
    rng = np.random.default_rng(17)
    for trial in range(250):
        m = int(rng.integers(1, 9))
        c = [Q(int(v), 64) for v in rng.integers(1, 65, m)] if trial % 2 else \
            [Q(float(v)) for v in rng.uniform(0.5, 1.0, m)]
        positions = sorted(rng.choice(64, m, replace=False).tolist())
        perm = rng.permutation(m)
        c = [c[i] for i in perm]
        for rule in ["profile", "factor"]:
            for f in [0.25, 0.75, 1.0, 2.0]:
                best, sets = subset_brute_force(c, positions, rule, f)
                r = select_block([float(1 - v) for v in c], [float(v) for v in c], positions, rule, f)
                if best == 0:
                    assert r.n_commit == 1
                    top = max(range(m), key=lambda k: (c[k], -positions[k]))
                    assert r.committed == [positions[top]]
                else:
                    assert r.n_commit == best
                    assert r.committed in sets


def test_subset_bruteforce():
    check_subset_bruteforce()


def _random_joint(rng, n, V, peak):
    """A random joint over V^n with mass `peak` on one random tuple."""
    P = rng.dirichlet(np.full(V ** n, 0.3)).reshape((V,) * n)
    if peak:
        idx = tuple(rng.integers(0, V, n))
        P = (1 - peak) * P
        P[idx] += peak
    return P


def check_frechet_bound_and_greedy_theorem(frechet_quantities=oracle.frechet_quantities):
    """Frechet-Bonferroni lemma and the greedy-equivalence theorem on tiny joints."""
    rng = np.random.default_rng(23)
    certified = 0
    for trial in range(600):
        n = int(rng.integers(1, 4))
        V = int(rng.integers(2, 5))
        P = _random_joint(rng, n, V, rng.choice([0.0, 0.5, 0.8, 0.95]))
        marg = [P.sum(axis=tuple(a for a in range(n) if a != j)) for j in range(n)]
        xs = tuple(int(np.argmax(mj)) for mj in marg)
        cj = [float(marg[j][xs[j]]) for j in range(n)]
        order = sorted(range(n), key=lambda j: -cj[j])
        eps_sorted = [1.0 - cj[j] for j in order]
        q = frechet_quantities(eps_sorted)[-1]
        joint_correct = float(P[xs])
        assert joint_correct >= float(q["L"]) - 1e-12           # lemma
        if q["L"] > q["U"]:                                      # theorem
            certified += 1
            flat = P.ravel()
            top = np.argsort(flat)[::-1]
            assert np.unravel_index(top[0], P.shape) == xs
            assert flat[top[0]] > flat[top[1]] if flat.size > 1 else True
    assert certified > 100
    # sharpness: complements disjoint -> P(all correct) == L_n exactly
    for _ in range(50):
        n = int(rng.integers(2, 5))
        miss = rng.dirichlet(np.ones(n + 1))[:n] * rng.uniform(0, 1)
        eps_sorted = sorted(float(v) for v in miss)
        q = frechet_quantities(eps_sorted)[-1]
        assert float(q["L"]) == pytest.approx(1 - sum(miss), abs=1e-12)


def test_frechet_bound_and_greedy_theorem():
    check_frechet_bound_and_greedy_theorem()


def test_fallback_and_empty():
    assert oracle.select_block([], [], [], "profile", 1.0).n_commit == 0
    assert oracle.select_block([], [], [], "threshold", 0.9).n_commit == 0
    r = oracle.select_block([0.9, 0.9], [0.1, 0.1], [4, 2], "profile", 0.1)
    assert r.n_commit == 1 and r.committed == [2]


def test_batch_select_matches_blocks():
    rng = np.random.default_rng(2)
    B, L = 5, 20
    eps = rng.uniform(0, 0.5, (B, L))
    conf = 1 - eps
    mask = (rng.random((B, L)) < 0.6).astype(np.uint8)
    start = np.array([0, 3, 10, 19, 20])
    end = np.array([8, 20, 10, 20, 20])
    for rule, p in [("profile", 0.75), ("factor", 1.0), ("threshold", 0.8)]:
        commit, n_commit, flagged, res = oracle.select(eps, conf, mask, start, end, rule, p)
        for b in range(B):
            pos = [i for i in range(start[b], end[b]) if mask[b, i]]
            r = oracle.select_block([eps[b, i] for i in pos], [conf[b, i] for i in pos], pos, rule, p)
            assert n_commit[b] == r.n_commit
            assert sorted(np.nonzero(commit[b])[0].tolist()) == r.committed
            assert set(r.committed) <= set(pos)


def check_robust_rule(select_block=oracle.select_block, frechet_quantities=oracle.frechet_quantities):
    """Calibration-robust rule: eta = 0 is the profile rule; the calibration
    penalty G^(eta)_n = G^_n - (n+1) eta holds exactly where its assumptions
    hold; commits never grow with a larger uniform eta."""
    rng = np.random.default_rng(41)
    pen = 0
    for eps in random_profiles(rng, 400, quantise=None) + random_profiles(rng, 200, quantise=64):
        m = len(eps)
        pos = list(range(m))
        conf = [1 - e for e in eps]
        for f in (0.5, 0.75, 1.0, 2.0):
            a = select_block(eps, conf, pos, "profile", f)
            b = select_block(eps, conf, pos, "robust", f, eta=[0.0] * m)
            assert (a.n_commit, a.committed) == (b.n_commit, b.committed)
            prev = m + 1
            for eta in (0.0, 0.01, 0.05, 0.2, 0.6):
                r = select_block(eps, conf, pos, "robust", f, eta=[eta] * m)
                assert r.n_commit <= prev
                prev = r.n_commit
        eta = float(rng.choice([0.01, 0.03, 0.1]))
        plain = frechet_quantities(eps)
        rob = frechet_quantities(oracle.robust_eps(eps, [eta] * m))
        c = [1 - Q(e) for e in eps]
        for qp, qr in zip(plain, rob):
            n = qp["n"]
            no_clip = all(c[j] >= Q(eta) for j in range(n))
            if no_clip and qr["sum_c"] - (n - 1) > 0:
                pen += 1
                assert qr["G"] == qp["G"] - (n + 1) * Q(eta)
    assert pen > 300


def check_robust_subsets_and_certificate(select_block=oracle.select_block,
                                         frechet_quantities=oracle.frechet_quantities):
    rng = np.random.default_rng(43)
    for trial in range(150):
        m = int(rng.integers(1, 8))
        c = [Q(int(v), 64) for v in rng.integers(1, 65, m)]
        eta = [Q(int(v), 64) for v in rng.integers(0, 9, m)]
        low = [max(Q(0), ci - hi) for ci, hi in zip(c, eta)]
        positions = list(range(m))
        for f in (0.25, 0.75, 1.0):
            best, sets = subset_brute_force(low, positions, "profile", f)
            r = select_block([float(1 - v) for v in c], [float(v) for v in c], positions, "robust", f,
                             eta=[float(h) for h in eta])
            if best == 0:
                top = max(range(m), key=lambda k: (low[k], -positions[k]))
                assert r.n_commit == 1 and r.committed == [positions[top]]
            else:
                assert r.n_commit == best and r.committed in sets
    # robust certificate on tiny joints: any envelope c_low <= true marginal
    certified = 0
    for trial in range(500):
        n = int(rng.integers(1, 4))
        V = int(rng.integers(2, 5))
        P = _random_joint(rng, n, V, rng.choice([0.0, 0.8, 0.95]))
        marg = [P.sum(axis=tuple(a for a in range(n) if a != j)) for j in range(n)]
        xs = tuple(int(np.argmax(mj)) for mj in marg)
        r_true = [float(marg[j][xs[j]]) for j in range(n)]
        eta = rng.uniform(0, 0.05, n)
        c_low = [max(0.0, r - h) for r, h in zip(r_true, eta)]
        q = frechet_quantities(sorted(1.0 - v for v in c_low))[-1]
        if q["L"] > q["U"]:
            certified += 1
            flat = P.ravel()
            top = np.argsort(flat)[::-1]
            assert np.unravel_index(top[0], P.shape) == xs and flat[top[0]] > flat[top[1]]
    assert certified > 50


def test_robust_rule():
    check_robust_rule()


def test_robust_subsets_and_certificate():
    check_robust_subsets_and_certificate()
