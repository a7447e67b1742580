"""The oracle's pins catch plausible mistakes.

Each case plants one mistake in a copy of an oracle function (on the CPU,
never in the GPU path) and checks that at least one pin rejects it.
"""
import math
from fractions import Fraction as Q

import numpy as np
import pytest

import oracle
from oracle import rules

import test_oracle_confidence as tc
import test_oracle_select as ts

_PROFILE_LHS = rules.profile_lhs
_FRECHET_Q = rules.frechet_quantities


def _conf_variant(kind):
    def fn(row):
        r = np.asarray(row, dtype=np.float64).ravel()
        M = float(r.max())
        t = int(np.argmax(r))
        if kind == "argmax_last":
            t = len(r) - 1 - int(np.argmax(r[::-1]))
        terms = np.exp(r - M)
        if kind != "keep_greedy_term":
            terms[t] = 0.0
        s = math.fsum(terms.tolist())
        c = 1.0 / (1.0 + s)
        eps = s / (1.0 + s)
        lse = M + math.log1p(s)
        if kind == "eps_by_cancellation":
            eps = 1.0 - c
        if kind == "lse_drops_one":
            lse = M + math.log(s) if s > 0 else M
        if kind == "conf_from_sum_with_greedy":
            c = 1.0 / (2.0 + s)
        return t, c, eps, lse
    return fn


CONF_CHECKS = [tc.check_constant_row, tc.check_two_equal_maxima, tc.check_spike_closed_form,
               tc.check_against_scipy, tc.check_decimal_bruteforce]


@pytest.mark.parametrize("kind", ["argmax_last", "keep_greedy_term", "eps_by_cancellation",
                                  "lse_drops_one", "conf_from_sum_with_greedy"])
def test_confidence_mutants_are_caught(kind):
    fn = _conf_variant(kind)
    caught = 0
    for chk in CONF_CHECKS:
        try:
            chk(fn)
        except AssertionError:
            caught += 1
    assert caught >= 1, kind


def test_unmutated_confidence_passes_all():
    fn = _conf_variant("none")
    for chk in CONF_CHECKS:
        chk(fn)


SELECT_MUTANTS = {
    # factor uses n instead of n+1
    "factor_n_not_n_plus_1": ("factor_lhs",
        lambda eps: [n * Q(eps[n - 1]) for n in range(1, len(eps) + 1)]),
    # profile left side with the bonus added instead of subtracted
    "bonus_sign": ("profile_lhs",
        lambda eps: [v + 2 * (( n + 1) * Q(eps[n - 1]) - v)
                     for n, v in enumerate(_PROFILE_LHS(eps), start=1)]),
    # sort by confidence ascending
    "sort_ascending": ("sorted_order",
        lambda eps, pos: sorted(range(len(eps)), key=lambda k: (-float(eps[k]), int(pos[k])))),
    # ties to the higher position
    "ties_high_position": ("sorted_order",
        lambda eps, pos: sorted(range(len(eps)), key=lambda k: (float(eps[k]), -int(pos[k])))),
    # threshold strict
    "threshold_strict": ("threshold_set",
        lambda conf, order, tau: ([k for k in range(len(conf)) if Q(float(conf[k])) > Q(float(tau))]
                                  or ([order[0]] if len(order) else []))),
    # no progress fallback
    "no_fallback": ("_fallback", lambda m: 0),
    # robust rule: allowance added to the confidence instead of subtracted
    "robust_sign": ("robust_eps",
        lambda eps, eta: [max(Q(0), Q(float(e)) - Q(float(h))) for e, h in zip(eps, eta)]),
    # robust rule: lower confidence not clipped at zero
    "robust_no_clip": ("robust_eps",
        lambda eps, eta: [Q(float(e)) + Q(float(h)) for e, h in zip(eps, eta)]),
}


def _frechet_variant(kind):
    def fq(eps_sorted, with_bonus=True):
        out = _FRECHET_Q(eps_sorted, with_bonus)
        for q in out:
            n = q["n"]
            c = [1 - Q(e) for e in eps_sorted]
            if kind == "U_uses_first":
                q["U"] = 1 - c[0]
            if kind == "L_without_n_minus_1":
                q["L"] = max(Q(0), q["sum_c"])
            if kind == "no_clip":
                q["L"] = q["sum_c"] - (n - 1)
            q["G"] = q["L"] - q["U"]
        return out
    return fq


@pytest.mark.parametrize("kind", sorted(SELECT_MUTANTS))
def test_select_mutants_are_caught(kind, monkeypatch):
    name, fn = SELECT_MUTANTS[kind]
    monkeypatch.setattr(rules, name, fn)
    caught = 0
    for chk in [ts.run_golden, ts.check_subset_bruteforce, ts.check_robust_rule]:
        try:
            chk()
        except AssertionError:
            caught += 1
    assert caught >= 1, kind


@pytest.mark.parametrize("kind", ["U_uses_first", "L_without_n_minus_1", "no_clip"])
def test_frechet_quantity_mutants_are_caught(kind, monkeypatch):
    monkeypatch.setattr(rules, "frechet_quantities", _frechet_variant(kind))
    caught = 0
    for chk in [ts.run_golden, ts.check_subset_bruteforce, ts.check_bonus_decomposition,
                ts.check_literal_equals_adaptive, ts.check_frechet_bound_and_greedy_theorem]:
        try:
            chk() if chk not in (ts.check_bonus_decomposition, ts.check_frechet_bound_and_greedy_theorem) \
                else chk(rules.frechet_quantities)
        except AssertionError:
            caught += 1
    assert caught >= 1, kind
