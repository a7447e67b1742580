"""Commit-set selection rules (oracle; test infrastructure only).

Each rule takes the candidates of one block -- their complements
eps_i = 1 - c_i, their confidences c_i and their positions -- and returns how
many / which candidates to reveal.  All decisions are made in exact rational
arithmetic on the given floating-point values, so strict and non-strict
inequalities are decided exactly.

Order.  Alg. 1 sorts the confidences descending, c_(1) >= ... >= c_(m).  The
candidates are ordered by eps ascending, which is the same order; equal values
go to the lower position first (the paper leaves ties open).  Within one
sorted profile c_(j) is taken as exactly 1 - eps_(j).

Rules (n runs over 1..m):
  * factor (Sec. 2 and Sec. 5 "Baselines"): accept n when
        (n+1) (1 - c_(n)) < f ;
  * Frechet profile, literal (Sec. 3 "Frechet profile quantities", Alg. 1):
        L_n = max{0, sum_{j<=n} c_(j) - (n-1)},  U_n = 1 - c_(n),
        G_n = L_n - U_n,  accept n when G_n > delta,  delta = 1 - f
    (the matched parameterisation f = 1 - delta of the equal-confidence
    corollary and Sec. 5 "Baselines");
  * Frechet profile, adaptive-factor form (Remark "Adaptive-factor
    interpretation", eq. adaptive_factor): accept n when
        (n+1)(1 - c_(n)) < f + B_n,   B_n = sum_{j<n} (c_(j) - c_(n)),
    i.e. G_n without the clip at 0 (heterogeneity-bonus proposition).
    For f <= 1 (delta >= 0, the paper's domain) both forms accept exactly the
    same n; for f > 1 (delta < 0) the paper gives no rule and the
    adaptive-factor form is used, which keeps the equal-confidence reduction
    exact for every f;
  * threshold (Sec. 2 "Confidence-Aware Parallel Decoding"): commit every
    candidate with c_i >= tau;
  * calibration-robust profile (appendix "Calibration-Robust Frechet
    Certificates"): the Frechet profile rule on the conservative lower
    confidences c_low_i = max{0, c^_i - eta_i}, sorted by c_low.  The paper
    states the robust certificate L_eta(S) > U_eta(S) for a set S; for a
    fixed size the top-|S| set by c_low maximises both sum c_low and
    min c_low, so the selector takes the largest prefix of the c_low order
    whose robust score exceeds delta (the same reading as the plain rule).

n* is the largest accepted n; when no n is accepted one candidate is still
committed (Sec. 3 "with the convention n* = 1 ... ensuring progress"; for the
threshold rule, "commits the single highest-confidence token").  The factor
rule takes the same fallback (the paper does not state one for it).  An empty
block commits nothing.

Margin flags.  A block is flagged when its decision sits within FLAG_WINDOW of
a boundary, where a float32 implementation may legitimately decide otherwise:
  * factor / profile: |f - LHS_{n*}| <= w when n* was accepted,
    |f - LHS_{n*+1}| <= w when n* < m, or c_(n*) - c_(n*+1) <= w;
    LHS_n = (n+1) eps_(n) for factor and (n+1) eps_(n) - B_n for profile;
  * threshold: some |c_i - tau| <= w, or, on a fallback, c_(1) - c_(2) <= w.
"""
from __future__ import annotations

import dataclasses
from fractions import Fraction as Q
from typing import List, Optional, Sequence

import numpy as np

FLAG_WINDOW = 1e-6


def _q(v) -> Q:
    return v if isinstance(v, Q) else Q(float(v))


def sorted_order(eps: Sequence[float], positions: Sequence[int]) -> List[int]:
    """Candidate indices by confidence descending (eps ascending), ties by position."""
    return sorted(range(len(eps)), key=lambda k: (_q(eps[k]), int(positions[k])))


def robust_eps(eps: Sequence[float], eta: Sequence[float]) -> List[Q]:
    """1 - c_low for the calibration-robust rule, exactly.

    Appendix "Calibration-Robust Frechet Certificates": the reported
    confidence c^_i is replaced by the conservative lower confidence
    c_low_i = max{0, c^_i - eta_i}, i.e. eps_low_i = min{1, eps^_i + eta_i}.
    The allowance eta_i is >= 0 in the paper; a negative value is taken as 0.
    """
    return [min(Q(1), _q(e) + max(Q(0), _q(h))) for e, h in zip(eps, eta)]


def frechet_quantities(eps_sorted: Sequence[float], with_bonus: bool = True):
    """Exact L_n, U_n, G_n, F_n, B_n for n = 1..m of a sorted profile.

    Sec. 3 (L_n, U_n, G_n) and the heterogeneity-bonus proposition
    (F_n = (n+1) c_(n) - n, B_n = sum_{j<n} (c_(j) - c_(n))), with
    c_(j) = 1 - eps_(j).  Returns a list of dicts of Fractions.  B_n is summed
    term by term (quadratic in m); with_bonus=False leaves it out (None).
    """
    c = [1 - _q(e) for e in eps_sorted]
    out = []
    running = Q(0)
    for n in range(1, len(c) + 1):
        running += c[n - 1]
        L = max(Q(0), running - (n - 1))
        U = 1 - c[n - 1]
        F = (n + 1) * c[n - 1] - n
        B = sum((c[j] - c[n - 1] for j in range(n - 1)), Q(0)) if with_bonus else None
        out.append(dict(n=n, L=L, U=U, G=L - U, F=F, B=B, sum_c=running))
    return out


def _fallback(m: int) -> int:
    return 1 if m >= 1 else 0


def factor_lhs(eps_sorted: Sequence[float]) -> List[Q]:
    """(n+1)(1 - c_(n)) for n = 1..m."""
    return [(n + 1) * _q(eps_sorted[n - 1]) for n in range(1, len(eps_sorted) + 1)]


def profile_lhs(eps_sorted: Sequence[float]) -> List[Q]:
    """(n+1)(1 - c_(n)) - B_n for n = 1..m (the adaptive-factor left side)."""
    c = [1 - _q(e) for e in eps_sorted]
    out = []
    total = Q(0)                                   # sum_{j<n} c_(j)
    for n in range(1, len(c) + 1):
        B = total - (n - 1) * c[n - 1]             # sum_{j<n} (c_(j) - c_(n))
        out.append((n + 1) * (1 - c[n - 1]) - B)
        total += c[n - 1]
    return out


def factor_n_star(eps_sorted: Sequence[float], f: float) -> int:
    """Largest n with (n+1)(1 - c_(n)) < f; 1 when none (0 for an empty block)."""
    fq = _q(f)
    acc = [n for n, lhs in enumerate(factor_lhs(eps_sorted), start=1) if lhs < fq]
    return max(acc) if acc else _fallback(len(eps_sorted))


def profile_literal_n_star(eps_sorted: Sequence[float], f: float) -> int:
    """n* = max{n : L_n - U_n > delta}, delta = 1 - f, literal clipped L_n."""
    delta = 1 - _q(f)
    acc = [q["n"] for q in frechet_quantities(eps_sorted, with_bonus=False) if q["G"] > delta]
    return max(acc) if acc else _fallback(len(eps_sorted))


def profile_adaptive_n_star(eps_sorted: Sequence[float], f: float) -> int:
    """n* = max{n : (n+1)(1 - c_(n)) < f + B_n} (adaptive-factor remark)."""
    fq = _q(f)
    acc = [n for n, lhs in enumerate(profile_lhs(eps_sorted), start=1) if lhs < fq]
    return max(acc) if acc else _fallback(len(eps_sorted))


def profile_n_star(eps_sorted: Sequence[float], f: float) -> int:
    """The Frechet profile rule at matched factor f (delta = 1 - f).

    Literal definition for f <= 1; adaptive-factor form for f > 1.
    """
    if f <= 1.0:
        return profile_literal_n_star(eps_sorted, f)
    return profile_adaptive_n_star(eps_sorted, f)


def threshold_set(conf: Sequence[float], order: Sequence[int], tau: float) -> List[int]:
    """Indices with c_i >= tau; else the single first index of `order`."""
    tq = _q(tau)
    s = [k for k in range(len(conf)) if _q(conf[k]) >= tq]
    if not s and len(order):
        s = [order[0]]
    return s


@dataclasses.dataclass
class SelectResult:
    n_commit: int
    committed: List[int]            # positions
    flagged: bool
    reasons: List[str]
    order: List[int]                # candidate indices in sorted order


def select_block(eps: Sequence[float], conf: Sequence[float], positions: Sequence[int],
                 rule: str, param: float, window: float = FLAG_WINDOW,
                 eta: Optional[Sequence[float]] = None) -> SelectResult:
    """Commit set of one block's candidates under `rule`.

    rule is one of profile, factor, threshold, robust; `eta` (per candidate)
    is the calibration allowance of the robust rule.
    """
    m = len(eps)
    if m == 0:
        return SelectResult(0, [], False, [], [])
    if rule == "robust":
        eps = robust_eps(eps, eta if eta is not None else [0.0] * m)
    order = sorted_order(eps, positions)
    eps_s = [_q(eps[k]) for k in order]
    reasons: List[str] = []
    wq = _q(window)
    if rule == "threshold":
        chosen = threshold_set(conf, order, param)
        tq = _q(param)
        for k in range(m):
            if abs(_q(conf[k]) - tq) <= wq:
                reasons.append(f"|c-tau| small at position {positions[k]}")
        if len(chosen) == 1 and _q(conf[chosen[0]]) < tq and m >= 2:
            if _q(eps_s[1]) - _q(eps_s[0]) <= wq:
                reasons.append("fallback with near-tied top two")
        committed = sorted(int(positions[k]) for k in chosen)
        return SelectResult(len(chosen), committed, bool(reasons), reasons, order)
    if rule == "factor":
        n_star = factor_n_star(eps_s, param)
        lhs = factor_lhs(eps_s)
    elif rule in ("profile", "robust"):
        n_star = profile_n_star(eps_s, param)
        lhs = profile_lhs(eps_s)
    else:
        raise ValueError(f"unknown rule {rule!r}")
    fq = _q(param)
    accepted = lhs[n_star - 1] < fq
    if accepted and abs(fq - lhs[n_star - 1]) <= wq:
        reasons.append(f"|f-LHS| small at n*={n_star}")
    if n_star < m:
        if abs(fq - lhs[n_star]) <= wq:
            reasons.append(f"|f-LHS| small at n*+1={n_star + 1}")
        if _q(eps_s[n_star]) - _q(eps_s[n_star - 1]) <= wq:
            reasons.append(f"c_(n*) - c_(n*+1) small at n*={n_star}")
    committed = sorted(int(positions[k]) for k in order[:n_star])
    return SelectResult(n_star, committed, bool(reasons), reasons, order)


def select(eps, conf, mask, start, end, rule: str, param: float, eta=None):
    """Selection for a batch of blocks given per-position eps/conf arrays [B, L].

    Candidates of sequence b: masked positions in [start[b], end[b]).
    `eta` ([B, L] array or scalar) is the robust rule's calibration allowance.
    Returns (commit [B,L] uint8, n_commit [B] int64, flagged [B] bool, results).
    """
    eps = np.asarray(eps)
    conf = np.asarray(conf)
    mask = np.asarray(mask)
    eta_arr = None if eta is None else np.broadcast_to(np.asarray(eta, dtype=np.float64), mask.shape)
    B, L = mask.shape
    commit = np.zeros((B, L), dtype=np.uint8)
    n_commit = np.zeros((B,), dtype=np.int64)
    flagged = np.zeros((B,), dtype=bool)
    results = []
    for b in range(B):
        lo, hi = int(start[b]), int(end[b])
        if not (0 <= lo <= hi <= L):
            raise ValueError(f"bad block bounds for sequence {b}: [{lo},{hi}) with L={L}")
        pos = [i for i in range(lo, hi) if mask[b, i]]
        r = select_block([eps[b, i] for i in pos], [conf[b, i] for i in pos], pos, rule, param,
                         eta=None if eta_arr is None else [eta_arr[b, i] for i in pos])
        for i in r.committed:
            commit[b, i] = 1
        n_commit[b] = r.n_commit
        flagged[b] = r.flagged
        results.append(r)
    return commit, n_commit, flagged, results
