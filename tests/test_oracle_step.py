"""Pins of the oracle's whole decoding step (confidence -> select -> reveal)."""
import itertools
import math
from fractions import Fraction as Q

import numpy as np
import pytest

import oracle
import workloads


def brute_step(logits, mask, start, end, x, rule, param):
    """Independent tiny-case step: softmax by definition, subsets by enumeration."""
    B, L, V = logits.shape
    x = x.copy()
    mask = mask.copy()
    n_commit = np.zeros(B, dtype=np.int64)
    for b in range(B):
        cand = [i for i in range(start[b], end[b]) if mask[b, i]]
        if not cand:
            continue
        tok, c = {}, {}
        for i in cand:
            p = np.exp(logits[b, i] - logits[b, i].max())
            p = p / p.sum()
            tok[i] = min(v for v in range(V) if logits[b, i, v] == logits[b, i].max())
            c[i] = float(p.max())
        if rule == "threshold":
            S = [i for i in cand if c[i] >= param] or [max(cand, key=lambda i: (c[i], -i))]
        else:
            def passes(sub):
                k, lo = len(sub), min(c[i] for i in sub)
                if rule == "factor":
                    return (k + 1) * (1 - lo) < param
                raw = sum(c[i] for i in sub) - (k - 1)
                return (raw if param > 1 else max(0.0, raw)) - (1 - lo) > 1 - param

            best = 0
            for k in range(1, len(cand) + 1):
                if any(passes(sub) for sub in itertools.combinations(cand, k)):
                    best = k
            ranked = sorted(cand, key=lambda i: (-c[i], i))
            S = ranked[:max(best, 1)]
            if best:
                assert passes(S)          # the top-k set is a passing set of that size
        for i in S:
            x[b, i] = tok[i]
            mask[b, i] = 0
        n_commit[b] = len(S)
    return x, mask, n_commit


def test_step_against_bruteforce():
    rng = np.random.default_rng(31)
    for trial in range(60):
        B, L, V = int(rng.integers(1, 4)), int(rng.integers(1, 9)), int(rng.integers(2, 17))
        logits = rng.standard_normal((B, L, V)) * rng.choice([1.0, 3.0])
        spikes = rng.integers(0, V, (B, L))
        logits[np.arange(B)[:, None], np.arange(L)[None, :], spikes] += rng.uniform(0, 9, (B, L))
        mask = (rng.random((B, L)) < 0.7).astype(np.uint8)
        start = rng.integers(0, L + 1, B)
        end = np.array([int(rng.integers(s, L + 1)) for s in start])
        x = np.where(mask == 1, -1, rng.integers(0, V, (B, L)))
        for rule, p in [("profile", 0.75), ("profile", 1.0), ("profile", 2.0), ("factor", 0.75),
                        ("factor", 1.0), ("threshold", 0.9), ("threshold", 0.5)]:
            r = oracle.decode_step(logits, B, L, mask, start, end, x, rule, p)
            bx, bm, bn = brute_step(logits, mask, start, end, x, rule, p)
            ok = ~r.flagged
            assert np.array_equal(r.n_commit[ok], bn[ok])
            assert np.array_equal(r.x[ok], bx[ok])
            assert np.array_equal(r.mask[ok], bm[ok])


def test_step_semantics():
    B, L, V = 2, 8, 12
    rng = np.random.default_rng(4)
    logits = rng.standard_normal((B, L, V))
    logits[:, :, 3] += 12.0                  # confident everywhere
    mask = np.ones((B, L), dtype=np.uint8)
    mask[0, 2] = 0
    x = np.where(mask == 1, -1, 77)
    start, end = np.array([1, 0]), np.array([6, 0])
    r = oracle.decode_step(logits, B, L, mask, start, end, x, "profile", 1.0)
    # only candidates of sequence 0 (positions 1,3,4,5) can change
    assert r.n_commit.tolist() == [4, 0]
    assert r.commit[0].tolist() == [0, 1, 0, 1, 1, 1, 0, 0]
    assert r.x[0].tolist() == [-1, 3, 77, 3, 3, 3, -1, -1]
    assert r.mask[0].tolist() == [1, 0, 0, 0, 0, 0, 1, 1]
    assert np.array_equal(r.x[1], x[1]) and np.array_equal(r.mask[1], mask[1])
    assert (r.tokens[0] == np.array([-1, 3, -1, 3, 3, 3, -1, -1])).all()
    # inputs untouched
    assert x[0, 1] == -1 and mask[0, 1] == 1


def test_workload_shapes_small():
    import torch
    inp = workloads.random_case(3, 10, 40, torch.bfloat16, seed=5)
    assert inp.logits.shape == (3, 10, 40) and inp.logits.dtype == torch.bfloat16
    assert inp.mask.dtype == torch.uint8 and inp.x.dtype == torch.int32
    assert ((inp.end - inp.start) <= 10).all() and (inp.start >= 0).all()
    again = workloads.random_case(3, 10, 40, torch.bfloat16, seed=5)
    assert torch.equal(inp.logits.view(torch.int16), again.logits.view(torch.int16))
    # candidates are finite, everything else is poison
    for b in range(3):
        for i in range(10):
            cand = int(inp.start[b]) <= i < int(inp.end[b]) and inp.mask[b, i]
            assert bool(torch.isfinite(inp.logits[b, i].float()).all()) == bool(cand)


def test_single_block_recipe():
    inp = workloads.single_block_b1_l32(V=4096)
    lg = inp.logits[0].double().numpy()
    # exactly two rows carry an exact tie at the maximum
    ties = sum(int((row == row.max()).sum() >= 2) for row in lg)
    assert ties >= 2
    r = oracle.decode_step(lg[None], 1, 32, inp.mask.numpy(), inp.start.numpy(), inp.end.numpy(),
                           inp.x.numpy(), "profile", 1.0)
    assert r.n_commit[0] >= 1


def test_advance_blocks():
    """Alg. 1 outer loop: a finished block hands over to the next block with a
    masked position; hand-derived windows."""
    G, blk = 10, 4                                   # blocks [0,4) [4,8) [8,10)
    mask = np.array([[0, 0, 0, 0, 1, 0, 0, 0, 0, 0],     # first block done -> [4,8)
                     [1, 0, 0, 0, 0, 0, 0, 0, 0, 0],     # stays
                     [0, 0, 0, 0, 0, 0, 0, 0, 0, 1],     # skips an empty block -> [8,10)
                     [0] * 10,                           # finished -> [10,10)
                     [0, 0, 0, 0, 0, 0, 0, 0, 1, 1]], dtype=np.uint8)
    start = np.array([0, 0, 0, 0, 8])
    end = np.array([4, 4, 4, 4, 10])
    n = oracle.advance_blocks(mask, start, end, G, blk)
    assert start.tolist() == [4, 0, 8, 10, 8] and end.tolist() == [8, 4, 10, 10, 10]
    assert n == 4
