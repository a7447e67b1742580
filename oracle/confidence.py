"""Per-position greedy token and confidence (oracle; test infrastructure only).

Follows Sec. 3 "Notation" of the paper: for a masked position i the model gives
a marginal distribution p_i(v) over the vocabulary; the marginal greedy token
is x*_i = argmax_v p_i(v) and its confidence is c_i = p_i(x*_i).  Alg. 1
computes both for every masked position of the active block.  Decoding is
greedy at temperature 1 (Sec. 5, "Model and Hardware"), so p_i is the plain
softmax of the logits l_i:

    M   = max_v l_iv
    t   = smallest v with l_iv = M              (ties -> lowest index)
    s'  = sum_{v != t} exp(l_iv - M)            (other maxima contribute 1 each)
    c   = 1 / (1 + s')
    eps = s' / (1 + s') = 1 - c                 (computed without cancellation)
    lse = M + log1p(s') = log sum_v exp(l_iv)

The paper leaves the tie rule for the argmax open; the lowest index is used.
"""
from __future__ import annotations

import math
from typing import Callable, Union

import numpy as np


def position_confidence(row) -> tuple[int, float, float, float]:
    """(t, c, eps, lse) of one position's logits, in float64.

    ``row`` is any 1-D array-like of finite numbers (the exact value of each
    entry is used).  Raises ValueError for an empty or non-finite row.
    """
    r = np.asarray(row, dtype=np.float64).ravel()
    if r.size == 0:
        raise ValueError("empty logits row")
    if not np.all(np.isfinite(r)):
        raise ValueError("logits must be finite")
    M = float(r.max())
    t = int(np.argmax(r))                 # numpy returns the first maximum
    terms = np.exp(r - M)
    terms[t] = 0.0                        # the greedy token's own term is 1
    s = math.fsum(terms.tolist())
    c = 1.0 / (1.0 + s)
    eps = s / (1.0 + s)
    lse = M + math.log1p(s)
    return t, c, eps, lse


RowSource = Union[np.ndarray, Callable[[int, int], np.ndarray]]


def _row(logits: RowSource, b: int, i: int) -> np.ndarray:
    if callable(logits):
        return logits(b, i)
    return logits[b][i]


def confidence(logits: RowSource, B: int, L: int, mask, start, end):
    """Greedy tokens / confidences for every candidate position of a batch.

    Candidates of sequence b are the masked positions i with
    start[b] <= i < end[b] (Alg. 1 iterates over the masked positions of the
    active block).  Non-candidate entries get token -1, c = 0, eps = 1,
    lse = 0 and their logits are not touched.

    Returns float64/int arrays (tokens [B,L] int64, conf, eps, lse [B,L]).
    """
    mask = np.asarray(mask)
    tokens = np.full((B, L), -1, dtype=np.int64)
    conf = np.zeros((B, L), dtype=np.float64)
    eps = np.ones((B, L), dtype=np.float64)
    lse = np.zeros((B, L), dtype=np.float64)
    for b in range(B):
        lo, hi = int(start[b]), int(end[b])
        if not (0 <= lo <= hi <= L):
            raise ValueError(f"bad block bounds for sequence {b}: [{lo},{hi}) with L={L}")
        for i in range(lo, hi):
            if mask[b, i]:
                tokens[b, i], conf[b, i], eps[b, i], lse[b, i] = position_confidence(_row(logits, b, i))
    return tokens, conf, eps, lse
