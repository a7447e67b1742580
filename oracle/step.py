"""One decoding step of Fast-dLLM++ (oracle; test infrastructure only).

Alg. 1, body of the per-block while loop, after the model call: compute the
greedy token and confidence of every masked position of the active block,
choose the commit set with the selected rule, and reveal the chosen
positions (x_i <- x*_i; the position stops being masked).
"""
from __future__ import annotations

import dataclasses

import numpy as np

from .confidence import confidence
from .rules import select


@dataclasses.dataclass
class StepResult:
    tokens: np.ndarray      # [B, L] int64, -1 for non-candidates
    conf: np.ndarray        # [B, L] float64
    eps: np.ndarray         # [B, L] float64
    lse: np.ndarray         # [B, L] float64
    commit: np.ndarray      # [B, L] uint8
    n_commit: np.ndarray    # [B] int64
    x: np.ndarray           # [B, L] updated sequence
    mask: np.ndarray        # [B, L] updated mask
    flagged: np.ndarray     # [B] bool
    details: list


def decode_step(logits, B: int, L: int, mask, start, end, x, rule: str, param: float,
                eta=None) -> StepResult:
    """Oracle decode step.

    ``logits`` is a [B][L] indexable of 1-D rows or a callable row(b, i);
    only candidate rows are read.  ``mask``/``x`` are [B, L] arrays and are
    not modified; the updated copies are returned.  ``eta`` is the robust
    rule's calibration allowance ([B, L] or scalar).
    """
    mask = np.array(mask, dtype=np.uint8, copy=True)
    x = np.array(x, dtype=np.int64, copy=True)
    tokens, conf, eps, lse = confidence(logits, B, L, mask, start, end)
    commit, n_commit, flagged, details = select(eps, conf, mask, start, end, rule, param, eta=eta)
    hit = commit.astype(bool)
    x[hit] = tokens[hit]
    mask[hit] = 0
    return StepResult(tokens, conf, eps, lse, commit, n_commit, x, mask, flagged, details)
