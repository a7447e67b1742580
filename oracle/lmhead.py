"""Logits from hidden states (oracle; test infrastructure only).

Alg. 1's model call ends in the output projection: the logits of a masked
position are the dot products of its final hidden state with every row of
the output embedding, l_v = sum_k h_k W_vk; the per-position confidence
(Sec. 3 "Notation") is then taken on those logits exactly as for given
logits.  Here the dot products are formed in float64 by a library matrix
product on the exact float64 values of the bf16 operands: every product
h_k W_vk is exact in float64, and the float64 sums carry a relative error of
at most about d * 2^-53, negligible next to the float32 accumulation of the
matrix cores.
"""
from __future__ import annotations

import numpy as np


def logits_rows(hidden_rows: np.ndarray, weight: np.ndarray) -> np.ndarray:
    """[n, V] float64 logits of n hidden rows [n, d] against weight [V, d]."""
    h = np.asarray(hidden_rows, dtype=np.float64)
    w = np.asarray(weight, dtype=np.float64)
    return h @ w.T


def row_source(hidden: np.ndarray, weight: np.ndarray):
    """Row accessor row(b, i) -> float64 logits of position (b, i), computed on demand.

    ``hidden`` is [B, L, d] and ``weight`` [V, d], both exact float64 copies
    of the bf16 operands."""
    w = np.asarray(weight, dtype=np.float64)
    h = np.asarray(hidden, dtype=np.float64)

    def row(b, i):
        return w @ h[b, i]
    return row


def accumulation_bound(hidden_row: np.ndarray, weight: np.ndarray, unit: float) -> float:
    """max_v sum_k |h_k W_vk| * unit: a bound on how far any floating-point
    evaluation of the row's logits with relative rounding `unit` per
    accumulated term may stray from the exact values."""
    h = np.abs(np.asarray(hidden_row, dtype=np.float64))
    w = np.abs(np.asarray(weight, dtype=np.float64))
    return float((w @ h).max() * unit)
