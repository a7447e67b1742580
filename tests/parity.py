"""Helpers shared by the GPU parity tests: run the HIP path and the oracle on
the same seeded inputs and compare them.

Bars (from the method's precision needs):
  * tokens, commit masks, n_commit, x, mask: bit-exact, except blocks the
    oracle flags as within 1e-6 of a decision boundary (reported);
  * conf and lse: relative error <= 1e-5 (lse relative to max(|lse|, 1));
  * eps: relative error <= 1e-5, or absolute error <= EPS_ATOL = 2^-48: the
    GPU forms s' = (S - e_M) / e_M from a double sum S that holds the greedy
    term e_M (about 1) next to the others, so below eps ~ 1e-11 the double's
    last bits (2^-53 of S per addition) dominate the relative error.
"""
from __future__ import annotations

import sys
from typing import Iterable, List, Optional, Sequence, Tuple

import numpy as np
import torch

import oracle

CONF_RTOL = 1e-5
LSE_RTOL = 1e-5
EPS_RTOL = 1e-5
EPS_ATOL = 2.0 ** -48
MAX_BLOCK = 1024        # longest block the library accepts (FDLLM_MAX_BLOCK)


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def row_source(logits: torch.Tensor):
    """Oracle row accessor reading single rows of a (GPU) tensor exactly as float64."""
    def row(b, i):
        return logits[b, i].to(torch.float64).cpu().numpy()
    return row


def candidates(mask: np.ndarray, start: np.ndarray, end: np.ndarray, bs: Iterable[int]):
    out = []
    for b in bs:
        for i in range(int(start[b]), int(end[b])):
            if mask[b, i]:
                out.append((b, i))
    return out


def compare_rows(g_tok, g_conf, g_eps, g_lse, o_tok, o_conf, o_eps, o_lse, cells) -> dict:
    """Compare per-position outputs at `cells`; returns error statistics."""
    bad = []
    worst = dict(conf=0.0, eps=0.0, lse=0.0)
    for (b, i) in cells:
        if int(g_tok[b, i]) != int(o_tok[b, i]):
            bad.append(("token", b, i, int(g_tok[b, i]), int(o_tok[b, i])))
        ec = abs(float(g_conf[b, i]) - o_conf[b, i]) / max(abs(o_conf[b, i]), 1e-30)
        de = abs(float(g_eps[b, i]) - o_eps[b, i])
        ee = de / max(abs(o_eps[b, i]), 1e-30) if de > EPS_ATOL else 0.0
        el = abs(float(g_lse[b, i]) - o_lse[b, i]) / max(abs(o_lse[b, i]), 1.0)
        worst["conf"] = max(worst["conf"], ec)
        worst["eps"] = max(worst["eps"], ee)
        worst["lse"] = max(worst["lse"], el)
        if ec > CONF_RTOL:
            bad.append(("conf", b, i, float(g_conf[b, i]), o_conf[b, i]))
        if ee > EPS_RTOL:
            bad.append(("eps", b, i, float(g_eps[b, i]), o_eps[b, i]))
        if el > LSE_RTOL:
            bad.append(("lse", b, i, float(g_lse[b, i]), o_lse[b, i]))
    assert not bad, f"{len(bad)} mismatches, first: {bad[:5]}"
    return worst


def gpu_confidence(fd, inp):
    B, L, V = inp.logits.shape
    dev = inp.logits.device
    tok = torch.full((B, L), -7, dtype=torch.int32, device=dev)
    conf = torch.full((B, L), -7.0, dtype=torch.float32, device=dev)
    eps = torch.full((B, L), -7.0, dtype=torch.float32, device=dev)
    lse = torch.full((B, L), -7.0, dtype=torch.float32, device=dev)
    fd.fdllm_confidence(inp.logits, inp.mask, inp.start, inp.end, tok, conf, eps, lse)
    torch.cuda.synchronize()
    return tok, conf, eps, lse


def oracle_confidence_subset(inp, bs: Sequence[int]):
    """Oracle outputs for the sequences in bs (others left at defaults)."""
    B, L, V = inp.logits.shape
    mask = inp.mask.cpu().numpy()
    start = inp.start.cpu().numpy()
    end = inp.end.cpu().numpy()
    sub_mask = np.zeros_like(mask)
    for b in bs:
        sub_mask[b] = mask[b]
    return oracle.confidence(row_source(inp.logits), B, L, sub_mask, start, end)


def check_defaults(g_tok, g_conf, g_eps, g_lse, mask, start, end, bs):
    for b in bs:
        for i in range(mask.shape[1]):
            cand = int(start[b]) <= i < int(end[b]) and mask[b, i] and int(end[b]) - int(start[b]) <= MAX_BLOCK
            if not cand:
                assert (int(g_tok[b, i]), float(g_conf[b, i]), float(g_eps[b, i]), float(g_lse[b, i])) \
                    == (-1, 0.0, 1.0, 0.0), (b, i)


def compare_selection(g_commit, g_n, o_commit, o_n, flagged, bs) -> Tuple[int, int]:
    """Commit masks and counts must match on every unflagged block in bs.

    Returns (number flagged, number of flagged blocks that still match)."""
    nflag, nflag_match = 0, 0
    bad = []
    for b in bs:
        same = np.array_equal(g_commit[b], o_commit[b]) and int(g_n[b]) == int(o_n[b])
        if flagged[b]:
            nflag += 1
            nflag_match += int(same)
        elif not same:
            bad.append(b)
    assert not bad, f"unflagged blocks differ: {bad[:10]}"
    return nflag, nflag_match
