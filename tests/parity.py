"""Helpers shared by the GPU parity tests: run the HIP path and the oracle on
the same seeded inputs and compare them.

Bars (from the method's precision needs):
  * tokens, commit masks, n_commit, x, mask: bit-exact, except blocks the
    oracle flags as within 1e-6 of a decision boundary (reported);
  * conf and lse: relative error <= 1e-5 (lse relative to max(|lse|, 1));
  * eps: relative error <= 1e-5, or absolute error <= EPS_ATOL = 1e-30 (the
    vocabulary pass sums every term but the greedy one, so eps keeps its
    relative accuracy until the float32 terms underflow).  The LM-head folds
    keep the greedy term e_M (about 1) in their double sum and form
    s' = (S - e_M) / e_M, so below eps ~ 1e-11 the double's last bits set
    the error there: EPS_ATOL_LMHEAD = 2^-48.
"""
from __future__ import annotations

import os
import sys
from typing import Iterable, List, Optional, Sequence, Tuple

if __name__ == "__main__":      # run as a script: the repository root is not on the path
    sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))

import numpy as np
import torch

import oracle

CONF_RTOL = 1e-5
LSE_RTOL = 1e-5
EPS_RTOL = 1e-5
EPS_ATOL = 1e-30
EPS_ATOL_LMHEAD = 2.0 ** -48
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
    """Non-candidate positions of the sequences bs hold the default outputs."""
    bs = np.asarray(list(bs), dtype=np.int64)
    if bs.size == 0:
        return
    L = mask.shape[1]
    pos = np.arange(L)[None, :]
    s = np.asarray(start)[bs][:, None].astype(np.int64)
    e = np.asarray(end)[bs][:, None].astype(np.int64)
    cand = (pos >= s) & (pos < e) & (np.asarray(mask)[bs] != 0) & ((e - s) <= MAX_BLOCK)
    dead = ~cand
    ok = ((np.asarray(g_tok)[bs] == -1) & (np.asarray(g_conf)[bs] == 0.0) &
          (np.asarray(g_eps)[bs] == 1.0) & (np.asarray(g_lse)[bs] == 0.0))
    bad = np.argwhere(dead & ~ok)
    assert bad.size == 0, f"default outputs wrong at {[(int(bs[r]), int(c)) for r, c in bad[:5]]}"


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


# ---------------------------------------------------------------------------
# whole-workload checks: the oracle in worker processes (oracle.parallel)
# ---------------------------------------------------------------------------
def check_bounds(start: np.ndarray, end: np.ndarray, L: int):
    """The oracle's bounds rule (it raises on a bad window)."""
    for b in range(len(start)):
        lo, hi = int(start[b]), int(end[b])
        if not (0 <= lo <= hi <= L):
            raise ValueError(f"bad block bounds for sequence {b}: [{lo},{hi}) with L={L}")


def pool_confidence(pool, logits: torch.Tensor, mask: np.ndarray, start: np.ndarray,
                    end: np.ndarray, bs: Optional[Sequence[int]] = None):
    """Oracle (tokens, conf, eps, lse) [B, L] of every candidate of the
    sequences bs (all when None), rows copied from the GPU tensor's exact bits;
    non-candidates and other sequences keep the oracle's defaults."""
    from oracle.parallel import scatter_confidence
    B, L, V = logits.shape
    check_bounds(start, end, L)
    bs = range(B) if bs is None else bs
    cells = candidates(mask, start, end, bs)
    kind = "bf16" if logits.dtype == torch.bfloat16 else "f32"
    flat = logits.view(B * L, V)
    idx = torch.tensor([b * L + i for b, i in cells], dtype=torch.long, device=logits.device)

    def fill(first, cnt, out):
        rows = flat.index_select(0, idx[first:first + cnt])
        torch.from_numpy(out).copy_(rows.view(torch.int16) if kind == "bf16" else rows)

    res = pool.rows_confidence(fill, len(cells), V, kind)
    return scatter_confidence(B, L, cells, res)


def sub_mask(mask: np.ndarray, bs: Sequence[int]) -> np.ndarray:
    m = np.zeros_like(mask)
    idx = list(bs)
    m[idx] = mask[idx]
    return m


def selection_stats(g_commit, g_n, o_commit, o_n, flagged, bs) -> dict:
    """Counts of a selection comparison on the blocks bs (no assertion)."""
    st = dict(blocks=0, mismatches=0, flagged=0, flagged_matching=0, bad=[])
    for b in bs:
        same = np.array_equal(g_commit[b], o_commit[b]) and int(g_n[b]) == int(o_n[b])
        st["blocks"] += 1
        if flagged[b]:
            st["flagged"] += 1
            st["flagged_matching"] += int(same)
        elif not same:
            st["mismatches"] += 1
            st["bad"].append(int(b))
    return st


class ParityTally:
    """Per-workload totals of the comparisons, printed and, when the
    environment names a file (FDLLM_PARITY_REPORT), appended to it as JSON."""

    def __init__(self, workload: str, **info):
        self.d = dict(workload=workload, block_checks=0, mismatches=0, flagged=0,
                      flagged_matching=0, rows=0, worst=dict(conf=0.0, eps=0.0, lse=0.0),
                      rules={}, **info)

    def rows_checked(self, n: int, worst: dict):
        self.d["rows"] += n
        for k, v in worst.items():
            self.d["worst"][k] = max(self.d["worst"][k], v)

    def selection(self, rule: str, st: dict):
        r = self.d["rules"].setdefault(rule, dict(block_checks=0, mismatches=0, flagged=0,
                                                  flagged_matching=0))
        for key, src in (("block_checks", "blocks"), ("mismatches", "mismatches"),
                         ("flagged", "flagged"), ("flagged_matching", "flagged_matching")):
            r[key] += st[src]
            self.d[key] += st[src]
        assert st["mismatches"] == 0, f"{rule}: unflagged blocks differ: {st['bad'][:10]}"

    def note(self, **kv):
        self.d.update(kv)

    def finish(self):
        import json
        import os
        say(f"  parity {self.d['workload']}: {self.d['block_checks']} block checks, "
            f"{self.d['mismatches']} mismatches, {self.d['flagged']} flagged "
            f"({self.d['flagged_matching']} matching), {self.d['rows']} rows, worst {self.d['worst']}")
        path = os.environ.get("FDLLM_PARITY_REPORT")
        if path:
            with open(path, "a") as fh:
                fh.write(json.dumps(self.d) + "\n")
        return self.d


SHAPES = {
    "single_block_b1_l32": "B=1, one block of 32, fp32; one step, every row",
    "generation_b8_g256": ("B=8, 256 positions in blocks of 32, bf16; seven whole generations (one "
                           "driven by each rule), every step, every sequence"),
    "sparse_b64_g512": "B=64, span 512, 1..32 masked per block, bf16; one step, every candidate row",
    "bimodal_b256_g1024": ("B=256, 1024 positions in blocks of 64, bf16; the whole generation (profile "
                           "f=1 drives it): every step for the 16 flat sequences and 4 others, every "
                           "sequence at step 0"),
    "stress_b1024_l32": "B=1024, L=32, bf16, 8.3 GB; one step, every block",
}
ORDER = list(SHAPES)


def render_report(records) -> str:
    """Markdown summary of the JSON lines ParityTally appends to FDLLM_PARITY_REPORT."""
    recs = sorted(records, key=lambda r: ORDER.index(r["workload"]) if r["workload"] in ORDER else 99)
    out = ["| workload | what is checked | block checks | unflagged mismatches | flagged | flagged and "
           "matching | row comparisons | worst rel. err conf / eps / lse |",
           "|---|---|---|---|---|---|---|---|"]
    tot = dict(block_checks=0, mismatches=0, flagged=0, flagged_matching=0, rows=0)
    for r in recs:
        w = r["worst"]
        out.append(f"| {r['workload']} | {SHAPES.get(r['workload'], '')} | {r['block_checks']} | "
                   f"{r['mismatches']} | {r['flagged']} | {r['flagged_matching']} | {r['rows']} | "
                   f"{w['conf']:.1e} / {w['eps']:.1e} / {w['lse']:.1e} |")
        for k in tot:
            tot[k] += r[k]
    out.append(f"| **all** | | **{tot['block_checks']}** | **{tot['mismatches']}** | {tot['flagged']} | "
               f"{tot['flagged_matching']} | {tot['rows']} | |")
    out += ["", "Per rule:", "",
            "| workload | rule | block checks | mismatches | flagged | flagged and matching |",
            "|---|---|---|---|---|---|"]
    for r in recs:
        for rule, st in r["rules"].items():
            out.append(f"| {r['workload']} | {rule} | {st['block_checks']} | {st['mismatches']} | "
                       f"{st['flagged']} | {st['flagged_matching']} |")
    notes = []
    for r in recs:
        if "steps_per_generation" in r:
            notes.append(f"* {r['workload']} steps per whole generation (NFE): " +
                         ", ".join(f"{k} {v}" for k, v in r["steps_per_generation"].items()) + ".")
        if "every_step_sequences" in r:
            notes.append(f"* {r['workload']}: {r.get('steps')} steps; sequences checked at every step: "
                         f"{r['every_step_sequences']} (flat: {r.get('flat_sequences')}).")
    if notes:
        out += [""] + notes
    return "\n".join(out) + "\n"


if __name__ == "__main__":
    # python tests/parity.py REPORT.jsonl: the markdown tables of a parity run
    import json
    import sys
    with open(sys.argv[1]) as fh:
        print(render_report([json.loads(line) for line in fh if line.strip()]), end="")
