"""Logit magnitudes up to the documented bound, and the opt-in input check.

* Parity at large offsets: every logit shifted by 1e4, 1e6 or close to the
  bound |logit| <= 1e7 (values beyond it clamped to the bound, so rows hold
  ties exactly at it), float32 and bf16, fused and split plans.  The oracle
  computes in float64 on the exact shifted values.
* fdllm_check_inputs: windows out of the span or too long, and NaN / inf /
  out-of-range logits in candidate rows, reported to the host; bad values in
  rows that are not candidates are ignored.
"""
import numpy as np
import pytest
import torch

import paper_2606_02955_amd as fd
import workloads
from parity import (say, candidates, compare_rows, check_defaults, pool_confidence, sub_mask,
                    selection_stats)

pytestmark = pytest.mark.gpu

BOUND = fd.MAX_ABS_LOGIT


# the largest magnitude of each dtype within the bound (1e7 is not a bf16 value)
DT_BOUND = {torch.float32: BOUND, torch.bfloat16: 9961472.0}


def _shifted(B, L, V, dt, offset, seed):
    inp = workloads.random_case(B, L, V, torch.float32, device="cuda", seed=seed, poison=False)
    lim = DT_BOUND[dt]
    lg = (inp.logits.double() + offset).clamp_(-lim, lim).to(dt)
    inp.logits = lg.contiguous()
    return inp


OFFSETS = [
    (torch.float32, 1e4), (torch.float32, -1e4), (torch.float32, 1e6),
    (torch.float32, BOUND - 8), (torch.float32, -(BOUND - 8)),
    (torch.bfloat16, 1e4), (torch.bfloat16, -1e6), (torch.bfloat16, 9928700.0),  # about halfway between the two top bf16 values: rows of two values, ties at the bound
]


@pytest.mark.parametrize("dt,offset", OFFSETS)
@pytest.mark.parametrize("B,L,V", [(4, 32, 126464), (130, 8, 5000), (260, 8, 5000)])
def test_large_offset_parity(gpu, oracle_pool, dt, offset, B, L, V):
    say(f"[offset] B={B} L={L} V={V} {dt} offset {offset:g}")
    inp = _shifted(B, L, V, dt, offset, seed=int(abs(offset)) % 97 + B)
    top = float(inp.logits.abs().max())
    assert top <= BOUND, top
    st, counts = gpu.fdllm_check_inputs(inp.logits, inp.mask, inp.start, inp.end)
    assert st == fd.OK and counts == [0, 0, 0]
    mask, x = inp.mask.clone(), inp.x.clone()
    o = dict(tokens=torch.empty((B, L), dtype=torch.int32, device="cuda"),
             conf=torch.empty((B, L), device="cuda"), eps=torch.empty((B, L), device="cuda"),
             lse=torch.empty((B, L), device="cuda"),
             commit=torch.empty((B, L), dtype=torch.uint8, device="cuda"),
             n_commit=torch.empty((B,), dtype=torch.int32, device="cuda"))
    gpu.fdllm_decode_step(inp.logits, mask, inp.start, inp.end, x, "profile", 1.0, **o)
    torch.cuda.synchronize()
    g = {k: v.cpu().numpy() for k, v in o.items()}
    assert np.isfinite(g["conf"]).all() and np.isfinite(g["eps"]).all() and np.isfinite(g["lse"]).all()
    m, s, e = inp.mask.cpu().numpy(), inp.start.cpu().numpy(), inp.end.cpu().numpy()
    tok, conf, eps, lse = pool_confidence(oracle_pool, inp.logits, m, s, e)
    cells = candidates(m, s, e, range(B))
    worst = compare_rows(g["tokens"], g["conf"], g["eps"], g["lse"], tok, conf, eps, lse, cells)
    check_defaults(g["tokens"], g["conf"], g["eps"], g["lse"], m, s, e, range(B))
    oc, on, fl = oracle_pool.select(eps, conf, m, s, e, "profile", 1.0)
    stt = selection_stats(g["commit"], g["n_commit"], oc, on, fl, range(B))
    assert stt["mismatches"] == 0, stt
    say(f"  {len(cells)} rows, worst {worst}, flagged {stt['flagged']}")


def _clean(B, L, V, dt, seed=3):
    inp = workloads.random_case(B, L, V, dt, device="cuda", seed=seed)   # bf16: NaN-poisoned non-candidates
    return inp


def _first_candidate(inp):
    m, s, e = inp.mask.cpu().numpy(), inp.start.cpu().numpy(), inp.end.cpu().numpy()
    cells = candidates(m, s, e, range(inp.B))
    assert cells
    return cells[len(cells) // 2]


@pytest.mark.parametrize("B,L,V,dt", [(5, 40, 1000, torch.bfloat16), (3, 30, 997, torch.bfloat16),
                                      (4, 20, 2048, torch.float32), (2, 16, 333, torch.float32)])
def test_check_inputs_values(gpu, B, L, V, dt):
    say(f"[check inputs] B={B} L={L} V={V} {dt}")
    inp = _clean(B, L, V, dt)
    st, counts = gpu.fdllm_check_inputs(inp.logits, inp.mask, inp.start, inp.end)
    assert st == fd.OK and counts == [0, 0, 0]          # NaN poison outside the candidates is ignored
    b, i = _first_candidate(inp)
    v = V // 3
    keep = inp.logits[b, i, v].clone()
    for bad, want in ((float("nan"), fd.ERR_NONFINITE), (float("inf"), fd.ERR_NONFINITE),
                      (-float("inf"), fd.ERR_NONFINITE), (2.0e7, fd.ERR_NONFINITE),
                      (-1.5e7, fd.ERR_NONFINITE), (BOUND, fd.OK), (-BOUND, fd.OK)):
        inp.logits[b, i, v] = bad
        st, counts = gpu.fdllm_check_inputs(inp.logits, inp.mask, inp.start, inp.end)
        if dt == torch.bfloat16 and abs(bad) == BOUND:
            # 1e7 is not a bf16 value: it rounds to 9961472 or 10027008
            want = fd.OK if float(inp.logits[b, i, v].float().abs()) <= BOUND else fd.ERR_NONFINITE
        assert st == want, (bad, st, counts)
        assert counts[:2] == [0, 0] and counts[2] == (0 if want == fd.OK else 1)
    inp.logits[b, i, v] = keep
    # the same value in a row that is not a candidate: not scanned
    inp.mask[b, i] = 0
    inp.logits[b, i, v] = float("nan")
    st, counts = gpu.fdllm_check_inputs(inp.logits, inp.mask, inp.start, inp.end)
    assert st == fd.OK and counts == [0, 0, 0]


def test_check_inputs_windows(gpu):
    B, L, V = 6, 1100, 64
    inp = workloads.random_case(B, L, V, torch.bfloat16, device="cuda", seed=9, window=64)
    st, counts = gpu.fdllm_check_inputs(inp.logits, inp.mask, inp.start, inp.end)
    assert st == fd.OK and counts == [0, 0, 0]
    s0, e0 = inp.start.clone(), inp.end.clone()
    inp.start[1], inp.end[1] = 10, 5                      # start > end
    inp.end[3] = L + 1                                    # end beyond the span
    st, counts = gpu.fdllm_check_inputs(inp.logits, inp.mask, inp.start, inp.end)
    assert st == fd.ERR_BOUNDS and counts[0] == 2
    inp.start.copy_(s0); inp.end.copy_(e0)
    inp.start[2], inp.end[2] = 0, 1025                    # longer than the block limit
    inp.start[4], inp.end[4] = 50, 50 + 1024              # exactly the limit: fine
    st, counts = gpu.fdllm_check_inputs(inp.logits, inp.mask, inp.start, inp.end)
    assert st == fd.ERR_BLOCK_TOO_LARGE and counts[:2] == [0, 1]
    # n_commit reports the bad window of the decode step as -1
    n = torch.empty(B, dtype=torch.int32, device="cuda")
    inp.mask.zero_()                                      # nothing to read anywhere
    gpu.fdllm_decode_step(inp.logits, inp.mask, inp.start, inp.end, inp.x, "profile", 1.0, n_commit=n)
    torch.cuda.synchronize()
    assert int(n[2]) == -1 and int(n[4]) == 0
