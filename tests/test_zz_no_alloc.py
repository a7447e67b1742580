"""fdllm_decode_step_static (the decode step with the library's static
scratch, for callers that cannot allocate) against fdllm_decode_step given a
workspace: bitwise the same outputs, on calls in a row whose inputs shrink,
called through the C ABI."""
import ctypes

import pytest
import torch

import paper_2606_02955_amd as fd
import workloads
from parity import say

pytestmark = pytest.mark.gpu

SEL = {"profile": 2, "factor": 1, "threshold": 0, "robust": 3}


def _p(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _outs(B, L, dev, with_scores=True):
    o = dict(tokens=torch.full((B, L), -7, dtype=torch.int32, device=dev),
             conf=torch.full((B, L), -7.0, device=dev), eps=torch.full((B, L), -7.0, device=dev),
             lse=torch.full((B, L), -7.0, device=dev),
             commit=torch.full((B, L), 7, dtype=torch.uint8, device=dev),
             n_commit=torch.full((B,), -7, dtype=torch.int32, device=dev))
    if not with_scores:
        o["tokens"] = o["conf"] = o["eps"] = None
    return o


def _run(lib, static, inp, rule, param, with_scores, eta_uniform=0.0):
    B, L, V = inp.logits.shape
    dev = inp.logits.device
    mask, x = inp.mask.clone(), inp.x.clone()
    o = _outs(B, L, dev, with_scores)
    dt = 0 if inp.logits.dtype == torch.bfloat16 else 1
    stream = ctypes.c_void_p(torch.cuda.current_stream(dev).cuda_stream)
    head = [_p(inp.logits), dt, B, L, V, _p(mask), _p(inp.start), _p(inp.end), _p(x), SEL[rule],
            ctypes.c_float(param), None, ctypes.c_float(eta_uniform), _p(o["tokens"]), _p(o["conf"]),
            _p(o["eps"]), _p(o["lse"]), _p(o["commit"]), _p(o["n_commit"])]
    if static:
        st = lib.fdllm_decode_step_static(*head, stream)
        ws = None
    else:
        n = ctypes.c_size_t(0)
        assert lib.fdllm_workspace_size(B, L, V, dt, ctypes.byref(n)) == 0
        ws = torch.empty(max(int(n.value), 1), dtype=torch.uint8, device=dev)
        st = lib.fdllm_decode_step(*head, _p(ws), ctypes.c_size_t(int(n.value)), stream)
    assert st == 0, fd.status_string(st)
    torch.cuda.synchronize()
    o.update(mask=mask, x=x)
    return {k: v for k, v in o.items() if v is not None}


def _same(a, b):
    assert a.keys() == b.keys()
    for k in a:
        assert torch.equal(a[k].view(torch.uint8), b[k].view(torch.uint8)), k


# shrinking inputs: every plan that uses scratch (rows split over several
# workgroups with their parts in scratch; rows split within a workgroup; wide
# spans), large batches (one workgroup per sequence, their last sequences
# beyond a multiple of the CU count as a small batch: on a side stream for
# fdllm_decode_step, after the one-kernel part for the static call), and
# calls without tokens / conf / eps, whose values then live in the scratch
CASES = [
    (8, 32, 126464, torch.bfloat16, "profile", 1.0, True),
    (2, 16, 126464, torch.bfloat16, "factor", 1.0, False),
    (40, 64, 50000, torch.bfloat16, "threshold", 0.9, True),
    (3, 32, 5000, torch.float32, "robust", 0.9, False),
    (300, 8, 4096, torch.float32, "threshold", 0.9, False),
    (260, 8, 4096, torch.bfloat16, "profile", 0.75, True),
    (24, 200, 8000, torch.bfloat16, "profile", 1.0, False),
    (1, 32, 126464, torch.float32, "profile", 1.0, False),
]


def test_static_matches_workspace_calls_in_a_row(gpu):
    lib = fd.load()
    for k, (B, L, V, dt, rule, param, scores) in enumerate(CASES):
        say(f"[static scratch] call {k}: B={B} L={L} V={V} {dt} {rule}({param}) scores={scores}")
        inp = workloads.random_case(B, L, V, dt, device="cuda", seed=70 + k,
                                    window=min(L, 160))
        eta = 0.01 if rule == "robust" else 0.0
        ref = _run(lib, False, inp, rule, param, scores, eta)
        got = _run(lib, True, inp, rule, param, scores, eta)
        _same(got, ref)
        # again, right after: the scratch keeps the last call's contents
        got2 = _run(lib, True, inp, rule, param, scores, eta)
        _same(got2, ref)
        say(f"  commits {int(ref['n_commit'].clamp(min=0).sum())}: identical")
