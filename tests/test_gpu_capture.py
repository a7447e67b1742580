"""The decode step captured into a HIP graph (torch.cuda.CUDAGraph) and
replayed: a large batch whose last sequences run on the library's side stream
(forked from and joined back to the capturing stream by events), the same
with those sequences' conf and eps in the workspace, small batches (two
launches; one of them with windows wider than a wavefront), and the
static-scratch entry point.  Every replay, with eager work
between replays, must give the eager call's outputs bit for bit."""
import pytest
import torch

import workloads
from parity import say

pytestmark = pytest.mark.gpu


def _outs(B, L, dev, scores):
    o = dict(commit=torch.full((B, L), 9, dtype=torch.uint8, device=dev),
             n_commit=torch.full((B,), -9, dtype=torch.int32, device=dev),
             lse=torch.full((B, L), -9.0, device=dev))
    if scores:
        o.update(tokens=torch.full((B, L), -9, dtype=torch.int32, device=dev),
                 conf=torch.full((B, L), -9.0, device=dev), eps=torch.full((B, L), -9.0, device=dev))
    return o


@pytest.mark.parametrize("B,L,V,dt,scores,static", [
    (260, 8, 4096, torch.bfloat16, True, False),    # 4 sequences beyond 256 CUs, outputs given
    (300, 8, 2048, torch.float32, False, False),    # 44 beyond, their conf / eps in the workspace
    (8, 32, 20000, torch.bfloat16, False, False),   # a small batch: the pass, then the selection
    (16, 300, 3000, torch.bfloat16, True, False),   # 32 row groups over 300-wide windows, wide selection
    (300, 8, 2048, torch.float32, False, True),     # the static entry point: no side stream
    (8, 32, 20000, torch.bfloat16, False, True),
])
def test_decode_step_graph_replays(gpu, B, L, V, dt, scores, static):
    inp = workloads.random_case(B, L, V, dt, device="cuda", seed=3 * B + L, window=L)
    dev = inp.logits.device
    say(f"[graph capture] B={B} L={L} V={V} {dt} scores={scores} static={static}")
    need = gpu.fdllm_workspace_size(B, L, V, dt)
    ws = torch.empty(max(need, 1), dtype=torch.uint8, device=dev)
    mask0, x0 = inp.mask.clone(), inp.x.clone()

    # eager reference (also creates whatever the library sets up on first use)
    mask, x = mask0.clone(), x0.clone()
    ref = _outs(B, L, dev, scores)
    gpu.fdllm_decode_step(inp.logits, mask, inp.start, inp.end, x, "profile", 1.0, workspace=ws, **ref)
    torch.cuda.synchronize()
    ref.update(mask=mask, x=x)

    gmask, gx = mask0.clone(), x0.clone()
    gout = _outs(B, L, dev, scores)
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        gmask.copy_(mask0)
        gx.copy_(x0)
        if static:
            gpu.fdllm_decode_step_static(inp.logits, gmask, inp.start, inp.end, gx, "profile", 1.0, **gout)
        else:
            gpu.fdllm_decode_step(inp.logits, gmask, inp.start, inp.end, gx, "profile", 1.0, workspace=ws,
                                  **gout)
    torch.cuda.synchronize()
    gout.update(mask=gmask, x=gx)
    for r in range(3):
        # eager work between replays: poison every output the replay must rewrite
        for t in gout.values():
            t.fill_(7 + r)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for k in ref:
            assert torch.equal(gout[k].view(torch.uint8), ref[k].view(torch.uint8)), (r, k)
    say(f"  3 replays identical ({int(ref['n_commit'].clamp(min=0).sum())} commits)")
