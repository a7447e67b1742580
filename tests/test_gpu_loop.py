"""The device-resident decoding loop (Alg. 1 outer loops) against the oracle.

The synthetic logits producer and the block advance are checked bit for bit
against their CPU implementations in workloads.synth; whole generations are
replayed on the CPU with the oracle's decode step, step by step, on logits
the CPU builds itself from the same counter-based recipe.
"""
import numpy as np
import pytest
import torch

import oracle
from parity import say
from workloads import synth

pytestmark = pytest.mark.gpu

BF16_SENTINEL = 0x7FC0


@pytest.mark.parametrize("V", [1000, 1001, 126464])
def test_synth_logits_match_cpu_recipe(gpu, V):
    B, L, blk, seed, step = 3, 40, 8, 0x1234_5678_9ABC_DEF0, 5
    logits = torch.empty((B, L, V), dtype=torch.bfloat16, device="cuda")
    logits.view(torch.int16).fill_(BF16_SENTINEL)
    spans = [(0, 8), (16, 24), (40, 40)]
    start = torch.tensor([s for s, _ in spans], dtype=torch.int32, device="cuda")
    end = torch.tensor([e for _, e in spans], dtype=torch.int32, device="cuda")
    say(f"[synth] V={V}")
    gpu.fdllm_synth_logits(logits, start, end, blk, seed, step)
    torch.cuda.synchronize()
    got = logits.view(torch.int16).cpu().numpy().view(np.uint16)
    for b, (s, e) in enumerate(spans):
        for i in range(L):
            if s <= i < e:
                assert np.array_equal(got[b, i], synth.row_bits(seed, b, i, step, V)), (b, i)
            elif i % 7 == 0:
                assert (got[b, i] == BF16_SENTINEL).all(), (b, i)


def test_advance_blocks_match_cpu(gpu):
    rng = np.random.default_rng(3)
    B, G, blk = 50, 100, 16                         # the last block is partial
    mask = (rng.random((B, G)) < 0.05).astype(np.uint8)
    mask[::7] = 0                                   # some finished sequences
    start = (rng.integers(0, 7, B) * blk).astype(np.int32)
    end = np.minimum(start + blk, G).astype(np.int32)
    s_d, e_d = torch.from_numpy(start).cuda(), torch.from_numpy(end).cuda()
    n_d = torch.full((1,), -5, dtype=torch.int32, device="cuda")
    gpu.fdllm_advance_blocks(torch.from_numpy(mask).cuda(), s_d, e_d, blk, n_d)
    torch.cuda.synchronize()
    n = oracle.advance_blocks(mask, start, end, G, blk)
    assert s_d.cpu().numpy().tolist() == start.tolist()
    assert e_d.cpu().numpy().tolist() == end.tolist()
    assert int(n_d[0]) == n


def _replay(seed, B, G, blk, V, rule, p, eta, hist, steps_gpu, x_gpu):
    """The oracle's generation on CPU-built logits; compares every step."""
    mask = np.ones((B, G), dtype=np.uint8)
    x = np.full((B, G), -1, dtype=np.int64)
    start = np.zeros(B, dtype=np.int64)
    end = np.full(B, min(blk, G), dtype=np.int64)
    diverged = set()
    t, active, flagged_total = 0, B, 0
    while active:
        r = oracle.decode_step(lambda b, i: synth.row(seed, b, i, t, V), B, G, mask, start, end, x,
                               rule, p, eta=eta)
        for b in range(B):
            if b in diverged:
                continue
            if int(r.n_commit[b]) != int(hist[t, b]):
                assert r.flagged[b], (t, b, int(r.n_commit[b]), int(hist[t, b]))
                diverged.add(b)
            flagged_total += int(r.flagged[b])
        mask, x = r.mask, r.x
        active = oracle.advance_blocks(mask, start, end, G, blk)
        t += 1
    assert not mask.any()
    for b in range(B):
        if b not in diverged:
            assert np.array_equal(x[b], x_gpu[b]), b
    if not diverged:
        assert t == steps_gpu
    return t, diverged, flagged_total


@pytest.mark.parametrize("rule,p", [("profile", 1.0), ("profile", 2.0), ("factor", 1.0),
                                    ("threshold", 0.9), ("robust", 0.75)])
def test_generation_vs_oracle(gpu, rule, p):
    B, G, blk, V, seed = 4, 48, 16, 2048, 99
    eta_u = 0.03 if rule == "robust" else 0.0
    say(f"[generation] {rule}({p}) B={B} G={G} blk={blk} V={V}")
    gen = gpu.Generation(B, G, blk, V, seed, rule, p, eta_uniform=eta_u, chunk=4, use_graph=True)
    steps = gen.run()
    torch.cuda.synchronize()
    hist = gen.hist.cpu().numpy()
    x_gpu = gen.x.cpu().numpy()
    assert not gen.mask.any()
    t, diverged, nflag = _replay(seed, B, G, blk, V, rule, p, eta_u if rule == "robust" else None,
                                 hist, steps, x_gpu)
    say(f"  steps {steps} (oracle {t}), diverged after a flagged step: {sorted(diverged)}, flagged {nflag}")
    gen.close()


def test_generation_eta_tensor_vs_oracle(gpu):
    """The robust rule with a per-position allowance [B, G] (some entries
    negative, which count as 0) through the whole device loop."""
    B, G, blk, V, seed = 5, 40, 8, 1500, 7
    rng = np.random.default_rng(11)
    eta = rng.uniform(-0.01, 0.06, (B, G)).astype(np.float32)
    eta[1] = 0.0
    say(f"[generation eta tensor] B={B} G={G} blk={blk} V={V}")
    gen = gpu.Generation(B, G, blk, V, seed, "robust", 0.8, eta=torch.from_numpy(eta).cuda(),
                         chunk=3, use_graph=True)
    steps = gen.run()
    torch.cuda.synchronize()
    t, diverged, nflag = _replay(seed, B, G, blk, V, "robust", 0.8, eta, gen.hist.cpu().numpy(),
                                 steps, gen.x.cpu().numpy())
    say(f"  steps {steps} (oracle {t}), diverged {sorted(diverged)}, flagged {nflag}")
    gen.close()


@pytest.mark.parametrize("B,G,blk,V", [(8, 256, 32, 126464), (130, 64, 16, 512), (260, 64, 16, 512)])
def test_generation_graph_equals_eager(gpu, B, G, blk, V):
    """Graph replay in chunks, direct launches with a host check every step,
    and a second run of the same object all give the same generation."""
    seed = 2026
    say(f"[generation graph vs eager] B={B} G={G} blk={blk} V={V}")
    a = gpu.Generation(B, G, blk, V, seed, "profile", 1.0, chunk=8, use_graph=True)
    b = gpu.Generation(B, G, blk, V, seed, "profile", 1.0, chunk=1, use_graph=False)
    sa, sb = a.run(), b.run()
    torch.cuda.synchronize()
    assert sa == sb
    assert torch.equal(a.x, b.x) and torch.equal(a.mask, b.mask) and torch.equal(a.hist, b.hist)
    x1, h1 = a.x.clone(), a.hist.clone()
    assert a.run() == sa
    torch.cuda.synchronize()
    assert torch.equal(a.x, x1) and torch.equal(a.hist, h1)
    # invariants: every position revealed exactly once, within G steps
    assert not a.mask.any()
    assert bool(((a.x >= 0) & (a.x < V)).all())
    assert 1 <= sa <= G
    assert int(a.hist.sum()) == B * G
    say(f"  {sa} steps, {B * G / sa:.2f} tokens per step")
    a.close()
    b.close()
