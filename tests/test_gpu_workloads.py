"""GPU parity on the five workload recipes at their full sizes.

The single-block and sparse-block recipes are checked on every candidate
row; the throughput stress (8.3 GB of logits) on a seeded sample of blocks
plus properties that hold at any size; the simulated generations run in
lockstep with the oracle for their first steps.
"""
import gc

import numpy as np
import pytest
import torch

import oracle
import workloads
from parity import (say, row_source, candidates, compare_rows, gpu_confidence,
                    oracle_confidence_subset, check_defaults, compare_selection)

pytestmark = pytest.mark.gpu


def _free():
    gc.collect()
    torch.cuda.empty_cache()


def _decode(gpu, inp, rule, p, mask=None, x=None, eta=None, eta_uniform=0.0):
    B, L, V = inp.logits.shape
    mask = inp.mask.clone() if mask is None else mask
    x = inp.x.clone() if x is None else x
    o = dict(tokens=torch.empty((B, L), dtype=torch.int32, device="cuda"),
             conf=torch.empty((B, L), device="cuda"), eps=torch.empty((B, L), device="cuda"),
             lse=torch.empty((B, L), device="cuda"),
             commit=torch.empty((B, L), dtype=torch.uint8, device="cuda"),
             n_commit=torch.empty((B,), dtype=torch.int32, device="cuda"))
    gpu.fdllm_decode_step(inp.logits, mask, inp.start, inp.end, x, rule, p, eta=eta,
                          eta_uniform=eta_uniform, **o)
    torch.cuda.synchronize()
    return mask, x, o


def _oracle_step(inp, bs, rule, p):
    B, L, V = inp.logits.shape
    m = inp.mask.cpu().numpy().copy()
    keep = np.zeros(B, dtype=bool)
    keep[list(bs)] = True
    m[~keep] = 0
    return oracle.decode_step(row_source(inp.logits), B, L, m, inp.start.cpu().numpy(),
                              inp.end.cpu().numpy(), inp.x.cpu().numpy(), rule, p)


def _check_step(inp, o, bs, rule, p):
    r = _oracle_step(inp, bs, rule, p)
    nf, nfm = compare_selection(o["commit"].cpu().numpy(), o["n_commit"].cpu().numpy(),
                                r.commit, r.n_commit, r.flagged, bs)
    cells = candidates(inp.mask.cpu().numpy(), inp.start.cpu().numpy(), inp.end.cpu().numpy(), bs)
    g = [o[k].cpu().numpy() for k in ("tokens", "conf", "eps", "lse")]
    worst = compare_rows(*g, r.tokens, r.conf, r.eps, r.lse, cells)
    return nf, nfm, worst, r


def test_single_block_b1_l32_full(gpu):
    say("[single block] B=1 L=32 V=126464 fp32")
    inp = workloads.single_block_b1_l32(device="cuda")
    for rule, p in [("profile", 1.0), ("factor", 1.0), ("threshold", 0.9)]:
        mask, x, o = _decode(gpu, inp, rule, p)
        nf, nfm, worst, r = _check_step(inp, o, [0], rule, p)
        assert int(o["n_commit"][0]) >= 1
        say(f"  {rule}({p}): n*={int(o['n_commit'][0])} flagged={nf} worst={worst}")
    # two rows hold exact ties at their maximum: lowest index wins
    tok = o["tokens"][0].cpu().numpy()
    rows = inp.logits[0].cpu().numpy()
    for i in range(32):
        assert tok[i] == int(np.argmax(rows[i]))


def test_sparse_b64_g512_full(gpu):
    say("[sparse blocks] B=64 L=512 V=126464 bf16, poisoned non-candidate rows")
    inp = workloads.sparse_b64_g512(device="cuda")
    g = gpu_confidence(gpu, inp)
    assert all(bool(torch.isfinite(t.float()).all()) for t in g[1:])
    for rule, p in [("profile", 1.0), ("profile", 0.75), ("factor", 1.0), ("factor", 0.75),
                    ("threshold", 0.9)]:
        mask, x, o = _decode(gpu, inp, rule, p)
        for name, t in zip(("tokens", "conf", "eps", "lse"), g):
            assert torch.equal(o[name].view(torch.int32), t.view(torch.int32))
        if rule == "profile" and p == 1.0:
            nf, nfm, worst, r = _check_step(inp, o, range(64), rule, p)
            say(f"  {rule}({p}): rows={int(inp.mask.sum())} flagged={nf} worst={worst}")
        else:
            # selection on the oracle's own confidences, reusing the last oracle pass
            oc, on, fl, _ = oracle.select(r.eps, r.conf, inp.mask.cpu().numpy(), inp.start.cpu().numpy(),
                                          inp.end.cpu().numpy(), rule, p)
            nf, nfm = compare_selection(o["commit"].cpu().numpy(), o["n_commit"].cpu().numpy(),
                                        oc, on, fl, range(64))
            say(f"  {rule}({p}): commits={int(o['n_commit'].sum())} flagged={nf}")
    del inp, g
    _free()


def test_stress_b1024_l32_sampled(gpu):
    say("[throughput stress] B=1024 L=32 V=126464 bf16 (8.3 GB), fused decode step")
    inp = workloads.stress_b1024_l32(device="cuda")
    B, L, V = inp.logits.shape
    rng = np.random.default_rng(2026)
    sample = sorted(rng.choice(B, 24, replace=False).tolist())
    conf_ref = gpu_confidence(gpu, inp)
    res = {}
    for rule, p in [("profile", 1.0), ("factor", 1.0), ("profile", 0.75), ("factor", 0.75),
                    ("threshold", 0.9)]:
        mask, x, o = _decode(gpu, inp, rule, p)
        res[(rule, p)] = o
        n = o["n_commit"]
        assert int(n.min()) >= 1 and int(n.max()) <= L
        assert torch.equal(o["commit"].sum(1, dtype=torch.int32), n)
        assert not (o["commit"].bool() & mask.bool()).any()             # committed -> unmasked
        assert torch.equal(torch.where(o["commit"].bool(), o["tokens"], x), x)
        for name, t in zip(("tokens", "conf", "eps", "lse"), conf_ref):
            assert torch.equal(o[name].view(torch.int32), t.view(torch.int32))
        c2 = torch.empty_like(o["commit"]); n2 = torch.empty_like(n)
        gpu.select(rule, conf_ref[1], conf_ref[2], inp.mask, inp.start, inp.end, p, c2, n2)
        torch.cuda.synchronize()
        assert torch.equal(c2, o["commit"]) and torch.equal(n2, n)
        say(f"  {rule}({p}): mean commits/block {float(n.float().mean()):.3f}")
    # matched-factor dominance holds exactly in the GPU arithmetic
    for p in (1.0, 0.75):
        assert (res[("profile", p)]["n_commit"] >= res[("factor", p)]["n_commit"]).all()
    # the calibration-robust rule never commits more than the plain rule
    mask_r, x_r, o_r = _decode(gpu, inp, "robust", 1.0, eta_uniform=0.02)
    assert (o_r["n_commit"] <= res[("profile", 1.0)]["n_commit"]).all()
    assert (o_r["n_commit"] >= 1).all()
    say(f"  robust(1.0, eta=0.02): mean commits/block {float(o_r['n_commit'].float().mean()):.3f}")
    nf, nfm, worst, r = _check_step(inp, res[("profile", 1.0)], sample, "profile", 1.0)
    say(f"  oracle on {len(sample)} blocks: flagged={nf} worst={worst}")
    res[("robust", 1.0)] = o_r
    for rule, p in [("factor", 1.0), ("threshold", 0.9), ("profile", 0.75), ("robust", 1.0)]:
        oc, on, fl, _ = oracle.select(r.eps, r.conf, np.where(np.isin(np.arange(B), sample)[:, None],
                                      inp.mask.cpu().numpy(), 0), inp.start.cpu().numpy(),
                                      inp.end.cpu().numpy(), rule, p,
                                      eta=0.02 if rule == "robust" else None)
        o = res[(rule, p)]
        nf, nfm = compare_selection(o["commit"].cpu().numpy(), o["n_commit"].cpu().numpy(), oc, on, fl, sample)
        say(f"  {rule}({p}) on sample: flagged={nf}")
    del inp, conf_ref, res
    _free()


def _simulate(gpu, recipe, rules, steps, check_bs, B=None):
    sim = workloads.SimulatedGeneration(recipe, device="cuda", B=B)
    flagged_total = 0
    for s in range(steps):
        if sim.done():
            break
        inp = sim.prepare_step()
        say(f"  step {s}: active rows {int(sum((inp.end - inp.start).tolist()))}")
        outs = {}
        for rule, p in rules:
            mask, x, o = _decode(gpu, inp, rule, p)
            outs[(rule, p)] = (mask, x, o)
        # oracle in lockstep on the checked sequences, first rule drives the trajectory
        for k, (rule, p) in enumerate(rules):
            mask, x, o = outs[(rule, p)]
            if k == 0:
                nf, nfm, worst, r = _check_step(inp, o, check_bs, rule, p)
            else:
                oc, on, fl, _ = oracle.select(r.eps, r.conf, _sub_mask(inp, check_bs),
                                              inp.start.cpu().numpy(), inp.end.cpu().numpy(), rule, p)
                nf, nfm = compare_selection(o["commit"].cpu().numpy(), o["n_commit"].cpu().numpy(),
                                            oc, on, fl, check_bs)
            flagged_total += nf
        yield sim, inp, outs
        mask, x, _ = outs[rules[0]]
        sim.mask.copy_(mask)
        sim.x.copy_(x)
    say(f"  flagged blocks in total: {flagged_total}")


def _sub_mask(inp, bs):
    m = inp.mask.cpu().numpy().copy()
    keep = np.zeros(m.shape[0], dtype=bool)
    keep[list(bs)] = True
    m[~keep] = 0
    return m


def test_generation_b8_g256_simulation(gpu):
    say("[generation] B=8 gen 256 in blocks of 32, lockstep with the oracle")
    rules = [("profile", 1.0), ("factor", 1.0), ("profile", 0.5), ("factor", 0.5),
             ("profile", 2.0), ("factor", 2.0), ("threshold", 0.9)]
    for sim, inp, outs in _simulate(gpu, workloads.GENERATION, rules, steps=6, check_bs=range(8)):
        for f in (0.5, 1.0, 2.0):
            assert (outs[("profile", f)][2]["n_commit"] >= outs[("factor", f)][2]["n_commit"]).all()
    _free()


def test_bimodal_b256_g1024_simulation(gpu):
    say("[bimodal generation] B=256 gen 1024 in blocks of 64, lockstep on a subset incl. all flat sequences")
    sim_probe = workloads.SimulatedGeneration(workloads.BIMODAL_GENERATION, device="cpu", V=8)
    flat = [b for b in range(256) if sim_probe.flat[b]]
    check = sorted(set(flat) | {0, 1, 100, 255})
    rules = [("profile", 1.0), ("factor", 1.0), ("profile", 0.75), ("factor", 0.75), ("threshold", 0.9)]
    for sim, inp, outs in _simulate(gpu, workloads.BIMODAL_GENERATION, rules, steps=2, check_bs=check):
        for f in (0.75, 1.0):
            npf = outs[("profile", f)][2]["n_commit"].cpu().numpy()
            nfa = outs[("factor", f)][2]["n_commit"].cpu().numpy()
            assert (npf >= nfa).all()
            # flat blocks: profile == factor, bit-exactly on the GPU
            assert (npf[flat] == nfa[flat]).all()
            for b in flat:
                assert torch.equal(outs[("profile", f)][2]["commit"][b], outs[("factor", f)][2]["commit"][b])
        # rows of a flat block are identical, so their confidences are identical bits
        eps = outs[rules[0]][2]["eps"]
        for b in flat:
            s, e = int(inp.start[b]), int(inp.end[b])
            m = inp.mask[b, s:e].bool()
            v = eps[b, s:e][m].view(torch.int32)
            assert (v == v[0]).all()
    _free()
