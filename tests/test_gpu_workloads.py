"""GPU parity on the five workload recipes at their full sizes, whole.

Every candidate row of every checked step is compared with the oracle
(tokens bit-exact, conf / eps / lse within the tolerances of parity.py), and
every checked block's commit set with the oracle's selection on the oracle's
own confidences (level 3: logits in, commits out), bit for bit unless the
oracle flags the block as within 1e-6 of a decision boundary.  The oracle
runs in worker processes (oracle.parallel) on exact copies of the rows the
GPU read.

  * single block (B=1, L=32, fp32): every row, three rules;
  * generation (B=8, 256 positions in blocks of 32): seven whole
    generations, one driven by each rule, every step and every sequence;
  * sparse blocks (B=64, span 512): every candidate row, five rules;
  * bimodal generation (B=256, 1024 positions in blocks of 64): the whole
    generation driven by the profile rule; every step of the 16 flat
    sequences and four others, all five rules, and every sequence at step 0;
  * throughput stress (B=1024, L=32, 8.3 GB): every one of the 1024 blocks,
    six rules.
"""
import gc

import numpy as np
import pytest
import torch

import oracle
import workloads
from parity import (say, candidates, compare_rows, check_defaults, pool_confidence, sub_mask,
                    selection_stats, ParityTally)

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


def _host(o):
    return {k: v.cpu().numpy() for k, v in o.items()}


class _Step:
    """One step's inputs on the host plus the oracle's confidences of the
    checked sequences."""

    def __init__(self, pool, inp, bs):
        self.inp = inp
        self.mask = inp.mask.cpu().numpy()
        self.start = inp.start.cpu().numpy()
        self.end = inp.end.cpu().numpy()
        self.x = inp.x.cpu().numpy()
        self.bs = list(bs)
        self.pool = pool
        self.cells = candidates(self.mask, self.start, self.end, self.bs)
        self.tokens, self.conf, self.eps, self.lse = pool_confidence(pool, inp.logits, self.mask,
                                                                     self.start, self.end, self.bs)

    def check_rows(self, tally, go):
        worst = compare_rows(go["tokens"], go["conf"], go["eps"], go["lse"], self.tokens, self.conf,
                             self.eps, self.lse, self.cells)
        check_defaults(go["tokens"], go["conf"], go["eps"], go["lse"], self.mask, self.start,
                       self.end, self.bs)
        tally.rows_checked(len(self.cells), worst)

    def check_rules(self, tally, runs):
        """Level 3 for several rules on this step's inputs: the oracle's
        selection on the oracle's confidences, then the reveal, against each
        GPU run's commits, n_commit, x and mask.  runs: (rule, p, eta, outputs,
        mask after, x after)."""
        sel = self.pool.select_many(self.eps, self.conf, self.mask, self.start, self.end,
                                    [(r[0], r[1], r[2]) for r in runs], blocks=self.bs)
        stats = []
        for (rule, p, eta, go, g_mask, g_x), (oc, on, fl) in zip(runs, sel):
            st = selection_stats(go["commit"], go["n_commit"], oc, on, fl, self.bs)
            tally.selection(f"{rule}({p})" if eta is None else f"{rule}({p}, eta={eta})", st)
            hit = oc.astype(bool)
            ox, om = self.x.copy(), self.mask.copy()
            ox[hit] = self.tokens[hit]
            om[hit] = 0
            for b in self.bs:
                if not fl[b]:
                    assert np.array_equal(g_x[b], ox[b]) and np.array_equal(g_mask[b], om[b]), b
            stats.append(st)
        return stats


def test_single_block_b1_l32_full(gpu, oracle_pool):
    say("[single block] B=1 L=32 V=126464 fp32")
    inp = workloads.single_block_b1_l32(device="cuda")
    tally = ParityTally("single_block_b1_l32", B=1, L=32, steps=1)
    step = _Step(oracle_pool, inp, [0])
    runs = []
    for rule, p in [("profile", 1.0), ("factor", 1.0), ("threshold", 0.9)]:
        mask, x, o = _decode(gpu, inp, rule, p)
        go = _host(o)
        step.check_rows(tally, go)
        runs.append((rule, p, None, go, mask.cpu().numpy(), x.cpu().numpy()))
        assert int(go["n_commit"][0]) >= 1
    step.check_rules(tally, runs)
    # two rows hold exact ties at their maximum: lowest index wins
    rows = inp.logits[0].cpu().numpy()
    for i in range(32):
        assert go["tokens"][0, i] == int(np.argmax(rows[i]))
    tally.finish()


def test_sparse_b64_g512_full(gpu, oracle_pool):
    say("[sparse blocks] B=64 L=512 V=126464 bf16, poisoned non-candidate rows")
    inp = workloads.sparse_b64_g512(device="cuda")
    tally = ParityTally("sparse_b64_g512", B=64, L=512, steps=1)
    step = _Step(oracle_pool, inp, range(64))
    runs = []
    for rule, p in [("profile", 1.0), ("profile", 0.75), ("factor", 1.0), ("factor", 0.75),
                    ("threshold", 0.9)]:
        mask, x, o = _decode(gpu, inp, rule, p)
        go = _host(o)
        step.check_rows(tally, go)
        runs.append((rule, p, None, go, mask.cpu().numpy(), x.cpu().numpy()))
    step.check_rules(tally, runs)
    tally.finish()
    del inp
    _free()


def test_stress_b1024_l32_full(gpu, oracle_pool):
    say("[throughput stress] B=1024 L=32 V=126464 bf16 (8.3 GB), fused decode step, every block")
    inp = workloads.stress_b1024_l32(device="cuda")
    B, L, V = inp.logits.shape
    tally = ParityTally("stress_b1024_l32", B=B, L=L, steps=1)
    step = _Step(oracle_pool, inp, range(B))
    say(f"  oracle: {len(step.cells)} rows")
    res, runs = {}, []
    rules = [("profile", 1.0, None), ("factor", 1.0, None), ("profile", 0.75, None),
             ("factor", 0.75, None), ("threshold", 0.9, None), ("robust", 1.0, 0.02)]
    for rule, p, eta in rules:
        mask, x, o = _decode(gpu, inp, rule, p, eta_uniform=eta or 0.0)
        go = _host(o)
        res[(rule, p)] = go
        step.check_rows(tally, go)
        runs.append((rule, p, eta, go, mask.cpu().numpy(), x.cpu().numpy()))
        assert int(go["n_commit"].min()) >= 1 and int(go["n_commit"].max()) <= L
    for (rule, p, eta, go, _, _), st in zip(runs, step.check_rules(tally, runs)):
        say(f"  {rule}({p}): mean commits/block {float(go['n_commit'].mean()):.3f}, "
            f"flagged {st['flagged']}")
    # matched-factor dominance holds exactly in the GPU arithmetic
    for p in (1.0, 0.75):
        assert (res[("profile", p)]["n_commit"] >= res[("factor", p)]["n_commit"]).all()
    # the calibration-robust rule never commits more than the plain rule
    assert (res[("robust", 1.0)]["n_commit"] <= res[("profile", 1.0)]["n_commit"]).all()
    tally.finish()
    del inp
    _free()


def _generation(gpu, pool, recipe, drive, side, check_every, check_first, tally, max_steps,
                on_step=None):
    """A whole simulated generation driven by the GPU's `drive` rule.  At every
    step the sequences `check_every` (at step 0 also `check_first`) are
    compared with the oracle for the driving rule and every rule of `side`
    (run on the same inputs, not driving).  Returns the number of steps."""
    sim = workloads.SimulatedGeneration(recipe, device="cuda")
    steps = 0
    # the host loop's windows follow the oracle's block advance (Alg. 1 outer loop)
    w_start = np.zeros(sim.B, dtype=np.int64)
    w_end = np.full(sim.B, sim.blk, dtype=np.int64)
    while not sim.done():
        assert steps < max_steps, "generation did not finish"
        inp = sim.prepare_step()
        oracle.advance_blocks(sim.mask.cpu().numpy(), w_start, w_end, sim.G, sim.blk)
        live = w_end > w_start
        assert np.array_equal(inp.start.cpu().numpy()[live], w_start[live])
        assert np.array_equal(inp.end.cpu().numpy()[live], w_end[live])
        assert np.array_equal(inp.end.cpu().numpy()[~live], inp.start.cpu().numpy()[~live])
        bs = sorted(set(check_every) | (set(check_first) if steps == 0 else set()))
        bs = [b for b in bs if int(inp.end[b]) > int(inp.start[b])]
        step = _Step(pool, inp, bs)
        rule, p = drive
        mask, x, o = _decode(gpu, inp, rule, p)
        go = _host(o)
        step.check_rows(tally, go)
        runs = [(rule, p, None, go, mask.cpu().numpy(), x.cpu().numpy())]
        outs = {drive: go}
        for srule, sp in side:
            m2, x2, o2 = _decode(gpu, inp, srule, sp)
            g2 = _host(o2)
            for k in ("tokens", "conf", "eps", "lse"):
                assert np.array_equal(g2[k].view(np.int32), go[k].view(np.int32))
            runs.append((srule, sp, None, g2, m2.cpu().numpy(), x2.cpu().numpy()))
            outs[(srule, sp)] = g2
        step.check_rules(tally, runs)
        if on_step is not None:
            on_step(sim, inp, outs)
        sim.mask.copy_(mask)
        sim.x.copy_(x)
        steps += 1
    # every position revealed, with the token its step proposed
    assert not bool(sim.mask.any()) and bool((sim.x >= 0).all())
    return steps


GEN_RULES = [("profile", 1.0), ("factor", 1.0), ("profile", 0.5), ("factor", 0.5),
             ("profile", 2.0), ("factor", 2.0), ("threshold", 0.9)]


def test_generation_b8_g256_whole(gpu, oracle_pool):
    say("[generation] B=8 gen 256 in blocks of 32: a whole generation per rule, every step checked")
    tally = ParityTally("generation_b8_g256", B=8, G=256, blk=32)
    nfe = {}
    for drive in GEN_RULES:
        side = [("factor", drive[1])] if drive[0] == "profile" else []

        def dominance(sim, inp, outs, f=drive[1], prof=drive[0] == "profile"):
            if prof:
                assert (outs[("profile", f)]["n_commit"] >= outs[("factor", f)]["n_commit"]).all()

        nfe[f"{drive[0]}({drive[1]})"] = _generation(gpu, oracle_pool, workloads.GENERATION, drive,
                                                     side, range(8), (), tally, max_steps=256,
                                                     on_step=dominance)
        say(f"  {drive[0]}({drive[1]}): {nfe[f'{drive[0]}({drive[1]})']} steps")
    tally.note(steps_per_generation=nfe)
    tally.finish()
    _free()


def test_bimodal_b256_g1024_whole(gpu, oracle_pool):
    say("[bimodal generation] B=256 gen 1024 in blocks of 64: whole generation, flat + 4 others every "
        "step, all 256 at step 0")
    probe = workloads.SimulatedGeneration(workloads.BIMODAL_GENERATION, device="cpu", V=8)
    flat = [b for b in range(256) if probe.flat[b]]
    others = [b for b in (0, 1, 100, 255) if b not in flat]
    while len(others) < 4:
        others.append(next(b for b in range(2, 256) if b not in flat and b not in others))
    check = sorted(set(flat) | set(others))
    tally = ParityTally("bimodal_b256_g1024", B=256, G=1024, blk=64, flat_sequences=flat,
                        every_step_sequences=check)
    side = [("factor", 1.0), ("profile", 0.75), ("factor", 0.75), ("threshold", 0.9)]

    def flat_checks(sim, inp, outs):
        for f in (0.75, 1.0):
            npf = outs[("profile", f)]["n_commit"]
            nfa = outs[("factor", f)]["n_commit"]
            assert (npf >= nfa).all()
            # flat blocks: profile == factor, bit for bit on the GPU
            assert (npf[flat] == nfa[flat]).all()
            for b in flat:
                assert np.array_equal(outs[("profile", f)]["commit"][b], outs[("factor", f)]["commit"][b])
        # rows of a flat block are identical, so their confidences are identical bits
        eps = outs[("profile", 1.0)]["eps"]
        m = inp.mask.cpu().numpy()
        for b in flat:
            s, e = int(inp.start[b]), int(inp.end[b])
            v = eps[b, s:e][m[b, s:e] != 0].view(np.int32)
            assert (v == v[:1]).all()

    steps = _generation(gpu, oracle_pool, workloads.BIMODAL_GENERATION, ("profile", 1.0), side,
                        check, range(256), tally, max_steps=1024, on_step=flat_checks)
    tally.note(steps=steps)
    tally.finish()
    _free()
