#!/usr/bin/env python3
"""Throughput of one Fast-dLLM++ decoding step on one MI355X.

Workload (throughput stress recipe): B=1024 sequences, an active block of
L=32 all-masked positions each, V=126464 bf16 logits per position (8.29 GB
per step, Gumbel(0,1) background with 10% planted near-ties), resident in HBM.
A step is the whole hot path in one fused launch: the vocabulary pass
(greedy token, confidence, eps, lse for all 32768 positions), the Frechet
profile selection (f = 1.0) of every block and the reveal.  Each timed step
works on its own copy of the step's input mask/x, staged in HBM before the
timed region, so every step does the same work.  Ahead of each timed run's untimed warm-up steps, a
settle phase of about 100 ms of back-to-back read-only streams brings the
GPU's clocks to their loaded steady state, so the timed steps see what a
continuously decoding server sees rather than the ramp after an idle pause.

Prints one JSON line.  `value` is masked positions per second over the whole
timed region; `roofline` relates the fused kernel's algorithmic bytes to its
average launch time measured with HIP events on the launch stream, and to a
read-only stream of the same logits buffer (libfdllm_bench.so).
`parity` compares the outputs of the timed step with the CPU oracle run on
exact host copies of every one of its logits rows, and `cpu_baseline` times
that oracle run (all host cores, one worker process per core) and a one-core
run on a seeded sample of its blocks.  `--per-workload` adds the other workload recipes (one sequence fp32;
eight-sequence and 256-sequence simulated generations; 64 sequences in a
512-position span), cold and cache-hot, the device-resident generation loop
and the LM head fused with the pass, and can write them as a markdown table.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import math
import multiprocessing as mp
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "masked positions selected/sec + logits-read HBM GB/s (% of peak), 1 GPU"
HBM_PEAK_GBPS = 8000.0
IO_BYTES_PER_POSITION = 18   # mask read, commit, tokens, conf, eps, lse (1+1+4+4+4+4)
# sources of the vocabulary pass kernels (the fused decode step and its helpers)
SRCS = [os.path.join(ROOT, "paper_2606_02955_amd", "csrc", f) for f in ("fdllm.hip", "pass_common.h")]
TRAFFIC = os.path.join(ROOT, "profiles", "traffic_fused_decode_b1024_l32.json")
MAX_HOST_WORKERS = 16        # host CPU share of one GPU


def log(msg: str):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def _code_only(text: str) -> str:
    """C++ source without comments and with whitespace collapsed, so that an
    edit to comments or layout does not count as a change of the kernel."""
    import re
    out, i, n = [], 0, len(text)
    while i < n:
        c = text[i]
        if c in "\"'":                      # string or character literal, kept whole
            j = i + 1
            while j < n and text[j] != c:
                j += 2 if text[j] == "\\" else 1
            out.append(text[i:j + 1])
            i = j + 1
        elif text.startswith("//", i):
            j = text.find("\n", i)
            i = n if j < 0 else j
        elif text.startswith("/*", i):
            j = text.find("*/", i + 2)
            i = n if j < 0 else j + 2
            out.append(" ")
        else:
            out.append(c)
            i += 1
    return re.sub(r"\s+", " ", "".join(out)).strip()


def source_digest() -> str:
    """Hash of the k_fused sources (code only: comments and layout do not
    count) and the device compiler flags they build with."""
    from paper_2606_02955_amd import build as _build
    h = hashlib.sha256()
    for f in SRCS:
        h.update(_code_only(open(f, encoding="utf-8").read()).encode())
    h.update(" ".join(_build.HIPCC_FLAGS).encode())
    return h.hexdigest()[:16]


def measured_traffic():
    """HBM bytes per launch from committed rocprofv3 counter runs, if current."""
    try:
        t = json.load(open(TRAFFIC))
    except (OSError, ValueError):
        return None
    if t.get("source_sha256_16") != source_digest():
        return None
    return t.get("hbm_bytes_per_launch")


def _counter_means(csv_path: str, counter: str):
    """Mean value per dispatch of `counter` for the calibration kernel (the
    elementwise add of the uint8 copy reference) and the fused decode step,
    from a rocprofv3 counter_collection csv."""
    import csv
    sums = {"copy": [0.0, 0], "fused": [0.0, 0]}
    with open(csv_path) as fh:
        for row in csv.DictReader(fh):
            if row.get("Counter_Name") != counter:
                continue
            name = row.get("Kernel_Name", "")
            # the calibration is torch.add(uint8 tensor, 1): its functor names the dtype
            key = "fused" if "k_fused<" in name else "copy" if "add<unsigned char>" in name else None
            if key:
                sums[key][0] += float(row["Counter_Value"])
                sums[key][1] += 1
    if not sums["copy"][1] or not sums["fused"][1]:
        raise SystemExit(f"{csv_path}: no {counter} rows for the elementwise add and k_fused")
    return {k: v[0] / v[1] for k, v in sums.items()}, {k: v[1] for k, v in sums.items()}


def traffic_from(fetch_csv: str, write_csv: str, out_path: str, copy_mb: int):
    """HBM bytes per fused-step launch from the FETCH_SIZE and WRITE_SIZE runs
    (KiB per dispatch), each scaled by what the counter reads for the
    elementwise add of copy_mb MiB (which reads and writes exactly that)."""
    n = copy_mb << 20
    f, fc = _counter_means(fetch_csv, "FETCH_SIZE")
    w, wc = _counter_means(write_csv, "WRITE_SIZE")
    fetch_scale = n / (f["copy"] * 1024.0)
    write_scale = n / (w["copy"] * 1024.0)
    t = {"kernel": "k_fused (stress_b1024_l32 decode step)",
         "workload": "throughput stress B=1024 L=32 V=126464 bf16",
         "source_sha256_16": source_digest(),
         "fetch_kib_per_dispatch": f["fused"], "write_kib_per_dispatch": w["fused"],
         "dispatches": {"fetch": fc, "write": wc},
         "fetch_scale": fetch_scale, "write_scale": write_scale,
         "hbm_bytes_per_launch": (f["fused"] * fetch_scale + w["fused"] * write_scale) * 1024.0}
    with open(out_path, "w") as fh:
        json.dump(t, fh, indent=1)
        fh.write("\n")
    print(json.dumps(t))


def cpu_model() -> str:
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def under_profiler() -> bool:
    return "rocprof" in os.environ.get("LD_PRELOAD", "") or any(
        k.startswith("ROCPROF") for k in os.environ)


# ---------------------------------------------------------------------------
# CPU oracle: parity of the timed step and the CPU baseline.  The worker
# processes (oracle.parallel) are spawned before this process touches the GPU;
# after the GPU timing they run the oracle on exact host copies of the timed
# step's logits rows and the outputs of its last run are compared with it.
# ---------------------------------------------------------------------------
def oracle_parity(pool, inp, saved, rule: str, param: float):
    """Oracle on every candidate row of the timed step (all host cores), and
    the comparison with the saved GPU outputs of that step."""
    import numpy as np
    import torch
    from oracle.parallel import scatter_confidence
    B, L, V = inp.logits.shape
    mask = inp.mask0.cpu().numpy()
    start, end = inp.start.cpu().numpy(), inp.end.cpu().numpy()
    cells = [(b, i) for b in range(B) for i in range(int(start[b]), int(end[b])) if mask[b, i]]
    flat = inp.logits.view(B * L, V)
    idx = torch.tensor([b * L + i for b, i in cells], dtype=torch.long, device=inp.logits.device)

    def fill(first, cnt, out):
        rows = flat.index_select(0, idx[first:first + cnt])
        torch.from_numpy(out).copy_(rows.view(torch.int16))

    s0 = pool.seconds
    res = pool.rows_confidence(fill, len(cells), V, "bf16")
    tok, conf, eps, lse = scatter_confidence(B, L, cells, res)
    commit, n_commit, flagged = pool.select(eps, conf, mask, start, end, rule, param)
    secs = pool.seconds - s0
    g = {k: v.cpu().numpy() for k, v in saved.items()}
    ci = tuple(np.array(c) for c in zip(*cells))
    rel = lambda a, b, floor: np.abs(a[ci].astype(np.float64) - b[ci]) / np.maximum(np.abs(b[ci]), floor)
    e_conf, e_lse = rel(g["conf"], conf, 1e-30), rel(g["lse"], lse, 1.0)
    d_eps = np.abs(g["eps"][ci].astype(np.float64) - eps[ci])
    e_eps = np.where(d_eps > 2.0 ** -48, d_eps / np.maximum(np.abs(eps[ci]), 1e-30), 0.0)
    same = np.array([np.array_equal(g["commit"][b], commit[b]) and int(g["n_commit"][b]) == int(n_commit[b])
                     for b in range(B)])
    hit = commit.astype(bool)
    ox, om = inp.x0.cpu().numpy().copy(), mask.copy()
    ox[hit] = tok[hit]
    om[hit] = 0
    same_seq = np.array([np.array_equal(g["x"][b], ox[b]) and np.array_equal(g["mask"][b], om[b])
                         for b in range(B)])
    parity = {"rule": f"{rule}({param})", "checked_blocks": B, "checked_positions": len(cells),
              "token_mismatches": int((g["tokens"][ci] != tok[ci]).sum()),
              "value_mismatches": int(((e_conf > 1e-5) | (e_eps > 1e-5) | (e_lse > 1e-5)).sum()),
              "mismatches": int((~same & ~flagged).sum() + (~same_seq & ~flagged).sum()),
              "flagged": int(flagged.sum()), "flagged_matching": int((same & flagged).sum()),
              "max_rel_err": {"conf": float(e_conf.max()), "eps": float(e_eps.max()),
                              "lse": float(e_lse.max())},
              "oracle": "oracle.position_confidence (float64, fsum) + oracle.select (exact rationals) "
                        "on device-to-host copies of the timed step's rows"}
    base = {"value": len(cells) / secs, "unit": "masked positions/s", "cores": pool.workers,
            "kind": "oracle",
            "sample": f"the whole timed step: {B} blocks, {len(cells)} positions "
                      f"({len(cells) * V * 2 / 1e9:.2f} GB of bf16 logits copied device-to-host), "
                      f"{rule} f={param}; {pool.workers} processes, NumPy float64 + exact rational "
                      f"selection; {secs:.1f} s inside the oracle calls (staging copies excluded)",
            "seconds": secs, "logits_GBps": len(cells) * V * 2 / secs / 1e9}
    return parity, base


def cpu_baseline_single(inp, saved, n_blocks: int, rule: str, param: float):
    """The oracle in this process (one core) on a seeded sample of blocks of the
    timed step, checked against the saved GPU outputs of those blocks."""
    import numpy as np
    import torch
    import oracle
    B, L, V = inp.logits.shape
    rng = np.random.default_rng(7)
    blocks = sorted(rng.choice(B, n_blocks, replace=False).tolist())
    rows = inp.logits[blocks].to("cpu")                      # [n, L, V] bf16, outside the timing
    mask = inp.mask0[blocks].cpu().numpy()
    start, end = inp.start[blocks].cpu().numpy(), inp.end[blocks].cpu().numpy()
    x = inp.x0[blocks].cpu().numpy()
    get = lambda b, i: rows[b, i].to(dtype=torch.float64).numpy()
    t0 = time.perf_counter()
    r = oracle.decode_step(get, n_blocks, L, mask, start, end, x, rule, param)
    dt = time.perf_counter() - t0
    n_pos = int(mask.sum())
    gc_, gn = saved["commit"][blocks].cpu().numpy(), saved["n_commit"][blocks].cpu().numpy()
    same = np.array([np.array_equal(gc_[k], r.commit[k]) and int(gn[k]) == int(r.n_commit[k])
                     for k in range(n_blocks)])
    return {"value": n_pos / dt, "unit": "masked positions/s", "cores": 1, "kind": "oracle",
            "sample": f"{n_blocks} of {B} blocks ({n_pos} positions, {n_pos * V * 2 / 1e9:.2f} GB of "
                      f"bf16 logits) of the timed step, {rule} f={param}; one process, NumPy float64 "
                      f"+ exact rational selection; {dt:.1f} s",
            "seconds": dt, "logits_GBps": n_pos * V * 2 / dt / 1e9, "commits": int(r.n_commit.sum()),
            "blocks_matching_gpu": int(same.sum()), "blocks_flagged": int(r.flagged.sum())}


# ---------------------------------------------------------------------------
# per-workload report
# ---------------------------------------------------------------------------
def _candidates(inp) -> int:
    import torch
    L = inp.logits.shape[1]
    pos = torch.arange(L, device=inp.mask.device).view(1, L)
    inwin = (pos >= inp.start.view(-1, 1)) & (pos < inp.end.view(-1, 1))
    return int((inwin & inp.mask.bool()).sum())


def _time_steps(fd, torch, inp, selector, p, reps, scratch=None, settle=None):
    """Average decode-step kernel time (HIP events) over reps, input state restored;
    `settle` (if given) brings the clocks to their loaded state first."""
    B = inp.logits.shape[0]
    mask0, x0 = inp.mask.clone(), inp.x.clone()
    mask, x = mask0.clone(), x0.clone()
    nc = torch.empty((B,), dtype=torch.int32, device=inp.logits.device)
    ws = fd.fdllm_decode_step(inp.logits, mask, inp.start, inp.end, x, selector, p, n_commit=nc)
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in range(reps)]
    if settle is not None:
        settle()
    for _ in range(2):                       # warm-up on this workload's own buffers
        mask.copy_(mask0)
        x.copy_(x0)
        fd.fdllm_decode_step(inp.logits, mask, inp.start, inp.end, x, selector, p, n_commit=nc,
                             workspace=ws)
    for k in range(reps):
        mask.copy_(mask0)
        x.copy_(x0)
        if scratch is not None:
            scratch.fill_(k & 0x7F)          # evicts the logits from L2 and the Infinity Cache
        evs[k][0].record()
        fd.fdllm_decode_step(inp.logits, mask, inp.start, inp.end, x, selector, p, n_commit=nc,
                             workspace=ws)
        evs[k][1].record()
    torch.cuda.synchronize()
    t = sorted(a.elapsed_time(b) * 1e-3 for a, b in evs)
    return sum(t) / len(t), t[len(t) // 2], float(nc.clamp(min=0).float().mean())


def _row(name, shape, sel, positions, bytes_, t_cold, t_hot, stream_gbps, extra=None):
    d = {"workload": name, "shape": shape, "selector": sel, "positions_per_step": positions,
         "logits_bytes_per_step": bytes_, "kernel_ms_cold": 1e3 * t_cold,
         "kernel_ms_hot": None if t_hot is None else 1e3 * t_hot,
         "positions_per_s": positions / t_cold, "logits_GBps": bytes_ / t_cold / 1e9,
         "frac_of_peak": bytes_ / t_cold / 1e9 / HBM_PEAK_GBPS,
         "frac_of_stream": bytes_ / t_cold / 1e9 / stream_gbps if stream_gbps else None}
    if extra:
        d.update(extra)
    return d


def per_workload_report(fd, torch, workloads, dev, stream_gbps, reps, settle=None):
    import gc
    rows = []
    scratch = torch.empty(512 << 20, dtype=torch.uint8, device=dev)
    sels = {k: [(s, p) for s in v["selectors"] for p in v["params"][s]]
            for k, v in workloads.RECIPES.items()}
    name = workloads.RECIPE_NAMES

    def static(k, inp, label, cold_needed=True):
        B, L, V = inp.logits.shape
        pos = _candidates(inp)
        nbytes = pos * V * inp.logits.element_size()
        # one untimed pass over the workload's fresh buffers first, so that no
        # selector's figure carries their first use
        _time_steps(fd, torch, inp, sels[k][0][0], sels[k][0][1], 2, None, settle)
        for sel, p in sels[k]:
            tc, _, commits = _time_steps(fd, torch, inp, sel, p, reps, scratch if cold_needed else None,
                                         settle)
            th = _time_steps(fd, torch, inp, sel, p, reps, settle=settle)[0] if cold_needed else None
            extra = {"mean_commits_per_block": commits}
            if not cold_needed:
                extra["note"] = "cold by size: the step reads far more than the caches hold"
            rows.append(_row(name[k], label, f"{sel}({p})", pos, nbytes, tc, th, stream_gbps, extra))
            log(f"{name[k]} {sel}({p}): {1e3 * tc:.3f} ms cold, {nbytes / tc / 1e9:.0f} GB/s")

    log("per-workload: single block")
    inp = workloads.single_block_b1_l32(device=dev)
    static(workloads.SINGLE_BLOCK, inp, "B=1 L=32 V=126464 fp32")
    del inp
    log("per-workload: sparse blocks")
    inp = workloads.sparse_b64_g512(device=dev)
    static(workloads.SPARSE_BLOCKS, inp, "B=64 span 512, m_b~U{1..32}, V=126464 bf16")
    del inp
    gc.collect()
    torch.cuda.empty_cache()
    # whole simulated generations (B=8 of 256), one per selector
    for sel, p in sels[workloads.GENERATION]:
        gen = workloads.SimulatedGeneration(workloads.GENERATION, device=dev)
        nc = torch.empty((gen.B,), dtype=torch.int32, device=dev)
        steps, commits, positions, ktime, ws = 0, 0, 0, 0.0, None
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        while not gen.done() and steps < 4096:
            inp = gen.prepare_step()
            positions += _candidates(inp)
            e0.record()
            ws = fd.fdllm_decode_step(inp.logits, inp.mask, inp.start, inp.end, inp.x, sel, p,
                                      n_commit=nc, workspace=ws)
            e1.record()
            torch.cuda.synchronize()
            ktime += e0.elapsed_time(e1) * 1e-3
            commits += int(nc.clamp(min=0).sum())
            steps += 1
        nbytes = positions * gen.V * 2
        rows.append(_row(workloads.RECIPE_NAMES[workloads.GENERATION],
                         "B=8 gen 256 in blocks of 32, V=126464 bf16 (whole generation)",
                         f"{sel}({p})", positions / steps, nbytes / steps, ktime / steps, None,
                         stream_gbps, {"steps": steps, "commits_per_step": commits / steps,
                                       "note": "hot: each step's rows were just written"}))
        log(f"generation_b8_g256 {sel}({p}): {steps} steps, {commits / steps:.2f} commits/step")
        del gen
    gc.collect()
    torch.cuda.empty_cache()
    # the same eight-sequence generation shape, run by the device-resident loop
    # with the counter-based logits producer in place of the model call
    loop_modes = [("graph, 8 steps per launch", 8, True),
                  ("direct launches, 8 steps per host check", 8, False),
                  ("direct launches, host check every step", 1, False)]
    for V_loop, (mode, chunk, graph) in [(v, m) for v in (workloads.V_LLADA, 4096) for m in loop_modes]:
        gen = fd.Generation(8, 256, 32, V_loop, 2026, "profile", 1.0, chunk=chunk,
                            use_graph=graph, record_history=False, device=dev)
        gen.run()                                    # warm-up
        walls = []
        for _ in range(5):
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            steps = gen.run()
            walls.append(time.perf_counter() - t0)
        w = sorted(walls)[len(walls) // 2]
        rows.append({"workload": "device-loop", "shape": f"B=8 gen 256 in blocks of 32, V={V_loop} bf16",
                     "selector": "profile(1.0)", "mode": mode, "steps": steps,
                     "ms_per_generation": 1e3 * w, "us_per_step": 1e6 * w / steps,
                     "tokens_per_s": 8 * 256 / w})
        log(f"device loop ({mode}): {steps} steps, {1e3 * w:.2f} ms per generation")
        gen.close()
        del gen
    # LM head fused with the vocabulary pass (hidden states in, no logits in HBM)
    # against the unfused pair: a hipBLASLt GEMM writing bf16 logits, then the pass
    d_model = 4096
    gw = torch.Generator(device=dev).manual_seed(2606)
    weight = (torch.randn((workloads.V_LLADA, d_model), generator=gw, device=dev) / 64).to(torch.bfloat16)
    for B_lm in (1, 2, 8, 128):
        L_lm = 32
        hid = torch.randn((B_lm, L_lm, d_model), generator=gw, device=dev).to(torch.bfloat16)
        mk = torch.ones((B_lm, L_lm), dtype=torch.uint8, device=dev)
        st_ = torch.zeros(B_lm, dtype=torch.int32, device=dev)
        en_ = torch.full((B_lm,), L_lm, dtype=torch.int32, device=dev)
        tok = torch.empty((B_lm, L_lm), dtype=torch.int32, device=dev)
        cf = torch.empty((B_lm, L_lm), device=dev)
        ws = fd.fdllm_lmhead_confidence(hid, weight, mk, st_, en_, tok, cf)
        lg = torch.empty((B_lm * L_lm, workloads.V_LLADA), dtype=torch.bfloat16, device=dev)
        torch.matmul(hid.view(-1, d_model), weight.t(), out=lg)
        torch.cuda.synchronize()
        # each event pair brackets `burst` back-to-back calls, so the queue
        # stays full and host launch gaps stay out of the per-call times
        burst = 4
        tf, tg, tp = [], [], []
        if settle is not None:
            settle()
        for _ in range(max(3, reps // 2)):
            e0, e1, e2, e3 = (torch.cuda.Event(enable_timing=True) for _ in range(4))
            e0.record()
            for _ in range(burst):
                fd.fdllm_lmhead_confidence(hid, weight, mk, st_, en_, tok, cf, workspace=ws)
            e1.record()
            for _ in range(burst):
                torch.matmul(hid.view(-1, d_model), weight.t(), out=lg)
            e2.record()
            for _ in range(burst):
                fd.fdllm_confidence(lg.view(B_lm, L_lm, -1), mk, st_, en_, tok, cf)
            e3.record()
            torch.cuda.synchronize()
            tf.append(e0.elapsed_time(e1) * 1e-3 / burst)
            tg.append(e1.elapsed_time(e2) * 1e-3 / burst)
            tp.append(e2.elapsed_time(e3) * 1e-3 / burst)
        med = lambda v: sorted(v)[len(v) // 2]
        flops = 2.0 * B_lm * L_lm * d_model * workloads.V_LLADA
        rows.append({"workload": "lmhead", "shape": f"{B_lm * L_lm} positions, d={d_model}, V={workloads.V_LLADA}",
                     "fused_ms": 1e3 * med(tf), "fused_TFLOPs": flops / med(tf) / 1e12,
                     "frac_of_bf16_peak": flops / med(tf) / 2.5e15,
                     "W_TBps": 2.0 * workloads.V_LLADA * d_model / med(tf) / 1e12,
                     "unfused_gemm_ms": 1e3 * med(tg), "unfused_pass_ms": 1e3 * med(tp),
                     "unfused_TFLOPs": flops / (med(tg) + med(tp)) / 1e12,
                     "logits_bytes_avoided": B_lm * L_lm * workloads.V_LLADA * 2})
        log(f"lmhead {B_lm * L_lm} positions: fused {1e3 * med(tf):.3f} ms, "
            f"hipBLASLt {1e3 * med(tg):.3f} ms + pass {1e3 * med(tp):.3f} ms")
        del hid, lg, ws
    del weight
    gc.collect()
    torch.cuda.empty_cache()
    log("per-workload: bimodal generation (its first step)")
    gen = workloads.SimulatedGeneration(workloads.BIMODAL_GENERATION, device=dev)
    inp = gen.prepare_step()
    static(workloads.BIMODAL_GENERATION, inp, "B=256 span 1024 (66 GB allocated), block 64, V=126464 bf16", cold_needed=False)
    del inp, gen
    gc.collect()
    torch.cuda.empty_cache()
    del scratch
    return rows


def per_workload_markdown(rows, stress, stream_gbps, cmd) -> str:
    out = ["# Decode-step throughput per workload recipe (one MI355X)", "",
           "Command (from the repository root):", "", f"    {cmd}", "",
           f"Read-only stream reference (`fdllm_stream_read` over the 8.29 GB logits buffer): "
           f"{stream_gbps:.0f} GB/s.  Kernel times are HIP-event averages of `fdllm_decode_step`; "
           "`cold` overwrites a 512 MB buffer before every step (evicting L2 and the Infinity "
           "Cache), `hot` does not (with no long kernel queued ahead, a hot step's event window also holds "
           "the host's launch gaps between its kernels).  The per-step traffic of the B=8 generation is "
           "8x32 rows, so its steps are launch-bound.", "",
           "| workload | shape | selector | positions/step | kernel ms (cold) | kernel ms (hot) | "
           "positions/s | logits GB/s | % of 8 TB/s | % of stream | commits |",
           "|---|---|---|---|---|---|---|---|---|---|---|"]
    loop = [r for r in rows if r["workload"] == "device-loop"]
    lm = [r for r in rows if r["workload"] == "lmhead"]
    rows = [r for r in rows if r["workload"] not in ("device-loop", "lmhead")]
    for r in rows + stress:
        hot = f"{r['kernel_ms_hot']:.4f}" if r["kernel_ms_hot"] is not None else "—"
        cold = f"{r['kernel_ms_cold']:.4f}"
        if str(r.get("note", "")).startswith("hot"):      # steps timed right after their rows were written
            cold, hot = "—", cold
        commits = (f"{r['commits_per_step']:.2f}/step, {r['steps']} steps" if "steps" in r
                   else f"{r.get('mean_commits_per_block', 0):.2f}/block")
        fs = f"{100 * r['frac_of_stream']:.1f}" if r["frac_of_stream"] else "—"
        out.append(f"| {r['workload']} | {r['shape']} | {r['selector']} | {r['positions_per_step']:.0f} | "
                   f"{cold} | {hot} | {r['positions_per_s']:.4g} | "
                   f"{r['logits_GBps']:.0f} | {100 * r['frac_of_peak']:.1f} | {fs} | {commits} |")
    if loop:
        out += ["", "Whole generations in the device-resident loop (`fdllm_generation_run`: "
                "counter-based logits producer, decode step, block advance; wall clock of "
                "`run()`, median of 5, the producer's time included):", "",
                "| shape | mode | steps | ms per generation | µs per step | tokens/s |",
                "|---|---|---|---|---|---|"]
        for r in loop:
            out.append(f"| {r['shape']} | {r['mode']} | {r['steps']} | {r['ms_per_generation']:.3f} | "
                       f"{r['us_per_step']:.1f} | {r['tokens_per_s']:.4g} |")
    if lm:
        out += ["", "LM head fused with the vocabulary pass (`fdllm_lmhead_confidence`: bf16 hidden "
                "states x bf16 output embedding on the matrix cores, online softmax in the epilogue, no "
                "logits stored) against the unfused pair (hipBLASLt GEMM to bf16 logits via torch.matmul, "
                "then `fdllm_confidence`); HIP-event medians, each event pair around 4 back-to-back calls.  "
                "32 positions run the streaming kernel (bound by the read of W, 2 V d bytes), 64 the "
                "two-part streaming kernel, larger shapes the tiled MFMA kernel:", "",
                "| shape | fused ms | fused TFLOP/s | % of 2.5 PFLOP/s | W read TB/s | GEMM ms | pass ms | unfused TFLOP/s | logits not stored |",
                "|---|---|---|---|---|---|---|---|---|"]
        for r in lm:
            out.append(f"| {r['shape']} | {r['fused_ms']:.3f} | {r['fused_TFLOPs']:.0f} | "
                       f"{100 * r['frac_of_bf16_peak']:.1f} | {r['W_TBps']:.2f} | {r['unfused_gemm_ms']:.3f} | "
                       f"{r['unfused_pass_ms']:.3f} | {r['unfused_TFLOPs']:.0f} | "
                       f"{r['logits_bytes_avoided'] / 1e6:.0f} MB |")
    return "\n".join(out) + "\n"


def plan_sweep(reps: int, md_path):
    """Cold decode-step times over the batch size B and the masked rows per
    block m (L = 32, V = 126464 bf16, profile f = 1): the plan the library
    picks at each B (one workgroup per sequence from 256 sequences, rows split
    over waves plus a selection launch below; up to 64 sequences beyond a
    multiple of the CU count take the split plan on a side stream beside the
    fused kernel).  One JSON line; optionally a markdown table."""
    import torch
    import paper_2606_02955_amd as fd
    fd.load()
    dev = torch.device("cuda", 0)
    V, L = 126464, 32
    Bs = (64, 96, 128, 160, 192, 224, 256, 320, 384, 512, 1024)
    ms = (32, 16, 8, 4, 1)
    g = torch.Generator(device=dev).manual_seed(5)
    big = torch.empty((max(Bs), L, V), dtype=torch.bfloat16, device=dev)
    for b0 in range(0, big.shape[0], 64):
        big[b0:b0 + 64].normal_(generator=g)
    scratch = torch.empty(512 << 20, dtype=torch.uint8, device=dev)
    cus = torch.cuda.get_device_properties(dev).multi_processor_count

    def plan_name(B):
        if B < 256:
            return "rows split over waves + selection"
        rem = B % cus
        if 0 < rem <= 64:
            return f"one workgroup per sequence for {B - rem}, split rows for {rem} on a side stream"
        return "one workgroup per sequence"

    res = []
    for B in Bs:
        logits = big[:B]
        start = torch.zeros(B, dtype=torch.int32, device=dev)
        end = torch.full((B,), L, dtype=torch.int32, device=dev)
        x0 = torch.full((B, L), -1, dtype=torch.int32, device=dev)
        nc = torch.empty(B, dtype=torch.int32, device=dev)
        for m in ms:
            mask0 = torch.zeros((B, L), dtype=torch.uint8, device=dev)
            mask0.scatter_(1, torch.rand((B, L), generator=g, device=dev).argsort(1)[:, :m], 1)
            mask, x = mask0.clone(), x0.clone()
            ws = fd.fdllm_decode_step(logits, mask, start, end, x, "profile", 1.0, n_commit=nc)
            ts = []
            for k in range(reps + 2):
                mask.copy_(mask0)
                x.copy_(x0)
                scratch.fill_(k & 0x7F)            # evicts the logits from L2 and the Infinity Cache
                e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                e0.record()
                fd.fdllm_decode_step(logits, mask, start, end, x, "profile", 1.0, n_commit=nc, workspace=ws)
                e1.record()
                torch.cuda.synchronize()
                if k >= 2:
                    ts.append(e0.elapsed_time(e1) * 1e-3)
            t = sorted(ts)[len(ts) // 2]
            nbytes = B * m * V * 2
            res.append({"B": B, "m": m, "us": t * 1e6, "GBps": nbytes / t / 1e9,
                        "plan": plan_name(B)})
            log(f"plan sweep B={B} m={m}: {t * 1e6:.1f} us, {nbytes / t / 1e9:.0f} GB/s")
    print(json.dumps({"metric": "decode-step time over batch size and masked rows per block (cold)",
                      "L": L, "V": V, "dtype": "bf16", "reps": reps, "rows": res}), flush=True)
    if md_path:
        out = ["# Decode-step plan sweep (one MI355X)", "", "Command (from the repository root):", "",
               f"    python bench.py --plan-sweep --plan-sweep-md <file>", "",
               "Cold decode steps (512 MB overwritten before each), L = 32, V = 126464 bf16, profile f = 1, "
               f"median of {reps}; m of the 32 positions of every block masked.  B >= 256 runs one workgroup "
               "per sequence, smaller batches the split rows plus a selection launch; beyond a multiple of "
               f"the {cus} CUs, up to 64 sequences run the split plan on a side stream beside the fused "
               "kernel (B = 320 here).  Cells: µs (logits GB/s).", "",
               "| B | " + " | ".join(f"m = {m}" for m in ms) + " |", "|---|" + "---|" * len(ms)]
        for B in Bs:
            cells = [r for r in res if r["B"] == B]
            out.append(f"| {B} | " + " | ".join(f"{r['us']:.1f} ({r['GBps']:.0f})" for r in cells) + " |")
        with open(md_path, "w") as fh:
            fh.write("\n".join(out) + "\n")


def lmhead_only(n, steps, warmup):
    """Times fdllm_lmhead_confidence on n positions (one sequence's block of
    up to 32, or n / 32 of them) with random bf16 hidden states and output
    embedding; prints one JSON line."""
    import torch
    import paper_2606_02955_amd as fd
    import workloads
    fd.load()
    dev = torch.device("cuda", 0)
    d, V = 4096, workloads.V_LLADA
    L = min(n, 32)
    B = (n + L - 1) // L
    g = torch.Generator(device=dev).manual_seed(2606)
    weight = (torch.randn((V, d), generator=g, device=dev) / 64).to(torch.bfloat16)
    hid = torch.randn((B, L, d), generator=g, device=dev).to(torch.bfloat16)
    mk = torch.ones((B, L), dtype=torch.uint8, device=dev)
    mk.view(-1)[n:] = 0
    st_ = torch.zeros(B, dtype=torch.int32, device=dev)
    en_ = torch.full((B,), L, dtype=torch.int32, device=dev)
    tok = torch.empty((B, L), dtype=torch.int32, device=dev)
    cf = torch.empty((B, L), device=dev)
    ws = fd.fdllm_lmhead_confidence(hid, weight, mk, st_, en_, tok, cf)
    for _ in range(warmup):
        fd.fdllm_lmhead_confidence(hid, weight, mk, st_, en_, tok, cf, workspace=ws)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(steps):
        fd.fdllm_lmhead_confidence(hid, weight, mk, st_, en_, tok, cf, workspace=ws)
    e1.record()
    torch.cuda.synchronize()
    t = e0.elapsed_time(e1) * 1e-3 / steps
    print(json.dumps({"metric": "fused LM head + vocabulary pass, one GPU", "value": n / t,
                      "unit": "positions/s", "ms_per_call": 1e3 * t, "steps": steps, "warmup": warmup,
                      "positions": n, "B": B, "L": L, "d": d, "V": V, "dtype": "bf16",
                      "W_read_TBps": 2.0 * V * d / t / 1e12, "data": "synthetic"}), flush=True)


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--selector", default="profile", choices=["profile", "factor", "threshold"])
    ap.add_argument("--param", type=float, default=None, help="f (default 1.0) or tau (default 0.9)")
    ap.add_argument("--cpu-blocks", type=int, default=90, help="blocks in the one-core oracle sample")
    ap.add_argument("--cpu-workers", type=int, default=0,
                    help="processes of the all-core oracle run (0: host CPUs, at most 16)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-selector-sweep", action="store_true")
    ap.add_argument("--per-workload", action="store_true", help="also time the other workload recipes")
    ap.add_argument("--per-workload-md", default=None, help="write the per-workload table here")
    ap.add_argument("--settle-ms", type=float, default=100.0,
                    help="untimed back-to-back read-only streams (GPU ms) right before each timed run's "
                         "warm-up steps, so the clocks are at their loaded steady state (0: none)")
    ap.add_argument("--copy-calibration-mb", type=int, default=1024,
                    help="size of a plain device copy timed (and counted by rocprofv3) for reference")
    ap.add_argument("--plan-sweep", action="store_true",
                    help="instead: cold decode-step times over batch size and masked rows per block")
    ap.add_argument("--plan-sweep-md", default=None, help="write the plan sweep as a markdown table here")
    ap.add_argument("--lmhead-positions", type=int, default=0,
                    help="instead: time only the fused LM head on this many positions "
                         "(d=4096, V=126464 bf16; one JSON line)")
    ap.add_argument("--traffic-from", nargs=2, metavar=("FETCH_CSV", "WRITE_CSV"), default=None,
                    help="instead: turn the counter_collection csv files of two rocprofv3 runs of "
                         "this script (--pmc FETCH_SIZE, then --pmc WRITE_SIZE) into the fused "
                         "step's HBM traffic, written to --traffic-out")
    ap.add_argument("--traffic-out", default=TRAFFIC)
    args = ap.parse_args()
    if args.traffic_from:
        traffic_from(args.traffic_from[0], args.traffic_from[1], args.traffic_out,
                     args.copy_calibration_mb)
        return
    if args.gpus != 1:
        print(f"bench.py measures one GPU only; --gpus {args.gpus} is not supported "
              f"(sequences shard across GPUs with no exchange, so the per-GPU figure is the one-GPU run)",
              file=sys.stderr)
        sys.exit(2)
    param = args.param if args.param is not None else (0.9 if args.selector == "threshold" else 1.0)
    if args.lmhead_positions > 0:
        lmhead_only(args.lmhead_positions, args.steps, args.warmup)
        return
    if args.plan_sweep:
        plan_sweep(10, args.plan_sweep_md)
        return

    pool, pool_note = None, None
    if not args.no_cpu_baseline:
        if under_profiler():
            # the profiler's preloaded library has initialised the GPU already,
            # and processes are not spawned from such a process
            pool_note = "oracle run (parity and all-core baseline) skipped under a profiler"
        else:
            try:
                from oracle.parallel import OraclePool
                pool = OraclePool(args.cpu_workers or min(MAX_HOST_WORKERS, len(os.sched_getaffinity(0))))
                log(f"cpu_baseline: started {pool.workers} oracle processes")
            except Exception as e:          # no process support: one-core figure only
                pool_note = f"all-core oracle run unavailable: {e!r}"

    import torch
    import paper_2606_02955_amd as fd
    import workloads

    fd.load()
    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    log(f"generating the throughput-stress inputs on {torch.cuda.get_device_name(dev)}")
    inp = workloads.stress_b1024_l32(device=dev, progress=log)
    B, L, V = inp.logits.shape
    positions = int(inp.mask.sum())
    logits_bytes = positions * V * inp.logits.element_size()
    algo_bytes = logits_bytes + B * L * IO_BYTES_PER_POSITION + B * 12
    mask0, x0 = inp.mask.clone(), inp.x.clone()
    mask, x = inp.mask.clone(), inp.x.clone()
    outs = dict(tokens=torch.empty((B, L), dtype=torch.int32, device=dev),
                conf=torch.empty((B, L), device=dev), eps=torch.empty((B, L), device=dev),
                lse=torch.empty((B, L), device=dev),
                commit=torch.empty((B, L), dtype=torch.uint8, device=dev),
                n_commit=torch.empty((B,), dtype=torch.int32, device=dev))
    torch.cuda.synchronize()

    copy_ref = None
    if args.copy_calibration_mb > 0:
        n = args.copy_calibration_mb << 20
        # an elementwise kernel that reads n bytes and writes n bytes: its
        # FETCH_SIZE / WRITE_SIZE counters calibrate the fused kernel's
        src = torch.empty(n, dtype=torch.uint8, device=dev).fill_(1)
        dst = torch.empty_like(src)
        torch.add(src, 1, out=dst)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record()
        for _ in range(5):
            torch.add(src, 1, out=dst)
        e1.record()
        torch.cuda.synchronize()
        t = e0.elapsed_time(e1) * 1e-3 / 5
        copy_ref = {"bytes_read": n, "bytes_written": n, "seconds": t,
                    "read_plus_write_GBps": 2 * n / t / 1e9}
        del src, dst

    # read-only stream of the same logits buffer: the measured bandwidth ceiling
    sink = torch.zeros(1, dtype=torch.int32, device=dev)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    fd.fdllm_stream_read(inp.logits, sink)
    e1.record()
    torch.cuda.synchronize()
    stream_est_ms = max(e0.elapsed_time(e1), 0.05)

    def settle():
        # After an idle pause the GPU's clocks need ~25 ms of load to return to
        # their loaded steady state (the first timed steps then run up to 25%
        # slower); back-to-back untimed reads of the logits, queued right
        # before the warm-up steps, bring them there.
        for _ in range(int(math.ceil(args.settle_ms / stream_est_ms))):
            fd.fdllm_stream_read(inp.logits, sink)

    settle()
    sevs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
            for _ in range(5)]
    for a, b in sevs:
        a.record()
        fd.fdllm_stream_read(inp.logits, sink)
        b.record()
    torch.cuda.synchronize()
    stream_s = sum(a.elapsed_time(b) for a, b in sevs) * 1e-3 / len(sevs)
    stream_bytes = inp.logits.numel() * inp.logits.element_size()
    stream_gbps = stream_bytes / stream_s / 1e9
    log(f"stream read: {stream_gbps:.0f} GB/s")

    def run(selector, p, steps, warmup, label):
        evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
               for _ in range(steps)]
        # every timed step gets its own copy of the step's input mask and x,
        # staged before the timed region, so each does the same work and the
        # timed region holds the decode steps only
        masks = mask0.unsqueeze(0).repeat(steps, 1, 1)
        xs = x0.unsqueeze(0).repeat(steps, 1, 1)
        settle()
        for _ in range(warmup):
            mask.copy_(mask0); x.copy_(x0)
            fd.fdllm_decode_step(inp.logits, mask, inp.start, inp.end, x, selector, p, **outs)
        torch.cuda.synchronize()
        log(f"{label}: timing {steps} steps")
        t0 = time.perf_counter()
        for k in range(steps):
            evs[k][0].record()
            fd.fdllm_decode_step(inp.logits, masks[k], inp.start, inp.end, xs[k], selector, p, **outs)
            evs[k][1].record()
        torch.cuda.synchronize()
        wall = time.perf_counter() - t0
        mask.copy_(masks[-1]); x.copy_(xs[-1])
        kern = [a.elapsed_time(b) * 1e-3 for a, b in evs]
        return wall, sum(kern) / len(kern), min(kern)

    wall, kavg, kmin = run(args.selector, param, args.steps, args.warmup, f"{args.selector}({param})")
    commits = float(outs["n_commit"].float().mean())
    # the headline run's outputs (every timed step computes the same), kept for the parity check
    saved = {k: v.clone() for k, v in outs.items()}
    saved.update(mask=mask.clone(), x=x.clone())
    inp.mask0, inp.x0 = mask0, x0
    sweep = {}
    stress_rows = [_row(workloads.RECIPE_NAMES[workloads.STRESS], "B=1024 L=32 V=126464 bf16", f"{args.selector}({param})", positions,
                    logits_bytes, kavg, None, stream_gbps, {"mean_commits_per_block": commits})]
    if not args.no_selector_sweep:
        for sel, p in [("profile", 1.0), ("profile", 0.75), ("factor", 1.0), ("factor", 0.75),
                       ("threshold", 0.9)]:
            if sel == args.selector and p == param:
                continue
            n2 = max(5, args.steps // 4)
            w2, k2, _ = run(sel, p, n2, 1, f"{sel}({p})")
            mc = float(outs["n_commit"].float().mean())
            sweep[f"{sel}({p})"] = {"ms_per_step": 1e3 * w2 / n2, "kernel_ms": 1e3 * k2,
                                    "mean_commits_per_block": mc}
            stress_rows.append(_row(workloads.RECIPE_NAMES[workloads.STRESS], "B=1024 L=32 V=126464 bf16", f"{sel}({p})", positions,
                                logits_bytes, k2, None, stream_gbps, {"mean_commits_per_block": mc}))
    ms = 1e3 * wall / args.steps
    value = positions * args.steps / wall
    achieved = algo_bytes / kavg / 1e9
    traffic = measured_traffic()
    line = {
        "metric": METRIC,
        "value": value,
        "unit": "masked positions/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "settle_ms": args.settle_ms,
        "ms_per_step": ms,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": "throughput stress: B=1024 blocks x L=32 masked positions, "
                               "V=126464 bf16 logits (Gumbel(0,1), 10% planted near-ties), one fused "
                               f"decode step ({args.selector} {'tau' if args.selector == 'threshold' else 'f'}={param})",
                   "B": B, "L": L, "V": V, "logits_dtype": "bf16", "selector": args.selector,
                   "param": param, "parallelism": "none (1 GPU)"},
        "logits_read_GBps": logits_bytes * args.steps / wall / 1e9,
        "logits_read_frac_of_peak": logits_bytes * args.steps / wall / 1e9 / HBM_PEAK_GBPS,
        "kernel_ms_avg": 1e3 * kavg,
        "kernel_ms_min": 1e3 * kmin,
        "mean_commits_per_block": commits,
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                     "frac": achieved / HBM_PEAK_GBPS,
                     "traffic": traffic,
                     "kernel": "k_fused (one launch per step)",
                     "algorithmic_bytes_per_launch": algo_bytes,
                     "stream_read_GBps": stream_gbps,
                     "frac_of_stream_read": achieved / stream_gbps},
        "selectors": sweep,
        "copy_reference": copy_ref,
        "source_sha256_16": source_digest(),
    }
    if args.per_workload:
        rows = per_workload_report(fd, torch, workloads, dev, stream_gbps, reps=10, settle=settle)
        line["per_workload"] = rows + stress_rows
        if args.per_workload_md:
            cmd = "python bench.py " + " ".join(sys.argv[1:])
            with open(args.per_workload_md, "w") as fh:
                fh.write(per_workload_markdown(rows, stress_rows, stream_gbps, cmd))
    if not args.no_cpu_baseline:
        base = None
        if pool is not None:
            log(f"parity: oracle on every block of the timed step, {pool.workers} processes")
            try:
                parity, base = oracle_parity(pool, inp, saved, args.selector, param)
                line["parity"] = parity
                log(f"parity: {parity['mismatches']} mismatches, {parity['flagged']} flagged, "
                    f"{parity['token_mismatches']} token / {parity['value_mismatches']} value mismatches")
            except Exception as e:
                pool_note = f"all-core oracle run failed: {e!r}"
            finally:
                pool.close()
        log(f"cpu_baseline: oracle on {args.cpu_blocks} blocks, one core")
        single = cpu_baseline_single(inp, saved, args.cpu_blocks, args.selector, param)
        single["cpu_model"] = cpu_model()
        if base is None:
            base = dict(single)
            if pool_note:
                base["note"] = pool_note
        else:
            base.update(cpu_model=cpu_model(), single_core=single)
        base["host_cpus_available"] = len(os.sched_getaffinity(0))
        line["cpu_baseline"] = base
    else:
        line["cpu_baseline"] = None
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
