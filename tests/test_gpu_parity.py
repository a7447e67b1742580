"""GPU parity: the HIP path against the CPU oracle on the same seeded inputs.

Level 1: per-position outputs of fdllm_confidence vs the oracle.
Level 2: fdllm_select_* vs the oracle's rules fed the GPU's own conf/eps.
Level 3: fdllm_decode_step end to end vs the oracle's decode step.
"""
import numpy as np
import pytest
import torch

import oracle
import workloads
from parity import (say, row_source, candidates, compare_rows, gpu_confidence,
                    oracle_confidence_subset, check_defaults, compare_selection, sub_mask)

pytestmark = pytest.mark.gpu

RULES = [("profile", 1.0), ("profile", 0.75), ("profile", 2.0), ("factor", 1.0),
         ("factor", 0.75), ("threshold", 0.9), ("robust", 1.0), ("robust", 0.75)]


def _eta(rule, B, L, seed):
    """(eta tensor or None, uniform value, oracle eta) for a rule: per-position
    allowances for robust(1.0), a uniform one for robust(0.75)."""
    if rule != "robust":
        return None, 0.0, None
    g = torch.Generator(device="cuda").manual_seed(seed)
    eta = torch.rand((B, L), generator=g, device="cuda") * 0.1
    return eta, 0.0, eta.double().cpu().numpy()


def _eta_for(rule, p, B, L, seed):
    if rule == "robust" and p == 0.75:
        return None, 0.03, 0.03
    return _eta(rule, B, L, seed)

SMALL = [
    # (B, L, V, dtype, window)  -- vector and scalar paths, ragged wave-loads
    (3, 20, 16, torch.bfloat16, None),
    (2, 9, 13, torch.bfloat16, None),
    (4, 40, 1000, torch.bfloat16, None),
    (2, 70, 5003, torch.float32, None),
    (5, 8, 8200, torch.bfloat16, None),
    (3, 33, 126464, torch.bfloat16, 33),
    (2, 17, 126464, torch.float32, 17),
    (2, 64, 6000, torch.float32, 64),
    (130, 8, 520, torch.bfloat16, None),      # below 256 sequences: split plan
    (260, 8, 520, torch.bfloat16, None),      # enough sequences for the fused plan
    (160, 12, 1024, torch.float32, 12),
    (320, 12, 1024, torch.float32, 12),
    (129, 3, 7, torch.bfloat16, None),        # split plan, scalar path
    (257, 3, 7, torch.bfloat16, None),        # fused plan, scalar path
    (2, 24, 40000, torch.bfloat16, 24),       # rows split 8 ways (decode: two workgroups per row)
    (1, 20, 70001, torch.bfloat16, None),     # split 16 ways, scalar path
    (8, 64, 6000, torch.float32, 64),         # from 8 sequences: 32 row groups, two rows each
    (7, 48, 3000, torch.bfloat16, None),      # below 8 sequences: 64 row groups
    (16, 40, 20000, torch.bfloat16, 40),      # 32 row groups, windows of 33-40 rows
]

# blocks beyond one wavefront (block-size ablation): workgroup selection
WIDE = [
    (3, 200, 1000, torch.bfloat16, 200),      # two-kernel plan
    (2, 1024, 300, torch.float32, 1024),      # largest block
    (260, 100, 64, torch.bfloat16, 100),      # fused plan
    (129, 700, 40, torch.bfloat16, 700),      # split plan
    (257, 700, 40, torch.bfloat16, 700),
    (256, 1024, 13, torch.float32, 1024),     # fused plan, scalar path, largest block
]


def _case(B, L, V, dt, window, seed=0):
    return workloads.random_case(B, L, V, dt, device="cuda", seed=seed, window=window)


@pytest.mark.parametrize("B,L,V,dt,window", SMALL + WIDE)
def test_confidence_vs_oracle(gpu, B, L, V, dt, window):
    inp = _case(B, L, V, dt, window, seed=B * 7 + L)
    say(f"[confidence] {inp.name}")
    g = [t.cpu().numpy() for t in gpu_confidence(gpu, inp)]
    o = oracle_confidence_subset(inp, range(B))
    mask, start, end = inp.mask.cpu().numpy(), inp.start.cpu().numpy(), inp.end.cpu().numpy()
    cells = candidates(mask, start, end, range(B))
    worst = compare_rows(*g, *o, cells)
    check_defaults(*g, mask, start, end, range(B))
    say(f"  {len(cells)} rows, worst rel err {worst}")


@pytest.mark.parametrize("B,L,V,dt,window", SMALL[:6] + SMALL[8:9] + WIDE[:3])
def test_select_vs_oracle_on_gpu_confidences(gpu, B, L, V, dt, window):
    inp = _case(B, L, V, dt, window, seed=B * 11 + L)
    say(f"[select] {inp.name}")
    tok, conf, eps, lse = gpu_confidence(gpu, inp)
    mask, start, end = inp.mask.cpu().numpy(), inp.start.cpu().numpy(), inp.end.cpu().numpy()
    for use_eps in (True, False):
        e_in = eps if use_eps else None
        e_or = eps.double().cpu().numpy() if use_eps else 1.0 - conf.double().cpu().numpy()
        for rule, p in RULES:
            eta, eta_u, eta_o = _eta_for(rule, p, B, L, B + L)
            commit = torch.full((B, L), 9, dtype=torch.uint8, device="cuda")
            n = torch.full((B,), -9, dtype=torch.int32, device="cuda")
            gpu.select(rule, conf, e_in, inp.mask, inp.start, inp.end, p, commit, n, eta=eta, eta_uniform=eta_u)
            torch.cuda.synchronize()
            oc, on, flagged, _ = oracle.select(e_or, conf.double().cpu().numpy(), mask, start, end, rule, p,
                                               eta=eta_o)
            nf, nfm = compare_selection(commit.cpu().numpy(), n.cpu().numpy(), oc, on, flagged, range(B))
            say(f"  {rule}({p}) eps={'gpu' if use_eps else '1-conf'}: flagged {nf} (matching {nfm})")


def _decode(gpu, inp, rule, p, with_outputs=True, eta=None, eta_uniform=0.0):
    B, L, V = inp.logits.shape
    d = "cuda"
    mask, x = inp.mask.clone(), inp.x.clone()
    outs = dict(tokens=torch.full((B, L), -7, dtype=torch.int32, device=d),
                conf=torch.full((B, L), -7.0, device=d), eps=torch.full((B, L), -7.0, device=d),
                lse=torch.full((B, L), -7.0, device=d),
                commit=torch.full((B, L), 9, dtype=torch.uint8, device=d),
                n_commit=torch.full((B,), -9, dtype=torch.int32, device=d))
    if not with_outputs:
        outs = dict(commit=outs["commit"], n_commit=outs["n_commit"])
    gpu.fdllm_decode_step(inp.logits, mask, inp.start, inp.end, x, rule, p, eta=eta,
                          eta_uniform=eta_uniform, **outs)
    torch.cuda.synchronize()
    return mask, x, outs


@pytest.mark.parametrize("B,L,V,dt,window", SMALL + WIDE)
def test_decode_step_vs_oracle(gpu, B, L, V, dt, window):
    inp = _case(B, L, V, dt, window, seed=B * 13 + L)
    say(f"[decode] {inp.name}")
    m0, x0 = inp.mask.cpu().numpy(), inp.x.cpu().numpy()
    start, end = inp.start.cpu().numpy(), inp.end.cpu().numpy()
    ref_conf = gpu_confidence(gpu, inp)
    rows = row_source(inp.logits.cpu())
    for rule, p in RULES:
        eta, eta_u, eta_o = _eta_for(rule, p, B, L, B * 3 + L)
        mask, x, o = _decode(gpu, inp, rule, p, eta=eta, eta_uniform=eta_u)
        r = oracle.decode_step(rows, B, L, m0, start, end, x0, rule, p, eta=eta_o)
        nf, nfm = compare_selection(o["commit"].cpu().numpy(), o["n_commit"].cpu().numpy(),
                                    r.commit, r.n_commit, r.flagged, range(B))
        ok = ~r.flagged
        assert np.array_equal(x.cpu().numpy()[ok], r.x[ok])
        assert np.array_equal(mask.cpu().numpy()[ok], r.mask[ok])
        # bitwise the same per-position outputs as fdllm_confidence
        for name, t in zip(("tokens", "conf", "eps", "lse"), ref_conf):
            assert torch.equal(o[name].view(torch.int32), t.view(torch.int32)), name
        # and the same commits as fdllm_select_* fed those outputs, then reveal
        c2 = torch.zeros((B, L), dtype=torch.uint8, device="cuda")
        n2 = torch.zeros((B,), dtype=torch.int32, device="cuda")
        gpu.select(rule, ref_conf[1], ref_conf[2], inp.mask, inp.start, inp.end, p, c2, n2,
                   eta=eta, eta_uniform=eta_u)
        m2, x2 = inp.mask.clone(), inp.x.clone()
        gpu.fdllm_reveal(c2, ref_conf[0], x2, m2)
        torch.cuda.synchronize()
        assert torch.equal(c2, o["commit"]) and torch.equal(n2, o["n_commit"])
        assert torch.equal(m2, mask) and torch.equal(x2, x)
        # outputs are optional
        mask3, x3, o3 = _decode(gpu, inp, rule, p, with_outputs=False, eta=eta, eta_uniform=eta_u)
        assert torch.equal(mask3, mask) and torch.equal(x3, x) and torch.equal(o3["commit"], o["commit"])
        say(f"  {rule}({p}): commits {int(o['n_commit'].clamp(min=0).sum())}, flagged {nf} (matching {nfm})")


def test_crafted_profiles_on_gpu(gpu):
    """The hand-derived worked examples, fed to the GPU selectors as float32."""
    import test_oracle_select as ts
    cases = ts.load_golden()
    B, L = len(cases), 16
    conf = torch.zeros((B, L)); eps = torch.ones((B, L)); eta = torch.zeros((B, L))
    mask = torch.zeros((B, L), dtype=torch.uint8)
    for b, cs in enumerate(cases):
        for k, (c, pos) in enumerate(zip(cs["c"], cs["pos"])):
            conf[b, pos % L] = float(c)
            eps[b, pos % L] = float(1 - c)
            mask[b, pos % L] = 1
            if cs["eta"] is not None:
                eta[b, pos % L] = cs["eta"][k]
    start = torch.zeros(B, dtype=torch.int32); end = torch.full((B,), L, dtype=torch.int32)
    args = [t.cuda() for t in (conf, eps, mask, start, end)]
    eta = eta.cuda()
    for b, cs in enumerate(cases):
        commit = torch.zeros((B, L), dtype=torch.uint8, device="cuda")
        n = torch.zeros((B,), dtype=torch.int32, device="cuda")
        gpu.select(cs["rule"], *args[:2], *args[2:], cs["param"], commit, n, eta=eta)
        torch.cuda.synchronize()
        got = sorted(np.nonzero(commit[b].cpu().numpy())[0].tolist())
        assert int(n[b]) == cs["n_star"], cs
        assert got == sorted(p % L for p in cs["committed"]), cs


def test_invalid_bounds_on_device(gpu):
    V = 64
    for (BB, LL) in [(6, 20), (130, 100), (260, 100), (7, 1100), (130, 1030), (260, 1030)]:
        case = workloads.random_case(BB, LL, V, torch.bfloat16, device="cuda", seed=7, poison=False)
        s = torch.zeros(BB, dtype=torch.int32); e = torch.zeros(BB, dtype=torch.int32)
        bounds = [(0, LL), (5, 4), (-1, 3), (0, LL + 1), (3, 3), (10, 10 + 65), (2, 2 + 1025)]
        for b in range(BB):
            s[b], e[b] = bounds[b % len(bounds)]
        case.start.copy_(s); case.end.copy_(e)
        say(f"[bounds] B={BB} L={LL}")
        mask, x, o = _decode(gpu, case, "profile", 1.0)
        n = o["n_commit"].cpu().numpy()
        for b in range(BB):
            lo, hi = bounds[b % len(bounds)]
            bad = not (0 <= lo <= hi <= LL and hi - lo <= gpu.MAX_BLOCK)
            if bad:
                assert n[b] == -1
                assert not o["commit"][b].any()
                assert torch.equal(mask[b], case.mask[b]) and torch.equal(x[b], case.x[b])
                assert (o["tokens"][b] == -1).all()
            elif hi == lo:
                assert n[b] == 0


def test_determinism_and_identical_rows(gpu):
    B, L, V = 260, 16, 126464
    g = torch.Generator(device="cuda").manual_seed(5)
    one = torch.randn((1, 1, V), generator=g, device="cuda") * 2
    one[0, 0, 123] += 15.0
    logits = one.expand(B, L, V).to(torch.bfloat16).contiguous()
    mask = torch.ones((B, L), dtype=torch.uint8, device="cuda")
    start = torch.zeros(B, dtype=torch.int32, device="cuda")
    end = torch.full((B,), L, dtype=torch.int32, device="cuda")
    x = torch.full((B, L), -1, dtype=torch.int32, device="cuda")
    inp = workloads.StepInputs(logits, mask, start, end, x, "identical")
    say("[determinism] fused plan, identical rows")
    a = gpu_confidence(gpu, inp)
    b_ = gpu_confidence(gpu, inp)
    for t1, t2 in zip(a, b_):
        assert torch.equal(t1.view(torch.int32), t2.view(torch.int32))
        flat = t1.view(torch.int32).flatten()
        assert (flat == flat[0]).all()                 # identical rows -> identical bits
    for f in (0.5, 0.75, 1.0, 2.0):
        _, _, op = _decode(gpu, inp, "profile", f)
        _, _, of = _decode(gpu, inp, "factor", f)
        assert torch.equal(op["commit"], of["commit"]) and torch.equal(op["n_commit"], of["n_commit"])


REPEATED_MAX = [
    # (B, L, V, dtype): the row maximum repeats in many lanes and batches
    (260, 3, 126464, torch.bfloat16),         # fused plan for the decode step
    (2, 24, 40000, torch.bfloat16),           # rows split 8 ways
    (1, 20, 70001, torch.bfloat16),           # split 16 ways, scalar path
    (2, 9, 126464, torch.float32),
]


def _repeated_max_case(B, L, V, dt, seed):
    """Integer logits in [-8, 8], so the value 8 appears about V/17 times per
    row.  Position 0 of every sequence is a constant row (every element is a
    maximum), position 1 has its only maximum at the last element and
    position 2 at the first and the last."""
    g = torch.Generator(device="cuda").manual_seed(seed)
    logits = torch.randint(-8, 9, (B, L, V), generator=g, device="cuda").to(dt)
    logits[:, 0, :] = 3
    logits[:, 1:3, :] = logits[:, 1:3, :].clamp(max=7)
    logits[:, 1, V - 1] = 8
    logits[:, 2, 0] = 8
    logits[:, 2, V - 1] = 8
    mask = torch.ones((B, L), dtype=torch.uint8, device="cuda")
    start = torch.zeros(B, dtype=torch.int32, device="cuda")
    end = torch.full((B,), L, dtype=torch.int32, device="cuda")
    x = torch.full((B, L), -1, dtype=torch.int32, device="cuda")
    return workloads.StepInputs(logits, mask, start, end, x, f"repeated maxima B={B} L={L} V={V} {dt}")


@pytest.mark.parametrize("B,L,V,dt", REPEATED_MAX)
def test_argmax_with_repeated_maxima(gpu, B, L, V, dt):
    """Ties broken to the lowest index when the maximum value repeats
    thousands of times per row, across lanes, batches and split parts."""
    inp = _repeated_max_case(B, L, V, dt, seed=B + L + V)
    say(f"[repeated max] {inp.name}")
    gt = gpu_confidence(gpu, inp)
    g = [t.cpu().numpy() for t in gt]
    first = inp.logits.float().cpu().numpy().argmax(axis=-1)   # numpy: first occurrence
    assert np.array_equal(g[0], first)
    assert (g[0][:, 0] == 0).all() and (g[0][:, 1] == V - 1).all() and (g[0][:, 2] == 0).all()
    o = oracle_confidence_subset(inp, range(B))
    mask, start, end = inp.mask.cpu().numpy(), inp.start.cpu().numpy(), inp.end.cpu().numpy()
    worst = compare_rows(*g, *o, candidates(mask, start, end, range(B)))
    _, _, od = _decode(gpu, inp, "profile", 1.0)
    for name, t in zip(("tokens", "conf", "eps", "lse"), gt):
        assert torch.equal(od[name].view(torch.int32), t.view(torch.int32)), name
    say(f"  worst rel err {worst}")


def _tied_profiles(B, L, seed):
    """conf on a coarse grid (many exact ties) with a few large gaps."""
    g = torch.Generator().manual_seed(seed)
    q = torch.randint(40, 65, (B, L), generator=g).float() / 64
    fine = torch.rand((B, L), generator=g) < 0.5
    conf = torch.where(fine, 1 - torch.rand((B, L), generator=g) ** 3 * 0.05, q)
    mask = (torch.rand((B, L), generator=g) < 0.8).to(torch.uint8)
    return conf, mask


@pytest.mark.parametrize("B,L", [(7, 1024), (130, 700)])
def test_wide_blocks_select_vs_oracle(gpu, B, L):
    """Windows from empty to 1024 slots, exact ties, both kernels' selection paths."""
    conf, mask = _tied_profiles(B, L, seed=B + L)
    spans = [(0, L), (0, 65), (L // 10, L - L // 7), (5, 5 + 64), (3, 3 + 128), (L - 777 % L, L),
             (1, 1), (0, 1), (0, 63)]
    start = torch.tensor([spans[b % len(spans)][0] for b in range(B)], dtype=torch.int32)
    end = torch.tensor([min(spans[b % len(spans)][1], L) for b in range(B)], dtype=torch.int32)
    eps = 1 - conf                                    # exact for these values
    c_d, e_d, m_d, s_d, en_d = (t.cuda() for t in (conf, eps, mask, start, end))
    eta = torch.rand((B, L), generator=torch.Generator().manual_seed(3)) * 0.05
    say(f"[wide select] B={B} L={L}")
    for use_eps in (True, False):
        for rule, p in RULES:
            eta_d = eta.cuda() if rule == "robust" and p == 1.0 else None
            eta_u = 0.03 if rule == "robust" and p == 0.75 else 0.0
            eta_o = eta.double().numpy() if eta_d is not None else (eta_u if rule == "robust" else None)
            commit = torch.full((B, L), 9, dtype=torch.uint8, device="cuda")
            n = torch.full((B,), -9, dtype=torch.int32, device="cuda")
            gpu.select(rule, c_d, e_d if use_eps else None, m_d, s_d, en_d, p, commit, n,
                       eta=eta_d, eta_uniform=eta_u)
            torch.cuda.synchronize()
            oc, on, flagged, _ = oracle.select(eps.double().numpy(), conf.double().numpy(),
                                               mask.numpy(), start.numpy(), end.numpy(), rule, p,
                                               eta=eta_o)
            nf, nfm = compare_selection(commit.cpu().numpy(), n.cpu().numpy(), oc, on, flagged,
                                        range(B))
            say(f"  {rule}({p}) eps={use_eps}: flagged {nf} (matching {nfm})")


@pytest.mark.parametrize("B", [3, 130])
def test_wide_flat_block_profile_equals_factor(gpu, B):
    """A block of 1024 identical rows: B_n = 0, so profile and factor agree bitwise."""
    L, V = 1024, 256
    g = torch.Generator(device="cuda").manual_seed(11)
    one = torch.randn((1, 1, V), generator=g, device="cuda")
    one[0, 0, 17] += 9.0
    logits = one.expand(B, L, V).to(torch.bfloat16).contiguous()
    mask = torch.ones((B, L), dtype=torch.uint8, device="cuda")
    start = torch.zeros(B, dtype=torch.int32, device="cuda")
    end = torch.full((B,), L, dtype=torch.int32, device="cuda")
    x = torch.full((B, L), -1, dtype=torch.int32, device="cuda")
    inp = workloads.StepInputs(logits, mask, start, end, x, "identical-wide")
    say(f"[wide flat] B={B}")
    for f in (0.5, 1.0, 2.0, 50.0):
        _, _, op = _decode(gpu, inp, "profile", f)
        _, _, of = _decode(gpu, inp, "factor", f)
        assert torch.equal(op["commit"], of["commit"]) and torch.equal(op["n_commit"], of["n_commit"])
        n = int(op["n_commit"][0])
        e = float(op["eps"][0, 0])
        want = max([k for k in range(1, L + 1) if (k + 1) * e < f] or [1])
        assert (op["n_commit"] == n).all() and n == want, (n, want)
        # ties go to the lower positions: the first n* slots commit
        assert int(op["commit"][:, :n].sum()) == B * n and int(op["commit"][:, n:].sum()) == 0


@pytest.mark.parametrize("B,L,V,dt,window", [(2, 17, 126464, torch.float32, 17),
                                              (2, 24, 40000, torch.bfloat16, 24)])
def test_decode_step_row_parts_match_single_workgroup(gpu, B, L, V, dt, window):
    """A small batch's rows streamed by several workgroups (the workspace holds
    their partials) give the same bits as one workgroup per row (no workspace)."""
    inp = _case(B, L, V, dt, window, seed=B + L + V)
    say(f"[decode parts vs single workgroup] {inp.name}")
    outs = []
    for ws in (None, torch.empty(1, dtype=torch.uint8, device="cuda")):
        mask, x = inp.mask.clone(), inp.x.clone()
        o = {"tokens": torch.full((B, L), -7, dtype=torch.int32, device="cuda"),
             "conf": torch.full((B, L), -7.0, device="cuda"),
             "eps": torch.full((B, L), -7.0, device="cuda"),
             "lse": torch.full((B, L), -7.0, device="cuda"),
             "commit": torch.full((B, L), 9, dtype=torch.uint8, device="cuda"),
             "n_commit": torch.full((B,), -9, dtype=torch.int32, device="cuda")}
        gpu.fdllm_decode_step(inp.logits, mask, inp.start, inp.end, x, "profile", 1.0, workspace=ws, **o)
        torch.cuda.synchronize()
        outs.append((mask, x, o))
    (m1, x1, o1), (m2, x2, o2) = outs
    assert torch.equal(m1, m2) and torch.equal(x1, x2)
    for k in o1:
        assert torch.equal(o1[k].view(torch.uint8), o2[k].view(torch.uint8)), k


@pytest.mark.parametrize("B,L,V,dt,window", [(260, 32, 126464, torch.bfloat16, 32),
                                              (300, 12, 20000, torch.float32, 12),
                                              (257, 70, 3000, torch.bfloat16, 70),
                                              # the remainder's limits on a 256-CU part: 64 beyond
                                              # one and two CU multiples, then 65 (all fused)
                                              (320, 8, 4096, torch.bfloat16, 8),
                                              (576, 8, 2048, torch.float32, 8),
                                              (321, 8, 4096, torch.float32, 8)])
def test_fused_step_remainder_bits(gpu, B, L, V, dt, window):
    """Sequences beyond a multiple of the CU count take the small-batch plan
    beside the fused kernel: the decode step gives fdllm_confidence's bits for
    every row, the same with and without a workspace, and the oracle's
    results (checked on the remainder and a few fused sequences)."""
    inp = _case(B, L, V, dt, window, seed=B + L)
    say(f"[fused step remainder] {inp.name}")
    ref = gpu_confidence(gpu, inp)
    outs = []
    for ws in ("default", None):
        mask, x = inp.mask.clone(), inp.x.clone()
        o = {"tokens": torch.full((B, L), -7, dtype=torch.int32, device="cuda"),
             "conf": torch.full((B, L), -7.0, device="cuda"),
             "eps": torch.full((B, L), -7.0, device="cuda"),
             "lse": torch.full((B, L), -7.0, device="cuda"),
             "commit": torch.full((B, L), 9, dtype=torch.uint8, device="cuda"),
             "n_commit": torch.full((B,), -9, dtype=torch.int32, device="cuda")}
        kw = {} if ws == "default" else {"workspace": torch.empty(1, dtype=torch.uint8, device="cuda")}
        gpu.fdllm_decode_step(inp.logits, mask, inp.start, inp.end, x, "profile", 1.0, **kw, **o)
        torch.cuda.synchronize()
        outs.append((mask, x, o))
    (m1, x1, o1), (m2, x2, o2) = outs
    assert torch.equal(m1, m2) and torch.equal(x1, x2)
    for k in o1:
        assert torch.equal(o1[k].view(torch.uint8), o2[k].view(torch.uint8)), k
    for k, t in zip(("tokens", "conf", "eps", "lse"), ref):
        assert torch.equal(o1[k].view(torch.uint8), t.view(torch.uint8)), k
    bs = [0, 1, 100] + list(range(B - 8, B))
    m0, x0 = sub_mask(inp.mask.cpu().numpy(), bs), inp.x.cpu().numpy()
    r = oracle.decode_step(row_source(inp.logits), B, L, m0, inp.start.cpu().numpy(),
                           inp.end.cpu().numpy(), x0, "profile", 1.0)
    compare_selection(o1["commit"].cpu().numpy(), o1["n_commit"].cpu().numpy(), r.commit,
                      r.n_commit, r.flagged, bs)


def _random_shapes(n, seed=2606):
    """Seeded small-batch shapes: odd spans, windows above one wavefront, rows
    long enough to be split, both dtypes."""
    rng = np.random.default_rng(seed)
    out = []
    for k in range(n):
        B = int(rng.integers(1, 7))
        L = int(rng.choice([1, 7, 31, 64, 65, 130, 300]))
        V = int(rng.choice([5, 129, 2047, 9000, 40000]))
        dt = torch.bfloat16 if k % 2 == 0 else torch.float32
        lo = 65 if (k % 3 == 0 and L > 64) else 1          # every third: beyond a wavefront
        window = int(rng.integers(lo, min(L, 1024) + 1))
        out.append((B, L, V, dt, window))
    return out


@pytest.mark.parametrize("B,L,V,dt,window", _random_shapes(12))
def test_decode_step_random_shapes(gpu, B, L, V, dt, window):
    """Random small-batch shapes through the two-kernel plans: the oracle's
    selection, defaults outside the windows, and the same bits as
    fdllm_confidence."""
    inp = _case(B, L, V, dt, window, seed=B * 101 + L * 7 + V)
    say(f"[decode random] {inp.name} window {window}")
    m0, x0 = inp.mask.cpu().numpy(), inp.x.cpu().numpy()
    start, end = inp.start.cpu().numpy(), inp.end.cpu().numpy()
    ref_conf = gpu_confidence(gpu, inp)
    check_defaults(*[t.cpu().numpy() for t in ref_conf], m0, start, end, range(B))
    rows = row_source(inp.logits.cpu())
    for rule, p in [("profile", 1.0), ("threshold", 0.9), ("robust", 0.75)]:
        eta, eta_u, eta_o = _eta_for(rule, p, B, L, B + L)
        mask, x, o = _decode(gpu, inp, rule, p, eta=eta, eta_uniform=eta_u)
        r = oracle.decode_step(rows, B, L, m0, start, end, x0, rule, p, eta=eta_o)
        compare_selection(o["commit"].cpu().numpy(), o["n_commit"].cpu().numpy(), r.commit,
                          r.n_commit, r.flagged, range(B))
        ok = ~r.flagged
        assert np.array_equal(x.cpu().numpy()[ok], r.x[ok])
        assert np.array_equal(mask.cpu().numpy()[ok], r.mask[ok])
        for name, t in zip(("tokens", "conf", "eps", "lse"), ref_conf):
            assert torch.equal(o[name].view(torch.int32), t.view(torch.int32)), name


@pytest.mark.parametrize("B,L,V,dt", [(3, 24, 5000, torch.float32), (2, 16, 126464, torch.bfloat16),
                                      (260, 4, 3000, torch.bfloat16), (4, 9, 8191, torch.float32)])
def test_very_confident_rows_eps(gpu, B, L, V, dt):
    """Rows whose greedy token stands 22-85 above an N(0,1) background: eps
    from ~1e-6 down to ~1e-32.  The pass never sums the greedy term, so eps
    matches the oracle to 1e-5 relative down to the float32 terms' underflow."""
    g = torch.Generator().manual_seed(B * 1000 + V)
    rows = torch.randn((B * L, V), generator=g)
    tok = torch.randint(0, V, (B * L,), generator=g)
    h = 22.0 + 63.0 * torch.rand((B * L,), generator=g)
    rows[torch.arange(B * L), tok] = h
    logits = rows.view(B, L, V).to(dt).to("cuda")
    mask = torch.ones((B, L), dtype=torch.uint8, device="cuda")
    start = torch.zeros(B, dtype=torch.int32, device="cuda")
    end = torch.full((B,), L, dtype=torch.int32, device="cuda")
    inp = workloads.StepInputs(logits, mask, start, end, torch.full((B, L), -1, dtype=torch.int32,
                                                                    device="cuda"), "very confident")
    say(f"[very confident] B={B} L={L} V={V} {dt}")
    gc = [t.cpu().numpy() for t in gpu_confidence(gpu, inp)]
    o = oracle_confidence_subset(inp, range(B))
    cells = candidates(mask.cpu().numpy(), start.cpu().numpy(), end.cpu().numpy(), range(B))
    worst = compare_rows(*gc, *o, cells)
    assert float(np.min(o[2][mask.cpu().numpy() != 0])) < 1e-25
    # the decode step's pass gives the same bits
    d = dict(tokens=torch.empty((B, L), dtype=torch.int32, device="cuda"),
             conf=torch.empty((B, L), device="cuda"), eps=torch.empty((B, L), device="cuda"),
             lse=torch.empty((B, L), device="cuda"))
    gpu.fdllm_decode_step(logits, mask.clone(), start, end, inp.x.clone(), "profile", 1.0, **d)
    torch.cuda.synchronize()
    for k, t in zip(("tokens", "conf", "eps", "lse"), gc):
        assert np.array_equal(d[k].cpu().numpy().view(np.int32), t.view(np.int32)), k
    say(f"  worst {worst}")
