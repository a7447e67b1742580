"""GPU parity of the fused LM head + vocabulary pass against the oracle.

The oracle forms every candidate row's logits as float64 dot products of the
bf16 hidden state with the bf16 output embedding (oracle.lmhead), then takes
the per-position confidence and the selection exactly as for given logits.

* "exact" inputs are built so that every logit is exact in float32 whatever
  the accumulation order: tokens must match bit for bit and conf / eps / lse
  within the vocabulary pass's 1e-5;
* "random" inputs carry float32 accumulation error on the GPU: tokens must
  match wherever the oracle's top-two gap exceeds twice the row's rounding
  bound delta, and conf / eps / lse stay within 3 delta (+1e-6).
"""
import numpy as np
import pytest
import torch

import oracle
import workloads
from parity import (say, candidates, compare_rows, check_defaults, compare_selection, CONF_RTOL,
                    EPS_ATOL_LMHEAD)

pytestmark = pytest.mark.gpu

CASES = [
    # B, L, d, V, recipe, window
    (3, 40, 64, 1000, "exact", 40),          # one hidden stage, partial last vocabulary tile
    (20, 32, 256, 4096, "exact", 32),        # 640 rows: three row tiles, the last partial
    (2, 16, 4096, 126464, "exact", 16),      # LLaDA's hidden size and vocabulary
    (3, 100, 128, 777, "exact", 100),        # blocks beyond one wavefront
    (4, 32, 512, 2000, "random", 32),
    (2, 24, 4096, 8192, "random", 24),
    # at most 32 positions and d a multiple of 512 up to 4096: the streaming kernel
    (1, 32, 4096, 1001, "exact", 32),        # one sequence, partial last row block
    (1, 13, 2048, 3000, "random", 13),
    (1, 5, 4096, 10, "exact", 5),            # two row blocks, one per workgroup
    (1, 32, 1024, 1001, "exact", 32),
    (1, 20, 512, 3001, "random", 20),
    (1, 32, 1536, 2000, "exact", 32),
    (4, 8, 1024, 2500, "exact", 5),          # several sequences, windows inside them
    (1, 1, 512, 100, "exact", 1),            # a single position
    (1, 32, 64, 1000, "exact", 32),          # d not a multiple of 512: the tiled kernel
    # 33..64 positions, d a multiple of 1024: the k-split kernel
    (2, 32, 4096, 126464, "exact", 32),      # two sequences' blocks at LLaDA's sizes
    (1, 64, 1024, 3001, "random", 64),
    (2, 20, 3072, 999, "exact", 20),
    (1, 50, 4096, 700, "random", 50),        # fewer row blocks than workgroup groups
    (1, 33, 2048, 1234, "random", 33),       # one position past a single block
    # more positions: the tiled kernel
    (4, 32, 2048, 5000, "exact", 32),
    (3, 40, 4096, 2000, "random", 40),
    (1, 100, 2048, 777, "exact", 100),
    (2, 30, 192, 777, "exact", 30),          # 33..64 positions
    (1, 7, 128, 5000, "random", 7),
]


def _case(B, L, d, V, kind, window, seed):
    return workloads.lmhead_case(B, L, d, V, kind, device="cuda", seed=seed, window=window)


def _oracle_rows(hidden, weight, cells):
    """float64 logits of the candidate cells, one matrix product over W."""
    h = hidden.double().cpu().numpy()
    w = weight.double().cpu().numpy()
    if not cells:
        return {}
    rows = np.stack([h[b, i] for b, i in cells])
    lg = oracle.lmhead.logits_rows(rows, w)
    return {c: lg[k] for k, c in enumerate(cells)}, h, w


def _gpu_conf(gpu, hidden, weight, mask, start, end):
    B, L, _ = hidden.shape
    out = [torch.full((B, L), -7, dtype=torch.int32, device="cuda")] + \
          [torch.full((B, L), -7.0, device="cuda") for _ in range(3)]
    gpu.fdllm_lmhead_confidence(hidden, weight, mask, start, end, *out)
    torch.cuda.synchronize()
    return out


@pytest.mark.parametrize("B,L,d,V,kind,window", CASES)
def test_lmhead_confidence_vs_oracle(gpu, B, L, d, V, kind, window):
    hidden, weight, mask, start, end, x, name = _case(B, L, d, V, kind, window, seed=B + L + d)
    say(f"[lmhead confidence] {name}")
    g = [t.cpu().numpy() for t in _gpu_conf(gpu, hidden, weight, mask, start, end)]
    m, s, e = mask.cpu().numpy(), start.cpu().numpy(), end.cpu().numpy()
    cells = candidates(m, s, e, range(B))
    check_defaults(*g, m, s, e, range(B))
    if not cells:
        return
    lg, h64, w64 = _oracle_rows(hidden, weight, cells)
    unit = (d / 16 + 32) * 2.0 ** -24
    worst = dict(conf=0.0, eps=0.0, lse=0.0)
    near = 0
    for (b, i) in cells:
        t, c, ep, lse = oracle.position_confidence(lg[(b, i)])
        if kind == "exact":
            tol_c = tol_e = CONF_RTOL
            tol_l = CONF_RTOL * max(abs(lse), 1.0)
            assert int(g[0][b, i]) == t, (b, i, int(g[0][b, i]), t)
        else:
            delta = oracle.lmhead.accumulation_bound(h64[b, i], w64, unit)
            top2 = np.partition(lg[(b, i)], -2)[-2:]
            if top2[1] - top2[0] > 2 * delta:
                assert int(g[0][b, i]) == t, (b, i, int(g[0][b, i]), t, delta)
            else:
                near += 1
            tol_c = tol_e = 3 * delta + 1e-6
            tol_l = delta + CONF_RTOL * max(abs(lse), 1.0)
        rc = abs(float(g[1][b, i]) - c) / c
        de = abs(float(g[2][b, i]) - ep)
        re_ = de / max(ep, 1e-30) if de > EPS_ATOL_LMHEAD else 0.0
        rl = abs(float(g[3][b, i]) - lse)
        assert rc <= tol_c and re_ <= max(tol_e, 1e-5) and rl <= tol_l, (b, i, rc, re_, rl, tol_c)
        worst["conf"] = max(worst["conf"], rc)
        worst["eps"] = max(worst["eps"], re_)
        worst["lse"] = max(worst["lse"], rl)
    say(f"  {len(cells)} rows, worst {worst}, near ties {near}")


@pytest.mark.parametrize("B,L,d,V,kind,window", [c for c in CASES if c[4] == "exact"])
def test_lmhead_decode_step_vs_oracle(gpu, B, L, d, V, kind, window):
    hidden, weight, mask, start, end, x, name = _case(B, L, d, V, kind, window, seed=7 * B + L)
    say(f"[lmhead decode] {name}")
    m0, x0 = mask.cpu().numpy(), x.cpu().numpy()
    s, e = start.cpu().numpy(), end.cpu().numpy()
    cells = candidates(m0, s, e, range(B))
    lg = _oracle_rows(hidden, weight, cells)[0] if cells else {}
    rows = lambda b, i: lg[(b, i)]
    ref = _gpu_conf(gpu, hidden, weight, mask, start, end)
    for rule, p in [("profile", 1.0), ("profile", 2.0), ("factor", 1.0), ("threshold", 0.9),
                    ("robust", 0.75)]:
        eta_u = 0.03 if rule == "robust" else 0.0
        mk, xx = mask.clone(), x.clone()
        commit = torch.full((B, L), 9, dtype=torch.uint8, device="cuda")
        n = torch.full((B,), -9, dtype=torch.int32, device="cuda")
        tok = torch.empty((B, L), dtype=torch.int32, device="cuda")
        conf = torch.empty((B, L), device="cuda")
        gpu.fdllm_lmhead_decode_step(hidden, weight, mk, start, end, xx, rule, p, tokens=tok,
                                     conf=conf, commit=commit, n_commit=n, eta_uniform=eta_u)
        torch.cuda.synchronize()
        r = oracle.decode_step(rows, B, L, m0, s, e, x0, rule, p, eta=eta_u if rule == "robust" else None)
        nf, nfm = compare_selection(commit.cpu().numpy(), n.cpu().numpy(), r.commit, r.n_commit,
                                    r.flagged, range(B))
        ok = ~r.flagged
        assert np.array_equal(xx.cpu().numpy()[ok], r.x[ok])
        assert np.array_equal(mk.cpu().numpy()[ok], r.mask[ok])
        # the step's per-position outputs are those of fdllm_lmhead_confidence
        assert torch.equal(tok, ref[0]) and torch.equal(conf.view(torch.int32), ref[1].view(torch.int32))
        say(f"  {rule}({p}): commits {int(n.clamp(min=0).sum())}, flagged {nf} (matching {nfm})")


def test_lmhead_decode_step_eta_tensor(gpu):
    """The robust rule with a per-position allowance, LM-head form."""
    B, L, d, V, window = 6, 24, 128, 3000, 24
    hidden, weight, mask, start, end, x, name = _case(B, L, d, V, "exact", window, seed=5)
    say(f"[lmhead decode eta tensor] {name}")
    m0, x0 = mask.cpu().numpy(), x.cpu().numpy()
    s, e = start.cpu().numpy(), end.cpu().numpy()
    cells = candidates(m0, s, e, range(B))
    lg = _oracle_rows(hidden, weight, cells)[0] if cells else {}
    eta = np.random.default_rng(2).uniform(-0.02, 0.08, (B, L)).astype(np.float32)
    mk, xx = mask.clone(), x.clone()
    commit = torch.empty((B, L), dtype=torch.uint8, device="cuda")
    n = torch.empty((B,), dtype=torch.int32, device="cuda")
    gpu.fdllm_lmhead_decode_step(hidden, weight, mk, start, end, xx, "robust", 0.9, commit=commit,
                                 n_commit=n, eta=torch.from_numpy(eta).cuda())
    torch.cuda.synchronize()
    r = oracle.decode_step(lambda b, i: lg[(b, i)], B, L, m0, s, e, x0, "robust", 0.9, eta=eta)
    nf, nfm = compare_selection(commit.cpu().numpy(), n.cpu().numpy(), r.commit, r.n_commit,
                                r.flagged, range(B))
    ok = ~r.flagged
    assert np.array_equal(xx.cpu().numpy()[ok], r.x[ok])
    assert np.array_equal(mk.cpu().numpy()[ok], r.mask[ok])
    say(f"  commits {int(n.clamp(min=0).sum())}, flagged {nf} (matching {nfm})")


@pytest.mark.parametrize("L,d", [(16, 512), (16, 4096), (16, 192), (30, 4096), (50, 2048)])
def test_lmhead_no_candidates(gpu, L, d):
    """No masked position inside any window: every output is the default."""
    B, V = 2, 700
    g = torch.Generator().manual_seed(d)
    hidden = torch.randn((B, L, d), generator=g).to(torch.bfloat16).cuda()
    weight = torch.randn((V, d), generator=g).to(torch.bfloat16).cuda()
    mask = torch.zeros((B, L), dtype=torch.uint8)
    mask[1, 10:] = 1                                   # masked, but outside the window
    start = torch.tensor([0, 2], dtype=torch.int32)
    end = torch.tensor([16, 8], dtype=torch.int32)
    say(f"[lmhead no candidates] L={L} d={d}")
    out = _gpu_conf(gpu, hidden, weight, mask.cuda(), start.cuda(), end.cuda())
    check_defaults(*[t.cpu().numpy() for t in out], mask.numpy(), start.numpy(), end.numpy(),
                   range(B))
    assert not candidates(mask.numpy(), start.numpy(), end.numpy(), range(B))


def test_lmhead_rejects_bad_shapes(gpu):
    hidden = torch.zeros((1, 4, 96), dtype=torch.bfloat16, device="cuda")     # d not a multiple of 64
    weight = torch.zeros((10, 96), dtype=torch.bfloat16, device="cuda")
    m = torch.ones((1, 4), dtype=torch.uint8, device="cuda")
    s = torch.zeros(1, dtype=torch.int32, device="cuda")
    e = torch.full((1,), 4, dtype=torch.int32, device="cuda")
    out = [torch.empty((1, 4), dtype=torch.int32, device="cuda"), torch.empty((1, 4), device="cuda")]
    with pytest.raises(gpu.FdllmError):
        gpu.fdllm_lmhead_confidence(hidden, weight, m, s, e, *out,
                                    workspace=torch.empty(1 << 20, dtype=torch.uint8, device="cuda"))
