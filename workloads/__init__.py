"""Seeded synthetic inputs for the commit-selector hot path.

This module only draws random numbers and lays them out; it holds none of the
selector's arithmetic (no softmax, no argmax, no sorting, no prefix test).  Both
the HIP path's tests/benchmark and the CPU oracle's harness take their inputs
from here, so the two sides see the very same tensors.

The paper's workloads are model logits of LLaDA-8B on reasoning/code benchmarks
(Sec. 5, "Model and Hardware", "Benchmarks"); neither the model nor the
datasets are available, so these generators stand in for them.  They keep the
paper's decoding geometry: block size 32 (Table 1 caption), generation lengths
256/512/1024 (Table 2), greedy decoding at temperature 1 (Sec. 5), and the
operating points tau=0.9, f=0.75/1.0, delta=0.25 (Sec. 5, "Parameter
selection"; Table 5).  The vocabulary size V=126464 is LLaDA's.

Every draw comes from a ``torch.Generator`` seeded by ``seed_for(recipe,
step, b)``, so a sequence's logits at a step are reproducible on the same
device type.  CPU and GPU generators produce different streams: a parity
check always hands the oracle a host copy of the exact tensor the GPU read.

Layouts (all contiguous, row-major):
  logits  [B, L, V]  bfloat16 or float32
  mask    [B, L]     uint8, 1 = position still masked
  x       [B, L]     int32, sequence tokens; MASK_ID where masked
  start, end [B]     int32, the active block [start_b, end_b) of sequence b
"""
from __future__ import annotations

import dataclasses
import math
from typing import Callable, Optional

import torch

V_LLADA = 126464          # LLaDA-8B vocabulary
MASK_ID = -1              # token id stored in x for a still-masked position
BASE_SEED = 20260601      # recipe k draws from BASE_SEED + k

# the seed salts of the five benchmark recipes
SINGLE_BLOCK = 1          # B=1, one block of 32, fp32
GENERATION = 2            # B=8, generation of 256 in blocks of 32
SPARSE_BLOCKS = 3         # B=64, span 512, partly masked blocks of 32
BIMODAL_GENERATION = 4    # B=256, generation of 1024 in blocks of 64
STRESS = 5                # B=1024, L=32, all masked
RECIPE_NAMES = {SINGLE_BLOCK: "single_block_b1_l32", GENERATION: "generation_b8_g256",
                SPARSE_BLOCKS: "sparse_b64_g512", BIMODAL_GENERATION: "bimodal_b256_g1024",
                STRESS: "stress_b1024_l32"}
BF16_NAN = 0x7FC0         # poison for logits rows that must never be read


def seed_for(recipe: int, step: int, b: int) -> int:
    """Deterministic 63-bit seed for (recipe, step, sequence)."""
    h = (BASE_SEED + recipe) * 0x9E3779B97F4A7C15
    h ^= (step + 1) * 0xBF58476D1CE4E5B9
    h ^= (b + 1) * 0x94D049BB133111EB
    h &= (1 << 64) - 1
    h ^= h >> 31
    return h & ((1 << 63) - 1)


def _gen(recipe: int, step: int, b: int, device) -> torch.Generator:
    g = torch.Generator(device=device)
    g.manual_seed(seed_for(recipe, step, b))
    return g


def _uniform(g, shape, lo, hi, device):
    return torch.rand(shape, generator=g, device=device, dtype=torch.float32) * (hi - lo) + lo


def _gumbel(g, shape, device):
    u = torch.rand(shape, generator=g, device=device, dtype=torch.float32)
    u = u.clamp_(min=1e-30, max=1.0 - 2.0 ** -24)
    return -torch.log(-torch.log(u))


def _distinct_tokens(g, n_rows, k, V, device):
    """k distinct random token ids per row (rejection-free: offsets mod V)."""
    first = torch.randint(0, V, (n_rows, 1), generator=g, device=device)
    if k == 1:
        return first
    steps = torch.randint(1, max(2, V // k), (n_rows, k - 1), generator=g, device=device)
    return (first + torch.cat([torch.zeros_like(first), steps.cumsum(1)], 1)) % V


def _put(rows: torch.Tensor, toks: torch.Tensor, vals: torch.Tensor, add: bool):
    """rows[r, toks[r, j]] (+)= vals[r, j]."""
    if add:
        rows.scatter_add_(1, toks, vals.to(rows.dtype))
    else:
        rows.scatter_(1, toks, vals.to(rows.dtype))


@dataclasses.dataclass
class StepInputs:
    """One decode step's inputs; tensors live on one device."""
    logits: torch.Tensor      # [B, L, V]
    mask: torch.Tensor        # [B, L] uint8
    start: torch.Tensor       # [B] int32
    end: torch.Tensor         # [B] int32
    x: torch.Tensor           # [B, L] int32
    name: str
    notes: str = ""

    @property
    def B(self):
        return self.logits.shape[0]

    @property
    def L(self):
        return self.logits.shape[1]

    @property
    def V(self):
        return self.logits.shape[2]


# ---------------------------------------------------------------------------
# single block: B=1, one block of 32 all-masked positions, fp32, N(0,1)+U(0,12)
# spike; 4 positions get a second spike (2 exact ties, 2 gaps in [1e-6,1e-3]).
# ---------------------------------------------------------------------------
def single_block_b1_l32(device="cpu", V: int = V_LLADA, L: int = 32) -> StepInputs:
    g = _gen(SINGLE_BLOCK, 0, 0, device)
    rows = torch.randn((L, V), generator=g, device=device, dtype=torch.float32)
    tok = _distinct_tokens(g, L, 2, V, device)
    h = _uniform(g, (L, 1), 0.0, 12.0, device)
    _put(rows, tok[:, :1], h, add=True)
    # four positions with a second, (near-)tied spike; their first spike is
    # drawn from U(8,12) so that it stands above the N(0,1) background
    special = torch.randperm(L, generator=g, device=device)[:4]
    gaps = _uniform(g, (4,), 1e-6, 1e-3, device)
    hs = _uniform(g, (4,), 8.0, 12.0, device)
    for j in range(4):
        r = int(special[j])
        top = rows[r, tok[r, 0]] - h[r, 0] + hs[j]
        rows[r, tok[r, 0]] = top
        rows[r, tok[r, 1]] = top if j < 2 else top - gaps[j]
    logits = rows.view(1, L, V)
    mask = torch.ones((1, L), dtype=torch.uint8, device=device)
    start = torch.zeros((1,), dtype=torch.int32, device=device)
    end = torch.full((1,), L, dtype=torch.int32, device=device)
    x = torch.full((1, L), MASK_ID, dtype=torch.int32, device=device)
    return StepInputs(logits, mask, start, end, x, "single_block_b1_l32",
                      "B=1 L=32 fp32 N(0,1)+U(0,12) spike, 2 exact ties + 2 near ties")


# ---------------------------------------------------------------------------
# generations (B=8 of 256, B=256 of 1024): full simulated generations.  The whole generation span
# is one logits tensor [B, G, V] ("no-cache" layout); each step fills only the
# rows of every sequence's active block, which start/end select.
# ---------------------------------------------------------------------------
@dataclasses.dataclass
class Generation:
    recipe: int
    B: int
    G: int                    # generation length
    blk: int                  # block size
    V: int
    dtype: torch.dtype
    fill_rows: Callable       # (rows [n,V] fp32 out, b, step, positions, g, device) -> None

    @property
    def n_blocks(self):
        return self.G // self.blk


def _c2_fill(rows, b, step, pos, gen_tok, g, device):
    n, V = rows.shape
    rows.normal_(generator=g)
    conf = torch.rand((n,), generator=g, device=device) < 0.6
    h = torch.where(conf, _uniform(g, (n,), 8.0, 14.0, device), _uniform(g, (n,), 0.0, 6.0, device))
    _put(rows, gen_tok[pos].view(n, 1), h.view(n, 1), add=True)


def _c4_fill(rows, b, step, pos, gen_tok, g, device, flat: bool, temp: float):
    n, V = rows.shape
    if flat:
        # one row repeated over the whole block: a flat confidence profile.
        # Spike heights U(14.5,19) over an N(0,1) background put the greedy
        # probability roughly in (0.9, 0.999) at V=126464.
        one = torch.randn((1, V), generator=g, device=device)
        hh = _uniform(g, (1, 1), 14.5, 19.0, device)
        _put(one, gen_tok[pos[:1]].view(1, 1), hh, add=True)
        rows.copy_(one.expand(n, V))
        return
    rows.normal_(generator=g)
    u = torch.rand((n,), generator=g, device=device)
    beta = torch.sin(0.5 * math.pi * u) ** 2          # Beta(1/2, 1/2)
    _put(rows, gen_tok[pos].view(n, 1), (14.0 * beta).view(n, 1), add=True)
    rows.div_(temp)


class SimulatedGeneration:
    """Host-side state of a semi-autoregressive generation (Alg. 1 outer loops).

    Holds x/mask over the whole generation span and, per step, fills the
    logits rows of each sequence's active block (the first block that still
    has a masked position).  Selection itself is not done here.
    """

    def __init__(self, recipe: int, device="cpu", B=None, V: int = V_LLADA):
        if recipe == GENERATION:
            self.B, self.G, self.blk = (B or 8), 256, 32
        elif recipe == BIMODAL_GENERATION:
            self.B, self.G, self.blk = (B or 256), 1024, 64
        else:
            raise ValueError("simulated generations are GENERATION and BIMODAL_GENERATION")
        self.recipe, self.V, self.device = recipe, V, device
        self.dtype = torch.bfloat16
        g = _gen(recipe, 0, 10_000, device)
        # per-(sequence, position) spike token, fixed for the whole generation
        self.tok = torch.randint(0, V, (self.B, self.G), generator=g, device=device)
        if recipe == BIMODAL_GENERATION:
            self.temp = _uniform(g, (self.B,), 0.5, 2.0, device).tolist()
            self.flat = torch.zeros(self.B, dtype=torch.bool)
            self.flat[torch.randperm(self.B, generator=torch.Generator().manual_seed(seed_for(BIMODAL_GENERATION, 0, 0)))[:16 * self.B // 256 or 1]] = True
            for b in range(self.B):
                if self.flat[b]:
                    self.temp[b] = 1.0
        self.x = torch.full((self.B, self.G), MASK_ID, dtype=torch.int32, device=device)
        self.mask = torch.ones((self.B, self.G), dtype=torch.uint8, device=device)
        self.logits = torch.empty((self.B, self.G, V), dtype=self.dtype, device=device)
        self.start = torch.zeros((self.B,), dtype=torch.int32, device=device)
        self.end = torch.zeros((self.B,), dtype=torch.int32, device=device)
        self.step_no = 0

    def active_blocks(self):
        """Per sequence, the first block with a masked position (-1 when done)."""
        m = self.mask.view(self.B, self.G // self.blk, self.blk).any(dim=2).to("cpu")
        out = []
        for b in range(self.B):
            nz = torch.nonzero(m[b]).flatten()
            out.append(int(nz[0]) if nz.numel() else -1)
        return out

    def done(self) -> bool:
        return not bool(self.mask.any())

    def prepare_step(self) -> StepInputs:
        """Fill the active rows' logits and set start/end; returns the inputs."""
        blocks = self.active_blocks()
        s = torch.zeros(self.B, dtype=torch.int32)
        e = torch.zeros(self.B, dtype=torch.int32)
        for b, k in enumerate(blocks):
            if k < 0:
                continue                      # finished: empty window
            lo, hi = k * self.blk, (k + 1) * self.blk
            s[b], e[b] = lo, hi
            g = _gen(self.recipe, self.step_no, b, self.device)
            rows = torch.empty((self.blk, self.V), dtype=torch.float32, device=self.device)
            pos = torch.arange(lo, hi, device=self.device)
            if self.recipe == GENERATION:
                _c2_fill(rows, b, self.step_no, pos, self.tok[b], g, self.device)
            else:
                _c4_fill(rows, b, self.step_no, pos, self.tok[b], g, self.device,
                         bool(self.flat[b]), float(self.temp[b]))
            self.logits[b, lo:hi].copy_(rows.to(self.dtype))
        self.start.copy_(s)
        self.end.copy_(e)
        self.step_no += 1
        return StepInputs(self.logits, self.mask, self.start, self.end, self.x,
                          f"{RECIPE_NAMES[self.recipe]}-step{self.step_no - 1}")


# ---------------------------------------------------------------------------
# sparse blocks: B=64, gen 512 in blocks of 32, no-cache layout [64,512,V] bf16;
# sequence b is at a seeded block k_b with m_b ~ U{1..32} masked positions.
# Background N(0, sd=2) plus Zipf(1.1)-ranked spikes on 5 tokens.
# ---------------------------------------------------------------------------
def sparse_b64_g512(device="cpu", V: int = V_LLADA, B: int = 64, G: int = 512, blk: int = 32,
            poison: bool = True) -> StepInputs:
    g0 = _gen(SPARSE_BLOCKS, 0, 10_000, device)
    k = torch.randint(0, G // blk, (B,), generator=g0, device="cpu" if device == "cpu" else device).cpu()
    m = torch.randint(1, blk + 1, (B,), generator=g0, device="cpu" if device == "cpu" else device).cpu()
    logits = torch.empty((B, G, V), dtype=torch.bfloat16, device=device)
    if poison:
        logits.view(torch.int16).fill_(BF16_NAN)
    mask = torch.zeros((B, G), dtype=torch.uint8, device=device)
    x = torch.randint(0, V, (B, G), generator=g0, device=device).to(torch.int32)
    ranks = torch.arange(1, 6, device=device, dtype=torch.float32)
    for b in range(B):
        g = _gen(SPARSE_BLOCKS, 0, b, device)
        lo = int(k[b]) * blk
        sel = torch.randperm(blk, generator=g, device=device)[: int(m[b])] + lo
        mask[b, sel] = 1
        x[b, sel] = MASK_ID
        n = sel.numel()
        rows = torch.randn((n, V), generator=g, device=device) * 2.0
        H = _uniform(g, (n, 1), 8.0, 20.0, device)
        toks = _distinct_tokens(g, n, 5, V, device)
        _put(rows, toks, H * ranks.pow(-1.1).view(1, 5), add=True)
        logits[b, sel] = rows.to(torch.bfloat16)
    start = (k * blk).to(torch.int32).to(device)
    end = ((k + 1) * blk).to(torch.int32).to(device)
    return StepInputs(logits, mask, start, end, x, "sparse_b64_g512",
                      "B=64 no-cache [64,512,V] bf16, m_b~U{1..32}, N(0,2)+Zipf(1.1) top-5 spikes")


# ---------------------------------------------------------------------------
# throughput stress: B=1024, L=32, all masked, bf16 Gumbel(0,1)
# background; 10% of positions carry a planted pair with gap U(0,1e-3).
# ---------------------------------------------------------------------------
def stress_b1024_l32_rows(b: int, device="cpu", V: int = V_LLADA, L: int = 32) -> torch.Tensor:
    """The [L, V] bf16 logits of sequence b (its own seeded stream per device)."""
    g = _gen(STRESS, 0, b, device)
    rows = _gumbel(g, (L, V), device)
    tie = torch.rand((L,), generator=g, device=device) < 0.10
    toks = _distinct_tokens(g, L, 2, V, device)
    H = _uniform(g, (L, 1), 13.0, 17.0, device)
    gap = _uniform(g, (L, 1), 0.0, 1e-3, device)
    idx = torch.nonzero(tie).flatten()
    if idx.numel():
        pair = torch.cat([H[idx], H[idx] - gap[idx]], 1)
        rows[idx] = rows[idx].scatter(1, toks[idx], pair)
    return rows.to(torch.bfloat16)


def stress_b1024_l32(device="cpu", V: int = V_LLADA, B: int = 1024, L: int = 32,
            chunk: int = 32, progress: Optional[Callable[[str], None]] = None) -> StepInputs:
    logits = torch.empty((B, L, V), dtype=torch.bfloat16, device=device)
    for b0 in range(0, B, chunk):
        if progress is not None and b0 % 256 == 0:
            progress(f"stress inputs: sequences {b0}..{min(B, b0 + 256) - 1}")
        for b in range(b0, min(B, b0 + chunk)):
            logits[b] = stress_b1024_l32_rows(b, device, V, L)
    mask = torch.ones((B, L), dtype=torch.uint8, device=device)
    start = torch.zeros((B,), dtype=torch.int32, device=device)
    end = torch.full((B,), L, dtype=torch.int32, device=device)
    x = torch.full((B, L), MASK_ID, dtype=torch.int32, device=device)
    return StepInputs(logits, mask, start, end, x, "stress_b1024_l32",
                      "B=1024 L=32 bf16 Gumbel(0,1), 10% planted near-ties gap<1e-3")


# ---------------------------------------------------------------------------
# small generic cases for parity tests: any (B, L, V, dtype), a random window
# and a random mask inside it, N(0, sd) + one spike per row.
# ---------------------------------------------------------------------------
def random_case(B: int, L: int, V: int, dtype=torch.bfloat16, device="cpu", seed: int = 0,
                window: Optional[int] = None, p_mask: float = 0.7, sd: float = 1.0,
                spike_hi: float = 14.0, ties: float = 0.1, poison: bool = True) -> StepInputs:
    """A generic seeded case: per-sequence window of <= window rows, random mask.

    A fraction `ties` of rows get a second token equal to the first spike's
    value (an exact tie in the row's dtype).
    """
    g = torch.Generator(device=device)
    g.manual_seed(seed_for(100 + seed % 1000, seed // 1000, 0))
    window = min(L, 64) if window is None else window
    lens = torch.randint(0, window + 1, (B,), generator=g, device=device).cpu()
    starts = []
    for b in range(B):
        starts.append(int(torch.randint(0, L - int(lens[b]) + 1, (1,), generator=g, device=device)))
    start = torch.tensor(starts, dtype=torch.int32)
    end = start + lens.to(torch.int32)
    mask = (torch.rand((B, L), generator=g, device=device) < p_mask).to(torch.uint8)
    rows = torch.randn((B * L, V), generator=g, device=device) * sd
    toks = _distinct_tokens(g, B * L, 2, V, device)
    h = _uniform(g, (B * L, 1), 0.0, spike_hi, device)
    _put(rows, toks[:, :1], h, add=True)
    tie = torch.nonzero(torch.rand((B * L,), generator=g, device=device) < ties).flatten()
    if tie.numel() and V > 1:
        top = rows[tie].gather(1, toks[tie, :1])
        rows[tie] = rows[tie].scatter(1, toks[tie, 1:2], top)
    logits = rows.view(B, L, V).to(dtype)
    if poison and dtype == torch.bfloat16:
        # rows outside the window or unmasked are never read by the selector
        inwin = torch.zeros((B, L), dtype=torch.bool)
        for b in range(B):
            inwin[b, int(start[b]):int(end[b])] = True
        dead = ~(inwin.to(device) & mask.bool())
        logits.view(torch.int16)[dead] = BF16_NAN
    x = torch.where(mask.bool(), torch.full((B, L), MASK_ID, device=device),
                    torch.randint(0, V, (B, L), generator=g, device=device)).to(torch.int32)
    return StepInputs(logits, mask, start.to(device), end.to(device), x,
                      f"random(B={B},L={L},V={V},{str(dtype).split('.')[-1]},seed={seed})")


RECIPES = {
    SINGLE_BLOCK: dict(B=1, L=32, V=V_LLADA, dtype="f32", selectors=["profile", "factor", "threshold"],
            params=dict(profile=[1.0], factor=[1.0], threshold=[0.9])),
    GENERATION: dict(B=8, L=256, V=V_LLADA, dtype="bf16", block=32,
            selectors=["profile", "factor", "threshold"],
            params=dict(profile=[0.5, 1.0, 2.0], factor=[0.5, 1.0, 2.0], threshold=[0.9])),
    SPARSE_BLOCKS: dict(B=64, L=512, V=V_LLADA, dtype="bf16", block=32,
            selectors=["profile", "factor", "threshold"],
            params=dict(profile=[1.0, 0.75], factor=[1.0, 0.75], threshold=[0.9])),
    BIMODAL_GENERATION: dict(B=256, L=1024, V=V_LLADA, dtype="bf16", block=64,
            selectors=["profile", "factor", "threshold"],
            params=dict(profile=[0.75, 1.0], factor=[0.75, 1.0], threshold=[0.9])),
    STRESS: dict(B=1024, L=32, V=V_LLADA, dtype="bf16", selectors=["profile", "factor", "threshold"],
            params=dict(profile=[1.0, 0.75], factor=[1.0, 0.75], threshold=[0.9])),
}


# ---------------------------------------------------------------------------
# LM-head inputs: hidden states [B, L, d] and an output embedding [V, d], both
# bf16, for the fused LM head + vocabulary pass.  Two recipes:
#   exact:  W entries in {-3..3}/4; a candidate row aimed at token t has
#           h = (s * W[t] + 4 r) / 4 * 2^(q-7) with r in {-3..3}/4, a per-row
#           strength s in {0..16} and q = round(log2(4096/d)).  Up to the
#           power of two, every product is a multiple of 2^-11 and every
#           partial sum stays below 2^20 of those units, so the logits are
#           exact in float32 whatever the order of accumulation.  Some rows
#           aim at token pairs with identical W rows (exact ties).
#   random: W ~ N(0, 1/d), h = a W[t] / |W[t]|^2 + N(0, 1) with a ~ U(0, 24)
#           (a spike of height a over a unit-variance background), general
#           bf16 values (results compared within rounding bounds).
# ---------------------------------------------------------------------------
def lmhead_case(B: int, L: int, d: int, V: int, kind: str = "exact", device="cpu", seed: int = 0,
                window: Optional[int] = None, p_mask: float = 0.8, tie_pairs: int = 4):
    g = torch.Generator(device="cpu")
    g.manual_seed(seed_for(200 + seed % 1000, seed // 1000, 0))
    window = min(L, 64) if window is None else window
    lens = torch.randint(0, window + 1, (B,), generator=g)
    start = torch.tensor([int(torch.randint(0, L - int(lens[b]) + 1, (1,), generator=g)) for b in range(B)],
                         dtype=torch.int32)
    end = start + lens.to(torch.int32)
    mask = (torch.rand((B, L), generator=g) < p_mask).to(torch.uint8)
    target = torch.randint(0, V, (B, L), generator=g)
    if kind == "exact":
        w = torch.randint(-3, 4, (V, d), generator=g).float() / 4
        # tie pairs: W[t2] = W[t1], some rows aimed at t1 or t2
        pairs = torch.randint(0, V, (tie_pairs, 2), generator=g)
        for t1, t2 in pairs.tolist():
            if t1 != t2:
                w[max(t1, t2)] = w[min(t1, t2)]
        flat = target.view(-1)
        aim = torch.rand(flat.shape, generator=g) < 0.1
        flat[aim] = pairs[torch.randint(0, tie_pairs, (int(aim.sum()),), generator=g),
                          torch.randint(0, 2, (int(aim.sum()),), generator=g)]
        s = torch.randint(0, 17, (B, L, 1), generator=g).float()
        r = torch.randint(-3, 4, (B, L, d), generator=g).float() / 4
        # a power of two keeps every value exact and the spike's logit near 2 s for any d
        scale = 2.0 ** (round(math.log2(4096 / d)) - 7)
        h = (s * w[target] + 4 * r) / 4 * scale
    elif kind == "random":
        w = torch.randn((V, d), generator=g) / math.sqrt(d)
        a = torch.rand((B, L, 1), generator=g) * 24.0
        wt = w[target]
        h = a * wt / (wt * wt).sum(-1, keepdim=True) + torch.randn((B, L, d), generator=g)
    else:
        raise ValueError(f"unknown LM-head recipe {kind!r}")
    hidden = h.to(torch.bfloat16).to(device)
    weight = w.to(torch.bfloat16).to(device)
    x = torch.full((B, L), MASK_ID, dtype=torch.int32)
    return (hidden, weight, mask.to(device), start.to(device), end.to(device), x.to(device),
            f"lmhead-{kind}(B={B},L={L},d={d},V={V},seed={seed})")
