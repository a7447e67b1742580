"""Counter-based synthetic logits for device-resident generations.

The device-resident step loop produces every step's logits on the GPU, so
that no host work sits between steps.  This module implements the same
recipe on the CPU, from the generator's published definition, so that the
oracle's harness builds identical logits without reading anything the GPU
produced.  It draws random numbers and lays them out; none of the selector's
arithmetic is here.

Generator: Philox4x32-10 (Salmon, Moraes, Dror and Shaw, "Parallel random
numbers: as easy as 1, 2, 3", SC 2011).  A 128-bit counter (c0, c1, c2, c3)
and a 64-bit key (k0, k1) give four 32-bit words after ten rounds; a round
multiplies c0 by 0xD2511F53 and c2 by 0xCD9E8D57 (full 64-bit products) and
outputs (hi(c2*M1) ^ c1 ^ k0, lo(c2*M1), hi(c0*M0) ^ c3 ^ k1, lo(c0*M0)); the
key is bumped by (0x9E3779B9, 0xBB67AE85) between rounds.

Recipe of one generation (B sequences over a span of G positions, blocks of
blk positions, vocabulary V, 64-bit seed; key = (seed mod 2^32, seed >> 32)).
The logits of row (b, i) at step t, for vocabulary index v:
  * background: w = philox((v >> 2, i, b, t))[v & 3]; the sum of w's four
    bytes minus 510, times 2^-7 (exact in float32; sd 1.15, |bg| < 4);
  * spike token of (b, i), fixed across steps:
    philox((0xFFFFFFFF, i, b, 0xFFFFFFFF))[0] mod V;
  * spike height at step t: y = philox((0xFFFFFFFE, i, b, t)),
    u1 = (y[0] >> 8) 2^-24, u2 = (y[1] >> 8) 2^-24; h = 8 + 6 u2 when
    u1 < 0.6, else 6 u2 (a confident and an unconfident mode, as in the
    eight-sequence simulated generation); float32, every operation rounded
    to nearest, no fused multiply-add;
  * logit = bf16(bg + h) at the spike token and bf16(bg) elsewhere, bf16 by
    round-to-nearest-even of the float32 bits.
Only the rows of each sequence's active block are produced at a step.
"""
from __future__ import annotations

from typing import Sequence

import numpy as np

M0, M1 = np.uint64(0xD2511F53), np.uint64(0xCD9E8D57)
W0, W1 = 0x9E3779B9, 0xBB67AE85
MASK32 = np.uint64(0xFFFFFFFF)
SPIKE_TOKEN_C0 = 0xFFFFFFFF
SPIKE_TOKEN_C3 = 0xFFFFFFFF
SPIKE_HEIGHT_C0 = 0xFFFFFFFE


def philox4x32_10(c0, c1, c2, c3, k0: int, k1: int):
    """Philox4x32-10 on arrays of counters (broadcast); returns four uint32 arrays."""
    c = [np.asarray(v, dtype=np.uint64) & MASK32 for v in (c0, c1, c2, c3)]
    c = list(np.broadcast_arrays(*c))
    ka, kb = k0 & 0xFFFFFFFF, k1 & 0xFFFFFFFF
    for r in range(10):
        if r:
            ka = (ka + W0) & 0xFFFFFFFF
            kb = (kb + W1) & 0xFFFFFFFF
        p0 = M0 * c[0]
        p1 = M1 * c[2]
        c = [((p1 >> np.uint64(32)) ^ c[1] ^ np.uint64(ka)) & MASK32, p1 & MASK32,
             ((p0 >> np.uint64(32)) ^ c[3] ^ np.uint64(kb)) & MASK32, p0 & MASK32]
    return [v.astype(np.uint32) for v in c]


def key_of(seed: int):
    return seed & 0xFFFFFFFF, (seed >> 32) & 0xFFFFFFFF


def bf16_bits(x: np.ndarray) -> np.ndarray:
    """float32 -> bf16 bit patterns, round to nearest even (finite inputs)."""
    u = np.asarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    r = (u + np.uint64(0x7FFF) + ((u >> np.uint64(16)) & np.uint64(1))) >> np.uint64(16)
    return r.astype(np.uint16)


def bf16_to_f32(bits: np.ndarray) -> np.ndarray:
    return (np.asarray(bits, dtype=np.uint32) << np.uint32(16)).view(np.float32)


def spike_token(seed: int, b: int, i: int, V: int) -> int:
    k0, k1 = key_of(seed)
    return int(philox4x32_10(SPIKE_TOKEN_C0, i, b, SPIKE_TOKEN_C3, k0, k1)[0]) % V


def spike_height(seed: int, b: int, i: int, t: int) -> np.float32:
    k0, k1 = key_of(seed)
    y = philox4x32_10(SPIKE_HEIGHT_C0, i, b, t, k0, k1)
    u1 = np.float32(int(y[0]) >> 8) * np.float32(2.0 ** -24)
    u2 = np.float32(int(y[1]) >> 8) * np.float32(2.0 ** -24)
    six_u2 = np.float32(np.float32(6.0) * u2)
    return np.float32(np.float32(8.0) + six_u2) if u1 < np.float32(0.6) else six_u2


def row_bits(seed: int, b: int, i: int, t: int, V: int) -> np.ndarray:
    """bf16 bit patterns [V] of row (b, i) at step t."""
    k0, k1 = key_of(seed)
    v = np.arange(V, dtype=np.uint64)
    words = philox4x32_10(v >> np.uint64(2), i, b, t, k0, k1)
    sel = (v & np.uint64(3)).astype(np.int64)
    w = np.choose(sel, words).astype(np.uint32)
    bytesum = ((w & 0xFF) + ((w >> 8) & 0xFF) + ((w >> 16) & 0xFF) + (w >> 24)).astype(np.int32)
    bg = (bytesum - 510).astype(np.float32) * np.float32(2.0 ** -7)
    tok = spike_token(seed, b, i, V)
    bg[tok] = np.float32(bg[tok] + spike_height(seed, b, i, t))
    return bf16_bits(bg)


def row(seed: int, b: int, i: int, t: int, V: int) -> np.ndarray:
    """Row (b, i) at step t as float64 (exact values of the bf16 logits)."""
    return bf16_to_f32(row_bits(seed, b, i, t, V)).astype(np.float64)
