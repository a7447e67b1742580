"""Block advance of the decoding loop (oracle; test infrastructure only).

Alg. 1 decodes the blocks of a sequence left to right: the model call and
the decode step repeat on the active block until none of its positions is
masked, then the next block becomes active.  A sequence moves to its first
block, from the current one on, that still has a masked position; when no
block is left the sequence is finished and gets the empty window [G, G).
"""
from __future__ import annotations

import numpy as np


def advance_blocks(mask: np.ndarray, start: np.ndarray, end: np.ndarray, G: int, blk: int) -> int:
    """Moves every sequence's window [start[b], end[b]) to its first block of
    blk positions, from the current one on, holding a masked position (the
    last block may be shorter); [G, G) when none is left.  Updates start and
    end in place and returns the number of sequences with an active block."""
    active = 0
    for b in range(mask.shape[0]):
        s = int(start[b])
        while s < G and not mask[b, s:min(s + blk, G)].any():
            s += blk
        if s >= G:
            start[b] = end[b] = G
        else:
            start[b], end[b] = s, min(s + blk, G)
            active += 1
    return active
