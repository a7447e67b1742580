"""Process-parallel driver of the oracle (test infrastructure only).

The oracle's per-position confidence (``position_confidence``) is plain
float64 NumPy plus ``math.fsum`` and takes a few milliseconds per row of
126464 logits; checking whole workloads (tens of thousands of rows per step)
needs many host cores.  This module only distributes the oracle's own
functions over worker processes: it adds no arithmetic of the method.

Rows travel through a staging file mapped by every process (``/dev/shm`` when
it has room, else the temporary directory): the caller fills the staging array
with the raw logits bits of a chunk of rows, and the workers read them from
there, so no logits pass through pipes.  Raw bits are converted to float64
exactly (bf16 -> float32 by a 16-bit shift, float32 -> float64 by NumPy).

Workers are spawned, never forked, and each imports only NumPy and this
package.  A caller that touches a GPU must create the pool before it
initialises the GPU runtime (a spawn from a process holding GPU state is not
allowed on every platform).
"""
from __future__ import annotations

import multiprocessing as mp
import os
import tempfile
import time
import uuid
from typing import Callable, List, Optional, Sequence, Tuple

import numpy as np

from .confidence import position_confidence
from .rules import select

KINDS = {"bf16": np.int16, "f32": np.float32}

_maps = {}   # worker side: (path, kind, rows, V) -> memmap


def _stage_map(path: str, kind: str, rows: int, V: int, mode: str = "r") -> np.memmap:
    return np.memmap(path, dtype=KINDS[kind], mode=mode, shape=(rows, V))


def _row_values(raw: np.ndarray, kind: str) -> np.ndarray:
    if kind == "bf16":
        return (raw.view(np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)
    return raw


def _conf_task(path: str, kind: str, rows: int, V: int, lo: int, hi: int):
    key = (path, kind, rows, V)
    mm = _maps.get(key)
    if mm is None:
        _maps.clear()
        mm = _maps[key] = _stage_map(path, kind, rows, V)
    return [position_confidence(_row_values(np.asarray(mm[k]), kind)) for k in range(lo, hi)]


def _select_task(eps, conf, mask, start, end, rule, param, eta):
    commit, n_commit, flagged, _ = select(eps, conf, mask, start, end, rule, param, eta=eta)
    return commit, n_commit, flagged


def _noop(_=None):
    return os.getpid()


def default_workers(cap: int = 16) -> int:
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:
        n = os.cpu_count() or 1
    return max(1, min(cap, n))


def _stage_dir(nbytes: int) -> str:
    for d in ("/dev/shm", tempfile.gettempdir()):
        try:
            st = os.statvfs(d)
            if st.f_bavail * st.f_frsize > nbytes + (512 << 20):
                return d
        except OSError:
            continue
    raise RuntimeError(f"no room for a {nbytes >> 20} MiB oracle staging file")


class OraclePool:
    """A pool of spawned processes that run the oracle on staged logits rows.

    ``stage_rows`` x ``V`` raw values are staged at a time; larger requests
    run in chunks.  ``seconds`` accumulates the time spent inside the
    workers' oracle calls (wall clock of the parallel sections, staging
    copies excluded).
    """

    def __init__(self, workers: Optional[int] = None):
        self.workers = workers or default_workers()
        self._pool = mp.get_context("spawn").Pool(self.workers)
        # make sure every worker has started and imported the oracle
        self._pool.map(_noop, range(self.workers), chunksize=1)
        self._stage = None            # (path, kind, rows, V, memmap)
        self.seconds = 0.0
        self.rows_done = 0

    # ------------------------------------------------------------------ staging
    def _staging(self, kind: str, rows: int, V: int) -> Tuple[str, np.memmap]:
        s = self._stage
        if s is not None and s[1] == kind and s[2] >= rows and s[3] == V:
            return s[0], s[4]
        self._drop_stage()
        nbytes = rows * V * np.dtype(KINDS[kind]).itemsize
        path = os.path.join(_stage_dir(nbytes), f"fdllm-oracle-{os.getpid()}-{uuid.uuid4().hex}.bin")
        mm = _stage_map(path, kind, rows, V, mode="w+")
        self._stage = (path, kind, rows, V, mm)
        return path, mm

    def _drop_stage(self):
        if self._stage is not None:
            path = self._stage[0]
            self._stage = None
            try:
                os.unlink(path)
            except OSError:
                pass

    # ------------------------------------------------------------------ oracle
    def rows_confidence(self, fill: Callable[[int, int, np.ndarray], None], n: int, V: int,
                        kind: str, chunk_rows: int = 2048) -> List[tuple]:
        """(t, c, eps, lse) of n rows.  ``fill(first, count, out)`` writes the
        raw values (int16 bf16 bits, or float32) of rows first..first+count-1
        into ``out`` [count, V]."""
        if kind not in KINDS:
            raise ValueError(f"unknown logits kind {kind!r}")
        out: List[tuple] = []
        if n == 0:
            return out
        rows = min(n, chunk_rows)
        path, mm = self._staging(kind, rows, V)
        stage_rows = self._stage[2]
        for first in range(0, n, rows):
            cnt = min(rows, n - first)
            fill(first, cnt, mm[:cnt])
            mm.flush()
            per = max(1, -(-cnt // (4 * self.workers)))
            tasks = [(path, kind, stage_rows, V, lo, min(cnt, lo + per)) for lo in range(0, cnt, per)]
            t0 = time.perf_counter()
            for part in self._pool.starmap(_conf_task, tasks):
                out.extend(part)
            self.seconds += time.perf_counter() - t0
            self.rows_done += cnt
        return out

    def select_many(self, eps, conf, mask, start, end, rules: Sequence[tuple],
                    blocks: Optional[Sequence[int]] = None, blocks_per_task: int = 16):
        """oracle.select for several (rule, param, eta) on one batch, the blocks
        of every rule spread over the workers in one round.  Only the blocks
        in ``blocks`` (all when None) are decided; the others get no commits.
        Returns one (commit [B,L] uint8, n_commit [B] int64, flagged [B] bool)
        per rule."""
        eps, conf, mask = np.asarray(eps), np.asarray(conf), np.asarray(mask)
        start, end = np.asarray(start), np.asarray(end)
        B, L = mask.shape
        bl = np.arange(B) if blocks is None else np.asarray(sorted(blocks), dtype=np.int64)
        tasks, where = [], []
        for k, (rule, param, eta) in enumerate(rules):
            eta_arr = None if eta is None else np.broadcast_to(np.asarray(eta, dtype=np.float64),
                                                               mask.shape)
            for j in range(0, len(bl), blocks_per_task):
                sel = bl[j:j + blocks_per_task]
                tasks.append((eps[sel], conf[sel], mask[sel], start[sel], end[sel], rule, param,
                              None if eta_arr is None else np.ascontiguousarray(eta_arr[sel])))
                where.append((k, sel))
        t0 = time.perf_counter()
        parts = self._pool.starmap(_select_task, tasks) if tasks else []
        self.seconds += time.perf_counter() - t0
        out = [(np.zeros((B, L), np.uint8), np.zeros((B,), np.int64), np.zeros((B,), bool))
               for _ in rules]
        for (k, sel), (c, n, f) in zip(where, parts):
            out[k][0][sel], out[k][1][sel], out[k][2][sel] = c, n, f
        return out

    def select(self, eps, conf, mask, start, end, rule: str, param: float, eta=None,
               blocks_per_task: int = 16):
        """oracle.select over a batch, blocks spread over the workers.
        Returns (commit [B,L] uint8, n_commit [B] int64, flagged [B] bool)."""
        return self.select_many(eps, conf, mask, start, end, [(rule, param, eta)],
                                blocks_per_task=blocks_per_task)[0]

    def close(self):
        self._drop_stage()
        if self._pool is not None:
            self._pool.close()
            self._pool.join()
            self._pool = None

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()


def scatter_confidence(B: int, L: int, cells: Sequence[Tuple[int, int]], results: Sequence[tuple]):
    """Arrays [B, L] from per-cell oracle results; defaults elsewhere (token -1,
    c = 0, eps = 1, lse = 0, as ``oracle.confidence`` leaves them)."""
    tokens = np.full((B, L), -1, dtype=np.int64)
    conf = np.zeros((B, L), dtype=np.float64)
    eps = np.ones((B, L), dtype=np.float64)
    lse = np.zeros((B, L), dtype=np.float64)
    for (b, i), (t, c, e, s) in zip(cells, results):
        tokens[b, i], conf[b, i], eps[b, i], lse[b, i] = t, c, e, s
    return tokens, conf, eps, lse
