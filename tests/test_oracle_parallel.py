"""The process-parallel oracle driver returns exactly what the oracle's own
functions return (it adds no arithmetic): rows staged as raw bf16 bits or
float32 values, and selections split over workers."""
import numpy as np
import torch

import oracle
import workloads
from oracle.parallel import OraclePool, scatter_confidence
from parity import candidates, pool_confidence


def _ref(inp):
    B, L, V = inp.logits.shape
    return oracle.confidence(lambda b, i: inp.logits[b, i].to(torch.float64).numpy(), B, L,
                             inp.mask.numpy(), inp.start.numpy(), inp.end.numpy())


def test_pool_matches_oracle():
    with OraclePool(workers=2) as pool:
        for dt in (torch.bfloat16, torch.float32):
            inp = workloads.random_case(6, 40, 777, dt, device="cpu", seed=5, poison=False)
            mask, s, e = inp.mask.numpy(), inp.start.numpy(), inp.end.numpy()
            got = pool_confidence(pool, inp.logits, mask, s, e)
            want = _ref(inp)
            for g, w in zip(got, want):
                assert g.dtype == w.dtype and np.array_equal(g, w)
            # small chunks: several staging rounds
            cells = candidates(mask, s, e, range(6))
            flat = inp.logits.view(-1, 777)

            def fill(first, cnt, out):
                rows = flat[[b * 40 + i for b, i in cells[first:first + cnt]]]
                out[...] = (rows.view(torch.int16) if dt == torch.bfloat16 else rows).numpy()

            kind = "bf16" if dt == torch.bfloat16 else "f32"
            res = pool.rows_confidence(fill, len(cells), 777, kind, chunk_rows=7)
            for g, w in zip(scatter_confidence(6, 40, cells, res), want):
                assert np.array_equal(g, w)
            for rule, p in [("profile", 1.0), ("factor", 0.75), ("threshold", 0.9), ("robust", 1.0)]:
                eta = 0.01 if rule == "robust" else None
                c1, n1, f1 = pool.select(want[2], want[1], mask, s, e, rule, p, eta=eta, blocks_per_task=2)
                c2, n2, f2, _ = oracle.select(want[2], want[1], mask, s, e, rule, p, eta=eta)
                assert np.array_equal(c1, c2) and np.array_equal(n1, n2) and np.array_equal(f1, f2)
        assert pool.rows_done > 0 and pool.seconds > 0


def test_pool_empty_request():
    with OraclePool(workers=1) as pool:
        assert pool.rows_confidence(lambda *a: None, 0, 10, "bf16") == []
