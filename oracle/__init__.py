"""CPU oracle for the Fast-dLLM++ commit selector (arXiv 2606.02955).

TEST INFRASTRUCTURE ONLY.  This package is a plain, slow and obviously correct
CPU restatement of what one decoding step of the paper's method computes:

  * per masked position of the active block, the greedy token, its softmax
    confidence, the complement 1 - c and the log-sum-exp of the logits
    (Sec. 3 "Notation"; Alg. 1, the per-position loop);
  * per block, the commit set chosen by the Frechet profile rule (Sec. 3,
    "Frechet profile quantities"; Alg. 1 selection), by its calibration-robust
    variant (appendix "Calibration-Robust Frechet Certificates"), by
    Fast-dLLM's factor rule and by the threshold rule (Sec. 2,
    "Confidence-Aware Parallel Decoding"; Sec. 5, "Baselines");
  * the reveal of the chosen tokens (Alg. 1, reveal step), and the move of
    a finished block's window to the next block (Alg. 1, outer loop);
  * for the LM-head form, the logits as float64 dot products of hidden
    states with the output embedding (``lmhead``).

It shares no code with the HIP library and imports nothing from it.  Only the
tests, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import it; the product path never does.

Precision: the vocabulary pass is done in float64 on the exact float64 value
of every logit (bf16 and fp32 inputs convert exactly); the sum of the
non-greedy softmax terms uses ``math.fsum`` (correctly rounded).  Selection
is decided in exact rational arithmetic (``fractions.Fraction``) on the float64
confidence values, so ties and strict inequalities are decided exactly.

Every function is pinned by the CPU tests (``-m "not gpu"``) against closed
forms, library routines, brute force on tiny inputs and the paper's
propositions; see the docstrings for which passage each one follows.
"""
from .confidence import position_confidence, confidence
from .rules import (sorted_order, factor_n_star, profile_n_star, profile_literal_n_star,
                     profile_adaptive_n_star, threshold_set, select_block, select, SelectResult,
                     frechet_quantities, robust_eps, FLAG_WINDOW)
from .step import decode_step, StepResult
from .loop import advance_blocks
from . import lmhead

__all__ = [
    "position_confidence", "confidence", "sorted_order", "factor_n_star", "profile_n_star",
    "profile_literal_n_star", "profile_adaptive_n_star", "threshold_set", "select_block",
    "select", "SelectResult", "frechet_quantities", "robust_eps", "FLAG_WINDOW", "decode_step", "StepResult",
    "advance_blocks", "lmhead",
]
