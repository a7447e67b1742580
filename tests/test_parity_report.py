"""The markdown summary of a parity run (tests/parity.py render_report)."""
import os
import sys

sys.path.insert(0, os.path.dirname(os.path.abspath(__file__)))
import parity  # noqa: E402


def _rec(workload, checks, flagged, rows, **extra):
    return dict(workload=workload, block_checks=checks, mismatches=0, flagged=flagged,
                flagged_matching=flagged, rows=rows, worst=dict(conf=1.5e-7, eps=2e-7, lse=6e-8),
                rules={"profile(1.0)": dict(block_checks=checks, mismatches=0, flagged=flagged,
                                            flagged_matching=flagged)}, **extra)


def test_totals_order_and_notes():
    md = parity.render_report([
        _rec("stress_b1024_l32", 1024, 0, 32768),
        _rec("generation_b8_g256", 100, 2, 900, steps_per_generation={"profile(1.0)": 150}),
        _rec("single_block_b1_l32", 1, 0, 32),
    ])
    lines = md.splitlines()
    # workloads in the benchmark description's order, then the totals
    assert lines[2].startswith("| single_block_b1_l32 |")
    assert lines[3].startswith("| generation_b8_g256 |")
    assert lines[4].startswith("| stress_b1024_l32 |")
    assert lines[5] == "| **all** | | **1125** | **0** | 2 | 2 | 33700 | |"
    assert "1.5e-07 / 2.0e-07 / 6.0e-08" in lines[2]
    assert "generation_b8_g256 steps per whole generation (NFE): profile(1.0) 150." in md
