"""The calibration step runs on the GPU: it times one attention layer's CP
step over a small grid of (C, R, P) and fits the prefill-time model's
attention term (paper Sec. 3.2, alpha W / C).  Only that the measurement
works is checked here -- every time finite and positive, a fit with a
positive slope.  The timing claims (the line explains the times, its slope
is a plausible kernel rate) depend on a quiet GPU and are checked by
``python -m paper_2609_04774_amd.calibrate --check``, not by this suite."""

import math

import pytest

from paper_2609_04774_amd import calibrate as cal

pytestmark = pytest.mark.gpu


def test_attention_calibration_runs():
    grid = [(C, R, P) for C in (1, 4) for R in (4096, 16384) for P in (0, 8192)]
    samples = cal.measure_attention(grid, n_heads_q=32, n_heads_kv=8, reps=2, warmup_seconds=0.2)
    assert [(C, R, P) for C, R, P, _ in samples] == grid
    for C, R, P, t in samples:
        print(f"C={C} R={R} P={P} W/C={cal.remaining_workload(R, P) / C:.3e} t={t * 1e3:.4f} ms")
        assert math.isfinite(t) and t > 0
    fit = cal.fit_attention_term(samples)
    print("alpha", fit.alpha, "d0", fit.d0, "r2", fit.r2)
    assert fit.alpha > 0
