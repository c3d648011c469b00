"""Host checks of the prefill-time model fits (paper Sec. 3.2) on synthetic
timings generated from known coefficients, plus the workload W(R, P)
against the oracle's (pinned) definition."""

import numpy as np
import pytest

from oracle import plan as oplan
from paper_2609_04774_amd import calibrate as cal

GRID = [(C, R, P) for C in (1, 2, 4, 8) for R in (512, 3000, 8192) for P in (0, 4096, 16384)]


def test_workload_matches_the_oracle():
    for R, P in [(1, 0), (7, 3), (32768, 0), (16384, 49152), (300, 17)]:
        assert cal.remaining_workload(R, P) == oplan.remaining_workload(R, P)


def test_attention_term_recovered_exactly():
    d0, alpha = 12e-6, 1.7e-13
    samples = [(C, R, P, d0 + alpha * cal.remaining_workload(R, P) / C) for C, R, P in GRID]
    fit = cal.fit_attention_term(samples)
    assert abs(fit.d0 - d0) <= 1e-12 and abs(fit.alpha - alpha) / alpha <= 1e-9
    assert fit.r2 > 1 - 1e-12 and fit.max_rel_err < 1e-9
    assert abs(fit.predict(4, 1000, 0) - (d0 + alpha * 500500 / 4)) < 1e-15


def test_attention_term_with_noise():
    rng = np.random.default_rng(1)
    d0, alpha = 20e-6, 2.0e-13
    samples = [(C, R, P, (d0 + alpha * cal.remaining_workload(R, P) / C) * (1 + 0.01 * rng.standard_normal()))
               for C, R, P in GRID]
    fit = cal.fit_attention_term(samples)
    assert abs(fit.alpha - alpha) / alpha < 0.03
    assert fit.r2 > 0.99


def test_full_prefill_model_recovered_exactly():
    coef = dict(d=3e-3, a=2e-7, b=4e-8, c=9e-6, alpha=1.1e-12)
    samples = [(C, R, P, coef["d"] + coef["a"] * R + coef["b"] * P
                + (coef["c"] * R + coef["alpha"] * cal.remaining_workload(R, P)) / C) for C, R, P in GRID]
    fit = cal.fit_prefill_model(samples)
    for k, v in coef.items():
        assert abs(getattr(fit, k) - v) <= 1e-6 * abs(v) + 1e-15, k
    assert fit.max_rel_err < 1e-9


def test_degenerate_grids_are_rejected():
    with pytest.raises(ValueError):
        cal.fit_attention_term([(1, 100, 0, 1.0)])
    with pytest.raises(ValueError):
        cal.fit_attention_term([(1, 100, 0, 1.0), (1, 100, 0, 1.1)])
    # One degree only: R and R / C are collinear, so a and c cannot be told apart.
    with pytest.raises(ValueError):
        cal.fit_prefill_model([(1, R, P, 1.0) for _, R, P in GRID])


def test_linearity_check_flags_what_it_claims():
    d0, alpha = 50e-6, 1.5e-11
    flop = 4 * 128 * 32
    good = [(C, R, P, d0 + alpha * cal.remaining_workload(R, P) / C) for C, R, P in GRID]
    assert cal.check_linearity(good, cal.fit_attention_term(good), flop) == []
    # One large shard 60% slow: the line no longer explains the times (it
    # drags the fit, so R^2 drops and shards are flagged off the line).
    bad = [(C, R, P, t * (1.6 if (C, R, P) == (1, 8192, 16384) else 1.0)) for C, R, P, t in good]
    msgs = cal.check_linearity(bad, cal.fit_attention_term(bad), flop)
    assert any(m.startswith("R^2") for m in msgs) and any("off the line" in m for m in msgs)
    # A slope implying more than the bf16 peak is flagged.
    fast = [(C, R, P, d0 + 1e-13 * cal.remaining_workload(R, P) / C) for C, R, P in GRID]
    assert any("TFLOP/s" in m for m in cal.check_linearity(fast, cal.fit_attention_term(fast), flop))
