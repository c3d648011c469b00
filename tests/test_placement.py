"""Host checks of the adaptive placement cost (paper Sec. 5.3), with J worked
out by hand from its definition on small cases, and the behaviours the paper
describes for beta (prefix locality) and lambda (GPU-time price)."""

import pytest

from paper_2609_04774_amd import placement as pl

MODEL = pl.PrefillModel(d=1.0, alpha=1e-3)      # E_C(R, P) = 1 + 1e-3 W(R, P) / C


def test_costs_by_hand():
    workers = [pl.Worker(C=1, outstanding=[2.0]), pl.Worker(C=2), pl.Worker(C=4, eligible=False)]
    # L = 100, no prefix: W = 5050; s_1 = 6.05, s_2 = 3.525; C_min = 1 (the C = 4 worker is ineligible).
    costs = pl.placement_costs(100, workers, MODEL, beta=1.5, lam=0.5)
    assert costs[2] is None
    assert costs[0] == pytest.approx(2.0 + 1.5 * 6.05 + 0.5 * (6.05 - 6.05))
    assert costs[1] == pytest.approx(0.0 + 1.5 * 3.525 + 0.5 * (2 * 3.525 - 6.05))
    assert pl.place(100, workers, MODEL, beta=1.5, lam=0.5) == 1
    assert workers[1].outstanding == [pytest.approx(3.525)]     # reserved at placement


def test_prefix_hit_uses_the_worker_specific_prefix():
    # L = 100 with 80 cached tokens: R = 20, W = 20 * 80 + 210 = 1810.
    w = pl.Worker(C=2, prefix_for=lambda _r, L: 80)
    (j,) = pl.placement_costs(100, [w], MODEL, beta=1.0, lam=0.0)
    assert j == pytest.approx(1.0 + 1e-3 * 1810 / 2)


def test_lambda_prices_extra_gpus():
    short = 64
    assert pl.preferred_degree(short, 0, MODEL, lam=0.0) == 8     # latency only: more ranks are faster
    # W = 2080: s_C = 1 + 2.08 / C.  With lambda = 2: J_1 = 3.08, J_2 = 2.04 + 2 (2 s_2 - s_1) = 4.04, ...
    assert pl.preferred_degree(short, 0, MODEL, lam=2.0) == 1     # short request: the extra GPU time dominates
    long_model = pl.PrefillModel(d=1e-3, alpha=1e-6)
    assert pl.preferred_degree(65536, 0, long_model, lam=0.05) == 8  # compute-heavy: the speedup wins
    picks = [pl.preferred_degree(L, 0, long_model, lam=0.05) for L in (256, 2048, 16384, 65536)]
    assert picks == sorted(picks)                                  # longer requests never pick fewer ranks


def test_beta_favours_the_cache_holder():
    def workers():
        return [pl.Worker(C=2, name="idle, no cache"),
                pl.Worker(C=2, name="cache, busy", outstanding=[4.1], prefix_for=lambda _r, L: L - 100)]
    model = pl.PrefillModel(d=0.1, alpha=1e-6)
    L = 4096
    # Idle worker: W = 4096 * 4097 / 2, s = 0.1 + 4.195 = 4.295.  Cache holder: R = 100, P = 3996,
    # W = 404,650, s = 0.302, behind 4.1 s of queued work.
    # beta = 1: predicted TTFT, recomputing on the idle worker (4.295) beats waiting (4.402).
    assert pl.place(L, workers(), model, beta=1.0) == 0
    # Large beta amplifies the prefix hit's shorter service time.
    assert pl.place(L, workers(), model, beta=8.0) == 1


def test_queue_delay_steers_away_from_loaded_workers():
    ws = [pl.Worker(C=4, outstanding=[5.0]), pl.Worker(C=4)]
    assert pl.place(1000, ws, MODEL) == 1
    assert pl.place(1000, ws, MODEL) == 1 or ws[1].queue_delay() > 5.0


def test_invalid_arguments():
    with pytest.raises(ValueError):
        pl.placement_costs(10, [pl.Worker(C=1)], MODEL, beta=0.5)
    with pytest.raises(ValueError):
        pl.placement_costs(10, [pl.Worker(C=1)], MODEL, lam=-1.0)
    with pytest.raises(ValueError):
        pl.place(10, [pl.Worker(C=1, eligible=False)], MODEL)
