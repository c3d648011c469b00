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


# PreferDegree on a prefill-time model of the form the calibration fits:
# E_C(R, P) = d0 + alpha W(R, P) / C, d0 = 100 us, alpha = 1.5e-11 s per pair.
# With beta = lambda = 1 on idle workers of degrees 1, 2, 4, 8 (C_min = 1):
#   J_C = s_C + (C s_C - s_1) = d0 + alpha W / C + (C - 1) d0.
FIT = pl.PrefillModel(d=1e-4, alpha=1.5e-11)


@pytest.mark.parametrize("L,P,J,pick", [
    # W = 2,098,176: alpha W = 3.147264e-5.
    (2048, 0, [1.3147264e-4, 2.15736320e-4, 4.07868160e-4, 8.03934080e-4], 1),
    # W = 33,558,528: alpha W = 5.0337792e-4.
    (8192, 0, [6.0337792e-4, 4.5168896e-4, 5.2584448e-4, 8.6292224e-4], 2),
    # W = 134,225,920: alpha W = 2.0133888e-3.
    (16384, 0, [2.1133888e-3, 1.2066944e-3, 9.033472e-4, 1.0516736e-3], 4),
    # R = P = 8192: W = 8192 * 8192 + 33,558,528 = 100,667,392; alpha W = 1.51001088e-3.
    (16384, 8192, [1.61001088e-3, 9.5500544e-4, 7.7750272e-4, 9.8875136e-4], 4),
    # W = 536,887,296: alpha W = 8.05330944e-3.
    (32768, 0, [8.15330944e-3, 4.22665472e-3, 2.41332736e-3, 1.80666368e-3], 8),
])
def test_prefer_degree_on_a_fitted_model_by_hand(L, P, J, pick):
    workers = [pl.Worker(C=C, prefix_for=lambda _r, _L: P) for C in pl.DEGREES]
    costs = pl.placement_costs(L, workers, FIT, beta=pl.DEFAULT_BETA, lam=pl.DEFAULT_LAMBDA)
    assert costs == pytest.approx(J, rel=1e-9)
    assert pl.preferred_degree(L, P, FIT, pl.DEGREES, pl.DEFAULT_BETA, pl.DEFAULT_LAMBDA) == pick
    assert pl.choose_degrees([(L, P)], "cost", FIT) == [pick]


def test_length_rule_buckets():
    assert [pl.degree_by_length(L) for L in (256, 8191, 8192, 32767, 32768, 65535, 65536, 131072)] == \
        [1, 1, 2, 2, 4, 4, 8, 8]
    assert pl.choose_degrees([(100, 0), (40000, 16)], "length") == [1, 4]
    with pytest.raises(ValueError):
        pl.choose_degrees([(100, 0)], "cost")
    with pytest.raises(ValueError):
        pl.choose_degrees([(100, 0)], "size")


def test_model_from_calibration(tmp_path):
    f = tmp_path / "cal.json"
    f.write_text('{"fit": {"d0_s": 0.0001, "alpha_s_per_pair": 1.5e-11, "r2": 0.999}}')
    m = pl.model_from_calibration(str(f))
    assert m.predict(2, 8192, 0) == pytest.approx(1e-4 + 1.5e-11 * 33558528 / 2)
