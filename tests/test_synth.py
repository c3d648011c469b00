"""The seeded synthetic inputs: the heterogeneous mix's seed follows its
stated rule (data statistics only; no attention arithmetic here)."""

import synth


def _meets_rule(reqs):
    total = sum(L for L, _ in reqs)
    return abs(total - synth.HETERO_TOTAL) <= 0.05 * synth.HETERO_TOTAL and \
        any(L >= synth.HETERO_LONG for L, _ in reqs)


def test_hetero_seed_is_the_first_that_meets_the_rule():
    assert _meets_rule(synth.hetero_requests(seed=synth.HETERO_SEED))
    for seed in range(1005, synth.HETERO_SEED):
        assert not _meets_rule(synth.hetero_requests(seed=seed)), seed


def test_hetero_mix_shape():
    reqs = synth.hetero_requests()
    assert len(reqs) == synth.HETERO_REQUESTS
    assert sum(1 for _, P in reqs if P) == synth.HETERO_PREFIXED
    for L, P in reqs:
        assert synth.HETERO_MIN <= L <= synth.HETERO_MAX
        assert P % synth.BLOCK_TOKENS == 0 and (P == 0 or 0.2 * L - 16 <= P <= 0.8 * L)
