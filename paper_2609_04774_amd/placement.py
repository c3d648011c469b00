"""CP-aware request placement: the adaptive placement cost of Sec. 5.3.

For request i and an eligible worker w (CP degree C_w, reusable prefix
P_{i,w}, uncached suffix R_{i,w} = L_i - P_{i,w}):

    s_{i,w} = E_{C_w}(R_{i,w}, P_{i,w})                        (service time)
    q_w     = sum of E_{C_w}(R_j, P_j) over unfinished requests j at w
    J_{i,w} = q_w + beta s_{i,w}
              + lambda [C_w s_{i,w} - C_min E_{C_min}(R_{i,w}, P_{i,w})]

with C_min the smallest degree among the eligible workers, beta >= 1 the
weight on cache-aware service time and lambda >= 0 the price of extra GPU
time.  The request goes to the worker of least J, which then reserves the
request's predicted service time (Sec. 5.2) so that later arrivals see it.

E_C(R, P) is the prefill-time model of Sec. 3.2 (``PrefillModel``), e.g. with
the attention term calibrated by ``calibrate.fit_attention_term`` or all five
coefficients by ``calibrate.fit_prefill_model``.  This is host-side policy:
no GPU is involved.
"""

from __future__ import annotations

from dataclasses import dataclass, field
from typing import Callable, List, Optional, Sequence


# Readings (the paper gives the roles of beta and lambda, not their values):
# beta = 1 makes q_w + s_{i,w} the predicted worker-dependent TTFT (Sec. 5.3);
# lambda = 1 weighs one GPU-second of extra occupancy like one second of it.
DEFAULT_BETA = 1.0
DEFAULT_LAMBDA = 1.0
DEGREES = (1, 2, 4, 8)


def remaining_workload(R: int, P: int) -> int:
    """W(R, P) = R P + R (R + 1) / 2 (Sec. 2.2)."""
    return R * P + R * (R + 1) // 2


@dataclass
class PrefillModel:
    """E_C(R, P) = d + a R + b P + (c R + alpha W(R, P)) / C  (Sec. 3.2)."""
    d: float = 0.0
    a: float = 0.0
    b: float = 0.0
    c: float = 0.0
    alpha: float = 0.0

    def predict(self, C: int, R: int, P: int) -> float:
        return self.d + self.a * R + self.b * P + (self.c * R + self.alpha * remaining_workload(R, P)) / C


@dataclass
class Worker:
    """A CP worker as the scheduler sees it (Sec. 5.2): its degree, the
    predicted service times of the requests it has not finished, and which
    prefix of a request it can reuse (``prefix_for(tokens_id, L)`` returns a
    cached length <= L; the default caches nothing)."""
    C: int
    name: str = ""
    eligible: bool = True
    outstanding: List[float] = field(default_factory=list)
    prefix_for: Optional[Callable[[object, int], int]] = None

    def queue_delay(self) -> float:
        return float(sum(self.outstanding))

    def reusable_prefix(self, request_id, L: int) -> int:
        return 0 if self.prefix_for is None else max(0, min(L, int(self.prefix_for(request_id, L))))


def placement_costs(L: int, workers: Sequence[Worker], model: PrefillModel, beta: float = 1.0,
                    lam: float = 0.0, request_id=None) -> List[Optional[float]]:
    """J_{i,w} for every worker (None for an ineligible one)."""
    if beta < 1.0 or lam < 0.0:
        raise ValueError("beta >= 1 and lambda >= 0 (Sec. 5.3)")
    cand = [w for w in workers if w.eligible]
    if not cand:
        return [None] * len(workers)
    c_min = min(w.C for w in cand)
    out: List[Optional[float]] = []
    for w in workers:
        if not w.eligible:
            out.append(None)
            continue
        P = w.reusable_prefix(request_id, L)
        R = L - P
        s = model.predict(w.C, R, P)
        extra = w.C * s - c_min * model.predict(c_min, R, P)
        out.append(w.queue_delay() + beta * s + lam * extra)
    return out


def place(L: int, workers: Sequence[Worker], model: PrefillModel, beta: float = 1.0, lam: float = 0.0,
          request_id=None) -> int:
    """Index of the least-cost eligible worker (first on ties); reserves the
    request's predicted service time at that worker."""
    costs = placement_costs(L, workers, model, beta, lam, request_id)
    best = None
    for i, j in enumerate(costs):
        if j is not None and (best is None or j < costs[best]):
            best = i
    if best is None:
        raise ValueError("no eligible worker")
    w = workers[best]
    P = w.reusable_prefix(request_id, L)
    w.outstanding.append(model.predict(w.C, L - P, P))
    return best


def preferred_degree(L: int, P: int, model: PrefillModel, degrees: Sequence[int] = (1, 2, 4, 8),
                     beta: float = 1.0, lam: float = 0.0) -> int:
    """The CP degree J picks for a request of L tokens with a P-token prefix
    hit on idle workers of every degree (the per-request choice of C that
    replaces a fixed length rule)."""
    workers = [Worker(C=C, prefix_for=lambda _r, _L: P) for C in degrees]
    return workers[place(L, workers, model, beta, lam)].C


def degree_by_length(L: int) -> int:
    """The fixed length rule the placement cost replaces: C = 1 below 8K
    tokens, 2 below 32K, 4 below 64K, else 8 (the paper's short / medium /
    long buckets, Sec. 3 and its TTFT SLO table)."""
    if L < 8192:
        return 1
    if L < 32768:
        return 2
    if L < 65536:
        return 4
    return 8


def model_from_calibration(path: str) -> PrefillModel:
    """E_C(R, P) = d0 + alpha W(R, P) / C from a calibration file written by
    ``python -m paper_2609_04774_amd.calibrate --out`` (the attention term of
    Sec. 3.2 measured on this GPU; the model's other terms are not measured
    here and stay 0)."""
    import json
    with open(path) as f:
        fit = json.load(f)["fit"]
    return PrefillModel(d=float(fit["d0_s"]), alpha=float(fit["alpha_s_per_pair"]))


def choose_degrees(requests, rule: str, model: Optional[PrefillModel] = None, beta: float = DEFAULT_BETA,
                   lam: float = DEFAULT_LAMBDA, degrees: Sequence[int] = DEGREES) -> List[int]:
    """Per-request CP degree of [(L, P)]: rule "cost" takes PreferDegree over
    idle workers of every degree (Sec. 7.1: the placement cost without the
    queue term), rule "length" the fixed length buckets."""
    if rule == "length":
        return [degree_by_length(L) for L, _ in requests]
    if rule != "cost":
        raise ValueError("rule must be 'cost' or 'length'")
    if model is None:
        raise ValueError("the cost rule needs a prefill-time model")
    return [preferred_degree(L, P, model, degrees, beta, lam) for L, P in requests]
