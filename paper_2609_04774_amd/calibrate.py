"""Calibration of the prefill-time model's attention term from kernel timings.

The paper's cache-aware prefill-time model (Sec. 3.2, equation
"prefill-performance-model") predicts a request's prefill time on a degree-C
worker as

    E_C(R, P) = d + a R + b P + (c R + alpha W(R, P)) / C,
    W(R, P)   = R P + R (R + 1) / 2      (Sec. 2.2, "remaining-attention"),

with coefficients fitted from queue-free profiles.  Of its terms, the
attention kernel supplies alpha W / C: zigzag sharding gives every rank about
W / C visible (query, key) pairs, and the CP step waits for its slowest rank.
``measure_attention`` times one attention layer's CP step (every rank's shard,
the maximum over ranks) on the GPU over a grid of (C, R, P);
``fit_attention_term`` fits t = d0 + alpha W / C to such samples and reports
how well a straight line in W / C explains them; ``fit_prefill_model`` fits
the paper's full five-coefficient model when end-to-end times are available.
The fits are ordinary least squares in numpy (host only).
"""

from __future__ import annotations

from dataclasses import dataclass
from typing import Iterable, List, Sequence, Tuple

import numpy as np


def remaining_workload(R: int, P: int) -> int:
    """W(R, P) = R P + R (R + 1) / 2: the causal (query, key) pairs of R new
    tokens after a cached prefix of P tokens."""
    return R * P + R * (R + 1) // 2


@dataclass
class AttentionFit:
    d0: float          # seconds: fixed cost of a CP step's attention (launch, ramp-up)
    alpha: float       # seconds per (query, key) pair per rank, for the whole layer's heads
    r2: float          # coefficient of determination of t against W / C
    max_rel_err: float  # largest |predicted - measured| / measured over the samples

    def predict(self, C: int, R: int, P: int) -> float:
        return self.d0 + self.alpha * remaining_workload(R, P) / C


@dataclass
class PrefillFit:
    d: float
    a: float
    b: float
    c: float
    alpha: float
    max_rel_err: float

    def predict(self, C: int, R: int, P: int) -> float:
        return self.d + self.a * R + self.b * P + (self.c * R + self.alpha * remaining_workload(R, P)) / C


def _rel_err(pred: np.ndarray, t: np.ndarray) -> float:
    return float(np.max(np.abs(pred - t) / t))


def fit_attention_term(samples: Iterable[Tuple[int, int, int, float]]) -> AttentionFit:
    """Least-squares t = d0 + alpha * W(R, P) / C over samples (C, R, P, t)."""
    rows = [(C, R, P, t) for C, R, P, t in samples]
    if len(rows) < 2:
        raise ValueError("need at least two samples")
    x = np.array([remaining_workload(R, P) / C for C, R, P, _ in rows], dtype=np.float64)
    t = np.array([s[3] for s in rows], dtype=np.float64)
    if np.ptp(x) == 0:
        raise ValueError("the samples must span more than one W / C")
    A = np.stack([np.ones_like(x), x], axis=1)
    (d0, alpha), *_ = np.linalg.lstsq(A, t, rcond=None)
    pred = A @ np.array([d0, alpha])
    ss_res = float(np.sum((t - pred) ** 2))
    ss_tot = float(np.sum((t - t.mean()) ** 2))
    r2 = 1.0 - ss_res / ss_tot if ss_tot > 0 else 1.0
    return AttentionFit(float(d0), float(alpha), r2, _rel_err(pred, t))


def fit_prefill_model(samples: Iterable[Tuple[int, int, int, float]]) -> PrefillFit:
    """Least-squares fit of the paper's five coefficients (d, a, b, c, alpha)
    over samples (C, R, P, t); the grid must vary C, R and P enough for the
    five regressors 1, R, P, R / C, W / C to be independent."""
    rows = [(C, R, P, t) for C, R, P, t in samples]
    A = np.array([[1.0, R, P, R / C, remaining_workload(R, P) / C] for C, R, P, _ in rows], dtype=np.float64)
    t = np.array([s[3] for s in rows], dtype=np.float64)
    if len(rows) < 5 or np.linalg.matrix_rank(A) < 5:
        raise ValueError("the samples do not determine all five coefficients")
    coef, *_ = np.linalg.lstsq(A, t, rcond=None)
    return PrefillFit(*(float(v) for v in coef), _rel_err(A @ coef, t))


def measure_attention(grid: Sequence[Tuple[int, int, int]], n_heads_q: int = 32, n_heads_kv: int = 8,
                      reps: int = 5, seed: int = 0, warmup: int = 3,
                      warmup_seconds: float = 1.0) -> List[Tuple[int, int, int, float]]:
    """GPU time (seconds) of one attention layer's CP step for each (C, R, P):
    every rank's partial over all its visible keys (prefix through a paged
    cache), each rank timed alone with HIP events on the launch stream; the
    step time is the slowest rank's (median of ``reps`` runs, after
    ``warmup`` untimed launches).  The first grid point is also run untimed
    for ``warmup_seconds`` before anything is measured: a cold GPU (clocks
    still rising, fresh allocations) measured up to 20% slow on the first
    points of a grid."""
    import time

    import torch

    from . import cpattn as cp

    D, B = cp.CP_HEAD_DIM, cp.CP_KV_BLOCK_TOKENS
    dev = torch.device("cuda", torch.cuda.current_device())
    stream = torch.cuda.current_stream()
    g = torch.Generator(device=dev)
    g.manual_seed(seed)
    warm_left = float(warmup_seconds)
    out = []
    for C, R, P in grid:
        if P % B:
            raise ValueError("P must be a multiple of 16")
        k = torch.randn((R, n_heads_kv, D), generator=g, device=dev).to(torch.bfloat16)
        v = torch.randn((R, n_heads_kv, D), generator=g, device=dev).to(torch.bfloat16)
        kc = vc = table = None
        if P:
            nb = P // B
            kc = torch.randn((nb, B, n_heads_kv, D), generator=g, device=dev).to(torch.bfloat16)
            vc = torch.randn((nb, B, n_heads_kv, D), generator=g, device=dev).to(torch.bfloat16)
            table = torch.randperm(nb, generator=g, device=dev).to(torch.int32)
        worst = 0.0
        for r in range(C):
            plan, _ = cp.shard_plan(P, R, C, r, with_rows=False)
            if plan.n_rows == 0:
                continue
            q = torch.randn((plan.n_rows, n_heads_q, D), generator=g, device=dev).to(torch.bfloat16)
            o = torch.empty((plan.n_rows, n_heads_q, D), dtype=torch.float32, device=dev)
            lse = torch.empty((plan.n_rows, n_heads_q), dtype=torch.float32, device=dev)
            desc = cp.make_desc(plan, q, k, v, o, lse, kc, vc, table, include_prefix=True)
            ws = torch.empty(max(256, cp.workspace_size([desc], n_heads_q, n_heads_kv)), dtype=torch.uint8,
                             device=dev)
            for _ in range(max(1, warmup)):
                cp.attn_partial([desc], n_heads_q, n_heads_kv, ws, stream=stream)
            if warm_left > 0:
                t_end = time.perf_counter() + warm_left
                while time.perf_counter() < t_end:
                    cp.attn_partial([desc], n_heads_q, n_heads_kv, ws, stream=stream)
                    torch.cuda.synchronize()
                warm_left = 0.0
            times = []
            for _ in range(reps):
                a = torch.cuda.Event(enable_timing=True)
                b = torch.cuda.Event(enable_timing=True)
                a.record(stream)
                cp.attn_partial([desc], n_heads_q, n_heads_kv, ws, stream=stream)
                b.record(stream)
                b.synchronize()
                times.append(a.elapsed_time(b) * 1e-3)
            worst = max(worst, float(np.median(times)))
        out.append((C, R, P, worst))
    return out


DEFAULT_GRID = [(C, R, P) for C in (1, 2, 4, 8) for R in (4096, 8192, 16384, 32768) for P in (0, 16384)]


def check_linearity(samples, fit, flop_per_pair: float, min_pairs: float = 3e7) -> List[str]:
    """The linearity claims of the attention term on measured samples: a
    straight line in W / C explains them (R^2 > 0.98); every shard large
    enough to fill the GPU (W / C >= min_pairs) sits within 25% of the line
    (smaller ones finish faster than the intercept); the slope's implied rate
    lies between 10% and 100% of the bf16 peak.  Returns the failures (empty
    when all hold).  Timing claims: run by ``main --check`` on a quiet GPU,
    not by the parity tests."""
    bad = []
    if not fit.alpha > 0:
        bad.append(f"alpha = {fit.alpha} is not positive")
    if not fit.r2 > 0.98:
        bad.append(f"R^2 = {fit.r2:.4f} <= 0.98")
    for C, R, P, t in samples:
        if remaining_workload(R, P) / C >= min_pairs and abs(fit.predict(C, R, P) - t) / t >= 0.25:
            bad.append(f"(C={C}, R={R}, P={P}): {t * 1e3:.3f} ms is more than 25% off the line")
    tflops = flop_per_pair / fit.alpha / 1e12 if fit.alpha > 0 else 0.0
    if not 250 < tflops < 2500:
        bad.append(f"implied {tflops:.0f} TFLOP/s outside 250..2500")
    return bad


def main(argv=None):
    """Measure the default grid (Llama-3-8B attention shape: 32 query heads,
    8 KV heads, D = 128) and print the samples and the attention-term fit as
    JSON; --out also writes that JSON to a file (the fit the placement
    policy reads); --check exits non-zero when the linearity claims of
    ``check_linearity`` fail."""
    import argparse
    import json
    import sys

    ap = argparse.ArgumentParser(description=main.__doc__)
    ap.add_argument("--heads-q", type=int, default=32)
    ap.add_argument("--heads-kv", type=int, default=8)
    ap.add_argument("--reps", type=int, default=5)
    ap.add_argument("--out", default=None, help="also write the JSON to this file")
    ap.add_argument("--check", action="store_true", help="exit 1 if the linearity claims fail")
    args = ap.parse_args(argv)
    samples = measure_attention(DEFAULT_GRID, args.heads_q, args.heads_kv, args.reps)
    fit = fit_attention_term(samples)
    flop_per_pair = 4 * 128 * args.heads_q
    failures = check_linearity(samples, fit, flop_per_pair)
    text = json.dumps({
        "shape": {"Hq": args.heads_q, "Hkv": args.heads_kv, "D": 128},
        "samples": [{"C": C, "R": R, "P": P, "W_over_C": remaining_workload(R, P) / C, "seconds": t}
                    for C, R, P, t in samples],
        "fit": {"d0_s": fit.d0, "alpha_s_per_pair": fit.alpha, "r2": fit.r2, "max_rel_err": fit.max_rel_err,
                "implied_tflops": flop_per_pair / fit.alpha / 1e12},
        "linearity_failures": failures,
    }, indent=1)
    print(text, flush=True)
    if args.out:
        with open(args.out, "w") as f:
            f.write(text + "\n")
    if args.check and failures:
        print("linearity check failed: " + "; ".join(failures), file=sys.stderr)
        sys.exit(1)


if __name__ == "__main__":
    main()
