"""Scheduling ablation on the synthetic augmented trace: the ranking (theta,
FCFS, SSJF) and the budget mode (static T_max, or the memory-derived budget
clipped to [0.5, 2] x T_max) of the batch former, each served over the same
seeded 2000-request trace, with request-level results (time to first token,
normalized latency, goodput under the SLOs TTFT < 1 s and normalized latency
< 10 x the base iteration time). When nothing fits, the serving loop
preempts a running request by recomputation (as an engine does); the count
is reported, and no run is cut short for it.

This is the synthetic analogue of the paper's ablation (Base = FCFS with a
fixed budget, +B = dynamic budget, +S = state-aware ranking, Aug = both) and
of its SSJF baseline; the absolute numbers depend on the trace and the
iteration-time model, not on any measured engine.

    python -m synth.scheduling [--budget 2048] [--seed 0] [--rate 3.0]
"""

from __future__ import annotations

import argparse
import json
import time
from typing import Callable, List

from .sweep import former_params, run_budget

ORDERS = {"theta": 0, "fcfs": 1, "ssjf": 2}


def ablation(make_former: Callable[[dict], Callable], make_lifecycle: Callable[[], object],
             budget: int = 2048, seed: int = 0, orders=("fcfs", "ssjf", "theta"),
             modes=(False, True), max_steps: int = 30_000, rate: float = 3.0,
             admit_whole_prompt: bool = False) -> List[dict]:
    """One row per (order, budget mode): the former is ``make_former(params)``
    with the sweep's former parameters for ``budget``."""
    rows = []
    for order in orders:
        for dynamic in modes:
            t0 = time.perf_counter()
            run = run_budget(budget, make_former(former_params(budget, dynamic, ORDERS[order], chunk_cap=512)),
                             make_lifecycle(), seed=seed, dynamic=dynamic, max_steps=max_steps, rate=rate,
                             max_preemptions=1_000_000, admit_whole_prompt=admit_whole_prompt)
            m = dict(run.metrics)
            m.update(admission="whole prompt" if admit_whole_prompt else "none", order=order, budget_mode="dynamic" if dynamic else "static", t_max=budget, rate=rate,
                     complete=run.complete, iterations=len(run.steps), sim_seconds=round(run.sim_seconds, 1),
                     wall_s=round(time.perf_counter() - t0, 2))
            rows.append(m)
    return rows


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--budget", type=int, default=2048)
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--rate", type=float, default=3.0, help="arrivals per second")
    ap.add_argument("--admit-whole-prompt", action="store_true",
                    help="offer a new request to the former only when its whole prompt fits the free blocks")
    a = ap.parse_args()
    from paper_2512_04013_amd import runtime as rt
    for row in ablation(lambda p: rt.serving_former(**p), rt.serving_lifecycle, a.budget, a.seed, rate=a.rate,
                        admit_whole_prompt=a.admit_whole_prompt):
        print(json.dumps(row), flush=True)


if __name__ == "__main__":
    main()
