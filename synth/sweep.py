"""The token-budget sweep: formed batches of a synthetic augmented trace laid
out on a 64-query-head, 8-KV-head, head_dim 128 layer with bf16 queries and an
fp8 E4M3FN KV cache (one fp32 scale per block, KV head and K|V).

The trace is ``synth.trace.make_trace`` (2000 requests, Poisson arrivals at 3
per second, lognormal prompts and outputs, 0-4 external calls with
exponential pauses and 20-800 returned tokens). ``run_budget`` drives a batch
former -- any callable, normally the library's -- over it through
``ServingLoop`` and returns the step records: which requests ran, with how
many query tokens and how many keys. This module only chooses and lays out
batches; the budget, costs, priorities and packing come from the former.

Every budget of the sweep serves the whole trace at 3 requests per second
(prefill chunks are capped at half the budget). A budget too small for a
heavier trace leaves the loop overloaded: requests pile up until the pool
thrashes. Such a run stops at ``max_steps`` iterations (or when the loop
reports thrashing) and is marked incomplete.
"""

from __future__ import annotations

import dataclasses
from typing import Callable, Dict, List, Optional, Sequence

import numpy as np

from .attn_inputs import AttnBatch, make_batch_from_lengths
from .trace import ServingLoop, SimConfig, StepRecord, make_trace

BUDGETS = (256, 512, 1024, 2048, 4096, 8192)
HEADS_Q, HEADS_KV, HEAD_DIM = 64, 8, 128
POOL_BLOCKS = 16384          # the serving loop's pool (blocks of 16 tokens)

# Former parameters of the sweep (field names of the former's parameter
# record); ``t_max`` is the budget being swept, and the dynamic mode clips the
# memory-derived budget to [0.5, 2] x t_max while the static mode pins it.
FORMER_PARAMS = dict(beta=5e-5, t_iter=0.02, fwd_a=0.0175, fwd_b=20.5e-9, swap_s_per_tok=4.1e-8,
                     n_fwd_max=1)


def sweep_chunk_cap(budget: int) -> int:
    """Prefill tokens one request may take per iteration under reference
    budget T_max: half of it (at least 64). A prompt, a call's returned tokens
    or a recomputed context then never fills a batch on its own, so decodes
    always fit beside a chunk (with a fixed 512-token cap, budget 256 could
    place a chunk only in an empty batch and could not serve the trace), and
    larger budgets take longer chunks, as an engine without chunking would
    take a whole prompt that fits its token limit."""
    return max(64, int(budget) // 2)


def former_params(budget: int, dynamic: bool = True, order: int = 0, chunk_cap: Optional[int] = None) -> dict:
    p = dict(FORMER_PARAMS, t_max=int(budget), order=int(order),
             chunk_cap=int(sweep_chunk_cap(budget) if chunk_cap is None else chunk_cap))
    p.update(beta_low=0.5, beta_high=2.0) if dynamic else p.update(beta_low=1.0, beta_high=1.0)
    return p


@dataclasses.dataclass
class SweepRun:
    budget: int
    dynamic: bool
    steps: List[StepRecord]          # non-empty iterations only
    complete: bool                   # every request of the trace finished
    finished: int                    # requests that finished
    sim_seconds: float
    metrics: dict                    # request-level results (ServingLoop.metrics)
    former_stats: Optional[dict] = None   # per-iteration former time, when the former records it


def run_budget(budget: int, former: Callable, lifecycle, seed: int = 0, dynamic: bool = True,
               max_steps: int = 40_000, n_requests: int = 2000, rate: float = 3.0,
               max_preemptions: int = 200, admit_whole_prompt: bool = False) -> SweepRun:
    """Serve the seeded trace (``rate`` arrivals per second) with ``former``
    (built for this budget) and the request-record ``lifecycle`` (arrival and
    call return)."""
    trace = make_trace(n=n_requests, seed=seed, rate=rate)
    loop = ServingLoop(trace, SimConfig(num_blocks=POOL_BLOCKS, max_preemptions=max_preemptions,
                                        admit_whole_prompt=admit_whole_prompt), lifecycle)
    try:
        loop.run(former, max_steps=max_steps)
    except RuntimeError as e:          # thrashing: the budget cannot serve the trace
        if "thrashing" not in str(e):
            raise
    steps = [s for s in loop.steps if s.ids]
    return SweepRun(budget=budget, dynamic=dynamic, steps=steps,
                    complete=len(loop.done) == n_requests, finished=len(loop.done),
                    sim_seconds=loop.now, metrics=dict(loop.metrics(), preemptions=loop.preemptions),
                    former_stats=former_overhead(getattr(former, "timings", None)))


# bins of paused requests for the per-iteration former time (the paper's
# scheduling-overhead table groups iterations the same way)
PAUSED_BINS = ((0, 50), (50, 100), (100, 150), (150, 200), (200, 10 ** 9))


def former_overhead(timings) -> Optional[dict]:
    """Per-iteration time of the former call (mean, p50, p99, in us), overall
    and by number of paused requests, from (seconds, records, paused) tuples."""
    if not timings:
        return None
    t = np.array([x[0] for x in timings]) * 1e6
    n = np.array([x[1] for x in timings])
    pz = np.array([x[2] for x in timings])
    out = {"iterations": int(t.size), "us_mean": round(float(t.mean()), 1),
           "us_p50": round(float(np.median(t)), 1), "us_p99": round(float(np.percentile(t, 99)), 1),
           "records_mean": round(float(n.mean()), 1), "records_max": int(n.max()), "by_paused": {}}
    for lo, hi in PAUSED_BINS:
        sel = (pz >= lo) & (pz < hi)
        if sel.any():
            key = f"{lo}-{hi}" if hi < 10 ** 9 else f">={lo}"
            out["by_paused"][key] = {"iterations": int(sel.sum()), "us_mean": round(float(t[sel].mean()), 1)}
    return out


def prefill_pairs(step: StepRecord) -> int:
    """Query-key pairs of the step's multi-row (prefill) requests: row j of a
    request with q rows and ctx keys attends ctx - q + j + 1 keys."""
    n = 0
    for q, c in zip(step.q_len, step.ctx_len):
        if q > 1:
            n += q * (c - q) + q * (q + 1) // 2
    return n


def select_steps(steps: Sequence[StepRecord], n_random: int, seed: int) -> Dict[str, int]:
    """Indices of the batches a test or benchmark looks at: the one with the
    most query tokens, the one with the most prefill query-key pairs, the one
    with the most context tokens, and ``n_random`` seeded others."""
    q = np.array([sum(s.q_len) for s in steps])
    pairs = np.array([prefill_pairs(s) for s in steps])
    ctx = np.array([sum(s.ctx_len) for s in steps])
    out = {"most_tokens": int(np.argmax(q)), "most_prefill": int(np.argmax(pairs)),
           "most_context": int(np.argmax(ctx))}
    rng = np.random.default_rng(seed)
    for k, i in enumerate(rng.choice(len(steps), size=min(n_random, len(steps)), replace=False)):
        out[f"random{k}"] = int(i)
    return out


def batch_for_step(step: StepRecord, seed: int, name: str = "sweep-64x8-fp8",
                   n_pool_blocks: Optional[int] = None, sharp: bool = False) -> AttnBatch:
    """Lay one formed batch out on the 64/8-head fp8 layer: bf16 Q ~ N(0,1),
    K/V ~ N(0,1)/sqrt(128) (N(0,1) when ``sharp``) encoded per block (scale
    max|x|/448), blocks dealt from a random permutation of the pool, unused
    slots NaN."""
    need = int(sum(-(-c // 16) for c in step.ctx_len))
    pool = n_pool_blocks or max(POOL_BLOCKS, need + 64)
    return make_batch_from_lengths(
        name, step.q_len, step.ctx_len, num_q_heads=HEADS_Q, num_kv_heads=HEADS_KV,
        head_dim=HEAD_DIM, q_dtype="bf16", kv_dtype="fp8", out_dtype="bf16", n_pool_blocks=pool,
        seed=seed, kv_std=1.0 if sharp else 1.0 / np.sqrt(HEAD_DIM))
