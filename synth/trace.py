"""Synthetic augmented-LLM request trace and a discrete-event serving loop.

The trace: Poisson arrivals; prompt and output lengths lognormal; each
request makes 0-4 external calls fired at equal splits of its output; each
call pauses the request for an exponential time and returns a number of
tokens that the request then prefills (the returned-tokens stage of a
segment). Predictions of segment output lengths and call durations are the
true values times (1 + e) with e = +-p chosen at random, output lengths
rounded up to 50-token buckets (the noise model and bucket size the paper
uses for its predictor).

The loop keeps every request in the scheduler's record format. Records are
created on arrival and renewed when a call returns by a ``lifecycle`` object
(``arrive`` and ``on_return``: Algorithm 1, steps (1)-(2), normally the
library's). Each iteration the loop asks a batch former (any callable) for a
plan, then applies it:
evictions (park or free), resumes, the chunk or decode token of every
scheduled request, pauses, call returns with the policy that was actually
realised (Swap if the context was parked, Discard if it was freed, Preserve
if it stayed), completions, and a simulated clock. It contains none of the
scheduler's arithmetic: budget, cost, priority, policy choice and packing all
come from the former and the record transitions from the lifecycle, so the
oracle and the C++ library can be driven in lock step. Iteration time follows a simple linear model of a large model on
one GPU: t = t0 + a * (query tokens) + b * (context tokens).
"""

from __future__ import annotations

import dataclasses
from typing import Callable, Dict, List, Optional, Tuple

import numpy as np

WAITING, RUNNING, SWAPPED, PAUSED = 0, 1, 2, 3
NONE, PRESERVE, DISCARD, SWAP = 0, 1, 2, 3
BLOCK = 16

FIELDS = ("id", "arrival", "last_sched", "pred_call", "pause_start", "state", "seg", "prev_policy",
          "cur_policy", "seg_ctx", "seg_prefill", "pred_out", "has_next_call", "ctx_len", "pending",
          "blocks_on_gpu")


@dataclasses.dataclass
class TraceRequest:
    id: int
    arrival: float
    prompt: int
    output: int
    call_after: List[int]          # generated-token counts at which calls fire
    pause: List[float]             # true call durations (s)
    ret: List[int]                 # tokens each call returns
    pred_sign: List[int]           # +-1 per segment, prediction error direction


def _bucket(x: float, size: int = 50) -> int:
    return max(size, int(-(-x // size)) * size)


def make_trace(n: int = 2000, rate: float = 3.0, seed: int = 0, prompt_median: float = 800.0,
               out_median: float = 200.0, sigma: float = 0.8, max_calls: int = 4,
               pause_mean: float = 0.5, ret_lo: int = 20, ret_hi: int = 800,
               max_prompt: int = 8192, max_output: int = 2048) -> List[TraceRequest]:
    rng = np.random.default_rng(seed)
    arrivals = np.cumsum(rng.exponential(1.0 / rate, size=n))
    prompts = np.clip(np.rint(rng.lognormal(np.log(prompt_median), sigma, size=n)), 1, max_prompt)
    outputs = np.clip(np.rint(rng.lognormal(np.log(out_median), sigma, size=n)), 1, max_output)
    reqs = []
    for i in range(n):
        out = int(outputs[i])
        c = int(rng.integers(0, max_calls + 1))
        c = min(c, out - 1) if out > 1 else 0
        after = sorted({int(round(k * out / (c + 1))) for k in range(1, c + 1)} - {0, out})
        c = len(after)
        reqs.append(TraceRequest(
            id=i, arrival=float(arrivals[i]), prompt=int(prompts[i]), output=out, call_after=after,
            pause=[float(x) for x in rng.exponential(pause_mean, size=c)],
            ret=[int(x) for x in rng.integers(ret_lo, ret_hi + 1, size=c)],
            pred_sign=[int(x) for x in rng.choice([-1, 1], size=c + 1)]))
    return reqs


@dataclasses.dataclass
class _Live:
    rec: Dict[str, float]          # scheduler record (FIELDS)
    tr: TraceRequest
    generated: int = 0
    seg_index: int = 0             # index of the current segment (0-based)
    logical_ctx: int = 0           # tokens of the context, whether or not its KV is held
    pause_end: float = 0.0
    parked: bool = False
    freed: bool = False
    admitted: bool = False         # scheduled at least once


@dataclasses.dataclass
class SimConfig:
    num_blocks: int = 16384
    t0: float = 0.0175             # iteration time model
    per_query_token: float = 56e-6
    per_context_token: float = 20.5e-9
    pred_err: float = 0.2
    max_iters: int = 10 ** 7
    max_preemptions: int = 100_000   # recompute preemptions before the loop gives up (thrashing)
    # an engine's admission rule, not part of the paper's algorithm: a request
    # that has never run is offered to the former only while the free blocks
    # (less those set aside for requests admitted earlier in the same
    # iteration) cover its whole prompt
    admit_whole_prompt: bool = False


@dataclasses.dataclass
class StepRecord:
    now: float
    budget: int
    ids: List[int]
    q_len: List[int]
    ctx_len: List[int]             # keys of each scheduled request after this step's tokens
    n_resume: int
    n_park: int
    n_free: int
    resume_blocks: int
    park_blocks: int


class ServingLoop:
    """Drives a batch former over a trace. ``former(records, free_blocks, now)``
    receives a list of dicts with the FIELDS keys and returns a dict with
    budget, ids, q_len, resume_ids, park_ids, free_ids and policy (per record)."""

    def __init__(self, trace: List[TraceRequest], cfg: SimConfig, lifecycle):
        self.lifecycle = lifecycle
        self.trace = sorted(trace, key=lambda t: (t.arrival, t.id))
        self.cfg = cfg
        self.now = 0.0
        self.free = cfg.num_blocks
        self.live: Dict[int, _Live] = {}
        self.next_arrival = 0
        self.done: Dict[int, Tuple[float, float, float]] = {}   # id -> (arrival, first token, finish)
        self.first_token: Dict[int, float] = {}
        self.steps: List[StepRecord] = []
        self.preemptions = 0
        self.last_ids = set()                                   # requests of the last non-empty iteration

    # ---- segment bookkeeping ------------------------------------------------------

    def _segment_len(self, lv: _Live) -> int:
        tr, k = lv.tr, lv.seg_index
        end = tr.call_after[k] if k < len(tr.call_after) else tr.output
        start = tr.call_after[k - 1] if k > 0 else 0
        return end - start

    def _predictions(self, lv: _Live):
        tr, k = lv.tr, lv.seg_index
        e = self.cfg.pred_err * tr.pred_sign[k]
        pred_out = _bucket(self._segment_len(lv) * (1.0 + e))
        has_call = k < len(tr.call_after)
        pred_call = tr.pause[k] * (1.0 + e) if has_call else 0.0
        return pred_out, pred_call, int(has_call)

    def _arrive(self, tr: TraceRequest):
        lv = _Live(rec={}, tr=tr)
        pred_out, pred_call, has_call = self._predictions(lv)
        lv.rec = self.lifecycle.arrive(id=tr.id, arrival=tr.arrival, prompt_tokens=tr.prompt,
                                       pred_out=pred_out, pred_call=pred_call, has_next_call=has_call)
        self.live[tr.id] = lv

    def _return(self, lv: _Live):
        # the policy actually realised during the wait: Swap if the context was
        # parked, Discard if it was freed, Preserve if it stayed
        realised = SWAP if lv.parked else DISCARD if lv.freed else PRESERVE
        ret = lv.tr.ret[lv.seg_index]
        lv.seg_index += 1
        pred_out, pred_call, has_call = self._predictions(lv)
        lv.rec = self.lifecycle.on_return(lv.rec, realised=realised, context_tokens=lv.logical_ctx,
                                          ret_tokens=ret, pred_out=pred_out, pred_call=pred_call,
                                          has_next_call=has_call)
        lv.parked = lv.freed = False

    # ---- one iteration -------------------------------------------------------------

    def next_event_time(self) -> Optional[float]:
        times = []
        if self.next_arrival < len(self.trace):
            times.append(self.trace[self.next_arrival].arrival)
        times += [lv.pause_end for lv in self.live.values() if lv.rec["state"] == PAUSED]
        return min(times) if times else None

    def records(self) -> List[dict]:
        return [dict(self.live[i].rec) for i in sorted(self.live)]

    def step(self, former: Callable) -> Optional[StepRecord]:
        while self.next_arrival < len(self.trace) and self.trace[self.next_arrival].arrival <= self.now:
            self._arrive(self.trace[self.next_arrival])
            self.next_arrival += 1
        for i in sorted(self.live):
            lv = self.live[i]
            if lv.rec["state"] == PAUSED and lv.pause_end <= self.now:
                self._return(lv)
        if not self.live:
            t = self.next_event_time()
            if t is None:
                return None
            self.now = max(self.now, t)
            return self.step(former)

        recs = self.records()
        if self.cfg.admit_whole_prompt:
            room, offered = self.free, []
            for r in recs:
                if r["state"] == WAITING and not self.live[r["id"]].admitted:
                    need = -(-(r["ctx_len"] + r["pending"]) // BLOCK)
                    if need > room:
                        continue
                    room -= need
                offered.append(r)
            recs = offered
        plan = former(recs, self.free, self.now)
        order = [r["id"] for r in recs]
        policy = {order[k]: plan["policy"][k] for k in range(len(order))}
        park_blocks = 0
        for vid in plan["park_ids"]:
            lv = self.live[int(vid)]
            park_blocks += lv.rec["blocks_on_gpu"]
            self.free += lv.rec["blocks_on_gpu"]
            lv.rec["blocks_on_gpu"] = 0
            lv.parked = True
        for vid in plan["free_ids"]:
            lv = self.live[int(vid)]
            self.free += lv.rec["blocks_on_gpu"]
            lv.rec.update(blocks_on_gpu=0, ctx_len=0)
            lv.freed = True
        resume_blocks = 0
        ids, qls, ctxs = [], [], []
        batch_q = batch_ctx = 0
        finished = []
        for rid, t in zip(plan["ids"], plan["q_len"]):
            rid, t = int(rid), int(t)
            lv = self.live[rid]
            r = lv.rec
            if r["state"] == SWAPPED:
                resume_blocks += -(-r["ctx_len"] // BLOCK)
            have = 0 if r["state"] == SWAPPED else r["blocks_on_gpu"]
            need_total = -(-(r["ctx_len"] + t) // BLOCK)
            self.free -= need_total - have
            assert self.free >= 0, "former scheduled more blocks than exist"
            r["blocks_on_gpu"] = need_total
            r["last_sched"] = self.now
            lv.admitted = True
            r["state"] = RUNNING
            if r["pending"] > 0:
                r["ctx_len"] += t
                r["pending"] -= t
                if lv.logical_ctx < r["ctx_len"]:
                    lv.logical_ctx = r["ctx_len"]
            else:
                r["ctx_len"] += 1
                lv.logical_ctx = r["ctx_len"]
                lv.generated += 1
                self.first_token.setdefault(rid, self.now)
            ids.append(rid)
            qls.append(t)
            ctxs.append(r["ctx_len"])
            batch_q += t
            batch_ctx += r["ctx_len"]
        dt = self.cfg.t0 + self.cfg.per_query_token * batch_q + self.cfg.per_context_token * batch_ctx
        end = self.now + dt
        for rid in ids:
            lv = self.live[rid]
            r = lv.rec
            if r["pending"] > 0:
                continue
            seg_end = lv.tr.call_after[lv.seg_index] if lv.seg_index < len(lv.tr.call_after) else lv.tr.output
            if r["pending"] == 0 and lv.generated >= seg_end:
                if lv.seg_index < len(lv.tr.call_after):
                    r.update(state=PAUSED, cur_policy=policy[rid], pause_start=end)
                    lv.pause_end = end + lv.tr.pause[lv.seg_index]
                else:
                    finished.append(rid)
        for rid in finished:
            lv = self.live.pop(rid)
            self.free += lv.rec["blocks_on_gpu"]
            self.done[rid] = (lv.tr.arrival, self.first_token.get(rid, end), end)
        rec = StepRecord(now=self.now, budget=int(plan["budget"]), ids=ids, q_len=qls, ctx_len=ctxs,
                         n_resume=len(plan["resume_ids"]), n_park=len(plan["park_ids"]),
                         n_free=len(plan["free_ids"]), resume_blocks=resume_blocks,
                         park_blocks=park_blocks)
        if ids:
            self.now = end
        else:
            t = self.next_event_time()
            if t is None:
                # Nothing fits and no pause or arrival will change that: every
                # block is held by runnable requests. Like an engine preempting by
                # recomputation, drop the KV of the latest-arriving holder, sparing
                # the requests that ran in the previous iteration (so a request is
                # never dropped right after it was given blocks) unless no other
                # holder is left.
                holders = [lv for lv in self.live.values()
                           if lv.rec["state"] in (RUNNING, SWAPPED, WAITING) and lv.rec["blocks_on_gpu"] > 0]
                if not holders:
                    raise RuntimeError("serving loop cannot make progress (a request exceeds the pool)")
                idle = [lv for lv in holders if lv.tr.id not in self.last_ids]
                v = max(idle or holders, key=lambda lv: (lv.tr.arrival, lv.tr.id))
                self.free += v.rec["blocks_on_gpu"]
                v.rec.update(state=WAITING, blocks_on_gpu=0, ctx_len=0, pending=v.logical_ctx + v.rec["pending"])
                self.preemptions += 1
                if self.preemptions > self.cfg.max_preemptions:
                    raise RuntimeError("serving loop is thrashing: the pool is far smaller than the "
                                       "contexts the scheduled requests need")
                t = end
            self.now = max(end, t)
        if ids:
            self.last_ids = set(ids)
        self.steps.append(rec)
        return rec

    def metrics(self, slo_ttft: float = 1.0, slo_norm: Optional[float] = None) -> dict:
        """Request-level results of the finished requests: time to first token
        (queueing included), normalized latency (end-to-end latency over output
        tokens) and goodput (requests per second meeting both SLOs, over the
        time from the first arrival to the last completion). The default
        normalized-latency SLO is ten times the model's base iteration time."""
        if slo_norm is None:
            slo_norm = 10.0 * self.cfg.t0
        ids = sorted(self.done)
        if not ids:
            return dict(finished=0, ttft_mean=None, ttft_p50=None, ttft_p99=None, norm_latency_mean=None,
                        goodput=0.0, slo_ttft=slo_ttft, slo_norm=slo_norm)
        out_len = {t.id: t.output for t in self.trace}
        ttft = np.array([self.done[i][1] - self.done[i][0] for i in ids])
        norm = np.array([(self.done[i][2] - self.done[i][0]) / max(1, out_len[i]) for i in ids])
        span = max(self.done[i][2] for i in ids) - min(self.done[i][0] for i in ids)
        good = int(np.count_nonzero((ttft < slo_ttft) & (norm < slo_norm)))
        return dict(finished=len(ids), ttft_mean=float(ttft.mean()), ttft_p50=float(np.median(ttft)),
                    ttft_p99=float(np.percentile(ttft, 99)), norm_latency_mean=float(norm.mean()),
                    goodput=good / span if span > 0 else 0.0, slo_met=good, slo_ttft=slo_ttft,
                    slo_norm=slo_norm)

    def run(self, former: Callable, max_steps: Optional[int] = None) -> List[StepRecord]:
        n = 0
        while self.live or self.next_arrival < len(self.trace):
            if self.step(former) is None:
                break
            n += 1
            if max_steps is not None and n >= max_steps:
                break
            if n >= self.cfg.max_iters:
                raise RuntimeError("serving loop exceeded its iteration cap")
        return self.steps
