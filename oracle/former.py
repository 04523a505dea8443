"""Oracle for the token-budget batch former (pure Python, float64).

Follows the paper's scheduler in its own order:

* Waste of each context-handling policy during an external call and the
  policy that minimises it (Appendix B, Eqs. waste_preserve, waste_discard,
  waste_swap, waste_si; ties resolved in the order the paper lists the
  policies: Preserve, Discard, Swap);
* the space-time cost C_{i,k} as the integral of memory occupancy over the
  segment (Eq. cost), built before the first call from predictions
  (Eq. context_policy and the C_{i,1} / C^call equations) and after a call
  returns from the realised policy and return length (Eqs. c_fb, c_ik_new);
* the value V = 1 + beta * w (Eq. value) and the priority theta = V / C
  (Eq. theta), w being the time since the request was last scheduled;
* the dynamic token budget B = floor((G_free + G_preempt) / mu), clipped to
  [beta_low * T_max, beta_high * T_max] (Eq. token; Algorithm 1 step (3));
* ranking by theta and greedy packing that stops at the first request that
  does not fit (Algorithm 1 step (4)).

Readings of points the paper leaves open (all of them also listed in the
design notes):

* memory occupancy m(t) is counted in KV tokens and time in seconds; one
  engine iteration lasts ``t_iter``; memory is counted after each iteration's
  tokens are added, so a prefill of X tokens onto L0 cached ones in chunks of
  ``chunk_cap`` costs t_iter * sum_{j=1..ceil(X/cap)} (L0 + min(j*cap, X)),
  and l decode steps from L0 cost t_iter * sum_{j=1..l} (L0 + j);
* the per-token footprint M (or mu) is one token, so it drops out of Waste and
  the budget is (G_free + G_preempt) * block_size tokens when G is counted in
  blocks;
* tau_fwd(L) = fwd_a + fwd_b * L and tau_swap(L) = swap_s_per_tok * L;
  L_other is the summed context of the other runnable requests;
* swap-out / swap-in cost tau_swap(L) * L, recomputation costs a prefill of
  the whole context from nothing, and the return-token cost is a prefill of
  the returned tokens onto the context;
* w is measured in milliseconds (beta = 5e-5 is the paper's default);
* candidates are the running, swapped and waiting queues; a request
  contributes min(pending, chunk_cap, B) tokens (at least 1) while it has
  prompt, returned or recompute tokens pending, else 1 decode token, so a
  prefill chunk never exceeds the budget on its own; active tokens start at 0;
* ties in theta go to the earlier arrival, then the smaller id;
* a request also needs ceil((ctx + tokens) / block) pool blocks beyond those
  it holds (all of them if swapped out); if free plus reclaimable blocks
  cannot cover it, it is passed over for this iteration and packing goes on
  (the algorithm's stop is the token-budget test alone; memory enters it
  through the budget). Blocks are reclaimed lazily from
  paused Swap/Discard requests, longest predicted remaining pause first
  (ties by id): Swap victims are parked, Discard victims are freed;
* ``skip_instead_of_break`` replaces the stop with a skip (the greedy of the
  approximation appendix, which adds every request that fits);
* ``order`` swaps the ranking key for the baselines the paper compares
  against: FCFS ranks by arrival, SSJF by the predicted output length of the
  current segment (shortest first); both break ties like theta does.

Steps (1) and (2) of Algorithm 1 change a request's record: on arrival it
waits to prefill its prompt in segment 1 (``arrive``); when an external call
returns, the next segment starts from the realised policy of the wait, which
decides the queue it rejoins and what it must prefill (``on_return``).

All arithmetic is on Python floats (IEEE binary64) and ints, in a fixed order,
so the C++ former reproduces it bit for bit.
"""

from __future__ import annotations

import dataclasses
import math
from typing import List

WAITING, RUNNING, SWAPPED, PAUSED = 0, 1, 2, 3
NONE, PRESERVE, DISCARD, SWAP = 0, 1, 2, 3
ORDER_THETA, ORDER_FCFS, ORDER_SSJF = 0, 1, 2


@dataclasses.dataclass
class Request:
    id: int
    arrival: float
    last_sched: float = -1.0      # < 0: never scheduled
    state: int = WAITING
    seg: int = 1                  # k
    prev_policy: int = NONE       # realised policy of the previous wait (k >= 2)
    cur_policy: int = NONE        # PAUSED: policy chosen for the current wait
    seg_ctx: int = 0              # context at the segment start (before returned tokens)
    seg_prefill: int = 0          # prompt (k = 1) or returned tokens (k >= 2)
    pred_out: int = 1             # predicted tokens generated in this segment
    pred_call: float = 0.0        # predicted duration of the call ending it (s)
    has_next_call: int = 0
    ctx_len: int = 0              # tokens with KV now
    pending: int = 0              # tokens to prefill before the next decode
    blocks_on_gpu: int = 0
    pause_start: float = 0.0


@dataclasses.dataclass
class Params:
    beta: float = 5e-5
    t_max: int = 2048
    beta_low: float = 0.5
    beta_high: float = 2.0
    chunk_cap: int = 512
    t_iter: float = 0.02
    fwd_a: float = 0.015
    fwd_b: float = 2.0e-8
    swap_s_per_tok: float = 2.0e-6
    n_fwd_max: int = 1
    skip_instead_of_break: int = 0
    order: int = 0                # ORDER_THETA, ORDER_FCFS or ORDER_SSJF


@dataclasses.dataclass
class Plan:
    budget: int
    ids: List[int]
    q_len: List[int]
    theta: List[float]
    resume_ids: List[int]
    park_ids: List[int]
    free_ids: List[int]
    policy: List[int]            # per input request: predicted policy (NONE if not a candidate)
    cost: List[float]            # per input request: C (0.0 if not a candidate)


# ---- space-time cost pieces (Eq. cost under the readings above) -------------

def prefill_cost(p: Params, l0: int, x: int) -> float:
    if x <= 0:
        return 0.0
    n_chunks = -(-x // p.chunk_cap)
    token_iters = 0
    for j in range(1, n_chunks + 1):
        token_iters += l0 + min(j * p.chunk_cap, x)
    return float(token_iters) * p.t_iter


def decode_cost(p: Params, l0: int, n: int) -> float:
    token_iters = 0
    for j in range(1, n + 1):
        token_iters += l0 + j
    return float(token_iters) * p.t_iter


def fwd_time(p: Params, length: float) -> float:
    return p.fwd_a + p.fwd_b * length


def swap_time(p: Params, length: float) -> float:
    return p.swap_s_per_tok * length


# ---- Appendix B: waste of each policy and the argmin ------------------------

def waste(p: Params, l_tilde: int, tau_call: float, l_other: int):
    lt = float(l_tilde)
    w_preserve = tau_call * lt
    f = fwd_time(p, lt)
    w_discard = f * lt + f * float(l_other)
    w_swap = 2.0 * swap_time(p, lt) * float(p.n_fwd_max)
    return w_preserve, w_discard, w_swap


def select_policy(p: Params, l_tilde: int, tau_call: float, l_other: int) -> int:
    w_p, w_d, w_s = waste(p, l_tilde, tau_call, l_other)
    best, best_w = PRESERVE, w_p
    if w_d < best_w:
        best, best_w = DISCARD, w_d
    if w_s < best_w:
        best, best_w = SWAP, w_s
    return best


def call_cost(p: Params, policy: int, l_tilde: int, tau_call: float) -> float:
    lt = float(l_tilde)
    if policy == PRESERVE:
        return tau_call * lt
    if policy == SWAP:
        return swap_time(p, lt) * lt
    return 0.0


def resumption_cost(p: Params, prev_policy: int, l_ctx: int) -> float:
    if prev_policy == DISCARD:
        return prefill_cost(p, 0, l_ctx)
    if prev_policy == SWAP:
        return swap_time(p, float(l_ctx)) * float(l_ctx)
    return 0.0


def segment_cost(p: Params, r: Request, l_other: int):
    """(C_{i,k}, predicted policy) of the request's current segment."""
    l0 = r.seg_ctx
    x = r.seg_prefill
    l_tilde = l0 + x + r.pred_out
    if r.has_next_call:
        pol = select_policy(p, l_tilde, r.pred_call, l_other)
        c_call = call_cost(p, pol, l_tilde, r.pred_call)
    else:
        pol = NONE
        c_call = 0.0
    c_decode = decode_cost(p, l0 + x, r.pred_out)
    if r.seg <= 1:
        c_prefill = prefill_cost(p, l0, x)
        return (c_prefill + c_decode) + c_call, pol
    c_fb = prefill_cost(p, l0, x) + resumption_cost(p, r.prev_policy, l0)
    return (c_fb + c_decode) + c_call, pol


def waiting_ms(r: Request, now: float) -> float:
    since = r.last_sched if r.last_sched >= 0.0 else r.arrival
    return (now - since) * 1000.0


def priority(p: Params, c: float, w_ms: float) -> float:
    return (1.0 + p.beta * w_ms) / c


# ---- Eq. token ---------------------------------------------------------------

def token_budget(p: Params, free_blocks: int, preempt_blocks: int, block_size: int) -> int:
    raw = (free_blocks + preempt_blocks) * block_size
    lo = math.floor(p.beta_low * float(p.t_max))
    hi = math.floor(p.beta_high * float(p.t_max))
    return min(max(raw, lo), hi)


def tokens_of(p: Params, r: Request, budget: int) -> int:
    return min(r.pending, p.chunk_cap, max(1, budget)) if r.pending > 0 else 1


def greedy_pack(sizes, budget, skip_instead_of_break=False):
    """Indices chosen by scanning ``sizes`` in order (Algorithm 1 step (4))."""
    chosen, active = [], 0
    for i, s in enumerate(sizes):
        if active + s <= budget:
            chosen.append(i)
            active += s
        elif not skip_instead_of_break:
            break
    return chosen


# ---- the whole formation step ------------------------------------------------

def form_batch(reqs: List[Request], free_blocks: int, block_size: int, now: float,
               p: Params) -> Plan:
    cands = [i for i, r in enumerate(reqs) if r.state in (WAITING, RUNNING, SWAPPED)]
    total_ctx = 0
    for i in cands:
        total_ctx += reqs[i].ctx_len

    policy = [NONE] * len(reqs)
    cost = [0.0] * len(reqs)
    theta = {}
    for i in cands:
        r = reqs[i]
        c, pol = segment_cost(p, r, total_ctx - r.ctx_len)
        policy[i], cost[i] = pol, c
        theta[i] = priority(p, c, waiting_ms(r, now))

    victims = [i for i, r in enumerate(reqs)
               if r.state == PAUSED and r.cur_policy in (SWAP, DISCARD) and r.blocks_on_gpu > 0]
    preempt = 0
    for i in victims:
        preempt += reqs[i].blocks_on_gpu
    budget = token_budget(p, free_blocks, preempt, block_size)

    def remaining_pause(i):
        r = reqs[i]
        return r.pred_call - (now - r.pause_start)

    victims.sort(key=lambda i: (-remaining_pause(i), reqs[i].id))
    if p.order == ORDER_FCFS:
        ranked = sorted(cands, key=lambda i: (reqs[i].arrival, reqs[i].id))
    elif p.order == ORDER_SSJF:
        ranked = sorted(cands, key=lambda i: (reqs[i].pred_out, reqs[i].arrival, reqs[i].id))
    else:
        ranked = sorted(cands, key=lambda i: (-theta[i], reqs[i].arrival, reqs[i].id))

    free_now, reclaim_left, vi, active = free_blocks, preempt, 0, 0
    ids, q_len, th, resume_ids, park_ids, free_ids = [], [], [], [], [], []
    for i in ranked:
        r = reqs[i]
        t = tokens_of(p, r, budget)
        if active + t > budget:
            if p.skip_instead_of_break:
                continue
            break
        have = 0 if r.state == SWAPPED else r.blocks_on_gpu
        need = max(0, -(-(r.ctx_len + t) // block_size) - have)
        if need > free_now + reclaim_left:
            continue            # no memory for it now: not a budget stop, later ones may fit
        while need > free_now:
            v = reqs[victims[vi]]
            vi += 1
            free_now += v.blocks_on_gpu
            reclaim_left -= v.blocks_on_gpu
            (park_ids if v.cur_policy == SWAP else free_ids).append(v.id)
        free_now -= need
        active += t
        ids.append(r.id)
        q_len.append(t)
        th.append(theta[i])
        if r.state == SWAPPED:
            resume_ids.append(r.id)
    return Plan(budget, ids, q_len, th, resume_ids, park_ids, free_ids, policy, cost)


# ---- Algorithm 1, steps (1) and (2): the request record -------------------------

def arrive(id: int, arrival: float, prompt_tokens: int, pred_out: int, pred_call: float,
           has_next_call: int) -> Request:
    """A new request waits to prefill its prompt in its first segment."""
    return Request(id=id, arrival=arrival, last_sched=-1.0, state=WAITING, seg=1, prev_policy=NONE,
                   cur_policy=NONE, seg_ctx=0, seg_prefill=prompt_tokens, pred_out=pred_out,
                   pred_call=pred_call if has_next_call else 0.0, has_next_call=1 if has_next_call else 0,
                   ctx_len=0, pending=prompt_tokens, blocks_on_gpu=0, pause_start=0.0)


def on_return(r: Request, realised: int, context_tokens: int, ret_tokens: int, pred_out: int,
              pred_call: float, has_next_call: int) -> Request:
    """The record after the external call of a paused request returned:
    the next segment starts at the full context and prefills the returned
    tokens; the realised policy of the wait decides the queue (Preserve:
    running; Swap: swapped; Discard: waiting, recomputing the whole context)."""
    assert r.state == PAUSED
    out = dataclasses.replace(r, seg=r.seg + 1, prev_policy=realised, cur_policy=NONE,
                              seg_ctx=context_tokens, seg_prefill=ret_tokens, pred_out=pred_out,
                              pred_call=pred_call if has_next_call else 0.0,
                              has_next_call=1 if has_next_call else 0)
    if realised == PRESERVE:
        out.state, out.pending = RUNNING, ret_tokens
    elif realised == SWAP:
        out.state, out.pending = SWAPPED, ret_tokens
    else:
        out.state, out.ctx_len, out.blocks_on_gpu = WAITING, 0, 0
        out.pending = context_tokens + ret_tokens
    return out
