"""Pins of the batch-former oracle: hand-worked budget, Waste and ranking
cases, the cost closed forms against step-by-step integration of memory
occupancy, and the knapsack half-approximation by brute force (CPU only)."""

import itertools
import math

import numpy as np
import pytest

from oracle import former as of
from oracle.former import (DISCARD, NONE, PAUSED, PRESERVE, RUNNING, SWAP, SWAPPED,
                           WAITING, Params, Request)


# ---- Eq. token -----------------------------------------------------------------------

def test_budget_hand_cases():
    p = Params(t_max=2048, beta_low=0.5, beta_high=2.0)
    assert of.token_budget(p, 100, 20, 16) == 1920
    assert of.token_budget(p, 3, 0, 16) == 1024          # raw 48 -> low clip
    assert of.token_budget(p, 62500, 0, 16) == 4096      # raw 1e6 -> high clip
    static = Params(t_max=2048, beta_low=1.0, beta_high=1.0)
    assert of.token_budget(static, 100, 20, 16) == 2048
    assert of.token_budget(Params(t_max=1000, beta_low=0.33, beta_high=1.5), 0, 0, 16) == 330


def test_budget_counts_only_preemptable_paused_blocks():
    p = Params(t_max=256, beta_low=0.0, beta_high=100.0)
    reqs = [Request(id=0, arrival=0.0, state=PAUSED, cur_policy=SWAP, blocks_on_gpu=5),
            Request(id=1, arrival=0.0, state=PAUSED, cur_policy=DISCARD, blocks_on_gpu=7),
            Request(id=2, arrival=0.0, state=PAUSED, cur_policy=PRESERVE, blocks_on_gpu=11),
            Request(id=3, arrival=0.0, state=RUNNING, ctx_len=10, blocks_on_gpu=1, pred_out=3)]
    plan = of.form_batch(reqs, free_blocks=4, block_size=16, now=1.0, p=p)
    assert plan.budget == (4 + 5 + 7) * 16


# ---- Appendix B -----------------------------------------------------------------------

def test_waste_argmin_cases():
    p = Params(fwd_a=0.01, fwd_b=1e-6, swap_s_per_tok=1e-5, n_fwd_max=1)
    assert of.select_policy(p, 1000, 0.0, 0) == PRESERVE                  # instant call
    cheap_recompute = Params(fwd_a=1e-6, fwd_b=0.0, swap_s_per_tok=1.0, n_fwd_max=1)
    assert of.select_policy(cheap_recompute, 1000, 100.0, 0) == DISCARD
    cheap_swap = Params(fwd_a=1.0, fwd_b=0.0, swap_s_per_tok=1e-9, n_fwd_max=1)
    assert of.select_policy(cheap_swap, 1000, 100.0, 0) == SWAP
    # all three equal -> the first listed (Preserve); Discard/Swap tie -> Discard
    tie = Params(fwd_a=0.5, fwd_b=0.0, swap_s_per_tok=0.25 / 1000, n_fwd_max=1)
    assert of.waste(tie, 1000, 0.5, 0) == (500.0, 500.0, 0.5)
    tie2 = Params(fwd_a=0.5, fwd_b=0.0, swap_s_per_tok=0.25, n_fwd_max=1000)
    w = of.waste(tie2, 1000, 0.5, 0)
    assert w[0] == w[1] == 500.0 and w[2] == 2.0 * 250.0 * 1000.0
    assert of.select_policy(tie2, 1000, 0.5, 0) == PRESERVE
    tie3 = Params(fwd_a=0.5, fwd_b=0.0, swap_s_per_tok=0.25 / 1000, n_fwd_max=1000)
    assert of.waste(tie3, 1000, 9.0, 0)[1:] == (500.0, 500.0)
    assert of.select_policy(tie3, 1000, 9.0, 0) == DISCARD
    # other runnable context makes Discard dearer (interference term)
    p2 = Params(fwd_a=0.01, fwd_b=0.0, swap_s_per_tok=1.0, n_fwd_max=1)
    assert of.select_policy(p2, 100, 0.02, 0) == DISCARD
    assert of.select_policy(p2, 100, 0.02, 10_000) == PRESERVE


# ---- Eq. cost against step-by-step integration -------------------------------------------

def _integrate_segment(p, r, policy):
    """Step the segment iteration by iteration, adding memory x t_iter after each
    iteration, then the call phase: an independent statement of the integral."""
    token_iters = 0.0
    mem = r.seg_ctx
    if r.seg >= 2 and r.prev_policy == DISCARD:        # recompute the context from nothing
        mem = 0
        left = r.seg_ctx
        while left > 0:
            step = min(left, p.chunk_cap)
            mem += step
            left -= step
            token_iters += mem * p.t_iter
    extra = 0.0
    if r.seg >= 2 and r.prev_policy == SWAP:
        extra += p.swap_s_per_tok * r.seg_ctx * r.seg_ctx
    left = r.seg_prefill
    while left > 0:
        step = min(left, p.chunk_cap)
        mem += step
        left -= step
        token_iters += mem * p.t_iter
    for _ in range(r.pred_out):
        mem += 1
        token_iters += mem * p.t_iter
    if policy == PRESERVE:
        extra += r.pred_call * mem
    elif policy == SWAP:
        extra += p.swap_s_per_tok * mem * mem
    return token_iters + extra


@pytest.mark.parametrize("seg,prev", [(1, NONE), (2, PRESERVE), (2, DISCARD), (3, SWAP)])
@pytest.mark.parametrize("has_call", [0, 1])
def test_segment_cost_equals_stepwise_integral(seg, prev, has_call):
    rng = np.random.default_rng(seg * 7 + prev + 13 * has_call)
    p = Params(chunk_cap=128, t_iter=0.017, fwd_a=0.01, fwd_b=3e-6, swap_s_per_tok=4e-6)
    for _ in range(20):
        r = Request(id=1, arrival=0.0, seg=seg, prev_policy=prev,
                    seg_ctx=0 if seg == 1 else int(rng.integers(1, 3000)),
                    seg_prefill=int(rng.integers(1, 1500)), pred_out=int(rng.integers(1, 400)),
                    pred_call=float(rng.uniform(0.01, 3.0)), has_next_call=has_call)
        c, pol = of.segment_cost(p, r, int(rng.integers(0, 50000)))
        assert (pol == NONE) == (not has_call)
        assert math.isclose(c, _integrate_segment(p, r, pol), rel_tol=1e-12)


def test_prefill_cost_hand_example():
    p = Params(chunk_cap=512, t_iter=0.5)
    # 1100 tokens onto 100: chunks end at 612, 1124, 1200 -> 2936 token-iterations
    assert of.prefill_cost(p, 100, 1100) == 2936 * 0.5
    assert of.decode_cost(p, 10, 3) == (11 + 12 + 13) * 0.5


# ---- ranking --------------------------------------------------------------------------

def _running(i, ctx, out, arrival=0.0, last=-1.0):
    return Request(id=i, arrival=arrival, last_sched=last, state=RUNNING, seg_ctx=0,
                   seg_prefill=ctx, pred_out=out, ctx_len=ctx, blocks_on_gpu=-(-ctx // 16) + 1)


def test_beta_zero_orders_by_ascending_cost():
    p = Params(beta=0.0, t_max=10_000, beta_low=1, beta_high=1)
    rng = np.random.default_rng(0)
    reqs = [_running(i, int(rng.integers(10, 2000)), int(rng.integers(1, 300)),
                     arrival=float(rng.uniform(0, 5))) for i in range(40)]
    plan = of.form_batch(reqs, free_blocks=10**6, block_size=16, now=10.0, p=p)
    costs = [plan.cost[i] for i in plan.ids]
    assert len(plan.ids) == 40 and costs == sorted(costs)


def test_equal_cost_longest_waiting_first():
    p = Params(beta=5e-5, t_max=10_000, beta_low=1, beta_high=1)
    reqs = [_running(i, 100, 10, arrival=0.0, last=float(s)) for i, s in
            enumerate([3.0, 1.0, 2.5, 0.5, 4.0])]
    plan = of.form_batch(reqs, free_blocks=10**6, block_size=16, now=5.0, p=p)
    assert plan.ids == [3, 1, 2, 0, 4]
    # never scheduled: w counts from arrival, so FCFS
    reqs = [Request(id=i, arrival=a, state=WAITING, seg_prefill=100, pending=100, pred_out=10)
            for i, a in enumerate([0.3, 0.1, 0.2])]
    plan = of.form_batch(reqs, free_blocks=10**6, block_size=16, now=1.0, p=p)
    assert plan.ids == [1, 2, 0]
    # exact ties fall back to arrival, then id
    reqs = [Request(id=i, arrival=0.0, state=WAITING, seg_prefill=100, pending=100, pred_out=10)
            for i in (7, 3, 5)]
    assert of.form_batch(reqs, 10**6, 16, 1.0, p).ids == [3, 5, 7]


def test_fcfs_ranks_by_arrival_whatever_the_cost():
    rng = np.random.default_rng(3)
    reqs = [_running(i, int(rng.integers(10, 2000)), int(rng.integers(1, 300)),
                     arrival=float(rng.uniform(0, 5)), last=float(rng.uniform(5, 6))) for i in range(30)]
    p = Params(t_max=10_000, beta_low=1, beta_high=1, order=of.ORDER_FCFS)
    plan = of.form_batch(reqs, free_blocks=10**6, block_size=16, now=10.0, p=p)
    assert plan.ids == [r.id for r in sorted(reqs, key=lambda r: r.arrival)]
    # theta order differs on the same requests, so the key really changed
    theta_plan = of.form_batch(reqs, 10**6, 16, 10.0, Params(t_max=10_000, beta_low=1, beta_high=1))
    assert theta_plan.ids != plan.ids and sorted(theta_plan.ids) == sorted(plan.ids)


def test_ssjf_ranks_by_predicted_output_then_arrival():
    outs = [300, 50, 50, 1000, 2, 50]
    reqs = [_running(i, 100 + 37 * i, o, arrival=float(5 - i)) for i, o in enumerate(outs)]
    p = Params(t_max=10_000, beta_low=1, beta_high=1, order=of.ORDER_SSJF)
    plan = of.form_batch(reqs, free_blocks=10**6, block_size=16, now=10.0, p=p)
    # pred_out 2, then the three 50s by arrival (ids 5, 2, 1 arrived at 0, 3, 4), then 300, 1000
    assert plan.ids == [4, 5, 2, 1, 0, 3]


def test_prefill_takes_one_chunk_capped_by_chunk_cap_and_budget():
    # a 1500-token prompt runs 512 tokens per iteration; with a 300-token
    # budget the chunk is cut to the budget, so it can still run alone
    r = Request(id=0, arrival=0.0, state=WAITING, seg_prefill=1500, pending=1500, pred_out=10)
    plan = of.form_batch([r], free_blocks=10**6, block_size=16, now=1.0,
                         p=Params(t_max=2048, beta_low=1, beta_high=1, chunk_cap=512))
    assert plan.q_len == [512]
    plan = of.form_batch([r], free_blocks=10**6, block_size=16, now=1.0,
                         p=Params(t_max=300, beta_low=1, beta_high=1, chunk_cap=512))
    assert plan.budget == 300 and plan.q_len == [300]
    # the last chunk takes what is left
    r2 = Request(id=1, arrival=0.0, state=RUNNING, seg_prefill=1500, ctx_len=1024, pending=476,
                 blocks_on_gpu=64, pred_out=10)
    plan = of.form_batch([r2], free_blocks=10**6, block_size=16, now=1.0,
                         p=Params(t_max=2048, beta_low=1, beta_high=1, chunk_cap=512))
    assert plan.q_len == [476]


# ---- packing ---------------------------------------------------------------------------

def _mixed_2048_requests(extra_decode=False):
    rng = np.random.default_rng(42)
    reqs = []
    for i in range(3):
        prior = int(rng.integers(0, 4097))
        reqs.append(Request(id=i, arrival=0.1 * i, state=WAITING, seg_prefill=prior + 512,
                            ctx_len=prior, pending=512, pred_out=100,
                            blocks_on_gpu=-(-prior // 16)))
    for i in range(3, 515 + int(extra_decode)):
        ctx = int(np.clip(np.rint(rng.lognormal(np.log(1500), 0.8)), 1, 8192))
        swapped = rng.random() < 0.3
        reqs.append(Request(id=i, arrival=0.01 * i, last_sched=1.0, state=SWAPPED if swapped else RUNNING,
                            seg_prefill=ctx, ctx_len=ctx, pred_out=50,
                            blocks_on_gpu=0 if swapped else -(-ctx // 16)))
    return reqs


def test_mixed_budget_2048_selects_all_515():
    p = Params(t_max=2048, beta_low=0.5, beta_high=1.0, chunk_cap=512)
    reqs = _mixed_2048_requests()
    plan = of.form_batch(reqs, free_blocks=131_072, block_size=16, now=2.0, p=p)
    assert plan.budget == 2048 and len(plan.ids) == 515 and sum(plan.q_len) == 2048
    assert sorted(plan.q_len)[-3:] == [512, 512, 512]
    assert sorted(plan.resume_ids) == sorted(r.id for r in reqs if r.state == SWAPPED)


def test_one_more_decode_is_excluded_by_break():
    p = Params(t_max=2048, beta_low=0.5, beta_high=1.0, chunk_cap=512)
    reqs = _mixed_2048_requests(extra_decode=True)
    plan = of.form_batch(reqs, free_blocks=131_072, block_size=16, now=2.0, p=p)
    assert len(plan.ids) == 515 and sum(plan.q_len) == 2048
    theta = {i: t for i, t in zip(plan.ids, plan.theta)}
    left = [r.id for r in reqs if r.id not in theta][0]
    assert min(theta.values()) >= of.priority(p, plan.cost[left], of.waiting_ms(reqs[left], 2.0))


def test_break_stops_where_skip_continues():
    p = Params(beta=0.0, t_max=100, beta_low=1, beta_high=1, chunk_cap=512)
    # ranked by cost: a(60 tok) < b(50 tok, dearer) < c(1 tok decode, dearest)
    reqs = [Request(id=0, arrival=0.0, state=WAITING, seg_prefill=60, pending=60, pred_out=1),
            Request(id=1, arrival=0.0, state=WAITING, seg_prefill=50, pending=50, pred_out=40),
            Request(id=2, arrival=0.0, state=RUNNING, seg_prefill=900, ctx_len=900, pred_out=90,
                    blocks_on_gpu=57)]
    stop = of.form_batch(reqs, 1000, 16, 1.0, p)
    assert stop.ids == [0]
    p.skip_instead_of_break = 1
    skip = of.form_batch(reqs, 1000, 16, 1.0, p)
    assert skip.ids == [0, 2]


def test_block_shortage_evicts_longest_remaining_pause_first():
    p = Params(beta=0.0, t_max=4096, beta_low=1, beta_high=1, chunk_cap=512)
    reqs = [Request(id=10, arrival=0.0, state=PAUSED, cur_policy=SWAP, blocks_on_gpu=8,
                    pred_call=2.0, pause_start=0.5),           # remaining 1.5
            Request(id=11, arrival=0.0, state=PAUSED, cur_policy=DISCARD, blocks_on_gpu=8,
                    pred_call=3.0, pause_start=0.0),           # remaining 2.0
            Request(id=12, arrival=0.0, state=PAUSED, cur_policy=PRESERVE, blocks_on_gpu=50,
                    pred_call=9.0, pause_start=0.0),
            Request(id=1, arrival=0.0, state=WAITING, seg_prefill=300, pending=300, pred_out=5)]
    plan = of.form_batch(reqs, free_blocks=12, block_size=16, now=1.0, p=p)
    # needs 19 blocks: 12 free + Discard victim (8) is enough
    assert plan.ids == [1] and plan.free_ids == [11] and plan.park_ids == []
    plan = of.form_batch(reqs, free_blocks=4, block_size=16, now=1.0, p=p)
    assert plan.ids == [1] and plan.free_ids == [11] and plan.park_ids == [10]
    plan = of.form_batch(reqs, free_blocks=2, block_size=16, now=1.0, p=p)
    assert plan.ids == [] and plan.free_ids == [] and plan.park_ids == []


def test_form_batch_packing_is_the_plain_greedy_when_blocks_are_ample():
    rng = np.random.default_rng(7)
    p = Params(t_max=3000, beta_low=1, beta_high=1, chunk_cap=256)
    reqs = []
    for i in range(60):
        if rng.random() < 0.3:
            n = int(rng.integers(1, 900))
            reqs.append(Request(id=i, arrival=float(rng.uniform(0, 3)), state=WAITING,
                                seg_prefill=n, pending=n, pred_out=int(rng.integers(1, 200))))
        else:
            c = int(rng.integers(1, 4000))
            reqs.append(Request(id=i, arrival=float(rng.uniform(0, 3)), state=RUNNING,
                                seg_prefill=c, ctx_len=c, pred_out=int(rng.integers(1, 200)),
                                blocks_on_gpu=-(-c // 16) + 1))
    plan = of.form_batch(reqs, 10**7, 16, 4.0, p)
    ranked = sorted(range(60), key=lambda i: (-of.priority(p, plan.cost[i], of.waiting_ms(reqs[i], 4.0)),
                                             reqs[i].arrival, reqs[i].id))
    sizes = [of.tokens_of(p, reqs[i], plan.budget) for i in ranked]
    chosen = of.greedy_pack(sizes, plan.budget)
    assert plan.ids == [reqs[ranked[c]].id for c in chosen]


# ---- Appendix F: the better of break-greedy and the best singleton is >= OPT/2 --------------

def test_density_greedy_half_approximation_by_brute_force():
    rng = np.random.default_rng(123)
    for _ in range(3000):
        n = int(rng.integers(1, 11))
        c = rng.integers(1, 60, size=n)
        v = rng.uniform(0.1, 10.0, size=n)
        budget = int(rng.integers(1, 150))
        feasible = [i for i in range(n) if c[i] <= budget]      # infeasible singletons removed
        if not feasible:
            continue
        order = sorted(feasible, key=lambda i: -v[i] / c[i])
        g = of.greedy_pack([int(c[i]) for i in order], budget)
        v_g = sum(v[order[i]] for i in g)
        v_s = max(v[i] for i in feasible)
        opt = 0.0
        for mask in itertools.product([0, 1], repeat=n):
            if sum(c[i] for i in range(n) if mask[i]) <= budget:
                opt = max(opt, sum(v[i] for i in range(n) if mask[i]))
        assert v_g + v_s >= opt - 1e-9
        assert max(v_g, v_s) >= opt / 2 - 1e-9
