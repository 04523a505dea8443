"""The serving loop over a synthetic augmented trace, driven by the oracle
former and the C++ former in lock step (CPU only)."""

import os

import numpy as np
import pytest

import paper_2512_04013_amd as aug
from oracle import former as of
from synth import sweep
from synth.trace import PAUSED, ServingLoop, SimConfig, make_trace
from tests.former_drivers import LockstepLifecycle, OracleLifecycle, library_former, lockstep, oracle_former

pytestmark = pytest.mark.skipif(not os.path.exists(aug.LIB_PATH), reason="libaug.so not built")


def params_for(budget, dynamic):
    return of.Params(**sweep.former_params(budget, dynamic))


def small_trace(seed, n=60):
    # short prompts, outputs and returns keep the pure-Python oracle former fast
    return make_trace(n=n, seed=seed, rate=6.0, prompt_median=150, out_median=30, ret_lo=20, ret_hi=200)


def test_trace_is_seeded_and_shaped():
    a, b = make_trace(n=300, seed=4), make_trace(n=300, seed=4)
    assert [(t.arrival, t.prompt, t.output, t.call_after, t.ret) for t in a] == \
           [(t.arrival, t.prompt, t.output, t.call_after, t.ret) for t in b]
    assert all(0 < c < t.output for t in a for c in t.call_after)
    assert all(len(t.call_after) <= 4 and len(t.pause) == len(t.ret) == len(t.call_after) for t in a)
    assert all(20 <= r <= 800 for t in a for r in t.ret)
    gaps = np.diff([t.arrival for t in a])
    assert 0.25 < gaps.mean() < 0.45          # Poisson at 3 requests per second


@pytest.mark.parametrize("budget,dynamic,blocks", [(256, False, 1024), (512, True, 384), (2048, True, 384),
                                                   (8192, True, 384)])
def test_loop_runs_both_formers_in_lock_step(budget, dynamic, blocks):
    trace = small_trace(seed=budget)
    p = params_for(budget, dynamic)
    loop = ServingLoop(trace, SimConfig(num_blocks=blocks), LockstepLifecycle())
    steps = loop.run(lockstep(oracle_former(p), library_former(p)))
    assert len(loop.done) == len(trace)
    assert all(sum(s.q_len) <= s.budget for s in steps)
    assert loop.free == blocks
    if dynamic:
        # the budget follows the free pool: below T_max only when memory is short
        assert min(s.budget for s in steps) >= budget // 2 and max(s.budget for s in steps) <= 2 * budget
    if blocks == 384:
        # memory pressure made the formers evict paused contexts at least once
        assert sum(s.n_park + s.n_free for s in steps) > 0


def test_paused_requests_are_never_scheduled():
    trace = small_trace(seed=9)
    p = params_for(1024, True)
    lib = library_former(p)
    loop = ServingLoop(trace, SimConfig(num_blocks=384), OracleLifecycle())

    def checked(recs, free, now):
        plan = lib(recs, free, now)
        paused = {r["id"] for r in recs if r["state"] == PAUSED}
        assert not (set(int(i) for i in plan["ids"]) & paused)
        return plan

    loop.run(checked)
    assert len(loop.done) == len(trace)


def test_whole_prompt_admission_offers_only_new_requests_that_fit():
    """With the admission rule on, every never-run request offered to the
    former has its whole prompt covered by the free blocks, after those of
    the new requests offered before it; the trace still completes, in lock
    step between the two formers."""
    from synth.trace import BLOCK, WAITING
    trace = small_trace(seed=11)
    p = params_for(1024, True)
    both = lockstep(oracle_former(p), library_former(p))
    loop = ServingLoop(trace, SimConfig(num_blocks=384, admit_whole_prompt=True), LockstepLifecycle())
    held_back = []

    def checked(recs, free, now):
        room = free
        offered = {r["id"] for r in recs}
        for r in recs:
            if r["state"] == WAITING and not loop.live[r["id"]].admitted:
                need = -(-(r["ctx_len"] + r["pending"]) // BLOCK)
                assert need <= room
                room -= need
        held_back.append(len(loop.live) - len(offered))
        return both(recs, free, now)

    loop.run(checked)
    assert len(loop.done) == len(trace)
    assert max(held_back) > 0          # the rule did hold requests back


def test_a_pool_far_too_small_is_reported_not_looped_on():
    trace = small_trace(seed=256)
    loop = ServingLoop(trace, SimConfig(num_blocks=48, max_preemptions=200), OracleLifecycle())
    with pytest.raises(RuntimeError, match="thrashing"):
        loop.run(library_former(params_for(256, False)))


@pytest.mark.parametrize("budget", [256, 8192])
def test_lock_step_on_a_prefix_of_the_full_size_trace(budget):
    """2000 requests with the full-size length distributions and a 16,384-block
    pool; the first 400 iterations (the whole trace is about 25k iterations,
    too long for the pure-Python former in the CPU suite)."""
    trace = make_trace(n=2000, seed=1, rate=3.0)
    p = params_for(budget, True)
    loop = ServingLoop(trace, SimConfig(num_blocks=16384), LockstepLifecycle())
    steps = loop.run(lockstep(oracle_former(p), library_former(p)), max_steps=400)
    assert len(steps) == 400
    assert all(sum(s.q_len) <= s.budget for s in steps)


def _lock_step_whole_trace(budget, dynamic, seed=0):
    """Serve the whole 2000-request sweep trace with both formers in lock
    step; returns (finished requests, iterations, whether the loop stopped
    because it was thrashing)."""
    p = params_for(budget, dynamic)
    loop = ServingLoop(make_trace(n=2000, seed=seed, rate=3.0),
                       SimConfig(num_blocks=sweep.POOL_BLOCKS, max_preemptions=200), LockstepLifecycle())
    try:
        loop.run(lockstep(oracle_former(p), library_former(p)))
        thrashing = False
    except RuntimeError as e:
        if "thrashing" not in str(e):
            raise
        thrashing = True
    return len(loop.done), len(loop.steps), thrashing


@pytest.mark.slow
def test_lock_step_over_the_whole_sweep_trace_at_every_budget():
    """The oracle former and the library's agree (ids, token counts, theta
    bit for bit, resume / park / free lists, policies, budgets) at every
    iteration of the whole 2000-request trace of the budget sweep, for every
    budget, in dynamic mode for trace seeds 0, 1 and 2 and in static mode for
    seed 0 (23k-25k iterations each). Every run serves all 2000 requests
    except static mode at budget 256: a budget pinned at 256 tokens cannot
    keep up with 3 requests per second, and both formers agree at every
    iteration until the loop reports thrashing. The 24 runs go to worker
    processes."""
    import concurrent.futures as cf
    import multiprocessing as mp
    jobs = [(b, True, seed) for seed in (0, 1, 2) for b in sweep.BUDGETS] + [(b, False, 0) for b in sweep.BUDGETS]
    jobs.sort(key=lambda j: (j[0] != 256, j[1]))     # the longest runs first
    workers = max(1, min(len(jobs), len(os.sched_getaffinity(0))))
    with cf.ProcessPoolExecutor(max_workers=workers, mp_context=mp.get_context("spawn")) as ex:
        results = list(ex.map(_lock_step_whole_trace, *zip(*jobs)))
    for (budget, dynamic, seed), (finished, iters, thrashing) in zip(jobs, results):
        if (budget, dynamic) == (256, False):
            assert thrashing and iters > 5000, (finished, iters)
        else:
            assert finished == 2000 and not thrashing, (budget, dynamic, seed, finished)
            assert iters > 20000, (budget, dynamic, seed, iters)


def test_serving_former_marshals_like_the_test_driver():
    """The runtime's former callable (used by the benchmark and the GPU sweep)
    returns the same plans as the test driver's, which is checked against the
    oracle above; first 300 iterations of the full-size trace."""
    from paper_2512_04013_amd import runtime as rt
    p = sweep.former_params(1024)
    product, driver = rt.serving_former(**p), library_former(of.Params(**p))

    def both(recs, free, now):
        a, b = product(recs, free, now), driver(recs, free, now)
        for k in ("ids", "q_len", "resume_ids", "park_ids", "free_ids", "policy"):
            assert list(a[k]) == list(b[k]), k
        assert a["budget"] == b["budget"]
        assert np.array_equal(np.asarray(a["theta"]).view(np.uint64), np.asarray(b["theta"]).view(np.uint64))
        return a

    loop = ServingLoop(make_trace(n=2000, seed=2), SimConfig(num_blocks=16384), rt.serving_lifecycle())
    assert len(loop.run(both, max_steps=300)) == 300


def test_every_sweep_budget_serves_the_whole_trace_with_its_own_batches():
    """Every request of the 2000-request trace finishes under every budget of
    the sweep (16,384-block pool, chunks capped at half the budget), and each
    budget forms batches of its own: the largest formed batch grows with the
    budget, and budgets 4096 and 8192 form prefill-dominated batches that no
    smaller budget can hold. A fixed 512-token chunk cap starves budget 256
    (a chunk then fits only in an empty batch), which the loop reports."""
    from paper_2512_04013_amd import runtime as rt
    largest, biggest_prefill = [], []
    for budget in sweep.BUDGETS:
        run = sweep.run_budget(budget, rt.serving_former(**sweep.former_params(budget)), rt.serving_lifecycle())
        assert run.complete and run.finished == 2000, budget
        assert all(sum(s.q_len) <= s.budget for s in run.steps)
        assert all(max(s.q_len) <= sweep.sweep_chunk_cap(budget) for s in run.steps)
        largest.append(max(sum(s.q_len) for s in run.steps))
        biggest_prefill.append(max(sum(q for q in s.q_len if q > 1) for s in run.steps))
    assert all(a < b for a, b in zip(largest, largest[1:])), largest
    assert biggest_prefill[-1] > biggest_prefill[-2] > 2048 >= biggest_prefill[2], biggest_prefill
    small = sweep.run_budget(256, rt.serving_former(**sweep.former_params(256, chunk_cap=512)),
                             rt.serving_lifecycle(), max_steps=2000)
    assert not small.complete


@pytest.mark.parametrize("order", [of.ORDER_FCFS, of.ORDER_SSJF])
def test_baseline_orders_run_both_formers_in_lock_step(order):
    trace = small_trace(seed=30 + order)
    p = of.Params(**sweep.former_params(1024, True, order=order))
    loop = ServingLoop(trace, SimConfig(num_blocks=384), LockstepLifecycle())
    steps = loop.run(lockstep(oracle_former(p), library_former(p)))
    assert len(loop.done) == len(trace)
    assert all(sum(s.q_len) <= s.budget for s in steps)


def test_request_records_match_the_oracle_on_every_transition_kind():
    """Arrival, and a return under each realised policy, through the library
    and the oracle, compared field by field."""
    lc = LockstepLifecycle()
    rec = lc.arrive(id=7, arrival=2.5, prompt_tokens=300, pred_out=150, pred_call=0.4, has_next_call=1)
    assert rec["state"] == of.WAITING and rec["pending"] == 300 and rec["seg"] == 1
    for realised, state in ((of.PRESERVE, of.RUNNING), (of.SWAP, of.SWAPPED), (of.DISCARD, of.WAITING)):
        paused = dict(rec, state=of.PAUSED, ctx_len=0 if realised == of.DISCARD else 460,
                      blocks_on_gpu=0 if realised != of.PRESERVE else 29, cur_policy=realised)
        out = lc.on_return(paused, realised=realised, context_tokens=460, ret_tokens=90, pred_out=50,
                           pred_call=0.0, has_next_call=0)
        assert out["state"] == state and out["seg"] == 2 and out["prev_policy"] == realised
        assert out["pending"] == (550 if realised == of.DISCARD else 90)
        assert out["seg_ctx"] == 460 and out["seg_prefill"] == 90 and out["pred_call"] == 0.0


def test_library_rejects_bad_record_transitions():
    from paper_2512_04013_amd import REQUEST_DTYPE, AugError
    with pytest.raises(AugError):
        aug.aug_request_arrive(1, 0.0, 0, 10, 0.0, 0)            # empty prompt
    rec = aug.aug_request_arrive(1, 0.0, 10, 10, 0.0, 0)
    with pytest.raises(AugError):
        aug.aug_request_return(rec, of.PRESERVE, 10, 5, 10, 0.0, 0)   # not paused
    rec["state"] = of.PAUSED
    with pytest.raises(AugError):
        aug.aug_request_return(rec, 9, 10, 5, 10, 0.0, 0)              # unknown policy
    assert REQUEST_DTYPE.itemsize > 0
