"""The serving loop over a synthetic augmented trace, driven by the oracle
former and the C++ former in lock step (CPU only)."""

import os

import numpy as np
import pytest

import paper_2512_04013_amd as aug
from oracle import former as of
from synth import sweep
from synth.trace import PAUSED, ServingLoop, SimConfig, make_trace
from tests.former_drivers import library_former, lockstep, oracle_former

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
    loop = ServingLoop(trace, SimConfig(num_blocks=blocks))
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
    loop = ServingLoop(trace, SimConfig(num_blocks=384))

    def checked(recs, free, now):
        plan = lib(recs, free, now)
        paused = {r["id"] for r in recs if r["state"] == PAUSED}
        assert not (set(int(i) for i in plan["ids"]) & paused)
        return plan

    loop.run(checked)
    assert len(loop.done) == len(trace)


def test_a_pool_far_too_small_is_reported_not_looped_on():
    trace = small_trace(seed=256)
    loop = ServingLoop(trace, SimConfig(num_blocks=256, max_preemptions=200))
    with pytest.raises(RuntimeError, match="thrashing"):
        loop.run(library_former(params_for(256, False)))


@pytest.mark.parametrize("budget", [256, 8192])
def test_lock_step_on_a_prefix_of_the_full_size_trace(budget):
    """2000 requests with the full-size length distributions and a 16,384-block
    pool; the first 400 iterations (the whole trace is about 25k iterations,
    too long for the pure-Python former in the CPU suite)."""
    trace = make_trace(n=2000, seed=1, rate=3.0)
    p = params_for(budget, True)
    loop = ServingLoop(trace, SimConfig(num_blocks=16384))
    steps = loop.run(lockstep(oracle_former(p), library_former(p)), max_steps=400)
    assert len(steps) == 400
    assert all(sum(s.q_len) <= s.budget for s in steps)


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

    loop = ServingLoop(make_trace(n=2000, seed=2), SimConfig(num_blocks=16384))
    assert len(loop.run(both, max_steps=300)) == 300


def test_sweep_budgets_from_512_serve_the_whole_trace():
    """Every request of the 2000-request trace finishes under budget 512 with
    the 16,384-block pool; budget 256 overloads it (the loop stops early)."""
    from paper_2512_04013_amd import runtime as rt
    run = sweep.run_budget(512, rt.serving_former(**sweep.former_params(512)))
    assert run.complete and run.finished == 2000
    assert all(sum(s.q_len) <= s.budget for s in run.steps)
    small = sweep.run_budget(256, rt.serving_former(**sweep.former_params(256)), max_steps=2000)
    assert not small.complete
