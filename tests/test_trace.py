"""The serving loop over a synthetic augmented trace, driven by the oracle
former and the C++ former in lock step (CPU only)."""

import os

import numpy as np
import pytest

import paper_2512_04013_amd as aug
from oracle import former as of
from synth.trace import PAUSED, ServingLoop, SimConfig, make_trace
from tests.former_drivers import library_former, lockstep, oracle_former

pytestmark = pytest.mark.skipif(not os.path.exists(aug.LIB_PATH), reason="libaug.so not built")


def params_for(budget, dynamic):
    return of.Params(beta=5e-5, t_max=budget, beta_low=0.5 if dynamic else 1.0,
                     beta_high=2.0 if dynamic else 1.0, chunk_cap=512, t_iter=0.02, fwd_a=0.0175,
                     fwd_b=20.5e-9, swap_s_per_tok=4.1e-8, n_fwd_max=1)


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
