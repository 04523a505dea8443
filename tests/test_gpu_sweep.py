"""GPU parity on the token-budget sweep: batches that the library's former
forms from the 2000-request augmented trace under budgets 256 ... 8192, laid
out on the 64-query-head, 8-KV-head, head_dim 128 layer with bf16 queries and
an fp8 E4M3FN KV cache, run through the C ABI and compared with the oracle.

Per budget: the batch with the most query tokens, the one with the most
prefill query-key pairs, and one seeded random batch (identical batches of
different budgets are run once). Every row of every batch is compared with the
oracle; the most prefill-heavy batch of each budget also with sharp inputs
(K/V ~ N(0,1)).
"""

import pytest

torch = pytest.importorskip("torch")

from oracle import attention as oa  # noqa: E402
from synth import sweep  # noqa: E402
from tests.gpu_util import compare, say  # noqa: E402

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a GPU")]

@pytest.fixture(scope="module")
def formed_batches():
    from paper_2512_04013_amd import runtime as rt
    seen, cases = set(), []
    for budget in sweep.BUDGETS:
        run = sweep.run_budget(budget, rt.serving_former(**sweep.former_params(budget)), rt.serving_lifecycle())
        say(f"[sweep] budget {budget}: {len(run.steps)} batches, complete={run.complete}")
        assert run.complete
        picks = sweep.select_steps(run.steps, 1, seed=budget)
        for what in ("most_tokens", "most_prefill", "random0"):
            s = run.steps[picks[what]]
            key = (tuple(s.q_len), tuple(s.ctx_len))
            if key in seen:
                continue
            seen.add(key)
            cases.append((budget, what, s))
    return cases


def test_every_budget_contributes_batches(formed_batches):
    """Every budget forms batches of its own; the most prefill-heavy batches
    of budgets 4096 and 8192 hold more prefill rows than any smaller budget
    can (chunks are capped at half the budget)."""
    assert {b for b, _, _ in formed_batches} == set(sweep.BUDGETS)
    most_prefill = {b: sum(q for q in s.q_len if q > 1) for b, w, s in formed_batches if w == "most_prefill"}
    assert set(most_prefill) == set(sweep.BUDGETS)
    assert most_prefill[8192] > most_prefill[4096] > 2048 >= most_prefill[1024]


SLOTS = 18


@pytest.mark.parametrize("index", range(SLOTS))
def test_formed_batch_matches_oracle(formed_batches, index):
    assert len(formed_batches) <= SLOTS
    if index >= len(formed_batches):
        pytest.skip("fewer distinct batches than slots")
    budget, what, step = formed_batches[index]
    _check_step(budget, what, step, seed=1000 + index, sharp=False)


@pytest.mark.parametrize("budget", sweep.BUDGETS)
def test_most_prefill_batch_sharp(formed_batches, budget):
    (what, step), = [(w, s) for b, w, s in formed_batches if b == budget and w == "most_prefill"]
    _check_step(budget, what, step, seed=2000 + budget, sharp=True)


def _check_step(budget, what, step, seed, sharp):
    from paper_2512_04013_amd import runtime as rt
    b = sweep.batch_for_step(step, seed=seed, n_pool_blocks=sum(-(-c // 16) for c in step.ctx_len) + 64,
                             sharp=sharp)
    say(f"[sweep] budget={budget} {what} sharp={sharp}: {b.num_reqs} requests, {b.total_q} rows, "
        f"{int(b.ctx_len.sum())} keys")
    shape, kv, q, bids = rt.upload_batch(b, staging_bytes=1 << 20)
    att = rt.MixedAttention(shape, kv, b.q_start, b.ctx_len, b.bt_start, b.block_ids, bids)
    got = rt.to_host_f64(att.run(q))
    torch.cuda.synchronize()
    want = oa.attention_for(b)
    compare(got, want, "bf16", what=f"budget {budget} {what} sharp={sharp} (all {b.total_q} rows) "
                                    f"tiles={att.info.num_prefill_items} items={att.info.num_items}")
