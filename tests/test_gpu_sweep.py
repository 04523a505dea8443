"""GPU parity on the token-budget sweep: batches that the library's former
forms from the 2000-request augmented trace under budgets 256 ... 8192, laid
out on the 64-query-head, 8-KV-head, head_dim 128 layer with bf16 queries and
an fp8 E4M3FN KV cache, run through the C ABI and compared with the oracle.

Per budget: the batch with the most query tokens, the one with the most
prefill query-key pairs, and one seeded random batch (identical batches of
different budgets are run once). Every prefill request of a batch and up to 24
of its decodes are compared row by row.
"""

import numpy as np
import pytest

torch = pytest.importorskip("torch")

from oracle import attention as oa  # noqa: E402
from synth import sweep  # noqa: E402
from tests.gpu_util import compare, rows_of, say  # noqa: E402

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a GPU")]

# budgets far below what the trace needs overload the serving loop; a prefix
# of their iterations is enough to sample formed batches
MAX_STEPS = {256: 3000}


@pytest.fixture(scope="module")
def formed_batches():
    from paper_2512_04013_amd import runtime as rt
    seen, cases = set(), []
    for budget in sweep.BUDGETS:
        run = sweep.run_budget(budget, rt.serving_former(**sweep.former_params(budget)), rt.serving_lifecycle(),
                               max_steps=MAX_STEPS.get(budget, 40_000))
        say(f"[sweep] budget {budget}: {len(run.steps)} batches, complete={run.complete}")
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
    assert {b for b, _, _ in formed_batches} >= {256, 512, 1024, 2048}
    assert any(max(s.q_len) > 1 for _, _, s in formed_batches)


@pytest.mark.parametrize("index", range(16))
def test_formed_batch_matches_oracle(formed_batches, index):
    from paper_2512_04013_amd import runtime as rt
    if index >= len(formed_batches):
        pytest.skip("fewer distinct batches than slots")
    budget, what, step = formed_batches[index]
    b = sweep.batch_for_step(step, seed=1000 + index,
                             n_pool_blocks=sum(-(-c // 16) for c in step.ctx_len) + 64)
    say(f"[sweep] budget={budget} {what}: {b.num_reqs} requests, {b.total_q} rows, "
        f"{int(b.ctx_len.sum())} keys")
    shape, kv, q, bids = rt.upload_batch(b, staging_bytes=1 << 20)
    att = rt.MixedAttention(shape, kv, b.q_start, b.ctx_len, b.bt_start, b.block_ids, bids)
    got = rt.to_host_f64(att.run(q))
    torch.cuda.synchronize()
    pre = [r for r in range(b.num_reqs) if b.q_len[r] > 1]
    dec = [r for r in range(b.num_reqs) if b.q_len[r] == 1]
    rng = np.random.default_rng(index)
    dec = sorted(rng.choice(dec, size=min(24, len(dec)), replace=False).tolist()) if dec else []
    reqs = sorted(pre + dec)
    want = oa.attention_for(b, requests=reqs)
    compare(got, want, "bf16", rows=rows_of(b, reqs),
            what=f"budget {budget} {what} tiles={att.info.num_prefill_items} items={att.info.num_items}")
