"""aug_attn_mixed_noalloc (split-K partials in the library's own device array,
no workspace argument) against aug_attn_mixed with a caller workspace, on two
calls in a row (the second with a smaller batch), and both against the
oracle."""

import numpy as np
import pytest

torch = pytest.importorskip("torch")

from oracle import attention as oa  # noqa: E402
from synth.attn_inputs import make_batch_from_lengths  # noqa: E402
from tests.gpu_util import compare, say  # noqa: E402

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a GPU")]

# (q_lens, ctx_lens, kv dtype, split): split decode rows merged in the launch
# and split prefill tiles merged by the second launch, then a smaller batch
CALLS = [
    ([1024, 1, 1, 1, 1], [17024, 5000, 20000, 3, 700], "bf16", 512),
    ([40, 1, 1], [1500, 3000, 64], "bf16", 256),
]


def _batch(q_lens, ctx_lens, kv, seed):
    return make_batch_from_lengths("noalloc", q_lens, ctx_lens, num_q_heads=32, num_kv_heads=8, head_dim=128,
                                   q_dtype="bf16", kv_dtype=kv, out_dtype="bf16",
                                   n_pool_blocks=int(sum(-(-c // 16) for c in ctx_lens)) + 16, seed=seed,
                                   kv_std=1.0)


def test_noalloc_entry_point_matches_the_workspace_entry_point_on_two_calls():
    import paper_2512_04013_amd as aug
    from paper_2512_04013_amd import runtime as rt
    for k, (q_lens, ctx_lens, kv, split) in enumerate(CALLS):
        b = _batch(q_lens, ctx_lens, kv, seed=90 + k)
        say(f"[noalloc] call {k}: q={q_lens} ctx={ctx_lens} split={split}")
        shape, kvp, q, bids = rt.upload_batch(b)
        att = rt.MixedAttention(shape, kvp, b.q_start, b.ctx_len, b.bt_start, b.block_ids, bids,
                                kv_split_tokens=split)
        info = att.info
        assert info.num_partials > 0 and info.num_merge_groups > info.num_tile_merge_groups
        assert 0 < info.workspace_bytes <= aug.NOALLOC_SCRATCH_BYTES
        if k == 0:
            assert info.num_tile_merge_groups > 0
        ref = att.run(q).clone()
        out = torch.full_like(ref, float("nan"))
        aug.aug_attn_mixed_noalloc(shape, info, att.plan_dev, q, kvp.k_cache, kvp.v_cache, kvp.k_scale,
                                   kvp.v_scale, bids, kvp.num_pool_blocks, out)
        torch.cuda.synchronize()
        # the same kernels and partial layout: the same bits
        assert torch.equal(out.view(torch.int16), ref.view(torch.int16)), f"call {k}"
        got = rt.to_host_f64(out)
        compare(got, oa.attention_for(b), "bf16", what=f"noalloc call {k} parts={info.num_partials}")
        # the plan image's completion counters are back at zero after both launches
        counters_off = int(np.frombuffer(att.plan_host.numpy()[40:44].tobytes(), np.int32)[0])
        cnt = att.plan_dev[counters_off:counters_off + 4 * info.num_merge_groups].cpu().numpy()
        assert not cnt.any()


def test_noalloc_refuses_a_plan_larger_than_its_array():
    import paper_2512_04013_amd as aug
    from paper_2512_04013_amd import runtime as rt
    q_lens, ctx_lens, kv, split = CALLS[1]
    b = _batch(q_lens, ctx_lens, kv, seed=99)
    shape, kvp, q, bids = rt.upload_batch(b)
    att = rt.MixedAttention(shape, kvp, b.q_start, b.ctx_len, b.bt_start, b.block_ids, bids, kv_split_tokens=split)
    big = aug.aug_attn_plan_info.from_buffer_copy(att.info)
    big.workspace_bytes = aug.NOALLOC_SCRATCH_BYTES + 256
    with pytest.raises(aug.AugError) as e:
        aug.aug_attn_mixed_noalloc(shape, big, att.plan_dev, q, kvp.k_cache, kvp.v_cache, None, None, bids,
                                   kvp.num_pool_blocks, att.out)
    assert e.value.status == aug.AUG_ERR_NO_SPACE
