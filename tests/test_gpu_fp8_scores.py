"""GPU parity of the opt-in fp8 score products of prefill tiles
(AUG_TILES_FP8_QK): against the oracle with the chunk rows' queries rounded
to E4M3 the same way (the path's own arithmetic) at the bf16 gate, on plain
and sharp inputs; against the exact oracle at the bf16 gate on the plain
inputs, where the option meets it, and within the stated error law on the
sharp ones, where it does not."""

import numpy as np
import pytest

torch = pytest.importorskip("torch")

import synth  # noqa: E402
from oracle import attention as oa  # noqa: E402
from synth.attn_inputs import make_batch_from_lengths  # noqa: E402
from tests.gpu_util import compare, say  # noqa: E402

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a GPU")]

FP8_QK = 2

# (q_lens, ctx_lens, hq, hkv) on fp8 KV, head_dim 128: ragged chunks, decodes
# beside them, split tiles, G = 1, 2, 4, 8
CASES = [
    ([1, 3, 1, 1], [400, 40, 1, 77], 64, 8),
    ([130, 1, 64, 17], [1500, 700, 64, 3000], 64, 8),
    ([40, 1, 100], [2100, 33, 100], 32, 8),
    ([9, 33, 1], [9, 2000, 500], 16, 8),
    ([70, 2, 1], [300, 4100, 64], 16, 16),
]


def _run(batch, kv_split=0, tile_path=FP8_QK):
    from paper_2512_04013_amd import runtime as rt
    shape, kv, q, bids = rt.upload_batch(batch, staging_bytes=1 << 26)
    att = rt.MixedAttention(shape, kv, batch.q_start, batch.ctx_len, batch.bt_start, batch.block_ids,
                            bids, kv_split_tokens=kv_split, tile_path=tile_path)
    assert att.info.tile_path == tile_path
    out = att.run(q)
    torch.cuda.synchronize()
    return rt.to_host_f64(out), att


# Error law of the option against the exact oracle: each query element moves
# by up to 2^-4 of itself (3 mantissa bits), so a logit moves by about
# 2^-5 |q| |k| scale (random signs), and an output by that much of |v|. On the
# sharp inputs (q, k, v ~ N(0, 1), head_dim 128, scale 128^-1/2) that is
# about 0.04 of a logit and a few 1e-2 of an output; measured on the host
# with the same rounding: max-abs up to 5e-2 and row relative L2 up to 6e-2
# on short contexts. The bounds below sit above those figures.
SHARP_LAW = dict(max_abs=1.5e-1, mean_abs=1e-2, rel_l2=1.5e-1)


@pytest.mark.parametrize("case", range(len(CASES)))
@pytest.mark.parametrize("sharp", [False, True])
def test_fp8_scores_match_rounded_query_oracle(case, sharp):
    q_lens, ctx_lens, hq, hkv = CASES[case]
    b = make_batch_from_lengths(f"fp8qk{case}", q_lens, ctx_lens, num_q_heads=hq, num_kv_heads=hkv,
                                head_dim=128, q_dtype="bf16", kv_dtype="fp8", out_dtype="bf16",
                                n_pool_blocks=1024, seed=300 + case,
                                kv_std=1.0 if sharp else 1.0 / np.sqrt(128))
    say(f"[fp8 scores] case={case} sharp={sharp} G={hq // hkv}")
    want_rounded = oa.attention_for(b, fp8_chunk_queries=True)
    want_exact = oa.attention_for(b)
    for split in (0, 48):
        got, att = _run(b, kv_split=split)
        what = f"case{case} sharp={sharp} split={split} tiles={att.info.num_prefill_items}"
        compare(got, want_rounded, "bf16", what=what + " vs rounded-Q oracle")
        if not sharp:
            compare(got, want_exact, "bf16", what=what + " vs exact oracle")
        else:
            diff = np.abs(got - want_exact)
            max_abs = float((diff / np.maximum(1.0, np.abs(want_exact))).max())
            rel = float((np.sqrt(((got - want_exact) ** 2).sum(-1)) /
                         np.maximum(np.sqrt((want_exact ** 2).sum(-1)), 1e-6)).max())
            say(f"  {what} vs exact oracle (departure): max_abs={max_abs:.3e} mean_abs={diff.mean():.3e} "
                f"rel_l2={rel:.3e}")
            assert max_abs <= SHARP_LAW["max_abs"] and diff.mean() <= SHARP_LAW["mean_abs"]
            assert rel <= SHARP_LAW["rel_l2"]


@pytest.mark.parametrize("sharp", [False, True])
def test_fp8_scores_prefill_batch_full_size(sharp):
    """The 16 x 512-row prefill batch on the 64/8-head fp8 layer, every row."""
    b = synth.make_prefill_gqa8_fp8(seed=0, sharp=sharp)
    say(f"[fp8 scores] prefill-fp8-64x8 sharp={sharp}, every row")
    got, att = _run(b)
    compare(got, oa.attention_for(b, fp8_chunk_queries=True), "bf16",
            what=f"prefill-fp8-64x8 sharp={sharp} vs rounded-Q oracle")
    if not sharp:
        compare(got, oa.attention_for(b), "bf16", what="prefill-fp8-64x8 vs exact oracle")


def test_fp8_scores_are_opt_in_and_refused_elsewhere():
    import paper_2512_04013_amd as aug
    b = make_batch_from_lengths("optin", [5, 1], [50, 20], num_q_heads=16, num_kv_heads=2, head_dim=128,
                                q_dtype="bf16", kv_dtype="fp8", out_dtype="bf16", n_pool_blocks=64, seed=9)
    _, att = _run(b, tile_path=0 + 1)
    assert att.info.tile_path == aug.AUG_TILES_BF16
    info, _ = aug.aug_attn_plan(aug.make_shape(16, 2, 128, "bf16", "fp8", "bf16", 0.088), b.q_start,
                                b.ctx_len, b.bt_start, b.num_pool_blocks)
    assert info.tile_path == aug.AUG_TILES_BF16


def test_fp8_scores_zero_and_tiny_query_vectors():
    """Query vectors that are all zero, or whose largest magnitude is below
    2^-100, round to zero: their rows attend uniformly (the oracle of the
    rounded queries says the same), with no overflow of the reciprocal scale."""
    b = make_batch_from_lengths("fp8qz", [40, 1], [300, 90], num_q_heads=16, num_kv_heads=2, head_dim=128,
                                q_dtype="bf16", kv_dtype="fp8", out_dtype="bf16", n_pool_blocks=128, seed=21)
    q = b.q.copy()                       # bf16 bit patterns [rows][heads][dim]
    q[3, 0, :] = 0
    q[5, 9, :] = 0
    q[7, 4, :] = 0
    q[7, 4, 11] = 0x0380                 # 2^-120
    b.q = q
    got, _ = _run(b)
    want = oa.attention_for(b, fp8_chunk_queries=True)
    compare(got, want, "bf16", what="zero and tiny query vectors vs rounded-Q oracle")
    assert np.isfinite(got).all()


def test_fp8_scores_relaunch_repeats_the_bits():
    """Split tiles and split decode rows on the fp8 score path: the same plan
    image launched three times gives the same bits (the counters it uses are
    back at zero after each launch)."""
    q_lens, ctx_lens, hq, hkv = CASES[1]
    b = make_batch_from_lengths("fp8qk-relaunch", q_lens, ctx_lens, num_q_heads=hq, num_kv_heads=hkv,
                                head_dim=128, q_dtype="bf16", kv_dtype="fp8", out_dtype="bf16",
                                n_pool_blocks=1024, seed=77)
    first, att = _run(b, kv_split=48)
    assert att.info.num_merge_groups > 0 and att.info.num_prefill_items > 0
    from paper_2512_04013_amd import runtime as rt
    for _ in range(2):
        shape, kv, q, bids = rt.upload_batch(b, staging_bytes=1 << 26)
        out = att.run(q, kv=kv, block_ids=bids)
        torch.cuda.synchronize()
        assert np.array_equal(rt.to_host_f64(out), first)
