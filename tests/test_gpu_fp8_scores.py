"""GPU parity of the opt-in fp8 products of prefill tiles.

Scores only (AUG_TILES_FP8_QK): against the oracle with the chunk rows'
queries rounded to E4M3 the same way (the path's own arithmetic) at the bf16
gate, on plain and sharp inputs; against the exact oracle at the bf16 gate on
the plain inputs, where the option meets it, and within the stated error law
on the sharp ones, where it does not.

Scores and values (AUG_TILES_FP8): the probabilities are rounded to E4M3 in
the order the kernel meets the keys, which no plain oracle reproduces, so the
outputs are held to an error law derived from that rounding (against both
oracles), decode rows of the same launches to the bf16 gate, and two cases
pin what the rounding must leave exact: a single dominant key returns its
value, and split spans whose values have different scales merge correctly."""

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
FP8 = 3

# (q_lens, ctx_lens, hq, hkv) on fp8 KV, head_dim 128: ragged chunks, decodes
# beside them, split tiles, G = 1, 2, 4, 8
CASES = [
    ([1, 3, 1, 1], [400, 40, 1, 77], 64, 8),
    ([130, 1, 64, 17], [1500, 700, 64, 3000], 64, 8),
    ([40, 1, 100], [2100, 33, 100], 32, 8),
    ([9, 33, 1], [9, 2000, 500], 16, 8),
    ([70, 2, 1], [300, 4100, 64], 16, 16),
]


def _run(batch, kv_split=0, tile_path=FP8_QK, row_path=0):
    from paper_2512_04013_amd import runtime as rt
    shape, kv, q, bids = rt.upload_batch(batch, staging_bytes=1 << 26)
    att = rt.MixedAttention(shape, kv, batch.q_start, batch.ctx_len, batch.bt_start, batch.block_ids,
                            bids, kv_split_tokens=kv_split, tile_path=tile_path, row_path=row_path)
    assert att.info.tile_path == tile_path
    assert row_path == 0 or att.info.row_path == row_path
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


# Error law of fp8 probabilities (on top of the rounded queries): each
# probability carries a relative error of at most 2^-4 (3 mantissa bits), and
# the row sum adds the same rounded values, so an output moves by
# sum_k d_k p_k (v_k - o) / sum_k p_k. With independent d_k (standard
# deviation 2^-4 / sqrt(3) = 0.036) that is about 3.6 % of o's own spread for
# near-uniform attention: a row's relative L2 error of a few per cent
# (measured median 2.5 %, largest 4.3 % on these cases), while the absolute
# errors of the plain inputs (outputs of order 0.1 or less) stay inside the
# bf16 gate's 1e-2 / 1e-3. On the sharp inputs (v ~ N(0, 1)) a few keys share
# the weight and the worst case is 2^-4 max|v_k - o|: measured max-abs up to
# 0.13 and relative L2 up to 0.11 against the exact oracle.
PV_PLAIN_LAW = dict(max_abs=1e-2, mean_abs=1e-3, rel_l2=8e-2)
PV_SHARP_LAW = dict(max_abs=2.5e-1, mean_abs=1e-2, rel_l2=2e-1)


def _check_law(got, want, law, what):
    diff = np.abs(got - want)
    max_abs = float((diff / np.maximum(1.0, np.abs(want))).max())
    rel = float((np.sqrt(((got - want) ** 2).sum(-1)) /
                 np.maximum(np.sqrt((want ** 2).sum(-1)), 1e-6)).max())
    say(f"  {what}: max_abs={max_abs:.3e} mean_abs={diff.mean():.3e} rel_l2={rel:.3e} (law {law})")
    assert np.isfinite(got).all(), what
    assert max_abs <= law["max_abs"] and diff.mean() <= law["mean_abs"] and rel <= law["rel_l2"], what


def _rows(b, decode):
    return np.concatenate([np.arange(b.q_start[r], b.q_start[r + 1]) for r in range(b.num_reqs)
                           if (b.q_len[r] == 1) == decode] or [np.zeros(0, np.int64)]).astype(np.int64)


@pytest.mark.parametrize("case", range(len(CASES)))
@pytest.mark.parametrize("sharp", [False, True])
def test_fp8_values_ragged_cases(case, sharp):
    q_lens, ctx_lens, hq, hkv = CASES[case]
    b = make_batch_from_lengths(f"fp8pv{case}", q_lens, ctx_lens, num_q_heads=hq, num_kv_heads=hkv,
                                head_dim=128, q_dtype="bf16", kv_dtype="fp8", out_dtype="bf16",
                                n_pool_blocks=1024, seed=300 + case,
                                kv_std=1.0 if sharp else 1.0 / np.sqrt(128))
    say(f"[fp8 values] case={case} sharp={sharp} G={hq // hkv}")
    want_rounded = oa.attention_for(b, fp8_chunk_queries=True)
    want_exact = oa.attention_for(b)
    law = PV_SHARP_LAW if sharp else PV_PLAIN_LAW
    chunk, dec = _rows(b, False), _rows(b, True)
    for split in (0, 48):
        got, att = _run(b, kv_split=split, tile_path=FP8)
        what = f"case{case} sharp={sharp} split={split} tiles={att.info.num_prefill_items}"
        _check_law(got[chunk], want_rounded[chunk], law, what + " chunk rows vs rounded-Q oracle")
        _check_law(got[chunk], want_exact[chunk], law, what + " chunk rows vs exact oracle")
        if len(dec):
            compare(got, want_exact, "bf16", rows=dec, what=what + " decode rows")


@pytest.mark.parametrize("sharp", [False, True])
def test_fp8_values_prefill_batch_full_size(sharp):
    """The 16 x 512-row prefill batch on the 64/8-head fp8 layer, every row."""
    b = synth.make_prefill_gqa8_fp8(seed=0, sharp=sharp)
    say(f"[fp8 values] prefill-fp8-64x8 sharp={sharp}, every row")
    got, _ = _run(b, tile_path=FP8)
    law = PV_SHARP_LAW if sharp else PV_PLAIN_LAW
    _check_law(got, oa.attention_for(b, fp8_chunk_queries=True), law, f"prefill-fp8-64x8 sharp={sharp} vs rounded-Q")
    _check_law(got, oa.attention_for(b), law, f"prefill-fp8-64x8 sharp={sharp} vs exact")


def test_fp8_values_single_dominant_key():
    """Every query (all ones) scores key 0 (all twos, unit scale) about 2^32
    times higher than the other keys (zero): each row's output is key 0's
    value. The probability of key 0 is rounded to E4M3 after scaling by its
    block's V scale over the largest one (not a power of two here), so the
    output is exact only because the row sum adds the same rounded value: each
    output must be the oracle's value rounded to bf16, within the half-ulp
    bound 2^-8 |o| of round-to-nearest (a row sum of the unrounded value would
    miss by up to 2^-4). The values are N(0, 1), so the outputs are of order
    1 and the absolute bf16 gate would measure the output rounding itself."""
    b = make_batch_from_lengths("fp8pv-dominant", [200, 70, 1], [200, 1500, 900], num_q_heads=64, num_kv_heads=8,
                                head_dim=128, q_dtype="bf16", kv_dtype="fp8", out_dtype="bf16",
                                n_pool_blocks=256, seed=31)
    b.q = np.full_like(b.q, 0x3F80)                       # bf16 1.0
    k = np.zeros_like(b.k_cache)
    for r in range(b.num_reqs):
        k[b.block_ids[b.bt_start[r]], :, 0, :] = 0x40     # E4M3 2.0: key 0 of each request
    b.k_cache = k
    b.k_scale = np.ones_like(b.k_scale)
    assert np.ptp(b.v_scale[b.block_ids]) > 0             # V scales differ between blocks
    got, _ = _run(b, tile_path=FP8)
    want = oa.attention_for(b)
    err = np.abs(got - want) / np.maximum(np.abs(want), 1e-30)
    say(f"  single dominant key (fp8 values): largest relative error {err.max():.3e} (bound 2^-8 = 3.906e-03)")
    assert np.isfinite(got).all() and err.max() <= 2.0 ** -8 * (1 + 1e-3)


def test_fp8_values_split_spans_with_different_value_scales():
    """A 128-row chunk behind 8,000 cached tokens, split into key spans that
    the tile merge launch combines; the values of the later half of the
    context are scaled up 8 times, so the spans' largest V scales (which set
    each span's probability codes) differ and the partials must carry that
    factor in their maxima to merge correctly."""
    q_lens, ctx_lens = [128, 1, 1], [8128, 5000, 40]
    b = make_batch_from_lengths("fp8pv-spans", q_lens, ctx_lens, num_q_heads=64, num_kv_heads=8, head_dim=128,
                                q_dtype="bf16", kv_dtype="fp8", out_dtype="bf16",
                                n_pool_blocks=int(sum(-(-c // 16) for c in ctx_lens)) + 16, seed=41,
                                kv_std=1.0 / np.sqrt(128))
    table = b.block_ids[b.bt_start[0]:b.bt_start[1]]
    vs = b.v_scale.copy()
    vs[table[len(table) // 2:]] *= 8.0
    b.v_scale = vs
    got, att = _run(b, tile_path=FP8)
    assert att.info.num_tile_merge_groups > 0
    chunk = _rows(b, False)
    _check_law(got[chunk], oa.attention_for(b, fp8_chunk_queries=True)[chunk], PV_PLAIN_LAW,
               f"split spans ({att.info.num_tile_merge_groups} tile merges) vs rounded-Q oracle")


def test_fp8_values_relaunch_repeats_the_bits():
    q_lens, ctx_lens, hq, hkv = CASES[1]
    b = make_batch_from_lengths("fp8pv-relaunch", q_lens, ctx_lens, num_q_heads=hq, num_kv_heads=hkv,
                                head_dim=128, q_dtype="bf16", kv_dtype="fp8", out_dtype="bf16",
                                n_pool_blocks=1024, seed=78)
    first, att = _run(b, kv_split=48, tile_path=FP8)
    from paper_2512_04013_amd import runtime as rt
    for _ in range(2):
        shape, kv, q, bids = rt.upload_batch(b, staging_bytes=1 << 26)
        out = att.run(q, kv=kv, block_ids=bids)
        torch.cuda.synchronize()
        assert np.array_equal(rt.to_host_f64(out), first)


def test_fp8_values_blocks_of_zero_values_keep_their_weight():
    """Blocks whose values are all zero (V scale 0) or far smaller than the
    item's largest scale round their probability codes to zero; their keys
    must still count in the softmax denominator. Every third block of each
    chunk's context is zeroed (codes and scale) and one more is scaled down
    2^-12: outputs within the plain-input law of the exact oracle (without
    the mass of those keys the outputs would grow by about half)."""
    q_lens, ctx_lens = [100, 40, 1], [1700, 900, 600]
    b = make_batch_from_lengths("fp8pv-zero-v", q_lens, ctx_lens, num_q_heads=64, num_kv_heads=8, head_dim=128,
                                q_dtype="bf16", kv_dtype="fp8", out_dtype="bf16", n_pool_blocks=256, seed=51,
                                kv_std=1.0 / np.sqrt(128))
    v = b.v_cache.copy()
    vs = b.v_scale.copy()
    for r in range(2):
        table = b.block_ids[b.bt_start[r]:b.bt_start[r + 1]]
        zero = table[::3]
        v[zero] = 0
        vs[zero] = 0.0
        vs[table[1]] *= 2.0 ** -12
    b.v_cache, b.v_scale = v, vs
    got, _ = _run(b, tile_path=FP8)
    chunk = _rows(b, False)
    _check_law(got[chunk], oa.attention_for(b)[chunk], PV_PLAIN_LAW, "zero and tiny value blocks vs exact oracle")


@pytest.mark.parametrize("tile_path", [FP8_QK, FP8])
@pytest.mark.parametrize("sharp", [False, True])
def test_fp8_tiles_beside_four_head_mfma_rows(tile_path, sharp):
    """Four-head groups on the opt-in MFMA rows next to the opt-in fp8 tile
    products, in one launch (an instantiation of its own): decode rows at the
    bf16 gate against the exact oracle, chunk rows against both oracles
    within the tile path's law, with and without split decode rows."""
    q_lens, ctx_lens, hq, hkv = CASES[2]
    assert hq == 4 * hkv
    b = make_batch_from_lengths(f"fp8-mfma4-{tile_path}", q_lens, ctx_lens, num_q_heads=hq, num_kv_heads=hkv,
                                head_dim=128, q_dtype="bf16", kv_dtype="fp8", out_dtype="bf16",
                                n_pool_blocks=1024, seed=310, kv_std=1.0 if sharp else 1.0 / np.sqrt(128))
    say(f"[fp8 tiles + MFMA rows] G=4 tile_path={tile_path} sharp={sharp}")
    want_rounded = oa.attention_for(b, fp8_chunk_queries=True)
    want_exact = oa.attention_for(b)
    chunk, dec = _rows(b, False), _rows(b, True)
    for split in (0, 48):
        got, att = _run(b, kv_split=split, tile_path=tile_path, row_path=2)
        what = f"G=4 MFMA rows, tile path {tile_path}, sharp={sharp}, split={split}"
        compare(got, want_exact, "bf16", rows=dec, what=what + " decode rows")
        if tile_path == FP8:
            law = PV_SHARP_LAW if sharp else PV_PLAIN_LAW
            _check_law(got[chunk], want_rounded[chunk], law, what + " chunk rows vs rounded-Q oracle")
            _check_law(got[chunk], want_exact[chunk], law, what + " chunk rows vs exact oracle")
        else:
            compare(got, want_rounded, "bf16", rows=chunk, what=what + " chunk rows vs rounded-Q oracle")
            if sharp:
                _check_law(got[chunk], want_exact[chunk], SHARP_LAW, what + " chunk rows vs exact oracle")
            else:
                compare(got, want_exact, "bf16", rows=chunk, what=what + " chunk rows vs exact oracle")
