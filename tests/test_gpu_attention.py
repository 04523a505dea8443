"""GPU parity of aug_attn_mixed against the oracle (through the C ABI)."""

import copy

import numpy as np
import pytest

torch = pytest.importorskip("torch")

import synth  # noqa: E402
from oracle import attention as oa  # noqa: E402
from oracle import kvpark  # noqa: E402
from synth.attn_inputs import make_batch_from_lengths  # noqa: E402
from tests.gpu_util import compare, say  # noqa: E402

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a GPU")]


def _run(batch, kv_split=0, staging_bytes=1 << 26, row_path=0):
    from paper_2512_04013_amd import runtime as rt
    shape, kv, q, bids = rt.upload_batch(batch, staging_bytes=staging_bytes)
    att = rt.MixedAttention(shape, kv, batch.q_start, batch.ctx_len, batch.bt_start, batch.block_ids,
                            bids, kv_split_tokens=kv_split, row_path=row_path)
    out = att.run(q)
    torch.cuda.synchronize()
    return rt.to_host_f64(out), att


# ---- tiny fp32 mixed batch: every row, several splits ------------------------------------

@pytest.mark.parametrize("seed", [0, 1, 2])
@pytest.mark.parametrize("split", [0, 32, 64])
def test_tiny_mixed_fp32(seed, split):
    b = synth.make_tiny_mixed(seed=seed)
    say(f"[tiny-mixed fp32] seed={seed} split={split}")
    got, att = _run(b, kv_split=split)
    want = oa.attention_for(b)
    compare(got, want, "f32", what=f"tiny seed={seed} split={split} parts={att.info.num_partials}")


# ---- ragged shapes across group sizes, head dims and dtypes ---------------------------------

CASES = [
    # (q_lens, ctx_lens, hq, hkv, d, q/kv dtype)
    ([1, 1, 1, 5, 1, 40], [1, 17, 300, 5, 16, 333], 8, 8, 64, "bf16"),        # G=1, ctx=1, q=ctx
    ([1, 70, 1, 3], [200, 70, 1000, 29], 8, 4, 128, "bf16"),                 # G=2
    ([33, 1, 129, 1], [100, 1, 500, 2049], 32, 8, 128, "bf16"),              # G=4, >1 tile
    ([17, 1, 1, 16], [17, 64, 65, 600], 64, 8, 128, "bf16"),                 # G=8
    ([1, 9, 1], [513, 100, 48], 16, 4, 64, "bf16"),                          # D=64 tiles
    ([1, 3, 1, 1], [400, 40, 1, 77], 64, 8, 128, "fp8"),                     # fp8 KV, small tile
    ([2, 1, 1], [35, 250, 16], 8, 2, 128, "f32"),                            # f32 D=128, G=4
    ([70, 1, 5], [2600, 1500, 2100], 32, 8, 128, "bf16"),                    # split tiles (3 spans)
    ([20, 130], [1100, 2200], 16, 2, 64, "bf16"),                            # split tiles, D=64, G=8
    ([130, 1, 64, 17], [1500, 700, 64, 3000], 64, 8, 128, "fp8"),            # fp8 KV tiles, split, G=8
    ([40, 1, 100], [2100, 33, 100], 32, 8, 128, "fp8"),                      # fp8 KV tiles, G=4
]


def _row_paths(hq, hkv, d, dt):
    """The automatic row path, and for four-head groups (head_dim 128, bf16
    queries) also the opt-in MFMA row path."""
    return (0, 2) if hq == 4 * hkv and d == 128 and dt in ("bf16", "fp8") else (0,)


@pytest.mark.parametrize("case", range(len(CASES)))
@pytest.mark.parametrize("sharp", [False, True])
def test_ragged_shapes(case, sharp):
    q_lens, ctx_lens, hq, hkv, d, dt = CASES[case]
    qd = "f32" if dt == "f32" else "bf16"
    b = make_batch_from_lengths(f"case{case}", q_lens, ctx_lens, num_q_heads=hq, num_kv_heads=hkv,
                                head_dim=d, q_dtype=qd, kv_dtype=dt, out_dtype=qd,
                                n_pool_blocks=512, seed=100 + case,
                                kv_std=1.0 if sharp else 1.0 / np.sqrt(d))
    say(f"[ragged] case={case} sharp={sharp} G={hq // hkv} D={d} kv={dt}")
    want = oa.attention_for(b)
    for row_path in _row_paths(hq, hkv, d, dt):
        for split in (0, 48):
            got, att = _run(b, kv_split=split, row_path=row_path)
            assert row_path == 0 or att.info.row_path == row_path
            compare(got, want, qd, what=f"case{case} sharp={sharp} split={split} row path {att.info.row_path} "
                                        f"tiles={att.info.num_prefill_items}")


def test_relaunching_one_plan_image_repeats_the_bits():
    """Split decode rows are merged inside the launch through completion
    counters in the plan image, which the launch returns to zero: the same
    device copy launched again gives the same bits, and the counters read
    zero afterwards."""
    q_lens, ctx_lens, hq, hkv, d, dt = CASES[9]
    b = make_batch_from_lengths("relaunch", q_lens, ctx_lens, num_q_heads=hq, num_kv_heads=hkv,
                                head_dim=d, q_dtype="bf16", kv_dtype=dt, out_dtype="bf16",
                                n_pool_blocks=512, seed=77, kv_std=1.0 / np.sqrt(d))
    say("[relaunch] fp8 G=8, split rows and tiles, 4 launches of one plan image")
    first, att = _run(b, kv_split=32)
    assert att.info.num_merge_groups > att.info.num_tile_merge_groups > 0
    compare(first, oa.attention_for(b), "bf16", what="relaunch first")
    from paper_2512_04013_amd import runtime as rt
    q = rt.to_device_array(b.q, b.q_dtype, "cuda")
    for i in range(3):
        att.out.zero_()
        got = rt.to_host_f64(att.run(q))
        torch.cuda.synchronize()
        assert np.array_equal(got.view(np.uint64), first.view(np.uint64)), f"launch {i + 2} differs"
    image = att.plan_dev.cpu().numpy()
    hdr = image[:64].view(np.int32)
    counters = image[hdr[10]:hdr[10] + 4 * att.info.num_merge_groups].view(np.int32)
    assert not counters.any()


# ---- the 8B-shaped decode batch at full size ----------------------------------------------------

@pytest.fixture(scope="module")
def decode_8b():
    return synth.make_decode_8b(seed=0)


@pytest.fixture(scope="module")
def decode_8b_want(decode_8b):
    return oa.attention_for(decode_8b)


@pytest.mark.parametrize("split", [0, 128, 1024])
@pytest.mark.parametrize("row_path", [0, 2])
def test_decode_8b_full(decode_8b, decode_8b_want, split, row_path):
    """All 256 rows of the 8B decode batch (32/8 heads), on the planner's row
    path (vector ALU) and on the opt-in MFMA row path for four-head groups."""
    b = decode_8b
    say(f"[decode-8b] 256 decodes, split={split} row_path={row_path}")
    got, att = _run(b, kv_split=split, row_path=row_path)
    assert att.info.row_path == (row_path or 1)
    compare(got, decode_8b_want, "bf16", what=f"decode-8b split={split} row path {att.info.row_path} "
                                             f"items={att.info.num_items}")


@pytest.mark.parametrize("kv", ["fp8", "bf16"])
@pytest.mark.parametrize("sharp", [False, True])
@pytest.mark.parametrize("row_path", [2, 1])
def test_gqa8_decode_batch_full_size(kv, sharp, row_path):
    """512 decodes on the 64/8-head layer (the shape of the budget sweep),
    contexts lognormal (median 2500, sigma 0.8, cap 16384): the 8-way grouped
    decode rows on the MFMA row path (the planner's default for this shape)
    and on the vector-ALU row path. Every row against the oracle."""
    if kv == "fp8":
        b = synth.make_decode_gqa8_fp8(seed=0, sharp=sharp)      # the decode-fp8-64x8 bench workload
        ctx = b.ctx_len.astype(int)
    else:
        rng = np.random.default_rng(21)
        ctx = np.clip(np.rint(rng.lognormal(np.log(2500), 0.8, 512)), 1, 16384).astype(int)
        b = make_batch_from_lengths("gqa8-decode", [1] * 512, ctx.tolist(), num_q_heads=64, num_kv_heads=8,
                                    head_dim=128, q_dtype="bf16", kv_dtype=kv, out_dtype="bf16",
                                    n_pool_blocks=int(sum(-(-c // 16) for c in ctx)) + 64, seed=22,
                                    kv_std=1.0 if sharp else 1.0 / np.sqrt(128.0))
    say(f"[gqa8 decode] kv={kv} sharp={sharp} row_path={row_path} keys={int(ctx.sum())}")
    got, att = _run(b, row_path=row_path)
    assert att.info.row_path == row_path
    compare(got, oa.attention_for(b), "bf16", what=f"gqa8 decode {kv} sharp={sharp} row path {row_path} (all 512 rows)")


@pytest.mark.parametrize("row_path", [0, 2])
def test_decode_8b_sharp_full(row_path):
    b = synth.make_decode_8b(seed=1, sharp=True)
    say(f"[decode-8b sharp] 256 decodes row_path={row_path}")
    got, att = _run(b, row_path=row_path)
    assert att.info.row_path == (row_path or 1)
    compare(got, oa.attention_for(b), "bf16", what=f"decode-8b sharp row path {att.info.row_path}")


def test_block_permutation_gives_identical_bits(decode_8b):
    b = synth.make_decode_8b(seed=5, n_req=48, n_pool_blocks=8192)
    say("[permutation] 48 decodes")
    got, _ = _run(b)
    perm = np.random.default_rng(9).permutation(b.num_pool_blocks)
    b2 = copy.copy(b)
    b2.k_cache = np.empty_like(b.k_cache)
    b2.v_cache = np.empty_like(b.v_cache)
    b2.k_cache[perm] = b.k_cache
    b2.v_cache[perm] = b.v_cache
    b2.block_ids = perm[b.block_ids].astype(np.int32)
    got2, _ = _run(b2)
    assert np.array_equal(got.view(np.uint64), got2.view(np.uint64))


def test_results_do_not_depend_on_the_split_beyond_tolerance(decode_8b):
    b = synth.make_decode_8b(seed=6, n_req=32, n_pool_blocks=8192, sharp=True)
    say("[split independence] 32 decodes")
    outs = [_run(b, kv_split=s)[0] for s in (16, 64, 256, 4096)]
    for o in outs[1:]:
        assert np.abs(o - outs[0]).max() <= 1e-2


# ---- the mixed batch: resume parked requests, then attention ----------------------------------

def _park_resume_then_attend(b, split=0, staging_bytes=1 << 26, sample=None, row_path=0):
    from paper_2512_04013_amd import runtime as rt
    shape, kv, q, bids = rt.upload_batch(b, staging_bytes=staging_bytes)
    pk = b.park
    dev = kv.k_cache.device
    src = torch.from_numpy(pk.resume_src_blocks).to(dev)
    dst = torch.from_numpy(pk.resume_blocks).to(dev)
    host = kv.host_buffer(len(pk.resume_src_blocks))
    kv.park(pk.resume_src_blocks, src, host)
    torch.cuda.synchronize()
    image = host.numpy()[:len(pk.resume_src_blocks) * kv.record_bytes]
    want_img = kvpark.park(b.k_cache, b.v_cache, b.k_scale, b.v_scale, b.kv_dtype, pk.resume_src_blocks)
    assert np.array_equal(image, want_img), "parked image differs from the oracle's"
    # the source blocks are free now: poison them, then resume into the new blocks
    kv.k_cache.view(torch.uint8)[src.long()] = 0xFF
    kv.v_cache.view(torch.uint8)[src.long()] = 0xFF
    kv.resume(pk.resume_blocks, dst, host)
    att = rt.MixedAttention(shape, kv, b.q_start, b.ctx_len, b.bt_start, b.block_ids, bids,
                            kv_split_tokens=split, row_path=row_path)
    assert row_path == 0 or att.info.row_path == row_path
    out = att.run(q)
    parked_others = None
    if len(pk.park_blocks):
        pb = torch.from_numpy(pk.park_blocks).to(dev)
        parked_others = kv.host_buffer(len(pk.park_blocks))
        kv.park(pk.park_blocks, pb, parked_others)
    torch.cuda.synchronize()
    k_res, v_res, _, _ = kvpark.resume(b.k_cache, b.v_cache, b.k_scale, b.v_scale, b.kv_dtype,
                                       pk.resume_blocks, want_img)
    if parked_others is not None:
        want_other = kvpark.park(b.k_cache, b.v_cache, b.k_scale, b.v_scale, b.kv_dtype, pk.park_blocks)
        assert np.array_equal(parked_others.numpy()[:want_other.size], want_other)
    # resumed blocks hold exactly the parked bytes
    rb = torch.from_numpy(pk.resume_blocks).long().to(dev)
    dev_k = kv.k_cache.view(torch.uint8)[rb].cpu().numpy() if b.kv_dtype == "fp8" else \
        kv.k_cache[rb].view(torch.int16 if b.kv_dtype == "bf16" else torch.int32).cpu().numpy()
    host_k = b.k_cache[pk.resume_src_blocks]
    assert np.array_equal(dev_k.view(np.uint8), np.ascontiguousarray(host_k).view(np.uint8))
    return rt.to_host_f64(out), att, (k_res, v_res)


def test_mixed_8b_small_all_rows():
    b = synth.make_mixed_8b(seed=3, n_dec=64, n_pre=2, n_pool_blocks=16384)
    say("[mixed-8b small] 2 prefill chunks + 64 decodes, resume 30%")
    got, att, (k_res, v_res) = _park_resume_then_attend(b)
    assert att.info.num_prefill_items > 0
    want = oa.attention_for(b, k_cache=k_res, v_cache=v_res)
    compare(got, want, "bf16", what="mixed-8b small")


@pytest.mark.parametrize("sharp,row_path", [(False, 0), (True, 0), (False, 2), (True, 2)])
def test_mixed_8b_full_size_every_row(sharp, row_path):
    """The full mixed batch (3 x 512-row prefill chunks and 512 decodes, 30 %
    of them resumed after a real park round trip), in the launch configuration
    the benchmark times (planner's split): every row against the oracle, plain
    (K/V ~ N(0,1)/sqrt(128)) and sharp (K/V ~ N(0,1)); decode rows on the
    planner's vector-ALU rows and on the opt-in MFMA rows."""
    b = synth.make_mixed_8b(seed=0, sharp=sharp)
    say(f"[mixed-8b full] sharp={sharp} row_path={row_path} {b.num_reqs} requests, {b.total_q} rows, "
        f"resume {len(b.park.resume_blocks)} blocks")
    got, att, (k_res, v_res) = _park_resume_then_attend(b, staging_bytes=1 << 27, row_path=row_path)
    assert att.info.num_prefill_items > 0
    want = oa.attention_for(b, k_cache=k_res, v_cache=v_res)
    compare(got, want, "bf16", what=f"mixed-8b full sharp={sharp} row path {att.info.row_path} "
                                    f"(all {b.total_q} rows)")


@pytest.mark.parametrize("sharp,row_path", [(False, 0), (True, 0), (True, 2)])
def test_long_context_every_row(sharp, row_path):
    """64 decodes over 16k-32k keys (split-K, merged inside the launch) after
    8 requests were parked and 8 resumed: all 64 rows against the oracle, on
    the planner's row path and (sharp inputs) on the opt-in MFMA rows."""
    b = synth.make_long_context(seed=0, sharp=sharp)
    say(f"[long-context] sharp={sharp} row_path={row_path} 64 decodes 16k-32k, resume 8, park 8 "
        f"({len(b.park.park_blocks)} blocks)")
    got, att, (k_res, v_res) = _park_resume_then_attend(b, staging_bytes=1 << 28, row_path=row_path)
    assert att.info.num_merge_groups > 0
    want = oa.attention_for(b, k_cache=k_res, v_cache=v_res)
    compare(got, want, "bf16", what=f"long-context sharp={sharp} row path {att.info.row_path} (all 64 rows)")


@pytest.mark.parametrize("workload,sharp", [("prefill-fp8-64x8", False), ("prefill-fp8-64x8", True),
                                             ("prefill-8b", False), ("prefill-8b", True)])
def test_prefill_workloads_full_size_every_row(workload, sharp):
    """The prefill-dominated benchmark batches at full size, in the launch
    configuration the benchmark times (automatic split): 16 x 512-row chunks
    on the 64/8-head fp8 layer, 8 x 512-row chunks on the 8B bf16 layer.
    Every row of every chunk against the oracle."""
    b = (synth.make_prefill_gqa8_fp8 if workload == "prefill-fp8-64x8" else synth.make_prefill_8b)(
        seed=0, sharp=sharp)
    ctx = b.ctx_len.astype(int)
    say(f"[{workload}] sharp={sharp} {b.num_reqs} chunks, {b.total_q} rows, keys={int(ctx.sum())}")
    got, att = _run(b)
    assert att.info.num_prefill_items > 0
    want = oa.attention_for(b)
    compare(got, want, "bf16", what=f"{workload} sharp={sharp} (all {b.total_q} rows)")


def test_long_chunk_over_long_prior_context():
    """One 1024-row chunk behind 16,000 cached tokens (tiles split along
    keys, merged by the tile merge launch) next to two decodes, every row
    against the oracle."""
    q_lens, ctx_lens = [1024, 1, 1], [17024, 9000, 3]
    b = make_batch_from_lengths("long-chunk", q_lens, ctx_lens, num_q_heads=32, num_kv_heads=8, head_dim=128,
                                q_dtype="bf16", kv_dtype="bf16", out_dtype="bf16",
                                n_pool_blocks=int(sum(-(-c // 16) for c in ctx_lens)) + 16, seed=77, kv_std=1.0)
    say("[long chunk] 1024 rows over 16k prior keys + 2 decodes, sharp")
    got, att = _run(b)
    assert att.info.num_prefill_items > 0
    compare(got, oa.attention_for(b), "bf16",
            what=f"long chunk items={att.info.num_items} tile merges={att.info.num_tile_merge_groups}")


@pytest.mark.parametrize("kv,row_path", [("bf16", 0), ("bf16", 2), ("fp8", 2)])
def test_decodes_at_very_long_contexts(kv, row_path):
    """Decodes over 131,072 and 131,071 keys (8192 blocks each, many split
    spans merged inside the launch) beside a one-key decode, four heads per
    KV head: the vector-ALU rows and the opt-in MFMA rows."""
    hq = 32
    ctx_lens = [131072, 131071, 1]
    b = make_batch_from_lengths("long-decodes", [1, 1, 1], ctx_lens, num_q_heads=hq, num_kv_heads=8, head_dim=128,
                                q_dtype="bf16", kv_dtype=kv, out_dtype="bf16",
                                n_pool_blocks=int(sum(-(-c // 16) for c in ctx_lens)) + 8, seed=78, kv_std=1.0)
    say(f"[long decodes] kv={kv} row_path={row_path} ctx={ctx_lens}")
    got, att = _run(b, row_path=row_path)
    assert att.info.num_merge_groups >= 2 and att.info.row_path == (row_path or 1)
    compare(got, oa.attention_for(b), "bf16", what=f"long decodes {kv} row path {att.info.row_path} "
                                                   f"items={att.info.num_items}")


@pytest.mark.parametrize("hq,kv,row_path", [(32, "bf16", 0), (32, "fp8", 2), (64, "fp8", 0), (64, "bf16", 0)])
def test_decode_rows_with_a_thousand_spans(hq, kv, row_path):
    """Decode rows split into about 1250 spans each (16-key spans over 20,000
    keys), merged inside the launch by the workgroup that finishes last:
    the merge loop over many partials, on the vector-ALU rows (four heads per
    KV head) and on the eight-wave MFMA rows (eight heads, fp8 and bf16; four
    heads when asked for)."""
    ctx_lens = [20000, 19999, 700, 1]
    b = make_batch_from_lengths("many-spans", [1, 1, 1, 1], ctx_lens, num_q_heads=hq, num_kv_heads=8,
                                head_dim=128, q_dtype="bf16", kv_dtype=kv, out_dtype="bf16",
                                n_pool_blocks=int(sum(-(-c // 16) for c in ctx_lens)) + 8, seed=79, kv_std=1.0)
    say(f"[many spans] G={hq // 8} kv={kv} row_path={row_path}")
    got, att = _run(b, kv_split=16, row_path=row_path)
    assert row_path == 0 or att.info.row_path == row_path
    assert att.info.num_partials >= 2 * 8 * 1250
    compare(got, oa.attention_for(b), "bf16", what=f"many spans G={hq // 8} {kv} parts={att.info.num_partials}")
