"""CPU tests of the C ABI library: it loads without a GPU, exports every
symbol include/aug.h declares, the planner validates batches and covers every
key of every row exactly once, and the C++ batch former equals the oracle
former bit for bit. No device call is made here."""

import os
import re

import numpy as np
import pytest

import paper_2512_04013_amd as aug
from paper_2512_04013_amd import AugError
import synth
from synth.attn_inputs import make_batch_from_lengths

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

pytestmark = pytest.mark.skipif(not os.path.exists(aug.LIB_PATH), reason="libaug.so not built")


def test_library_exports_every_declared_symbol():
    header = open(os.path.join(ROOT, "include", "aug.h")).read()
    declared = set(re.findall(r"\b(aug_[a-z_]+)\s*\(", header))
    assert declared == set(aug.EXPORTED)
    L = aug.lib()
    for name in declared:
        assert hasattr(L, name), name
    assert aug.aug_abi_version() >> 16 == 3
    assert aug.aug_status_string(aug.AUG_ERR_NO_SPACE) == "AUG_ERR_NO_SPACE"


def _shape(b):
    return aug.make_shape(b.num_q_heads, b.num_kv_heads, b.head_dim, b.q_dtype, b.kv_dtype,
                          b.out_dtype, b.softmax_scale)


def _decode_plan(plan):
    hdr = plan[:64].view(np.int32)
    assert hdr[0] == 0x4E4C5041 and hdr[1] == 4
    n_items, n_groups = hdr[2], hdr[4]
    item_t = np.dtype([("kvh", "<i2"), ("kind", "i1"), ("res", "i1"), ("q_row0", "<i4"),
                       ("n_rows", "<i2"), ("stride", "<i2"), ("kb", "<i4"), ("ke", "<i4"),
                       ("pos0", "<i4"), ("bt_off", "<i4"), ("part", "<i4"), ("group", "<i4"),
                       ("res2", "<i4", (3,))])
    assert item_t.itemsize == 48
    items = plan[hdr[8]:hdr[8] + 48 * n_items].view(item_t)
    groups = plan[hdr[9]:hdr[9] + 16 * n_groups].view(np.int32).reshape(-1, 4)
    counters = plan[hdr[10]:hdr[10] + 4 * n_groups].view(np.int32)
    assert hdr[10] == hdr[9] + 16 * n_groups
    # the append list follows the counters, 16-byte aligned, and ends the image
    assert hdr[11] == (hdr[10] + 4 * n_groups + 15) // 16 * 16 and hdr[11] + 16 * hdr[12] == len(plan)
    assert not plan[hdr[10] + 4 * n_groups:hdr[11]].any()
    assert not counters.any(), "completion counters start at zero"
    return hdr, items, groups


@pytest.mark.parametrize("cfg", [1, 3])
@pytest.mark.parametrize("split", [0, 32, 256])
def test_plan_covers_every_key_of_every_row_once(cfg, split):
    if cfg == 3:
        b = synth.make_mixed_8b(seed=1, n_dec=40, n_pre=2, n_pool_blocks=8192)
    else:
        b = synth.make_tiny_mixed(seed=3)
    info, plan = aug.aug_attn_plan(_shape(b), b.q_start, b.ctx_len, b.bt_start, b.num_pool_blocks,
                                   b.block_ids, kv_split_tokens=split)
    hdr, items, groups = _decode_plan(plan)
    assert info.num_items == len(items) and info.num_merge_groups == len(groups)
    g = b.num_q_heads // b.num_kv_heads
    tiled = b.q_dtype == "bf16" and b.kv_dtype == "bf16"
    cover = {}
    parts_seen = set()
    tile_slots = set()
    for it in items:
        kind, kvh, q_row0, n_rows = int(it["kind"]), int(it["kvh"]), int(it["q_row0"]), int(it["n_rows"])
        kb, ke, pos0, bt_off, part, stride = (int(it[f]) for f in ("kb", "ke", "pos0", "bt_off", "part", "stride"))
        r = int(np.searchsorted(b.q_start, q_row0, side="right") - 1)
        assert bt_off == b.bt_start[r]
        q_len = b.q_start[r + 1] - b.q_start[r]
        if kind == 1:
            assert tiled and q_len > 1 and kb % 64 == 0
            assert n_rows <= 128 // g
            for j in range(n_rows):
                row = q_row0 + j
                pos = b.ctx_len[r] - q_len + (row - b.q_start[r])
                assert pos0 + j == pos
                lo, hi = kb, min(ke, pos + 1)
                if hi > lo:
                    cover.setdefault((row, kvh), []).append((lo, hi))
                if part >= 0:
                    slot = part + j * stride
                    assert slot not in tile_slots
                    tile_slots.add(slot)
                    # row j's merge group lists this slot among its spans
                    q_row, g_kvh, part0, n = groups[int(it["group"]) + j]
                    assert q_row == row and g_kvh == kvh and part0 <= slot < part0 + n
            if part < 0:
                assert int(it["group"]) == -1
        else:
            assert n_rows == 1 and kb % 16 == 0
            pos = b.ctx_len[r] - q_len + (q_row0 - b.q_start[r])
            assert pos0 == pos and ke <= pos + 1
            cover.setdefault((q_row0, kvh), []).append((kb, ke))
            if part >= 0:
                assert part not in parts_seen
                parts_seen.add(part)
                q_row, g_kvh, part0, n = groups[int(it["group"])]
                assert q_row == q_row0 and g_kvh == kvh and part0 <= part < part0 + n
            else:
                assert int(it["group"]) == -1
    assert not (tile_slots & parts_seen)
    parts_seen |= tile_slots
    for r in range(b.num_reqs):
        for row in range(b.q_start[r], b.q_start[r + 1]):
            pos = b.ctx_len[r] - (b.q_start[r + 1] - b.q_start[r]) + (row - b.q_start[r])
            for h in range(b.num_kv_heads):
                spans = sorted(cover[(row, h)])
                assert spans[0][0] == 0 and spans[-1][1] == pos + 1
                assert all(a[1] == c[0] for a, c in zip(spans, spans[1:]))
    assert parts_seen == set(range(info.num_partials))
    for q_row, kvh, part0, n in groups:
        assert n > 1 and len(cover[(q_row, kvh)]) <= n


def test_plan_rejects_invalid_batches():
    b = synth.make_tiny_mixed(seed=0)
    s = _shape(b)

    def plan(**kw):
        args = dict(q_start=b.q_start, ctx_len=b.ctx_len, bt_start=b.bt_start,
                    num_pool_blocks=b.num_pool_blocks, block_ids=b.block_ids)
        args.update(kw)
        return aug.aug_attn_plan(s, **args)

    plan()
    bad_ctx = b.ctx_len.copy()
    bad_ctx[np.argmax(b.q_len > 1)] = 5           # fewer keys than rows
    with pytest.raises(AugError) as e:
        plan(ctx_len=bad_ctx)
    assert e.value.status == aug.AUG_ERR_INVALID
    bad_ids = b.block_ids.copy()
    bad_ids[3] = b.num_pool_blocks
    with pytest.raises(AugError):
        plan(block_ids=bad_ids)
    plan(block_ids=None, num_pool_blocks=b.num_pool_blocks)    # unchecked table is accepted
    bad_bt = b.bt_start.copy()
    bad_bt[1:] -= 1                                # first request one block short
    with pytest.raises(AugError):
        plan(bt_start=bad_bt)
    bad_q = b.q_start.copy()
    bad_q[2] = bad_q[1]                            # an empty request
    with pytest.raises(AugError):
        plan(q_start=bad_q)
    with pytest.raises(AugError) as e:
        aug.aug_attn_plan(aug.make_shape(4, 4, 96, "f32", "f32", "f32", 0.1), b.q_start, b.ctx_len,
                          b.bt_start, b.num_pool_blocks)
    assert e.value.status == aug.AUG_ERR_UNSUPPORTED
    with pytest.raises(AugError) as e:
        aug.aug_attn_plan(aug.make_shape(6, 4, 64, "f32", "f32", "f32", 0.1), b.q_start, b.ctx_len,
                          b.bt_start, b.num_pool_blocks)
    assert e.value.status == aug.AUG_ERR_INVALID
    info, p = aug.aug_attn_plan(s, np.zeros(1, np.int32), np.zeros(0, np.int32),
                                np.zeros(1, np.int32), 8)
    assert info.num_items == 0


def test_park_and_attention_reject_bad_arguments_without_touching_the_gpu():
    s = aug.make_shape(32, 8, 128, "bf16", "bf16", "bf16", 0.088)
    assert aug.aug_kv_record_bytes(s) == 2 * 8 * 16 * 128 * 2
    s8 = aug.make_shape(64, 8, 128, "bf16", "fp8", "bf16", 0.088)
    assert aug.aug_kv_record_bytes(s8) == 2 * 8 * 16 * 128 + 2 * 8 * 4
    L = aug.lib()
    ids = np.array([0, 5, 99], np.int32)
    # id 99 is outside a 50-block pool: refused on the host before any launch
    st = L.aug_kv_park(aug.C.byref(s), 8, 8, None, None, 8, ids.ctypes.data, 3, 50, 8, 1 << 30, 8,
                       1 << 20, None)
    assert st == aug.AUG_ERR_INVALID and "outside" in aug.aug_last_error()
    st = L.aug_kv_park(aug.C.byref(s), 8, 8, None, None, 8, None, 3, 50, 8, 100, 8, 1 << 20, None)
    assert st == aug.AUG_ERR_NO_SPACE
    st = L.aug_kv_resume(aug.C.byref(s8), 8, 8, None, None, 8, None, 3, 50, 8, 1 << 30, 8, 1 << 20, None)
    assert st == aug.AUG_ERR_INVALID             # fp8 without scales
    assert L.aug_kv_park(aug.C.byref(s), None, None, None, None, None, None, 0, 50, None, 0, None, 0,
                         None) == aug.AUG_OK     # nothing to do
    # the host copy of the ids is required, so that every id is checked before a launch
    for f in (L.aug_kv_park, L.aug_kv_resume):
        st = f(aug.C.byref(s), 8, 8, None, None, 8, None, 3, 50, 8, 1 << 30, 8, 1 << 20, None)
        assert st == aug.AUG_ERR_INVALID and "block_ids_host" in aug.aug_last_error()
    b = synth.make_tiny_mixed(seed=0)
    info, _ = aug.aug_attn_plan(_shape(b), b.q_start, b.ctx_len, b.bt_start, b.num_pool_blocks)
    if info.num_partials == 0:
        info, _ = aug.aug_attn_plan(_shape(b), b.q_start, b.ctx_len, b.bt_start, b.num_pool_blocks,
                                    kv_split_tokens=32)
    assert info.num_partials > 0
    st = L.aug_attn_mixed(aug.C.byref(_shape(b)), aug.C.byref(info), 8, 8, 8, 8, None, None, 8,
                          b.num_pool_blocks, 8, None, 0, None)
    assert st == aug.AUG_ERR_NO_SPACE
    st = L.aug_attn_mixed(aug.C.byref(_shape(b)), aug.C.byref(info), None, 8, 8, 8, None, None, 8,
                          b.num_pool_blocks, 8, 8, 1 << 30, None)
    assert st == aug.AUG_ERR_INVALID


def test_plan_header_and_info_record_the_shape():
    b = synth.make_mixed_8b(seed=1, n_dec=8, n_pre=1, n_pool_blocks=4096)
    info, plan = aug.aug_attn_plan(_shape(b), b.q_start, b.ctx_len, b.bt_start, b.num_pool_blocks)
    hdr16 = plan[52:58].view(np.int16)
    assert hdr16.tolist() == [32, 8, 128]
    assert plan[58:61].view(np.int8).tolist() == [aug.AUG_BF16] * 3
    assert (info.num_q_heads, info.num_kv_heads, info.head_dim) == (32, 8, 128)
    assert (info.q_dtype, info.kv_dtype, info.out_dtype) == (aug.AUG_BF16,) * 3


def test_workspace_size_query_matches_the_plan():
    rng = np.random.default_rng(2)
    ctx = [int(c) for c in rng.integers(1, 6000, 40)] + [700, 3000]
    b = make_batch_from_lengths("ws", [1] * 40 + [100, 512], ctx, num_q_heads=32, num_kv_heads=8, head_dim=128,
                                q_dtype="bf16", kv_dtype="bf16", out_dtype="bf16",
                                n_pool_blocks=sum(-(-c // 16) for c in ctx) + 8, seed=2)
    for split in (0, 32, 256):
        info, _ = aug.aug_attn_plan(_shape(b), b.q_start, b.ctx_len, b.bt_start, b.num_pool_blocks,
                                    b.block_ids, kv_split_tokens=split)
        ws = aug.aug_attn_workspace_size(_shape(b), b.q_start, b.ctx_len, b.bt_start, b.num_pool_blocks,
                                         b.block_ids, kv_split_tokens=split)
        assert ws == info.workspace_bytes
        assert (ws > 0) == (info.num_partials > 0)
    with pytest.raises(AugError) as e:
        aug.aug_attn_workspace_size(_shape(b), b.q_start, b.ctx_len[:-1] * 0, b.bt_start, b.num_pool_blocks)
    assert e.value.status == aug.AUG_ERR_INVALID
    L = aug.lib()
    assert L.aug_attn_workspace_size(aug.C.byref(_shape(b)), None, 0, None) == aug.AUG_ERR_INVALID


@pytest.mark.parametrize("split", [2 ** 31 - 1, 2 ** 31 - 100, 2 ** 24 + 1])
def test_plan_rejects_a_huge_requested_split(split):
    """A requested split near INT32_MAX must be refused, not overflow the
    span arithmetic (which once divided by zero)."""
    b = synth.make_tiny_mixed(seed=0)
    with pytest.raises(AugError) as e:
        aug.aug_attn_plan(_shape(b), b.q_start, b.ctx_len, b.bt_start, b.num_pool_blocks,
                          kv_split_tokens=split)
    assert e.value.status == aug.AUG_ERR_INVALID and "kv_split_tokens" in str(e.value)
    info, _ = aug.aug_attn_plan(_shape(b), b.q_start, b.ctx_len, b.bt_start, b.num_pool_blocks,
                                kv_split_tokens=2 ** 24)
    assert info.kv_split_tokens == 2 ** 24


def test_plan_rejects_contexts_beyond_its_limit():
    s = aug.make_shape(8, 8, 64, "bf16", "bf16", "bf16", 0.125)
    ctx = 2 ** 24 + 1
    with pytest.raises(AugError) as e:
        aug.aug_attn_plan(s, [0, 1], [ctx], [0, -(-ctx // 16)], 1 << 21)
    assert e.value.status == aug.AUG_ERR_UNSUPPORTED
    # the limit itself is accepted: a decode and a 300-row chunk over 2^24 keys,
    # every key of every row covered by the spans (largest requested split too)
    ctx = 2 ** 24
    for q_len, split in ((1, 0), (300, 0), (1, 2 ** 24)):
        info, plan = aug.aug_attn_plan(s, [0, q_len], [ctx], [0, ctx // 16], 1 << 21, kv_split_tokens=split)
        hdr, items, groups = _decode_plan(plan)
        for j in (0, q_len - 1):
            pos = ctx - q_len + j
            mine = items[(items["kvh"] == 0) & (items["q_row0"] <= j) & (j < items["q_row0"] + items["n_rows"])]
            spans = sorted((int(a), min(int(b), pos + 1)) for a, b in zip(mine["kb"], mine["ke"]) if a <= pos)
            assert spans[0][0] == 0 and spans[-1][1] == pos + 1
            assert all(x[1] == y[0] for x, y in zip(spans, spans[1:]))


def test_empty_batches_launch_nothing():
    L = aug.lib()
    s = aug.make_shape(32, 8, 128, "bf16", "bf16", "bf16", 0.088)
    info, plan = aug.aug_attn_plan(s, [0], [], [0], 64)
    assert info.num_items == 0 and info.num_append_items == 0 and info.workspace_bytes == 0
    assert aug.aug_attn_workspace_size(s, [0], [], [0], 64) == 0
    # every device pointer NULL: nothing is launched, so nothing is dereferenced
    assert L.aug_attn_mixed(aug.C.byref(s), aug.C.byref(info), None, None, None, None, None, None, None, 64, None,
                            None, 0, None) == aug.AUG_OK
    assert L.aug_attn_mixed_noalloc(aug.C.byref(s), aug.C.byref(info), None, None, None, None, None, None, None, 64,
                                    None, None) == aug.AUG_OK


def test_a_plan_for_one_shape_is_refused_for_another():
    """A plan built for 8 query heads per KV head (or any other head count,
    head_dim or dtype set) is refused by a call with another shape, before
    anything is launched: its items, partial sizes and workspace would not fit."""
    L = aug.lib()
    q_lens, ctx_lens = [40, 1, 1], [300, 700, 2100]
    s4 = aug.make_shape(32, 8, 128, "bf16", "bf16", "bf16", 0.088)    # G = 4
    b = make_batch_from_lengths("shape", q_lens, ctx_lens, num_q_heads=32, num_kv_heads=8, head_dim=128,
                                q_dtype="bf16", kv_dtype="bf16", out_dtype="bf16", n_pool_blocks=256, seed=4)
    info, _ = aug.aug_attn_plan(s4, b.q_start, b.ctx_len, b.bt_start, b.num_pool_blocks, kv_split_tokens=64)
    assert info.num_partials > 0
    others = [aug.make_shape(64, 8, 128, "bf16", "bf16", "bf16", 0.088),     # G = 8
              aug.make_shape(32, 4, 128, "bf16", "bf16", "bf16", 0.088),     # other KV heads
              aug.make_shape(32, 8, 64, "bf16", "bf16", "bf16", 0.125),      # other head_dim
              aug.make_shape(32, 8, 128, "bf16", "fp8", "bf16", 0.088)]      # other KV dtype
    for s in others:
        st = L.aug_attn_mixed(aug.C.byref(s), aug.C.byref(info), 8, 8, 8, 8, 8, 8, 8, b.num_pool_blocks, 8, 8,
                              1 << 40, None)
        assert st == aug.AUG_ERR_INVALID and "plan was built for" in aug.aug_last_error()
        st = L.aug_kv_append(aug.C.byref(s), aug.C.byref(info), 8, 8, 8, 8, 8, 8, 8, 8, b.num_pool_blocks, None)
        assert st == aug.AUG_ERR_INVALID and "plan was built for" in aug.aug_last_error()
    # the softmax scale is not part of the plan: another scale is accepted by the checks
    # (a NULL output pointer then stops the call, still before any launch)
    s4b = aug.make_shape(32, 8, 128, "bf16", "bf16", "bf16", 0.5)
    st = L.aug_attn_mixed(aug.C.byref(s4b), aug.C.byref(info), 8, 8, 8, 8, None, None, 8, b.num_pool_blocks,
                          None, 8, 1 << 40, None)
    assert st == aug.AUG_ERR_INVALID and "NULL" in aug.aug_last_error()


def test_row_path_option_resolves_and_is_checked():
    """AUTO runs eight-head groups (head_dim 128, bf16 or fp8 KV) on the MFMA
    row path and everything else on the vector ALUs; VALU can be asked for
    anywhere, MFMA only where it exists (groups of eight or four heads). The
    resolved path is in the info and the plan header, and a call refuses an
    info naming a path its shape lacks."""
    L = aug.lib()
    ctx = [700, 3000, 17]
    q_start, bt_start = [0, 1, 2, 3], np.concatenate([[0], np.cumsum([-(-c // 16) for c in ctx])])
    pool = int(bt_start[-1]) + 4
    g8 = aug.make_shape(64, 8, 128, "bf16", "fp8", "bf16", 0.088)
    g4 = aug.make_shape(32, 8, 128, "bf16", "bf16", "bf16", 0.088)
    info, plan = aug.aug_attn_plan(g8, q_start, ctx, bt_start, pool)
    assert info.row_path == aug.AUG_ROWS_MFMA and plan[61] == aug.AUG_ROWS_MFMA
    info, plan = aug.aug_attn_plan(g8, q_start, ctx, bt_start, pool, row_path=aug.AUG_ROWS_VALU)
    assert info.row_path == aug.AUG_ROWS_VALU and plan[61] == aug.AUG_ROWS_VALU
    info4, _ = aug.aug_attn_plan(g4, q_start, ctx, bt_start, pool)
    assert info4.row_path == aug.AUG_ROWS_VALU
    info4m, plan4m = aug.aug_attn_plan(g4, q_start, ctx, bt_start, pool, row_path=aug.AUG_ROWS_MFMA)
    assert info4m.row_path == aug.AUG_ROWS_MFMA and plan4m[61] == aug.AUG_ROWS_MFMA
    for hq, hkv, d, kv in [(16, 8, 128, "bf16"), (64, 8, 64, "bf16"), (32, 8, 128, "f32"), (64, 4, 128, "bf16")]:
        other = aug.make_shape(hq, hkv, d, "f32" if kv == "f32" else "bf16", kv, "f32" if kv == "f32" else "bf16",
                               0.088)
        with pytest.raises(AugError) as e:
            aug.aug_attn_plan(other, q_start, ctx, bt_start, pool, row_path=aug.AUG_ROWS_MFMA)
        assert e.value.status == aug.AUG_ERR_UNSUPPORTED, (hq, hkv, d, kv)
    with pytest.raises(AugError) as e:
        aug.aug_attn_plan(g8, q_start, ctx, bt_start, pool, row_path=7)
    assert e.value.status == aug.AUG_ERR_INVALID
    desc, keep = aug._batch_desc(q_start, ctx, bt_start, pool)
    opts = aug.aug_plan_options(0, 0)
    opts.reserved = 3
    out = aug.aug_attn_plan_info()
    assert L.aug_attn_plan_opts(aug.C.byref(g8), aug.C.byref(desc), aug.C.byref(opts), None, 0,
                                aug.C.byref(out)) == aug.AUG_ERR_INVALID
    g2 = aug.make_shape(16, 8, 128, "bf16", "bf16", "bf16", 0.088)
    info2, _ = aug.aug_attn_plan(g2, q_start, ctx, bt_start, pool)
    assert info2.row_path == aug.AUG_ROWS_VALU
    bad = aug.aug_attn_plan_info.from_buffer_copy(info2)
    bad.row_path = aug.AUG_ROWS_MFMA
    st = L.aug_attn_mixed(aug.C.byref(g2), aug.C.byref(bad), 8, 8, 8, 8, None, None, 8, pool, 8, 8, 1 << 40, None)
    assert st == aug.AUG_ERR_INVALID and "row path" in aug.aug_last_error()


def test_default_split_doubles_for_mfma_rows_without_tiles():
    """A launch of MFMA row items alone runs eight-wave workgroups and takes
    decode spans twice as long as four-wave row items: 1024 instead of 512
    keys on a small batch, 8192 on a large one. Four-wave row items keep 512
    on a small batch and go up to 6144 keys in a launch of their own, 4096
    beside prefill tiles; an explicit split is taken as given."""
    def plan(shape, q_len, ctx, **kw):
        q_start = np.concatenate([[0], np.cumsum(q_len)])
        bt_start = np.concatenate([[0], np.cumsum([-(-c // 16) for c in ctx])])
        info, _ = aug.aug_attn_plan(shape, q_start, ctx, bt_start, int(bt_start[-1]) + 4, **kw)
        return info
    g8 = aug.make_shape(64, 8, 128, "bf16", "fp8", "bf16", 0.088)
    small, large = [2000] * 20, [3000] * 512
    assert plan(g8, [1] * 20, small).kv_split_tokens == 1024
    assert plan(g8, [1] * 20, small, row_path=aug.AUG_ROWS_VALU).kv_split_tokens == 512
    assert plan(g8, [1] * 19 + [64], small).kv_split_tokens == 512      # one prefill chunk: tiles
    assert plan(g8, [1] * 512, large).kv_split_tokens == 8192
    assert plan(g8, [1] * 512, large, row_path=aug.AUG_ROWS_VALU).kv_split_tokens == 6144
    assert plan(g8, [1] * 511 + [64], large).kv_split_tokens == 4096              # beside tiles
    assert plan(g8, [1] * 511 + [64], large, row_path=aug.AUG_ROWS_VALU).kv_split_tokens == 4096
    assert plan(g8, [1] * 20, small, kv_split_tokens=300).kv_split_tokens == 304
    g4 = aug.make_shape(32, 8, 128, "bf16", "bf16", "bf16", 0.088)
    assert plan(g4, [1] * 20, small).kv_split_tokens == 512
    assert plan(g4, [1] * 20, small, row_path=aug.AUG_ROWS_MFMA).kv_split_tokens == 1024


def test_tile_path_option_resolves_and_is_checked():
    """fp8 products on the tiles are opt-in: AUTO resolves to bf16; FP8_QK
    (scores) and FP8 (scores and values) are accepted for fp8 KV with bf16
    queries (head_dim 128) and refused for other dtype sets; the resolved
    path is in the info and the plan header, and a call refuses an info
    naming a path its shape lacks."""
    L = aug.lib()
    q_start, ctx = [0, 5, 6], [50, 20]
    bt_start = np.concatenate([[0], np.cumsum([-(-c // 16) for c in ctx])])
    pool = int(bt_start[-1]) + 4
    f8 = aug.make_shape(16, 2, 128, "bf16", "fp8", "bf16", 0.088)
    b16 = aug.make_shape(16, 2, 128, "bf16", "bf16", "bf16", 0.088)
    info, plan = aug.aug_attn_plan(f8, q_start, ctx, bt_start, pool)
    assert info.tile_path == aug.AUG_TILES_BF16 and plan[62] == aug.AUG_TILES_BF16
    for tp in (aug.AUG_TILES_FP8_QK, aug.AUG_TILES_FP8):
        info, plan = aug.aug_attn_plan(f8, q_start, ctx, bt_start, pool, tile_path=tp)
        assert info.tile_path == tp and plan[62] == tp
    info16, _ = aug.aug_attn_plan(b16, q_start, ctx, bt_start, pool, tile_path=aug.AUG_TILES_BF16)
    assert info16.tile_path == aug.AUG_TILES_BF16
    f8_d64 = aug.make_shape(16, 2, 64, "bf16", "fp8", "bf16", 0.125)
    for shape in (b16, f8_d64):
        for tp in (aug.AUG_TILES_FP8_QK, aug.AUG_TILES_FP8):
            with pytest.raises(AugError) as e:
                aug.aug_attn_plan(shape, q_start, ctx, bt_start, pool, tile_path=tp)
            assert e.value.status == aug.AUG_ERR_UNSUPPORTED
    with pytest.raises(AugError) as e:
        aug.aug_attn_plan(f8, q_start, ctx, bt_start, pool, tile_path=9)
    assert e.value.status == aug.AUG_ERR_INVALID
    for tp in (aug.AUG_TILES_FP8_QK, aug.AUG_TILES_FP8, 4):
        bad = aug.aug_attn_plan_info.from_buffer_copy(info16)
        bad.tile_path = tp
        st = L.aug_attn_mixed(aug.C.byref(b16), aug.C.byref(bad), 8, 8, 8, 8, None, None, 8, pool, 8, 8, 1 << 40,
                              None)
        assert st == aug.AUG_ERR_INVALID and "tile path" in aug.aug_last_error()


def test_noalloc_attention_rejects_bad_arguments_without_touching_the_gpu():
    L = aug.lib()
    b = synth.make_tiny_mixed(seed=0)
    info, _ = aug.aug_attn_plan(_shape(b), b.q_start, b.ctx_len, b.bt_start, b.num_pool_blocks,
                                kv_split_tokens=32)
    assert info.num_partials > 0
    args = (8, 8, 8, 8, None, None, 8, b.num_pool_blocks, 8, None)
    big = aug.aug_attn_plan_info.from_buffer_copy(info)
    big.workspace_bytes = aug.NOALLOC_SCRATCH_BYTES + 256
    assert L.aug_attn_mixed_noalloc(aug.C.byref(_shape(b)), aug.C.byref(big), *args) == aug.AUG_ERR_NO_SPACE
    assert "scratch" in aug.aug_last_error()
    assert L.aug_attn_mixed_noalloc(aug.C.byref(_shape(b)), aug.C.byref(info), None, *args[1:]) == \
        aug.AUG_ERR_INVALID
    other = aug.make_shape(8, 4, 64, "f32", "f32", "f32", 0.125)
    assert L.aug_attn_mixed_noalloc(aug.C.byref(other), aug.C.byref(info), *args) == aug.AUG_ERR_INVALID


def test_kv_append_rejects_bad_arguments_without_touching_the_gpu():
    L = aug.lib()
    b = synth.make_tiny_mixed(seed=0)
    shape = _shape(b)
    info, _ = aug.aug_attn_plan(shape, b.q_start, b.ctx_len, b.bt_start, b.num_pool_blocks)
    assert info.num_append_items > 0
    args = (8, 8, 8, 8, 8, None, None, 8, b.num_pool_blocks, None)
    # NULL plan image / rows / cache
    assert L.aug_kv_append(aug.C.byref(shape), aug.C.byref(info), None, *args[1:]) == aug.AUG_ERR_INVALID
    assert L.aug_kv_append(aug.C.byref(shape), aug.C.byref(info), 8, None, *args[2:]) == aug.AUG_ERR_INVALID
    # info that does not describe a plan image of this layout
    bad = aug.aug_attn_plan_info.from_buffer_copy(info)
    bad.plan_bytes += 16
    assert L.aug_kv_append(aug.C.byref(shape), aug.C.byref(bad), *args) == aug.AUG_ERR_INVALID
    bad = aug.aug_attn_plan_info.from_buffer_copy(info)
    bad.num_append_items = -1
    assert L.aug_kv_append(aug.C.byref(shape), aug.C.byref(bad), *args) == aug.AUG_ERR_INVALID
    # fp8 cache without scales
    s8 = aug.make_shape(64, 8, 128, "bf16", "fp8", "bf16", 0.088)
    b8 = make_batch_from_lengths("a8", [3, 1], [40, 17], num_q_heads=64, num_kv_heads=8, head_dim=128,
                                 q_dtype="bf16", kv_dtype="fp8", out_dtype="bf16", n_pool_blocks=16, seed=1)
    info8, _ = aug.aug_attn_plan(s8, b8.q_start, b8.ctx_len, b8.bt_start, b8.num_pool_blocks)
    assert L.aug_kv_append(aug.C.byref(s8), aug.C.byref(info8), 8, 8, 8, 8, 8, None, None, 8, 16,
                           None) == aug.AUG_ERR_INVALID
    assert "scales" in aug.aug_last_error()
    # an empty batch appends nothing and launches nothing
    info0, _ = aug.aug_attn_plan(shape, [0], [], [0], b.num_pool_blocks)
    assert info0.num_append_items == 0
    assert L.aug_kv_append(aug.C.byref(shape), aug.C.byref(info0), None, None, None, None, None, None, None,
                           None, b.num_pool_blocks, None) == aug.AUG_OK


def test_planning_from_several_threads_gives_the_serial_plans():
    """The binding releases the GIL inside the planner; plans made on eight
    threads at once must equal the plans made one after another."""
    import threading
    shape = aug.make_shape(32, 8, 128, "bf16", "bf16", "bf16", 0.088)
    batches = []
    for k in range(8):                  # batch descriptions only: the planner reads no KV
        rng = np.random.default_rng(k)
        n = 64 + 32 * k
        q = np.where(rng.random(n) < 0.1, rng.integers(2, 300, n), 1)
        ctx = q + rng.integers(0, 3000, n)
        nblk = (ctx + 15) // 16
        q_start = np.concatenate([[0], np.cumsum(q)])
        bt_start = np.concatenate([[0], np.cumsum(nblk)])
        pool = int(bt_start[-1]) + 16
        batches.append((q_start, ctx, bt_start, pool, rng.permutation(pool)[:bt_start[-1]]))
    want = [aug.aug_attn_plan(shape, *b)[1] for b in batches]
    bad = []

    def worker(k):
        for _ in range(30):
            _, plan = aug.aug_attn_plan(shape, *batches[k])
            if not np.array_equal(plan, want[k]):
                bad.append(k)

    threads = [threading.Thread(target=worker, args=(k,)) for k in range(len(batches))]
    for t in threads:
        t.start()
    for t in threads:
        t.join()
    assert not bad


def test_plan_upload_rejects_bad_arguments_without_touching_the_gpu():
    L = aug.lib()
    # nothing to copy: nothing enqueued, whatever the pointers
    assert L.aug_plan_upload(None, None, 0, None) == aug.AUG_OK
    assert L.aug_plan_upload(None, 4096, 16, None) == aug.AUG_ERR_INVALID
    assert L.aug_plan_upload(4096, None, 16, None) == aug.AUG_ERR_INVALID
    assert "NULL" in aug.aug_last_error()
    # both pointers must be 16-byte aligned
    assert L.aug_plan_upload(4096 + 8, 8192, 64, None) == aug.AUG_ERR_INVALID
    assert L.aug_plan_upload(4096, 8192 + 4, 64, None) == aug.AUG_ERR_INVALID
    assert "aligned" in aug.aug_last_error()


# ---- the former, bit-exact against the oracle --------------------------------------------

from oracle import former as of  # noqa: E402


def _to_c(reqs):
    arr = np.zeros(len(reqs), aug.REQUEST_DTYPE)
    for i, r in enumerate(reqs):
        for f in ("id", "arrival", "last_sched", "pred_call", "pause_start", "state", "seg",
                  "prev_policy", "cur_policy", "seg_ctx", "seg_prefill", "pred_out",
                  "has_next_call", "ctx_len", "pending", "blocks_on_gpu"):
            arr[i][f] = getattr(r, f)
    return arr


def _c_params(p: of.Params, block_size=16):
    return aug.former_params(beta=p.beta, t_max=p.t_max, beta_low=p.beta_low, beta_high=p.beta_high,
                             chunk_cap=p.chunk_cap, t_iter=p.t_iter, fwd_a=p.fwd_a, fwd_b=p.fwd_b,
                             swap_s_per_tok=p.swap_s_per_tok, n_fwd_max=p.n_fwd_max,
                             skip_instead_of_break=p.skip_instead_of_break, block_size=block_size)


def random_requests(rng, n, now):
    reqs = []
    for i in range(n):
        state = int(rng.choice([0, 1, 2, 3], p=[0.25, 0.4, 0.15, 0.2]))
        seg = int(rng.integers(1, 4))
        ctx = int(rng.integers(0, 6000))
        r = of.Request(
            id=int(rng.integers(0, 1 << 40)), arrival=float(rng.uniform(0, now)),
            last_sched=float(rng.uniform(0, now)) if rng.random() < 0.7 else -1.0,
            state=state, seg=seg,
            prev_policy=int(rng.integers(1, 4)) if seg > 1 else 0,
            cur_policy=int(rng.integers(1, 4)) if state == 3 else 0,
            seg_ctx=0 if seg == 1 else int(rng.integers(1, 5000)),
            seg_prefill=int(rng.integers(1, 3000)), pred_out=int(rng.integers(1, 800)),
            pred_call=float(rng.exponential(0.5)), has_next_call=int(rng.random() < 0.6),
            ctx_len=ctx, pending=int(rng.integers(0, 2000)) if rng.random() < 0.4 else 0,
            blocks_on_gpu=0 if state == 2 else -(-ctx // 16), pause_start=float(rng.uniform(0, now)))
        reqs.append(r)
    return reqs


def _compare(reqs, free_blocks, now, p):
    want = of.form_batch(reqs, free_blocks, 16, now, p)
    got = aug.aug_form_batch(_to_c(reqs), free_blocks, now, _c_params(p))
    assert got["budget"] == want.budget
    assert got["ids"].tolist() == want.ids
    assert got["q_len"].tolist() == want.q_len
    assert got["theta"].view(np.uint64).tolist() == np.array(want.theta, np.float64).view(np.uint64).tolist()
    assert got["resume_ids"].tolist() == want.resume_ids
    assert got["park_ids"].tolist() == want.park_ids
    assert got["free_ids"].tolist() == want.free_ids
    assert got["policy"].tolist() == want.policy
    assert got["cost"].view(np.uint64).tolist() == np.array(want.cost, np.float64).view(np.uint64).tolist()
    return want


def test_former_matches_oracle_bit_for_bit_on_random_sets():
    rng = np.random.default_rng(2024)
    nonempty = 0
    for trial in range(300):
        now = float(rng.uniform(1, 100))
        p = of.Params(beta=float(rng.choice([0.0, 5e-5, 1e-3])), t_max=int(rng.choice([256, 2048, 8192])),
                      beta_low=float(rng.choice([0.5, 1.0])), beta_high=float(rng.choice([1.0, 2.0])),
                      chunk_cap=int(rng.choice([256, 512])), t_iter=float(rng.uniform(0.005, 0.05)),
                      fwd_a=float(rng.uniform(0.001, 0.05)), fwd_b=float(rng.uniform(1e-9, 1e-6)),
                      swap_s_per_tok=float(rng.uniform(1e-7, 1e-5)), n_fwd_max=int(rng.integers(1, 8)),
                      skip_instead_of_break=int(rng.random() < 0.3))
        reqs = random_requests(rng, int(rng.integers(0, 120)), now)
        want = _compare(reqs, int(rng.integers(0, 3000)), now, p)
        nonempty += bool(want.ids)
        if want.park_ids or want.free_ids:
            nonempty += 0
    assert nonempty > 200


def test_former_matches_oracle_on_the_2048_token_mixed_batch():
    from tests.test_oracle_former import _mixed_2048_requests
    p = of.Params(t_max=2048, beta_low=0.5, beta_high=1.0, chunk_cap=512)
    want = _compare(_mixed_2048_requests(), 131_072, 2.0, p)
    assert len(want.ids) == 515
    _compare(_mixed_2048_requests(extra_decode=True), 131_072, 2.0, p)


def test_former_rejects_bad_inputs():
    p = _c_params(of.Params())
    bad = _to_c([of.Request(id=1, arrival=0.0, state=1, pred_out=0)])
    with pytest.raises(AugError):
        aug.aug_form_batch(bad, 10, 1.0, p)
    bad = _to_c([of.Request(id=1, arrival=0.0, state=7, pred_out=1)])
    with pytest.raises(AugError):
        aug.aug_form_batch(bad, 10, 1.0, p)
    q = _c_params(of.Params(t_iter=0.0))
    with pytest.raises(AugError):
        aug.aug_form_batch(_to_c([]), 10, 1.0, q)
    assert aug.aug_form_batch(_to_c([]), 10, 1.0, p)["ids"].size == 0
