"""Pins of the KV-append oracle (CPU only): the E4M3FN encoder against the
OCP value table by brute force, the placement of new rows against the
attention oracle's independent gather, the fp8 scale rule's error bounds, and
the plan image's append list against the oracle's segments."""

import os

import numpy as np
import pytest

from oracle import attention as oa
from oracle import codecs, kvappend
import synth
from synth.attn_inputs import make_batch_from_lengths

import paper_2512_04013_amd as aug


def _batch(q_lens, ctx_lens, kv="f32", hq=4, hkv=2, d=8, seed=0, pool=96):
    qd = "f32" if kv == "f32" else "bf16"
    return make_batch_from_lengths("a", q_lens, ctx_lens, num_q_heads=hq, num_kv_heads=hkv, head_dim=d,
                                   q_dtype=qd, kv_dtype=kv, out_dtype=qd, n_pool_blocks=pool, seed=seed)


def _bf16_to_f32(bits):
    return (np.asarray(bits, np.uint32) << 16).view(np.float32)


# ---- the encoder --------------------------------------------------------------

FINITE = np.array([c for c in range(256) if (c & 0x7F) != 0x7F], np.uint8)


def test_encoder_round_trips_every_finite_code():
    vals = codecs.E4M3FN_TABLE[FINITE].astype(np.float32)
    assert np.array_equal(codecs.e4m3fn_encode(vals), FINITE)


def test_encoder_is_nearest_value_by_brute_force():
    rng = np.random.default_rng(5)
    x = np.concatenate([rng.standard_normal(20000) * 50, rng.standard_normal(20000) * 0.01,
                        rng.uniform(-470, 470, 5000)]).astype(np.float32)
    got = codecs.e4m3fn_encode(x)
    vals = codecs.E4M3FN_TABLE[FINITE]
    # distance of every input to every finite value; the encoder's pick must be one of the nearest
    dist = np.abs(np.minimum(np.abs(x.astype(np.float64)), 448.0)[:, None] * np.sign(x)[:, None] - vals[None, :])
    best = dist.min(axis=1)
    got_val = codecs.E4M3FN_TABLE[got]
    assert np.all(np.abs(np.clip(x, -448, 448) - got_val) == best)


def test_encoder_ties_go_to_even_mantissa_and_large_values_saturate():
    vals = codecs.E4M3FN_TABLE[:0x7F]
    mids = ((vals[:-1] + vals[1:]) / 2).astype(np.float32)
    exact = mids.astype(np.float64) == (vals[:-1] + vals[1:]) / 2
    codes = codecs.e4m3fn_encode(mids[exact]).astype(int)
    assert np.all(codes % 2 == 0)
    assert np.all(np.isin(codes, np.nonzero(exact)[0]) | np.isin(codes, np.nonzero(exact)[0] + 1))
    big = np.array([448.0, 449.0, 464.0, 1e6, 3e38], np.float32)
    assert np.all(codecs.e4m3fn_encode(big) == 0x7E)
    assert np.all(codecs.e4m3fn_encode(-big) == 0xFE)
    assert codecs.e4m3fn_encode(np.array([-0.0], np.float32))[0] == 0x80
    # smallest subnormal 2^-9: half of it is a tie that goes to zero, a bit more rounds up
    assert codecs.e4m3fn_encode(np.array([2.0 ** -10], np.float32))[0] == 0
    assert codecs.e4m3fn_encode(np.array([2.0 ** -10 * 1.01], np.float32))[0] == 1


# ---- placement ----------------------------------------------------------------

@pytest.mark.parametrize("kv", ["f32", "bf16"])
def test_append_puts_row_j_at_position_ctx_minus_q_plus_j(kv):
    # prefill chunks that start mid-block, span several blocks and end mid-block; decodes at slot 0 and 15
    b = synth.poison_new_slots(_batch([20, 1, 1, 33, 1], [25, 17, 16, 70, 1], kv=kv, seed=2))
    k_new, v_new = synth.make_new_kv(b, seed=9)
    k, v, _, _ = kvappend.append(b.k_cache, b.v_cache, None, None, kv, k_new, v_new, b.q_start,
                                 b.ctx_len, b.bt_start, b.block_ids)
    to64 = (lambda x: x.astype(np.float64)) if kv == "f32" else (lambda x: _bf16_to_f32(x).astype(np.float64))
    for r in range(b.num_reqs):
        ctx, q = int(b.ctx_len[r]), int(b.q_len[r])
        got_k = oa.materialise_kv(k, None, kv, b.blocks_of(r), ctx)
        got_v = oa.materialise_kv(v, None, kv, b.blocks_of(r), ctx)
        old_k = oa.materialise_kv(b.k_cache, None, kv, b.blocks_of(r), ctx)
        rows = slice(int(b.q_start[r]), int(b.q_start[r + 1]))
        assert np.array_equal(got_k[ctx - q:], to64(k_new[rows]))
        assert np.array_equal(got_v[ctx - q:], to64(v_new[rows]))
        assert np.array_equal(got_k[:ctx - q], old_k[:ctx - q])         # earlier context untouched
    assert np.isfinite(oa.attention_for(b, k_cache=k, v_cache=v)).all()
    # every byte outside the new positions is unchanged (the poison past each context included)
    changed = np.zeros(b.k_cache.shape[:1] + b.k_cache.shape[2:3], bool)   # [block, slot]
    for r in range(b.num_reqs):
        for p in range(int(b.ctx_len[r]) - int(b.q_len[r]), int(b.ctx_len[r])):
            changed[b.blocks_of(r)[p // 16], p % 16] = True
    same = ~changed
    kb = b.k_cache.transpose(0, 2, 1, 3)[same]
    assert np.array_equal(k.transpose(0, 2, 1, 3)[same].view(np.uint8), kb.view(np.uint8))


def test_segments_cover_each_row_once_within_one_block():
    q_start = np.array([0, 40, 41, 58], np.int32)
    ctx_len = np.array([47, 1, 400], np.int32)
    bt_start = np.array([0, 3, 4, 29], np.int32)
    segs = kvappend.append_segments(q_start, ctx_len, bt_start)
    rows = np.concatenate([np.arange(r0, r0 + n) for _, _, r0, n, _ in segs])
    assert np.array_equal(np.sort(rows), np.arange(58))
    for r, blk, r0, n, slot0 in segs:
        assert 1 <= n and slot0 + n <= 16
        pos0 = int(ctx_len[r]) - int(q_start[r + 1] - q_start[r]) + (r0 - int(q_start[r]))
        assert pos0 // 16 == blk and pos0 % 16 == slot0


# ---- fp8 scale rule -----------------------------------------------------------

def _fp8_case(q_lens, ctx_lens, seed, std):
    b = synth.poison_new_slots(_batch(q_lens, ctx_lens, kv="fp8", hq=8, hkv=2, d=128, seed=seed))
    k_new, v_new = synth.make_new_kv(b, seed=seed + 100, std=std)
    k, v, ks, vs = kvappend.append(b.k_cache, b.v_cache, b.k_scale, b.v_scale, "fp8", k_new, v_new,
                                   b.q_start, b.ctx_len, b.bt_start, b.block_ids)
    return b, k_new, v_new, k, v, ks, vs


def _max_err_bound(x, scale):
    # E4M3 keeps 3 mantissa bits: half an ulp is 2^-4 of the value for normal
    # codes, and 2^-10 of the scale (half the subnormal step) near zero
    return np.maximum(np.abs(x) * 2.0 ** -4, scale * 2.0 ** -10) * (1 + 1e-6)


@pytest.mark.parametrize("std", [0.2, 1.0, 5.0])
def test_fp8_append_new_rows_decode_within_half_an_ulp(std):
    b, k_new, _, k, _, ks, _ = _fp8_case([20, 1, 1, 33], [25, 17, 40, 70], seed=3, std=std)
    x_all = _bf16_to_f32(k_new).astype(np.float64)
    for r in range(b.num_reqs):
        ctx, q = int(b.ctx_len[r]), int(b.q_len[r])
        got = oa.materialise_kv(k, ks, "fp8", b.blocks_of(r), ctx)[ctx - q:]
        x = x_all[int(b.q_start[r]):int(b.q_start[r + 1])]
        for j in range(q):
            p = ctx - q + j
            s = ks[b.blocks_of(r)[p // 16]].astype(np.float64)          # [H_kv]
            assert np.all(np.abs(got[j] - x[j]) <= _max_err_bound(x[j], s[:, None]))


def test_fp8_block_opened_at_slot_zero_takes_new_max_over_448():
    b, k_new, _, k, _, ks, _ = _fp8_case([16], [32], seed=4, std=1.0)   # exactly block 1 of the request
    blk = b.blocks_of(0)[1]
    x = _bf16_to_f32(k_new).reshape(16, 2, 128)
    want = np.abs(x).max(axis=(0, 2)).astype(np.float32) / np.float32(448.0)
    assert np.array_equal(ks[blk].view(np.uint32), want.view(np.uint32))
    # the largest element of each head encodes to +-448
    assert np.all((k[blk] & 0x7F).max(axis=(1, 2)) == 0x7E)


def test_fp8_growing_scale_reencodes_earlier_tokens_within_bounds():
    # decode into a half-full block with new values far above the block's range
    b, k_new, _, k, _, ks, _ = _fp8_case([1], [24], seed=6, std=40.0)
    blk = b.blocks_of(0)[1]
    old = oa.materialise_kv(b.k_cache, b.k_scale, "fp8", b.blocks_of(0), 23)[16:23]   # slots 0..6
    new = oa.materialise_kv(k, ks, "fp8", b.blocks_of(0), 23)[16:23]
    assert np.all(ks[blk] > b.k_scale[blk])
    # re-encoding one value at the new, coarser scale: error within half an ulp at that scale
    s = ks[blk].astype(np.float64)[None, :, None]
    assert np.all(np.abs(new - old) <= _max_err_bound(old, s))
    assert np.array_equal(k[blk, :, 8:], b.k_cache[blk, :, 8:])        # poison past the context kept


def test_fp8_shrinking_values_keep_the_block_scale_and_codes():
    b, _, _, k, _, ks, _ = _fp8_case([1], [24], seed=6, std=1e-3)
    blk = b.blocks_of(0)[1]
    assert np.array_equal(ks[blk].view(np.uint32), b.k_scale[blk].view(np.uint32))
    assert np.array_equal(k[blk, :, :7], b.k_cache[blk, :, :7])


def test_fp8_token_by_token_decode_matches_its_own_replay():
    # 16 decode steps filling one block one token at a time; each step appends
    # into the cache the previous one produced. The end state has every token
    # within the error bound of the block's final scale accumulated over the
    # re-encodes (each re-encode adds at most half an ulp at a scale no larger
    # than the final one).
    b = synth.poison_new_slots(_batch([16], [16], kv="fp8", hq=8, hkv=2, d=128, seed=8))
    k_all, v_all = synth.make_new_kv(b, seed=1, std=1.0)
    kc, vc, ks, vs = b.k_cache.copy(), b.v_cache.copy(), b.k_scale.copy(), b.v_scale.copy()
    for t in range(16):
        qs = np.array([0, 1], np.int32)
        cl = np.array([t + 1], np.int32)
        kc, vc, ks, vs = kvappend.append(kc, vc, ks, vs, "fp8", k_all[t:t + 1], v_all[t:t + 1], qs, cl,
                                         b.bt_start, b.block_ids)
    got = oa.materialise_kv(kc, ks, "fp8", b.blocks_of(0), 16)
    x = _bf16_to_f32(k_all).astype(np.float64)
    s = ks[b.blocks_of(0)[0]].astype(np.float64)[None, :, None]
    assert np.all(np.abs(got - x) <= 16 * _max_err_bound(x, s))
    assert np.allclose(s[0, :, 0], np.abs(x).max(axis=(0, 2)) / 448, rtol=1e-6)


# ---- the plan image's append list (host code of the library) ---------------------

@pytest.mark.skipif(not os.path.exists(aug.LIB_PATH), reason="libaug.so not built")
def test_plan_append_items_match_oracle_segments():
    b = _batch([20, 1, 1, 33, 1, 7], [25, 17, 16, 70, 1, 7], kv="bf16", hq=8, hkv=2, d=64, seed=2)
    shape = aug.make_shape(8, 2, 64, "bf16", "bf16", "bf16", 0.125)
    info, plan = aug.aug_attn_plan(shape, b.q_start, b.ctx_len, b.bt_start, b.num_pool_blocks, b.block_ids)
    hdr = plan[:64].view(np.int32)
    off, n = int(hdr[11]), int(hdr[12])
    assert n == info.num_append_items
    items = plan[off:off + 16 * n].view(np.int32).reshape(n, 4)
    segs = kvappend.append_segments(b.q_start, b.ctx_len, b.bt_start)
    assert n == len(segs)
    for (r, blk, r0, cnt, slot0), it in zip(segs, items):
        assert it[0] == r0
        assert (it[1] & 0xFFFF) == cnt and (it[1] >> 16) == slot0
        assert it[2] == int(b.bt_start[r]) + blk


@pytest.mark.skipif(not os.path.exists(aug.LIB_PATH), reason="libaug.so not built")
def test_plan_rejects_a_block_receiving_new_tokens_twice():
    shape = aug.make_shape(4, 4, 64, "f32", "f32", "f32", 0.125)
    q_start, ctx_len, bt_start = [0, 1, 2], [5, 9], [0, 1, 2]
    with pytest.raises(aug.AugError):
        aug.aug_attn_plan(shape, q_start, ctx_len, bt_start, 8, block_ids=[3, 3])
    info, _ = aug.aug_attn_plan(shape, q_start, ctx_len, bt_start, 8, block_ids=[3, 4])
    assert info.num_append_items == 2
