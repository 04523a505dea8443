"""Pins of the attention and park/resume oracles against closed forms,
invariants, brute force and library codecs (CPU only)."""

import copy

import numpy as np
import pytest
import torch

from oracle import attention as oa
from oracle import brute, codecs, kvpark
import synth
from synth.attn_inputs import make_batch_from_lengths


def _tiny(q_lens, ctx_lens, hq=4, hkv=2, d=8, kv="f32", qd="f32", seed=0, pool=64, **kw):
    return make_batch_from_lengths("t", q_lens, ctx_lens, num_q_heads=hq, num_kv_heads=hkv,
                                   head_dim=d, q_dtype=qd, kv_dtype=kv, out_dtype="f32",
                                   n_pool_blocks=pool, seed=seed, **kw)


def _set_token(b, cache, r, t, g, vec):
    blk = b.blocks_of(r)[t // 16]
    cache[blk, g, t % 16, :] = vec


# ---- closed forms -------------------------------------------------------------

def test_single_key_returns_v_exactly():
    b = _tiny([1], [1])
    out = oa.attention_for(b)
    v0 = b.v_cache[b.blocks_of(0)[0], :, 0, :].astype(np.float64)   # [H_kv, D]
    for h in range(4):
        assert np.array_equal(out[0, h], v0[h // 2])


def test_identical_keys_give_prefix_mean_of_v():
    b = _tiny([5], [40], seed=3)
    rng = np.random.default_rng(1)
    kvec = rng.standard_normal((2, 8)).astype(np.float32)
    for t in range(40):
        for g in range(2):
            _set_token(b, b.k_cache, 0, t, g, kvec[g])
    out = oa.attention_for(b)
    v = oa.materialise_kv(b.v_cache, None, "f32", b.blocks_of(0), 40)
    for j in range(5):
        pos = 40 - 5 + j
        for h in range(4):
            np.testing.assert_allclose(out[j, h], v[:pos + 1, h // 2].mean(axis=0), rtol=0, atol=1e-12)


def test_dominant_logit_selects_its_value():
    b = _tiny([1], [50], seed=4)
    q = b.q[0].astype(np.float64)
    # make key 17 of every KV head 60x the (group-mean) query: its logit dwarfs the rest
    for g in range(2):
        _set_token(b, b.k_cache, 0, 17, g, (60.0 * q[2 * g]).astype(np.float32))
        _set_token(b, b.k_cache, 0, 17, g, (60.0 * q[2 * g]).astype(np.float32))
    out = oa.attention_for(b)
    v17 = oa.materialise_kv(b.v_cache, None, "f32", b.blocks_of(0), 50)[17]
    np.testing.assert_allclose(out[0, 0], v17[0], atol=1e-9)
    np.testing.assert_allclose(out[0, 2], v17[1], atol=1e-9)


# ---- invariants ------------------------------------------------------------------

def test_shift_invariance_of_keys():
    b = _tiny([3, 1], [30, 70], seed=5)
    base = oa.attention_for(b)
    u = np.random.default_rng(2).standard_normal((2, 8)).astype(np.float32)
    b2 = copy.deepcopy(b)
    for r in range(2):
        for t in range(int(b.ctx_len[r])):
            for g in range(2):
                blk = b.blocks_of(r)[t // 16]
                b2.k_cache[blk, g, t % 16] = b.k_cache[blk, g, t % 16] + u[g]
    # the shift adds q.u to every logit of a row; the f32 sum k+u rounds, so compare loosely
    np.testing.assert_allclose(oa.attention_for(b2), base, atol=2e-5)


def test_linearity_in_values():
    # values with 8-bit significands, so 2*v1 - 3*v2 is exact in float32 storage
    def coarse(x):
        return (synth.round_to_bf16_bits(x).astype(np.uint32) << 16).view(np.float32)
    b = _tiny([4, 1], [20, 33], seed=6)
    b.v_cache = coarse(np.nan_to_num(b.v_cache))
    b2 = copy.deepcopy(b)
    b2.v_cache = coarse(np.random.default_rng(3).standard_normal(b.v_cache.shape).astype(np.float32))
    b3 = copy.deepcopy(b)
    b3.v_cache = (np.float32(2.0) * b.v_cache - np.float32(3.0) * b2.v_cache)
    assert np.array_equal(b3.v_cache.astype(np.float64),
                          2.0 * b.v_cache.astype(np.float64) - 3.0 * b2.v_cache.astype(np.float64))
    o1, o2, o3 = oa.attention_for(b), oa.attention_for(b2), oa.attention_for(b3)
    np.testing.assert_allclose(o3, 2.0 * o1 - 3.0 * o2, atol=1e-10)


def test_decode_row_equals_last_row_of_full_prefill():
    full = _tiny([37], [37], seed=7)
    dec = copy.deepcopy(full)
    dec.q = full.q[36:37].copy()
    dec.q_start = np.array([0, 1], np.int32)
    o_full = oa.attention_for(full)
    o_dec = oa.attention_for(dec)
    np.testing.assert_allclose(o_dec[0], o_full[36], rtol=0, atol=1e-13)


def test_two_chunks_equal_one_chunk():
    one = _tiny([32], [80], seed=8)
    two = copy.deepcopy(one)
    # same request split as two requests over the same blocks: rows 0..15 (ctx 64), 16..31 (ctx 80)
    two.q_start = np.array([0, 16, 32], np.int32)
    two.ctx_len = np.array([64, 80], np.int32)
    blocks = one.blocks_of(0)
    two.bt_start = np.array([0, 4, 4 + len(blocks)], np.int32)
    two.block_ids = np.concatenate([blocks[:4], blocks]).astype(np.int32)
    np.testing.assert_allclose(oa.attention_for(two), oa.attention_for(one), rtol=0, atol=1e-13)


def test_gqa_equals_mha_with_replicated_kv_heads():
    g = _tiny([3, 1], [25, 40], hq=4, hkv=2, seed=9)
    m = copy.deepcopy(g)
    m.num_kv_heads = 4
    m.k_cache = np.repeat(g.k_cache, 2, axis=1)
    m.v_cache = np.repeat(g.v_cache, 2, axis=1)
    np.testing.assert_array_equal(oa.attention_for(m), oa.attention_for(g))


def test_block_permutation_is_bit_identical():
    b = synth.make_tiny_mixed(seed=11)
    base = oa.attention_for(b)
    perm = np.random.default_rng(5).permutation(b.num_pool_blocks)
    b2 = copy.deepcopy(b)
    b2.k_cache = np.empty_like(b.k_cache)
    b2.v_cache = np.empty_like(b.v_cache)
    b2.k_cache[perm] = b.k_cache
    b2.v_cache[perm] = b.v_cache
    b2.block_ids = perm[b.block_ids].astype(np.int32)
    np.testing.assert_array_equal(oa.attention_for(b2), base)


def test_unused_slots_are_nan_and_never_read():
    b = synth.make_tiny_mixed(seed=12)
    # the generator poisons every slot outside the contexts
    r = int(np.argmax(b.ctx_len % 16 != 0))
    last = b.blocks_of(r)[-1]
    assert np.isnan(b.k_cache[last, :, int(b.ctx_len[r]) % 16:]).all()
    out = oa.attention_for(b)
    assert np.isfinite(out).all()
    # poisoning a slot inside a context does reach the output
    b.v_cache[b.blocks_of(r)[0], 0, 0, 0] = np.nan
    assert np.isnan(oa.attention_for(b)).any()


def test_requests_subset_matches_full():
    b = synth.make_tiny_mixed(seed=13)
    full = oa.attention_for(b)
    part = oa.attention_for(b, requests=[1, 4])
    for r in (1, 4):
        s = slice(b.q_start[r], b.q_start[r + 1])
        np.testing.assert_array_equal(part[s], full[s])
    assert np.isnan(part[b.q_start[0]:b.q_start[1]]).all()


# ---- brute force ---------------------------------------------------------------------

@pytest.mark.parametrize("seed", [0, 1])
def test_numpy_oracle_matches_scalar_brute_force_on_tiny_mixed(seed):
    b = synth.make_tiny_mixed(seed=seed)
    # trim to keep the scalar loops to a few seconds: 1 prefill + 3 decodes
    keep = [int(np.argmax(b.q_len > 1))] + [int(i) for i in np.nonzero(b.q_len == 1)[0][:3]]
    ref = oa.attention_for(b)
    got = brute.brute_attention(b.q, "f32", b.k_cache, b.v_cache, None, None, "f32",
                                b.q_start, b.ctx_len, b.bt_start, b.block_ids, 4, 4,
                                b.softmax_scale)
    got = np.array(got)
    for r in keep:
        s = slice(b.q_start[r], b.q_start[r + 1])
        np.testing.assert_allclose(got[s], ref[s], rtol=0, atol=1e-12)


@pytest.mark.parametrize("kv", ["bf16", "fp8"])
def test_numpy_oracle_matches_brute_force_low_precision(kv):
    b = _tiny([3, 1, 2], [20, 35, 17], hq=4, hkv=2, d=16, kv=kv, qd="bf16", seed=21)
    ref = oa.attention_for(b)
    got = np.array(brute.brute_attention(b.q, "bf16", b.k_cache, b.v_cache, b.k_scale, b.v_scale,
                                         kv, b.q_start, b.ctx_len, b.bt_start, b.block_ids, 4, 2,
                                         b.softmax_scale))
    np.testing.assert_allclose(got, ref, rtol=0, atol=1e-12)


# ---- codecs --------------------------------------------------------------------------

def test_e4m3fn_decoder_matches_torch_for_all_codes():
    codes = np.arange(256, dtype=np.uint8)
    ours = codecs.e4m3fn_bits_to_f64(codes)
    theirs = torch.from_numpy(codes).view(torch.float8_e4m3fn).double().numpy()
    assert np.array_equal(np.isnan(ours), np.isnan(theirs))
    ok = ~np.isnan(ours)
    assert np.array_equal(ours[ok], theirs[ok])


def test_e4m3fn_spec_points():
    v = codecs.e4m3fn_value
    assert v(0x7E) == 448.0 and v(0xFE) == -448.0
    assert v(0x01) == 2.0 ** -9 and v(0x08) == 2.0 ** -6 and v(0x07) == 7 * 2.0 ** -9
    assert v(0x38) == 1.0 and v(0xC0) == -2.0 and v(0x30) == 0.5
    assert np.isnan(v(0x7F)) and np.isnan(v(0xFF))
    pos = [v(c) for c in range(0x7F)]
    assert all(a < b for a, b in zip(pos, pos[1:]))


def test_bf16_decoder_matches_torch():
    u = np.random.default_rng(0).integers(0, 65536, size=4096).astype(np.uint16)
    u = u[((u >> 7) & 0xFF) != 0xFF]                       # drop inf/nan patterns
    ours = codecs.bf16_bits_to_f64(u)
    theirs = torch.from_numpy(u.view(np.int16)).view(torch.bfloat16).double().numpy()
    assert np.array_equal(ours, theirs)


def test_input_encoders_agree_with_torch():
    x = np.random.default_rng(1).standard_normal(20000).astype(np.float32) * 50
    bf = synth.round_to_bf16_bits(x)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(bf, ref)
    y = np.clip(x, -440, 440)
    f8 = synth.encode_e4m3fn_bits(y)
    ref8 = torch.from_numpy(y).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    assert np.array_equal(f8, ref8)
    assert synth.encode_e4m3fn_bits(np.array([1e6, -1e6], np.float32)).tolist() == [0x7E, 0xFE]


# ---- park / resume -----------------------------------------------------------------

def test_park_image_layout_hand_example():
    k = np.arange(2 * 1 * 16 * 2, dtype=np.uint16).reshape(2, 1, 16, 2)
    v = (1000 + np.arange(2 * 1 * 16 * 2, dtype=np.uint16)).reshape(2, 1, 16, 2)
    img = kvpark.park(k, v, None, None, "bf16", [1])
    assert img.size == kvpark.record_bytes(1, 2, "bf16") == 128
    words = img.view(np.uint16)
    assert words[:32].tolist() == list(range(32, 64))
    assert words[32:].tolist() == list(range(1032, 1064))


def test_park_then_resume_elsewhere_restores_bytes_fp8():
    b = _tiny([1, 1], [40, 70], hq=8, hkv=2, d=16, kv="fp8", qd="bf16", seed=31,
              extra_reqs_ctx=[50])
    src = b.park.park_blocks
    used = set(b.block_ids.tolist()) | set(src.tolist())
    dst = np.array(sorted(set(range(b.num_pool_blocks)) - used)[:len(src)], np.int32)
    img = kvpark.park(b.k_cache, b.v_cache, b.k_scale, b.v_scale, "fp8", src)
    assert img.size == len(src) * kvpark.record_bytes(2, 16, "fp8")
    k2, v2, ks2, vs2 = kvpark.resume(b.k_cache, b.v_cache, b.k_scale, b.v_scale, "fp8", dst, img)
    assert np.array_equal(k2[dst], b.k_cache[src]) and np.array_equal(v2[dst], b.v_cache[src])
    assert np.array_equal(ks2[dst], b.k_scale[src]) and np.array_equal(vs2[dst], b.v_scale[src])
    others = np.setdiff1d(np.arange(b.num_pool_blocks), dst)
    assert np.array_equal(k2[others].view(np.uint8), b.k_cache[others].view(np.uint8))


def test_resumed_batch_attention_equals_original_placement():
    b = synth.make_mixed_8b(seed=2, n_dec=24, n_pre=1, n_pool_blocks=4096)
    pk = b.park
    img = kvpark.park(b.k_cache, b.v_cache, None, None, "bf16", pk.resume_src_blocks)
    k2, v2, _, _ = kvpark.resume(b.k_cache, b.v_cache, None, None, "bf16", pk.resume_blocks, img)
    # before the resume the destination blocks are NaN, after it every row is finite
    assert np.isnan(oa.attention_for(b)).any()
    out = oa.attention_for(b, k_cache=k2, v_cache=v2)
    assert np.isfinite(out).all()


# ---- queries rounded to E4M3 (the opt-in fp8 score arithmetic of prefill tiles) ----------

def _nearest_by_search(x, scale):
    """Brute force: the E4M3FN value times `scale` nearest to x (ties to the
    even code), over all 254 finite codes, element by element."""
    table = codecs.E4M3FN_TABLE
    finite = [c for c in range(256) if np.isfinite(table[c])]
    out = np.empty_like(x)
    for i, xi in enumerate(x.ravel()):
        best, best_d = None, None
        for c in finite:
            d = abs(table[c] * scale - xi)
            if best is None or d < best_d or (d == best_d and (c & 1) == 0 and (best & 1) == 1):
                best, best_d = c, d
        out.ravel()[i] = table[best] * scale
    return out


def test_rounded_queries_on_the_grid_are_unchanged():
    # a vector whose largest magnitude is 448 x 2^-5 and whose entries are all
    # E4M3 values times 2^-5: scale 2^-5 exactly, so rounding changes nothing
    rng = np.random.default_rng(0)
    codes = rng.integers(0, 0x7F, size=(3, 2, 128)).astype(np.uint8)
    vals = codecs.e4m3fn_bits_to_f64(codes) * np.where(rng.random((3, 2, 128)) < 0.5, -1, 1)
    vals[..., 7] = 448.0
    q = vals * 2.0 ** -5
    np.testing.assert_array_equal(oa.round_query_rows_e4m3(q), q)


def test_rounded_queries_are_the_nearest_scaled_e4m3_values():
    rng = np.random.default_rng(1)
    q = torch.from_numpy(rng.standard_normal((2, 2, 32))).to(torch.bfloat16).double().numpy()
    got = oa.round_query_rows_e4m3(q)
    for r in range(2):
        for h in range(2):
            amax = np.float32(np.abs(q[r, h]).max())
            scale = float(amax * np.float32(1.0 / 448.0))
            x = q[r, h].astype(np.float32) * (np.float32(448.0) / amax)
            want = _nearest_by_search(x.astype(np.float64), 1.0) * scale
            np.testing.assert_array_equal(got[r, h], want)
    # relative error of 3 mantissa bits in the normal range, and the largest
    # magnitude maps to 448 x scale (the vector's own maximum, up to rounding)
    rel = np.abs(got - q) / np.maximum(np.abs(q), 1e-30)
    normal = np.abs(q) >= np.abs(q).max(axis=-1, keepdims=True) * 2.0 ** -6 / 448   # E4M3 normals
    assert (rel[normal] <= 2.0 ** -4 + 1e-7).all()
    np.testing.assert_allclose(np.abs(got).max(axis=-1), np.abs(q).max(axis=-1), rtol=2e-7)


def test_rounded_queries_zero_vector_and_chunk_rows_only():
    assert (oa.round_query_rows_e4m3(np.zeros((1, 1, 16))) == 0).all()
    tiny = np.zeros((1, 1, 16))
    tiny[0, 0, 3] = 2.0 ** -120          # its reciprocal scale would overflow float32
    assert (oa.round_query_rows_e4m3(tiny) == 0).all()
    b = make_batch_from_lengths("fp8q", [1, 5, 1], [40, 70, 33], num_q_heads=8, num_kv_heads=2,
                                head_dim=128, q_dtype="bf16", kv_dtype="fp8", out_dtype="bf16",
                                n_pool_blocks=64, seed=5)
    plain = oa.attention_for(b)
    rounded = oa.attention_for(b, fp8_chunk_queries=True)
    dec = np.r_[0, 6]                      # the two decode rows: untouched
    np.testing.assert_array_equal(rounded[dec], plain[dec])
    assert not np.array_equal(rounded[1:6], plain[1:6])
