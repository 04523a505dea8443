"""Oracle for appending a step's new K/V rows to the paged cache.

TEST INFRASTRUCTURE ONLY: imported by the test suite, the smoke check and the
benchmark's CPU-baseline leg, never by the library or its binding.

Every query row of a formed batch is a token whose K and V the step's forward
pass produces (the chunk or decode token scheduled in Algorithm 1, step (5);
prefill, returned-token and recompute stages of the problem formulation).
Before attention reads the cache, those K/V rows are written into the
request's blocks: row j of request r sits at context position
p = ctx_len[r] - q_len[r] + j, in slot p mod 16 of block
block_ids[bt_start[r] + p // 16], for every KV head.

The paper fixes no cache format; the reading taken here:

* f32 and bf16 caches: the new rows come in the cache's own format and are
  stored unchanged (a byte copy).
* fp8 E4M3FN caches keep one float32 scale per (block, KV head), separately
  for K and V (value = code * scale). New rows come as bf16. For each block
  and KV head that receives new tokens, with a = the largest |x| among them:
    - if the request's first new token in the block lands in slot 0 (the block
      holds nothing of the request yet): s = a / 448;
    - otherwise s = max(s_old, a / 448), and if s > s_old every earlier token
      of the block is re-encoded: code <- enc((dec(code) * s_old) / s);
    - new tokens: code = enc(x / s), or 0 when s == 0;
    - the block's scale becomes s.
  enc is round-to-nearest-even to E4M3FN saturating at +-448
  (``codecs.e4m3fn_encode``); every product and quotient above is one IEEE
  float32 operation, in the order written.
"""

from __future__ import annotations

import numpy as np

from .codecs import E4M3FN_TABLE, bf16_bits_to_f64, e4m3fn_encode

BLOCK = 16
FP8_MAX = np.float32(448.0)


def append_segments(q_start, ctx_len, bt_start):
    """(request, block index within the request, first row, rows, first slot)
    for every block that receives new tokens, in request order."""
    out = []
    for r in range(len(ctx_len)):
        q = int(q_start[r + 1] - q_start[r])
        first = int(ctx_len[r]) - q
        p = first
        while p < int(ctx_len[r]):
            blk = p // BLOCK
            end = min(int(ctx_len[r]), (blk + 1) * BLOCK)
            out.append((r, blk, int(q_start[r]) + p - first, end - p, p % BLOCK))
            p = end
    return out


def _append_fp8(cache, scale, new_bits, segs, bt_start, block_ids, h_kv):
    for r, blk, row0, n, slot0 in segs:
        b = int(block_ids[int(bt_start[r]) + blk])
        for h in range(h_kv):
            x = bf16_bits_to_f64(new_bits[row0:row0 + n, h, :]).astype(np.float32)
            a = np.float32(np.abs(x).max())
            need = np.float32(a / FP8_MAX)
            s_old = np.float32(scale[b, h])
            if slot0 == 0:
                s = need
            else:
                s = need if need > s_old else s_old
                if s > s_old:
                    old = E4M3FN_TABLE[cache[b, h, :slot0, :]].astype(np.float32)
                    cache[b, h, :slot0, :] = e4m3fn_encode(np.float32(old * s_old) / s)
            if s == 0:
                codes = np.zeros(x.shape, np.uint8)
            else:
                codes = e4m3fn_encode(x / s)
            cache[b, h, slot0:slot0 + n, :] = codes
            scale[b, h] = s


def append(k_cache, v_cache, k_scale, v_scale, kv_dtype, k_new, v_new, q_start, ctx_len, bt_start,
           block_ids):
    """Return copies of (k_cache, v_cache, k_scale, v_scale) after appending
    k_new, v_new ([rows][H_kv][D]: float32 for f32 caches, bf16 bit patterns
    otherwise) for the batch (q_start, ctx_len, bt_start, block_ids)."""
    k, v = k_cache.copy(), v_cache.copy()
    ks = None if k_scale is None else k_scale.copy()
    vs = None if v_scale is None else v_scale.copy()
    segs = append_segments(q_start, ctx_len, bt_start)
    h_kv = k.shape[1]
    if kv_dtype == "fp8":
        _append_fp8(k, ks, np.asarray(k_new, np.uint16), segs, bt_start, block_ids, h_kv)
        _append_fp8(v, vs, np.asarray(v_new, np.uint16), segs, bt_start, block_ids, h_kv)
        return k, v, ks, vs
    for r, blk, row0, n, slot0 in segs:
        b = int(block_ids[int(bt_start[r]) + blk])
        k[b, :, slot0:slot0 + n, :] = np.asarray(k_new[row0:row0 + n]).transpose(1, 0, 2)
        v[b, :, slot0:slot0 + n, :] = np.asarray(v_new[row0:row0 + n]).transpose(1, 0, 2)
    return k, v, ks, vs
