"""Oracle for mixed-batch paged attention (numpy, float64).

The paper runs every request's prefill, incremental prefill of returned tool
tokens (P^ret), recomputation after Discard and decoding through one engine
iteration (request lifecycle, Eq. 1 and the segment definition in the problem
formulation; Algorithm 1, step (5) "forward(scheduled)"). It does not write
the attention itself down, so this module is the textbook definition of
scaled dot-product attention with a causal mask, applied to each request of
the batch:

    for request r with q_r query rows and ctx_r keys (this step's rows included),
    row j sits at position pos_j = ctx_r - q_r + j and attends keys 0..pos_j;
    query head h reads KV head g = h // (H_q / H_kv)  (grouped-query attention);
    s_t = scale * <q_{j,h}, k_{t,g}>,  p = softmax(s),  o_{j,h} = sum_t p_t v_{t,g}.

The paged cache is first materialised into contiguous per-request K/V by
walking the request's block table, then truncated to ctx_r tokens, so slots
past the context never take part. Inputs are decoded exactly to float64 (fp8
codes times their per-(block, KV head) float32 scale) and all arithmetic is
float64.
"""

from __future__ import annotations

from typing import Iterable, Optional

import numpy as np

from .codecs import e4m3fn_bits_to_f64, e4m3fn_encode, storage_to_f64

BLOCK = 16


def materialise_kv(cache: np.ndarray, scale: Optional[np.ndarray], kv_dtype: str,
                   blocks: np.ndarray, ctx: int) -> np.ndarray:
    """Contiguous [ctx, H_kv, D] float64 K or V of one request."""
    nblk = -(-ctx // BLOCK)
    blocks = np.asarray(blocks[:nblk], dtype=np.int64)
    raw = storage_to_f64(cache[blocks], kv_dtype)            # [nblk, H_kv, 16, D]
    if kv_dtype == "fp8":
        raw = raw * scale[blocks].astype(np.float64)[:, :, None, None]
    h_kv, d = raw.shape[1], raw.shape[3]
    return raw.transpose(0, 2, 1, 3).reshape(nblk * BLOCK, h_kv, d)[:ctx]


def attend_request(q_rows: np.ndarray, k: np.ndarray, v: np.ndarray, num_q_heads: int,
                   num_kv_heads: int, softmax_scale: float) -> np.ndarray:
    """Causal GQA attention of one request: q_rows [q, H_q, D] float64 against
    k, v [ctx, H_kv, D] float64; returns [q, H_q, D] float64."""
    q_len, ctx = q_rows.shape[0], k.shape[0]
    group = num_q_heads // num_kv_heads
    pos = ctx - q_len + np.arange(q_len)
    masked = np.arange(ctx)[None, :] > pos[:, None]          # [q, ctx]
    out = np.empty_like(q_rows)
    for h in range(num_q_heads):
        g = h // group
        s = (q_rows[:, h, :] @ k[:, g, :].T) * softmax_scale
        s[masked] = -np.inf
        s -= s.max(axis=1, keepdims=True)
        p = np.exp(s)
        p /= p.sum(axis=1, keepdims=True)
        out[:, h, :] = p @ v[:, g, :]
    return out


def round_query_rows_e4m3(q_rows: np.ndarray) -> np.ndarray:
    """Query vectors as an fp8 score product sees them. This is not the
    paper's arithmetic but an opt-in arithmetic of the kernel for prefill
    chunks over an fp8 cache, defined here so that it can be checked: each
    (row, head) vector of head_dim values is divided by its scale, the
    largest magnitude over 448, rounded to the nearest E4M3FN value (ties to
    even) and multiplied back by the scale. The scale and its reciprocal are
    float32 values (reciprocal = 448 / largest magnitude, correctly rounded;
    scale = largest magnitude times float32(1/448)), and the division is a
    float32 product with the reciprocal, as the kernel computes them; a
    vector whose largest magnitude is below 2^-100 (all zero, in practice)
    becomes zero. q_rows [n, H, D] float64 (bf16 values)."""
    q32 = np.asarray(q_rows, dtype=np.float32)
    amax = np.abs(q32).max(axis=-1, keepdims=True)
    zero = ~(amax >= np.float32(2.0 ** -100))
    inv = np.where(zero, np.float32(0.0), np.float32(448.0) / np.where(zero, np.float32(1.0), amax))
    scale = np.where(zero, np.float32(1.0), amax * np.float32(1.0 / 448.0)).astype(np.float32)
    x = (q32 * inv.astype(np.float32)).astype(np.float32)
    codes = e4m3fn_encode(x)
    return e4m3fn_bits_to_f64(codes) * scale.astype(np.float64)


def paged_attention(q, q_dtype, k_cache, v_cache, k_scale, v_scale, kv_dtype,
                    q_start, ctx_len, bt_start, block_ids, num_q_heads, num_kv_heads,
                    softmax_scale, requests: Optional[Iterable[int]] = None,
                    fp8_chunk_queries: bool = False) -> np.ndarray:
    """Output rows [sum_q, H_q, D] float64. With ``requests`` given, only those
    requests' rows are computed and every other row is NaN. With
    ``fp8_chunk_queries`` the query rows of every request with more than one
    row (a prefill chunk) pass through ``round_query_rows_e4m3`` first."""
    total_q = int(q_start[-1])
    d = q.shape[-1]
    out = np.full((total_q, num_q_heads, d), np.nan, dtype=np.float64)
    reqs = range(len(ctx_len)) if requests is None else requests
    for r in reqs:
        r = int(r)
        q0, q1 = int(q_start[r]), int(q_start[r + 1])
        ctx = int(ctx_len[r])
        blocks = block_ids[int(bt_start[r]):int(bt_start[r + 1])]
        k = materialise_kv(k_cache, k_scale, kv_dtype, blocks, ctx)
        v = materialise_kv(v_cache, v_scale, kv_dtype, blocks, ctx)
        q_rows = storage_to_f64(q[q0:q1], q_dtype)
        if fp8_chunk_queries and q1 - q0 > 1:
            q_rows = round_query_rows_e4m3(q_rows)
        out[q0:q1] = attend_request(q_rows, k, v, num_q_heads, num_kv_heads, softmax_scale)
    return out


def attention_for(batch, requests=None, k_cache=None, v_cache=None, k_scale=None, v_scale=None,
                  fp8_chunk_queries=False):
    """Run ``paged_attention`` on a batch object carrying the standard fields;
    the cache arguments override the batch's own pool (e.g. after a resume)."""
    return paged_attention(
        batch.q, batch.q_dtype,
        batch.k_cache if k_cache is None else k_cache,
        batch.v_cache if v_cache is None else v_cache,
        batch.k_scale if k_scale is None else k_scale,
        batch.v_scale if v_scale is None else v_scale,
        batch.kv_dtype, batch.q_start, batch.ctx_len, batch.bt_start, batch.block_ids,
        batch.num_q_heads, batch.num_kv_heads, batch.softmax_scale, requests, fp8_chunk_queries)
