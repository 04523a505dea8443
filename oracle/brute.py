"""Brute-force attention in scalar Python (float64, ``math.exp``), tiny shapes only.

An independent second statement of the same definition as ``oracle.attention``
(scaled dot-product attention, causal with bottom-right alignment, grouped
query heads), reading the paged cache slot by slot through the block table
instead of materialising it, and using no numpy arithmetic. It pins the numpy
oracle.
"""

import math

from .codecs import bf16_bits_to_f64, e4m3fn_value

BLOCK = 16


def _val(x, dtype):
    if dtype == "f32":
        return float(x)
    if dtype == "bf16":
        return float(bf16_bits_to_f64(x))
    if dtype == "fp8":
        return e4m3fn_value(int(x))
    raise ValueError(dtype)


def brute_attention(q, q_dtype, k_cache, v_cache, k_scale, v_scale, kv_dtype, q_start,
                    ctx_len, bt_start, block_ids, num_q_heads, num_kv_heads, softmax_scale):
    """Nested lists out[row][head][dim] of Python floats."""
    d = len(q[0][0])
    group = num_q_heads // num_kv_heads
    out = []
    for r in range(len(ctx_len)):
        q0, q1 = int(q_start[r]), int(q_start[r + 1])
        ctx = int(ctx_len[r])
        table = [int(b) for b in block_ids[int(bt_start[r]):int(bt_start[r + 1])]]

        def key(t, g, i):
            b = table[t // BLOCK]
            x = _val(k_cache[b][g][t % BLOCK][i], kv_dtype)
            return x * float(k_scale[b][g]) if kv_dtype == "fp8" else x

        def value(t, g, i):
            b = table[t // BLOCK]
            x = _val(v_cache[b][g][t % BLOCK][i], kv_dtype)
            return x * float(v_scale[b][g]) if kv_dtype == "fp8" else x

        for j in range(q1 - q0):
            pos = ctx - (q1 - q0) + j
            row = []
            for h in range(num_q_heads):
                g = h // group
                qv = [_val(q[q0 + j][h][i], q_dtype) for i in range(d)]
                scores = []
                for t in range(pos + 1):
                    acc = 0.0
                    for i in range(d):
                        acc += qv[i] * key(t, g, i)
                    scores.append(acc * softmax_scale)
                mx = max(scores)
                w = [math.exp(s - mx) for s in scores]
                tot = sum(w)
                o = []
                for i in range(d):
                    acc = 0.0
                    for t in range(pos + 1):
                        acc += w[t] * value(t, g, i)
                    o.append(acc / tot)
                row.append(o)
            out.append(row)
    return out
