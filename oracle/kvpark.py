"""Oracle for parking (swap-out) and resuming (swap-in) KV blocks.

Under the Swap policy a paused request's context is moved to host memory for
the length of its external call and restored when the call returns (context-
handling policies in the background section and Appendix B; Algorithm 1,
step (2), the swapped queue). The oracle fixes the byte image on the host:
the listed blocks one after another, each one record of

    K[block]  (H_kv x 16 x D elements, the pool's own bit patterns)
    V[block]  (same)
    k_scale[block], v_scale[block]  (H_kv float32 each; fp8 caches only)

Park and resume are pure byte moves, so they are checked bit for bit.
"""

import numpy as np


def record_bytes(num_kv_heads: int, head_dim: int, kv_dtype: str) -> int:
    elem = {"f32": 4, "bf16": 2, "fp8": 1}[kv_dtype]
    scales = 2 * num_kv_heads * 4 if kv_dtype == "fp8" else 0
    return 2 * num_kv_heads * 16 * head_dim * elem + scales


def park(k_cache, v_cache, k_scale, v_scale, kv_dtype, blocks) -> np.ndarray:
    """Host image (uint8) of ``blocks`` in the given order."""
    parts = []
    for b in np.asarray(blocks, dtype=np.int64):
        parts.append(np.ascontiguousarray(k_cache[b]).view(np.uint8).ravel())
        parts.append(np.ascontiguousarray(v_cache[b]).view(np.uint8).ravel())
        if kv_dtype == "fp8":
            parts.append(np.ascontiguousarray(k_scale[b], dtype=np.float32).view(np.uint8).ravel())
            parts.append(np.ascontiguousarray(v_scale[b], dtype=np.float32).view(np.uint8).ravel())
    if not parts:
        return np.zeros(0, dtype=np.uint8)
    return np.concatenate(parts)


def resume(k_cache, v_cache, k_scale, v_scale, kv_dtype, blocks, image):
    """Write the records of ``image`` into ``blocks`` of copies of the pool and
    return the copies (k_cache, v_cache, k_scale, v_scale)."""
    k_out, v_out = k_cache.copy(), v_cache.copy()
    ks_out = None if k_scale is None else k_scale.copy()
    vs_out = None if v_scale is None else v_scale.copy()
    blk_bytes = k_cache[0].nbytes
    sc_bytes = 0 if kv_dtype != "fp8" else k_scale[0].nbytes
    rec = 2 * blk_bytes + 2 * sc_bytes
    image = np.asarray(image, dtype=np.uint8)
    assert image.size == rec * len(blocks)
    for i, b in enumerate(np.asarray(blocks, dtype=np.int64)):
        off = i * rec
        k_out[b] = image[off:off + blk_bytes].view(k_cache.dtype).reshape(k_cache.shape[1:])
        off += blk_bytes
        v_out[b] = image[off:off + blk_bytes].view(v_cache.dtype).reshape(v_cache.shape[1:])
        off += blk_bytes
        if kv_dtype == "fp8":
            ks_out[b] = image[off:off + sc_bytes].view(np.float32)
            off += sc_bytes
            vs_out[b] = image[off:off + sc_bytes].view(np.float32)
    return k_out, v_out, ks_out, vs_out
