"""Seeded synthetic attention batches over a paged KV cache.

Layout of every batch (one attention layer):

* ``q``        [sum_q, H_q, D]            query rows of all requests, request after request
* ``k_cache``  [n_blocks, H_kv, 16, D]    pool of 16-token blocks, head-major inside a block
* ``v_cache``  same as ``k_cache``
* ``k_scale``, ``v_scale`` [n_blocks, H_kv] float32, only for fp8 caches
* ``q_start``  [R+1] int32  row offsets of each request into ``q``
* ``ctx_len``  [R]   int32  keys of each request, counting this step's query tokens
* ``bt_start`` [R+1] int32  CSR offsets of each request into ``block_ids``
* ``block_ids``[nnz] int32  pool block of each 16-token slice of each request

Query token j of request r sits at position ``ctx_len[r] - q_len + j`` of its
context. Every pool slot that no request reads (the tail of a last block,
blocks owned by nobody, blocks that a resume has yet to fill) holds NaN, so a
consumer that reads outside the context shows it at once.

The five workloads follow the configurations the attention step is measured
on: a tiny fp32 mixed batch, an 8B-shaped (32 query heads, 8 KV heads,
head_dim 128) decode batch, the same shape as a mixed batch under a 2048-token
budget with parked and resumed requests, a long-context decode batch, and the
64/8-head fp8 shape used by the budget sweep.
"""

from __future__ import annotations

import concurrent.futures as cf
import dataclasses
import os
from typing import List, Optional, Sequence

import numpy as np

BLOCK = 16
BF16_NAN = np.uint16(0x7FC0)
FP8_NAN = np.uint8(0x7F)
F32_NAN = np.float32(np.nan)


@dataclasses.dataclass
class ParkCase:
    """Blocks that a step parks to host memory and resumes from it.

    ``park_blocks`` hold live data and are copied out this step. For a resume,
    the data a request expects at ``resume_blocks`` starts out at
    ``resume_src_blocks`` (where the request lived before it was paused); the
    caller parks those first, poisons them, then resumes into ``resume_blocks``.
    """

    park_blocks: np.ndarray
    resume_src_blocks: np.ndarray
    resume_blocks: np.ndarray
    park_req_ctx: List[int] = dataclasses.field(default_factory=list)
    resume_req_ctx: List[int] = dataclasses.field(default_factory=list)


@dataclasses.dataclass
class AttnBatch:
    name: str
    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    q_dtype: str          # "f32" | "bf16"
    kv_dtype: str         # "f32" | "bf16" | "fp8"
    out_dtype: str        # "f32" | "bf16"
    softmax_scale: float
    q: np.ndarray
    k_cache: np.ndarray
    v_cache: np.ndarray
    k_scale: Optional[np.ndarray]
    v_scale: Optional[np.ndarray]
    q_start: np.ndarray
    ctx_len: np.ndarray
    bt_start: np.ndarray
    block_ids: np.ndarray
    park: Optional[ParkCase] = None
    seed: int = 0

    @property
    def num_reqs(self) -> int:
        return int(self.ctx_len.shape[0])

    @property
    def num_pool_blocks(self) -> int:
        return int(self.k_cache.shape[0])

    @property
    def q_len(self) -> np.ndarray:
        return np.diff(self.q_start).astype(np.int32)

    @property
    def total_q(self) -> int:
        return int(self.q_start[-1])

    def blocks_of(self, r: int) -> np.ndarray:
        return self.block_ids[self.bt_start[r]:self.bt_start[r + 1]]


# ---------------------------------------------------------------------------
# bit-pattern encoders (input preparation only)
# ---------------------------------------------------------------------------

def round_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """float32 -> bf16 bit patterns, round to nearest even (finite inputs)."""
    u = np.array(x, dtype=np.float32, copy=True).view(np.uint32)
    u += ((u >> np.uint32(16)) & np.uint32(1)) + np.uint32(0x7FFF)
    return np.ascontiguousarray(u.view(np.uint16)[..., 1::2])


def encode_e4m3fn_bits(y: np.ndarray) -> np.ndarray:
    """float32 -> OCP FP8 E4M3FN bit patterns, round to nearest even, saturating.

    E4M3FN: 1 sign bit, 4 exponent bits with bias 7, 3 mantissa bits, no
    infinities, S.1111.111 is NaN, largest finite magnitude 448, subnormals are
    multiples of 2^-9.
    """
    y = np.asarray(y, dtype=np.float64)
    sign = (y < 0) | ((y == 0) & np.signbit(y))
    a = np.minimum(np.abs(y), 448.0)
    code = np.zeros(a.shape, dtype=np.int64)
    sub = a < 2.0 ** -6
    code[sub] = np.rint(a[sub] * 2.0 ** 9).astype(np.int64)
    f, ex = np.frexp(a[~sub])            # a = f * 2^ex, f in [0.5, 1)
    e = ex.astype(np.int64) - 1
    m = np.rint((2.0 * f - 1.0) * 8.0).astype(np.int64)
    carry = m == 8
    e[carry] += 1
    m[carry] = 0
    code[~sub] = ((e + 7) << 3) | m
    code = np.minimum(code, 0x7E)
    return (code | (sign.astype(np.int64) << 7)).astype(np.uint8)


# ---------------------------------------------------------------------------
# pool filling
# ---------------------------------------------------------------------------

def _empty_pool(n_blocks, h_kv, d, kv_dtype):
    shape = (n_blocks, h_kv, BLOCK, d)
    if kv_dtype == "f32":
        return np.full(shape, F32_NAN, dtype=np.float32)
    if kv_dtype == "bf16":
        return np.full(shape, BF16_NAN, dtype=np.uint16)
    if kv_dtype == "fp8":
        return np.full(shape, FP8_NAN, dtype=np.uint8)
    raise ValueError(kv_dtype)


def _to_storage(x: np.ndarray, dtype: str) -> np.ndarray:
    if dtype == "f32":
        return x.astype(np.float32)
    if dtype == "bf16":
        return round_to_bf16_bits(x)
    raise ValueError(dtype)


def _write_tokens(pool, scale, vals, blocks, ctx, kv_dtype):
    """Write ``vals`` [ctx, H_kv, D] (float32) into ``pool`` at ``blocks``; the
    slots past ``ctx`` in the last block keep their NaN poison."""
    nblk = -(-ctx // BLOCK)
    h_kv, d = vals.shape[1], vals.shape[2]
    blocks = np.asarray(blocks[:nblk], dtype=np.int64)
    full = ctx // BLOCK
    if kv_dtype == "fp8":
        pad = np.zeros((nblk * BLOCK, h_kv, d), dtype=np.float32)
        pad[:ctx] = vals
        per_block = pad.reshape(nblk, BLOCK, h_kv, d)
        amax = np.abs(per_block).max(axis=(1, 3))               # [nblk, H_kv]
        s = np.where(amax > 0, amax / 448.0, 1.0).astype(np.float32)
        scale[blocks] = s
        codes = encode_e4m3fn_bits(per_block / s[:, None, :, None]).transpose(0, 2, 1, 3)
        if full:
            pool[blocks[:full]] = codes[:full]
        tail = ctx - full * BLOCK
        if tail:
            pool[blocks[full], :, :tail, :] = codes[full, :, :tail, :]
        return
    stored = _to_storage(vals, kv_dtype)
    if full:
        pool[blocks[:full]] = stored[:full * BLOCK].reshape(full, BLOCK, h_kv, d).transpose(0, 2, 1, 3)
    tail = ctx - full * BLOCK
    if tail:
        pool[blocks[full], :, :tail, :] = stored[full * BLOCK:].transpose(1, 0, 2)


def make_batch_from_lengths(
    name: str,
    q_lens: Sequence[int],
    ctx_lens: Sequence[int],
    *,
    num_q_heads: int,
    num_kv_heads: int,
    head_dim: int,
    q_dtype: str,
    kv_dtype: str,
    out_dtype: str,
    n_pool_blocks: int,
    seed: int,
    q_std: float = 1.0,
    kv_std: float = 1.0,
    extra_reqs_ctx: Sequence[int] = (),
    resume_mask: Optional[Sequence[bool]] = None,
) -> AttnBatch:
    """Lay out a batch with the given per-request (q_len, ctx_len).

    Blocks come from one random permutation of the pool, dealt to requests in
    order. ``extra_reqs_ctx`` adds paused requests that are not in the batch
    but own live blocks (they are the ones a step parks). ``resume_mask``
    marks batch requests whose KV must be resumed before the step: their data
    starts in other blocks (``resume_src_blocks``).
    """
    rng = np.random.default_rng(seed)
    q_lens = np.asarray(q_lens, dtype=np.int64)
    ctx_lens = np.asarray(ctx_lens, dtype=np.int64)
    assert np.all(q_lens >= 1) and np.all(ctx_lens >= q_lens)
    n_req = len(q_lens)
    resume_mask = np.zeros(n_req, bool) if resume_mask is None else np.asarray(resume_mask, bool)
    nblk = -(-ctx_lens // BLOCK)
    extra = np.asarray(extra_reqs_ctx, dtype=np.int64)
    extra_nblk = -(-extra // BLOCK)
    need = int(nblk.sum() + nblk[resume_mask].sum() + extra_nblk.sum())
    if need > n_pool_blocks:
        raise ValueError(f"pool of {n_pool_blocks} blocks cannot hold {need}")
    perm = rng.permutation(n_pool_blocks).astype(np.int32)

    cursor = 0
    tables = []
    for r in range(n_req):
        tables.append(perm[cursor:cursor + nblk[r]])
        cursor += int(nblk[r])
    src_tables = {}
    for r in np.nonzero(resume_mask)[0]:
        src_tables[int(r)] = perm[cursor:cursor + nblk[r]]
        cursor += int(nblk[r])
    extra_tables = []
    for e in range(len(extra)):
        extra_tables.append(perm[cursor:cursor + extra_nblk[e]])
        cursor += int(extra_nblk[e])

    # queries
    total_q = int(q_lens.sum())
    qf = rng.standard_normal((total_q, num_q_heads, head_dim), dtype=np.float32) * np.float32(q_std)
    q = _to_storage(qf, q_dtype)
    del qf

    k_cache = _empty_pool(n_pool_blocks, num_kv_heads, head_dim, kv_dtype)
    v_cache = _empty_pool(n_pool_blocks, num_kv_heads, head_dim, kv_dtype)
    if kv_dtype == "fp8":
        k_scale = np.full((n_pool_blocks, num_kv_heads), np.nan, dtype=np.float32)
        v_scale = np.full((n_pool_blocks, num_kv_heads), np.nan, dtype=np.float32)
    else:
        k_scale = v_scale = None

    # every request (and every paused extra request) draws from its own stream,
    # so the bytes do not depend on how the work is spread over threads
    kv_std32 = np.float32(kv_std)
    jobs = [(r, int(ctx_lens[r]), src_tables.get(r, tables[r])) for r in range(n_req)]
    jobs += [(n_req + e, int(extra[e]), extra_tables[e]) for e in range(len(extra))]

    def fill(job):
        key, ctx, where = job
        g = np.random.default_rng([seed, 7, key])
        for cache, scale in ((k_cache, k_scale), (v_cache, v_scale)):
            x = g.standard_normal((ctx, num_kv_heads, head_dim), dtype=np.float32)
            x *= kv_std32
            _write_tokens(cache, scale, x, where, ctx, kv_dtype)

    workers = min(16, os.cpu_count() or 1)
    if workers > 1 and len(jobs) > 1:
        with cf.ThreadPoolExecutor(workers) as ex:
            list(ex.map(fill, jobs))
    else:
        for j in jobs:
            fill(j)

    q_start = np.zeros(n_req + 1, dtype=np.int32)
    q_start[1:] = np.cumsum(q_lens)
    bt_start = np.zeros(n_req + 1, dtype=np.int32)
    bt_start[1:] = np.cumsum(nblk)
    block_ids = (np.concatenate(tables) if n_req else np.zeros(0, np.int64)).astype(np.int32)

    park = None
    if len(extra) or resume_mask.any():
        rs = sorted(src_tables)
        park = ParkCase(
            park_blocks=(np.concatenate(extra_tables) if len(extra) else np.zeros(0)).astype(np.int32),
            resume_src_blocks=(np.concatenate([src_tables[r] for r in rs]) if rs else np.zeros(0)).astype(np.int32),
            resume_blocks=(np.concatenate([tables[r] for r in rs]) if rs else np.zeros(0)).astype(np.int32),
            park_req_ctx=[int(c) for c in extra],
            resume_req_ctx=[int(ctx_lens[r]) for r in rs],
        )

    return AttnBatch(
        name=name,
        num_q_heads=num_q_heads,
        num_kv_heads=num_kv_heads,
        head_dim=head_dim,
        q_dtype=q_dtype,
        kv_dtype=kv_dtype,
        out_dtype=out_dtype,
        softmax_scale=float(1.0 / np.sqrt(head_dim)),
        q=q,
        k_cache=k_cache,
        v_cache=v_cache,
        k_scale=k_scale,
        v_scale=v_scale,
        q_start=q_start,
        ctx_len=ctx_lens.astype(np.int32),
        bt_start=bt_start,
        block_ids=block_ids,
        park=park,
        seed=seed,
    )


# ---------------------------------------------------------------------------
# the five workloads
# ---------------------------------------------------------------------------

def make_new_kv(batch: AttnBatch, seed: int, std: float = 1.0):
    """The step's new K and V rows, each [total_q, H_kv, D] drawn N(0, std^2):
    float32 for f32 caches, bf16 bit patterns for bf16 and fp8 caches (an fp8
    cache receives bf16 rows and encodes them itself)."""
    rng = np.random.default_rng(seed)
    shape = (batch.total_q, batch.num_kv_heads, batch.head_dim)
    dt = "f32" if batch.kv_dtype == "f32" else "bf16"
    k = _to_storage(rng.standard_normal(shape, dtype=np.float32) * np.float32(std), dt)
    v = _to_storage(rng.standard_normal(shape, dtype=np.float32) * np.float32(std), dt)
    return k, v


def poison_new_slots(batch: AttnBatch, copy: bool = True) -> AttnBatch:
    """``batch`` (a copy unless ``copy`` is False) whose slots at this step's
    query positions (the ones an append fills) hold the NaN poison, as before
    the step's K/V exist. Scales are left as they are."""
    out = dataclasses.replace(batch, k_cache=batch.k_cache.copy(), v_cache=batch.v_cache.copy()) \
        if copy else batch
    nan = {"f32": F32_NAN, "bf16": BF16_NAN, "fp8": FP8_NAN}[batch.kv_dtype]
    q_len = batch.q_len
    for r in range(batch.num_reqs):
        blocks = batch.blocks_of(r)
        for p in range(int(batch.ctx_len[r]) - int(q_len[r]), int(batch.ctx_len[r])):
            out.k_cache[blocks[p // BLOCK], :, p % BLOCK, :] = nan
            out.v_cache[blocks[p // BLOCK], :, p % BLOCK, :] = nan
    return out


def _lognormal_ctx(rng, n, median, sigma, lo, hi):
    x = np.rint(rng.lognormal(np.log(median), sigma, size=n))
    return np.clip(x, lo, hi).astype(np.int64)


def make_tiny_mixed(seed: int = 0, sharp: bool = True) -> AttnBatch:
    """8 requests, 4/4 heads, head_dim 64, fp32: 2 prefill chunks of 32 rows
    with prior context U{0..64}, 6 decodes with context U{16..256}, order
    shuffled; a 128-block pool; 1 paused request of U{49..64} tokens (4
    blocks) to park and resume."""
    rng = np.random.default_rng(seed)
    kinds = np.array([1, 1, 0, 0, 0, 0, 0, 0])
    rng.shuffle(kinds)
    q_lens, ctx_lens = [], []
    for kd in kinds:
        if kd:
            q_lens.append(32)
            ctx_lens.append(32 + int(rng.integers(0, 65)))
        else:
            q_lens.append(1)
            ctx_lens.append(int(rng.integers(16, 257)))
    paused_ctx = int(rng.integers(49, 65))
    b = make_batch_from_lengths(
        "tiny-mixed-fp32", q_lens, ctx_lens, num_q_heads=4, num_kv_heads=4, head_dim=64,
        q_dtype="f32", kv_dtype="f32", out_dtype="f32", n_pool_blocks=128,
        seed=seed + 1000, extra_reqs_ctx=[paused_ctx])
    # the paused request's blocks are parked, then resumed into 4 free blocks
    used = set(b.block_ids.tolist()) | set(b.park.park_blocks.tolist())
    free = np.array(sorted(set(range(128)) - used), dtype=np.int32)
    dst = np.random.default_rng(seed + 2000).choice(free, size=len(b.park.park_blocks), replace=False)
    b.park.resume_src_blocks = b.park.park_blocks.copy()
    b.park.resume_blocks = dst.astype(np.int32)
    b.park.resume_req_ctx = [paused_ctx]
    return b


def make_decode_8b(seed: int = 0, sharp: bool = False, n_req: int = 256,
                   n_pool_blocks: int = 80_000) -> AttnBatch:
    """Llama-3-8B-shaped layer, decode only: 32/8 heads, head_dim 128, bf16;
    256 decodes with context lognormal(median 1200, sigma 0.8) capped at 8192;
    K/V N(0,1)/sqrt(128) (N(0,1) when ``sharp``); an 80k-block pool."""
    rng = np.random.default_rng(seed)
    ctx = _lognormal_ctx(rng, n_req, 1200, 0.8, 1, 8192)
    return make_batch_from_lengths(
        "decode-8b-bf16", [1] * n_req, ctx, num_q_heads=32, num_kv_heads=8, head_dim=128,
        q_dtype="bf16", kv_dtype="bf16", out_dtype="bf16", n_pool_blocks=n_pool_blocks,
        seed=seed + 1000, kv_std=1.0 if sharp else 1.0 / np.sqrt(128.0))


def mixed_8b_lengths(seed: int = 0, n_dec: int = 512, n_pre: int = 3, chunk: int = 512):
    """Per-request lengths of the 2048-token mixed batch: prefill chunks of 512
    rows with prior context U{0..4096}, decodes with context lognormal(median
    1500, sigma 0.8) capped at 8192, 30% of decodes carrying U{50..500}
    appended tool-output tokens and resumed from host memory."""
    rng = np.random.default_rng(seed)
    pre_ctx = chunk + rng.integers(0, 4097, size=n_pre)
    dec_ctx = _lognormal_ctx(rng, n_dec, 1500, 0.8, 1, 8192)
    resumed = rng.random(n_dec) < 0.3
    dec_ctx = dec_ctx + np.where(resumed, rng.integers(50, 501, size=n_dec), 0)
    q_lens = [chunk] * n_pre + [1] * n_dec
    ctx_lens = list(pre_ctx) + list(dec_ctx)
    mask = [False] * n_pre + list(resumed)
    return q_lens, ctx_lens, mask


def make_mixed_8b(seed: int = 0, sharp: bool = False, n_dec: int = 512, n_pre: int = 3,
                  n_pool_blocks: int = 131_072) -> AttnBatch:
    q_lens, ctx_lens, mask = mixed_8b_lengths(seed, n_dec, n_pre)
    return make_batch_from_lengths(
        "mixed-8b-bf16-budget2048", q_lens, ctx_lens, num_q_heads=32, num_kv_heads=8,
        head_dim=128, q_dtype="bf16", kv_dtype="bf16", out_dtype="bf16",
        n_pool_blocks=n_pool_blocks, seed=seed + 1000,
        kv_std=1.0 if sharp else 1.0 / np.sqrt(128.0), resume_mask=mask)


def make_long_context(seed: int = 0, sharp: bool = False, n_req: int = 64, n_move: int = 8,
                      lo: int = 16384, hi: int = 32768, n_pool_blocks: int = 163_840) -> AttnBatch:
    """64 decodes with context U{16k..32k} (split-K path); each step resumes 8
    of them from host memory and parks 8 paused requests of the same length
    distribution (up to 2048 blocks each)."""
    rng = np.random.default_rng(seed)
    ctx = rng.integers(lo, hi + 1, size=n_req)
    parked_ctx = rng.integers(lo, hi + 1, size=n_move)
    mask = np.zeros(n_req, bool)
    mask[rng.choice(n_req, size=n_move, replace=False)] = True
    return make_batch_from_lengths(
        "long-context-8b-bf16", [1] * n_req, ctx, num_q_heads=32, num_kv_heads=8, head_dim=128,
        q_dtype="bf16", kv_dtype="bf16", out_dtype="bf16", n_pool_blocks=n_pool_blocks,
        seed=seed + 1000, kv_std=1.0 if sharp else 1.0 / np.sqrt(128.0),
        extra_reqs_ctx=parked_ctx, resume_mask=mask)


def make_decode_gqa8_fp8(seed: int = 0, sharp: bool = False, n_req: int = 512) -> AttnBatch:
    """A decode-only batch on the budget sweep's layer (64 query heads, 8 KV
    heads, head_dim 128, bf16 Q, fp8 E4M3FN KV with per-block scales):
    ``n_req`` decodes with contexts lognormal (median 2500, sigma 0.8, capped
    at 16384), the decode-dominated end of the batches a large budget forms."""
    rng = np.random.default_rng(seed)
    ctx = np.clip(np.rint(rng.lognormal(np.log(2500.0), 0.8, n_req)), 1, 16384).astype(np.int64)
    pool = int(((ctx + BLOCK - 1) // BLOCK).sum()) * 5 // 4 + 64
    return make_batch_from_lengths(
        "decode-fp8-64x8", [1] * n_req, ctx.tolist(), num_q_heads=64, num_kv_heads=8, head_dim=128,
        q_dtype="bf16", kv_dtype="fp8", out_dtype="bf16", n_pool_blocks=pool, seed=seed + 2000,
        kv_std=1.0 if sharp else 1.0 / np.sqrt(128.0))


def make_prefill_8b(seed: int = 0, sharp: bool = False, n_chunks: int = 8, chunk: int = 512) -> AttnBatch:
    """A prefill-only batch on the 8B layer (32/8 heads, head_dim 128, bf16):
    ``n_chunks`` chunks of ``chunk`` rows, each behind a prior context drawn
    U{0..4096}, the prefill part of the mixed batch at a 4096-token budget."""
    rng = np.random.default_rng(seed)
    ctx = chunk + rng.integers(0, 4097, size=n_chunks)
    # room beside the batch for the memory-derived budget to reach 4096 tokens
    pool = int(((ctx + BLOCK - 1) // BLOCK).sum()) * 5 // 4 + 1024
    return make_batch_from_lengths(
        "prefill-8b-bf16", [chunk] * n_chunks, ctx.tolist(), num_q_heads=32, num_kv_heads=8, head_dim=128,
        q_dtype="bf16", kv_dtype="bf16", out_dtype="bf16", n_pool_blocks=pool, seed=seed + 3000,
        kv_std=1.0 if sharp else 1.0 / np.sqrt(128.0))


def make_prefill_gqa8_fp8(seed: int = 0, sharp: bool = False, n_chunks: int = 16, chunk: int = 512) -> AttnBatch:
    """The prefill-dominated end of the batches an 8192-token budget forms on
    the budget sweep's layer (64/8 heads, head_dim 128, bf16 Q, fp8 E4M3FN KV
    with per-block scales): ``n_chunks`` chunks of ``chunk`` rows, each behind
    a prior context drawn U{0..2048} (prompts of the trace have a median of
    800 tokens, so most chunks sit one to four chunks into their prompt)."""
    rng = np.random.default_rng(seed)
    ctx = chunk + rng.integers(0, 2049, size=n_chunks)
    # room beside the batch for the memory-derived budget to reach 8192 tokens
    pool = int(((ctx + BLOCK - 1) // BLOCK).sum()) * 5 // 4 + 1024
    return make_batch_from_lengths(
        "prefill-fp8-64x8", [chunk] * n_chunks, ctx.tolist(), num_q_heads=64, num_kv_heads=8, head_dim=128,
        q_dtype="bf16", kv_dtype="fp8", out_dtype="bf16", n_pool_blocks=pool, seed=seed + 4000,
        kv_std=1.0 if sharp else 1.0 / np.sqrt(128.0))


def make_config(cfg: int, seed: int = 0, sharp: bool = False, **kw) -> AttnBatch:
    if cfg == 1:
        return make_tiny_mixed(seed, **kw)
    if cfg == 2:
        return make_decode_8b(seed, sharp=sharp, **kw)
    if cfg == 3:
        return make_mixed_8b(seed, sharp=sharp, **kw)
    if cfg == 4:
        return make_long_context(seed, sharp=sharp, **kw)
    raise ValueError(f"no attention batch generator for workload {cfg}")
