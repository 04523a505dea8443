"""Device-side plumbing around the C ABI: torch tensors for the pool, the
plan image and the workspace, and one call per step of the hot path.

Everything here is argument marshalling and memory management (torch owns
the device memory and the stream); the arithmetic runs in libaug.so.
"""

from __future__ import annotations

import time

import numpy as np
import torch

from . import (aug_attn_mixed, aug_attn_plan, aug_kv_append, aug_kv_park, aug_kv_record_bytes, aug_kv_resume,
               aug_plan_upload, make_shape)

_TORCH_STORAGE = {"f32": torch.float32, "bf16": torch.bfloat16, "fp8": torch.uint8}


def to_device_array(x: np.ndarray, dtype: str, device) -> torch.Tensor:
    """Host bit patterns (float32 / uint16 bf16 / uint8 fp8) -> device tensor."""
    if dtype == "bf16":
        return torch.from_numpy(np.ascontiguousarray(x).view(np.int16)).view(torch.bfloat16).to(device)
    if dtype == "fp8":
        return torch.from_numpy(np.ascontiguousarray(x, dtype=np.uint8)).to(device)
    return torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).to(device)


def to_host_f64(t: torch.Tensor) -> np.ndarray:
    return t.detach().float().cpu().numpy().astype(np.float64)


class PagedKV:
    """A KV pool on the device plus its park/resume staging."""

    def __init__(self, shape, k_cache, v_cache, k_scale=None, v_scale=None, staging_bytes=1 << 28):
        self.shape = shape
        self.k_cache, self.v_cache = k_cache, v_cache
        self.k_scale, self.v_scale = k_scale, v_scale
        self.num_pool_blocks = int(k_cache.shape[0])
        self.record_bytes = aug_kv_record_bytes(shape)
        staging_bytes = max(self.record_bytes, (staging_bytes // self.record_bytes) * self.record_bytes)
        self.staging = torch.empty(staging_bytes, dtype=torch.uint8, device=k_cache.device)

    def host_buffer(self, n_blocks: int) -> torch.Tensor:
        return torch.empty(max(1, n_blocks * self.record_bytes), dtype=torch.uint8, pin_memory=True)

    def park(self, blocks_host: np.ndarray, blocks_dev: torch.Tensor, host_dst: torch.Tensor, stream=None):
        aug_kv_park(self.shape, self.k_cache, self.v_cache, self.k_scale, self.v_scale, blocks_dev,
                    len(blocks_host), self.num_pool_blocks, host_dst, self.staging,
                    block_ids_host=blocks_host, stream=stream)

    def resume(self, blocks_host: np.ndarray, blocks_dev: torch.Tensor, host_src: torch.Tensor, stream=None):
        aug_kv_resume(self.shape, self.k_cache, self.v_cache, self.k_scale, self.v_scale, blocks_dev,
                      len(blocks_host), self.num_pool_blocks, host_src, self.staging,
                      block_ids_host=blocks_host, stream=stream)


class MixedAttention:
    """One planned mixed batch: its plan image and workspace on the device,
    its output tensor, and the launch."""

    def __init__(self, shape, kv: PagedKV, q_start, ctx_len, bt_start, block_ids_host,
                 block_ids_dev: torch.Tensor, kv_split_tokens: int = 0, check_blocks: bool = True,
                 row_path: int = 0, tile_path: int = 0):
        self.shape, self.kv = shape, kv
        device = kv.k_cache.device
        self.info, plan = aug_attn_plan(shape, q_start, ctx_len, bt_start, kv.num_pool_blocks,
                                        block_ids_host if check_blocks else None,
                                        kv_split_tokens=kv_split_tokens, row_path=row_path,
                                        tile_path=tile_path)
        # pinned staging kept alive with the batch; the library's copy kernel
        # moves it on the current stream of the cache's device
        self.plan_host = torch.from_numpy(plan.copy()).pin_memory()
        self.plan_dev = torch.empty(max(1, plan.size), dtype=torch.uint8, device=device)
        aug_plan_upload(self.plan_host, self.plan_dev, plan.size)
        self.workspace = torch.empty(max(256, int(self.info.workspace_bytes)), dtype=torch.uint8,
                                     device=device)
        self.block_ids = block_ids_dev
        rows = int(self.info.total_rows)
        out_dtype = torch.float32 if shape.out_dtype == 0 else torch.bfloat16
        self.out = torch.empty((rows, shape.num_q_heads, shape.head_dim), dtype=out_dtype, device=device)

    def run(self, q: torch.Tensor, stream=None, kv: "PagedKV" = None, block_ids: torch.Tensor = None,
            out: torch.Tensor = None):
        """Enqueue the batch's attention. ``kv``, ``block_ids`` and ``out``
        default to the planned ones; another layer of the same batch passes its
        own pool, block ids (same table shape) and output, and reuses the plan."""
        kv = self.kv if kv is None else kv
        out = self.out if out is None else out
        aug_attn_mixed(self.shape, self.info, self.plan_dev, q, kv.k_cache, kv.v_cache,
                       kv.k_scale, kv.v_scale, self.block_ids if block_ids is None else block_ids,
                       kv.num_pool_blocks, out, self.workspace, stream=stream)
        return out

    def append(self, k_new: torch.Tensor, v_new: torch.Tensor, stream=None, kv: "PagedKV" = None,
               block_ids: torch.Tensor = None):
        """Write the batch's new K/V rows ([rows][H_kv][D]) into the pool
        (``kv`` and ``block_ids`` as for ``run``)."""
        kv = self.kv if kv is None else kv
        want = (int(self.info.total_rows), self.shape.num_kv_heads, self.shape.head_dim)
        dtype = torch.float32 if self.shape.kv_dtype == 0 else torch.bfloat16
        for t in (k_new, v_new):
            if tuple(t.shape) != want or t.dtype != dtype or not t.is_contiguous():
                raise ValueError(f"new K/V rows must be contiguous {dtype} of shape {want}, got "
                                 f"{t.dtype} {tuple(t.shape)}")
        aug_kv_append(self.shape, self.info, self.plan_dev, k_new, v_new, kv.k_cache,
                      kv.v_cache, kv.k_scale, kv.v_scale, self.block_ids if block_ids is None else block_ids,
                      kv.num_pool_blocks, stream=stream)


def shape_of(batch) -> object:
    return make_shape(batch.num_q_heads, batch.num_kv_heads, batch.head_dim, batch.q_dtype,
                      batch.kv_dtype, batch.out_dtype, batch.softmax_scale)


def upload_batch(batch, device="cuda", staging_bytes=1 << 28):
    """Move a host batch (fields as produced by the seeded generators) to the
    device: returns (shape, PagedKV, q tensor, block_ids tensor)."""
    shape = shape_of(batch)
    k = to_device_array(batch.k_cache, batch.kv_dtype, device)
    v = to_device_array(batch.v_cache, batch.kv_dtype, device)
    ks = vs = None
    if batch.kv_dtype == "fp8":
        ks = torch.from_numpy(batch.k_scale).to(device)
        vs = torch.from_numpy(batch.v_scale).to(device)
    kv = PagedKV(shape, k, v, ks, vs, staging_bytes=staging_bytes)
    q = to_device_array(batch.q, batch.q_dtype, device)
    bids = torch.from_numpy(np.ascontiguousarray(batch.block_ids, dtype=np.int32)).to(device)
    return shape, kv, q, bids


def serving_former(**params):
    """A batch former for the serving loop (``synth.trace.ServingLoop``):
    ``former(records, free_blocks, now)`` packs the records (dicts with the
    request-record field names) into the library's request layout, calls
    ``aug_form_batch`` and returns its plan dict. ``params`` are the fields of
    the former's parameter record."""
    from . import REQUEST_DTYPE, aug_form_batch, former_params
    p = former_params(**params)
    names = REQUEST_DTYPE.names

    def run(recs, free_blocks, now):
        arr = np.zeros(len(recs), REQUEST_DTYPE)
        for k in names:
            if k != "reserved":
                arr[k] = [r[k] for r in recs]
        t0 = time.perf_counter()
        plan = aug_form_batch(arr, free_blocks, now, p)
        run.timings.append((time.perf_counter() - t0, len(recs), int(np.count_nonzero(arr["state"] == 3))))
        return plan
    # (seconds in the library call, records, paused records) per iteration
    run.timings = []
    return run


class _LibraryLifecycle:
    """Request records of a serving loop, created and renewed by the library
    (Algorithm 1, steps (1)-(2)). Records are dicts with the field names of
    the library's request record."""

    def __init__(self):
        from . import REQUEST_DTYPE
        self.dtype = REQUEST_DTYPE
        self.names = [k for k in REQUEST_DTYPE.names if k != "reserved"]

    def _dict(self, rec):
        return {k: rec[k].item() for k in self.names}

    def arrive(self, id, arrival, prompt_tokens, pred_out, pred_call, has_next_call):
        from . import aug_request_arrive
        return self._dict(aug_request_arrive(id, arrival, prompt_tokens, pred_out, pred_call, has_next_call))

    def on_return(self, rec, realised, context_tokens, ret_tokens, pred_out, pred_call, has_next_call):
        from . import aug_request_return
        arr = np.zeros(1, self.dtype)
        for k in self.names:
            arr[0][k] = rec[k]
        return self._dict(aug_request_return(arr[0], realised, context_tokens, ret_tokens, pred_out,
                                             pred_call, has_next_call))


def serving_lifecycle():
    """The library's request-record transitions for ``synth.trace.ServingLoop``."""
    return _LibraryLifecycle()
