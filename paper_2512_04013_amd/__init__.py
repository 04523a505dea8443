"""Python binding of libaug.so (the C ABI declared in include/aug.h).

Argument marshalling only: every function below converts its arguments
(numpy arrays, torch tensors, ints) to the plain pointers and sizes of the C
signature of the same name and calls it; all computation happens in the
library's HIP kernels and C++ host code. Device tensors are torch tensors
(PyTorch provides device memory and streams); the stream defaults to
torch's current stream on the tensors' device.

The library must have been built in-tree (``paper_2512_04013_amd.build``);
importing this module does not load it, the first call does, and fails loudly
when it is missing.
"""

from __future__ import annotations

import ctypes as C
import os
import threading
from typing import Optional

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libaug.so")
# Test runs of the host code under the sanitizers load a host-only build of
# the planner and former instead (no device entry points: calling one raises).
_HOST_ONLY_LIB = os.environ.get("AUG_HOST_ONLY_LIB")

AUG_OK, AUG_ERR_INVALID, AUG_ERR_UNSUPPORTED, AUG_ERR_NO_SPACE, AUG_ERR_HIP = 0, -1, -2, -3, -4
AUG_F32, AUG_BF16, AUG_FP8_E4M3FN = 0, 1, 2
AUG_WAITING, AUG_RUNNING, AUG_SWAPPED, AUG_PAUSED = 0, 1, 2, 3
AUG_POL_NONE, AUG_PRESERVE, AUG_DISCARD, AUG_SWAP = 0, 1, 2, 3
AUG_ROWS_AUTO, AUG_ROWS_VALU, AUG_ROWS_MFMA = 0, 1, 2
AUG_TILES_AUTO, AUG_TILES_BF16, AUG_TILES_FP8_QK, AUG_TILES_FP8 = 0, 1, 2, 3

DTYPE_CODES = {"f32": AUG_F32, "bf16": AUG_BF16, "fp8": AUG_FP8_E4M3FN}

EXPORTED = ["aug_request_arrive", "aug_request_return", "aug_attn_plan", "aug_attn_plan_opts",
            "aug_attn_workspace_size",
            "aug_plan_upload", "aug_attn_mixed", "aug_attn_mixed_noalloc",
            "aug_kv_append", "aug_kv_record_bytes", "aug_kv_park", "aug_kv_resume", "aug_form_batch",
            "aug_status_string", "aug_last_error", "aug_abi_version"]


class AugError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(message)
        self.status = status


# ---- C structs ----------------------------------------------------------------

class aug_attn_shape(C.Structure):
    _fields_ = [("num_q_heads", C.c_int32), ("num_kv_heads", C.c_int32), ("head_dim", C.c_int32),
                ("block_size", C.c_int32), ("q_dtype", C.c_int32), ("kv_dtype", C.c_int32),
                ("out_dtype", C.c_int32), ("softmax_scale", C.c_float)]


class aug_batch_desc(C.Structure):
    _fields_ = [("num_reqs", C.c_int32), ("q_start", C.POINTER(C.c_int32)),
                ("ctx_len", C.POINTER(C.c_int32)), ("bt_start", C.POINTER(C.c_int32)),
                ("block_ids", C.POINTER(C.c_int32)), ("num_pool_blocks", C.c_int32)]


class aug_attn_plan_info(C.Structure):
    _fields_ = [("plan_bytes", C.c_int64), ("workspace_bytes", C.c_int64), ("num_items", C.c_int32),
                ("num_prefill_items", C.c_int32), ("num_merge_groups", C.c_int32),
                ("num_partials", C.c_int32), ("kv_split_tokens", C.c_int32),
                ("total_rows", C.c_int32), ("num_reqs", C.c_int32),
                ("num_tile_merge_groups", C.c_int32), ("num_append_items", C.c_int32),
                ("num_q_heads", C.c_int32), ("num_kv_heads", C.c_int32), ("head_dim", C.c_int32),
                ("q_dtype", C.c_int32), ("kv_dtype", C.c_int32), ("out_dtype", C.c_int32),
                ("row_path", C.c_int32), ("tile_path", C.c_int32)]


class aug_plan_options(C.Structure):
    _fields_ = [("kv_split_tokens", C.c_int32), ("row_path", C.c_int32), ("tile_path", C.c_int32),
                ("reserved", C.c_int32)]


class aug_request(C.Structure):
    _fields_ = [("id", C.c_int64), ("arrival", C.c_double), ("last_sched", C.c_double),
                ("pred_call", C.c_double), ("pause_start", C.c_double), ("state", C.c_int32),
                ("seg", C.c_int32), ("prev_policy", C.c_int32), ("cur_policy", C.c_int32),
                ("seg_ctx", C.c_int32), ("seg_prefill", C.c_int32), ("pred_out", C.c_int32),
                ("has_next_call", C.c_int32), ("ctx_len", C.c_int32), ("pending", C.c_int32),
                ("blocks_on_gpu", C.c_int32), ("reserved", C.c_int32)]


class aug_former_params(C.Structure):
    _fields_ = [("beta", C.c_double), ("beta_low", C.c_double), ("beta_high", C.c_double),
                ("t_iter", C.c_double), ("fwd_a", C.c_double), ("fwd_b", C.c_double),
                ("swap_s_per_tok", C.c_double), ("n_fwd_max", C.c_int64), ("t_max", C.c_int32),
                ("chunk_cap", C.c_int32), ("block_size", C.c_int32),
                ("skip_instead_of_break", C.c_int32), ("order", C.c_int32), ("reserved", C.c_int32)]


class aug_batch_plan(C.Structure):
    _fields_ = [("cap", C.c_int32), ("budget", C.c_int32), ("n_sched", C.c_int32),
                ("n_resume", C.c_int32), ("n_park", C.c_int32), ("n_free", C.c_int32),
                ("ids", C.POINTER(C.c_int64)), ("q_len", C.POINTER(C.c_int32)),
                ("theta", C.POINTER(C.c_double)), ("resume_ids", C.POINTER(C.c_int64)),
                ("park_ids", C.POINTER(C.c_int64)), ("free_ids", C.POINTER(C.c_int64)),
                ("policy_out", C.POINTER(C.c_int32)), ("cost_out", C.POINTER(C.c_double))]


REQUEST_DTYPE = np.dtype([("id", "<i8"), ("arrival", "<f8"), ("last_sched", "<f8"),
                          ("pred_call", "<f8"), ("pause_start", "<f8"), ("state", "<i4"),
                          ("seg", "<i4"), ("prev_policy", "<i4"), ("cur_policy", "<i4"),
                          ("seg_ctx", "<i4"), ("seg_prefill", "<i4"), ("pred_out", "<i4"),
                          ("has_next_call", "<i4"), ("ctx_len", "<i4"), ("pending", "<i4"),
                          ("blocks_on_gpu", "<i4"), ("reserved", "<i4")])
assert REQUEST_DTYPE.itemsize == C.sizeof(aug_request)

# ---- loading ---------------------------------------------------------------------

_lib = None


def lib():
    """The loaded library; raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    path = _HOST_ONLY_LIB or LIB_PATH
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is missing: build it with "
                           "`python -m paper_2512_04013_amd.build` (or __graft_entry__.build())")
    L = C.CDLL(path)
    if _HOST_ONLY_LIB:
        L = _HostOnly(L)
    P = C.c_void_p
    L.aug_attn_plan.argtypes = [C.POINTER(aug_attn_shape), C.POINTER(aug_batch_desc), C.c_int32, P,
                                C.c_size_t, C.POINTER(aug_attn_plan_info)]
    L.aug_attn_plan_opts.argtypes = [C.POINTER(aug_attn_shape), C.POINTER(aug_batch_desc),
                                     C.POINTER(aug_plan_options), P, C.c_size_t, C.POINTER(aug_attn_plan_info)]
    L.aug_attn_workspace_size.argtypes = [C.POINTER(aug_attn_shape), C.POINTER(aug_batch_desc), C.c_int32,
                                          C.POINTER(C.c_size_t)]
    L.aug_attn_mixed.argtypes = [C.POINTER(aug_attn_shape), C.POINTER(aug_attn_plan_info), P, P, P, P,
                                 P, P, P, C.c_int32, P, P, C.c_size_t, P]
    L.aug_attn_mixed_noalloc.argtypes = [C.POINTER(aug_attn_shape), C.POINTER(aug_attn_plan_info), P, P, P, P,
                                         P, P, P, C.c_int32, P, P]
    L.aug_kv_append.argtypes = [C.POINTER(aug_attn_shape), C.POINTER(aug_attn_plan_info), P, P, P, P, P,
                                P, P, P, C.c_int32, P]
    L.aug_plan_upload.argtypes = [P, P, C.c_size_t, P]
    L.aug_kv_record_bytes.argtypes = [C.POINTER(aug_attn_shape)]
    L.aug_kv_record_bytes.restype = C.c_size_t
    L.aug_kv_park.argtypes = [C.POINTER(aug_attn_shape), P, P, P, P, P, P, C.c_int32, C.c_int32, P,
                              C.c_size_t, P, C.c_size_t, P]
    L.aug_kv_resume.argtypes = [C.POINTER(aug_attn_shape), P, P, P, P, P, P, C.c_int32, C.c_int32, P,
                                C.c_size_t, P, C.c_size_t, P]
    L.aug_form_batch.argtypes = [P, C.c_int32, C.c_int64, C.c_double, C.POINTER(aug_former_params),
                                 C.POINTER(aug_batch_plan)]
    L.aug_request_arrive.argtypes = [P, C.c_int64, C.c_double, C.c_int32, C.c_int32, C.c_double, C.c_int32]
    L.aug_request_return.argtypes = [P, C.c_int32, C.c_int32, C.c_int32, C.c_int32, C.c_double, C.c_int32]
    for f in ("aug_attn_plan", "aug_attn_plan_opts", "aug_attn_workspace_size", "aug_plan_upload", "aug_attn_mixed",
              "aug_attn_mixed_noalloc", "aug_kv_append", "aug_kv_park", "aug_kv_resume",
              "aug_form_batch", "aug_request_arrive", "aug_request_return"):
        getattr(L, f).restype = C.c_int
    L.aug_status_string.argtypes = [C.c_int]
    L.aug_status_string.restype = C.c_char_p
    L.aug_last_error.argtypes = []
    L.aug_last_error.restype = C.c_char_p
    L.aug_abi_version.restype = C.c_int32
    _lib = L
    return L


class _HostOnly:
    """A host-only build: its functions, and for each device entry point it
    lacks a stand-in that raises when called."""

    def __init__(self, L):
        self._L = L

    def __getattr__(self, name):
        try:
            return getattr(self._L, name)
        except AttributeError:
            def missing(*a, **k):
                raise RuntimeError(f"{name} is not in the host-only library {_HOST_ONLY_LIB}")
            missing.argtypes = missing.restype = None
            setattr(self, name, missing)
            return missing


def aug_status_string(status: int) -> str:
    return lib().aug_status_string(status).decode()


def aug_last_error() -> str:
    return lib().aug_last_error().decode()


def aug_abi_version() -> int:
    return int(lib().aug_abi_version())


def _check(status: int, who: str):
    if status != AUG_OK:
        raise AugError(status, f"{who}: {aug_status_string(status)}: {aug_last_error()}")


def _ptr(x) -> Optional[int]:
    """Address of a torch tensor / numpy array / int / None."""
    if x is None:
        return None
    if isinstance(x, int):
        return x
    if isinstance(x, np.ndarray):
        assert x.flags.c_contiguous
        return x.ctypes.data
    dp = getattr(x, "data_ptr", None)
    if dp is not None:
        assert x.is_contiguous()
        return x.data_ptr()
    raise TypeError(f"cannot take the address of {type(x)}")


def _stream(stream, *tensors):
    if stream is not None:
        return stream if isinstance(stream, int) else stream.cuda_stream
    import torch
    for t in tensors:
        if t is not None and hasattr(t, "is_cuda") and t.is_cuda:
            return torch.cuda.current_stream(t.device).cuda_stream
    return None


def _i32(a) -> np.ndarray:
    return np.ascontiguousarray(a, dtype=np.int32)


# ---- attention ---------------------------------------------------------------------

def make_shape(num_q_heads, num_kv_heads, head_dim, q_dtype, kv_dtype, out_dtype,
               softmax_scale, block_size=16) -> aug_attn_shape:
    code = lambda d: d if isinstance(d, int) else DTYPE_CODES[d]
    return aug_attn_shape(num_q_heads, num_kv_heads, head_dim, block_size, code(q_dtype),
                          code(kv_dtype), code(out_dtype), softmax_scale)


def _batch_desc(q_start, ctx_len, bt_start, num_pool_blocks, block_ids=None):
    """The C batch description and the int32 arrays it points into (which the
    caller keeps alive for the call)."""
    qs, cl, bs = _i32(q_start), _i32(ctx_len), _i32(bt_start)
    bi = None if block_ids is None else _i32(block_ids)
    p32 = C.POINTER(C.c_int32)
    desc = aug_batch_desc(len(cl), qs.ctypes.data_as(p32), cl.ctypes.data_as(p32),
                          bs.ctypes.data_as(p32), None if bi is None else bi.ctypes.data_as(p32),
                          int(num_pool_blocks))
    return desc, (qs, cl, bs, bi)


def aug_attn_plan(shape: aug_attn_shape, q_start, ctx_len, bt_start, num_pool_blocks: int,
                  block_ids=None, kv_split_tokens: int = 0, row_path: int = AUG_ROWS_AUTO,
                  tile_path: int = AUG_TILES_AUTO):
    """Validate a batch (host arrays) and build its plan image (aug_attn_plan,
    or aug_attn_plan_opts when a row or tile path is requested). Returns
    (info, plan) with plan a numpy uint8 array of info.plan_bytes bytes."""
    L = lib()
    desc, keep = _batch_desc(q_start, ctx_len, bt_start, num_pool_blocks, block_ids)
    opts = aug_plan_options(int(kv_split_tokens), int(row_path), int(tile_path))
    info = aug_attn_plan_info()
    # one scratch image per thread: ctypes releases the GIL during the call
    buf = getattr(_plan_scratch, "buf", None)
    if buf is None:
        buf = _plan_scratch.buf = np.zeros(1 << 20, dtype=np.uint8)
    while True:
        if row_path == AUG_ROWS_AUTO and tile_path == AUG_TILES_AUTO:
            st = L.aug_attn_plan(C.byref(shape), C.byref(desc), int(kv_split_tokens), buf.ctypes.data,
                                 buf.nbytes, C.byref(info))
        else:
            st = L.aug_attn_plan_opts(C.byref(shape), C.byref(desc), C.byref(opts), buf.ctypes.data, buf.nbytes,
                                      C.byref(info))
        if st == AUG_ERR_NO_SPACE and info.plan_bytes > buf.nbytes:
            buf = _plan_scratch.buf = np.zeros(int(info.plan_bytes) * 2, dtype=np.uint8)
            continue
        _check(st, "aug_attn_plan")
        return info, buf[:int(info.plan_bytes)].copy()


_plan_scratch = threading.local()


def aug_attn_workspace_size(shape: aug_attn_shape, q_start, ctx_len, bt_start, num_pool_blocks: int,
                            block_ids=None, kv_split_tokens: int = 0) -> int:
    """Bytes of device workspace aug_attn_mixed needs for this batch and split."""
    desc, keep = _batch_desc(q_start, ctx_len, bt_start, num_pool_blocks, block_ids)
    n = C.c_size_t(0)
    _check(lib().aug_attn_workspace_size(C.byref(shape), C.byref(desc), int(kv_split_tokens), C.byref(n)),
           "aug_attn_workspace_size")
    del keep
    return int(n.value)


def aug_plan_upload(host_src, dev_dst, nbytes: Optional[int] = None, stream=None):
    """Enqueue the copy of ``nbytes`` bytes (default: all of ``host_src``)
    from a pinned host tensor to a device tensor by the library's copy kernel
    on ``stream`` (default: the current stream of ``dev_dst``)."""
    if nbytes is None:
        nbytes = host_src.numel() * host_src.element_size()
    st = _stream(stream, dev_dst, dev_dst)
    _check(lib().aug_plan_upload(_ptr(host_src), _ptr(dev_dst), int(nbytes), st), "aug_plan_upload")


def aug_attn_mixed(shape: aug_attn_shape, info: aug_attn_plan_info, plan_dev, q, k_cache, v_cache,
                   k_scale, v_scale, block_ids, num_pool_blocks: int, out, workspace,
                   workspace_bytes: Optional[int] = None, stream=None):
    """Enqueue the attention of a planned batch (all device arguments are torch
    tensors or raw device addresses)."""
    if workspace_bytes is None:
        workspace_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    st = _stream(stream, q, out)
    _check(lib().aug_attn_mixed(C.byref(shape), C.byref(info), _ptr(plan_dev), _ptr(q),
                                _ptr(k_cache), _ptr(v_cache), _ptr(k_scale), _ptr(v_scale),
                                _ptr(block_ids), int(num_pool_blocks), _ptr(out), _ptr(workspace),
                                int(workspace_bytes), st), "aug_attn_mixed")


def aug_attn_mixed_noalloc(shape: aug_attn_shape, info: aug_attn_plan_info, plan_dev, q, k_cache, v_cache,
                           k_scale, v_scale, block_ids, num_pool_blocks: int, out, stream=None):
    """Enqueue the attention of a planned batch with the split-K partials in
    the library's own device array (no workspace argument)."""
    st = _stream(stream, q, out)
    _check(lib().aug_attn_mixed_noalloc(C.byref(shape), C.byref(info), _ptr(plan_dev), _ptr(q), _ptr(k_cache),
                                        _ptr(v_cache), _ptr(k_scale), _ptr(v_scale), _ptr(block_ids),
                                        int(num_pool_blocks), _ptr(out), st), "aug_attn_mixed_noalloc")


NOALLOC_SCRATCH_BYTES = 64 << 20


def aug_kv_append(shape: aug_attn_shape, info: aug_attn_plan_info, plan_dev, k_new, v_new, k_cache,
                  v_cache, k_scale, v_scale, block_ids, num_pool_blocks: int, stream=None):
    """Enqueue the write of the planned batch's new K/V rows into the pool
    (all device arguments are torch tensors or raw device addresses)."""
    st = _stream(stream, k_new, k_cache)
    _check(lib().aug_kv_append(C.byref(shape), C.byref(info), _ptr(plan_dev), _ptr(k_new), _ptr(v_new),
                               _ptr(k_cache), _ptr(v_cache), _ptr(k_scale), _ptr(v_scale),
                               _ptr(block_ids), int(num_pool_blocks), st), "aug_kv_append")


# ---- park / resume -------------------------------------------------------------------

def aug_kv_record_bytes(shape: aug_attn_shape) -> int:
    return int(lib().aug_kv_record_bytes(C.byref(shape)))


def aug_kv_park(shape, k_cache, v_cache, k_scale, v_scale, block_ids_dev, n_blocks: int,
                num_pool_blocks: int, host_dst, staging, block_ids_host=None, stream=None):
    hb = None if block_ids_host is None else _i32(block_ids_host)
    st = _stream(stream, k_cache)
    _check(lib().aug_kv_park(C.byref(shape), _ptr(k_cache), _ptr(v_cache), _ptr(k_scale),
                             _ptr(v_scale), _ptr(block_ids_dev), _ptr(hb), int(n_blocks),
                             int(num_pool_blocks), _ptr(host_dst),
                             host_dst.numel() * host_dst.element_size(), _ptr(staging),
                             staging.numel() * staging.element_size(), st), "aug_kv_park")


def aug_kv_resume(shape, k_cache, v_cache, k_scale, v_scale, block_ids_dev, n_blocks: int,
                  num_pool_blocks: int, host_src, staging, block_ids_host=None, stream=None):
    hb = None if block_ids_host is None else _i32(block_ids_host)
    st = _stream(stream, k_cache)
    _check(lib().aug_kv_resume(C.byref(shape), _ptr(k_cache), _ptr(v_cache), _ptr(k_scale),
                               _ptr(v_scale), _ptr(block_ids_dev), _ptr(hb), int(n_blocks),
                               int(num_pool_blocks), _ptr(host_src),
                               host_src.numel() * host_src.element_size(), _ptr(staging),
                               staging.numel() * staging.element_size(), st), "aug_kv_resume")


# ---- batch former ----------------------------------------------------------------------

AUG_ORDER_THETA, AUG_ORDER_FCFS, AUG_ORDER_SSJF = 0, 1, 2


def former_params(beta=5e-5, t_max=2048, beta_low=0.5, beta_high=2.0, chunk_cap=512, t_iter=0.02,
                  fwd_a=0.015, fwd_b=2.0e-8, swap_s_per_tok=2.0e-6, n_fwd_max=1,
                  skip_instead_of_break=0, block_size=16, order=AUG_ORDER_THETA) -> aug_former_params:
    return aug_former_params(beta, beta_low, beta_high, t_iter, fwd_a, fwd_b, swap_s_per_tok,
                             int(n_fwd_max), int(t_max), int(chunk_cap), int(block_size),
                             int(skip_instead_of_break), int(order), 0)


_former_scratch = threading.local()


def _former_outputs(cap: int):
    """The calling thread's output arrays of aug_form_batch (at least ``cap``
    entries each) and the aug_batch_plan pointing at them, reused across
    calls; callers copy what they return."""
    sc = getattr(_former_scratch, "v", None)
    if sc is None or sc[-1].cap < cap:
        cap = max(cap, 64 if sc is None else 2 * sc[-1].cap)
        arrs = [np.zeros(cap, t) for t in (np.int64, np.int32, np.float64, np.int64, np.int64, np.int64,
                                            np.int32, np.float64)]
        P64, P32, PD = C.POINTER(C.c_int64), C.POINTER(C.c_int32), C.POINTER(C.c_double)
        ptrs = [a.ctypes.data_as(pt) for a, pt in zip(arrs, (P64, P32, PD, P64, P64, P64, P32, PD))]
        sc = _former_scratch.v = (*arrs, aug_batch_plan(cap, 0, 0, 0, 0, 0, *ptrs))
    return sc


def aug_form_batch(reqs: np.ndarray, free_blocks: int, now: float, params: aug_former_params):
    """Form one batch from a structured array of REQUEST_DTYPE. Returns a dict
    with budget, ids, q_len, theta, resume_ids, park_ids, free_ids, policy, cost."""
    reqs = np.ascontiguousarray(reqs, dtype=REQUEST_DTYPE)
    n = len(reqs)
    ids, q_len, theta, res, park, free, pol, cost, out = _former_outputs(max(n, 1))
    out.budget = out.n_sched = out.n_resume = out.n_park = out.n_free = 0
    _check(lib().aug_form_batch(reqs.ctypes.data if n else None, n, int(free_blocks), float(now),
                                C.byref(params), C.byref(out)), "aug_form_batch")
    k = out.n_sched
    return dict(budget=out.budget, ids=ids[:k].copy(), q_len=q_len[:k].copy(),
                theta=theta[:k].copy(), resume_ids=res[:out.n_resume].copy(),
                park_ids=park[:out.n_park].copy(), free_ids=free[:out.n_free].copy(),
                policy=pol[:n].copy(), cost=cost[:n].copy())


# ---- request records (Algorithm 1, steps (1)-(2)) ------------------------------------

def aug_request_arrive(id: int, arrival: float, prompt_tokens: int, pred_out: int, pred_call: float,
                       has_next_call: int) -> np.ndarray:
    """The record (one REQUEST_DTYPE element) of a newly arrived request."""
    rec = np.zeros(1, REQUEST_DTYPE)
    _check(lib().aug_request_arrive(rec.ctypes.data, int(id), float(arrival), int(prompt_tokens),
                                    int(pred_out), float(pred_call), int(has_next_call)),
           "aug_request_arrive")
    return rec[0]


def aug_request_return(rec: np.ndarray, realised: int, context_tokens: int, ret_tokens: int,
                       pred_out: int, pred_call: float, has_next_call: int) -> np.ndarray:
    """The record after a paused request's external call returned (a new
    REQUEST_DTYPE element; `rec` is not modified)."""
    out = np.array([rec], REQUEST_DTYPE)
    _check(lib().aug_request_return(out.ctypes.data, int(realised), int(context_tokens), int(ret_tokens),
                                    int(pred_out), float(pred_call), int(has_next_call)),
           "aug_request_return")
    return out[0]
