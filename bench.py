"""Benchmark of one mixed-batch serving step on one MI355X.

A step is one pass of the hot path over one batch: the host batch former
(token budget, cost, priority, greedy packing), the host planner, the
upload of the work list, the append of the step's new K/V rows to the paged
cache, and the attention launch(es) over it.
Inputs are synthetic, seeded, and resident in HBM before timing starts.
Workloads that move paused requests (mixed-8b, long-context-8b) also time
their resume and park on their own, after the steps, and report them in
``park_resume`` as GB/s of the host link beside a plain pinned-memory copy of
the same size; those host transfers are not part of ``value``.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload mixed-8b] [--also a,b]

Prints one JSON line. The main workload is the mixed batch of 3 x 512-row
prefill chunks and 512 decodes under a 2048-token budget on the 8B-shaped
layer; the decode-only batch, the long-context split-K batch and the
prefill-dominated 64/8-head fp8 batch follow in the same run, each reported
under ``workloads`` with its own roofline. ``value`` is query tokens per second of whole steps;
``roofline`` relates the attention launches' algorithmic bytes (each KV byte
a request reads counted once, plus Q, O and block ids) to their duration,
measured with HIP events on the launch stream; ``cpu_baseline`` times the
CPU oracle on a bounded sample of the same batch.
"""

from __future__ import annotations

import argparse
import gc
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
MFMA_BF16_PEAK_TFS = 2516.6
MFMA_FP8_PEAK_TFS = 2 * MFMA_BF16_PEAK_TFS

WORKLOADS = {
    "tiny-mixed": 1,
    "decode-8b": 2,
    "mixed-8b": 3,
    "long-context-8b": 4,
    # batches the library's former forms from the 2000-request augmented trace
    # under an 8192-token budget, on the 64/8-head fp8-KV layer
    "sweep-prefill-fp8": 5,   # the batch with the most prefill query-key pairs
    "sweep-context-fp8": 5,   # the batch with the most context tokens
    # a typical small batch: under a 512-token budget, the formed batch with the
    # median number of context tokens
    "sweep-median-512-fp8": 5,
    # 512 decodes on the same 64/8-head fp8 layer (decode-dominated, full size)
    "decode-fp8-64x8": 7,
    # prefill-dominated batches: 16 x 512-row chunks on the 64/8-head fp8
    # layer (an 8192-token budget), 8 x 512-row chunks on the 8B bf16 layer
    "prefill-fp8-64x8": 8,
    "prefill-8b": 9,
    # every budget 256 ... 8192: a sample of the formed batches replayed on one pool
    "budget-sweep-fp8": 6,
}
# timed after the main (mixed-batch) workload in the default run, each with its own roofline
# (a workload name followed by "@valu" runs its row items on the vector ALUs instead of the
# planner's default, which is MFMA for eight query heads per KV head; "@mfma" runs four-head
# groups' row items on the MFMA row path, which they take only when asked; "@fp8qk" runs the
# prefill tiles' score products on fp8 MFMAs and "@fp8" both of their products, opt-in arithmetic)
DEFAULT_ALSO = ("mixed-8b@mfma", "decode-8b", "decode-8b@mfma", "long-context-8b", "prefill-fp8-64x8",
                "prefill-fp8-64x8@fp8qk", "prefill-fp8-64x8@fp8", "decode-fp8-64x8", "decode-fp8-64x8@valu")
PATHS = {"": (0, 0), "valu": (1, 0), "mfma": (2, 0), "fp8qk": (0, 2), "fp8": (0, 3)}   # suffix -> (rows, tiles)
PATH_NOTES = {"": "", "valu": " (vector-ALU rows)", "mfma": " (MFMA rows)", "fp8qk": " (fp8 scores)",
              "fp8": " (fp8 scores and values)"}


def algorithmic_bytes(b) -> float:
    elem = {"f32": 4, "bf16": 2, "fp8": 1}
    kv = float(np.sum(b.ctx_len.astype(np.int64))) * b.num_kv_heads * 2 * b.head_dim * elem[b.kv_dtype]
    nblk = np.sum((b.ctx_len.astype(np.int64) + 15) // 16)
    scales = float(nblk) * b.num_kv_heads * 2 * 4 if b.kv_dtype == "fp8" else 0.0
    qo = float(b.total_q) * b.num_q_heads * b.head_dim * (elem[b.q_dtype] + elem[b.out_dtype])
    return kv + scales + qo + float(nblk) * 4


def prefill_flops(b) -> float:
    q = b.q_len.astype(np.int64)
    ctx = b.ctx_len.astype(np.int64)
    pre = q > 1
    # rows j attend pos_j + 1 keys: sum = q*(ctx-q) + q(q+1)/2
    keys = (q * (ctx - q) + q * (q + 1) // 2)[pre]
    return float(4 * b.head_dim * b.num_q_heads * keys.sum())


def append_bytes(b, info) -> float:
    """Algorithmic bytes of one append: every new row's K and V read once in
    the caller's format and written once in the cache's, per KV head; for fp8
    caches one scale read and written per (block, KV head, K|V); the append
    list and block ids. Re-encoding earlier tokens when a scale grows depends
    on the data and is not counted."""
    row_in = 4 if b.kv_dtype == "f32" else 2
    row_out = {"f32": 4, "bf16": 2, "fp8": 1}[b.kv_dtype]
    n = float(b.total_q) * b.num_kv_heads * b.head_dim * 2 * (row_in + row_out)
    items = int(info.num_append_items)
    if b.kv_dtype == "fp8":
        n += items * b.num_kv_heads * 2 * 8
    return n + items * (16 + 4)


def traffic_key(workload_name: str, row_path: int = 0, tile_path: int = 0):
    """Name of a workload's counter record: the workload itself on the
    planner's default paths, ``<workload>@<suffix>`` on an opt-in path (the
    suffixes of PATHS)."""
    for suffix, paths in PATHS.items():
        if paths == (row_path, tile_path):
            return workload_name + ("@" + suffix if suffix else "")
    return None


def measured_traffic(workload_name):
    """HBM bytes per attention call from the committed rocprofv3 counter
    summary, or None when the summary does not cover this workload (or path)
    or the kernel and planner sources have changed since the counters were
    taken."""
    import hashlib
    if workload_name is None:
        return None
    path = os.path.join(ROOT, "profiles", "hbm_traffic.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        rec = json.load(f)
    h = hashlib.sha256()
    for name in rec.get("source_files", []):
        with open(os.path.join(ROOT, name), "rb") as f:
            h.update(f.read())
    if h.hexdigest() != rec.get("source_sha256"):
        return None
    w = rec.get("workloads", {}).get(workload_name)
    return None if w is None else int(w["bytes_per_call"])


def request_records(b, aug):
    """Scheduler view of the batch: prefill chunks as waiting requests with
    pending tokens, decodes as running requests."""
    recs = np.zeros(b.num_reqs, aug.REQUEST_DTYPE)
    for r in range(b.num_reqs):
        q, ctx = int(b.q_len[r]), int(b.ctx_len[r])
        rec = recs[r]
        rec["id"] = r
        rec["arrival"] = 0.001 * r
        rec["last_sched"] = -1.0
        rec["seg"] = 1
        rec["seg_prefill"] = ctx if q == 1 else ctx
        rec["pred_out"] = 64
        rec["ctx_len"] = ctx - q
        rec["pending"] = q if q > 1 else 0
        rec["state"] = aug.AUG_WAITING if q > 1 else aug.AUG_RUNNING
        rec["blocks_on_gpu"] = (ctx - q + 15) // 16 if q > 1 else (ctx + 15) // 16
    return recs


def cpu_baseline(b, budget_s: float = 15.0):
    """Time the oracle on a prefix of the batch's requests (about budget_s of
    CPU work), reported in query tokens per second."""
    from oracle import attention as oa
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:  # noqa: BLE001
        threads = len(os.sched_getaffinity(0))
    order = list(range(b.num_reqs))
    elem = {"f32": 4, "bf16": 2, "fp8": 1}[b.kv_dtype]
    kv_per_token = 2 * b.num_kv_heads * b.head_dim * elem     # K and V bytes of one context token
    done_rows, t_used, n_done, kv_bytes = 0, 0.0, 0, 0
    for r in order:
        t0 = time.perf_counter()
        oa.attention_for(b, requests=[r])
        t_used += time.perf_counter() - t0
        done_rows += int(b.q_len[r])
        kv_bytes += int(b.ctx_len[r]) * kv_per_token
        n_done += 1
        if t_used >= budget_s:
            break
    res = {"value": done_rows / t_used, "unit": "query-tokens/s", "cores": int(threads),
           "affinity_cores": len(os.sched_getaffinity(0)),
           "kv_gbs": round(kv_bytes / t_used / 1e9, 4), "kind": "oracle",
           "sample": f"first {n_done} of {b.num_reqs} requests ({done_rows} query rows), float64 numpy, "
                     f"{t_used:.1f} s"}
    # the same sample again with numpy's BLAS held to one thread
    try:
        from threadpoolctl import threadpool_limits
    except Exception:  # noqa: BLE001
        return res
    t1, rows1, n1 = 0.0, 0, 0
    with threadpool_limits(limits=1):
        for r in order[:n_done]:
            t0 = time.perf_counter()
            oa.attention_for(b, requests=[r])
            t1 += time.perf_counter() - t0
            rows1 += int(b.q_len[r])
            n1 += 1
            if t1 >= budget_s / 3:
                break
    res["single_core"] = {"value": rows1 / t1, "unit": "query-tokens/s", "cores": 1,
                          "sample": f"first {n1} requests ({rows1} query rows), {t1:.1f} s"}
    return res


PCIE_PEAK_GBS = 64.0   # PCIe Gen5 x16, per direction


def park_resume_rates(b, kv, log, reps: int = 3):
    """Time aug_kv_resume of the batch's resumed requests and aug_kv_park of
    the requests it parks (HIP events on the launch stream, mean of `reps`),
    and a plain hipMemcpyAsync between pinned host memory and the device of
    the same byte counts for comparison."""
    import torch
    pk = b.park
    dev = kv.k_cache.device
    stream = torch.cuda.current_stream(dev)
    res_ids = np.asarray(pk.resume_blocks, np.int32)
    src_ids = np.asarray(pk.resume_src_blocks, np.int32)
    park_ids = np.asarray(pk.park_blocks if len(pk.park_blocks) else pk.resume_src_blocks, np.int32)
    res_dev = torch.from_numpy(res_ids).to(dev)
    src_dev = torch.from_numpy(src_ids).to(dev)
    park_dev = torch.from_numpy(park_ids).to(dev)
    img = kv.host_buffer(len(src_ids))
    kv.park(src_ids, src_dev, img)            # the parked image the resume reads back
    out = kv.host_buffer(len(park_ids))
    torch.cuda.synchronize()

    def timed(fn):
        fn()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(reps):
            fn()
        e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) * 1e-3 / reps

    res_bytes = len(res_ids) * kv.record_bytes
    park_bytes = len(park_ids) * kv.record_bytes
    t_res = timed(lambda: kv.resume(res_ids, res_dev, img))
    t_park = timed(lambda: kv.park(park_ids, park_dev, out))
    d_buf = torch.empty(max(res_bytes, park_bytes), dtype=torch.uint8, device=dev)
    t_h2d = timed(lambda: d_buf[:res_bytes].copy_(img[:res_bytes], non_blocking=True))
    t_d2h = timed(lambda: out[:park_bytes].copy_(d_buf[:park_bytes], non_blocking=True))
    r = {"resume_blocks": int(len(res_ids)), "resume_bytes": int(res_bytes),
         "resume_gbs": round(res_bytes / t_res / 1e9, 2),
         "park_blocks": int(len(park_ids)), "park_bytes": int(park_bytes),
         "park_gbs": round(park_bytes / t_park / 1e9, 2),
         "h2d_copy_gbs": round(res_bytes / t_h2d / 1e9, 2), "d2h_copy_gbs": round(park_bytes / t_d2h / 1e9, 2),
         "pcie_peak_gbs": PCIE_PEAK_GBS, "reps": reps}
    log(f"park/resume: {r}")
    return r


class TimingEvent:
    """A HIP timing event created with hipEventDisableSystemFence: its
    timestamp is taken when the stream reaches it, without the system-scope
    cache write-back and invalidation of an ordinary event, which would
    otherwise fall inside the measured window and delay the next launch (the
    HIP runtime documents the flag for timing-only events). Same record /
    elapsed_time interface as torch.cuda.Event."""

    DISABLE_SYSTEM_FENCE = 0x20000000
    _hip = None

    def __init__(self):
        import ctypes as C
        if TimingEvent._hip is None:
            # the HIP runtime torch has already loaded, so that its streams are valid here
            loaded = sorted({ln.split()[-1] for ln in open("/proc/self/maps") if "libamdhip64" in ln})
            L = C.CDLL(loaded[0] if loaded else "libamdhip64.so.7")
            L.hipEventCreateWithFlags.argtypes = [C.POINTER(C.c_void_p), C.c_uint]
            L.hipEventRecord.argtypes = [C.c_void_p, C.c_void_p]
            L.hipEventSynchronize.argtypes = [C.c_void_p]
            L.hipEventElapsedTime.argtypes = [C.POINTER(C.c_float), C.c_void_p, C.c_void_p]
            TimingEvent._hip = L
        self._c = C
        self.h = C.c_void_p()
        if self._hip.hipEventCreateWithFlags(C.byref(self.h), self.DISABLE_SYSTEM_FENCE) != 0:
            raise RuntimeError("hipEventCreateWithFlags failed")

    def record(self, stream):
        if self._hip.hipEventRecord(self.h, self._c.c_void_p(stream.cuda_stream)) != 0:
            raise RuntimeError("hipEventRecord failed")

    def elapsed_time(self, end: "TimingEvent") -> float:
        """Milliseconds from this event to ``end`` (waits for ``end``)."""
        ms = self._c.c_float()
        if self._hip.hipEventSynchronize(end.h) != 0 or \
                self._hip.hipEventElapsedTime(self._c.byref(ms), self.h, end.h) != 0:
            raise RuntimeError("hipEventElapsedTime failed")
        return ms.value


def time_layers(n_layers, shape, info, plan_dev, k_new, v_new, q, pools, bids, num_pool_blocks, out, ws,
                stream, log, reps: int = 20):
    """One planned batch run as ``n_layers`` layers (per layer: the KV append
    and the attention call, layer l on pool copy l mod copies), launched one
    call at a time and as one captured HIP graph. Returns per-step and
    per-layer times of both (medians over ``reps``)."""
    import torch
    import paper_2512_04013_amd as aug

    def layers(st):
        for l in range(n_layers):
            kc, vc, ksc, vsc = pools[l % len(pools)]
            aug.aug_kv_append(shape, info, plan_dev, k_new, v_new, kc, vc, ksc, vsc, bids, num_pool_blocks,
                              stream=st)
            aug.aug_attn_mixed(shape, info, plan_dev, q, kc, vc, ksc, vsc, bids, num_pool_blocks, out, ws,
                               stream=st)

    def timed(fn):
        ts = []
        for _ in range(reps + 3):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            fn()
            e1.record(stream)
            e1.synchronize()
            ts.append(e0.elapsed_time(e1))
        return float(np.median(ts[3:]))

    eager_ms = timed(lambda: layers(stream.cuda_stream))
    side = torch.cuda.Stream()
    side.wait_stream(stream)
    with torch.cuda.stream(side):
        layers(side.cuda_stream)
    stream.wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        layers(torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    graph_ms = timed(g.replay)
    log(f"{n_layers} layers: {eager_ms:.3f} ms launched one by one, {graph_ms:.3f} ms as one graph")
    return {"n": n_layers, "what": "KV append + attention per layer, one plan, layer l on pool copy l mod copies",
            "eager_ms_per_step": round(eager_ms, 4), "graph_ms_per_step": round(graph_ms, 4),
            "eager_us_per_layer": round(1e3 * eager_ms / n_layers, 2),
            "graph_us_per_layer": round(1e3 * graph_ms / n_layers, 2)}


def make_workload(name: str, seed: int, log):
    """The workload's batch and the budget T_max it is formed under."""
    import synth
    cfg = WORKLOADS[name]
    if cfg == 7:
        return synth.make_decode_gqa8_fp8(seed=seed), 8192
    if cfg == 8:
        return synth.make_prefill_gqa8_fp8(seed=seed), 8192
    if cfg == 9:
        return synth.make_prefill_8b(seed=seed), 4096
    if cfg != 5:
        return synth.make_config(cfg, seed=seed), 2048
    from synth import sweep
    from paper_2512_04013_amd import runtime as rt
    budget = 512 if name == "sweep-median-512-fp8" else 8192
    t0 = time.time()
    run = sweep.run_budget(budget, rt.serving_former(**sweep.former_params(budget)), rt.serving_lifecycle(),
                           seed=seed)
    if name == "sweep-median-512-fp8":
        ctx = np.array([sum(st.ctx_len) for st in run.steps])
        pick = int(np.argsort(ctx, kind="stable")[len(ctx) // 2])
    else:
        pick = sweep.select_steps(run.steps, 0, seed)["most_prefill" if name == "sweep-prefill-fp8" else "most_context"]
    log(f"trace served under budget {budget}: {len(run.steps)} batches in {time.time() - t0:.1f} s; "
        f"batch {pick} chosen")
    return sweep.batch_for_step(run.steps[pick], seed=seed + 1000, name=f"{name}-budget{budget}"), budget


def budget_sweep(args, log):
    """Token-budget sweep: for each budget, serve the 2000-request trace with
    the library's former, then replay a sample of the batches it formed (up
    to --sweep-batches, evenly spaced over the run, plus its largest and most
    prefill-heavy batch) through planner, upload and attention on one 65,536-
    block fp8 pool of random codes and scales. Reports per budget and overall:
    query tokens per second of the attention launches (HIP events) and of
    whole replayed steps, and the fractions of the HBM and MFMA roofs. Each
    replayed batch also runs as --sweep-layers layers back to back (each layer
    on its own random blocks of the pool, one plan for all), timed as one
    window: the per-layer figures of a multi-layer step, where no launch
    waits on the host."""
    import torch
    import paper_2512_04013_amd as aug
    from paper_2512_04013_amd import runtime as rt
    from synth import sweep

    dev = torch.device("cuda:0")
    rng = np.random.default_rng(args.seed)
    runs = {}
    for budget in sweep.BUDGETS:
        t0 = time.time()
        run = sweep.run_budget(budget, rt.serving_former(**sweep.former_params(budget)), rt.serving_lifecycle(),
                               seed=args.seed, max_steps=40_000)
        n = len(run.steps)
        pick = sorted(set(np.linspace(0, n - 1, min(n, args.sweep_batches)).astype(int).tolist())
                      | {sweep.select_steps(run.steps, 0, 0)[k] for k in ("most_tokens", "most_prefill")})
        runs[budget] = (run, pick)
        log(f"budget {budget}: {n} batches formed ({'whole trace' if run.complete else 'overloaded, stopped'}), "
            f"{len(pick)} replayed ({time.time() - t0:.1f} s)")
    hq, hkv, d = sweep.HEADS_Q, sweep.HEADS_KV, sweep.HEAD_DIM
    # the device pool is four times the simulator's, so the random blocks of
    # consecutive batches rarely meet in the 256 MB last-level cache
    nb = 4 * sweep.POOL_BLOCKS
    gen = torch.Generator(device=dev).manual_seed(args.seed)
    shape_kv = (nb, hkv, 16, d)
    sign = torch.randint(0, 2, shape_kv, device=dev, dtype=torch.uint8, generator=gen) << 7
    k_cache = torch.randint(0, 0x7F, shape_kv, device=dev, dtype=torch.uint8, generator=gen) | sign
    sign = torch.randint(0, 2, shape_kv, device=dev, dtype=torch.uint8, generator=gen) << 7
    v_cache = torch.randint(0, 0x7F, shape_kv, device=dev, dtype=torch.uint8, generator=gen) | sign
    del sign
    k_scale = torch.rand((nb, hkv), device=dev, generator=gen) * 1e-3 + 1e-4
    v_scale = torch.rand((nb, hkv), device=dev, generator=gen) * 1e-3 + 1e-4
    pool_perm = rng.permutation(nb).astype(np.int32)
    max_rows = max(sum(r.steps[i].q_len) for r, pick in runs.values() for i in pick)
    q = torch.randn((max_rows, hq, d), device=dev, generator=gen).to(torch.bfloat16)
    out = torch.empty((max_rows, hq, d), device=dev, dtype=torch.bfloat16)
    shape = aug.make_shape(hq, hkv, d, "bf16", "fp8", "bf16", float(1.0 / np.sqrt(d)))
    stream = torch.cuda.current_stream(dev)
    up_dev = torch.empty(64 << 20, dtype=torch.uint8, device=dev)   # plan image, then block ids
    ws_dev = torch.empty(256 << 20, dtype=torch.uint8, device=dev)
    host = [torch.empty(64 << 20, dtype=torch.uint8, pin_memory=True) for _ in range(2)]
    host_ev = [None, None]

    class B:   # the fields algorithmic_bytes / prefill_flops read
        pass

    results = {}
    t_all, q_all, bytes_all, flops_all, wall_all, t_all_l = 0.0, 0, 0.0, 0.0, 0.0, 0.0
    n_layers = max(1, int(args.sweep_layers))
    # every budget's batches are replayed twice; only the second pass is timed, so
    # no budget pays for first launches (code loading, clocks ramping up)
    for budget, (run, pick), timed_pass in [(b, rp, p) for p in (False, True) for b, rp in runs.items()]:
        evs, qsum, nbytes, nflops = [], 0, 0.0, 0.0
        kinds = []          # per replayed batch: (prefill-dominated?, bytes, flops)
        torch.cuda.synchronize()
        w0 = time.perf_counter()
        for k, i in enumerate(pick):
            step = run.steps[i]
            q_len = np.asarray(step.q_len, np.int32)
            ctx = np.asarray(step.ctx_len, np.int32)
            nblk = (ctx.astype(np.int64) + 15) // 16
            q_start = np.zeros(len(q_len) + 1, np.int32)
            q_start[1:] = np.cumsum(q_len)
            bt_start = np.zeros(len(q_len) + 1, np.int32)
            bt_start[1:] = np.cumsum(nblk)
            # a random window of one fixed random permutation of the pool
            # (distinct blocks, O(batch) host work per step)
            n_bt = int(bt_start[-1])
            bids = np.concatenate([np.take(pool_perm, rng.integers(nb) + np.arange(n_bt), mode="wrap")
                                   for _ in range(n_layers)])
            info, plan = aug.aug_attn_plan(shape, q_start, ctx, bt_start, nb, None)
            slot = k & 1
            if host_ev[slot] is not None:
                host_ev[slot].synchronize()
            hb = host[slot]
            off = -(-plan.size // 256) * 256
            hb.numpy()[:plan.size] = plan
            hb.numpy()[off:off + bids.nbytes] = bids.view(np.uint8)
            aug.aug_plan_upload(hb, up_dev, off + bids.nbytes, stream=stream.cuda_stream)
            plan_dev = up_dev[:plan.size]
            bid_all = up_dev[off:off + bids.nbytes].view(torch.int32)
            host_ev[slot] = torch.cuda.Event()
            host_ev[slot].record(stream)
            e0, e1, e2 = TimingEvent(), TimingEvent(), TimingEvent()
            e0.record(stream)
            for layer in range(n_layers):
                aug.aug_attn_mixed(shape, info, plan_dev, q, k_cache, v_cache, k_scale, v_scale,
                                   bid_all[layer * n_bt:(layer + 1) * n_bt], nb, out, ws_dev,
                                   stream=stream.cuda_stream)
                if layer == 0:
                    e1.record(stream)
            e2.record(stream)
            evs.append((e0, e1, e2))
            b = B()
            b.q_len, b.ctx_len, b.total_q = q_len, ctx, int(q_start[-1])
            b.num_kv_heads, b.num_q_heads, b.head_dim = hkv, hq, d
            b.kv_dtype, b.q_dtype, b.out_dtype = "fp8", "bf16", "bf16"
            qsum += b.total_q
            bb, ff = algorithmic_bytes(b), prefill_flops(b)
            nbytes += bb
            nflops += ff
            kinds.append((ff / (MFMA_BF16_PEAK_TFS * 1e12) > bb / (HBM_PEAK_GBS * 1e9), bb, ff))
        torch.cuda.synchronize()
        wall = time.perf_counter() - w0
        if not timed_pass:
            continue
        times = [a.elapsed_time(c) * 1e-3 for a, c, _ in evs]
        t = sum(times)
        # per layer of an n_layers-layer step: the window over all layers / n_layers
        times_l = [a.elapsed_time(e) * 1e-3 / n_layers for a, _, e in evs]
        t_l = sum(times_l)

        def by_bound(ts_all):
            out_k = {}
            for label, pre in (("prefill_dominated", True), ("decode_dominated", False)):
                sel = [(tt, bb, ff) for tt, (p_dom, bb, ff) in zip(ts_all, kinds) if p_dom == pre]
                if sel:
                    ts = sum(x[0] for x in sel)
                    out_k[label] = {"batches": len(sel), "attn_us_per_batch": round(1e6 * ts / len(sel), 1),
                                    "mfma_frac": round(sum(x[2] for x in sel) / ts / (MFMA_BF16_PEAK_TFS * 1e12), 4),
                                    "hbm_frac": round(sum(x[1] for x in sel) / ts / (HBM_PEAK_GBS * 1e9), 4)}
            return out_k
        by_kind = by_bound(times)
        results[budget] = {"batches_formed": len(run.steps), "trace_complete": bool(run.complete),
                           "by_bound": by_kind,
                           "batches_replayed": len(pick), "query_tokens": int(qsum),
                           "attn_query_tokens_per_s": round(qsum / t, 1), "step_query_tokens_per_s": round(qsum / wall, 1),
                           "hbm_frac": round(nbytes / t / (HBM_PEAK_GBS * 1e9), 4),
                           "mfma_frac": round(nflops / t / (MFMA_BF16_PEAK_TFS * 1e12), 4),
                           "attn_ms_per_batch": round(1e3 * t / len(pick), 4),
                           "per_layer": {"layers": n_layers, "attn_ms_per_batch": round(1e3 * t_l / len(pick), 4),
                                         "hbm_frac": round(nbytes / t_l / (HBM_PEAK_GBS * 1e9), 4),
                                         "mfma_frac": round(nflops / t_l / (MFMA_BF16_PEAK_TFS * 1e12), 4),
                                         "by_bound": by_bound(times_l)},
                           # the library former's own time per iteration over the whole trace
                           # (the paper's per-iteration scheduling overhead, Table 3)
                           "former_per_iteration": run.former_stats}
        log(f"budget {budget}: {results[budget]}")
        t_all += t
        t_all_l += t_l
        wall_all += wall
        q_all += qsum
        bytes_all += nbytes
        flops_all += nflops
    achieved_gbs = bytes_all / t_all / 1e9
    achieved_tfs = flops_all / t_all / 1e12
    if flops_all / (MFMA_BF16_PEAK_TFS * 1e12) > bytes_all / (HBM_PEAK_GBS * 1e9):
        roof = {"bound": "mfma", "achieved": round(achieved_tfs, 1), "peak": MFMA_BF16_PEAK_TFS, "unit": "TFLOP/s",
                "frac": round(achieved_tfs / MFMA_BF16_PEAK_TFS, 4), "traffic": None}
    else:
        roof = {"bound": "hbm", "achieved": round(achieved_gbs, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": round(achieved_gbs / HBM_PEAK_GBS, 4), "traffic": None}
    roof.update({"kernel": "aug_attn_mixed launches over all replayed batches",
                 "prefill_mfma_tflops": round(achieved_tfs, 2), "hbm_gbs": round(achieved_gbs, 1),
                 "per_layer": {"layers": n_layers, "hbm_gbs": round(bytes_all / t_all_l / 1e9, 1),
                               "hbm_frac": round(bytes_all / t_all_l / 1e9 / HBM_PEAK_GBS, 4),
                               "prefill_mfma_tflops": round(flops_all / t_all_l / 1e12, 2),
                               "what": "each batch's attention as layers back to back, one window over all "
                                       "layers divided by their number"}})
    n_rep = sum(len(p) for _, p in runs.values())
    result = {
        "metric": "mixed-batch attn query-tokens/s + % peak HBM GB/s (decode) / % MFMA (prefill)",
        "value": round(q_all / wall_all, 1), "unit": "query-tokens/s", "n_gpus": 1, "steps": n_rep, "warmup": 0,
        "ms_per_step": round(1e3 * wall_all / n_rep, 4), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16-q/fp8e4m3-kv", "data": "synthetic",
        "config": {"workload": "budget-sweep-fp8", "trace_requests": 2000, "q_heads": hq, "kv_heads": hkv,
                   "head_dim": d, "block_size": 16, "pool_blocks": nb, "seed": args.seed,
                   "budgets": {str(k): v for k, v in results.items()}},
        "roofline": roof,
    }
    print(json.dumps(result), flush=True)


def run_workload(name: str, args, log, full: bool = True, row_path: int = 0, tile_path: int = 0) -> dict:
    """Time ``args.steps`` whole steps of one workload (after ``args.warmup``
    untimed ones) and return its result record: query tokens per second of
    whole steps, the attention call's roofline and the KV append's rate; with
    ``full`` also park/resume, the several-layer timing and the CPU oracle."""
    import torch
    import paper_2512_04013_amd as aug
    from paper_2512_04013_amd import runtime as rt
    import synth

    dev = torch.device("cuda:0")
    t0 = time.time()
    b, t_max = make_workload(name, args.seed, log)
    log(f"workload {b.name}: {b.num_reqs} requests, {b.total_q} query rows, "
        f"{int(b.ctx_len.sum())} context tokens ({time.time() - t0:.1f} s to generate)")
    shape, kv, q, bids = rt.upload_batch(b, device=dev)
    # identical copies of the pool, used in turn, so that consecutive steps
    # never find a small batch's KV in the 256 MB last-level cache
    touched = algorithmic_bytes(b)
    n_copies = args.pool_copies or int(min(8, max(1, np.ceil((1 << 30) / touched))))
    pools = [(kv.k_cache, kv.v_cache, kv.k_scale, kv.v_scale)]
    for _ in range(n_copies - 1):
        pools.append(tuple(None if x is None else x.clone() for x in pools[0]))
    torch.cuda.synchronize()
    log(f"{n_copies} copies of the pool, used in turn")

    recs = request_records(b, aug)
    used_blocks = int(np.sum((b.ctx_len.astype(np.int64) + 15) // 16))
    free_blocks = b.num_pool_blocks - used_blocks
    if WORKLOADS[name] == 5:
        # a trace-formed batch is re-formed with the sweep's own former parameters
        # (dynamic budget up to twice T_max, chunks capped at half of it)
        from synth import sweep
        params = aug.former_params(**sweep.former_params(t_max))
    else:
        params = aug.former_params(t_max=t_max, beta_low=0.5, beta_high=1.0, chunk_cap=512)
    stream = torch.cuda.current_stream(dev)
    plan_dev = torch.empty(64 << 20, dtype=torch.uint8, device=dev)
    plan_host = [torch.empty(64 << 20, dtype=torch.uint8, pin_memory=True) for _ in range(2)]
    plan_ev = [None, None]
    ws_dev = torch.empty(256 << 20, dtype=torch.uint8, device=dev)
    out = torch.empty((b.total_q, b.num_q_heads, b.head_dim),
                      dtype=torch.float32 if b.out_dtype == "f32" else torch.bfloat16, device=dev)
    ev = []
    ev_append = []
    # the step's new K/V rows, written into the pool ahead of its attention
    new_std = 1.0 / np.sqrt(b.head_dim) if WORKLOADS[name] != 1 else 1.0
    k_new_h, v_new_h = synth.make_new_kv(b, seed=args.seed + 7, std=new_std)
    new_dt = "f32" if b.kv_dtype == "f32" else "bf16"
    k_new = rt.to_device_array(k_new_h, new_dt, dev)
    v_new = rt.to_device_array(v_new_h, new_dt, dev)
    del k_new_h, v_new_h

    def step(i, timed):
        now = 1.0 + 0.02 * i
        formed = aug.aug_form_batch(recs, free_blocks, now, params)
        sel = np.sort(formed["ids"]).astype(np.int64)          # slot order of the selected requests
        q_len = np.zeros(b.num_reqs, np.int32)
        q_len[formed["ids"]] = formed["q_len"]
        assert np.array_equal(q_len[sel], b.q_len[sel]), "former must select the generated batch"
        assert len(sel) == b.num_reqs, "the synthetic batch is sized to fit one budget"
        q_start = np.zeros(len(sel) + 1, np.int32)
        q_start[1:] = np.cumsum(q_len[sel])
        info, plan = aug.aug_attn_plan(shape, q_start, b.ctx_len, b.bt_start, kv.num_pool_blocks,
                                       None, kv_split_tokens=args.kv_split, row_path=row_path,
                                       tile_path=tile_path)
        # double-buffered pinned staging: a buffer is rewritten only after the
        # copy that last read it has completed
        slot = i & 1
        if plan_ev[slot] is not None:
            plan_ev[slot].synchronize()
        host = plan_host[slot]
        host.numpy()[:plan.size] = plan
        # the library's copy kernel on the launch stream: it starts as soon
        # as the previous step's attention has finished
        aug.aug_plan_upload(host, plan_dev, plan.size, stream=stream.cuda_stream)
        plan_ev[slot] = torch.cuda.Event()
        plan_ev[slot].record(stream)
        e0, e1, a0 = TimingEvent(), TimingEvent(), TimingEvent()
        kc, vc, ksc, vsc = pools[i % len(pools)]
        a0.record(stream)
        aug.aug_kv_append(shape, info, plan_dev, k_new, v_new, kc, vc, ksc, vsc, bids, kv.num_pool_blocks,
                          stream=stream.cuda_stream)
        e0.record(stream)
        aug.aug_attn_mixed(shape, info, plan_dev, q, kc, vc, ksc, vsc,
                           bids, kv.num_pool_blocks, out, ws_dev, stream=stream.cuda_stream)
        e1.record(stream)
        if timed:
            ev.append((e0, e1))
            ev_append.append((a0, e0))
        return info

    if args.copy_probe_mib > 0:
        n = args.copy_probe_mib << 20
        src = torch.empty(n, dtype=torch.uint8, device=dev).fill_(1)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        log(f"copy probe: 3 copies of {n} bytes")
        del src, dst

    # everything allocated so far lives until the end: keep the collector
    # from rescanning it (a full pass over torch's objects stalls a step by
    # tens of milliseconds)
    gc.collect()
    gc.freeze()
    info = None
    for i in range(args.warmup):
        info = step(i, False)
    torch.cuda.synchronize()
    log(f"plan: {info.num_items} items ({info.num_prefill_items} tiles), {info.num_merge_groups} merge "
        f"groups, split {info.kv_split_tokens} keys")
    t_start = time.perf_counter()
    for i in range(args.steps):
        step(args.warmup + i, True)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t_start
    ms_per_step = 1e3 * elapsed / args.steps
    launch_ms = np.array([a.elapsed_time(c) for a, c in ev])
    attn_ms = float(launch_ms.mean())
    rows = b.total_q
    value = rows / (elapsed / args.steps)

    nbytes = algorithmic_bytes(b)
    flops = prefill_flops(b)
    achieved_gbs = nbytes / (attn_ms * 1e-3) / 1e9
    achieved_tfs = flops / (attn_ms * 1e-3) / 1e12
    traffic = measured_traffic(traffic_key(b.name, row_path, tile_path))
    # the matrix peak of the prefill work: bf16; with fp8 score products half
    # of the flops (Q K^T) at the fp8 peak and half (P V) at the bf16 one; with
    # both products in fp8 the fp8 peak
    mfma_peak = {2: 2.0 / (1.0 / MFMA_FP8_PEAK_TFS + 1.0 / MFMA_BF16_PEAK_TFS),
                 3: MFMA_FP8_PEAK_TFS}.get(tile_path, MFMA_BF16_PEAK_TFS)
    # the batch is bound by whichever roof its algorithmic work reaches first
    if flops / (mfma_peak * 1e12) > nbytes / (HBM_PEAK_GBS * 1e9):
        roof = {"bound": "mfma", "achieved": round(achieved_tfs, 1), "peak": round(mfma_peak, 1),
                "unit": "TFLOP/s", "frac": round(achieved_tfs / mfma_peak, 4),
                "traffic": traffic, "hbm_gbs": round(achieved_gbs, 1)}
        if tile_path in (2, 3):
            roof["peak_note"] = ("Q K^T at the fp8 MFMA peak, P V at the bf16 one (half of the flops each)"
                                 if tile_path == 2 else "both products at the fp8 MFMA peak")
            roof["frac_of_bf16_peak"] = round(achieved_tfs / MFMA_BF16_PEAK_TFS, 4)
    else:
        roof = {"bound": "hbm", "achieved": round(achieved_gbs, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": round(achieved_gbs / HBM_PEAK_GBS, 4), "traffic": traffic}
        if flops > 0:
            roof["prefill_mfma_tflops"] = round(achieved_tfs, 2)
    # decode rows' flops (4 D H_q per key): on the vector ALUs for up to four
    # heads per KV head, on MFMA for eight; reported beside the HBM figure
    dec_flops = 4.0 * b.head_dim * b.num_q_heads * float(b.ctx_len[b.q_len == 1].sum())
    if dec_flops > 0:
        roof["decode_tflops"] = round(dec_flops / (attn_ms * 1e-3) / 1e12, 2)
        roof["decode_tflops_frac_of_fp32_valu"] = round(dec_flops / (attn_ms * 1e-3) / 157.3e12, 4)
    roof.update({"kernel": "aug_attn_mixed launches (attention + split-K merge)",
                 "algorithmic_bytes_per_launch": int(nbytes), "prefill_flops_per_launch": int(flops),
                 "launch_ms": round(attn_ms, 4), "launch_ms_median": round(float(np.median(launch_ms)), 4),
                 "launch_ms_p10": round(float(np.percentile(launch_ms, 10)), 4),
                 "launch_ms_p90": round(float(np.percentile(launch_ms, 90)), 4)})

    result = {
        "metric": "mixed-batch attn query-tokens/s + % peak HBM GB/s (decode) / % MFMA (prefill)",
        "value": round(value, 1), "unit": "query-tokens/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(ms_per_step, 4), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "bf16" if b.kv_dtype == "bf16" else "bf16-q/fp8e4m3-kv" if b.kv_dtype == "fp8" else "f32",
        "data": "synthetic",
        "config": {"workload": b.name, "requests": b.num_reqs, "query_rows": rows,
                   "context_tokens": int(b.ctx_len.sum()), "q_heads": b.num_q_heads,
                   "kv_heads": b.num_kv_heads, "head_dim": b.head_dim, "block_size": 16,
                   "kv_split_tokens": int(info.kv_split_tokens), "seed": args.seed, "pool_copies": n_copies,
                   "row_path": {1: "vector ALU", 2: "MFMA"}[int(info.row_path)],
                   "tile_path": {1: "bf16", 2: "fp8 scores (opt-in)",
                                 3: "fp8 scores and values (opt-in)"}[int(info.tile_path)]},
        "roofline": roof,
    }
    app_ms = np.array([a.elapsed_time(c) for a, c in ev_append])
    app_bytes = append_bytes(b, info)
    result["kv_append"] = {
        "kernel": "aug_kv_append (the step's new K/V rows into the pool, before attention)",
        "algorithmic_bytes_per_launch": int(app_bytes), "launch_ms": round(float(app_ms.mean()), 4),
        "launch_ms_median": round(float(np.median(app_ms)), 4),
        "gbs": round(app_bytes / (float(app_ms.mean()) * 1e-3) / 1e9, 1),
        "frac_hbm": round(app_bytes / (float(app_ms.mean()) * 1e-3) / 1e9 / HBM_PEAK_GBS, 4)}
    if full and getattr(b, "park", None) is not None and len(b.park.resume_blocks) and not args.no_park_resume:
        result["park_resume"] = park_resume_rates(b, kv, log)
    if full and args.layers > 0:
        result["layers"] = time_layers(args.layers, shape, info, plan_dev, k_new, v_new, q, pools, bids,
                                       kv.num_pool_blocks, out, ws_dev, stream, log)
    if full and not args.no_cpu_baseline:
        log("timing the CPU oracle on a sample")
        result["cpu_baseline"] = cpu_baseline(b, args.cpu_budget_s)
    gc.unfreeze()
    return result



def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="mixed-8b", choices=sorted(WORKLOADS))
    ap.add_argument("--also", default=None,
                    help="comma-separated workloads timed after the main one in the same run, each reported "
                         "with its own roofline under 'workloads' (default for mixed-8b: " +
                         ",".join(DEFAULT_ALSO) + "; 'none' for no others)")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--tile-path", choices=("auto", "fp8qk", "fp8"), default="auto",
                    help="fp8qk: the prefill tiles' score products on fp8 MFMAs; fp8: both of their products "
                         "(opt-in arithmetic)")
    ap.add_argument("--row-path", choices=("auto", "valu", "mfma"), default="auto",
                    help="where the main workload's row items run: the planner's choice (MFMA for eight query "
                         "heads per KV head), the vector ALUs, or MFMA (eight or four heads per KV head)")
    ap.add_argument("--kv-split", type=int, default=0, help="keys per decode work item (0: planner's choice)")
    ap.add_argument("--pool-copies", type=int, default=0,
                    help="copies of the KV pool used in turn (0: enough for 1 GiB of KV reads between "
                         "two uses of one copy, at most 8)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-park-resume", action="store_true",
                    help="skip the separate park/resume timing of workloads that move paused requests")
    ap.add_argument("--cpu-budget-s", type=float, default=15.0)
    ap.add_argument("--sweep-layers", type=int, default=8,
                    help="budget sweep: layers per replayed batch for the per-layer figures")
    ap.add_argument("--sweep-batches", type=int, default=200,
                    help="budget-sweep-fp8: formed batches replayed per budget")
    ap.add_argument("--layers", type=int, default=8,
                    help="after the steps, time this many layers of the planned batch (each an append and "
                         "an attention call on its own pool copy) launched one by one and as one HIP graph "
                         "(0: skip)")
    ap.add_argument("--copy-probe-mib", type=int, default=0,
                    help="before timing, copy a buffer of this many MiB a few times (a kernel of known "
                         "traffic for calibrating hardware byte counters)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(json.dumps({"error": "this benchmark runs on exactly one GPU; the step needs no "
                                   "collectives and multi-GPU runs are not part of it",
                          "n_gpus": args.gpus}))
        sys.exit(2)

    import torch

    def log(msg):
        print(f"[bench] {msg}", file=sys.stderr, flush=True)

    torch.cuda.set_device(0)
    if args.workload == "budget-sweep-fp8":
        budget_sweep(args, log)
        return
    result = run_workload(args.workload, args, log, full=True,
                          row_path={"auto": 0, "valu": 1, "mfma": 2}[args.row_path],
                          tile_path={"auto": 0, "fp8qk": 2, "fp8": 3}[args.tile_path])
    if args.also is None:
        also = list(DEFAULT_ALSO) if args.workload == "mixed-8b" else []
    else:
        also = [w for w in args.also.split(",") if w and w != "none"]
    if also:
        result["workloads"] = {}
    for entry in also:
        name, _, path = entry.partition("@")
        if name not in WORKLOADS or name == "budget-sweep-fp8" or entry == args.workload or path not in PATHS:
            raise SystemExit(f"--also: {entry} is not a single-batch workload other than the main one")
        gc.collect()
        torch.cuda.empty_cache()
        sub = run_workload(name, args, log, full=False, row_path=PATHS[path][0], tile_path=PATHS[path][1])
        keep = ("value", "unit", "steps", "warmup", "ms_per_step", "dtype", "config", "roofline", "kv_append")
        key = sub["config"]["workload"] + PATH_NOTES[path]
        result["workloads"][key] = {k: sub[k] for k in keep}
        log(f"{name}: {sub['value']:.0f} query-tokens/s, {sub['roofline']['unit']} frac "
            f"{sub['roofline']['frac']}")
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
