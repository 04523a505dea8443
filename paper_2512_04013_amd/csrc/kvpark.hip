// Park (swap-out) and resume (swap-in) of KV blocks for requests paused on
// external calls (Swap policy of the paper's context-handling policies,
// Appendix B; the swapped queue of Algorithm 1, step (2)).
//
// One (block, all KV heads) of the pool is contiguous: K[block] is
// num_kv_heads * 16 * head_dim elements, likewise V[block]. A parked record
// is K[block] | V[block] | k_scale[block] | v_scale[block] (scales for fp8
// caches only). Park gathers the listed blocks' records into a contiguous
// device staging buffer with one kernel (16-byte loads and stores, one
// workgroup per block) and drains it to pinned host memory with one
// asynchronous copy (the DMA engine), chunk by chunk when staging is smaller
// than the whole image; resume runs the same two steps backwards and
// scatters into the (new) destination blocks. The bytes are moved, never
// reinterpreted, so the round trip is exact.

#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdint>

#include "aug.h"
#include "checks.h"
#include "status.h"

namespace {

constexpr int kThreads = 256;

struct RecordGeom {
  int64_t kv_bytes;     // bytes of K[block] (and of V[block])
  int64_t scale_bytes;  // bytes of k_scale[block] (and of v_scale[block]); 0 unless fp8
  int64_t rec_bytes;
};

RecordGeom geom(const aug_attn_shape& s) {
  const int64_t elem = s.kv_dtype == AUG_F32 ? 4 : s.kv_dtype == AUG_BF16 ? 2 : 1;
  RecordGeom g{};
  g.kv_bytes = static_cast<int64_t>(s.num_kv_heads) * s.block_size * s.head_dim * elem;
  g.scale_bytes = s.kv_dtype == AUG_FP8_E4M3FN ? static_cast<int64_t>(s.num_kv_heads) * 4 : 0;
  g.rec_bytes = 2 * g.kv_bytes + 2 * g.scale_bytes;
  return g;
}

// Copy `bytes` (a multiple of 4) between two buffers with the widest aligned
// vector width, cooperatively across the workgroup.
__device__ __forceinline__ void wg_copy(char* dst, const char* src, int64_t bytes) {
  const bool a16 = ((reinterpret_cast<uintptr_t>(dst) | reinterpret_cast<uintptr_t>(src) | bytes) & 15) == 0;
  if (a16) {
    const int64_t n = bytes / 16;
    const uint4* s = reinterpret_cast<const uint4*>(src);
    uint4* d = reinterpret_cast<uint4*>(dst);
    for (int64_t i = threadIdx.x; i < n; i += kThreads) d[i] = s[i];
  } else {
    const int64_t n = bytes / 4;
    const uint32_t* s = reinterpret_cast<const uint32_t*>(src);
    uint32_t* d = reinterpret_cast<uint32_t*>(dst);
    for (int64_t i = threadIdx.x; i < n; i += kThreads) d[i] = s[i];
  }
}

// Zero `bytes` (a multiple of 4) cooperatively across the workgroup.
__device__ __forceinline__ void wg_zero(char* dst, int64_t bytes) {
  uint32_t* d = reinterpret_cast<uint32_t*>(dst);
  for (int64_t i = threadIdx.x; i < bytes / 4; i += kThreads) d[i] = 0u;
}

__global__ __launch_bounds__(kThreads) void gather_kernel(
    const char* k_cache, const char* v_cache, const char* k_scale, const char* v_scale,
    const int32_t* ids, int32_t first, int32_t num_pool_blocks, RecordGeom g, char* staging) {
  const int32_t bid = ids[first + blockIdx.x];
  char* rec = staging + static_cast<int64_t>(blockIdx.x) * g.rec_bytes;
  if (static_cast<uint32_t>(bid) >= static_cast<uint32_t>(num_pool_blocks)) {
    // never dereferenced; the record reads as zero bytes rather than stale staging
    wg_zero(rec, g.rec_bytes);
    return;
  }
  wg_copy(rec, k_cache + static_cast<int64_t>(bid) * g.kv_bytes, g.kv_bytes);
  wg_copy(rec + g.kv_bytes, v_cache + static_cast<int64_t>(bid) * g.kv_bytes, g.kv_bytes);
  if (g.scale_bytes) {
    wg_copy(rec + 2 * g.kv_bytes, k_scale + static_cast<int64_t>(bid) * g.scale_bytes, g.scale_bytes);
    wg_copy(rec + 2 * g.kv_bytes + g.scale_bytes, v_scale + static_cast<int64_t>(bid) * g.scale_bytes,
            g.scale_bytes);
  }
}

__global__ __launch_bounds__(kThreads) void scatter_kernel(
    char* k_cache, char* v_cache, char* k_scale, char* v_scale, const int32_t* ids, int32_t first,
    int32_t num_pool_blocks, RecordGeom g, const char* staging) {
  const int32_t bid = ids[first + blockIdx.x];
  if (static_cast<uint32_t>(bid) >= static_cast<uint32_t>(num_pool_blocks)) return;
  const char* rec = staging + static_cast<int64_t>(blockIdx.x) * g.rec_bytes;
  wg_copy(k_cache + static_cast<int64_t>(bid) * g.kv_bytes, rec, g.kv_bytes);
  wg_copy(v_cache + static_cast<int64_t>(bid) * g.kv_bytes, rec + g.kv_bytes, g.kv_bytes);
  if (g.scale_bytes) {
    wg_copy(k_scale + static_cast<int64_t>(bid) * g.scale_bytes, rec + 2 * g.kv_bytes, g.scale_bytes);
    wg_copy(v_scale + static_cast<int64_t>(bid) * g.scale_bytes, rec + 2 * g.kv_bytes + g.scale_bytes,
            g.scale_bytes);
  }
}

aug_status check_common(const char* who, const aug_attn_shape* s, const void* k, const void* v,
                        const void* ks, const void* vs, const int32_t* ids_dev,
                        const int32_t* ids_host, int32_t n_blocks, int32_t num_pool_blocks,
                        const void* host, size_t host_bytes, const void* staging,
                        size_t staging_bytes, RecordGeom* g) {
  if (aug_status st = aug::check_shape(s, who); st != AUG_OK) return st;
  if (n_blocks < 0) return aug::fail(AUG_ERR_INVALID, "%s: n_blocks %d < 0", who, n_blocks);
  if (num_pool_blocks < 1) return aug::fail(AUG_ERR_INVALID, "%s: empty pool", who);
  *g = geom(*s);
  if (n_blocks == 0) return AUG_OK;
  if (!k || !v || !ids_dev || !host || !staging)
    return aug::fail(AUG_ERR_INVALID, "%s: NULL pointer", who);
  if (s->kv_dtype == AUG_FP8_E4M3FN && (!ks || !vs))
    return aug::fail(AUG_ERR_INVALID, "%s: fp8 KV needs scale arrays", who);
  if (host_bytes < static_cast<size_t>(g->rec_bytes) * static_cast<size_t>(n_blocks))
    return aug::fail(AUG_ERR_NO_SPACE, "%s: host buffer %zu < %lld bytes", who, host_bytes,
                     (long long)(g->rec_bytes * n_blocks));
  if (staging_bytes < static_cast<size_t>(g->rec_bytes))
    return aug::fail(AUG_ERR_NO_SPACE, "%s: staging %zu < one record (%lld bytes)", who,
                     staging_bytes, (long long)g->rec_bytes);
  if (!ids_host) return aug::fail(AUG_ERR_INVALID, "%s: block_ids_host is required", who);
  {
    for (int32_t i = 0; i < n_blocks; ++i)
      if (ids_host[i] < 0 || ids_host[i] >= num_pool_blocks)
        return aug::fail(AUG_ERR_INVALID, "%s: block id %d (entry %d) outside a pool of %d", who,
                         ids_host[i], i, num_pool_blocks);
  }
  return AUG_OK;
}

}  // namespace

extern "C" size_t aug_kv_record_bytes(const aug_attn_shape* s) {
  if (!s || aug::check_shape(s, "aug_kv_record_bytes") != AUG_OK) return 0;
  return static_cast<size_t>(geom(*s).rec_bytes);
}

extern "C" aug_status aug_kv_park(const aug_attn_shape* s, const void* k_cache, const void* v_cache,
                                  const float* k_scale, const float* v_scale,
                                  const int32_t* ids_dev, const int32_t* ids_host, int32_t n_blocks,
                                  int32_t num_pool_blocks, void* host_dst, size_t host_bytes,
                                  void* staging, size_t staging_bytes, void* stream) {
  RecordGeom g{};
  if (aug_status st = check_common("aug_kv_park", s, k_cache, v_cache, k_scale, v_scale, ids_dev,
                                   ids_host, n_blocks, num_pool_blocks, host_dst, host_bytes,
                                   staging, staging_bytes, &g);
      st != AUG_OK || n_blocks == 0)
    return st;
  hipStream_t st = static_cast<hipStream_t>(stream);
  const int64_t per_chunk = static_cast<int64_t>(staging_bytes) / g.rec_bytes;
  for (int64_t first = 0; first < n_blocks; first += per_chunk) {
    const int64_t cnt = std::min<int64_t>(per_chunk, n_blocks - first);
    hipLaunchKernelGGL(gather_kernel, dim3(static_cast<uint32_t>(cnt)), dim3(kThreads), 0, st,
                       static_cast<const char*>(k_cache), static_cast<const char*>(v_cache),
                       reinterpret_cast<const char*>(k_scale), reinterpret_cast<const char*>(v_scale),
                       ids_dev, static_cast<int32_t>(first), num_pool_blocks, g,
                       static_cast<char*>(staging));
    if (hipError_t e = hipGetLastError(); e != hipSuccess)
      return aug::fail(AUG_ERR_HIP, "aug_kv_park: gather launch: %s", hipGetErrorString(e));
    if (hipError_t e = hipMemcpyAsync(static_cast<char*>(host_dst) + first * g.rec_bytes, staging,
                                      static_cast<size_t>(cnt * g.rec_bytes), hipMemcpyDeviceToHost, st);
        e != hipSuccess)
      return aug::fail(AUG_ERR_HIP, "aug_kv_park: copy to host: %s", hipGetErrorString(e));
  }
  return AUG_OK;
}

extern "C" aug_status aug_kv_resume(const aug_attn_shape* s, void* k_cache, void* v_cache,
                                    float* k_scale, float* v_scale, const int32_t* ids_dev,
                                    const int32_t* ids_host, int32_t n_blocks,
                                    int32_t num_pool_blocks, const void* host_src,
                                    size_t host_bytes, void* staging, size_t staging_bytes,
                                    void* stream) {
  RecordGeom g{};
  if (aug_status st = check_common("aug_kv_resume", s, k_cache, v_cache, k_scale, v_scale, ids_dev,
                                   ids_host, n_blocks, num_pool_blocks, host_src, host_bytes,
                                   staging, staging_bytes, &g);
      st != AUG_OK || n_blocks == 0)
    return st;
  hipStream_t st = static_cast<hipStream_t>(stream);
  const int64_t per_chunk = static_cast<int64_t>(staging_bytes) / g.rec_bytes;
  for (int64_t first = 0; first < n_blocks; first += per_chunk) {
    const int64_t cnt = std::min<int64_t>(per_chunk, n_blocks - first);
    if (hipError_t e = hipMemcpyAsync(staging, static_cast<const char*>(host_src) + first * g.rec_bytes,
                                      static_cast<size_t>(cnt * g.rec_bytes), hipMemcpyHostToDevice, st);
        e != hipSuccess)
      return aug::fail(AUG_ERR_HIP, "aug_kv_resume: copy from host: %s", hipGetErrorString(e));
    hipLaunchKernelGGL(scatter_kernel, dim3(static_cast<uint32_t>(cnt)), dim3(kThreads), 0, st,
                       static_cast<char*>(k_cache), static_cast<char*>(v_cache),
                       reinterpret_cast<char*>(k_scale), reinterpret_cast<char*>(v_scale), ids_dev,
                       static_cast<int32_t>(first), num_pool_blocks, g,
                       static_cast<const char*>(staging));
    if (hipError_t e = hipGetLastError(); e != hipSuccess)
      return aug::fail(AUG_ERR_HIP, "aug_kv_resume: scatter launch: %s", hipGetErrorString(e));
  }
  return AUG_OK;
}
