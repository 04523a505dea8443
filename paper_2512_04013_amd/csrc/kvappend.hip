// Append of a step's new K/V rows to the paged cache: every query row of a
// formed batch is a token that the step's forward pass produces (Algorithm 1,
// step (5)), and its K and V go into the request's blocks before attention
// reads them.
//
// The work list is the plan image's append section: one item per block that
// receives tokens (first row, row count, first slot, block-table index). One
// wave handles one (item, KV head, K or V): it streams the item's rows from
// the [rows][H_kv][D] input with 16-byte lane loads and writes them to
// consecutive slots of the block. For fp8 caches the wave also reduces the
// rows' largest magnitude, derives the block's new scale from it and the old
// one, re-encodes the block's earlier codes when the scale grows, and encodes
// the new rows (round to nearest even, saturating at +-448).
//
// HBM-bound and tiny next to attention: bytes per new token and KV head are
// the input row (D * 2 or 4) plus the cache row (D * 1, 2 or 4), for K and V.

#include <hip/hip_runtime.h>

#include <cstdint>

#include "aug.h"
#include "checks.h"
#include "plan_format.h"
#include "status.h"


namespace {

using aug::AppendItem;
using aug::kBlock;

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / 64;

struct AppendArgs {
  const AppendItem* items;
  int32_t num_items;
  int32_t hkv;
  const char* k_new;
  const char* v_new;
  char* k_cache;
  char* v_cache;
  float* k_scale;
  float* v_scale;
  const int32_t* block_ids;
  int32_t num_pool_blocks;
};

// E4M3FN code -> float, exact: exponent field 0 holds multiples of 2^-9,
// otherwise (1 + m/8) * 2^(e - 7).
__device__ __forceinline__ float fp8_value(uint32_t c) {
  const uint32_t e = (c >> 3) & 15u, m = c & 7u;
  const float mag = e == 0 ? static_cast<float>(m) * 0x1p-9f
                           : __uint_as_float(((e + 120u) << 23) | (m << 20));
  return (c & 0x80u) ? -mag : mag;
}

// float -> E4M3FN code: round to nearest, ties to an even mantissa, every
// magnitude from 448 up saturates to +-448, the sign of zero is kept.
__device__ __forceinline__ uint32_t fp8_code(float y) {
  const uint32_t sign = (__float_as_uint(y) >> 24) & 0x80u;
  const float a = fabsf(y);
  uint32_t code;
  if (!(a < 448.f)) {
    code = 0x7Eu;
  } else if (a < 0x1p-6f) {
    code = static_cast<uint32_t>(__builtin_rintf(a * 512.f));   // subnormal steps of 2^-9 (8 = 2^-6)
  } else {
    const uint32_t b = __float_as_uint(a);
    const uint32_t e = (b >> 23) - 120u;                         // E4M3 exponent field, 1..15
    const uint32_t m = b & 0x7FFFFFu;
    const uint32_t rest = m & 0xFFFFFu;
    uint32_t r = m >> 20;
    r += (rest > 0x80000u) | ((rest == 0x80000u) & (r & 1u));
    code = min((e << 3) + r, 0x7Eu);                             // r == 8 carries into the exponent
  }
  return code | sign;
}

// An append item read with one 16-byte load (the index is the same for the
// whole wave, so it goes through the scalar cache).
__device__ __forceinline__ AppendItem load_item(const AppendItem* items, int64_t idx) {
  static_assert(sizeof(AppendItem) == 16, "one 16-byte load");
  const uint4 raw = *reinterpret_cast<const uint4*>(items + idx);
  AppendItem it;
  __builtin_memcpy(&it, &raw, sizeof(it));
  return it;
}

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }

// f32 and bf16 caches: the rows are stored as they come.
template <int EB, int D>
__global__ __launch_bounds__(kThreads) void append_copy_kernel(AppendArgs a) {
  constexpr int LPR = D * EB / 16;     // lanes per row (16 bytes each)
  constexpr int RPP = 64 / LPR;        // rows per pass
  const int lane = threadIdx.x & 63;
  const int64_t unit = static_cast<int64_t>(blockIdx.x) * kWaves + __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  if (unit >= static_cast<int64_t>(a.num_items) * a.hkv * 2) return;
  const AppendItem it = load_item(a.items, unit / (2 * a.hkv));
  const int kvh = static_cast<int>((unit >> 1) % a.hkv);
  const bool is_v = unit & 1;
  const int32_t bid = a.block_ids[it.bt_index];
  if (static_cast<uint32_t>(bid) >= static_cast<uint32_t>(a.num_pool_blocks)) return;
  const char* src = is_v ? a.v_new : a.k_new;
  char* dst = is_v ? a.v_cache : a.k_cache;
  const int64_t row_bytes = static_cast<int64_t>(D) * EB;
  char* blk = dst + ((static_cast<int64_t>(bid) * a.hkv + kvh) * kBlock + it.slot0) * row_bytes;
  for (int r = lane / LPR; r < it.n_rows; r += RPP) {
    const int64_t in = ((static_cast<int64_t>(it.q_row0) + r) * a.hkv + kvh) * row_bytes;
    const int col = (lane % LPR) * 16;
    *reinterpret_cast<uint4*>(blk + r * row_bytes + col) = *reinterpret_cast<const uint4*>(src + in + col);
  }
}

// fp8 caches (head_dim 128): bf16 rows in, codes and the block scale out.
__global__ __launch_bounds__(kThreads) void append_fp8_kernel(AppendArgs a) {
  constexpr int D = 128;
  constexpr int LPR = D / 8;           // lanes per row: 8 bf16 in, 8 codes out
  constexpr int RPP = 64 / LPR;        // 4 rows per pass
  constexpr int PASSES = kBlock / RPP;
  const int lane = threadIdx.x & 63;
  const int64_t unit = static_cast<int64_t>(blockIdx.x) * kWaves + __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  if (unit >= static_cast<int64_t>(a.num_items) * a.hkv * 2) return;
  const AppendItem it = load_item(a.items, unit / (2 * a.hkv));
  const int kvh = static_cast<int>((unit >> 1) % a.hkv);
  const bool is_v = unit & 1;
  // the block id and the new rows are fetched together, the block's current
  // scale as soon as the id is known: no load waits on another it does not need
  const int32_t bid = a.block_ids[it.bt_index];
  const bool bid_ok = static_cast<uint32_t>(bid) < static_cast<uint32_t>(a.num_pool_blocks);
  const uint16_t* src = reinterpret_cast<const uint16_t*>(is_v ? a.v_new : a.k_new);
  uint8_t* blk = reinterpret_cast<uint8_t*>(is_v ? a.v_cache : a.k_cache) +
                 (static_cast<int64_t>(bid) * a.hkv + kvh) * kBlock * D;
  float* scale = (is_v ? a.v_scale : a.k_scale) + static_cast<int64_t>(bid) * a.hkv + kvh;
  const int col = (lane % LPR) * 8;
  const int r0 = lane / LPR;

  float x[PASSES][8];
  float amax = 0.f;
#pragma unroll
  for (int p = 0; p < PASSES; ++p) {
    const int r = r0 + p * RPP;
    uint4 w{0u, 0u, 0u, 0u};
    if (r < it.n_rows)
      w = *reinterpret_cast<const uint4*>(src + ((static_cast<int64_t>(it.q_row0) + r) * a.hkv + kvh) * D + col);
    x[p][0] = bf16_lo(w.x); x[p][1] = bf16_hi(w.x);
    x[p][2] = bf16_lo(w.y); x[p][3] = bf16_hi(w.y);
    x[p][4] = bf16_lo(w.z); x[p][5] = bf16_hi(w.z);
    x[p][6] = bf16_lo(w.w); x[p][7] = bf16_hi(w.w);
#pragma unroll
    for (int e = 0; e < 8; ++e) amax = fmaxf(amax, fabsf(x[p][e]));
  }
  const float s_old = bid_ok && it.slot0 > 0 ? *scale : 0.f;
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) amax = fmaxf(amax, __shfl_xor(amax, off, 64));
  if (!bid_ok) return;

  const float need = amax / 448.f;
  float s = need;
  if (it.slot0 > 0) {
    if (need > s_old) {
      // the scale grows: re-encode the block's earlier tokens
      for (int r = r0; r < it.slot0; r += RPP) {
        uint2* q = reinterpret_cast<uint2*>(blk + r * D + col);
        const uint2 c = *q;
        uint32_t lo = 0, hi = 0;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float v0 = (fp8_value((c.x >> (8 * e)) & 0xFFu) * s_old) / need;
          const float v1 = (fp8_value((c.y >> (8 * e)) & 0xFFu) * s_old) / need;
          lo |= fp8_code(v0) << (8 * e);
          hi |= fp8_code(v1) << (8 * e);
        }
        *q = uint2{lo, hi};
      }
    } else {
      s = s_old;
    }
  }
#pragma unroll
  for (int p = 0; p < PASSES; ++p) {
    const int r = r0 + p * RPP;
    if (r >= it.n_rows) break;
    uint32_t lo = 0, hi = 0;
    if (s != 0.f) {
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        lo |= fp8_code(x[p][e] / s) << (8 * e);
        hi |= fp8_code(x[p][4 + e] / s) << (8 * e);
      }
    }
    *reinterpret_cast<uint2*>(blk + (it.slot0 + r) * D + col) = uint2{lo, hi};
  }
  if (lane == 0) *scale = s;
}

}  // namespace

extern "C" aug_status aug_kv_append(const aug_attn_shape* s, const aug_attn_plan_info* info,
                                    const void* plan_dev, const void* k_new, const void* v_new,
                                    void* k_cache, void* v_cache, float* k_scale, float* v_scale,
                                    const int32_t* block_ids, int32_t num_pool_blocks, void* stream) {
  const char* who = "aug_kv_append";
  if (aug_status st = aug::check_shape(s, who); st != AUG_OK) return st;
  if (aug_status st = aug::check_plan_info(info, s, who); st != AUG_OK) return st;
  const int64_t append_off = aug::append_offset(info->num_items, info->num_merge_groups);
  if (info->num_append_items == 0) return AUG_OK;
  if (!plan_dev || !k_new || !v_new || !k_cache || !v_cache || !block_ids)
    return aug::fail(AUG_ERR_INVALID, "%s: NULL device pointer", who);
  const bool fp8 = s->kv_dtype == AUG_FP8_E4M3FN;
  if (fp8 && (!k_scale || !v_scale)) return aug::fail(AUG_ERR_INVALID, "%s: fp8 cache without scales", who);
  if (num_pool_blocks < 1) return aug::fail(AUG_ERR_INVALID, "%s: empty pool", who);

  AppendArgs a{};
  a.items = reinterpret_cast<const AppendItem*>(static_cast<const char*>(plan_dev) + append_off);
  a.num_items = info->num_append_items;
  a.hkv = s->num_kv_heads;
  a.k_new = static_cast<const char*>(k_new);
  a.v_new = static_cast<const char*>(v_new);
  a.k_cache = static_cast<char*>(k_cache);
  a.v_cache = static_cast<char*>(v_cache);
  a.k_scale = k_scale;
  a.v_scale = v_scale;
  a.block_ids = block_ids;
  a.num_pool_blocks = num_pool_blocks;
  const int64_t units = static_cast<int64_t>(a.num_items) * a.hkv * 2;
  const int64_t grid = (units + kWaves - 1) / kWaves;
  if (grid > INT32_MAX) return aug::fail(AUG_ERR_UNSUPPORTED, "%s: %lld units", who, (long long)units);
  hipStream_t st = static_cast<hipStream_t>(stream);
  if (fp8) {
    hipLaunchKernelGGL(append_fp8_kernel, dim3(grid), dim3(kThreads), 0, st, a);
  } else if (s->kv_dtype == AUG_BF16) {
    if (s->head_dim == 64) hipLaunchKernelGGL((append_copy_kernel<2, 64>), dim3(grid), dim3(kThreads), 0, st, a);
    else hipLaunchKernelGGL((append_copy_kernel<2, 128>), dim3(grid), dim3(kThreads), 0, st, a);
  } else {
    if (s->head_dim == 64) hipLaunchKernelGGL((append_copy_kernel<4, 64>), dim3(grid), dim3(kThreads), 0, st, a);
    else hipLaunchKernelGGL((append_copy_kernel<4, 128>), dim3(grid), dim3(kThreads), 0, st, a);
  }
  if (hipError_t e = hipGetLastError(); e != hipSuccess)
    return aug::fail(AUG_ERR_HIP, "%s: launch failed: %s", who, hipGetErrorString(e));
  return AUG_OK;
}
