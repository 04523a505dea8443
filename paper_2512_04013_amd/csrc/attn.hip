// Mixed-batch paged attention for gfx950 (MI355X).
//
// One launch runs every work item of a plan (plan_format.h):
//
//  * Row items (decodes; prefill rows of dtype sets without a tile path): one
//    query row and the G query heads that share one KV head, against a span of
//    that request's keys. A 256-thread workgroup streams the span's 16-token
//    blocks, each wave its own blocks (wave w takes blocks w, w+4, ...). A
//    block of one KV head is 16 contiguous rows of head_dim elements, so a
//    wave reads it with fully coalesced 16-byte (8-byte for fp8) lane loads:
//    LPT lanes cover one token row, 64/LPT tokens per load instruction. Scores
//    are reduced across the LPT lanes of a token with DPP row operations, the
//    softmax is online in the log2 domain, and every lane group keeps its own
//    running (max, sum, output) state; the states are merged across lane
//    groups with cross-lane shuffles and across waves through LDS. Each KV byte
//    is read once for all G heads (grouped-query sharing). Arithmetic runs on
//    the vector ALUs in fp32, except for groups of eight (or, when asked for,
//    four) query heads (bf16 or fp8 KV, head_dim 128), whose products run on
//    16x16 bf16 MFMAs with the same item, split and merge structure
//    (row_item_mfma).
//  * Tile items (bf16 chunked prefill): 128 query rows (positions x group
//    heads) of one chunk, causal against keys 0 .. last row's position. K and V
//    are staged through LDS 64 keys at a time (V read back through transposing
//    LDS loads), and
//    both products run on bf16 MFMA 32x32x16 with fp32 accumulation:
//    S^T = K Q^T puts one query row per lane column, so the row max/sum are
//    lane-local plus one exchange between the two lane halves, and
//    O^T = V^T P^T takes P straight from the S^T accumulators.
//
// Keys past a request's context (tail of its last block) and blocks it does
// not list never reach the arithmetic: their loads are skipped (zero-filled)
// and their scores masked, so NaN or garbage in unused slots cannot leak.
// Block ids outside the pool are treated the same way (never dereferenced).
//
// Split-K: an item whose keys were split writes an unnormalised partial
// (o, m, l) per row to the workspace. A decode row's span then counts itself
// done on its group's counter in the plan image, and the workgroup that
// finishes the row's last span merges its partials by log-sum-exp (and
// resets the counter) in the same launch. Split prefill tiles, whose rows
// would make one workgroup merge many rows serially, are merged by a second
// launch, one workgroup per (row, KV head).

#include <hip/hip_runtime.h>

#include <cstdint>
#include <mutex>
#include <type_traits>

#include "aug.h"
#include "checks.h"
#include "plan_format.h"
#include "status.h"

namespace {

using aug::kBlock;
using aug::MergeGroup;
using aug::WorkItem;

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef int v8i_t __attribute__((ext_vector_type(8)));   // 32 fp8 codes: one 32x32x64 MFMA operand

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kNegBig = -1.0e30f;   // finite "minus infinity" for running maxima
// A running maximum is only moved (and the running sums rescaled) when a new
// score exceeds it by more than this many powers of two; until then
// probabilities are taken against the stale maximum and stay below 2^8, which
// fp32 sums and bf16 probabilities carry without loss. Numerator and
// denominator always share one reference, so the result is unchanged.
constexpr float kRescaleSlack = 8.0f;
constexpr int kThreads = 256;


enum : int { KV_F32 = 0, KV_BF16 = 1, KV_FP8 = 2 };

struct AttnArgs {
  const WorkItem* items;
  const void* q;
  const void* k_cache;
  const void* v_cache;
  const float* k_scale;
  const float* v_scale;
  const int32_t* block_ids;
  void* out;
  float* partials;
  const MergeGroup* groups;   // split groups of the plan
  int32_t* counters;          // per group: spans finished in this launch (zero between launches)
  int32_t num_pool_blocks;
  int32_t hq;
  int32_t hkv;
  float scale_log2;    // softmax_scale * log2(e)
};

// ---------------------------------------------------------------------------
// small helpers
// ---------------------------------------------------------------------------

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }

__device__ __forceinline__ uint32_t f32_to_bf16_bits(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);   // round to nearest even (inputs are finite)
  return u >> 16;
}

typedef __bf16 bf16x2v_t __attribute__((ext_vector_type(2)));

__device__ __forceinline__ bf16x8_t as_bf16x8(uint4 v) { return __builtin_bit_cast(bf16x8_t, v); }
constexpr uint32_t kBf16PairOne = 0x3F803F80u;   // (1.0, 1.0) as packed bf16

// two floats -> packed bf16 pair, round to nearest even (v_cvt_pk_bf16_f32)
__device__ __forceinline__ uint32_t pack_bf16(float lo, float hi) {
  const bf16x2v_t v = {static_cast<__bf16>(lo), static_cast<__bf16>(hi)};
  return __builtin_bit_cast(uint32_t, v);
}

// OCP E4M3FN byte pair (bytes 0-1, or 2-3 with HI) -> exact bf16 pair
template <bool HI>
__device__ __forceinline__ uint32_t fp8x2_to_bf16x2(uint32_t w) {
  return __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(w, 1.0f, HI));
}

template <int CTRL>
__device__ __forceinline__ float dpp(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xF, 0xF, true));
}

// Sum over aligned groups of LANES lanes (4, 8, 16 or 32); every lane of a
// group receives the group's sum.
template <int LANES>
__device__ __forceinline__ float group_sum(float v) {
  v += dpp<0xB1>(v);                  // quad_perm [1,0,3,2]: lane ^ 1
  v += dpp<0x4E>(v);                  // quad_perm [2,3,0,1]: lane ^ 2
  if constexpr (LANES >= 8) v += dpp<0x141>(v);   // row_half_mirror: pairs quads of 8
  if constexpr (LANES >= 16) v += dpp<0x140>(v);  // row_mirror: pairs halves of 16
  if constexpr (LANES >= 32) v += __shfl_xor(v, 16);
  return v;
}

// ---------------------------------------------------------------------------
// KV element formats for the row path
// ---------------------------------------------------------------------------

template <int KVT> struct KvFmt;
template <> struct KvFmt<KV_F32> {
  static constexpr int VEC = 4;       // elements per lane load (16 bytes)
  using raw_t = uint4;
  __device__ static void to_f32(const raw_t& r, float* f) {
    f[0] = __uint_as_float(r.x); f[1] = __uint_as_float(r.y);
    f[2] = __uint_as_float(r.z); f[3] = __uint_as_float(r.w);
  }
};
template <> struct KvFmt<KV_BF16> {
  static constexpr int VEC = 8;       // 16 bytes
  using raw_t = uint4;
  __device__ static void to_f32(const raw_t& r, float* f) {
    f[0] = bf16_lo(r.x); f[1] = bf16_hi(r.x); f[2] = bf16_lo(r.y); f[3] = bf16_hi(r.y);
    f[4] = bf16_lo(r.z); f[5] = bf16_hi(r.z); f[6] = bf16_lo(r.w); f[7] = bf16_hi(r.w);
  }
};
template <> struct KvFmt<KV_FP8> {
  static constexpr int VEC = 8;       // 8 bytes
  using raw_t = uint2;
  __device__ static void to_f32(const raw_t& r, float* f) {
    // gfx950 converts OCP E4M3FN codes exactly to fp32, two at a time
    auto a = __builtin_amdgcn_cvt_pk_f32_fp8(r.x, false);
    auto b = __builtin_amdgcn_cvt_pk_f32_fp8(r.x, true);
    auto c = __builtin_amdgcn_cvt_pk_f32_fp8(r.y, false);
    auto d = __builtin_amdgcn_cvt_pk_f32_fp8(r.y, true);
    f[0] = a[0]; f[1] = a[1]; f[2] = b[0]; f[3] = b[1];
    f[4] = c[0]; f[5] = c[1]; f[6] = d[0]; f[7] = d[1];
  }
};

template <int OT>
__device__ __forceinline__ void store_out(void* out, int64_t off, float v) {
  if constexpr (OT == AUG_F32) {
    static_cast<float*>(out)[off] = v;
  } else {
    static_cast<uint16_t*>(out)[off] = static_cast<uint16_t>(f32_to_bf16_bits(v));
  }
}

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));

__device__ __forceinline__ float dot2_bf16(uint32_t a, uint32_t b, float c) {
  return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, a), __builtin_bit_cast(bf16x2_t, b),
                                         c, false);
}

// Per-lane query slice and the q.k partial product of one lane's VEC
// elements. bf16 K against bf16 Q uses packed dot2 on the raw pairs (no
// conversion of K); other KV formats convert K to fp32 first.
template <int KVT, int QT> struct RowMath;

template <> struct RowMath<KV_BF16, AUG_BF16> {
  static constexpr int QW = 4;                 // packed bf16 pairs per lane (8 elements)
  using q_t = uint32_t;
  using k_t = uint4;
  __device__ static const uint4& prep(const uint4& k) { return k; }
  __device__ static void load(const void* q, int64_t off, q_t* dst) {
    const uint4 v = *reinterpret_cast<const uint4*>(static_cast<const uint16_t*>(q) + off);
    dst[0] = v.x; dst[1] = v.y; dst[2] = v.z; dst[3] = v.w;
  }
  __device__ static float dot(const q_t* qh, const uint4& k) {
    float acc = dot2_bf16(k.x, qh[0], 0.f);
    acc = dot2_bf16(k.y, qh[1], acc);
    acc = dot2_bf16(k.z, qh[2], acc);
    return dot2_bf16(k.w, qh[3], acc);
  }
};

template <> struct RowMath<KV_F32, AUG_F32> {
  static constexpr int QW = 4;
  using q_t = float;
  using k_t = uint4;
  __device__ static const uint4& prep(const uint4& k) { return k; }
  __device__ static void load(const void* q, int64_t off, q_t* dst) {
    const float4 v = *reinterpret_cast<const float4*>(static_cast<const float*>(q) + off);
    dst[0] = v.x; dst[1] = v.y; dst[2] = v.z; dst[3] = v.w;
  }
  __device__ static float dot(const q_t* qh, const uint4& k) {
    float acc = qh[0] * __uint_as_float(k.x);
    acc = fmaf(qh[1], __uint_as_float(k.y), acc);
    acc = fmaf(qh[2], __uint_as_float(k.z), acc);
    return fmaf(qh[3], __uint_as_float(k.w), acc);
  }
};

// fp8 K is converted once per load to packed bf16 (exact for OCP E4M3FN)
// and dotted with the bf16 query pairs like the bf16 cache.
template <> struct RowMath<KV_FP8, AUG_BF16> {
  static constexpr int QW = 4;
  using q_t = uint32_t;
  using k_t = uint4;
  __device__ static void load(const void* q, int64_t off, q_t* dst) {
    RowMath<KV_BF16, AUG_BF16>::load(q, off, dst);
  }
  __device__ static uint4 prep(const uint2& k) {
    uint4 o;
    o.x = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(k.x, 1.0f, false));
    o.y = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(k.x, 1.0f, true));
    o.z = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(k.y, 1.0f, false));
    o.w = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(k.y, 1.0f, true));
    return o;
  }
  __device__ static float dot(const q_t* qh, const uint4& k) { return RowMath<KV_BF16, AUG_BF16>::dot(qh, k); }
};

// ---------------------------------------------------------------------------
// split-K merge inside the launch
// ---------------------------------------------------------------------------

// Partials cross workgroups that may run on different XCDs, whose L2 caches
// are not coherent with each other. They are therefore stored and loaded as
// device-scope relaxed atomics (write-through / coherent accesses), and a
// writer waits for its stores to complete before it counts its span done;
// no release fence, which would write back and invalidate the whole L2.
__device__ __forceinline__ void store_partial(float* p, float v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ float load_partial(const float* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ float2 load_partial2(const float* p) {
  const uint64_t v = __hip_atomic_load(reinterpret_cast<const uint64_t*>(p), __ATOMIC_RELAXED,
                                       __HIP_MEMORY_SCOPE_AGENT);
  return float2{__uint_as_float(static_cast<uint32_t>(v)), __uint_as_float(static_cast<uint32_t>(v >> 32))};
}

// Merge of one (row, KV head) group without LDS or barriers: every thread
// folds four output dims of one head over all spans online, its loads of
// (m, l) and of the partial values all independent (device-scope loads,
// since the partials come from other workgroups of this launch).
template <int D, int G, int OT, int NT>
__device__ __forceinline__ void merge_group_direct(const MergeGroup& g, const float* partials, void* out,
                                                   int32_t hq) {
  const int64_t pf = aug::partial_floats(G, D);
  const float* base = partials + static_cast<int64_t>(g.part0) * pf;
  for (int c = threadIdx.x; c < G * D / 4; c += NT) {
    const int h = (4 * c) / D;
    float mx = kNegBig, l = 0.f, o0 = 0.f, o1 = 0.f, o2 = 0.f, o3 = 0.f;
    int s = 0;
    auto fold = [&](float ms, float ls, float2 x01, float2 x23) {
      const float mn = fmaxf(mx, ms);
      const float a0 = __builtin_amdgcn_exp2f(mx - mn), a1 = __builtin_amdgcn_exp2f(ms - mn);
      l = l * a0 + ls * a1;
      o0 = o0 * a0 + x01.x * a1;
      o1 = o1 * a0 + x01.y * a1;
      o2 = o2 * a0 + x23.x * a1;
      o3 = o3 * a0 + x23.y * a1;
      mx = mn;
    };
    for (; s + 4 <= g.n_parts; s += 4) {
      float ms[4], ls[4];
      float2 x01[4], x23[4];
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const float* p = base + static_cast<int64_t>(s + k) * pf;
        ms[k] = load_partial(p + G * D + h);
        ls[k] = load_partial(p + G * D + G + h);
        x01[k] = load_partial2(p + 4 * c);
        x23[k] = load_partial2(p + 4 * c + 2);
      }
#pragma unroll
      for (int k = 0; k < 4; ++k) fold(ms[k], ls[k], x01[k], x23[k]);
    }
    for (; s < g.n_parts; ++s) {
      const float* p = base + static_cast<int64_t>(s) * pf;
      fold(load_partial(p + G * D + h), load_partial(p + G * D + G + h), load_partial2(p + 4 * c),
           load_partial2(p + 4 * c + 2));
    }
    const float inv = 1.f / l;
    const int64_t off = (static_cast<int64_t>(g.q_row) * hq + static_cast<int64_t>(g.kvh) * G) * D + 4 * c;
    store_out<OT>(out, off + 0, o0 * inv);
    store_out<OT>(out, off + 1, o1 * inv);
    store_out<OT>(out, off + 2, o2 * inv);
    store_out<OT>(out, off + 3, o3 * inv);
  }
}

// Called by every thread of a split item after it stored its partials. The
// workgroup that finishes a group's last span merges the group's rows
// (merge groups `group` .. `group + n_rows - 1`, which share their spans) and
// returns the counter to zero, so the plan image can be launched again.
// `lds` needs one int and must be free when this is called.
template <int D, int G, int OT, int NT>
__device__ __forceinline__ void finish_split(const AttnArgs& a, int group, int n_rows, float* lds) {
  __builtin_amdgcn_s_waitcnt(0);   // this thread's partial stores have completed
  __syncthreads();
  int* flag = reinterpret_cast<int*>(lds);
  if (threadIdx.x == 0) {
    const int done = __hip_atomic_fetch_add(a.counters + group, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    const bool last = done == a.groups[group].n_parts - 1;
    if (last) __hip_atomic_store(a.counters + group, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    *flag = last;
  }
  __syncthreads();
  if (!*flag) return;
  for (int r = 0; r < n_rows; ++r) merge_group_direct<D, G, OT, NT>(a.groups[group + r], a.partials, a.out, a.hq);
}

// ---------------------------------------------------------------------------
// row items (VALU)
// ---------------------------------------------------------------------------

// Last step of a row item: every wave has written its unnormalised output
// o[G][D], running maximum and row sum to lds[wave][head][D + 2]; the waves'
// results are merged (log-sum-exp) and stored as the output rows, or as the
// item's split-K partial.
template <int D, int G, int OT, int NW>
__device__ __forceinline__ void row_merge_waves(const WorkItem& it, const AttnArgs& a, float* lds) {
  constexpr int ROW = D + 2;
  const int kvh = it.kvh;
  __syncthreads();
  for (int idx = threadIdx.x; idx < G * D; idx += 64 * NW) {
    const int h = idx / D;
    const int d = idx % D;
    float mw[NW];
    float mx = kNegBig;
#pragma unroll
    for (int w = 0; w < NW; ++w) {
      mw[w] = lds[(w * G + h) * ROW + D];
      mx = fmaxf(mx, mw[w]);
    }
    float ls = 0.f, os = 0.f;
#pragma unroll
    for (int w = 0; w < NW; ++w) {
      const float f = __builtin_amdgcn_exp2f(mw[w] - mx);
      ls += lds[(w * G + h) * ROW + D + 1] * f;
      os += lds[(w * G + h) * ROW + d] * f;
    }
    if (it.part < 0) {
      const int64_t off = (static_cast<int64_t>(it.q_row0) * a.hq + static_cast<int64_t>(kvh) * G + h) * D + d;
      store_out<OT>(a.out, off, os / ls);
    } else {
      float* pp = a.partials + static_cast<int64_t>(it.part) * aug::partial_floats(G, D);
      store_partial(pp + h * D + d, os);
      if (d == 0) {
        store_partial(pp + G * D + h, mx);
        store_partial(pp + G * D + G + h, ls);
      }
    }
  }
  if (it.part >= 0) finish_split<D, G, OT, 64 * NW>(a, it.group, 1, lds);
}


template <int KVT, int D, int G, int QT, int OT, bool PREFETCH, int NW>
__device__ void row_item(const WorkItem& it, const AttnArgs& a, float* lds) {
  using F = KvFmt<KVT>;
  using M = RowMath<KVT, QT>;
  constexpr int VEC = F::VEC;
  constexpr int LPT = D / VEC;        // lanes per token row
  constexpr int TPI = 64 / LPT;       // tokens per load instruction
  constexpr int NLD = kBlock / TPI;   // load instructions per 16-token block
  constexpr int EB = KVT == KV_F32 ? 4 : KVT == KV_BF16 ? 2 : 1;
  static_assert(LPT >= 4 && LPT <= 32 && NLD >= 1, "row-path lane mapping");
  using elem_t = typename F::raw_t;

  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int dl = lane % LPT;
  const int tsub = lane / LPT;
  const int d0 = dl * VEC;
  const int kvh = it.kvh;

  typename M::q_t q[G][M::QW];
  {
    const int64_t qoff = (static_cast<int64_t>(it.q_row0) * a.hq + static_cast<int64_t>(kvh) * G) * D + d0;
#pragma unroll
    for (int h = 0; h < G; ++h) M::load(a.q, qoff + static_cast<int64_t>(h) * D, q[h]);
  }
  const float sc = a.scale_log2;

  float m[G], l[G], o[G][VEC];
#pragma unroll
  for (int h = 0; h < G; ++h) {
    m[h] = kNegBig;
    l[h] = 0.f;
#pragma unroll
    for (int e = 0; e < VEC; ++e) o[h][e] = 0.f;
  }

  const int blk0 = it.key_begin / kBlock;
  const int nblk = (it.key_end - it.key_begin + kBlock - 1) / kBlock;
  const int64_t head_stride = static_cast<int64_t>(kBlock) * D;   // elements of one (block, head)
  const char* kc = static_cast<const char*>(a.k_cache);
  const char* vc = static_cast<const char*>(a.v_cache);

  // The block id of a wave's next block is fetched one iteration ahead, so
  // the K/V loads of a block never wait on the block-table load. With
  // PREFETCH the K/V of the next block are in flight too while the current
  // one is computed.
  constexpr int kWaves = NW;
  const int32_t* table = a.block_ids + it.bt_off + blk0;
  auto load_block = [&](int bid, elem_t* kr, elem_t* vr) {
    const bool ok = static_cast<uint32_t>(bid) < static_cast<uint32_t>(a.num_pool_blocks);
    const int64_t base = ((static_cast<int64_t>(bid) * a.hkv + kvh) * head_stride + d0) * EB;
#pragma unroll
    for (int i = 0; i < NLD; ++i) {
      if (ok) {
        const int64_t off = base + static_cast<int64_t>(i * TPI + tsub) * D * EB;
        kr[i] = *reinterpret_cast<const elem_t*>(kc + off);
        vr[i] = *reinterpret_cast<const elem_t*>(vc + off);
      } else {
        kr[i] = elem_t{};
        vr[i] = elem_t{};
      }
    }
  };
  int bid_next = wave < nblk ? table[wave] : 0;
  elem_t kpre[PREFETCH ? NLD : 1], vpre[PREFETCH ? NLD : 1];
  int bid_pre = 0;
  if constexpr (PREFETCH) {
    if (wave < nblk) {
      bid_pre = __builtin_amdgcn_readfirstlane(bid_next);
      load_block(bid_pre, kpre, vpre);
      if (wave + kWaves < nblk) bid_next = table[wave + kWaves];
    }
  }
  for (int bi = wave; bi < nblk; bi += kWaves) {
    const int blk = blk0 + bi;
    int bid;
    elem_t kraw[NLD], vraw[NLD];
    if constexpr (PREFETCH) {
      bid = bid_pre;
#pragma unroll
      for (int i = 0; i < NLD; ++i) {
        kraw[i] = kpre[i];
        vraw[i] = vpre[i];
      }
      if (bi + kWaves < nblk) {
        bid_pre = __builtin_amdgcn_readfirstlane(bid_next);
        load_block(bid_pre, kpre, vpre);
        if (bi + 2 * kWaves < nblk) bid_next = table[bi + 2 * kWaves];
      }
    } else {
      bid = __builtin_amdgcn_readfirstlane(bid_next);
      if (bi + kWaves < nblk) bid_next = table[bi + kWaves];
      load_block(bid, kraw, vraw);
    }
    const bool bid_ok = static_cast<uint32_t>(bid) < static_cast<uint32_t>(a.num_pool_blocks);
    const int tok0 = blk * kBlock;
    float ksc = sc, vsc = 1.f, vlog = 0.f, vinv = 1.f;
    if constexpr (KVT == KV_FP8) {
      if (bid_ok) {
        ksc = sc * a.k_scale[static_cast<int64_t>(bid) * a.hkv + kvh];
        vsc = a.v_scale[static_cast<int64_t>(bid) * a.hkv + kvh];
        // bf16 probabilities carry the V scale through its log2 and the row
        // sum weighs it back (a zero scale is taken as 2^-100)
        const float vs = fmaxf(vsc, 0x1p-100f);
        vlog = __builtin_amdgcn_logf(vs);
        vinv = __builtin_amdgcn_rcpf(vs);
      }
    }
    // a block is either entirely inside the span (no masking at all) or the
    // span's tail block / an unusable block (masked token by token)
    const bool full = bid_ok && tok0 + kBlock <= it.key_end;

    float s[NLD][G];
#pragma unroll
    for (int i = 0; i < NLD; ++i) {
      const typename M::k_t kb = M::prep(kraw[i]);
#pragma unroll
      for (int h = 0; h < G; ++h) s[i][h] = group_sum<LPT>(M::dot(q[h], kb)) * ksc;
    }
    if (!full) {
#pragma unroll
      for (int i = 0; i < NLD; ++i) {
        const bool valid = bid_ok && (tok0 + i * TPI + tsub) < it.key_end;
#pragma unroll
        for (int h = 0; h < G; ++h) s[i][h] = valid ? s[i][h] : -INFINITY;
        if (!valid) vraw[i] = elem_t{};   // zero, so 0 * value never meets NaN
      }
    }

    float mn[G];
    bool moved = false;
#pragma unroll
    for (int h = 0; h < G; ++h) {
      float mb = s[0][h];
#pragma unroll
      for (int i = 1; i < NLD; ++i) mb = fmaxf(mb, s[i][h]);
      mn[h] = fmaxf(m[h], mb);
      moved |= mn[h] > m[h] + kRescaleSlack;
    }
    // rescale only when some running maximum moved far (see kRescaleSlack)
    if (__any(moved)) {
#pragma unroll
      for (int h = 0; h < G; ++h) {
        const float alpha = __builtin_amdgcn_exp2f(m[h] - mn[h]);
        l[h] *= alpha;
#pragma unroll
        for (int e = 0; e < VEC; ++e) o[h][e] *= alpha;
        m[h] = mn[h];
      }
    }
    if constexpr (KVT == KV_F32) {
#pragma unroll
      for (int i = 0; i < NLD; ++i) {
        float vf[VEC];
        F::to_f32(vraw[i], vf);
#pragma unroll
        for (int h = 0; h < G; ++h) {
          const float p = __builtin_amdgcn_exp2f(s[i][h] - m[h]);
          l[h] += p;
          const float pv = p * vsc;
#pragma unroll
          for (int e = 0; e < VEC; ++e) o[h][e] = fmaf(pv, vf[e], o[h][e]);
        }
      }
    } else {
      // The lane's tokens go in pairs (loads i and i + 1 of the block): their
      // probabilities are packed to one bf16 pair, the values of each dim to
      // another, and one packed dot product adds both tokens' terms. The row
      // sum adds exactly the packed probabilities, as the MFMA paths do.
      static_assert(NLD % 2 == 0 && VEC == 8, "row tokens pair up, eight dims per lane");
#pragma unroll
      for (int i = 0; i < NLD; i += 2) {
        uint32_t vp[VEC];   // dim e of tokens i and i + 1, as one bf16 pair
        if constexpr (KVT == KV_BF16) {
          const uint32_t a0[4] = {vraw[i].x, vraw[i].y, vraw[i].z, vraw[i].w};
          const uint32_t a1[4] = {vraw[i + 1].x, vraw[i + 1].y, vraw[i + 1].z, vraw[i + 1].w};
#pragma unroll
          for (int k = 0; k < 4; ++k) {
            vp[2 * k] = __builtin_amdgcn_perm(a1[k], a0[k], 0x05040100u);
            vp[2 * k + 1] = __builtin_amdgcn_perm(a1[k], a0[k], 0x07060302u);
          }
        } else {
          // fp8: interleave the two tokens' codes, then convert each byte
          // pair exactly to a bf16 pair
#pragma unroll
          for (int k = 0; k < 2; ++k) {
            const uint32_t x0 = k ? vraw[i].y : vraw[i].x, x1 = k ? vraw[i + 1].y : vraw[i + 1].x;
            const uint32_t lo = __builtin_amdgcn_perm(x1, x0, 0x05010400u);   // dims 4k, 4k+1
            const uint32_t hi = __builtin_amdgcn_perm(x1, x0, 0x07030602u);   // dims 4k+2, 4k+3
            vp[4 * k + 0] = fp8x2_to_bf16x2<false>(lo);
            vp[4 * k + 1] = fp8x2_to_bf16x2<true>(lo);
            vp[4 * k + 2] = fp8x2_to_bf16x2<false>(hi);
            vp[4 * k + 3] = fp8x2_to_bf16x2<true>(hi);
          }
        }
#pragma unroll
        for (int h = 0; h < G; ++h) {
          const float bias = vlog - m[h];
          const uint32_t pp = pack_bf16(__builtin_amdgcn_exp2f(s[i][h] + bias),
                                        __builtin_amdgcn_exp2f(s[i + 1][h] + bias));
          const float psum = dot2_bf16(pp, kBf16PairOne, 0.f);
          l[h] = KVT == KV_FP8 ? fmaf(psum, vinv, l[h]) : l[h] + psum;
#pragma unroll
          for (int e = 0; e < VEC; ++e) o[h][e] = dot2_bf16(pp, vp[e], o[h][e]);
        }
      }
    }
  }

  // merge the TPI lane groups of this wave (lanes with equal dl)
#pragma unroll
  for (int mask = LPT; mask < 64; mask <<= 1) {
#pragma unroll
    for (int h = 0; h < G; ++h) {
      const float mo = __shfl_xor(m[h], mask);
      const float lo = __shfl_xor(l[h], mask);
      const float mn = fmaxf(m[h], mo);
      const float a1 = __builtin_amdgcn_exp2f(m[h] - mn);
      const float a2 = __builtin_amdgcn_exp2f(mo - mn);
      l[h] = l[h] * a1 + lo * a2;
#pragma unroll
      for (int e = 0; e < VEC; ++e) o[h][e] = o[h][e] * a1 + __shfl_xor(o[h][e], mask) * a2;
      m[h] = mn;
    }
  }

  // merge the four waves through LDS: [wave][head][D + 2]
  constexpr int ROW = D + 2;
  if (tsub == 0) {
#pragma unroll
    for (int h = 0; h < G; ++h) {
      float* dst = lds + (wave * G + h) * ROW;
#pragma unroll
      for (int e = 0; e < VEC; ++e) dst[d0 + e] = o[h][e];
      if (dl == 0) {
        dst[D] = m[h];
        dst[D + 1] = l[h];
      }
    }
  }
  row_merge_waves<D, G, OT, NW>(it, a, lds);
}

// ---------------------------------------------------------------------------
// row items of 8-way (and 4-way) grouped-query attention (MFMA)
// ---------------------------------------------------------------------------
//
// With eight query heads per KV head, a decode row's work per KV byte (two
// bf16 dot products of D per head and key) is more than the vector ALUs keep
// up with next to fp8 decoding, so the eight heads go through 16x16 bf16
// MFMAs instead (heads 8..15 of each MFMA are zero padding). Groups of four
// heads take the same path with heads 4..15 as padding: the vector ALUs keep
// up there, and the MFMA form only frees issue slots for the loads. Per
// 16-token block and wave:
//   S^T[16 keys][16 heads] = K Q^T with four 16x16x32 MFMAs over head_dim.
//     Lane l holds token l % 16 and dims 32g .. 32g + 31 (g = l / 16) of the
//     block's K rows; k-step s takes dims 32g + 8s .. + 8 of both K and Q (a
//     permutation of the reduction dimension shared by both operands).
//   The S^T accumulator gives lane l head l % 16 and keys 4g .. 4g + 3, which
//   is exactly the B operand layout of a 16x16x16 MFMA over those keys, so
//   the probabilities feed PV without any exchange.
//   O^T[128 dims][16 heads] += V^T P^T with eight 16x16x16 MFMAs, one per dim
//     block b: row m of block b is dim 8m + b, so lane l loads dims 8m .. 8m + 7
//     (m = l % 16) of its four tokens 4g .. 4g + 3 with contiguous loads and
//     only regroups them into (token, token) pairs per dim.
// The resulting accumulators give lane l head l % 16 and dims 32g .. 32g + 31.

// max and sum over the four lanes l, l ^ 16, l ^ 32, l ^ 48
__device__ __forceinline__ float group4_max(float v) {
  const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  const float m = fmaxf(__uint_as_float(a[0]), __uint_as_float(a[1]));
  const auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(m), __float_as_uint(m), false, false);
  return fmaxf(__uint_as_float(b[0]), __uint_as_float(b[1]));
}
__device__ __forceinline__ float group4_sum(float v) {
  const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  const float m = __uint_as_float(a[0]) + __uint_as_float(a[1]);
  const auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(m), __float_as_uint(m), false, false);
  return __uint_as_float(b[0]) + __uint_as_float(b[1]);
}

typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef short s16x4_t __attribute__((ext_vector_type(4)));


template <int KVT> struct MfmaRowKv;
template <> struct MfmaRowKv<KV_BF16> {
  struct K { uint4 w[4]; };      // token l % 16, dims 32g .. 32g + 31
  struct V { uint4 w[4]; };      // tokens 4g + t, dims 8m .. 8m + 7
  static constexpr int EB = 2;
  __device__ static void load_k(const char* p, K& k) {
#pragma unroll
    for (int i = 0; i < 4; ++i) k.w[i] = reinterpret_cast<const uint4*>(p)[i];
  }
  __device__ static void load_v(const char* p, int64_t row_bytes, V& v) {
#pragma unroll
    for (int t = 0; t < 4; ++t) v.w[t] = *reinterpret_cast<const uint4*>(p + t * row_bytes);
  }
  __device__ static uint4 k_operand(const K& k, int s) { return k.w[s]; }
  __device__ static void zero_v(V& v, int t) { v.w[t] = uint4{0, 0, 0, 0}; }
  // (token 4g + 0..3) values of dim 8m + b, as two bf16 pairs
  __device__ static void v_operands(const V& v, uint2 (&op)[8]) {
    const uint32_t* x0 = reinterpret_cast<const uint32_t*>(&v.w[0]);
    const uint32_t* x1 = reinterpret_cast<const uint32_t*>(&v.w[1]);
    const uint32_t* x2 = reinterpret_cast<const uint32_t*>(&v.w[2]);
    const uint32_t* x3 = reinterpret_cast<const uint32_t*>(&v.w[3]);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      op[2 * i] = uint2{__builtin_amdgcn_perm(x1[i], x0[i], 0x05040100u), __builtin_amdgcn_perm(x3[i], x2[i], 0x05040100u)};
      op[2 * i + 1] = uint2{__builtin_amdgcn_perm(x1[i], x0[i], 0x07060302u), __builtin_amdgcn_perm(x3[i], x2[i], 0x07060302u)};
    }
  }
};
template <> struct MfmaRowKv<KV_FP8> {
  struct K { uint4 w[2]; };
  struct V { uint2 w[4]; };
  static constexpr int EB = 1;
  __device__ static void load_k(const char* p, K& k) {
    k.w[0] = reinterpret_cast<const uint4*>(p)[0];
    k.w[1] = reinterpret_cast<const uint4*>(p)[1];
  }
  __device__ static void load_v(const char* p, int64_t row_bytes, V& v) {
#pragma unroll
    for (int t = 0; t < 4; ++t) v.w[t] = *reinterpret_cast<const uint2*>(p + t * row_bytes);
  }
  __device__ static uint4 k_operand(const K& k, int s) {
    const uint4& w = k.w[s >> 1];
    const uint32_t lo = (s & 1) ? w.z : w.x, hi = (s & 1) ? w.w : w.y;
    return uint4{fp8x2_to_bf16x2<false>(lo), fp8x2_to_bf16x2<true>(lo), fp8x2_to_bf16x2<false>(hi),
                 fp8x2_to_bf16x2<true>(hi)};
  }
  __device__ static void zero_v(V& v, int t) { v.w[t] = uint2{0, 0}; }
  __device__ static void v_operands(const V& v, uint2 (&op)[8]) {
    // interleave the bytes of tokens (0, 1) and (2, 3), then each byte pair
    // converts to the bf16 pair (token, token + 1) of one dim
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const uint32_t a0 = i ? v.w[0].y : v.w[0].x, a1 = i ? v.w[1].y : v.w[1].x;
      const uint32_t a2 = i ? v.w[2].y : v.w[2].x, a3 = i ? v.w[3].y : v.w[3].x;
      const uint32_t p01lo = __builtin_amdgcn_perm(a1, a0, 0x05010400u);   // dims 4i, 4i+1
      const uint32_t p01hi = __builtin_amdgcn_perm(a1, a0, 0x07030602u);   // dims 4i+2, 4i+3
      const uint32_t p23lo = __builtin_amdgcn_perm(a3, a2, 0x05010400u);
      const uint32_t p23hi = __builtin_amdgcn_perm(a3, a2, 0x07030602u);
      op[4 * i + 0] = uint2{fp8x2_to_bf16x2<false>(p01lo), fp8x2_to_bf16x2<false>(p23lo)};
      op[4 * i + 1] = uint2{fp8x2_to_bf16x2<true>(p01lo), fp8x2_to_bf16x2<true>(p23lo)};
      op[4 * i + 2] = uint2{fp8x2_to_bf16x2<false>(p01hi), fp8x2_to_bf16x2<false>(p23hi)};
      op[4 * i + 3] = uint2{fp8x2_to_bf16x2<true>(p01hi), fp8x2_to_bf16x2<true>(p23hi)};
    }
  }
};

template <int KVT, int OT, int NW, int G>
__device__ void row_item_mfma(const WorkItem& it, const AttnArgs& a, float* lds) {
  static_assert(G == 8 || G == 4, "one 16-column MFMA holds the group's heads");
  constexpr int D = 128;
  constexpr bool FP8 = KVT == KV_FP8;
  using KV = MfmaRowKv<KVT>;
  constexpr int EB = KV::EB;
  const int lane = threadIdx.x & 63;
  // wave-uniform, so block ids and scales come through scalar loads instead
  // of queueing behind the K/V loads
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int j = lane & 15;            // query head of the group (G..15: padding)
  const int g = lane >> 4;            // keys 4g .. 4g + 3 of a block
  const int kvh = it.kvh;

  // Q^T operands of the four k-steps: dims 32g + 8s .. + 8 of head j
  uint4 qop[4];
  {
    const uint16_t* qb = static_cast<const uint16_t*>(a.q) +
                         (static_cast<int64_t>(it.q_row0) * a.hq + static_cast<int64_t>(kvh) * G + (j < G ? j : 0)) * D + 32 * g;
#pragma unroll
    for (int s = 0; s < 4; ++s) qop[s] = j < G ? *reinterpret_cast<const uint4*>(qb + 8 * s) : uint4{0, 0, 0, 0};
  }
  const float sc = a.scale_log2;
  float m_run = kNegBig, l_run = 0.f;
  f32x4_t oacc[8];
#pragma unroll
  for (int b = 0; b < 8; ++b) oacc[b] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  const int blk0 = it.key_begin / kBlock;
  const int nblk = (it.key_end - it.key_begin + kBlock - 1) / kBlock;
  constexpr int64_t kRow = static_cast<int64_t>(D) * EB;                 // bytes of one token row
  constexpr int64_t kHead = kBlock * kRow;                               // bytes of one (block, head)
  const char* kc = static_cast<const char*>(a.k_cache);
  const char* vc = static_cast<const char*>(a.v_cache);
  const int64_t k_lane = (j * D + 32 * g) * EB;                          // token j, dims 32g..
  const int64_t v_lane = (4 * g * D + 8 * j) * EB;                       // tokens 4g.., dims 8j..
  constexpr int kWaves = NW;
  const int32_t* table = a.block_ids + it.bt_off + blk0;
  // a block's K and V, and (fp8) its two scales, loaded together so the
  // scales arrive with the data instead of a memory round trip later
  struct Scales { float k, v; };
  auto load_block = [&](int bid, typename KV::K& k, typename KV::V& v, Scales& sc2) {
    if (static_cast<uint32_t>(bid) < static_cast<uint32_t>(a.num_pool_blocks)) {
      const int64_t base = (static_cast<int64_t>(bid) * a.hkv + kvh) * kHead;
      KV::load_k(kc + base + k_lane, k);
      KV::load_v(vc + base + v_lane, kRow, v);
      if constexpr (FP8) {
        sc2.k = a.k_scale[static_cast<int64_t>(bid) * a.hkv + kvh];
        sc2.v = a.v_scale[static_cast<int64_t>(bid) * a.hkv + kvh];
      }
    } else {
      k = typename KV::K{};
      v = typename KV::V{};
      sc2 = Scales{1.f, 1.f};
    }
  };

  // the next block's K/V (and scales) in flight while one is computed, its
  // id read one iteration before that (deeper prefetch measured no faster)
  typename KV::K kpre{};
  typename KV::V vpre{};
  Scales spre{1.f, 1.f};
  int bid_pre = wave < nblk ? __builtin_amdgcn_readfirstlane(table[wave]) : 0;
  if (wave < nblk) load_block(bid_pre, kpre, vpre, spre);
  int bid_next = wave + kWaves < nblk ? table[wave + kWaves] : 0;
  for (int bi = wave; bi < nblk; bi += kWaves) {
    const int tok0 = (blk0 + bi) * kBlock;
    const int bid = bid_pre;
    typename KV::K kraw = kpre;
    typename KV::V vraw = vpre;
    const Scales bsc = spre;
    // the next block's loads are issued ahead of the other waves' work on
    // this SIMD (measured 1-2 % on decode batches)
    __builtin_amdgcn_s_setprio(1);
    if (bi + kWaves < nblk) {
      bid_pre = __builtin_amdgcn_readfirstlane(bid_next);
      load_block(bid_pre, kpre, vpre, spre);
      if (bi + 2 * kWaves < nblk) bid_next = table[bi + 2 * kWaves];
    }
    __builtin_amdgcn_s_setprio(0);
    const bool bid_ok = static_cast<uint32_t>(bid) < static_cast<uint32_t>(a.num_pool_blocks);
    float ksc = sc, vlog = 0.f, vinv = 1.f;
    if constexpr (FP8) {
      if (bid_ok) {
        ksc = sc * bsc.k;
        // the V scale enters each probability through its log2 and leaves the
        // row sum through its reciprocal (a zero scale is taken as 2^-100)
        const float vs = fmaxf(bsc.v, 0x1p-100f);
        vlog = __builtin_amdgcn_logf(vs);
        vinv = __builtin_amdgcn_rcpf(vs);
      }
    }

    f32x4_t sacc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int s = 0; s < 4; ++s)
      sacc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(KV::k_operand(kraw, s)), as_bf16x8(qop[s]), sacc,
                                                     0, 0, 0);
    // a block is inside the span (no masking) or the span's tail / an unusable block
    const bool full = bid_ok && tok0 + kBlock <= it.key_end;
    float sv[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) sv[r] = sacc[r] * ksc;
    if (!full) {
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const bool valid = bid_ok && tok0 + 4 * g + r < it.key_end;
        sv[r] = valid ? sv[r] : -INFINITY;
        if (!valid) KV::zero_v(vraw, r);   // zero, so 0 * value never meets NaN
      }
    }
    const float bm = group4_max(fmaxf(fmaxf(sv[0], sv[1]), fmaxf(sv[2], sv[3])));
    const float mn = fmaxf(m_run, bm);
    if (__any(mn > m_run + kRescaleSlack)) {
      const float alpha = __builtin_amdgcn_exp2f(m_run - mn);
      l_run *= alpha;
#pragma unroll
      for (int b = 0; b < 8; ++b) oacc[b] *= alpha;
      m_run = mn;
    }
    const float bias = vlog - m_run;
    const uint32_t p01 = pack_bf16(__builtin_amdgcn_exp2f(sv[0] + bias), __builtin_amdgcn_exp2f(sv[1] + bias));
    const uint32_t p23 = pack_bf16(__builtin_amdgcn_exp2f(sv[2] + bias), __builtin_amdgcn_exp2f(sv[3] + bias));
    // the row sum adds exactly the packed probabilities
    const float bsum = dot2_bf16(p23, kBf16PairOne, dot2_bf16(p01, kBf16PairOne, 0.f));
    l_run = FP8 ? fmaf(bsum, vinv, l_run) : l_run + bsum;
    const s16x4_t pop = __builtin_bit_cast(s16x4_t, uint2{p01, p23});
    uint2 vop[8];
    KV::v_operands(vraw, vop);
#pragma unroll
    for (int b = 0; b < 8; ++b)
      oacc[b] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(__builtin_bit_cast(s16x4_t, vop[b]), pop, oacc[b], 0, 0, 0);
  }

  // this wave's result for head j: dims 32g + 8r + b from oacc[b][r]
  constexpr int ROW = D + 2;
  const float l_tot = group4_sum(l_run);
  if (j < G) {
    float* dst = lds + (wave * G + j) * ROW;
#pragma unroll
    for (int r = 0; r < 4; ++r)
#pragma unroll
      for (int b = 0; b < 8; ++b) dst[32 * g + 8 * r + b] = oacc[b][r];
    if (g == 0) {
      dst[D] = m_run;
      dst[D + 1] = l_tot;
    }
  }
  row_merge_waves<D, G, OT, NW>(it, a, lds);
}

// ---------------------------------------------------------------------------
// tile items (bf16 MFMA)
// ---------------------------------------------------------------------------

template <int D>
struct TileLds {
  static constexpr int KS = D + 8;    // K row stride (elements): 16-byte aligned, conflict-free reads
  static constexpr int KS8 = D + 16;  // K row stride (bytes) of fp8 keys kept as codes
  // fp8 values kept as codes, transposed: one row of 64 key bytes per
  // dimension (16 bytes of padding spread a 16-row read over all banks)
  static constexpr int VT8 = 80;
  // V row stride (elements): rows 64 bytes apart modulo the 256-byte bank
  // width, so the transposing reads of four consecutive rows hit distinct banks
  static constexpr int VS = D + 32;
  static constexpr int STAGE = 64 * (KS + VS) * 2;       // bytes of one K + V stage
  static constexpr int IDS = aug::kTileSpanMax / kBlock + 8; // block ids of one item's key span
  // fp8, per stage and block of the tile: the K scale times the softmax
  // coefficient, log2 of the V scale, and the V scale's reciprocal
  static constexpr int NSC = 12;
  static constexpr int SCALES = 2 * NSC * 4;
  static constexpr int BYTES = 2 * STAGE + IDS * 4 + SCALES;
  static_assert(D * VT8 <= 64 * VS * 2, "transposed fp8 values fit the V region of a stage");
};

// Staging of one thread's share of a key tile: 16-byte bf16 chunks, or
// 8-byte fp8 chunks converted (exactly) to bf16 on the way into LDS.
template <int KVT> struct TileStage;
template <> struct TileStage<KV_BF16> {
  using raw_t = uint4;
  __device__ static uint4 to_bf16(const raw_t& r) { return r; }
};
template <> struct TileStage<KV_FP8> {
  using raw_t = uint2;
  __device__ static uint4 to_bf16(const raw_t& r) {
    // OCP E4M3FN codes are exactly representable in bf16
    uint4 o;
    o.x = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(r.x, 1.0f, false));
    o.y = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(r.x, 1.0f, true));
    o.z = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(r.y, 1.0f, false));
    o.w = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(r.y, 1.0f, true));
    return o;
  }
};


typedef __bf16 bf16x4_t __attribute__((ext_vector_type(4)));
typedef bf16x4_t __attribute__((address_space(3))) lds_bf16x4_t;

// ds_read_b64_tr_b16: 8 bytes per lane, transposed across each 16-lane group
__device__ __forceinline__ uint2 ds_read_tr16(const uint16_t* p) {
  return __builtin_bit_cast(uint2, __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4_t*)(p)));
}

// v_permlane32_swap hands lane i the register of lane i + 32 (and back), so
// combining both results pairs every lane with its partner in the other half.
__device__ __forceinline__ float max_across_halves(float v) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float sum_across_halves(float v) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}


template <bool B> using bool_tag = std::integral_constant<bool, B>;

// One tile item: up to 128 query rows (kTileRows / G positions x G heads of
// one KV head) against keys [key_begin, key_end) of the request. Key tiles of
// 64 go through two LDS stages: while tile t is multiplied, tile t+1 sits in
// the other stage and tile t+2 is on its way from HBM into registers.
//
// Tiles that every row reads in full (all keys at or below the first row's
// position and inside the span, all block ids inside the pool) take a path
// without per-key conditions; only the diagonal and span-end tiles mask.
//
// F8 selects the arithmetic of the two products: 0 both bf16; 1 the score
// products S = Q K^T on fp8 MFMAs (queries rounded to E4M3 per row); 2 also
// P V on fp8 MFMAs (probabilities rounded to E4M3, values as stored).
template <int KVT, int D, int G, int OT, int F8>
__device__ void tile_item(const WorkItem& it, const AttnArgs& a, unsigned char* smem) {
  using L = TileLds<D>;
  using TS = TileStage<KVT>;
  using raw_t = typename TS::raw_t;
  constexpr bool FP8 = KVT == KV_FP8;
  constexpr bool QK8 = F8 >= 1;
  constexpr bool PV8 = F8 >= 2;
  static_assert(!QK8 || (FP8 && D == 128), "fp8 score products need fp8 keys and head_dim 128");
  // fp8 probabilities: a lane's P values are stored as E4M3 codes of
  // p * (vs_b / vref) * 2^kPv8Log2, with vs_b the block's V scale and vref the
  // largest V scale of the item; p stays below 2^kSlack between rescales, so
  // the codes stay below 2^(kSlack + kPv8Log2) = 256 (E4M3 reaches 448) and
  // probabilities down to 2^-15 of the row maximum remain nonzero
  constexpr float kSlack = PV8 ? 2.f : kRescaleSlack;
  constexpr float kPv8Log2 = 6.f;
  constexpr int EB = FP8 ? 1 : 2;     // bytes per K/V element
  constexpr int KSTEPS = D / 16;      // k-steps of S^T over head_dim
  constexpr int DB = D / 32;          // 32-dim blocks of O^T
  constexpr int CPR = D / 8;          // 16-byte chunks per key row
  constexpr int KPT = 64 * CPR / kThreads;   // keys staged per thread (4 or 2)
  static_assert(KPT == 2 || KPT == 4, "tile staging map");

  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int n = lane & 31;            // MFMA column: query row within the wave
  const int hh = lane >> 5;           // lane half: which 8 of the 16 k-slots
  const int kvh = it.kvh;
  const int row = wave * 32 + n;
  const int p = row / G;
  const int gh = row % G;
  const bool row_ok = p < it.n_rows;
  const int pos = it.pos0 + p;
  const uint16_t* qb = static_cast<const uint16_t*>(a.q);
  // lane (dimension m = lane % 32, k-slot half hh) reads keys 4hh + {0..3}
  // (and +8) of a 16-key step at dimension m of a 32-dim block
  const int v_lane_off = (4 * hh + (lane & 15) / 4) * L::VS + 16 * ((lane >> 4) & 1) + 4 * (lane & 3);

  // bf16 scores: Q^T operands of the KSTEPS k-steps, dims 16s + 8hh .. + 7.
  // fp8 scores: the row rounded to E4M3 after division by its scale qscale
  // (largest magnitude / 448), as the B operands of the two 64-dim k-steps:
  // lane half hh holds dims 64h + 32hh .. + 31 of k-step h.
  uint4 qreg[QK8 ? 1 : KSTEPS];
  v8i_t q8[2];
  float qscale = 1.f;
  {
    const int64_t qoff = (static_cast<int64_t>(it.q_row0 + p) * a.hq + static_cast<int64_t>(kvh) * G + gh) * D;
    if constexpr (!QK8) {
#pragma unroll
      for (int s = 0; s < KSTEPS; ++s)
        qreg[s] = row_ok ? *reinterpret_cast<const uint4*>(qb + qoff + 16 * s + 8 * hh) : uint4{0, 0, 0, 0};
    } else {
      uint4 raw[2][4];
#pragma unroll
      for (int h = 0; h < 2; ++h)
#pragma unroll
        for (int c4 = 0; c4 < 4; ++c4)
          raw[h][c4] = row_ok ? *reinterpret_cast<const uint4*>(qb + qoff + 64 * h + 32 * hh + 8 * c4)
                              : uint4{0, 0, 0, 0};
      float amax = 0.f;
#pragma unroll
      for (int h = 0; h < 2; ++h)
#pragma unroll
        for (int c4 = 0; c4 < 4; ++c4) {
          const uint32_t w[4] = {raw[h][c4].x, raw[h][c4].y, raw[h][c4].z, raw[h][c4].w};
#pragma unroll
          for (int e = 0; e < 4; ++e)
            amax = fmaxf(amax, fmaxf(fabsf(__uint_as_float(w[e] << 16)), fabsf(__uint_as_float(w[e] & 0xFFFF0000u))));
        }
      amax = max_across_halves(amax);
      // a vector below 2^-100 (all zero, in practice) rounds to zero: its
      // reciprocal scale would overflow
      const bool tiny = !(amax >= 0x1p-100f);
      qscale = tiny ? 1.f : amax * (1.f / 448.f);
      const float inv = tiny ? 0.f : 448.f / amax;
#pragma unroll
      for (int h = 0; h < 2; ++h)
#pragma unroll
        for (int c4 = 0; c4 < 4; ++c4) {
          const uint32_t w[4] = {raw[h][c4].x, raw[h][c4].y, raw[h][c4].z, raw[h][c4].w};
          // eight dims -> two dwords of four E4M3 codes (dim order kept)
          int lo = __builtin_amdgcn_cvt_pk_fp8_f32(__uint_as_float(w[0] << 16) * inv,
                                                  __uint_as_float(w[0] & 0xFFFF0000u) * inv, 0, false);
          lo = __builtin_amdgcn_cvt_pk_fp8_f32(__uint_as_float(w[1] << 16) * inv,
                                              __uint_as_float(w[1] & 0xFFFF0000u) * inv, lo, true);
          int hi = __builtin_amdgcn_cvt_pk_fp8_f32(__uint_as_float(w[2] << 16) * inv,
                                                  __uint_as_float(w[2] & 0xFFFF0000u) * inv, 0, false);
          hi = __builtin_amdgcn_cvt_pk_fp8_f32(__uint_as_float(w[3] << 16) * inv,
                                              __uint_as_float(w[3] & 0xFFFF0000u) * inv, hi, true);
          q8[h][2 * c4] = lo;
          q8[h][2 * c4 + 1] = hi;
        }
    }
  }

  f32x16_t acc_o[DB];
#pragma unroll
  for (int db = 0; db < DB; ++db)
#pragma unroll
    for (int e = 0; e < 16; ++e) acc_o[db][e] = 0.f;
  float m_run = kNegBig, l_run = 0.f;
  const float c = a.scale_log2;

  const int tc = threadIdx.x % CPR;
  const int tk = threadIdx.x / CPR;
  // fp8 values are staged transposed; their loads put the key groups on
  // neighbouring threads instead, so each wave's transposed LDS writes
  // spread over the banks (the loads then take 32-byte pieces of 16 rows)
  const int tkv = PV8 ? threadIdx.x % (64 / KPT) : tk;
  const int tcv = PV8 ? threadIdx.x / (64 / KPT) : tc;
  const int key_end = it.key_end;
  const int t0 = it.key_begin / 64;
  const int t1 = (key_end + 63) / 64;
  const char* kc = static_cast<const char*>(a.k_cache);
  const char* vc = static_cast<const char*>(a.v_cache);
  const int64_t head_stride = static_cast<int64_t>(kBlock) * D;

  // the item's block ids (at most IDS: spans are capped by the planner) are
  // read once into LDS, so staging a key tile costs one round trip
  int32_t* ids = reinterpret_cast<int32_t*>(smem + 2 * L::STAGE);
  float* stage_scales = reinterpret_cast<float*>(smem + 2 * L::STAGE + L::IDS * 4);
  const int blk_first = it.key_begin / kBlock;
  const int n_ids = (key_end + kBlock - 1) / kBlock - blk_first;
  int bad = 0;
  float vmax = 0.f;   // fp8 probabilities: the item's largest V scale
  for (int i = threadIdx.x; i < n_ids && i < L::IDS; i += kThreads) {
    const int32_t id = a.block_ids[it.bt_off + blk_first + i];
    ids[i] = id;
    const bool id_ok = static_cast<uint32_t>(id) < static_cast<uint32_t>(a.num_pool_blocks);
    bad |= !id_ok;
    if constexpr (PV8) {
      if (id_ok) vmax = fmaxf(vmax, a.v_scale[static_cast<int64_t>(id) * a.hkv + kvh]);
    }
  }
  if constexpr (PV8) {
    // per-wave maxima into the second stage's scale slots, which are free
    // until the first step's barrier
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) vmax = fmaxf(vmax, __shfl_xor(vmax, o));
    if (lane == 0) stage_scales[L::NSC + wave] = vmax;
  }
  bad = __syncthreads_or(bad);
  // exponent offset of the fp8 probabilities: log2(2^kPv8Log2 / vref) (a zero
  // scale counts as 2^-100, as for the blocks)
  float vbias = 0.f, vref = 1.f, vsmall = 0.f;
  if constexpr (PV8) {
    vref = 0x1p-100f;
#pragma unroll
    for (int w = 0; w < kThreads / 64; ++w) vref = fmaxf(vref, stage_scales[L::NSC + w]);
    vbias = kPv8Log2 - __builtin_amdgcn_logf(vref);
    // A block whose V scale is below 2^-8 of vref (an all-zero block has
    // scale 0) would round its probability codes to zero or nearly, and its
    // keys would drop out of the row sum. Such a block is staged with zero
    // values and vref's own scale terms instead: its keys keep their weight,
    // and its values, at most 2^-8 of the item's largest, are left out.
    vsmall = vref * 0x1p-8f;
  }
  const int t_full = bad ? t0 : max(t0, min(t1, min(it.pos0 + 1, key_end) / 64));

  // a thread stages KPT consecutive keys of one block (KPT divides 16)
  raw_t kr[KPT], vr[KPT];
  float sc_reg = 1.f;   // fp8: thread t < 8 carries scale t of the tile (k0..3, v0..3)
  float vsc_reg = 1.f;  // fp8 values: the V scale of the block this thread stages
  // KPT consecutive key rows (dims 8 tcx .. 8 tcx + 7) of `src`, zero where
  // past the span or in a block outside the pool
  auto load_rows = [&](const char* src, int k0, int tkx, int tcx, raw_t (&dst)[KPT], auto full_tag) -> int {
    constexpr bool FULL = decltype(full_tag)::value;
    const int tok0 = k0 + tkx * KPT;
    const int slot = (tok0 >> 4) - blk_first;
    const int bid = FULL || tok0 < key_end ? ids[slot] : -1;
    const bool ok = FULL || static_cast<uint32_t>(bid) < static_cast<uint32_t>(a.num_pool_blocks);
    const int64_t base = ((static_cast<int64_t>(bid) * a.hkv + kvh) * head_stride +
                          static_cast<int64_t>(tok0 & 15) * D + 8 * tcx) * EB;
#pragma unroll
    for (int u = 0; u < KPT; ++u)
      dst[u] = FULL || (ok && tok0 + u < key_end) ? *reinterpret_cast<const raw_t*>(src + base + static_cast<int64_t>(u) * D * EB)
                                                  : raw_t{};
    return ok ? bid : -1;
  };
  auto load_tile = [&](int k0, auto full_tag) {
    constexpr bool FULL = decltype(full_tag)::value;
    const int tok0 = k0 + tk * KPT;
    const int slot = (tok0 >> 4) - blk_first;
    if constexpr (PV8) {
      load_rows(kc, k0, tk, tc, kr, full_tag);
      const int vbid = load_rows(vc, k0, tkv, tcv, vr, full_tag);
      vsc_reg = vbid >= 0 ? a.v_scale[static_cast<int64_t>(vbid) * a.hkv + kvh] : 1.f;
    } else if constexpr (FULL) {
      const int64_t base = ((static_cast<int64_t>(ids[slot]) * a.hkv + kvh) * head_stride +
                            static_cast<int64_t>(tok0 & 15) * D + 8 * tc) * EB;
#pragma unroll
      for (int u = 0; u < KPT; ++u) {
        kr[u] = *reinterpret_cast<const raw_t*>(kc + base + static_cast<int64_t>(u) * D * EB);
        vr[u] = *reinterpret_cast<const raw_t*>(vc + base + static_cast<int64_t>(u) * D * EB);
      }
    } else {
      const int bid = tok0 < key_end ? ids[slot] : -1;
      const bool ok = static_cast<uint32_t>(bid) < static_cast<uint32_t>(a.num_pool_blocks);
      const int64_t base = ((static_cast<int64_t>(bid) * a.hkv + kvh) * head_stride +
                            static_cast<int64_t>(tok0 & 15) * D + 8 * tc) * EB;
#pragma unroll
      for (int u = 0; u < KPT; ++u) {
        if (ok && tok0 + u < key_end) {
          kr[u] = *reinterpret_cast<const raw_t*>(kc + base + static_cast<int64_t>(u) * D * EB);
          vr[u] = *reinterpret_cast<const raw_t*>(vc + base + static_cast<int64_t>(u) * D * EB);
        } else {
          kr[u] = raw_t{};
          vr[u] = raw_t{};
        }
      }
    }
    if constexpr (FP8) {
      if (threadIdx.x < 8) {
        const int b = (k0 >> 4) + (threadIdx.x & 3) - blk_first;
        const int sb = (k0 + 16 * (threadIdx.x & 3)) < key_end ? ids[b] : -1;
        const float* sa = threadIdx.x < 4 ? a.k_scale : a.v_scale;
        sc_reg = static_cast<uint32_t>(sb) < static_cast<uint32_t>(a.num_pool_blocks)
                     ? sa[static_cast<int64_t>(sb) * a.hkv + kvh] : 1.f;
      }
    }
  };
  auto store_tile = [&](int stage) {
    uint16_t* ks = reinterpret_cast<uint16_t*>(smem + stage * L::STAGE);
    uint16_t* vs = ks + 64 * L::KS;
#pragma unroll
    for (int u = 0; u < KPT; ++u) {
      if constexpr (QK8) {
        // keys stay fp8: rows of KS8 bytes
        *reinterpret_cast<raw_t*>(reinterpret_cast<unsigned char*>(ks) + (tk * KPT + u) * L::KS8 + 8 * tc) = kr[u];
      } else {
        *reinterpret_cast<uint4*>(ks + (tk * KPT + u) * L::KS + 8 * tc) = TS::to_bf16(kr[u]);
      }
      if constexpr (!PV8) *reinterpret_cast<uint4*>(vs + (tk * KPT + u) * L::VS + 8 * tc) = TS::to_bf16(vr[u]);
    }
    if constexpr (PV8) {
      // V^T: the thread's four keys 4 tkv + t become byte t of one dword per
      // dimension. In a row, key 32mb + 8j + 4h + t sits at byte
      // 32h + 16mb + 4j + t, so a lane half's 32 keys of the score layout
      // (those with bit 2 equal to h) are one contiguous 32-byte operand.
      unsigned char* vt = reinterpret_cast<unsigned char*>(vs);
      const int pos = 32 * (tkv & 1) + 16 * (tkv >> 3) + 4 * ((tkv & 7) >> 1);
      const uint32_t keep = fmaxf(vsc_reg, 0x1p-100f) < vsmall ? 0u : 0xFFFFFFFFu;
#pragma unroll
      for (int half = 0; half < 2; ++half) {
        const uint32_t x0 = (half ? vr[0].y : vr[0].x) & keep, x1 = (half ? vr[1].y : vr[1].x) & keep;
        const uint32_t x2 = (half ? vr[2].y : vr[2].x) & keep, x3 = (half ? vr[3].y : vr[3].x) & keep;
        const uint32_t t01lo = __builtin_amdgcn_perm(x1, x0, 0x05010400u);   // keys 0, 1 of dims 0, 1
        const uint32_t t01hi = __builtin_amdgcn_perm(x1, x0, 0x07030602u);   // keys 0, 1 of dims 2, 3
        const uint32_t t23lo = __builtin_amdgcn_perm(x3, x2, 0x05010400u);
        const uint32_t t23hi = __builtin_amdgcn_perm(x3, x2, 0x07030602u);
        const uint32_t col[4] = {__builtin_amdgcn_perm(t23lo, t01lo, 0x05040100u),
                                 __builtin_amdgcn_perm(t23lo, t01lo, 0x07060302u),
                                 __builtin_amdgcn_perm(t23hi, t01hi, 0x05040100u),
                                 __builtin_amdgcn_perm(t23hi, t01hi, 0x07060302u)};
#pragma unroll
        for (int d = 0; d < 4; ++d)
          *reinterpret_cast<uint32_t*>(vt + (8 * tcv + 4 * half + d) * L::VT8 + pos) = col[d];
      }
    }
    if constexpr (FP8) {
      // K: the score coefficient of the block; V: its scale enters each
      // probability as 2^(log2 vs) inside the exponential, and the row sum
      // weighs the block by 1/vs. A zero scale (an all-zero block) is taken
      // as 2^-100, which changes no result representable in fp32.
      float* ss = stage_scales + stage * L::NSC;
      if (threadIdx.x < 4) {
        ss[threadIdx.x] = c * sc_reg;
      } else if (threadIdx.x < 8) {
        float v = fmaxf(sc_reg, 0x1p-100f);
        if constexpr (PV8) v = v < vsmall ? vref : v;   // staged as zeros (see vsmall)
        ss[threadIdx.x] = __builtin_amdgcn_logf(v);
        ss[threadIdx.x + 4] = __builtin_amdgcn_rcpf(v);
      }
    }
  };

  auto step = [&](int t, auto mask_tag) {
    constexpr bool MASK = decltype(mask_tag)::value;
    const int k0 = t * 64;
    const int stage = (t - t0) & 1;
    __syncthreads();   // stage `stage` is written; the other stage's readers are done
    if (t + 1 < t1) {
      store_tile(stage ^ 1);
      if (t + 2 < t1) {
        if (t + 2 < t_full) load_tile(k0 + 128, bool_tag<true>{});
        else load_tile(k0 + 128, bool_tag<false>{});
      }
    }
    const uint16_t* ks = reinterpret_cast<const uint16_t*>(smem + stage * L::STAGE);
    const uint16_t* vs = ks + 64 * L::KS;

    // S^T = K Q^T for keys k0..k0+63. All K operands of the tile are read
    // from LDS first, so the reads stream while the MFMAs consume them in order.
    f32x16_t sacc[2];
    if constexpr (QK8) {
      // fp8: K rows of 128 codes against the rounded Q, two 64-dim k-steps
      // per 32 keys on 32x32x64 fp8 MFMAs (unit block scales)
      const unsigned char* k8 = reinterpret_cast<const unsigned char*>(ks);
      v8i_t kop[2][2];
#pragma unroll
      for (int mb = 0; mb < 2; ++mb)
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          const unsigned char* src = k8 + (32 * mb + n) * L::KS8 + 64 * h + 32 * hh;
          const uint4 lo = *reinterpret_cast<const uint4*>(src);
          const uint4 hi = *reinterpret_cast<const uint4*>(src + 16);
          kop[mb][h] = v8i_t{static_cast<int>(lo.x), static_cast<int>(lo.y), static_cast<int>(lo.z),
                             static_cast<int>(lo.w), static_cast<int>(hi.x), static_cast<int>(hi.y),
                             static_cast<int>(hi.z), static_cast<int>(hi.w)};
        }
      __builtin_amdgcn_sched_barrier(0);
      __builtin_amdgcn_s_setprio(0);
#pragma unroll
      for (int mb = 0; mb < 2; ++mb) {
#pragma unroll
        for (int e = 0; e < 16; ++e) sacc[mb][e] = 0.f;
#pragma unroll
        for (int h = 0; h < 2; ++h)
          sacc[mb] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(kop[mb][h], q8[h], sacc[mb], 0, 0, 0, 127, 0, 127);
      }
    } else {
      uint4 kop[2][KSTEPS];
#pragma unroll
      for (int mb = 0; mb < 2; ++mb)
#pragma unroll
        for (int s = 0; s < KSTEPS; ++s)
          kop[mb][s] = *reinterpret_cast<const uint4*>(ks + (32 * mb + n) * L::KS + 16 * s + 8 * hh);
      __builtin_amdgcn_sched_barrier(0);
      // back to normal issue priority for the matrix work (raised below)
      __builtin_amdgcn_s_setprio(0);
#pragma unroll
      for (int mb = 0; mb < 2; ++mb) {
#pragma unroll
        for (int e = 0; e < 16; ++e) sacc[mb][e] = 0.f;
#pragma unroll
        for (int s = 0; s < KSTEPS; ++s)
          sacc[mb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(kop[mb][s]), as_bf16x8(qreg[s]), sacc[mb], 0, 0, 0);
      }
    }
    // V^T operands of the tile, read now so their latency hides behind the
    // softmax. V sits row-major in LDS; the transposing LDS read gives lane i
    // of a 16-lane group element (i % 4) of the 8-byte chunks addressed by
    // lanes i/4, 4 + i/4, 8 + i/4 and 12 + i/4 of its group, so addressing
    // row (lane % 16) / 4 at column 4 (lane % 4) hands each lane four
    // consecutive keys of one dimension: the operand layout of V^T.
    uint4 vop[PV8 ? 1 : 4][PV8 ? 1 : DB];
    // fp8 values: lane (dimension n of a 32-dim block, half hh) takes the 32
    // codes of its dimension for the keys whose bit 2 is hh
    v8i_t vop8[PV8 ? DB : 1];
    if constexpr (PV8) {
      const unsigned char* vt = reinterpret_cast<const unsigned char*>(vs);
#pragma unroll
      for (int db = 0; db < DB; ++db) {
        const unsigned char* src = vt + (32 * db + n) * L::VT8 + 32 * hh;
        const uint4 lo = *reinterpret_cast<const uint4*>(src);
        const uint4 hi = *reinterpret_cast<const uint4*>(src + 16);
        vop8[db] = v8i_t{static_cast<int>(lo.x), static_cast<int>(lo.y), static_cast<int>(lo.z),
                         static_cast<int>(lo.w), static_cast<int>(hi.x), static_cast<int>(hi.y),
                         static_cast<int>(hi.z), static_cast<int>(hi.w)};
      }
    } else {
#pragma unroll
      for (int s = 0; s < 4; ++s)
#pragma unroll
        for (int db = 0; db < DB; ++db) {
          const uint16_t* v0 = vs + (16 * s) * L::VS + 32 * db + v_lane_off;
          const uint2 lo = ds_read_tr16(v0);
          const uint2 hi = ds_read_tr16(v0 + 8 * L::VS);
          vop[s][db] = uint4{lo.x, lo.y, hi.x, hi.y};
        }
    }

    // Entry (mb, i, j) of this lane is key k0 + 32mb + 8i + 4hh + j, which
    // lies in block b = 2mb + i/2 of the tile; b is also the PV step that
    // consumes it. Keys past the row's position (or past key_end) are masked
    // on boundary tiles.
    const int lim = MASK ? min(pos, key_end - 1) - k0 - 4 * hh : 0;
    auto live = [&](int mb, int e) { return !MASK || 32 * mb + 8 * (e >> 2) + (e & 3) <= lim; };
    if constexpr (MASK) {
#pragma unroll
      for (int mb = 0; mb < 2; ++mb)
#pragma unroll
        for (int e = 0; e < 16; ++e)
          if (!live(mb, e)) sacc[mb][e] = -INFINITY;
    }
    // log2-domain coefficient of the raw score, per block (fp8: K scale folded in)
    float coef[4], vlog[4], vinv[4];
#pragma unroll
    for (int b = 0; b < 4; ++b) {
      coef[b] = FP8 ? stage_scales[stage * L::NSC + b] * (QK8 ? qscale : 1.f) : c;
      vlog[b] = FP8 ? stage_scales[stage * L::NSC + 4 + b] : 0.f;
      vinv[b] = FP8 ? stage_scales[stage * L::NSC + 8 + b] : 1.f;
    }
    // row maximum of the scaled scores: block maxima of the raw scores times
    // the (non-negative) block coefficients. The raw scores are finite or
    // -inf (masked), so the NaN-propagating maximum (three operands per
    // instruction, no canonicalising of its inputs) gives the same value;
    // fp8 blocks combine with fmaxf, which drops the NaN of a masked block
    // under a zero key scale.
    float smax;
    if constexpr (FP8) {
      smax = -INFINITY;
#pragma unroll
      for (int b = 0; b < 4; ++b) {
        const int mb = b >> 1, e0 = 8 * (b & 1);
        float bm = sacc[mb][e0];
#pragma unroll
        for (int e = 1; e < 8; ++e) bm = __builtin_elementwise_maximum(bm, sacc[mb][e0 + e]);
        smax = fmaxf(smax, bm * coef[b]);
      }
    } else {
      // one coefficient for the whole tile: one chain over its 32 entries
      smax = sacc[0][0];
#pragma unroll
      for (int e = 1; e < 32; ++e) smax = __builtin_elementwise_maximum(smax, sacc[e >> 4][e & 15]);
      smax *= c;
    }
    smax = max_across_halves(smax);
    const float mn = fmaxf(m_run, smax);
    if (__any(mn > m_run + kSlack)) {
      const float alpha = __builtin_amdgcn_exp2f(m_run - mn);
      l_run *= alpha;
#pragma unroll
      for (int db = 0; db < DB; ++db)
#pragma unroll
        for (int e = 0; e < 16; ++e) acc_o[db][e] *= alpha;
      m_run = mn;
    }

    // p = 2^(s * coef - m) (fp8: times the block's V scale, through its log2),
    // packed to bf16 pairs for the PV MFMAs; the row sum adds exactly the
    // packed values (fp8: weighted back by 1/vs)
    // O^T += V^T P^T, 16 keys (one block) per step; k-slots of lane half hh
    // are keys {16s+4hh+j, 16s+8+4hh+j}, exactly the S^T entries this lane holds
    if constexpr (PV8) {
      // O^T += V^T P^T for all 64 keys at once, one 32x32x64 fp8 MFMA per
      // 32-dim block. Codes p * (vs_b / vref) * 2^kPv8Log2: dword 2s + i of
      // the operand holds block s's entries 4i .. 4i + 3 of this lane, the
      // byte order of the V^T rows. The row sum adds the rounded codes
      // (exact in bf16) weighed back by 1/vs_b.
      v8i_t pop8;
#pragma unroll
      for (int s = 0; s < 4; ++s) {
        const int mb = s >> 1, e0 = 8 * (s & 1);
        const float bias = vlog[s] + vbias - m_run;
        float pv[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const float x = __builtin_amdgcn_exp2f(fmaf(sacc[mb][e0 + e], coef[s], bias));
          pv[e] = live(mb, e0 + e) ? x : 0.f;
        }
        int w0 = __builtin_amdgcn_cvt_pk_fp8_f32(pv[0], pv[1], 0, false);
        w0 = __builtin_amdgcn_cvt_pk_fp8_f32(pv[2], pv[3], w0, true);
        int w1 = __builtin_amdgcn_cvt_pk_fp8_f32(pv[4], pv[5], 0, false);
        w1 = __builtin_amdgcn_cvt_pk_fp8_f32(pv[6], pv[7], w1, true);
        pop8[2 * s] = w0;
        pop8[2 * s + 1] = w1;
        const float bsum = dot2_bf16(fp8x2_to_bf16x2<true>(w1), kBf16PairOne,
                           dot2_bf16(fp8x2_to_bf16x2<false>(w1), kBf16PairOne,
                           dot2_bf16(fp8x2_to_bf16x2<true>(w0), kBf16PairOne,
                           dot2_bf16(fp8x2_to_bf16x2<false>(w0), kBf16PairOne, 0.f))));
        l_run = fmaf(bsum, vinv[s], l_run);
      }
#pragma unroll
      for (int db = 0; db < DB; ++db)
        acc_o[db] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(vop8[db], pop8, acc_o[db], 0, 0, 0, 127, 0, 127);
    } else {
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      const int mb = s >> 1, e0 = 8 * (s & 1);
      const float bias = vlog[s] - m_run;
      float pv[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float x = __builtin_amdgcn_exp2f(fmaf(sacc[mb][e0 + e], coef[s], bias));
        pv[e] = live(mb, e0 + e) ? x : 0.f;
      }
      uint4 pw;
      pw.x = pack_bf16(pv[0], pv[1]);
      pw.y = pack_bf16(pv[2], pv[3]);
      pw.z = pack_bf16(pv[4], pv[5]);
      pw.w = pack_bf16(pv[6], pv[7]);
      // bf16 KV adds the packed probabilities straight into the row sum;
      // fp8 weighs the block's sum by 1/vs first
      const float bsum = dot2_bf16(pw.w, kBf16PairOne, dot2_bf16(pw.z, kBf16PairOne,
                         dot2_bf16(pw.y, kBf16PairOne, dot2_bf16(pw.x, kBf16PairOne, FP8 ? 0.f : l_run))));
      l_run = FP8 ? fmaf(bsum, vinv[s], l_run) : bsum;
      const bf16x8_t pop = as_bf16x8(pw);
#pragma unroll
      for (int db = 0; db < DB; ++db)
        acc_o[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(vop[s][db]), pop, acc_o[db], 0, 0, 0);
    }
    }
    // From here to the next tile's score MFMAs (barrier, staging of the tile
    // after next, reads of the K operands) this wave issues ahead of the
    // other wave of its SIMD, which is then usually in its matrix phase:
    // the memory requests start sooner and the MFMAs fill the gap
    // (measured 2-3 % on prefill-dominated batches).
    __builtin_amdgcn_s_setprio(1);
  };

  if (t0 < t_full) load_tile(t0 * 64, bool_tag<true>{});
  else load_tile(t0 * 64, bool_tag<false>{});
  store_tile(0);
  if (t0 + 1 < t1) {
    if (t0 + 1 < t_full) load_tile((t0 + 1) * 64, bool_tag<true>{});
    else load_tile((t0 + 1) * 64, bool_tag<false>{});
  }
  int t = t0;
  for (; t < t_full; ++t) step(t, bool_tag<false>{});
  for (; t < t1; ++t) step(t, bool_tag<true>{});

  const float l_tot = sum_across_halves(l_run);
  if (it.part < 0) {
    if (!row_ok) return;
    const float inv = 1.f / l_tot;
    const int64_t ooff = (static_cast<int64_t>(it.q_row0 + p) * a.hq + static_cast<int64_t>(kvh) * G + gh) * D;
#pragma unroll
    for (int db = 0; db < DB; ++db)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int dim = 32 * db + 8 * i + 4 * hh;
        if constexpr (OT == AUG_BF16) {
          uint2 w;
          w.x = pack_bf16(acc_o[db][4 * i + 0] * inv, acc_o[db][4 * i + 1] * inv);
          w.y = pack_bf16(acc_o[db][4 * i + 2] * inv, acc_o[db][4 * i + 3] * inv);
          *reinterpret_cast<uint2*>(static_cast<uint16_t*>(a.out) + ooff + dim) = w;
        } else {
          float4 w{acc_o[db][4 * i] * inv, acc_o[db][4 * i + 1] * inv, acc_o[db][4 * i + 2] * inv,
                   acc_o[db][4 * i + 3] * inv};
          *reinterpret_cast<float4*>(static_cast<float*>(a.out) + ooff + dim) = w;
        }
      }
  } else {
    // split tile: unnormalised partial of this row for head gh, merged by
    // the tile merge launch after this one
    if (!row_ok) return;
    float* pp = a.partials + static_cast<int64_t>(it.part + p * it.part_stride) * aug::partial_floats(G, D);
#pragma unroll
    for (int db = 0; db < DB; ++db)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int dim = 32 * db + 8 * i + 4 * hh;
        *reinterpret_cast<float4*>(pp + gh * D + dim) =
            float4{acc_o[db][4 * i], acc_o[db][4 * i + 1], acc_o[db][4 * i + 2], acc_o[db][4 * i + 3]};
      }
    if (hh == 0) {
      // fp8 probabilities carry the item's factor 2^vbias in both the
      // outputs and the row sum: it enters the partial's maximum
      pp[G * D + gh] = PV8 ? m_run - vbias : m_run;
      pp[G * D + G + gh] = l_tot;
    }
  }
}

// ---------------------------------------------------------------------------
// kernels
// ---------------------------------------------------------------------------

template <int D, int G, int NW>
constexpr int row_lds_bytes() { return NW * G * (D + 2) * 4; }

// Whether row items of this instantiation can run on the 16x16 MFMA row
// path (eight or four query heads per KV head, head_dim 128, bf16 or fp8 KV).
template <int KVT, int D, int G, int QT>
constexpr bool row_mfma_capable() {
  return (G == 8 || G == 4) && D == 128 && (KVT == KV_BF16 || KVT == KV_FP8) && QT == AUG_BF16;
}

template <int KVT, int D, int G, int QT, int OT, bool TILES, bool ROW_MFMA, int NW, int F8 = 0>
__device__ __forceinline__ void attn_body(const AttnArgs& a) {
  static_assert(!TILES || NW == kThreads / 64, "tile items run on four-wave workgroups");
  constexpr int RB = row_lds_bytes<D, G, NW>();
  constexpr int TB = TILES ? TileLds<D>::BYTES : 0;
  static_assert(RB >= 4 && (!TILES || TB >= 4), "a split item's workgroup keeps its merge flag in LDS");
  __shared__ __align__(16) unsigned char smem[RB > TB ? RB : TB];
  const WorkItem it = a.items[blockIdx.x];
  if constexpr (TILES) {
    if (it.kind == aug::kTileItem) {
      tile_item<KVT, D, G, OT, F8>(it, a, smem);
      return;
    }
  }
  // row items always fetch a wave's next block while the current one is
  // computed: short spans (small batches) are latency bound otherwise
  if constexpr (ROW_MFMA && row_mfma_capable<KVT, D, G, QT>())
    row_item_mfma<KVT, OT, NW, G>(it, a, reinterpret_cast<float*>(smem));
  else
    row_item<KVT, D, G, QT, OT, true, NW>(it, a, reinterpret_cast<float*>(smem));
}

// Batches without prefill tiles: row items only, on workgroups of NW waves.
template <int KVT, int D, int G, int QT, int OT, bool ROW_MFMA, int NW>
__global__ __launch_bounds__(64 * NW) void attn_rows_kernel(AttnArgs a) {
  attn_body<KVT, D, G, QT, OT, false, ROW_MFMA, NW>(a);
}

// Mixed batches: MFMA tiles and row items in one launch. The tile path's
// accumulators set the register budget (two waves per SIMD); the row path
// spends the same budget on prefetching the next block.
template <int KVT, int D, int G, int QT, int OT, bool ROW_MFMA, int F8>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(2, 2))) void attn_mixed_kernel(AttnArgs a) {
  attn_body<KVT, D, G, QT, OT, true, ROW_MFMA, kThreads / 64, F8>(a);
}

// Merge launch for split prefill tiles: one workgroup per (row, KV head)
// group; the attention launch before it wrote the partials.
template <int D, int G, int OT>
__global__ __launch_bounds__(kThreads) void tile_merge_kernel(AttnArgs a) {
  // Every thread merges four consecutive output dims of one head on its own:
  // it reads each span's (m, l) of that head and its four partial values,
  // all independent loads, and folds them in online (log-sum-exp), so the
  // group costs one memory round trip per eight spans and no barrier. The
  // partials come from the previous launch, so plain loads see them.
  const MergeGroup g = a.groups[blockIdx.x];
  const int64_t pf = aug::partial_floats(G, D);
  const float* base = a.partials + static_cast<int64_t>(g.part0) * pf;
  for (int c = threadIdx.x; c < G * D / 4; c += kThreads) {
    const int h = (4 * c) / D;
    float mx = kNegBig, l = 0.f;
    float4 o = {0.f, 0.f, 0.f, 0.f};
    int s = 0;
    for (; s + 8 <= g.n_parts; s += 8) {
      float ms[8], ls[8];
      float4 os[8];
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        const float* p = base + static_cast<int64_t>(s + k) * pf;
        ms[k] = p[G * D + h];
        ls[k] = p[G * D + G + h];
        os[k] = *reinterpret_cast<const float4*>(p + 4 * c);
      }
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        const float mn = fmaxf(mx, ms[k]);
        const float a0 = __builtin_amdgcn_exp2f(mx - mn), a1 = __builtin_amdgcn_exp2f(ms[k] - mn);
        l = l * a0 + ls[k] * a1;
        o.x = o.x * a0 + os[k].x * a1;
        o.y = o.y * a0 + os[k].y * a1;
        o.z = o.z * a0 + os[k].z * a1;
        o.w = o.w * a0 + os[k].w * a1;
        mx = mn;
      }
    }
    for (; s < g.n_parts; ++s) {
      const float* p = base + static_cast<int64_t>(s) * pf;
      const float ms = p[G * D + h], ls = p[G * D + G + h];
      const float4 os = *reinterpret_cast<const float4*>(p + 4 * c);
      const float mn = fmaxf(mx, ms);
      const float a0 = __builtin_amdgcn_exp2f(mx - mn), a1 = __builtin_amdgcn_exp2f(ms - mn);
      l = l * a0 + ls * a1;
      o.x = o.x * a0 + os.x * a1;
      o.y = o.y * a0 + os.y * a1;
      o.z = o.z * a0 + os.z * a1;
      o.w = o.w * a0 + os.w * a1;
      mx = mn;
    }
    const float inv = 1.f / l;
    const int64_t off = (static_cast<int64_t>(g.q_row) * a.hq + static_cast<int64_t>(g.kvh) * G) * D + 4 * c;
    store_out<OT>(a.out, off + 0, o.x * inv);
    store_out<OT>(a.out, off + 1, o.y * inv);
    store_out<OT>(a.out, off + 2, o.z * inv);
    store_out<OT>(a.out, off + 3, o.w * inv);
  }
}

template <int KVT, int D, int G, int QT, int OT, bool ROW_MFMA>
aug_status launch_rows(const AttnArgs& a, const aug_attn_plan_info& info, hipStream_t st) {
  if (info.num_prefill_items > 0) {
    if constexpr ((KVT == KV_BF16 || KVT == KV_FP8) && QT == AUG_BF16) {
      if (info.tile_path == AUG_TILES_FP8_QK || info.tile_path == AUG_TILES_FP8) {
        if constexpr (KVT == KV_FP8 && D == 128) {
          if (info.tile_path == AUG_TILES_FP8)
            hipLaunchKernelGGL((attn_mixed_kernel<KVT, D, G, QT, OT, ROW_MFMA, 2>), dim3(info.num_items),
                               dim3(kThreads), 0, st, a);
          else
            hipLaunchKernelGGL((attn_mixed_kernel<KVT, D, G, QT, OT, ROW_MFMA, 1>), dim3(info.num_items),
                               dim3(kThreads), 0, st, a);
        } else {
          return aug::fail(AUG_ERR_UNSUPPORTED, "aug_attn_mixed: fp8 tile products need fp8 KV and head_dim 128");
        }
      } else {
        hipLaunchKernelGGL((attn_mixed_kernel<KVT, D, G, QT, OT, ROW_MFMA, 0>), dim3(info.num_items),
                           dim3(kThreads), 0, st, a);
      }
    } else {
      return aug::fail(AUG_ERR_UNSUPPORTED, "aug_attn_mixed: plan has tiles for a dtype set without them");
    }
  } else {
    // MFMA row items without tiles beside them run eight waves per
    // workgroup (the planner gives them spans twice as long): a typical
    // context is then one item merged in LDS instead of two or more spans
    // merged through partials. The VALU row path keeps four waves: its
    // register use would leave a compute unit a single eight-wave workgroup.
    constexpr int NW = ROW_MFMA && row_mfma_capable<KVT, D, G, QT>() ? 8 : 4;
    hipLaunchKernelGGL((attn_rows_kernel<KVT, D, G, QT, OT, ROW_MFMA, NW>), dim3(info.num_items), dim3(64 * NW), 0,
                       st, a);
  }
  return AUG_OK;
}

template <int KVT, int D, int G, int QT, int OT>
aug_status launch(const AttnArgs& a, const aug_attn_plan_info& info, hipStream_t st) {
  if (info.num_items > 0) {
    aug_status rs;
    if constexpr (row_mfma_capable<KVT, D, G, QT>()) {
      rs = info.row_path == AUG_ROWS_VALU ? launch_rows<KVT, D, G, QT, OT, false>(a, info, st)
                                          : launch_rows<KVT, D, G, QT, OT, true>(a, info, st);
    } else {
      rs = launch_rows<KVT, D, G, QT, OT, false>(a, info, st);
    }
    if (rs != AUG_OK) return rs;
    if (hipError_t e = hipGetLastError(); e != hipSuccess)
      return aug::fail(AUG_ERR_HIP, "aug_attn_mixed: launch failed: %s", hipGetErrorString(e));
  }
  if (info.num_tile_merge_groups > 0) {
    hipLaunchKernelGGL((tile_merge_kernel<D, G, OT>), dim3(info.num_tile_merge_groups), dim3(kThreads), 0, st, a);
    if (hipError_t e = hipGetLastError(); e != hipSuccess)
      return aug::fail(AUG_ERR_HIP, "aug_attn_mixed: merge launch failed: %s", hipGetErrorString(e));
  }
  return AUG_OK;
}

template <int KVT, int QT, int OT>
aug_status dispatch_dg(int d, int g, const AttnArgs& a, const aug_attn_plan_info& info,
                       hipStream_t st) {
#define AUG_CASE(DD, GG) \
  if (d == DD && g == GG) return launch<KVT, DD, GG, QT, OT>(a, info, st);
  if constexpr (KVT != KV_FP8) {
    AUG_CASE(64, 1) AUG_CASE(64, 2) AUG_CASE(64, 4) AUG_CASE(64, 8)
  }
  AUG_CASE(128, 1) AUG_CASE(128, 2) AUG_CASE(128, 4) AUG_CASE(128, 8)
#undef AUG_CASE
  return aug::fail(AUG_ERR_UNSUPPORTED, "aug_attn_mixed: head_dim %d with group %d", d, g);
}

// Checks shared by both entry points (everything but the workspace).
aug_status check_call(const char* who, const aug_attn_shape* s, const aug_attn_plan_info* info, void* plan_dev,
                      const void* q, const void* k_cache, const void* v_cache, const float* k_scale,
                      const float* v_scale, const int32_t* block_ids, int32_t num_pool_blocks, void* out) {
  if (aug_status st = aug::check_shape(s, who); st != AUG_OK) return st;
  if (aug_status st = aug::check_plan_info(info, s, who); st != AUG_OK) return st;
  if (info->num_items == 0) return AUG_OK;
  if (!plan_dev || !q || !k_cache || !v_cache || !block_ids || !out)
    return aug::fail(AUG_ERR_INVALID, "%s: NULL device pointer", who);
  if (s->kv_dtype == AUG_FP8_E4M3FN && (!k_scale || !v_scale))
    return aug::fail(AUG_ERR_INVALID, "%s: fp8 KV needs k_scale and v_scale", who);
  if (num_pool_blocks < 1) return aug::fail(AUG_ERR_INVALID, "%s: empty pool", who);
  return AUG_OK;
}

aug_status enqueue(const aug_attn_shape* s, const aug_attn_plan_info* info, void* plan_dev, const void* q,
                   const void* k_cache, const void* v_cache, const float* k_scale, const float* v_scale,
                   const int32_t* block_ids, int32_t num_pool_blocks, void* out, void* workspace,
                   void* stream) {
  AttnArgs a{};
  auto* base = static_cast<unsigned char*>(plan_dev);
  const size_t groups_off = sizeof(aug::PlanHeader) + static_cast<size_t>(info->num_items) * sizeof(WorkItem);
  a.items = reinterpret_cast<const WorkItem*>(base + sizeof(aug::PlanHeader));
  a.groups = reinterpret_cast<const MergeGroup*>(base + groups_off);
  a.counters = reinterpret_cast<int32_t*>(base + groups_off +
                                          static_cast<size_t>(info->num_merge_groups) * sizeof(MergeGroup));
  a.q = q;
  a.k_cache = k_cache;
  a.v_cache = v_cache;
  a.k_scale = k_scale;
  a.v_scale = v_scale;
  a.block_ids = block_ids;
  a.out = out;
  a.partials = static_cast<float*>(workspace);
  a.num_pool_blocks = num_pool_blocks;
  a.hq = s->num_q_heads;
  a.hkv = s->num_kv_heads;
  a.scale_log2 = s->softmax_scale * kLog2e;
  const int g = s->num_q_heads / s->num_kv_heads;
  hipStream_t st = static_cast<hipStream_t>(stream);
  if (s->kv_dtype == AUG_F32) return dispatch_dg<KV_F32, AUG_F32, AUG_F32>(s->head_dim, g, a, *info, st);
  if (s->kv_dtype == AUG_BF16) return dispatch_dg<KV_BF16, AUG_BF16, AUG_BF16>(s->head_dim, g, a, *info, st);
  return dispatch_dg<KV_FP8, AUG_BF16, AUG_BF16>(s->head_dim, g, a, *info, st);
}

}  // namespace

extern "C" aug_status aug_attn_mixed(const aug_attn_shape* s, const aug_attn_plan_info* info,
                                     void* plan_dev, const void* q, const void* k_cache,
                                     const void* v_cache, const float* k_scale, const float* v_scale,
                                     const int32_t* block_ids, int32_t num_pool_blocks, void* out,
                                     void* workspace, size_t workspace_bytes, void* stream) {
  const char* who = "aug_attn_mixed";
  if (aug_status st = check_call(who, s, info, plan_dev, q, k_cache, v_cache, k_scale, v_scale, block_ids,
                                 num_pool_blocks, out);
      st != AUG_OK || info->num_items == 0)
    return st;
  if (info->num_partials > 0 && (!workspace || workspace_bytes < static_cast<size_t>(info->workspace_bytes)))
    return aug::fail(AUG_ERR_NO_SPACE, "%s: workspace %zu < %lld bytes", who, workspace_bytes,
                     (long long)info->workspace_bytes);
  return enqueue(s, info, plan_dev, q, k_cache, v_cache, k_scale, v_scale, block_ids, num_pool_blocks, out,
                 workspace, stream);
}

// ---------------------------------------------------------------------------
// the same launch with the split-K partials in a library-owned device array
// ---------------------------------------------------------------------------

// Device memory for the split-K partials of aug_attn_mixed_noalloc: one copy
// per GPU, held until the process ends. In host code this name stands for the
// array only symbolically; its device address comes from hipGetSymbolAddress.
static __device__ __align__(256) unsigned char scratch[AUG_NOALLOC_SCRATCH_BYTES];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// The device address of `scratch` on the current device, looked up on the
// first call there and kept.
aug_status scratch_on_current_device(void** ptr, const char* who) {
  int dev = -1;
  if (hipError_t e = hipGetDevice(&dev); e != hipSuccess)
    return aug::fail(AUG_ERR_HIP, "%s: hipGetDevice: %s", who, hipGetErrorString(e));
  if (dev < 0 || dev >= kMaxDevices) return aug::fail(AUG_ERR_UNSUPPORTED, "%s: device %d", who, dev);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    if (hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)); e != hipSuccess || !p)
      return aug::fail(AUG_ERR_HIP, "%s: hipGetSymbolAddress of the scratch array: %s", who,
                       hipGetErrorString(e));
    g_scratch_ptr[dev] = p;
  }
  *ptr = g_scratch_ptr[dev];
  return AUG_OK;
}

}  // namespace

extern "C" aug_status aug_attn_mixed_noalloc(const aug_attn_shape* s, const aug_attn_plan_info* info,
                                             void* plan_dev, const void* q, const void* k_cache,
                                             const void* v_cache, const float* k_scale, const float* v_scale,
                                             const int32_t* block_ids, int32_t num_pool_blocks, void* out,
                                             void* stream) {
  const char* who = "aug_attn_mixed_noalloc";
  if (aug_status st = check_call(who, s, info, plan_dev, q, k_cache, v_cache, k_scale, v_scale, block_ids,
                                 num_pool_blocks, out);
      st != AUG_OK || info->num_items == 0)
    return st;
  if (info->workspace_bytes > static_cast<int64_t>(AUG_NOALLOC_SCRATCH_BYTES))
    return aug::fail(AUG_ERR_NO_SPACE, "%s: the plan needs %lld bytes of split-K partials, more than the %lld "
                     "of the library's scratch array (plan with a larger kv_split_tokens, or call "
                     "aug_attn_mixed with a workspace)", who, (long long)info->workspace_bytes,
                     (long long)AUG_NOALLOC_SCRATCH_BYTES);
  void* ws = nullptr;
  if (info->num_partials > 0)
    if (aug_status st = scratch_on_current_device(&ws, who); st != AUG_OK) return st;
  return enqueue(s, info, plan_dev, q, k_cache, v_cache, k_scale, v_scale, block_ids, num_pool_blocks, out, ws,
                 stream);
}
