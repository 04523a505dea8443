// Host planner of the mixed-batch attention launch.
//
// It turns a formed batch (per request: query rows, context length, block
// table) into a work list for one kernel launch:
//  * chunked-prefill requests with bf16 Q/K/V become MFMA tiles of
//    kTileRows query rows (positions x the G query heads of one KV head),
//    each reading keys 0 .. its last row's position;
//  * every other row (decodes, and prefill rows of dtype sets without an MFMA
//    path) becomes row items: one row, the G heads of one KV head, and a span
//    of keys; long contexts are split into spans of nearly equal length whose
//    partial softmax states a second launch merges (split-K).
// Items are ordered longest first so the long ones start early. The planner
// is deterministic and validates the batch completely before any launch.

#include <algorithm>
#include <cstdint>
#include <cmath>
#include <cstring>
#include <vector>

#include "aug.h"
#include "checks.h"
#include "plan_format.h"
#include "status.h"

namespace aug {

bool dtype_set_supported(const aug_attn_shape& s) {
  if (s.q_dtype == AUG_F32 && s.kv_dtype == AUG_F32 && s.out_dtype == AUG_F32) return true;
  if (s.q_dtype == AUG_BF16 && s.kv_dtype == AUG_BF16 && s.out_dtype == AUG_BF16) return true;
  if (s.q_dtype == AUG_BF16 && s.kv_dtype == AUG_FP8_E4M3FN && s.out_dtype == AUG_BF16) return true;
  return false;
}

bool row_mfma_supported(const aug_attn_shape& s) {
  return (s.num_q_heads == 8 * s.num_kv_heads || s.num_q_heads == 4 * s.num_kv_heads) && s.head_dim == 128 && s.q_dtype == AUG_BF16 &&
         (s.kv_dtype == AUG_BF16 || s.kv_dtype == AUG_FP8_E4M3FN);
}

bool tiles_supported(const aug_attn_shape& s) {
  return s.q_dtype == AUG_BF16 && (s.kv_dtype == AUG_BF16 || s.kv_dtype == AUG_FP8_E4M3FN);
}

// fp8 score products on the tiles: fp8 keys (head_dim 128) and bf16 queries
bool tile_fp8qk_supported(const aug_attn_shape& s) {
  return s.q_dtype == AUG_BF16 && s.kv_dtype == AUG_FP8_E4M3FN && s.head_dim == 128;
}

aug_status check_shape(const aug_attn_shape* s, const char* who) {
  if (!s) return fail(AUG_ERR_INVALID, "%s: shape is NULL", who);
  if (s->num_q_heads < 1 || s->num_kv_heads < 1 || s->num_q_heads % s->num_kv_heads != 0)
    return fail(AUG_ERR_INVALID, "%s: heads %d/%d are not a positive multiple", who,
                s->num_q_heads, s->num_kv_heads);
  if (s->num_kv_heads > 1024)
    return fail(AUG_ERR_UNSUPPORTED, "%s: %d KV heads (supported: up to 1024)", who, s->num_kv_heads);
  const int g = s->num_q_heads / s->num_kv_heads;
  if (g != 1 && g != 2 && g != 4 && g != 8)
    return fail(AUG_ERR_UNSUPPORTED, "%s: group size %d (supported: 1, 2, 4, 8)", who, g);
  if (s->head_dim != 64 && s->head_dim != 128)
    return fail(AUG_ERR_UNSUPPORTED, "%s: head_dim %d (supported: 64, 128)", who, s->head_dim);
  if (s->block_size != kBlock)
    return fail(AUG_ERR_UNSUPPORTED, "%s: block_size %d (supported: 16)", who, s->block_size);
  if (!dtype_set_supported(*s))
    return fail(AUG_ERR_UNSUPPORTED, "%s: dtype set q=%d kv=%d out=%d", who, s->q_dtype,
                s->kv_dtype, s->out_dtype);
  if (s->kv_dtype == AUG_FP8_E4M3FN && s->head_dim != 128)
    return fail(AUG_ERR_UNSUPPORTED, "%s: fp8 KV needs head_dim 128", who);
  if (!std::isfinite(s->softmax_scale) || !(s->softmax_scale > 0.f))
    return fail(AUG_ERR_INVALID, "%s: softmax_scale must be finite and positive", who);
  return AUG_OK;
}

aug_status check_plan_info(const aug_attn_plan_info* info, const aug_attn_shape* s, const char* who) {
  if (!info) return fail(AUG_ERR_INVALID, "%s: info is NULL", who);
  if (info->num_items < 0 || info->num_merge_groups < 0 || info->num_partials < 0 ||
      info->num_tile_merge_groups < 0 || info->num_tile_merge_groups > info->num_merge_groups ||
      info->num_append_items < 0 || info->num_prefill_items < 0 || info->num_prefill_items > info->num_items ||
      info->workspace_bytes < 0 ||
      info->plan_bytes != plan_image_bytes(info->num_items, info->num_merge_groups, info->num_append_items))
    return fail(AUG_ERR_INVALID, "%s: info is not consistent with a plan image", who);
  if (info->num_q_heads != s->num_q_heads || info->num_kv_heads != s->num_kv_heads ||
      info->head_dim != s->head_dim || info->q_dtype != s->q_dtype || info->kv_dtype != s->kv_dtype ||
      info->out_dtype != s->out_dtype)
    return fail(AUG_ERR_INVALID,
                "%s: the plan was built for heads %d/%d, head_dim %d, dtypes %d/%d/%d; called with "
                "%d/%d, %d, %d/%d/%d",
                who, info->num_q_heads, info->num_kv_heads, info->head_dim, info->q_dtype, info->kv_dtype,
                info->out_dtype, s->num_q_heads, s->num_kv_heads, s->head_dim, s->q_dtype, s->kv_dtype,
                s->out_dtype);
  if (info->row_path != AUG_ROWS_VALU && !(info->row_path == AUG_ROWS_MFMA && row_mfma_supported(*s)))
    return fail(AUG_ERR_INVALID, "%s: info names row path %d, which this shape cannot run", who, info->row_path);
  if (info->tile_path != AUG_TILES_BF16 &&
      !((info->tile_path == AUG_TILES_FP8_QK || info->tile_path == AUG_TILES_FP8) && tile_fp8qk_supported(*s)))
    return fail(AUG_ERR_INVALID, "%s: info names tile path %d, which this shape cannot run", who,
                info->tile_path);
  return AUG_OK;
}

namespace {

struct Sized {
  WorkItem item;
  double weight;    // estimated ns: longest first
  int64_t order;    // creation order, to keep the sort deterministic
};

// Estimated run time of a work item while the GPU is full (about 512
// workgroups resident, two per compute unit), used to order items longest
// first (so prefill tiles, compute bound, run beside decode spans, memory
// bound, and no long item starts last) and to choose how far to split long
// tiles. Calibrated on MI355X: a row item streams its K/V at about 11.5 GB/s
// per resident workgroup (5.9 TB/s over 512); a tile item costs about 3 us
// of set-up and write-out plus 2.6 us per 64-key step of its 128 rows; the
// split-K merge launch about 5 us plus its partials read at 1.5 TB/s.
constexpr int kSlots = 512;
double row_item_ns(int64_t keys, int32_t head_dim, int32_t kv_bytes) {
  return static_cast<double>(keys) * head_dim * kv_bytes * 2 / 11.5;
}
double tile_item_ns(int64_t key_tiles) { return 3000.0 + static_cast<double>(key_tiles) * 2600.0; }
double merge_ns(int64_t partial_bytes) {
  return partial_bytes > 0 ? 5000.0 + static_cast<double>(partial_bytes) / 1500.0 : 0.0;
}

// Lower bound of a launch's makespan on kSlots slots: its longest item, or
// its total work spread evenly.
double makespan_bound(double longest, double total) { return std::max(longest, total / kSlots); }

int32_t choose_split(int64_t total_row_keys, int32_t requested, bool wide_rows, bool rows_only) {
  if (requested > 0) return ((requested + kBlock - 1) / kBlock) * kBlock;   // requested <= kMaxSplit
  // About four row items per compute unit (256 CUs), but never spans under
  // 512 keys (on small batches an item's fixed latency, query load, state
  // merge and partial write, outweighs shorter streams); on large batches
  // spans of 4096 keys, long enough that those fixed costs are a few percent
  // of an item's streaming time while lognormal context mixes still balance.
  // Eight-wave row items (MFMA rows without tiles) take spans twice as long,
  // so that each wave streams as many keys as in a four-wave item. Four-wave
  // row items of a launch without tiles go up to 6144 keys (measured 3.5 %
  // faster on 64 decodes over 16k-32k keys; beside tiles 4096 stays best).
  const int32_t f = wide_rows ? 2 : 1;
  int64_t s = (total_row_keys + 1024 / f - 1) / (1024 / f);
  s = std::max<int64_t>(s, 512 * f);
  s = std::min<int64_t>(s, wide_rows ? 8192 : rows_only ? 6144 : 4096);
  return static_cast<int32_t>(((s + kBlock - 1) / kBlock) * kBlock);
}

}  // namespace
}  // namespace aug

using namespace aug;

extern "C" aug_status aug_attn_plan(const aug_attn_shape* s, const aug_batch_desc* b,
                                    int32_t kv_split_tokens, void* plan_host, size_t plan_cap,
                                    aug_attn_plan_info* info) {
  const aug_plan_options opts{kv_split_tokens, AUG_ROWS_AUTO, AUG_TILES_AUTO, 0};
  return aug_attn_plan_opts(s, b, &opts, plan_host, plan_cap, info);
}

extern "C" aug_status aug_attn_plan_opts(const aug_attn_shape* s, const aug_batch_desc* b,
                                         const aug_plan_options* opts, void* plan_host, size_t plan_cap,
                                         aug_attn_plan_info* info) {
  const char* who = "aug_attn_plan";
  if (aug_status st = check_shape(s, who); st != AUG_OK) return st;
  if (!opts) return fail(AUG_ERR_INVALID, "%s: options are NULL", who);
  if (opts->reserved != 0) return fail(AUG_ERR_INVALID, "%s: the reserved option field must be zero", who);
  const int32_t kv_split_tokens = opts->kv_split_tokens;
  int32_t row_path = opts->row_path;
  if (row_path != AUG_ROWS_AUTO && row_path != AUG_ROWS_VALU && row_path != AUG_ROWS_MFMA)
    return fail(AUG_ERR_INVALID, "%s: unknown row path %d", who, row_path);
  if (row_path == AUG_ROWS_MFMA && !row_mfma_supported(*s))
    return fail(AUG_ERR_UNSUPPORTED, "%s: the MFMA row path needs 8 or 4 query heads per KV head, head_dim 128 "
                "and bf16 or fp8 KV", who);
  // AUTO takes the MFMA rows only for eight-head groups, where the vector ALUs
  // cannot keep up with the KV stream; four-head groups stay on the vector ALUs
  // unless asked for
  if (row_path == AUG_ROWS_AUTO)
    row_path = row_mfma_supported(*s) && s->num_q_heads == 8 * s->num_kv_heads ? AUG_ROWS_MFMA : AUG_ROWS_VALU;
  int32_t tile_path = opts->tile_path;
  if (tile_path != AUG_TILES_AUTO && tile_path != AUG_TILES_BF16 && tile_path != AUG_TILES_FP8_QK &&
      tile_path != AUG_TILES_FP8)
    return fail(AUG_ERR_INVALID, "%s: unknown tile path %d", who, tile_path);
  if ((tile_path == AUG_TILES_FP8_QK || tile_path == AUG_TILES_FP8) && !tile_fp8qk_supported(*s))
    return fail(AUG_ERR_UNSUPPORTED, "%s: fp8 tile products need fp8 KV, bf16 queries and head_dim 128", who);
  if (tile_path == AUG_TILES_AUTO) tile_path = AUG_TILES_BF16;   // fp8 tile products are opt-in
  if (!b || !info) return fail(AUG_ERR_INVALID, "%s: batch or info is NULL", who);
  const int32_t n = b->num_reqs;
  if (n < 0) return fail(AUG_ERR_INVALID, "%s: num_reqs %d < 0", who, n);
  if (n > 0 && (!b->q_start || !b->ctx_len || !b->bt_start))
    return fail(AUG_ERR_INVALID, "%s: batch arrays are NULL", who);
  if (b->num_pool_blocks < 1) return fail(AUG_ERR_INVALID, "%s: empty pool", who);
  if (kv_split_tokens > kMaxSplit)
    return fail(AUG_ERR_INVALID, "%s: kv_split_tokens %d > %d", who, kv_split_tokens, kMaxSplit);
  if (n > 0 && b->q_start[0] != 0) return fail(AUG_ERR_INVALID, "%s: q_start[0] != 0", who);
  const int32_t hkv = s->num_kv_heads;
  const int32_t g = s->num_q_heads / hkv;
  int64_t total_row_keys = 0;
  bool any_tiled = false;
  for (int32_t r = 0; r < n; ++r) {
    const int64_t q = static_cast<int64_t>(b->q_start[r + 1]) - b->q_start[r];
    const int64_t ctx = b->ctx_len[r];
    if (q < 1) return fail(AUG_ERR_INVALID, "%s: request %d has %lld rows", who, r, (long long)q);
    if (ctx < q)
      return fail(AUG_ERR_INVALID, "%s: request %d has ctx_len %lld < rows %lld", who, r,
                  (long long)ctx, (long long)q);
    if (ctx > kMaxContext)
      return fail(AUG_ERR_UNSUPPORTED, "%s: request %d has ctx_len %lld > %d", who, r, (long long)ctx,
                  kMaxContext);
    const int64_t need = (ctx + kBlock - 1) / kBlock;
    const int64_t have = static_cast<int64_t>(b->bt_start[r + 1]) - b->bt_start[r];
    if (b->bt_start[r] < 0 || have < need)
      return fail(AUG_ERR_INVALID, "%s: request %d lists %lld blocks, needs %lld", who, r,
                  (long long)have, (long long)need);
    if (b->block_ids) {
      for (int64_t i = 0; i < need; ++i) {
        const int32_t id = b->block_ids[b->bt_start[r] + i];
        if (id < 0 || id >= b->num_pool_blocks)
          return fail(AUG_ERR_INVALID, "%s: request %d block %lld is %d, pool has %d", who, r,
                      (long long)i, id, b->num_pool_blocks);
      }
    }
    const bool tiled = q > 1 && tiles_supported(*s);
    any_tiled = any_tiled || tiled;
    if (!tiled) {
      // rows at positions ctx-q .. ctx-1 read pos+1 keys each
      total_row_keys += (q * (2 * ctx - q + 1) / 2) * hkv;
    }
  }
  const int64_t total_rows = n > 0 ? b->q_start[n] : 0;
  if (total_rows > (int64_t{1} << 30))
    return fail(AUG_ERR_UNSUPPORTED, "%s: %lld rows", who, (long long)total_rows);

  // blocks that receive this step's new K/V rows (aug_kv_append); with the
  // host block table, no block may receive tokens of two requests (or twice
  // from one), which concurrent appends could not merge
  int64_t n_append = 0;
  for (int32_t r = 0; r < n; ++r) {
    const int64_t first = b->ctx_len[r] - (b->q_start[r + 1] - b->q_start[r]);
    n_append += (b->ctx_len[r] - 1) / kBlock - first / kBlock + 1;
  }
  if (b->block_ids && n_append > 0) {
    std::vector<int32_t> touched;
    touched.reserve(static_cast<size_t>(n_append));
    for (int32_t r = 0; r < n; ++r) {
      const int64_t first = b->ctx_len[r] - (b->q_start[r + 1] - b->q_start[r]);
      for (int64_t blk = first / kBlock; blk <= (b->ctx_len[r] - 1) / kBlock; ++blk)
        touched.push_back(b->block_ids[b->bt_start[r] + blk]);
    }
    std::sort(touched.begin(), touched.end());
    const auto dup = std::adjacent_find(touched.begin(), touched.end());
    if (dup != touched.end())
      return fail(AUG_ERR_INVALID, "%s: block %d receives new tokens more than once", who, *dup);
  }

  // a launch without tiles runs MFMA row items on eight-wave workgroups
  const int32_t split = choose_split(total_row_keys, kv_split_tokens, !any_tiled && row_path == AUG_ROWS_MFMA, !any_tiled);
  const int32_t pos_per_tile = kTileRows / g;
  const int32_t kv_bytes_all = s->kv_dtype == AUG_F32 ? 4 : s->kv_dtype == AUG_BF16 ? 2 : 1;

  // Keys per span of a split prefill tile. Splitting evens out the items but
  // costs a partial per row and span and their merge, so each candidate span
  // is priced as the makespan of the whole launch (row items included) plus
  // its merge, and the cheapest wins (ties: the longer span).
  int32_t tile_span = kTileSpanMax;
  int32_t longest_tile = 0;
  for (int32_t r = 0; r < n && tiles_supported(*s); ++r)
    if (b->q_start[r + 1] - b->q_start[r] > 1) longest_tile = std::max(longest_tile, b->ctx_len[r]);
  if (longest_tile > kTileSpanMin) {
    double row_total = 0.0, row_longest = 0.0;
    int64_t row_partial_bytes = 0;
    for (int32_t r = 0; r < n; ++r) {
      const int32_t q = b->q_start[r + 1] - b->q_start[r];
      if (q > 1) continue;
      const int32_t ctx = b->ctx_len[r];
      const int32_t nspan = (ctx + split - 1) / split;
      const int32_t span = (((ctx + nspan - 1) / nspan + kBlock - 1) / kBlock) * kBlock;
      const int32_t nsp = (ctx + span - 1) / span;
      const double t = row_item_ns(std::min(span, ctx), s->head_dim, kv_bytes_all);
      row_longest = std::max(row_longest, t);
      row_total += row_item_ns(ctx, s->head_dim, kv_bytes_all) * hkv;
      if (nsp > 1) row_partial_bytes += static_cast<int64_t>(nsp) * hkv * partial_floats(g, s->head_dim) * 4;
    }
    double best = 0.0;
    bool have = false;
    for (const int32_t cand : {kTileSpanMax, 4096, 2048, 1024, 512, kTileSpanMin}) {
      if (have && longest_tile <= cand) continue;   // nothing splits: same as the longer span
      if (have && longest_tile / cand > 1024) continue;   // at most ~1k spans per tile row
      double total = row_total, longest = row_longest;
      int64_t partial_bytes = row_partial_bytes;
      for (int32_t r = 0; r < n; ++r) {
        const int32_t q = b->q_start[r + 1] - b->q_start[r];
        if (q <= 1) continue;
        const int32_t ctx = b->ctx_len[r];
        for (int32_t j0 = 0; j0 < q; j0 += pos_per_tile) {
          const int32_t nr = std::min(pos_per_tile, q - j0);
          const int32_t key_end = ctx - q + j0 + nr;
          const int32_t nsplit = (key_end + cand - 1) / cand;
          const int32_t span = (((key_end + nsplit - 1) / nsplit + kKeyTile - 1) / kKeyTile) * kKeyTile;
          const int32_t nsp = (key_end + span - 1) / span;
          longest = std::max(longest, tile_item_ns((std::min(span, key_end) + kKeyTile - 1) / kKeyTile));
          total += (tile_item_ns(0) * nsp + tile_item_ns((key_end + kKeyTile - 1) / kKeyTile) - tile_item_ns(0)) * hkv;
          if (nsp > 1) partial_bytes += static_cast<int64_t>(nr) * nsp * hkv * partial_floats(g, s->head_dim) * 4;
        }
      }
      const double cost = makespan_bound(longest, total) + merge_ns(partial_bytes);
      if (!have || cost < best) {
        best = cost;
        tile_span = cand;
        have = true;
      }
    }
  }

  // Row items: a request's spans are equal (within one block), so ordering
  // requests by span length orders their items longest first.
  struct RowReq {
    int32_t r, span, nspan;
    double ns;      // estimated time of one of its items
  };
  const int32_t kv_bytes = s->kv_dtype == AUG_F32 ? 4 : s->kv_dtype == AUG_BF16 ? 2 : 1;
  std::vector<RowReq> row_reqs;
  std::vector<Sized> tiles;
  std::vector<MergeGroup> tile_groups;
  int64_t n_row_items = 0, n_groups = 0, tile_parts = 0, row_parts = 0;
  int64_t order = 0;
  for (int32_t r = 0; r < n; ++r) {
    const int32_t q = b->q_start[r + 1] - b->q_start[r];
    const int32_t ctx = b->ctx_len[r];
    if (q > 1 && tiles_supported(*s)) {
      for (int32_t j0 = 0; j0 < q; j0 += pos_per_tile) {
        const int32_t nr = std::min(pos_per_tile, q - j0);
        const int32_t pos0 = ctx - q + j0;
        const int32_t key_end = pos0 + nr;
        // long tiles are split into near-equal spans of whole key tiles; each
        // row of a split tile then has one partial per span, stored together
        const int32_t nsplit = (key_end + tile_span - 1) / tile_span;
        int32_t span = (key_end + nsplit - 1) / nsplit;
        span = ((span + kKeyTile - 1) / kKeyTile) * kKeyTile;
        const int32_t nsp = (key_end + span - 1) / span;
        static_assert(kTileSpanMax % kKeyTile == 0 && kTileSpanMin % kKeyTile == 0,
                      "tile spans are whole key tiles");
        // span <= tile_span <= kTileSpanMax, so the kernel's per-item block-id buffer suffices
        for (int32_t h = 0; h < hkv; ++h) {
          const int32_t g0 = static_cast<int32_t>(tile_groups.size());
          for (int32_t sidx = 0; sidx < nsp; ++sidx) {
            WorkItem it{};
            it.kvh = static_cast<int16_t>(h);
            it.kind = kTileItem;
            it.q_row0 = b->q_start[r] + j0;
            it.n_rows = static_cast<int16_t>(nr);
            it.part_stride = static_cast<int16_t>(nsp);
            it.key_begin = sidx * span;
            it.key_end = std::min(key_end, (sidx + 1) * span);
            it.pos0 = pos0;
            it.bt_off = b->bt_start[r];
            it.part = nsp > 1 ? static_cast<int32_t>(tile_parts) + sidx : -1;
            it.group = nsp > 1 ? g0 : -1;
            const int64_t steps = (it.key_end - it.key_begin + kKeyTile - 1) / kKeyTile;
            tiles.push_back({it, tile_item_ns(steps), order++});
          }
          if (nsp > 1) {
            for (int32_t j = 0; j < nr; ++j)
              tile_groups.push_back(MergeGroup{b->q_start[r] + j0 + j, h,
                                               static_cast<int32_t>(tile_parts) + j * nsp, nsp});
            tile_parts += static_cast<int64_t>(nr) * nsp;
            n_groups += nr;
          }
        }
      }
      continue;
    }
    // decodes have one row; rows of an untiled prefill get spans of their own length
    const int32_t keys = ctx;  // the longest row of the request
    const int32_t nspan = (keys + split - 1) / split;
    int32_t span = (keys + nspan - 1) / nspan;
    span = ((span + kBlock - 1) / kBlock) * kBlock;
    row_reqs.push_back({r, span, (keys + span - 1) / span, row_item_ns(span, s->head_dim, kv_bytes)});
    for (int32_t j = 0; j < q; ++j) {
      const int32_t k = ctx - q + j + 1;
      const int64_t ns = (k + span - 1) / span;
      n_row_items += ns * hkv;
      if (ns > 1) {
        n_groups += hkv;
        row_parts += ns * hkv;
      }
    }
  }
  std::sort(tiles.begin(), tiles.end(), [](const Sized& a, const Sized& c) {
    if (a.weight != c.weight) return a.weight > c.weight;
    return a.order < c.order;
  });
  std::stable_sort(row_reqs.begin(), row_reqs.end(),
                   [](const RowReq& a, const RowReq& c) { return a.ns > c.ns; });
  (void)order;

  const int64_t n_items = static_cast<int64_t>(tiles.size()) + n_row_items;
  if (n_items > (int64_t{1} << 30))
    return fail(AUG_ERR_UNSUPPORTED, "%s: %lld work items", who, (long long)n_items);
  const int64_t items_off = sizeof(PlanHeader);
  const int64_t groups_off = items_off + n_items * static_cast<int64_t>(sizeof(WorkItem));
  const int64_t n_parts = tile_parts + row_parts;
  if (n_parts > (int64_t{1} << 30))
    return fail(AUG_ERR_UNSUPPORTED, "%s: %lld split-K partials", who, (long long)n_parts);
  const int64_t counters_off = groups_off + n_groups * static_cast<int64_t>(sizeof(MergeGroup));
  const int64_t append_off = append_offset(n_items, n_groups);
  const int64_t plan_bytes = plan_image_bytes(n_items, n_groups, n_append);
  if (plan_bytes > INT32_MAX)
    return fail(AUG_ERR_UNSUPPORTED, "%s: plan image of %lld bytes", who, (long long)plan_bytes);
  const int64_t ws = ((n_parts * partial_floats(g, s->head_dim) * 4 + 255) / 256) * 256;

  std::memset(info, 0, sizeof(*info));
  info->plan_bytes = plan_bytes;
  info->workspace_bytes = ws;
  info->num_items = static_cast<int32_t>(n_items);
  info->num_prefill_items = static_cast<int32_t>(tiles.size());
  info->num_merge_groups = static_cast<int32_t>(n_groups);
  info->num_partials = static_cast<int32_t>(n_parts);
  info->kv_split_tokens = split;
  info->total_rows = static_cast<int32_t>(total_rows);
  info->num_reqs = n;
  info->num_tile_merge_groups = static_cast<int32_t>(tile_groups.size());
  info->num_append_items = static_cast<int32_t>(n_append);
  info->num_q_heads = s->num_q_heads;
  info->num_kv_heads = hkv;
  info->head_dim = s->head_dim;
  info->q_dtype = s->q_dtype;
  info->kv_dtype = s->kv_dtype;
  info->out_dtype = s->out_dtype;
  info->row_path = row_path;
  info->tile_path = tile_path;
  if (!plan_host) return AUG_OK;
  if (plan_cap < static_cast<size_t>(plan_bytes))
    return fail(AUG_ERR_NO_SPACE, "%s: plan buffer %zu < %lld bytes", who, plan_cap,
                (long long)plan_bytes);

  auto* base = static_cast<unsigned char*>(plan_host);
  PlanHeader hdr{};
  hdr.magic = kPlanMagic;
  hdr.version = kPlanVersion;
  hdr.num_items = info->num_items;
  hdr.num_tile_items = info->num_prefill_items;
  hdr.num_groups = info->num_merge_groups;
  hdr.num_partials = info->num_partials;
  hdr.kv_split = split;
  hdr.total_rows = info->total_rows;
  hdr.items_offset = static_cast<int32_t>(items_off);
  hdr.groups_offset = static_cast<int32_t>(groups_off);
  hdr.counters_offset = static_cast<int32_t>(counters_off);
  hdr.append_offset = static_cast<int32_t>(append_off);
  hdr.num_append_items = static_cast<int32_t>(n_append);
  hdr.num_q_heads = static_cast<int16_t>(s->num_q_heads);
  hdr.num_kv_heads = static_cast<int16_t>(hkv);
  hdr.head_dim = static_cast<int16_t>(s->head_dim);
  hdr.q_dtype = static_cast<int8_t>(s->q_dtype);
  hdr.kv_dtype = static_cast<int8_t>(s->kv_dtype);
  hdr.out_dtype = static_cast<int8_t>(s->out_dtype);
  hdr.row_path = static_cast<int8_t>(row_path);
  hdr.tile_path = static_cast<int8_t>(tile_path);
  std::memcpy(base, &hdr, sizeof(hdr));
  auto* items = reinterpret_cast<WorkItem*>(base + items_off);
  auto* groups = reinterpret_cast<MergeGroup*>(base + groups_off);
  size_t k = 0;
  int32_t ng = 0;
  for (const MergeGroup& mg : tile_groups) groups[ng++] = mg;
  int32_t parts = static_cast<int32_t>(tile_parts);
  size_t ti = 0;
  auto emit_tiles_longer_than = [&](double ns) {
    while (ti < tiles.size() && tiles[ti].weight >= ns) items[k++] = tiles[ti++].item;
  };
  for (const RowReq& rr : row_reqs) {
    emit_tiles_longer_than(rr.ns);
    const int32_t r = rr.r;
    const int32_t q = b->q_start[r + 1] - b->q_start[r];
    const int32_t ctx = b->ctx_len[r];
    for (int32_t j = 0; j < q; ++j) {
      const int32_t pos = ctx - q + j;
      const int32_t keys = pos + 1;
      const int32_t nspan = (keys + rr.span - 1) / rr.span;
      for (int32_t h = 0; h < hkv; ++h) {
        const int32_t part0 = nspan > 1 ? parts : -1;
        const int32_t group = nspan > 1 ? ng : -1;
        if (nspan > 1) {
          groups[ng++] = MergeGroup{b->q_start[r] + j, h, part0, nspan};
          parts += nspan;
        }
        for (int32_t sidx = 0; sidx < nspan; ++sidx) {
          WorkItem it{};
          it.kvh = static_cast<int16_t>(h);
          it.kind = kRowItem;
          it.q_row0 = b->q_start[r] + j;
          it.n_rows = 1;
          it.part_stride = 1;
          it.key_begin = sidx * rr.span;
          it.key_end = std::min(keys, (sidx + 1) * rr.span);
          it.pos0 = pos;
          it.bt_off = b->bt_start[r];
          it.part = nspan > 1 ? part0 + sidx : -1;
          it.group = group;
          items[k++] = it;
        }
      }
    }
  }
  emit_tiles_longer_than(-1.0);
  std::memset(base + counters_off, 0, static_cast<size_t>(append_off - counters_off));
  auto* app = reinterpret_cast<AppendItem*>(base + append_off);
  int64_t na = 0;
  for (int32_t r = 0; r < n; ++r) {
    const int32_t first = b->ctx_len[r] - (b->q_start[r + 1] - b->q_start[r]);
    for (int32_t p = first; p < b->ctx_len[r];) {
      const int32_t blk = p / kBlock;
      const int32_t end = std::min(b->ctx_len[r], (blk + 1) * kBlock);
      app[na++] = AppendItem{b->q_start[r] + (p - first), static_cast<int16_t>(end - p),
                             static_cast<int16_t>(p % kBlock), b->bt_start[r] + blk, 0};
      p = end;
    }
  }
  return AUG_OK;
}

extern "C" aug_status aug_attn_workspace_size(const aug_attn_shape* s, const aug_batch_desc* b,
                                              int32_t kv_split_tokens, size_t* bytes) {
  if (!bytes) return fail(AUG_ERR_INVALID, "aug_attn_workspace_size: bytes is NULL");
  aug_attn_plan_info info;
  if (aug_status st = aug_attn_plan(s, b, kv_split_tokens, nullptr, 0, &info); st != AUG_OK) return st;
  *bytes = static_cast<size_t>(info.workspace_bytes);
  return AUG_OK;
}
