// Work-list ("plan image") of one attention launch, written by the host
// planner and read by the kernels. Plain data, position independent.
#pragma once

#include <cstdint>

namespace aug {

constexpr int32_t kPlanMagic = 0x4E4C5041;  // "APLN"
constexpr int32_t kPlanVersion = 4;
constexpr int32_t kBlock = 16;              // tokens per KV block
constexpr int32_t kKeyTile = 64;            // keys per MFMA tile (4 blocks)
constexpr int32_t kTileRows = 128;          // query rows (positions x group heads) per MFMA tile
constexpr int32_t kTileSpanMin = 256;       // a tile is never split into spans shorter than this
constexpr int32_t kTileSpanMax = 8192;      // longest key span of one tile item (its block ids fit in LDS)
constexpr int32_t kMaxContext = 1 << 24;    // longest context of one request the planner accepts
constexpr int32_t kMaxSplit = 1 << 24;      // largest requested decode split (keys per work item)

enum ItemKind : int32_t {
  kRowItem = 0,   // one query row (all heads of one KV head group) against a key span, VALU
  kTileItem = 1,  // a tile of consecutive query rows of one chunk, causal, MFMA
};

struct PlanHeader {          // 64 bytes
  int32_t magic;
  int32_t version;
  int32_t num_items;
  int32_t num_tile_items;
  int32_t num_groups;
  int32_t num_partials;
  int32_t kv_split;
  int32_t total_rows;
  int32_t items_offset;      // bytes from the start of the image
  int32_t groups_offset;
  int32_t counters_offset;   // int32 per merge group, zero in the image
  int32_t append_offset;     // AppendItem list (16-byte aligned)
  int32_t num_append_items;
  // the layer shape the image was planned for
  int16_t num_q_heads;
  int16_t num_kv_heads;
  int16_t head_dim;
  int8_t q_dtype;
  int8_t kv_dtype;
  int8_t out_dtype;
  int8_t row_path;           // aug_row_path of the row items (resolved)
  int8_t tile_path;          // aug_tile_path of the prefill tiles (resolved)
  int8_t reserved1;
};

struct WorkItem {            // 48 bytes
  int16_t kvh;               // KV head
  int8_t kind;               // ItemKind
  int8_t reserved0;
  int32_t q_row0;            // first global row of Q/O
  int16_t n_rows;            // rows (context positions) in the item
  int16_t part_stride;       // tiles: distance between the partial slots of consecutive rows
  int32_t key_begin;         // first key (row items: multiple of kBlock; tiles: of kKeyTile)
  int32_t key_end;           // one past the last key any row reads
  int32_t pos0;              // context position of the first row
  int32_t bt_off;            // offset of the request's block table in block_ids
  int32_t part;              // partial slot of the first row, -1 = write O directly
  // split items: merge group of the first row (the item's rows own groups
  // group .. group + n_rows - 1, which share their spans); that group's
  // counter counts finished spans and its n_parts is the number of spans.
  // -1 when not split.
  int32_t group;
  int32_t reserved[3];
};

struct MergeGroup {          // 16 bytes
  int32_t q_row;
  int32_t kvh;
  int32_t part0;
  int32_t n_parts;
};

// One block that receives new tokens of the step: rows q_row0 .. q_row0 +
// n_rows - 1 of Q (and of the new K/V rows) go to slots slot0 .. slot0 +
// n_rows - 1 of block block_ids[bt_index]; slot0 == 0 means the block holds
// nothing of the request yet.
struct AppendItem {          // 16 bytes
  int32_t q_row0;
  int16_t n_rows;
  int16_t slot0;
  int32_t bt_index;
  int32_t reserved;
};

static_assert(sizeof(PlanHeader) == 64, "plan header layout");
static_assert(sizeof(AppendItem) == 16, "append item layout");
static_assert(sizeof(WorkItem) == 48, "work item layout");
static_assert(sizeof(MergeGroup) == 16, "merge group layout");

// Layout of the image: header, work items, merge groups, one int32 counter
// per merge group, then (16-byte aligned) the append items.
constexpr int64_t append_offset(int64_t num_items, int64_t num_groups) {
  return ((static_cast<int64_t>(sizeof(PlanHeader)) + num_items * static_cast<int64_t>(sizeof(WorkItem)) +
           num_groups * static_cast<int64_t>(sizeof(MergeGroup) + 4) + 15) / 16) * 16;
}
constexpr int64_t plan_image_bytes(int64_t num_items, int64_t num_groups, int64_t num_append) {
  return append_offset(num_items, num_groups) + num_append * static_cast<int64_t>(sizeof(AppendItem));
}

// Split-K partial of one (row, KV head, key span): unnormalised o[G][D]
// relative to the running maximum, then m[G] (log2 domain) and l[G], padded to
// a multiple of 4 floats so every slot starts 16-byte aligned.
constexpr int64_t partial_floats(int32_t group, int32_t head_dim) {
  return ((static_cast<int64_t>(group) * (head_dim + 2) + 3) / 4) * 4;
}

}  // namespace aug
