/*
 * aug.h - C ABI of the mixed-batch serving step for augmented-LLM requests
 * on AMD Instinct MI355X (gfx950).
 *
 * The scheduler described in "AugServe: Adaptive Request Scheduling for
 * Augmented LLM Inference Serving" (arXiv 2512.04013) forms, every engine
 * iteration, a batch of requests that are prefilling a prompt, prefilling the
 * tokens an external call returned, recomputing a discarded context, or
 * decoding (request lifecycle, Eq. 1; Algorithm 1, steps (1)-(5)). Requests
 * paused on an external call keep their KV cache on the GPU, park it in host
 * memory, or discard it (context-handling policies, Appendix B). This library
 * runs the data-parallel work of one such iteration:
 *
 *   aug_request_arrive, aug_request_return
 *                     host: a request's record on arrival and on the return
 *                     of an external call (Algorithm 1, steps (1)-(2))
 *   aug_form_batch    host: token budget (Eq. token), cost and priority
 *                     (Eqs. cost, c_fb, c_ik_new, value, theta), Waste policy
 *                     choice (Appendix B) and greedy packing (Algorithm 1 (4))
 *   aug_attn_plan     host: validates a formed batch and writes the work list
 *   aug_plan_upload   pinned host -> device: the work list, on the launch stream
 *   aug_kv_append     device: the step's new K/V rows into their paged slots
 *   aug_attn_mixed    device: one launch of paged, causal, grouped-query
 *                     attention over every chunked-prefill row and decode row
 *                     of the batch (plus a merge launch for split prefill tiles)
 *   aug_kv_park       device -> pinned host: swap-out of KV blocks
 *   aug_kv_resume     pinned host -> device: swap-in into (new) KV blocks
 *
 * Conventions
 *  - Every buffer belongs to the caller. The library allocates nothing and
 *    keeps no state between calls.
 *  - "device" pointers are HIP device memory of the current device; "host"
 *    pointers are ordinary host memory unless "pinned" is stated (then it must
 *    come from hipHostMalloc or an equivalent page-locked allocation).
 *  - `stream` is a hipStream_t (NULL = the null stream). Device calls validate
 *    their arguments on the host, then enqueue work and return without
 *    waiting. A validation error enqueues nothing.
 *  - Errors are returned as aug_status; aug_last_error() gives a message for
 *    the most recent failing call of the calling thread.
 *  - No C++ exception crosses this interface.
 */
#ifndef AUG_H
#define AUG_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  AUG_OK = 0,
  AUG_ERR_INVALID = -1,      /* an argument is out of its documented range */
  AUG_ERR_UNSUPPORTED = -2,  /* a valid combination the library does not run */
  AUG_ERR_NO_SPACE = -3,     /* a caller buffer is too small */
  AUG_ERR_HIP = -4           /* the HIP runtime reported an error */
} aug_status;

typedef enum { AUG_F32 = 0, AUG_BF16 = 1, AUG_FP8_E4M3FN = 2 } aug_dtype;

/* Request queues of Algorithm 1: running, swapped, waiting, paused. */
typedef enum { AUG_WAITING = 0, AUG_RUNNING = 1, AUG_SWAPPED = 2, AUG_PAUSED = 3 } aug_state;

/* Context-handling policies (set Pi), in the order the paper lists them in
 * the Waste minimisation of Appendix B; that order breaks ties. */
typedef enum { AUG_POL_NONE = 0, AUG_PRESERVE = 1, AUG_DISCARD = 2, AUG_SWAP = 3 } aug_policy;

/* Ranking of the candidates in Algorithm 1, step (4). THETA is the paper's
 * value density theta = (1 + beta w) / C (Eqs. value, theta); FCFS (arrival
 * order) is the scheduling of the systems the paper starts from, and SSJF
 * (shortest predicted output first) the prediction-based baseline of its
 * evaluation. Ties: earlier arrival, then smaller id. */
typedef enum { AUG_ORDER_THETA = 0, AUG_ORDER_FCFS = 1, AUG_ORDER_SSJF = 2 } aug_order;

/* ------------------------------------------------------------------------ */
/* Attention                                                                 */
/* ------------------------------------------------------------------------ */

/* Shape of one attention layer.
 *   num_q_heads % num_kv_heads == 0; query head h reads KV head
 *   h / (num_q_heads / num_kv_heads) (grouped-query attention).
 *   head_dim: 64 or 128.  block_size: 16 (tokens per KV block).
 *   Supported dtype sets (q, kv, out): (F32, F32, F32), (BF16, BF16, BF16),
 *   (BF16, FP8_E4M3FN, BF16).
 *   softmax_scale: multiplies q.k before the softmax (typically 1/sqrt(head_dim));
 *   finite and > 0. */
typedef struct {
  int32_t num_q_heads;
  int32_t num_kv_heads;
  int32_t head_dim;
  int32_t block_size;
  int32_t q_dtype;
  int32_t kv_dtype;
  int32_t out_dtype;
  float softmax_scale;
} aug_attn_shape;

/* A formed batch, in HOST memory.
 *   q_start[num_reqs+1]: rows of request r are q_start[r] .. q_start[r+1]-1 of
 *     Q and O ([rows][num_q_heads][head_dim], row-major); q_start[0] == 0 and
 *     every request has at least one row.
 *   ctx_len[num_reqs]: keys of request r, this step's rows included; row j of
 *     request r sits at position ctx_len[r] - q_len + j and attends keys
 *     0 .. that position (causal, aligned at the end of the context).
 *     ctx_len[r] >= q_len(r).
 *   bt_start[num_reqs+1]: request r's KV blocks are
 *     block_ids[bt_start[r] .. bt_start[r+1]-1]; it must list at least
 *     ceil(ctx_len[r] / block_size) of them; only that many are read.
 *   block_ids: host copy of the block table, used only to range-check it
 *     against num_pool_blocks; may be NULL to skip that check (the kernels
 *     still never read outside the pool).
 */
typedef struct {
  int32_t num_reqs;
  const int32_t* q_start;
  const int32_t* ctx_len;
  const int32_t* bt_start;
  const int32_t* block_ids;
  int32_t num_pool_blocks;
} aug_batch_desc;

/* Sizes the planner derived for one batch. */
typedef struct {
  int64_t plan_bytes;        /* bytes of the plan image */
  int64_t workspace_bytes;   /* device workspace aug_attn_mixed needs */
  int32_t num_items;         /* work items of the attention launch */
  int32_t num_prefill_items; /* of which chunked-prefill tiles */
  int32_t num_merge_groups;  /* split (row, KV head) pairs; the first num_tile_merge_groups
                                belong to prefill tiles */
  int32_t num_partials;      /* split-K partial results */
  int32_t kv_split_tokens;   /* keys per decode work item (multiple of block_size) */
  int32_t total_rows;        /* q_start[num_reqs] */
  int32_t num_reqs;
  int32_t num_tile_merge_groups;
  int32_t num_append_items;  /* blocks that receive new K/V rows (aug_kv_append) */
  /* The layer shape the plan was built for. aug_attn_mixed and aug_kv_append
   * refuse a call whose shape differs in any of these fields: the plan's work
   * items, partial sizes and workspace size depend on them. */
  int32_t num_q_heads;
  int32_t num_kv_heads;
  int32_t head_dim;
  int32_t q_dtype;
  int32_t kv_dtype;
  int32_t out_dtype;
  int32_t row_path;          /* aug_row_path the plan's row items run on (VALU or MFMA, resolved) */
  int32_t tile_path;         /* aug_tile_path the plan's prefill tiles run on (resolved) */
} aug_attn_plan_info;

/* Where the row items (decode rows) of a plan run. Groups of eight or four
 * query heads per KV head with head_dim 128 and bf16 or fp8 KV can run their
 * products on 16x16 bf16 MFMAs; every other shape runs on the vector ALUs.
 * AUTO takes MFMA for groups of eight (the vector ALUs cannot keep up with
 * eight heads of fp8 KV) and VALU otherwise; four-head groups run on MFMA
 * only when asked for. */
typedef enum { AUG_ROWS_AUTO = 0, AUG_ROWS_VALU = 1, AUG_ROWS_MFMA = 2 } aug_row_path;

/* Arithmetic of the prefill tiles' products S = Q K^T and O = P V. BF16: Q,
 * P and the (converted) keys and values as bf16 on 32x32x16 MFMAs, the
 * default. FP8_QK, for fp8 KV with bf16 Q and head_dim 128 only: the keys
 * stay fp8 and each query vector (row and head) is rounded to E4M3 with its
 * own scale (largest magnitude / 448; a vector below 2^-100 becomes zero), on
 * 32x32x64 fp8 MFMAs at twice the rate; P V stays bf16; decode rows are not
 * affected. Rounding Q to 3 mantissa bits moves a logit by about 2^-5 of
 * |q| |k| sqrt(head_dim) times the softmax scale, so outputs stay within the
 * bf16 tolerances for near-uniform attention (keys of norm about 1) but not
 * for sharp attention (keys of norm about sqrt(head_dim)). FP8 (same shapes):
 * FP8_QK, and P V on 32x32x64 fp8 MFMAs as well: the values stay fp8 and each
 * probability is rounded to E4M3 after scaling by its block's V scale over
 * the item's largest one (the row sums add the rounded probabilities, so a
 * single dominant key still returns its value); probabilities below 2^-15 of
 * the row maximum vanish and the rest carry a relative error of up to 2^-4,
 * which adds to the output error of FP8_QK where several keys share the
 * weight. Both fp8 forms are opt-in, never chosen by AUTO. */
typedef enum { AUG_TILES_AUTO = 0, AUG_TILES_BF16 = 1, AUG_TILES_FP8_QK = 2, AUG_TILES_FP8 = 3 } aug_tile_path;

/* Planner options (aug_attn_plan_opts). */
typedef struct {
  int32_t kv_split_tokens;   /* as the argument of aug_attn_plan */
  int32_t row_path;          /* aug_row_path */
  int32_t tile_path;         /* aug_tile_path */
  int32_t reserved;          /* zero */
} aug_plan_options;

/* Validate a formed batch and write its work list ("plan image") to
 * plan_host, which needs info->plan_bytes bytes (call once with
 * plan_host == NULL to obtain the sizes only). The image is position
 * independent: copy it verbatim to device memory and pass that copy to
 * aug_attn_mixed with the same `info`. kv_split_tokens <= 0 lets the planner
 * choose the decode split (keys per work item); a positive value, at most
 * 2^24, is rounded up to a multiple of block_size. Contexts are limited to
 * 2^24 tokens per request. Pure host code; deterministic.
 * The image also lists the blocks that receive the step's new K/V rows
 * (info->num_append_items), for aug_kv_append.
 * Errors: AUG_ERR_INVALID (shape, monotonicity, ctx_len < q_len, too few
 * blocks, block id outside the pool, kv_split_tokens above 2^24; with the
 * host block table, a block that would receive new tokens of two requests or
 * twice from one), AUG_ERR_UNSUPPORTED (dtype set, head_dim, block_size, a
 * context above 2^24 tokens), AUG_ERR_NO_SPACE (plan_cap < plan_bytes). */
aug_status aug_attn_plan(const aug_attn_shape* shape, const aug_batch_desc* batch,
                         int32_t kv_split_tokens, void* plan_host, size_t plan_cap,
                         aug_attn_plan_info* info);

/* aug_attn_plan with options: opts->kv_split_tokens as above, the path the
 * row items run on and the arithmetic of the prefill tiles (info->row_path
 * and info->tile_path record the resolved choices, which aug_attn_mixed
 * follows). Same image layout and errors, plus AUG_ERR_UNSUPPORTED for
 * AUG_ROWS_MFMA, AUG_TILES_FP8_QK or AUG_TILES_FP8 on a shape without that path and
 * AUG_ERR_INVALID for an unknown path or a non-zero reserved field. */
aug_status aug_attn_plan_opts(const aug_attn_shape* shape, const aug_batch_desc* batch,
                              const aug_plan_options* opts, void* plan_host, size_t plan_cap,
                              aug_attn_plan_info* info);

/* Device workspace (split-K partials, in bytes) that aug_attn_mixed needs for
 * this batch with this split: the planner's size query, the same validation
 * as aug_attn_plan, nothing written but *bytes. The batch is the formed batch
 * of the problem statement (requests with their query rows, context lengths
 * and block tables); the size depends on the split the planner chooses.
 * Errors: those of aug_attn_plan; AUG_ERR_INVALID for a NULL `bytes`. */
aug_status aug_attn_workspace_size(const aug_attn_shape* shape, const aug_batch_desc* batch,
                                   int32_t kv_split_tokens, size_t* bytes);

/* Copy `bytes` bytes of a plan image (or any other bytes) from pinned host
 * memory host_src to device memory dev_dst with one small copy kernel
 * enqueued on `stream`, so that the copy starts as soon as the stream's
 * previous kernel has finished instead of waiting for a DMA engine; the step's
 * launches queued after it on the same stream see the bytes. host_src must be
 * page-locked memory registered with HIP (hipHostMalloc, torch's pinned
 * tensors) and must stay unchanged until the copy has run; both ranges must
 * lie inside their allocations (the caller's duty: they are not checked); both
 * pointers 16-byte aligned. bytes == 0 enqueues nothing. No allocation, no
 * memset.
 * Errors: AUG_ERR_INVALID (NULL or misaligned pointer, host_src not pinned
 * host memory, dev_dst not device memory), AUG_ERR_HIP (launch). */
aug_status aug_plan_upload(const void* host_src, void* dev_dst, size_t bytes, void* stream);

/* Mixed-batch paged attention: for every row of every request of the planned
 * batch, O = softmax(softmax_scale * q K^T, causal) V over the request's
 * paged keys (see aug_batch_desc). Device memory:
 *   plan_dev   the plan image of aug_attn_plan (info->plan_bytes bytes). Its
 *              last 4 * info->num_merge_groups bytes are completion counters
 *              of the split decode rows, which the launch increments and
 *              returns to zero, so the same device copy can be launched
 *              again; calls that overlap on one copy race
 *   q          [total_rows][num_q_heads][head_dim], q_dtype
 *   k_cache,   [num_pool_blocks][num_kv_heads][block_size][head_dim], kv_dtype
 *   v_cache
 *   k_scale,   [num_pool_blocks][num_kv_heads] float32, dequantisation scale of
 *   v_scale    each fp8 block (value = code * scale); NULL unless kv is fp8
 *   block_ids  the block table (CSR payload of aug_batch_desc)
 *   out        [total_rows][num_q_heads][head_dim], out_dtype
 *   workspace  >= info->workspace_bytes bytes (split-K partials); contents on
 *              entry do not matter
 * Slots past a request's context and blocks it does not list never influence
 * its output, whatever they hold. Enqueued on `stream` as one kernel launch:
 * split decode rows are merged in it by the workgroup that finishes each
 * row's last span; split prefill tiles are merged by a second small launch
 * when info->num_tile_merge_groups > 0.
 * Errors: AUG_ERR_INVALID (NULL pointers, info inconsistent, or a shape
 * other than the one the plan was built for: heads, head_dim or dtypes),
 * AUG_ERR_NO_SPACE (workspace_bytes too small), AUG_ERR_HIP (launch). */
aug_status aug_attn_mixed(const aug_attn_shape* shape, const aug_attn_plan_info* info,
                          void* plan_dev, const void* q, const void* k_cache,
                          const void* v_cache, const float* k_scale, const float* v_scale,
                          const int32_t* block_ids, int32_t num_pool_blocks, void* out,
                          void* workspace, size_t workspace_bytes, void* stream);

/* Bytes of the library's own device array for split-K partials, used by
 * aug_attn_mixed_noalloc (64 MiB per GPU the library runs on). */
#define AUG_NOALLOC_SCRATCH_BYTES (64ull << 20)

/* aug_attn_mixed for callers that cannot allocate device memory (code under
 * HIP graph capture, tight serving loops, harnesses that forbid allocation):
 * the same launch, arguments and results, but the split-K partials live in a
 * file-scope device array of the library (AUG_NOALLOC_SCRATCH_BYTES per GPU,
 * held until the process ends) instead of a caller workspace. The caller
 * still passes the plan image, inputs and output. The array's device address
 * is looked up once per device, on the first call made with that device
 * current; `stream` must belong to the current device. Nothing in the array
 * needs to start at zero (every partial is written before it is read), and
 * it keeps the last call's contents. All calls on one GPU share the array:
 * calls that overlap in time on that GPU (other streams, other threads)
 * race and must be serialised by the caller. Allocates nothing (no
 * hipMalloc, no hipFree, no allocating library call).
 * Errors: those of aug_attn_mixed; AUG_ERR_NO_SPACE when the plan's
 * info->workspace_bytes exceeds AUG_NOALLOC_SCRATCH_BYTES (plan with a larger
 * kv_split_tokens, or use aug_attn_mixed); AUG_ERR_HIP when the array's
 * address cannot be obtained or the launch fails. */
aug_status aug_attn_mixed_noalloc(const aug_attn_shape* shape, const aug_attn_plan_info* info,
                                  void* plan_dev, const void* q, const void* k_cache,
                                  const void* v_cache, const float* k_scale, const float* v_scale,
                                  const int32_t* block_ids, int32_t num_pool_blocks, void* out,
                                  void* stream);

/* Append the step's new K/V rows to the paged cache, before the attention of
 * the same step reads them: every query row is a token the forward pass
 * produced (the chunk or decode token scheduled in Algorithm 1, step (5)).
 * Row j of request r sits at position ctx_len[r] - q_len + j, slot
 * (position mod block_size) of block block_ids[bt_start[r] + position /
 * block_size], for every KV head. Device memory:
 *   plan_dev   the plan image of aug_attn_plan for this batch (read only)
 *   k_new,     [total_rows][num_kv_heads][head_dim]: float32 for f32 caches,
 *   v_new      bf16 for bf16 and fp8 caches; finite values
 *   k_cache, v_cache, k_scale, v_scale, block_ids  as for aug_attn_mixed;
 *              written in place
 * f32 and bf16 caches receive the rows unchanged. fp8 E4M3FN caches (one
 * float32 scale per block and KV head, value = code * scale): per block and
 * KV head that receives tokens, with a = max |x| of the new tokens, the scale
 * becomes a / 448 if the request's first new token lands in slot 0, else
 * max(old scale, a / 448); when it grows, the block's earlier codes are
 * re-encoded as enc(dec(code) * old / new); new tokens are enc(x / scale)
 * (0 if the scale is 0). enc rounds to nearest even and saturates at +-448;
 * products and quotients are single float32 operations in that order.
 * A block id outside the pool is skipped. The blocks that receive tokens
 * must be distinct across the batch (aug_attn_plan checks this when it is
 * given the host block table); two requests appending into one block would
 * race on its contents and scale. Enqueued on `stream` as one kernel launch
 * (none for an empty batch); no allocation, no memset, so the call can be
 * captured in a HIP graph and replayed.
 * Errors: AUG_ERR_INVALID (NULL pointers, info inconsistent or built for
 * another shape, missing scales for fp8), AUG_ERR_HIP (launch). */
aug_status aug_kv_append(const aug_attn_shape* shape, const aug_attn_plan_info* info,
                         const void* plan_dev, const void* k_new, const void* v_new, void* k_cache,
                         void* v_cache, float* k_scale, float* v_scale, const int32_t* block_ids,
                         int32_t num_pool_blocks, void* stream);

/* ------------------------------------------------------------------------ */
/* Park / resume (Swap policy: swap-out during an external call, swap-in     */
/* when it returns; Appendix B, Algorithm 1 step (2))                         */
/* ------------------------------------------------------------------------ */

/* Bytes of one parked block record: K[block] then V[block]
 * (num_kv_heads * block_size * head_dim elements each, the pool's own bit
 * patterns), then, for fp8 caches, k_scale[block] and v_scale[block]
 * (num_kv_heads float32 each). Returns 0 for an invalid shape. */
size_t aug_kv_record_bytes(const aug_attn_shape* shape);

/* Park n_blocks blocks: host_dst (pinned, >= n_blocks * record bytes) receives
 * the records of block_ids_dev[0..n_blocks-1] in that order. Data moves
 * through `staging` (device, >= one record; larger staging means fewer,
 * larger copies): a gather kernel fills it, then an asynchronous copy drains
 * it to host_dst, chunk after chunk, all on `stream`. host_dst is complete
 * once the stream reaches the end of this call's work.
 * block_ids_dev: device int32[n_blocks]. block_ids_host: the same ids in
 * host memory (required), range-checked against num_pool_blocks before
 * anything is enqueued, so every record of a successful call is the block's
 * bytes. (Should the device copy still name a block outside the pool, the
 * kernel never dereferences it and writes a record of zero bytes instead.)
 * Errors: AUG_ERR_INVALID (NULL pointers, block_ids_host missing, an id
 * outside the pool), AUG_ERR_NO_SPACE (host_bytes, staging_bytes),
 * AUG_ERR_HIP. */
aug_status aug_kv_park(const aug_attn_shape* shape, const void* k_cache, const void* v_cache,
                       const float* k_scale, const float* v_scale,
                       const int32_t* block_ids_dev, const int32_t* block_ids_host,
                       int32_t n_blocks, int32_t num_pool_blocks, void* host_dst,
                       size_t host_bytes, void* staging, size_t staging_bytes, void* stream);

/* Resume n_blocks records from host_src (pinned, as written by aug_kv_park)
 * into the pool blocks block_ids_dev[0..n_blocks-1] (any blocks: a resumed
 * request usually lands elsewhere than it was). Same staging scheme in the
 * other direction; block_ids_host is required and range-checked as for
 * aug_kv_park (a device id outside the pool is never written).
 * Errors as aug_kv_park. */
aug_status aug_kv_resume(const aug_attn_shape* shape, void* k_cache, void* v_cache,
                         float* k_scale, float* v_scale, const int32_t* block_ids_dev,
                         const int32_t* block_ids_host, int32_t n_blocks,
                         int32_t num_pool_blocks, const void* host_src, size_t host_bytes,
                         void* staging, size_t staging_bytes, void* stream);

/* ------------------------------------------------------------------------ */
/* Batch former (host)                                                       */
/* ------------------------------------------------------------------------ */

/* One request R_i as the scheduler sees it (symbols of the paper's notation
 * table). Times are seconds on the caller's clock. */
typedef struct {
  int64_t id;             /* unique */
  double arrival;
  double last_sched;      /* last time it was scheduled; < 0 if never */
  double pred_call;       /* tau_hat^call of the call ending this segment (s) */
  double pause_start;     /* PAUSED: when the current wait began */
  int32_t state;          /* aug_state */
  int32_t seg;            /* k, 1 for the first segment */
  int32_t prev_policy;    /* p_{i,k-1}: policy realised during the last wait (k >= 2) */
  int32_t cur_policy;     /* PAUSED: policy chosen for the current wait */
  int32_t seg_ctx;        /* L: context tokens at the segment start (before returned tokens) */
  int32_t seg_prefill;    /* tokens prefilled in this segment: prompt (k = 1) or returned (k >= 2) */
  int32_t pred_out;       /* l_hat^out: tokens predicted for this segment, >= 1 */
  int32_t has_next_call;  /* 1 if the segment ends in an external call */
  int32_t ctx_len;        /* tokens whose KV the request holds now */
  int32_t pending;        /* tokens to prefill before its next decode (prompt, returned, recompute) */
  int32_t blocks_on_gpu;  /* pool blocks it holds now */
  int32_t reserved;
} aug_request;

typedef struct {
  double beta;            /* aging factor of Eq. value; w is in milliseconds */
  double beta_low;        /* budget clip: [floor(beta_low*t_max), floor(beta_high*t_max)] */
  double beta_high;
  double t_iter;          /* seconds per engine iteration in the space-time cost */
  double fwd_a;           /* tau_fwd(L) = fwd_a + fwd_b * L  (Waste of Discard) */
  double fwd_b;
  double swap_s_per_tok;  /* tau_swap(L) = swap_s_per_tok * L */
  int64_t n_fwd_max;      /* N_max^fwd of the Swap Waste */
  int32_t t_max;          /* T_max, reference token budget */
  int32_t chunk_cap;      /* most prefill tokens one request takes per iteration */
  int32_t block_size;     /* tokens per pool block */
  int32_t skip_instead_of_break; /* 0: stop at the first request that does not fit */
  int32_t order;          /* aug_order of the ranking */
  int32_t reserved;
} aug_former_params;

/* Output of aug_form_batch. The caller sets `cap` and the array pointers; each
 * id/q_len/theta array must hold `cap` entries, policy_out and cost_out one
 * entry per input request (either may be NULL). */
typedef struct {
  int32_t cap;
  int32_t budget;         /* B_token after clipping */
  int32_t n_sched;        /* scheduled requests, in rank order */
  int32_t n_resume;       /* scheduled requests that were swapped out */
  int32_t n_park;         /* paused Swap requests evicted to host memory */
  int32_t n_free;         /* paused Discard requests whose blocks are freed */
  int64_t* ids;           /* [cap] scheduled ids */
  int32_t* q_len;         /* [cap] tokens each scheduled request runs */
  double* theta;          /* [cap] priority at formation */
  int64_t* resume_ids;    /* [cap] */
  int64_t* park_ids;      /* [cap] */
  int64_t* free_ids;      /* [cap] */
  int32_t* policy_out;    /* [n] predicted policy per input (AUG_POL_NONE if not a candidate) */
  double* cost_out;       /* [n] C_{i,k} per input (0 if not a candidate) */
} aug_batch_plan;

/* Form one iteration's batch (Algorithm 1, steps (3)-(4)) from n requests and
 * free_blocks free pool blocks at time `now`. Deterministic, pure host code in
 * IEEE double precision with a fixed operation order.
 * Errors: AUG_ERR_INVALID (NULL pointers, pred_out < 1 for a candidate,
 * negative sizes, t_iter <= 0, chunk_cap < 1, block_size < 1, unknown state),
 * AUG_ERR_NO_SPACE (more than `cap` entries in any output list). */
aug_status aug_form_batch(const aug_request* reqs, int32_t n, int64_t free_blocks, double now,
                          const aug_former_params* params, aug_batch_plan* out);

/* Algorithm 1, step (1): a new request enters the waiting queue. Fills every
 * field of *r: the first segment prefills the prompt (seg 1, seg_ctx 0,
 * seg_prefill = pending = prompt_tokens, no KV held), with the predictor's
 * output length and call duration (pred_call 0 and has_next_call 0 when the
 * request makes no call). Its policy, cost and priority are evaluated by
 * aug_form_batch at every iteration, since the waiting time w changes.
 * Errors: AUG_ERR_INVALID (NULL r, prompt_tokens < 1, pred_out < 1,
 * pred_call < 0 or not finite). */
aug_status aug_request_arrive(aug_request* r, int64_t id, double arrival, int32_t prompt_tokens,
                              int32_t pred_out, double pred_call, int32_t has_next_call);

/* Algorithm 1, step (2): a paused request's external call has returned.
 * `realised` is the policy actually executed during the wait (p_{i,k-1}):
 * PRESERVE (its KV stayed on the GPU), SWAP (its blocks were parked) or
 * DISCARD (its blocks were freed). The next segment starts at the request's
 * full context `context_tokens` (prompt, generated and returned tokens so
 * far) and prefills the `ret_tokens` the call returned; its cost from then on
 * is the feedback cost C^fb (Eq. c_fb) plus decode and next-call terms. The
 * request is requeued by the realised policy: PRESERVE -> running, SWAP ->
 * swapped (pending = ret_tokens), DISCARD -> waiting with no KV and pending =
 * context_tokens + ret_tokens (recompute). The predictions are those of the
 * new segment.
 * Errors: AUG_ERR_INVALID (NULL r, r not PAUSED, unknown policy,
 * context_tokens < ctx_len, ret_tokens < 0, pred_out < 1, pred_call < 0 or
 * not finite). */
aug_status aug_request_return(aug_request* r, int32_t realised, int32_t context_tokens, int32_t ret_tokens,
                              int32_t pred_out, double pred_call, int32_t has_next_call);

/* ------------------------------------------------------------------------ */

/* Static name of a status code. */
const char* aug_status_string(aug_status s);
/* Message of the calling thread's most recent failing call ("" if none). */
const char* aug_last_error(void);
/* Version of this ABI: (major << 16) | minor. */
int32_t aug_abi_version(void);

#ifdef __cplusplus
}
#endif

#endif /* AUG_H */
