// Token-budget batch former: Algorithm 1, steps (3)-(4), of the paper, and
// the request records of steps (1)-(2) (arrival, return of an external call).
//
// Per candidate request (running, swapped and waiting queues) it builds the
// space-time cost C_{i,k} (Eq. cost) from the request's segment inputs -
// before the first call from predictions (Eq. context_policy and the C_{i,1},
// C^call equations), after a call from the realised policy and return length
// (Eqs. c_fb, c_ik_new) - picks the context-handling policy that minimises
// Waste (Appendix B), and ranks by theta = (1 + beta w) / C (Eqs. value,
// theta). The token budget is floor((G_free + G_preempt) / mu), clipped
// (Eq. token). Packing walks the ranking and stops at the first request whose
// tokens do not fit the budget; a request whose blocks cannot be found is
// passed over. Blocks are reclaimed lazily from paused Swap (parked) and
// Discard (freed) requests. A prefill request takes min(pending, chunk_cap,
// budget) tokens.
//
// Memory occupancy is counted in KV tokens after each iteration's tokens are
// added, one iteration lasting t_iter seconds; mu is one token, so a budget
// in blocks is (free + preemptable) * block_size tokens. Token-iteration sums
// are exact integers converted to double once. Compiled without FMA
// contraction or fast-math; every floating-point expression keeps a fixed
// order, so results are reproducible bit for bit.

#include <algorithm>
#include <cmath>
#include <cstdint>
#include <vector>

#include "aug.h"
#include "status.h"

namespace {

struct Cost {
  double c;
  int32_t policy;
};

double prefill_cost(const aug_former_params& p, int64_t l0, int64_t x) {
  if (x <= 0) return 0.0;
  const int64_t cap = p.chunk_cap;
  const int64_t n = (x + cap - 1) / cap;
  // chunks 1..n-1 end at j*cap, the last at x
  const int64_t token_iters = n * l0 + cap * (n * (n - 1) / 2) + x;
  return static_cast<double>(token_iters) * p.t_iter;
}

double decode_cost(const aug_former_params& p, int64_t l0, int64_t n) {
  const int64_t token_iters = n * l0 + n * (n + 1) / 2;
  return static_cast<double>(token_iters) * p.t_iter;
}

double fwd_time(const aug_former_params& p, double len) { return p.fwd_a + p.fwd_b * len; }
double swap_time(const aug_former_params& p, double len) { return p.swap_s_per_tok * len; }

// Appendix B with the per-token footprint M dropped (it scales all three).
int32_t select_policy(const aug_former_params& p, int64_t l_tilde, double tau_call,
                      int64_t l_other) {
  const double lt = static_cast<double>(l_tilde);
  const double w_preserve = tau_call * lt;
  const double f = fwd_time(p, lt);
  const double w_discard = f * lt + f * static_cast<double>(l_other);
  const double w_swap = 2.0 * swap_time(p, lt) * static_cast<double>(p.n_fwd_max);
  int32_t best = AUG_PRESERVE;
  double best_w = w_preserve;
  if (w_discard < best_w) { best = AUG_DISCARD; best_w = w_discard; }
  if (w_swap < best_w) { best = AUG_SWAP; best_w = w_swap; }
  return best;
}

double call_cost(const aug_former_params& p, int32_t policy, int64_t l_tilde, double tau_call) {
  const double lt = static_cast<double>(l_tilde);
  if (policy == AUG_PRESERVE) return tau_call * lt;
  if (policy == AUG_SWAP) return swap_time(p, lt) * lt;
  return 0.0;
}

double resumption_cost(const aug_former_params& p, int32_t prev, int64_t l_ctx) {
  if (prev == AUG_DISCARD) return prefill_cost(p, 0, l_ctx);
  if (prev == AUG_SWAP) {
    const double l = static_cast<double>(l_ctx);
    return swap_time(p, l) * l;
  }
  return 0.0;
}

Cost segment_cost(const aug_former_params& p, const aug_request& r, int64_t l_other) {
  const int64_t l0 = r.seg_ctx, x = r.seg_prefill;
  const int64_t l_tilde = l0 + x + r.pred_out;
  Cost out{0.0, AUG_POL_NONE};
  double c_call = 0.0;
  if (r.has_next_call) {
    out.policy = select_policy(p, l_tilde, r.pred_call, l_other);
    c_call = call_cost(p, out.policy, l_tilde, r.pred_call);
  }
  const double c_decode = decode_cost(p, l0 + x, r.pred_out);
  if (r.seg <= 1) {
    const double c_prefill = prefill_cost(p, l0, x);
    out.c = (c_prefill + c_decode) + c_call;
  } else {
    const double c_fb = prefill_cost(p, l0, x) + resumption_cost(p, r.prev_policy, l0);
    out.c = (c_fb + c_decode) + c_call;
  }
  return out;
}

int64_t token_budget(const aug_former_params& p, int64_t free_blocks, int64_t preempt) {
  const int64_t raw = (free_blocks + preempt) * p.block_size;
  const int64_t lo = static_cast<int64_t>(std::floor(p.beta_low * static_cast<double>(p.t_max)));
  const int64_t hi = static_cast<int64_t>(std::floor(p.beta_high * static_cast<double>(p.t_max)));
  return std::min(std::max(raw, lo), hi);
}

bool is_candidate(int32_t s) { return s == AUG_WAITING || s == AUG_RUNNING || s == AUG_SWAPPED; }

}  // namespace

extern "C" aug_status aug_form_batch(const aug_request* reqs, int32_t n, int64_t free_blocks,
                                     double now, const aug_former_params* params,
                                     aug_batch_plan* out) {
  if (!params || !out || n < 0 || (n > 0 && !reqs))
    return aug::fail(AUG_ERR_INVALID, "aug_form_batch: NULL argument or negative count");
  const aug_former_params& p = *params;
  if (!(p.t_iter > 0.0) || p.chunk_cap < 1 || p.block_size < 1 || p.t_max < 0 ||
      free_blocks < 0 || out->cap < 0 || p.order < AUG_ORDER_THETA || p.order > AUG_ORDER_SSJF)
    return aug::fail(AUG_ERR_INVALID, "aug_form_batch: bad parameters");
  if (out->cap > 0 && (!out->ids || !out->q_len || !out->theta || !out->resume_ids ||
                       !out->park_ids || !out->free_ids))
    return aug::fail(AUG_ERR_INVALID, "aug_form_batch: NULL output array");
  for (int32_t i = 0; i < n; ++i) {
    const aug_request& r = reqs[i];
    if (r.state < AUG_WAITING || r.state > AUG_PAUSED)
      return aug::fail(AUG_ERR_INVALID, "aug_form_batch: request %d has unknown state", i);
    if (r.ctx_len < 0 || r.pending < 0 || r.blocks_on_gpu < 0 || r.seg_ctx < 0 ||
        r.seg_prefill < 0)
      return aug::fail(AUG_ERR_INVALID, "aug_form_batch: request %d has a negative size", i);
    if (is_candidate(r.state) && r.pred_out < 1)
      return aug::fail(AUG_ERR_INVALID, "aug_form_batch: request %d has pred_out < 1", i);
  }

  int64_t total_ctx = 0;
  for (int32_t i = 0; i < n; ++i)
    if (is_candidate(reqs[i].state)) total_ctx += reqs[i].ctx_len;

  std::vector<int32_t> cand;
  std::vector<double> theta(n, 0.0);
  cand.reserve(n);
  for (int32_t i = 0; i < n; ++i) {
    if (out->policy_out) out->policy_out[i] = AUG_POL_NONE;
    if (out->cost_out) out->cost_out[i] = 0.0;
    const aug_request& r = reqs[i];
    if (!is_candidate(r.state)) continue;
    const Cost c = segment_cost(p, r, total_ctx - r.ctx_len);
    const double since = r.last_sched >= 0.0 ? r.last_sched : r.arrival;
    const double w_ms = (now - since) * 1000.0;
    theta[i] = (1.0 + p.beta * w_ms) / c.c;
    if (out->policy_out) out->policy_out[i] = c.policy;
    if (out->cost_out) out->cost_out[i] = c.c;
    cand.push_back(i);
  }

  std::vector<int32_t> victims;
  int64_t preempt = 0;
  for (int32_t i = 0; i < n; ++i) {
    const aug_request& r = reqs[i];
    if (r.state == AUG_PAUSED && (r.cur_policy == AUG_SWAP || r.cur_policy == AUG_DISCARD) &&
        r.blocks_on_gpu > 0) {
      victims.push_back(i);
      preempt += r.blocks_on_gpu;
    }
  }
  const int64_t budget = token_budget(p, free_blocks, preempt);

  std::vector<double> remaining(n, 0.0);
  for (int32_t i : victims) remaining[i] = reqs[i].pred_call - (now - reqs[i].pause_start);
  std::sort(victims.begin(), victims.end(), [&](int32_t a, int32_t b) {
    if (remaining[a] != remaining[b]) return remaining[a] > remaining[b];
    return reqs[a].id < reqs[b].id;
  });
  std::sort(cand.begin(), cand.end(), [&](int32_t a, int32_t b) {
    if (p.order == AUG_ORDER_THETA && theta[a] != theta[b]) return theta[a] > theta[b];
    if (p.order == AUG_ORDER_SSJF && reqs[a].pred_out != reqs[b].pred_out)
      return reqs[a].pred_out < reqs[b].pred_out;
    if (reqs[a].arrival != reqs[b].arrival) return reqs[a].arrival < reqs[b].arrival;
    return reqs[a].id < reqs[b].id;
  });

  int64_t free_now = free_blocks, reclaim_left = preempt, active = 0;
  size_t vi = 0;
  int32_t n_sched = 0, n_resume = 0, n_park = 0, n_free = 0;
  const int64_t bs = p.block_size;
  // a prefill chunk is capped by the budget too, so it can always fit alone
  const int64_t chunk = std::min<int64_t>(p.chunk_cap, std::max<int64_t>(1, budget));
  for (int32_t i : cand) {
    const aug_request& r = reqs[i];
    const int64_t t = r.pending > 0 ? std::min<int64_t>(r.pending, chunk) : 1;
    if (active + t > budget) {
      if (p.skip_instead_of_break) continue;
      break;
    }
    const int64_t have = r.state == AUG_SWAPPED ? 0 : r.blocks_on_gpu;
    const int64_t need = std::max<int64_t>(0, (r.ctx_len + t + bs - 1) / bs - have);
    // no memory for it now: passed over (the algorithm stops at the token
    // budget only; memory enters through the budget)
    if (need > free_now + reclaim_left) continue;
    while (need > free_now) {
      const aug_request& v = reqs[victims[vi++]];
      free_now += v.blocks_on_gpu;
      reclaim_left -= v.blocks_on_gpu;
      if (v.cur_policy == AUG_SWAP) {
        if (n_park >= out->cap) return aug::fail(AUG_ERR_NO_SPACE, "aug_form_batch: park list over cap");
        out->park_ids[n_park++] = v.id;
      } else {
        if (n_free >= out->cap) return aug::fail(AUG_ERR_NO_SPACE, "aug_form_batch: free list over cap");
        out->free_ids[n_free++] = v.id;
      }
    }
    free_now -= need;
    active += t;
    if (n_sched >= out->cap) return aug::fail(AUG_ERR_NO_SPACE, "aug_form_batch: batch over cap");
    out->ids[n_sched] = r.id;
    out->q_len[n_sched] = static_cast<int32_t>(t);
    out->theta[n_sched] = theta[i];
    ++n_sched;
    if (r.state == AUG_SWAPPED) {
      if (n_resume >= out->cap) return aug::fail(AUG_ERR_NO_SPACE, "aug_form_batch: resume list over cap");
      out->resume_ids[n_resume++] = r.id;
    }
  }
  out->budget = static_cast<int32_t>(budget);
  out->n_sched = n_sched;
  out->n_resume = n_resume;
  out->n_park = n_park;
  out->n_free = n_free;
  return AUG_OK;
}

namespace {

bool prediction_ok(int32_t pred_out, double pred_call) {
  return pred_out >= 1 && std::isfinite(pred_call) && pred_call >= 0.0;
}

}  // namespace

extern "C" aug_status aug_request_arrive(aug_request* r, int64_t id, double arrival, int32_t prompt_tokens,
                                         int32_t pred_out, double pred_call, int32_t has_next_call) {
  if (!r || prompt_tokens < 1 || !prediction_ok(pred_out, pred_call) || !std::isfinite(arrival))
    return aug::fail(AUG_ERR_INVALID, "aug_request_arrive: NULL record or bad prompt/prediction");
  aug_request q{};
  q.id = id;
  q.arrival = arrival;
  q.last_sched = -1.0;
  q.pred_call = has_next_call ? pred_call : 0.0;
  q.pause_start = 0.0;
  q.state = AUG_WAITING;
  q.seg = 1;
  q.prev_policy = AUG_POL_NONE;
  q.cur_policy = AUG_POL_NONE;
  q.seg_ctx = 0;
  q.seg_prefill = prompt_tokens;
  q.pred_out = pred_out;
  q.has_next_call = has_next_call ? 1 : 0;
  q.ctx_len = 0;
  q.pending = prompt_tokens;
  q.blocks_on_gpu = 0;
  *r = q;
  return AUG_OK;
}

extern "C" aug_status aug_request_return(aug_request* r, int32_t realised, int32_t context_tokens,
                                         int32_t ret_tokens, int32_t pred_out, double pred_call,
                                         int32_t has_next_call) {
  if (!r) return aug::fail(AUG_ERR_INVALID, "aug_request_return: NULL record");
  if (r->state != AUG_PAUSED)
    return aug::fail(AUG_ERR_INVALID, "aug_request_return: request %lld is not paused", (long long)r->id);
  if (realised != AUG_PRESERVE && realised != AUG_SWAP && realised != AUG_DISCARD)
    return aug::fail(AUG_ERR_INVALID, "aug_request_return: unknown realised policy %d", realised);
  if (context_tokens < r->ctx_len || ret_tokens < 0 || !prediction_ok(pred_out, pred_call))
    return aug::fail(AUG_ERR_INVALID, "aug_request_return: bad context, return length or prediction");
  r->seg += 1;
  r->prev_policy = realised;
  r->cur_policy = AUG_POL_NONE;
  r->seg_ctx = context_tokens;
  r->seg_prefill = ret_tokens;
  r->pred_out = pred_out;
  r->pred_call = has_next_call ? pred_call : 0.0;
  r->has_next_call = has_next_call ? 1 : 0;
  if (realised == AUG_PRESERVE) {
    r->state = AUG_RUNNING;
    r->pending = ret_tokens;
  } else if (realised == AUG_SWAP) {
    r->state = AUG_SWAPPED;
    r->pending = ret_tokens;
  } else {
    r->state = AUG_WAITING;
    r->ctx_len = 0;
    r->blocks_on_gpu = 0;
    r->pending = context_tokens + ret_tokens;
  }
  return AUG_OK;
}
