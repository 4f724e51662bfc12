// Host scheduler for streamed prefill requests: lifecycle, LCP invalidation, the
// two-phase step, cost-based preemption and the four priority orders (Stream2LLM
// Sec. 4.1-4.4).  The contract, and the readings taken where the paper is silent, are in
// include/s2l_sched.h.
#include "s2l_sched.h"

#include <algorithm>
#include <chrono>
#include <cstdint>
#include <unordered_map>
#include <vector>

#include "status.h"

// The cost comparison must round as written (no fused multiply-add).
#pragma STDC FP_CONTRACT OFF

namespace {

using s2l::fail;
using s2l::ok;
using Clock = std::chrono::steady_clock;

constexpr int32_t kBlockTokens = 16;

int32_t blocks_for(int64_t tokens) { return (int32_t)((tokens + kBlockTokens - 1) / kBlockTokens); }

int64_t ns_since(Clock::time_point t0) {
  return std::chrono::duration_cast<std::chrono::nanoseconds>(Clock::now() - t0).count();
}

// Free-block pool that hands out the lowest free indices first: a bitmap with a hint to
// the lowest word that may hold a free bit.
class BlockPool {
 public:
  explicit BlockPool(int32_t n) : n_(n), free_(n), bits_((n + 63) / 64, ~0ull) {
    if (n % 64) bits_.back() = (1ull << (n % 64)) - 1;
    if (n == 0) bits_.clear();
  }
  int32_t free_count() const { return free_; }
  // appends the `k` lowest free blocks to `out` (k <= free_count)
  void take(int32_t k, std::vector<int32_t>& out) {
    free_ -= k;
    for (size_t w = lo_; k > 0; ++w) {
      while (bits_[w] && k > 0) {
        const int b = __builtin_ctzll(bits_[w]);
        bits_[w] &= bits_[w] - 1;
        out.push_back((int32_t)(w * 64 + b));
        --k;
      }
      if (!bits_[w]) lo_ = w + 1;
    }
  }
  void give(int32_t b) {
    bits_[b >> 6] |= 1ull << (b & 63);
    if ((size_t)(b >> 6) < lo_) lo_ = b >> 6;
    ++free_;
  }
  template <typename It>
  void give(It first, It last) {
    for (; first != last; ++first) give(*first);
  }

 private:
  int32_t n_, free_;
  size_t lo_ = 0;
  std::vector<uint64_t> bits_;
};

struct Request {
  int64_t id;
  std::vector<int32_t> ids;
  bool complete;
  double arrival, last_chunk;
  int64_t seq;
  int32_t computed = 0;
  std::vector<int32_t> gpu, cpu;
  int32_t state = S2L_REQ_WAITING;
  int64_t invalidated = 0;
  int32_t n_swap = 0, n_recompute = 0;
};

}  // namespace

struct s2l_sched {
  s2l_sched_config cfg;
  std::vector<double> rec_x, rec_y;
  BlockPool gpu, cpu;
  std::vector<int32_t> deferred_cpu;
  std::vector<Request> reqs;                   // indexed by slot, in admission order
  std::unordered_map<int64_t, int32_t> slot;   // request id -> slot
  std::vector<int32_t> live;                   // unfinished slots, admission order
  std::vector<int32_t> running, waiting;       // DEFAULT queues (front first)
  // per-step scratch
  std::vector<int32_t> order, not_sched, sel, sel_n, tmp;

  explicit s2l_sched(const s2l_sched_config& c)
      : cfg(c), gpu(c.num_gpu_blocks), cpu(c.num_cpu_blocks) {}

  double recompute_latency(double x) const {
    const std::vector<double>& xs = rec_x;
    const std::vector<double>& ys = rec_y;
    if (xs.size() == 1) return ys[0] * (x / xs[0]);
    size_t k = 0;
    while (k < xs.size() - 2 && x > xs[k + 1]) ++k;
    return ys[k] + (ys[k + 1] - ys[k]) * ((x - xs[k]) / (xs[k + 1] - xs[k]));
  }

  static void erase_value(std::vector<int32_t>& v, int32_t x) {
    auto it = std::find(v.begin(), v.end(), x);
    if (it != v.end()) v.erase(it);
  }

  // Sec. 4.4: the priority order of the unfinished requests, into `order`
  void priority_order() {
    order.clear();
    const int policy = cfg.policy;
    if (policy == S2L_SCHED_DEFAULT) {
      order.insert(order.end(), running.begin(), running.end());
      order.insert(order.end(), waiting.begin(), waiting.end());
      return;
    }
    order.assign(live.begin(), live.end());
    const Request* R = reqs.data();
    if (policy == S2L_SCHED_FCFS) {
      std::sort(order.begin(), order.end(), [R](int32_t a, int32_t b) {
        const Request &x = R[a], &y = R[b];
        if (x.complete != y.complete) return x.complete;
        if (x.arrival != y.arrival) return x.arrival < y.arrival;
        return x.seq < y.seq;
      });
    } else if (policy == S2L_SCHED_MCPS) {
      std::sort(order.begin(), order.end(), [R](int32_t a, int32_t b) {
        const Request &x = R[a], &y = R[b];
        if (x.computed != y.computed) return x.computed > y.computed;
        if (x.arrival != y.arrival) return x.arrival < y.arrival;
        return x.seq < y.seq;
      });
    } else {
      std::sort(order.begin(), order.end(), [R](int32_t a, int32_t b) {
        const Request &x = R[a], &y = R[b];
        if (x.complete != y.complete) return x.complete;
        if (x.last_chunk != y.last_chunk) return x.last_chunk > y.last_chunk;
        if (x.arrival != y.arrival) return x.arrival < y.arrival;
        return x.seq < y.seq;
      });
    }
  }

  void preempt(int32_t v, s2l_sched_step_out* out) {
    Request& r = reqs[v];
    const int32_t held = (int32_t)r.gpu.size();
    const double swap_cost = cfg.swap_fixed_seconds + cfg.swap_seconds_per_block * (double)held;
    const double rec_cost = recompute_latency((double)r.computed);
    int32_t kind;
    if (swap_cost < rec_cost && cpu.free_count() >= held) {
      r.cpu.clear();
      cpu.take(held, r.cpu);
      for (int32_t i = 0; i < held; ++i) {
        out->swap_out[2 * (out->num_swap_out + i)] = r.gpu[i];
        out->swap_out[2 * (out->num_swap_out + i) + 1] = r.cpu[i];
      }
      out->num_swap_out += held;
      gpu.give(r.gpu.begin(), r.gpu.end());
      r.gpu.clear();
      r.state = S2L_REQ_SWAPPED;
      ++r.n_swap;
      kind = S2L_EV_PREEMPT_SWAP;
    } else {
      gpu.give(r.gpu.begin(), r.gpu.end());
      r.gpu.clear();
      r.computed = 0;
      r.state = S2L_REQ_WAITING;
      ++r.n_recompute;
      kind = S2L_EV_PREEMPT_RECOMPUTE;
    }
    out->event_ids[out->num_events] = r.id;
    out->event_kinds[out->num_events] = kind;
    ++out->num_events;
    if (cfg.policy == S2L_SCHED_DEFAULT) {
      erase_value(running, v);
      waiting.insert(waiting.begin(), v);
    }
  }

  void step(s2l_sched_step_out* out) {
    const auto t0 = Clock::now();
    out->num_reqs = out->num_events = out->num_swap_out = out->num_swap_in = 0;
    out->total_tokens = 0;
    cpu.give(deferred_cpu.begin(), deferred_cpu.end());
    deferred_cpu.clear();

    // requests whose input is complete and fully computed finish
    tmp.clear();
    for (int32_t v : live) {
      Request& r = reqs[v];
      if (r.complete && r.computed == (int32_t)r.ids.size()) {
        gpu.give(r.gpu.begin(), r.gpu.end());
        cpu.give(r.cpu.begin(), r.cpu.end());
        r.gpu.clear();
        r.cpu.clear();
        r.state = S2L_REQ_FINISHED;
        out->event_ids[out->num_events] = r.id;
        out->event_kinds[out->num_events] = S2L_EV_FINISHED;
        ++out->num_events;
        if (cfg.policy == S2L_SCHED_DEFAULT) {
          erase_value(running, v);
          erase_value(waiting, v);
        }
      } else {
        tmp.push_back(v);
      }
    }
    live.swap(tmp);

    // Phase 1: order, then feasibility (no state changes)
    const auto t1 = Clock::now();
    priority_order();
    out->order_ns = ns_since(t1);
    int64_t budget = cfg.token_budget, claimed = 0;
    sel.clear();
    sel_n.clear();
    not_sched.clear();
    for (int32_t v : order) {
      const Request& r = reqs[v];
      const int64_t n = std::min<int64_t>((int64_t)r.ids.size() - r.computed, budget);
      const int32_t need = blocks_for(r.computed + std::max<int64_t>(n, 0));
      if (n <= 0 || claimed + need > cfg.num_gpu_blocks) {
        not_sched.push_back(v);
        continue;
      }
      claimed += need;
      budget -= n;
      sel.push_back(v);
      sel_n.push_back((int32_t)n);
    }

    // Phase 2: acquire blocks in priority order; preempt from the lowest priority up
    const int32_t M = cfg.max_blocks_per_req;
    size_t scan = not_sched.size();   // victims are taken from the end; a preempted request
                                      // holds no GPU blocks, so the scan never moves back
    for (size_t k = 0; k < sel.size(); ++k) {
      Request& r = reqs[sel[k]];
      const int32_t n = sel_n[k];
      const int32_t total = blocks_for((int64_t)r.computed + n);
      const bool swapped = r.state == S2L_REQ_SWAPPED;
      const int32_t missing = total - (swapped ? 0 : (int32_t)r.gpu.size());
      while (gpu.free_count() < missing) {
        while (scan > 0 && reqs[not_sched[scan - 1]].gpu.empty()) --scan;
        // phase 1 charged at most the whole pool, so a holder is always left
        preempt(not_sched[scan - 1], out);
      }
      if (swapped) {
        const int32_t nb = (int32_t)r.cpu.size();
        r.gpu.clear();
        gpu.take(nb, r.gpu);
        for (int32_t i = 0; i < nb; ++i) {
          out->swap_in[2 * (out->num_swap_in + i)] = r.cpu[i];
          out->swap_in[2 * (out->num_swap_in + i) + 1] = r.gpu[i];
        }
        out->num_swap_in += nb;
        deferred_cpu.insert(deferred_cpu.end(), r.cpu.begin(), r.cpu.end());
        r.cpu.clear();
      }
      gpu.take(total - (int32_t)r.gpu.size(), r.gpu);
      if (r.state != S2L_REQ_RUNNING) {
        r.state = S2L_REQ_RUNNING;
        if (cfg.policy == S2L_SCHED_DEFAULT) {
          erase_value(waiting, sel[k]);
          running.push_back(sel[k]);
        }
      }
      const int32_t q = out->num_reqs++;
      out->req_ids[q] = r.id;
      out->prefix_lens[q] = r.computed;
      out->chunk_lens[q] = n;
      int32_t* row = out->block_tables + (int64_t)q * M;
      std::copy(r.gpu.begin(), r.gpu.end(), row);
      std::fill(row + r.gpu.size(), row + M, cfg.table_pad);
      out->total_tokens += n;
      r.computed += n;
    }
    out->step_ns = ns_since(t0);
  }
};

namespace {

s2l_status find_live(s2l_sched* s, int64_t id, Request** r) {
  auto it = s->slot.find(id);
  if (it == s->slot.end()) return fail(S2L_EINVAL, "request %lld is unknown", (long long)id);
  Request& q = s->reqs[it->second];
  if (q.state == S2L_REQ_FINISHED) return fail(S2L_EINVAL, "request %lld has finished", (long long)id);
  if (q.complete) return fail(S2L_EINVAL, "request %lld: its input is already complete", (long long)id);
  *r = &q;
  return S2L_OK;
}

s2l_status check_ids(const int32_t* ids, int32_t n) {
  if (n < 0) return fail(S2L_EINVAL, "negative token count %d", n);
  if (n > 0 && !ids) return fail(S2L_EINVAL, "token ids are NULL");
  return S2L_OK;
}

}  // namespace

extern "C" {

int32_t s2l_lcp_len(const int32_t* a, int32_t na, const int32_t* b, int32_t nb) {
  const int32_t n = std::min(std::max(na, 0), std::max(nb, 0));
  if (n > 0 && (!a || !b)) return 0;
  int32_t k = 0;
  while (k < n && a[k] == b[k]) ++k;
  return k;
}

s2l_status s2l_sched_create(const s2l_sched_config* cfg, s2l_sched** out) {
  if (!cfg || !out) return fail(S2L_EINVAL, "config or output is NULL");
  const s2l_sched_config& c = *cfg;
  if (c.policy < S2L_SCHED_DEFAULT || c.policy > S2L_SCHED_LCAS) return fail(S2L_EINVAL, "unknown policy %d", c.policy);
  if (c.num_gpu_blocks < 1 || c.num_cpu_blocks < 0 || c.token_budget < 1 || c.max_blocks_per_req < 1)
    return fail(S2L_EINVAL, "pool sizes, budget and table length must be positive");
  if (c.reserved != 0) return fail(S2L_EINVAL, "reserved must be 0");
  if (c.num_recompute_points < 1 || !c.recompute_tokens || !c.recompute_seconds)
    return fail(S2L_EINVAL, "the recomputation model needs at least one point");
  for (int32_t i = 0; i < c.num_recompute_points; ++i) {
    if (!(c.recompute_tokens[i] > 0) || (i > 0 && !(c.recompute_tokens[i] > c.recompute_tokens[i - 1])))
      return fail(S2L_EINVAL, "recompute_tokens must be positive and strictly ascending");
  }
  s2l_sched* s = new s2l_sched(c);
  s->rec_x.assign(c.recompute_tokens, c.recompute_tokens + c.num_recompute_points);
  s->rec_y.assign(c.recompute_seconds, c.recompute_seconds + c.num_recompute_points);
  s->cfg.recompute_tokens = s->rec_x.data();
  s->cfg.recompute_seconds = s->rec_y.data();
  *out = s;
  return ok();
}

void s2l_sched_destroy(s2l_sched* s) { delete s; }

s2l_status s2l_sched_new_stream(s2l_sched* s, int64_t req_id, const int32_t* ids, int32_t n,
                                int32_t input_complete, double now) {
  if (!s) return fail(S2L_EINVAL, "scheduler is NULL");
  if (s2l_status st = check_ids(ids, n)) return st;
  if (s->slot.count(req_id)) return fail(S2L_EINVAL, "request %lld exists", (long long)req_id);
  if (blocks_for(n) > s->cfg.max_blocks_per_req)
    return fail(S2L_ERANGE, "%d tokens need more than %d blocks", n, s->cfg.max_blocks_per_req);
  Request r;
  r.id = req_id;
  r.ids.assign(ids, ids + n);
  r.complete = input_complete != 0;
  r.arrival = r.last_chunk = now;
  r.seq = (int64_t)s->reqs.size();
  const int32_t v = (int32_t)s->reqs.size();
  s->reqs.push_back(std::move(r));
  s->slot[req_id] = v;
  s->live.push_back(v);
  s->waiting.push_back(v);
  return ok();
}

s2l_status s2l_sched_append(s2l_sched* s, int64_t req_id, const int32_t* ids, int32_t n,
                            int32_t input_complete, double now) {
  if (!s) return fail(S2L_EINVAL, "scheduler is NULL");
  if (s2l_status st = check_ids(ids, n)) return st;
  Request* r;
  if (s2l_status st = find_live(s, req_id, &r)) return st;
  if (blocks_for((int64_t)r->ids.size() + n) > s->cfg.max_blocks_per_req)
    return fail(S2L_ERANGE, "%lld tokens need more than %d blocks", (long long)r->ids.size() + n,
                s->cfg.max_blocks_per_req);
  r->ids.insert(r->ids.end(), ids, ids + n);
  r->complete = input_complete != 0;
  r->last_chunk = now;
  return ok();
}

s2l_status s2l_sched_update(s2l_sched* s, int64_t req_id, const int32_t* ids, int32_t n,
                            int32_t input_complete, double now, int32_t* lcp_out) {
  if (!s) return fail(S2L_EINVAL, "scheduler is NULL");
  if (s2l_status st = check_ids(ids, n)) return st;
  Request* r;
  if (s2l_status st = find_live(s, req_id, &r)) return st;
  if (blocks_for(n) > s->cfg.max_blocks_per_req)
    return fail(S2L_ERANGE, "%d tokens need more than %d blocks", n, s->cfg.max_blocks_per_req);
  const int32_t lcp = s2l_lcp_len(r->ids.data(), (int32_t)r->ids.size(), ids, n);
  const int32_t keep = std::min(r->computed, lcp);
  r->invalidated += r->computed - keep;
  r->computed = keep;
  const int32_t nb = blocks_for(keep);
  if (r->state == S2L_REQ_SWAPPED) {
    s->cpu.give(r->cpu.begin() + nb, r->cpu.end());
    r->cpu.resize(nb);
    if (keep == 0) r->state = S2L_REQ_WAITING;
  } else {
    s->gpu.give(r->gpu.begin() + std::min<size_t>(nb, r->gpu.size()), r->gpu.end());
    if ((size_t)nb < r->gpu.size()) r->gpu.resize(nb);
  }
  r->ids.assign(ids, ids + n);
  r->complete = input_complete != 0;
  r->last_chunk = now;
  if (lcp_out) *lcp_out = lcp;
  return ok();
}

s2l_status s2l_sched_step(s2l_sched* s, s2l_sched_step_out* out) {
  if (!s || !out) return fail(S2L_EINVAL, "scheduler or output is NULL");
  if (!out->req_ids || !out->prefix_lens || !out->chunk_lens || !out->block_tables || !out->event_ids ||
      !out->event_kinds || !out->swap_out || !out->swap_in)
    return fail(S2L_EINVAL, "an output array is NULL");
  if (out->cap_reqs < (int32_t)s->live.size())
    return fail(S2L_ERANGE, "cap_reqs %d < %zu unfinished requests", out->cap_reqs, s->live.size());
  if (out->cap_swap < s->cfg.num_gpu_blocks)
    return fail(S2L_ERANGE, "cap_swap %d < num_gpu_blocks %d", out->cap_swap, s->cfg.num_gpu_blocks);
  s->step(out);
  return ok();
}

s2l_status s2l_sched_priority_order(s2l_sched* s, int64_t* ids, int32_t cap, int32_t* n, int64_t* order_ns) {
  if (!s || !n || (cap > 0 && !ids)) return fail(S2L_EINVAL, "scheduler, ids or n is NULL");
  const auto t0 = Clock::now();
  s->priority_order();
  if (order_ns) *order_ns = ns_since(t0);
  *n = (int32_t)s->order.size();
  for (int32_t i = 0; i < std::min(cap, *n); ++i) ids[i] = s->reqs[s->order[i]].id;
  return ok();
}

s2l_status s2l_sched_request(const s2l_sched* s, int64_t req_id, s2l_sched_req_info* info,
                             int32_t* gpu_blocks, int32_t* cpu_blocks) {
  if (!s || !info) return fail(S2L_EINVAL, "scheduler or info is NULL");
  auto it = s->slot.find(req_id);
  if (it == s->slot.end()) return fail(S2L_EINVAL, "request %lld is unknown", (long long)req_id);
  const Request& r = s->reqs[it->second];
  info->state = r.state;
  info->num_tokens = (int32_t)r.ids.size();
  info->num_computed_tokens = r.computed;
  info->input_complete = r.complete;
  info->total_tokens_invalidated = r.invalidated;
  info->num_preempt_swap = r.n_swap;
  info->num_preempt_recompute = r.n_recompute;
  info->num_gpu_blocks = (int32_t)r.gpu.size();
  info->num_cpu_blocks = (int32_t)r.cpu.size();
  info->arrival_time = r.arrival;
  info->last_chunk_arrival_time = r.last_chunk;
  if (gpu_blocks) std::copy(r.gpu.begin(), r.gpu.end(), gpu_blocks);
  if (cpu_blocks) std::copy(r.cpu.begin(), r.cpu.end(), cpu_blocks);
  return ok();
}

s2l_status s2l_sched_stats_get(const s2l_sched* s, s2l_sched_stats* st) {
  if (!s || !st) return fail(S2L_EINVAL, "scheduler or stats is NULL");
  st->num_unfinished = (int32_t)s->live.size();
  st->free_gpu_blocks = s->gpu.free_count();
  st->free_cpu_blocks = s->cpu.free_count();
  st->reserved = 0;
  return ok();
}

}  // extern "C"
