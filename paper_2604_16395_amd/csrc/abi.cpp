// C-ABI entry points: host-side validation, the host mirror of the work partition, and
// kernel launches.  Declarations and the full contract are in include/s2l.h.
#include "s2l.h"

#include <hip/hip_runtime_api.h>

#include <algorithm>
#include <cmath>
#include <cstddef>
#include <cstdarg>
#include <cstdio>
#include <string>
#include <vector>

#include "launch.h"
#include "plan_rules.h"
#include "status.h"

namespace {
thread_local std::string g_err;
}  // namespace

static_assert(offsetof(s2l::PlanHeader, status) == S2L_PLAN_STATUS_OFFSET,
              "the plan status word sits where the header says");

namespace s2l {

s2l_status fail(s2l_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  std::vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return st;
}

s2l_status ok() {
  g_err.clear();
  return S2L_OK;
}

}  // namespace s2l

namespace {

using s2l::fail;
using s2l::ok;

s2l_status hip_fail(const char* what, hipError_t e) {
  return fail(S2L_EHIP, "%s: %s", what, hipGetErrorString(e));
}

struct Resolved {
  int32_t target_items, min_split_keys, max_splits, tile_cols, key_halves;
};

// Automatic tile width: 16-column decode tiles when every request fits one (C * G <= 16:
// decode-shaped batches, bound by reading the keys); otherwise 256-column tiles (8-wave
// workgroups sharing each K/V tile, with a four-stage copy ring; the fastest layout
// measured on the 8K-prefix, 512-token step) unless they would be less than half full on
// average, as in batches of mostly decode-like rows; then 128.
int32_t auto_tile_cols(int32_t R, const int32_t* C, int32_t hq, int32_t hkv) {
  const int64_t g = hq / hkv;
  bool decode = g <= s2l::kDecodeTileCols;
  for (int32_t r = 0; r < R && decode; ++r) decode = (int64_t)C[r] * g <= s2l::kDecodeTileCols;
  if (decode) return s2l::kDecodeTileCols;
  int64_t used = 0, alloc = 0;
  for (int32_t r = 0; r < R; ++r) {
    const int64_t cols = (int64_t)C[r] * g;
    used += cols;
    alloc += s2l::ceil_div64(cols, s2l::kMaxTileCols) * s2l::kMaxTileCols;
  }
  return 2 * used >= alloc ? s2l::kMaxTileCols : s2l::kMinTileCols;
}

s2l_status resolve_opts(const s2l_plan_opts* o, bool need_cus, int32_t num_cus, int32_t R, const int32_t* C,
                        int32_t hq, int32_t hkv, Resolved* r) {
  int32_t t = o ? o->target_items : 0, m = o ? o->min_split_keys : 0, x = o ? o->max_splits : 0;
  int32_t tc = o ? o->tile_cols : 0, kh = o ? o->key_halves : 0;
  if (t < 0 || m < 0 || x < 0) return fail(S2L_EINVAL, "plan opts must be >= 0");
  if (tc != 0 && tc != s2l::kDecodeTileCols && tc != s2l::kMinTileCols && tc != s2l::kMaxTileCols)
    return fail(S2L_ENOTSUP, "tile_cols %d unsupported (0, 16, 128 or 256)", tc);
  if (tc == s2l::kDecodeTileCols && hq / hkv > s2l::kDecodeTileCols)
    return fail(S2L_ENOTSUP, "16-column tiles need at most 16 query heads per kv head (have %d)", hq / hkv);
  if (kh < 0 || kh > 2) return fail(S2L_ENOTSUP, "key_halves %d unsupported (0, 1 or 2)", kh);
  r->tile_cols = tc != 0 ? tc : auto_tile_cols(R, C, hq, hkv);
  if (r->tile_cols != s2l::kMinTileCols && kh == 2)
    return fail(S2L_ENOTSUP, "key_halves 2 needs 128-column tiles");
  r->key_halves = kh != 0 ? kh : (r->tile_cols == s2l::kMinTileCols ? 2 : 1);
  if (t == 0) {
    if (num_cus <= 0 && need_cus) {
      int dev = 0, n = 0;
      hipError_t e = hipGetDevice(&dev);
      if (e == hipSuccess) e = hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev);
      if (e != hipSuccess) return hip_fail("querying the CU count", e);
      num_cus = n;
    }
    if (num_cus <= 0) return fail(S2L_EINVAL, "num_cus must be > 0 when target_items is 0");
    t = s2l::items_per_cu(r->tile_cols, r->key_halves) * num_cus;
  }
  r->target_items = t;
  r->min_split_keys = (int32_t)s2l::align_up(m > 0 ? m : s2l::kDefaultMinSplitKeys, s2l::kKvTile);
  r->max_splits = x > 0 ? (x < s2l::kMaxSplitsCap ? x : s2l::kMaxSplitsCap) : s2l::kDefaultMaxSplits;
  return S2L_OK;
}

s2l_status check_heads(int32_t hq, int32_t hkv) {
  if (hq <= 0 || hkv <= 0) return fail(S2L_EINVAL, "head counts must be > 0 (hq=%d hkv=%d)", hq, hkv);
  if (hq % hkv != 0) return fail(S2L_EINVAL, "num_q_heads %d is not a multiple of num_kv_heads %d", hq, hkv);
  if (hq / hkv > s2l::kMinTileCols)
    return fail(S2L_ENOTSUP, "query heads per kv head %d exceeds %d", hq / hkv, s2l::kMinTileCols);
  return S2L_OK;
}

// Lengths from the host copies; device pointers checked only when `device` is set.
s2l_status check_batch(const s2l_batch* b, bool device, int64_t* total_tokens) {
  if (!b) return fail(S2L_EINVAL, "batch is NULL");
  if (b->num_reqs < 0) return fail(S2L_EINVAL, "num_reqs %d < 0", b->num_reqs);
  *total_tokens = 0;
  if (b->num_reqs == 0) return S2L_OK;
  if (!b->prefix_lens_host || !b->chunk_lens_host) return fail(S2L_EINVAL, "host length copies are NULL");
  if (device && (!b->prefix_lens || !b->chunk_lens || !b->cu_chunk || !b->block_tables))
    return fail(S2L_EINVAL, "a device batch array is NULL");
  if (device && b->max_pages_per_req <= 0) return fail(S2L_EINVAL, "max_pages_per_req must be > 0");
  int64_t t = 0;
  for (int32_t r = 0; r < b->num_reqs; ++r) {
    const int64_t p = b->prefix_lens_host[r], c = b->chunk_lens_host[r];
    if (p < 0 || c < 0) return fail(S2L_EINVAL, "request %d: negative length (P=%lld C=%lld)", r, (long long)p, (long long)c);
    if (p + c > ((int64_t)1 << 30)) return fail(S2L_EINVAL, "request %d: P+C=%lld exceeds 2^30", r, (long long)(p + c));
    if (device && p + c > (int64_t)b->max_pages_per_req * s2l::kPageSize)
      return fail(S2L_ERANGE, "request %d: P+C=%lld needs more than max_pages_per_req=%d pages", r,
                  (long long)(p + c), b->max_pages_per_req);
    t += c;
  }
  if (t >= ((int64_t)1 << 31)) return fail(S2L_EINVAL, "total chunk tokens %lld too large", (long long)t);
  *total_tokens = t;
  return S2L_OK;
}

s2l_status check_cache(const s2l_kv_cache* c, const s2l_batch* b) {
  if (!c) return fail(S2L_EINVAL, "cache is NULL");
  if (c->head_dim != s2l::kHeadDim) return fail(S2L_ENOTSUP, "head_dim %d unsupported (only 128)", c->head_dim);
  if (c->page_size != s2l::kPageSize) return fail(S2L_ENOTSUP, "page_size %d unsupported (only 16)", c->page_size);
  if (!c->k_pages || !c->v_pages) return fail(S2L_EINVAL, "k_pages/v_pages is NULL");
  if (c->num_pages <= 0 || c->num_kv_heads <= 0) return fail(S2L_EINVAL, "num_pages and num_kv_heads must be > 0");
  if (c->dtype == S2L_KV_FP8_E4M3) {
    if (!c->k_scale || !c->v_scale) return fail(S2L_EINVAL, "fp8 cache needs k_scale and v_scale");
  } else if (c->dtype == S2L_KV_BF16) {
    if (c->k_scale || c->v_scale) return fail(S2L_EINVAL, "bf16 cache must pass NULL scales");
  } else {
    return fail(S2L_EINVAL, "unknown kv dtype %d", c->dtype);
  }
  (void)b;
  return S2L_OK;
}

s2l::KvLaunch kv_launch(const s2l_kv_cache* c, const s2l_batch* b) {
  s2l::KvLaunch a;
  a.kpool = c->k_pages;
  a.vpool = c->v_pages;
  a.kscale = c->k_scale;
  a.vscale = c->v_scale;
  a.prefix_lens = b->prefix_lens;
  a.chunk_lens = b->chunk_lens;
  a.cu_chunk = b->cu_chunk;
  a.block_tables = b->block_tables;
  a.max_pages = b->max_pages_per_req;
  a.hkv = c->num_kv_heads;
  a.num_reqs = b->num_reqs;
  a.num_pages = c->num_pages;
  a.fp8 = c->dtype == S2L_KV_FP8_E4M3;
  return a;
}

// Items of the batch when every request is cut into pieces of at most split_keys keys.
int64_t items_for(int32_t R, const int32_t* P, const int32_t* C, int32_t hkv, int32_t tq, int32_t split_keys,
                  int32_t max_splits) {
  int64_t n = 0;
  for (int32_t r = 0; r < R; ++r)
    n += (int64_t)hkv * s2l::num_qtiles(C[r], tq) * s2l::req_splits(P[r], C[r], split_keys, max_splits);
  return n;
}

// Piece length of the batch: 0 (no split) when the batch already has at least target_items
// query tiles; else the shortest multiple of 64 keys (at least min_split_keys) for which
// cutting every request into ceil((P + C) / length) pieces (at most max_splits) gives no
// more than target_items items, so that one round of workgroups covers the launch and the
// longest item is as short as that allows.  Item counts fall as the length grows, so the
// shortest such length is found by bisection.
int32_t choose_split_keys(int32_t R, const int32_t* P, const int32_t* C, int32_t hkv, int32_t tq,
                          const Resolved& o) {
  int64_t tiles = 0, longest = 0;
  for (int32_t r = 0; r < R; ++r) {
    tiles += (int64_t)hkv * s2l::num_qtiles(C[r], tq);
    if (C[r] > 0 && (int64_t)P[r] + C[r] > longest) longest = (int64_t)P[r] + C[r];
  }
  if (tiles == 0 || tiles >= o.target_items) return 0;
  const int64_t lo_keys = s2l::align_up(o.min_split_keys, s2l::kKvTile);
  int64_t lo = lo_keys / s2l::kKvTile, hi = std::max(lo, s2l::ceil_div64(longest, s2l::kKvTile));
  if (items_for(R, P, C, hkv, tq, (int32_t)(lo * s2l::kKvTile), o.max_splits) <= o.target_items) return (int32_t)(lo * s2l::kKvTile);
  while (hi - lo > 1) {   // items(lo) > target >= items(hi); hi keys give one piece per tile
    const int64_t mid = (lo + hi) / 2;
    if (items_for(R, P, C, hkv, tq, (int32_t)(mid * s2l::kKvTile), o.max_splits) <= o.target_items) hi = mid;
    else lo = mid;
  }
  return (int32_t)(hi * s2l::kKvTile);
}

// Binned item order (plan_rules.h): requests ranked as the device plan ranks them, their
// (request, kv head) groups placed greedily.  Fills group_bin (if not NULL) by ranked slot and
// kv head, sets *len to the longest bin's item count, and returns whether the bins balance.
bool bin_groups(int32_t R, const int32_t* P, const int32_t* C, int32_t hkv, int32_t tq, int32_t split_keys,
                int32_t max_splits, uint8_t* group_bin, int32_t* len) {
  std::vector<int32_t> order(R);
  for (int32_t r = 0; r < R; ++r) order[r] = r;
  auto key = [&](int32_t r) { return C[r] > 0 ? P[r] + C[r] : -1; };
  std::stable_sort(order.begin(), order.end(), [&](int32_t a, int32_t b) { return key(a) > key(b); });
  s2l::XcdBins bins;
  s2l::bins_init(&bins);
  for (int32_t k = 0; k < R; ++k) {
    const int32_t r = order[k];
    const int32_t ns = s2l::req_splits(P[r], C[r], split_keys, max_splits);
    const int32_t n = s2l::num_qtiles(C[r], tq) * ns;
    const int64_t cost = s2l::group_cost(P[r], C[r], tq, ns);
    for (int32_t gg = 0; gg < hkv; ++gg) {
      int32_t pos;
      const int32_t x = s2l::bins_place(&bins, cost, n, &pos);
      if (group_bin) group_bin[k * hkv + gg] = (uint8_t)x;
    }
  }
  *len = s2l::bins_len(bins);
  return s2l::bins_balanced(bins);
}

// Host plan: the partition the device plan kernel stores (same rules, same order).
void host_plan(int32_t R, const int32_t* P, const int32_t* C, int32_t hq, int32_t hkv, const Resolved& o,
               s2l_plan_info* info, int32_t* items, int64_t cap) {
  const int32_t g = hq / hkv, tq = s2l::tile_tokens(g, o.tile_cols);
  int64_t tokens = 0;
  for (int32_t r = 0; r < R; ++r) tokens += C[r];
  const int32_t split_keys = choose_split_keys(R, P, C, hkv, tq, o);
  int64_t n_items = 0, part = 0, n_tiles = 0;
  int32_t n_split = 0;
  for (int32_t r = 0; r < R; ++r) {
    const int32_t ns = s2l::req_splits(P[r], C[r], split_keys, o.max_splits);
    const int32_t nqt = s2l::num_qtiles(C[r], tq);
    if (items) {
      for (int32_t gg = 0; gg < hkv; ++gg)
        for (int32_t qt = 0; qt < nqt; ++qt)
          for (int32_t s = 0; s < ns; ++s) {
            const int64_t k = n_items + ((int64_t)gg * nqt + qt) * ns + s;
            if (k >= cap) continue;
            const int32_t i0 = qt * tq, i1 = i0 + tq < C[r] ? i0 + tq : C[r];
            int32_t lo, hi;
            s2l::piece_range(P[r] + i1, ns, s, &lo, &hi);
            int32_t* row = items + 8 * k;
            row[0] = r; row[1] = gg; row[2] = i0; row[3] = i1;
            row[4] = lo; row[5] = hi; row[6] = s; row[7] = ns;
          }
    }
    n_items += (int64_t)hkv * nqt * ns;
    n_tiles += (int64_t)hkv * nqt;
    part += s2l::req_part_floats(ns, C[r], hq);
    n_split += ns > 1 ? 1 : 0;
  }
  info->num_items = (int32_t)n_items;
  info->num_split_reqs = n_split;
  info->split_keys = split_keys;
  info->num_q_heads = hq;
  info->num_kv_heads = hkv;
  info->num_reqs = R;
  info->total_tokens = tokens;
  info->workspace_bytes = s2l::plan_layout(R, n_items, n_tiles, part).end;
  info->tile_cols = o.tile_cols;
  info->num_tiles = (int32_t)n_tiles;
  info->part_floats = part;
  info->key_halves = o.key_halves;
  // item key ranges: tile t of request r covers keys [0, P + i1), cut into ns pieces
  int64_t keys_sum = 0, keys_max = 0;
  for (int32_t r = 0; r < R; ++r) {
    const int32_t ns = s2l::req_splits(P[r], C[r], split_keys, o.max_splits);
    const int32_t nqt = s2l::num_qtiles(C[r], tq);
    for (int32_t qt = 0; qt < nqt; ++qt) {
      const int32_t i1 = std::min((qt + 1) * tq, C[r]);
      const int64_t len = s2l::ceil_div64((int64_t)P[r] + i1, ns);
      keys_sum += len * ns * hkv;
      keys_max = std::max(keys_max, len);
    }
  }
  const bool uniform = n_items > 0 && keys_max * n_items <= keys_sum + keys_sum / 4;
  info->flags = uniform ? S2L_PLAN_UNIFORM : 0;
  // binned order (plan_rules.h) for batches of items of unequal cost, when its bins balance
  int32_t bin_len = 0;
  if (!uniform && n_items > 0 && R <= s2l::kBinnedMaxReqs && (int64_t)R * hkv <= s2l::kBinnedMaxGroups) {
    if (bin_groups(R, P, C, hkv, tq, split_keys, o.max_splits, nullptr, &bin_len)) {
      const int64_t padded = (int64_t)s2l::kNumXcds * bin_len;
      if (items)   // the rows past the real items are the bins' no-op padding
        for (int64_t k = n_items; k < padded && k < cap; ++k) {
          int32_t* row = items + 8 * k;
          row[0] = -1;
          for (int j = 1; j < 8; ++j) row[j] = 0;
        }
      info->num_items = (int32_t)padded;
      info->workspace_bytes = s2l::plan_layout(R, padded, n_tiles, part).end;
      info->flags = S2L_PLAN_BINNED;
    }
  }
}

s2l::PlanDims plan_dims(const s2l_plan_info* p) {
  s2l::PlanDims d;
  d.num_reqs = p->num_reqs;
  d.num_items = p->num_items;
  d.num_tiles = p->num_tiles;
  d.part_floats = p->part_floats;
  return d;
}

s2l_status check_plan(const s2l_plan_info* plan, const s2l_batch* b, int32_t hq, int32_t hkv, int64_t T,
                      const void* ws, size_t ws_bytes) {
  if (!plan) return fail(S2L_EINVAL, "plan info is NULL");
  if (plan->num_q_heads != hq || plan->num_kv_heads != hkv || plan->num_reqs != b->num_reqs ||
      plan->total_tokens != T)
    return fail(S2L_EINVAL, "plan was made for another batch or head count");
  if (plan->tile_cols != s2l::kDecodeTileCols && plan->tile_cols != s2l::kMinTileCols &&
      plan->tile_cols != s2l::kMaxTileCols)
    return fail(S2L_EINVAL, "plan info has an invalid tile width %d", plan->tile_cols);
  if (plan->tile_cols == s2l::kDecodeTileCols && hq / hkv > s2l::kDecodeTileCols)
    return fail(S2L_EINVAL, "plan info has 16-column tiles for %d query heads per kv head", hq / hkv);
  if (plan->key_halves != 1 && (plan->key_halves != 2 || plan->tile_cols != s2l::kMinTileCols))
    return fail(S2L_EINVAL, "plan info has an invalid key_halves %d", plan->key_halves);
  if (plan->num_items < 0 || plan->num_tiles < 0 || plan->part_floats < 0 ||
      s2l::plan_layout(plan->num_reqs, plan->num_items, plan->num_tiles, plan->part_floats).end !=
          plan->workspace_bytes)
    return fail(S2L_EINVAL, "plan info is inconsistent (not as returned by s2l_attn_plan)");
  if (!ws) return fail(S2L_EWORKSPACE, "workspace is NULL");
  if ((int64_t)ws_bytes < plan->workspace_bytes)
    return fail(S2L_EWORKSPACE, "workspace %zu bytes < %lld needed", ws_bytes, (long long)plan->workspace_bytes);
  return S2L_OK;
}

s2l_status attn_common(const s2l_kv_cache* cache, const s2l_batch* batch, const void* q, int32_t hq,
                       float scale, void* out, const s2l_plan_info* plan, const void* ws, size_t ws_bytes,
                       int64_t* T) {
  s2l_status st;
  if ((st = check_cache(cache, batch)) != S2L_OK) return st;
  if ((st = check_batch(batch, true, T)) != S2L_OK) return st;
  if ((st = check_heads(hq, cache->num_kv_heads)) != S2L_OK) return st;
  if (!(scale > 0.0f) || !std::isfinite(scale)) return fail(S2L_EINVAL, "softmax_scale must be finite and > 0");
  if (*T > 0 && (!q || !out)) return fail(S2L_EINVAL, "q/out is NULL");
  return check_plan(plan, batch, hq, cache->num_kv_heads, *T, ws, ws_bytes);
}

s2l_status attn_launch(const s2l_kv_cache* cache, const s2l_batch* batch, const void* q, int32_t num_q_heads,
                       float softmax_scale, void* out, float* lse, const s2l_plan_info* plan, void* workspace,
                       size_t ws_bytes, void* stream, const void* k_new = nullptr, const void* v_new = nullptr,
                       bool q8 = false) {
  int64_t T = 0;
  s2l_status st = attn_common(cache, batch, q, num_q_heads, softmax_scale, out, plan, workspace, ws_bytes, &T);
  if (st != S2L_OK) return st;
  s2l::AttnLaunch a;
  a.kv = kv_launch(cache, batch);
  a.q = q;
  a.out = out;
  a.lse = lse;
  a.hq = num_q_heads;
  a.softmax_scale = softmax_scale;
  a.workspace = workspace;
  a.dims = plan_dims(plan);
  a.tile_cols = plan->tile_cols;
  a.key_halves = plan->key_halves;
  a.group_by_xcd = (plan->flags & (S2L_PLAN_UNIFORM | S2L_PLAN_BINNED)) != 0;
  a.knew = k_new;
  a.vnew = v_new;
  a.q8 = q8;
  a.total_rows = T;
  (void)hipGetLastError();
  hipError_t e = s2l::launch_attn_main(a, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail("attn_main launch", e);
  return ok();
}

}  // namespace

extern "C" {

int32_t s2l_abi_version(void) { return S2L_ABI_VERSION; }

const char* s2l_last_error(void) { return g_err.c_str(); }

s2l_status s2l_calib_stream_read(const void* buf, size_t bytes, uint32_t* sink, int32_t grid, void* stream) {
  if (!buf || !sink) return fail(S2L_EINVAL, "buffer or sink is NULL");
  if (bytes == 0 || bytes % 16 != 0) return fail(S2L_EINVAL, "bytes must be a positive multiple of 16");
  if (grid <= 0) return fail(S2L_EINVAL, "grid must be > 0");
  (void)hipGetLastError();
  hipError_t e = s2l::launch_stream_read(buf, bytes, sink, grid, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail("stream_read launch", e);
  return ok();
}

s2l_status s2l_calib_mfma_bf16(int64_t iters, float* sink, int32_t grid, int64_t* flops_out, void* stream) {
  if (!sink) return fail(S2L_EINVAL, "sink is NULL");
  if (iters <= 0 || grid <= 0) return fail(S2L_EINVAL, "iters and grid must be > 0");
  (void)hipGetLastError();
  hipError_t e = s2l::launch_mfma_loop(iters, sink, grid, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail("mfma loop launch", e);
  if (flops_out) *flops_out = s2l::mfma_loop_flops(iters, grid);
  return ok();
}

s2l_status s2l_kv_append(const s2l_kv_cache* cache, const s2l_batch* batch, const void* k_new, const void* v_new,
                         void* stream) {
  s2l_status st;
  int64_t T = 0;
  if ((st = check_cache(cache, batch)) != S2L_OK) return st;
  if ((st = check_batch(batch, true, &T)) != S2L_OK) return st;
  if (T > 0 && (!k_new || !v_new)) return fail(S2L_EINVAL, "k_new/v_new is NULL");
  if (batch->num_reqs > 65535 || cache->num_kv_heads > 65535)
    return fail(S2L_ENOTSUP, "kv_append supports at most 65535 requests and kv heads");
  int32_t max_touched = 0;
  for (int32_t r = 0; r < batch->num_reqs; ++r) {
    const int32_t p = batch->prefix_lens_host[r], c = batch->chunk_lens_host[r];
    if (c <= 0) continue;
    const int32_t n = (p + c - 1) / s2l::kPageSize - p / s2l::kPageSize + 1;
    if (n > max_touched) max_touched = n;
  }
  (void)hipGetLastError();
  hipError_t e = s2l::launch_kv_append(kv_launch(cache, batch), k_new, v_new, max_touched,
                                       static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail("kv_append launch", e);
  return ok();
}

s2l_status s2l_check_tables(const s2l_kv_cache* cache, const s2l_batch* batch, int32_t* counts, void* stream) {
  s2l_status st;
  int64_t T = 0;
  if ((st = check_cache(cache, batch)) != S2L_OK) return st;
  if ((st = check_batch(batch, true, &T)) != S2L_OK) return st;
  if (!counts) return fail(S2L_EINVAL, "counts is NULL");
  int32_t max_used = 0;
  for (int32_t r = 0; r < batch->num_reqs; ++r) {
    const int64_t n = (int64_t)batch->prefix_lens_host[r] + batch->chunk_lens_host[r];
    max_used = std::max<int32_t>(max_used, (int32_t)((n + s2l::kPageSize - 1) / s2l::kPageSize));
  }
  (void)hipGetLastError();
  hipError_t e = s2l::launch_check_tables(kv_launch(cache, batch), max_used, counts, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail("check_tables launch", e);
  return ok();
}

// Swap between the device page pools and pinned host pools of the same layout.
static s2l_status kv_swap(const char* what, const s2l_kv_cache* cache, const int32_t* pairs, int32_t n,
                          const void* host_k, const void* host_v, int32_t num_host_pages, bool to_host,
                          void* stream) {
  s2l_status st;
  if ((st = check_cache(cache, nullptr)) != S2L_OK) return st;
  if (n < 0) return fail(S2L_EINVAL, "%s: negative pair count %d", what, n);
  if (n == 0) return ok();
  if (n > 65535 * 1024) return fail(S2L_EINVAL, "%s: %d pairs exceed one launch", what, n);
  if (!pairs) return fail(S2L_EINVAL, "%s: pairs is NULL", what);
  if (num_host_pages <= 0) return fail(S2L_EINVAL, "%s: num_host_pages must be > 0", what);
  void* dev_view[2] = {nullptr, nullptr};
  const void* host[2] = {host_k, host_v};
  for (int i = 0; i < 2; ++i) {
    if (!host[i]) return fail(S2L_EINVAL, "%s: host pool is NULL", what);
    hipPointerAttribute_t attr;
    hipError_t e = hipPointerGetAttributes(&attr, host[i]);
    (void)hipGetLastError();
    if (e != hipSuccess || attr.type != hipMemoryTypeHost || !attr.devicePointer)
      return fail(S2L_EINVAL, "%s: host pool %c is not pinned host memory (allocate it with hipHostMalloc)",
                  what, i ? 'v' : 'k');
    dev_view[i] = attr.devicePointer;
  }
  const int64_t page_bytes = (int64_t)cache->num_kv_heads * s2l::kPageSize * s2l::kHeadDim *
                             (cache->dtype == S2L_KV_FP8_E4M3 ? 1 : 2);
  (void)hipGetLastError();
  hipError_t e = to_host
      ? s2l::launch_kv_page_copy(cache->k_pages, cache->v_pages, dev_view[0], dev_view[1], pairs, n,
                                 cache->num_pages, num_host_pages, page_bytes, static_cast<hipStream_t>(stream))
      : s2l::launch_kv_page_copy(dev_view[0], dev_view[1], cache->k_pages, cache->v_pages, pairs, n,
                                 num_host_pages, cache->num_pages, page_bytes, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(what, e);
  return ok();
}

s2l_status s2l_kv_swap_out(const s2l_kv_cache* cache, const int32_t* pairs, int32_t n, void* host_k, void* host_v,
                           int32_t num_host_pages, void* stream) {
  return kv_swap("kv_swap_out", cache, pairs, n, host_k, host_v, num_host_pages, true, stream);
}

s2l_status s2l_kv_swap_in(const s2l_kv_cache* cache, const int32_t* pairs, int32_t n, const void* host_k,
                          const void* host_v, int32_t num_host_pages, void* stream) {
  return kv_swap("kv_swap_in", cache, pairs, n, host_k, host_v, num_host_pages, false, stream);
}

s2l_status s2l_kv_gather(const s2l_kv_cache* cache, const s2l_batch* batch, int32_t include_chunk,
                         const int32_t* cu_out, void* k_out, void* v_out, void* stream) {
  s2l_status st;
  int64_t T = 0;
  if ((st = check_cache(cache, batch)) != S2L_OK) return st;
  if ((st = check_batch(batch, true, &T)) != S2L_OK) return st;
  if (include_chunk != 0 && include_chunk != 1) return fail(S2L_EINVAL, "include_chunk must be 0 or 1");
  int32_t max_read = 0;
  for (int32_t r = 0; r < batch->num_reqs; ++r) {
    const int32_t n = batch->prefix_lens_host[r] + (include_chunk ? batch->chunk_lens_host[r] : 0);
    const int32_t pages = (n + s2l::kPageSize - 1) / s2l::kPageSize;
    if (pages > max_read) max_read = pages;
  }
  if (max_read > 0 && (!cu_out || !k_out || !v_out)) return fail(S2L_EINVAL, "cu_out/k_out/v_out is NULL");
  (void)hipGetLastError();
  hipError_t e = s2l::launch_kv_gather(kv_launch(cache, batch), include_chunk, cu_out, k_out, v_out, max_read,
                                       static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail("kv_gather launch", e);
  return ok();
}

s2l_status s2l_attn_workspace_bytes(const s2l_batch* batch, int32_t num_q_heads, int32_t num_kv_heads,
                                    const s2l_plan_opts* opts, size_t* bytes_out) {
  s2l_status st;
  int64_t T = 0;
  if (!bytes_out) return fail(S2L_EINVAL, "bytes_out is NULL");
  if ((st = check_batch(batch, false, &T)) != S2L_OK) return st;
  if ((st = check_heads(num_q_heads, num_kv_heads)) != S2L_OK) return st;
  Resolved o;
  if ((st = resolve_opts(opts, true, 0, batch->num_reqs, batch->chunk_lens_host, num_q_heads, num_kv_heads, &o)) !=
      S2L_OK)
    return st;
  s2l_plan_info info;
  host_plan(batch->num_reqs, batch->prefix_lens_host, batch->chunk_lens_host, num_q_heads, num_kv_heads, o, &info,
            nullptr, 0);
  *bytes_out = (size_t)info.workspace_bytes;
  return ok();
}

s2l_status s2l_attn_plan(const s2l_batch* batch, int32_t num_q_heads, int32_t num_kv_heads,
                         const s2l_plan_opts* opts, void* workspace, size_t ws_bytes, s2l_plan_info* info,
                         void* stream) {
  s2l_status st;
  int64_t T = 0;
  if (!info) return fail(S2L_EINVAL, "info is NULL");
  if ((st = check_batch(batch, true, &T)) != S2L_OK) return st;
  if (batch->num_reqs > 0 && !batch->cu_chunk) return fail(S2L_EINVAL, "cu_chunk is NULL");
  if ((st = check_heads(num_q_heads, num_kv_heads)) != S2L_OK) return st;
  Resolved o;
  if ((st = resolve_opts(opts, true, 0, batch->num_reqs, batch->chunk_lens_host, num_q_heads, num_kv_heads, &o)) !=
      S2L_OK)
    return st;
  s2l_plan_info pi;
  host_plan(batch->num_reqs, batch->prefix_lens_host, batch->chunk_lens_host, num_q_heads, num_kv_heads, o, &pi,
            nullptr, 0);
  if (!workspace) return fail(S2L_EWORKSPACE, "workspace is NULL");
  if ((int64_t)ws_bytes < pi.workspace_bytes)
    return fail(S2L_EWORKSPACE, "workspace %zu bytes < %lld needed", ws_bytes, (long long)pi.workspace_bytes);
  if (batch->num_reqs == 0 && !batch->cu_chunk) {
    *info = pi;  // empty batch: nothing for the kernels to read
    return ok();
  }
  s2l::PlanLaunch a;
  a.prefix_lens = batch->prefix_lens;
  a.chunk_lens = batch->chunk_lens;
  a.cu_chunk = batch->cu_chunk;
  a.num_reqs = batch->num_reqs;
  a.hq = num_q_heads;
  a.hkv = num_kv_heads;
  a.split_keys = pi.split_keys;
  a.max_splits = o.max_splits;
  a.tile_cols = o.tile_cols;
  a.binned = (pi.flags & S2L_PLAN_BINNED) != 0;
  if (a.binned) {
    int32_t len;
    const int32_t tq = s2l::tile_tokens(num_q_heads / num_kv_heads, o.tile_cols);
    bin_groups(batch->num_reqs, batch->prefix_lens_host, batch->chunk_lens_host, num_kv_heads, tq, pi.split_keys,
               o.max_splits, a.group_bin, &len);
  }
  a.ws_bytes = (int64_t)ws_bytes;
  a.workspace = workspace;
  (void)hipGetLastError();
  hipError_t e = s2l::launch_attn_plan(a, plan_dims(&pi), static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail("attn_plan launch", e);
  *info = pi;
  return ok();
}

s2l_status s2l_attn_main(const s2l_kv_cache* cache, const s2l_batch* batch, const void* q, int32_t num_q_heads,
                         float softmax_scale, void* out, float* lse, const s2l_plan_info* plan, void* workspace,
                         size_t ws_bytes, void* stream) {
  return attn_launch(cache, batch, q, num_q_heads, softmax_scale, out, lse, plan, workspace, ws_bytes, stream);
}

s2l_status s2l_split_reduce(const s2l_batch* batch, int32_t num_q_heads, void* out, float* lse,
                            const s2l_plan_info* plan, const void* workspace, size_t ws_bytes, void* stream) {
  int64_t T = 0;
  s2l_status st;
  if ((st = check_batch(batch, false, &T)) != S2L_OK) return st;
  if (!plan) return fail(S2L_EINVAL, "plan info is NULL");
  if ((st = check_plan(plan, batch, num_q_heads, plan->num_kv_heads, T, workspace, ws_bytes)) != S2L_OK) return st;
  if (plan->num_split_reqs == 0) return ok();
  if (!out) return fail(S2L_EINVAL, "out is NULL");
  s2l::ReduceLaunch a;
  a.out = out;
  a.lse = lse;
  a.workspace = workspace;
  a.hq = num_q_heads;
  a.num_reqs = batch->num_reqs;
  a.total_tokens = T;
  a.dims = plan_dims(plan);
  (void)hipGetLastError();
  hipError_t e = s2l::launch_split_reduce(a, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail("split_reduce launch", e);
  return ok();
}

s2l_status s2l_append_chunk_prefill_attn(const s2l_kv_cache* cache, const s2l_batch* batch, const void* k_new,
                                         const void* v_new, const void* q, int32_t num_q_heads, float softmax_scale,
                                         void* out, float* lse, const s2l_plan_info* plan, void* workspace,
                                         size_t ws_bytes, int32_t* fused_out, void* stream) {
  s2l_status st;
  int64_t T = 0;
  // Every argument of both halves is checked before anything is enqueued.
  if ((st = attn_common(cache, batch, q, num_q_heads, softmax_scale, out, plan, workspace, ws_bytes, &T)) != S2L_OK)
    return st;
  if (T > 0 && (!k_new || !v_new)) return fail(S2L_EINVAL, "k_new/v_new is NULL");
  bool fuse = cache->dtype == S2L_KV_BF16 && plan->tile_cols != s2l::kDecodeTileCols;
  for (int32_t r = 0; r < batch->num_reqs && fuse; ++r) fuse = batch->prefix_lens_host[r] % s2l::kPageSize == 0;
  if (!fuse && (batch->num_reqs > 65535 || cache->num_kv_heads > 65535))
    return fail(S2L_ENOTSUP, "kv_append supports at most 65535 requests and kv heads");
  if (fused_out) *fused_out = fuse ? 1 : 0;
  if (!fuse) {
    if ((st = s2l_kv_append(cache, batch, k_new, v_new, stream)) != S2L_OK) return st;
    return s2l_chunk_prefill_attn(cache, batch, q, num_q_heads, softmax_scale, out, lse, plan, workspace, ws_bytes,
                                  stream);
  }
  st = attn_launch(cache, batch, q, num_q_heads, softmax_scale, out, lse, plan, workspace, ws_bytes, stream,
                   T > 0 ? k_new : nullptr, T > 0 ? v_new : nullptr);
  if (st != S2L_OK) return st;
  return s2l_split_reduce(batch, num_q_heads, out, lse, plan, workspace, ws_bytes, stream);
}

s2l_status s2l_chunk_prefill_attn(const s2l_kv_cache* cache, const s2l_batch* batch, const void* q,
                                  int32_t num_q_heads, float softmax_scale, void* out, float* lse,
                                  const s2l_plan_info* plan, void* workspace, size_t ws_bytes, void* stream) {
  s2l_status st = attn_launch(cache, batch, q, num_q_heads, softmax_scale, out, lse, plan, workspace, ws_bytes,
                              stream);
  if (st != S2L_OK) return st;
  return s2l_split_reduce(batch, num_q_heads, out, lse, plan, workspace, ws_bytes, stream);
}

s2l_status s2l_chunk_prefill_attn_q8(const s2l_kv_cache* cache, const s2l_batch* batch, const void* q,
                                     int32_t num_q_heads, float softmax_scale, void* out, float* lse,
                                     const s2l_plan_info* plan, void* workspace, size_t ws_bytes, void* stream) {
  if (cache && cache->dtype != S2L_KV_FP8_E4M3)
    return fail(S2L_ENOTSUP, "the quantised-Q path needs an e4m3 cache");
  if (plan && plan->tile_cols == s2l::kDecodeTileCols)
    return fail(S2L_ENOTSUP, "the quantised-Q path has no 16-column (decode) tiles: plan with tile_cols 128 or 256");
  s2l_status st = attn_launch(cache, batch, q, num_q_heads, softmax_scale, out, lse, plan, workspace, ws_bytes,
                              stream, nullptr, nullptr, true);
  if (st != S2L_OK) return st;
  return s2l_split_reduce(batch, num_q_heads, out, lse, plan, workspace, ws_bytes, stream);
}

s2l_status s2l_chunk_prefill_attn_noalloc(const s2l_kv_cache* cache, const s2l_batch* batch, const void* q,
                                          int32_t num_q_heads, float softmax_scale, void* out, float* lse,
                                          const s2l_plan_opts* opts, s2l_plan_info* plan_out, void* stream) {
  s2l_status st;
  int64_t T = 0;
  if ((st = check_cache(cache, batch)) != S2L_OK) return st;
  if ((st = check_batch(batch, true, &T)) != S2L_OK) return st;
  if ((st = check_heads(num_q_heads, cache->num_kv_heads)) != S2L_OK) return st;
  if (!(softmax_scale > 0.0f) || !std::isfinite(softmax_scale))
    return fail(S2L_EINVAL, "softmax_scale must be finite and > 0");
  if (T > 0 && (!q || !out)) return fail(S2L_EINVAL, "q/out is NULL");
  Resolved o;
  if ((st = resolve_opts(opts, true, 0, batch->num_reqs, batch->chunk_lens_host, num_q_heads, cache->num_kv_heads,
                         &o)) != S2L_OK)
    return st;
  s2l_plan_info pi;
  host_plan(batch->num_reqs, batch->prefix_lens_host, batch->chunk_lens_host, num_q_heads, cache->num_kv_heads, o,
            &pi, nullptr, 0);
  if (pi.workspace_bytes > (int64_t)s2l::kNoAllocScratchBytes)
    return fail(S2L_EWORKSPACE,
                "this batch needs %lld bytes of workspace, more than the %zu bytes of scratch the allocation-free "
                "call holds; use s2l_chunk_prefill_attn with a caller workspace",
                (long long)pi.workspace_bytes, s2l::kNoAllocScratchBytes);
  void* ws = nullptr;
  hipError_t e = s2l::noalloc_scratch(&ws);
  if (e != hipSuccess) return hip_fail("taking the scratch array's device address", e);
  s2l_plan_info info;
  if ((st = s2l_attn_plan(batch, num_q_heads, cache->num_kv_heads, opts, ws, s2l::kNoAllocScratchBytes, &info,
                          stream)) != S2L_OK)
    return st;
  if ((st = s2l_chunk_prefill_attn(cache, batch, q, num_q_heads, softmax_scale, out, lse, &info, ws,
                                   s2l::kNoAllocScratchBytes, stream)) != S2L_OK)
    return st;
  if (plan_out) *plan_out = info;
  return ok();
}

s2l_status s2l_plan_host(int32_t num_reqs, const int32_t* prefix_lens_host, const int32_t* chunk_lens_host,
                         int32_t num_q_heads, int32_t num_kv_heads, const s2l_plan_opts* opts, int32_t num_cus,
                         s2l_plan_info* info, int32_t* items_out, int64_t item_capacity) {
  s2l_status st;
  if (!info) return fail(S2L_EINVAL, "info is NULL");
  s2l_batch b = {};
  b.num_reqs = num_reqs;
  b.prefix_lens_host = prefix_lens_host;
  b.chunk_lens_host = chunk_lens_host;
  int64_t T = 0;
  if ((st = check_batch(&b, false, &T)) != S2L_OK) return st;
  if ((st = check_heads(num_q_heads, num_kv_heads)) != S2L_OK) return st;
  Resolved o;
  if ((st = resolve_opts(opts, false, num_cus, num_reqs, chunk_lens_host, num_q_heads, num_kv_heads, &o)) !=
      S2L_OK)
    return st;
  if (item_capacity < 0) return fail(S2L_EINVAL, "item_capacity < 0");
  host_plan(num_reqs, prefix_lens_host, chunk_lens_host, num_q_heads, num_kv_heads, o, info, items_out,
            item_capacity);
  return ok();
}

}  // extern "C"
