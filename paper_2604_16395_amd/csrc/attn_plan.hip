// Device plan kernel: computes the varlen work partition of one step from the device
// length arrays (rules in plan_rules.h, identical to the host's) and stores it at the start
// of the caller's workspace: per-request arrays and one ItemRec per work item (so that an
// attention workgroup finds all it needs in one scalar load).  One workgroup.  The piece
// length comes from the host planner, which chose it from its copies of the lengths, and so
// does, for the binned item order, the XCD bin of each (request, kv head) group.
#include "launch.h"
#include "plan_rules.h"

namespace s2l {

namespace {

constexpr int kPlanThreads = 256;
constexpr int kPlanWaves = kPlanThreads / 64;
constexpr int kLdsReqs = 1024;   // batches up to this size keep their per-request values in LDS
constexpr int kRankReqs = kPlanThreads;   // batches up to this size are laid out longest first
static_assert(kRankReqs == kBinnedMaxReqs, "the binned order needs the ranking");

// Block-wide exclusive scan of N int64 values; returns the block totals in tot[].
template <int N>
__device__ void block_scan(const int64_t (&v)[N], int64_t (&excl)[N], int64_t (&tot)[N],
                           int64_t (*sh)[kPlanWaves]) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  int64_t x[N];
  for (int k = 0; k < N; ++k) x[k] = v[k];
  for (int o = 1; o < 64; o <<= 1) {
    for (int k = 0; k < N; ++k) {
      const int64_t y = __shfl_up(x[k], o);
      if (lane >= o) x[k] += y;
    }
  }
  if (lane == 63)
    for (int k = 0; k < N; ++k) sh[k][w] = x[k];
  __syncthreads();
  for (int k = 0; k < N; ++k) {
    int64_t before = 0, all = 0;
    for (int i = 0; i < kPlanWaves; ++i) {
      before += i < w ? sh[k][i] : 0;
      all += sh[k][i];
    }
    excl[k] = before + x[k] - v[k];
    tot[k] = all;
  }
}

// Largest r with a[r] <= x, for a non-decreasing a[0..n] with a[0] <= x < a[n].
template <typename A>
__device__ inline int upper_index(const A& a, int n, int x) {
  int lo = 0, hi = n;
  while (hi - lo > 1) {
    int mid = (lo + hi) >> 1;
    if (a[mid] <= x) lo = mid; else hi = mid;
  }
  return lo;
}

// Item order.  Up to kRankReqs requests are laid out longest first (by P + C, the key range
// of their longest tile; ties by index), so that when the items take several rounds of
// workgroups the longest start first and the dispatcher balances the tail; larger batches
// keep request order.  Then one pass over the requests in that order (a contiguous segment
// of slots per thread): pieces per request from the host's piece length, then a block scan
// of items, partial floats, tiles, split requests and tokens gives every offset and total.
__global__ __launch_bounds__(kPlanThreads) void attn_plan_kernel(PlanLaunch a, PlanPtrs pp) {
  __shared__ int64_t sh[5][kPlanWaves];
  __shared__ int32_t s_item_off[kLdsReqs + 1];
  __shared__ int32_t s_req[kLdsReqs], s_tile_off[kLdsReqs], s_ns[kLdsReqs], s_p[kLdsReqs], s_c[kLdsReqs],
      s_cu[kLdsReqs];
  __shared__ int64_t s_part[kLdsReqs];
  __shared__ int32_t s_key[kRankReqs], s_order[kRankReqs];
  __shared__ int64_t sh_bins[kNumXcds][kPlanWaves];
  __shared__ int32_t s_bin_cnt[kNumXcds];
  const int R = a.num_reqs;
  const int G = a.hq / a.hkv;
  const int tq = tile_tokens(G, a.tile_cols);
  const int split_keys = a.split_keys;
  const bool ranked = R <= kRankReqs;
  if (ranked) {
    const int t = threadIdx.x;
    int key = -1;
    if (t < R) {
      const int P = a.prefix_lens[t], C = a.chunk_lens[t];
      key = C > 0 ? P + C : -1;
      s_key[t] = key;
    }
    __syncthreads();
    if (t < R) {
      int rank = 0;
      for (int o = 0; o < R; ++o) {
        const int ko = s_key[o];
        rank += ko > key || (ko == key && o < t);
      }
      s_order[rank] = t;
    }
    __syncthreads();
  }
  auto req_at = [&](int k) { return ranked ? s_order[k] : k; };

  const int seg = (R + kPlanThreads - 1) / kPlanThreads;
  const int k0 = threadIdx.x * seg, k1 = min(R, k0 + seg);
  int64_t v[5] = {0, 0, 0, 0, 0}, excl[5], tot[5];
  for (int k = k0; k < k1; ++k) {
    const int r = req_at(k);
    const int P = a.prefix_lens[r], C = a.chunk_lens[r];
    const int ns = req_splits(P, C, split_keys, a.max_splits);
    const int64_t tiles = (int64_t)a.hkv * num_qtiles(C, tq);
    v[0] += tiles * ns;
    v[1] += req_part_floats(ns, C, a.hq);
    v[2] += tiles;
    v[3] += ns > 1 ? 1 : 0;
    v[4] += C;
  }
  block_scan<5>(v, excl, tot, sh);
  const int64_t num_items = tot[0], part_floats = tot[1], num_tiles = tot[2];
  int64_t items = excl[0], part = excl[1], tiles = excl[2];
  for (int k = k0; k < k1; ++k) {
    const int r = req_at(k);
    const int P = a.prefix_lens[r], C = a.chunk_lens[r];
    const int ns = req_splits(P, C, split_keys, a.max_splits);
    const int nqt = num_qtiles(C, tq);
    pp.item_off[r] = (int32_t)items;
    pp.ns[r] = ns;
    pp.c[r] = C;
    pp.cu[r] = a.cu_chunk[r];
    pp.part_off[r] = part;
    if (R <= kLdsReqs) {   // slot-ordered copies for the item search below
      s_item_off[k] = (int32_t)items;
      s_req[k] = r;
      s_tile_off[k] = (int32_t)tiles;
      s_ns[k] = ns;
      s_p[k] = P;
      s_c[k] = C;
      s_cu[k] = a.cu_chunk[r];
      s_part[k] = part;
    }
    items += (int64_t)a.hkv * nqt * ns;
    part += req_part_floats(ns, C, a.hq);
    tiles += (int64_t)a.hkv * nqt;
  }
  // Binned order (plan_rules.h): the host's bin of each (request, kv head) group, groups in
  // ranked order; a block scan of the bins' item counts over contiguous segments of groups
  // places every group's items in its bin.
  const bool binned = a.binned != 0 && ranked && R * a.hkv <= kBinnedMaxGroups;
  const int ngroups = R * a.hkv;
  const int gseg = (ngroups + kPlanThreads - 1) / kPlanThreads;
  const int q0 = min(ngroups, (int)threadIdx.x * gseg), q1 = min(ngroups, q0 + gseg);
  auto group_items = [&](int q) { const int k = q / a.hkv; return num_qtiles(s_c[k], tq) * s_ns[k]; };
  int64_t bin_before[kNumXcds], bin_total[kNumXcds];
  int64_t records = num_items;
  int bin_len = 0;
  if (binned) {
    __syncthreads();   // the slot-ordered request values are in LDS
    int64_t cnt[kNumXcds];
#pragma unroll
    for (int x = 0; x < kNumXcds; ++x) cnt[x] = 0;
    for (int q = q0; q < q1; ++q) {
      const int b = a.group_bin[q], n = group_items(q);
#pragma unroll
      for (int x = 0; x < kNumXcds; ++x) cnt[x] += x == b ? n : 0;
    }
    block_scan<kNumXcds>(cnt, bin_before, bin_total, sh_bins);
#pragma unroll
    for (int x = 0; x < kNumXcds; ++x) bin_len = max(bin_len, (int)bin_total[x]);
    if (threadIdx.x < kNumXcds) {
#pragma unroll
      for (int x = 0; x < kNumXcds; ++x)
        if (x == (int)threadIdx.x) s_bin_cnt[x] = (int)bin_total[x];
    }
    records = (int64_t)kNumXcds * bin_len;
  }
  const bool fits = records <= pp.cap_items && num_tiles <= pp.cap_tiles && part_floats <= pp.cap_part_floats;
  if (threadIdx.x == 0) {
    pp.item_off[R] = (int32_t)num_items;
    pp.cu[R] = a.cu_chunk[R];
    if (R <= kLdsReqs) s_item_off[R] = (int32_t)num_items;
    PlanHeader* h = pp.hdr;
    h->magic = kPlanMagic;
    h->num_reqs = R;
    h->hq = a.hq;
    h->hkv = a.hkv;
    h->g = G;
    h->tq = tq;
    h->num_items = fits ? (int32_t)records : 0;
    h->num_split_reqs = (int32_t)tot[3];
    h->split_keys = split_keys;
    h->status = fits ? 0 : 1;
    h->tile_cols = a.tile_cols;
    h->num_tiles = (int32_t)num_tiles;
    h->part_floats = part_floats;
    h->total_tokens = tot[4];
  }
  if (!fits) return;
  __syncthreads();   // request arrays (global and LDS) complete

  // The record of item `local` of the request at ranked slot k (request-local items: kv head
  // g, then query tile, then piece).
  auto make_rec = [&](int k, int local) {
    int r, tile0, P, C, ns, row0;
    int64_t part_off;
    if (R <= kLdsReqs) {
      r = s_req[k];
      tile0 = s_tile_off[k];
      P = s_p[k], C = s_c[k], ns = s_ns[k], row0 = s_cu[k], part_off = s_part[k];
    } else {   // request order (no ranking above kRankReqs requests), offsets in global memory
      r = k;
      tile0 = 0;
      for (int j = 0; j < r; ++j) tile0 += a.hkv * num_qtiles(a.chunk_lens[j], tq);
      P = a.prefix_lens[r], C = a.chunk_lens[r], ns = pp.ns[r], row0 = a.cu_chunk[r];
      part_off = pp.part_off[r];
    }
    const int nqt = num_qtiles(C, tq);
    const Item it = decode_local(local, nqt, ns);
    ItemRec rec;
    rec.r = r;
    rec.g = it.g;
    rec.i0 = it.qt * tq;
    rec.i1 = min(rec.i0 + tq, C);
    piece_range(P + rec.i1, ns, it.s, &rec.lo, &rec.hi);
    rec.s = it.s;
    rec.ns = ns;
    rec.p = P;
    rec.c = C;
    rec.row0 = row0;
    rec.tile = tile0 + it.g * nqt + it.qt;
    rec.part_off = part_off;
    rec.pad0 = rec.pad1 = 0;
    return rec;
  };
  if (binned) {
    // this thread's groups at their places in their bins, then the bins' padding (request -1)
    const int N = bin_len;
    int64_t at[kNumXcds];
#pragma unroll
    for (int x = 0; x < kNumXcds; ++x) at[x] = bin_before[x];
    for (int q = q0; q < q1; ++q) {
      const int k = q / a.hkv, gg = q % a.hkv, b = a.group_bin[q], n = group_items(q);
      int64_t pos = 0;
#pragma unroll
      for (int x = 0; x < kNumXcds; ++x)
        if (x == b) {
          pos = at[x];
          at[x] += n;
        }
      const int64_t base = (int64_t)b * N + pos;
      for (int j = 0; j < n; ++j) pp.items[base + j] = make_rec(k, gg * n + j);
    }
    for (int w = threadIdx.x; w < kNumXcds * N; w += kPlanThreads)
      if (w % N >= s_bin_cnt[w / N]) {
        ItemRec rec = {};
        rec.r = -1;
        pp.items[w] = rec;
      }
    return;
  }
  // one record per item; the request of item w is found by binary search over item offsets
  for (int w = threadIdx.x; w < (int)num_items; w += kPlanThreads) {
    const int k = R <= kLdsReqs ? upper_index(s_item_off, R, w) : upper_index(pp.item_off, R, w);
    const int off = R <= kLdsReqs ? s_item_off[k] : pp.item_off[k];
    pp.items[w] = make_rec(k, w - off);
  }
}

}  // namespace

hipError_t launch_attn_plan(const PlanLaunch& a, const PlanDims& dims, hipStream_t stream) {
  attn_plan_kernel<<<1, kPlanThreads, 0, stream>>>(a, plan_ptrs(a.workspace, dims));
  return hipGetLastError();
}

}  // namespace s2l
