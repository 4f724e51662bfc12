// Device plan kernel: computes the varlen work partition of one step from the device
// length arrays (rules in plan_rules.h, identical to the host's) and stores it, with a
// snapshot of the lengths, at the start of the caller's workspace.  One workgroup.
#include "launch.h"
#include "plan_rules.h"

namespace s2l {

namespace {

constexpr int kPlanThreads = 256;
constexpr int kPlanWaves = kPlanThreads / 64;

// Block-wide exclusive scan of three int64 values; returns the block totals in tot[].
__device__ void block_scan3(int64_t v[3], int64_t excl[3], int64_t tot[3], int64_t (*sh)[kPlanWaves]) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  int64_t x[3] = {v[0], v[1], v[2]};
  for (int o = 1; o < 64; o <<= 1) {
    for (int k = 0; k < 3; ++k) {
      int64_t y = __shfl_up(x[k], o);
      if (lane >= o) x[k] += y;
    }
  }
  if (lane == 63)
    for (int k = 0; k < 3; ++k) sh[k][w] = x[k];
  __syncthreads();
  if (threadIdx.x == 0) {
    int64_t run[3] = {0, 0, 0};
    for (int i = 0; i < kPlanWaves; ++i)
      for (int k = 0; k < 3; ++k) {
        int64_t t = sh[k][i];
        sh[k][i] = run[k];
        run[k] += t;
      }
    for (int k = 0; k < 3; ++k) tot[k] = run[k];
  }
  __syncthreads();
  for (int k = 0; k < 3; ++k) excl[k] = sh[k][w] + x[k] - v[k];
}

__global__ __launch_bounds__(kPlanThreads) void attn_plan_kernel(PlanLaunch a, PlanPtrs pp) {
  __shared__ int64_t sh[3][kPlanWaves];
  __shared__ int64_t tot[3];
  const int R = a.num_reqs;
  const int G = a.hq / a.hkv;
  const int tq = tile_tokens(G, a.tile_cols);
  int32_t* item_off = pp.item_off;
  int32_t* nqt_a = pp.nqt;
  int32_t* ns_a = pp.ns;
  int32_t* p_a = pp.p;
  int32_t* c_a = pp.c;
  int32_t* cu_a = pp.cu;
  int64_t* po_a = pp.part_off;

  // pass 1: tiles and keys of the whole batch
  const int seg = (R + kPlanThreads - 1) / kPlanThreads;
  const int r0 = threadIdx.x * seg, r1 = min(R, r0 + seg);
  int64_t v[3] = {0, 0, 0}, excl[3];
  for (int r = r0; r < r1; ++r) {
    const int P = a.prefix_lens[r], C = a.chunk_lens[r];
    v[0] += (int64_t)num_qtiles(C, tq) * a.hkv;
    v[1] += req_work(P, C, tq) * a.hkv;
    v[2] += C;
  }
  block_scan3(v, excl, tot, sh);
  const int64_t base_items = tot[0], total_work = tot[1], total_tokens = tot[2];
  const int32_t split_keys = split_keys_for(base_items, total_work, a.target_items, a.min_split_keys);
  __syncthreads();

  // pass 2: per-request pieces, item offsets and partial offsets
  v[0] = v[1] = v[2] = 0;
  for (int r = r0; r < r1; ++r) {
    const int P = a.prefix_lens[r], C = a.chunk_lens[r];
    const int ns = req_splits(P, C, split_keys, a.max_splits);
    v[0] += (int64_t)a.hkv * num_qtiles(C, tq) * ns;
    v[1] += req_part_floats(ns, C, a.hq);
    v[2] += ns > 1 ? 1 : 0;
  }
  block_scan3(v, excl, tot, sh);
  const int64_t num_items = tot[0], part_floats = tot[1], num_split = tot[2];
  const bool fits = workspace_bytes_for(R, part_floats) <= a.ws_bytes && num_items < ((int64_t)1 << 31);
  int64_t items = excl[0], part = excl[1];
  for (int r = r0; r < r1; ++r) {
    const int P = a.prefix_lens[r], C = a.chunk_lens[r];
    const int ns = req_splits(P, C, split_keys, a.max_splits);
    const int nqt = num_qtiles(C, tq);
    item_off[r] = (int32_t)items;
    nqt_a[r] = nqt;
    ns_a[r] = ns;
    p_a[r] = P;
    c_a[r] = C;
    cu_a[r] = a.cu_chunk[r];
    po_a[r] = part;
    items += (int64_t)a.hkv * nqt * ns;
    part += req_part_floats(ns, C, a.hq);
  }
  if (threadIdx.x == 0) {
    item_off[R] = (int32_t)num_items;
    cu_a[R] = a.cu_chunk[R];
    PlanHeader* h = pp.hdr;
    h->magic = kPlanMagic;
    h->num_reqs = R;
    h->hq = a.hq;
    h->hkv = a.hkv;
    h->g = G;
    h->tq = tq;
    h->num_items = fits ? (int32_t)num_items : 0;
    h->num_split_reqs = (int32_t)num_split;
    h->split_keys = split_keys;
    h->status = fits ? 0 : 1;
    h->tile_cols = a.tile_cols;
    h->pad1 = 0;
    h->part_floats = part_floats;
    h->total_tokens = total_tokens;
  }
}

}  // namespace

hipError_t launch_attn_plan(const PlanLaunch& a, hipStream_t stream) {
  attn_plan_kernel<<<1, kPlanThreads, 0, stream>>>(a, plan_ptrs(a.workspace, a.num_reqs));
  return hipGetLastError();
}

}  // namespace s2l
