// Varlen work partition for chunked-prefill attention: rules shared by the host
// (workspace sizing, grid sizing, s2l_plan_host) and the device plan kernel, so both
// derive the same partition from the same lengths.
//
// Work item = (request r, kv head g, query tile, key-range piece).  A query tile is
// tile_cols (128 or 256) packed columns of one kv head: tq = tile_cols / G consecutive
// chunk tokens times the G query heads that share kv head g (token-major: column n is
// token n / G, head g*G + n % G), so a tile's causal diagonal spans only tq tokens.  A
// tile with chunk tokens [i0, i1) needs keys [0, P + i1); that range is cut into `ns`
// pieces of a multiple of kKvTile keys when the batch has too few tiles to fill the GPU.
#pragma once
#include <stdint.h>

#if defined(__HIPCC__)
#define S2L_HD __host__ __device__
#else
#define S2L_HD
#endif

namespace s2l {

constexpr int kHeadDim = 128;
constexpr int kPageSize = 16;
constexpr int kMinTileCols = 128;   // packed (token, head) columns per work item: 4 waves x 32
constexpr int kMaxTileCols = 256;   //   or 8 waves x 32
constexpr int kKvTile = 64;         // keys per LDS tile
constexpr int kMaxSplitsCap = 64;
constexpr int kDefaultMinSplitKeys = 512;
constexpr int kDefaultMaxSplits = 16;
constexpr int kDefaultItemsPerCu = 2;
constexpr int32_t kPlanMagic = 0x53324c50;  // "S2LP"

struct PlanHeader {           // first 256 bytes of the workspace
  int32_t magic;
  int32_t num_reqs;
  int32_t hq, hkv, g, tq;
  int32_t num_items;
  int32_t num_split_reqs;
  int32_t split_keys;
  int32_t status;             // 0 ok, 1 = partials exceed the workspace (nothing planned)
  int32_t tile_cols;
  int32_t pad1;
  int64_t part_floats;
  int64_t total_tokens;
};

// a must be a power of two
S2L_HD inline int64_t align_up(int64_t x, int64_t a) {
  return (int64_t)(((uint64_t)x + (uint64_t)(a - 1)) & ~(uint64_t)(a - 1));
}
S2L_HD inline int32_t ceil_div(int32_t a, int32_t b) { return (a + b - 1) / b; }
S2L_HD inline int64_t ceil_div64(int64_t a, int64_t b) { return (a + b - 1) / b; }

S2L_HD inline int32_t tile_tokens(int32_t g, int32_t tile_cols) { return tile_cols / g; }
S2L_HD inline int32_t num_qtiles(int32_t c, int32_t tq) { return c > 0 ? ceil_div(c, tq) : 0; }

// Keys summed over the query tiles of one (request, kv head): tile t covers tokens
// [t*tq, min((t+1)*tq, C)) and reads keys [0, P + min((t+1)*tq, C)).
S2L_HD inline int64_t req_work(int32_t p, int32_t c, int32_t tq) {
  int64_t n = num_qtiles(c, tq);
  if (n == 0) return 0;
  return n * (int64_t)p + (int64_t)tq * (n - 1) * n / 2 + c;
}

// Piece length (keys) for the batch: 0 (no split) when the batch already has at least
// target_items tiles, else total keys / target_items, at least min_split_keys, rounded
// up to a multiple of kKvTile.
S2L_HD inline int32_t split_keys_for(int64_t base_items, int64_t total_work, int32_t target_items,
                                     int32_t min_split_keys) {
  if (base_items >= target_items || base_items == 0) return 0;
  int64_t l = ceil_div64(total_work, target_items);
  if (l < min_split_keys) l = min_split_keys;
  l = align_up(l, kKvTile);
  if (l > (int64_t)1 << 30) l = (int64_t)1 << 30;
  return (int32_t)l;
}

S2L_HD inline int32_t req_splits(int32_t p, int32_t c, int32_t split_keys, int32_t max_splits) {
  if (split_keys <= 0 || c <= 0) return 1;
  int64_t n = ceil_div64((int64_t)p + c, split_keys);
  if (n < 1) n = 1;
  if (n > max_splits) n = max_splits;
  return (int32_t)n;
}

// Key range [lo, hi) of piece s (of ns) of a tile whose range is [0, kv_end); may be empty.
S2L_HD inline void piece_range(int32_t kv_end, int32_t ns, int32_t s, int32_t* lo, int32_t* hi) {
  int32_t len = (int32_t)align_up(ceil_div(kv_end, ns), kKvTile);
  int32_t a = s * len;
  int32_t b = a + len < kv_end ? a + len : kv_end;
  *lo = a;
  *hi = b > a ? b : a;
}

// Floats of split partials for one request: ns pieces x C rows x Hq heads x (D + 4): the
// unnormalised output row, then (m, l_b, l_f, 0) per row.
S2L_HD inline int64_t req_part_floats(int32_t ns, int32_t c, int32_t hq) {
  return ns > 1 ? (int64_t)ns * c * hq * (kHeadDim + 4) : 0;
}

// Workspace layout (byte offsets), a function of R only.
struct PlanLayout {
  int64_t item_off;   // int32 [R+1]
  int64_t nqt;        // int32 [R]
  int64_t ns;         // int32 [R]
  int64_t p;          // int32 [R]
  int64_t c;          // int32 [R]
  int64_t cu;         // int32 [R+1]
  int64_t part_off;   // int64 [R]
  int64_t partials;   // float [part_floats]
};

S2L_HD inline PlanLayout plan_layout(int32_t r) {
  PlanLayout L;
  int64_t o = 256;
  L.item_off = o; o += 4 * (int64_t)(r + 1);
  L.nqt = o;      o += 4 * (int64_t)r;
  L.ns = o;       o += 4 * (int64_t)r;
  L.p = o;        o += 4 * (int64_t)r;
  L.c = o;        o += 4 * (int64_t)r;
  L.cu = o;       o += 4 * (int64_t)(r + 1);
  o = align_up(o, 8);
  L.part_off = o; o += 8 * (int64_t)r;
  L.partials = align_up(o, 256);
  return L;
}

S2L_HD inline int64_t workspace_bytes_for(int32_t r, int64_t part_floats) {
  return plan_layout(r).partials + align_up(part_floats * 4, 256);
}

// Typed pointers into a workspace, computed once on the host and passed to every kernel
// by value.  (Kernels never rebuild them from the layout arithmetic: a scalar load whose
// address the compiler splits into a misaligned base plus a misaligned immediate offset
// reads the wrong dwords on this hardware.)
struct PlanPtrs {
  PlanHeader* hdr;
  int32_t* item_off;
  int32_t* nqt;
  int32_t* ns;
  int32_t* p;
  int32_t* c;
  int32_t* cu;
  int64_t* part_off;
  float* partials;
};

inline PlanPtrs plan_ptrs(void* ws, int32_t r) {
  char* b = static_cast<char*>(ws);
  PlanLayout L = plan_layout(r);
  PlanPtrs q;
  q.hdr = reinterpret_cast<PlanHeader*>(b);
  q.item_off = reinterpret_cast<int32_t*>(b + L.item_off);
  q.nqt = reinterpret_cast<int32_t*>(b + L.nqt);
  q.ns = reinterpret_cast<int32_t*>(b + L.ns);
  q.p = reinterpret_cast<int32_t*>(b + L.p);
  q.c = reinterpret_cast<int32_t*>(b + L.c);
  q.cu = reinterpret_cast<int32_t*>(b + L.cu);
  q.part_off = reinterpret_cast<int64_t*>(b + L.part_off);
  q.partials = reinterpret_cast<float*>(b + L.partials);
  return q;
}

// Decode work item w of request r (local index = w - item_off[r]):
// local = ((g * nqt) + t) * ns + s.
struct Item {
  int32_t g, qt, s;
};
S2L_HD inline Item decode_local(int32_t local, int32_t nqt, int32_t ns) {
  Item it;
  it.s = local % ns;
  int32_t t = local / ns;
  it.qt = t % nqt;
  it.g = t / nqt;
  return it;
}

// WG dispatch goes round-robin over the 8 XCDs (each with its own L2).  Map workgroup b
// to a logical item so that each XCD receives one contiguous range of logical items:
// consecutive items share a (request, kv head) and hence its K/V pages.
constexpr int kNumXcds = 8;
S2L_HD inline int32_t xcd_logical(int32_t b, int32_t n) {
  int32_t x = b % kNumXcds, k = b / kNumXcds;
  int32_t per = n / kNumXcds, rem = n % kNumXcds;
  return x * per + (x < rem ? x : rem) + k;
}

}  // namespace s2l
