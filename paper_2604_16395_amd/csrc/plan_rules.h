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
constexpr int kDecodeTileCols = 16; // decode-shaped items: 16 columns, four waves over the keys
constexpr int kKvTile = 64;         // keys per LDS tile
constexpr int kMaxSplitsCap = 64;
constexpr int kDefaultMinSplitKeys = 512;
constexpr int kDefaultMaxSplits = 16;
constexpr int32_t kPlanMagic = 0x53324c50;  // "S2LP"

// Work items resident per CU: a 128-column item is a 4-wave workgroup with a two-stage
// K/V ring (64 KiB of LDS), two per CU, or with two key-range groups an 8-wave workgroup
// with two such rings (128 KiB), one per CU; a 256-column item is an 8-wave workgroup with
// a four-stage ring (128 KiB), one per CU; a 16-column item is a 4-wave workgroup whose
// waves hold two tiles of K and V in registers each (up to 512 registers), one per CU.
S2L_HD inline int32_t items_per_cu(int32_t tile_cols, int32_t key_halves) {
  return tile_cols == kMaxTileCols || tile_cols == kDecodeTileCols || key_halves == 2 ? 1 : 2;
}

struct PlanHeader {           // first 256 bytes of the workspace
  int32_t magic;
  int32_t num_reqs;
  int32_t hq, hkv, g, tq;
  int32_t num_items;
  int32_t num_split_reqs;
  int32_t split_keys;
  int32_t status;             // 0 ok, 1 = the device partition does not fit the host's sizing
  int32_t tile_cols;
  int32_t num_tiles;
  int64_t part_floats;
  int64_t total_tokens;
};

// One work item as the attention kernel reads it (a single 64-byte scalar load).
struct ItemRec {
  int32_t r, g, i0, i1;       // request, kv head, chunk tokens [i0, i1)
  int32_t lo, hi, s, ns;      // key range [lo, hi), piece s of ns
  int32_t p, c, row0, tile;   // P_r, C_r, first row of the request, query-tile index
  int64_t part_off;           // floats: start of the request's partials
  int32_t pad0, pad1;
};
static_assert(sizeof(ItemRec) == 64, "ItemRec is one 64-byte scalar load");

// a must be a power of two
S2L_HD inline int64_t align_up(int64_t x, int64_t a) {
  return (int64_t)(((uint64_t)x + (uint64_t)(a - 1)) & ~(uint64_t)(a - 1));
}
S2L_HD inline int32_t ceil_div(int32_t a, int32_t b) { return (a + b - 1) / b; }
S2L_HD inline int64_t ceil_div64(int64_t a, int64_t b) { return (a + b - 1) / b; }

S2L_HD inline int32_t tile_tokens(int32_t g, int32_t tile_cols) { return tile_cols / g; }
S2L_HD inline int32_t num_qtiles(int32_t c, int32_t tq) { return c > 0 ? ceil_div(c, tq) : 0; }

// Pieces of a request with piece length split_keys (0 = no split): every tile of the
// request is cut into the same number, set by its longest key range [0, P + C).
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
// unnormalised output row, then (m, l, 0, 0) per row.
S2L_HD inline int64_t req_part_floats(int32_t ns, int32_t c, int32_t hq) {
  return ns > 1 ? (int64_t)ns * c * hq * (kHeadDim + 4) : 0;
}

// Workspace layout (byte offsets), a function of the request count R, the item count W,
// the tile count NT and the partial floats (all four known to the host planner).
struct PlanLayout {
  int64_t item_off;   // int32 [R+1]   first item of each request
  int64_t ns;         // int32 [R]     pieces per request
  int64_t c;          // int32 [R]
  int64_t cu;         // int32 [R+1]
  int64_t part_off;   // int64 [R]
  int64_t items;      // ItemRec [W]
  int64_t partials;   // float [part_floats]
  int64_t end;
};

S2L_HD inline PlanLayout plan_layout(int32_t r, int64_t w, int64_t nt, int64_t part_floats) {
  PlanLayout L;
  int64_t o = 256;
  L.item_off = o; o += 4 * (int64_t)(r + 1);
  L.ns = o;       o += 4 * (int64_t)r;
  L.c = o;        o += 4 * (int64_t)r;
  L.cu = o;       o += 4 * (int64_t)(r + 1);
  o = align_up(o, 8);
  L.part_off = o; o += 8 * (int64_t)r;
  o = align_up(o, 64);
  L.items = o;    o += 64 * w;
  (void)nt;
  L.partials = align_up(o, 256);
  L.end = L.partials + align_up(part_floats * 4, 256);
  return L;
}

// The sizes a plan was made for (host plan); the layout and every launch derive from them.
struct PlanDims {
  int32_t num_reqs;
  int64_t num_items, num_tiles, part_floats;
};

// Typed pointers into a workspace, computed once on the host and passed to every kernel
// by value.  (Kernels never rebuild them from the layout arithmetic: a scalar load whose
// address the compiler splits into a misaligned base plus a misaligned immediate offset
// reads the wrong dwords on this hardware.)
struct PlanPtrs {
  PlanHeader* hdr;
  int32_t* item_off;
  int32_t* ns;
  int32_t* c;
  int32_t* cu;
  int64_t* part_off;
  ItemRec* items;
  float* partials;
  int64_t cap_items, cap_tiles, cap_part_floats;   // sizes the workspace was laid out for
};

inline PlanPtrs plan_ptrs(void* ws, const PlanDims& d) {
  char* b = static_cast<char*>(ws);
  PlanLayout L = plan_layout(d.num_reqs, d.num_items, d.num_tiles, d.part_floats);
  PlanPtrs q;
  q.hdr = reinterpret_cast<PlanHeader*>(b);
  q.item_off = reinterpret_cast<int32_t*>(b + L.item_off);
  q.ns = reinterpret_cast<int32_t*>(b + L.ns);
  q.c = reinterpret_cast<int32_t*>(b + L.c);
  q.cu = reinterpret_cast<int32_t*>(b + L.cu);
  q.part_off = reinterpret_cast<int64_t*>(b + L.part_off);
  q.items = reinterpret_cast<ItemRec*>(b + L.items);
  q.partials = reinterpret_cast<float*>(b + L.partials);
  q.cap_items = d.num_items;
  q.cap_tiles = d.num_tiles;
  q.cap_part_floats = d.part_floats;
  return q;
}

// Decode the local index of an item within its request: local = ((g * nqt) + t) * ns + s.
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

// Binned item order, for batches whose items differ in cost.  The (request, kv head) groups,
// requests longest first (by P + C; ties by index), each go whole to the XCD bin with the
// least work so far (lowest index on ties), so that a group's K/V pages are read by one
// L2; a bin's items then run in that order on its XCD.  Bins are padded with no-op records
// (request -1) to the length N of the longest, so logical item x N + k is item k of bin x and
// xcd_logical over 8 N workgroups sends bin x to XCD x.  Used when the bins' work is within
// 4% of their mean; otherwise items keep the longest-request-first order over all XCDs.  The
// host planner assigns the bins (it sizes the launch with them) and hands the device plan one
// bin per group; the device places each group's items with a scan of the bins' item counts.
constexpr int kBinnedMaxReqs = 256;      // requests the device plan ranks
constexpr int kBinnedMaxGroups = 1024;   // (request, kv head) groups a plan launch carries bins for
constexpr int64_t kItemCostKeys = 192;   // a work item's fixed cost (prologue and tail), in keys

// Work of one (request, kv head) group: the key ranges [0, P + i1) of its query tiles, plus
// the fixed cost of each of its nqt x ns items.
S2L_HD inline int64_t group_cost(int32_t p, int32_t c, int32_t tq, int32_t ns) {
  const int32_t nqt = num_qtiles(c, tq);
  int64_t k = 0;
  for (int32_t qt = 0; qt < nqt; ++qt) {
    const int32_t e = (qt + 1) * tq;
    k += (int64_t)p + (e < c ? e : c);
  }
  return k + kItemCostKeys * nqt * ns;
}

struct XcdBins {
  int64_t load[kNumXcds];
  int32_t count[kNumXcds];
};
S2L_HD inline void bins_init(XcdBins* b) {
  for (int x = 0; x < kNumXcds; ++x) {
    b->load[x] = 0;
    b->count[x] = 0;
  }
}
// The bin with the least work (lowest index on ties) takes a group of n items costing `cost`;
// returns the bin and sets *pos to the group's first position in it.
S2L_HD inline int32_t bins_place(XcdBins* b, int64_t cost, int32_t n, int32_t* pos) {
  // every index is a constant after unrolling, so the bins stay in registers on the device
  int32_t x = 0;
  int64_t least = b->load[0];
#pragma unroll
  for (int y = 1; y < kNumXcds; ++y)
    if (b->load[y] < least) {
      least = b->load[y];
      x = y;
    }
#pragma unroll
  for (int y = 0; y < kNumXcds; ++y)
    if (y == x) {
      *pos = b->count[y];
      b->count[y] += n;
      b->load[y] += cost;
    }
  return x;
}
S2L_HD inline int32_t bins_len(const XcdBins& b) {
  int32_t n = 0;
  for (int x = 0; x < kNumXcds; ++x) n = b.count[x] > n ? b.count[x] : n;
  return n;
}
S2L_HD inline bool bins_balanced(const XcdBins& b) {
  int64_t sum = 0, mx = 0;
  for (int x = 0; x < kNumXcds; ++x) {
    sum += b.load[x];
    mx = b.load[x] > mx ? b.load[x] : mx;
  }
  return sum > 0 && mx * kNumXcds * 25 <= sum * 26;
}

}  // namespace s2l
