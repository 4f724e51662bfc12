// Chunk-prefill attention over a paged KV cache, and the split-KV merge, for gfx950.
//
// What is computed (Stream2LLM Sec. 2.1 prefill over the pages of Sec. 2.2, resumed at
// num_computed_tokens as in Sec. 4.2): query i of a request's new chunk (absolute position
// t = P + i) attends to keys 0..t of that request, read through its block table.
//
// One workgroup = one work item of the plan: kv head g, 32 kColWaves packed query columns
// (tq tokens x G heads, token-major) and a key range [lo, hi).  With kHalves = 2 the
// workgroup has two groups of kColWaves waves on the same columns, each taking one half of
// the key range (in whole 64-key tiles) with its own K/V ring; the second group hands its
// (O, m, l) to the first through LDS at the end and the first merges them (the log-sum-exp
// merge of the online softmax), so a key range is split in two without any partials in
// memory.  The item's description is one 64-byte record written by the plan kernel (a
// single scalar load).
//
// Data movement.  K and V tiles of 64 keys x 128 are staged in LDS, one key row of 256
// bytes each, 16-byte chunks permuted per row (K: chunk c of row r at c ^ (r & 15); V: at
// c ^ 4 (r & 3)) so that the MFMA operand reads below hit 64 distinct banks.  bf16 pages
// are copied straight from HBM into LDS (buffer_load ... lds), each wave moving its share of
// one page of the tile; the buffer descriptor of a page ends at key `hi`, so keys past it
// arrive as zeros.  The tiles rotate through a ring of kStages LDS stages (four for the
// 8-wave bf16 kernel, which runs alone on its CU; two otherwise): K(t) and V(t) are fetched
// kStages - 1 iterations ahead of their use and each wave waits only for the copies that the
// next step reads (vmcnt(N), N > 0), so HBM latency hides behind several tiles of MFMA
// work.  Page ids: each wave keeps the page of 64 consecutive tiles in one VGPR (lane l:
// tile w0 + l; v_readlane picks a tile's), refilled from a window that an LDS-direct load
// fetched 64 tiles earlier, so the loop issues no scalar loads (their lgkmcnt would serialise
// the LDS operand waits).  E4M3 pages go through registers and are widened to bf16 on the way
// (exact), with a two-stage ring.
//
// Compute, per wave (32 query columns, one per lane pair), per 32-key sub-block b:
//   * S^T(b) = K Q^T with v_mfma_f32_32x32x16_bf16: A = K rows from LDS, B = Q held in
//     registers, so every lane owns one query column and 16 of the sub-block's scores;
//   * online softmax in the exp2 domain against a per-column reference m, set to the exact
//     max of the item's first sub-block (lane pair combined by v_permlane32_swap); later
//     probabilities exp2(s c - m) are accumulated against it as they come, so a sub-block
//     costs no max; only when one of them would exceed 2^64 (the row sum shows it) is m
//     raised to that sub-block's max and the sub-block redone.  The final division by the
//     accumulated sum makes the result independent of m;
//   * O^T += V^T P^T with the same MFMA: A = V^T read from the key-major V tile with the
//     transposing LDS read (ds_read_b64_tr_b16), B = bf16 P straight from the registers.
//     The row sum l adds up exactly these bf16 probabilities (v_dot2_f32_bf16), so O / l
//     applies weights that are normalised exactly; the log-sum-exp is m + log2 l.
// The sub-blocks are software pipelined: while the softmax of sub-block b runs on the
// VALU, the MFMA unit computes S(b+1) and O += P(b-1) V(b-1); P(b-1) is checked for
// overflow at the start of step b, before it enters O.  The causal mask is applied only to
// sub-blocks that reach past the first query token's position.
//
// Quantised-Q variant (e4m3 pages only): each lane pair encodes its column of Q to e4m3 with
// the column's own scale, K's codes stay e4m3 in LDS (same permuted chunk positions), and the
// two MFMAs of a step's S are v_mfma_f32_32x32x64_f8f6f4 (64 dims each); P V is unchanged.
//
// Unsplit items write bf16 O = acc / l (and LSE).  Split items write fp32 partials
// (acc, m, l) that split_reduce_kernel merges (the standard log-sum-exp merge of partial
// softmaxes); in the one-group bf16 layouts they are staged through LDS and stored as whole
// rows with write-through stores.
#include "launch.h"
#include "plan_rules.h"
#include "s2l_device.h"

namespace s2l {

namespace {

constexpr int kRowBytes = kHeadDim * 2;              // one bf16 key row in LDS
constexpr int kTileBytes = kKvTile * kRowBytes;      // 16 KiB
constexpr int kSubBytes = 32 * kRowBytes;            // one 32-key sub-block of a tile
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;
constexpr float kOverflow = 18446744073709551616.0f;   // 2^64: largest probability kept

// Raw buffer loads: a resource descriptor (base, size in bytes) in SGPRs plus a per-lane
// byte offset.  Offsets at or past the size read as zero.
constexpr int32_t kRsrcWord3 = 0x00020000;   // gfx9-family raw buffer: 32-bit dword format
__device__ inline __amdgpu_buffer_rsrc_t make_rsrc(const void* base, int32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, bytes, kRsrcWord3);
}

typedef __attribute__((address_space(3))) void lds_void;
typedef short v4i16 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) v4i16 lds_v4i16;

__device__ inline int clamp16(int x) { return x < 0 ? 0 : (x > 16 ? 16 : x); }

// LDS-direct copy: 64 lanes x 16 bytes from a raw buffer (descriptor words in SGPRs) to the
// 1 KiB of LDS at byte address `lds`, lane l's bytes at lds + 16 l.  Issued as inline
// assembly so that the compiler does not treat every later LDS read as waiting on it; the
// caller waits for the copy's vmcnt and synchronises before the destination is read.
typedef int32_t i32x4 __attribute__((ext_vector_type(4)));
__device__ inline i32x4 sgpr_rsrc(const void* base, int32_t bytes) {
  const uint64_t a = reinterpret_cast<uint64_t>(base);
  return i32x4{(int32_t)__builtin_amdgcn_readfirstlane((uint32_t)a),
               (int32_t)(__builtin_amdgcn_readfirstlane((uint32_t)(a >> 32)) & 0xffff),
               __builtin_amdgcn_readfirstlane(bytes), kRsrcWord3};
}
__device__ inline void lds_dma_b128(const i32x4& rs, uint32_t voff, uint32_t lds) {
  __asm__ volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tbuffer_load_dwordx4 %1, %2, 0 offen lds"
                   :: "s"(lds), "v"(voff), "s"(rs) : "m0");
}

// Wait until at most N vector-memory operations of this wave are outstanding (the older
// ones, issued first, are then complete); lgkm and exp counters are not waited for.
template <int N>
__device__ inline void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt is six bits");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}
// Lane `lane` of v into an SGPR, ordered with the surrounding assembly (the copies whose
// descriptor it feeds and the waits before it).  The nops cover the lane-select read of an
// SGPR written by SALU and the SGPR written here being read by a later buffer load.
__device__ inline int32_t readlane_ordered(int32_t v, int32_t lane) {
  int32_t r;
  __asm__ volatile("s_nop 4\n\tv_readlane_b32 %0, %1, %2\n\ts_nop 4" : "=s"(r) : "v"(v), "s"(lane));
  return r;
}
// LDS-direct copy of one dword per lane (lane l's dword to lds + 4 l), as lds_dma_b128.
__device__ inline void lds_dma_b32(const i32x4& rs, uint32_t voff, uint32_t lds) {
  __asm__ volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tbuffer_load_dword %1, %2, 0 offen lds"
                   :: "s"(lds), "v"(voff), "s"(rs) : "m0");
}

// Wait until this wave's LDS operations are complete (before a barrier that publishes them).
__device__ inline void wait_lgkmcnt0() { __builtin_amdgcn_s_waitcnt(15 | (3 << 14) | (7 << 4)); }

// Sub-block max of the 16 scores a lane holds, then over the lane pair (l, l ^ 32).  The
// scores come straight from MFMAs: the max must be ordinary code (the compiler forms
// v_max3 chains), so that the wait states an MFMA result needs before a VALU read are
// inserted; an assembly max here can read a partly accumulated score.
__device__ inline float block_max(const f32x16& s) {
  float mx = __builtin_fmaxf(s[0], s[1]);
#pragma unroll
  for (int e = 2; e < 16; ++e) mx = __builtin_fmaxf(mx, s[e]);
  return max_with_partner(mx);
}

// Instruction order the scheduler is asked for in one slot of a pipelined step: each MFMA
// followed by the LDS reads of a later slot and a few VALU instructions of the softmax.
template <bool kQK, bool kReads>
__device__ inline void slot_schedule() {
  if constexpr (kQK) {
    // the LDS reads go right after each MFMA, ahead of the VALU work (measured ~4% fewer
    // cycles per tile than VALU first)
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);     // MFMA (S)
    if constexpr (kReads) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);   // LDS read (K)
    __builtin_amdgcn_sched_group_barrier(0x002, 4, 0);     // VALU
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);     // MFMA (O)
    if constexpr (kReads) __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);   // LDS reads (V)
    __builtin_amdgcn_sched_group_barrier(0x002, 2, 0);
  } else {
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
    __builtin_amdgcn_sched_group_barrier(0x002, 6, 0);
    if constexpr (kReads) __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
  }
}

// Weight 2^(m_s - m*) of a piece in the log-sum-exp merge (0 for an empty piece).
__device__ inline float merge_weight(float m_s, float mstar) {
  return m_s == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(m_s - mstar);
}

// LDS of one group of waves: a K/V ring of kStages 16 KiB tiles each (four stages for the
// 8-column-wave bf16 kernel, which runs alone on its CU; two otherwise).
template <bool kFp8, int kColWaves, int kHalves>
struct Ring {
  static constexpr int kStages = (!kFp8 && kColWaves == 8) ? 4 : 2;
  static constexpr int kGroupBytes = 2 * kStages * kTileBytes;
  static constexpr int kBytes = kHalves * kGroupBytes;
};

template <bool kFp8, int kColWaves, int kHalves, bool kFused, bool kQ8>
__global__ __launch_bounds__(kColWaves * kHalves * 64, 8 / (kColWaves * kHalves)) void attn_main_kernel(
    const uint16_t* __restrict__ q, uint16_t* __restrict__ out, float* __restrict__ lse,
    void* kpool, void* vpool, const float* __restrict__ kscale,
    const float* __restrict__ vscale, const int32_t* __restrict__ block_tables, int32_t max_pages, int32_t hq,
    int32_t hkv, float scale_log2, PlanPtrs pv, int32_t group_by_xcd, const uint16_t* __restrict__ knew,
    const uint16_t* __restrict__ vnew, int64_t total_rows) {
  using RingT = Ring<kFp8, kColWaves, kHalves>;
  constexpr int kWaves = kColWaves * kHalves;
  constexpr int kS = RingT::kStages;
  static_assert(kHalves == 1 || kHalves == 2, "one or two key-range groups");
  static_assert(kHalves == 1 || kColWaves * 32 * 128 * 4 + kColWaves * 64 * 8 <= RingT::kBytes,
                "the second group's (O, m, l) fits in the LDS of the rings");
  constexpr int kQuarters = kColWaves / 4;           // waves sharing one page of a tile
  constexpr int kRowsPerWave = 16 / kQuarters;       // key rows each wave moves per tile
  constexpr int kDma = kRowsPerWave / 4;             // bf16: 1 KiB LDS-direct loads per wave
  constexpr int kF8Loads = kRowsPerWave / 8;         // e4m3: 16-byte loads per lane
  constexpr int kRun = kFp8 ? 16 * 128 : 16 * 128 * 2;   // bytes of one (page, kv head)
  constexpr int kKeyBytes = kRun / 16;
  __shared__ __attribute__((aligned(1024))) uint8_t smem[RingT::kBytes];
  __shared__ __attribute__((aligned(256))) int32_t s_pages[kWaves][2][64];   // next page windows

  // the item (one scalar load) and the device plan's item count, fetched together.  When
  // the items cost about the same, consecutive items (one kv head's pages) go to one XCD's
  // L2; otherwise workgroups take items in plan order (longest request first), which the
  // round-robin dispatch spreads evenly over the XCDs.
  const int w_item = group_by_xcd ? xcd_logical(blockIdx.x, gridDim.x) : (int)blockIdx.x;
  const ItemRec it = pv.items[w_item];
  const int W = pv.hdr->num_items;
  if (pv.hdr->status != 0) {   // the device plan did not fit this launch: nothing planned
    poison_outputs(out, lse, total_rows, hq);
    return;
  }
  if (w_item >= W || it.r < 0) return;   // past the plan's items, or a bin's padding
  const int P = it.p, C = it.c, row0 = it.row0, ns = it.ns, g = it.g;
  const int i0 = it.i0, i1 = it.i1;
  const int G = hq / hkv;
  const int tq = tile_tokens(G, 32 * kColWaves);
  const int32_t* bt = block_tables + (int64_t)it.r * max_pages;

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int grp = wave / kColWaves;                  // key-range group (0 or 1)
  const int cw = wave % kColWaves;                   // column wave within the group
  const int n = lane & 31, half = lane >> 5;
  const int col = cw * 32 + n;
  // This group's key range: the item's [it.lo, it.hi) cut into two halves of whole tiles
  // (the second may be a tile shorter, or empty); both groups step through nt0 tiles.
  const int nt_all = it.hi > it.lo ? ceil_div(it.hi - it.lo, kKvTile) : 0;
  const int nt0 = kHalves == 2 ? (nt_all + 1) >> 1 : nt_all;
  const int lo = it.lo + grp * nt0 * kKvTile;
  const int hi = kHalves == 2 && grp == 0 ? min(it.hi, lo + nt0 * kKvTile) : max(it.hi, lo);
  // LDS offsets below are relative to the group's ring at grp_base (folded into the per-lane
  // operand offsets and the copy destinations); K stages first, then V stages.
  const int grp_base = grp * RingT::kGroupBytes;
  constexpr int kKBase = 0;
  constexpr int kVBase = kS * kTileBytes;
  const int tok = i0 + col / G;
  const int hq_col = g * G + col % G;
  const bool valid = col < tq * G && tok < i1;
  const int horizon = valid ? P + tok : P + i1 - 1;   // last visible key of this column

  float c_log2 = scale_log2;
  float v_mul = 1.0f;
  if constexpr (kFp8) {
    c_log2 *= kscale[g];
    v_mul = vscale[g];
  }

  // Q^T operand: lane (n, half) holds Q[col][16 ks + 8 half .. +7] for ks = 0..7.
  bf16x8 qf[8];
  // kQ8: the column quantised to e4m3 with its own scale sq = max |Q[col]| / 448 (1 for a
  // zero column; both divisions correctly rounded, codes RNE with saturation, as the page
  // encoder); for the fp8 MFMA of k-half j lane (n, half) holds the codes of
  // Q[col][32 (2 j + half) + b], b < 32, and the scores take sq in their scale.
  i32x8 q8[2];
  if constexpr (!kQ8) {
    const uint16_t* qrow = q + ((int64_t)(row0 + (valid ? tok : 0)) * hq + (valid ? hq_col : 0)) * 128 + 8 * half;
#pragma unroll
    for (int ks = 0; ks < 8; ++ks) {
      u32x4 x = valid ? *reinterpret_cast<const u32x4*>(qrow + 16 * ks) : u32x4{0, 0, 0, 0};
      qf[ks] = __builtin_bit_cast(bf16x8, x);
    }
  } else {
    const uint16_t* qrow = q + ((int64_t)(row0 + (valid ? tok : 0)) * hq + (valid ? hq_col : 0)) * 128 + 32 * half;
    u32x4 x[8];   // x[4 j + i]: dims 32 (2 j + half) + 8 i .. + 7
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int i = 0; i < 4; ++i)
        x[4 * j + i] = valid ? *reinterpret_cast<const u32x4*>(qrow + 64 * j + 8 * i) : u32x4{0, 0, 0, 0};
    float amax = 0.f;
#pragma unroll
    for (int k = 0; k < 8; ++k)
#pragma unroll
      for (int w = 0; w < 4; ++w)
        amax = fmaxf(amax, fmaxf(fabsf(u2f(x[k][w] << 16)), fabsf(u2f(x[k][w] & 0xffff0000u))));
    amax = max_with_partner(amax);
    const float sq = amax > 0.f ? __fdiv_rn(amax, 448.f) : 1.f;
    const float inv = __fdiv_rn(1.f, sq);
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          const uint32_t w0 = x[4 * j + i][2 * h], w1 = x[4 * j + i][2 * h + 1];
          q8[j][2 * i + h] = (int)f32x4_to_fp8x4(u2f(w0 << 16) * inv, u2f(w0 & 0xffff0000u) * inv,
                                                 u2f(w1 << 16) * inv, u2f(w1 & 0xffff0000u) * inv);
        }
    c_log2 *= sq;
  }

  // LDS byte offsets of the operand reads, relative to a tile buffer.
  // K (A of S^T = K Q^T), k-step ks, sub-block 0: row n, chunk 2 ks + half.
  uint32_t ka[8];
#pragma unroll
  for (int ks = 0; ks < 8; ++ks) ka[ks] = grp_base + n * kRowBytes + ((((2 * ks + half) ^ (n & 15))) << 4);
  // kQ8: K stays e4m3 in LDS, the 8 16-byte chunks of a key's codes in the same permuted
  // positions of its 256-byte row slot (chunk c at c ^ (r & 15)); the fp8 MFMA of k-half j
  // reads chunks 4 j + 2 half and 4 j + 2 half + 1 of row n.
  uint32_t ka8[2][2];
#pragma unroll
  for (int j = 0; j < 2; ++j)
#pragma unroll
    for (int t = 0; t < 2; ++t) ka8[j][t] = grp_base + n * kRowBytes + (((4 * j + 2 * half + t) ^ (n & 15)) << 4);
  // V^T (A of O^T += V^T P^T), d-block db, first 4-key set of k-step 0: within each group
  // of 16 lanes, lane j addresses key row (j >> 2) at column 32 db + 16 ((l >> 4) & 1) +
  // 4 (j & 3); the transposing read hands lane i the four keys of column base + i, so lane
  // (n, half) receives V[keys 4 half + {0..3}, then (second read, +8 rows) 8 + 4 half +
  // {0..3}][32 db + n]: the k-slot order of the score registers it multiplies.
  uint32_t va[4];
  {
    const int j = lane & 15, b4 = (lane >> 4) & 1;
    const int row = 4 * half + (j >> 2);
#pragma unroll
    for (int db = 0; db < 4; ++db) {
      // The V stages start at kVBase (64 KiB with four stages): that base is added here, and
      // hidden from constant folding, so that the offsets within the V ring (below 64 KiB)
      // fit the LDS instructions' 16-bit immediate instead of costing an add per read.
      va[db] = kVBase + grp_base + row * kRowBytes + ((4 * (db ^ ((j >> 2) & 3)) + 2 * b4 + ((j >> 1) & 1)) << 4) +
               8 * (j & 1);
      __asm__ volatile("" : "+v"(va[db]));
    }
  }

  // Tile loads: column wave cw moves rows [s0, s0 + kRowsPerWave) of page pw of each tile.
  const int pw = cw / kQuarters;
  const int s0 = (cw % kQuarters) * kRowsPerWave;
  uint32_t kvo[kFp8 ? kF8Loads : kDma], vvo[kFp8 ? kF8Loads : kDma];
  // Fused append (bf16, page-aligned prefixes): keys at or past P, the chunk's own, are
  // copied straight from the new K/V rows (row stride hkv * 256 bytes) instead of the pages,
  // which this same launch writes; kno / vno are the lane offsets for that source.
  static_assert(!(kFp8 && kFused), "the fused append is for bf16 pages");
  static_assert(!kQ8 || kFp8, "Q is quantised only against e4m3 pages");
  const uint32_t new_stride = (uint32_t)hkv * kRowBytes;
  uint32_t kno[kFp8 ? 1 : kDma], vno[kFp8 ? 1 : kDma];
  if constexpr (!kFp8) {
    // LDS-direct load d writes tile rows 16 pw + s0 + 4d + (l >> 4), chunk l & 15: it
    // fetches the source chunk that the row's permutation puts there.
#pragma unroll
    for (int d = 0; d < kDma; ++d) {
      const int slot = s0 + 4 * d + (lane >> 4), c = lane & 15;
      kvo[d] = slot * kRowBytes + ((c ^ slot) << 4);
      vvo[d] = slot * kRowBytes + ((c ^ ((slot & 3) << 2)) << 4);
      kno[d] = slot * new_stride + ((c ^ slot) << 4);
      vno[d] = slot * new_stride + ((c ^ ((slot & 3) << 2)) << 4);
    }
  } else {
    // lane l loads bytes [16 f, 16 f + 16) of key slot s0 + l / kLpr (f as below)
#pragma unroll
    for (int i = 0; i < kF8Loads; ++i) {
      constexpr int kLpr = 8 / kF8Loads;
      const int slot = s0 + lane / kLpr, f = (lane % kLpr) * kF8Loads + i;
      kvo[i] = vvo[i] = slot * 128 + 16 * f;
    }
  }
  const char* kpb = static_cast<const char*>(kpool) + (int64_t)g * kRun;
  const char* vpb = static_cast<const char*>(vpool) + (int64_t)g * kRun;
  const int64_t page_stride = (int64_t)hkv * kRun;

  const int ntiles = nt0;                            // tile steps (the same in both groups)
  const int last_page = hi > lo ? (hi - 1) >> 4 : (it.hi > it.lo ? (it.hi - 1) >> 4 : 0);
  // Page ids.  Lane l of pg_win holds the physical page of this wave's page of tile
  // win0 + l (block-table entry lo/16 + 4 (win0 + l) + pw, clamped to the item's last
  // page, whose entry exists: a tile past the range is copied with a size-0 descriptor).
  // The next 64-tile window is copied into this wave's LDS slot 64 tiles before it is
  // needed, by an LDS-direct load that the per-iteration vmcnt waits cover (it is older than
  // the copies they wait for), and read into pg_win when the window moves on.  Page ids
  // never come from scalar loads inside the loop: those share lgkmcnt with the LDS reads,
  // whose waits would then all be full waits.
  const i32x4 bt_rs = sgpr_rsrc(bt, 4 * (last_page + 1));
  auto win_offset = [&](int w0) -> uint32_t {
    const int idx = (lo >> 4) + 4 * (w0 + lane) + pw;
    return 4u * (uint32_t)(idx < last_page ? idx : last_page);
  };
  int32_t pg_win = bt[(win_offset(0) >> 2)];     // tracked load, waited for with the Q loads
  int win0 = 0, win_slot = 0;
  auto fetch_window = [&](int w0, int slot) {
    lds_dma_b32(bt_rs, win_offset(w0),
                __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)(lds_void*)&s_pages[wave][slot][0]));
  };
  auto page_of = [&](int j) -> int32_t { return readlane_ordered(pg_win, j - win0); };

  // Page pg of the tile at key kb into the buffer at LDS byte `dst` (bf16: LDS-direct).
  auto dma_rows = [&](bool is_k, int32_t pg, int kb, int dst) {
    const uint32_t lds0 = (uint32_t)(uintptr_t)(lds_void*)smem;
    const int key0 = kb + 16 * pw;
    const int n = clamp16(hi - key0);
    if (kFused && key0 >= P) {
      // chunk rows of this kv head: new row (row0 + key0 - P + slot), one per key
      const char* nb = reinterpret_cast<const char*>(is_k ? knew : vnew) +
                       ((int64_t)(row0 + key0 - P) * hkv + g) * kRowBytes;
      const int bytes = __builtin_amdgcn_readfirstlane(n > 0 ? (n - 1) * (int)new_stride + kRowBytes : 0);
      const i32x4 rs = sgpr_rsrc(nb, bytes);
      const uint32_t* no = is_k ? kno : vno;
#pragma unroll
      for (int d = 0; d < kDma; ++d) {
        const int row = 16 * pw + s0 + 4 * d;
        lds_dma_b128(rs, no[d], __builtin_amdgcn_readfirstlane(lds0 + grp_base + dst + row * kRowBytes));
      }
      return;
    }
    const int bytes = __builtin_amdgcn_readfirstlane(n * kKeyBytes);
    const i32x4 rs = sgpr_rsrc((is_k ? kpb : vpb) + (int64_t)pg * page_stride, bytes);
    const uint32_t* vo = is_k ? kvo : vvo;
#pragma unroll
    for (int d = 0; d < kDma; ++d) {
      const int row = 16 * pw + s0 + 4 * d;
      lds_dma_b128(rs, vo[d], __builtin_amdgcn_readfirstlane(lds0 + grp_base + dst + row * kRowBytes));
    }
  };
  struct F8Stage {
    u32x4 x[kF8Loads];
  };
  auto f8_load = [&](F8Stage& st, const char* base, int32_t pg, int kb, const uint32_t* vo) {
    const int bytes = __builtin_amdgcn_readfirstlane(clamp16(hi - (kb + 16 * pw)) * kKeyBytes);
    const auto rs = make_rsrc(base + (int64_t)pg * page_stride, bytes);
#pragma unroll
    for (int i = 0; i < kF8Loads; ++i)
      st.x[i] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(rs, vo[i], 0, 0));
  };
  // e4m3 -> bf16 into the permuted rows: 16 codes = bf16 chunks 2f, 2f + 1.
  auto f8_store = [&](const F8Stage& st, int dst, bool is_k) {
#pragma unroll
    for (int i = 0; i < kF8Loads; ++i) {
      constexpr int kLpr = 8 / kF8Loads;
      const int row = 16 * pw + s0 + lane / kLpr, f = (lane % kLpr) * kF8Loads + i;
      if (kQ8 && is_k) {   // the codes as they are, chunk f at f ^ (row & 15)
        *reinterpret_cast<u32x4*>(smem + grp_base + dst + row * kRowBytes + ((f ^ (row & 15)) << 4)) = st.x[i];
        continue;
      }
      const int sw = is_k ? (row & 15) : ((row & 3) << 2);
      const u32x2 a = fp8x4_to_bf16x4(st.x[i][0]);
      const u32x2 b = fp8x4_to_bf16x4(st.x[i][1]);
      const u32x2 c = fp8x4_to_bf16x4(st.x[i][2]);
      const u32x2 d = fp8x4_to_bf16x4(st.x[i][3]);
      uint8_t* rp = smem + grp_base + dst + row * kRowBytes;
      *reinterpret_cast<u32x4*>(rp + (((2 * f) ^ sw) << 4)) = u32x4{a[0], a[1], b[0], b[1]};
      *reinterpret_cast<u32x4*>(rp + (((2 * f + 1) ^ sw) << 4)) = u32x4{c[0], c[1], d[0], d[1]};
    }
  };

  f32x16 o[4];
#pragma unroll
  for (int db = 0; db < 4; ++db) o[db] = f32x16{};
  float m_run = 0.f;
  float l_run = 0.f;   // sum of the bf16 probabilities exactly as P.V uses them

  // kQ8: the e4m3 codes of K for the fp8 MFMA of k-half j, sub-block at LDS byte `kofs`.
  auto read_k8 = [&](int kofs, int j) {
    const u32x4 lo = *reinterpret_cast<const u32x4*>(smem + kofs + ka8[j][0]);
    const u32x4 hi = *reinterpret_cast<const u32x4*>(smem + kofs + ka8[j][1]);
    return i32x8{(int)lo[0], (int)lo[1], (int)lo[2], (int)lo[3], (int)hi[0], (int)hi[1], (int)hi[2], (int)hi[3]};
  };
  // S^T += K Q^T over 64 dims in e4m3 (both operands' codes; their scales are in c_log2)
  auto mfma_q8 = [&](const i32x8& a, const i32x8& b, const f32x16& c) {
    return __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a, b, c, 0, 0, 0, 0, 0, 0);
  };
  // S(b+1) = K(b+1) Q^T from the sub-block at LDS byte `kofs`.
  auto qk = [&](int kofs) {
    f32x16 s = f32x16{};
    if constexpr (kQ8) {
      s = mfma_q8(read_k8(kofs, 0), q8[0], s);
      s = mfma_q8(read_k8(kofs, 1), q8[1], s);
    } else {
#pragma unroll
      for (int ks = 0; ks < 8; ++ks) {
        const bf16x8 a = *reinterpret_cast<const bf16x8*>(smem + kofs + ka[ks]);
        s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qf[ks], s, 0, 0, 0);
      }
    }
    return s;
  };
  // One A fragment of O^T += V^T P^T: keys 16 k2 + (4-key sets of this lane half), d-block db.
  auto read_v = [&](int vofs, int k2, int db) {
    const uint8_t* base = smem + (vofs - kVBase) + 16 * k2 * kRowBytes + va[db];
    const v4i16 x = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16*)(base));
    const v4i16 y = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16*)(base + 8 * kRowBytes));
    const u32x2 ux = __builtin_bit_cast(u32x2, x), uy = __builtin_bit_cast(u32x2, y);
    return __builtin_bit_cast(bf16x8, u32x4{ux[0], ux[1], uy[0], uy[1]});
  };
  // O += P V over the sub-block whose V rows start at LDS byte `vofs`.
  auto pv_acc = [&](const u32x4* p, int vofs) {
#pragma unroll
    for (int k2 = 0; k2 < 2; ++k2) {
      const bf16x8 pb = __builtin_bit_cast(bf16x8, p[k2]);
#pragma unroll
      for (int db = 0; db < 4; ++db) o[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(read_v(vofs, k2, db), pb, o[db], 0, 0, 0);
    }
  };
  auto read_k = [&](int kofs, int ks) { return *reinterpret_cast<const bf16x8*>(smem + kofs + ka[ks]); };
  // Operands of a step's first two slots, read before its (branchy) softmax prologue.
  struct Pre {
    bf16x8 k[2], v[2];
    i32x8 k8[2];   // kQ8: both fp8 K operands of the step
  };
  auto prefetch = [&](int kofs, int vofs, auto with_qk) {
    Pre f;
    if constexpr (decltype(with_qk)::value) {
      if constexpr (kQ8) {
        f.k8[0] = read_k8(kofs, 0);
        f.k8[1] = read_k8(kofs, 1);
      } else {
        f.k[0] = read_k(kofs, 0);
        f.k[1] = read_k(kofs, 1);
      }
    }
    f.v[0] = read_v(vofs, 0, 0);
    f.v[1] = read_v(vofs, 0, 1);
    return f;
  };
  // Pipelined step in eight slots; slot i issues S(b+1) += K_i Q_i (k-step i), O_db +=
  // V^T P(b-1) (k2 = i / 4, db = i % 4) and the probabilities of score elements 2i, 2i+1
  // of sub-block b, while the operands of slot i + 2 are read from LDS.  With a next step
  // in the same tile (with_next), slots 6 and 7 also read that step's first two operands
  // (at nkofs / nvofs) into nxt, so its reads are not exposed behind its softmax prologue.
  auto step_main = [&](const f32x16& s, const u32x4* pp, u32x4* po, int kofs, int vofs, const Pre& f,
                       auto with_qk, float& lsum, auto with_next, int nkofs, int nvofs, Pre& nxt, auto&& hook) {
    constexpr bool kQK = decltype(with_qk)::value;
    constexpr bool kNext = decltype(with_next)::value;
    f32x16 sn = f32x16{};
    bf16x8 kf[10], vf[10];
    kf[0] = f.k[0];
    kf[1] = f.k[1];
    vf[0] = f.v[0];
    vf[1] = f.v[1];
    float l0 = 0.f, l1 = 0.f;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      if (i + 2 < 8) {
        if constexpr (kQK && !kQ8) kf[i + 2] = read_k(kofs, i + 2);
        vf[i + 2] = read_v(vofs, (i + 2) >> 2, (i + 2) & 3);
      } else if constexpr (kNext) {
        if constexpr (kQ8) nxt.k8[i - 6] = read_k8(nkofs, i - 6);
        else nxt.k[i - 6] = read_k(nkofs, i - 6);
        nxt.v[i - 6] = read_v(nvofs, 0, i - 6);
      }
      if constexpr (kQK && kQ8) {
        if (i < 2) sn = mfma_q8(f.k8[i], q8[i], sn);   // the two fp8 MFMAs in the first slots
      } else if constexpr (kQK) {
        sn = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[i], qf[i], sn, 0, 0, 0);
      }
      o[i & 3] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf[i], __builtin_bit_cast(bf16x8, pp[i >> 2]), o[i & 3],
                                                          0, 0, 0);
      const float p0 = __builtin_amdgcn_exp2f(__builtin_fmaf(s[2 * i], c_log2, -m_run));
      const float p1 = __builtin_amdgcn_exp2f(__builtin_fmaf(s[2 * i + 1], c_log2, -m_run));
      const uint32_t pk = pack_bf16x2(p0, p1);
      po[i >> 2][i & 3] = pk;
      if (i & 1) l1 = sum_bf16x2(pk, l1);
      else l0 = sum_bf16x2(pk, l0);
      if (i == 1) hook();
    }
    lsum = l0 + l1;
    __asm__ volatile("" ::"v"(po[0]), "v"(po[1]), "v"(lsum));   // produced here, not sunk
    if constexpr (!kQ8) {
      slot_schedule<kQK, true>();
      slot_schedule<kQK, true>();
      slot_schedule<kQK, true>();
      slot_schedule<kQK, true>();
      slot_schedule<kQK, true>();
      slot_schedule<kQK, true>();
      slot_schedule<kQK, kNext>();
      slot_schedule<kQK, kNext>();
    }
    return sn;
  };
  // Mask of sub-block sb0 (element e of a lane's scores is key sb0 + 8 (e / 4) + 4 half +
  // e % 4): keys past the column's position (causal) or at or past the group's range end,
  // applied only where the sub-block reaches past the first query token or the range end.
  const int mask_from = min(P + i0, hi - 1);
  const int key_lim = min(horizon, hi - 1);
  auto mask = [&](f32x16& s, int sb0) {
    if (sb0 + 31 > mask_from) {
      __asm__ volatile("" ::);   // keep this a branch (not predicated into every sub-block)
      const int lim = key_lim - sb0 - 4 * half;
#pragma unroll
      for (int e = 0; e < 16; ++e) s[e] = 8 * (e >> 2) + (e & 3) > lim ? -INFINITY : s[e];
    }
  };
  // exp2(s c - m) -> bf16 pairs (k-slot order of the B operand) and their row sum.
  auto probs = [&](const f32x16& s, u32x4* p, float& lsum) {
    float l0 = 0.f, l1 = 0.f;
#pragma unroll
    for (int e = 0; e < 16; e += 4) {
      const float p0 = __builtin_amdgcn_exp2f(__builtin_fmaf(s[e], c_log2, -m_run));
      const float p1 = __builtin_amdgcn_exp2f(__builtin_fmaf(s[e + 1], c_log2, -m_run));
      const float p2 = __builtin_amdgcn_exp2f(__builtin_fmaf(s[e + 2], c_log2, -m_run));
      const float p3 = __builtin_amdgcn_exp2f(__builtin_fmaf(s[e + 3], c_log2, -m_run));
      const uint32_t pk0 = pack_bf16x2(p0, p1), pk1 = pack_bf16x2(p2, p3);
      p[e >> 3][(e >> 1) & 3] = pk0;
      p[e >> 3][((e >> 1) & 3) + 1] = pk1;
      l0 = sum_bf16x2(pk0, l0);
      l1 = sum_bf16x2(pk1, l1);
    }
    lsum = l0 + l1;
  };
  // Settles the probabilities P of the previous sub-block (scores s, row sum lsum) before
  // they enter O.  They were computed against the running reference m; only when one of
  // them exceeds 2^64 (seen in the row sum, an overflow to inf included) is the column's
  // reference raised to that sub-block's exact max: O and l, which hold only earlier
  // sub-blocks, are rescaled and P is recomputed (rare branch).  Then the sum joins l.  The
  // reference of a column is shared by its lane pair, and so is the decision.
  auto settle = [&](const f32x16& s, u32x4* p, float& lsum) {
    if (__builtin_amdgcn_ballot_w64(lsum > kOverflow) != 0) {
      __asm__ volatile("" ::);
      const bool over = max_with_partner(lsum) > kOverflow;
      const float t = block_max(s) * c_log2;
      const float m_new = over ? t : m_run;
      const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
#pragma unroll
      for (int db = 0; db < 4; ++db) o[db] *= alpha;
      l_run *= alpha;
      m_run = m_new;
      probs(s, p, lsum);
    }
    l_run += lsum;
  };

  f32x16 sp, sc;                 // scores of the previous and the current sub-block
  u32x4 pa[2], pb[2];
  float lsum_p = 0.f;            // row sum of the probabilities not yet settled
  int32_t pg_klast = 0;          // page of the last K tile whose copy was issued
  int32_t pg_knext = 0;          // page of the next K tile (loaded one iteration ahead)
  F8Stage kst, vst;

  // Moves the page window on when tile u leaves it (uniform, once per 64 tiles) and fetches
  // the window after it into the other slot.  The new window's copy was issued 64 tiles
  // earlier, before every copy the waits at the top of the last iterations covered, so it
  // is in LDS.
  auto advance_window = [&](int u) {
    if (u - win0 == 64) {
      pg_win = s_pages[wave][win_slot][lane];
      win0 += 64;
      win_slot ^= 1;
      if (ntiles > win0 + 64 - kS - 2) fetch_window(win0 + 64, win_slot);
    }
  };

  // Iteration t: copies V(t + kS - 1) and K(t + kS); sub-blocks 2t+1 and 2t+2 take the
  // softmax, their successors S from K(t + 1), their predecessors O += P V from V(t).
  // The ring stage of tile t is t % kS (a compile-time constant in each unrolled copy).
  auto iteration = [&](int t, auto stage) {
    constexpr int kJ = decltype(stage)::value;
    const int kcur = kKBase + ((kJ + 1) % kS) * kTileBytes;   // K(t + 1)
    const int vcur = kVBase + kJ * kTileBytes;                // V(t)
    if constexpr (!kFp8) {
      // K(t + 1) and V(t) are this wave's copies issued before the last 2 kS - 4 groups of
      // kDma; after the barrier every wave's share of them is in LDS, and every wave has
      // finished iteration t - 1, whose stages the copies below overwrite.
      wait_vmcnt<(2 * kS - 4) * kDma>();
      __builtin_amdgcn_s_barrier();
      advance_window(t + kS + 1);
    } else {
      wait_lgkmcnt0();
      __builtin_amdgcn_s_barrier();   // the stores of iteration t - 1 are visible
      f8_load(vst, vpb, pg_klast, lo + (t + 1) * kKvTile, vvo);
      f8_load(kst, kpb, pg_knext, lo + (t + 2) * kKvTile, kvo);
      pg_klast = pg_knext;
      advance_window(t + 3);
      pg_knext = page_of(t + 3);
    }

    // The copies into the stages just freed are issued from inside the first step (after its
    // second slot), where the MFMAs already in flight hide their scalar address work.
    auto copies = [&]() {
      if constexpr (!kFp8) {
        dma_rows(false, pg_klast, lo + (t + kS - 1) * kKvTile, kVBase + ((kJ + kS - 1) % kS) * kTileBytes);
        dma_rows(true, pg_knext, lo + (t + kS) * kKvTile, kKBase + kJ * kTileBytes);
        pg_klast = pg_knext;
        pg_knext = page_of(t + kS + 1);
      }
    };
    auto no_hook = []() {};
    const int sb1 = lo + (2 * t + 1) * 32;
    constexpr std::true_type kWithQK{}, kWithNext{};
    constexpr std::false_type kNoNext{};
    Pre f2;   // first operands of the second step, read during the first step's last slots
    // sub-block 2t+1 (scores sc; P(2t) in pa, from scores sp)
    {
      const Pre f = prefetch(kcur, vcur, kWithQK);
      settle(sp, pa, lsum_p);
      mask(sc, sb1);
      float ls;
      const f32x16 sn =
          step_main(sc, pa, pb, kcur, vcur, f, kWithQK, ls, kWithNext, kcur + kSubBytes, vcur + kSubBytes, f2, copies);
      sp = sc;
      sc = sn;
      lsum_p = ls;
    }
    // sub-block 2t+2 (P(2t+1) in pb)
    {
      settle(sp, pb, lsum_p);
      mask(sc, sb1 + 32);
      float ls;
      const f32x16 sn =
          step_main(sc, pb, pa, kcur + kSubBytes, vcur + kSubBytes, f2, kWithQK, ls, kNoNext, 0, 0, f2, no_hook);
      sp = sc;
      sc = sn;
      lsum_p = ls;
    }
    if constexpr (kFp8) {
      // K(t + 2) into stage t % 2 (K(t) there was last read in iteration t - 1), V(t + 1)
      // into stage (t + 1) % 2 (V(t - 1) there likewise)
      f8_store(kst, kKBase + kJ * kTileBytes, true);
      f8_store(vst, kVBase + ((kJ + 1) % 2) * kTileBytes, false);
    }
  };

  // Fused append: the first key-range piece of each (kv head, query tile) writes the tile's
  // chunk rows of kv head g into their pages (slots P + i, i in [i0, i1)); nothing in this
  // launch reads those slots from the pages.  Its loads and stores overlap the Q loads and
  // are covered by the wait below.
  if (kFused && it.s == 0) {
    constexpr int kThreads = kWaves * 64;
    const int units = (i1 - i0) * 2 * 16;   // (token, K or V, 16-byte chunk)
    for (int u = threadIdx.x; u < units; u += kThreads) {
      const int c = u & 15, kv = (u >> 4) & 1, i = i0 + (u >> 5);
      const int pos = P + i;
      const int64_t page = bt[pos >> 4];
      const uint16_t* src = (kv ? vnew : knew) + ((int64_t)(row0 + i) * hkv + g) * kHeadDim + 8 * c;
      char* dst = static_cast<char*>(kv ? vpool : kpool) +
                  ((page * hkv + g) * 16 + (pos & 15)) * kRowBytes + 16 * c;
      *reinterpret_cast<u32x4*>(dst) = *reinterpret_cast<const u32x4*>(src);
    }
  }

  // Page ids of the first tiles are requested while the Q loads are in flight; the Q loads
  // are then waited for on every path, before any LDS-direct copy is issued: the compiler's
  // wait-count bookkeeping does not see those copies, and a Q load it still counted as
  // pending would make it wait for every copy in each step of the loop.
  wait_vmcnt<0>();
  int32_t pg[kS + 1];
#pragma unroll
  for (int j = 0; j <= kS; ++j) pg[j] = page_of(j);
  if (ntiles > 64 - kS - 2) fetch_window(64, 0);

  if (ntiles > 0) {
    // Prologue: copies K(0), V(0), K(1), V(1), ..., K(kS - 2), V(kS - 2), K(kS - 1); waits
    // for K(0); sub-block 0 sets the reference to its own max (a lane with no visible key
    // there has none in the group's range, as its visible keys form a prefix of it).
    if constexpr (!kFp8) {
#pragma unroll
      for (int j = 0; j < kS - 1; ++j) {
        dma_rows(true, pg[j], lo + j * kKvTile, kKBase + j * kTileBytes);
        dma_rows(false, pg[j], lo + j * kKvTile, kVBase + j * kTileBytes);
      }
      dma_rows(true, pg[kS - 1], lo + (kS - 1) * kKvTile, kKBase + (kS - 1) * kTileBytes);
      pg_klast = pg[kS - 1];
      pg_knext = pg[kS];
      wait_vmcnt<(2 * kS - 2) * kDma>();   // K(0), the first of these copies
    } else {
      const int32_t pg0 = pg[0], pg1 = pg[1];
      f8_load(kst, kpb, pg0, lo, kvo);
      f8_load(vst, vpb, pg0, lo, vvo);
      f8_store(kst, kKBase, true);
      f8_store(vst, kVBase, false);
      f8_load(kst, kpb, pg1, lo + kKvTile, kvo);
      f8_store(kst, kKBase + kTileBytes, true);
      pg_klast = pg1;
      pg_knext = pg[2];
      wait_lgkmcnt0();
    }
    __builtin_amdgcn_s_barrier();

    sp = qk(kKBase);
    mask(sp, lo);
    {
      const float t = block_max(sp) * c_log2;
      m_run = t == -INFINITY ? 0.f : t;
    }
    probs(sp, pa, lsum_p);
    sc = qk(kKBase + kSubBytes);
  }

  int t = 0;
  if constexpr (kS == 4) {
    for (; t + 4 < ntiles; t += 4) {
      iteration(t, std::integral_constant<int, 0>{});
      iteration(t + 1, std::integral_constant<int, 1>{});
      iteration(t + 2, std::integral_constant<int, 2>{});
      iteration(t + 3, std::integral_constant<int, 3>{});
    }
    if (t + 1 < ntiles) {
      iteration(t, std::integral_constant<int, 0>{});
      ++t;
      if (t + 1 < ntiles) {
        iteration(t, std::integral_constant<int, 1>{});
        ++t;
        if (t + 1 < ntiles) {
          iteration(t, std::integral_constant<int, 2>{});
          ++t;
        }
      }
    }
  } else {
    for (; t + 2 < ntiles; t += 2) {
      iteration(t, std::integral_constant<int, 0>{});
      iteration(t + 1, std::integral_constant<int, 1>{});
    }
    if (t + 1 < ntiles) {
      iteration(t, std::integral_constant<int, 0>{});
      ++t;
    }
  }
  if (ntiles > 0) {
    // last tile (t = ntiles - 1): sub-block 2t+1 takes the softmax, P(2t) V, then P(2t+1) V
    if constexpr (!kFp8) wait_vmcnt<0>();
    else wait_lgkmcnt0();
    __builtin_amdgcn_s_barrier();
    const int vlast = kVBase + (t % kS) * kTileBytes;
    constexpr std::false_type kNoQK{};
    Pre f = prefetch(0, vlast, kNoQK);
    settle(sp, pa, lsum_p);
    mask(sc, lo + (2 * t + 1) * 32);
    float ls;
    step_main(sc, pa, pb, 0, vlast, f, kNoQK, ls, std::false_type{}, 0, 0, f, [] {});
    settle(sc, pb, ls);
    pv_acc(pb, vlast + kSubBytes);
  }

  float l_fin = sum_with_partner(l_run);
  float m_fin = l_fin > 0.f ? m_run : -INFINITY;     // -inf: no visible key in this range
  if constexpr (kHalves == 2) {
    // The second group's (O, m, l) to the first through LDS (the rings are free once every
    // wave is past its last tile): column wave cw of both groups holds the same elements in
    // the same lanes; element group k = 4 db + j of lane l is at ((k kColWaves + cw) 64 + l)
    // x 16 bytes, so each store or load of 64 lanes covers 1 KiB without bank conflicts.
    __builtin_amdgcn_s_barrier();
    float* xo = reinterpret_cast<float*>(smem);
    float* xml = xo + 16 * kColWaves * 64 * 4;
    if (grp == 1) {
#pragma unroll
      for (int db = 0; db < 4; ++db)
#pragma unroll
        for (int j = 0; j < 4; ++j)
          *reinterpret_cast<f32x4*>(xo + (((4 * db + j) * kColWaves + cw) * 64 + lane) * 4) =
              f32x4{o[db][4 * j], o[db][4 * j + 1], o[db][4 * j + 2], o[db][4 * j + 3]};
      *reinterpret_cast<f32x2*>(xml + (cw * 64 + lane) * 2) = f32x2{m_fin, l_fin};
    }
    wait_lgkmcnt0();
    __builtin_amdgcn_s_barrier();
    if (grp == 1) return;
    const f32x2 ml1 = *reinterpret_cast<const f32x2*>(xml + (cw * 64 + lane) * 2);
    const float mstar = fmaxf(m_fin, ml1[0]);
    const float a0 = merge_weight(m_fin, mstar), a1 = merge_weight(ml1[0], mstar);
#pragma unroll
    for (int db = 0; db < 4; ++db)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const f32x4 x = *reinterpret_cast<const f32x4*>(xo + (((4 * db + j) * kColWaves + cw) * 64 + lane) * 4);
#pragma unroll
        for (int e = 0; e < 4; ++e) o[db][4 * j + e] = a0 * o[db][4 * j + e] + a1 * x[e];
      }
    l_fin = a0 * l_fin + a1 * ml1[1];
    m_fin = mstar;
  }
  // Split piece, when the ring can hold the whole tile's rows (bf16 pages; one key group):
  // the fp32 partial is staged through LDS, row-major with each row's 16-byte chunks
  // permuted by (column mod 16) so that both the register-order writes and the row reads
  // are free of bank conflicts, and then stored a row run at a time (the G head rows of a
  // token are adjacent) with device-scope (sc1) stores, which write through the L2: no
  // dirty partial lines are left for the write-back at the end of the launch.  The row sum
  // and max follow with the same policy.
  float* const acc = pv.partials + it.part_off;
  const int64_t acc_bytes = (int64_t)ns * C * hq * (kHeadDim + 4) * 4;
  if (kHalves == 1 && RingT::kBytes >= kColWaves * 32 * kHeadDim * 4 && ns > 1 && acc_bytes <= 0x7fffffff) {
    constexpr int kSc1 = 16;   // cache policy: device scope
    __builtin_amdgcn_s_barrier();   // every wave is past its last read of the ring
    float* xs = reinterpret_cast<float*>(smem);
#pragma unroll
    for (int db = 0; db < 4; ++db)
#pragma unroll
      for (int j = 0; j < 4; ++j)
        *reinterpret_cast<f32x4*>(xs + (col * 32 + ((8 * db + 2 * j + half) ^ (col & 15))) * 4) =
            f32x4{o[db][4 * j] * v_mul, o[db][4 * j + 1] * v_mul, o[db][4 * j + 2] * v_mul,
                  o[db][4 * j + 3] * v_mul};
    wait_lgkmcnt0();
    __builtin_amdgcn_s_barrier();
    const auto prs = make_rsrc(acc, (int32_t)acc_bytes);
    const int ncols = min(tq * G, (i1 - i0) * G);   // the valid columns of this tile
    // row of column c: (s C + i0 + c / G) hq + g G + c % G = rbase + c + (c / G)(hq - G);
    // c / G = (c ginv) >> 24 exactly for c < 256 and G < 2^16
    const int64_t rbase = ((int64_t)it.s * C + i0) * hq + g * G;
    const uint32_t ginv = ((1u << 24) + (uint32_t)G - 1) / (uint32_t)G;
    constexpr int kThreads = kColWaves * 64;
#pragma unroll
    for (int u0 = 0; u0 < 32 * kColWaves * 32; u0 += kThreads) {
      const int u = u0 + (int)threadIdx.x;
      const int c = u >> 5, k = u & 31;   // column, 16-byte chunk
      if (c < ncols) {
        const f32x4 x = *reinterpret_cast<const f32x4*>(xs + (c * 32 + (k ^ (c & 15))) * 4);
        const int64_t pr = rbase + c + (int64_t)(((uint32_t)c * ginv) >> 24) * (hq - G);
        __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, x), prs, (uint32_t)(pr * 512 + 16 * k), 0,
                                               kSc1);
      }
    }
    if (valid && half == 0) {
      const int64_t prow = ((int64_t)it.s * C + tok) * hq + hq_col;
      const int64_t ml_off = (int64_t)ns * C * hq * kHeadDim * 4 + 16 * prow;
      __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, f32x4{m_fin, l_fin, 0.f, 0.f}), prs,
                                             (uint32_t)ml_off, 0, kSc1);
    }
    return;
  }
  if (!valid) return;
  if (ns == 1) {
    const float inv = v_mul / l_fin;
    uint16_t* orow = out + ((int64_t)(row0 + tok) * hq + hq_col) * 128 + 4 * half;
#pragma unroll
    for (int db = 0; db < 4; ++db)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const u32x2 w = {pack_bf16x2(o[db][4 * j] * inv, o[db][4 * j + 1] * inv),
                         pack_bf16x2(o[db][4 * j + 2] * inv, o[db][4 * j + 3] * inv)};
        *reinterpret_cast<u32x2*>(orow + 32 * db + 8 * j) = w;
      }
    if (lse != nullptr && half == 0) lse[(int64_t)(row0 + tok) * hq + hq_col] = (m_fin + __log2f(l_fin)) * kLn2;
    return;
  }
  // Split piece (other layouts): fp32 partial (acc row, then (m, l, 0, 0)), stored from the
  // registers; a column with no visible key in this piece has (-inf, 0): the merge skips it.
  float* ml = acc + (int64_t)ns * C * hq * kHeadDim;
  const int64_t prow = ((int64_t)it.s * C + tok) * hq + hq_col;
  float* arow = acc + prow * kHeadDim + 4 * half;
#pragma unroll
  for (int db = 0; db < 4; ++db)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const f32x4 w = {o[db][4 * j] * v_mul, o[db][4 * j + 1] * v_mul, o[db][4 * j + 2] * v_mul,
                       o[db][4 * j + 3] * v_mul};
      *reinterpret_cast<f32x4*>(arow + 32 * db + 8 * j) = w;
    }
  if (half == 0) *reinterpret_cast<f32x4*>(ml + 4 * prow) = f32x4{m_fin, l_fin, 0.f, 0.f};
}

// Largest r with a[r] <= x, for a non-decreasing a[0..n] with a[0] <= x < a[n].
__device__ inline int upper_index(const int32_t* a, int n, int x) {
  int lo = 0, hi = n;  // invariant: a[lo] <= x < a[hi]
  while (hi - lo > 1) {
    int mid = (lo + hi) >> 1;
    if (a[mid] <= x) lo = mid; else hi = mid;
  }
  return lo;
}

// Merge of split partials: workgroup (row, y) merges heads 8y .. 8y+7 of one chunk row;
// each thread owns 4 dims of one head.  Up to kFastPieces pieces are read in one round trip.
constexpr int kFastPieces = 4;
__global__ __launch_bounds__(256) void split_reduce_kernel(uint16_t* __restrict__ out, float* __restrict__ lse,
                                                           PlanPtrs pv, int32_t num_reqs, int32_t hq) {
  const int row = blockIdx.x;
  if (num_reqs == 0 || pv.hdr->status != 0 || row >= pv.cu[num_reqs]) return;
  const int r = upper_index(pv.cu, num_reqs, row);
  const int ns = pv.ns[r];
  if (ns <= 1) return;
  const int C = pv.c[r];
  const int tok = row - pv.cu[r];
  const float* acc = pv.partials + pv.part_off[r];
  const float* ml = acc + (int64_t)ns * C * hq * kHeadDim;
  const int u = blockIdx.y * 256 + threadIdx.x;
  if (u < hq * 32) {
    const int h = u >> 5, d4 = (u & 31) * 4;
    const int64_t piece = (int64_t)C * hq;                 // rows of one piece
    const int64_t prow0 = (int64_t)tok * hq + h;
    float mstar = -INFINITY, lb = 0.f;
    f32x4 a = {0.f, 0.f, 0.f, 0.f};
    if (ns <= kFastPieces) {
      // every piece's (m, l) and values loaded at once (one round trip)
      f32x4 mls[kFastPieces], xs[kFastPieces];
#pragma unroll
      for (int s = 0; s < kFastPieces; ++s)
        if (s < ns) {
          mls[s] = *reinterpret_cast<const f32x4*>(ml + 4 * (s * piece + prow0));
          xs[s] = *reinterpret_cast<const f32x4*>(acc + (s * piece + prow0) * kHeadDim + d4);
        }
#pragma unroll
      for (int s = 0; s < kFastPieces; ++s)
        if (s < ns) mstar = fmaxf(mstar, mls[s][0]);
#pragma unroll
      for (int s = 0; s < kFastPieces; ++s)
        if (s < ns && mls[s][0] != -INFINITY) {
          const float wgt = merge_weight(mls[s][0], mstar);
          lb += wgt * mls[s][1];
          a += wgt * xs[s];
        }
    } else {
      for (int s = 0; s < ns; ++s) mstar = fmaxf(mstar, ml[4 * (s * piece + prow0)]);
      for (int s = 0; s < ns; ++s) {
        const int64_t prow = s * piece + prow0;
        const f32x4 mlp = *reinterpret_cast<const f32x4*>(ml + 4 * prow);
        if (mlp[0] == -INFINITY) continue;
        const float wgt = merge_weight(mlp[0], mstar);
        lb += wgt * mlp[1];
        a += wgt * *reinterpret_cast<const f32x4*>(acc + prow * kHeadDim + d4);
      }
    }
    const float inv = 1.0f / lb;
    const u32x2 w = {pack_bf16x2(a[0] * inv, a[1] * inv), pack_bf16x2(a[2] * inv, a[3] * inv)};
    *reinterpret_cast<u32x2*>(out + ((int64_t)row * hq + h) * kHeadDim + d4) = w;
    if (lse != nullptr && d4 == 0) lse[(int64_t)row * hq + h] = (mstar + __log2f(lb)) * kLn2;
  }
}

}  // namespace

template <bool kFp8, int kColWaves, int kHalves, bool kFused, bool kQ8 = false>
void launch_main_variant(const AttnLaunch& a, hipStream_t stream) {
  attn_main_kernel<kFp8, kColWaves, kHalves, kFused, kQ8><<<(unsigned)a.dims.num_items, kColWaves * kHalves * 64, 0, stream>>>(
      static_cast<const uint16_t*>(a.q), static_cast<uint16_t*>(a.out), a.lse, a.kv.kpool, a.kv.vpool,
      a.kv.kscale, a.kv.vscale, a.kv.block_tables, a.kv.max_pages, a.hq, a.kv.hkv, a.softmax_scale * kLog2e,
      plan_ptrs(a.workspace, a.dims), a.group_by_xcd ? 1 : 0, static_cast<const uint16_t*>(a.knew),
      static_cast<const uint16_t*>(a.vnew), a.total_rows);
}

template <bool kFp8>
void launch_main_dtype(const AttnLaunch& a, hipStream_t stream) {
  constexpr bool kF = false;
  if (!kFp8 && a.knew != nullptr) {
    // append fused into this launch (bf16 pages only)
    if (a.tile_cols == kMaxTileCols) launch_main_variant<false, 8, 1, true>(a, stream);
    else if (a.key_halves == 2) launch_main_variant<false, 4, 2, true>(a, stream);
    else launch_main_variant<false, 4, 1, true>(a, stream);
    return;
  }
  if (kFp8 && a.q8) {
    // Q quantised to e4m3 and S = Q K^T on the fp8 MFMA (e4m3 pages only)
    if (a.tile_cols == kMaxTileCols) launch_main_variant<true, 8, 1, false, true>(a, stream);
    else if (a.key_halves == 2) launch_main_variant<true, 4, 2, false, true>(a, stream);
    else launch_main_variant<true, 4, 1, false, true>(a, stream);
    return;
  }
  if (a.tile_cols == kMaxTileCols) launch_main_variant<kFp8, 8, 1, kF>(a, stream);
  else if (a.key_halves == 2) launch_main_variant<kFp8, 4, 2, kF>(a, stream);
  else launch_main_variant<kFp8, 4, 1, kF>(a, stream);
}

hipError_t launch_attn_main(const AttnLaunch& a, hipStream_t stream) {
  if (a.dims.num_items <= 0) return hipSuccess;
  if (a.tile_cols == kDecodeTileCols) return launch_attn_decode(a, stream);
  if (a.kv.fp8) launch_main_dtype<true>(a, stream);
  else launch_main_dtype<false>(a, stream);
  return hipGetLastError();
}

hipError_t launch_split_reduce(const ReduceLaunch& a, hipStream_t stream) {
  if (a.total_tokens <= 0) return hipSuccess;
  dim3 grid((unsigned)a.total_tokens, (unsigned)((a.hq * 32 + 255) / 256));
  split_reduce_kernel<<<grid, 256, 0, stream>>>(static_cast<uint16_t*>(a.out), a.lse,
                                                plan_ptrs(const_cast<void*>(a.workspace), a.dims), a.num_reqs, a.hq);
  return hipGetLastError();
}

}  // namespace s2l
