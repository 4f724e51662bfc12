// Chunk-prefill attention over a paged KV cache, and the split-KV merge, for gfx950.
//
// What is computed (Stream2LLM Sec. 2.1 prefill over the pages of Sec. 2.2, resumed at
// num_computed_tokens as in Sec. 4.2): query i of a request's new chunk (absolute position
// t = P + i) attends to keys 0..t of that request, read through its block table.
//
// One workgroup = 4 waves = one work item of the plan: kv head g, 128 packed query
// columns (tq tokens x G heads, token-major) and a key range [lo, hi).  Per 64-key tile:
//   * K and V (64 keys x 128) are staged in LDS, double buffered; pages are read through
//     the block table with raw buffer loads, keys at or past `hi` are zero-filled;
//   * each wave computes S^T = K Q^T for its 32 columns with v_mfma_f32_32x32x16_bf16
//     (A = K rows from LDS, B = Q held in registers), so every lane owns one query column
//     and 32 of the tile's scores;
//   * online softmax in the exp2 domain, row max shared with lane ^ 32 by
//     v_permlane32_swap; the running maximum is only raised (and O rescaled) when the new
//     maximum exceeds it by more than 2^8, else probabilities up to 2^8 are accumulated
//     against the stale maximum (exact after the final division);
//   * O^T += V^T P^T with the same MFMA: A = V^T read from the key-major V tile with the
//     gfx950 transposing LDS read (ds_read_b64_tr_b16), B = P (bf16) straight from the
//     score registers, the A operand's k-slots ordered as the keys each lane half holds;
//   * the causal mask is evaluated only on tiles that reach past the first query token's
//     position (the chunk-diagonal tiles).
// Unsplit items write bf16 O = acc / l (and LSE); split items write fp32 partials
// (acc, m, l) that split_reduce merges.
#include "launch.h"
#include "plan_rules.h"
#include "s2l_device.h"

namespace s2l {

namespace {

constexpr int kWaves = 4;
constexpr int kThreads = kWaves * 64;
#ifndef S2L_VROW_PAD
#define S2L_VROW_PAD 32   // 320-byte rows: the transposing reads hit distinct banks
#endif
constexpr int kKRow = 128 + 8;                     // bf16 per K row in LDS (272 B: bank-shifted rows)
constexpr int kVRow = 128 + S2L_VROW_PAD;          // bf16 per V row in LDS
constexpr int kKTile = kKvTile * kKRow;            // elements
constexpr int kVTile = kKvTile * kVRow;
constexpr int kBufElems = kKTile + kVTile;         // one stage buffer (35840 B)
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;
constexpr float kRescaleSlack = 8.0f;              // log2 units

// Largest r with a[r] <= x, for a non-decreasing a[0..n] with a[0] <= x < a[n].
__device__ inline int upper_index(const int32_t* a, int n, int x) {
  int lo = 0, hi = n;  // invariant: a[lo] <= x < a[hi]
  while (hi - lo > 1) {
    int mid = (lo + hi) >> 1;
    if (a[mid] <= x) lo = mid; else hi = mid;
  }
  return lo;
}

// Registers holding one tile's global loads until they are written to LDS.
struct Stage {
  u32x4 k[4];
  u32x4 v[4];
};

// Raw buffer loads: a resource descriptor (base, size in bytes) in SGPRs plus a per-lane
// byte offset.  Offsets at or past the size read as zero.
constexpr int32_t kRsrcWord3 = 0x00020000;   // gfx9-family raw buffer: 32-bit dword format
__device__ inline __amdgpu_buffer_rsrc_t make_rsrc(const void* base, int32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, bytes, kRsrcWord3);
}

// Page ids of the four 16-key pages of the tile at key kb (lane l loads entry l & 3).
// Entries past the item's last page read as 0, a valid page: the keys they would hold are
// at or past `hi` and are zeroed before use.
__device__ inline int32_t tile_page_entry(const int32_t* bt, int kb, int last_page, uint32_t lane_off) {
  const int first = kb >> 4;
  const int n = last_page + 1 - first;
  return (int32_t)__builtin_amdgcn_raw_buffer_load_b32(make_rsrc(bt + first, 4 * (n > 0 ? n : 0)), lane_off, 0, 0);
}
struct Pages {
  int32_t p[4];
};
__device__ inline Pages broadcast_pages(int32_t v) {
  Pages pg;
  pg.p[0] = __builtin_amdgcn_readlane(v, 0);
  pg.p[1] = __builtin_amdgcn_readlane(v, 1);
  pg.p[2] = __builtin_amdgcn_readlane(v, 2);
  pg.p[3] = __builtin_amdgcn_readlane(v, 3);
  return pg;
}
__device__ inline int32_t pick(const Pages& pg, int j) {  // j wave-uniform
  return j == 0 ? pg.p[0] : (j == 1 ? pg.p[1] : (j == 2 ? pg.p[2] : pg.p[3]));
}

// Global loads of one tile.  bf16 cache: thread t loads K rows (t>>4) + 16j (page j, slot
// t>>4), 16-byte chunk t&15, and V rows 4(t>>4) + i (page t>>6, slot 4((t>>4)&3) + i) of the
// same chunk.  fp8 cache: K rows (t>>3) + 32j (page 2j + (t>>7)), 16-byte chunk t&7; V rows
// as for bf16 with 8-byte chunks t&15, kept raw in .xy.  The loads are unconditional (pages
// are clamped to valid ones); keys at or past `hi` are zeroed in store_tile, once the data
// has arrived, so no instruction waits on a load before the tile's compute is done.
// Per-thread byte offsets of the tile loads inside a (page, kv head) run; loop invariant,
// so the address of every load is a uniform base (pool + page stride, in SGPRs) plus one of
// these (VGPRs never overwritten while a load is in flight).
struct LoadOffsets {
  uint32_t k;      // K row / chunk offset
  uint32_t v[4];   // V rows 4((t>>4)&3) + i
};
template <bool kFp8>
__device__ inline LoadOffsets load_offsets() {
  const int t = threadIdx.x;
  LoadOffsets o;
  if constexpr (!kFp8) {
    o.k = (uint32_t)(((t >> 4) * 128 + (t & 15) * 8) * 2);
#pragma unroll
    for (int i = 0; i < 4; ++i) o.v[i] = (uint32_t)(((4 * ((t >> 4) & 3) + i) * 128 + (t & 15) * 8) * 2);
  } else {
    o.k = (uint32_t)(((t >> 3) & 15) * 128 + (t & 7) * 16);
#pragma unroll
    for (int i = 0; i < 4; ++i) o.v[i] = (uint32_t)((4 * ((t >> 4) & 3) + i) * 128 + (t & 15) * 8);
  }
  return o;
}

template <bool kFp8>
__device__ inline void load_tile(Stage& st, const char* kpool, const char* vpool, const Pages& pg,
                                 int64_t head, int hkv, const LoadOffsets& lo) {
  constexpr int32_t kRun = kFp8 ? 16 * 128 : 16 * 128 * 2;   // bytes of one (page, kv head)
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const auto vr = make_rsrc(vpool + ((int64_t)pick(pg, wave) * hkv + head) * kRun, kRun);
  if constexpr (!kFp8) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const auto kr = make_rsrc(kpool + ((int64_t)pg.p[j] * hkv + head) * kRun, kRun);
      st.k[j] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(kr, lo.k, 0, 0));
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) st.v[i] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(vr, lo.v[i], 0, 0));
  } else {
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const auto kr = make_rsrc(kpool + ((int64_t)pick(pg, 2 * j + (wave >> 1)) * hkv + head) * kRun, kRun);
      st.k[j] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(kr, lo.k, 0, 0));
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const u32x2 w = __builtin_bit_cast(u32x2, __builtin_amdgcn_raw_buffer_load_b64(vr, lo.v[i], 0, 0));
      st.v[i] = u32x4{w[0], w[1], 0, 0};
    }
  }
}

// Zero the staged keys at or past `hi` (only the last tile of an item can have any).
template <bool kFp8>
__device__ inline void mask_tile(Stage& st, int kb0, int hi) {
  const int t = threadIdx.x;
  if constexpr (!kFp8) {
#pragma unroll
    for (int j = 0; j < 4; ++j)
      if (kb0 + (t >> 4) + 16 * j >= hi) st.k[j] = u32x4{0, 0, 0, 0};
  } else {
#pragma unroll
    for (int j = 0; j < 2; ++j)
      if (kb0 + (t >> 3) + 32 * j >= hi) st.k[j] = u32x4{0, 0, 0, 0};
  }
#pragma unroll
  for (int i = 0; i < 4; ++i)
    if (kb0 + 4 * (t >> 4) + i >= hi) st.v[i] = u32x4{0, 0, 0, 0};
}

// K and V tiles are stored in LDS as they are in the pages, one key per row (row strides
// kKRow / kVRow elements).  Thread t writes its staged rows: bf16 K rows (t>>4) + 16j and V
// rows 4(t>>4) + i, 16-byte chunk t&15; fp8 data is converted to bf16 on the way (exact).
template <bool kFp8>
__device__ inline void store_tile(const Stage& st, uint16_t* buf) {
  const int t = threadIdx.x;
  uint16_t* kl = buf;
  uint16_t* vl = buf + kKTile;
  if constexpr (!kFp8) {
    const int c = t & 15;
#pragma unroll
    for (int j = 0; j < 4; ++j)
      *reinterpret_cast<u32x4*>(kl + ((t >> 4) + 16 * j) * kKRow + c * 8) = st.k[j];
#pragma unroll
    for (int i = 0; i < 4; ++i)
      *reinterpret_cast<u32x4*>(vl + (4 * (t >> 4) + i) * kVRow + c * 8) = st.v[i];
  } else {
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const u32x2 a = fp8x4_to_bf16x4(st.k[j][0]);
      const u32x2 b = fp8x4_to_bf16x4(st.k[j][1]);
      const u32x2 c = fp8x4_to_bf16x4(st.k[j][2]);
      const u32x2 d = fp8x4_to_bf16x4(st.k[j][3]);
      uint16_t* row = kl + ((t >> 3) + 32 * j) * kKRow + (t & 7) * 16;
      *reinterpret_cast<u32x4*>(row) = u32x4{a[0], a[1], b[0], b[1]};
      *reinterpret_cast<u32x4*>(row + 8) = u32x4{c[0], c[1], d[0], d[1]};
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const u32x2 a = fp8x4_to_bf16x4(st.v[i][0]);
      const u32x2 b = fp8x4_to_bf16x4(st.v[i][1]);
      *reinterpret_cast<u32x4*>(vl + (4 * (t >> 4) + i) * kVRow + (t & 15) * 8) = u32x4{a[0], a[1], b[0], b[1]};
    }
  }
}

// A operand of O^T += V^T P^T for k-step ks (keys 16ks..16ks+15 of the tile) and d-block db,
// read transposed from the key-major V tile with two ds_read_b64_tr_b16.  Within each group
// of 16 lanes, lane j addresses key row (j>>2) of a 4-key set at column base + 4(j&3); the
// hardware hands lane i the four keys of column base + i.  Lane (n, half) thereby receives
// V[keys 4 half + {0..3}, then 8 + 4 half + {0..3}][32 db + n]: the k-slot order of the
// score registers it multiplies.
typedef short v4i16 __attribute__((ext_vector_type(4)));
__device__ inline bf16x8 read_vt(const uint16_t* vl, int ks, int db) {
  const int l = threadIdx.x & 63;
  const int j = l & 15, half = l >> 5;
  const int col = 32 * db + 16 * ((l >> 4) & 1) + 4 * (j & 3);
  const int row0 = 16 * ks + 4 * half + (j >> 2);
  typedef __attribute__((address_space(3))) v4i16 lds_v4i16;
  const lds_v4i16* p0 = (const lds_v4i16*)(vl + row0 * kVRow + col);
  const lds_v4i16* p1 = (const lds_v4i16*)(vl + (row0 + 8) * kVRow + col);
  const v4i16 a = __builtin_amdgcn_ds_read_tr16_b64_v4i16(const_cast<lds_v4i16*>(p0));
  const v4i16 b = __builtin_amdgcn_ds_read_tr16_b64_v4i16(const_cast<lds_v4i16*>(p1));
  const u32x2 ua = __builtin_bit_cast(u32x2, a), ub = __builtin_bit_cast(u32x2, b);
  return __builtin_bit_cast(bf16x8, u32x4{ua[0], ua[1], ub[0], ub[1]});
}

// kQB blocks of 32 query columns per wave: the workgroup's tile is 4 * 32 * kQB columns.
template <bool kFp8, int kQB>
__global__ __launch_bounds__(kThreads, kQB == 1 ? 2 : 1) void attn_main_kernel(
    const uint16_t* __restrict__ q, uint16_t* __restrict__ out, float* __restrict__ lse,
    const void* __restrict__ kpool, const void* __restrict__ vpool, const float* __restrict__ kscale,
    const float* __restrict__ vscale, const int32_t* __restrict__ block_tables, int32_t max_pages,
    int32_t num_reqs, int32_t hq, int32_t hkv, float scale_log2, PlanPtrs pv) {
  __shared__ __attribute__((aligned(16))) uint16_t smem[2 * kBufElems];
  const int W = pv.hdr->num_items;
  if ((int)blockIdx.x >= W) return;
  const int w_item = xcd_logical(blockIdx.x, gridDim.x < (unsigned)W ? gridDim.x : W);
  const int r = upper_index(pv.item_off, num_reqs, w_item);
  const int nqt = pv.nqt[r], ns = pv.ns[r];
  const Item it = decode_local(w_item - pv.item_off[r], nqt, ns);
  const int P = pv.p[r], C = pv.c[r], row0 = pv.cu[r];
  const int G = hq / hkv;
  const int tq = tile_tokens(G, 128 * kQB);
  const int i0 = it.qt * tq;
  const int i1 = min(i0 + tq, C);
  int lo, hi;
  piece_range(P + i1, ns, it.s, &lo, &hi);
  const int g = it.g;
  const int32_t* bt = block_tables + (int64_t)r * max_pages;

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int n = lane & 31, half = lane >> 5;
  int tok[kQB], hq_col[kQB], horizon[kQB];
  bool valid[kQB];
#pragma unroll
  for (int qb = 0; qb < kQB; ++qb) {
    const int col = (wave * kQB + qb) * 32 + n;
    tok[qb] = i0 + col / G;
    hq_col[qb] = g * G + col % G;
    valid[qb] = col < tq * G && tok[qb] < i1;
    horizon[qb] = valid[qb] ? P + tok[qb] : P + i1 - 1;   // last visible key of this column
  }

  float c_log2 = scale_log2;
  float v_mul = 1.0f;
  if constexpr (kFp8) {
    c_log2 *= kscale[g];
    v_mul = vscale[g];
  }

  // Q^T operand: lane (n, half) holds Q[col][16 ks + 8 half .. +7] for ks = 0..7.
  bf16x8 qf[kQB][8];
#pragma unroll
  for (int qb = 0; qb < kQB; ++qb) {
    const uint16_t* qrow =
        q + ((int64_t)(row0 + (valid[qb] ? tok[qb] : 0)) * hq + (valid[qb] ? hq_col[qb] : 0)) * 128 + 8 * half;
#pragma unroll
    for (int ks = 0; ks < 8; ++ks) {
      u32x4 x = valid[qb] ? *reinterpret_cast<const u32x4*>(qrow + 16 * ks) : u32x4{0, 0, 0, 0};
      qf[qb][ks] = __builtin_bit_cast(bf16x8, x);
    }
  }

  f32x16 o[kQB][4];
  float m_run[kQB], l_run[kQB];
#pragma unroll
  for (int qb = 0; qb < kQB; ++qb) {
#pragma unroll
    for (int db = 0; db < 4; ++db) o[qb][db] = f32x16{};
    m_run[qb] = 0.f;
    l_run[qb] = 0.f;
  }

  const int ntiles = hi > lo ? ceil_div(hi - lo, kKvTile) : 0;
  bool first = true;   // wave-uniform: the next sub-block is the item's first
  const int last_page = hi > lo ? (hi - 1) >> 4 : 0;
  Stage st;
  int32_t page_next = 0;   // (vector) page-id entry of the tile after the one being loaded
  const LoadOffsets loff = load_offsets<kFp8>();
  const uint32_t page_lane_off = 4u * (threadIdx.x & 3);
  const char* kpb = static_cast<const char*>(kpool);
  const char* vpb = static_cast<const char*>(vpool);
  if (ntiles > 0) {
    const Pages pg0 = broadcast_pages(tile_page_entry(bt, lo, last_page, page_lane_off));
    load_tile<kFp8>(st, kpb, vpb, pg0, g, hkv, loff);
    if (ntiles > 1) page_next = tile_page_entry(bt, lo + kKvTile, last_page, page_lane_off);
    if (lo + kKvTile > hi) mask_tile<kFp8>(st, lo, hi);
    store_tile<kFp8>(st, smem);
  }
  // Nothing loaded before the loop may remain in flight at its head: otherwise the compiler's
  // wait-count bookkeeping, merging the entry and back edges, puts a full wait for vector
  // loads in front of every iteration's first MFMA, serialising the prefetch.
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();

  for (int ti = 0; ti < ntiles; ++ti) {
    const int kb0 = lo + ti * kKvTile;
    const uint16_t* kl = smem + (ti & 1) * kBufElems;
    const uint16_t* vl = kl + kKTile;
    const bool more = ti + 1 < ntiles;
    if (more) {
      const int kb1 = kb0 + kKvTile;
      const Pages pg = broadcast_pages(page_next);
      if (ti + 2 < ntiles) page_next = tile_page_entry(bt, kb1 + kKvTile, last_page, page_lane_off);
      load_tile<kFp8>(st, kpb, vpb, pg, g, hkv, loff);
    }

    // S^T = K Q^T for both 32-key sub-blocks (two independent MFMA chains); element e of
    // sc[kb][qb] is key kb0 + 32 kb + 8(e/4) + 4 half + e%4.  Softmax and P.V then run one
    // sub-block at a time.
    f32x16 sc[2][kQB];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int qb = 0; qb < kQB; ++qb) sc[kb][qb] = f32x16{};
#pragma unroll
    for (int ks = 0; ks < 8; ++ks) {
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
        const bf16x8 a = *reinterpret_cast<const bf16x8*>(kl + (32 * kb + n) * kKRow + 16 * ks + 8 * half);
#pragma unroll
        for (int qb = 0; qb < kQB; ++qb)
          sc[kb][qb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qf[qb][ks], sc[kb][qb], 0, 0, 0);
      }
    }
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
      f32x16* s = sc[kb];

      // Online softmax in the log2 domain against the running reference m_run: x = s c - m.
      // The reference is set on the item's first sub-block and afterwards only raised when a
      // score exceeds it by more than 2^8 (probabilities up to 2^8 are accumulated against a
      // stale reference; the final division makes the result exact).  A lane whose first
      // sub-block is fully masked sees no key in the whole piece (its keys only grow), so its
      // reference can stay unset.
      const int sb0 = kb0 + 32 * kb;
      float xmax[kQB];
      bool over = false;
#pragma unroll
      for (int qb = 0; qb < kQB; ++qb) {
#pragma unroll
        for (int e = 0; e < 16; ++e) s[qb][e] = __builtin_fmaf(s[qb][e], c_log2, -m_run[qb]);
      }
      if (sb0 + 31 > P + i0) {   // chunk-diagonal sub-block: causal mask
        __asm__ volatile("" ::);  // keep this a branch (not predicated into every sub-block)
#pragma unroll
        for (int qb = 0; qb < kQB; ++qb)
#pragma unroll
          for (int e = 0; e < 16; ++e) {
            const int key = sb0 + 8 * (e >> 2) + 4 * half + (e & 3);
            s[qb][e] = key > horizon[qb] ? -INFINITY : s[qb][e];
          }
      }
#pragma unroll
      for (int qb = 0; qb < kQB; ++qb) {
        float mx = vmax3(s[qb][0], s[qb][1], s[qb][2]);
#pragma unroll
        for (int e = 3; e < 15; e += 2) mx = vmax3(mx, s[qb][e], s[qb][e + 1]);
        mx = vmax2(mx, s[qb][15]);
        xmax[qb] = max_with_partner(mx);
        over |= xmax[qb] > kRescaleSlack;
      }
      if (first || __any(over)) {
        __asm__ volatile("" ::);
#pragma unroll
        for (int qb = 0; qb < kQB; ++qb) {
          // new reference: the block maximum (first block) or the larger of old and new
          const float cand = xmax[qb] + m_run[qb];
          const float m_new = xmax[qb] == -INFINITY ? m_run[qb] : (first ? cand : fmaxf(m_run[qb], cand));
          const float alpha = first ? 0.0f : __builtin_amdgcn_exp2f(m_run[qb] - m_new);
          const float shift = m_new - m_run[qb];
          m_run[qb] = m_new;
          l_run[qb] *= alpha;
#pragma unroll
          for (int db = 0; db < 4; ++db) o[qb][db] *= alpha;
#pragma unroll
          for (int e = 0; e < 16; ++e) s[qb][e] -= shift;
        }
        first = false;
      }
      uint32_t pk[kQB][8];
#pragma unroll
      for (int qb = 0; qb < kQB; ++qb) {
        float lsum = 0.f;
#pragma unroll
        for (int e = 0; e < 16; e += 2) {
          const float p0 = __builtin_amdgcn_exp2f(s[qb][e]);
          const float p1 = __builtin_amdgcn_exp2f(s[qb][e + 1]);
          lsum += p0 + p1;
          pk[qb][e >> 1] = pack_bf16x2(p0, p1);
        }
        l_run[qb] += lsum;
      }

      // O^T += V^T P^T over the sub-block's two k-steps of 16 keys.
#pragma unroll
      for (int k2 = 0; k2 < 2; ++k2) {
        const int ks = 2 * kb + k2;
        bf16x8 pb[kQB];
#pragma unroll
        for (int qb = 0; qb < kQB; ++qb)
          pb[qb] = __builtin_bit_cast(bf16x8, u32x4{pk[qb][4 * k2], pk[qb][4 * k2 + 1], pk[qb][4 * k2 + 2],
                                                    pk[qb][4 * k2 + 3]});
#pragma unroll
        for (int db = 0; db < 4; ++db) {
          const bf16x8 a = read_vt(vl, ks, db);
#pragma unroll
          for (int qb = 0; qb < kQB; ++qb)
            o[qb][db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, pb[qb], o[qb][db], 0, 0, 0);
        }
      }
    }
    if (more) {
      if (kb0 + 2 * kKvTile > hi) mask_tile<kFp8>(st, kb0 + kKvTile, hi);
      store_tile<kFp8>(st, smem + ((ti + 1) & 1) * kBufElems);
    }
    __syncthreads();
  }

#pragma unroll
  for (int qb = 0; qb < kQB; ++qb) {
    const float l_tot = sum_with_partner(l_run[qb]);
    if (!valid[qb]) continue;
    if (ns == 1) {
      const float inv = v_mul / l_tot;
      uint16_t* orow = out + ((int64_t)(row0 + tok[qb]) * hq + hq_col[qb]) * 128 + 4 * half;
#pragma unroll
      for (int db = 0; db < 4; ++db)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const u32x2 w = {pack_bf16x2(o[qb][db][4 * j] * inv, o[qb][db][4 * j + 1] * inv),
                           pack_bf16x2(o[qb][db][4 * j + 2] * inv, o[qb][db][4 * j + 3] * inv)};
          *reinterpret_cast<u32x2*>(orow + 32 * db + 8 * j) = w;
        }
      if (lse != nullptr && half == 0)
        lse[(int64_t)(row0 + tok[qb]) * hq + hq_col[qb]] = (m_run[qb] + __log2f(l_tot)) * kLn2;
    } else {
      float* acc = pv.partials + pv.part_off[r];
      float* ml = acc + (int64_t)ns * C * hq * kHeadDim;
      const int64_t prow = ((int64_t)it.s * C + tok[qb]) * hq + hq_col[qb];
      float* arow = acc + prow * kHeadDim + 4 * half;
#pragma unroll
      for (int db = 0; db < 4; ++db)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const f32x4 w = {o[qb][db][4 * j] * v_mul, o[qb][db][4 * j + 1] * v_mul, o[qb][db][4 * j + 2] * v_mul,
                           o[qb][db][4 * j + 3] * v_mul};
          *reinterpret_cast<f32x4*>(arow + 32 * db + 8 * j) = w;
        }
      // a column with no visible key in this piece: (m, l) = (-inf, 0), skipped by the merge
      if (half == 0) *reinterpret_cast<f32x2*>(ml + 2 * prow) = f32x2{l_tot > 0.f ? m_run[qb] : -INFINITY, l_tot};
    }
  }
}

// Merge of split partials: workgroup (row, y) merges heads 8y .. 8y+7 of one chunk row;
// each thread owns 4 dims of one head.
__global__ __launch_bounds__(256) void split_reduce_kernel(uint16_t* __restrict__ out, float* __restrict__ lse,
                                                           PlanPtrs pv, int32_t num_reqs, int32_t hq) {
  const int row = blockIdx.x;
  if (num_reqs == 0 || row >= pv.cu[num_reqs]) return;
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
    float mstar = -INFINITY;
    for (int s = 0; s < ns; ++s) mstar = fmaxf(mstar, ml[2 * (((int64_t)s * C + tok) * hq + h)]);
    float lstar = 0.f;
    f32x4 a = {0.f, 0.f, 0.f, 0.f};
    for (int s = 0; s < ns; ++s) {
      const int64_t prow = ((int64_t)s * C + tok) * hq + h;
      const float ms = ml[2 * prow];
      if (ms == -INFINITY) continue;
      const float wgt = __builtin_amdgcn_exp2f(ms - mstar);
      lstar += wgt * ml[2 * prow + 1];
      const f32x4 x = *reinterpret_cast<const f32x4*>(acc + prow * kHeadDim + d4);
      a += wgt * x;
    }
    const float inv = 1.0f / lstar;
    const u32x2 w = {pack_bf16x2(a[0] * inv, a[1] * inv), pack_bf16x2(a[2] * inv, a[3] * inv)};
    *reinterpret_cast<u32x2*>(out + ((int64_t)row * hq + h) * kHeadDim + d4) = w;
    if (lse != nullptr && d4 == 0) lse[(int64_t)row * hq + h] = (mstar + __log2f(lstar)) * kLn2;
  }
}

}  // namespace

template <bool kFp8, int kQB>
void launch_main_variant(const AttnLaunch& a, hipStream_t stream) {
  attn_main_kernel<kFp8, kQB><<<a.num_items, kThreads, 0, stream>>>(
      static_cast<const uint16_t*>(a.q), static_cast<uint16_t*>(a.out), a.lse, a.kv.kpool, a.kv.vpool,
      a.kv.kscale, a.kv.vscale, a.kv.block_tables, a.kv.max_pages, a.kv.num_reqs, a.hq, a.kv.hkv,
      a.softmax_scale * kLog2e, plan_ptrs(a.workspace, a.kv.num_reqs));
}

hipError_t launch_attn_main(const AttnLaunch& a, hipStream_t stream) {
  if (a.num_items <= 0) return hipSuccess;
  const bool wide = a.tile_cols == kMaxTileCols;
  if (a.kv.fp8) {
    if (wide) launch_main_variant<true, 2>(a, stream);
    else launch_main_variant<true, 1>(a, stream);
  } else {
    if (wide) launch_main_variant<false, 2>(a, stream);
    else launch_main_variant<false, 1>(a, stream);
  }
  return hipGetLastError();
}

hipError_t launch_split_reduce(const ReduceLaunch& a, hipStream_t stream) {
  if (a.total_tokens <= 0) return hipSuccess;
  dim3 grid((unsigned)a.total_tokens, (unsigned)((a.hq * 32 + 255) / 256));
  split_reduce_kernel<<<grid, 256, 0, stream>>>(
      static_cast<uint16_t*>(a.out), a.lse, plan_ptrs(const_cast<void*>(a.workspace), a.num_reqs), a.num_reqs,
      a.hq);
  return hipGetLastError();
}

}  // namespace s2l
