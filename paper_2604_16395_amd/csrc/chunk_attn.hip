// Chunk-prefill attention over a paged KV cache, and the split-KV merge, for gfx950.
//
// What is computed (Stream2LLM Sec. 2.1 prefill over the pages of Sec. 2.2, resumed at
// num_computed_tokens as in Sec. 4.2): query i of a request's new chunk (absolute position
// t = P + i) attends to keys 0..t of that request, read through its block table.
//
// One workgroup = kWaves waves (4 or 8) = one work item of the plan: kv head g, 32 kWaves
// packed query columns (tq tokens x G heads, token-major) and a key range [lo, hi).
//
// Data movement.  K and V tiles of 64 keys x 128 are staged in LDS, one key row of 256
// bytes each, 16-byte chunks permuted per row (K: chunk c of row r at c ^ (r & 15); V: at
// c ^ 4 (r & 3)) so that the MFMA operand reads below hit 64 distinct banks.  bf16 pages
// are copied straight from HBM into LDS (buffer_load ... lds), each wave moving one page of
// the tile; the buffer descriptor of a page ends at key `hi`, so keys past it arrive as
// zeros.  E4M3 pages go through registers and are widened to bf16 on the way (exact).  K
// is fetched one tile ahead of V; both are double buffered.
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
// The sub-blocks are software pipelined: while the softmax of sub-block b runs on the
// VALU, the MFMA unit computes S(b+1) and O += P(b-1) V(b-1); P(b-1) is checked for
// overflow at the start of step b, before it enters O.  The causal mask is applied only to
// sub-blocks that reach past the first query token's position.
//
// Unsplit items write bf16 O = acc / l (and LSE); split items write fp32 partials
// (acc, m, l) that split_reduce merges (log-sum-exp merge of Sec. 2.1's softmax).
#include "launch.h"
#include "plan_rules.h"
#include "s2l_device.h"

namespace s2l {

namespace {

constexpr int kRowBytes = kHeadDim * 2;              // one bf16 key row in LDS
constexpr int kTileBytes = kKvTile * kRowBytes;      // 16 KiB
constexpr int kSubBytes = 32 * kRowBytes;            // one 32-key sub-block of a tile
constexpr int kKBuf = 0;                             // K tiles at 0 and 16 KiB
constexpr int kVBuf = 2 * kTileBytes;                // V tiles at 32 and 48 KiB
constexpr int kLdsBytes = 4 * kTileBytes;
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;
constexpr float kOverflow = 18446744073709551616.0f;   // 2^64: largest probability kept

// Largest r with a[r] <= x, for a non-decreasing a[0..n] with a[0] <= x < a[n].
__device__ inline int upper_index(const int32_t* a, int n, int x) {
  int lo = 0, hi = n;  // invariant: a[lo] <= x < a[hi]
  while (hi - lo > 1) {
    int mid = (lo + hi) >> 1;
    if (a[mid] <= x) lo = mid; else hi = mid;
  }
  return lo;
}

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

// Block-table entry `idx` of the request (0 past its last page: the descriptor of such a
// page then has size 0 and nothing is read from it).  Every lane loads the same entry.
// The index goes into the scalar offset: a load with a VGPR address would make every later
// write of that VGPR wait for the load.
__device__ inline int32_t table_entry(const int32_t* bt, int idx, int last_page) {
  const int n = last_page + 1;
  return (int32_t)__builtin_amdgcn_raw_buffer_load_b32(make_rsrc(bt, 4 * n), 0u,
                                                       __builtin_amdgcn_readfirstlane(4 * idx), 0);
}

// LDS-direct copy: 64 lanes x 16 bytes from a raw buffer (descriptor words in SGPRs) to the
// 1 KiB of LDS at byte address `lds`, lane l's bytes at lds + 16 l.  Issued as inline
// assembly so that the compiler does not treat every later LDS read as waiting on it; the
// caller waits for vmcnt(0) and synchronises before the destination is read.
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
// followed by a few VALU instructions of the softmax and the LDS reads of a later slot.
template <bool kQK, bool kReads>
__device__ inline void slot_schedule() {
  if constexpr (kQK) {
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);     // MFMA
    __builtin_amdgcn_sched_group_barrier(0x002, 4, 0);     // VALU
    if constexpr (kReads) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);   // LDS read (K)
  }
  __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
  __builtin_amdgcn_sched_group_barrier(0x002, kQK ? 3 : 7, 0);
  if constexpr (kReads) __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);     // LDS reads (V)
}

template <bool kFp8, int kWaves>
__global__ __launch_bounds__(kWaves * 64, 8 / kWaves) void attn_main_kernel(
    const uint16_t* __restrict__ q, uint16_t* __restrict__ out, float* __restrict__ lse,
    const void* __restrict__ kpool, const void* __restrict__ vpool, const float* __restrict__ kscale,
    const float* __restrict__ vscale, const int32_t* __restrict__ block_tables, int32_t max_pages,
    int32_t num_reqs, int32_t hq, int32_t hkv, float scale_log2, PlanPtrs pv) {
  constexpr int kQuarters = kWaves / 4;              // waves sharing one page of a tile
  constexpr int kRowsPerWave = 16 / kQuarters;       // key rows each wave moves per tile
  constexpr int kDma = kRowsPerWave / 4;             // bf16: 1 KiB LDS-direct loads per wave
  constexpr int kF8Loads = kRowsPerWave / 8;         // e4m3: 16-byte loads per lane
  constexpr int kRun = kFp8 ? 16 * 128 : 16 * 128 * 2;   // bytes of one (page, kv head)
  constexpr int kKeyBytes = kRun / 16;
  __shared__ __attribute__((aligned(1024))) uint8_t smem[kLdsBytes];

  const int W = pv.hdr->num_items;
  if ((int)blockIdx.x >= W) return;
  const int w_item = xcd_logical(blockIdx.x, gridDim.x < (unsigned)W ? gridDim.x : W);
  const int r = upper_index(pv.item_off, num_reqs, w_item);
  const int nqt = pv.nqt[r], ns = pv.ns[r];
  const Item it = decode_local(w_item - pv.item_off[r], nqt, ns);
  const int P = pv.p[r], C = pv.c[r], row0 = pv.cu[r];
  const int G = hq / hkv;
  const int tq = tile_tokens(G, 32 * kWaves);
  const int i0 = it.qt * tq;
  const int i1 = min(i0 + tq, C);
  int lo, hi;
  piece_range(P + i1, ns, it.s, &lo, &hi);
  const int g = it.g;
  const int32_t* bt = block_tables + (int64_t)r * max_pages;

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int n = lane & 31, half = lane >> 5;
  const int col = wave * 32 + n;
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
  {
    const uint16_t* qrow = q + ((int64_t)(row0 + (valid ? tok : 0)) * hq + (valid ? hq_col : 0)) * 128 + 8 * half;
#pragma unroll
    for (int ks = 0; ks < 8; ++ks) {
      u32x4 x = valid ? *reinterpret_cast<const u32x4*>(qrow + 16 * ks) : u32x4{0, 0, 0, 0};
      qf[ks] = __builtin_bit_cast(bf16x8, x);
    }
  }

  // LDS byte offsets of the operand reads, relative to a tile buffer.
  // K (A of S^T = K Q^T), k-step ks, sub-block 0: row n, chunk 2 ks + half.
  uint32_t ka[8];
#pragma unroll
  for (int ks = 0; ks < 8; ++ks) ka[ks] = n * kRowBytes + ((((2 * ks + half) ^ (n & 15))) << 4);
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
    for (int db = 0; db < 4; ++db)
      va[db] = row * kRowBytes + ((4 * (db ^ ((j >> 2) & 3)) + 2 * b4 + ((j >> 1) & 1)) << 4) + 8 * (j & 1);
  }

  // Tile loads: wave w moves rows [s0, s0 + kRowsPerWave) of page pw of each tile.
  const int pw = wave / kQuarters;
  const int s0 = (wave % kQuarters) * kRowsPerWave;
  uint32_t kvo[kFp8 ? kF8Loads : kDma], vvo[kFp8 ? kF8Loads : kDma];
  if constexpr (!kFp8) {
    // LDS-direct load d writes tile rows 16 pw + s0 + 4d + (l >> 4), chunk l & 15: it
    // fetches the source chunk that the row's permutation puts there.
#pragma unroll
    for (int d = 0; d < kDma; ++d) {
      const int slot = s0 + 4 * d + (lane >> 4), c = lane & 15;
      kvo[d] = slot * kRowBytes + ((c ^ slot) << 4);
      vvo[d] = slot * kRowBytes + ((c ^ ((slot & 3) << 2)) << 4);
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

  // Page pg of the tile at key kb into the K or V buffer at `dst` (bf16: LDS-direct).
  struct F8Stage {
    u32x4 x[kF8Loads];
  };
  auto dma_rows = [&](const char* base, int32_t pg, int kb, int dst, const uint32_t* vo, bool is_k) {
    const int bytes = __builtin_amdgcn_readfirstlane(clamp16(hi - (kb + 16 * pw)) * kKeyBytes);
    const i32x4 rs = sgpr_rsrc(base + (int64_t)pg * page_stride, bytes);
    const uint32_t lds0 = (uint32_t)(uintptr_t)(lds_void*)smem;
#pragma unroll
    for (int d = 0; d < kDma; ++d) {
      const int row = 16 * pw + s0 + 4 * d;
      lds_dma_b128(rs, vo[d], __builtin_amdgcn_readfirstlane(lds0 + dst + row * kRowBytes));
    }
    (void)is_k;
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
      const int sw = is_k ? (row & 15) : ((row & 3) << 2);
      const u32x2 a = fp8x4_to_bf16x4(st.x[i][0]);
      const u32x2 b = fp8x4_to_bf16x4(st.x[i][1]);
      const u32x2 c = fp8x4_to_bf16x4(st.x[i][2]);
      const u32x2 d = fp8x4_to_bf16x4(st.x[i][3]);
      uint8_t* rp = smem + dst + row * kRowBytes;
      *reinterpret_cast<u32x4*>(rp + (((2 * f) ^ sw) << 4)) = u32x4{a[0], a[1], b[0], b[1]};
      *reinterpret_cast<u32x4*>(rp + (((2 * f + 1) ^ sw) << 4)) = u32x4{c[0], c[1], d[0], d[1]};
    }
  };

  f32x16 o[4];
#pragma unroll
  for (int db = 0; db < 4; ++db) o[db] = f32x16{};
  // Row sums per lane: b sums the bf16 probabilities exactly as P.V uses them (O is
  // normalised by it), f sums them unrounded in fp32 (the log-sum-exp).
  struct Sums {
    float b, f;
  };
  float m_run = 0.f;
  Sums l_run = {0.f, 0.f};

  // S(b+1) = K(b+1) Q^T from the sub-block at LDS byte `kofs`.
  auto qk = [&](int kofs) {
    f32x16 s = f32x16{};
#pragma unroll
    for (int ks = 0; ks < 8; ++ks) {
      const bf16x8 a = *reinterpret_cast<const bf16x8*>(smem + kofs + ka[ks]);
      s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qf[ks], s, 0, 0, 0);
    }
    return s;
  };
  // O += P V over the sub-block whose V rows start at LDS byte `vofs`.
  auto pv_acc = [&](const u32x4* p, int vofs) {
#pragma unroll
    for (int k2 = 0; k2 < 2; ++k2) {
      const bf16x8 pb = __builtin_bit_cast(bf16x8, p[k2]);
#pragma unroll
      for (int db = 0; db < 4; ++db) {
        const uint8_t* base = smem + vofs + 16 * k2 * kRowBytes + va[db];
        const v4i16 x = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16*)(base));
        const v4i16 y = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16*)(base + 8 * kRowBytes));
        const u32x2 ux = __builtin_bit_cast(u32x2, x), uy = __builtin_bit_cast(u32x2, y);
        const bf16x8 a = __builtin_bit_cast(bf16x8, u32x4{ux[0], ux[1], uy[0], uy[1]});
        o[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, pb, o[db], 0, 0, 0);
      }
    }
  };
  // One A fragment of O^T += V^T P^T: keys 16 k2 + (4-key sets of this lane half), d-block db.
  auto read_v = [&](int vofs, int k2, int db) {
    const uint8_t* base = smem + vofs + 16 * k2 * kRowBytes + va[db];
    const v4i16 x = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16*)(base));
    const v4i16 y = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16*)(base + 8 * kRowBytes));
    const u32x2 ux = __builtin_bit_cast(u32x2, x), uy = __builtin_bit_cast(u32x2, y);
    return __builtin_bit_cast(bf16x8, u32x4{ux[0], ux[1], uy[0], uy[1]});
  };
  auto read_k = [&](int kofs, int ks) { return *reinterpret_cast<const bf16x8*>(smem + kofs + ka[ks]); };
  // Operands of a step's first two slots, read before its (branchy) softmax prologue.
  struct Pre {
    bf16x8 k[2], v[2];
  };
  auto prefetch = [&](int kofs, int vofs, auto with_qk) {
    Pre f;
    if constexpr (decltype(with_qk)::value) {
      f.k[0] = read_k(kofs, 0);
      f.k[1] = read_k(kofs, 1);
    }
    f.v[0] = read_v(vofs, 0, 0);
    f.v[1] = read_v(vofs, 0, 1);
    return f;
  };
  // Pipelined step in eight slots; slot i issues S(b+1) += K_i Q_i (k-step i), O_db +=
  // V^T P(b-1) (k2 = i / 4, db = i % 4) and the probabilities of score elements 2i, 2i+1
  // of sub-block b, while the operands of slot i + 2 are read from LDS.
  auto step_main = [&](const f32x16& s, const u32x4* pp, u32x4* po, int kofs, int vofs, const Pre& f,
                       auto with_qk, Sums& lsum) {
    constexpr bool kQK = decltype(with_qk)::value;
    f32x16 sn = f32x16{};
    bf16x8 kf[10], vf[10];
    kf[0] = f.k[0];
    kf[1] = f.k[1];
    vf[0] = f.v[0];
    vf[1] = f.v[1];
    float l0 = 0.f, l1 = 0.f, f0 = 0.f, f1 = 0.f;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      if (i + 2 < 8) {
        if constexpr (kQK) kf[i + 2] = read_k(kofs, i + 2);
        vf[i + 2] = read_v(vofs, (i + 2) >> 2, (i + 2) & 3);
      }
      if constexpr (kQK) sn = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[i], qf[i], sn, 0, 0, 0);
      o[i & 3] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf[i], __builtin_bit_cast(bf16x8, pp[i >> 2]), o[i & 3],
                                                          0, 0, 0);
      const float p0 = __builtin_amdgcn_exp2f(__builtin_fmaf(s[2 * i], c_log2, -m_run));
      const float p1 = __builtin_amdgcn_exp2f(__builtin_fmaf(s[2 * i + 1], c_log2, -m_run));
      const uint32_t pk = pack_bf16x2(p0, p1);
      po[i >> 2][i & 3] = pk;
      if (i & 1) {
        l1 = sum_bf16x2(pk, l1);
        f1 += p0 + p1;
      } else {
        l0 = sum_bf16x2(pk, l0);
        f0 += p0 + p1;
      }
    }
    lsum = Sums{l0 + l1, f0 + f1};
    __asm__ volatile("" ::"v"(po[0]), "v"(po[1]), "v"(lsum.b), "v"(lsum.f));   // produced here, not sunk
    slot_schedule<kQK, true>();
    slot_schedule<kQK, true>();
    slot_schedule<kQK, true>();
    slot_schedule<kQK, true>();
    slot_schedule<kQK, true>();
    slot_schedule<kQK, true>();
    slot_schedule<kQK, false>();
    slot_schedule<kQK, false>();
    return sn;
  };
  // Causal mask of sub-block sb0 (element e of a lane's scores is key sb0 + 8 (e / 4) +
  // 4 half + e % 4), applied only where the sub-block reaches past the first query token.
  auto mask = [&](f32x16& s, int sb0) {
    if (sb0 + 31 > P + i0) {
      __asm__ volatile("" ::);   // keep this a branch (not predicated into every sub-block)
      const int lim = horizon - sb0 - 4 * half;
#pragma unroll
      for (int e = 0; e < 16; ++e) s[e] = 8 * (e >> 2) + (e & 3) > lim ? -INFINITY : s[e];
    }
  };
  // exp2(s c - m) -> bf16 pairs (k-slot order of the B operand) and both row sums.
  auto probs = [&](const f32x16& s, u32x4* p, Sums& lsum) {
    float l0 = 0.f, l1 = 0.f, f0 = 0.f, f1 = 0.f;
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
      f0 += p0 + p1;
      f1 += p2 + p3;
    }
    lsum = Sums{l0 + l1, f0 + f1};
  };
  // Settles the probabilities P of the previous sub-block (scores s, row sum lsum) before
  // they enter O.  They were computed against the running reference m; only when one of
  // them exceeds 2^64 (seen in the row sum, an overflow to inf included) is the column's
  // reference raised to that sub-block's exact max: O and l, which hold only earlier
  // sub-blocks, are rescaled and P is recomputed (rare branch).  Then the sum joins l.  The
  // reference of a column is shared by its lane pair, and so is the decision.
  auto settle = [&](const f32x16& s, u32x4* p, Sums& lsum) {
    if (__builtin_amdgcn_ballot_w64(lsum.f > kOverflow) != 0) {
      __asm__ volatile("" ::);
      const bool over = max_with_partner(lsum.f) > kOverflow;
      const float t = block_max(s) * c_log2;
      const float m_new = over ? t : m_run;
      const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
#pragma unroll
      for (int db = 0; db < 4; ++db) o[db] *= alpha;
      l_run.b *= alpha;
      l_run.f *= alpha;
      m_run = m_new;
      probs(s, p, lsum);
    }
    l_run.b += lsum.b;
    l_run.f += lsum.f;
  };

  const int ntiles = hi > lo ? ceil_div(hi - lo, kKvTile) : 0;
  const int last_page = hi > lo ? (hi - 1) >> 4 : 0;
  const int P_i0 = P + i0;
  (void)P_i0;

  auto load_k = [&](int t, int32_t pg, int buf) {  // K of tile t into K buffer buf
    if constexpr (!kFp8) dma_rows(kpb, pg, lo + t * kKvTile, kKBuf + buf * kTileBytes, kvo, true);
  };
  auto load_v = [&](int t, int32_t pg, int buf) {
    if constexpr (!kFp8) dma_rows(vpb, pg, lo + t * kKvTile, kVBuf + buf * kTileBytes, vvo, false);
  };

  f32x16 sp, sc;                 // scores of the previous and the current sub-block
  u32x4 pa[2], pb[2];
  Sums lsum_p = {0.f, 0.f};      // row sums of the probabilities not yet settled
  int32_t pg_next_v = 0;       // page (this wave's) of the tile whose V is loaded next
  int32_t pid_v = 0;           // vector copy of a page-table entry loaded ahead
  F8Stage kst, vst;

  if (ntiles > 0) {
    const int e0 = table_entry(bt, (lo >> 4) + pw, last_page);
    const int e1 = ntiles > 1 ? table_entry(bt, ((lo + kKvTile) >> 4) + pw, last_page) : 0;
    if (ntiles > 2) pid_v = table_entry(bt, ((lo + 2 * kKvTile) >> 4) + pw, last_page);
    __builtin_amdgcn_s_waitcnt(0);
    const int32_t pg0 = __builtin_amdgcn_readfirstlane(e0);
    const int32_t pg1 = __builtin_amdgcn_readfirstlane(e1);
    if constexpr (!kFp8) {
      load_k(0, pg0, 0);
      load_v(0, pg0, 0);
      if (ntiles > 1) load_k(1, pg1, 1);
    } else {
      f8_load(kst, kpb, pg0, lo, kvo);
      f8_load(vst, vpb, pg0, lo, vvo);
      __builtin_amdgcn_s_waitcnt(0);
      f8_store(kst, kKBuf, true);
      f8_store(vst, kVBuf, false);
      if (ntiles > 1) {
        f8_load(kst, kpb, pg1, lo + kKvTile, kvo);
        __builtin_amdgcn_s_waitcnt(0);
        f8_store(kst, kKBuf + kTileBytes, true);
      }
    }
    pg_next_v = pg1;
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();

    // Sub-block 0 sets the reference to its own max (a lane with no visible key there has
    // none in the whole piece, as its visible keys form a prefix of the range).
    sp = qk(kKBuf);
    mask(sp, lo);
    {
      const float t = block_max(sp) * c_log2;
      m_run = t == -INFINITY ? 0.f : t;
    }
    probs(sp, pa, lsum_p);
    sc = qk(kKBuf + kSubBytes);
    __syncthreads();   // K tile 0 is overwritten by the first iteration's loads
  }

  // Iteration t: loads K(t + 2), V(t + 1); sub-blocks 2t+1 and 2t+2 take the softmax, their
  // successors S from K(t + 1), their predecessors O += P V from V(t).  kPar = t & 1.
  auto iteration = [&](int t, auto par) {
    constexpr int kPar = decltype(par)::value;
    const int kcur = kKBuf + (kPar ^ 1) * kTileBytes;   // K(t + 1)
    const int vcur = kVBuf + kPar * kTileBytes;         // V(t)
    const int32_t pg_v = pg_next_v;
    if (t + 2 < ntiles) {
      const int32_t pg_k = __builtin_amdgcn_readfirstlane(pid_v);
      if (t + 3 < ntiles) pid_v = table_entry(bt, ((lo + (t + 3) * kKvTile) >> 4) + pw, last_page);
      if constexpr (!kFp8) load_k(t + 2, pg_k, kPar);
      else f8_load(kst, kpb, pg_k, lo + (t + 2) * kKvTile, kvo);
      pg_next_v = pg_k;
    }
    if constexpr (!kFp8) load_v(t + 1, pg_v, kPar ^ 1);
    else f8_load(vst, vpb, pg_v, lo + (t + 1) * kKvTile, vvo);

    const int sb1 = lo + (2 * t + 1) * 32;
    constexpr std::true_type kWithQK{};
    // sub-block 2t+1 (scores sc; P(2t) in pa, from scores sp)
    {
      const Pre f = prefetch(kcur, vcur, kWithQK);
      settle(sp, pa, lsum_p);
      mask(sc, sb1);
      Sums ls;
      const f32x16 sn = step_main(sc, pa, pb, kcur, vcur, f, kWithQK, ls);
      sp = sc;
      sc = sn;
      lsum_p = ls;
    }
    // sub-block 2t+2 (P(2t+1) in pb)
    {
      const Pre f = prefetch(kcur + kSubBytes, vcur + kSubBytes, kWithQK);
      settle(sp, pb, lsum_p);
      mask(sc, sb1 + 32);
      Sums ls;
      const f32x16 sn = step_main(sc, pb, pa, kcur + kSubBytes, vcur + kSubBytes, f, kWithQK, ls);
      sp = sc;
      sc = sn;
      lsum_p = ls;
    }
    if constexpr (kFp8) {
      __builtin_amdgcn_s_waitcnt(0);
      if (t + 2 < ntiles) f8_store(kst, kKBuf + kPar * kTileBytes, true);
      f8_store(vst, kVBuf + (kPar ^ 1) * kTileBytes, false);
    }
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
  };

  // Every load issued so far is complete here on every path (also ntiles == 0, which skips
  // the block above): otherwise the compiler's bookkeeping keeps the Q loads pending at the
  // loop head and waits for all vector memory, LDS-direct copies included, in each step.
  __builtin_amdgcn_s_waitcnt(0);
  int t = 0;
  for (; t + 2 < ntiles; t += 2) {
    iteration(t, std::integral_constant<int, 0>{});
    iteration(t + 1, std::integral_constant<int, 1>{});
  }
  if (t + 1 < ntiles) {
    iteration(t, std::integral_constant<int, 0>{});
    ++t;
  }
  if (ntiles > 0) {
    // last tile (t = ntiles - 1): sub-block 2t+1 takes the softmax, P(2t) V, then P(2t+1) V
    const int vlast = kVBuf + (t & 1) * kTileBytes;
    constexpr std::false_type kNoQK{};
    const Pre f = prefetch(0, vlast, kNoQK);
    settle(sp, pa, lsum_p);
    mask(sc, lo + (2 * t + 1) * 32);
    Sums ls;
    step_main(sc, pa, pb, 0, vlast, f, kNoQK, ls);
    settle(sc, pb, ls);
    pv_acc(pb, vlast + kSubBytes);
  }

  const float lb_tot = sum_with_partner(l_run.b);
  const float lf_tot = sum_with_partner(l_run.f);
  if (!valid) return;
  if (ns == 1) {
    const float inv = v_mul / lb_tot;
    uint16_t* orow = out + ((int64_t)(row0 + tok) * hq + hq_col) * 128 + 4 * half;
#pragma unroll
    for (int db = 0; db < 4; ++db)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const u32x2 w = {pack_bf16x2(o[db][4 * j] * inv, o[db][4 * j + 1] * inv),
                         pack_bf16x2(o[db][4 * j + 2] * inv, o[db][4 * j + 3] * inv)};
        *reinterpret_cast<u32x2*>(orow + 32 * db + 8 * j) = w;
      }
    if (lse != nullptr && half == 0) lse[(int64_t)(row0 + tok) * hq + hq_col] = (m_run + __log2f(lf_tot)) * kLn2;
  } else {
    float* acc = pv.partials + pv.part_off[r];
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
    // (m, l_b, l_f, 0); a column with no visible key in this piece has (-inf, 0, 0): the
    // merge skips it
    if (half == 0)
      *reinterpret_cast<f32x4*>(ml + 4 * prow) = f32x4{lf_tot > 0.f ? m_run : -INFINITY, lb_tot, lf_tot, 0.f};
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
    for (int s = 0; s < ns; ++s) mstar = fmaxf(mstar, ml[4 * (((int64_t)s * C + tok) * hq + h)]);
    float lb = 0.f, lf = 0.f;
    f32x4 a = {0.f, 0.f, 0.f, 0.f};
    for (int s = 0; s < ns; ++s) {
      const int64_t prow = ((int64_t)s * C + tok) * hq + h;
      const f32x4 mlp = *reinterpret_cast<const f32x4*>(ml + 4 * prow);
      if (mlp[0] == -INFINITY) continue;
      const float wgt = __builtin_amdgcn_exp2f(mlp[0] - mstar);
      lb += wgt * mlp[1];
      lf += wgt * mlp[2];
      const f32x4 x = *reinterpret_cast<const f32x4*>(acc + prow * kHeadDim + d4);
      a += wgt * x;
    }
    const float inv = 1.0f / lb;
    const u32x2 w = {pack_bf16x2(a[0] * inv, a[1] * inv), pack_bf16x2(a[2] * inv, a[3] * inv)};
    *reinterpret_cast<u32x2*>(out + ((int64_t)row * hq + h) * kHeadDim + d4) = w;
    if (lse != nullptr && d4 == 0) lse[(int64_t)row * hq + h] = (mstar + __log2f(lf)) * kLn2;
  }
}

}  // namespace

template <bool kFp8, int kWaves>
void launch_main_variant(const AttnLaunch& a, hipStream_t stream) {
  attn_main_kernel<kFp8, kWaves><<<a.num_items, kWaves * 64, 0, stream>>>(
      static_cast<const uint16_t*>(a.q), static_cast<uint16_t*>(a.out), a.lse, a.kv.kpool, a.kv.vpool,
      a.kv.kscale, a.kv.vscale, a.kv.block_tables, a.kv.max_pages, a.kv.num_reqs, a.hq, a.kv.hkv,
      a.softmax_scale * kLog2e, plan_ptrs(a.workspace, a.kv.num_reqs));
}

hipError_t launch_attn_main(const AttnLaunch& a, hipStream_t stream) {
  if (a.num_items <= 0) return hipSuccess;
  const bool wide = a.tile_cols == kMaxTileCols;
  if (a.kv.fp8) {
    if (wide) launch_main_variant<true, 8>(a, stream);
    else launch_main_variant<true, 4>(a, stream);
  } else {
    if (wide) launch_main_variant<false, 8>(a, stream);
    else launch_main_variant<false, 4>(a, stream);
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
