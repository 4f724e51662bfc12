// Chunk-prefill attention over a paged KV cache, and the split-KV merge, for gfx950.
//
// What is computed (Stream2LLM Sec. 2.1 prefill over the pages of Sec. 2.2, resumed at
// num_computed_tokens as in Sec. 4.2): query i of a request's new chunk (absolute position
// t = P + i) attends to keys 0..t of that request, read through its block table.
//
// One workgroup = 4 waves = one work item of the plan: kv head g, 128 packed query
// columns (tq tokens x G heads, token-major) and a key range [lo, hi).  Per 64-key tile:
//   * K (64 x 128) and V^T (128 x 64) are staged in LDS, double buffered; pages are read
//     through the block table, 16-byte loads, keys at or past `hi` are zero-filled;
//   * each wave computes S^T = K Q^T for its 32 columns with v_mfma_f32_32x32x16_bf16
//     (A = K rows from LDS, B = Q held in registers), so every lane owns one query column
//     and 32 of the tile's scores;
//   * online softmax in the exp2 domain, row max shared with lane ^ 32 by
//     v_permlane32_swap; the running maximum is only raised (and O rescaled) when the new
//     maximum exceeds it by more than 2^8, else probabilities up to 2^8 are accumulated
//     against the stale maximum (exact after the final division);
//   * O^T += V^T P^T with the same MFMA: A = V^T from LDS, B = P (bf16) straight from the
//     score registers.  V is transposed while it is written to LDS, keys of each 16-key
//     group stored in the order {0-3, 8-11, 4-7, 12-15} so that the MFMA k-slots of a
//     lane half match the keys that half holds in the score layout;
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
constexpr int kKRow = 128 + 8;                     // bf16 per K row in LDS (272 B: bank-shifted rows)
constexpr int kVRow = kKvTile + 8;                 // bf16 per V^T row in LDS (144 B)
constexpr int kKTile = kKvTile * kKRow;            // elements
constexpr int kVTile = kHeadDim * kVRow;
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

// bf16 cache: thread t loads K rows (t>>4) + 16j, 16-byte chunk t&15, and V rows
// 4(t>>4) .. 4(t>>4)+3 of the same chunk.
template <bool kFp8>
__device__ inline void load_tile(Stage& st, const void* kpool, const void* vpool, const int32_t* bt,
                                 int64_t head_base, int hkv, int kb0, int hi) {
  const int t = threadIdx.x;
  if constexpr (!kFp8) {
    const uint16_t* kp = static_cast<const uint16_t*>(kpool);
    const uint16_t* vp = static_cast<const uint16_t*>(vpool);
    const int c = t & 15;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int key = kb0 + (t >> 4) + 16 * j;
      if (key < hi) {
        const int64_t page = bt[key >> 4];
        st.k[j] = *reinterpret_cast<const u32x4*>(kp + ((page * hkv + head_base) * 16 + (key & 15)) * 128 + c * 8);
      } else {
        st.k[j] = u32x4{0, 0, 0, 0};
      }
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int key = kb0 + 4 * (t >> 4) + i;
      if (key < hi) {
        const int64_t page = bt[key >> 4];
        st.v[i] = *reinterpret_cast<const u32x4*>(vp + ((page * hkv + head_base) * 16 + (key & 15)) * 128 + c * 8);
      } else {
        st.v[i] = u32x4{0, 0, 0, 0};
      }
    }
  } else {
    // fp8 cache (128-byte rows): K rows (t>>3) + 32j, 16-byte chunk t&7 (16 codes);
    // V rows 4(t>>4)+i, 8-byte chunk t&15 (8 codes), kept raw in st.v[i].xy.
    const uint8_t* kp = static_cast<const uint8_t*>(kpool);
    const uint8_t* vp = static_cast<const uint8_t*>(vpool);
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int key = kb0 + (t >> 3) + 32 * j;
      if (key < hi) {
        const int64_t page = bt[key >> 4];
        st.k[j] = *reinterpret_cast<const u32x4*>(kp + ((page * hkv + head_base) * 16 + (key & 15)) * 128 + (t & 7) * 16);
      } else {
        st.k[j] = u32x4{0, 0, 0, 0};
      }
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int key = kb0 + 4 * (t >> 4) + i;
      if (key < hi) {
        const int64_t page = bt[key >> 4];
        const u32x2 w = *reinterpret_cast<const u32x2*>(vp + ((page * hkv + head_base) * 16 + (key & 15)) * 128 + (t & 15) * 8);
        st.v[i] = u32x4{w[0], w[1], 0, 0};
      } else {
        st.v[i] = u32x4{0, 0, 0, 0};
      }
    }
  }
}

// Position (in elements) of 4-key group q4 (keys 4 q4 .. 4 q4 + 3 of a 16-key group) in
// the V^T row: groups are stored in the order 0, 2, 1, 3.
__device__ inline int vt_group_pos(int q4) { return ((q4 & 1) << 1) | (q4 >> 1); }

template <bool kFp8>
__device__ inline void store_tile(const Stage& st, uint16_t* buf) {
  const int t = threadIdx.x;
  uint16_t* kl = buf;
  uint16_t* vl = buf + kKTile;
  u32x4 v[4];
  if constexpr (!kFp8) {
    const int c = t & 15;
#pragma unroll
    for (int j = 0; j < 4; ++j)
      *reinterpret_cast<u32x4*>(kl + ((t >> 4) + 16 * j) * kKRow + c * 8) = st.k[j];
#pragma unroll
    for (int i = 0; i < 4; ++i) v[i] = st.v[i];
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
      v[i] = u32x4{a[0], a[1], b[0], b[1]};
    }
  }
  // V^T: thread holds keys 4kg..4kg+3 x dims 8c..8c+7; dword m of each key row holds
  // dims 2m (low half) and 2m+1 (high half).
  const int c = t & 15, kg = t >> 4;
  const int pos = 16 * (kg >> 2) + 4 * vt_group_pos(kg & 3);
#pragma unroll
  for (int m = 0; m < 4; ++m) {
    const uint32_t lo01 = __builtin_amdgcn_perm(v[1][m], v[0][m], 0x05040100u);
    const uint32_t lo23 = __builtin_amdgcn_perm(v[3][m], v[2][m], 0x05040100u);
    const uint32_t hi01 = __builtin_amdgcn_perm(v[1][m], v[0][m], 0x07060302u);
    const uint32_t hi23 = __builtin_amdgcn_perm(v[3][m], v[2][m], 0x07060302u);
    *reinterpret_cast<u32x2*>(vl + (8 * c + 2 * m) * kVRow + pos) = u32x2{lo01, lo23};
    *reinterpret_cast<u32x2*>(vl + (8 * c + 2 * m + 1) * kVRow + pos) = u32x2{hi01, hi23};
  }
}

template <bool kFp8>
__global__ __launch_bounds__(kThreads, 2) void attn_main_kernel(
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
  const int tq = tile_tokens(G);
  const int i0 = it.qt * tq;
  const int i1 = min(i0 + tq, C);
  int lo, hi;
  piece_range(P + i1, ns, it.s, &lo, &hi);
  const int g = it.g;
  const int32_t* bt = block_tables + (int64_t)r * max_pages;

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
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

  f32x16 o[4];
#pragma unroll
  for (int db = 0; db < 4; ++db) o[db] = f32x16{};
  float m_run = -INFINITY, l_run = 0.f;

  const int ntiles = hi > lo ? ceil_div(hi - lo, kKvTile) : 0;
  Stage st;
  if (ntiles > 0) {
    load_tile<kFp8>(st, kpool, vpool, bt, g, hkv, lo, hi);
    store_tile<kFp8>(st, smem);
  }
  __syncthreads();

  for (int ti = 0; ti < ntiles; ++ti) {
    const int kb0 = lo + ti * kKvTile;
    const uint16_t* kl = smem + (ti & 1) * kBufElems;
    const uint16_t* vl = kl + kKTile;
    const bool more = ti + 1 < ntiles;
    if (more) load_tile<kFp8>(st, kpool, vpool, bt, g, hkv, kb0 + kKvTile, hi);

    // S^T for keys kb0 + [0,32) and kb0 + [32,64): element r of s0 is key 8(r/4) + 4 half + r%4.
    f32x16 s0 = f32x16{}, s1 = f32x16{};
#pragma unroll
    for (int ks = 0; ks < 8; ++ks) {
      const bf16x8 a0 = *reinterpret_cast<const bf16x8*>(kl + n * kKRow + 16 * ks + 8 * half);
      const bf16x8 a1 = *reinterpret_cast<const bf16x8*>(kl + (32 + n) * kKRow + 16 * ks + 8 * half);
      s0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a0, qf[ks], s0, 0, 0, 0);
      s1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a1, qf[ks], s1, 0, 0, 0);
    }
    if (kb0 + kKvTile - 1 > P + i0) {     // chunk-diagonal tile: causal mask
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int key = kb0 + 8 * (e >> 2) + 4 * half + (e & 3);
        if (key > horizon) s0[e] = -INFINITY;
        if (key + 32 > horizon) s1[e] = -INFINITY;
      }
    }
    float mx = -INFINITY;
#pragma unroll
    for (int e = 0; e < 16; ++e) mx = fmaxf(mx, fmaxf(s0[e], s1[e]));
    mx = max_with_partner(mx);
    const float m_tile = mx * c_log2;
    const float m_new = fmaxf(m_run, m_tile);
    if (__any(m_new > m_run + kRescaleSlack)) {
      const float alpha = m_new == m_run ? 1.0f : __builtin_amdgcn_exp2f(m_run - m_new);
      m_run = m_new;
      l_run *= alpha;
#pragma unroll
      for (int db = 0; db < 4; ++db)
#pragma unroll
        for (int e = 0; e < 16; ++e) o[db][e] *= alpha;
    }
    const float mu = m_run == -INFINITY ? 0.0f : m_run;
    uint32_t pk[16];
    float lsum = 0.f;
#pragma unroll
    for (int e = 0; e < 16; e += 2) {
      const float p0 = __builtin_amdgcn_exp2f(__builtin_fmaf(s0[e], c_log2, -mu));
      const float p1 = __builtin_amdgcn_exp2f(__builtin_fmaf(s0[e + 1], c_log2, -mu));
      const float p2 = __builtin_amdgcn_exp2f(__builtin_fmaf(s1[e], c_log2, -mu));
      const float p3 = __builtin_amdgcn_exp2f(__builtin_fmaf(s1[e + 1], c_log2, -mu));
      lsum += (p0 + p1) + (p2 + p3);
      pk[e >> 1] = pack_bf16x2(p0, p1);
      pk[8 + (e >> 1)] = pack_bf16x2(p2, p3);
    }
    l_run += lsum;

    // O^T += V^T P^T over the 4 k-steps of 16 keys.
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      const bf16x8 pb = __builtin_bit_cast(bf16x8, u32x4{pk[4 * ks], pk[4 * ks + 1], pk[4 * ks + 2], pk[4 * ks + 3]});
#pragma unroll
      for (int db = 0; db < 4; ++db) {
        const bf16x8 a = *reinterpret_cast<const bf16x8*>(vl + (32 * db + n) * kVRow + 16 * ks + 8 * half);
        o[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, pb, o[db], 0, 0, 0);
      }
    }
    if (more) store_tile<kFp8>(st, smem + ((ti + 1) & 1) * kBufElems);
    __syncthreads();
  }

  const float l_tot = sum_with_partner(l_run);
  if (!valid) return;
  if (ns == 1) {
    const float inv = v_mul / l_tot;
    uint16_t* orow = out + ((int64_t)(row0 + tok) * hq + hq_col) * 128 + 4 * half;
#pragma unroll
    for (int db = 0; db < 4; ++db)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const u32x2 w = {pack_bf16x2(o[db][4 * j] * inv, o[db][4 * j + 1] * inv),
                         pack_bf16x2(o[db][4 * j + 2] * inv, o[db][4 * j + 3] * inv)};
        *reinterpret_cast<u32x2*>(orow + 32 * db + 8 * j) = w;
      }
    if (lse != nullptr && half == 0) lse[(int64_t)(row0 + tok) * hq + hq_col] = (m_run + __log2f(l_tot)) * kLn2;
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
    if (half == 0) *reinterpret_cast<f32x2*>(ml + 2 * prow) = f32x2{m_run, l_tot};
  }
}

// Merge of split partials: one workgroup per chunk row (token), all heads.
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
  for (int u = threadIdx.x; u < hq * 32; u += 256) {
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

hipError_t launch_attn_main(const AttnLaunch& a, hipStream_t stream) {
  if (a.num_items <= 0) return hipSuccess;
  const float scale_log2 = a.softmax_scale * kLog2e;
  if (a.kv.fp8) {
    attn_main_kernel<true><<<a.num_items, kThreads, 0, stream>>>(
        static_cast<const uint16_t*>(a.q), static_cast<uint16_t*>(a.out), a.lse, a.kv.kpool, a.kv.vpool,
        a.kv.kscale, a.kv.vscale, a.kv.block_tables, a.kv.max_pages, a.kv.num_reqs, a.hq, a.kv.hkv, scale_log2,
        plan_ptrs(a.workspace, a.kv.num_reqs));
  } else {
    attn_main_kernel<false><<<a.num_items, kThreads, 0, stream>>>(
        static_cast<const uint16_t*>(a.q), static_cast<uint16_t*>(a.out), a.lse, a.kv.kpool, a.kv.vpool,
        nullptr, nullptr, a.kv.block_tables, a.kv.max_pages, a.kv.num_reqs, a.hq, a.kv.hkv, scale_log2,
        plan_ptrs(a.workspace, a.kv.num_reqs));
  }
  return hipGetLastError();
}

hipError_t launch_split_reduce(const ReduceLaunch& a, hipStream_t stream) {
  if (a.total_tokens <= 0) return hipSuccess;
  split_reduce_kernel<<<(unsigned)a.total_tokens, 256, 0, stream>>>(
      static_cast<uint16_t*>(a.out), a.lse, plan_ptrs(const_cast<void*>(a.workspace), a.num_reqs), a.num_reqs,
      a.hq);
  return hipGetLastError();
}

}  // namespace s2l
