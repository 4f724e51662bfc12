// Chunk attention for decode-shaped work items (16 query columns: C * G <= 16 per kv head,
// e.g. one new token of Llama-3's 4 or 8 query heads per kv head), for gfx950.
//
// What is computed is exactly what the main kernel computes (Stream2LLM Sec. 2.1 prefill
// over the pages of Sec. 2.2, resumed at num_computed_tokens as in Sec. 4.2): query i of a
// request's chunk (position t = P + i) attends to keys 0..t through the block table; an
// unsplit item writes bf16 O and the LSE, a split item writes the same fp32 partials
// (acc, m, l) that the split merge combines.
//
// Such items read a whole key range for very few queries, so they are bound by HBM, not by
// the MFMA: the main kernel's 128-column tiles would spend 8-32x the necessary MFMA and
// softmax work on empty columns.  Here one workgroup of four waves takes one item; the
// waves run independently over the item's 64-key tiles (wave w takes tiles w, w+4, ...),
// each with its own online softmax, and merge their (O, m, l) through LDS at the end.
//
// Per wave and tile (16 columns, one per lane j = l % 16; q = l / 16 picks a key group):
//   * K goes from HBM straight into the A operand of S^T = K Q^T
//     (v_mfma_f32_16x16x32_bf16): lane (j, q) loads key j of the tile's page b, dims
//     32 ks + 8 q .. + 7, a 16-byte load (fp8: 8 bytes, widened to bf16 exactly);
//   * S^T lands as keys 16 b + 4 q + v of column j in lane (j, q);
//   * softmax in the exp2 domain against a per-column reference m (the exact max of the
//     wave's first tile; raised, with O and l rescaled, only if a probability would exceed
//     2^64), probabilities rounded to bf16, the row sum adding exactly those;
//   * V is staged through this wave's private 16 KiB of LDS (key-major rows, 16-byte chunks
//     permuted by 2 (row & 7) so that the transposing reads below hit every bank at most
//     twice) and read with ds_read_b64_tr_b16 as the A operand of O^T += V^T P^T; the key
//     order of both operands is the one the score registers already have, so P goes to the
//     MFMA without any shuffle.
// Loads run one tile ahead (the next tile's K and V, and the page ids two tiles ahead, are
// in flight during a tile's MFMAs).  All loads are ordinary compiler-visible loads, so
// the compiler's own wait counts are exact; the loop is unrolled by two so that the two K
// and V register sets alternate without copies.  No barrier inside the loop: every LDS
// byte a wave reads it wrote itself.
#include "launch.h"
#include "plan_rules.h"
#include "s2l_device.h"

namespace s2l {

namespace {

constexpr int kDecodeWaves = 4;
constexpr int kDTile = 64;                      // keys per tile (four 16-key pages)
constexpr int kVRow = kHeadDim * 2;             // bf16 key row in LDS
constexpr int kVWaveBytes = kDTile * kVRow;     // one wave's V tile: 16 KiB
constexpr float kDLn2 = 0.6931471805599453f;
constexpr float kDOverflow = 18446744073709551616.0f;   // 2^64
constexpr int32_t kDRsrcWord3 = 0x00020000;

typedef short dv4i16 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) dv4i16 lds_dv4i16;

__device__ inline __amdgpu_buffer_rsrc_t page_rsrc(const char* base, int32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<char*>(base), (short)0, bytes, kDRsrcWord3);
}

__device__ inline int clamp16i(int x) { return x < 0 ? 0 : (x > 16 ? 16 : x); }

__device__ inline float xmax16(float x) {   // over the four lanes of one column
  x = fmaxf(x, __shfl_xor(x, 16));
  return fmaxf(x, __shfl_xor(x, 32));
}
__device__ inline float xsum16(float x) {
  x += __shfl_xor(x, 16);
  return x + __shfl_xor(x, 32);
}
__device__ inline float dmerge_weight(float m_s, float mstar) {
  return m_s == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(m_s - mstar);
}

// One tile's K (A operands) and V (rows on their way to LDS), in registers.
template <bool kFp8>
struct TileRegs {
  bf16x8 k[4][4];                     // [page b][k-step ks]
  u32x4 v[kFp8 ? 8 : 16];             // bf16: [page b][4 row groups]; fp8: [page b][2]
};

template <bool kFp8>
__global__ __launch_bounds__(kDecodeWaves * 64, 1) void attn_decode_kernel(
    const uint16_t* __restrict__ q, uint16_t* __restrict__ out, float* __restrict__ lse,
    const void* __restrict__ kpool, const void* __restrict__ vpool, const float* __restrict__ kscale,
    const float* __restrict__ vscale, const int32_t* __restrict__ block_tables, int32_t max_pages, int32_t hq,
    int32_t hkv, float scale_log2, PlanPtrs pv, int32_t group_by_xcd, int64_t total_rows) {
  __shared__ __attribute__((aligned(1024))) uint8_t smem[kDecodeWaves * kVWaveBytes];

  const int w_item = group_by_xcd ? xcd_logical(blockIdx.x, gridDim.x) : (int)blockIdx.x;
  const ItemRec it = pv.items[w_item];
  if (pv.hdr->status != 0) {   // the device plan did not fit this launch: nothing planned
    poison_outputs(out, lse, total_rows, hq);
    return;
  }
  if (w_item >= pv.hdr->num_items || it.r < 0) return;   // past the plan's items, or a bin's padding
  const int P = it.p, C = it.c, row0 = it.row0, ns = it.ns, g = it.g;
  const int i0 = it.i0, i1 = it.i1, lo = it.lo, hi = it.hi;
  const int G = hq / hkv;
  const int tq = tile_tokens(G, kDecodeTileCols);
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int j = lane & 15, qg = lane >> 4;

  // this lane's column: token i0 + j / G, query head g G + j % G (token-major packing)
  const int tok = i0 + j / G;
  const int hq_col = g * G + j % G;
  const bool valid = j < tq * G && tok < i1;
  const int horizon = valid ? P + tok : P + i1 - 1;
  const int key_lim = min(horizon, hi - 1);     // last key this column may see
  const int mask_from = min(P + i0, hi - 1);    // tiles ending past it need the mask

  float c_log2 = scale_log2, v_mul = 1.0f;
  if constexpr (kFp8) {
    c_log2 *= kscale[g];
    v_mul = vscale[g];
  }

  // Q^T (B operand): lane (j, q) holds Q[column j][32 ks + 8 q .. + 7]
  bf16x8 qf[4];
  {
    const uint16_t* qrow = q + ((int64_t)(row0 + (valid ? tok : 0)) * hq + (valid ? hq_col : 0)) * kHeadDim + 8 * qg;
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      const u32x4 x = valid ? *reinterpret_cast<const u32x4*>(qrow + 32 * ks) : u32x4{0, 0, 0, 0};
      qf[ks] = __builtin_bit_cast(bf16x8, x);
    }
  }

  constexpr int kRun = kFp8 ? 16 * kHeadDim : 16 * kHeadDim * 2;   // one (page, kv head)
  constexpr int kKeyBytes = kRun / 16;
  const char* kpb = static_cast<const char*>(kpool) + (int64_t)g * kRun;
  const char* vpb = static_cast<const char*>(vpool) + (int64_t)g * kRun;
  const int64_t page_stride = (int64_t)hkv * kRun;
  const int32_t* bt = block_tables + (int64_t)it.r * max_pages;

  const int nt = hi > lo ? ceil_div(hi - lo, kDTile) : 0;
  const int my_n = nt > wave ? (nt - wave + kDecodeWaves - 1) / kDecodeWaves : 0;
  const int last_page = hi > lo ? (hi - 1) >> 4 : 0;
  uint8_t* vbuf = smem + wave * kVWaveBytes;

  // Page ids of my k-th tile (tile wave + 4 k): lanes with the same lane % 4 = b load the
  // table entry of page b (clamped to the range's last page, whose entry exists).
  auto load_pages = [&](int k) -> int32_t {
    const int idx = (lo >> 4) + 4 * (wave + kDecodeWaves * k) + (lane & 3);
    return bt[idx < last_page ? idx : last_page];
  };
  // Issue the loads of my k-th tile (pages in lanes 0..3 of pg).  Keys at or past `hi`
  // (and every key of a tile past my last) read as zeros.
  auto issue = [&](int k, int32_t pg, TileRegs<kFp8>& t) {
    const int key0 = lo + (wave + kDecodeWaves * k) * kDTile;
#pragma unroll
    for (int b = 0; b < 4; ++b) {
      const int64_t page = __builtin_amdgcn_readlane(pg, b);
      // uniform by construction; readfirstlane lets the compiler see it (a descriptor it
      // must treat as per-lane costs a loop around every load)
      const int bytes = __builtin_amdgcn_readfirstlane(k < my_n ? clamp16i(hi - (key0 + 16 * b)) * kKeyBytes : 0);
      const auto kr = page_rsrc(kpb + page * page_stride, bytes);
      const auto vr = page_rsrc(vpb + page * page_stride, bytes);
      if constexpr (!kFp8) {
#pragma unroll
        for (int ks = 0; ks < 4; ++ks)
          t.k[b][ks] = __builtin_bit_cast(
              bf16x8, __builtin_amdgcn_raw_buffer_load_b128(kr, j * kKeyBytes + 64 * ks + 16 * qg, 0, 0));
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          // LDS row 16 b + 4 i + q, position j holds source chunk j ^ 2 (row & 7)
          const int slot = 4 * i + qg, row = 16 * b + slot;
          t.v[4 * b + i] = __builtin_bit_cast(
              u32x4, __builtin_amdgcn_raw_buffer_load_b128(vr, slot * kKeyBytes + 16 * (j ^ (2 * (row & 7))), 0, 0));
        }
      } else {
#pragma unroll
        for (int ks = 0; ks < 4; ++ks) {
          const u32x2 c8 = __builtin_bit_cast(
              u32x2, __builtin_amdgcn_raw_buffer_load_b64(kr, j * kKeyBytes + 32 * ks + 8 * qg, 0, 0));
          const u32x2 lo4 = fp8x4_to_bf16x4(c8[0]), hi4 = fp8x4_to_bf16x4(c8[1]);
          t.k[b][ks] = __builtin_bit_cast(bf16x8, u32x4{lo4[0], lo4[1], hi4[0], hi4[1]});
        }
#pragma unroll
        for (int i = 0; i < 2; ++i)   // key slot 8 i + l / 8, fp8 dims 16 (l % 8) .. + 15
          t.v[2 * b + i] = __builtin_bit_cast(
              u32x4, __builtin_amdgcn_raw_buffer_load_b128(vr, (8 * i + (lane >> 3)) * kKeyBytes + 16 * (lane & 7), 0, 0));
      }
    }
  };
  // V rows of a tile from registers into this wave's LDS (key-major, permuted chunks).
  auto stage_v = [&](const TileRegs<kFp8>& t) {
    if constexpr (!kFp8) {
#pragma unroll
      for (int b = 0; b < 4; ++b)
#pragma unroll
        for (int i = 0; i < 4; ++i)
          *reinterpret_cast<u32x4*>(vbuf + (16 * b + 4 * i + qg) * kVRow + 16 * j) = t.v[4 * b + i];
    } else {
#pragma unroll
      for (int b = 0; b < 4; ++b)
#pragma unroll
        for (int i = 0; i < 2; ++i) {
          const int row = 16 * b + 8 * i + (lane >> 3), c0 = 2 * (lane & 7), sw = 2 * (row & 7);
          const u32x4 x = t.v[2 * b + i];
          const u32x2 a = fp8x4_to_bf16x4(x[0]), bb = fp8x4_to_bf16x4(x[1]);
          const u32x2 c = fp8x4_to_bf16x4(x[2]), d = fp8x4_to_bf16x4(x[3]);
          *reinterpret_cast<u32x4*>(vbuf + row * kVRow + 16 * (c0 ^ sw)) = u32x4{a[0], a[1], bb[0], bb[1]};
          *reinterpret_cast<u32x4*>(vbuf + row * kVRow + 16 * ((c0 + 1) ^ sw)) = u32x4{c[0], c[1], d[0], d[1]};
        }
    }
  };
  // A operand of O^T += V^T P^T for dims 16 db .. + 15 and keys 32 kk + (4 q + 0..3, then
  // 16 + 4 q + 0..3): lane (i, q) of the transposing read addresses key row
  // 32 kk + 4 q + i / 4 (+ 16), dims 16 db + 4 (i % 4) .. + 3, and receives the four keys of
  // dim 16 db + i.
  auto read_vt = [&](int kk, int db) {
    const int row = 32 * kk + 4 * qg + (j >> 2);
    const int chunk = 2 * db + ((j >> 1) & 1);
    const uint8_t* a0 = vbuf + row * kVRow + 16 * (chunk ^ (2 * (row & 7))) + 8 * (j & 1);
    const uint8_t* a1 = vbuf + (row + 16) * kVRow + 16 * (chunk ^ (2 * ((row + 16) & 7))) + 8 * (j & 1);
    const dv4i16 x = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_dv4i16*)a0);
    const dv4i16 y = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_dv4i16*)a1);
    const u32x2 ux = __builtin_bit_cast(u32x2, x), uy = __builtin_bit_cast(u32x2, y);
    return __builtin_bit_cast(bf16x8, u32x4{ux[0], ux[1], uy[0], uy[1]});
  };

  f32x4 o[8];
#pragma unroll
  for (int db = 0; db < 8; ++db) o[db] = f32x4{0.f, 0.f, 0.f, 0.f};
  float m_run = 0.f, l_run = 0.f;

  // One tile: scores, mask, probabilities (settling the reference), P V.
  auto compute = [&](int k, const TileRegs<kFp8>& t) {
    const int key0 = lo + (wave + kDecodeWaves * k) * kDTile;
    f32x4 s[4];
#pragma unroll
    for (int b = 0; b < 4; ++b) {
      s[b] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < 4; ++ks) s[b] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(t.k[b][ks], qf[ks], s[b], 0, 0, 0);
    }
    if (key0 + kDTile - 1 > mask_from) {
      const int lim = key_lim - key0 - 4 * qg;
#pragma unroll
      for (int b = 0; b < 4; ++b)
#pragma unroll
        for (int v = 0; v < 4; ++v) s[b][v] = 16 * b + v > lim ? -INFINITY : s[b][v];
    }
    if (k == 0) {   // the reference: this column's exact max over the wave's first tile
      float mx = s[0][0];
#pragma unroll
      for (int b = 0; b < 4; ++b)
#pragma unroll
        for (int v = 0; v < 4; ++v) mx = fmaxf(mx, s[b][v]);
      const float t0 = xmax16(mx) * c_log2;
      m_run = t0 == -INFINITY ? 0.f : t0;
    }
    uint32_t pk[8];
    float lsum = 0.f;
    auto probs = [&]() {
      lsum = 0.f;
#pragma unroll
      for (int b = 0; b < 4; ++b) {
        pk[2 * b] = pack_bf16x2(__builtin_amdgcn_exp2f(__builtin_fmaf(s[b][0], c_log2, -m_run)),
                                __builtin_amdgcn_exp2f(__builtin_fmaf(s[b][1], c_log2, -m_run)));
        pk[2 * b + 1] = pack_bf16x2(__builtin_amdgcn_exp2f(__builtin_fmaf(s[b][2], c_log2, -m_run)),
                                    __builtin_amdgcn_exp2f(__builtin_fmaf(s[b][3], c_log2, -m_run)));
        lsum = sum_bf16x2(pk[2 * b], lsum);
        lsum = sum_bf16x2(pk[2 * b + 1], lsum);
      }
    };
    probs();
    if (__builtin_amdgcn_ballot_w64(lsum > kDOverflow) != 0) {
      // rare: a probability above 2^64 (or inf) in some column; that column's reference
      // becomes this tile's max, O and l (earlier tiles only) are rescaled, P is redone
      const bool over = xmax16(lsum) > kDOverflow;
      float mx = s[0][0];
#pragma unroll
      for (int b = 0; b < 4; ++b)
#pragma unroll
        for (int v = 0; v < 4; ++v) mx = fmaxf(mx, s[b][v]);
      const float tmax = xmax16(mx) * c_log2;
      const float m_new = over ? tmax : m_run;
      const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
#pragma unroll
      for (int db = 0; db < 8; ++db) o[db] *= alpha;
      l_run *= alpha;
      m_run = m_new;
      probs();
    }
    l_run += lsum;
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) {
      const bf16x8 pb = __builtin_bit_cast(bf16x8, u32x4{pk[4 * kk], pk[4 * kk + 1], pk[4 * kk + 2], pk[4 * kk + 3]});
#pragma unroll
      for (int db = 0; db < 8; ++db) o[db] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(read_vt(kk, db), pb, o[db], 0, 0, 0);
    }
  };

  if (my_n > 0) {
    TileRegs<kFp8> ta, tb;
    int32_t pg0 = load_pages(0);
    int32_t pg1 = load_pages(1);
    issue(0, pg0, ta);
    int32_t pg2 = load_pages(2);
    // step k: issue tile k+1 (pages known), stage V(k), compute tile k
    auto step = [&](int k, TileRegs<kFp8>& cur, TileRegs<kFp8>& nxt, int32_t& pnext, int32_t& pafter) {
      const int32_t p3 = load_pages(k + 3);
      issue(k + 1, pnext, nxt);
      stage_v(cur);
      compute(k, cur);
      pnext = pafter;
      pafter = p3;
    };
    for (int k = 0; k < my_n; k += 2) {
      step(k, ta, tb, pg1, pg2);
      step(k + 1, tb, ta, pg1, pg2);   // past my last tile: zero-size loads, fully masked
    }
  }

  // merge the four waves' (O, m, l) through LDS, then each wave finishes two dim blocks
  const float l_col = xsum16(l_run);
  const float m_col = l_col > 0.f ? m_run : -INFINITY;   // -inf: no visible key here
  __syncthreads();
  float* xo = reinterpret_cast<float*>(smem);                              // [wave][db][lane][4]
  float* xml = xo + kDecodeWaves * 8 * 64 * 4;                            // [wave][lane][2]
#pragma unroll
  for (int db = 0; db < 8; ++db) *reinterpret_cast<f32x4*>(xo + ((wave * 8 + db) * 64 + lane) * 4) = o[db];
  *reinterpret_cast<f32x2*>(xml + (wave * 64 + lane) * 2) = f32x2{m_col, l_col};
  __syncthreads();
  float mw[kDecodeWaves], lw[kDecodeWaves], mstar = -INFINITY;
#pragma unroll
  for (int w = 0; w < kDecodeWaves; ++w) {
    const f32x2 ml = *reinterpret_cast<const f32x2*>(xml + (w * 64 + lane) * 2);
    mw[w] = ml[0];
    lw[w] = ml[1];
    mstar = fmaxf(mstar, ml[0]);
  }
  float lstar = 0.f, aw[kDecodeWaves];
#pragma unroll
  for (int w = 0; w < kDecodeWaves; ++w) {
    aw[w] = dmerge_weight(mw[w], mstar);
    lstar += aw[w] * lw[w];
  }
  if (!valid) return;
  const float m_fin = lstar > 0.f ? mstar : -INFINITY;
  float* acc = pv.partials + it.part_off;
  float* mlp = acc + (int64_t)ns * C * hq * kHeadDim;
  const int64_t prow = ((int64_t)it.s * C + tok) * hq + hq_col;
  const float inv = v_mul / lstar;
#pragma unroll
  for (int d = 0; d < 2; ++d) {
    const int db = 2 * wave + d;
    f32x4 x = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int w = 0; w < kDecodeWaves; ++w) x += aw[w] * *reinterpret_cast<const f32x4*>(xo + ((w * 8 + db) * 64 + lane) * 4);
    const int dim = 16 * db + 4 * qg;   // this lane's four dims of the block
    if (ns == 1) {
      const u32x2 wv = {pack_bf16x2(x[0] * inv, x[1] * inv), pack_bf16x2(x[2] * inv, x[3] * inv)};
      *reinterpret_cast<u32x2*>(out + ((int64_t)(row0 + tok) * hq + hq_col) * kHeadDim + dim) = wv;
    } else {
      *reinterpret_cast<f32x4*>(acc + prow * kHeadDim + dim) = x * v_mul;
    }
  }
  if (wave == 0 && qg == 0) {
    if (ns == 1) {
      if (lse != nullptr) lse[(int64_t)(row0 + tok) * hq + hq_col] = (m_fin + __log2f(lstar)) * kDLn2;
    } else {
      *reinterpret_cast<f32x4*>(mlp + 4 * prow) = f32x4{m_fin, lstar, 0.f, 0.f};
    }
  }
}

}  // namespace

hipError_t launch_attn_decode(const AttnLaunch& a, hipStream_t stream) {
  if (a.dims.num_items <= 0) return hipSuccess;
  const float scale_log2 = a.softmax_scale * 1.4426950408889634f;
  if (a.kv.fp8) {
    attn_decode_kernel<true><<<(unsigned)a.dims.num_items, kDecodeWaves * 64, 0, stream>>>(
        static_cast<const uint16_t*>(a.q), static_cast<uint16_t*>(a.out), a.lse, a.kv.kpool, a.kv.vpool,
        a.kv.kscale, a.kv.vscale, a.kv.block_tables, a.kv.max_pages, a.hq, a.kv.hkv, scale_log2,
        plan_ptrs(a.workspace, a.dims), a.group_by_xcd ? 1 : 0, a.total_rows);
  } else {
    attn_decode_kernel<false><<<(unsigned)a.dims.num_items, kDecodeWaves * 64, 0, stream>>>(
        static_cast<const uint16_t*>(a.q), static_cast<uint16_t*>(a.out), a.lse, a.kv.kpool, a.kv.vpool,
        a.kv.kscale, a.kv.vscale, a.kv.block_tables, a.kv.max_pages, a.hq, a.kv.hkv, scale_log2,
        plan_ptrs(a.workspace, a.dims), a.group_by_xcd ? 1 : 0, a.total_rows);
  }
  return hipGetLastError();
}

}  // namespace s2l
