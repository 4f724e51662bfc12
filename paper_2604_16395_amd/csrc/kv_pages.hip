// Page append (scatter), gather and page-copy (swap) kernels for the paged KV cache.
//
// Paging (Stream2LLM Sec. 2.2): token p of a request lives in logical page p / 16, slot
// p % 16; the block table maps logical pages to physical ones.  Append (Sec. 4.2 /
// Sec. 5.1): a chunk of C new tokens after P cached ones occupies positions P .. P+C-1.
//
// Append: one workgroup per (logical page touched, kv head, request).  A page of one kv head
// is a contiguous 4 KiB (bf16) / 2 KiB (fp8) run of 16 slot rows; thread t moves 16 bytes
// of input (8 elements) of slot t / 16, chunk t % 16, for K and for V: one load and one
// store each, coalesced on both sides (a slot row is 256 contiguous input bytes).
#include "launch.h"
#include "s2l_device.h"

namespace s2l {

namespace {

template <bool kFp8>
__global__ __launch_bounds__(256) void kv_append_kernel(
    void* __restrict__ kpool, void* __restrict__ vpool, const float* __restrict__ kscale,
    const float* __restrict__ vscale, const uint16_t* __restrict__ knew, const uint16_t* __restrict__ vnew,
    const int32_t* __restrict__ prefix_lens, const int32_t* __restrict__ chunk_lens,
    const int32_t* __restrict__ cu_chunk, const int32_t* __restrict__ block_tables, int32_t max_pages,
    int32_t hkv) {
  const int r = blockIdx.z, h = blockIdx.y;
  const int P = prefix_lens[r], C = chunk_lens[r];
  if (C <= 0) return;
  const int lp = (P >> 4) + (int)blockIdx.x;
  if (lp > ((P + C - 1) >> 4)) return;
  const int slot = threadIdx.x >> 4, c = threadIdx.x & 15;
  const int pos = lp * 16 + slot;
  if (pos < P || pos >= P + C) return;
  const int64_t page = block_tables[(int64_t)r * max_pages + lp];
  const int64_t src = ((int64_t)(cu_chunk[r] + pos - P) * hkv + h) * 128 + c * 8;
  const int64_t dst = ((page * hkv + h) * 16 + slot) * 128 + c * 8;
  const u32x4 kx = *reinterpret_cast<const u32x4*>(knew + src);
  const u32x4 vx = *reinterpret_cast<const u32x4*>(vnew + src);
  if constexpr (!kFp8) {
    *reinterpret_cast<u32x4*>(static_cast<uint16_t*>(kpool) + dst) = kx;
    *reinterpret_cast<u32x4*>(static_cast<uint16_t*>(vpool) + dst) = vx;
  } else {
    // code = e4m3(fp32(x) * fp32(1/scale[h])), RNE, saturated
    const float ki = __fdiv_rn(1.0f, kscale[h]);
    const float vi = __fdiv_rn(1.0f, vscale[h]);
    u32x2 kq, vq;
    kq[0] = f32x4_to_fp8x4(bf16lo(kx[0]) * ki, bf16hi(kx[0]) * ki, bf16lo(kx[1]) * ki, bf16hi(kx[1]) * ki);
    kq[1] = f32x4_to_fp8x4(bf16lo(kx[2]) * ki, bf16hi(kx[2]) * ki, bf16lo(kx[3]) * ki, bf16hi(kx[3]) * ki);
    vq[0] = f32x4_to_fp8x4(bf16lo(vx[0]) * vi, bf16hi(vx[0]) * vi, bf16lo(vx[1]) * vi, bf16hi(vx[1]) * vi);
    vq[1] = f32x4_to_fp8x4(bf16lo(vx[2]) * vi, bf16hi(vx[2]) * vi, bf16lo(vx[3]) * vi, bf16hi(vx[3]) * vi);
    *reinterpret_cast<u32x2*>(static_cast<uint8_t*>(kpool) + dst) = kq;
    *reinterpret_cast<u32x2*>(static_cast<uint8_t*>(vpool) + dst) = vq;
  }
}

// Gather: rows cu_out[r] + p (p < n_r) <- stored elements of position p.  kEB = element bytes.
template <int kEB>
__global__ __launch_bounds__(256) void kv_gather_kernel(
    const void* __restrict__ kpool, const void* __restrict__ vpool, void* __restrict__ kout,
    void* __restrict__ vout, const int32_t* __restrict__ prefix_lens, const int32_t* __restrict__ chunk_lens,
    const int32_t* __restrict__ cu_out, const int32_t* __restrict__ block_tables, int32_t max_pages,
    int32_t hkv, int32_t include_chunk) {
  const int r = blockIdx.y;
  const int n = prefix_lens[r] + (include_chunk ? chunk_lens[r] : 0);
  const int lp = blockIdx.x;
  if (lp * 16 >= n) return;
  const int64_t page = block_tables[(int64_t)r * max_pages + lp];
  const int64_t row0 = cu_out[r];
  constexpr int kChunks = 128 * kEB / 16;  // 16-byte chunks per slot row
  const int units = hkv * 16 * kChunks;
  const char* kp = static_cast<const char*>(kpool);
  const char* vp = static_cast<const char*>(vpool);
  char* ko = static_cast<char*>(kout);
  char* vo = static_cast<char*>(vout);
  for (int u = threadIdx.x; u < units; u += 256) {
    const int c = u % kChunks, slot = (u / kChunks) & 15, h = u / (kChunks * 16);
    const int pos = lp * 16 + slot;
    if (pos >= n) continue;
    const int64_t src = (((page * hkv + h) * 16 + slot) * 128) * kEB + c * 16;
    const int64_t dst = (((row0 + pos) * hkv + h) * 128) * kEB + c * 16;
    *reinterpret_cast<u32x4*>(ko + dst) = *reinterpret_cast<const u32x4*>(kp + src);
    *reinterpret_cast<u32x4*>(vo + dst) = *reinterpret_cast<const u32x4*>(vp + src);
  }
}

// Page copy between two pools of the same layout (swap-out: device pool -> pinned host
// pool; swap-in: the reverse).  Workgroup (i, pool) copies pair i's whole page of K
// (pool 0) or V (pool 1): page_bytes contiguous bytes, as 16-byte units, eight loads in
// flight per thread before their stores (host memory is far: latency needs depth).  A
// pair with a page id outside its pool is skipped.
__global__ __launch_bounds__(256) void kv_page_copy_kernel(
    const char* __restrict__ src_k, const char* __restrict__ src_v, char* __restrict__ dst_k,
    char* __restrict__ dst_v, const int32_t* __restrict__ pairs, int32_t num_src, int32_t num_dst,
    int64_t page_bytes) {
  const int32_t sp = pairs[2 * blockIdx.x], dp = pairs[2 * blockIdx.x + 1];
  if (sp < 0 || sp >= num_src || dp < 0 || dp >= num_dst) return;
  const u32x4* src = reinterpret_cast<const u32x4*>((blockIdx.y ? src_v : src_k) + sp * page_bytes);
  u32x4* dst = reinterpret_cast<u32x4*>((blockIdx.y ? dst_v : dst_k) + dp * page_bytes);
  const int units = (int)(page_bytes / 16);
  constexpr int kDepth = 8;
  for (int u0 = threadIdx.x; u0 < units; u0 += 256 * kDepth) {
    u32x4 x[kDepth];
#pragma unroll
    for (int j = 0; j < kDepth; ++j)
      if (u0 + j * 256 < units) x[j] = src[u0 + j * 256];
#pragma unroll
    for (int j = 0; j < kDepth; ++j)
      if (u0 + j * 256 < units) dst[u0 + j * 256] = x[j];
  }
}

// Table check: workgroup (page block, request) looks at 256 logical pages of the request's
// used range [0, ceil((P + C) / 16)) and counts entries outside [0, num_pages) (vector
// atomics into counts[0]; counts[1] keeps the largest request index with a bad entry + 1).
__global__ __launch_bounds__(256) void check_tables_kernel(const int32_t* __restrict__ prefix_lens,
                                                           const int32_t* __restrict__ chunk_lens,
                                                           const int32_t* __restrict__ block_tables,
                                                           int32_t max_pages, int32_t num_pages, int32_t* counts) {
  const int r = blockIdx.y;
  const int used = (prefix_lens[r] + chunk_lens[r] + 15) >> 4;
  const int lp = blockIdx.x * 256 + threadIdx.x;
  if (lp >= used || lp >= max_pages) return;
  const int32_t page = block_tables[(int64_t)r * max_pages + lp];
  if (page < 0 || page >= num_pages) {
    atomicAdd(counts, 1);
    atomicMax(counts + 1, r + 1);
  }
}

__global__ void zero2_kernel(int32_t* counts) {
  if (threadIdx.x < 2) counts[threadIdx.x] = 0;
}

}  // namespace

hipError_t launch_check_tables(const KvLaunch& a, int32_t max_pages_used, int32_t* counts, hipStream_t stream) {
  zero2_kernel<<<1, 64, 0, stream>>>(counts);
  if (a.num_reqs > 0 && max_pages_used > 0) {
    dim3 grid((max_pages_used + 255) / 256, a.num_reqs);
    check_tables_kernel<<<grid, 256, 0, stream>>>(a.prefix_lens, a.chunk_lens, a.block_tables, a.max_pages,
                                                  a.num_pages, counts);
  }
  return hipGetLastError();
}

hipError_t launch_kv_page_copy(const void* src_k, const void* src_v, void* dst_k, void* dst_v,
                               const int32_t* pairs, int32_t n, int32_t num_src, int32_t num_dst,
                               int64_t page_bytes, hipStream_t stream) {
  if (n == 0) return hipSuccess;
  kv_page_copy_kernel<<<dim3(n, 2), 256, 0, stream>>>(
      static_cast<const char*>(src_k), static_cast<const char*>(src_v), static_cast<char*>(dst_k),
      static_cast<char*>(dst_v), pairs, num_src, num_dst, page_bytes);
  return hipGetLastError();
}

hipError_t launch_kv_append(const KvLaunch& a, const void* knew, const void* vnew, int32_t max_pages_touched,
                            hipStream_t stream) {
  if (a.num_reqs == 0 || max_pages_touched == 0) return hipSuccess;
  dim3 grid(max_pages_touched, a.hkv, a.num_reqs);
  if (a.fp8) {
    kv_append_kernel<true><<<grid, 256, 0, stream>>>(
        a.kpool, a.vpool, a.kscale, a.vscale, static_cast<const uint16_t*>(knew),
        static_cast<const uint16_t*>(vnew), a.prefix_lens, a.chunk_lens, a.cu_chunk, a.block_tables,
        a.max_pages, a.hkv);
  } else {
    kv_append_kernel<false><<<grid, 256, 0, stream>>>(
        a.kpool, a.vpool, nullptr, nullptr, static_cast<const uint16_t*>(knew),
        static_cast<const uint16_t*>(vnew), a.prefix_lens, a.chunk_lens, a.cu_chunk, a.block_tables,
        a.max_pages, a.hkv);
  }
  return hipGetLastError();
}

hipError_t launch_kv_gather(const KvLaunch& a, int32_t include_chunk, const int32_t* cu_out, void* kout,
                            void* vout, int32_t max_pages_read, hipStream_t stream) {
  if (a.num_reqs == 0 || max_pages_read == 0) return hipSuccess;
  dim3 grid(max_pages_read, a.num_reqs);
  if (a.fp8) {
    kv_gather_kernel<1><<<grid, 256, 0, stream>>>(a.kpool, a.vpool, kout, vout, a.prefix_lens, a.chunk_lens,
                                                  cu_out, a.block_tables, a.max_pages, a.hkv, include_chunk);
  } else {
    kv_gather_kernel<2><<<grid, 256, 0, stream>>>(a.kpool, a.vpool, kout, vout, a.prefix_lens, a.chunk_lens,
                                                  cu_out, a.block_tables, a.max_pages, a.hkv, include_chunk);
  }
  return hipGetLastError();
}

}  // namespace s2l
