// Measurement support: ceilings that the benchmark reports the kernels against, measured
// on the GPU at hand rather than taken from the data sheet (HBM read bandwidth reachable
// by a plain streaming kernel; bf16 MFMA rate of a register-only loop at the clock the
// chip holds under that load).  Not part of the attention path.
#include "launch.h"
#include "s2l_device.h"

namespace s2l {

namespace {

// Every thread reads 16-byte units with a grid stride, eight loads in flight, and folds
// them into one word it writes.
__global__ __launch_bounds__(256) void stream_read_kernel(const u32x4* __restrict__ x, uint64_t n16,
                                                          uint32_t* __restrict__ sink) {
  uint64_t i = blockIdx.x * 256ull + threadIdx.x;
  const uint64_t stride = (uint64_t)gridDim.x * 256;
  uint32_t acc = 0;
  for (; i + 7 * stride < n16; i += 8 * stride) {
    u32x4 v[8];
#pragma unroll
    for (int k = 0; k < 8; ++k) v[k] = __builtin_nontemporal_load(x + i + k * stride);
#pragma unroll
    for (int k = 0; k < 8; ++k) acc ^= v[k][0] ^ v[k][1] ^ v[k][2] ^ v[k][3];
  }
  for (; i < n16; i += stride) {
    const u32x4 v = x[i];
    acc ^= v[0] ^ v[1] ^ v[2] ^ v[3];
  }
  sink[blockIdx.x * 256ull + threadIdx.x] = acc;
}

// Four independent accumulation chains of v_mfma_f32_32x32x16_bf16 per wave on register
// operands; the sum of one accumulator element per lane is written at the end.
constexpr int kChains = 4;
__global__ __launch_bounds__(256) void mfma_loop_kernel(int64_t iters, float* __restrict__ sink) {
  const float x = (float)(threadIdx.x & 7) * 0.001f;
  bf16x8 a, b;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    a[e] = (__bf16)(x + e);
    b[e] = (__bf16)(x - e);
  }
  f32x16 acc[kChains];
#pragma unroll
  for (int c = 0; c < kChains; ++c) acc[c] = f32x16{};
  for (int64_t it = 0; it < iters; ++it) {
#pragma unroll
    for (int c = 0; c < kChains; ++c) acc[c] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc[c], 0, 0, 0);
  }
  float s = 0.f;
#pragma unroll
  for (int c = 0; c < kChains; ++c) s += acc[c][threadIdx.x & 15];
  sink[blockIdx.x * 256ull + threadIdx.x] = s;
}

}  // namespace

hipError_t launch_stream_read(const void* buf, uint64_t bytes, uint32_t* sink, int32_t grid, hipStream_t stream) {
  stream_read_kernel<<<grid, 256, 0, stream>>>(static_cast<const u32x4*>(buf), bytes / 16, sink);
  return hipGetLastError();
}

hipError_t launch_mfma_loop(int64_t iters, float* sink, int32_t grid, hipStream_t stream) {
  mfma_loop_kernel<<<grid, 256, 0, stream>>>(iters, sink);
  return hipGetLastError();
}

int64_t mfma_loop_flops(int64_t iters, int32_t grid) {
  return (int64_t)grid * 4 /* waves */ * kChains * iters * 32 * 32 * 16 * 2;
}

}  // namespace s2l
