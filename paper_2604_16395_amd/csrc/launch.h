// Internal launcher interface between the C-ABI layer (abi.cpp) and the kernel files.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "plan_rules.h"

namespace s2l {

struct KvLaunch {           // device pointers of one layer's cache and one batch
  void* kpool;
  void* vpool;
  const float* kscale;
  const float* vscale;
  const int32_t* prefix_lens;
  const int32_t* chunk_lens;
  const int32_t* cu_chunk;
  const int32_t* block_tables;
  int32_t max_pages;
  int32_t hkv;
  int32_t num_reqs;
  int32_t num_pages;
  bool fp8;
};

hipError_t launch_kv_append(const KvLaunch& a, const void* knew, const void* vnew, int32_t max_pages_touched,
                            hipStream_t stream);
hipError_t launch_kv_gather(const KvLaunch& a, int32_t include_chunk, const int32_t* cu_out, void* kout,
                            void* vout, int32_t max_pages_read, hipStream_t stream);
// Counts used block-table entries outside [0, num_pages) into counts[0] and the largest
// offending request + 1 into counts[1] (both cleared first).
hipError_t launch_check_tables(const KvLaunch& a, int32_t max_pages_used, int32_t* counts, hipStream_t stream);
// Copies whole (page, all kv heads) runs of K and V from pages pairs[i][0] of the source
// pools to pages pairs[i][1] of the destination pools (either side may be pinned host
// memory); pairs is a device array; pairs outside [0, num_src) x [0, num_dst) are skipped.
hipError_t launch_kv_page_copy(const void* src_k, const void* src_v, void* dst_k, void* dst_v,
                               const int32_t* pairs, int32_t n, int32_t num_src, int32_t num_dst,
                               int64_t page_bytes, hipStream_t stream);

struct PlanLaunch {
  const int32_t* prefix_lens;
  const int32_t* chunk_lens;
  const int32_t* cu_chunk;
  int32_t num_reqs, hq, hkv;
  int32_t split_keys, max_splits, tile_cols;   // split_keys chosen by the host planner
  int32_t binned;                              // the host chose the binned item order
  uint8_t group_bin[kBinnedMaxGroups];         // binned: XCD bin of group k Hkv + g (k = ranked slot)
  int64_t ws_bytes;
  void* workspace;
};
// Measurement support (calib.hip): a streaming read of `bytes` (a multiple of 16) over
// `grid` workgroups of 256 threads (sink: grid * 256 words), and a register-only loop of
// bf16 MFMAs (sink: grid * 256 floats; mfma_loop_flops gives its flop count).
hipError_t launch_stream_read(const void* buf, uint64_t bytes, uint32_t* sink, int32_t grid, hipStream_t stream);
hipError_t launch_mfma_loop(int64_t iters, float* sink, int32_t grid, hipStream_t stream);
int64_t mfma_loop_flops(int64_t iters, int32_t grid);

// Attention for a plan of kDecodeTileCols-column items (decode_attn.hip).
struct AttnLaunch;
hipError_t launch_attn_decode(const AttnLaunch& a, hipStream_t stream);

hipError_t launch_attn_plan(const PlanLaunch& a, const PlanDims& dims, hipStream_t stream);

struct AttnLaunch {
  KvLaunch kv;
  const void* q;
  void* out;
  float* lse;
  int32_t hq;
  float softmax_scale;
  void* workspace;
  PlanDims dims;            // host copy of the plan's sizes (grid = dims.num_items)
  int32_t tile_cols;        // 128 or 256 (host copy of the plan's tile width)
  int32_t key_halves;       // 1 or 2 wave groups per item, each on half of its key range
  bool group_by_xcd;        // items of near-equal cost: consecutive items onto one XCD
  const void* knew = nullptr;   // fused append (bf16, page-aligned prefixes): the chunk's
  const void* vnew = nullptr;   //   new K/V rows [T][Hkv][128], else null
  bool q8 = false;              // e4m3 pages: Q quantised per column, S on the fp8 MFMA
  int64_t total_rows = 0;       // T of the host lengths: rows of out / lse (written as NaN
                                //   when the device plan's status says it did not fit)
};
hipError_t launch_attn_main(const AttnLaunch& a, hipStream_t stream);

struct ReduceLaunch {
  void* out;
  float* lse;
  const void* workspace;
  int32_t hq;
  int32_t num_reqs;
  int64_t total_tokens;
  PlanDims dims;
};
hipError_t launch_split_reduce(const ReduceLaunch& a, hipStream_t stream);

// Size of the library-held scratch array of the allocation-free attention call, and its
// device address on the current device (taken on the first call there; noalloc.hip).
constexpr size_t kNoAllocScratchBytes = (size_t)64 << 20;
hipError_t noalloc_scratch(void** ptr);

}  // namespace s2l
