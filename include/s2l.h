/*
 * s2l.h - incremental chunked-prefill attention over a paged KV cache, for AMD MI355X (gfx950).
 *
 * The operation (Stream2LLM, arXiv 2604.16395):
 *   - prefill computes a key/value pair for every input token and keeps them as the KV
 *     cache (Sec. 2.1);
 *   - the cache is split into fixed blocks of page_size tokens, each placed anywhere in
 *     memory and found through a per-request block table; attention at position t reads
 *     every block covering positions 0..t (Sec. 2.2);
 *   - a streamed request that already holds num_computed_tokens = P cached tokens resumes
 *     prefill from there (Sec. 4.2): in append mode a newly arrived chunk of C tokens is
 *     added after them (Sec. 5.1), so its K/V are appended to the pages and its C queries
 *     attend to the P cached tokens fully and to themselves causally.
 *   Per scheduler step the engine runs a batch of such requests under a token budget
 *   (Sec. 4.1); these calls are that step for one attention layer.
 *
 * Notation: request r has P_r cached tokens and a chunk of C_r new tokens; T = sum C_r;
 * Hq query heads, Hkv kv heads, G = Hq / Hkv, head_dim D = 128, page_size S = 16.
 * Query head h reads kv head h / G.  Chunk token i of request r is absolute position
 * P_r + i and attends to keys 0 .. P_r + i inclusive.
 *
 * Memory and threading contract (all entry points):
 *   - Every tensor argument is a DEVICE pointer owned by the caller, except the fields
 *     documented as host pointers.  The library never allocates or frees memory and keeps
 *     no state between calls; all scratch memory is the caller's workspace.
 *   - Work is enqueued asynchronously on `stream` (a hipStream_t; NULL = the null stream).
 *     Same-stream order is the only ordering: append before attention for the same step.
 *   - Arguments are validated on the host before anything is enqueued.  On failure the call
 *     returns a negative s2l_status, enqueues nothing, and s2l_last_error() holds the reason.
 *     A failed launch returns S2L_EHIP.  Device faults surface at the caller's next sync.
 *   - Preconditions that are not checked (undefined behaviour if violated): block-table
 *     entries for the pages a request uses lie in [0, num_pages); device length arrays hold
 *     the same values as their host copies (a difference that needs more work than the
 *     host planned for is reported by the plan's status word, see s2l_attn_plan); pages
 *     written by an append belong to that request alone (shared prefix pages are
 *     read-only); no two in-flight calls share a workspace.
 */
#ifndef S2L_H
#define S2L_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define S2L_ABI_VERSION 3
#define S2L_HEAD_DIM 128
#define S2L_PAGE_SIZE 16
/* Byte offset, in a workspace that s2l_attn_plan has filled, of the plan's int32 status word
 * (see s2l_attn_plan). */
#define S2L_PLAN_STATUS_OFFSET 36

typedef enum s2l_status {
  S2L_OK = 0,
  S2L_EINVAL = -1,     /* a null pointer, negative length or inconsistent argument      */
  S2L_ERANGE = -2,     /* a request needs more pages than its block-table row holds      */
  S2L_EWORKSPACE = -3, /* workspace missing or smaller than the plan needs               */
  S2L_ENOTSUP = -4,    /* unsupported shape: head_dim != 128, page_size != 16, G > 128,  */
                       /* or a tile_cols other than 0, 128, 256                          */
  S2L_EHIP = -5        /* a HIP runtime call failed (launch or attribute query)          */
} s2l_status;

typedef enum s2l_kv_dtype {
  S2L_KV_BF16 = 0,     /* bf16 elements                                                  */
  S2L_KV_FP8_E4M3 = 1  /* OCP FP8 E4M3 (e4m3fn) codes with per-kv-head fp32 scales       */
} s2l_kv_dtype;

/*
 * One layer's paged KV cache (Sec. 2.2).  K and V are separate pools, each laid out
 * [num_pages][num_kv_heads][page_size][head_dim]: one (page, kv head) pair is a
 * contiguous run of page_size * head_dim elements (4 KiB in bf16, 2 KiB in fp8).
 *
 * fp8 cache: the stored code of value x of kv head h is e4m3(fp32(x) * fp32(1/scale[h]))
 * with round-to-nearest-even and saturation to +-448 (NaN stays NaN); the cached value it
 * stands for is decode(code) * scale[h].  Scales are static, chosen by the caller, > 0.
 */
typedef struct s2l_kv_cache {
  void* k_pages;          /* device; bf16 or uint8 codes                                   */
  void* v_pages;          /* device; same layout                                           */
  const float* k_scale;   /* device [num_kv_heads], fp8 only (must be NULL for bf16)       */
  const float* v_scale;   /* device [num_kv_heads], fp8 only                               */
  int32_t num_pages;
  int32_t num_kv_heads;
  int32_t head_dim;       /* must be 128                                                   */
  int32_t page_size;      /* must be 16                                                    */
  int32_t dtype;          /* s2l_kv_dtype                                                  */
  int32_t reserved;
} s2l_kv_cache;

/*
 * One scheduler step's varlen batch (Sec. 4.1: a continuous batch under a token budget).
 * prefix_lens is num_computed_tokens per request (Sec. 4.2).  chunk_lens may be 0 (the
 * request is skipped).  Row i of request r in q / k_new / v_new / out is row cu_chunk[r] + i.
 */
typedef struct s2l_batch {
  int32_t num_reqs;                /* R >= 0                                                */
  int32_t max_pages_per_req;       /* columns of block_tables                               */
  const int32_t* prefix_lens;      /* device [R]      P_r >= 0                              */
  const int32_t* chunk_lens;       /* device [R]      C_r >= 0                              */
  const int32_t* cu_chunk;         /* device [R+1]    exclusive prefix sum of chunk_lens     */
  const int32_t* block_tables;     /* device [R][max_pages_per_req] physical page ids       */
  const int32_t* prefix_lens_host; /* HOST [R], same values (validation and grid sizing)   */
  const int32_t* chunk_lens_host;  /* HOST [R], same values                                 */
} s2l_batch;

/* Tunables of the work partitioner; pass NULL for the defaults. */
typedef struct s2l_plan_opts {
  int32_t target_items;    /* work items wanted before prefixes are split; 0 = the number   */
                           /* of workgroups the GPU holds at once (CUs x 1 or x 2)          */
  int32_t min_split_keys;  /* smallest key range of a split piece; 0 = 512 (rounded to 64) */
  int32_t max_splits;      /* most pieces per request; 0 = 16 (at most 64)                  */
  int32_t tile_cols;       /* query columns (tokens x heads of one kv head) per work item:  */
                           /* 128 or 256; 0 = automatic: 256 unless such tiles would be     */
                           /* less than half full on average (mostly decode-like rows)      */
  int32_t key_halves;      /* wave groups per work item, each taking half of its key range: */
                           /* 1 (a 4-wave workgroup per 128 columns, two per CU; 8 waves,   */
                           /* one per CU, for 256) or 2 (128 columns only: an 8-wave        */
                           /* workgroup whose two groups merge their halves through LDS,    */
                           /* one per CU); 0 = automatic: 2 for 128 columns, else 1         */
} s2l_plan_opts;

/* What a plan contains, returned to the host by s2l_attn_plan. */
typedef struct s2l_plan_info {
  int32_t num_items;       /* attention work items (one workgroup each)                    */
  int32_t num_split_reqs;  /* requests whose key range is split (they need the reduction)  */
  int32_t split_keys;      /* target piece length in keys; 0 when nothing is split         */
  int32_t num_q_heads;
  int32_t num_kv_heads;
  int32_t num_reqs;
  int64_t total_tokens;    /* T                                                             */
  int64_t workspace_bytes; /* bytes of workspace this plan uses                            */
  int32_t tile_cols;       /* query columns per work item (128 or 256)                     */
  int32_t num_tiles;       /* query tiles (a split tile has one item per key-range piece)   */
  int64_t part_floats;     /* fp32 words of split partials in the workspace                 */
  int32_t key_halves;      /* wave groups per work item (1 or 2)                            */
  int32_t flags;           /* S2L_PLAN_UNIFORM: the items' key ranges are within 25% of     */
                           /* their mean, so consecutive items (one kv head's pages) are    */
                           /* grouped onto one XCD's L2.  S2L_PLAN_BINNED: items of unequal */
                           /* cost, each (request, kv head) group placed whole on the XCD   */
                           /* with the least work so far, longest request first; the bins   */
                           /* are padded with no-op items to equal length (num_items counts */
                           /* them).  Otherwise (the bins would not balance to within 4%)   */
                           /* items run longest request first, spread over the XCDs, so the */
                           /* dispatcher balances them                                      */
} s2l_plan_info;
#define S2L_PLAN_UNIFORM 1
#define S2L_PLAN_BINNED 2

/* ABI version (S2L_ABI_VERSION of the built library).  An ABI utility, not a step of the
 * method. */
int32_t s2l_abi_version(void);

/* Reason for the last failure on the calling thread ("" if none); valid until the next
 * call on this thread.  An ABI utility, not a step of the method. */
const char* s2l_last_error(void);

/*
 * Append each request's chunk K/V to its pages (Sec. 2.2 paging; Sec. 4.2 / Sec. 5.1 append).
 * For i in [0, C_r), h in [0, Hkv): position p = P_r + i goes to page
 * block_tables[r][p / 16], slot p % 16.  Only those slots are written; every other byte of
 * the pools is left untouched (a partially filled first page keeps its earlier slots).
 *   k_new, v_new : device bf16 [T][Hkv][128].
 * Errors: EINVAL (nulls, negative lengths, fp8 without scales), ERANGE (P_r + C_r >
 * max_pages_per_req * 16), ENOTSUP (head_dim/page_size), EHIP.
 */
s2l_status s2l_kv_append(const s2l_kv_cache* cache, const s2l_batch* batch,
                         const void* k_new, const void* v_new, void* stream);

/*
 * Read a request's cached K/V back out of its pages in position order: the inverse of the
 * block-table addressing of Sec. 2.2 (block j of a request holds tokens (j-1)k+1 .. jk,
 * anywhere in the pool), as a preempted request's blocks are copied out when it is swapped
 * to CPU memory (Sec. 2.2 swapping; Sec. 4.3 cost-based preemption).  Copies stored K/V
 * elements of positions 0..n_r-1 of every request, bit-exact (bf16 bits or fp8 codes, not
 * dequantised); n_r = P_r + C_r if include_chunk, else P_r.  Request r's rows go to rows
 * cu_out[r] .. cu_out[r] + n_r - 1 of k_out / v_out, each [rows][Hkv][128] elements of the
 * cache dtype.  Used by the tests and as the dense form of a swap-out.
 *   cu_out : device int32 [R+1] row offsets chosen by the caller (need not be dense).
 *   k_out, v_out: device, caller-owned, at least max_r(cu_out[r] + n_r) rows.
 * Errors: EINVAL (nulls, negative lengths), ERANGE (P_r + C_r > max_pages_per_req * 16),
 * ENOTSUP (head_dim/page_size), EHIP.
 */
s2l_status s2l_kv_gather(const s2l_kv_cache* cache, const s2l_batch* batch, int32_t include_chunk,
                         const int32_t* cu_out, void* k_out, void* v_out, void* stream);

/*
 * Validation of block-table contents on the device (the block tables of Sec. 2.2's paged
 * cache), a debugging aid: the other calls assume
 * the used entries are valid page ids and do not check them.  Counts the used entries of
 * every request (logical pages 0 .. ceil((P + C) / 16) - 1) that lie outside
 * [0, cache->num_pages).
 *   counts: DEVICE int32 [2]; receives (number of such entries, 1 + the largest request
 *           index that has one, or 0).  Asynchronous on `stream`; read after a sync.
 */
s2l_status s2l_check_tables(const s2l_kv_cache* cache, const s2l_batch* batch, int32_t* counts, void* stream);

/*
 * Swap-out and swap-in of KV pages (Sec. 4.3: a preempted request's blocks move to CPU
 * memory and come back when it resumes; Sec. 4.2: blocks past an update's LCP are simply
 * dropped).  One layer's pages move between the device pools of `cache` and two pinned
 * host pools host_k, host_v laid out like them, [num_host_pages][num_kv_heads][16][128]
 * of the cache's element type (bf16 or fp8 codes: pages move as bytes, bit-exact).
 *   pairs: DEVICE int32 [n][2]; swap_out copies device page pairs[i][0] to host page
 *          pairs[i][1]; swap_in copies host page pairs[i][0] to device page pairs[i][1]
 *          (the scheduler's swap_out / swap_in lists have exactly these forms).  A pair
 *          whose page ids fall outside [0, num_pages) or [0, num_host_pages) is skipped.
 *   host_k, host_v: pinned host memory (hipHostMalloc, or torch pin_memory) that the GPU
 *          reads or writes directly over the host link; anything else is S2L_EINVAL.
 *          The caller keeps them alive until the stream has passed the copy.
 * Pages of one call must be distinct on the destination side.  Asynchronous on `stream`.
 */
s2l_status s2l_kv_swap_out(const s2l_kv_cache* cache, const int32_t* pairs, int32_t n, void* host_k,
                           void* host_v, int32_t num_host_pages, void* stream);
s2l_status s2l_kv_swap_in(const s2l_kv_cache* cache, const int32_t* pairs, int32_t n, const void* host_k,
                          const void* host_v, int32_t num_host_pages, void* stream);

/*
 * Workspace bytes that s2l_attn_plan and the attention calls need for one scheduler step's
 * batch (Sec. 4.1: each step runs the continuous batch of selected requests, their new
 * tokens limited by the token budget; Sec. 6.1 runs 2048-8192 tokens per step): the plan
 * header, per-request arrays, one 64-byte record per work item and the fp32 partials of
 * split key ranges.  A host computation from the host length copies (opts as for
 * s2l_attn_plan); nothing is enqueued.
 *   bytes_out: HOST out.
 * Errors: EINVAL (nulls, negative lengths, bad head counts, negative opts), ENOTSUP
 * (tile_cols / key_halves), EHIP (the CU count query, when target_items is 0).
 */
s2l_status s2l_attn_workspace_bytes(const s2l_batch* batch, int32_t num_q_heads, int32_t num_kv_heads,
                                    const s2l_plan_opts* opts, size_t* bytes_out);

/*
 * Build the varlen work partition for one scheduler step (Sec. 4.1: a continuous batch of
 * requests, each with num_computed_tokens cached and a share of the step's token budget as
 * new tokens; Sec. 2.2 continuous batching) and store it in the workspace (a small kernel on
 * `stream`: per-request arrays and one 64-byte record per work item); reuse it for every
 * layer of the step.  Each request's chunk is cut into query tiles of
 * tile_cols / G tokens x G heads per kv head.  When the batch has fewer than target_items
 * tiles, each request's key range 0 .. P_r + i_end is split into up to max_splits pieces of
 * >= min_split_keys keys (never more items than target_items in total), so that long
 * prefixes spread over more workgroups (their partial results are merged by
 * s2l_split_reduce).  With key_halves = 2 a work item's own range is
 * further halved between two wave groups of its workgroup, merged in LDS.
 *   workspace : device, ws_bytes >= s2l_attn_workspace_bytes(...).
 *   info      : HOST out, describes the plan; pass it to the attention calls.
 * The device kernel plans from the device length arrays, sized by the host copies.  Its
 * int32 status word (workspace byte S2L_PLAN_STATUS_OFFSET, readable once the stream has
 * passed the plan) is 0 when the plan was stored, 1 when the device lengths need more work
 * items, tiles or partial space than the host copies planned for (the two disagree, which
 * the contract forbids): then nothing is planned, and every attention call on this plan
 * computes nothing and writes NaN to every element of out (and lse).  Device lengths that
 * differ from the host copies but fit are not detected.
 * Errors: as s2l_attn_workspace_bytes, plus EINVAL (device arrays NULL), ERANGE, EWORKSPACE
 * (workspace NULL or too small), EHIP (launch).
 */
s2l_status s2l_attn_plan(const s2l_batch* batch, int32_t num_q_heads, int32_t num_kv_heads,
                         const s2l_plan_opts* opts, void* workspace, size_t ws_bytes,
                         s2l_plan_info* info, void* stream);

/*
 * Chunk-prefill attention (Sec. 2.1 prefill over the pages of Sec. 2.2, restarted at
 * num_computed_tokens as in Sec. 4.2): for request r, chunk row i, query head h,
 * g = h / G, t = P_r + i:
 *   s_j = softmax_scale * <q[cu_chunk[r]+i][h], K_r[j][g]>   for j = 0..t
 *   out[cu_chunk[r]+i][h] = sum_j e^{s_j} V_r[j][g] / sum_j e^{s_j}     (bf16, RNE)
 *   lse[cu_chunk[r]+i][h] = ln sum_j e^{s_j}                             (fp32, optional)
 * K_r/V_r are read from the pages after the step's append (the chunk's own keys included;
 * for an fp8 cache these are its quantised values decode(code) * scale).  Precision: the
 * weights e^{s_j} / sum are applied as bf16 values normalised by their own sum, so out is
 * within about 2^-7 sum_j w_j |V_j - out| + 2^-8 |out| of the exact result; lse is the
 * log of the sum of those bf16 weights (within about 2^-8 of the exact value).
 *   q   : device bf16 [T][Hq][128] (post-RoPE).     out : device bf16 [T][Hq][128].
 *   lse : device fp32 [T][Hq] or NULL.               softmax_scale > 0 (e.g. 1/sqrt(128)).
 *   plan: the s2l_plan_info returned by s2l_attn_plan for this batch and head counts.
 * Equivalent to s2l_attn_main followed by s2l_split_reduce (which enqueues nothing when
 * no request is split).  Calls on one workspace must not overlap.
 */
s2l_status s2l_chunk_prefill_attn(const s2l_kv_cache* cache, const s2l_batch* batch,
                                  const void* q, int32_t num_q_heads, float softmax_scale,
                                  void* out, float* lse, const s2l_plan_info* plan,
                                  void* workspace, size_t ws_bytes, void* stream);

/*
 * Append and attention of one step in one call (Sec. 4.2 / Sec. 5.1: the chunk's K/V join
 * the cache and its queries attend to prefix and chunk): the same results as
 * s2l_kv_append followed by s2l_chunk_prefill_attn (arguments as there; k_new / v_new
 * bf16 [T][Hkv][128]), pages and outputs bit for bit.  When the cache is bf16, the plan's
 * tiles are 128 or 256 columns and every P_r is a multiple of 16, it is one attention
 * launch (plus the split merge): attention copies the chunk's own keys straight from
 * k_new / v_new, and the first key-range piece of each (kv head, query tile) writes that
 * tile's rows into the pages, which nothing in the launch reads; the append launch and its
 * gap leave the step.  Otherwise it issues the two calls.  *fused_out (may be NULL) = 1
 * if the single launch was used.
 */
s2l_status s2l_append_chunk_prefill_attn(const s2l_kv_cache* cache, const s2l_batch* batch, const void* k_new,
                                         const void* v_new, const void* q, int32_t num_q_heads, float softmax_scale,
                                         void* out, float* lse, const s2l_plan_info* plan, void* workspace,
                                         size_t ws_bytes, int32_t* fused_out, void* stream);

/*
 * s2l_chunk_prefill_attn (Sec. 2.1 attention over the paged cache) with Q quantised too, for
 * e4m3 caches: S = Q K^T runs on the fp8 MFMA (v_mfma_f32_32x32x64_f8f6f4) with K's codes
 * as stored, P V stays on bf16.  Each (token, head) row of Q is encoded as the pages are,
 * with its own scale s = max|q| / 448 (1 for an all-zero row), inv = 1 / s (both fp32,
 * correctly rounded), code = e4m3(fp32(q * inv)), round to nearest even, saturating; the
 * result is the attention of those dequantised rows (code * s) over the dequantised cache,
 * to the same rounding contract as s2l_chunk_prefill_attn.  Arguments as there.  Returns
 * S2L_ENOTSUP for a bf16 cache or a plan with 16-column (decode) tiles.  The quantisation is
 * not in the paper: it is a variant of this library for caches that are already e4m3.
 */
s2l_status s2l_chunk_prefill_attn_q8(const s2l_kv_cache* cache, const s2l_batch* batch, const void* q,
                                     int32_t num_q_heads, float softmax_scale, void* out, float* lse,
                                     const s2l_plan_info* plan, void* workspace, size_t ws_bytes, void* stream);

/*
 * s2l_chunk_prefill_attn for callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the same plan and the same
 * attention and merge launches, with the workspace replaced by a scratch array the library
 * holds on each GPU (S2L_NOALLOC_SCRATCH_BYTES, a file-scope device array that every GPU the
 * library runs on keeps until the process ends).  Plans the batch (opts as for s2l_attn_plan,
 * NULL for the defaults) and runs attention; results are bit-identical to s2l_attn_plan +
 * s2l_chunk_prefill_attn with a caller workspace and the same opts.  The caller still passes
 * q, out and lse; *plan_out (may be NULL) receives the plan's description.
 * Allocates nothing: no hipMalloc, hipFree or allocating library routine.  The scratch holds
 * the last call's plan and partials; every call writes all of it that it reads, so nothing
 * needs clearing.  All calls on one GPU share its scratch: calls that overlap in time on one
 * GPU (different streams or threads without ordering between them) race and give undefined
 * results.
 * Errors: as s2l_chunk_prefill_attn, plus EWORKSPACE when the batch needs more workspace than
 * the scratch holds (s2l_attn_workspace_bytes tells), EHIP when the scratch's device address
 * cannot be taken.
 */
#define S2L_NOALLOC_SCRATCH_BYTES ((size_t)64 << 20)
s2l_status s2l_chunk_prefill_attn_noalloc(const s2l_kv_cache* cache, const s2l_batch* batch, const void* q,
                                          int32_t num_q_heads, float softmax_scale, void* out, float* lse,
                                          const s2l_plan_opts* opts, s2l_plan_info* plan_out, void* stream);

/*
 * The main attention kernel alone: the prefill attention of Sec. 2.1 over the paged cache of
 * Sec. 2.2 (online softmax over the work items of the plan).  Running it and
 * s2l_split_reduce as two launches is this library's choice, not the paper's.
 * Unsplit requests get their final out/lse; split requests get fp32 partials (unnormalised
 * output, then reference max and running sum) in the workspace, merged by s2l_split_reduce.
 */
s2l_status s2l_attn_main(const s2l_kv_cache* cache, const s2l_batch* batch,
                         const void* q, int32_t num_q_heads, float softmax_scale,
                         void* out, float* lse, const s2l_plan_info* plan,
                         void* workspace, size_t ws_bytes, void* stream);

/*
 * Log-sum-exp merge of split partials (the standard online-softmax merge; no passage of the
 * paper describes it: it completes the exact softmax of Sec. 2.1 over key ranges that were
 * processed apart).  For each row and head of a
 * split request, m* = max_s m_s, l* = sum_s l_s 2^(m_s - m*), out = sum_s acc_s 2^(m_s - m*) / l*
 * (bf16), lse = ln(2) (m* + log2 l*) (m in the log2 domain).  Enqueues nothing when the
 * plan has no split request.
 */
s2l_status s2l_split_reduce(const s2l_batch* batch, int32_t num_q_heads, void* out, float* lse,
                            const s2l_plan_info* plan, const void* workspace, size_t ws_bytes,
                            void* stream);

/*
 * Host-only view of the partition of a scheduler step's batch (Sec. 4.1; no GPU needed), for
 * tests and sizing: fills, for each request, the number of
 * query tiles and of key-range pieces, and the workspace layout, exactly as s2l_attn_plan
 * would store them.  items_out, if not NULL, receives num_items rows of 8 int32:
 * {request, kv_head, token_begin, token_end, key_begin, key_end, piece, num_pieces}, the
 * items in request order, then (binned plans) the bins' no-op padding as rows {-1, 0, ...};
 * item_capacity is its row count.  num_cus stands in for the device's CU count.
 */
s2l_status s2l_plan_host(int32_t num_reqs, const int32_t* prefix_lens_host, const int32_t* chunk_lens_host,
                         int32_t num_q_heads, int32_t num_kv_heads, const s2l_plan_opts* opts,
                         int32_t num_cus, s2l_plan_info* info, int32_t* items_out, int64_t item_capacity);

/*
 * Measurement support (not part of the attention path, and not in the paper): ceilings
 * measured on the GPU at hand, for reporting the kernels against.
 *   s2l_calib_stream_read: one streaming read of `bytes` (device, a multiple of 16, > 0)
 *     by `grid` workgroups of 256 threads; each thread writes one word of `sink` (device,
 *     grid * 256 uint32).  Bytes read / kernel time = reachable HBM read bandwidth.
 *   s2l_calib_mfma_bf16: `iters` steps of four independent 32x32x16 bf16 MFMA chains per
 *     wave, `grid` workgroups of four waves, no memory traffic; `sink` (device, grid * 256
 *     floats) receives one result per thread; *flops_out = the MFMA flops it issues.
 * Both are asynchronous on `stream`; time them with events.
 */
s2l_status s2l_calib_stream_read(const void* buf, size_t bytes, uint32_t* sink, int32_t grid, void* stream);
s2l_status s2l_calib_mfma_bf16(int64_t iters, float* sink, int32_t grid, int64_t* flops_out, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* S2L_H */
