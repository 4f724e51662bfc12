/*
 * s2l_sched.h - host-side scheduler for streamed prefill requests (part of libs2l.so).
 *
 * What it implements (Stream2LLM, arXiv 2604.16395):
 *   - request lifecycle with streamed inputs (Sec. 4.2, Sec. 5.1): a request starts with
 *     some tokens (new_stream), receives further chunks (append mode) or a replacement of
 *     its whole input (update mode), and is told when its input is complete;
 *   - longest-common-prefix invalidation (Sec. 4.2): an update keeps the cached tokens of
 *     the LCP of the old and new inputs, frees the blocks (GPU or CPU) that hold only
 *     tokens past it, lowers num_computed_tokens to at most the LCP and counts the dropped
 *     computed tokens in total_tokens_invalidated;
 *   - the two-phase step (Sec. 4.1): phase 1 ranks every unfinished request with the
 *     selected policy and decides, changing nothing, which fit the token budget and the
 *     GPU block pool; phase 2 allocates blocks in priority order and, when the free pool
 *     is short, preempts the lowest-priority request that was not scheduled and still
 *     holds GPU blocks;
 *   - cost-based preemption (Sec. 4.3): a piecewise-linear recomputation_latency(tokens)
 *     and a swap_latency(blocks) model; the cheaper predicted strategy is taken;
 *   - the priority orders (Sec. 4.4): DEFAULT (running requests in their order, then the
 *     waiting queue FIFO by arrival with preempted requests re-queued at its front, so
 *     the last running request is evicted first), FCFS (complete inputs before partial,
 *     each by arrival), MCPS (most computed tokens first, ties by arrival), LCAS
 *     (complete before partial, each by the latest chunk arrival, newest first).
 *
 * Where the paper leaves a choice open:
 *   - ties in every order fall to arrival time, then to admission order;
 *   - phase 1 charges the whole GPU pool with the blocks each selected request will hold
 *     after the step; blocks of requests not selected count as reclaimable by preemption.
 *     A request with no uncomputed tokens is never selected.  The token budget is given
 *     out in priority order: a request gets min(its uncomputed tokens, budget left);
 *   - swap_latency(C) = swap_fixed_seconds + swap_seconds_per_block * C covers the round
 *     trip; swap is taken only when strictly cheaper than recomputing the victim's
 *     computed tokens and the CPU pool can hold its blocks, else the victim recomputes
 *     (its progress drops to zero);
 *   - free blocks are handed out lowest index first;
 *   - a request whose input is complete and fully computed finishes at the start of the
 *     next step and releases its blocks (the hand-off to decode is not modelled).
 *
 * Executing a step's copies (the caller's job, on one stream, in this order):
 *   1. every swap_out pair (GPU block -> CPU block): its GPU block may be handed to
 *      another request in the same step;
 *   2. every swap_in pair (CPU block -> GPU block); those CPU blocks become free only at
 *      the start of the next step;
 *   3. the appends and attention of the step's batch.
 *
 * Memory and threading: a scheduler is an opaque host object created and destroyed by
 * the caller; every array argument is a caller-owned HOST array.  Calls on one scheduler
 * must not overlap.  Errors return a negative s2l_status (s2l.h) with the reason in
 * s2l_last_error() and leave the scheduler unchanged.  No call touches the GPU.
 */
#ifndef S2L_SCHED_H
#define S2L_SCHED_H

#include "s2l.h"

#ifdef __cplusplus
extern "C" {
#endif

typedef struct s2l_sched s2l_sched;

typedef enum s2l_sched_policy {
  S2L_SCHED_DEFAULT = 0,
  S2L_SCHED_FCFS = 1,
  S2L_SCHED_MCPS = 2,
  S2L_SCHED_LCAS = 3
} s2l_sched_policy;

typedef enum s2l_req_state {
  S2L_REQ_WAITING = 0,    /* no blocks (new, or preempted by recomputation)               */
  S2L_REQ_RUNNING = 1,    /* holds GPU blocks for its computed tokens                     */
  S2L_REQ_SWAPPED = 2,    /* preempted by swapping: its blocks are on the CPU             */
  S2L_REQ_FINISHED = 3
} s2l_req_state;

typedef enum s2l_sched_event {
  S2L_EV_FINISHED = 1,
  S2L_EV_PREEMPT_SWAP = 2,
  S2L_EV_PREEMPT_RECOMPUTE = 3
} s2l_sched_event;

typedef struct s2l_sched_config {
  int32_t policy;               /* s2l_sched_policy                                          */
  int32_t num_gpu_blocks;       /* GPU KV pool size in blocks (pages of 16 tokens), >= 1     */
  int32_t num_cpu_blocks;       /* CPU swap pool size in blocks, >= 0                        */
  int32_t token_budget;         /* tokens per step, >= 1                                     */
  int32_t max_blocks_per_req;   /* block-table row length; longer inputs are rejected        */
  int32_t table_pad;            /* value of the unused entries of an output table row        */
  int32_t num_recompute_points; /* >= 1 points of the recomputation model                   */
  int32_t reserved;             /* must be 0                                                 */
  const double* recompute_tokens;   /* [num_recompute_points], strictly ascending, > 0       */
  const double* recompute_seconds;  /* [num_recompute_points]; between points the model is  */
                                    /* linear, past either end it extends the end segment;  */
                                    /* with one point it is the line through the origin     */
  double swap_fixed_seconds;
  double swap_seconds_per_block;
} s2l_sched_config;

/* One step's result.  The caller sets the array pointers and capacities; the step fills
 * the arrays and the counts.  cap_reqs must be at least the number of unfinished requests
 * (s2l_sched_stats), cap_swap at least num_gpu_blocks; otherwise S2L_ERANGE, nothing
 * changes.  Requests appear in priority order. */
typedef struct s2l_sched_step_out {
  int64_t* req_ids;         /* [cap_reqs] scheduled requests                                */
  int32_t* prefix_lens;     /* [cap_reqs] P: tokens already computed                         */
  int32_t* chunk_lens;      /* [cap_reqs] C: tokens computed in this step                    */
  int32_t* block_tables;    /* [cap_reqs][max_blocks_per_req] GPU blocks, then table_pad     */
  int64_t* event_ids;       /* [cap_reqs] requests finished or preempted in this step       */
  int32_t* event_kinds;     /* [cap_reqs] s2l_sched_event, in the order they happened       */
  int32_t* swap_out;        /* [cap_swap][2] (GPU block, CPU block)                          */
  int32_t* swap_in;         /* [cap_swap][2] (CPU block, GPU block)                          */
  int32_t cap_reqs;
  int32_t cap_swap;
  int32_t num_reqs;
  int32_t num_events;
  int32_t num_swap_out;
  int32_t num_swap_in;
  int32_t total_tokens;     /* sum of chunk_lens                                             */
  int32_t reserved;
  int64_t order_ns;         /* host time of the policy ordering (the sort)                   */
  int64_t step_ns;          /* host time of the whole step                                   */
} s2l_sched_step_out;

typedef struct s2l_sched_req_info {
  int32_t state;                  /* s2l_req_state                                           */
  int32_t num_tokens;             /* current input length                                    */
  int32_t num_computed_tokens;
  int32_t input_complete;
  int64_t total_tokens_invalidated;
  int32_t num_preempt_swap;
  int32_t num_preempt_recompute;
  int32_t num_gpu_blocks;
  int32_t num_cpu_blocks;
  double arrival_time;
  double last_chunk_arrival_time;
} s2l_sched_req_info;

typedef struct s2l_sched_stats {
  int32_t num_unfinished;
  int32_t free_gpu_blocks;
  int32_t free_cpu_blocks;        /* excluding blocks whose release waits for the next step  */
  int32_t reserved;
} s2l_sched_stats;

/* Length of the longest common prefix of two token-id sequences (Sec. 4.2). */
int32_t s2l_lcp_len(const int32_t* a, int32_t na, const int32_t* b, int32_t nb);

s2l_status s2l_sched_create(const s2l_sched_config* cfg, s2l_sched** out);
void s2l_sched_destroy(s2l_sched* s);

/* new_stream (Sec. 5.1; lifecycle of Sec. 4.2): a new request with `n` input tokens (n >= 0)
 * arriving at time `now` (seconds, any
 * origin, non-decreasing over calls).  req_id must be new.  S2L_ERANGE if the input
 * needs more than max_blocks_per_req blocks. */
s2l_status s2l_sched_new_stream(s2l_sched* s, int64_t req_id, const int32_t* ids, int32_t n,
                                int32_t input_complete, double now);
/* Append mode (Sec. 4.2, Sec. 5.1): n more tokens after the current input.  The request must
 * be unfinished
 * with its input not yet complete. */
s2l_status s2l_sched_append(s2l_sched* s, int64_t req_id, const int32_t* ids, int32_t n,
                            int32_t input_complete, double now);
/* Update mode (Sec. 4.2): the input becomes ids[0..n); LCP invalidation as above.  *lcp_out
 * (may be
 * NULL) receives the LCP length. */
s2l_status s2l_sched_update(s2l_sched* s, int64_t req_id, const int32_t* ids, int32_t n,
                            int32_t input_complete, double now, int32_t* lcp_out);
/* One scheduling step (Sec. 4.1; preemption by Sec. 4.3's cost model): finish completed
 * requests, phase 1, phase 2.  The scheduled
 * requests' computed tokens advance by their chunk lengths (the caller runs the step). */
s2l_status s2l_sched_step(s2l_sched* s, s2l_sched_step_out* out);

/* The current priority order of the unfinished requests under the configured policy
 * (Sec. 4.4; its sorting time is what Sec. 6.5 reports) (ids into `ids`, at most `cap`;
 * *n = the number of unfinished requests; *order_ns = host time of the ordering). */
s2l_status s2l_sched_priority_order(s2l_sched* s, int64_t* ids, int32_t cap, int32_t* n, int64_t* order_ns);
/* One request's state (the per-request bookkeeping of Sec. 4.1-4.3: computed tokens, held
 * GPU and CPU blocks); gpu_blocks / cpu_blocks (each [max_blocks_per_req], may be NULL)
 * receive its block lists. */
s2l_status s2l_sched_request(const s2l_sched* s, int64_t req_id, s2l_sched_req_info* info,
                             int32_t* gpu_blocks, int32_t* cpu_blocks);
s2l_status s2l_sched_stats_get(const s2l_sched* s, s2l_sched_stats* stats);

#ifdef __cplusplus
}
#endif

#endif /* S2L_SCHED_H */
