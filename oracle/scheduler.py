"""Streaming-request scheduler by definition: request lifecycle, longest-common-prefix
invalidation, the two-phase step, cost-based preemption and the four priority orders.

TEST INFRASTRUCTURE ONLY (see the package docstring).  Plain Python over lists and sets,
written to be checked against the paper by eye, not to be fast.

What it follows (Stream2LLM, arXiv 2604.16395):

* Sec. 4.1 (two-phase scheduling).  Phase 1 ranks every unfinished request with the
  selected policy and decides, without changing any state, which requests fit the token
  budget and the GPU blocks; the rest form ``not_scheduled`` in priority order.  Phase 2
  allocates blocks for the selected requests in priority order; when the free pool is
  short it preempts the lowest-priority request of ``not_scheduled`` that still holds GPU
  blocks, and repeats.  Lifecycle queues: waiting, running, finished; a preempted request
  returns to waiting (recompute resets its progress, swap keeps it on CPU blocks).
* Sec. 4.2 (KV cache invalidation).  An update replaces the input; the LCP of the old and
  new token ids is kept, blocks holding only tokens past it are freed (GPU or CPU),
  ``num_computed_tokens`` drops to at most the LCP, and ``total_tokens_invalidated``
  counts the computed tokens that were dropped.  Append adds tokens after the old ones.
* Sec. 4.3 (cost-based preemption).  recomputation_latency(T) is a piecewise-linear fit
  over token counts; swap_latency(C) is the time to move C blocks between GPU and CPU.
  The cheaper predicted strategy is taken.
* Sec. 4.4 (policies).  DEFAULT: running requests keep their order, waiting ones are
  FIFO by arrival, a preempted request goes to the front of the waiting queue and the
  last running request is the first evicted.  FCFS: complete inputs before partial
  ones, each tier by arrival.  MCPS: most computed tokens first, ties by arrival.
  LCAS: complete before partial, each tier by the latest chunk arrival, newest first.

Readings where the paper is silent (each also made by the library):

* Ties of every order are broken by arrival time, then by admission order.
* Phase 1 charges the GPU pool (all its blocks) with the blocks each selected request
  will hold after the step; blocks of requests that are not selected count as
  reclaimable, which is what lets Phase 2 preempt them.  A request with no new tokens is
  never selected.  The token budget is shared in priority order; a request gets
  min(its uncomputed tokens, the budget left) (chunked prefill).
* swap_latency covers the whole round trip (out and back in):
  swap_fixed + swap_per_block * C.  Swap is taken only when it is strictly cheaper than
  recomputation and the CPU pool can hold the victim's blocks; otherwise recompute.
* Free blocks are handed out lowest index first.  CPU blocks released by a swap-in
  become free only at the start of the next step (the step's copies still read them);
  GPU blocks released by a swap-out are reusable at once, so the caller runs the step's
  swap-outs, then its swap-ins, then its appends.
* At the start of a step, a request whose input is complete and fully computed finishes
  (hand-off to decode is out of scope) and releases its blocks.
* A request updated down to zero computed tokens while swapped returns to plain waiting.

Parity: pinned by ``tests/test_oracle_scheduler.py`` (the paper's worked LCP example,
hand-derived orders and evictions for each policy, the MCPS/LCAS update behaviour the
paper describes, and pool invariants over random event streams).
"""

PAGE_SIZE = 16

DEFAULT, FCFS, MCPS, LCAS = 0, 1, 2, 3
POLICY_NAMES = {DEFAULT: "DEFAULT", FCFS: "FCFS", MCPS: "MCPS", LCAS: "LCAS"}
WAITING, RUNNING, SWAPPED, FINISHED = 0, 1, 2, 3


def lcp_len(a, b):
    """Length of the longest common prefix of token sequences a and b (Sec. 4.2)."""
    n = 0
    while n < len(a) and n < len(b) and a[n] == b[n]:
        n += 1
    return n


def blocks_for(tokens):
    """Blocks of PAGE_SIZE tokens that hold `tokens` tokens."""
    return (tokens + PAGE_SIZE - 1) // PAGE_SIZE


def piecewise_linear(xs, ys, x):
    """The piecewise-linear function through (xs[k], ys[k]), xs ascending, extended past
    both ends by its first and last segments; one point means the line through 0."""
    if len(xs) == 1:
        return ys[0] * (x / xs[0])
    k = 0
    while k < len(xs) - 2 and x > xs[k + 1]:
        k += 1
    return ys[k] + (ys[k + 1] - ys[k]) * ((x - xs[k]) / (xs[k + 1] - xs[k]))


class Request:
    def __init__(self, rid, ids, complete, now, seq):
        self.rid = rid
        self.ids = list(ids)
        self.complete = bool(complete)
        self.arrival = now
        self.last_chunk = now
        self.seq = seq                  # admission order
        self.computed = 0               # num_computed_tokens
        self.gpu = []                   # GPU block table
        self.cpu = []                   # CPU blocks while swapped
        self.state = WAITING
        self.invalidated = 0            # total_tokens_invalidated
        self.n_swap = 0
        self.n_recompute = 0


class Scheduler:
    def __init__(self, policy, num_gpu_blocks, num_cpu_blocks, token_budget, max_blocks_per_req,
                 recompute_tokens, recompute_seconds, swap_fixed, swap_per_block, table_pad=0):
        self.policy = policy
        self.num_gpu = num_gpu_blocks
        self.token_budget = token_budget
        self.max_blocks = max_blocks_per_req
        self.rec_x = list(recompute_tokens)
        self.rec_y = list(recompute_seconds)
        self.swap_fixed = swap_fixed
        self.swap_per_block = swap_per_block
        self.table_pad = table_pad
        self.free_gpu = set(range(num_gpu_blocks))
        self.free_cpu = set(range(num_cpu_blocks))
        self.deferred_cpu = []
        self.reqs = {}
        self.next_seq = 0
        self.running = []               # DEFAULT: running queue
        self.waiting = []               # DEFAULT: waiting queue, front first

    # ---- lifecycle (Sec. 4.2, Sec. 5.1) ----
    def _live(self, rid):
        r = self.reqs.get(rid)
        if r is None or r.state == FINISHED:
            raise ValueError(f"request {rid} is unknown or finished")
        return r

    def new_stream(self, rid, ids, complete, now):
        if rid in self.reqs:
            raise ValueError(f"request {rid} exists")
        if blocks_for(len(ids)) > self.max_blocks:
            raise OverflowError("too many tokens")
        r = Request(rid, ids, complete, now, self.next_seq)
        self.next_seq += 1
        self.reqs[rid] = r
        self.waiting.append(r)

    def append(self, rid, ids, complete, now):
        r = self._live(rid)
        if r.complete:
            raise ValueError("input already complete")
        if blocks_for(len(r.ids) + len(ids)) > self.max_blocks:
            raise OverflowError("too many tokens")
        r.ids += list(ids)
        r.complete = bool(complete)
        r.last_chunk = now

    def update(self, rid, ids, complete, now):
        """Replace the input; keep the LCP, free the blocks past it.  Returns the LCP."""
        r = self._live(rid)
        if r.complete:
            raise ValueError("input already complete")
        if blocks_for(len(ids)) > self.max_blocks:
            raise OverflowError("too many tokens")
        lcp = lcp_len(r.ids, ids)
        keep = min(r.computed, lcp)
        r.invalidated += r.computed - keep
        r.computed = keep
        nb = blocks_for(keep)
        if r.state == SWAPPED:
            self.free_cpu.update(r.cpu[nb:])
            r.cpu = r.cpu[:nb]
            if keep == 0:
                r.state = WAITING
        else:
            self.free_gpu.update(r.gpu[nb:])
            r.gpu = r.gpu[:nb]
        r.ids = list(ids)
        r.complete = bool(complete)
        r.last_chunk = now
        return lcp

    # ---- priority orders (Sec. 4.4) ----
    def priority_order(self):
        live = [r for r in self.reqs.values() if r.state != FINISHED]
        if self.policy == DEFAULT:
            return list(self.running) + list(self.waiting)
        if self.policy == FCFS:
            key = lambda r: (0 if r.complete else 1, r.arrival, r.seq)
        elif self.policy == MCPS:
            key = lambda r: (-r.computed, r.arrival, r.seq)
        elif self.policy == LCAS:
            key = lambda r: (0 if r.complete else 1, -r.last_chunk, r.arrival, r.seq)
        else:
            raise ValueError("policy")
        return sorted(live, key=key)

    # ---- one step (Sec. 4.1, Sec. 4.3) ----
    def _take(self, pool, n):
        got = sorted(pool)[:n]
        assert len(got) == n
        pool.difference_update(got)
        return got

    def _preempt(self, v, out):
        held = len(v.gpu)
        swap_cost = self.swap_fixed + self.swap_per_block * held
        rec_cost = piecewise_linear(self.rec_x, self.rec_y, v.computed)
        if swap_cost < rec_cost and len(self.free_cpu) >= held:
            cpu = self._take(self.free_cpu, held)
            out["swap_out"] += list(zip(v.gpu, cpu))
            self.free_gpu.update(v.gpu)
            v.gpu, v.cpu = [], cpu
            v.state = SWAPPED
            v.n_swap += 1
            out["preempt_swap"].append(v.rid)
            out["events"].append((v.rid, "swap"))
        else:
            self.free_gpu.update(v.gpu)
            v.gpu = []
            v.computed = 0
            v.state = WAITING
            v.n_recompute += 1
            out["preempt_recompute"].append(v.rid)
            out["events"].append((v.rid, "recompute"))
        if self.policy == DEFAULT:
            self.running.remove(v)
            self.waiting.insert(0, v)

    def step(self):
        out = {"reqs": [], "swap_out": [], "swap_in": [], "preempt_swap": [],
               "preempt_recompute": [], "finished": [], "events": []}
        self.free_cpu.update(self.deferred_cpu)
        self.deferred_cpu = []
        for r in sorted(self.reqs.values(), key=lambda r: r.seq):
            if r.state != FINISHED and r.complete and r.computed == len(r.ids):
                self.free_gpu.update(r.gpu)
                self.free_cpu.update(r.cpu)
                r.gpu, r.cpu = [], []
                r.state = FINISHED
                out["finished"].append(r.rid)
                out["events"].append((r.rid, "finished"))
                if r in self.running:
                    self.running.remove(r)
                if r in self.waiting:
                    self.waiting.remove(r)

        # Phase 1: order, then feasibility; nothing is modified
        order = self.priority_order()
        budget = self.token_budget
        claimed = 0
        selected, not_scheduled = [], []
        for r in order:
            n = min(len(r.ids) - r.computed, budget)
            need = blocks_for(r.computed + n)
            if n <= 0 or claimed + need > self.num_gpu:
                not_scheduled.append(r)
                continue
            claimed += need
            budget -= n
            selected.append((r, n))

        # Phase 2: acquire blocks, preempting not_scheduled requests lowest priority first
        for r, n in selected:
            total = blocks_for(r.computed + n)
            have = len(r.cpu) if r.state == SWAPPED else len(r.gpu)
            while len(self.free_gpu) < total - (0 if r.state == SWAPPED else have):
                victim = next((v for v in reversed(not_scheduled) if v.gpu), None)
                assert victim is not None, "phase 1 accounting guarantees a victim"
                self._preempt(victim, out)
            if r.state == SWAPPED:
                back = self._take(self.free_gpu, len(r.cpu))
                out["swap_in"] += list(zip(r.cpu, back))
                self.deferred_cpu += r.cpu
                r.cpu, r.gpu = [], back
            r.gpu += self._take(self.free_gpu, total - len(r.gpu))
            if r.state != RUNNING:
                r.state = RUNNING
                if self.policy == DEFAULT:
                    self.waiting.remove(r)
                    self.running.append(r)
            table = r.gpu + [self.table_pad] * (self.max_blocks - len(r.gpu))
            out["reqs"].append((r.rid, r.computed, n, table))
            r.computed += n
        return out
