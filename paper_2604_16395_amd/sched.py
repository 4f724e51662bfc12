"""Python binding of the host scheduler in ``include/s2l_sched.h`` (libs2l.so).

Argument marshalling only: ordering, invalidation, feasibility, allocation and preemption
all run in the library's C++ (Stream2LLM Sec. 4.1-4.4).

    s = Scheduler(POLICY_LCAS, num_gpu_blocks=4096, num_cpu_blocks=8192, token_budget=8192,
                  max_blocks_per_req=2048, recompute=([1024, 131072], [0.01, 2.0]),
                  swap=(0.0005, 0.00004))
    s.new_stream(7, ids, complete=False, now=t)
    step = s.step()        # step.req_ids, step.prefix_lens, step.chunk_lens, step.block_tables,
                           # step.swap_out, step.swap_in, step.events
"""
import ctypes
from dataclasses import dataclass

import numpy as np

from . import _lib

POLICY_DEFAULT, POLICY_FCFS, POLICY_MCPS, POLICY_LCAS = 0, 1, 2, 3
POLICIES = {"DEFAULT": 0, "FCFS": 1, "MCPS": 2, "LCAS": 3}
REQ_WAITING, REQ_RUNNING, REQ_SWAPPED, REQ_FINISHED = 0, 1, 2, 3
EV_FINISHED, EV_PREEMPT_SWAP, EV_PREEMPT_RECOMPUTE = 1, 2, 3


def lcp_len(a, b):
    a = np.ascontiguousarray(a, dtype=np.int32)
    b = np.ascontiguousarray(b, dtype=np.int32)
    return _lib.lib().s2l_lcp_len(a.ctypes.data_as(_lib.P_i32), len(a), b.ctypes.data_as(_lib.P_i32), len(b))


@dataclass
class Step:
    req_ids: np.ndarray        # int64 [n]
    prefix_lens: np.ndarray    # int32 [n]
    chunk_lens: np.ndarray     # int32 [n]
    block_tables: np.ndarray   # int32 [n][max_blocks_per_req]
    swap_out: np.ndarray       # int32 [k][2] (GPU block, CPU block)
    swap_in: np.ndarray        # int32 [k][2] (CPU block, GPU block)
    events: list               # [(request id, kind)]
    total_tokens: int
    order_ns: int
    step_ns: int


def _ids(ids):
    a = np.ascontiguousarray(ids, dtype=np.int32)
    return a, a.ctypes.data_as(_lib.P_i32)


class Scheduler:
    def __init__(self, policy, num_gpu_blocks, num_cpu_blocks, token_budget, max_blocks_per_req,
                 recompute, swap, table_pad=0):
        xs = np.ascontiguousarray(recompute[0], dtype=np.float64)
        ys = np.ascontiguousarray(recompute[1], dtype=np.float64)
        cfg = _lib.s2l_sched_config(
            policy=policy, num_gpu_blocks=num_gpu_blocks, num_cpu_blocks=num_cpu_blocks,
            token_budget=token_budget, max_blocks_per_req=max_blocks_per_req, table_pad=table_pad,
            num_recompute_points=len(xs), reserved=0,
            recompute_tokens=xs.ctypes.data_as(ctypes.POINTER(ctypes.c_double)),
            recompute_seconds=ys.ctypes.data_as(ctypes.POINTER(ctypes.c_double)),
            swap_fixed_seconds=float(swap[0]), swap_seconds_per_block=float(swap[1]))
        h = ctypes.c_void_p()
        _lib.call("s2l_sched_create", ctypes.byref(cfg), ctypes.byref(h))
        self._h = h
        self._destroy = _lib.lib().s2l_sched_destroy
        self.max_blocks = max_blocks_per_req
        self.num_gpu_blocks = num_gpu_blocks
        self._cap = 0
        self._grow(64)

    def __del__(self):
        h = getattr(self, "_h", None)
        if h is not None and h.value:
            self._destroy(h)
            self._h = None

    def _grow(self, cap):
        self._cap = cap
        self._req_ids = np.zeros(cap, np.int64)
        self._p = np.zeros(cap, np.int32)
        self._c = np.zeros(cap, np.int32)
        self._tables = np.zeros((cap, self.max_blocks), np.int32)
        self._ev_ids = np.zeros(cap, np.int64)
        self._ev_kinds = np.zeros(cap, np.int32)
        self._swap_out = np.zeros((self.num_gpu_blocks, 2), np.int32)
        self._swap_in = np.zeros((self.num_gpu_blocks, 2), np.int32)

    def new_stream(self, rid, ids, complete, now):
        a, p = _ids(ids)
        _lib.call("s2l_sched_new_stream", self._h, int(rid), p, len(a), int(bool(complete)), float(now))

    def append(self, rid, ids, complete, now):
        a, p = _ids(ids)
        _lib.call("s2l_sched_append", self._h, int(rid), p, len(a), int(bool(complete)), float(now))

    def update(self, rid, ids, complete, now):
        a, p = _ids(ids)
        lcp = ctypes.c_int32()
        _lib.call("s2l_sched_update", self._h, int(rid), p, len(a), int(bool(complete)), float(now),
                  ctypes.byref(lcp))
        return lcp.value

    def stats(self):
        st = _lib.s2l_sched_stats()
        _lib.call("s2l_sched_stats_get", self._h, ctypes.byref(st))
        return st

    def step(self):
        live = self.stats().num_unfinished
        if live > self._cap:
            self._grow(max(live, 2 * self._cap))
        out = _lib.s2l_sched_step_out(
            req_ids=self._req_ids.ctypes.data, prefix_lens=self._p.ctypes.data, chunk_lens=self._c.ctypes.data,
            block_tables=self._tables.ctypes.data, event_ids=self._ev_ids.ctypes.data,
            event_kinds=self._ev_kinds.ctypes.data, swap_out=self._swap_out.ctypes.data,
            swap_in=self._swap_in.ctypes.data, cap_reqs=self._cap, cap_swap=self.num_gpu_blocks)
        _lib.call("s2l_sched_step", self._h, ctypes.byref(out))
        n = out.num_reqs
        return Step(self._req_ids[:n].copy(), self._p[:n].copy(), self._c[:n].copy(), self._tables[:n].copy(),
                    self._swap_out[:out.num_swap_out].copy(), self._swap_in[:out.num_swap_in].copy(),
                    [(int(self._ev_ids[i]), int(self._ev_kinds[i])) for i in range(out.num_events)],
                    out.total_tokens, out.order_ns, out.step_ns)

    def priority_order(self):
        n = ctypes.c_int32()
        ns = ctypes.c_int64()
        cap = max(self.stats().num_unfinished, 1)
        ids = np.zeros(cap, np.int64)
        _lib.call("s2l_sched_priority_order", self._h, ids.ctypes.data_as(ctypes.POINTER(ctypes.c_int64)), cap,
                  ctypes.byref(n), ctypes.byref(ns))
        return ids[:n.value].tolist(), ns.value

    def request(self, rid):
        info = _lib.s2l_sched_req_info()
        gpu = np.zeros(self.max_blocks, np.int32)
        cpu = np.zeros(self.max_blocks, np.int32)
        _lib.call("s2l_sched_request", self._h, int(rid), ctypes.byref(info), gpu.ctypes.data_as(_lib.P_i32),
                  cpu.ctypes.data_as(_lib.P_i32))
        return info, gpu[:info.num_gpu_blocks].tolist(), cpu[:info.num_cpu_blocks].tolist()
