"""Timing of the library on the named workloads other than the headline step (used by
bench.py).  Inputs are seeded and synthetic: lengths and page tables from the same numpy
recipes as the parity tests (workloads/), Q/K/V drawn on the GPU as N(0, 0.5^2) bf16 from a
seeded torch generator, the prefix written into the pages by the library's own append (for
an fp8 cache: E4M3 codes with per-kv-head scales max|X_h| / 448).  Every timed region is a
HIP graph of the launches, replayed, with HIP events on its stream around the replays.
"""
import math
import time

import numpy as np
import torch

import paper_2604_16395_amd as s2l

PEAK_BF16_TFLOPS = 2500.0
PEAK_FP8_TFLOPS = 5000.0
# The quantised-Q path runs half its FLOPs (Q K^T) on the fp8 MFMA and half (P V) on the bf16
# one: at both peaks at once its FLOPs take 0.5 / 5000 + 0.5 / 2500 s per PFLOP, a mixed peak
# of 3333 TFLOP/s.
PEAK_MIXED_Q8_TFLOPS = 1.0 / (0.5 / PEAK_FP8_TFLOPS + 0.5 / PEAK_BF16_TFLOPS)
PEAK_HBM_GBS = 8000.0
SCALE = 1.0 / math.sqrt(128.0)


class Layer:
    """One layer's pool with a request batch's prefix already in its pages."""

    def __init__(self, P, C, hq, hkv, pool_pages, tables, gen, fp8=False, copies=1, dev="cuda"):
        P = np.asarray(P, np.int32)
        C = np.asarray(C, np.int32)
        self.P, self.C, self.hq, self.hkv, self.fp8 = P, C, hq, hkv, fp8
        seq = P + C
        T = int(C.sum())
        kfull = (torch.randn((int(seq.sum()), hkv, 128), generator=gen, device=dev) * 0.5).to(torch.bfloat16)
        vfull = (torch.randn((int(seq.sum()), hkv, 128), generator=gen, device=dev) * 0.5).to(torch.bfloat16)
        self.q = (torch.randn((T, hq, 128), generator=gen, device=dev) * 0.5).to(torch.bfloat16)
        starts = np.concatenate([[0], np.cumsum(seq)[:-1]])
        pre_idx = np.concatenate([np.arange(s, s + p) for s, p in zip(starts, P)]) if P.sum() else np.zeros(0, np.int64)
        new_idx = np.concatenate([np.arange(s + p, s + p + c) for s, p, c in zip(starts, P, C)])
        pre_idx_t = torch.from_numpy(pre_idx.astype(np.int64)).to(dev)
        new_idx_t = torch.from_numpy(new_idx.astype(np.int64)).to(dev)
        self.k_new, self.v_new = kfull[new_idx_t].contiguous(), vfull[new_idx_t].contiguous()
        scales = None
        if fp8:
            ks = (kfull.float().abs().amax(dim=(0, 2)) / 448.0).contiguous()
            vs = (vfull.float().abs().amax(dim=(0, 2)) / 448.0).contiguous()
            scales = (ks, vs)
        self.caches = []
        for _ in range(copies):
            dt = torch.uint8 if fp8 else torch.bfloat16
            kp = torch.zeros((pool_pages, hkv, 16, 128), dtype=dt, device=dev)
            vp = torch.zeros_like(kp)
            cache = s2l.PagedKVCache(kp, vp, *(scales or (None, None)))
            if P.sum():
                pre = s2l.Batch(np.zeros_like(P), P, tables)
                s2l.s2l_kv_append(cache, pre, kfull[pre_idx_t].contiguous(), vfull[pre_idx_t].contiguous())
            self.caches.append(cache)
        del kfull, vfull
        self.batch = s2l.Batch(P, C, tables)
        self.out = torch.empty((T, hq, 128), dtype=torch.bfloat16, device=dev)
        self.lse = torch.empty((T, hq), dtype=torch.float32, device=dev)
        self.ws = torch.empty(s2l.s2l_attn_workspace_bytes(self.batch, hq, hkv), dtype=torch.uint8, device=dev)
        torch.cuda.synchronize()

    def step(self, copy, stream):
        c = self.caches[copy % len(self.caches)]
        s2l.s2l_kv_append(c, self.batch, self.k_new, self.v_new, stream)
        plan = s2l.s2l_attn_plan(self.batch, self.hq, self.hkv, self.ws, None, stream)
        s2l.s2l_attn_main(c, self.batch, self.q, self.hq, SCALE, self.out, self.lse, plan, self.ws, stream)
        s2l.s2l_split_reduce(self.batch, self.hq, self.out, self.lse, plan, self.ws, stream)
        return plan

    def attn(self, copy, plan, stream):
        c = self.caches[copy % len(self.caches)]
        s2l.s2l_attn_main(c, self.batch, self.q, self.hq, SCALE, self.out, self.lse, plan, self.ws, stream)

    def flops(self):
        P, C = self.P.astype(np.float64), self.C.astype(np.float64)
        return float(4.0 * 128 * self.hq * (C * P + C * (C + 1) / 2).sum())

    def kv_bytes(self):
        return float((self.P + self.C).astype(np.float64).sum() * self.hkv * 128 * 2 * (1 if self.fp8 else 2))

    def io_bytes(self):
        """Algorithmic HBM bytes of attention: K+V of every visible key, Q in and O out."""
        return self.kv_bytes() + float(self.C.sum()) * self.hq * 128 * 2 * 2


def timed_graph(fn, stream, reps=5, settle=0.25):
    """Average ms of one replay of a graph of fn's launches, after untimed replays for `settle`
    seconds (at least one) so that the clock has reached its loaded steady state."""
    g = torch.cuda.CUDAGraph()
    with torch.cuda.stream(stream):
        with torch.cuda.graph(g, stream=stream):
            fn()
    t0 = time.perf_counter()
    while True:
        with torch.cuda.stream(stream):
            g.replay()
        stream.synchronize()
        if time.perf_counter() - t0 >= settle:
            break
    with torch.cuda.stream(stream):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(stream)
        for _ in range(reps):
            g.replay()
        b.record(stream)
    torch.cuda.synchronize()
    return a.elapsed_time(b) / reps


def tables_for(P, C, pool_pages, rng):
    """Disjoint page slices of one random permutation of the pool, one row per request."""
    need = (np.asarray(P) + np.asarray(C) + 15) // 16
    perm = rng.permutation(pool_pages).astype(np.int32)
    width = int(need.max())
    bt = np.zeros((len(P), width), np.int32)
    o = 0
    for r, n in enumerate(need):
        bt[r, :n] = perm[o:o + n]
        o += n
    return bt


def measure_step(layer, stream, copies, reps=5):
    """(us per step, us per attention launch, plan) for the layer's batch."""
    with torch.cuda.stream(stream):
        plan = layer.step(0, stream)
    torch.cuda.synchronize()
    n = max(copies, 1)
    step_ms = timed_graph(lambda: [layer.step(i, stream) for i in range(n)], stream, reps) / n
    attn_ms = timed_graph(lambda: [layer.attn(i, plan, stream) for i in range(n)], stream, reps) / n
    return step_ms * 1e3, attn_ms * 1e3, plan


def cfg1(stream, gen):
    """The small single request (P = 256, C = 128, 8q/2kv, bf16 KV, 64-page pool): bound by
    launch latency, so reported in microseconds (a fraction of the MFMA peak means nothing here)."""
    rng = np.random.default_rng(1001)
    P, C = np.array([256]), np.array([128])
    layer = Layer(P, C, 8, 2, 64, tables_for(P, C, 64, rng), gen, copies=32)
    us, attn_us, plan = measure_step(layer, stream, 32)
    f = layer.flops()
    return {"workload": "one request, P = 256 cached + C = 128 new, 8q/2kv, bf16 KV, 32 rotating layer copies",
            "us_per_step": round(us, 2), "attn_us": round(attn_us, 2),
            "attn_tflops": round(f / attn_us / 1e6, 2), "work_items": plan.num_items,
            "tile_cols": plan.tile_cols,
            "step": "append, plan, attention, split merge (each layer copy in turn)"}


def cfg2(stream, gen):
    import workloads
    P, C, s = workloads.config2_lengths()
    rng = np.random.default_rng(s)
    layer = Layer(P, C, 32, 8, 4096, tables_for(P, C, 4096, rng), gen, copies=4)
    us, attn_us, plan = measure_step(layer, stream, 4)
    f = layer.flops()
    return {"workload": "8 requests, P ~ U{0..8192}, C = 512, 32q/8kv, bf16 KV, 4 rotating layer copies "
                        "(0.6 GB of visible K/V, over twice the 256 MB last-level cache)",
            "us_per_step": round(us, 2), "attn_us": round(attn_us, 2),
            "step_tflops": round(f / us / 1e6, 1), "attn_tflops": round(f / attn_us / 1e6, 1),
            "attn_pct_mfma_peak": round(100 * f / attn_us / 1e6 / PEAK_BF16_TFLOPS, 1),
            "work_items": plan.num_items, "tile_cols": plan.tile_cols}


def cfg3(stream, gen):
    """64 streaming steps: step s has P = 512 s, C = 512; every step timed on its own."""
    rng = np.random.default_rng(1003)
    per_step, tfl = [], []
    L = 32768
    kfull = (torch.randn((L, 8, 128), generator=gen, device="cuda") * 0.5).to(torch.bfloat16)
    vfull = (torch.randn((L, 8, 128), generator=gen, device="cuda") * 0.5).to(torch.bfloat16)
    q_all = (torch.randn((L, 32, 128), generator=gen, device="cuda") * 0.5).to(torch.bfloat16)
    copies = 32                                  # a 32-layer model's pools: 4 GiB, far past the 256 MB cache
    table = tables_for([0], [L], 2048, rng)
    caches = []
    for _ in range(copies):
        kp = torch.zeros((2048, 8, 16, 128), dtype=torch.bfloat16, device="cuda")
        vp = torch.zeros_like(kp)
        c = s2l.PagedKVCache(kp, vp)
        s2l.s2l_kv_append(c, s2l.Batch([0], [L], table), kfull, vfull)   # the whole stream in the pages
        caches.append(c)
    out = torch.empty((512, 32, 128), dtype=torch.bfloat16, device="cuda")
    lse = torch.empty((512, 32), dtype=torch.float32, device="cuda")
    for s in range(64):
        P = 512 * s
        batch = s2l.Batch([P], [512], table)
        ws = torch.empty(s2l.s2l_attn_workspace_bytes(batch, 32, 8), dtype=torch.uint8, device="cuda")
        kn, vn, q = kfull[P:P + 512].contiguous(), vfull[P:P + 512].contiguous(), q_all[P:P + 512].contiguous()

        def step(i, batch=batch, ws=ws, kn=kn, vn=vn, q=q):
            c = caches[i % copies]
            s2l.s2l_kv_append(c, batch, kn, vn, stream)
            plan = s2l.s2l_attn_plan(batch, 32, 8, ws, None, stream)
            s2l.s2l_attn_main(c, batch, q, 32, SCALE, out, lse, plan, ws, stream)
            s2l.s2l_split_reduce(batch, 32, out, lse, plan, ws, stream)

        us = timed_graph(lambda: [step(i) for i in range(copies)], stream, 3) / copies * 1e3
        f = 4.0 * 128 * 32 * (512 * P + 512 * 513 / 2)
        per_step.append(round(us, 1))
        tfl.append(f / us / 1e6)
    head = [t for s, t in enumerate(tfl) if 512 * s >= 8192]
    return {"workload": "one 32768-token context streamed as 64 chunks of 512 (32q/8kv, bf16 KV); step s: "
                        "P = 512 s; each step = append + plan + attention + merge, 32 rotating layer copies",
            "us_per_step": per_step, "cumulative_ms": round(sum(per_step) / 1e3, 3),
            "mean_step_tflops_p_ge_8192": round(float(np.mean(head)), 1),
            "pct_mfma_peak_p_ge_8192": round(100 * float(np.mean(head)) / PEAK_BF16_TFLOPS, 1),
            "cumulative_tflops": round(8.796e12 / (sum(per_step) * 1e-6) / 1e12, 1)}


def cfg4(stream, gen):
    import workloads
    P, C, rng = workloads.config4_lengths()
    pool = int(((P + C + 15) // 16).sum() * 1.25)
    layer = Layer(P, C, 32, 8, pool, tables_for(P, C, pool, rng), gen)
    us, attn_us, plan = measure_step(layer, stream, 1)
    f, b = layer.flops(), layer.io_bytes()
    t_bound_us = max(f / (PEAK_BF16_TFLOPS * 1e12), b / (PEAK_HBM_GBS * 1e9)) * 1e6
    res = {"workload": "64 requests, P ~ U{0..32768}, C = clip(floor(lognormal(ln 64, 4.118)), 1, 2048), "
                       "32q/8kv, bf16 KV",
           "us_per_step": round(us, 2), "attn_us": round(attn_us, 2), "attn_tflops": round(f / attn_us / 1e6, 1),
           "t_bound_us": round(t_bound_us, 2), "pct_of_t_bound": round(100 * t_bound_us / attn_us, 1),
           "work_items": plan.num_items, "tile_cols": plan.tile_cols, "key_halves": plan.key_halves}
    dec = np.flatnonzero(C == 1)
    del layer
    torch.cuda.empty_cache()
    if len(dec):
        Pd, Cd = P[dec], C[dec]
        poold = int(((Pd + Cd + 15) // 16).sum() + 16)
        d = Layer(Pd, Cd, 32, 8, poold, tables_for(Pd, Cd, poold, rng), gen, copies=4)
        _, dus, dplan = measure_step(d, stream, 4)
        res["decode_subset"] = {"requests": int(len(dec)), "attn_us": round(dus, 2),
                                "kv_gbs": round(d.kv_bytes() / dus / 1e3, 1),
                                "pct_hbm_peak": round(100 * d.kv_bytes() / dus / 1e3 / PEAK_HBM_GBS, 1),
                                "work_items": dplan.num_items, "tile_cols": dplan.tile_cols}
        del d
        torch.cuda.empty_cache()
        res["decode_64x32k"] = decode_64x32k(stream, gen)
    return res


def decode_64x32k(stream, gen, seed=1006):
    """64 decode rows (C = 1) over 32K-token prefixes each, 32q/8kv: a steady decode batch,
    bound by reading its 4.3 GB of K and V (two rotating pool copies)."""
    P64, C64 = np.full(64, 32768, np.int32), np.ones(64, np.int32)
    pool64 = int(((P64 + C64 + 15) // 16).sum() + 16)
    d = Layer(P64, C64, 32, 8, pool64, tables_for(P64, C64, pool64, np.random.default_rng(seed)), gen, copies=2)
    _, dus, dplan = measure_step(d, stream, 2)
    return {"attn_us": round(dus, 2), "kv_gbs": round(d.kv_bytes() / dus / 1e3, 1),
            "pct_hbm_peak": round(100 * d.kv_bytes() / dus / 1e3 / PEAK_HBM_GBS, 1),
            "kv_bytes_per_launch": d.kv_bytes(), "io_bytes_per_launch": d.io_bytes(),
            "work_items": dplan.num_items, "tile_cols": dplan.tile_cols}


def cfg5(stream, gen):
    rng = np.random.default_rng(1005)
    P, C = np.array([131072]), np.array([2048])
    layer = Layer(P, C, 64, 8, 10400, tables_for(P, C, 10400, rng), gen, fp8=True, copies=2)
    us, attn_us, plan = measure_step(layer, stream, 2, reps=3)
    f = layer.flops()
    # the quantised-Q variant on the same layer (Q rows to e4m3, Q K^T on the fp8 MFMA)
    q8_ms = timed_graph(lambda: [s2l.s2l_chunk_prefill_attn_q8(layer.caches[i], layer.batch, layer.q, 64, SCALE,
                                                               layer.out, layer.lse, plan, layer.ws, stream)
                                 for i in range(2)], stream, reps=3) / 2
    return {"workload": "Llama-3-70B layer share: P = 131072, C = 2048, 64q/8kv, fp8 E4M3 KV with per-head "
                        "scales, 2 rotating layer copies",
            "ms_per_step": round(us / 1e3, 3), "attn_ms": round(attn_us / 1e3, 3),
            "attn_tflops": round(f / attn_us / 1e6, 1),
            "attn_pct_mfma_peak": round(100 * f / attn_us / 1e6 / PEAK_BF16_TFLOPS, 1),
            "work_items": plan.num_items, "tile_cols": plan.tile_cols,
            "quantised_q": {"what": "s2l_chunk_prefill_attn_q8: Q rows quantised to e4m3, Q K^T on the fp8 MFMA, "
                                    "P V on bf16 (no split here, so this is the attention launch)",
                            "ms": round(q8_ms, 3), "tflops": round(f / q8_ms / 1e9, 1),
                            "mixed_peak_tflops": round(PEAK_MIXED_Q8_TFLOPS, 1),
                            "pct_mixed_mfma_peak": round(100 * f / q8_ms / 1e9 / PEAK_MIXED_Q8_TFLOPS, 1),
                            "peak_how": "half the FLOPs (Q K^T) at the 5.0 PFLOP/s fp8 peak, half (P V) at "
                                        "the 2.5 PFLOP/s bf16 peak"}}


def scheduler_latency(seed=2024, sizes=(50, 500), calls=2000):
    """Host latency of the scheduler's policy ordering (the sort) and of a whole two-phase
    step with `n` unfinished requests, per policy: median and P99 over `calls` calls.
    Requests come from the synthetic crawler/ANNS streams (all arrived, some chunks in)."""
    from . import sched as S
    from workloads.streams import stream_events
    out = {}
    for n in sizes:
        events = stream_events(seed, n, mode="mixed", rate=1e4, token_scale=0.25, max_tokens=8192)
        horizon = events[len(events) // 2][0]
        for name, pol in S.POLICIES.items():
            s = S.Scheduler(pol, num_gpu_blocks=65536, num_cpu_blocks=65536, token_budget=8192,
                            max_blocks_per_req=512, recompute=([1024.0, 131072.0], [0.02, 2.0]),
                            swap=(0.0005, 0.00004))
            for t, kind, rid, ids, complete in events:
                if t > horizon:
                    break
                getattr(s, "new_stream" if kind == "new" else kind)(rid, ids, complete, t)
            s.step()
            order = np.array([s.priority_order()[1] for _ in range(calls)], dtype=np.float64)
            live = s.stats().num_unfinished
            steps = []
            for _ in range(20):
                steps.append(s.step().step_ns)
            out[f"{name}_n{n}"] = {
                "unfinished": live,
                "order_us_p50": round(float(np.median(order)) / 1e3, 3),
                "order_us_p99": round(float(np.percentile(order, 99)) / 1e3, 3),
                "step_us_p50": round(float(np.median(steps)) / 1e3, 3)}
    out["paper_sort_us_at_50"] = {"FCFS": "15-16", "LCAS": "15-16", "MCPS": "12-13"}
    out["paper_p99_us_at_500"] = "< 165"
    return out


def measured_ceilings(stream=None):
    """HBM read bandwidth of a plain streaming kernel (best of several grid sizes) and the
    bf16 MFMA rate of a register-only loop, both measured here with the library's
    calibration kernels and HIP events."""
    stream = stream or torch.cuda.Stream()
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    buf = torch.ones(1 << 30, dtype=torch.float32, device="cuda")          # 4 GiB
    best = 0.0
    for per_cu in (2, 8, 16):
        sink = torch.empty(cus * per_cu * 256, dtype=torch.int32, device="cuda")
        ms = timed_graph(lambda: s2l.s2l_calib_stream_read(buf, sink, cus * per_cu, stream), stream, reps=5)
        best = max(best, buf.numel() * 4 / ms / 1e6)
    del buf
    sink = torch.empty(cus * 2 * 256, dtype=torch.float32, device="cuda")
    flops = 0

    def loop():
        nonlocal flops
        flops = s2l.s2l_calib_mfma_bf16(20000, sink, cus * 2, stream)

    ms = timed_graph(loop, stream, reps=3)
    torch.cuda.empty_cache()
    return {"hbm_read_gbs": round(best, 1), "mfma_bf16_tflops": round(flops / ms / 1e9, 1),
            "how": "streaming-read kernel over 4 GiB (best of 2, 8, 16 workgroups per CU); "
                   "register-only loop of 32x32x16 bf16 MFMAs, 8 waves per CU"}


def prefix_sweep(stream, gen):
    """The headline step's shape (one request, a 512-token chunk, 32q/8kv, bf16 pages) at prefixes
    from 2K to 128K tokens: per-layer step (append, plan, attention, merge) and attention alone,
    each over enough rotating layer pools to exceed the 256 MB last-level cache."""
    rng = np.random.default_rng(1003)
    out = []
    for P in (2048, 4096, 8192, 16384, 32768, 65536, 131072):
        pages = (P + 512 + 15) // 16
        copies = int(min(32, max(2, math.ceil(512e6 / (pages * 8 * 16 * 128 * 2 * 2)))))
        layer = Layer([P], [512], 32, 8, pages, tables_for([P], [512], pages, rng), gen, copies=copies)
        us, attn_us, plan = measure_step(layer, stream, copies)
        f = layer.flops()
        out.append({"prefix": P, "layer_copies": copies, "us_per_step": round(us, 2), "attn_us": round(attn_us, 2),
                    "attn_tflops": round(f / attn_us / 1e6, 1),
                    "attn_pct_mfma_peak": round(100 * f / attn_us / 1e6 / PEAK_BF16_TFLOPS, 1),
                    "work_items": plan.num_items})
        del layer
        torch.cuda.synchronize()
        torch.cuda.empty_cache()
    return {"workload": "one request, C = 512, 32q/8kv, bf16 KV, P from 2K to 128K", "points": out}


def tp_shares(stream, gen):
    """One GPU's share of a tensor-parallel layer (the kv heads split over the GPUs, each with
    its G query heads; attention needs no exchange): Llama-3-8B at TP = 2 (16q/4kv, bf16, the
    headline step's P = 8192, C = 512) and Llama-3-70B at TP = 8 (8q/1kv, e4m3, config 5's
    P = 131072, C = 2048), each over enough rotating layer pools to exceed the 256 MB cache."""
    rng = np.random.default_rng(1007)
    out = {}
    for name, P, C, hq, hkv, fp8 in (("llama3_8b_tp2", 8192, 512, 16, 4, False),
                                     ("llama3_70b_tp8", 131072, 2048, 8, 1, True)):
        pages = (P + C + 15) // 16
        per_copy = pages * hkv * 16 * 128 * 2 * (1 if fp8 else 2)
        copies = int(min(32, max(2, math.ceil(512e6 / per_copy))))
        layer = Layer([P], [C], hq, hkv, pages, tables_for([P], [C], pages, rng), gen, fp8=fp8, copies=copies)
        us, attn_us, plan = measure_step(layer, stream, copies, reps=3)
        f = layer.flops()
        out[name] = {"prefix": P, "chunk": C, "heads": f"{hq}q/{hkv}kv", "kv": "e4m3" if fp8 else "bf16",
                     "layer_copies": copies, "us_per_step": round(us, 2), "attn_us": round(attn_us, 2),
                     "attn_tflops": round(f / attn_us / 1e6, 1),
                     "attn_pct_mfma_peak": round(100 * f / attn_us / 1e6 / PEAK_BF16_TFLOPS, 1),
                     "work_items": plan.num_items}
        del layer
        torch.cuda.synchronize()
        torch.cuda.empty_cache()
    return out


def all_configs(seed=2024):
    """{config name: result or error string}; each config is measured independently."""
    stream = torch.cuda.Stream()
    res = {}
    for name, fn in (("config1", cfg1), ("config2", cfg2), ("config3", cfg3), ("config4", cfg4), ("config5", cfg5),
                     ("prefix_sweep", prefix_sweep), ("tp_shares", tp_shares)):
        gen = torch.Generator(device="cuda")
        gen.manual_seed(seed)
        try:
            res[name] = fn(stream, gen)
        except Exception as e:   # reported in the JSON line instead of failing the whole run
            res[name] = {"error": f"{type(e).__name__}: {e}"}
        torch.cuda.synchronize()
        torch.cuda.empty_cache()
    try:
        from . import costmodel
        swap = costmodel.measure_swap()
        rec = costmodel.measure_recompute(token_counts=(1024, 16384, 131072))
        res["cost_model"] = {
            "swap_kernel_gbs": {"out": round(swap["kernel_out_gbs"], 1), "in": round(swap["kernel_in_gbs"], 1)},
            "memcpy_gbs": {"d2h": round(swap["memcpy_d2h_gbs"], 1), "h2d": round(swap["memcpy_h2d_gbs"], 1)},
            "swap_fit_round_trip_s": swap["fit_round_trip_s"],
            "compare": costmodel.crossover(swap, rec)}
    except Exception as e:
        res["cost_model"] = {"error": f"{type(e).__name__}: {e}"}
    try:
        res["scheduler"] = scheduler_latency(seed)
    except Exception as e:
        res["scheduler"] = {"error": f"{type(e).__name__}: {e}"}
    return res


if __name__ == "__main__":
    # one named workload on its own (for profiling): python -m paper_2604_16395_amd.benchcfg decode_64x32k
    import json
    import sys
    g = torch.Generator(device="cuda")
    g.manual_seed(2024)
    fn = {"decode_64x32k": decode_64x32k, "config1": cfg1, "config2": cfg2, "config4": cfg4, "config5": cfg5,
          "prefix_sweep": prefix_sweep, "tp_shares": tp_shares}[sys.argv[1]]
    print(json.dumps(fn(torch.cuda.Stream(), g)), flush=True)
