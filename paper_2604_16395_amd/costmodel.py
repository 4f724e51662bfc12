"""Offline profile of the two preemption costs on this GPU (Stream2LLM Sec. 4.3), and the
scheduler cost model fitted to it.

* swap_latency(C): time to move C KV blocks to pinned host memory and back with the
  library's page-copy kernels (one launch per layer and direction).  A block is 16 tokens
  of every layer: for Llama-3.1-8B (32 layers, 8 kv heads, d = 128, bf16) 2 MiB, the
  block size the paper quotes.  Fitted as fixed + per_block * C (least squares).
* recomputation_latency(T): time to prefill T tokens from scratch.  The attention part is
  the library (append, plan, attention, split merge: one layer, times the layer count);
  the rest of a layer (QKV, output and MLP projections) is timed as plain bf16 GEMMs of
  the model's shapes, outside this library, only to give the model its full cost.  Used
  as a piecewise-linear model over the measured token counts.

Usage:  python -m paper_2604_16395_amd.costmodel --out cost_model.json
        recompute, swap = costmodel.load("cost_model.json")  # -> sched.Scheduler(...)

``cost_model_mi355x.json`` beside this file is such a profile, taken on an MI355X
(``load()`` with no argument reads it).
"""
import argparse
import json
import math
import os

import numpy as np
import torch

import paper_2604_16395_amd as s2l
from . import benchcfg

LLAMA3_8B = {"layers": 32, "hidden": 4096, "q_heads": 32, "kv_heads": 8, "head_dim": 128, "mlp": 14336}


def _events_ms(fn, stream, reps):
    ts = []
    for _ in range(reps):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        with torch.cuda.stream(stream):
            a.record(stream)
            fn()
            b.record(stream)
        torch.cuda.synchronize()
        ts.append(a.elapsed_time(b))
    return float(np.median(ts))


def measure_swap(block_counts=(1, 8, 64, 512), model=LLAMA3_8B, reps=5, dev="cuda"):
    L, hkv = model["layers"], model["kv_heads"]
    nmax = max(block_counts)
    stream = torch.cuda.Stream()
    shape = (nmax, hkv, 16, 128)
    dev_pools = [(torch.randn(shape, device=dev).to(torch.bfloat16), torch.randn(shape, device=dev).to(torch.bfloat16))
                 for _ in range(L)]
    host_pools = [(torch.empty(shape, dtype=torch.bfloat16).pin_memory(),
                   torch.empty(shape, dtype=torch.bfloat16).pin_memory()) for _ in range(L)]
    caches = [s2l.PagedKVCache(k, v) for k, v in dev_pools]
    rng = np.random.default_rng(0)
    res = {"blocks": [], "out_ms": [], "in_ms": [], "block_bytes": L * 2 * hkv * 16 * 128 * 2}
    for c in block_counts:
        gpu = rng.permutation(nmax)[:c]
        host = rng.permutation(nmax)[:c]
        out_pairs = torch.from_numpy(np.stack([gpu, host], 1).astype(np.int32)).to(dev)
        in_pairs = torch.from_numpy(np.stack([host, gpu], 1).astype(np.int32)).to(dev)

        def out_all():
            for cache, (hk, hv) in zip(caches, host_pools):
                s2l.s2l_kv_swap_out(cache, out_pairs, hk, hv, stream)

        def in_all():
            for cache, (hk, hv) in zip(caches, host_pools):
                s2l.s2l_kv_swap_in(cache, in_pairs, hk, hv, stream)

        out_all(), in_all()
        torch.cuda.synchronize()
        res["blocks"].append(int(c))
        res["out_ms"].append(_events_ms(out_all, stream, reps))
        res["in_ms"].append(_events_ms(in_all, stream, reps))
    # the copy engine on one contiguous buffer of the largest size, for reference
    nbytes = nmax * res["block_bytes"]
    src = torch.empty(nbytes, dtype=torch.uint8, device=dev)
    dst = torch.empty(nbytes, dtype=torch.uint8).pin_memory()
    d2h = _events_ms(lambda: dst.copy_(src, non_blocking=True), stream, reps)
    h2d = _events_ms(lambda: src.copy_(dst, non_blocking=True), stream, reps)
    res["memcpy_d2h_gbs"] = nbytes / d2h / 1e6
    res["memcpy_h2d_gbs"] = nbytes / h2d / 1e6
    big = res["blocks"].index(nmax)
    res["kernel_out_gbs"] = nbytes / res["out_ms"][big] / 1e6
    res["kernel_in_gbs"] = nbytes / res["in_ms"][big] / 1e6
    x = np.asarray(res["blocks"], np.float64)
    y = (np.asarray(res["out_ms"]) + np.asarray(res["in_ms"])) / 1e3
    A = np.stack([np.ones_like(x), x], 1)
    fixed, per = np.linalg.lstsq(A, y, rcond=None)[0]
    res["fit_round_trip_s"] = {"fixed": float(max(fixed, 0.0)), "per_block": float(per)}
    del dev_pools, host_pools, caches, src, dst
    torch.cuda.empty_cache()
    return res


def measure_recompute(token_counts=(1024, 4096, 16384, 65536, 131072), model=LLAMA3_8B, reps=3, dev="cuda"):
    L, H, hq, hkv, F = model["layers"], model["hidden"], model["q_heads"], model["kv_heads"], model["mlp"]
    stream = torch.cuda.Stream()
    gen = torch.Generator(device=dev)
    gen.manual_seed(1)
    res = {"tokens": [], "attention_ms": [], "linear_ms": [], "total_ms": []}
    for T in token_counts:
        pages = (T + 15) // 16
        layer = benchcfg.Layer([0], [T], hq, hkv, pages, np.arange(pages, dtype=np.int32)[None, :], gen)
        step_us, _, _ = benchcfg.measure_step(layer, stream, 1, reps)
        del layer
        x = torch.randn((T, H), device=dev).to(torch.bfloat16)
        w_qkv = torch.randn((H, (hq + 2 * hkv) * 128), device=dev).to(torch.bfloat16)
        w_o = torch.randn((hq * 128, H), device=dev).to(torch.bfloat16)
        w_up = torch.randn((H, 2 * F), device=dev).to(torch.bfloat16)
        w_down = torch.randn((F, H), device=dev).to(torch.bfloat16)

        def linear():
            torch.matmul(x, w_qkv)
            torch.matmul(x, w_o)
            h = torch.matmul(x, w_up)
            torch.matmul(h[:, :F], w_down)

        with torch.cuda.stream(stream):
            linear()
        torch.cuda.synchronize()
        lin_ms = _events_ms(linear, stream, reps)
        del x, w_qkv, w_o, w_up, w_down
        torch.cuda.empty_cache()
        res["tokens"].append(int(T))
        res["attention_ms"].append(step_us / 1e3 * L)
        res["linear_ms"].append(lin_ms * L)
        res["total_ms"].append(step_us / 1e3 * L + lin_ms * L)
    return res


def crossover(swap, rec):
    """Per measured T: predicted round-trip swap of ceil(T/16) blocks against recomputing T."""
    fit = swap["fit_round_trip_s"]
    rows = []
    for T, tot, att in zip(rec["tokens"], rec["total_ms"], rec["attention_ms"]):
        sw = (fit["fixed"] + fit["per_block"] * math.ceil(T / 16)) * 1e3
        rows.append({"tokens": T, "swap_ms": round(sw, 3), "recompute_ms": round(tot, 3),
                     "recompute_attention_only_ms": round(att, 3),
                     "cheaper": "swap" if sw < tot else "recompute"})
    return rows


def profile(block_counts=(1, 8, 64, 512), token_counts=(1024, 4096, 16384, 65536, 131072)):
    swap = measure_swap(block_counts)
    rec = measure_recompute(token_counts)
    return {"device": torch.cuda.get_device_name(0), "model": "Llama-3.1-8B shapes " + json.dumps(LLAMA3_8B),
            "swap": swap, "recompute": rec, "compare": crossover(swap, rec)}


DEFAULT_PROFILE = os.path.join(os.path.dirname(os.path.abspath(__file__)), "cost_model_mi355x.json")


def load(path=DEFAULT_PROFILE):
    """(recompute, swap) arguments of sched.Scheduler from a saved profile."""
    d = json.load(open(path))
    rec = (list(map(float, d["recompute"]["tokens"])), [t / 1e3 for t in d["recompute"]["total_ms"]])
    fit = d["swap"]["fit_round_trip_s"]
    return rec, (fit["fixed"], fit["per_block"])


if __name__ == "__main__":
    ap = argparse.ArgumentParser()
    ap.add_argument("--out", required=True)
    args = ap.parse_args()
    prof = profile()
    with open(args.out, "w") as f:
        json.dump(prof, f, indent=1)
    print(json.dumps(prof["compare"]))
