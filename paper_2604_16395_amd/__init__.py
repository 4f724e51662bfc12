"""Incremental chunked-prefill attention over a paged KV cache, for AMD MI355X (gfx950).

Python binding of the C ABI in ``include/s2l.h`` (libs2l.so, built from ``csrc/``).  The
functions below carry the C names and only marshal arguments: torch tensors supply device
memory and streams, every step of the computation runs in the library's HIP kernels.

Typical step for one layer (Stream2LLM append mode: a chunk of C tokens arrives for a
request that already holds P cached tokens)::

    batch = Batch(prefix_lens, chunk_lens, block_tables)       # P_r, C_r, page ids
    s2l_kv_append(cache, batch, k_new, v_new)                  # pages <- chunk K/V
    ws = torch.empty(s2l_attn_workspace_bytes(batch, Hq, Hkv), dtype=torch.uint8, device="cuda")
    plan = s2l_attn_plan(batch, Hq, Hkv, ws)                   # once per step, all layers
    s2l_chunk_prefill_attn(cache, batch, q, Hq, 128 ** -0.5, out, lse, plan, ws)
"""
import ctypes

import numpy as np
import torch

from . import _lib
from ._lib import (S2L_KV_BF16, S2L_KV_FP8_E4M3, S2LError, S2LLibraryMissing, s2l_plan_info,
                   s2l_plan_opts)

__all__ = ["PagedKVCache", "Batch", "plan_opts", "S2LError", "S2LLibraryMissing",
           "s2l_abi_version", "s2l_kv_append", "s2l_kv_gather", "s2l_kv_swap_out", "s2l_kv_swap_in",
           "s2l_check_tables", "s2l_append_chunk_prefill_attn", "s2l_calib_stream_read", "s2l_calib_mfma_bf16", "s2l_attn_workspace_bytes",
           "s2l_attn_plan", "s2l_chunk_prefill_attn", "s2l_chunk_prefill_attn_q8", "s2l_attn_main", "s2l_split_reduce",
           "s2l_plan_host", "library_path", "plan_status", "s2l_chunk_prefill_attn_noalloc"]

HEAD_DIM = 128
PAGE_SIZE = 16


def library_path():
    return _lib.LIB_PATH


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream):
    if stream is None:
        stream = torch.cuda.current_stream()
    if isinstance(stream, torch.cuda.Stream):
        stream = stream.cuda_stream
    return ctypes.c_void_p(int(stream))


def _check(t, dtype, name):
    if t is None:
        return
    if t.dtype != dtype or not t.is_contiguous():
        raise ValueError(f"{name} must be a contiguous {dtype} tensor (got {t.dtype}, "
                         f"contiguous={t.is_contiguous()})")


class PagedKVCache:
    """One layer's K and V page pools, each [num_pages][Hkv][16][128] (bf16, or uint8 E4M3)."""

    def __init__(self, k_pages, v_pages, k_scale=None, v_scale=None):
        fp8 = k_pages.dtype == torch.uint8
        _check(k_pages, torch.uint8 if fp8 else torch.bfloat16, "k_pages")
        _check(v_pages, k_pages.dtype, "v_pages")
        if fp8:
            _check(k_scale, torch.float32, "k_scale")
            _check(v_scale, torch.float32, "v_scale")
        self.k_pages, self.v_pages = k_pages, v_pages
        self.k_scale, self.v_scale = k_scale, v_scale
        self.fp8 = fp8

    @property
    def num_pages(self):
        return self.k_pages.shape[0]

    @property
    def num_kv_heads(self):
        return self.k_pages.shape[1]

    def c(self):
        return _lib.s2l_kv_cache(
            k_pages=self.k_pages.data_ptr(), v_pages=self.v_pages.data_ptr(),
            k_scale=self.k_scale.data_ptr() if self.fp8 else None,
            v_scale=self.v_scale.data_ptr() if self.fp8 else None,
            num_pages=self.k_pages.shape[0], num_kv_heads=self.k_pages.shape[1],
            head_dim=self.k_pages.shape[3], page_size=self.k_pages.shape[2],
            dtype=S2L_KV_FP8_E4M3 if self.fp8 else S2L_KV_BF16)


class Batch:
    """A step's varlen batch: device length/table arrays plus the host length copies."""

    def __init__(self, prefix_lens, chunk_lens, block_tables, device="cuda"):
        self.prefix_host = np.ascontiguousarray(prefix_lens, dtype=np.int32)
        self.chunk_host = np.ascontiguousarray(chunk_lens, dtype=np.int32)
        cu = np.zeros(len(self.chunk_host) + 1, dtype=np.int32)
        cu[1:] = np.cumsum(self.chunk_host)
        self.cu_host = cu
        bt = np.ascontiguousarray(block_tables, dtype=np.int32)
        if bt.ndim == 1:
            bt = bt.reshape(len(self.prefix_host), -1)
        self.tables_host = bt
        self.prefix_lens = torch.from_numpy(self.prefix_host).to(device)
        self.chunk_lens = torch.from_numpy(self.chunk_host).to(device)
        self.cu_chunk = torch.from_numpy(cu).to(device)
        self.block_tables = torch.from_numpy(bt).to(device)

    @property
    def num_reqs(self):
        return len(self.prefix_host)

    @property
    def total_tokens(self):
        return int(self.cu_host[-1])

    def c(self):
        return _lib.s2l_batch(
            num_reqs=self.num_reqs, max_pages_per_req=self.tables_host.shape[1],
            prefix_lens=self.prefix_lens.data_ptr(), chunk_lens=self.chunk_lens.data_ptr(),
            cu_chunk=self.cu_chunk.data_ptr(), block_tables=self.block_tables.data_ptr(),
            prefix_lens_host=self.prefix_host.ctypes.data_as(_lib.P_i32),
            chunk_lens_host=self.chunk_host.ctypes.data_as(_lib.P_i32))


def plan_opts(target_items=0, min_split_keys=0, max_splits=0, tile_cols=0, key_halves=0):
    return s2l_plan_opts(target_items=target_items, min_split_keys=min_split_keys,
                         max_splits=max_splits, tile_cols=tile_cols, key_halves=key_halves)


def _opts_ptr(opts):
    return None if opts is None else ctypes.byref(opts)


def s2l_abi_version():
    return _lib.lib().s2l_abi_version()


def s2l_kv_append(cache, batch, k_new, v_new, stream=None):
    _check(k_new, torch.bfloat16, "k_new")
    _check(v_new, torch.bfloat16, "v_new")
    cc, bc = cache.c(), batch.c()
    _lib.call("s2l_kv_append", ctypes.byref(cc), ctypes.byref(bc), _ptr(k_new), _ptr(v_new), _stream(stream))


def _swap(name, cache, pairs, host_k, host_v, stream):
    _check(pairs, torch.int32, "pairs")
    if pairs.dim() != 2 or pairs.shape[1] != 2 or not pairs.is_cuda:
        raise ValueError("pairs must be a device int32 tensor [n][2]")
    if host_k.is_cuda or host_v.is_cuda or host_k.dtype != cache.k_pages.dtype or host_v.dtype != host_k.dtype:
        raise ValueError("host pools must be host tensors of the cache's element type")
    if not (host_k.is_contiguous() and host_v.is_contiguous()) or host_k.shape != host_v.shape:
        raise ValueError("host pools must be contiguous and of one shape")
    cc = cache.c()
    _lib.call(name, ctypes.byref(cc), _ptr(pairs), pairs.shape[0], _ptr(host_k), _ptr(host_v),
              host_k.shape[0], _stream(stream))


def s2l_kv_swap_out(cache, pairs, host_k, host_v, stream=None):
    """Device pages pairs[i][0] -> pinned host pages pairs[i][1] (K and V)."""
    _swap("s2l_kv_swap_out", cache, pairs, host_k, host_v, stream)


def s2l_kv_swap_in(cache, pairs, host_k, host_v, stream=None):
    """Pinned host pages pairs[i][0] -> device pages pairs[i][1] (K and V)."""
    _swap("s2l_kv_swap_in", cache, pairs, host_k, host_v, stream)


def s2l_check_tables(cache, batch, counts, stream=None):
    """Count used block-table entries outside the pool into the device int32[2] `counts`."""
    _check(counts, torch.int32, "counts")
    cc, bc = cache.c(), batch.c()
    _lib.call("s2l_check_tables", ctypes.byref(cc), ctypes.byref(bc), _ptr(counts), _stream(stream))


def s2l_calib_stream_read(buf, sink, grid, stream=None):
    """One streaming read of the device tensor `buf` (measurement support)."""
    _lib.call("s2l_calib_stream_read", _ptr(buf), buf.numel() * buf.element_size(), _ptr(sink), int(grid),
              _stream(stream))


def s2l_calib_mfma_bf16(iters, sink, grid, stream=None):
    """A register-only bf16 MFMA loop (measurement support); returns its flop count."""
    flops = ctypes.c_int64()
    _lib.call("s2l_calib_mfma_bf16", int(iters), _ptr(sink), int(grid), ctypes.byref(flops), _stream(stream))
    return flops.value


def s2l_kv_gather(cache, batch, include_chunk, cu_out, k_out, v_out, stream=None):
    _check(cu_out, torch.int32, "cu_out")
    cc, bc = cache.c(), batch.c()
    _lib.call("s2l_kv_gather", ctypes.byref(cc), ctypes.byref(bc), int(include_chunk), _ptr(cu_out),
              _ptr(k_out), _ptr(v_out), _stream(stream))


def s2l_attn_workspace_bytes(batch, num_q_heads, num_kv_heads, opts=None):
    bc = batch.c()
    n = ctypes.c_size_t(0)
    _lib.call("s2l_attn_workspace_bytes", ctypes.byref(bc), num_q_heads, num_kv_heads, _opts_ptr(opts),
              ctypes.byref(n))
    return n.value


def s2l_attn_plan(batch, num_q_heads, num_kv_heads, workspace, opts=None, stream=None):
    _check(workspace, torch.uint8, "workspace")
    bc = batch.c()
    info = s2l_plan_info()
    _lib.call("s2l_attn_plan", ctypes.byref(bc), num_q_heads, num_kv_heads, _opts_ptr(opts),
              _ptr(workspace), workspace.numel(), ctypes.byref(info), _stream(stream))
    return info


PLAN_STATUS_OFFSET = 36      # S2L_PLAN_STATUS_OFFSET of include/s2l.h


def plan_status(workspace):
    """The plan's int32 status word in `workspace` (a device uint8 tensor that s2l_attn_plan
    filled), as a 0-dim device tensor: 0 = planned, 1 = the device length arrays needed more
    than the host copies planned for (the attention calls then write NaN and compute
    nothing).  Read it after the stream has passed the plan."""
    _check(workspace, torch.uint8, "workspace")
    return workspace[PLAN_STATUS_OFFSET:PLAN_STATUS_OFFSET + 4].view(torch.int32)[0]


def _attn(name, cache, batch, q, num_q_heads, softmax_scale, out, lse, plan, workspace, stream):
    _check(q, torch.bfloat16, "q")
    _check(out, torch.bfloat16, "out")
    _check(lse, torch.float32, "lse")
    _check(workspace, torch.uint8, "workspace")
    cc, bc = cache.c(), batch.c()
    _lib.call(name, ctypes.byref(cc), ctypes.byref(bc), _ptr(q), num_q_heads, float(softmax_scale),
              _ptr(out), _ptr(lse), ctypes.byref(plan), _ptr(workspace), workspace.numel(), _stream(stream))


def s2l_chunk_prefill_attn(cache, batch, q, num_q_heads, softmax_scale, out, lse, plan, workspace,
                           stream=None):
    _attn("s2l_chunk_prefill_attn", cache, batch, q, num_q_heads, softmax_scale, out, lse, plan,
          workspace, stream)


def s2l_chunk_prefill_attn_q8(cache, batch, q, num_q_heads, softmax_scale, out, lse, plan, workspace,
                              stream=None):
    """s2l_chunk_prefill_attn with Q quantised to e4m3 per (token, head) row and Q K^T on the
    fp8 MFMA (e4m3 caches only)."""
    _attn("s2l_chunk_prefill_attn_q8", cache, batch, q, num_q_heads, softmax_scale, out, lse, plan,
          workspace, stream)


def s2l_append_chunk_prefill_attn(cache, batch, k_new, v_new, q, num_q_heads, softmax_scale, out, lse, plan,
                                  workspace, stream=None):
    """s2l_kv_append + s2l_chunk_prefill_attn, in one attention launch where possible;
    returns True when the single launch was used."""
    for t, n in ((k_new, "k_new"), (v_new, "v_new"), (q, "q"), (out, "out")):
        _check(t, torch.bfloat16, n)
    _check(lse, torch.float32, "lse")
    _check(workspace, torch.uint8, "workspace")
    cc, bc = cache.c(), batch.c()
    fused = ctypes.c_int32()
    _lib.call("s2l_append_chunk_prefill_attn", ctypes.byref(cc), ctypes.byref(bc), _ptr(k_new), _ptr(v_new),
              _ptr(q), num_q_heads, float(softmax_scale), _ptr(out), _ptr(lse), ctypes.byref(plan),
              _ptr(workspace), workspace.numel(), ctypes.byref(fused), _stream(stream))
    return bool(fused.value)


NOALLOC_SCRATCH_BYTES = 64 << 20     # S2L_NOALLOC_SCRATCH_BYTES of include/s2l.h


def s2l_chunk_prefill_attn_noalloc(cache, batch, q, num_q_heads, softmax_scale, out, lse, opts=None, stream=None):
    """Plan + attention + merge with the library's own scratch (no workspace, no allocation);
    returns the plan's s2l_plan_info.  Calls overlapping on one GPU race (shared scratch)."""
    _check(q, torch.bfloat16, "q")
    _check(out, torch.bfloat16, "out")
    _check(lse, torch.float32, "lse")
    info = s2l_plan_info()
    cc, bc = cache.c(), batch.c()
    _lib.call("s2l_chunk_prefill_attn_noalloc", ctypes.byref(cc), ctypes.byref(bc), _ptr(q), num_q_heads,
              float(softmax_scale), _ptr(out), _ptr(lse), _opts_ptr(opts), ctypes.byref(info), _stream(stream))
    return info


def s2l_attn_main(cache, batch, q, num_q_heads, softmax_scale, out, lse, plan, workspace, stream=None):
    _attn("s2l_attn_main", cache, batch, q, num_q_heads, softmax_scale, out, lse, plan, workspace, stream)


def s2l_split_reduce(batch, num_q_heads, out, lse, plan, workspace, stream=None):
    _check(out, torch.bfloat16, "out")
    _check(lse, torch.float32, "lse")
    bc = batch.c()
    _lib.call("s2l_split_reduce", ctypes.byref(bc), num_q_heads, _ptr(out), _ptr(lse), ctypes.byref(plan),
              _ptr(workspace), workspace.numel(), _stream(stream))


def s2l_plan_host(prefix_lens, chunk_lens, num_q_heads, num_kv_heads, opts=None, num_cus=256,
                  with_items=False):
    """Host-only partition: returns (s2l_plan_info, items [num_items][8] int32 or None)."""
    P = np.ascontiguousarray(prefix_lens, dtype=np.int32)
    C = np.ascontiguousarray(chunk_lens, dtype=np.int32)
    info = s2l_plan_info()
    _lib.call("s2l_plan_host", len(P), P.ctypes.data_as(_lib.P_i32), C.ctypes.data_as(_lib.P_i32),
              num_q_heads, num_kv_heads, _opts_ptr(opts), num_cus, ctypes.byref(info), None, 0)
    if not with_items:
        return info, None
    items = np.zeros((max(info.num_items, 1), 8), dtype=np.int32)
    _lib.call("s2l_plan_host", len(P), P.ctypes.data_as(_lib.P_i32), C.ctypes.data_as(_lib.P_i32),
              num_q_heads, num_kv_heads, _opts_ptr(opts), num_cus, ctypes.byref(info),
              items.ctypes.data_as(_lib.P_i32), info.num_items)
    return info, items[:info.num_items]
