"""ctypes declarations of the C ABI in include/s2l.h and include/s2l_sched.h, and the
loader of libs2l.so.

Loading fails loudly (S2LLibraryMissing) when the built library is absent: there is no
fallback implementation of any entry point.
"""
import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
# S2L_LIBRARY selects another build of the same library (the host-sanitizer build of
# `python -m paper_2604_16395_amd.build --sanitize`); by default the in-tree libs2l.so.
LIB_PATH = os.environ.get("S2L_LIBRARY") or os.path.join(_HERE, "libs2l.so")

S2L_OK, S2L_EINVAL, S2L_ERANGE, S2L_EWORKSPACE, S2L_ENOTSUP, S2L_EHIP = 0, -1, -2, -3, -4, -5
S2L_KV_BF16, S2L_KV_FP8_E4M3 = 0, 1
STATUS_NAMES = {0: "S2L_OK", -1: "S2L_EINVAL", -2: "S2L_ERANGE", -3: "S2L_EWORKSPACE",
                -4: "S2L_ENOTSUP", -5: "S2L_EHIP"}

c_i32 = ctypes.c_int32
c_i64 = ctypes.c_int64
c_vp = ctypes.c_void_p
P_i32 = ctypes.POINTER(ctypes.c_int32)


class s2l_kv_cache(ctypes.Structure):
    _fields_ = [("k_pages", c_vp), ("v_pages", c_vp), ("k_scale", c_vp), ("v_scale", c_vp),
                ("num_pages", c_i32), ("num_kv_heads", c_i32), ("head_dim", c_i32),
                ("page_size", c_i32), ("dtype", c_i32), ("reserved", c_i32)]


class s2l_batch(ctypes.Structure):
    _fields_ = [("num_reqs", c_i32), ("max_pages_per_req", c_i32), ("prefix_lens", c_vp),
                ("chunk_lens", c_vp), ("cu_chunk", c_vp), ("block_tables", c_vp),
                ("prefix_lens_host", P_i32), ("chunk_lens_host", P_i32)]


class s2l_plan_opts(ctypes.Structure):
    _fields_ = [("target_items", c_i32), ("min_split_keys", c_i32), ("max_splits", c_i32),
                ("tile_cols", c_i32), ("key_halves", c_i32)]


class s2l_plan_info(ctypes.Structure):
    _fields_ = [("num_items", c_i32), ("num_split_reqs", c_i32), ("split_keys", c_i32),
                ("num_q_heads", c_i32), ("num_kv_heads", c_i32), ("num_reqs", c_i32),
                ("total_tokens", c_i64), ("workspace_bytes", c_i64), ("tile_cols", c_i32),
                ("num_tiles", c_i32), ("part_floats", c_i64), ("key_halves", c_i32), ("flags", c_i32)]


class s2l_sched_config(ctypes.Structure):
    _fields_ = [("policy", c_i32), ("num_gpu_blocks", c_i32), ("num_cpu_blocks", c_i32),
                ("token_budget", c_i32), ("max_blocks_per_req", c_i32), ("table_pad", c_i32),
                ("num_recompute_points", c_i32), ("reserved", c_i32),
                ("recompute_tokens", ctypes.POINTER(ctypes.c_double)),
                ("recompute_seconds", ctypes.POINTER(ctypes.c_double)),
                ("swap_fixed_seconds", ctypes.c_double), ("swap_seconds_per_block", ctypes.c_double)]


class s2l_sched_step_out(ctypes.Structure):
    _fields_ = [("req_ids", c_vp), ("prefix_lens", c_vp), ("chunk_lens", c_vp), ("block_tables", c_vp),
                ("event_ids", c_vp), ("event_kinds", c_vp), ("swap_out", c_vp), ("swap_in", c_vp),
                ("cap_reqs", c_i32), ("cap_swap", c_i32), ("num_reqs", c_i32), ("num_events", c_i32),
                ("num_swap_out", c_i32), ("num_swap_in", c_i32), ("total_tokens", c_i32),
                ("reserved", c_i32), ("order_ns", c_i64), ("step_ns", c_i64)]


class s2l_sched_req_info(ctypes.Structure):
    _fields_ = [("state", c_i32), ("num_tokens", c_i32), ("num_computed_tokens", c_i32),
                ("input_complete", c_i32), ("total_tokens_invalidated", c_i64),
                ("num_preempt_swap", c_i32), ("num_preempt_recompute", c_i32),
                ("num_gpu_blocks", c_i32), ("num_cpu_blocks", c_i32),
                ("arrival_time", ctypes.c_double), ("last_chunk_arrival_time", ctypes.c_double)]


class s2l_sched_stats(ctypes.Structure):
    _fields_ = [("num_unfinished", c_i32), ("free_gpu_blocks", c_i32), ("free_cpu_blocks", c_i32),
                ("reserved", c_i32)]


P_cache = ctypes.POINTER(s2l_kv_cache)
P_batch = ctypes.POINTER(s2l_batch)
P_opts = ctypes.POINTER(s2l_plan_opts)
P_info = ctypes.POINTER(s2l_plan_info)

# name -> (restype, argtypes); the list of every symbol include/s2l.h declares
SIGNATURES = {
    "s2l_abi_version": (c_i32, []),
    "s2l_last_error": (ctypes.c_char_p, []),
    "s2l_kv_append": (c_i32, [P_cache, P_batch, c_vp, c_vp, c_vp]),
    "s2l_kv_gather": (c_i32, [P_cache, P_batch, c_i32, c_vp, c_vp, c_vp, c_vp]),
    "s2l_check_tables": (c_i32, [P_cache, P_batch, c_vp, c_vp]),
    "s2l_kv_swap_out": (c_i32, [P_cache, c_vp, c_i32, c_vp, c_vp, c_i32, c_vp]),
    "s2l_kv_swap_in": (c_i32, [P_cache, c_vp, c_i32, c_vp, c_vp, c_i32, c_vp]),
    "s2l_attn_workspace_bytes": (c_i32, [P_batch, c_i32, c_i32, P_opts, ctypes.POINTER(ctypes.c_size_t)]),
    "s2l_attn_plan": (c_i32, [P_batch, c_i32, c_i32, P_opts, c_vp, ctypes.c_size_t, P_info, c_vp]),
    "s2l_chunk_prefill_attn": (c_i32, [P_cache, P_batch, c_vp, c_i32, ctypes.c_float, c_vp, c_vp, P_info,
                                       c_vp, ctypes.c_size_t, c_vp]),
    "s2l_chunk_prefill_attn_q8": (c_i32, [P_cache, P_batch, c_vp, c_i32, ctypes.c_float, c_vp, c_vp, P_info,
                                       c_vp, ctypes.c_size_t, c_vp]),
    "s2l_append_chunk_prefill_attn": (c_i32, [P_cache, P_batch, c_vp, c_vp, c_vp, c_i32, ctypes.c_float, c_vp,
                                              c_vp, P_info, c_vp, ctypes.c_size_t, P_i32, c_vp]),
    "s2l_chunk_prefill_attn_noalloc": (c_i32, [P_cache, P_batch, c_vp, c_i32, ctypes.c_float, c_vp, c_vp, P_opts,
                                               P_info, c_vp]),
    "s2l_attn_main": (c_i32, [P_cache, P_batch, c_vp, c_i32, ctypes.c_float, c_vp, c_vp, P_info,
                              c_vp, ctypes.c_size_t, c_vp]),
    "s2l_split_reduce": (c_i32, [P_batch, c_i32, c_vp, c_vp, P_info, c_vp, ctypes.c_size_t, c_vp]),
    "s2l_plan_host": (c_i32, [c_i32, P_i32, P_i32, c_i32, c_i32, P_opts, c_i32, P_info, P_i32, c_i64]),
    "s2l_calib_stream_read": (c_i32, [c_vp, ctypes.c_size_t, c_vp, c_i32, c_vp]),
    "s2l_calib_mfma_bf16": (c_i32, [c_i64, c_vp, c_i32, ctypes.POINTER(c_i64), c_vp]),
    # include/s2l_sched.h
    "s2l_lcp_len": (c_i32, [P_i32, c_i32, P_i32, c_i32]),
    "s2l_sched_create": (c_i32, [ctypes.POINTER(s2l_sched_config), ctypes.POINTER(c_vp)]),
    "s2l_sched_destroy": (None, [c_vp]),
    "s2l_sched_new_stream": (c_i32, [c_vp, c_i64, P_i32, c_i32, c_i32, ctypes.c_double]),
    "s2l_sched_append": (c_i32, [c_vp, c_i64, P_i32, c_i32, c_i32, ctypes.c_double]),
    "s2l_sched_update": (c_i32, [c_vp, c_i64, P_i32, c_i32, c_i32, ctypes.c_double, P_i32]),
    "s2l_sched_step": (c_i32, [c_vp, ctypes.POINTER(s2l_sched_step_out)]),
    "s2l_sched_priority_order": (c_i32, [c_vp, ctypes.POINTER(c_i64), c_i32, P_i32, ctypes.POINTER(c_i64)]),
    "s2l_sched_request": (c_i32, [c_vp, c_i64, ctypes.POINTER(s2l_sched_req_info), P_i32, P_i32]),
    "s2l_sched_stats_get": (c_i32, [c_vp, ctypes.POINTER(s2l_sched_stats)]),
}


class S2LLibraryMissing(ImportError):
    pass


class S2LError(RuntimeError):
    def __init__(self, fn, status, message):
        super().__init__(f"{fn} failed: {STATUS_NAMES.get(status, status)}: {message}")
        self.status = status
        self.message = message


_lib = None


def lib():
    """The loaded libs2l.so (raises S2LLibraryMissing if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise S2LLibraryMissing(
                f"{LIB_PATH} is missing: build it with `python -m paper_2604_16395_amd.build`")
        handle = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in SIGNATURES.items():
            f = getattr(handle, name)
            f.restype = res
            f.argtypes = args
        _lib = handle
    return _lib


def call(name, *args):
    """Call an entry point; raise S2LError on a negative status."""
    st = getattr(lib(), name)(*args)
    if st != S2L_OK:
        raise S2LError(name, st, lib().s2l_last_error().decode())
    return st
