"""C-ABI checks that need no GPU: the library loads, exports every symbol the header
declares, and rejects bad arguments with the documented status before launching anything.

Every call here fails host-side validation, so no kernel is ever enqueued (the device
pointers below are placeholders that are never dereferenced).
"""
import ctypes
import glob
import os
import re

import numpy as np
import pytest

from paper_2604_16395_amd import _lib

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
FAKE = 0x10000  # placeholder device address, never dereferenced (validation fails first)


def header_functions():
    names = set()
    for h in sorted(glob.glob(os.path.join(ROOT, "include", "*.h"))):
        text = re.sub(r"/\*.*?\*/", "", open(h).read(), flags=re.S)
        names |= set(re.findall(r"\b(s2l_[a-z0-9_]+)\s*\(", text))
    return names


def test_library_exports_every_declared_function():
    names = header_functions()
    assert names == set(_lib.SIGNATURES), names ^ set(_lib.SIGNATURES)
    lib = _lib.lib()
    for n in names:
        assert hasattr(lib, n), n


def test_abi_version():
    assert _lib.lib().s2l_abi_version() == 3


def _batch(P, C, max_pages=None, device=True):
    P = np.asarray(P, np.int32)
    C = np.asarray(C, np.int32)
    b = _lib.s2l_batch()
    b.num_reqs = len(P)
    b.max_pages_per_req = max_pages if max_pages is not None else 64
    if device:
        b.prefix_lens = b.chunk_lens = b.cu_chunk = b.block_tables = FAKE
    b.prefix_lens_host = P.ctypes.data_as(_lib.P_i32)
    b.chunk_lens_host = C.ctypes.data_as(_lib.P_i32)
    return b, (P, C)


def _cache(head_dim=128, page_size=16, dtype=0, scales=False, hkv=2):
    c = _lib.s2l_kv_cache()
    c.k_pages = c.v_pages = FAKE
    if scales:
        c.k_scale = c.v_scale = FAKE
    c.num_pages, c.num_kv_heads, c.head_dim, c.page_size, c.dtype = 64, hkv, head_dim, page_size, dtype
    return c


def _status(name, *args):
    st = getattr(_lib.lib(), name)(*args)
    msg = _lib.lib().s2l_last_error().decode()
    return st, msg


@pytest.mark.parametrize("cache_kw,status", [
    (dict(head_dim=64), _lib.S2L_ENOTSUP),
    (dict(page_size=32), _lib.S2L_ENOTSUP),
    (dict(dtype=1, scales=False), _lib.S2L_EINVAL),
    (dict(dtype=0, scales=True), _lib.S2L_EINVAL),
    (dict(dtype=7), _lib.S2L_EINVAL),
])
def test_append_rejects_bad_cache(cache_kw, status):
    b, keep = _batch([0], [4])
    c = _cache(**cache_kw)
    st, msg = _status("s2l_kv_append", ctypes.byref(c), ctypes.byref(b), FAKE, FAKE, None)
    assert st == status and msg


@pytest.mark.parametrize("P,C,maxp,status", [
    ([-1], [4], 64, _lib.S2L_EINVAL),
    ([0], [-4], 64, _lib.S2L_EINVAL),
    ([1000], [25], 64, _lib.S2L_ERANGE),          # 1025 > 64 pages * 16
    ([1 << 30], [1], 1 << 26, _lib.S2L_EINVAL),
])
def test_append_rejects_bad_lengths(P, C, maxp, status):
    b, keep = _batch(P, C, maxp)
    c = _cache()
    st, msg = _status("s2l_kv_append", ctypes.byref(c), ctypes.byref(b), FAKE, FAKE, None)
    assert st == status and msg


def test_append_rejects_null_inputs_and_null_structs():
    b, keep = _batch([0], [4])
    c = _cache()
    assert _status("s2l_kv_append", ctypes.byref(c), ctypes.byref(b), None, FAKE, None)[0] == _lib.S2L_EINVAL
    assert _status("s2l_kv_append", None, ctypes.byref(b), FAKE, FAKE, None)[0] == _lib.S2L_EINVAL
    assert _status("s2l_kv_append", ctypes.byref(c), None, FAKE, FAKE, None)[0] == _lib.S2L_EINVAL
    b.block_tables = None
    assert _status("s2l_kv_append", ctypes.byref(c), ctypes.byref(b), FAKE, FAKE, None)[0] == _lib.S2L_EINVAL


def test_gather_rejects_bad_flag():
    b, keep = _batch([3], [4])
    c = _cache()
    st, _ = _status("s2l_kv_gather", ctypes.byref(c), ctypes.byref(b), 2, FAKE, FAKE, FAKE, None)
    assert st == _lib.S2L_EINVAL


@pytest.mark.parametrize("hq,hkv,status", [(8, 3, _lib.S2L_EINVAL), (0, 2, _lib.S2L_EINVAL),
                                           (512, 2, _lib.S2L_ENOTSUP)])
def test_plan_rejects_bad_heads(hq, hkv, status):
    b, keep = _batch([3], [4])
    info = _lib.s2l_plan_info()
    opts = _lib.s2l_plan_opts(target_items=64)
    st, msg = _status("s2l_attn_plan", ctypes.byref(b), hq, hkv, ctypes.byref(opts), FAKE, 1 << 20,
                      ctypes.byref(info), None)
    assert st == status and msg


def test_plan_rejects_small_workspace():
    b, keep = _batch([300], [40])
    info = _lib.s2l_plan_info()
    opts = _lib.s2l_plan_opts(target_items=64)
    n = ctypes.c_size_t()
    assert _status("s2l_attn_workspace_bytes", ctypes.byref(b), 8, 2, ctypes.byref(opts), ctypes.byref(n))[0] == 0
    st, _ = _status("s2l_attn_plan", ctypes.byref(b), 8, 2, ctypes.byref(opts), FAKE, n.value - 1,
                    ctypes.byref(info), None)
    assert st == _lib.S2L_EWORKSPACE
    st, _ = _status("s2l_attn_plan", ctypes.byref(b), 8, 2, ctypes.byref(opts), None, n.value,
                    ctypes.byref(info), None)
    assert st == _lib.S2L_EWORKSPACE


def _plan(P, C, hq, hkv, target=64):
    P = np.asarray(P, np.int32)
    C = np.asarray(C, np.int32)
    info = _lib.s2l_plan_info()
    opts = _lib.s2l_plan_opts(target_items=target)
    assert _lib.lib().s2l_plan_host(len(P), P.ctypes.data_as(_lib.P_i32), C.ctypes.data_as(_lib.P_i32),
                                    hq, hkv, ctypes.byref(opts), 0, ctypes.byref(info), None, 0) == 0
    return info


def test_attention_rejects_mismatched_plan_scale_and_workspace():
    b, keep = _batch([30], [40])
    c = _cache(hkv=2)
    info = _plan([30], [40], 8, 2)
    ok_bytes = info.workspace_bytes
    args = lambda hq, scale, plan, ws, nbytes: (ctypes.byref(c), ctypes.byref(b), FAKE, hq, scale, FAKE, None,
                                                 plan, ws, nbytes, None)
    for name in ("s2l_attn_main", "s2l_chunk_prefill_attn"):
        assert _status(name, *args(8, 0.0, ctypes.byref(info), FAKE, ok_bytes))[0] == _lib.S2L_EINVAL
        assert _status(name, *args(8, float("nan"), ctypes.byref(info), FAKE, ok_bytes))[0] == _lib.S2L_EINVAL
        assert _status(name, *args(16, 0.1, ctypes.byref(info), FAKE, ok_bytes))[0] == _lib.S2L_EINVAL
        assert _status(name, *args(8, 0.1, None, FAKE, ok_bytes))[0] == _lib.S2L_EINVAL
        assert _status(name, *args(8, 0.1, ctypes.byref(info), FAKE, ok_bytes - 1))[0] == _lib.S2L_EWORKSPACE
        assert _status(name, *args(8, 0.1, ctypes.byref(info), None, ok_bytes))[0] == _lib.S2L_EWORKSPACE
    other = _plan([31], [40], 8, 2)
    assert _status("s2l_attn_main", *args(8, 0.1, ctypes.byref(other), FAKE, ok_bytes))[0] == _lib.S2L_EINVAL \
        or other.total_tokens == info.total_tokens


def test_last_error_is_cleared_by_success():
    b, keep = _batch([3], [4], device=False)
    n = ctypes.c_size_t()
    opts = _lib.s2l_plan_opts(target_items=16)
    assert _status("s2l_attn_workspace_bytes", ctypes.byref(b), 8, 3, ctypes.byref(opts), ctypes.byref(n))[1]
    st, msg = _status("s2l_attn_workspace_bytes", ctypes.byref(b), 8, 2, ctypes.byref(opts), ctypes.byref(n))
    assert st == 0 and msg == "" and n.value > 0


def test_append_and_attention_checks_every_argument_before_enqueueing():
    """The two-call fallback (P not a multiple of 16) must not enqueue the append when the
    attention half is invalid: the call fails with EINVAL or EWORKSPACE from the host checks
    (an enqueued launch would have reached HIP here, where there is no device, and failed
    with EHIP instead)."""
    b, keep = _batch([30], [40])
    c = _cache(hkv=2)
    info = _plan([30], [40], 8, 2)
    ok_bytes = info.workspace_bytes
    fused = ctypes.c_int32(-1)

    def call(hq=8, scale=0.1, plan=ctypes.byref(info), q=FAKE, nbytes=ok_bytes, kn=FAKE):
        return _status("s2l_append_chunk_prefill_attn", ctypes.byref(c), ctypes.byref(b), kn, FAKE, q, hq, scale,
                       FAKE, None, plan, FAKE, nbytes, ctypes.byref(fused), None)[0]

    assert call(hq=16) == _lib.S2L_EINVAL
    assert call(scale=0.0) == _lib.S2L_EINVAL
    assert call(plan=None) == _lib.S2L_EINVAL
    assert call(q=None) == _lib.S2L_EINVAL
    assert call(kn=None) == _lib.S2L_EINVAL
    assert call(nbytes=ok_bytes - 1) == _lib.S2L_EWORKSPACE
    assert fused.value == -1                       # nothing decided, nothing enqueued


def test_noalloc_call_rejects_a_plan_larger_than_its_scratch():
    """16 pieces of a 512-token chunk with 32 query heads need 138 MB of partials: more than
    the 64 MiB scratch of the allocation-free call; rejected on the host, nothing launched."""
    b, _keep = _batch([8192], [512], max_pages=1024)
    c = _cache(hkv=8)
    o = _lib.s2l_plan_opts(target_items=1 << 20, min_split_keys=64, max_splits=16)
    info = _lib.s2l_plan_info()
    st = _lib.lib().s2l_chunk_prefill_attn_noalloc(ctypes.byref(c), ctypes.byref(b), FAKE, 32, 0.088, FAKE, None,
                                                   ctypes.byref(o), ctypes.byref(info), None)
    assert st == _lib.S2L_EWORKSPACE
    assert b"allocation-free" in _lib.lib().s2l_last_error()
