"""Paged KV cache by definition: addressing, append (scatter) and gather.

Sec. 2.2 splits a sequence's KV cache into blocks of k tokens, block j (1-based) holding
tokens (j-1)k+1 .. min(jk, l), with blocks placed anywhere in physical memory; a
per-request table maps logical block j to a physical page.  With 0-based positions,
token p lives in logical page p // k at slot p % k.  This library uses k = 16 (the
vLLM default quoted with the 2 MB block size in Sec. 4.3).

Cache layout (one layer; the library's contract): separate K and V pools, each
``[num_pages][num_kv_heads][page_size][head_dim]``; a (page, kv head) pair is one
contiguous run of ``page_size * head_dim`` stored elements.  Stored elements are bf16
bit patterns (uint16) or OCP E4M3 codes (uint8, see :mod:`oracle.fp8_e4m3`).

Append (Sec. 4.2 / Sec. 5.1): request r holds P_r cached tokens (``num_computed_tokens``)
and receives C_r new ones; the new token i (0 <= i < C_r) is token P_r + i of the
sequence.  Only its slot is written; no other stored element changes.

Parity: pinned by the page-formula, round-trip and sentinel tests in
``tests/test_oracle_paging.py`` (bit-exact).
"""
import numpy as np

from .fp8_e4m3 import e4m3_decode, quantise_kv

PAGE_SIZE = 16


def page_slot(p, page_size=PAGE_SIZE):
    """0-based token position -> (logical page, slot)."""
    return p // page_size, p % page_size


def ref_append(k_pool, v_pool, block_tables, prefix_lens, chunk_lens, cu_chunk,
               k_new, v_new, kv_dtype="bf16", k_scale=None, v_scale=None):
    """Write each request's new K/V rows into their pages, in place.

    k_pool, v_pool : uint16 (bf16 bits) or uint8 (e4m3 codes) [num_pages][Hkv][16][D]
    block_tables   : int [R][max_pages]
    prefix_lens, chunk_lens : int [R]      (P_r, C_r)
    cu_chunk       : int [R+1]             row offset of request r's chunk in k_new/v_new
    k_new, v_new   : uint16 bf16 bits [T][Hkv][D]
    kv_dtype       : "bf16" stores the bits unchanged; "fp8" stores
                     e4m3(fp32(x) * fp32(1/scale[h])) per kv head h.
    """
    num_pages, hkv, ps, d = k_pool.shape
    for r in range(len(prefix_lens)):
        P, C, row0 = int(prefix_lens[r]), int(chunk_lens[r]), int(cu_chunk[r])
        if C == 0:
            continue
        p = P + np.arange(C)                       # absolute positions of the new tokens
        lp, slot = page_slot(p, ps)
        page = np.asarray(block_tables[r])[lp].astype(np.int64)
        kb = k_new[row0:row0 + C]                  # [C][Hkv][D]
        vb = v_new[row0:row0 + C]
        if kv_dtype == "bf16":
            k_pool[page, :, slot, :] = kb
            v_pool[page, :, slot, :] = vb
        else:
            k_pool[page, :, slot, :] = quantise_kv(bf16_bits_to_f32(kb), k_scale)
            v_pool[page, :, slot, :] = quantise_kv(bf16_bits_to_f32(vb), v_scale)


def ref_gather(pool, block_tables, r, n):
    """Stored elements of positions 0..n-1 of request r, shape [n][Hkv][D] (same dtype)."""
    ps = pool.shape[2]
    out = np.empty((n,) + pool.shape[1:2] + pool.shape[3:], dtype=pool.dtype)
    for p in range(n):
        lp, slot = page_slot(p, ps)
        out[p] = pool[int(block_tables[r][lp]), :, slot]
    return out


def bf16_bits_to_f32(bits):
    """bf16 bit patterns -> float32 (exact: a bf16 is the top half of a float32)."""
    b = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16
    return b.view(np.float32)


def decode_stored(stored, kv_dtype="bf16", scale=None):
    """Stored elements [n][Hkv][D] -> float64 values.

    bf16: exact conversion.  fp8: e4m3 decode times the per-kv-head scale, in float64.
    """
    if kv_dtype == "bf16":
        return bf16_bits_to_f32(stored).astype(np.float64)
    vals = e4m3_decode(stored)
    return vals * np.asarray(scale, dtype=np.float64)[None, :, None]


def kv_bytes_per_page(num_kv_heads, head_dim, page_size=PAGE_SIZE, elem_bytes=2):
    """Bytes of one page of ONE pool (K or V) for one layer."""
    return num_kv_heads * page_size * head_dim * elem_bytes
