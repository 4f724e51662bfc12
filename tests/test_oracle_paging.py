"""Pins of the oracle's paged-KV addressing, append and gather (CPU only)."""
import json
import math
import os

import numpy as np
import pytest

from oracle.paged_kv import (bf16_bits_to_f32, decode_stored, kv_bytes_per_page, page_slot,
                             ref_append, ref_gather)
from oracle.fp8_e4m3 import quantise_kv
from workloads import BF16_SENTINEL, FP8_SENTINEL, make_case

GOLD = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "paper_kv_geometry.json")))


def test_page_formula_matches_the_papers_block_intervals():
    g = GOLD["block_interval"]
    for k in g["k_values"]:
        for ell in range(1, g["ell_max"] + 1):
            for j in range(1, math.ceil(ell / k) + 1):           # paper: 1-based blocks/tokens
                for t in range((j - 1) * k + 1, min(j * k, ell) + 1):
                    lp, slot = page_slot(t - 1, k)
                    assert lp == j - 1 and slot == (t - 1) - (j - 1) * k
            # attention at position t reads blocks 1..ceil(t/k): the pages of positions < t
            for t in range(1, ell + 1):
                pages = {page_slot(p, k)[0] for p in range(t)}
                assert pages == set(range(math.ceil(t / k)))


def test_block_and_cache_sizes_match_the_paper():
    kv = GOLD["kv_cache_per_request"]
    blk = GOLD["block"]
    hkv, head_dim = kv["h_kv"], kv["d"] // kv["h"]
    per_layer_page_k = kv_bytes_per_page(hkv, head_dim, blk["k"], kv["b"])
    assert per_layer_page_k == 32 * 1024                          # 32 KiB of K per page per layer
    m_block = 2 * kv["L"] * per_layer_page_k                       # K and V, all layers
    assert m_block == blk["M_block_MB_printed"] * 2 ** 20
    m_kv = (kv["ell"] // blk["k"]) * m_block
    assert m_kv == 2 * kv["L"] * kv["ell"] * kv["d"] * kv["h_kv"] // kv["h"] * kv["b"]
    assert round(m_kv / 2 ** 30, 1) == kv["M_KV_GB_printed"]


def _empty_pools(case, dtype):
    shape = (case.num_pages, case.num_kv_heads, 16, 128)
    if dtype == "bf16":
        return np.full(shape, BF16_SENTINEL, np.uint16), np.full(shape, BF16_SENTINEL, np.uint16)
    return np.full(shape, FP8_SENTINEL, np.uint8), np.full(shape, FP8_SENTINEL, np.uint8)


def _append_all(case, kp, vp, splits):
    """Append every request's full sequence in chunks given by ``splits`` (cut points)."""
    R = case.num_reqs
    seq = case.prefix_lens + case.chunk_lens
    cuts = [0] + list(splits) + [int(seq.max())]
    for a, b in zip(cuts[:-1], cuts[1:]):
        P = np.minimum(seq, a).astype(np.int32)
        C = (np.minimum(seq, b) - P).astype(np.int32)
        cu = np.zeros(R + 1, np.int32)
        cu[1:] = np.cumsum(C)
        rows_k = np.concatenate([case.k_full_bits[case.cu_seq[r] + P[r]:case.cu_seq[r] + P[r] + C[r]]
                                 for r in range(R)])
        rows_v = np.concatenate([case.v_full_bits[case.cu_seq[r] + P[r]:case.cu_seq[r] + P[r] + C[r]]
                                 for r in range(R)])
        ref_append(kp, vp, case.block_tables, P, C, cu, rows_k, rows_v, case.kv_dtype,
                   case.k_scale, case.v_scale)


@pytest.mark.parametrize("splits", [[], [5], [16, 33], [1, 2, 3, 17, 31, 32, 48]])
def test_round_trip_is_bit_exact_and_chunking_does_not_matter(splits):
    case = make_case("t", [0, 0, 0], [37, 50, 16], 4, 2, seed=11, pool_pages=20)
    kp, vp = _empty_pools(case, "bf16")
    _append_all(case, kp, vp, splits)
    for r in range(case.num_reqs):
        n = int(case.chunk_lens[r])
        want_k = case.k_full_bits[case.cu_seq[r]:case.cu_seq[r] + n]
        assert np.array_equal(ref_gather(kp, case.block_tables, r, n), want_k)
        want_v = case.v_full_bits[case.cu_seq[r]:case.cu_seq[r] + n]
        assert np.array_equal(ref_gather(vp, case.block_tables, r, n), want_v)
    # one-shot append gives the same pools byte for byte
    kp1, vp1 = _empty_pools(case, "bf16")
    _append_all(case, kp1, vp1, [])
    assert np.array_equal(kp, kp1) and np.array_equal(vp, vp1)


def test_only_slots_of_the_chunk_change():
    case = make_case("t", [21, 0], [9, 3], 2, 2, seed=12, pool_pages=8)
    kp, vp = _empty_pools(case, "bf16")
    before = kp.copy()
    ref_append(kp, vp, case.block_tables, case.prefix_lens, case.chunk_lens, case.cu_chunk,
               case.new_rows(case.k_full_bits), case.new_rows(case.v_full_bits))
    changed = np.argwhere(np.any(kp != before, axis=-1))           # (page, head, slot)
    expect = set()
    for r, (P, C) in enumerate(zip(case.prefix_lens, case.chunk_lens)):
        for p in range(P, P + C):
            for h in range(case.num_kv_heads):
                expect.add((int(case.block_tables[r][p // 16]), h, p % 16))
    assert {tuple(map(int, x)) for x in changed} == expect
    # request 0 starts mid-page (P=21): slots 0..4 of its second page keep the sentinel
    page = int(case.block_tables[0][1])
    assert np.all(kp[page, :, :5] == BF16_SENTINEL)
    assert np.all(kp[page, :, 14:] == BF16_SENTINEL)               # 21+9 = 30 -> slots 5..13


def test_fp8_pages_hold_the_quantised_rows():
    case = make_case("t", [0], [40], 2, 2, seed=13, kv_dtype="fp8", pool_pages=4)
    kp, vp = _empty_pools(case, "fp8")
    _append_all(case, kp, vp, [7])
    got = ref_gather(kp, case.block_tables, 0, 40)
    want = quantise_kv(bf16_bits_to_f32(case.k_full_bits[:40]), case.k_scale)
    assert np.array_equal(got, want)
    # decode(scale) reproduces the inputs to within half an fp8 step (relative 2^-4)
    x = bf16_bits_to_f32(case.k_full_bits[:40]).astype(np.float64)
    y = decode_stored(got, "fp8", case.k_scale)
    assert np.all(np.abs(y - x) <= np.maximum(np.abs(x) * 2.0 ** -4, case.k_scale.max() * 2.0 ** -9))
