"""Pins of the oracle's chunk attention (CPU only).

Each test checks the oracle against something other than itself: a dense brute-force
causal attention, scipy's softmax/logsumexp, closed forms of textbook special cases, the
invariant that any chunking of a sequence gives the same outputs as prefilling it whole,
and the Llama repeat-kv head order.
"""
import itertools

import numpy as np
import pytest
from scipy.special import logsumexp, softmax

from oracle.attention import (default_scale, lse_merge, ref_attn_key_range, ref_batch_attn,
                              ref_chunk_attn_blocked, ref_chunk_attn_loops, ref_full_causal)
from oracle.paged_kv import bf16_bits_to_f32, ref_append
from workloads import BF16_SENTINEL, make_case

SHAPES = [(1, 1), (2, 1), (4, 2), (8, 2), (8, 8), (6, 2)]


def _rand(rng, n, h, d, sigma=0.5):
    return rng.standard_normal((n, h, d)) * sigma


def _rel(a, b):
    return np.abs(a - b).max() / max(np.abs(b).max(), 1e-300)


@pytest.mark.parametrize("d", [8, 16, 128])
@pytest.mark.parametrize("hq,hkv", SHAPES)
def test_loops_equal_dense_causal_on_the_chunk_rows(d, hq, hkv):
    rng = np.random.default_rng(100 + d + hq * 7 + hkv)
    for P, C in [(0, 5), (7, 1), (13, 9), (40, 24), (90, 6)]:
        n = P + C
        q, k, v = _rand(rng, n, hq, d), _rand(rng, n, hkv, d), _rand(rng, n, hkv, d)
        sc = default_scale(d)
        o, l = ref_chunk_attn_loops(q[P:], k, v, P, sc)
        of, lf = ref_full_causal(q, k, v, sc)
        assert _rel(o, of[P:]) < 1e-12 and _rel(l, lf[P:]) < 1e-12


@pytest.mark.parametrize("hq,hkv", SHAPES)
def test_blocked_equals_loops(hq, hkv):
    rng = np.random.default_rng(5 + hq + hkv)
    d = 16
    for P, C in [(0, 33), (50, 17), (3, 64)]:
        n = P + C
        q, k, v = _rand(rng, n, hq, d), _rand(rng, n, hkv, d), _rand(rng, n, hkv, d)
        o1, l1 = ref_chunk_attn_loops(q[P:], k, v, P, 0.3)
        o2, l2 = ref_chunk_attn_blocked(q[P:], k, v, P, 0.3, q_block=7, k_block=10)
        assert _rel(o2, o1) < 1e-12 and _rel(l2, l1) < 1e-12
        rows = [0, 3, C - 1]
        o3, l3 = ref_chunk_attn_blocked(q[P:], k, v, P, 0.3, rows=rows, k_block=9)
        assert _rel(o3, o1[rows]) < 1e-12 and _rel(l3, l1[rows]) < 1e-12


def _compositions(n):
    for cuts in itertools.product([0, 1], repeat=n - 1):
        parts, last = [], 0
        for i, c in enumerate(cuts, start=1):
            if c:
                parts.append(i - last)
                last = i
        parts.append(n - last)
        yield parts


@pytest.mark.parametrize("n", [1, 2, 5, 9, 12])
def test_any_chunking_equals_whole_prefill(n):
    rng = np.random.default_rng(n)
    hq, hkv, d = 4, 2, 8
    q, k, v = _rand(rng, n, hq, d, 1.5), _rand(rng, n, hkv, d, 1.5), _rand(rng, n, hkv, d)
    whole_o, whole_l = ref_full_causal(q, k, v, 0.35)
    for parts in _compositions(n):
        outs, lses, P = [], [], 0
        for C in parts:
            o, l = ref_chunk_attn_blocked(q[P:P + C], k[:P + C], v[:P + C], P, 0.35, k_block=4)
            outs.append(o)
            lses.append(l)
            P += C
        assert _rel(np.concatenate(outs), whole_o) < 1e-12
        assert _rel(np.concatenate(lses), whole_l) < 1e-12


def test_first_row_without_prefix_returns_v0_exactly():
    rng = np.random.default_rng(1)
    q, k, v = _rand(rng, 6, 4, 16), _rand(rng, 6, 2, 16), _rand(rng, 6, 2, 16)
    for f in (ref_chunk_attn_loops, ref_chunk_attn_blocked):
        o, l = f(q, k, v, 0, 0.25)
        assert np.array_equal(o[0, :2], np.repeat(v[0, :1], 2, axis=0))
        assert np.array_equal(o[0, 2:], np.repeat(v[0, 1:], 2, axis=0))
        assert np.allclose(l[0], 0.25 * np.einsum("hd,hd->h", q[0], np.repeat(k[0], 2, axis=0)),
                           rtol=0, atol=1e-15)


def test_constant_keys_give_the_mean_of_visible_values():
    rng = np.random.default_rng(2)
    P, C, d = 11, 7, 16
    q = _rand(rng, C, 4, d)
    k = np.ones((P + C, 2, d)) * 0.3
    v = _rand(rng, P + C, 2, d)
    for f in (ref_chunk_attn_loops, ref_chunk_attn_blocked):
        o, _ = f(q, k, v, P, 0.2)
        for i in range(C):
            for h in range(4):
                assert np.allclose(o[i, h], v[:P + i + 1, h // 2].mean(axis=0), rtol=1e-13, atol=1e-15)


def test_one_hot_values_expose_scipy_softmax_probabilities():
    rng = np.random.default_rng(3)
    P, C, d = 9, 4, 16
    n = P + C
    q, k = _rand(rng, C, 2, d, 2.0), _rand(rng, n, 1, d, 2.0)
    v = np.zeros((n, 1, d))
    v[np.arange(n), 0, np.arange(n)] = 1.0
    o, l = ref_chunk_attn_blocked(q, k, v, P, 0.5, k_block=5)
    for i in range(C):
        for h in range(2):
            s = 0.5 * (k[:P + i + 1, 0] @ q[i, h])
            p = softmax(s)
            assert np.allclose(o[i, h, :P + i + 1], p, rtol=1e-13, atol=1e-16)
            assert np.all(o[i, h, P + i + 1:] == 0.0)
            assert abs(l[i, h] - logsumexp(s)) < 1e-12


def test_decode_row_equals_textbook_attention():
    rng = np.random.default_rng(4)
    P, d = 300, 128
    q, k, v = _rand(rng, 1, 8, d), _rand(rng, P + 1, 2, d), _rand(rng, P + 1, 2, d)
    sc = 1.0 / np.sqrt(128.0)
    o, l = ref_chunk_attn_blocked(q, k, v, P, sc, k_block=64)
    for h in range(8):
        p = softmax(sc * (k[:, h // 4] @ q[0, h]))
        assert _rel(o[0, h], p @ v[:, h // 4]) < 1e-12
        assert abs(l[0, h] - logsumexp(sc * (k[:, h // 4] @ q[0, h]))) < 1e-12


def test_gqa_equals_mha_with_llama_repeat_kv():
    rng = np.random.default_rng(5)
    P, C, d, G = 20, 10, 16, 3
    q, k, v = _rand(rng, C, 6, d), _rand(rng, P + C, 2, d), _rand(rng, P + C, 2, d)
    o1, l1 = ref_chunk_attn_blocked(q, k, v, P, 0.3)
    k_rep, v_rep = np.repeat(k, G, axis=1), np.repeat(v, G, axis=1)   # head h <- kv head h // G
    o2, l2 = ref_chunk_attn_loops(q, k_rep, v_rep, P, 0.3)
    assert _rel(o1, o2) < 1e-12 and _rel(l1, l2) < 1e-12


@pytest.mark.parametrize("cuts", [[5], [16, 32], [1, 2, 40], [64]])
def test_lse_merge_of_key_ranges_equals_unsplit(cuts):
    rng = np.random.default_rng(6)
    P, C, d = 50, 20, 16
    q, k, v = _rand(rng, C, 4, d, 2.0), _rand(rng, P + C, 2, d), _rand(rng, P + C, 2, d)
    bounds = [0] + cuts + [P + C]
    parts = [ref_attn_key_range(q, k, v, P, 0.4, a, b) for a, b in zip(bounds[:-1], bounds[1:])]
    om, lm = lse_merge([p[0] for p in parts], [p[1] for p in parts])
    o, l = ref_chunk_attn_loops(q, k, v, P, 0.4)
    assert _rel(om, o) < 1e-12 and _rel(lm, l) < 1e-12


def test_batch_through_paged_pools_equals_dense_per_request():
    case = make_case("t", [0, 37, 16, 5], [19, 8, 1, 40], 4, 2, seed=21, pool_pages=16)
    shape = (case.num_pages, 2, 16, 128)
    kp, vp = np.full(shape, BF16_SENTINEL, np.uint16), np.full(shape, BF16_SENTINEL, np.uint16)
    full_cu = np.zeros(case.num_reqs + 1, np.int32)
    full_cu[1:] = np.cumsum(case.prefix_lens + case.chunk_lens)
    ref_append(kp, vp, case.block_tables, np.zeros(case.num_reqs, np.int32),
               case.prefix_lens + case.chunk_lens, full_cu, case.k_full_bits, case.v_full_bits)
    q = bf16_bits_to_f32(case.q_bits).astype(np.float64)
    sc = default_scale(128)
    o, l = ref_batch_attn(q, kp, vp, case.block_tables, case.prefix_lens, case.chunk_lens,
                          case.cu_chunk, 4, sc)
    for r in range(case.num_reqs):
        P, C = int(case.prefix_lens[r]), int(case.chunk_lens[r])
        kf = bf16_bits_to_f32(case.k_full_bits[case.cu_seq[r]:case.cu_seq[r + 1]]).astype(np.float64)
        vf = bf16_bits_to_f32(case.v_full_bits[case.cu_seq[r]:case.cu_seq[r + 1]]).astype(np.float64)
        qf = np.concatenate([np.zeros((P, 4, 128)), q[case.cu_chunk[r]:case.cu_chunk[r + 1]]])
        of, lf = ref_full_causal(qf, kf, vf, sc)
        assert _rel(o[case.cu_chunk[r]:case.cu_chunk[r + 1]], of[P:]) < 1e-12
        assert _rel(l[case.cu_chunk[r]:case.cu_chunk[r + 1]], lf[P:]) < 1e-12
    # a sampled-row call returns the same rows
    o2, _ = ref_batch_attn(q, kp, vp, case.block_tables, case.prefix_lens, case.chunk_lens,
                           case.cu_chunk, 4, sc, sample_rows={1: [0, 7], 3: [39]})
    assert np.array_equal(o2[case.cu_chunk[1] + np.array([0, 7])], o[case.cu_chunk[1] + np.array([0, 7])])
    assert np.isnan(o2[0]).all()


def test_weighted_abs_values_are_the_same_weights_on_abs_v():
    rng = np.random.default_rng(8)
    P, C, d = 30, 9, 16
    q, k, v = _rand(rng, C, 4, d), _rand(rng, P + C, 2, d), _rand(rng, P + C, 2, d)
    o, l, oa, od = ref_chunk_attn_blocked(q, k, v, P, 0.3, k_block=7, with_abs=True)
    o2, _ = ref_chunk_attn_blocked(q, k, np.abs(v), P, 0.3)
    assert np.allclose(oa, o2, rtol=1e-13, atol=0)
    assert np.all(oa >= np.abs(o) - 1e-15)
    # B = sum_j w_j |V_j - O| from the softmax weights written out one row at a time
    for i in (0, 4, C - 1):
        for h in range(4):
            keys = np.arange(P + i + 1)
            s = np.array([0.3 * float(q[i, h] @ k[j, h // 2]) for j in keys])
            w = np.exp(s - s.max())
            w /= w.sum()
            dev = (w[:, None] * np.abs(v[keys, h // 2] - o[i, h][None, :])).sum(axis=0)
            assert np.allclose(od[i, h], dev, rtol=1e-12, atol=1e-15)
    assert np.all(od >= 0) and np.all(od <= oa + np.abs(o) + 1e-12)


def test_weighted_deviation_is_zero_when_all_values_agree():
    rng = np.random.default_rng(9)
    P, C, d = 20, 5, 8
    q, k = _rand(rng, C, 2, d), _rand(rng, P + C, 1, d)
    v = np.broadcast_to(_rand(rng, 1, 1, d), (P + C, 1, d)).copy()
    o, _, oa, od = ref_chunk_attn_blocked(q, k, v, P, 0.5, k_block=6, with_abs=True)
    assert np.allclose(o, v[0, 0][None, None, :], rtol=1e-13, atol=1e-15)
    assert np.all(od < 1e-13)
