"""Work-partition checks on the host mirror of the plan (CPU only).

The partition's layout is a design choice with no counterpart in the paper; what is pinned
is coverage: every (request, query head, chunk token, visible key) is computed by exactly
one work item, and the piece/tile bookkeeping is consistent.
"""
import numpy as np
import pytest

from paper_2604_16395_amd import plan_opts, s2l_plan_host
import workloads


def _coverage(P, C, hq, hkv, items):
    G = hq // hkv
    for r in range(len(P)):
        for g in range(hkv):
            mine = items[(items[:, 0] == r) & (items[:, 1] == g)]
            if C[r] == 0:
                assert len(mine) == 0
                continue
            # query tiles partition [0, C) with tq = 128 // G tokens
            tiles = sorted({(int(a), int(b)) for a, b in mine[:, 2:4]})
            tq = 128 // G
            assert tiles == [(t, min(t + tq, C[r])) for t in range(0, C[r], tq)]
            for (i0, i1) in tiles:
                pcs = mine[(mine[:, 2] == i0)]
                ns = int(pcs[0, 7])
                assert len(pcs) == ns and sorted(pcs[:, 6]) == list(range(ns))
                # pieces partition [0, P + i1): disjoint, ordered, 64-aligned starts
                pcs = pcs[np.argsort(pcs[:, 6])]
                cover = np.zeros(P[r] + i1, dtype=np.int32)
                for lo, hi in pcs[:, 4:6]:
                    assert lo % 64 == 0 and lo <= hi
                    cover[lo:hi] += 1
                assert np.all(cover == 1)
                # every token of the tile sees its keys 0..P+i in this tile's pieces
                assert P[r] + i1 - 1 < len(cover) + 1


@pytest.mark.parametrize("target", [1, 64, 1 << 20])
@pytest.mark.parametrize("hq,hkv", [(8, 2), (32, 8), (6, 2), (4, 4), (64, 8)])
def test_items_cover_each_visible_pair_once(target, hq, hkv):
    rng = np.random.default_rng(target + hq)
    P = rng.integers(0, 3000, size=7).astype(np.int32)
    C = rng.integers(0, 300, size=7).astype(np.int32)
    P[0], C[0] = 0, 1
    C[1] = 0
    P[2] = 17
    info, items = s2l_plan_host(P, C, hq, hkv, plan_opts(target_items=target, min_split_keys=64), with_items=True)
    assert info.num_items == len(items)
    _coverage(P, C, hq, hkv, items)
    assert info.total_tokens == C.sum()


def test_plan_is_deterministic_and_independent_of_call():
    P, C, _ = workloads.config4_lengths()
    a, ia = s2l_plan_host(P, C, 32, 8, with_items=True)
    b, ib = s2l_plan_host(P, C, 32, 8, with_items=True)
    assert np.array_equal(ia, ib) and a.workspace_bytes == b.workspace_bytes


def test_split_policy_on_the_named_workloads():
    # one 512-token chunk at an 8K prefix: 128 tiles < 512 wanted -> the prefix is split
    info, _ = s2l_plan_host([8192], [512], 32, 8, num_cus=256)
    assert info.num_split_reqs == 1 and info.num_items >= 512 and info.split_keys % 64 == 0
    # 8 x 512-token chunks: 1024 tiles already -> no split
    P2, C2, _ = workloads.config2_lengths()
    info, _ = s2l_plan_host(P2, C2, 32, 8, num_cus=256)
    assert info.num_split_reqs == 0 and info.num_items == 8 * 8 * 16
    # 70B share: 2048 tokens x 8 heads / 16 tokens per tile = 1024 tiles -> no split
    info, _ = s2l_plan_host([131072], [2048], 64, 8, num_cus=256)
    assert info.num_split_reqs == 0 and info.num_items == 1024


def test_workspace_grows_with_partials_only_for_split_requests():
    a, _ = s2l_plan_host([8192], [512], 32, 8, num_cus=256)
    b, _ = s2l_plan_host([8192], [512], 32, 8, plan_opts(target_items=1), num_cus=256)
    assert b.num_split_reqs == 0 and b.workspace_bytes < a.workspace_bytes
    ns = a.num_items // (8 * 16)
    assert a.workspace_bytes >= ns * 512 * 32 * 130 * 4


def test_empty_and_degenerate_batches():
    info, items = s2l_plan_host([], [], 32, 8, plan_opts(target_items=8), with_items=True)
    assert info.num_items == 0 and info.workspace_bytes > 0
    info, items = s2l_plan_host([5, 0], [0, 0], 32, 8, plan_opts(target_items=8), with_items=True)
    assert info.num_items == 0
    info, items = s2l_plan_host([0], [1], 8, 8, plan_opts(target_items=8), with_items=True)
    assert info.num_items == 8 and set(map(tuple, items[:, 2:6])) == {(0, 1, 0, 1)}
