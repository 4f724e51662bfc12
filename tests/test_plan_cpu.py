"""Work-partition checks on the host mirror of the plan (CPU only).

The partition's layout is a design choice with no counterpart in the paper; what is pinned
is coverage: every (request, query head, chunk token, visible key) is computed by exactly
one work item, and the piece/tile bookkeeping is consistent.
"""
import numpy as np
import pytest

from paper_2604_16395_amd import plan_opts, s2l_plan_host
import workloads

UNIFORM, BINNED = 1, 2


def _coverage(P, C, hq, hkv, items, tile_cols):
    G = hq // hkv
    for r in range(len(P)):
        for g in range(hkv):
            mine = items[(items[:, 0] == r) & (items[:, 1] == g)]
            if C[r] == 0:
                assert len(mine) == 0
                continue
            # query tiles partition [0, C) with tq = tile_cols // G tokens
            tiles = sorted({(int(a), int(b)) for a, b in mine[:, 2:4]})
            tq = tile_cols // G
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


@pytest.mark.parametrize("tile_cols,halves", [(0, 0), (128, 1), (256, 0)])
@pytest.mark.parametrize("target", [1, 64, 1 << 20])
@pytest.mark.parametrize("hq,hkv", [(8, 2), (32, 8), (6, 2), (4, 4), (64, 8)])
def test_items_cover_each_visible_pair_once(target, hq, hkv, tile_cols, halves):
    rng = np.random.default_rng(target + hq)
    P = rng.integers(0, 3000, size=7).astype(np.int32)
    C = rng.integers(0, 300, size=7).astype(np.int32)
    P[0], C[0] = 0, 1
    C[1] = 0
    P[2] = 17
    info, items = s2l_plan_host(P, C, hq, hkv, plan_opts(target_items=target, min_split_keys=64,
                                                         tile_cols=tile_cols, key_halves=halves),
                                with_items=True)
    assert info.num_items == len(items)
    real, pad = items[items[:, 0] >= 0], items[items[:, 0] < 0]
    assert np.all(pad == [-1, 0, 0, 0, 0, 0, 0, 0])            # no-op padding of the XCD bins
    if info.flags & BINNED:
        assert info.num_items % 8 == 0 and len(pad) < info.num_items
    else:
        assert len(pad) == 0
    assert tile_cols == 0 or info.tile_cols == tile_cols
    _coverage(P, C, hq, hkv, real, info.tile_cols)
    assert info.total_tokens == C.sum()
    # one tile per (request, kv head, query tile); the items of a tile are its pieces
    assert info.num_tiles == len({(r, g, i0) for r, g, i0 in real[:, 0:3]})


def test_plan_is_deterministic_and_independent_of_call():
    P, C, _ = workloads.config4_lengths()
    a, ia = s2l_plan_host(P, C, 32, 8, with_items=True)
    b, ib = s2l_plan_host(P, C, 32, 8, with_items=True)
    assert np.array_equal(ia, ib) and a.workspace_bytes == b.workspace_bytes


def test_split_policy_on_the_named_workloads():
    # one 512-token chunk at an 8K prefix: 256-column tiles (64 tokens x 4 heads), 64 tiles
    # for 256 one-per-CU workgroups -> every tile cut into 4 pieces: exactly 256 items
    info, items = s2l_plan_host([8192], [512], 32, 8, num_cus=256, with_items=True)
    assert info.tile_cols == 256 and info.key_halves == 1 and info.num_tiles == 64
    assert info.num_split_reqs == 1 and info.num_items == 256 and info.split_keys % 64 == 0
    assert set(items[:, 7]) == {4}
    # 128-column tiles with two key-range wave groups, one workgroup per CU: 2 pieces
    info, _ = s2l_plan_host([8192], [512], 32, 8, plan_opts(tile_cols=128), num_cus=256)
    assert info.key_halves == 2 and info.num_tiles == 128 and info.num_items == 256
    # 4-wave workgroups, two per CU: 128 tiles -> 4 pieces
    info, _ = s2l_plan_host([8192], [512], 32, 8, plan_opts(tile_cols=128, key_halves=1), num_cus=256)
    assert info.num_tiles == 128 and info.num_items == 512
    # 8 x 512-token chunks: 512 tiles already -> no split
    P2, C2, _ = workloads.config2_lengths()
    info, _ = s2l_plan_host(P2, C2, 32, 8, num_cus=256)
    assert info.num_split_reqs == 0 and info.num_items == 8 * 8 * 8
    # 70B share: 2048 tokens x 8 heads / 32 tokens per tile = 512 tiles -> no split
    info, _ = s2l_plan_host([131072], [2048], 64, 8, num_cus=256)
    assert info.num_split_reqs == 0 and info.num_items == 512


def test_automatic_tile_width():
    # every request fits a 16-column tile (C * G <= 16): the decode kernel's tiles
    info, _ = s2l_plan_host([4000] * 16, [1] * 16, 32, 8, num_cus=256)
    assert info.tile_cols == 16 and info.key_halves == 1
    info, _ = s2l_plan_host([4000, 10], [4, 2], 32, 8, num_cus=256)      # 16 and 8 columns
    assert info.tile_cols == 16 and info.num_tiles == 2 * 8
    info, _ = s2l_plan_host([4000], [2], 64, 8, num_cus=256)             # G = 8: 16 columns
    assert info.tile_cols == 16
    # one request past 16 columns: decode-like rows fill 256-column tiles to 2%: 128
    info, _ = s2l_plan_host([4000] * 15 + [4000], [1] * 15 + [5], 32, 8, num_cus=256)
    assert info.tile_cols == 128 and info.key_halves == 2
    info, _ = s2l_plan_host([4000], [1], 32, 1, num_cus=256)             # G = 32 > 16
    assert info.tile_cols == 128
    info, _ = s2l_plan_host([100, 5000], [300, 700], 32, 8, num_cus=256)
    assert info.tile_cols == 256 and info.key_halves == 1


@pytest.mark.parametrize("seed", range(20))
def test_splitting_never_exceeds_the_target(seed):
    rng = np.random.default_rng(seed)
    R = int(rng.integers(1, 12))
    P = rng.integers(0, 40000, size=R).astype(np.int32)
    C = rng.integers(1, 700, size=R).astype(np.int32)
    target = int(rng.integers(8, 600))
    info, _ = s2l_plan_host(P, C, 32, 8, plan_opts(target_items=target, min_split_keys=64))
    assert info.num_items <= max(target, info.num_tiles)


def test_option_validation():
    with pytest.raises(Exception):
        s2l_plan_host([100], [10], 32, 8, plan_opts(tile_cols=256, key_halves=2))
    with pytest.raises(Exception):
        s2l_plan_host([100], [10], 32, 8, plan_opts(key_halves=3))
    with pytest.raises(Exception):
        s2l_plan_host([100], [1], 32, 8, plan_opts(tile_cols=16, key_halves=2))
    with pytest.raises(Exception):
        s2l_plan_host([100], [1], 32, 1, plan_opts(tile_cols=16))         # G = 32
    with pytest.raises(Exception):
        s2l_plan_host([100], [1], 32, 8, plan_opts(tile_cols=64))
    # a 16-column tile holds 16 / G tokens: longer chunks take several tiles
    info, _ = s2l_plan_host([100], [10], 32, 8, plan_opts(tile_cols=16, target_items=1))
    assert info.num_tiles == 8 * 3 and info.num_items == 8 * 3


def test_workspace_grows_with_partials_only_for_split_requests():
    a, _ = s2l_plan_host([8192], [512], 32, 8, num_cus=256)
    b, _ = s2l_plan_host([8192], [512], 32, 8, plan_opts(target_items=1), num_cus=256)
    assert b.num_split_reqs == 0 and b.workspace_bytes < a.workspace_bytes
    ns = a.num_items // a.num_tiles
    assert a.part_floats == ns * 512 * 32 * 132 and b.part_floats == 0
    assert a.workspace_bytes >= ns * 512 * 32 * 132 * 4 + 64 * a.num_items


def test_empty_and_degenerate_batches():
    info, items = s2l_plan_host([], [], 32, 8, plan_opts(target_items=8), with_items=True)
    assert info.num_items == 0 and info.workspace_bytes > 0
    info, items = s2l_plan_host([5, 0], [0, 0], 32, 8, plan_opts(target_items=8), with_items=True)
    assert info.num_items == 0
    info, items = s2l_plan_host([0], [1], 8, 8, plan_opts(target_items=8), with_items=True)
    assert info.num_items == 8 and set(map(tuple, items[:, 2:6])) == {(0, 1, 0, 1)}


def test_uniform_items_flag():
    # one request: every item's key range within a few percent of the mean
    info, _ = s2l_plan_host([8192], [512], 32, 8, num_cus=256)
    assert info.flags & 1
    info, _ = s2l_plan_host([131072], [2048], 64, 8, num_cus=256)
    assert info.flags & 1
    # the mixed 64-request batch: ranges from a handful of keys to 34K
    P, C, _ = workloads.config4_lengths()
    info, _ = s2l_plan_host(P, C, 32, 8, num_cus=256)
    assert not (info.flags & 1)


def _binned_len(P, C, hq, hkv, info, items):
    """A second statement of the binned order's rule: (request, kv head) groups, requests by
    P + C descending (ties by index, requests without new tokens last), each to the bin with the
    least work so far (lowest index on ties); work of a group = the key ranges [0, P + i1) of its
    query tiles + 192 keys per item.  Returns (bins balanced within 4%, padded item count)."""
    tq = info.tile_cols // (hq // hkv)
    real = items[items[:, 0] >= 0]
    order = sorted(range(len(P)), key=lambda r: (-(P[r] + C[r] if C[r] > 0 else -1), r))
    load, count = [0] * 8, [0] * 8
    for r in order:
        mine = real[(real[:, 0] == r) & (real[:, 1] == 0)]
        n = len(mine)
        cost = sum(int(P[r]) + min(t + tq, int(C[r])) for t in range(0, int(C[r]), tq)) + 192 * n
        for _ in range(hkv):
            x = min(range(8), key=lambda y: (load[y], y))
            load[x] += cost
            count[x] += n
    return max(load) * 8 * 25 <= sum(load) * 26, 8 * max(count)


@pytest.mark.parametrize("which", ["config2", "config4", "ragged", "uniform"])
def test_binned_order_follows_its_rule(which):
    if which == "config2":
        P, C, _ = workloads.config2_lengths()
    elif which == "config4":
        P, C, _ = workloads.config4_lengths()
    elif which == "ragged":
        rng = np.random.default_rng(3)
        P, C = rng.integers(0, 20000, 40), rng.integers(1, 700, 40)
    else:
        P, C = np.full(8, 4096), np.full(8, 512)
    P, C = np.asarray(P, np.int32), np.asarray(C, np.int32)
    info, items = s2l_plan_host(P, C, 32, 8, num_cus=256, with_items=True)
    real = items[items[:, 0] >= 0]
    if info.flags & UNIFORM:
        assert which == "uniform" and len(real) == info.num_items
        return
    balanced, padded = _binned_len(P, C, 32, 8, info, items)
    if balanced:
        assert info.flags == BINNED and info.num_items == padded
    else:
        assert info.flags == 0 and info.num_items == len(real)
    if which in ("config2", "config4"):
        assert info.flags == BINNED   # the named mixed batches do balance
