"""CPU: the planted-key inputs of the rescale tests do what they are for.

The host replay of the kernels' softmax references (gpu_util.rescale_excess) on the planned
work items shows a later key more than 64 log2 units above its key group's reference in every
layout, split and dtype the GPU tests run (so the rescale branch runs there), and the planted
keys sit where no key group's reference block can hold them.  Pools come from the oracle's
append, so no GPU is needed."""
import types

import numpy as np
import pytest

import paper_2604_16395_amd as s2l
import workloads
from oracle.paged_kv import ref_append
from tests.gpu_util import LOG2E, SCALE, plant_dots_for, rescale_excess, sentinel_pools

FORCE_SPLIT = dict(target_items=1 << 20, min_split_keys=64, max_splits=16)
DOTS = plant_dots_for(72.0, 4)
TWIN = 1.0 / (SCALE * LOG2E)


def _setup(case):
    kp, vp = sentinel_pools(case)
    R = case.num_reqs
    seq = (case.prefix_lens + case.chunk_lens).astype(np.int32)
    cu = np.zeros(R + 1, np.int32)
    cu[1:] = np.cumsum(seq)
    ref_append(kp, vp, case.block_tables, np.zeros(R, np.int32), seq, cu, case.k_full_bits, case.v_full_bits,
               case.kv_dtype, case.k_scale, case.v_scale)
    return types.SimpleNamespace(case=case, kp_ref=kp, vp_ref=vp, tables=case.block_tables)


@pytest.mark.parametrize("kv_dtype,q8", [("bf16", False), ("fp8", True)])
def test_planted_keys_pass_the_rescale_threshold_in_every_layout(kv_dtype, q8):
    case = workloads.make_case("planted", [3000, 100, 700], [300, 64, 1], 32, 8, seed=40, kv_dtype=kv_dtype,
                               plant_dots=DOTS, plant_twin_gap=TWIN)
    st = _setup(case)
    for layout in [(128, 1), (128, 2), (256, 1)]:
        for extra in ({}, FORCE_SPLIT):
            excess, above = rescale_excess(st, s2l.plan_opts(tile_cols=layout[0], key_halves=layout[1], **extra),
                                           q8=q8)
            assert 64 < excess and above > 0, (layout, extra, excess)


def test_planted_keys_pass_the_rescale_threshold_in_the_decode_kernel():
    case = workloads.make_case("planted_dec", [6000, 300, 9000, 40], [1, 1, 1, 1], 32, 8, seed=41,
                               plant_dots=DOTS, plant_twin_gap=TWIN)
    st = _setup(case)
    for extra in ({}, FORCE_SPLIT):
        excess, above = rescale_excess(st, s2l.plan_opts(**extra))
        assert 64 < excess and above > 0, (extra, excess)


def test_planted_positions_avoid_every_reference_block():
    case = workloads.make_case("planted", [3000, 100, 700], [300, 64, 1], 32, 8, seed=40,
                               plant_dots=DOTS, plant_twin_gap=TWIN)
    for r, pos in case.meta["planted"].items():
        for j in pos:
            assert j % 64 >= 32 and (j + 1) % 64 >= 32      # never among a tile's first 32 keys
            assert j + 1 < case.prefix_lens[r] + case.chunk_lens[r]
    # the planted rows are exactly the aligned keys: dot product with the target query
    G = 4
    q = (case.q_bits[299, 0].astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    j = case.meta["planted"][0][0]
    k = (case.k_full_bits[j, 0].astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    assert abs(k @ q - DOTS[0]) < 1e-2 * DOTS[0]
    assert G * 8 == case.num_q_heads
