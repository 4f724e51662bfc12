"""GPU: the rescale branch of the online softmax (both attention kernels) against the oracle.

The kernels accumulate probabilities against a per-column reference max taken from the first
keys a key group sees (the main kernel: the first 32 keys of its range; the decode kernel:
each wave's first 64-key tile).  Only when a later probability would exceed 2^64 do they raise
the reference, rescale O and l and redo the sub-block; the result must stay the exact softmax
of Sec. 2.1 at any score spread.  These inputs plant keys aligned with one query per kv head,
late in each request, each 72 log2 units above the one before (so the first is far above the
keys before it, and later ones overflow fp32 against the old reference), plus a twin one log2
unit below the last one, so the output mixes two keys.  Before each launch the host replays
the kernel's references on the plan's work items and asserts that some excess is above 64,
i.e. that the branch runs; the outputs are then checked against the fp64 oracle with the same
bound as every other parity test."""
import numpy as np
import pytest

import paper_2604_16395_amd as s2l
import workloads
from tests.gpu_util import LOG2E, SCALE, Setup, assert_attention_close, plant_dots_for, rescale_excess

pytestmark = pytest.mark.gpu

FORCE_SPLIT = dict(target_items=1 << 20, min_split_keys=64, max_splits=16)
LAYOUTS = [(128, 1), (128, 2), (256, 1)]
DOTS = plant_dots_for(72.0, 4)
TWIN = 1.0 / (SCALE * LOG2E)            # one log2 unit


def _case(name, P, C, hq, hkv, seed, kv_dtype):
    return workloads.make_case(name, P, C, hq, hkv, seed=seed, kv_dtype=kv_dtype, plant_dots=DOTS,
                               plant_twin_gap=TWIN)


@pytest.mark.parametrize("layout", LAYOUTS)
@pytest.mark.parametrize("split", [False, True])
@pytest.mark.parametrize("kv_dtype,q8", [("bf16", False), ("fp8", False), ("fp8", True)])
def test_planted_keys_main_kernel(kv_dtype, q8, split, layout):
    case = _case("planted", [3000, 100, 700], [300, 64, 1], 32, 8, 40, kv_dtype)
    s = Setup(case)
    s.append()
    opts = s2l.plan_opts(tile_cols=layout[0], key_halves=layout[1], **(FORCE_SPLIT if split else {}))
    excess, above = rescale_excess(s, opts, q8=q8)
    print(f"[rescale] {kv_dtype} q8={q8} split={split} layout={layout}: max excess {excess:.1f}, "
          f"{above} (item, group, column) over 64", flush=True)
    assert excess > 64 and above > 0
    out, lse = s.attention(opts, q8=q8)
    assert s.plan.tile_cols == layout[0]
    assert_attention_close(case, out, lse, s.oracle(q8=q8), what=f"planted {kv_dtype} q8={q8}")


@pytest.mark.parametrize("split", [False, True])
@pytest.mark.parametrize("kv_dtype", ["bf16", "fp8"])
def test_planted_keys_decode_kernel(kv_dtype, split):
    case = _case("planted_dec", [6000, 300, 9000, 40], [1, 1, 1, 1], 32, 8, 41, kv_dtype)
    s = Setup(case)
    s.append()
    opts = s2l.plan_opts(**(FORCE_SPLIT if split else {}))
    excess, above = rescale_excess(s, opts)
    print(f"[rescale] decode {kv_dtype} split={split}: max excess {excess:.1f}, {above} over 64", flush=True)
    assert excess > 64 and above > 0
    out, lse = s.attention(opts)
    assert s.plan.tile_cols == 16
    assert_attention_close(case, out, lse, s.oracle(), what=f"planted decode {kv_dtype}")


def test_planted_keys_output_is_the_blend_of_the_two_top_keys():
    """The target column (last token, first query head of each kv head) attends, to within
    2^-60, only to the last planted key and its twin (about one log2 unit below it once the keys
    are rounded to bf16, so both carry weight): the oracle's output equals that two-key softmax, and
    the GPU's is within the bound.  A check that the planted inputs are what they claim."""
    case = _case("planted_blend", [3000], [64], 32, 8, 42, "bf16")
    s = Setup(case)
    s.append()
    out, lse = s.attention()
    ref = s.oracle()
    assert_attention_close(case, out, lse, ref, what="planted blend")
    j = case.meta["planted"][0][-1]
    f64 = lambda bits: (bits.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    kf, vf = f64(case.k_full_bits[[j, j + 1]]), f64(case.v_full_bits[[j, j + 1]])
    for g in range(8):
        qv = f64(case.q_bits[63, 4 * g])
        sc = SCALE * (kf[:, g] @ qv)
        w = np.exp(sc - sc.max())
        assert 0.3 < w[1] / w[0] < 0.8                 # about one log2 unit apart (bf16-rounded keys)
        expect = (w[:, None] * vf[:, g]).sum(axis=0) / w.sum()
        assert np.abs(ref[0][63, 4 * g] - expect).max() < 1e-9
