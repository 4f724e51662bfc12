"""GPU: the decode kernel (16-column work items, chosen when every request has
C * G <= 16) against the fp64 oracle: single tokens and a few tokens per tile (causal
inside the tile), every G from 1 to 16, page-edge prefixes, split and unsplit key ranges
(including pieces too short for all four waves), bf16 and fp8 caches, growing scores, and
long prefixes."""
import zlib

import numpy as np
import pytest

import paper_2604_16395_amd as s2l
import workloads
from tests.gpu_util import Setup, assert_attention_close, sample_rows

pytestmark = pytest.mark.gpu

FORCE_SPLIT = dict(target_items=1 << 20, min_split_keys=64, max_splits=16)

CASES = [
    ("one_token", [17], [1], 32, 8),
    ("p0", [0], [1], 32, 8),
    ("page_edges", [0, 5, 15, 16, 31, 32, 63, 64, 65, 1000, 4095], [1] * 11, 32, 8),
    ("g8_two_tokens", [3000, 70], [2, 1], 64, 8),
    ("g4_four_tokens", [500, 31, 0], [4, 3, 4], 32, 8),
    ("g1_sixteen_tokens", [200, 0], [16, 9], 8, 8),
    ("g16", [129, 4000], [1, 1], 16, 1),
    ("g2_ragged", [777], [5], 4, 2),
    ("with_empty", [40, 90, 0, 3000], [1, 0, 0, 1], 32, 8),
]


@pytest.mark.parametrize("kv_dtype", ["bf16", "fp8"])
@pytest.mark.parametrize("split", [False, True])
@pytest.mark.parametrize("name,P,C,hq,hkv", CASES)
def test_decode_cases_match_oracle(name, P, C, hq, hkv, split, kv_dtype):
    case = workloads.make_case(name, P, C, hq, hkv, seed=zlib.crc32(name.encode()) % 1000, kv_dtype=kv_dtype)
    print(f"[decode] {name} split={split} {kv_dtype}", flush=True)
    s = Setup(case)
    s.append()
    opts = dict(FORCE_SPLIT) if split else {}
    out, lse = s.attention(s2l.plan_opts(**opts))
    assert s.plan.tile_cols == 16
    if split and max(P) > 128:
        assert s.plan.num_split_reqs > 0
    ref = s.oracle()
    assert_attention_close(case, out, lse, ref, what=f"{name} {kv_dtype}")


def test_decode_tiles_of_several_tokens_forced():
    # 16-column tiles asked for explicitly on a chunk of 37 tokens (G = 4: 10 tiles, the last
    # ragged), causal inside every tile
    case = workloads.make_case("c37", [1200], [37], 32, 8, seed=31)
    s = Setup(case)
    s.append()
    for opts in (s2l.plan_opts(tile_cols=16), s2l.plan_opts(tile_cols=16, **FORCE_SPLIT)):
        out, lse = s.attention(opts)
        assert s.plan.tile_cols == 16 and s.plan.num_tiles == 8 * 10
        assert_attention_close(case, out, lse, s.oracle(), what="c37")


@pytest.mark.parametrize("q_sigma,k_ramp", [(4.0, 3.0), (0.5, 6.0)])
def test_decode_rescale_path(q_sigma, k_ramp):
    """Keys that grow along the sequence: a wave's reference max (its first tile) is
    overtaken by far (probabilities up to about 2^30 against it, per the host replay
    gpu_util.rescale_excess; the rescale branch, above 2^64, is exercised by the planted keys
    of test_gpu_rescale.py)."""
    case = workloads.make_case("ramp", [6000, 300], [1, 1], 32, 8, seed=33, q_sigma=q_sigma, k_ramp=k_ramp)
    s = Setup(case)
    s.append()
    for opts in (None, s2l.plan_opts(**FORCE_SPLIT)):
        out, lse = s.attention(opts)
        assert s.plan.tile_cols == 16
        assert_attention_close(case, out, lse, s.oracle(), what=f"ramp{q_sigma},{k_ramp}")


def test_decode_long_prefixes():
    # ten decode rows over prefixes up to 32K (the decode-like share of the mixed batch)
    rng = np.random.default_rng(35)
    P = rng.integers(1000, 32768, size=10).astype(np.int32)
    case = workloads.make_case("long", P, [1] * 10, 32, 8, seed=36)
    s = Setup(case)
    s.append()
    out, lse = s.attention()
    assert s.plan.tile_cols == 16
    assert_attention_close(case, out, lse, s.oracle(), what="long decode")


def test_decode_matches_the_wide_tiles():
    # same inputs through 128-column tiles and through the decode kernel: both within the
    # oracle's bound, and close to each other
    case = workloads.make_case("both", [2500, 9000, 40], [1, 2, 3], 32, 8, seed=37)
    s = Setup(case)
    s.append()
    ref = s.oracle()
    a, la = s.attention(s2l.plan_opts(tile_cols=16))
    b, lb = s.attention(s2l.plan_opts(tile_cols=128))
    assert_attention_close(case, a, la, ref, what="decode tiles")
    assert_attention_close(case, b, lb, ref, what="128-column tiles")
