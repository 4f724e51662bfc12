"""GPU: the quantised-Q variant (s2l_chunk_prefill_attn_q8, e4m3 caches) against the fp64
oracle of the same definition: exact attention of the per-row e4m3-quantised queries over the
dequantised cache, to the same error bound as the bf16-Q path."""
import numpy as np
import pytest
import torch

import paper_2604_16395_amd as s2l
import workloads
from tests.gpu_util import DEV, SCALE, Setup, assert_attention_close, bf16_to_f64, sample_rows

pytestmark = pytest.mark.gpu

FORCE_SPLIT = dict(target_items=1 << 20, min_split_keys=64, max_splits=16)
LAYOUTS = [(128, 1), (128, 2), (256, 1)]
CASES = [
    ("fp8_small", [700, 0, 33], [130, 77, 1], 64, 8),
    ("g4_varlen", [5, 0, 300, 64, 9], [33, 129, 1, 64, 0], 32, 8),
    ("page_edges", [15, 16, 17, 31], [1, 16, 15, 33], 8, 2),
]


@pytest.mark.parametrize("layout", LAYOUTS)
@pytest.mark.parametrize("split", [False, True])
@pytest.mark.parametrize("name,P,C,hq,hkv", CASES)
def test_q8_matches_oracle_of_quantised_queries(name, P, C, hq, hkv, split, layout):
    case = workloads.make_case(name, P, C, hq, hkv, seed=21, kv_dtype="fp8")
    s = Setup(case)
    s.append()
    opts = dict(FORCE_SPLIT) if split else {}
    out, lse = s.attention(s2l.plan_opts(tile_cols=layout[0], key_halves=layout[1], **opts), q8=True)
    assert_attention_close(case, out, lse, s.oracle(q8=True), what=f"q8 {name}")


def test_q8_quantisation_is_applied():
    """The quantised-Q output follows its own oracle and not the bf16-Q one where they differ."""
    case = workloads.make_case("peaky_q8", [2000], [64], 32, 8, seed=22, kv_dtype="fp8", q_sigma=4.0)
    s = Setup(case)
    s.append()
    out, lse = s.attention(q8=True)
    ref8, ref = s.oracle(q8=True), s.oracle()
    assert_attention_close(case, out, lse, ref8, what="q8 peaky")
    o = bf16_to_f64(out)
    assert np.abs(o - ref8[0]).mean() < np.abs(o - ref[0]).mean()


def test_q8_config5_sampled_rows():
    case = workloads.config5()
    s = Setup(case)
    s.append()
    out, lse = s.attention(q8=True)
    rows = sample_rows(case, 12, np.random.default_rng(23))
    assert_attention_close(case, out, lse, s.oracle(rows, q8=True), rows, what="q8 cfg5")


def test_q8_rejects_bf16_cache_and_decode_tiles():
    bf = workloads.make_case("bf", [64], [16], 8, 2, seed=24)
    s = Setup(bf)
    s.append()
    with pytest.raises(s2l.S2LError, match="e4m3"):
        s.attention(q8=True)
    f8 = workloads.make_case("dec", [64], [1], 8, 2, seed=25, kv_dtype="fp8")
    s = Setup(f8)
    s.append()
    with pytest.raises(s2l.S2LError, match="decode"):
        s.attention(s2l.plan_opts(), q8=True)      # C * G = 4 columns: automatic 16-column tiles
