"""GPU: the quantised-Q variant (s2l_chunk_prefill_attn_q8, e4m3 caches) against the fp64
oracle of the same definition: exact attention of the per-row e4m3-quantised queries over the
dequantised cache, to the same error bound as the bf16-Q path."""
import numpy as np
import pytest
import torch

import paper_2604_16395_amd as s2l
import workloads
from tests.gpu_util import (DEV, SCALE, Setup, named_case, assert_attention_close, bf16_to_f64, count_rows,
                            dense_rows, to_bf16)

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
    case = named_case("config5")
    s = Setup(case)
    s.append()
    out, lse = s.attention(q8=True)
    rows = dense_rows(case, 32)
    assert count_rows(rows) >= 64
    assert_attention_close(case, out, lse, s.oracle(rows, q8=True, spread=False), rows, what="q8 cfg5")


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


def test_q8_streamed_chunks_equal_one_shot():
    """The quantised-Q path keeps the streaming invariant: a 4096-token context arriving as 16
    chunks of 256 into an e4m3 cache, each chunk attended with quantised Q over the growing
    prefix; the streamed outputs and the GPU's one-shot quantised-Q run both match the oracle
    of the quantised queries on every 32nd row and the first and last row of every chunk,
    with the exact B.  (Q is quantised per row, so the chunking does not change what is
    computed.)"""
    case = workloads.make_case("q8stream", [0], [4096], 32, 8, seed=28, kv_dtype="fp8")
    s = Setup(case)
    kp = s.cache.k_pages.clone()                 # the sentinel-filled pools, before any append
    vp = s.cache.v_pages.clone()
    s.append()                                   # the whole sequence in the pages (the oracle's view)
    one, _ = s.attention(q8=True)
    cache = s2l.PagedKVCache(kp, vp, s.k_scale, s.v_scale)
    k_all, v_all = to_bf16(s.k_new), to_bf16(s.v_new)
    out = torch.empty((4096, 32, 128), dtype=torch.bfloat16, device=DEV)
    for step in range(16):
        P = 256 * step
        b = s2l.Batch([P], [256], case.block_tables)
        s2l.s2l_kv_append(cache, b, k_all[P:P + 256].contiguous(), v_all[P:P + 256].contiguous())
        ws = torch.empty(s2l.s2l_attn_workspace_bytes(b, 32, 8), dtype=torch.uint8, device=DEV)
        plan = s2l.s2l_attn_plan(b, 32, 8, ws)
        s2l.s2l_chunk_prefill_attn_q8(cache, b, s.q[P:P + 256].contiguous(), 32, SCALE, out[P:P + 256], None,
                                      plan, ws)
    torch.cuda.synchronize()
    assert torch.equal(kp, s.cache.k_pages) and torch.equal(vp, s.cache.v_pages)   # same pages either way
    rows = dense_rows(case, 32, 256)
    assert count_rows(rows) == 144
    ref = s.oracle(rows, q8=True)
    assert_attention_close(case, out, None, ref, rows, what="q8 stream")
    assert_attention_close(case, one, None, ref, rows, what="q8 one-shot")
