"""GPU: append and attention in one call (s2l_append_chunk_prefill_attn) give the same
pages, outputs and LSE, bit for bit, as s2l_kv_append followed by s2l_chunk_prefill_attn;
the single-launch path is taken exactly when the cache is bf16, the tiles are 128 or 256
columns and every prefix is page-aligned, and both paths match the oracle."""
import numpy as np
import pytest
import torch

import paper_2604_16395_amd as s2l
import workloads
from oracle.paged_kv import ref_append
from tests.gpu_util import DEV, SCALE, Setup, assert_attention_close, to_bf16

pytestmark = pytest.mark.gpu

FORCE_SPLIT = dict(target_items=1 << 20, min_split_keys=64, max_splits=16)


def _run(case, opts, fused_call):
    s = Setup(case)
    c = case
    T, hq = c.total_tokens, c.num_q_heads
    ws = torch.empty(s2l.s2l_attn_workspace_bytes(s.batch, hq, c.num_kv_heads, opts), dtype=torch.uint8, device=DEV)
    plan = s2l.s2l_attn_plan(s.batch, hq, c.num_kv_heads, ws, opts)
    out = torch.full((T, hq, 128), float("nan"), dtype=torch.bfloat16, device=DEV)
    lse = torch.full((T, hq), float("nan"), dtype=torch.float32, device=DEV)
    k_new, v_new = to_bf16(s.k_new), to_bf16(s.v_new)
    if fused_call:
        used = s2l.s2l_append_chunk_prefill_attn(s.cache, s.batch, k_new, v_new, s.q, hq, SCALE, out, lse, plan, ws)
    else:
        s2l.s2l_kv_append(s.cache, s.batch, k_new, v_new)
        s2l.s2l_chunk_prefill_attn(s.cache, s.batch, s.q, hq, SCALE, out, lse, plan, ws)
        used = None
    torch.cuda.synchronize()
    return s, out, lse, used


CASES = [
    ("aligned_8k", [8192], [512], 32, 8),
    ("aligned_varlen", [0, 16, 4096, 320, 64], [33, 129, 300, 1, 64], 32, 8),
    ("aligned_g8", [2048, 0], [200, 77], 64, 8),
    ("unaligned", [17, 4000], [100, 31], 32, 8),
]


MATRIX = [(c, split, layout) for c in CASES for split in (False, True)
          for layout in ([(256, 1), (128, 1), (128, 2)] if c[0] == "aligned_varlen" else [(256, 1)])]


@pytest.mark.parametrize("case_spec,split,layout", MATRIX)
def test_fused_equals_separate_calls(case_spec, split, layout):
    name, P, C, hq, hkv = case_spec
    case = workloads.make_case(name, P, C, hq, hkv, seed=41)
    opts = s2l.plan_opts(tile_cols=layout[0], key_halves=layout[1], **(FORCE_SPLIT if split else {}))
    print(f"[fused] {name} split={split} layout={layout}", flush=True)
    a, oa, la, used = _run(case, opts, True)
    b, ob, lb, _ = _run(case, opts, False)
    assert used == all(p % 16 == 0 for p in P)
    assert torch.equal(a.cache.k_pages.view(torch.int16), b.cache.k_pages.view(torch.int16))
    assert torch.equal(a.cache.v_pages.view(torch.int16), b.cache.v_pages.view(torch.int16))
    assert torch.equal(oa.view(torch.int16), ob.view(torch.int16)) and torch.equal(la, lb)
    # the oracle's pools take the chunk too
    ref_append(a.kp_ref, a.vp_ref, a.tables, case.prefix_lens, case.chunk_lens, case.cu_chunk, a.k_new, a.v_new)
    assert_attention_close(case, oa, la, a.oracle(), what=name)


def test_fused_call_falls_back_for_fp8_and_decode_tiles():
    case = workloads.make_case("fp8", [512, 0], [64, 16], 64, 8, seed=43, kv_dtype="fp8")
    s = Setup(case)
    hq = case.num_q_heads
    ws = torch.empty(s2l.s2l_attn_workspace_bytes(s.batch, hq, 8), dtype=torch.uint8, device=DEV)
    plan = s2l.s2l_attn_plan(s.batch, hq, 8, ws)
    out = torch.empty((case.total_tokens, hq, 128), dtype=torch.bfloat16, device=DEV)
    lse = torch.empty((case.total_tokens, hq), dtype=torch.float32, device=DEV)
    used = s2l.s2l_append_chunk_prefill_attn(s.cache, s.batch, to_bf16(s.k_new), to_bf16(s.v_new), s.q, hq, SCALE,
                                             out, lse, plan, ws)
    torch.cuda.synchronize()
    assert not used
    ref_append(s.kp_ref, s.vp_ref, s.tables, case.prefix_lens, case.chunk_lens, case.cu_chunk, s.k_new, s.v_new,
               case.kv_dtype, case.k_scale, case.v_scale)
    assert_attention_close(case, out, lse, s.oracle(), what="fp8 fallback")
    dec = workloads.make_case("dec", [4096, 64], [1, 1], 32, 8, seed=44)
    a, oa, la, used = _run(dec, None, True)
    b, ob, lb, _ = _run(dec, None, False)
    assert not used                                # 16-column decode tiles: two calls
    assert torch.equal(oa.view(torch.int16), ob.view(torch.int16)) and torch.equal(la, lb)
