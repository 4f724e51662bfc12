"""GPU: one step of the path (append, plan, attention, split merge) captured into a HIP
graph and replayed gives the same bits as the eager calls, on every replay."""
import numpy as np
import pytest
import torch

import paper_2604_16395_amd as s2l
import workloads
from tests.gpu_util import DEV, SCALE, Setup, to_bf16

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("layout", [(256, 1), (128, 2)])
def test_graph_replays_equal_eager(layout):
    case = workloads.make_case("graph", [3000, 40], [300, 97], 32, 8, seed=21)
    s = Setup(case)
    hq, hkv, T = case.num_q_heads, case.num_kv_heads, case.total_tokens
    opts = s2l.plan_opts(tile_cols=layout[0], key_halves=layout[1], target_items=512)
    ws = torch.empty(s2l.s2l_attn_workspace_bytes(s.batch, hq, hkv, opts), dtype=torch.uint8, device=DEV)
    k_new, v_new = to_bf16(s.k_new), to_bf16(s.v_new)
    out = torch.empty((T, hq, 128), dtype=torch.bfloat16, device=DEV)
    lse = torch.empty((T, hq), dtype=torch.float32, device=DEV)
    stream = torch.cuda.Stream()

    def step():
        s2l.s2l_kv_append(s.cache, s.batch, k_new, v_new, stream)
        plan = s2l.s2l_attn_plan(s.batch, hq, hkv, ws, opts, stream)
        s2l.s2l_chunk_prefill_attn(s.cache, s.batch, s.q, hq, SCALE, out, lse, plan, ws, stream)
        return plan

    with torch.cuda.stream(stream):
        plan = step()
    torch.cuda.synchronize()
    assert plan.num_split_reqs > 0
    ref_out, ref_lse = out.clone(), lse.clone()

    g = torch.cuda.CUDAGraph()
    with torch.cuda.stream(stream):
        with torch.cuda.graph(g, stream=stream):
            step()
    torch.cuda.synchronize()
    for rep in range(3):
        out.fill_(float("nan"))
        lse.fill_(float("nan"))
        junk = torch.randn(1 << 20, device=DEV).sum()   # eager work between replays
        torch.cuda.synchronize()
        with torch.cuda.stream(stream):
            g.replay()
        torch.cuda.synchronize()
        assert torch.isfinite(junk)
        assert torch.equal(out.view(torch.int16), ref_out.view(torch.int16)), f"replay {rep}: out differs"
        assert torch.equal(lse, ref_lse), f"replay {rep}: lse differs"
