"""GPU: every finite e4m3 code through the attention kernels' widening to bf16.  One query row
with no prefix sees exactly one key, so its weight is exactly 1 and the output row is that
key's value row as the kernel decoded it (scale 1, so nothing is rounded).  The value rows of
the two kv heads hold the 254 finite codes (0x00-0x7E, 0x80-0xFE; NaN codes 0x7F and 0xFF
left out), written through the library's append (exact: each value is an e4m3 value).  The
decode kernel, the main kernel in its three layouts and the quantised-Q variant must return
the codes' values of the OCP E4M3 definition (the oracle's decoder) bit for bit; the unused
slots of the page hold NaN codes, which must not leak into the output."""
import numpy as np
import pytest
import torch

import paper_2604_16395_amd as s2l
from oracle.fp8_e4m3 import e4m3_decode
from tests.gpu_util import DEV, SCALE, bf16_to_f64, to_bf16

pytestmark = pytest.mark.gpu

HQ = HKV = 2
CODES = np.stack([np.r_[np.arange(0x00, 0x7F), 0x00], np.r_[np.arange(0x80, 0xFF), 0x80]]).astype(np.uint8)


def _bits_of(values):
    """bf16 bits of values that bf16 holds exactly."""
    f = values.astype(np.float32)
    bits = f.view(np.uint32)
    assert np.all(bits & 0xFFFF == 0)
    return (bits >> 16).astype(np.uint16)


@pytest.fixture(scope="module")
def layer():
    expect = e4m3_decode(CODES)                                # [2][128], exact
    assert np.isfinite(expect).all()
    v_new = _bits_of(expect)[None]                             # [1 token][2 heads][128]
    k_new = _bits_of(np.full((HKV, 128), 0.5))[None]
    kp = torch.full((1, HKV, 16, 128), 0x7F, dtype=torch.uint8, device=DEV)
    vp = torch.full((1, HKV, 16, 128), 0x7F, dtype=torch.uint8, device=DEV)
    ones = torch.ones(HKV, dtype=torch.float32, device=DEV)
    cache = s2l.PagedKVCache(kp, vp, ones, ones.clone())
    batch = s2l.Batch([0], [1], np.zeros((1, 1), np.int32))
    s2l.s2l_kv_append(cache, batch, to_bf16(k_new), to_bf16(v_new))
    torch.cuda.synchronize()
    assert np.array_equal(vp[0, :, 0].cpu().numpy(), CODES)   # the append stored the codes
    rng = np.random.default_rng(5)
    q_bits = (rng.standard_normal((1, HQ, 128)).astype(np.float32).view(np.uint32) >> 16).astype(np.uint16)
    return cache, batch, to_bf16(q_bits), expect


@pytest.mark.parametrize("how", ["planner", "128", "128x2", "256", "q8"])
def test_every_finite_code_decodes_exactly(layer, how):
    cache, batch, q, expect = layer
    opts = {"planner": None, "128": s2l.plan_opts(tile_cols=128, key_halves=1),
            "128x2": s2l.plan_opts(tile_cols=128, key_halves=2), "256": s2l.plan_opts(tile_cols=256),
            "q8": s2l.plan_opts(tile_cols=256)}[how]
    ws = torch.empty(s2l.s2l_attn_workspace_bytes(batch, HQ, HKV, opts), dtype=torch.uint8, device=DEV)
    plan = s2l.s2l_attn_plan(batch, HQ, HKV, ws, opts)
    out = torch.full((1, HQ, 128), float("nan"), dtype=torch.bfloat16, device=DEV)
    if how == "q8":
        s2l.s2l_chunk_prefill_attn_q8(cache, batch, q, HQ, SCALE, out, None, plan, ws)
    else:
        s2l.s2l_chunk_prefill_attn(cache, batch, q, HQ, SCALE, out, None, plan, ws)
    torch.cuda.synchronize()
    if how == "planner":
        assert plan.tile_cols == 16                          # one decode-shaped row: the decode kernel
    got = bf16_to_f64(out)[0]
    assert np.array_equal(got, expect), f"{how}: {np.count_nonzero(got != expect)} values differ"
