"""GPU: pages past the first 4 GiB of a pool.  A production pool on one 288 GB device is far
larger than 4 GiB, so every byte offset of a page must be formed in 64 bits.  Each case runs
twice on the GPU: in a small pool, and in a pool of just over 4 GiB per K/V tensor whose even
logical pages lie above the 4 GiB mark and odd ones below (so each request's pages straddle
it).  Pages, gathered rows, swapped pages and attention outputs must agree bit for bit; the
large-pool attention is also checked against the oracle."""
import numpy as np
import pytest
import torch

import paper_2604_16395_amd as s2l
import workloads
from tests.gpu_util import DEV, SCALE, Setup, assert_attention_close, to_bf16
from workloads import BF16_SENTINEL, FP8_SENTINEL

pytestmark = pytest.mark.gpu

MARK = 1 << 32                      # bytes


def _bits(t):
    return t.view(torch.uint8) if t.dtype == torch.uint8 else t.view(torch.int16)


class Run:
    """The case's prefix and chunk appended by the GPU into a small or a large pool."""

    def __init__(self, case, large):
        self.case = case
        fp8 = case.kv_dtype == "fp8"
        page_bytes = case.num_kv_heads * 16 * 128 * (1 if fp8 else 2)
        base = MARK // page_bytes if large else 0
        tables = case.block_tables.astype(np.int64)
        if large:
            lp = np.arange(tables.shape[1])[None, :]
            tables = np.where(lp % 2 == 0, tables + base, tables)
            assert tables.max() * page_bytes >= MARK
        self.base = base
        self.tables = tables.astype(np.int32)
        shape = (base + case.num_pages, case.num_kv_heads, 16, 128)
        if fp8:
            kp = torch.full(shape, FP8_SENTINEL, dtype=torch.uint8, device=DEV)
            vp = torch.full(shape, FP8_SENTINEL, dtype=torch.uint8, device=DEV)
            ks, vs = torch.from_numpy(case.k_scale).to(DEV), torch.from_numpy(case.v_scale).to(DEV)
        else:
            kp = torch.full(shape, BF16_SENTINEL, dtype=torch.int16, device=DEV).view(torch.bfloat16)
            vp = torch.full(shape, BF16_SENTINEL, dtype=torch.int16, device=DEV).view(torch.bfloat16)
            ks = vs = None
        if large:
            assert kp.numel() * kp.element_size() > MARK
        self.cache = s2l.PagedKVCache(kp, vp, ks, vs)
        R = case.num_reqs
        pre = s2l.Batch(np.zeros(R, np.int32), case.prefix_lens, self.tables)
        if case.prefix_lens.sum():
            s2l.s2l_kv_append(self.cache, pre, to_bf16(case.prefix_rows(case.k_full_bits)),
                              to_bf16(case.prefix_rows(case.v_full_bits)))
        self.batch = s2l.Batch(case.prefix_lens, case.chunk_lens, self.tables)
        self.k_new = to_bf16(case.new_rows(case.k_full_bits))
        self.v_new = to_bf16(case.new_rows(case.v_full_bits))
        self.q = to_bf16(case.q_bits)

    def append(self):
        s2l.s2l_kv_append(self.cache, self.batch, self.k_new, self.v_new)

    def gather(self):
        c = self.case
        n = c.prefix_lens + c.chunk_lens
        cu = np.zeros(c.num_reqs + 1, np.int32)
        cu[1:] = np.cumsum(n)
        ko = torch.empty((int(cu[-1]), c.num_kv_heads, 128), dtype=self.cache.k_pages.dtype, device=DEV)
        vo = torch.empty_like(ko)
        s2l.s2l_kv_gather(self.cache, self.batch, 1, torch.from_numpy(cu).to(DEV), ko, vo)
        torch.cuda.synchronize()
        return ko, vo

    def attention(self, how="plain", opts=None):
        c = self.case
        hq = c.num_q_heads
        ws = torch.empty(s2l.s2l_attn_workspace_bytes(self.batch, hq, c.num_kv_heads, opts), dtype=torch.uint8,
                         device=DEV)
        plan = s2l.s2l_attn_plan(self.batch, hq, c.num_kv_heads, ws, opts)
        out = torch.full((c.total_tokens, hq, 128), float("nan"), dtype=torch.bfloat16, device=DEV)
        lse = torch.full((c.total_tokens, hq), float("nan"), dtype=torch.float32, device=DEV)
        if how == "fused":
            assert s2l.s2l_append_chunk_prefill_attn(self.cache, self.batch, self.k_new, self.v_new, self.q, hq,
                                                     SCALE, out, lse, plan, ws)
        elif how == "q8":
            s2l.s2l_chunk_prefill_attn_q8(self.cache, self.batch, self.q, hq, SCALE, out, lse, plan, ws)
        else:
            s2l.s2l_chunk_prefill_attn(self.cache, self.batch, self.q, hq, SCALE, out, lse, plan, ws)
        torch.cuda.synchronize()
        self.plan = plan
        return out, lse


CASES = {
    "prefill": lambda: workloads.make_case("big_prefill", [700, 33, 0], [300, 90, 64], 32, 8, seed=31),
    "aligned": lambda: workloads.make_case("big_aligned", [704, 32], [300, 90], 32, 8, seed=32),
    "decode": lambda: workloads.make_case("big_decode", [5000, 300, 17], [1, 1, 1], 32, 8, seed=33),
    "fp8": lambda: workloads.make_case("big_fp8", [700, 0, 33], [130, 77, 1], 64, 8, seed=34, kv_dtype="fp8"),
}
FORCE_SPLIT = dict(target_items=1 << 20, min_split_keys=64, max_splits=16)


@pytest.mark.parametrize("name,how,split", [
    ("prefill", "plain", False), ("prefill", "plain", True), ("aligned", "fused", False),
    ("decode", "plain", False), ("decode", "plain", True), ("fp8", "plain", True), ("fp8", "q8", False),
])
def test_pages_past_4gib_give_the_same_bits(name, how, split):
    case = CASES[name]()
    print(f"[large pool] {name} {how} split={split}", flush=True)
    opts = s2l.plan_opts(**FORCE_SPLIT) if split else None
    outs = []
    for large in (False, True):
        r = Run(case, large)
        if how != "fused":
            r.append()
        outs.append(r.attention(how, opts) + r.gather())
        if split:
            assert r.plan.num_split_reqs > 0
        del r
        torch.cuda.empty_cache()
    (o0, l0, k0, v0), (o1, l1, k1, v1) = outs
    assert torch.equal(_bits(k0), _bits(k1)) and torch.equal(_bits(v0), _bits(v1)), "pages differ"
    assert torch.equal(o0.view(torch.int16), o1.view(torch.int16)) and torch.equal(l0, l1), "outputs differ"
    s = Setup(case)
    s.append()
    ref = s.oracle(q8=how == "q8")
    assert_attention_close(case, o1, l1, ref, what=f"large pool {name} {how}")


@pytest.mark.parametrize("fp8", [False, True])
def test_swap_of_pages_past_4gib(fp8):
    case = CASES["fp8" if fp8 else "prefill"]()
    r = Run(case, True)
    r.append()
    used = np.unique(r.tables[r.tables >= r.base])[:12]
    n = len(used)
    hk = torch.zeros((n, case.num_kv_heads, 16, 128), dtype=r.cache.k_pages.dtype).pin_memory()
    hv = torch.zeros_like(hk).pin_memory()
    pairs = torch.tensor(np.stack([used, np.arange(n)], 1), dtype=torch.int32, device=DEV)
    s2l.s2l_kv_swap_out(r.cache, pairs, hk, hv)
    torch.cuda.synchronize()
    idx = torch.from_numpy(used.astype(np.int64)).to(DEV)
    assert torch.equal(_bits(hk), _bits(r.cache.k_pages[idx].cpu()))
    assert torch.equal(_bits(hv), _bits(r.cache.v_pages[idx].cpu()))
    # back in, to pages past the mark that no table entry names
    dst = np.setdiff1d(r.base + np.arange(case.num_pages), r.tables)[:n]
    assert len(dst) == n
    back = torch.tensor(np.stack([np.arange(n), dst], 1), dtype=torch.int32, device=DEV)
    s2l.s2l_kv_swap_in(r.cache, back, hk, hv)
    torch.cuda.synchronize()
    didx = torch.from_numpy(dst.astype(np.int64)).to(DEV)
    assert torch.equal(_bits(r.cache.k_pages[didx]), _bits(r.cache.k_pages[idx]))
    assert torch.equal(_bits(r.cache.v_pages[didx]), _bits(r.cache.v_pages[idx]))
