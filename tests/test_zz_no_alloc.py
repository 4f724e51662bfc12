"""GPU: the allocation-free attention call (s2l_chunk_prefill_attn_noalloc), whose plan and
split partials live in the library's own scratch array, against the workspace call
(s2l_attn_plan + s2l_chunk_prefill_attn) on the same inputs: two calls in a row, the second
with a smaller batch (the scratch keeps the first call's contents), each bit-identical to the
workspace call (same plan, same kernels) and within the oracle's bound on sampled rows."""
import numpy as np
import pytest
import torch

import paper_2604_16395_amd as s2l
import workloads
from tests.gpu_util import DEV, SCALE, Setup, assert_attention_close, sample_rows

pytestmark = pytest.mark.gpu

CASES = [
    ("p8192_c512", [8192], [512], 32, 8),                       # split: the 33 MiB plan of the 8K step
    ("varlen_small", [300, 40, 1000], [77, 1, 129], 32, 8),     # smaller, unsplit
]


def test_noalloc_call_equals_the_workspace_call_twice_in_a_row():
    for name, P, C, hq, hkv in CASES:
        print(f"[noalloc] {name}", flush=True)
        case = workloads.make_case(name, P, C, hq, hkv, seed=60)
        s = Setup(case)
        s.append()
        ref_out, ref_lse = s.attention()                         # caller workspace
        out = torch.full_like(ref_out, float("nan"))
        lse = torch.full_like(ref_lse, float("nan"))
        info = s2l.s2l_chunk_prefill_attn_noalloc(s.cache, s.batch, s.q, hq, SCALE, out, lse)
        torch.cuda.synchronize()
        assert info.num_items == s.plan.num_items and info.num_split_reqs == s.plan.num_split_reqs
        assert info.workspace_bytes <= s2l.NOALLOC_SCRATCH_BYTES
        assert torch.equal(out.view(torch.int16), ref_out.view(torch.int16))
        assert torch.equal(lse, ref_lse)
        rows = sample_rows(case, 24, np.random.default_rng(61))
        assert_attention_close(case, out, lse, s.oracle(rows), rows, what=f"noalloc {name}")
