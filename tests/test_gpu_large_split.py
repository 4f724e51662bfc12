"""GPU: split partials on both sides of the 2 GiB limit of the staged store.  The wide-tile
kernel stages a split piece's fp32 partial through LDS and stores it with a buffer resource
whose byte offsets are 32-bit, so a request whose partials exceed 2^31 - 1 bytes takes the
direct store from the registers instead.  One 8192-token chunk (32q/8kv, bf16 pages) planned
with 16 pieces per tile has 2.2 GB of partials (direct path); with 8 pieces, 1.1 GB (staged
path).  Both outputs are checked against the oracle on a dense row set."""
import numpy as np
import pytest

import paper_2604_16395_amd as s2l
import workloads
from tests.gpu_util import Setup, assert_attention_close, count_rows, dense_rows

pytestmark = pytest.mark.gpu

LIMIT = (1 << 31) - 1
P, C, HQ, HKV = 256, 8192, 32, 8


@pytest.fixture(scope="module")
def setup():
    case = workloads.make_case("large_split", [P], [C], HQ, HKV, seed=77)
    s = Setup(case)
    s.append()
    rows = dense_rows(case, stride=64, chunk=512)
    return s, rows, s.oracle(sample_rows=rows)


@pytest.mark.parametrize("max_splits,over", [(16, True), (8, False)])
def test_partials_past_and_below_2gib(setup, max_splits, over):
    s, rows, ref = setup
    opts = s2l.plan_opts(target_items=1 << 20, min_split_keys=64, max_splits=max_splits, tile_cols=256,
                         key_halves=1)
    out, lse = s.attention(opts)
    part_bytes = s.plan.part_floats * 4
    print(f"[large split] {max_splits} pieces per tile: {s.plan.num_items} items, {part_bytes / 1e9:.2f} GB "
          f"of partials, {count_rows(rows)} oracle rows", flush=True)
    assert s.plan.tile_cols == 256 and s.plan.split_keys > 0
    assert (part_bytes > LIMIT) == over
    assert_attention_close(s.case, out, lse, ref, rows=rows, what=f"{max_splits} pieces, {part_bytes} bytes")
