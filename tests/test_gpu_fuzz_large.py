"""GPU: seeded random batches of larger requests against the oracle on dense rows.  Each case
draws 1-4 requests with prefixes up to 20K tokens (most ragged, some page-aligned) and chunks of
1-2048 tokens (log-uniform), a head layout (G from 1 to 16), bf16 or e4m3 pages (and for e4m3
the quantised-Q call or not), a tile layout or the planner's choice, and a forced key split or
not.  Every 32nd chunk row and each chunk's first and last rows are checked against the oracle
with the bound of every other parity test (the spread term bounded by the triangle inequality)."""
import numpy as np
import pytest

import paper_2604_16395_amd as s2l
import workloads
from tests.gpu_util import Setup, assert_attention_close, dense_rows
from tests.test_gpu_fuzz import LAYOUTS, MORE_HEADS

pytestmark = pytest.mark.gpu

NUM_CASES = 16


def draw(seed):
    rng = np.random.default_rng(50_000 + seed)
    R = int(rng.integers(1, 5))
    P = [int(rng.integers(0, 20000)) if rng.random() < 0.8 else 16 * int(rng.integers(0, 1200)) for _ in range(R)]
    C = [int(max(1, min(2048, np.exp(rng.uniform(0, 7.7))))) for _ in range(R)]
    hq, hkv = MORE_HEADS[int(rng.integers(0, len(MORE_HEADS)))]
    kv = "fp8" if rng.random() < 0.35 else "bf16"
    q8 = kv == "fp8" and rng.random() < 0.5
    layout = LAYOUTS[int(rng.integers(0, len(LAYOUTS)))]
    if q8 and layout is None:
        layout = (256, 1)      # quantised Q runs on the wide-tile kernel only
    split = bool(rng.random() < 0.5)
    return P, C, hq, hkv, kv, q8, layout, split


@pytest.mark.parametrize("seed", range(NUM_CASES))
def test_large_random_batch_matches_the_oracle(seed):
    P, C, hq, hkv, kv, q8, layout, split = draw(seed)
    case = workloads.make_case(f"fuzz_large{seed}", P, C, hq, hkv, seed=seed, kv_dtype=kv)
    s = Setup(case)
    s.append()
    kw = {}
    if layout is not None:
        kw.update(tile_cols=layout[0], key_halves=layout[1])
    if split:
        kw.update(target_items=1 << 20, min_split_keys=64, max_splits=16)
    out, lse = s.attention(s2l.plan_opts(**kw), q8=q8)
    rows = dense_rows(case, 32)
    what = (f"fuzz large {seed}: P={P} C={C} heads {hq}/{hkv} {kv} q8={q8} layout={layout} split={split} "
            f"-> {s.plan.tile_cols}-column tiles, {s.plan.num_items} items")
    print(what, flush=True)
    assert_attention_close(case, out, lse, s.oracle(sample_rows=rows, q8=q8, spread=False), rows=rows, what=what)
