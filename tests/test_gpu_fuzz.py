"""GPU: seeded random batches against the oracle on every row.  Each case draws from its own
seed a request count, prefix and chunk lengths (zero, page-aligned, ragged and one- or
two-token chunks among them, and now and then a request with no new tokens), a head layout
(G = 1, 2, 3, 4 or 8; in a second set also 5, 6, 7, 12 and 16, with one or two kv heads among
them), the page dtype, the tile layout or the planner's choice, a forced key
split or not, and for e4m3 pages the quantised-Q call.  Whatever the plan selects (the main
kernel in one of its three layouts, or the decode kernel for 16-column plans) runs through the
C ABI and is checked with the same bound as every other parity test."""
import numpy as np
import pytest

import paper_2604_16395_amd as s2l
import workloads
from tests.gpu_util import Setup, assert_attention_close

pytestmark = pytest.mark.gpu

HEADS = [(8, 8), (16, 8), (24, 8), (32, 8), (64, 8), (8, 4), (12, 4), (16, 4), (32, 4)]
MORE_HEADS = HEADS + [(32, 2), (16, 1), (40, 8), (56, 8), (6, 1), (48, 4), (24, 2)]
LAYOUTS = [None, (256, 1), (128, 1), (128, 2)]
NUM_CASES = 48
NUM_MORE = 24


def draw(seed, heads=HEADS):
    rng = np.random.default_rng(10_000 + seed)
    R = int(rng.integers(1, 6))
    P = []
    for _ in range(R):
        kind = int(rng.integers(0, 4))
        P.append(0 if kind == 0 else 16 * int(rng.integers(1, 160)) if kind == 1 else int(rng.integers(1, 2500)))
    decode = rng.random() < 0.25
    C = [int(rng.integers(1, 3)) if decode else int(max(1.0, min(600.0, np.exp(rng.uniform(0.0, 6.4)))))
         for _ in range(R)]
    if R > 1 and rng.random() < 0.2:
        C[int(rng.integers(0, R))] = 0
    hq, hkv = heads[int(rng.integers(0, len(heads)))]
    kv = "fp8" if rng.random() < 0.35 else "bf16"
    q8 = kv == "fp8" and rng.random() < 0.5
    layout = LAYOUTS[int(rng.integers(0, len(LAYOUTS)))]
    if q8 and layout is None:
        layout = (256, 1)      # quantised Q runs on the wide-tile kernel only (not on 16-column plans)
    split = bool(rng.random() < 0.5)
    return P, C, hq, hkv, kv, q8, layout, split


@pytest.mark.parametrize("seed", range(NUM_CASES))
def test_random_batch_matches_the_oracle(seed):
    _run(seed, HEADS)


@pytest.mark.parametrize("seed", range(NUM_CASES, NUM_CASES + NUM_MORE))
def test_random_batch_more_head_layouts(seed):
    _run(seed, MORE_HEADS)


def _run(seed, heads):
    P, C, hq, hkv, kv, q8, layout, split = draw(seed, heads)
    case = workloads.make_case(f"fuzz{seed}", P, C, hq, hkv, seed=seed, kv_dtype=kv)
    s = Setup(case)
    s.append()
    kw = {}
    if layout is not None:
        kw.update(tile_cols=layout[0], key_halves=layout[1])
    if split:
        kw.update(target_items=1 << 20, min_split_keys=64, max_splits=16)
    out, lse = s.attention(s2l.plan_opts(**kw), q8=q8)
    what = (f"fuzz {seed}: P={P} C={C} heads {hq}/{hkv} {kv} q8={q8} layout={layout} split={split} "
            f"-> {s.plan.tile_cols}-column tiles, {s.plan.num_items} items")
    print(what, flush=True)
    assert_attention_close(case, out, lse, s.oracle(q8=q8), what=what)
