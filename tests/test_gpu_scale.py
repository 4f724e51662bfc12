"""GPU: softmax scales other than 1/sqrt(d), against the oracle.  The scale is a call argument
(the paper leaves it open); the kernels fold it into the exp2 argument of every score, with
log2 e, and for e4m3 caches with the kv head's K scale, for quantised Q with each row's Q scale.
Every other parity test runs at 1/sqrt(128), so these cases pin the folding itself: the main
kernel (bf16, e4m3 pages, quantised Q; split and unsplit) and the decode kernel, at a scale that
flattens the softmax, one that sharpens it, and 1."""
import pytest

import paper_2604_16395_amd as s2l
import workloads
from tests.gpu_util import Setup, assert_attention_close

pytestmark = pytest.mark.gpu

SCALES = [0.02, 0.3, 1.0]
FORCE_SPLIT = dict(target_items=1 << 20, min_split_keys=64, max_splits=16)


@pytest.mark.parametrize("scale", SCALES)
@pytest.mark.parametrize("split", [False, True])
@pytest.mark.parametrize("kv_dtype,q8", [("bf16", False), ("fp8", False), ("fp8", True)])
def test_main_kernel_at_other_scales(kv_dtype, q8, split, scale):
    case = workloads.make_case("scale", [700, 40], [200, 33], 32, 8, seed=50, kv_dtype=kv_dtype)
    s = Setup(case)
    s.append()
    opts = s2l.plan_opts(**(FORCE_SPLIT if split else {}))
    out, lse = s.attention(opts, q8=q8, scale=scale)
    assert s.plan.tile_cols != 16
    assert_attention_close(case, out, lse, s.oracle(q8=q8, scale=scale), what=f"scale {scale} {kv_dtype} q8={q8}")


@pytest.mark.parametrize("scale", SCALES)
@pytest.mark.parametrize("kv_dtype", ["bf16", "fp8"])
def test_decode_kernel_at_other_scales(kv_dtype, scale):
    case = workloads.make_case("scale_dec", [3000, 17, 900], [1, 1, 1], 32, 8, seed=51, kv_dtype=kv_dtype)
    s = Setup(case)
    s.append()
    out, lse = s.attention(scale=scale)
    assert s.plan.tile_cols == 16
    assert_attention_close(case, out, lse, s.oracle(scale=scale), what=f"decode scale {scale} {kv_dtype}")
