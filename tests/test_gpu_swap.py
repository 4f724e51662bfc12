"""GPU: swap-out / swap-in of KV pages between the device pools and pinned host pools
(Stream2LLM Sec. 4.3).  Pages move as bytes: every copied page must be bit-identical, and
no other page on either side may change."""
import numpy as np
import pytest
import torch

import paper_2604_16395_amd as s2l
from paper_2604_16395_amd import _lib

pytestmark = pytest.mark.gpu
DEV = "cuda"


def _pools(num_pages, hkv, fp8, seed):
    g = torch.Generator(device="cpu").manual_seed(seed)
    shape = (num_pages, hkv, 16, 128)
    if fp8:
        k = torch.randint(0, 256, shape, dtype=torch.uint8, generator=g)
        v = torch.randint(0, 256, shape, dtype=torch.uint8, generator=g)
    else:
        k = torch.randint(-32768, 32768, shape, dtype=torch.int16, generator=g).view(torch.bfloat16)
        v = torch.randint(-32768, 32768, shape, dtype=torch.int16, generator=g).view(torch.bfloat16)
    return k, v


def _bits(t):
    return t.view(torch.uint8) if t.dtype == torch.uint8 else t.view(torch.int16)


def _cache(k, v, fp8):
    ks = vs = None
    if fp8:
        ks = torch.ones(k.shape[1], dtype=torch.float32, device=DEV)
        vs = torch.ones(k.shape[1], dtype=torch.float32, device=DEV)
    return s2l.PagedKVCache(k, v, ks, vs)


@pytest.mark.parametrize("fp8,hkv", [(False, 8), (True, 8), (False, 1)])
def test_swap_round_trip_is_bit_exact(fp8, hkv):
    nd, nh = 96, 64
    kd0, vd0 = _pools(nd, hkv, fp8, 1)
    kh0, vh0 = _pools(nh, hkv, fp8, 2)
    kd, vd = kd0.to(DEV), vd0.to(DEV)
    kh, vh = kh0.clone().pin_memory(), vh0.clone().pin_memory()
    cache = _cache(kd, vd, fp8)
    rng = np.random.default_rng(3)
    dev_pages = torch.as_tensor(rng.choice(nd, 40, replace=False))
    host_pages = torch.as_tensor(rng.choice(nh, 40, replace=False))
    out_pairs = torch.stack([dev_pages, host_pages], 1).to(torch.int32).to(DEV)
    s2l.s2l_kv_swap_out(cache, out_pairs, kh, vh)
    torch.cuda.synchronize()
    kh_exp, vh_exp = kh0.clone(), vh0.clone()
    kh_exp[host_pages] = kd0[dev_pages]
    vh_exp[host_pages] = vd0[dev_pages]
    assert torch.equal(_bits(kh), _bits(kh_exp)) and torch.equal(_bits(vh), _bits(vh_exp))
    # back in, to other device pages
    back = torch.as_tensor(rng.choice(nd, 40, replace=False))
    in_pairs = torch.stack([host_pages, back], 1).to(torch.int32).to(DEV)
    s2l.s2l_kv_swap_in(cache, in_pairs, kh, vh)
    torch.cuda.synchronize()
    kd_exp, vd_exp = kd0.clone(), vd0.clone()
    kd_exp[back] = kd0[dev_pages]
    vd_exp[back] = vd0[dev_pages]
    assert torch.equal(_bits(kd.cpu()), _bits(kd_exp)) and torch.equal(_bits(vd.cpu()), _bits(vd_exp))


def test_swap_skips_pairs_out_of_range():
    nd, nh, hkv = 8, 4, 2
    kd0, vd0 = _pools(nd, hkv, False, 5)
    kd, vd = kd0.to(DEV), vd0.to(DEV)
    kh = torch.zeros((nh, hkv, 16, 128), dtype=torch.bfloat16).pin_memory()
    vh = torch.zeros_like(kh).pin_memory()
    cache = _cache(kd, vd, False)
    pairs = torch.tensor([[1, 0], [nd, 1], [-1, 2], [2, nh], [3, 3]], dtype=torch.int32, device=DEV)
    s2l.s2l_kv_swap_out(cache, pairs, kh, vh)
    torch.cuda.synchronize()
    assert torch.equal(_bits(kh[0]), _bits(kd0[1])) and torch.equal(_bits(kh[3]), _bits(kd0[3]))
    assert not _bits(kh[1]).any() and not _bits(kh[2]).any()


def test_swap_rejects_unpinned_host_memory():
    kd, vd = _pools(4, 2, False, 6)
    cache = _cache(kd.to(DEV), vd.to(DEV), False)
    kh = torch.zeros((4, 2, 16, 128), dtype=torch.bfloat16)      # pageable
    pairs = torch.tensor([[0, 0]], dtype=torch.int32, device=DEV)
    with pytest.raises(_lib.S2LError) as e:
        s2l.s2l_kv_swap_out(cache, pairs, kh, kh.clone())
    assert e.value.status == _lib.S2L_EINVAL
