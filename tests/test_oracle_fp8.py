"""Pins of the oracle's OCP E4M3 codec (CPU only)."""
import json
import os

import numpy as np
import pytest
import torch

from oracle.fp8_e4m3 import e4m3_decode, e4m3_encode, quantise_kv, quantize_rows

GOLD = os.path.join(os.path.dirname(__file__), "golden", "ocp_e4m3_named_values.json")
ALL = np.arange(256, dtype=np.uint8)


def test_named_values_from_the_ocp_table():
    g = json.load(open(GOLD))
    for e in g["values"]:
        v = e4m3_decode(np.array([e["code"]], dtype=np.uint8))[0]
        assert v == e["value"] and np.signbit(v) == np.signbit(e["value"]), e
        assert e4m3_encode(np.array([e["value"]]))[0] == e["code"], e
    for c in g["nan_codes"]:
        assert np.isnan(e4m3_decode(np.array([c], dtype=np.uint8))[0])


def test_decode_matches_torch_float8_e4m3fn_for_every_code():
    ours = e4m3_decode(ALL)
    theirs = torch.from_numpy(ALL.copy()).view(torch.float8_e4m3fn).to(torch.float64).numpy()
    assert np.array_equal(np.isnan(ours), np.isnan(theirs))
    m = ~np.isnan(ours)
    assert np.array_equal(ours[m], theirs[m])
    assert np.array_equal(np.signbit(ours[m]), np.signbit(theirs[m]))


def test_encode_inverts_decode():
    vals = e4m3_decode(ALL)
    m = ~np.isnan(vals)
    assert np.array_equal(e4m3_encode(vals[m]), ALL[m])


def _brute_force_encode(x):
    """Nearest finite E4M3 value by exhaustive search; ties -> even code; |x|>448 -> 448."""
    codes = np.arange(0, 0x7F, dtype=np.uint8)             # non-negative finite codes 0..126
    mags = e4m3_decode(codes)
    out = np.empty(len(x), dtype=np.uint8)
    for n, v in enumerate(x):
        if np.isnan(v):
            out[n] = 0xFF if np.signbit(v) else 0x7F
            continue
        a = min(abs(v), 448.0)
        dist = np.abs(mags - a)
        best = np.flatnonzero(dist == dist.min())
        c = best[0] if len(best) == 1 else [b for b in best if b % 2 == 0][0]
        out[n] = c | (0x80 if np.signbit(v) else 0)
    return out


def test_encode_every_bf16_pattern_against_brute_force():
    bits = np.arange(1 << 16, dtype=np.uint32) << 16
    with np.errstate(invalid="ignore"):            # the signalling-NaN patterns widen to NaN
        x = bits.view(np.float32).astype(np.float64)
    ours = e4m3_encode(x)
    # brute force on a strided subset plus every pattern around the binade edges
    pick = np.unique(np.concatenate([np.arange(0, 1 << 16, 7),
                                     np.flatnonzero(np.abs(x) > 400),
                                     np.flatnonzero((np.abs(x) > 0) & (np.abs(x) < 0.03))]))
    ref = _brute_force_encode(x[pick])
    nan = np.isnan(x[pick])
    assert np.array_equal(ours[pick][~nan], ref[~nan])
    assert np.all((ours[pick][nan] & 0x7F) == 0x7F)


def test_encode_matches_torch_inside_the_finite_range():
    bits = np.arange(1 << 16, dtype=np.uint32) << 16
    x = bits.view(np.float32)
    m = np.isfinite(x) & (np.abs(x) <= 448.0)
    theirs = torch.from_numpy(x[m].copy()).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    assert np.array_equal(e4m3_encode(x[m].astype(np.float64)), theirs)


def test_saturation_and_nan():
    big = np.array([448.0, 449.0, 463.9, 464.0, 470.0, 1e30, np.inf, -np.inf, -1e9])
    assert list(e4m3_encode(big)) == [0x7E] * 7 + [0xFE, 0xFE]
    assert e4m3_encode(np.array([np.nan]))[0] & 0x7F == 0x7F


def test_round_half_to_even_at_a_midpoint():
    # 1.0 (0x38, mantissa 000) and 1.125 (0x39): midpoint 1.0625 -> even mantissa -> 0x38
    assert e4m3_encode(np.array([1.0625]))[0] == 0x38
    # 1.125 (0x39) and 1.25 (0x3A): midpoint 1.1875 -> 0x3A
    assert e4m3_encode(np.array([1.1875]))[0] == 0x3A
    # subnormal midpoint between 1 and 2 quanta of 2^-9 -> 2 (even)
    assert e4m3_encode(np.array([1.5 * 2.0 ** -9]))[0] == 0x02


@pytest.mark.parametrize("scale", [0.25, 2.0 ** -7, 3.0])
def test_quantise_with_power_of_two_and_generic_scale(scale):
    rng = np.random.default_rng(7)
    x = (rng.standard_normal((5, 2, 16)).astype(np.float32) * 0.5)
    q = quantise_kv(x, np.array([scale, scale], dtype=np.float32))
    # the float32 product x * (1/scale), then RNE; check via decode that the code is nearest
    y = x.astype(np.float32) * (np.float32(1) / np.float32(scale))
    dec = e4m3_decode(q)
    assert np.array_equal(q.reshape(-1), _brute_force_encode(y.astype(np.float64).reshape(-1)))
    if scale in (0.25, 2.0 ** -7):
        # power-of-two scale: the product is exact, so decode*scale equals RNE(x) exactly
        assert np.allclose(dec * scale, e4m3_decode(e4m3_encode(x / scale)) * scale, rtol=0, atol=0)


# --- per-row quantisation of Q (the quantised-Q attention variant) ---------------------------

def test_rows_of_exact_codes_with_a_power_of_two_scale_round_trip():
    """A row made of e4m3 values times 2^k whose largest magnitude is 448 * 2^k has scale
    2^k exactly, so every element comes back unchanged."""
    rng = np.random.default_rng(11)
    finite = ALL[(ALL & 0x7F) != 0x7F]
    for k in (-9, -3, 0, 2):
        codes = rng.choice(finite, size=(6, 128))
        codes[:, 5] = 0x7E                               # +448 in every row
        x = (e4m3_decode(codes) * 2.0 ** k).astype(np.float32)
        c, s, d = quantize_rows(x)
        assert np.all(s == np.float32(2.0 ** k))
        assert np.array_equal(d, x.astype(np.float64))


def test_row_quantisation_error_within_the_e4m3_bound():
    """Round to nearest in E4M3: within half a quantum, i.e. 2^-4 relative in the normal range
    (scaled |x| >= 2^-6) and 2^-10 absolute (times the scale) below it; the fp32 product
    before rounding adds at most 2^-23 relative."""
    rng = np.random.default_rng(12)
    x = (rng.standard_normal((64, 128)) * rng.choice([0.01, 0.5, 30.0], size=(64, 1))).astype(np.float32)
    x[3, :] = np.float32(0.0)
    x[4, 7] = np.float32(1e-3)                           # one tiny element among zeros
    x[4, :7] = 0
    x[4, 8:] = 0
    c, s, d = quantize_rows(x)
    xs = np.abs(x.astype(np.float64)) / s[:, None]
    err = np.abs(d - x.astype(np.float64)) / s[:, None]
    normal = xs >= 2.0 ** -6
    assert np.all(err[normal] <= (2.0 ** -4 + 2.0 ** -22) * xs[normal])
    assert np.all(err[~normal] <= 2.0 ** -10 + 2.0 ** -22 * xs[~normal])
    # the largest element of a non-zero row is 448 * scale (code 0x7E or 0xFE); a zero row
    # has scale 1 and zero codes
    nz = np.abs(x).max(axis=1) > 0
    amax_idx = np.abs(x).argmax(axis=1)
    assert np.all((c[np.arange(64), amax_idx][nz] & 0x7F) == 0x7E)
    assert s[3] == 1.0 and not c[3].any() and not d[3].any()


def test_row_quantisation_is_odd_and_commutes_with_powers_of_two():
    rng = np.random.default_rng(13)
    x = (rng.standard_normal((8, 128)) * 0.5).astype(np.float32)
    c, s, d = quantize_rows(x)
    cn, sn, dn = quantize_rows(-x)
    assert np.array_equal(cn, c ^ 0x80) and np.array_equal(sn, s) and np.array_equal(dn, -d)
    c4, s4, d4 = quantize_rows(x * np.float32(16.0))
    assert np.array_equal(c4, c) and np.array_equal(s4, s * np.float32(16.0)) and np.array_equal(d4, 16.0 * d)
