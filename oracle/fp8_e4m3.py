"""OCP 8-bit floating point, E4M3 variant (``e4m3fn``), written from the format definition.

The paper does not discuss a quantised KV cache; the fp8 cache is a workload of this
library (a Llama-3-70B layer share with an fp8 cache).  The encoding used is the OCP
OFP8 E4M3 format:

* 1 sign bit, 4 exponent bits (bias 7), 3 mantissa bits;
* exponent field 0 encodes subnormals ``(-1)^s * m/8 * 2^-6``;
* exponent fields 1..15 encode normals ``(-1)^s * (1 + m/8) * 2^(e-7)``,
  except that ``S.1111.111`` is NaN; there are no infinities;
* largest finite magnitude 448 (``S.1111.110``), smallest subnormal 2^-9.

Encoding a float32 value ``y`` (this library's contract):

* round to nearest, ties to the code whose mantissa LSB is 0 (RNE);
* saturate: any magnitude above 448, infinities included, becomes +-448 ("satfinite");
* NaN encodes to ``S.1111.111`` (0x7F / 0xFF).

Parity: pinned by exhaustive tests (every code; every bf16 bit pattern) against
brute-force nearest-value search and against torch's float8_e4m3fn conversion.
"""
import numpy as np

E4M3_MAX = 448.0
_MIN_NORMAL_EXP = -6          # exponent of the smallest normal, 2^-6
_SUBNORMAL_QUANTUM = 2.0 ** -9


def e4m3_decode(codes):
    """Decode E4M3 codes (uint8 array) to float64 values, exactly (NaN for 0x7F/0xFF)."""
    c = np.asarray(codes, dtype=np.uint8).astype(np.int64)
    sign = np.where((c >> 7) & 1, -1.0, 1.0)
    e = (c >> 3) & 0xF
    m = c & 0x7
    mag = np.where(e == 0,
                   m.astype(np.float64) / 8.0 * 2.0 ** _MIN_NORMAL_EXP,
                   (1.0 + m.astype(np.float64) / 8.0) * np.exp2(e.astype(np.float64) - 7.0))
    mag = np.where((e == 15) & (m == 7), np.nan, mag)
    return sign * mag


def e4m3_encode(y):
    """Encode float values (exact in float64) to E4M3 codes with RNE and satfinite.

    Steps: take sign and magnitude; clip the magnitude at 448; pick the quantum of the
    binade the magnitude falls in (2^-9 below 2^-6, else 2^(floor(log2|y|) - 3));
    round |y|/quantum to the nearest integer, ties to even; rebuild the code.  A
    rounding carry into the next binade (integer reaching 16) is handled by the code
    arithmetic, because E4M3 codes of one sign are consecutive integers in value order.
    """
    y = np.asarray(y, dtype=np.float64)
    nan = np.isnan(y)
    neg = np.signbit(y)
    a = np.abs(np.where(nan, 0.0, y))
    a = np.minimum(a, E4M3_MAX)                       # satfinite (also maps +-inf to 448)
    sub = a < 2.0 ** _MIN_NORMAL_EXP
    # exponent of the binade for normals; frexp returns a = f * 2^k with f in [0.5, 1)
    _, k = np.frexp(np.where(sub, 1.0, a))
    e_unb = k - 1                                     # a in [2^e_unb, 2^(e_unb+1))
    quantum = np.where(sub, _SUBNORMAL_QUANTUM, np.exp2(e_unb.astype(np.float64) - 3.0))
    q = np.rint(a / quantum).astype(np.int64)         # np.rint: round half to even
    # subnormal binade: code = q (q == 8 is the smallest normal, code 0x08, consistent)
    # normal binade: code = (e_unb + 7) * 8 + (q - 8); q == 16 carries into the next binade
    code = np.where(sub, q, (e_unb + 7) * 8 + (q - 8))
    code = np.minimum(code, 0x7E)                     # cannot exceed 448 after the clip
    code = np.where(nan, 0x7F, code)
    code = code | np.where(neg, 0x80, 0)
    return code.astype(np.uint8)


def f32_mul(x, s):
    """float32 product (IEEE RNE) of float32 operands, returned as float32.  A product past
    the float32 range is +-inf, as in IEEE arithmetic (the encoder then saturates it)."""
    with np.errstate(over="ignore"):
        return (np.asarray(x, dtype=np.float32) * np.asarray(s, dtype=np.float32)).astype(np.float32)


def f32_recip(s):
    """Correctly rounded float32 reciprocal 1/s (elementwise)."""
    return (np.float32(1.0) / np.asarray(s, dtype=np.float32)).astype(np.float32)


def quantise_kv(x_f32, scale_f32):
    """Cache encoding of values x [..][Hkv][D] with per-kv-head scales [Hkv]:
    e4m3(fp32(x) * fp32(1/scale[h])).

    Two roundings by definition: the float32 product, then the E4M3 encode.  A scalar
    scale applies to every head.
    """
    inv = f32_recip(scale_f32)
    if inv.ndim == 1:
        inv = inv[:, None]                         # broadcast over D for [..][Hkv][D]
    return e4m3_encode(f32_mul(x_f32, inv).astype(np.float64))


def quantize_rows(x):
    """Per-row e4m3 quantisation of float32 rows ``x`` [..., D] (the quantised-Q variant of the
    attention: each (token, head) row of Q gets its own scale).

    For each row: amax = max |x| (exact); scale = fp32(amax / 448), or 1 for an all-zero row;
    inv = fp32(1 / scale); codes = e4m3_encode(fp32(x * inv)) (RNE, satfinite).  All fp32
    operations are single IEEE roundings (numpy float32 arithmetic), as the page encoder's.
    Returns (codes uint8 [..., D], scale float32 [...], dequantised float64 [..., D] =
    decode(codes) * scale, exact).
    """
    x = np.asarray(x, dtype=np.float32)
    amax = np.max(np.abs(x), axis=-1)
    scale = np.where(amax > 0, amax / np.float32(E4M3_MAX), np.float32(1.0)).astype(np.float32)
    inv = f32_recip(scale)
    codes = e4m3_encode(f32_mul(x, inv[..., None]).astype(np.float64))
    deq = e4m3_decode(codes) * scale.astype(np.float64)[..., None]
    return codes, scale, deq
