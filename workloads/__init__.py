"""Seeded synthetic inputs for incremental chunked-prefill attention.

Shared by the tests, ``bench.py`` and ``smoke()``.  This module only draws inputs
(lengths, bf16 activations, block tables, per-head fp8 scales); it holds none of the
attention or paging arithmetic, and imports neither the oracle nor the GPU library.

The paper's retrieval traces, datasets and model weights are not available; these
shapes stand in for them (Llama-3-8B / Llama-3-70B attention layer shapes, prefixes up
to 32K tokens as in the workloads' P95 of 28.9K-31K tokens, 512-token chunks, per-step
token totals within or above the 2048-8192 token budget).

Recipe (every case): numpy ``default_rng(seed)``; draw order: lengths, then Q, K, V
(float32 standard normal times ``sigma``, per request, converted to bf16 with
round-to-nearest-even), then the page permutation.  K and V are drawn for all P+C
positions of each request; the chunk rows are the last C of them.
"""
from dataclasses import dataclass, field
from typing import Optional

import numpy as np

PAGE_SIZE = 16
HEAD_DIM = 128
BF16_SENTINEL = 0x7FBF      # a quiet-NaN bf16 pattern: any read of an unwritten slot shows
FP8_SENTINEL = 0x7F         # E4M3 NaN code


def bf16_bits(x):
    """float32 -> bf16 bit patterns, round to nearest even (inputs are finite)."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    r = ((u >> 16) & 1) + np.uint32(0x7FFF)
    return ((u + r) >> 16).astype(np.uint16)


@dataclass
class Case:
    name: str
    num_q_heads: int
    num_kv_heads: int
    kv_dtype: str                 # "bf16" or "fp8"
    prefix_lens: np.ndarray       # int32 [R]
    chunk_lens: np.ndarray        # int32 [R]
    cu_chunk: np.ndarray          # int32 [R+1]
    cu_seq: np.ndarray            # int64 [R+1] row offsets of each request's full K/V
    q_bits: np.ndarray            # uint16 [T][Hq][D]
    k_full_bits: np.ndarray       # uint16 [sum(P+C)][Hkv][D]
    v_full_bits: np.ndarray
    num_pages: int                # includes the trailing poison page
    block_tables: np.ndarray      # int32 [R][max_pages]; unused entries -> poison page
    k_scale: Optional[np.ndarray] = None   # float32 [Hkv] (fp8 only)
    v_scale: Optional[np.ndarray] = None
    meta: dict = field(default_factory=dict)

    @property
    def num_reqs(self):
        return len(self.prefix_lens)

    @property
    def total_tokens(self):
        return int(self.cu_chunk[-1])

    @property
    def poison_page(self):
        return self.num_pages - 1

    def new_rows(self, full):
        """Chunk rows (positions P..P+C-1 of each request) of a full K/V array."""
        parts = [full[self.cu_seq[r] + self.prefix_lens[r]:self.cu_seq[r + 1]]
                 for r in range(self.num_reqs)]
        return np.concatenate(parts) if parts else full[:0]

    def prefix_rows(self, full):
        parts = [full[self.cu_seq[r]:self.cu_seq[r] + self.prefix_lens[r]]
                 for r in range(self.num_reqs)]
        return np.concatenate(parts) if parts else full[:0]


def _draw(rng, shape, sigma):
    return bf16_bits(rng.standard_normal(shape, dtype=np.float32) * np.float32(sigma))


PLANT_OFFSET = 40   # planted keys sit at position 64 t + 40: never among the first 32 keys of a 64-key tile


def _plant_keys(q_bits, kf, P, C, seq_lo, q_row, num_q_heads, num_kv_heads, dots, twin_gap):
    """Keys aligned with one query (in place on the float32 keys ``kf`` of one request).

    For each kv head g, the query of the chunk's last token at query head g*G (it sees every
    key of the request) is the target: len(dots) keys at positions 64 t + PLANT_OFFSET, spread
    evenly over the request's 64-key tiles from the second on, are replaced by
    dots[i] * q / |q|^2, so that their dot product with the target query is dots[i] (before
    bf16 rounding); the position after the last planted key gets dots[-1] - twin_gap.
    Returns the planted positions."""
    n = P + C
    last_tile = (n - PLANT_OFFSET - 2) // 64          # 64 t + PLANT_OFFSET + 1 <= n - 1
    if C <= 0 or last_tile < 1 or not dots:
        return []
    cnt = len(dots)
    tiles = [1 + (t * (last_tile - 1)) // max(cnt - 1, 1) for t in range(cnt)]
    by_tile = dict(zip(tiles, dots))                  # a request too short for all: the later win
    pos = [64 * t + PLANT_OFFSET for t in sorted(by_tile)]
    dots = [by_tile[t] for t in sorted(by_tile)]
    G = num_q_heads // num_kv_heads
    for g in range(num_kv_heads):
        qb = q_bits[q_row + C - 1, g * G].astype(np.uint32) << 16
        qv = qb.view(np.float32).astype(np.float64)
        qq = float(qv @ qv)
        if qq == 0.0:
            continue
        for j, dot in zip(pos, dots):
            kf[seq_lo + j, g] = (dot / qq * qv).astype(np.float32)
        kf[seq_lo + pos[-1] + 1, g] = ((dots[-1] - twin_gap) / qq * qv).astype(np.float32)
    return pos


def make_case(name, prefix_lens, chunk_lens, num_q_heads, num_kv_heads, seed,
              kv_dtype="bf16", pool_pages=None, table_mode="disjoint", sigma=0.5,
              q_sigma=None, k_ramp=0.0, max_pages=None, rng=None, plant_dots=None, plant_twin_gap=0.0):
    """Build one case from explicit lengths.

    table_mode: "disjoint" - request r takes a consecutive slice of one random
                permutation of the pool; "identity" - pages in order (for invariance
                tests); "shared:<n>" - every request maps its first n pages to the same
                physical pages (read-only shared prefix).
    k_ramp:     K row j of a request is multiplied by (1 + k_ramp * j / n) before bf16
                rounding, so scores grow along the sequence.
    plant_dots: keys aligned with one query per kv head (see ``_plant_keys``): a few keys
                whose dot products with that query are these values, late in each request,
                so that its scores rise far above those of the keys before them.
    """
    rng = np.random.default_rng(seed) if rng is None else rng
    P = np.asarray(prefix_lens, dtype=np.int32)
    C = np.asarray(chunk_lens, dtype=np.int32)
    R = len(P)
    d = HEAD_DIM
    cu_chunk = np.zeros(R + 1, dtype=np.int32)
    cu_chunk[1:] = np.cumsum(C)
    seq = (P + C).astype(np.int64)
    cu_seq = np.zeros(R + 1, dtype=np.int64)
    cu_seq[1:] = np.cumsum(seq)
    q_sigma = sigma if q_sigma is None else q_sigma
    # Q, K, V (per request so that memory stays bounded per draw)
    q_bits = np.empty((int(cu_chunk[-1]), num_q_heads, d), dtype=np.uint16)
    k_bits = np.empty((int(cu_seq[-1]), num_kv_heads, d), dtype=np.uint16)
    v_bits = np.empty_like(k_bits)
    planted = {}
    for r in range(R):
        q_bits[cu_chunk[r]:cu_chunk[r + 1]] = _draw(rng, (int(C[r]), num_q_heads, d), q_sigma)
    for r in range(R):
        n = int(seq[r])
        kf = rng.standard_normal((n, num_kv_heads, d), dtype=np.float32) * np.float32(sigma)
        if k_ramp:
            kf *= (1.0 + k_ramp * np.arange(n, dtype=np.float32) / max(n, 1))[:, None, None]
        if plant_dots:
            planted[r] = _plant_keys(q_bits, kf, int(P[r]), int(C[r]), 0, int(cu_chunk[r]), num_q_heads,
                                     num_kv_heads, list(plant_dots), plant_twin_gap)
        k_bits[cu_seq[r]:cu_seq[r + 1]] = bf16_bits(kf)
        del kf
    for r in range(R):
        v_bits[cu_seq[r]:cu_seq[r + 1]] = _draw(rng, (int(seq[r]), num_kv_heads, d), sigma)
    # block tables
    pages_needed = (seq + PAGE_SIZE - 1) // PAGE_SIZE
    mp = int(max_pages) if max_pages is not None else max(1, int(pages_needed.max(initial=1)))
    total_needed = int(pages_needed.sum())
    data_pages = int(pool_pages) if pool_pages is not None else max(1, total_needed)
    num_pages = data_pages + 1                      # + poison page (never written)
    tables = np.full((R, mp), data_pages, dtype=np.int32)
    if table_mode == "identity":
        assert total_needed <= data_pages
        perm = np.arange(data_pages, dtype=np.int32)
    else:
        perm = rng.permutation(data_pages).astype(np.int32)
    if table_mode.startswith("shared:"):
        n_shared = int(table_mode.split(":")[1])
        shared = perm[:n_shared]
        off = n_shared
        for r in range(R):
            k = int(pages_needed[r])
            tables[r, :min(k, n_shared)] = shared[:min(k, n_shared)]
            rest = max(0, k - n_shared)
            tables[r, n_shared:n_shared + rest] = perm[off:off + rest]
            off += rest
        assert off <= data_pages
    else:
        assert total_needed <= data_pages, "pool too small for the drawn lengths"
        off = 0
        for r in range(R):
            k = int(pages_needed[r])
            tables[r, :k] = perm[off:off + k]
            off += k
    case = Case(name=name, num_q_heads=num_q_heads, num_kv_heads=num_kv_heads,
                kv_dtype=kv_dtype, prefix_lens=P, chunk_lens=C, cu_chunk=cu_chunk,
                cu_seq=cu_seq, q_bits=q_bits, k_full_bits=k_bits, v_full_bits=v_bits,
                num_pages=num_pages, block_tables=tables)
    if kv_dtype == "fp8":
        # caller-chosen static scales: max |x| of each kv head over the whole tensor / 448
        kf = (k_bits.astype(np.uint32) << 16).view(np.float32)
        vf = (v_bits.astype(np.uint32) << 16).view(np.float32)
        case.k_scale = (np.abs(kf).max(axis=(0, 2)) / np.float32(448.0)).astype(np.float32)
        case.v_scale = (np.abs(vf).max(axis=(0, 2)) / np.float32(448.0)).astype(np.float32)
    case.meta = dict(seed=seed, sigma=sigma, q_sigma=q_sigma, k_ramp=k_ramp, table_mode=table_mode,
                     planted=planted)
    return case


# --------------------------------------------------------------------------------------
# The five named workloads (seed = 1000 + index)
# --------------------------------------------------------------------------------------

def config1(seed=1001):
    """Single request: P=256 cached, C=128 new; 8 q heads / 2 kv heads; 64-page pool."""
    return make_case("p256_c128_h8kv2", [256], [128], 8, 2, seed, pool_pages=64)


def config2_lengths(seed=1002):
    """(P, C, seed actually used): P ~ U{0..8192}, C = 512, re-drawn with seed+1 until the
    8 requests fit the 4096-page pool."""
    s = seed
    while True:
        rng = np.random.default_rng(s)
        P = rng.integers(0, 8193, size=8)
        C = np.full(8, 512)
        if int(((P + C + 15) // 16).sum()) <= 4096:
            return P, C, s
        s += 1


def config2(seed=1002):
    """Llama-3-8B layer shape: 8 requests, P ~ U{0..8192}, C = 512; 32q/8kv; 4096-page pool."""
    P, C, s = config2_lengths(seed)
    rng = np.random.default_rng(s)
    rng.integers(0, 8193, size=8)            # replay the length draw, then Q/K/V follow
    return make_case("batch8_c512_pU8k_h32kv8", P, C, 32, 8, s, pool_pages=4096, rng=rng)


def config3_stream(seed=1003):
    """One 32768-token context streamed as 64 chunks of 512 (Llama-3-8B heads).

    Returned as a single request with P=0, C=32768: Q/K/V rows for all positions; the
    streaming driver feeds it 512 rows at a time (step s: P = 512 s, C = 512).
    """
    return make_case("stream32k_c512x64_h32kv8", [0], [32768], 32, 8, seed, pool_pages=2048)


def config3_step(step=16, seed=1003):
    """One step of the stream: P = 512*step cached tokens, a 512-token chunk (Llama-3-8B heads)."""
    return make_case(f"p{512 * step}_c512_h32kv8", [512 * step], [512], 32, 8, seed,
                     pool_pages=2048)


def config4_lengths(seed=1004):
    """P ~ U{0..32768}; C = clip(floor(exp(N(ln 64, 4.118^2))), 1, 2048) (about 20% of rows
    at C = 1 and 20% at 2048)."""
    rng = np.random.default_rng(seed)
    P = rng.integers(0, 32769, size=64)
    C = np.clip(np.floor(np.exp(rng.normal(np.log(64.0), 4.118, size=64))), 1, 2048).astype(np.int64)
    return P, C, rng


def config4(seed=1004):
    """Mixed batch: 64 requests, prefixes uniform in [0, 32768], log-normal chunk lengths."""
    P, C, rng = config4_lengths(seed)
    pages = int(((P + C + 15) // 16).sum())
    return make_case("mixed64_pU32k_clognormal_h32kv8", P, C, 32, 8, seed,
                     pool_pages=int(pages * 1.25), rng=rng)


def config5(seed=1005):
    """Llama-3-70B single-GPU layer share: P=131072, C=2048, 64q/8kv, fp8 e4m3 KV cache."""
    return make_case("p131072_c2048_h64kv8_fp8", [131072], [2048], 64, 8, seed,
                     kv_dtype="fp8", pool_pages=10400)


def attn_flops(prefix_lens, chunk_lens, num_q_heads, head_dim=HEAD_DIM):
    """Algorithmic FLOPs: 4*d*Hq per (query, visible key) pair, over unmasked pairs only."""
    P = np.asarray(prefix_lens, dtype=np.float64)
    C = np.asarray(chunk_lens, dtype=np.float64)
    pairs = C * P + C * (C + 1) / 2
    return float(4.0 * head_dim * num_q_heads * pairs.sum())
