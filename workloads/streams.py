"""Seeded synthetic streams of request events for the scheduler (inputs only: no
scheduling arithmetic; imports neither the oracle nor the library).

The paper's retrieval traces are not available; these distributions stand in for the
two workloads it summarises (Stream2LLM Sec. 5, workload table):

* crawler, append mode: total tokens per query log-normal with median 5.8K and mean 9.1K
  (sigma = 0.949; P95 about 27.6K against the printed 28.9K), delivered in 6-10 chunks
  whose arrivals spread over a retrieval time log-normal with median 9.3 s and mean 9.9 s;
* ANNS, update mode: total tokens log-normal with median 10K and mean 13K (sigma = 0.724;
  P95 about 32.9K against 31K), 2-5 successive inputs over a retrieval time with median
  3.9 s and mean 4.5 s; each new input keeps a uniformly drawn prefix of the previous one
  and continues with fresh tokens.

Requests arrive as a Poisson process.  ``token_scale`` shrinks every length (for tests).
Recipe: numpy ``default_rng(seed)``; per request, in arrival order: inter-arrival gap,
total tokens, chunk or input count, retrieval time, event times, then token ids.
"""
import numpy as np

CRAWLER_TOKENS = (np.log(5800.0), 0.949)
CRAWLER_SPAN_S = (np.log(9.3), 0.354)
ANNS_TOKENS = (np.log(10000.0), 0.724)
ANNS_SPAN_S = (np.log(3.9), 0.535)


def stream_events(seed, num_reqs, mode="append", rate=2.0, token_scale=1.0, max_tokens=32768,
                  vocab=32000):
    """Events (time, kind, request id, token ids, input complete) sorted by time; kind is
    "new", "append" or "update".  mode: "append", "update" or "mixed" (alternating)."""
    rng = np.random.default_rng(seed)
    events = []
    t = 0.0
    for rid in range(num_reqs):
        t += rng.exponential(1.0 / rate)
        m = mode if mode != "mixed" else ("append" if rid % 2 == 0 else "update")
        mu, sig = CRAWLER_TOKENS if m == "append" else ANNS_TOKENS
        total = int(np.clip(np.exp(rng.normal(mu, sig)) * token_scale, 1, max_tokens))
        if m == "append":
            k = int(rng.integers(6, 11))
            span = float(np.exp(rng.normal(*CRAWLER_SPAN_S)))
            times = np.sort(rng.uniform(0.0, span, k - 1))
            cuts = np.sort(rng.integers(0, total + 1, k - 1))
            sizes = np.diff(np.concatenate([[0], cuts, [total]]))
            ids = rng.integers(0, vocab, total).astype(np.int32)
            pos = int(sizes[0])
            events.append((t, "new", rid, ids[:pos].tolist(), k == 1))
            for j in range(1, k):
                n = int(sizes[j])
                events.append((t + float(times[j - 1]), "append", rid, ids[pos:pos + n].tolist(), j == k - 1))
                pos += n
        else:
            k = int(rng.integers(2, 6))
            span = float(np.exp(rng.normal(*ANNS_SPAN_S)))
            times = np.sort(rng.uniform(0.0, span, k - 1))
            cur = rng.integers(0, vocab, max(1, int(total * rng.uniform(0.3, 1.0)))).astype(np.int32).tolist()
            events.append((t, "new", rid, cur, False))
            for j in range(1, k):
                keep = int(rng.integers(0, len(cur) + 1))
                n_new = max(0, int(total * rng.uniform(0.5, 1.0)) - keep)
                cur = cur[:keep] + rng.integers(0, vocab, n_new).astype(np.int32).tolist()
                events.append((t + float(times[j - 1]), "update", rid, cur, j == k - 1))
    events.sort(key=lambda e: (e[0], e[2]))
    return events


def prefix_hashes(ids):
    """64-bit FNV-1a style rolling hash of every prefix ids[0..p], p = 0 .. len-1."""
    out = np.zeros(len(ids), dtype=np.uint64)
    h = 1469598103934665603
    for p, t in enumerate(ids):
        h = ((h ^ (int(t) + 1)) * 1099511628211) & 0xFFFFFFFFFFFFFFFF
        out[p] = h
    return out


def prefix_rows(ids, start, end, hq, hkv, seed, sigma=0.5, head_dim=128, memo=None):
    """bf16 bit rows (Q [n][hq][D], K and V [n][hkv][D]) of positions [start, end) of the
    token sequence `ids`.  Row p is drawn from a generator seeded by (seed, hash of
    ids[0..p]): sequences that share a prefix share exactly those rows, as a model's
    activations would.  `memo` (a dict) keeps rows by prefix hash across calls."""
    from . import bf16_bits
    hs = prefix_hashes(ids[:end])
    n = end - start
    q = np.empty((n, hq, head_dim), np.uint16)
    k = np.empty((n, hkv, head_dim), np.uint16)
    v = np.empty((n, hkv, head_dim), np.uint16)
    for i, p in enumerate(range(start, end)):
        h = int(hs[p])
        got = memo.get(h) if memo is not None else None
        if got is None:
            rng = np.random.default_rng([seed, h])
            got = (bf16_bits(rng.standard_normal((hq, head_dim), dtype=np.float32) * sigma),
                   bf16_bits(rng.standard_normal((hkv, head_dim), dtype=np.float32) * sigma),
                   bf16_bits(rng.standard_normal((hkv, head_dim), dtype=np.float32) * sigma))
            if memo is not None:
                memo[h] = got
        q[i], k[i], v[i] = got
    return q, k, v
