"""Chunk-prefill attention by definition, in float64.

Sec. 2.1: prefill computes attention for every input position and stores each position's
key/value pair; Sec. 2.2: attention at position t reads the cached pairs of positions up
to t, wherever their blocks live.  For a request with P cached tokens that receives a chunk
of C new tokens (Sec. 4.2, Sec. 5.1), query i of the chunk is absolute position t = P + i
and attends to keys 0..t inclusive: the P cached ones fully and the chunk causally.

Notation: Hq query heads, Hkv kv heads, G = Hq / Hkv, query head h reads kv head h // G
(consecutive query heads share a kv head).  For query row i, head h:

    s_j  = scale * <Q[i, h], K[j, h // G]>         for j = 0..P+i
    O    = sum_j exp(s_j - m) V[j, h // G] / sum_j exp(s_j - m),   m = max_j s_j
    LSE  = m + ln sum_j exp(s_j - m)

The paper leaves the softmax scale, the head mapping and the alignment of the causal mask
with a cached prefix unstated; the readings above are the library's contract.

Functions:

* :func:`ref_chunk_attn_loops`   - per (row, head) loops over keys; tiny inputs only.
* :func:`ref_chunk_attn_blocked` - the same definition with numpy float64 matmuls over
  query/key blocks and an exact two-pass softmax (max pass, then sum pass).
* :func:`ref_full_causal`        - brute-force dense causal attention over a whole sequence.
* :func:`ref_attn_key_range`     - the definition restricted to keys in [lo, hi).
* :func:`lse_merge`              - merge of results over disjoint key ranges.
* :func:`ref_batch_attn`         - a varlen batch read through paged pools.

Parity: all pinned in ``tests/test_oracle_attention.py`` (brute force, chunking
invariance, textbook special cases, scipy softmax, merge identity).
"""
import math

import numpy as np

from .paged_kv import decode_stored, ref_gather


def default_scale(head_dim):
    return 1.0 / math.sqrt(head_dim)


def ref_chunk_attn_loops(q, k, v, P, scale):
    """q: [C][Hq][D], k, v: [P+C][Hkv][D] (float64) -> (O [C][Hq][D], LSE [C][Hq])."""
    C, hq, d = q.shape
    hkv = k.shape[1]
    g_size = hq // hkv
    out = np.zeros((C, hq, d))
    lse = np.zeros((C, hq))
    for i in range(C):
        t = P + i
        for h in range(hq):
            g = h // g_size
            s = [scale * float(np.dot(q[i, h], k[j, g])) for j in range(t + 1)]
            m = max(s)
            w = [math.exp(x - m) for x in s]
            den = sum(w)
            acc = np.zeros(d)
            for j in range(t + 1):
                acc += w[j] * v[j, g]
            out[i, h] = acc / den
            lse[i, h] = m + math.log(den)
    return out, lse


def ref_chunk_attn_blocked(q, k, v, P, scale, q_block=512, k_block=4096, rows=None, with_abs=False,
                           spread=True):
    """Blocked form of the same definition.

    q: [C][Hq][D]; k, v: [>= P+C][Hkv][D] (float64).  ``rows`` optionally selects query
    rows (sorted indices into the chunk); only those are computed and returned.
    Pass 1 finds each row's maximum score over all visible keys; pass 2 sums
    exp(s - m) and exp(s - m) V.  Blocks only bound memory: no term is reordered
    beyond summation order.  Every contraction is a float64 matrix product (BLAS).

    ``with_abs`` also returns A = sum_j w_j |V_j| and B = sum_j w_j |V_j - O| (pass 3,
    once O is known), with w the softmax weights: per-element scales for rounding-error
    bounds of an implementation that rounds the weights.  With ``spread=False`` pass 3 is
    skipped and B is returned as NaN (A alone costs one more matrix product; B needs
    |V_j - O| for every key and row, which is not a matrix product).
    """
    C, hq, d = q.shape
    hkv = k.shape[1]
    g_size = hq // hkv
    rows = np.arange(C) if rows is None else np.asarray(rows, dtype=np.int64)
    n_rows = len(rows)
    out = np.zeros((n_rows, hq, d))
    out_abs = np.zeros((n_rows, hq, d)) if with_abs else None
    out_dev = np.full((n_rows, hq, d), np.nan) if with_abs else None
    lse = np.zeros((n_rows, hq))

    def scores(qb, kb):                                  # [nb][G][D] x [j][D] -> [nb][G][j]
        nb, gs, dd = qb.shape
        return scale * (qb.reshape(nb * gs, dd) @ np.ascontiguousarray(kb).T).reshape(nb, gs, kb.shape[0])

    def weighted(w, x):                                  # [nb][G][j] x [j][D] -> [nb][G][D]
        nb, gs, j = w.shape
        return (w.reshape(nb * gs, j) @ x).reshape(nb, gs, x.shape[1])

    for g in range(hkv):
        heads = slice(g * g_size, (g + 1) * g_size)
        for b0 in range(0, n_rows, q_block):
            rb = rows[b0:b0 + q_block]
            qb = q[rb, heads, :]                         # [nb][G][D]
            horizon = P + rb                             # last visible key per row
            kmax = int(horizon.max()) + 1
            m = np.full((len(rb), g_size), -np.inf)
            def visible(k0, nk):                         # None: every key of the block is visible
                if k0 + nk - 1 <= horizon.min():
                    return None
                keys = np.arange(k0, k0 + nk)
                return keys[None, None, :] <= horizon[:, None, None]

            for k0 in range(0, kmax, k_block):           # pass 1: maxima
                kb = k[k0:min(kmax, k0 + k_block), g, :]
                s = scores(qb, kb)
                vis = visible(k0, kb.shape[0])
                if vis is not None:
                    s = np.where(vis, s, -np.inf)
                m = np.maximum(m, s.max(axis=2))
            den = np.zeros((len(rb), g_size))
            acc = np.zeros((len(rb), g_size, d))
            acc_abs = np.zeros((len(rb), g_size, d)) if with_abs else None
            for k0 in range(0, kmax, k_block):           # pass 2: sums
                kb = k[k0:min(kmax, k0 + k_block), g, :]
                vb = v[k0:min(kmax, k0 + k_block), g, :]
                w = np.exp(scores(qb, kb) - m[:, :, None])
                vis = visible(k0, kb.shape[0])
                if vis is not None:
                    w = np.where(vis, w, 0.0)
                den += w.sum(axis=2)
                acc += weighted(w, vb)
                if with_abs:
                    acc_abs += weighted(w, np.abs(vb))
            o_blk = acc / den[:, :, None]
            out[b0:b0 + q_block, heads, :] = o_blk
            lse[b0:b0 + q_block, heads] = m + np.log(den)
            if with_abs:
                out_abs[b0:b0 + q_block, heads, :] = acc_abs / den[:, :, None]
            if with_abs and spread:
                dev = np.zeros((len(rb), g_size, d))
                for k0 in range(0, kmax, k_block):       # pass 3: spread about O, row by row
                    kb = k[k0:min(kmax, k0 + k_block), g, :]
                    vb = v[k0:min(kmax, k0 + k_block), g, :]
                    w = np.exp(scores(qb, kb) - m[:, :, None])
                    vis = visible(k0, kb.shape[0])
                    if vis is not None:
                        w = np.where(vis, w, 0.0)
                    for i in range(len(rb)):
                        for j0 in range(0, kb.shape[0], 512):   # [G][512][D] at a time
                            spread_i = np.abs(vb[None, j0:j0 + 512, :] - o_blk[i][:, None, :])
                            dev[i] += np.matmul(w[i][:, None, j0:j0 + 512], spread_i)[:, 0, :]
                out_dev[b0:b0 + q_block, heads, :] = dev / den[:, :, None]
    if with_abs:
        return out, lse, out_abs, out_dev
    return out, lse


def ref_full_causal(q, k, v, scale):
    """Dense causal attention over a whole sequence of n tokens (brute force).

    q: [n][Hq][D], k, v: [n][Hkv][D].  Scores [n][n] per head, entries above the
    diagonal set to -inf, row softmax, times V.
    """
    n, hq, d = q.shape
    hkv = k.shape[1]
    g_size = hq // hkv
    out = np.zeros((n, hq, d))
    lse = np.zeros((n, hq))
    upper = np.triu(np.ones((n, n), dtype=bool), k=1)
    for h in range(hq):
        g = h // g_size
        s = scale * (q[:, h, :] @ k[:, g, :].T)
        s[upper] = -np.inf
        m = s.max(axis=1, keepdims=True)
        e = np.exp(s - m)
        z = e.sum(axis=1, keepdims=True)
        out[:, h, :] = (e / z) @ v[:, g, :]
        lse[:, h] = m[:, 0] + np.log(z[:, 0])
    return out, lse


def ref_attn_key_range(q, k, v, P, scale, lo, hi):
    """The definition restricted to keys j in [lo, hi) (and j <= P + i).

    Rows with no visible key in the range get O = 0 and LSE = -inf.
    """
    C, hq, d = q.shape
    hkv = k.shape[1]
    g_size = hq // hkv
    out = np.zeros((C, hq, d))
    lse = np.full((C, hq), -np.inf)
    for i in range(C):
        top = min(hi, P + i + 1)
        if top <= lo:
            continue
        for h in range(hq):
            g = h // g_size
            s = scale * (k[lo:top, g, :] @ q[i, h])
            m = s.max()
            w = np.exp(s - m)
            out[i, h] = (w @ v[lo:top, g, :]) / w.sum()
            lse[i, h] = m + np.log(w.sum())
    return out, lse


def lse_merge(outs, lses):
    """Merge results over disjoint key ranges: weights exp(lse_s - lse*)."""
    lses = np.stack(lses)                               # [S][C][Hq]
    outs = np.stack(outs)                               # [S][C][Hq][D]
    top = lses.max(axis=0)
    w = np.exp(lses - top[None])
    w = np.where(np.isneginf(lses), 0.0, w)
    tot = w.sum(axis=0)
    lse = top + np.log(tot)
    out = (w[..., None] * outs).sum(axis=0) / tot[..., None]
    return out, lse


def ref_batch_attn(q_rows, k_pool, v_pool, block_tables, prefix_lens, chunk_lens, cu_chunk,
                   num_q_heads, scale, kv_dtype="bf16", k_scale=None, v_scale=None,
                   sample_rows=None, method="blocked", with_abs=False, spread=True):
    """Attention of a varlen batch whose K/V (prefix and chunk) are read through the pools.

    q_rows: float64 [T][Hq][D] (the chunk queries, request r at rows cu_chunk[r]..).
    Returns float64 O [T][Hq][D] and LSE [T][Hq] (rows not sampled are NaN when
    ``sample_rows`` is given as a dict r -> sorted chunk-row indices), and with
    ``with_abs`` the softmax-weighted means of |V| and of |V - O| [T][Hq][D] as a third and
    a fourth array (the fourth NaN with ``spread=False``, as in ``ref_chunk_attn_blocked``).
    """
    T = q_rows.shape[0]
    d = q_rows.shape[2]
    out = np.full((T, num_q_heads, d), np.nan)
    lse = np.full((T, num_q_heads), np.nan)
    out_abs = np.full((T, num_q_heads, d), np.nan) if with_abs else None
    out_dev = np.full((T, num_q_heads, d), np.nan) if with_abs else None
    for r in range(len(prefix_lens)):
        P, C, row0 = int(prefix_lens[r]), int(chunk_lens[r]), int(cu_chunk[r])
        if C == 0:
            continue
        rows = None if sample_rows is None else sample_rows.get(r, [])
        if rows is not None and len(rows) == 0:
            continue
        n = P + C if rows is None else P + int(max(rows)) + 1
        k = decode_stored(ref_gather(k_pool, block_tables, r, n), kv_dtype, k_scale)
        v = decode_stored(ref_gather(v_pool, block_tables, r, n), kv_dtype, v_scale)
        q = q_rows[row0:row0 + C]
        if method == "loops":
            assert rows is None and not with_abs
            o, l = ref_chunk_attn_loops(q, k, v, P, scale)
            out[row0:row0 + C], lse[row0:row0 + C] = o, l
        else:
            res = ref_chunk_attn_blocked(q, k, v, P, scale, rows=rows, with_abs=with_abs, spread=spread)
            idx = np.arange(C) if rows is None else np.asarray(rows)
            out[row0 + idx], lse[row0 + idx] = res[0], res[1]
            if with_abs:
                out_abs[row0 + idx] = res[2]
                out_dev[row0 + idx] = res[3]
    if with_abs:
        return out, lse, out_abs, out_dev
    return out, lse
