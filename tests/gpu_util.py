"""Helpers shared by the GPU parity tests: build a case on the device through the C ABI and
compute the oracle's answer for the same seeded inputs."""
import math

import numpy as np
import torch

import paper_2604_16395_amd as s2l
from oracle.attention import ref_batch_attn
from oracle.fp8_e4m3 import quantize_rows
from oracle.paged_kv import bf16_bits_to_f32, ref_append
import workloads
from workloads import BF16_SENTINEL, FP8_SENTINEL

DEV = "cuda"
SCALE = 1.0 / math.sqrt(128.0)


def to_bf16(bits):
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).to(DEV).view(torch.bfloat16)


def from_bf16(t):
    return t.contiguous().view(torch.int16).cpu().numpy().view(np.uint16)


def bf16_to_f64(t):
    return bf16_bits_to_f32(from_bf16(t)).astype(np.float64)


_NAMED = {}
_PREFIX_POOLS = {}
_ORACLE = {}


def named_case(name):
    """The named workload ``workloads.<name>()``, drawn once per test session: drawing the large
    ones (and paging their prefixes into the reference pools) takes tens of seconds on the host.
    Tests only read the returned case."""
    if name not in _NAMED:
        _NAMED[name] = getattr(workloads, name)()
    return _NAMED[name]


def sentinel_pools(case):
    shape = (case.num_pages, case.num_kv_heads, 16, 128)
    if case.kv_dtype == "fp8":
        return np.full(shape, FP8_SENTINEL, np.uint8), np.full(shape, FP8_SENTINEL, np.uint8)
    return np.full(shape, BF16_SENTINEL, np.uint16), np.full(shape, BF16_SENTINEL, np.uint16)


def pool_to_dev(pool):
    if pool.dtype == np.uint8:
        return torch.from_numpy(pool).to(DEV)
    return to_bf16(pool)


def pool_from_dev(t):
    if t.dtype == torch.uint8:
        return t.cpu().numpy()
    return from_bf16(t)


class Setup:
    """One step of a case: pools hold each request's prefix (written by the oracle's
    append), the chunk is appended by the GPU kernel (and by the oracle on its copy)."""

    def __init__(self, case, block_tables=None, prefix_on_gpu=False):
        self.case = case
        self.tables = case.block_tables if block_tables is None else block_tables
        self.named = block_tables is None and any(c is case for c in _NAMED.values())
        R = case.num_reqs
        zeros = np.zeros(R, np.int32)
        cu_pre = np.zeros(R + 1, np.int32)
        cu_pre[1:] = np.cumsum(case.prefix_lens)
        # a named case with its own tables pages its prefix into the reference pools once
        memo = self.named and not prefix_on_gpu
        if memo and case.name in _PREFIX_POOLS:
            self.kp_ref, self.vp_ref = (a.copy() for a in _PREFIX_POOLS[case.name])
        else:
            self.kp_ref, self.vp_ref = sentinel_pools(case)
            pre_k, pre_v = case.prefix_rows(case.k_full_bits), case.prefix_rows(case.v_full_bits)
        self.fp8 = case.kv_dtype == "fp8"
        self.k_scale = None if not self.fp8 else torch.from_numpy(case.k_scale).to(DEV)
        self.v_scale = None if not self.fp8 else torch.from_numpy(case.v_scale).to(DEV)
        if prefix_on_gpu:
            kd, vd = pool_to_dev(self.kp_ref), pool_to_dev(self.vp_ref)
            self.cache = s2l.PagedKVCache(kd, vd, self.k_scale, self.v_scale)
            pb = s2l.Batch(zeros, case.prefix_lens, self.tables)
            if len(pre_k):
                s2l.s2l_kv_append(self.cache, pb, to_bf16(pre_k), to_bf16(pre_v))
        if not (memo and case.name in _PREFIX_POOLS):
            ref_append(self.kp_ref, self.vp_ref, self.tables, zeros, case.prefix_lens, cu_pre, pre_k, pre_v,
                       case.kv_dtype, case.k_scale, case.v_scale)
            if memo:
                _PREFIX_POOLS[case.name] = (self.kp_ref.copy(), self.vp_ref.copy())
        if not prefix_on_gpu:
            self.cache = s2l.PagedKVCache(pool_to_dev(self.kp_ref), pool_to_dev(self.vp_ref),
                                          self.k_scale, self.v_scale)
        self.batch = s2l.Batch(case.prefix_lens, case.chunk_lens, self.tables)
        self.k_new = case.new_rows(case.k_full_bits)
        self.v_new = case.new_rows(case.v_full_bits)
        self.q = to_bf16(case.q_bits)
        self.appended = False

    def append(self):
        s2l.s2l_kv_append(self.cache, self.batch, to_bf16(self.k_new), to_bf16(self.v_new))
        ref_append(self.kp_ref, self.vp_ref, self.tables, self.case.prefix_lens, self.case.chunk_lens,
                   self.case.cu_chunk, self.k_new, self.v_new, self.case.kv_dtype, self.case.k_scale,
                   self.case.v_scale)
        self.appended = True

    def attention(self, opts=None, with_lse=True, use_main_and_reduce=False, q8=False, scale=SCALE):
        c = self.case
        T, hq = c.total_tokens, c.num_q_heads
        nbytes = s2l.s2l_attn_workspace_bytes(self.batch, hq, c.num_kv_heads, opts)
        ws = torch.empty(nbytes, dtype=torch.uint8, device=DEV)
        self._ws = ws
        plan = s2l.s2l_attn_plan(self.batch, hq, c.num_kv_heads, ws, opts)
        out = torch.full((T, hq, 128), float("nan"), dtype=torch.bfloat16, device=DEV)
        lse = torch.full((T, hq), float("nan"), dtype=torch.float32, device=DEV) if with_lse else None
        if q8:
            s2l.s2l_chunk_prefill_attn_q8(self.cache, self.batch, self.q, hq, scale, out, lse, plan, ws)
        elif use_main_and_reduce:
            s2l.s2l_attn_main(self.cache, self.batch, self.q, hq, scale, out, lse, plan, ws)
            s2l.s2l_split_reduce(self.batch, hq, out, lse, plan, ws)
        else:
            s2l.s2l_chunk_prefill_attn(self.cache, self.batch, self.q, hq, scale, out, lse, plan, ws)
        torch.cuda.synchronize()
        self.plan = plan
        return out, lse

    def oracle(self, sample_rows=None, q8=False, spread=True, scale=SCALE):
        """(O, LSE, A, B): the oracle's output, log-sum-exp and the softmax-weighted means of
        |V| and of |V - O|.  q8: of the queries quantised per (token, head) row to e4m3.
        spread=False skips B (NaN), which costs a pass over |V_j - O| for every key: the
        comparison then bounds B by A + |O| (triangle inequality)."""
        c = self.case
        # a named case's appended pools are the same in every test, so is the oracle's answer
        key = None
        if self.named and self.appended:
            rows_key = None if sample_rows is None else tuple((r, tuple(v)) for r, v in sorted(sample_rows.items()))
            key = (c.name, q8, rows_key, spread, scale)
            if key in _ORACLE:
                return _ORACLE[key]
        q = bf16_bits_to_f32(c.q_bits).astype(np.float64)
        if q8:
            q = quantize_rows(bf16_bits_to_f32(c.q_bits))[2]
        res = ref_batch_attn(q, self.kp_ref, self.vp_ref, self.tables, c.prefix_lens, c.chunk_lens,
                             c.cu_chunk, c.num_q_heads, scale, c.kv_dtype, c.k_scale, c.v_scale,
                             sample_rows=sample_rows, with_abs=True, spread=spread)
        if key is not None:
            _ORACLE[key] = res
        return res


def sample_rows(case, per_req, rng):
    """Chunk rows to check per request: first, last, and `per_req` distinct random others (every
    row of a chunk shorter than that)."""
    out = {}
    for r in range(case.num_reqs):
        C = int(case.chunk_lens[r])
        if C == 0:
            continue
        pick = {0, C - 1} | set(rng.choice(C, size=min(per_req, C), replace=False).tolist())
        out[r] = sorted(pick)
    return out


def dense_rows(case, stride=64, chunk=None):
    """Deterministic dense row set per request: every `stride`-th chunk row, plus the first
    and last row of each `chunk`-row piece of the request's chunk (the whole chunk if None),
    so that every page, tile and streaming-chunk boundary region is represented."""
    out = {}
    for r in range(case.num_reqs):
        C = int(case.chunk_lens[r])
        if C == 0:
            continue
        step = C if chunk is None else chunk
        pick = set(range(0, C, stride))
        for a in range(0, C, step):
            pick |= {a, min(C, a + step) - 1}
        out[r] = sorted(pick)
    return out


def count_rows(rows):
    return sum(len(v) for v in rows.values())


def assert_attention_close(case, out_gpu, lse_gpu, ref, rows=None, what=""):
    """Compare bf16 GPU output with the fp64 oracle ``ref`` = (O, LSE, A, B).

    Error budget of the GPU arithmetic (u = 2^-8, the unit roundoff of bf16).  The kernel
    rounds each probability to bf16, b_j = p_j (1 + d_j) with |d_j| <= u, multiplies V by
    the b_j and divides by their own sum, i.e. it applies the exactly normalised weights
    w'_j = b_j / sum b.  Since sum (w'_j - w_j) = 0, O' - O = sum (w'_j - w_j)(V_j - O),
    and |w'_j - w_j| <= w_j 2u / (1 - u), so |O' - O| <= 2u/(1-u) B, B = sum_j w_j |V_j - O|.
    The bf16 output adds u |O'|; fp32 accumulation adds far less (budgeted as 2^-16 A).
    Where the oracle was run without B (NaN), B <= A + |O| (triangle inequality) stands in.
    Checks:
      * max |err| <= 1e-2 (the stated contract);
      * per element |err| <= u |O| + 2.02 u B + 2^-16 A + 1e-6;
      * per request ||err||_2 / ||O||_2 <= 5e-3;
      * |LSE err| <= 2^-8 + 1e-4 (1 + |LSE|): the log-sum-exp is taken of the sum of the
        same bf16 weights, sum b_j = (1 + t) sum p_j with |t| <= u, so ln differs by at most
        -ln(1 - u) < 1.002 u; fp32 arithmetic (exp2 argument, sums, log2) adds < 1e-4 relative.
    """
    o_ref, l_ref, a_ref, b_ref = ref
    o = bf16_to_f64(out_gpu)
    cu = case.cu_chunk
    mask = np.zeros(case.total_tokens, dtype=bool)
    if rows is None:
        mask[:] = True
    else:
        for r, rr in rows.items():
            mask[cu[r] + np.asarray(rr, dtype=np.int64)] = True
    a, b = o[mask], o_ref[mask]
    assert np.isfinite(a).all(), f"{what}: non-finite output"
    err = np.abs(a - b)
    assert err.max() <= 1e-2, f"{what}: max abs err {err.max():.3e}"
    u = 2.0 ** -8
    spread = b_ref[mask]
    spread = np.where(np.isnan(spread), a_ref[mask] + np.abs(b), spread)
    bound = u * np.abs(b) + 2.02 * u * spread + 2.0 ** -16 * a_ref[mask] + 1e-6
    bad = err > bound
    assert not bad.any(), (f"{what}: {bad.sum()} elements over the elementwise bound; worst "
                           f"excess {(err - bound).max():.3e}, worst err/bound {(err / bound).max():.2f}")
    for r in range(case.num_reqs):
        sel = mask[cu[r]:cu[r + 1]]
        if not sel.any():
            continue
        ea = o[cu[r]:cu[r + 1]][sel] - o_ref[cu[r]:cu[r + 1]][sel]
        rel = np.linalg.norm(ea) / max(np.linalg.norm(o_ref[cu[r]:cu[r + 1]][sel]), 1e-30)
        assert rel <= 5e-3, f"{what}: request {r} relative L2 err {rel:.3e}"
    if lse_gpu is not None:
        lg = lse_gpu.cpu().numpy().astype(np.float64)[mask]
        lr = l_ref[mask]
        assert np.isfinite(lg).all()
        assert (np.abs(lg - lr) <= 2.0 ** -8 + 1e-4 * (1 + np.abs(lr))).all(), \
            f"{what}: lse err {np.abs(lg - lr).max():.3e}"
    return float(err.max())


LOG2E = 1.4426950408889634


def plant_dots_for(excess_log2, count, scale=SCALE):
    """Dot products whose scores (scale * dot, in log2 units: times log2 e) are excess_log2,
    2 excess_log2, ..., count excess_log2: each planted key far above every key before it."""
    c = scale * LOG2E
    return [excess_log2 * (t + 1) / c for t in range(count)]


def rescale_excess(setup, opts=None, q8=False, threshold=64.0):
    """Replay, on the host, the reference each attention workgroup's online softmax starts
    from, and return (largest excess, number of (item, key group, column) triples above
    `threshold`): for every work item of the plan that `opts` gives, every key group of its
    workgroup and every query column, the excess is the largest score of a later key over the
    group's reference, in the log2 domain (scale * log2 e * q.k).  The main kernel's key
    groups are the item's range (or its two halves of whole 64-key tiles with two key groups),
    each with the exact max of its first 32 keys as reference; the decode kernel's are its four
    waves, wave w taking 64-key tiles w, w + 4, ... with the max of its first tile.  A
    probability above 2^64 sends the kernel through its rescale branch, so an excess above 64
    means the branch runs.  Scores come from the stored keys (fp8: decoded times the scale)
    and the queries as the kernel uses them (q8: quantised per row)."""
    from oracle.paged_kv import decode_stored, ref_gather
    c = setup.case
    info, items = s2l.s2l_plan_host(c.prefix_lens, c.chunk_lens, c.num_q_heads, c.num_kv_heads, opts,
                                    with_items=True)
    G = c.num_q_heads // c.num_kv_heads
    q = bf16_bits_to_f32(c.q_bits).astype(np.float64)
    if q8:
        q = quantize_rows(bf16_bits_to_f32(c.q_bits))[2]
    cl2 = SCALE * LOG2E
    best, above = -np.inf, 0
    for r in range(c.num_reqs):
        P, C, row0 = int(c.prefix_lens[r]), int(c.chunk_lens[r]), int(c.cu_chunk[r])
        if C == 0:
            continue
        n = P + C
        k = decode_stored(ref_gather(setup.kp_ref, setup.tables, r, n), c.kv_dtype, c.k_scale)
        mine = items[items[:, 0] == r]
        for g in range(c.num_kv_heads):
            s = cl2 * np.matmul(q[row0:row0 + C, g * G:(g + 1) * G, :], k[:, g, :].T)   # [C][G][n]
            for it in mine[mine[:, 1] == g]:
                i0, i1, lo, hi = (int(x) for x in it[2:6])
                if hi <= lo:
                    continue
                if info.tile_cols == 16:
                    groups = []
                    for w in range(4):
                        tiles = list(range(lo + 64 * w, hi, 256))
                        if tiles:
                            groups.append((tiles[0], min(tiles[0] + 64, hi),
                                           [(a, min(a + 64, hi)) for a in tiles[1:]]))
                else:
                    nt = -(-(hi - lo) // 64)
                    nt0 = (nt + 1) // 2 if info.key_halves == 2 else nt
                    bounds = [(lo, min(hi, lo + 64 * nt0))]
                    if info.key_halves == 2:
                        bounds.append((lo + 64 * nt0, hi))
                    groups = [(a, min(a + 32, b), [(min(a + 32, b), b)]) for a, b in bounds if b > a]
                for ref_lo, ref_hi, later in groups:
                    for i in range(i0, i1):
                        top = P + i + 1                  # keys 0 .. P + i are visible
                        if top <= ref_lo:
                            continue
                        ref = s[i, :, ref_lo:min(ref_hi, top)].max(axis=1)           # [G]
                        lat = [s[i, :, a:min(b, top)] for a, b in later if min(b, top) > a]
                        if not lat:
                            continue
                        ex = np.concatenate(lat, axis=1).max(axis=1) - ref
                        best = max(best, float(ex.max()))
                        above += int((ex > threshold).sum())
    return best, above
