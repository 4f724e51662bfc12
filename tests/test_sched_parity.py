"""The library's scheduler (C++, include/s2l_sched.h) against the scheduler oracle, step
by step, on seeded synthetic request streams: every scheduled (request, P, C, block
table), every swap pair and event, every LCP, and every request's final state must be
identical (integer results: bit-exact).  Host code only: no GPU involved.
"""
import numpy as np
import pytest

from oracle import scheduler as O
from paper_2604_16395_amd import _lib
from paper_2604_16395_amd import sched as L
from workloads.streams import stream_events

EV = {"finished": L.EV_FINISHED, "swap": L.EV_PREEMPT_SWAP, "recompute": L.EV_PREEMPT_RECOMPUTE}
REC = ([1024.0, 8192.0, 65536.0], [0.02, 0.1, 1.2])
SWAP = (0.001, 0.0006)


def _pair(policy, gpu, cpu, budget, max_blocks, pad=7):
    o = O.Scheduler(policy, gpu, cpu, budget, max_blocks, REC[0], REC[1], SWAP[0], SWAP[1], table_pad=pad)
    l = L.Scheduler(policy, gpu, cpu, budget, max_blocks, REC, SWAP, table_pad=pad)
    return o, l


def _compare_step(o_out, l_out, where):
    o_reqs = [(rid, p, c, list(tab)) for rid, p, c, tab in o_out["reqs"]]
    l_reqs = [(int(r), int(p), int(c), t.tolist())
              for r, p, c, t in zip(l_out.req_ids, l_out.prefix_lens, l_out.chunk_lens, l_out.block_tables)]
    assert l_reqs == o_reqs, where
    assert [tuple(x) for x in l_out.swap_out.tolist()] == [tuple(x) for x in o_out["swap_out"]], where
    assert [tuple(x) for x in l_out.swap_in.tolist()] == [tuple(x) for x in o_out["swap_in"]], where
    assert l_out.events == [(rid, EV[k]) for rid, k in o_out["events"]], where
    assert l_out.total_tokens == sum(c for _, _, c, _ in o_out["reqs"])


def _compare_requests(o, l):
    for rid, r in o.reqs.items():
        info, gpu, cpu = l.request(rid)
        assert (info.state, info.num_tokens, info.num_computed_tokens, bool(info.input_complete)) == \
            (r.state, len(r.ids), r.computed, r.complete), rid
        assert (info.total_tokens_invalidated, info.num_preempt_swap, info.num_preempt_recompute) == \
            (r.invalidated, r.n_swap, r.n_recompute), rid
        assert (gpu, cpu) == (r.gpu, r.cpu), rid
        assert (info.arrival_time, info.last_chunk_arrival_time) == (r.arrival, r.last_chunk)


def _drive(policy, events, gpu, cpu, budget, max_blocks, dt):
    o, l = _pair(policy, gpu, cpu, budget, max_blocks)
    stats = {"steps": 0, "swap": 0, "recompute": 0, "finished": 0, "update_lcp_short": 0}
    t_next = 0.0

    def step():
        where = f"step {stats['steps']}"
        oo, lo = o.step(), l.step()
        _compare_step(oo, lo, where)
        assert [r.rid for r in o.priority_order()] == l.priority_order()[0], where
        stats["steps"] += 1
        for _, k in oo["events"]:
            stats[k] += 1

    for t, kind, rid, ids, complete in events:
        while t_next <= t:
            step()
            t_next += dt
        if kind == "new":
            o.new_stream(rid, ids, complete, t)
            l.new_stream(rid, ids, complete, t)
        elif kind == "append":
            o.append(rid, ids, complete, t)
            l.append(rid, ids, complete, t)
        else:
            a = o.update(rid, ids, complete, t)
            b = l.update(rid, ids, complete, t)
            assert a == b
            stats["update_lcp_short"] += a < len(ids) // 2
    for _ in range(10000):
        if not l.stats().num_unfinished:
            break
        step()
    assert l.stats().num_unfinished == 0
    _compare_requests(o, l)
    st = l.stats()
    assert st.free_gpu_blocks == gpu
    return stats


@pytest.mark.parametrize("policy", [L.POLICY_DEFAULT, L.POLICY_FCFS, L.POLICY_MCPS, L.POLICY_LCAS])
@pytest.mark.parametrize("mode", ["append", "update", "mixed"])
def test_scheduler_matches_oracle_on_synthetic_streams(policy, mode):
    events = stream_events(seed=100 + policy, num_reqs=40, mode=mode, rate=4.0, token_scale=0.05, max_tokens=1000)
    stats = _drive(policy, events, gpu=96, cpu=160, budget=256, max_blocks=128, dt=0.25)
    assert stats["finished"] == 40


def test_scheduler_parity_covers_swap_and_recompute():
    seen = {"swap": 0, "recompute": 0}
    for policy in (L.POLICY_MCPS, L.POLICY_LCAS):
        events = stream_events(seed=7, num_reqs=60, mode="mixed", rate=8.0, token_scale=0.05, max_tokens=1000)
        st = _drive(policy, events, gpu=64, cpu=96, budget=192, max_blocks=128, dt=0.2)
        seen["swap"] += st["swap"]
        seen["recompute"] += st["recompute"]
    assert seen["swap"] > 0 and seen["recompute"] > 0, seen


def test_lcp_len_matches_definition():
    rng = np.random.default_rng(3)
    for _ in range(200):
        a = rng.integers(0, 4, rng.integers(0, 30)).tolist()
        b = a[:rng.integers(0, len(a) + 1)] + rng.integers(0, 4, rng.integers(0, 10)).tolist()
        assert L.lcp_len(a, b) == O.lcp_len(a, b)


def test_scheduler_errors_leave_state_unchanged():
    l = L.Scheduler(L.POLICY_LCAS, 8, 0, 64, 4, REC, SWAP)
    l.new_stream(1, list(range(20)), False, 0.0)
    with pytest.raises(_lib.S2LError) as e:
        l.new_stream(1, [1], False, 0.0)
    assert e.value.status == _lib.S2L_EINVAL
    with pytest.raises(_lib.S2LError) as e:
        l.append(1, list(range(50)), False, 1.0)          # 70 tokens > 4 blocks
    assert e.value.status == _lib.S2L_ERANGE
    with pytest.raises(_lib.S2LError) as e:
        l.update(2, [1], False, 1.0)
    assert e.value.status == _lib.S2L_EINVAL
    info, gpu, _ = l.request(1)
    assert info.num_tokens == 20 and gpu == []
    step = l.step()
    assert step.req_ids.tolist() == [1] and step.chunk_lens.tolist() == [20]
    l.append(1, [5], True, 2.0)
    with pytest.raises(_lib.S2LError) as e:
        l.append(1, [5], False, 3.0)                     # input already complete
    assert e.value.status == _lib.S2L_EINVAL


def test_scheduler_rejects_bad_configs():
    for kw in ({"num_gpu_blocks": 0}, {"token_budget": 0}, {"max_blocks_per_req": 0}):
        args = dict(policy=L.POLICY_FCFS, num_gpu_blocks=8, num_cpu_blocks=0, token_budget=8,
                    max_blocks_per_req=4, recompute=REC, swap=SWAP)
        args.update(kw)
        with pytest.raises(_lib.S2LError):
            L.Scheduler(**args)
    with pytest.raises(_lib.S2LError):
        L.Scheduler(9, 8, 0, 8, 4, REC, SWAP)
    with pytest.raises(_lib.S2LError):
        L.Scheduler(0, 8, 0, 8, 4, ([10.0, 5.0], [1.0, 2.0]), SWAP)


def test_measured_cost_model_drives_the_scheduler():
    from paper_2604_16395_amd import costmodel
    rec, swap = costmodel.load()
    assert len(rec[0]) >= 2 and all(b > a for a, b in zip(rec[0], rec[0][1:]))
    assert all(t > 0 for t in rec[1]) and swap[1] > 0
    s = L.Scheduler(L.POLICY_MCPS, 4, 8, 1000, 8, rec, swap)
    o = O.Scheduler(L.POLICY_MCPS, 4, 8, 1000, 8, rec[0], rec[1], swap[0], swap[1])
    for x in (s, o):
        x.new_stream(1, list(range(48)), False, 0.0)
        x.step()
        x.new_stream(2, list(range(100, 164)), True, 1.0)
    a, b = s.step(), o.step()
    _compare_step(b, a, "cost model")
    # on this GPU moving 3 blocks over the host link beats recomputing 48 tokens
    assert a.events == [(1, L.EV_PREEMPT_SWAP)]
