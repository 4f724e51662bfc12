"""Pins of the scheduler oracle against what the paper fixes (Stream2LLM Sec. 4.1-4.4).

Every expected value below is derived by hand from the paper's definitions and written
out; none is computed by the oracle.
"""
import random

import pytest

from oracle import scheduler as S

PAD = 999


def make(policy, gpu=4, cpu=0, budget=1000, max_blocks=8, rec=((1000,), (1.0,)), swap=(0.0, 1.0)):
    return S.Scheduler(policy, gpu, cpu, budget, max_blocks, rec[0], rec[1], swap[0], swap[1],
                       table_pad=PAD)


def toks(n, base=0):
    return [base + i for i in range(n)]


# ---- Sec. 4.2: longest common prefix ----

def test_lcp_worked_example_of_the_paper():
    # [d1, d2, q, out1, out2] -> [d1, d2', q, out1, out2]: the LCP is [d1], length 1, and
    # the cache of tokens 1 onward is invalidated
    d1, d2, d2p, q, o1, o2 = 11, 22, 99, 33, 44, 55
    assert S.lcp_len([d1, d2, q, o1, o2], [d1, d2p, q, o1, o2]) == 1
    s = make(S.FCFS, gpu=4)
    s.new_stream(7, [d1, d2, q, o1, o2], False, 0.0)
    s.step()
    assert s.reqs[7].computed == 5
    assert s.update(7, [d1, d2p, q, o1, o2], False, 1.0) == 1
    assert s.reqs[7].computed == 1 and s.reqs[7].invalidated == 4
    assert s.reqs[7].gpu == [0]             # token 0's block stays


def test_lcp_special_cases():
    a = toks(40)
    assert S.lcp_len(a, a) == 40
    assert S.lcp_len(a, a + [7, 8]) == 40           # append expressed as an update
    assert S.lcp_len(a, [-1] + a[1:]) == 0
    assert S.lcp_len([], a) == 0
    assert S.lcp_len(a, a[:17]) == 17                 # truncation


def test_update_frees_blocks_past_the_lcp():
    # three documents of 20, 20 and 8 tokens = 48 tokens in blocks [0, 1, 2]; the second
    # document is replaced: LCP 20 keeps blocks 0 and 1 (block 1 holds tokens 16..19 of the
    # prefix), frees block 2, and 28 computed tokens are invalidated
    s = make(S.LCAS, gpu=4)
    old = toks(20, 0) + toks(20, 100) + toks(8, 200)
    s.new_stream(1, old, False, 0.0)
    out = s.step()
    assert out["reqs"] == [(1, 0, 48, [0, 1, 2] + [PAD] * 5)]
    new = toks(20, 0) + toks(20, 300) + toks(8, 200)
    assert s.update(1, new, False, 1.0) == 20
    r = s.reqs[1]
    assert (r.computed, r.invalidated, r.gpu) == (20, 28, [0, 1])
    assert s.free_gpu == {2, 3}
    # the next step recomputes tokens 20..47: the partial block 1 is written from slot 4
    out = s.step()
    assert out["reqs"] == [(1, 20, 28, [0, 1, 2] + [PAD] * 5)]


def test_update_with_identical_or_extended_input_invalidates_nothing():
    s = make(S.MCPS)
    s.new_stream(1, toks(30), False, 0.0)
    s.step()
    assert s.update(1, toks(30), False, 1.0) == 30
    assert s.update(1, toks(35), False, 2.0) == 30
    r = s.reqs[1]
    assert (r.computed, r.invalidated, len(r.gpu)) == (30, 0, 2)


# ---- Sec. 4.4: priority orders ----

def _four(policy):
    # A: arrived 0, complete, last chunk 0, 32 computed
    # B: arrived 1, partial,  last chunk 5, 64 computed
    # C: arrived 2, complete, last chunk 6,  0 computed
    # D: arrived 3, partial,  last chunk 4, 16 computed
    s = make(policy, gpu=64)
    spec = {"A": (0, True, 0, 32), "B": (1, False, 5, 64), "C": (2, True, 6, 0), "D": (3, False, 4, 16)}
    for i, (name, (arr, comp, last, done)) in enumerate(spec.items()):
        s.new_stream(name, toks(100), comp, float(arr))
        r = s.reqs[name]
        r.last_chunk, r.computed = float(last), done
    return [r.rid for r in s.priority_order()]


def test_order_fcfs_complete_tier_first_then_arrival():
    assert _four(S.FCFS) == ["A", "C", "B", "D"]


def test_order_mcps_most_computed_first():
    assert _four(S.MCPS) == ["B", "A", "D", "C"]


def test_order_lcas_complete_tier_first_then_newest_chunk():
    assert _four(S.LCAS) == ["C", "A", "B", "D"]


def test_order_ties_break_by_arrival():
    s = make(S.MCPS, gpu=64)
    for name, arr in (("late", 2.0), ("early", 1.0)):
        s.new_stream(name, toks(10), False, arr)
    assert [r.rid for r in s.priority_order()] == ["early", "late"]


# ---- Sec. 4.1 + Sec. 4.4: eviction follows reverse priority ----

def _evict_scenario(policy):
    # GPU pool of 4 blocks.  X: 40 tokens at t=0, Y: 16 tokens at t=1 (both partial),
    # step; then Z: 16 tokens, complete, at t=2, step.  Z needs one block and the pool is
    # full, so one idle request is evicted (no CPU blocks: recompute).
    s = make(policy, gpu=4)
    s.new_stream("X", toks(40), False, 0.0)
    s.new_stream("Y", toks(16, 500), False, 1.0)
    first = s.step()
    s.new_stream("Z", toks(16, 900), True, 2.0)
    second = s.step()
    return s, first, second


def test_eviction_mcps_evicts_fewest_computed():
    s, first, second = _evict_scenario(S.MCPS)
    # step 1, order X, Y (tie on 0 computed, X arrived first): X [0,1,2], Y [3]
    assert [(r[0], r[3][:3]) for r in first["reqs"]] == [("X", [0, 1, 2]), ("Y", [3, PAD, PAD])]
    # step 2, order X (40), Y (16), Z (0): Y is evicted, Z takes block 3
    assert second["preempt_recompute"] == ["Y"] and second["preempt_swap"] == []
    assert second["reqs"] == [("Z", 0, 16, [3] + [PAD] * 7)]
    assert s.reqs["Y"].computed == 0 and s.reqs["Y"].gpu == [] and s.reqs["Y"].n_recompute == 1


def test_eviction_lcas_evicts_oldest_chunk():
    s, first, second = _evict_scenario(S.LCAS)
    # step 1, partial tier newest chunk first: Y [0], X [1,2,3]
    assert [(r[0], r[3][:3]) for r in first["reqs"]] == [("Y", [0, PAD, PAD]), ("X", [1, 2, 3])]
    # step 2, order Z (complete), Y (chunk at 1), X (chunk at 0): X is evicted
    assert second["preempt_recompute"] == ["X"]
    assert second["reqs"] == [("Z", 0, 16, [1] + [PAD] * 7)]
    assert s.free_gpu == {2, 3}


def test_eviction_fcfs_reverse_scheduling_order():
    s, first, second = _evict_scenario(S.FCFS)
    assert [r[0] for r in first["reqs"]] == ["X", "Y"]
    assert second["preempt_recompute"] == ["Y"]
    assert second["reqs"] == [("Z", 0, 16, [3] + [PAD] * 7)]


def test_default_lifo_eviction_and_front_requeue():
    s = make(S.DEFAULT, gpu=4)
    s.new_stream("X", toks(48), False, 0.0)
    s.new_stream("V", [], False, 0.5)              # nothing to compute yet: stays waiting
    out = s.step()
    assert [r[0] for r in out["reqs"]] == ["X"]
    s.new_stream("Y", toks(16, 500), False, 1.0)
    out = s.step()
    assert out["reqs"] == [("Y", 0, 16, [3] + [PAD] * 7)]
    s.new_stream("Z", toks(16, 900), True, 2.0)
    out = s.step()
    # the last running request (Y) is evicted and re-queued at the front of the waiting
    # queue, ahead of V which arrived earlier
    assert out["preempt_recompute"] == ["Y"]
    assert out["reqs"] == [("Z", 0, 16, [3] + [PAD] * 7)]
    assert [r.rid for r in s.priority_order()] == ["X", "Z", "Y", "V"]


# ---- Sec. 4.4: MCPS is unstable under updates, LCAS boosts updated requests ----

def _update_scenario(policy):
    s = make(policy, gpu=64, max_blocks=16)
    s.new_stream("old", toks(200), False, 0.0)
    s.new_stream("new", toks(50, 1000), False, 1.0)
    s.step()
    # "old" gets an update with a short LCP (10 tokens) at t=5
    s.update("old", toks(10) + toks(190, 5000), False, 5.0)
    return [r.rid for r in s.priority_order()]


def test_mcps_drops_an_updated_request_to_lowest_priority():
    assert _update_scenario(S.MCPS) == ["new", "old"]


def test_lcas_boosts_an_updated_request():
    assert _update_scenario(S.LCAS) == ["old", "new"]


# ---- Sec. 4.3: cost-based choice between swap and recompute ----

def test_cost_based_preemption_swap_then_resume():
    # recompute model: 1 s per 1000 tokens; victim X holds 48 tokens in 3 blocks:
    # recompute 0.048 s; swap 0.01 + 0.001 * 3 = 0.013 s -> swap
    s = make(S.MCPS, gpu=4, cpu=8, rec=((1000,), (1.0,)), swap=(0.01, 0.001))
    s.new_stream("X", toks(48), False, 0.0)
    s.step()                                            # X: blocks 0, 1, 2
    s.new_stream("Z", toks(64, 700), True, 1.0)          # needs all 4 blocks
    out = s.step()
    # order X (48), Z (0): X idle -> not scheduled; Z needs 4 blocks, 1 free -> evict X
    assert out["preempt_swap"] == ["X"] and out["swap_out"] == [(0, 0), (1, 1), (2, 2)]
    assert out["reqs"] == [("Z", 0, 64, [0, 1, 2, 3, PAD, PAD, PAD, PAD])]
    x = s.reqs["X"]
    assert (x.state, x.computed, x.cpu, x.gpu) == (S.SWAPPED, 48, [0, 1, 2], [])
    # Z is complete and computed: it finishes at the next step; X gets 8 new tokens and
    # resumes: its three blocks come back, plus one new (56 tokens = 4 blocks)
    s.append("X", toks(8, 48), False, 2.0)
    out = s.step()
    assert out["finished"] == ["Z"]
    assert out["swap_in"] == [(0, 0), (1, 1), (2, 2)]
    assert out["reqs"] == [("X", 48, 8, [0, 1, 2, 3, PAD, PAD, PAD, PAD])]
    # the swapped-in CPU blocks are released only at the following step
    assert s.free_cpu == {3, 4, 5, 6, 7}
    s.step()
    assert s.free_cpu == set(range(8))


def test_cost_based_preemption_recompute_when_swap_is_dearer():
    # swap 0.01 + 0.02 * 3 = 0.07 s > recompute 0.048 s
    s = make(S.MCPS, gpu=4, cpu=8, rec=((1000,), (1.0,)), swap=(0.01, 0.02))
    s.new_stream("X", toks(48), False, 0.0)
    s.step()
    s.new_stream("Z", toks(64, 700), True, 1.0)
    out = s.step()
    assert out["preempt_recompute"] == ["X"] and out["swap_out"] == []
    assert s.reqs["X"].computed == 0


def test_update_of_a_swapped_request_frees_cpu_blocks():
    s = make(S.MCPS, gpu=4, cpu=8, rec=((1000,), (1.0,)), swap=(0.0, 0.001))
    s.new_stream("X", toks(48), False, 0.0)
    s.step()
    s.new_stream("Z", toks(64, 700), True, 1.0)
    s.step()
    assert s.reqs["X"].cpu == [0, 1, 2]
    # update with LCP 20: keep blocks_for(20) = 2 CPU blocks, free CPU block 2
    s.update("X", toks(20) + toks(30, 4000), False, 2.0)
    x = s.reqs["X"]
    assert (x.computed, x.invalidated, x.cpu, x.state) == (20, 28, [0, 1], S.SWAPPED)
    assert 2 in s.free_cpu
    out = s.step()          # Z finishes; X resumes: 2 blocks in, then 2 more for 50 tokens
    assert out["swap_in"] == [(0, 0), (1, 1)]
    assert out["reqs"] == [("X", 20, 30, [0, 1, 2, 3, PAD, PAD, PAD, PAD])]


def test_piecewise_linear_model():
    xs, ys = (1000, 2000, 4000), (1.0, 3.0, 4.0)
    f = lambda x: S.piecewise_linear(xs, ys, x)
    assert f(1000) == 1.0 and f(2000) == 3.0 and f(4000) == 4.0
    assert f(1500) == 2.0 and f(3000) == 3.5
    assert f(0) == -1.0 and f(6000) == 5.0        # the end segments extended
    assert S.piecewise_linear((100,), (2.0,), 50) == 1.0


def test_token_budget_is_shared_in_priority_order():
    s = make(S.FCFS, gpu=64, budget=100)
    s.new_stream("a", toks(70), True, 0.0)
    s.new_stream("b", toks(70, 100), True, 1.0)
    out = s.step()
    assert [(r[0], r[1], r[2]) for r in out["reqs"]] == [("a", 0, 70), ("b", 0, 30)]
    out = s.step()           # "a" completed in the first step: it finishes now
    assert out["finished"] == ["a"]
    assert [(r[0], r[1], r[2]) for r in out["reqs"]] == [("b", 30, 40)]
    out = s.step()
    assert out["finished"] == ["b"] and out["reqs"] == []


# ---- invariants over random event streams ----

def _check_invariants(s, out):
    held = {}
    for r in s.reqs.values():
        for b in r.gpu:
            assert b not in held, "a GPU block held twice"
            held[b] = r.rid
        if r.state == S.RUNNING:
            assert len(r.gpu) == S.blocks_for(r.computed)
        if r.state == S.SWAPPED:
            assert r.gpu == [] and len(r.cpu) == S.blocks_for(r.computed)
        if r.state in (S.WAITING, S.FINISHED):
            assert r.gpu == [] and r.cpu == []
        assert 0 <= r.computed <= len(r.ids)
    assert not (set(held) & s.free_gpu)
    assert len(held) + len(s.free_gpu) == s.num_gpu
    assert sum(r[2] for r in out["reqs"]) <= s.token_budget
    assert all(r[2] > 0 for r in out["reqs"])


@pytest.mark.parametrize("policy", [S.DEFAULT, S.FCFS, S.MCPS, S.LCAS])
def test_invariants_under_random_streams(policy):
    rng = random.Random(policy)
    s = make(policy, gpu=24, cpu=16, budget=96, max_blocks=16, rec=((64, 256), (0.01, 0.1)),
             swap=(0.002, 0.003))
    live, t = [], 0.0
    for it in range(400):
        t += 1.0
        k = rng.random()
        if k < 0.15 and len(live) < 10:
            rid = it
            s.new_stream(rid, [rng.randrange(50) for _ in range(rng.randrange(0, 60))], False, t)
            live.append(rid)
        elif k < 0.45 and live:
            rid = rng.choice(live)
            r = s.reqs[rid]
            extra = [rng.randrange(50) for _ in range(rng.randrange(0, 40))]
            if len(r.ids) + len(extra) <= 16 * 16:
                s.append(rid, extra, rng.random() < 0.2, t)
                if s.reqs[rid].complete:
                    live.remove(rid)
        elif k < 0.6 and live:
            rid = rng.choice(live)
            r = s.reqs[rid]
            keep = rng.randrange(0, len(r.ids) + 1)
            new = r.ids[:keep] + [rng.randrange(50) for _ in range(rng.randrange(0, 40))]
            if len(new) <= 16 * 16:
                lcp = s.update(rid, new, False, t)
                assert lcp >= keep
        out = s.step()
        _check_invariants(s, out)
