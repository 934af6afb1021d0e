"""Pins of the oracle's logical cache: the paper's worked example, exhaustive
replay against an independent log-scanning LRU, invariants and closed forms."""
import itertools
import json
import os

import numpy as np
import pytest

from oracle import brute, cache

HERE = os.path.dirname(os.path.abspath(__file__))


def test_paper_worked_example_reorder():
    g = json.load(open(os.path.join(HERE, "golden", "worked_example_reorder.json")))
    lc = cache.LayerCache(g["n_experts"], g["slots"], warm=g["warm"])
    lc.spec_plan(g["prefetched"])
    order, entries = lc.precise_plan(g["gate_selects"])
    assert order == g["expected_order"]
    assert [e.expert for e in entries if e.miss] == g["expected_misses"]
    assert lc.count["miss"] == 1 and lc.count["hit"] == 3
    # expert 3 was prefetched but not used: it is the LRU victim of the miss
    assert entries[-1].victim == 3 and lc.count["spec_wasted"] == 1 and lc.count["spec_used"] == 3


def _check_invariants(lc):
    res = [e for e in lc.slot_expert if e >= 0]
    assert len(res) == len(set(res)) <= lc.C
    for s, e in enumerate(lc.slot_expert):
        if e >= 0:
            assert lc.slot_of[e] == s
    for e, s in enumerate(lc.slot_of):
        if s >= 0:
            assert lc.slot_expert[s] == e
    c = lc.count
    assert c["hit"] + c["miss"] == c["prec_access"]
    assert c["spec_used"] + c["spec_wasted"] <= c["spec_issued"]


def _plans(E, C):
    out = []
    for n in range(1, E + 1):
        for P in itertools.combinations(range(E), n):
            out.append(("P", list(P)))
    for n in range(1, min(C, E) + 1):
        for Q in itertools.permutations(range(E), n):
            out.append(("Q", list(Q)))
    return out


def _replay(seq, E, C, warm=True, budget=-1, reorder=True, pinned=0):
    a = cache.LayerCache(E, C, warm, pinned)
    b = brute.NaiveLRU(E, C, warm, pinned)
    for kind, lst in seq:
        if kind == "Q":
            ea = a.spec_plan(lst, budget)
            eb = b.spec(lst, budget)
            assert [(x.expert, x.slot, x.new) for x in ea] == eb
        else:
            order, entries = a.precise_plan(lst, reorder)
            ob, sb = b.precise(lst, reorder)
            assert order == ob
            assert [x.slot for x in entries] == sb
            # the `after` dependency names the earlier position whose slot is reused;
            # a victim that is a member of the order is an earlier one (reordered) or
            # one not yet used (id order)
            for i, x in enumerate(entries):
                if x.after >= 0:
                    assert x.after < i and order[x.after] == x.victim and entries[x.after].slot == x.slot
                elif x.miss and x.victim >= 0:
                    assert x.victim not in order[:i]
                    if reorder:
                        assert x.victim not in order
            if pinned and warm:
                assert a.slot_expert[:pinned] == list(range(pinned))
        _check_invariants(a)
        assert a.count == b.c
        assert {e: s for e, s in enumerate(a.slot_of) if s >= 0} == b.where


@pytest.mark.parametrize("C", [1, 2, 3])
def test_exhaustive_replay_up_to_three_plans(C):
    E = 4
    plans = _plans(E, C)
    for n in (1, 2, 3):
        for seq in itertools.product(plans, repeat=n):
            _replay(seq, E, C)


@pytest.mark.parametrize("budget", [0, 1, 2])
def test_exhaustive_replay_with_fill_budget(budget):
    E, C = 4, 2
    plans = _plans(E, C)
    for n in (1, 2, 3):
        for seq in itertools.product(plans, repeat=n):
            _replay(seq, E, C, budget=budget)


@pytest.mark.parametrize("reorder,pinned", [(False, 0), (True, 1), (False, 1)])
def test_exhaustive_replay_id_order_and_static(reorder, pinned):
    E, C = 4, 2
    plans = _plans(E, C)
    for n in (1, 2, 3):
        for seq in itertools.product(plans, repeat=n):
            _replay(seq, E, C, reorder=reorder, pinned=pinned)


def test_random_replays_id_order_and_static():
    rng = np.random.default_rng(12)
    for trial in range(300):
        E = int(rng.integers(2, 9))
        C = int(rng.integers(2, E + 2))
        warm = bool(rng.integers(0, 2))
        pinned = int(rng.integers(0, C))
        plans = []
        for _ in range(int(rng.integers(1, 16))):
            if rng.random() < 0.5:
                plans.append(("P", list(rng.choice(E, size=int(rng.integers(1, E + 1)), replace=False))))
            else:
                plans.append(("Q", list(rng.choice(E, size=int(rng.integers(1, min(C, E) + 1)), replace=False))))
        _replay(plans, E, C, warm, reorder=bool(rng.integers(0, 2)), pinned=pinned)


def test_id_order_cyclic_scan_thrashes():
    # every expert routed each time, C < E: in id order LRU misses every access after
    # the first scan; reordered, the resident half hits
    E, C, n = 8, 4, 5
    a, b = cache.LayerCache(E, C), cache.LayerCache(E, C)
    for _ in range(n):
        a.precise_plan(range(E), reorder=False)
        b.precise_plan(range(E))
    assert a.count["miss"] == (E - C) + E * (n - 1) and a.count["hit"] == C
    assert b.count["miss"] == (E - C) * n and b.count["hit"] == C * n


def test_paper_example_without_reorder_keeps_id_order():
    g = json.load(open(os.path.join(HERE, "golden", "worked_example_reorder.json")))
    lc = cache.LayerCache(g["n_experts"], g["slots"], warm=g["warm"])
    lc.spec_plan(g["prefetched"])
    order, entries = lc.precise_plan(g["gate_selects"], reorder=False)
    assert order == sorted(g["gate_selects"])
    assert [e.expert for e in entries if e.miss] == g["expected_misses"]


def test_static_cache_closed_form():
    # pinned experts always hit; the two staging slots hold the latest two misses
    rng = np.random.default_rng(13)
    E, C = 12, 6
    lc = cache.LayerCache(E, C, pinned=C - 2)
    staging = [C - 2, C - 1]
    for _ in range(300):
        P = sorted(rng.choice(E, int(rng.integers(1, 5)), replace=False).tolist())
        resident = set(lc.slot_expert)
        before = dict(lc.count)
        order, entries = lc.precise_plan(P, reorder=False)
        # misses: at least the non-resident members, at most every non-pinned member
        m = lc.count["miss"] - before["miss"]
        assert len(set(P) - resident) <= m <= len([e for e in P if e >= C - 2])
        for x in entries:
            if x.expert < C - 2:
                assert not x.miss and x.slot == x.expert
            if x.miss:
                assert x.slot in staging
        assert lc.slot_expert[:C - 2] == list(range(C - 2))


def test_prediction_accuracy_counts():
    lc = cache.LayerCache(8, 4)
    lc.spec_plan([5, 6, 1])                 # predicted
    lc.precise_plan([1, 2, 6])              # 1 and 6 correct
    assert (lc.count["pred_n"], lc.count["pred_correct"]) == (3, 2)
    lc.precise_plan([5])                    # the prediction was consumed by the route
    assert lc.count["pred_correct"] == 2
    lc.spec_plan([7], predicted=False)      # a caller's push is not a prediction
    lc.precise_plan([7])
    assert (lc.count["pred_n"], lc.count["pred_correct"]) == (3, 2)
    # a perfect predictor of one token scores k of k
    rng = np.random.default_rng(14)
    p = cache.LayerCache(16, 6)
    for _ in range(50):
        P = rng.choice(16, 4, replace=False).tolist()
        p.spec_plan(P)
        p.precise_plan(P)
    assert p.count["pred_correct"] == p.count["pred_n"] == 200


def test_fill_budget_closed_forms():
    rng = np.random.default_rng(9)
    E, C = 16, 8
    # budget 0: predictions only refresh residents, so fills happen only on misses
    a = cache.LayerCache(E, C)
    for _ in range(200):
        Q = rng.choice(E, 4, replace=False).tolist()
        P = rng.choice(E, 3, replace=False).tolist()
        ea = a.spec_plan(Q, budget=0)
        assert not any(x.new for x in ea) and a.count["spec_issued"] == 0
        a.precise_plan(P)
    # a budget of at least |Q| equals no budget
    c1, c2 = cache.LayerCache(E, C), cache.LayerCache(E, C)
    for _ in range(200):
        Q = rng.choice(E, 4, replace=False).tolist()
        P = rng.choice(E, 3, replace=False).tolist()
        e1 = c1.spec_plan(Q, budget=4)
        e2 = c2.spec_plan(Q)
        assert [(x.expert, x.slot, x.new) for x in e1] == [(x.expert, x.slot, x.new) for x in e2]
        assert c1.precise_plan(P)[0] == c2.precise_plan(P)[0]
    assert c1.count == c2.count
    # fills per plan never exceed the budget
    d = cache.LayerCache(E, C)
    for _ in range(200):
        Q = rng.choice(E, 6, replace=False).tolist()
        before = d.count["spec_issued"]
        d.spec_plan(Q, budget=2)
        assert d.count["spec_issued"] - before <= 2
        d.precise_plan(rng.choice(E, 3, replace=False).tolist())


def test_random_long_replays():
    rng = np.random.default_rng(11)
    for trial in range(300):
        E = int(rng.integers(2, 9))
        C = int(rng.integers(1, E + 2))
        warm = bool(rng.integers(0, 2))
        plans = []
        for _ in range(int(rng.integers(1, 16))):
            if rng.random() < 0.5:
                plans.append(("P", list(rng.choice(E, size=int(rng.integers(1, E + 1)), replace=False))))
            else:
                plans.append(("Q", list(rng.choice(E, size=int(rng.integers(1, min(C, E) + 1)), replace=False))))
        _replay(plans, E, C, warm)


def test_capacity_at_least_e_misses_once():
    rng = np.random.default_rng(2)
    E, C = 6, 8
    lc = cache.LayerCache(E, C, warm=True)          # warm set 0..5 = everything
    for _ in range(50):
        lc.precise_plan(rng.choice(E, 3, replace=False))
    assert lc.count["miss"] == 0
    lc = cache.LayerCache(8, 8, warm=False)
    seen = set()
    for _ in range(50):
        P = set(rng.choice(8, 3, replace=False).tolist())
        lc.precise_plan(P)
        seen |= P
    assert lc.count["miss"] == len(seen)


def test_perfect_predictor_gives_no_misses():
    rng = np.random.default_rng(3)
    E, C, k = 16, 6, 4
    lc = cache.LayerCache(E, C)
    for _ in range(100):
        P = sorted(rng.choice(E, k, replace=False).tolist())
        lc.spec_plan(P)              # |Q| = k <= C, exactly the routed experts
        order, entries = lc.precise_plan(P)
        assert not any(x.miss for x in entries)
    assert lc.count["miss"] == 0 and lc.count["spec_used"] == lc.count["spec_issued"]


def test_lru_inclusion_property_demand_only():
    # pure LRU with one access per plan: misses(C+1) <= misses(C)
    rng = np.random.default_rng(4)
    E = 10
    for trial in range(50):
        seq = rng.integers(0, E, size=200)
        prev = None
        for C in range(1, E + 1):
            lc = cache.LayerCache(E, C, warm=False)
            for e in seq:
                lc.precise_plan([int(e)])
            m = lc.count["miss"]
            if prev is not None:
                assert m <= prev
            prev = m


def test_streaming_more_experts_than_slots():
    lc = cache.LayerCache(8, 2, warm=True)
    order, entries = lc.precise_plan(range(8))
    assert order == list(range(8))
    assert [x.slot for x in entries] == [0, 1, 0, 1, 0, 1, 0, 1]
    assert [x.after for x in entries] == [-1, -1, 0, 1, 2, 3, 4, 5]
    assert lc.count["miss"] == 6 and lc.count["hit"] == 2


def test_spec_touches_its_list_before_filling():
    # Alg. 2 counts the list's hits while pushing it; Alg. 1 replaces a slot only
    # when the worker starts a copy.  Warm 0, 1 (0 the least recent): the list
    # [2, 0] touches 0 first, so filling 2 evicts 1, not the listed 0.
    lc = cache.LayerCache(4, 2)
    e = lc.spec_plan([2, 0])
    assert [(x.expert, x.slot, x.new, x.victim) for x in e] == [(2, 1, True, 1), (0, 0, False, -1)]
    assert lc.resident() == {0, 2} and lc.count["evict"] == 1
    b = brute.NaiveLRU(4, 2)
    assert b.spec([2, 0]) == [(2, 1, True), (0, 0, False)]


def test_spec_never_evicts_a_predicted_expert():
    # every resident expert has a vote: the fill is skipped, nothing moves
    lc = cache.LayerCache(6, 3)
    e = lc.spec_plan([3], voted=[0, 1, 2, 3])
    assert e[0].skipped and e[0].slot == -1 and lc.count["spec_issued"] == 0 and lc.resident() == {0, 1, 2}
    # one unvoted resident (2): it is the victim, though 0 is older
    e = lc.spec_plan([3, 4], voted=[0, 1, 3, 4])
    assert (e[0].slot, e[0].victim, e[0].new) == (2, 2, True) and e[1].skipped
    assert lc.resident() == {0, 1, 3}
    # a free slot is always taken
    f = cache.LayerCache(6, 3, warm=False)
    assert f.spec_plan([5], voted=[5])[0].slot == 0


def test_random_replays_with_votes():
    rng = np.random.default_rng(21)
    for trial in range(300):
        E = int(rng.integers(2, 9))
        C = int(rng.integers(1, E + 1))
        a, b = cache.LayerCache(E, C), brute.NaiveLRU(E, C)
        for _ in range(int(rng.integers(1, 12))):
            if rng.random() < 0.5:
                Q = rng.choice(E, size=int(rng.integers(1, C + 1)), replace=False).tolist()
                voted = sorted(set(Q) | set(rng.choice(E, size=int(rng.integers(0, E + 1))).tolist()))
                budget = int(rng.integers(-1, 3))
                ea = a.spec_plan(Q, budget, voted=voted)
                eb = b.spec(Q, budget, voted=voted)
                assert [(x.expert, x.slot, x.new) for x in ea] == eb
                # no fill evicts a voted expert or a member of the list
                assert all(x.victim not in voted for x in ea if x.new)
            else:
                P = rng.choice(E, size=int(rng.integers(1, E + 1)), replace=False).tolist()
                order, entries = a.precise_plan(P)
                assert order == b.precise(P)[0]
            _check_invariants(a)
            assert a.count == b.c
