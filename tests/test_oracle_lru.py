"""Pins of the oracle's LRU slot table: hand traces, a brute-force key characterisation,
inclusion across cache sizes, and closed forms."""
import itertools

import numpy as np
import pytest

from conftest import golden_path
from oracle.lru import LayerLRU, simulate, slots_from_percent


def _golden_cases():
    cases, cur = [], None
    for line in open(golden_path("lru_hand_trace.txt")):
        line = line.split("#")[0].split()
        if not line:
            continue
        if line[0] == "case":
            cur = dict(name=line[1], E=int(line[3]), C=int(line[5]), calls=[], recs=[])
        elif line[0] == "call":
            cur["calls"].append([int(v) for v in line[1:]])
        elif line[0] == "rec":
            cur["recs"].append(tuple(int(v) for v in line[1:]))
        elif line[0] == "counters":
            cur["counters"] = tuple(int(v) for v in line[1:])
        elif line[0] == "end":
            cases.append(cur)
    return cases


@pytest.mark.parametrize("case", _golden_cases(), ids=lambda c: c["name"])
def test_hand_worked_traces(case):
    P = 1000
    recs, cnt = simulate(case["calls"], case["E"], case["C"], P)
    assert [r[1:] for r in recs] == case["recs"]
    h, m, ev = case["counters"]
    assert cnt.as_tuple() == (h, m, ev, m * P)


def _brute_force(calls, E, C):
    """Hits and victims from the key characterisation, valid while every call routes <= C experts.

    After call t the resident set is the C experts with the largest key
    (last call that routed it, expert id) among experts routed so far.  A routed
    expert is a hit iff it was resident before the call; the victims are the
    experts that leave the resident set, taken in ascending key order, and the
    ascending misses use the free slots (lowest first) and then the victims' slots.
    """
    last = {}
    slot_of = {}
    out = []
    for t, call in enumerate(calls):
        S = sorted(set(call))
        before = sorted(last, key=lambda e: (last[e], e))[-C:]
        for e in S:
            last[e] = t
        after = sorted(last, key=lambda e: (last[e], e))[-C:]
        leaving = sorted(set(before) - set(after), key=lambda e: (last[e], e))
        free = sorted(set(range(C)) - {slot_of[e] for e in before})
        misses = [e for e in S if e not in before]
        assign = {}
        for i, e in enumerate(misses):
            if i < len(free):
                assign[e] = (free[i], -1)
            else:
                v = leaving[i - len(free)]
                assign[e] = (slot_of.pop(v), v)
        assert len(misses) - len(free) == len(leaving) or (len(leaving) == 0 and len(misses) <= len(free))
        for e in S:
            if e in before:
                out.append((t, e, 1, slot_of[e], -1))
            else:
                s, v = assign[e]
                slot_of[e] = s
                out.append((t, e, 0, s, v))
    return out


def test_exhaustive_small_traces_match_brute_force():
    E = 4
    subsets = [c for r in (1, 2) for c in itertools.combinations(range(E), r)]
    n = 0
    for steps in range(1, 5):
        for calls in itertools.product(subsets, repeat=steps):
            kmax = max(len(c) for c in calls)
            for C in range(kmax, E + 1):
                recs, _ = simulate(calls, E, C, 1)
                assert [r[1:] for r in recs] == _brute_force(calls, E, C), (calls, C)
                n += 1
    assert n > 20000


def test_random_traces_match_brute_force():
    rng = np.random.default_rng(0)
    for trial in range(400):
        E = int(rng.integers(3, 40))
        k = int(rng.integers(1, min(E, 8) + 1))
        C = int(rng.integers(k, E + 1))
        calls = [rng.choice(E, size=k, replace=False) for _ in range(int(rng.integers(1, 40)))]
        recs, _ = simulate(calls, E, C, 1)
        assert [r[1:] for r in recs] == _brute_force(calls, E, C)


def test_inclusion_across_cache_sizes():
    rng = np.random.default_rng(1)
    for trial in range(100):
        E, k = 32, 4
        calls = [rng.choice(E, size=k, replace=False) for _ in range(60)]
        hits_prev = None
        for C in range(k, E + 1):
            recs, cnt = simulate(calls, E, C, 1)
            hits = {(r[1], r[2]) for r in recs if r[3]}
            if hits_prev is not None:
                assert hits_prev <= hits
            hits_prev = hits


def test_full_cache_closed_form():
    rng = np.random.default_rng(2)
    E, k = 16, 2
    calls = [rng.choice(E, size=k, replace=False) for _ in range(200)]
    recs, cnt = simulate(calls, E, E, 7)
    seen = set()
    for r in recs:
        assert r[5] == -1
        assert r[3] == (r[2] in seen)
        seen.add(r[2])
    assert cnt.evictions == 0 and cnt.misses == len(seen)
    # once every expert has been seen, the hit rate is 1
    first_all = next(i for i in range(len(calls)) if len(set(np.concatenate(calls[: i + 1]))) == E)
    assert all(r[3] == 1 for r in recs if r[1] > first_all)


def test_cold_overfull_call_closed_form():
    for E, C in ((128, 45), (20, 7), (9, 1)):
        lru = LayerLRU(E, C, 5)
        routed = list(range(0, E, 1))
        recs = lru.step(routed)
        for j, r in enumerate(recs):
            assert r[3] == 0
            assert r[4] == j % C
            assert r[5] == (routed[j - C] if j >= C else -1)
        assert lru.counters.as_tuple() == (0, E, E - C, 5 * E)


def test_bytes_invariant_and_record_counts():
    rng = np.random.default_rng(3)
    P = 5013504
    lru = LayerLRU(128, 19, P)
    total = 0
    for _ in range(300):
        ids = rng.choice(128, size=8, replace=False)
        recs = lru.step(ids)
        total += len(recs)
        assert [r[2] for r in recs] == sorted(ids.tolist())
    c = lru.counters
    assert c.materialized_bytes == c.misses * P
    assert c.hits + c.misses == total


def test_slot_rule_reproduces_named_budgets():
    # 15% of 128 experts -> 19 slots, 35% -> 45, 75% -> 96, 25% of 16 -> 4
    assert slots_from_percent(15, 128, 8) == 19
    assert slots_from_percent(35, 128, 8) == 45
    assert slots_from_percent(75, 128, 8) == 96
    assert slots_from_percent(25, 16, 2) == 4
    assert slots_from_percent(1, 128, 8) == 8
    assert slots_from_percent(100, 128, 8) == 128


def test_rejects_bad_sizes():
    with pytest.raises(ValueError):
        LayerLRU(8, 0, 1)
    with pytest.raises(ValueError):
        LayerLRU(8, 9, 1)
    with pytest.raises(ValueError):
        LayerLRU(8, 2, 1).step([8])


def test_score_policy_hand_worked():
    """Score eviction (one-token calls): the victim is the resident outside the call with the
    lowest logit, the higher id on a tie.  Worked by hand:
      call 0 routes {0, 1, 2}: three misses into slots 0, 1, 2;
      call 1 routes {3} with z = (0.5, -1, 2, 3, 0, 0): residents 0, 1, 2 have logits
             0.5, -1, 2, so expert 1 leaves slot 1 (LRU would evict expert 0);
      call 2 routes {0, 4} with z = (9, 0, 1, 1, 5, 0): 0 hits; 4 misses; residents outside
             the call are 2 and 3, both at logit 1: the higher id, 3, leaves slot 1."""
    lru = LayerLRU(6, 3, 10, 0, policy="score")
    assert lru.step([0, 1, 2], np.zeros(6)) == [(0, 0, 0, 0, 0, -1), (0, 0, 1, 0, 1, -1),
                                               (0, 0, 2, 0, 2, -1)]
    assert lru.step([3], np.array([0.5, -1.0, 2.0, 3.0, 0.0, 0.0])) == [(0, 1, 3, 0, 1, 1)]
    assert lru.step([0, 4], np.array([9.0, 0.0, 1.0, 1.0, 5.0, 0.0])) == [
        (0, 2, 0, 1, 0, -1), (0, 2, 4, 0, 1, 3)]
    assert lru.counters.as_tuple() == (1, 5, 2, 50)


def test_score_policy_with_recency_logits_is_lru():
    """Fed 'logits' that rank the residents by their last use (z[v] = a clock value taken by
    v at its last use, calls in order and ascending ids within a call), the score rule picks
    the least recently used resident: records equal the LRU table's."""
    rng = np.random.default_rng(17)
    for _ in range(200):
        E, C = int(rng.integers(4, 24)), 0
        k = int(rng.integers(1, 5))
        C = int(rng.integers(max(k, 1), E + 1))
        lru = LayerLRU(E, C, 3, 2)
        sc = LayerLRU(E, C, 3, 2, policy="score")
        last, clock = np.full(E, -1.0), 0
        for _ in range(int(rng.integers(1, 40))):
            S = rng.choice(E, size=k, replace=False)
            assert sc.step(S, last.copy()) == lru.step(S)
            for e in sorted(S.tolist()):
                clock += 1
                last[e] = clock
        assert sc.counters.as_tuple() == lru.counters.as_tuple()


def test_score_policy_bounds_and_nan():
    """Misses never below the offline bound; a NaN logit ranks lowest (evicted first)."""
    from oracle.policy import min_misses
    rng = np.random.default_rng(18)
    for _ in range(100):
        E, C, k = 16, int(rng.integers(2, 10)), 2
        calls = [rng.choice(E, size=k, replace=False) for _ in range(50)]
        sc = LayerLRU(E, C, 1, 0, policy="score")
        for S in calls:
            sc.step(S, rng.normal(size=E))
        assert sc.counters.misses >= min_misses(calls, E, C)
    sc = LayerLRU(4, 2, 1, 0, policy="score")
    sc.step([0, 1], np.zeros(4))
    assert sc.step([2], np.array([np.nan, 5.0, 0.0, 0.0]))[0][5] == 0
