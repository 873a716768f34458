"""Pins of the offline miss bound (oracle/policy.py, Belady's MIN for per-call expert sets):
the textbook reference string, exhaustive search over every demand policy on small traces,
and the bounds it must respect."""
import itertools

import numpy as np

from oracle.lru import simulate
from oracle.policy import min_misses


def brute_min(calls, n_slots):
    """Fewest misses over every demand policy: after a call the resident set R' holds the
    call's set S, at most n_slots experts, and nothing that was neither resident nor routed."""
    states = {frozenset(): 0}
    for S in calls:
        S = frozenset(S)
        nxt = {}
        for R, m in states.items():
            miss = len(S - R)
            keep = sorted(R - S)
            room = n_slots - len(S)
            for r in range(0, min(room, len(keep)) + 1):
                for extra in itertools.combinations(keep, r):
                    R2 = S | frozenset(extra)
                    if nxt.get(R2, 1 << 30) > m + miss:
                        nxt[R2] = m + miss
        states = nxt
    return min(states.values())


def test_textbook_reference_string():
    # Reference string 1 2 3 4 1 2 5 1 2 3 4 5 with 3 frames: the optimal policy faults 7
    # times and LRU 10 times (the operating-systems textbook example of page replacement).
    ref = [[p - 1] for p in (1, 2, 3, 4, 1, 2, 5, 1, 2, 3, 4, 5)]
    assert min_misses(ref, 5, 3) == 7
    assert simulate(ref, 5, 3, 1)[1].misses == 10
    assert min_misses(ref, 5, 4) == 6


def test_equals_exhaustive_search_on_small_traces():
    rng = np.random.default_rng(5)
    n = 0
    for _ in range(400):
        E, C = int(rng.integers(3, 7)), int(rng.integers(1, 4))
        k = int(rng.integers(1, C + 1))
        calls = [rng.choice(E, size=int(rng.integers(1, k + 1)), replace=False).tolist()
                 for _ in range(int(rng.integers(1, 8)))]
        assert min_misses(calls, E, C) == brute_min(calls, C), (E, C, calls)
        n += 1
    assert n == 400


def test_bounds():
    rng = np.random.default_rng(6)
    for _ in range(200):
        E, k = 32, 4
        calls = [rng.choice(E, size=k, replace=False) for _ in range(60)]
        distinct = len(set(np.concatenate(calls).tolist()))
        prev = None
        for C in range(k, E + 1, 4):
            m = min_misses(calls, E, C)
            assert distinct <= m <= simulate(calls, E, C, 1)[1].misses
            if prev is not None:
                assert m <= prev
            prev = m
        assert min_misses(calls, E, E) == distinct
