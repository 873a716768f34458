"""The library's offline miss bound (moe_policy_min, host code in libmoecache.so) against
the oracle's Belady MIN on random traces, exactly; argument errors."""
import os

import numpy as np
import pytest

from oracle.policy import min_misses as oracle_min


@pytest.fixture(scope="module")
def mc():
    from paper_2607_09686_amd import build, moecache
    if not os.path.exists(moecache.LIB_PATH):
        build.build()
    moecache.lib()
    return moecache


def test_matches_oracle_on_random_traces(mc):
    rng = np.random.default_rng(21)
    for _ in range(400):
        E = int(rng.integers(2, 140))
        C = int(rng.integers(1, E + 1))
        k = int(rng.integers(1, C + 1))
        calls = []
        for _ in range(int(rng.integers(0, 80))):
            ids = rng.choice(E, size=int(rng.integers(1, k + 1)), replace=False)
            if rng.random() < 0.3:   # duplicates and any order are allowed
                ids = np.concatenate([ids, ids[:1]])
            calls.append(ids)
        assert mc.min_misses(calls, E, C) == oracle_min(calls, E, C)


def test_textbook_reference_string(mc):
    ref = [[p - 1] for p in (1, 2, 3, 4, 1, 2, 5, 1, 2, 3, 4, 5)]
    assert mc.min_misses(ref, 5, 3) == 7


def test_bad_arguments(mc):
    with pytest.raises(mc.MoeError):
        mc.min_misses([[0, 1, 2]], 4, 2)      # more experts in a call than slots
    with pytest.raises(mc.MoeError):
        mc.min_misses([[0, 5]], 4, 2)         # id out of range
    with pytest.raises(mc.MoeError):
        mc.min_misses([[0]], 4, 0)
    assert mc.min_misses([], 4, 2) == 0
