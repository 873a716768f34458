"""Pins of the verification-window schedule (oracle/verify.py) and the seeded acceptance
draws: hand-worked schedules, the all-pass / none-pass / no-horizon closed forms, and the
union-of-experts lookups reducing to decode when a window has one token."""
import numpy as np

import synth
from oracle import router as oracle_router
from oracle.lru import simulate
from oracle.verify import schedule, window_union


def test_hand_worked_schedule():
    # n = 10, horizon 4.  Step 0 passes drafts 0, 1 then fails draft 2: 2 accepted, 3 tokens,
    # next window at 3.  Step 1 fails draft 0: 1 token, next at 4.  Step 2 passes all four:
    # 5 tokens, next at 9.  Step 3 passes all, but only 1 token is still wanted.
    acc = np.array([[1, 1, 0, 1], [0, 1, 1, 1], [1, 1, 1, 1], [1, 1, 1, 1]], bool)
    assert schedule(10, 4, acc) == [(0, 2, 3), (3, 0, 1), (4, 4, 5), (9, 4, 1)]


def test_closed_forms():
    n, h = 96, 4
    allp = np.ones((n, h), bool)
    s = schedule(n, h, allp)
    assert [t for t, _, _ in s] == list(range(0, n, h + 1))
    assert len(s) == -(-n // (h + 1))
    nonep = np.zeros((n, h), bool)
    assert schedule(n, h, nonep) == [(t, 0, 1) for t in range(n)]
    assert schedule(n, 0, np.zeros((n, 0), bool)) == [(t, 0, 1) for t in range(n)]


def test_schedule_invariants_on_random_draws():
    rng = np.random.default_rng(3)
    for _ in range(300):
        n, h = int(rng.integers(1, 60)), int(rng.integers(0, 7))
        acc = rng.random((n, h)) < rng.random()
        s = schedule(n, h, acc)
        assert sum(g for _, _, g in s) == n
        t = 0
        for start, a, g in s:
            assert start == t and 0 <= a <= h and 1 <= g <= a + 1
            # accepted = length of the leading run of passes
            row = acc[len([x for x in s if x[0] < start])]
            assert a == (h if row.all() else int(np.argmin(row)))
            t += g


def test_acceptance_draws():
    a = synth.acceptance(64, 4, 0.75, 2)
    assert a.shape == (64, 4) and a.dtype == bool
    assert np.array_equal(a, synth.acceptance(64, 4, 0.75, 2))
    # draft j of step s: top 53 bits of Philox word j under key(5, seed, 0, 0, 0)
    k0 = synth.key(5, 2, 0, 0, 0)
    for s in (0, 17, 63):
        words = synth.philox4x64((s, 0, 0, 0), (k0, 0))
        assert [bool((w >> 11) / 2.0 ** 53 < 0.75) for w in words] == a[s].tolist()
    big = synth.acceptance(4000, 4, 0.75, 9)
    assert abs(big.mean() - 0.75) < 0.02
    assert not synth.acceptance(10, 4, 0.0, 2).any() and synth.acceptance(10, 4, 1.0, 2).all()


def test_union_lookups_reduce_to_decode():
    """Windows of one token (horizon 0) give exactly the decode run's cache records; a window
    repeating one token routes to that token's k experts only."""
    wl = synth.WORKLOADS["tiny"]
    R = synth.router(wl)[0]
    X = synth.hidden(wl, n_tokens=24)
    idx, _, _ = oracle_router.topk(oracle_router.logits(X, R), wl.top_k)
    steps = schedule(24, 0, np.zeros((24, 0), bool))
    win = [window_union(idx[t:t + 1]) for t, _, _ in steps]
    dec = [np.unique(idx[t]) for t in range(24)]
    assert simulate(win, 16, 4, wl.payload_bytes) == simulate(dec, 16, 4, wl.payload_bytes)
    same = np.repeat(idx[:1], 5, axis=0)
    assert np.array_equal(window_union(same), np.unique(idx[0]))
    for t in range(20):
        u = window_union(idx[t:t + 5])
        assert len(u) <= min(wl.n_experts, 5 * wl.top_k)
        assert set(np.unique(idx[t])) <= set(u.tolist())
