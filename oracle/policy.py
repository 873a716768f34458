"""Offline lower bound on misses: Belady's MIN for per-call expert sets (oracle; test
infrastructure only).

The paper argues for an optimizer that minimises end-to-end latency under a memory
budget rather than a policy that maximises hit rate (its Discussion).  On a GPU
whose slots do not compete with host memory, the latency of a layer call is set by
the bytes it materialises, so the least possible number of misses for a recorded
route trace bounds every slot policy from below.

Belady's MIN (1966): on a miss with every slot taken, evict the resident block whose
next use lies farthest in the future.  Here a request is a layer call's set S of
distinct experts that must all be resident together (|S| <= C): the experts of S
are never evicted during their own call; among the other residents the victim is the
one used again last (never again counts as infinitely far; ties: the higher expert
id).  The number of misses does not depend on which slot a miss takes, so slots are
not modelled.
"""
import numpy as np

NEVER = 1 << 62


def next_uses(calls, n_experts):
    """nxt[i][e] = index of the first call after i that routes e (NEVER if none)."""
    n = len(calls)
    nxt = np.full((n + 1, n_experts), NEVER, np.int64)
    for i in range(n - 1, -1, -1):
        nxt[i] = nxt[i + 1]
        nxt[i][np.asarray(calls[i], np.int64)] = i
    return nxt[1:]  # row i: first use strictly after call i


def min_misses(calls, n_experts, n_slots):
    """Misses of MIN over the calls (each an iterable of expert ids) from a cold cache."""
    calls = [np.unique(np.asarray(c, np.int64)) for c in calls]
    for S in calls:
        if len(S) > n_slots:
            raise ValueError("a call routes more experts than there are slots")
    nxt = next_uses(calls, n_experts)
    resident = set()
    misses = 0
    for i, S in enumerate(calls):
        need = [e for e in S.tolist() if e not in resident]
        for e in need:
            misses += 1
            if len(resident) == n_slots:
                pinned = set(S.tolist())
                victim = max((v for v in resident if v not in pinned),
                             key=lambda v: (nxt[i][v], v))
                resident.remove(victim)
            resident.add(e)
    return misses
