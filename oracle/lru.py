"""Per-layer LRU expert-slot table with hit / miss accounting (oracle; test infrastructure only).

The paper's Native Serving Path section: each layer owns a fixed number of
slots for routed experts; a miss copies the expert's block into a free slot
and records which slot now holds that expert.  The paper states no eviction
rule; least-recently-used is used here, with these
readings:

For one layer call, S is the ascending set of distinct experts routed by any
token of the call (one lookup per distinct expert per call).

1. every e in S, ascending, gets stamp[e] = ++clock;
2. e in S that already has a slot is a hit;
3. the misses, ascending, are materialised one after another: the slot is the
   lowest-index free slot if any, otherwise the slot of the resident expert
   with the smallest stamp (it is evicted);  materialised_bytes grows by the
   payload size P per miss.

One record (layer, step, expert, hit, slot, evicted-or--1) is emitted per e in
S, in ascending expert order.

Policy "score" (an alternative for one-token calls, not the paper's): the victim
of rule 3 is instead the resident outside S whose router logit for the call's
token is lowest (ties: the higher id) -- the expert the current token wants
least, as a guess at the next token's routes.
"""
from dataclasses import dataclass, field
from typing import List


@dataclass
class Counters:
    hits: int = 0
    misses: int = 0
    evictions: int = 0
    materialized_bytes: int = 0

    def as_tuple(self):
        return (self.hits, self.misses, self.evictions, self.materialized_bytes)

    def __add__(self, o):
        return Counters(self.hits + o.hits, self.misses + o.misses,
                        self.evictions + o.evictions, self.materialized_bytes + o.materialized_bytes)


@dataclass
class LayerLRU:
    n_experts: int
    n_slots: int
    payload_bytes: int
    layer: int = 0
    policy: str = "lru"       # "lru", or "score": see step()
    slot_of: List[int] = field(default_factory=list)
    expert_in: List[int] = field(default_factory=list)
    stamp: List[int] = field(default_factory=list)
    clock: int = 0
    step_no: int = 0
    counters: Counters = field(default_factory=Counters)

    def __post_init__(self):
        if not (1 <= self.n_slots <= self.n_experts):
            raise ValueError("n_slots must lie in [1, n_experts]")
        self.reset()

    def reset(self):
        self.slot_of = [-1] * self.n_experts
        self.expert_in = [-1] * self.n_slots
        self.stamp = [0] * self.n_experts
        self.clock = 0
        self.step_no = 0
        self.counters = Counters()

    def step(self, routed, z=None):
        """Apply one layer call whose tokens routed the experts in ``routed``.

        With policy "score" (one-token calls), ``z`` holds the token's router logits
        for every expert, and the victim of a miss with every slot taken is the
        resident outside the call with the lowest logit (ties: the higher id) instead
        of the least recently used one.  Stamps are kept either way.

        Returns the list of records (layer, step, expert, hit, slot, evicted).
        """
        S = sorted(set(int(e) for e in routed))
        if self.policy == "score":
            if z is None or len(S) > self.n_slots:
                raise ValueError("the score policy needs the logits and at most n_slots experts")
        for e in S:
            if not (0 <= e < self.n_experts):
                raise ValueError("expert id out of range")
        for e in S:                                   # rule 1
            self.clock += 1
            self.stamp[e] = self.clock
        hit = {e: self.slot_of[e] >= 0 for e in S}    # rule 2
        rec = {}
        for e in S:
            if hit[e]:
                self.counters.hits += 1
                rec[e] = (self.slot_of[e], -1)
        for e in S:                                   # rule 3, ascending misses
            if hit[e]:
                continue
            self.counters.misses += 1
            self.counters.materialized_bytes += self.payload_bytes
            free = [s for s in range(self.n_slots) if self.expert_in[s] < 0]
            if free:
                s, victim = free[0], -1
            elif self.policy == "score":
                victim = min((v for v in self.expert_in if v not in S),
                             key=lambda v: (_logit_key(z[v]), -v))
                s = self.slot_of[victim]
                self.slot_of[victim] = -1
                self.counters.evictions += 1
            else:
                victim = min((self.expert_in[s] for s in range(self.n_slots)),
                             key=lambda v: self.stamp[v])
                s = self.slot_of[victim]
                self.slot_of[victim] = -1
                self.counters.evictions += 1
            self.expert_in[s] = e
            self.slot_of[e] = s
            rec[e] = (s, victim)
        out = [(self.layer, self.step_no, e, int(hit[e]), rec[e][0], rec[e][1]) for e in S]
        self.step_no += 1
        return out


def _logit_key(v):
    """A logit as an eviction key: NaN ranks below every number (evicted first)."""
    v = float(v)
    return float("-inf") if v != v else v


def simulate(calls, n_experts, n_slots, payload_bytes, layer=0):
    """Run a sequence of layer calls (each an iterable of routed ids) from cold.

    Returns (records, counters)."""
    lru = LayerLRU(n_experts, n_slots, payload_bytes, layer)
    recs = []
    for routed in calls:
        recs.extend(lru.step(routed))
    return recs, lru.counters


def slots_from_percent(percent, n_experts, top_k):
    """Slots per layer for a cache percentage: nearest integer to p*E, clamped to [k, E].

    The paper lists the inputs of the slot count (cache bytes, routed layer
    count, per-slot block size, active experts per token, experts per layer)
    but not the formula; with equal-size slots the cache percentage is p*E
    slots per layer, rounded half-up.
    """
    s = int(percent * n_experts / 100.0 + 0.5)
    return max(top_k, min(n_experts, s))
