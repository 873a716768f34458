"""Static budget planner (oracle; test infrastructure only).

The paper's Native Serving Path section: the slot count of every routed layer
is derived from the requested cache bytes, the routed layer count, the bytes
of one expert block (one slot), the active experts per token and the experts
per layer.  Its Static Budget Check section: with C the resident common
tensor bytes, E(p) the expert-cache bytes at cache percentage p, K(n) the
KV-cache bytes at context length n and O the runtime overhead,

    L(p, n) = C + E(p) + K(n)        static lower bound
    F(p, n) = C + E(p) + K(n) + O    runtime footprint

and a configuration is rejected before load when L already exceeds the
serving target.

Readings (the paper lists the inputs of the slot count but no formula):
* every layer gets the same number of equal-size slots, so the expert cache
  is E = n_layers * slots * P bytes;
* from a percentage p: slots = nearest integer to p/100 * n_experts (halves
  up); from a byte budget B: slots = floor(B / (n_layers * P)); either way
  clamped to [top_k, n_experts] (a layer must hold one token's top_k experts
  at once, and never needs more than all of them);
* K(n) = n * (KV bytes per token): the paper's KV figures for one model at
  4K and 32K context are in the ratio 8 : 1 exactly;
* the check compares L, not F, with the target ("rejected when the lower
  bound already exceeds the target"); F is reported.

Exact integer arithmetic throughout (percentages as exact fractions).
"""
from fractions import Fraction


def slots_for_percent(percent, n_experts, top_k):
    """(slots, clamped): nearest integer to percent/100 * n_experts, halves up, clamped to [k, E]."""
    want = Fraction(percent) * n_experts / 100
    s = (want + Fraction(1, 2)).__floor__()
    return _clamp(s, n_experts, top_k)


def slots_for_bytes(cache_bytes, n_layers, payload_bytes, n_experts, top_k):
    """(slots, clamped): floor(cache_bytes / (n_layers * P)), clamped to [k, E]."""
    s = cache_bytes // (n_layers * payload_bytes)
    return _clamp(s, n_experts, top_k)


def _clamp(s, n_experts, top_k):
    c = max(top_k, min(n_experts, s))
    return int(c), int(c != s)


def plan(slots, clamped, n_layers, payload_bytes, common_bytes, kv_bytes_per_token, overhead_bytes,
         target_bytes, context_tokens):
    """The static check for a given slot count.  Returns a dict of the plan's quantities."""
    e = n_layers * slots * payload_bytes
    k = context_tokens * kv_bytes_per_token
    lower = common_bytes + e + k
    return {"slots_per_layer": slots, "clamped": clamped, "expert_cache_bytes": e, "kv_bytes": k,
            "lower_bound_bytes": lower, "footprint_bytes": lower + overhead_bytes,
            "feasible": int(lower <= target_bytes)}


def plan_percent(m, percent, context_tokens):
    """m: dict with n_layers, n_experts, top_k, payload_bytes, common_bytes, kv_bytes_per_token,
    overhead_bytes, target_bytes."""
    s, c = slots_for_percent(percent, m["n_experts"], m["top_k"])
    return plan(s, c, m["n_layers"], m["payload_bytes"], m["common_bytes"], m["kv_bytes_per_token"],
                m["overhead_bytes"], m["target_bytes"], context_tokens)


def plan_bytes(m, cache_bytes, context_tokens):
    s, c = slots_for_bytes(cache_bytes, m["n_layers"], m["payload_bytes"], m["n_experts"], m["top_k"])
    return plan(s, c, m["n_layers"], m["payload_bytes"], m["common_bytes"], m["kv_bytes_per_token"],
                m["overhead_bytes"], m["target_bytes"], context_tokens)
