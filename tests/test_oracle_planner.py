"""Pins of the static budget planner oracle (oracle/planner.py) to the paper.

The paper prints no topology (layer counts, expert sizes), so its byte figures
cannot be recomputed from first principles.  What they do fix:
* a KV model linear in the context: one bytes-per-token constant reproduces
  both printed Gemma Q8 KV sizes;
* the planner's rule L = C + E(p) + K(n) against the target: the two rejected
  Gemma Q8 32K cells fix C and the expert-store size S (with E(p) = p S, the
  planner's slot count at a fine slot granularity); the rule then has to
  reproduce the accept / reject decision of the other eight Gemma Q8 cells the
  paper reports (all five 4K cells ran, 35 % at 32K ran);
* the slot counts of the configured workloads (nearest integer to p E).
"""
from fractions import Fraction

import pytest

from conftest import golden_path
from oracle import planner

GIB = 1 << 30


def golden():
    g = {"kv": {}, "reject": {}, "settings": {}, "ran": {}}
    for line in open(golden_path("static_plan_paper.txt")):
        line = line.split("#", 1)[0].split()
        if not line:
            continue
        key, rest = line[0], line[1:]
        if key == "kv":
            g["kv"][(rest[0], int(rest[1]))] = Fraction(rest[2])
        elif key == "reject":
            g["reject"][(rest[0], int(rest[1]), int(rest[2]))] = Fraction(rest[3])
        elif key == "settings":
            g["settings"][rest[0]] = [int(v) for v in rest[1:]]
        elif key == "ran":
            g["ran"][(rest[0], int(rest[1]))] = [int(v) for v in rest[2:]]
        else:
            g[key] = int(rest[0])
    return g


def gib4(b):
    """Bytes as GiB rounded to 4 decimals, as the paper prints them."""
    return round(Fraction(b, GIB), 4)


def test_slot_counts_of_the_workloads():
    assert planner.slots_for_percent(15, 128, 8) == (19, 0)
    assert planner.slots_for_percent(35, 128, 8) == (45, 0)
    assert planner.slots_for_percent(75, 128, 8) == (96, 0)
    assert planner.slots_for_percent(25, 16, 2) == (4, 0)
    assert planner.slots_for_percent(1, 128, 8) == (8, 1)      # below top_k: clamped up
    assert planner.slots_for_percent(100, 128, 8) == (128, 0)
    assert planner.slots_for_percent(12.5, 4, 1) == (1, 0)     # exact half rounds up: 0.5 -> 1
    assert planner.slots_for_percent(37.5, 4, 1) == (2, 0)     # 1.5 -> 2


def test_kv_linear_in_context():
    g = golden()
    k4, k32 = g["kv"][("gemma_q8", 4096)], g["kv"][("gemma_q8", 32768)]
    per_token = round(k32 * GIB / 32768)
    assert per_token * 32768 == k32 * GIB          # 6.8750 GiB is exact in bytes
    for n, k in ((4096, k4), (32768, k32)):
        p = planner.plan(19, 0, 1, 1, 0, per_token, 0, 0, n)
        assert gib4(p["kv_bytes"]) == k


def gemma_model(g):
    """C and S from the two rejected Gemma Q8 32K cells, as a planner model with 10^4 slots."""
    k32 = g["kv"][("gemma_q8", 32768)] * GIB
    l50 = g["reject"][("gemma_q8", 32768, 50)] * GIB
    l65 = g["reject"][("gemma_q8", 32768, 65)] * GIB
    S = (l65 - l50) / Fraction(15, 100)
    C = l50 - S / 2 - k32
    n_experts = 10000
    return {"n_layers": 1, "n_experts": n_experts, "top_k": 1, "payload_bytes": round(S / n_experts),
            "common_bytes": round(C), "kv_bytes_per_token": round(k32 / 32768), "overhead_bytes": 0,
            "target_bytes": g["target_gib"] * GIB}


def test_paper_decisions_for_gemma_q8():
    g = golden()
    m = gemma_model(g)
    ran = {(ctx, p) for (prof, ctx), ps in g["ran"].items() if prof == "gemma_q8" for p in ps}
    rejected = {(ctx, p) for (prof, ctx, p) in g["reject"] if prof == "gemma_q8"}
    assert len(ran) == 6 and len(rejected) == 2
    for ctx in (4096, 32768):
        for p in g["settings"]["gemma_q8"]:
            plan = planner.plan_percent(m, p, ctx)
            if (ctx, p) in rejected:
                assert plan["feasible"] == 0, (ctx, p)
                assert gib4(plan["lower_bound_bytes"]) == g["reject"][("gemma_q8", ctx, p)]
            elif (ctx, p) in ran:
                assert plan["feasible"] == 1, (ctx, p, float(Fraction(plan["lower_bound_bytes"], GIB)))


def test_rejected_cells_exceed_the_target_and_totals_add_up():
    g = golden()
    for v in g["reject"].values():
        assert v > g["target_gib"]
    n_cells = sum(len(s) for s in g["settings"].values()) * 2      # two contexts
    assert n_cells == g["unique_cells"]
    assert n_cells - len(g["reject"]) == g["feasible_cells"]


def test_bytes_round_trip_and_clamping():
    m = {"n_layers": 48, "n_experts": 128, "top_k": 8, "payload_bytes": 5013504, "common_bytes": 0,
         "kv_bytes_per_token": 0, "overhead_bytes": 0, "target_bytes": 1 << 62}
    for pct in (15, 35, 75):
        p = planner.plan_percent(m, pct, 0)
        q = planner.plan_bytes(m, p["expert_cache_bytes"], 0)
        assert q["slots_per_layer"] == p["slots_per_layer"] and q["clamped"] == 0
        # one byte short of the next slot in every layer still gives the same count
        q2 = planner.plan_bytes(m, p["expert_cache_bytes"] + 48 * 5013504 - 1, 0)
        assert q2["slots_per_layer"] == p["slots_per_layer"]
    assert planner.plan_bytes(m, 0, 0)["slots_per_layer"] == 8
    assert planner.plan_bytes(m, 0, 0)["clamped"] == 1
    big = planner.plan_bytes(m, 1 << 60, 0)
    assert big["slots_per_layer"] == 128 and big["clamped"] == 1


def test_lower_bound_monotone_and_footprint():
    m = {"n_layers": 30, "n_experts": 128, "top_k": 8, "payload_bytes": 6690816,
         "common_bytes": 3 * GIB, "kv_bytes_per_token": 98304, "overhead_bytes": GIB // 2,
         "target_bytes": 18 * GIB}
    prev = None
    for pct in range(1, 101):
        p = planner.plan_percent(m, pct, 32768)
        assert p["footprint_bytes"] == p["lower_bound_bytes"] + GIB // 2
        assert p["lower_bound_bytes"] == (3 * GIB + 30 * p["slots_per_layer"] * 6690816
                                          + 32768 * 98304)
        if prev:
            assert p["lower_bound_bytes"] >= prev["lower_bound_bytes"]
            assert p["feasible"] <= prev["feasible"]
        prev = p
    assert planner.plan_percent(m, 15, 4096)["lower_bound_bytes"] < \
        planner.plan_percent(m, 15, 32768)["lower_bound_bytes"]
