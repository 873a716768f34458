"""The library's static budget planner (moe_plan_percent / moe_plan_bytes, host code in
libmoecache.so) against the oracle planner, field by field, exactly; argument errors."""
import os

import numpy as np
import pytest

from oracle import planner


@pytest.fixture(scope="module")
def mc():
    from paper_2607_09686_amd import build, moecache
    if not os.path.exists(moecache.LIB_PATH):
        build.build()
    moecache.lib()
    return moecache


def random_model(rng):
    E = int(rng.integers(1, 300))
    return {"n_layers": int(rng.integers(1, 100)), "n_experts": E, "top_k": int(rng.integers(1, E + 1)),
            "payload_bytes": int(rng.integers(1, 1 << 34)), "common_bytes": int(rng.integers(0, 1 << 40)),
            "kv_bytes_per_token": int(rng.integers(0, 1 << 20)),
            "overhead_bytes": int(rng.integers(0, 1 << 32)), "target_bytes": int(rng.integers(0, 1 << 46))}


def test_percent_matches_oracle(mc):
    rng = np.random.default_rng(11)
    for i in range(3000):
        m = random_model(rng)
        pct = [int(rng.integers(1, 101)), float(rng.integers(1, 801)) / 8, 12.5, 100.0][i % 4]
        ctx = int(rng.integers(0, 1 << 18))
        assert mc.plan_percent(m, pct, ctx) == planner.plan_percent(m, pct, ctx), (m, pct, ctx)


def test_bytes_matches_oracle(mc):
    rng = np.random.default_rng(12)
    for _ in range(3000):
        m = random_model(rng)
        per = m["n_layers"] * m["payload_bytes"]
        cb = [int(rng.integers(0, 1 << 50)), per * int(rng.integers(0, 300)) + int(rng.integers(0, per)),
              per * m["top_k"] - 1, per * m["n_experts"]][int(rng.integers(0, 4))]
        ctx = int(rng.integers(0, 1 << 18))
        assert mc.plan_bytes(m, cb, ctx) == planner.plan_bytes(m, cb, ctx), (m, cb, ctx)


def test_workload_slot_counts(mc):
    a3b = {"n_layers": 48, "n_experts": 128, "top_k": 8, "payload_bytes": 5013504}
    assert [mc.plan_percent(a3b, p)["slots_per_layer"] for p in (15, 35, 75)] == [19, 45, 96]
    tiny = {"n_layers": 1, "n_experts": 16, "top_k": 2, "payload_bytes": 104448}
    assert mc.plan_percent(tiny, 25)["slots_per_layer"] == 4


@pytest.mark.parametrize("bad", [
    dict(n_layers=0), dict(n_experts=0), dict(top_k=0), dict(top_k=129), dict(payload_bytes=0)])
def test_bad_models_rejected(mc, bad):
    m = {"n_layers": 48, "n_experts": 128, "top_k": 8, "payload_bytes": 5013504}
    m.update(bad)
    with pytest.raises(mc.MoeError):
        mc.plan_percent(m, 15)
    with pytest.raises(mc.MoeError):
        mc.plan_bytes(m, 1 << 30)


def test_bad_arguments_and_overflow_rejected(mc):
    m = {"n_layers": 48, "n_experts": 128, "top_k": 8, "payload_bytes": 5013504}
    for pct in (0.0, -5.0, 100.5, float("nan"), float("inf")):
        with pytest.raises(mc.MoeError):
            mc.plan_percent(m, pct)
    with pytest.raises(mc.MoeError):
        mc.plan_percent(m, 15, -1)
    with pytest.raises(mc.MoeError):   # 48 * 128 * 2^60 bytes does not fit in 64 bits
        mc.plan_percent(dict(m, payload_bytes=1 << 60), 100)
    with pytest.raises(mc.MoeError):   # context * kv bytes per token overflows
        mc.plan_percent(dict(m, kv_bytes_per_token=1 << 40), 15, 1 << 30)
