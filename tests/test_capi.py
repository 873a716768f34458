"""CPU-side checks of the C ABI: the library loads and exports every declared symbol,
the HIP-free LRU slot table agrees bit-exactly with the oracle, argument errors."""
import ctypes
import os
import re

import numpy as np
import pytest

from conftest import ROOT, golden_path
from oracle.lru import LayerLRU

HEADER = os.path.join(ROOT, "include", "moecache.h")


@pytest.fixture(scope="module")
def mc():
    from paper_2607_09686_amd import build, moecache
    if not os.path.exists(moecache.LIB_PATH):
        build.build()
    moecache.lib()
    return moecache


def declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(moe_[a-z_0-9]+)\s*\(", src)))


def test_exports_every_declared_function(mc):
    names = declared_functions()
    assert len(names) >= 15
    L = ctypes.CDLL(mc.LIB_PATH)
    for n in names:
        assert hasattr(L, n), n


def test_lru_matches_oracle_on_random_traces(mc):
    rng = np.random.default_rng(7)
    for trial in range(200):
        E = int(rng.integers(2, 257))
        k = int(rng.integers(1, min(E, 16) + 1))
        C = int(rng.integers(1, E + 1))          # includes over-full calls (|S| > C)
        P = int(rng.integers(1, 1 << 40))
        ours = mc.SlotTable(E, C, P, layer=trial % 5)
        ref = LayerLRU(E, C, P, layer=trial % 5)
        for _ in range(int(rng.integers(1, 60))):
            T = int(rng.integers(1, 4))
            ids = rng.integers(0, E, size=T * k)           # duplicates on purpose
            assert ours.step(ids) == ref.step(ids)
        assert ours.counters().as_tuple() == ref.counters.as_tuple()


def test_lru_golden_traces(mc):
    from test_oracle_lru import _golden_cases
    for case in _golden_cases():
        t = mc.SlotTable(case["E"], case["C"], 1000)
        recs = []
        for call in case["calls"]:
            recs.extend(r[1:] for r in t.step(call))
        assert recs == case["recs"], case["name"]
        h, m, ev = case["counters"]
        assert t.counters().as_tuple() == (h, m, ev, 1000 * m)


def test_lru_rejects_bad_arguments(mc):
    with pytest.raises(mc.MoeError) as e:
        mc.SlotTable(8, 9, 1)
    assert e.value.code == mc.MOE_EINVAL
    t = mc.SlotTable(8, 2, 1)
    with pytest.raises(mc.MoeError):
        t.step([8])
    with pytest.raises(mc.MoeError):
        t.step([-1])


def test_create_rejects_bad_descriptors_before_touching_hip(mc):
    L = mc.lib()
    out = ctypes.c_void_p()
    assert L.moe_cache_create(None, 4, ctypes.byref(out)) == mc.MOE_EINVAL
    base = dict(n_layers=1, n_experts=16, top_k=2, hidden=256, inter=128, qtype=8,
                host_store=1, store_bytes=16 * 104448, hip_stream=None, flags=0)
    cases = [
        (dict(base), 1),                        # budget below top_k
        (dict(base), 17),                       # budget above n_experts
        (dict(base, hidden=96), 4),             # not a multiple of 64
        (dict(base, qtype=3), 4),               # unknown block type
        (dict(base, top_k=17, n_experts=32), 20),
        (dict(base, host_store=None), 4),
    ]
    for d, budget in cases:
        desc = mc.ModelDesc(**d)
        assert L.moe_cache_create(ctypes.byref(desc), budget, ctypes.byref(out)) == mc.MOE_EINVAL
        assert out.value is None
        assert L.moe_last_error()
    L.moe_cache_destroy(None)  # NULL-safe


def test_null_handle_calls_fail_cleanly(mc):
    L = mc.lib()
    c = mc.Counters()
    assert L.moe_cache_counters(None, -1, ctypes.byref(c)) == mc.MOE_EINVAL
    assert L.moe_cache_reset(None) == mc.MOE_EINVAL
    assert L.moe_layer_forward(None, None, 1, None, 0, None, None) == mc.MOE_EINVAL


def test_probes_reject_bad_arguments_before_touching_hip(mc):
    L = mc.lib()
    r, e = ctypes.c_double(), ctypes.c_double()
    for nbytes, iters in ((0, 10), (1000, 10), (16 << 30, 10), (1 << 20, 0), (1 << 20, 20000)):
        assert L.moe_probe_hbm_read(nbytes, iters, ctypes.byref(r), ctypes.byref(e)) == mc.MOE_EINVAL
    assert L.moe_probe_hbm_read(1 << 20, 10, None, ctypes.byref(e)) == mc.MOE_EINVAL
    g = ctypes.c_double()
    assert L.moe_probe_h2d(None, 1 << 20, 1, 1, ctypes.byref(g)) == mc.MOE_EINVAL
