"""GPU parity of the decode path (one token per layer call) through the C ABI, on
small workloads the oracle finishes in seconds, plus edge cases and error paths."""
import numpy as np
import pytest

import synth
from gpu_common import (check_routes, check_y, log, make_cache, oracle_layer_y, replay_trace,
                        residual_slack, store_buffer, torch_cuda)

pytestmark = pytest.mark.gpu


def run_decode(wl, budget, residual=False, device_store=False, n_tokens=None, store=None,
               timing=False, prenorm=False, copy_mode="kernel", X=None, poison=False):
    torch = torch_cuda()
    n_tokens = wl.n_tokens if n_tokens is None else n_tokens
    log(f"decode {wl.name} E={wl.n_experts} k={wl.top_k} H={wl.hidden} I={wl.inter} "
        f"{wl.qtype} L={wl.n_layers} C={budget} T={n_tokens} residual={residual} prenorm={prenorm} "
        f"copy={copy_mode}")
    keep, ptr, arr = store if store is not None else store_buffer(wl, device=device_store)
    R = synth.router(wl)
    X = synth.hidden(wl, n_tokens=n_tokens) if X is None else X
    Rd = torch.from_numpy(R).cuda()
    cache = make_cache(wl, ptr, budget, trace=True, residual=residual, timing=timing,
                       prenorm=prenorm, copy_mode=copy_mode)
    if poison:
        cache.fill_slots(0xFF)   # every slot scale reads NaN until its expert is copied in
    calls = [[] for _ in range(wl.n_layers)]
    worst = 0.0
    y = torch.empty(wl.hidden, dtype=torch.float32, device="cuda")
    for t in range(n_tokens):
        for l in range(wl.n_layers):
            xh = X[t] if l == 0 else (X[t] + 0.25 * l).astype(np.float32)
            x = torch.from_numpy(xh).cuda()
            delta, idx, w = cache.layer_forward(x, Rd[l], l, y, routes=True)
            torch.cuda.synchronize()
            ys = y.cpu().numpy()
            yg = ys.astype(np.float64)
            slack = None
            if residual:
                yg = yg - xh.astype(np.float64)
                slack = residual_slack(ys)[None]
            idx_or, w_or, z, flipped = check_routes(xh[None], R[l], wl.top_k, idx, w, prenorm)
            yo = oracle_layer_y(xh[None], R[l], arr, wl, l, idx_or, w_or, z, idx, flipped,
                                prenorm=prenorm)
            worst = max(worst, check_y(yg[None], yo, f"token {t} layer {l}", slack=slack))
            calls[l].append(idx[0])
            assert delta.hits + delta.misses == len(set(idx[0].tolist()))
            assert delta.materialized_bytes == delta.misses * wl.payload_bytes
    recs, cnt = replay_trace(calls, wl, budget)
    got = sorted(cache.read_trace(), key=lambda r: (r[0], r[1], r[2]))
    assert got == sorted(recs, key=lambda r: (r[0], r[1], r[2]))
    assert cache.counters().as_tuple() == cnt.as_tuple()
    log(f"  ok: worst err/rms {worst:.2e}, counters {cache.counters()}")
    return cache, calls, worst


@pytest.mark.parametrize("copy_mode", ["kernel", "split", "side", "sdma"])
def test_tiny_decode_parity(copy_mode):
    wl = synth.WORKLOADS["tiny"]
    cache, calls, worst = run_decode(wl, wl.budget_slots, copy_mode=copy_mode)
    c = cache.counters()
    assert c.misses > 0 and c.hits > 0 and c.evictions > 0
    cache.close()


def test_tiny_residual_mode():
    wl = synth.WORKLOADS["tiny"]
    run_decode(wl, wl.budget_slots, residual=True, n_tokens=16)[0].close()


@pytest.mark.parametrize("copy_mode", ["kernel", "split", "side", "sdma"])
def test_prenorm_residual_multi_layer(copy_mode):
    wl = synth.WORKLOADS["tiny"].with_(n_layers=4, name="tiny4")
    run_decode(wl, 4, residual=True, prenorm=True, n_tokens=16, copy_mode=copy_mode)[0].close()
    wl = wl.with_(qtype="q4_0", name="tiny4_q4")
    run_decode(wl, 5, residual=True, prenorm=True, n_tokens=8, copy_mode=copy_mode)[0].close()


def test_full_cache_reaches_hit_rate_one():
    wl = synth.WORKLOADS["tiny"]
    cache, calls, _ = run_decode(wl, wl.n_experts)
    seen, first_all = set(), None
    for t, ids in enumerate(calls[0]):
        seen |= set(ids.tolist())
        if len(seen) == wl.n_experts and first_all is None:
            first_all = t
    c = cache.counters()
    assert c.evictions == 0 and c.misses == len(seen)
    tr = replay_trace(calls, wl, wl.n_experts)[0]
    if first_all is not None:
        assert all(r[3] == 1 for r in tr if r[1] > first_all)
    cache.close()


def test_minimum_budget_equals_top_k():
    wl = synth.WORKLOADS["tiny"]
    run_decode(wl, wl.top_k, n_tokens=24)[0].close()


def test_q4_0_tiny():
    wl = synth.WORKLOADS["tiny"].with_(qtype="q4_0", name="tiny_q4")
    run_decode(wl, wl.budget_slots, n_tokens=24)[0].close()


@pytest.mark.parametrize("shape", [(64, 64, 1, 1, 1), (320, 192, 5, 3, 3), (1024, 384, 40, 6, 9),
                                   (768, 1408, 256, 8, 40), (2816, 704, 64, 16, 17),
                                   (8192, 64, 3, 2, 2), (128, 8192, 4, 1, 1),
                                   (1024, 768, 256, 16, 20)])  # E, top_k, top_k * inter at the limits
def test_other_shapes(shape):
    H, I, E, k, C = shape
    for qt in ("q8_0", "q4_0"):
        wl = synth.WORKLOADS["tiny"].with_(hidden=H, inter=I, n_experts=E, top_k=k, qtype=qt,
                                           name=f"shape{H}x{I}x{E}")
        run_decode(wl, C, n_tokens=6)[0].close()


@pytest.mark.parametrize("shape", [(320, 192, 5, 3, 3), (2816, 704, 64, 16, 17), (4096, 256, 32, 4, 6)])
def test_split_copy_matches_fused(shape):
    """The default decode launch (miss copies fused with gate/up) and the split
    launches (copy kernel, then gate/up) give bit-identical outputs and equal traces."""
    torch = torch_cuda()
    H, I, E, k, C = shape
    for qt in ("q8_0", "q4_0"):
        wl = synth.WORKLOADS["tiny"].with_(hidden=H, inter=I, n_experts=E, top_k=k, qtype=qt,
                                           n_layers=2, name=f"fuse{H}x{I}x{E}")
        keep, ptr, arr = store_buffer(wl)
        R = torch.from_numpy(synth.router(wl)).cuda()
        X = torch.from_numpy(synth.hidden(wl, n_tokens=10)).cuda()
        res = []
        for mode in ("kernel", "split"):
            cache = make_cache(wl, ptr, C, trace=True, residual=True, prenorm=True, copy_mode=mode)
            outs = []
            for t in range(X.shape[0]):
                x = X[t].contiguous()
                for l in range(wl.n_layers):
                    y = torch.empty_like(x)
                    cache.layer_forward(x, R[l], l, y)
                    x = y
                outs.append(x)
            res.append((torch.stack(outs).cpu().numpy(), sorted(cache.read_trace())))
            cache.close()
        np.testing.assert_array_equal(res[0][0].view(np.uint32), res[1][0].view(np.uint32))
        assert res[0][1] == res[1][1]


def test_multi_layer_and_reset():
    torch = torch_cuda()
    wl = synth.WORKLOADS["tiny"].with_(n_layers=3, name="tiny3")
    store = store_buffer(wl)
    cache, calls, _ = run_decode(wl, 4, n_tokens=10, store=store)
    per_layer = [cache.counters(l).as_tuple() for l in range(3)]
    tot = cache.counters().as_tuple()
    assert tuple(sum(v) for v in zip(*per_layer)) == tot
    cache.reset()
    assert cache.counters().as_tuple() == (0, 0, 0, 0)
    assert cache.read_trace() == []
    cache.close()


def test_all_experts_routed_with_identical_experts_is_dense_ffn():
    torch = torch_cuda()
    from oracle import ffn, quant
    wl = synth.WORKLOADS["tiny"].with_(top_k=16, name="tiny_dense")
    one = synth.expert_store(wl.with_(n_experts=1))
    from paper_2607_09686_amd import HostBuffer
    hb = HostBuffer(wl.store_bytes)
    hb.array[:] = np.tile(one, wl.n_experts)
    R = synth.router(wl)
    X = synth.hidden(wl, n_tokens=4)
    cache = make_cache(wl, hb.ptr, 16)
    wg, wu, wd = quant.expert_weights(one, "q8_0", 1, wl.hidden, wl.inter, 0, 0)
    y = torch.empty(wl.hidden, dtype=torch.float32, device="cuda")
    for t in range(4):
        cache.layer_forward(torch.from_numpy(X[t]).cuda(), torch.from_numpy(R[0]).cuda(), 0, y)
        dense = ffn.expert_ffn(X[t].astype(np.float64), wg, wu, wd)
        check_y(y.cpu().numpy()[None], dense[None], f"dense token {t}")
    cache.close()


def test_device_resident_store():
    wl = synth.WORKLOADS["tiny"]
    run_decode(wl, wl.budget_slots, device_store=True, n_tokens=16)[0].close()


def test_deterministic_outputs():
    torch = torch_cuda()
    wl = synth.WORKLOADS["tiny"]
    keep, ptr, arr = store_buffer(wl)
    R = torch.from_numpy(synth.router(wl)).cuda()
    X = torch.from_numpy(synth.hidden(wl, n_tokens=8)).cuda()
    outs = []
    for rep in range(2):
        cache = make_cache(wl, ptr, 4)
        ys = []
        for t in range(8):
            y = torch.empty(wl.hidden, dtype=torch.float32, device="cuda")
            cache.layer_forward(X[t].contiguous(), R[0], 0, y)
            ys.append(y)
        outs.append(torch.stack(ys).cpu().numpy())
        cache.close()
    np.testing.assert_array_equal(outs[0].view(np.uint32), outs[1].view(np.uint32))


def test_queued_calls_match_waited_calls():
    """Decode calls that only queue work (no routes or counters asked for, so the
    slot tables are stepped on the device with no host wait) give bit-identical
    outputs, trace and counters to calls that wait for every result."""
    torch = torch_cuda()
    wl = synth.WORKLOADS["tiny"].with_(n_layers=3, name="tiny3q")
    keep, ptr, arr = store_buffer(wl)
    R = torch.from_numpy(synth.router(wl)).cuda()
    X = torch.from_numpy(synth.hidden(wl, n_tokens=24)).cuda()
    res = []
    for wait in (True, False):
        cache = make_cache(wl, ptr, 5, trace=True, residual=True, prenorm=True)
        outs = []
        for t in range(X.shape[0]):
            x = X[t].contiguous()
            for l in range(wl.n_layers):
                y = torch.empty_like(x)
                cache.layer_forward(x, R[l], l, y, routes=wait)
                x = y
            outs.append(x)
        out = torch.stack(outs).cpu().numpy()
        res.append((out, sorted(cache.read_trace()), cache.counters().as_tuple()))
        cache.close()
    assert np.all(np.isfinite(res[0][0]))
    np.testing.assert_array_equal(res[0][0].view(np.uint32), res[1][0].view(np.uint32))
    assert res[0][1] == res[1][1] and len(res[0][1]) == 24 * 3 * wl.top_k
    assert res[0][2] == res[1][2]


@pytest.mark.parametrize("copy_mode", ["kernel", "side"])
def test_nonfinite_input_is_reported(copy_mode):
    """All-NaN logits leave no valid expert: the host-table modes fail the call, the
    device-table mode does no work for it and fails at the next synchronising call;
    the handle is poisoned afterwards either way."""
    torch = torch_cuda()
    from paper_2607_09686_amd import MoeError, moecache
    wl = synth.WORKLOADS["tiny"]
    keep, ptr, arr = store_buffer(wl)
    R = torch.from_numpy(synth.router(wl)).cuda()
    cache = make_cache(wl, ptr, 4, trace=True, copy_mode=copy_mode)
    x = torch.full((wl.hidden,), float("nan"), dtype=torch.float32, device="cuda")
    y = torch.zeros(wl.hidden, dtype=torch.float32, device="cuda")
    with pytest.raises(MoeError) as e:
        cache.layer_forward(x, R[0], 0, y)
        cache.counters()
    assert e.value.code == moecache.MOE_EHIP
    x = torch.from_numpy(synth.hidden(wl, n_tokens=1)[0]).cuda()
    with pytest.raises(MoeError) as e:
        cache.layer_forward(x, R[0], 0, y)
    assert e.value.code == moecache.MOE_ESTATE
    cache.close()


@pytest.mark.parametrize("copy_mode", ["kernel", "split"])
def test_timing_totals(copy_mode):
    """Event totals: copies and bytes counted by the copy launch itself; gate/up is a
    launch of its own only in the split mode (inside the copy launch otherwise)."""
    wl = synth.WORKLOADS["tiny"]
    from paper_2607_09686_amd import KIND_COPY, KIND_DOWN, KIND_GATEUP, KIND_ROUTER
    cache, calls, _ = run_decode(wl, wl.budget_slots, n_tokens=8, timing=True, copy_mode=copy_mode)
    c = cache.counters()
    cp = cache.kernel_stats(KIND_COPY)
    assert cp.launches == c.misses and cp.bytes == c.materialized_bytes and cp.total_ms > 0
    assert cache.kernel_stats(KIND_ROUTER).launches == 8
    gu = cache.kernel_stats(KIND_GATEUP)
    if copy_mode == "split":
        assert gu.bytes == 8 * wl.top_k * 2 * wl.payload_bytes // 3 and gu.total_ms > 0
    else:
        assert gu.launches == 0 and gu.bytes == 0
    assert cache.kernel_stats(KIND_DOWN).bytes == 8 * wl.top_k * wl.payload_bytes // 3
    cache.close()


def test_argument_errors():
    torch = torch_cuda()
    from paper_2607_09686_amd import MoeError, moecache
    wl = synth.WORKLOADS["tiny"]
    keep, ptr, arr = store_buffer(wl)
    cache = make_cache(wl, ptr, 4)
    x = torch.zeros(2 * wl.hidden, dtype=torch.float32, device="cuda")
    R = torch.zeros(wl.hidden * wl.n_experts, dtype=torch.float32, device="cuda")
    y = torch.zeros(wl.hidden, dtype=torch.float32, device="cuda")
    with pytest.raises(MoeError) as e:
        cache.layer_forward(x[:wl.hidden], R, 1, y)
    assert e.value.code == moecache.MOE_EINVAL
    with pytest.raises(MoeError):
        cache.layer_forward(x[:wl.hidden], R, 0, x[wl.hidden // 2: wl.hidden // 2 + wl.hidden])
    # an empty call is an argument error and leaves the table alone
    with pytest.raises(MoeError) as e:
        cache.layer_forward(x[:0], R, 0, y[:0], n_tokens=0)
    assert e.value.code == moecache.MOE_EINVAL
    assert moecache.lib().moe_layer_forward(cache.handle, x.data_ptr(), -1, R.data_ptr(), 0,
                                            y.data_ptr(), None) == moecache.MOE_EINVAL
    assert cache.counters().as_tuple() == (0, 0, 0, 0)
    cache.layer_forward(x[:wl.hidden], R, 0, y)     # still usable after argument errors
    cache.close()
    pageable = np.zeros(wl.store_bytes, np.uint8)
    with pytest.raises(MoeError) as e:
        make_cache(wl, pageable.ctypes.data, 4)
    assert e.value.code == moecache.MOE_EINVAL
    with pytest.raises(MoeError):
        make_cache(wl, ptr, 17)


def test_hbm_read_probe():
    """The reference launches: a plain read of 13 MB and of 256 MB takes longer than an empty
    launch, and neither is faster than the HBM peak (the loads are not dropped)."""
    torch_cuda()
    from paper_2607_09686_amd import probe_hbm_read
    for nbytes, iters in ((13369344, 20), (256 << 20, 5)):
        read_us, empty_us = probe_hbm_read(nbytes, iters)
        log(f"plain read of {nbytes} B: {read_us:.2f} us ({nbytes / read_us / 1e3:.0f} GB/s); "
            f"empty launch {empty_us:.2f} us")
        assert 0.0 < empty_us < read_us
        assert nbytes / read_us / 1e3 < 8000.0
