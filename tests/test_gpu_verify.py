"""GPU parity of speculative verification windows (1 + horizon tokens per layer call, the
multi-token path) through a residual + pre-norm layer stack:

* every route of every window token on every layer against the oracle router on the same
  layer input (near-ties exempt);
* the slot trace and counters bit-exact against the oracle LRU stepped once per window
  and layer with the union of the window's routed experts;
* layer outputs (all calls at the small shape, sampled calls at full size) against the
  oracle of the path each call takes: exact for the GEMVs (windows whose experts fit the
  slots, and the host-table path's chunks where the union GEMVs take the shape), bf16
  weights otherwise (MFMA GEMMs).

Windows follow the verification schedule of the seeded draft outcomes."""
import numpy as np
import pytest

import synth
from gpu_common import (TIE_GAP, check_routes, check_y, log, make_cache, oracle_layer_y,
                        replay_trace, small_call_exact, store_buffer, torch_cuda)
from oracle.verify import schedule, window_union

pytestmark = pytest.mark.gpu


def verify_chain(wl, budget, store, n_check, seed):
    torch = torch_cuda()
    keep, ptr, arr = store
    W = wl.horizon + 1
    R = synth.router(wl)
    Rd = torch.from_numpy(R).cuda()
    X = synth.hidden(wl, n_tokens=wl.n_tokens + wl.horizon)
    steps = schedule(wl.n_tokens, wl.horizon,
                     synth.acceptance(wl.n_tokens, wl.horizon, wl.accept_q, wl.hidden_seed))
    log(f"{wl.name}: C={budget} W={W}: {len(steps)} windows x {wl.n_layers} layers")
    cache = make_cache(wl, ptr, budget, trace=True, residual=True, prenorm=True)
    L = wl.n_layers
    inputs = np.empty((len(steps), L + 1, W, wl.hidden), np.float32)
    idx = np.empty((len(steps), L, W, wl.top_k), np.int32)
    wts = np.empty((len(steps), L, W, wl.top_k), np.float32)
    h = torch.empty((W, wl.hidden), dtype=torch.float32, device="cuda")
    y = torch.empty_like(h)
    for s, (t, _, _) in enumerate(steps):
        h.copy_(torch.from_numpy(np.ascontiguousarray(X[t:t + W])))
        for l in range(L):
            inputs[s, l] = h.cpu().numpy()
            _, i_, w_ = cache.layer_forward(h, Rd[l], l, y, n_tokens=W, routes=True)
            idx[s, l], wts[s, l] = i_, w_
            h, y = y, h
        inputs[s, L] = h.cpu().numpy()
    assert np.all(np.isfinite(inputs))
    flips = {}
    for s in range(len(steps)):
        for l in range(L):
            io, wo, z, fl = check_routes(inputs[s, l], R[l], wl.top_k, idx[s, l], wts[s, l],
                                         prenorm=True)
            if fl:
                flips[(s, l)] = (io, wo, z, fl)
    log(f"  near-tie flips: {len(flips)}; checking trace")
    calls = [[window_union(idx[s, l]) for s in range(len(steps))] for l in range(L)]
    recs, cnt = replay_trace(calls, wl, budget)
    assert sorted(cache.read_trace()) == sorted(recs)   # records carry (layer, step)
    assert cache.counters().as_tuple() == cnt.as_tuple()
    rng = np.random.default_rng(seed)
    picks = {(0, 0), (len(steps) - 1, L - 1)}
    all_calls = [(s, l) for s in range(len(steps)) for l in range(L)]
    if n_check >= len(all_calls):
        picks = set(all_calls)
    while len(picks) < min(n_check, len(all_calls)):
        picks.add((int(rng.integers(len(steps))), int(rng.integers(L))))
    worst, n_gemv = 0.0, 0
    for s, l in sorted(picks):
        xin = inputs[s, l]
        ymoe = inputs[s, l + 1].astype(np.float64) - xin.astype(np.float64)
        io, wo, z, fl = flips.get((s, l), (None, None, None, []))
        if io is None:
            io, wo, z, fl = check_routes(xin, R[l], wl.top_k, idx[s, l], wts[s, l], prenorm=True)
        # windows of at most 8 tokens run GEMVs (exact oracle): the union GEMVs, or with more
        # experts than slots the union GEMVs per chunk of the host-table path when the shape
        # fits them; others the bf16 MFMA GEMMs (bf16-weight oracle)
        gemv = small_call_exact(W, wl.hidden, wl.inter, len(window_union(idx[s, l])), budget)
        n_gemv += gemv
        yo = oracle_layer_y(xin, R[l], arr, wl, l, io, wo, z, idx[s, l], fl, bf16=not gemv,
                            prenorm=True)
        worst = max(worst, check_y(ymoe, yo, f"window {s} layer {l}"))
    c = cache.counters()
    log(f"  ok: {len(picks)} calls checked ({n_gemv} on the GEMVs), worst err/rms {worst:.2e}; hit rate "
        f"{c.hits / max(1, c.hits + c.misses):.3f}, mean union {(c.hits + c.misses) / len(all_calls):.2f}")
    cache.close()
    return c, steps


@pytest.mark.parametrize("qtype,budget,q", [("q8_0", 4, 0.6), ("q4_0", 6, 0.9), ("q8_0", 16, 0.0)])
def test_verify_small(qtype, budget, q):
    wl = synth.WORKLOADS["tiny"].with_(name="tiny_verify", qtype=qtype, n_layers=3, n_tokens=24,
                                       horizon=4, accept_q=q, mode="verify")
    st = store_buffer(wl)
    try:
        verify_chain(wl, budget, st, 10 ** 9, 1)
    finally:
        st[0].free()


def test_a3b_verify_full_size():
    """The A3B windows at their budget and at 19 slots (15 %), where most windows' unions
    exceed the slots and the device steps them in chunks."""
    wl = synth.WORKLOADS["a3b_verify"]
    st = store_buffer(wl)
    try:
        for budget, seed in ((wl.budget_slots, 5), (19, 6)):
            c, steps = verify_chain(wl, budget, st, 16, seed)
            assert sum(g for _, _, g in steps) == wl.n_tokens
            assert c.materialized_bytes == c.misses * wl.payload_bytes
    finally:
        st[0].free()


@pytest.mark.parametrize("qtype,H,I", [("q8_0", 512, 256), ("q4_0", 256, 384)])
def test_window_equals_decode_bitwise(qtype, H, I):
    """A window call of 5 tokens computes each token exactly as a decode call does: at hidden
    <= 512 the window router uses the decode router's 32-row partial blocks, so routes and
    weights match bit for bit, and the union GEMVs and the rank-order combine reproduce the
    decode GEMVs' outputs bit for bit (the slot tables differ: one step for the union against
    one per token, which changes where experts live, not what is computed)."""
    torch = torch_cuda()
    wl = synth.WORKLOADS["tiny"].with_(qtype=qtype, hidden=H, inter=I, n_experts=32, top_k=4,
                                       n_layers=2, name=f"win_eq_{qtype}")
    keep, ptr, arr = store_buffer(wl)
    R = synth.router(wl)
    Rd = torch.from_numpy(R).cuda()
    X = np.ascontiguousarray(synth.hidden(wl, n_tokens=5))
    win = make_cache(wl, ptr, 24, residual=True, prenorm=True)
    dec = make_cache(wl, ptr, 24, residual=True, prenorm=True)
    for l in range(wl.n_layers):
        x = torch.from_numpy(X).cuda()
        y = torch.empty_like(x)
        _, iw, ww = win.layer_forward(x, Rd[l], l, y, n_tokens=5, routes=True)
        yw = y.cpu().numpy()
        for t in range(5):
            xt = torch.from_numpy(np.ascontiguousarray(X[t:t + 1])).cuda()
            yt = torch.empty_like(xt)
            _, it, wt = dec.layer_forward(xt, Rd[l], l, yt, n_tokens=1, routes=True)
            assert np.array_equal(it.reshape(-1), iw[t]), (l, t)
            assert np.array_equal(wt.reshape(-1).view(np.uint32), ww[t].view(np.uint32)), (l, t)
            assert np.array_equal(yt.cpu().numpy()[0].view(np.uint32), yw[t].view(np.uint32)), (l, t)
        X = yw
    win.close()
    dec.close()


@pytest.mark.parametrize("qtype,H,I,T,E,k,C", [
    ("q8_0", 512, 256, 5, 32, 4, 20), ("q8_0", 1024, 384, 8, 32, 4, 32),
    ("q4_0", 256, 384, 2, 32, 4, 8), ("q4_0", 768, 256, 7, 32, 4, 28),
    # 8 tokens x 16 experts: the union lists at their 128-entry capacity
    ("q8_0", 512, 192, 8, 256, 16, 128),
    # fewer slots than some windows' unions: those calls take the host-table path in both modes
    ("q4_0", 512, 256, 6, 64, 8, 30)])
def test_window_fused_copy_equals_split_bitwise(qtype, H, I, T, E, k, C):
    """The default copy mode runs a window's gate/up inside the copy launch (copied experts
    from the rows in flight, resident ones alongside); the split mode copies first and then
    runs the union gate/up kernel.  Over a run of warm-cache windows both give the same routes,
    outputs and slot trace bit for bit."""
    torch = torch_cuda()
    wl = synth.WORKLOADS["tiny"].with_(qtype=qtype, hidden=H, inter=I, n_experts=E, top_k=k,
                                       n_layers=2, name=f"win_fuse_{qtype}_{E}")
    log(f"fused vs split window: {qtype} H={H} I={I} T={T} E={E} k={k} C={C}")
    keep, ptr, arr = store_buffer(wl)
    R = synth.router(wl)
    Rd = torch.from_numpy(R).cuda()
    X = np.ascontiguousarray(synth.hidden(wl, n_tokens=4 * T))
    caches = [make_cache(wl, ptr, C, residual=True, prenorm=True, trace=True, copy_mode=m)
              for m in ("kernel", "split")]
    for call in range(4):
        xs = np.ascontiguousarray(X[call * T:(call + 1) * T])
        for l in range(wl.n_layers):
            outs = []
            for c in caches:
                x = torch.from_numpy(xs).cuda()
                y = torch.empty_like(x)
                d, idx, w = c.layer_forward(x, Rd[l], l, y, n_tokens=T, routes=True)
                outs.append((d.as_tuple(), idx, w.view(np.uint32), y.cpu().numpy().view(np.uint32)))
            (d0, i0, w0, y0), (d1, i1, w1, y1) = outs
            assert d0 == d1 and np.array_equal(i0, i1) and np.array_equal(w0, w1), (call, l)
            assert np.array_equal(y0, y1), (call, l)
    assert caches[0].read_trace() == caches[1].read_trace()
    for c in caches:
        c.close()
