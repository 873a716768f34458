"""GPU parity of the multi-token path (many tokens per layer call): bf16 MFMA grouped
GEMMs compared with the bf16-weight oracle, and calls of at most 8 tokens (GEMVs) with the
exact oracle; routes, waves of slot reuse inside a call (more routed experts than slots),
trace and counters exact."""
import numpy as np
import pytest

import synth
from gpu_common import (TIE_GAP, check_routes, check_y, log, make_cache, residual_slack,
                        small_call_exact, softmax_of, store_buffer, torch_cuda)
from oracle import router as oracle_router
from oracle.layer import Shape, moe_layer, moe_layer_bf16, rms_normalize
from oracle.lru import LayerLRU

pytestmark = pytest.mark.gpu


def oracle_routes(x, wr, k, prenorm):
    z = oracle_router.logits(rms_normalize(x) if prenorm else x, wr)
    idx, w, gap = oracle_router.topk(z, k)
    return z, idx, w, gap


def gemv_call(T, idx, budget, H, I, qtype="q8_0"):
    """Whether a multi-token call takes the GEMVs (fp32-accurate) instead of the bf16 MFMA
    GEMMs."""
    return small_call_exact(T, H, I, len(np.unique(idx)), budget, qtype)


def check_call(x, wr, arr, wl, layer, idx_g, w_g, y_g, prenorm, residual, tokens=None, budget=None):
    """Routes of every token, y of `tokens` (default all) against the oracle of the path the
    call takes (bf16 weights for the MFMA GEMMs, exact for the decode GEMVs)."""
    z, idx, w, gap = oracle_routes(x, wr, wl.top_k, prenorm)
    flips = 0
    idx_use, w_use = idx.copy(), w.copy()
    for t in range(x.shape[0]):
        if set(idx[t].tolist()) != set(idx_g[t].tolist()):
            assert gap[t] < TIE_GAP, f"token {t}: top-k differs with gap {gap[t]}"
            idx_use[t] = idx_g[t]
            w_use[t] = softmax_of(z[t], idx_g[t])
            flips += 1
    toks = list(range(x.shape[0])) if tokens is None else list(tokens)
    exact = budget is not None and gemv_call(x.shape[0], idx_g, budget, wl.hidden, wl.inter, wl.qtype)
    fn = moe_layer if exact else moe_layer_bf16
    yo = fn(x, wr, arr, Shape.of(wl), layer, routes=(idx_use, w_use), tokens=toks,
            prenorm=prenorm)["y"][toks]
    yg = y_g[toks].astype(np.float64)
    slack = None
    if residual:
        yg = yg - x[toks].astype(np.float64)
        slack = residual_slack(y_g[toks])
    err = check_y(yg, yo, f"layer {layer}", slack=slack)
    return flips, err


def run_prefill(wl, budget, T, calls=1, prenorm=False, residual=False, store=None, seed_shift=0,
                copy_mode="kernel", xs=None, poison=False):
    torch = torch_cuda()
    log(f"prefill {wl.qtype} E={wl.n_experts} k={wl.top_k} H={wl.hidden} I={wl.inter} "
        f"L={wl.n_layers} C={budget} T={T} calls={calls} prenorm={prenorm} residual={residual} "
        f"copy_mode={copy_mode}")
    keep, ptr, arr = store if store is not None else store_buffer(wl)
    R = synth.router(wl)
    cache = make_cache(wl, ptr, budget, trace=True, residual=residual, prenorm=prenorm,
                       copy_mode=copy_mode)
    if poison:
        cache.fill_slots(0xFF)   # every slot scale reads NaN until its expert is copied in
    lrus = [LayerLRU(wl.n_experts, budget, wl.payload_bytes, l) for l in range(wl.n_layers)]
    want = []
    worst = 0.0
    for c in range(calls):
        X = synth.hidden(wl.with_(hidden_seed=wl.hidden_seed + 7 * c + seed_shift), rho=-1.0,
                         n_tokens=T) if xs is None else xs[c]
        for l in range(wl.n_layers):
            x = torch.from_numpy(X).cuda()
            y = torch.empty_like(x)
            delta, idx, w = cache.layer_forward(x, torch.from_numpy(R[l]).cuda(), l, y,
                                                n_tokens=T, routes=True)
            torch.cuda.synchronize()
            flips, err = check_call(X, R[l], arr, wl, l, idx, w, y.cpu().numpy(), prenorm, residual,
                                    budget=budget)
            worst = max(worst, err)
            want.extend(lrus[l].step(np.unique(idx)))
            assert delta.materialized_bytes == delta.misses * wl.payload_bytes
    got = cache.read_trace()
    assert got == want
    tot = sum((lr.counters for lr in lrus[1:]), lrus[0].counters)
    assert cache.counters().as_tuple() == tot.as_tuple()
    log(f"  ok: worst err/rms {worst:.2e}; counters {cache.counters()}")
    cache.close()
    return worst


def test_prefill_and_decode_share_slot_tables():
    """Prefill calls (slot table stepped on the host) and decode calls (stepped on
    the device) interleaved on one handle: the trace, in call order, and the
    counters equal one oracle table per layer stepped through all calls."""
    torch = torch_cuda()
    wl = synth.WORKLOADS["tiny"].with_(n_layers=2, name="tiny_mix")
    budget = 6
    keep, ptr, arr = store_buffer(wl)
    R = synth.router(wl)
    Rd = [torch.from_numpy(R[l]).cuda() for l in range(wl.n_layers)]
    cache = make_cache(wl, ptr, budget, trace=True)
    lrus = [LayerLRU(wl.n_experts, budget, wl.payload_bytes, l) for l in range(wl.n_layers)]
    want = []
    for phase, T in enumerate((37, 1, 20, 1, 2)):
        n_calls = 9 if T == 1 else 1
        X = synth.hidden(wl.with_(hidden_seed=wl.hidden_seed + 11 * phase), rho=-1.0,
                         n_tokens=max(T, n_calls))
        for c in range(n_calls):
            xs = np.ascontiguousarray(X[c:c + 1] if T == 1 else X)
            for l in range(wl.n_layers):
                x = torch.from_numpy(xs).cuda()
                y = torch.empty_like(x)
                delta, idx, w = cache.layer_forward(x, Rd[l], l, y, n_tokens=xs.shape[0],
                                                    routes=True)
                if T == 1:
                    check_routes(xs, R[l], wl.top_k, idx, w)
                else:
                    z, io, wo, gap = oracle_routes(xs, R[l], wl.top_k, False)
                    for t in range(xs.shape[0]):
                        if set(io[t].tolist()) != set(idx[t].tolist()):
                            assert gap[t] < TIE_GAP
                step = lrus[l].step(np.unique(idx))
                want.extend(step)
                assert delta.hits == sum(r[3] for r in step)
    assert cache.read_trace() == want
    tot = sum((lr.counters for lr in lrus[1:]), lrus[0].counters)
    assert cache.counters().as_tuple() == tot.as_tuple()
    cache.close()


@pytest.mark.parametrize("qtype", ["q8_0", "q4_0"])
@pytest.mark.parametrize("T,budget", [(2, 4), (37, 4), (300, 16), (300, 3), (129, 6)])
def test_prefill_small(qtype, T, budget):
    wl = synth.WORKLOADS["tiny"].with_(qtype=qtype, name="tiny_pf")
    run_prefill(wl, max(budget, wl.top_k), T)


@pytest.mark.parametrize("qtype", ["q8_0", "q4_0"])
@pytest.mark.parametrize("T,budget", [(3, 6), (5, 10), (8, 16), (8, 5), (9, 16)])
def test_small_calls_both_paths(qtype, T, budget):
    """Calls of up to 8 tokens whose experts fit the slots (union GEMVs), 8 tokens with 5
    slots (host-table path, slots reused inside the call, the union GEMVs per chunk) and 9
    tokens (MFMA GEMMs)."""
    # (H, I as in the warm-cache test below: large enough that a bf16 rounding flip on the
    # MFMA side stays far below the tolerance)
    wl = synth.WORKLOADS["tiny"].with_(qtype=qtype, n_layers=2, hidden=1024, inter=384,
                                       name="tiny_small")
    run_prefill(wl, budget, T, calls=3, prenorm=True, residual=True, seed_shift=T)


@pytest.mark.parametrize("copy_mode", ["side", "sdma"])
@pytest.mark.parametrize("T,budget", [(5, 10), (8, 5)])
def test_small_calls_host_table(copy_mode, T, budget):
    """The copy modes that keep the slot tables on the host: calls of up to 8 tokens whose
    experts fit the slots run the decode GEMVs once per token after the host's table step
    (5 tokens), those with more experts than slots the union GEMVs per chunk (8 tokens with
    5 slots)."""
    wl = synth.WORKLOADS["tiny"].with_(n_layers=2, hidden=1024, inter=384, name="tiny_small_host")
    run_prefill(wl, budget, T, calls=2, prenorm=True, residual=True, seed_shift=T,
                copy_mode=copy_mode)


@pytest.mark.parametrize("T", [3, 5])
def test_small_calls_wide_hidden(T):
    """Hidden 4096: 3 tokens run the union GEMVs (each routed expert's weights read once for
    all its tokens), 5 tokens the decode GEMVs once per token (five tokens' digit images
    exceed the union kernel's LDS budget)."""
    wl = synth.WORKLOADS["tiny"].with_(n_layers=2, hidden=4096, inter=256, name="tiny_wide")
    run_prefill(wl, 10, T, calls=3, prenorm=True, residual=True, seed_shift=T)


def test_prefill_warm_cache_prenorm_residual_multilayer():
    # (H, I large enough that one bf16 rounding flip of an input, ~4e-3 of its value,
    # stays far below the tolerance; at H 256 a single flip moves y by ~2e-3 x RMS)
    wl = synth.WORKLOADS["tiny"].with_(n_layers=3, hidden=1024, inter=384, name="pf3")
    run_prefill(wl, 5, 200, calls=3, prenorm=True, residual=True)


# 1088 = 17 x 64: the down GEMM's last 128-column tile holds 64 columns
@pytest.mark.parametrize("shape", [(1024, 384, 40, 6, 9, 260), (768, 1408, 64, 8, 20, 96),
                                   (1088, 320, 24, 4, 7, 180)])
def test_prefill_other_shapes(shape):
    H, I, E, k, C, T = shape
    for qt in ("q8_0", "q4_0"):
        wl = synth.WORKLOADS["tiny"].with_(hidden=H, inter=I, n_experts=E, top_k=k, qtype=qt,
                                           name=f"pf{H}x{I}x{E}")
        run_prefill(wl, C, T)


def test_prefill_tiles_past_the_table():
    """A warm call whose 65 536 (token, expert) pairs make more 128-row tiles than the
    grouped GEMMs' per-launch tile table holds (512): the kernels find their tile by the
    scan over the experts instead.  The first call copies every expert in; the second
    runs all 16 as hits in one launch.  Routes, trace, counters and every token's
    output against the bf16-weight oracle."""
    for qt in ("q8_0", "q4_0"):
        wl = synth.WORKLOADS["tiny"].with_(n_experts=16, top_k=8, qtype=qt, name=f"pftiles_{qt}")
        run_prefill(wl, 16, 8192, calls=2)


@pytest.mark.parametrize("name,budget,calls", [("a3b_prefill", None, 1), ("q4km_prefill", None, 1),
                                                ("a3b_prefill", 128, 2)])
def test_a3b_prefill_full_size(name, budget, calls):
    """4096 tokens through all 48 layers of the A3B stack (Q8_0, and the Q4_K_M mix:
    Q4_K gate/up, Q6_K down), pre-norm residual chain on the GPU: 45 slots from a cold
    cache, or every expert resident (128 slots, the second call all hits: each layer's
    128 experts in one launch of each grouped GEMM).  Every route and the whole trace
    checked, outputs of sampled tokens in sampled layers of the last call against the
    bf16 oracle."""
    torch = torch_cuda()
    wl = synth.WORKLOADS[name]
    C = wl.budget_slots if budget is None else budget
    keep, ptr, arr = store_buffer(wl)
    R = synth.router(wl)
    X = synth.hidden(wl)
    cache = make_cache(wl, ptr, C, trace=True, residual=True, prenorm=True)
    T, L = X.shape[0], wl.n_layers
    check_layers = {0, L // 2, L - 1}
    log(f"{name}: {T} tokens x {L} layers, C={C}, {calls} call(s)")
    lrus = [LayerLRU(wl.n_experts, C, wl.payload_bytes, l) for l in range(L)]
    want = []
    flips = 0
    for c in range(calls):
        inputs, outputs, routes = {}, {}, []
        h = torch.from_numpy(X).cuda()
        y = torch.empty_like(h)
        for l in range(L):
            xin = h.cpu().numpy()
            delta, idx, w = cache.layer_forward(h, torch.from_numpy(R[l]).cuda(), l, y, n_tokens=T,
                                                routes=True)
            routes.append((xin, idx, w))
            if l in check_layers:
                inputs[l] = xin
                outputs[l] = y.cpu().numpy()
            step = lrus[l].step(np.unique(idx))
            want.extend(step)
            assert delta.misses == sum(1 for r in step if not r[3])
            h, y = y, h
        assert np.all(np.isfinite(h.cpu().numpy()))
        for l, (xin, idx, w) in enumerate(routes):
            z, io, wo, gap = oracle_routes(xin, R[l], wl.top_k, True)
            for t in np.nonzero(np.any(np.sort(io, 1) != np.sort(idx, 1), axis=1))[0]:
                assert gap[t] < TIE_GAP, f"call {c} layer {l} token {t}: gap {gap[t]}"
                flips += 1
    log(f"  near-tie flips: {flips}; trace")
    assert cache.read_trace() == want
    rng = np.random.default_rng(5)
    worst = 0.0
    for l in sorted(check_layers):
        toks = sorted(rng.choice(T, size=6, replace=False).tolist())
        xin, idx, w = routes[l]
        _, err = check_call(xin, R[l], arr, wl, l, idx, w, outputs[l], True, True, tokens=toks,
                            budget=C)
        worst = max(worst, err)
    log(f"  ok: worst err/rms {worst:.2e}; counters {cache.counters()}")
    cache.close()
    keep.free()
