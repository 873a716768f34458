"""GPU parity of the score eviction policy (MOE_F_SCORE_EVICT: a miss with every slot taken
evicts the resident outside the call with the lowest router logit for the call's token):

* the logits the device slot-table step used (moe_cache_last_logits) against the oracle
  router's on the same layer input, and the routes (near-ties exempt);
* the slot trace and counters bit-exact against the oracle table with the score policy,
  replayed on the GPU's own routes and logits;
* sampled layer outputs against the oracle FFN;
* the argument errors of the flag.
"""
import numpy as np
import pytest

import synth
from gpu_common import check_routes, check_y, log, make_cache, oracle_layer_y, store_buffer, torch_cuda
from oracle import router as oracle_router
from oracle.layer import rms_normalize
from oracle.lru import LayerLRU

pytestmark = pytest.mark.gpu


def score_chain(wl, budget, store, rho, n_samples, seed):
    torch = torch_cuda()
    keep, ptr, arr = store
    R = synth.router(wl)
    Rd = torch.from_numpy(R).cuda()
    X = synth.hidden(wl, rho=rho)
    L, T = wl.n_layers, wl.n_tokens
    cache = make_cache(wl, ptr, budget, trace=True, residual=True, prenorm=True, score_evict=True)
    log(f"{wl.name}: score eviction, C={budget} rho={rho}: {T} tokens x {L} layers")
    inputs = np.empty((T, L + 1, wl.hidden), np.float32)
    idx = np.empty((T, L, wl.top_k), np.int32)
    wts = np.empty((T, L, wl.top_k), np.float32)
    zs = np.empty((T, L, wl.n_experts), np.float32)
    h = torch.empty(wl.hidden, dtype=torch.float32, device="cuda")
    y = torch.empty_like(h)
    for t in range(T):
        h.copy_(torch.from_numpy(X[t]))
        for l in range(L):
            inputs[t, l] = h.cpu().numpy()
            _, i_, w_ = cache.layer_forward(h, Rd[l], l, y, n_tokens=1, routes=True)
            idx[t, l], wts[t, l] = i_[0], w_[0]
            zs[t, l] = cache.last_logits()
            h, y = y, h
        inputs[t, L] = h.cpu().numpy()
    assert np.all(np.isfinite(inputs))
    flips, worst_z = {}, 0.0
    for t in range(T):
        for l in range(L):
            xin = inputs[t, l][None]
            zo = oracle_router.logits(rms_normalize(xin), R[l])[0]
            dz = np.abs(zs[t, l].astype(np.float64) - zo).max() / max(1.0, np.abs(zo).max())
            assert dz <= 1e-5, (t, l, dz)
            worst_z = max(worst_z, dz)
            io, wo, z, fl = check_routes(xin, R[l], wl.top_k, idx[t, l][None], wts[t, l][None],
                                         prenorm=True)
            if fl:
                flips[(t, l)] = (io, wo, z, fl)
    log(f"  logits within {worst_z:.1e} of the oracle's; near-tie flips {len(flips)}")
    want, cnt = [], None
    for l in range(L):
        lru = LayerLRU(wl.n_experts, budget, wl.payload_bytes, l, policy="score")
        for t in range(T):
            want.extend(lru.step(np.unique(idx[t, l]), zs[t, l]))
        cnt = lru.counters if cnt is None else cnt + lru.counters
    assert sorted(cache.read_trace()) == sorted(want)
    assert cache.counters().as_tuple() == cnt.as_tuple()
    rng = np.random.default_rng(seed)
    picks = {(0, 0), (T - 1, L - 1)}
    while len(picks) < min(n_samples, T * L):
        picks.add((int(rng.integers(T)), int(rng.integers(L))))
    worst = 0.0
    for t, l in sorted(picks):
        xin = inputs[t, l][None]
        ymoe = inputs[t, l + 1].astype(np.float64) - xin[0].astype(np.float64)
        io, wo, z, fl = flips.get((t, l)) or check_routes(xin, R[l], wl.top_k, idx[t, l][None],
                                                            wts[t, l][None], prenorm=True)
        yo = oracle_layer_y(xin, R[l], arr, wl, l, io, wo, z, idx[t, l][None], fl, prenorm=True)
        worst = max(worst, check_y(ymoe[None], yo, f"token {t} layer {l}"))
    c = cache.counters()
    log(f"  ok: worst err/rms {worst:.2e}; hit rate {c.hits / (c.hits + c.misses):.3f}, "
        f"misses {c.misses}")
    cache.close()
    return c


@pytest.mark.parametrize("qtype,budget", [("q8_0", 2), ("q8_0", 5), ("q4_0", 3), ("q4_0", 8)])
def test_score_policy_small(qtype, budget):
    wl = synth.WORKLOADS["tiny"].with_(name="tiny_score", qtype=qtype, n_layers=3, n_tokens=48)
    st = store_buffer(wl)
    try:
        score_chain(wl, budget, st, 0.8, 10 ** 9, 2)
    finally:
        st[0].free()


def test_score_policy_a3b_full_size():
    wl = synth.WORKLOADS["a3b_decode"]
    st = store_buffer(wl)
    try:
        score_chain(wl, wl.budget_slots, st, wl.rho, 16, 3)
    finally:
        st[0].free()


def test_score_policy_argument_errors():
    torch = torch_cuda()
    from paper_2607_09686_amd import MoeError, moecache
    wl = synth.WORKLOADS["tiny"]
    keep, ptr, arr = store_buffer(wl)
    for mode in ("side", "sdma"):
        with pytest.raises(MoeError) as e:
            make_cache(wl, ptr, 4, score_evict=True, copy_mode=mode)
        assert e.value.code == moecache.MOE_EINVAL
    cache = make_cache(wl, ptr, 4, score_evict=True)
    x = torch.zeros(2 * wl.hidden, dtype=torch.float32, device="cuda")
    R = torch.zeros(wl.hidden * wl.n_experts, dtype=torch.float32, device="cuda")
    y = torch.zeros_like(x)
    with pytest.raises(MoeError) as e:
        cache.layer_forward(x, R, 0, y, n_tokens=2)
    assert e.value.code == moecache.MOE_EINVAL
    cache.layer_forward(x[:wl.hidden], R, 0, y[:wl.hidden])   # one token still works
    assert np.array_equal(cache.last_logits(), np.zeros(wl.n_experts, np.float32))
    cache.close()
    side = make_cache(wl, ptr, 4, copy_mode="side")
    with pytest.raises(MoeError):
        side.last_logits()
    side.close()
    keep.free()
