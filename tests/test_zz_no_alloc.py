"""GPU check of moe_layer_forward_static (the one-token entry point that allocates nothing:
its per-call scratch lives in the library's static device array) against
moe_layer_forward on the same inputs, through the C ABI.

Two handles over one store, one driven through each entry point: outputs bit-identical
(the same kernels on the same data), traces and counters equal, and outputs within
2e-3 x RMS of the oracle with the routes exact except at near-ties.  Two runs in a row
share the static array: a larger shape first, then a smaller one (fewer experts per token,
a narrower model), so leftovers of the first would show in the second.  Argument errors:
more than one token, and a handle in a copy mode that keeps its tables on the host.
"""
import numpy as np
import pytest

import synth
from gpu_common import (check_routes, check_y, log, make_cache, oracle_layer_y, replay_trace,
                        store_buffer, torch_cuda)

pytestmark = pytest.mark.gpu


def run_pair(wl, budget, n_tokens):
    torch = torch_cuda()
    log(f"static vs regular: H={wl.hidden} I={wl.inter} E={wl.n_experts} k={wl.top_k} "
        f"L={wl.n_layers} C={budget} {wl.qtype} T={n_tokens}")
    keep, ptr, arr = store_buffer(wl)
    R = synth.router(wl)
    Rd = torch.from_numpy(R).cuda()
    X = synth.hidden(wl, n_tokens=n_tokens)
    reg = make_cache(wl, ptr, budget, trace=True, residual=True, prenorm=True)
    sta = make_cache(wl, ptr, budget, trace=True, residual=True, prenorm=True)
    calls = [[] for _ in range(wl.n_layers)]
    worst = 0.0
    for t in range(n_tokens):
        h_reg = torch.from_numpy(X[t]).cuda()
        h_sta = h_reg.clone()
        for l in range(wl.n_layers):
            xin = h_reg.cpu().numpy()
            y_reg = torch.empty_like(h_reg)
            y_sta = torch.empty_like(h_sta)
            d_reg, idx, w = reg.layer_forward(h_reg, Rd[l], l, y_reg, routes=True)
            d_sta = sta.layer_forward_static(h_sta, Rd[l], l, y_sta, counters=True)
            torch.cuda.synchronize()
            a, b = y_reg.cpu().numpy(), y_sta.cpu().numpy()
            np.testing.assert_array_equal(a.view(np.uint32), b.view(np.uint32))
            assert d_reg.as_tuple() == d_sta.as_tuple()
            idx_or, w_or, z, flipped = check_routes(xin[None], R[l], wl.top_k, idx, w, prenorm=True)
            yo = oracle_layer_y(xin[None], R[l], arr, wl, l, idx_or, w_or, z, idx, flipped,
                                prenorm=True)
            worst = max(worst, check_y((b.astype(np.float64) - xin)[None], yo, f"token {t} layer {l}",
                                       slack=np.spacing(np.abs(b)).astype(np.float64)[None]))
            calls[l].append(idx[0])
            h_reg, h_sta = y_reg, y_sta
    recs, cnt = replay_trace(calls, wl, budget)
    tr_reg, tr_sta = reg.read_trace(), sta.read_trace()
    assert tr_reg == tr_sta
    assert sorted(tr_sta) == sorted(recs)
    assert sta.counters().as_tuple() == reg.counters().as_tuple() == cnt.as_tuple()
    log(f"  ok: bit-identical, worst err/rms {worst:.2e}, counters {sta.counters()}")
    reg.close()
    sta.close()
    keep.free()


@pytest.mark.parametrize("qtype", ["q8_0", "q4_0"])
def test_static_entry_matches_regular(qtype):
    big = synth.WORKLOADS["tiny"].with_(qtype=qtype, n_layers=3, hidden=2048, inter=768,
                                        n_experts=32, top_k=8, name="static_big")
    run_pair(big, 10, 12)
    small = synth.WORKLOADS["tiny"].with_(qtype=qtype, n_layers=2, hidden=256, inter=128,
                                          n_experts=16, top_k=2, name="static_small")
    run_pair(small, 4, 12)


def test_static_entry_rejects_what_it_does_not_take():
    from paper_2607_09686_amd import MoeError
    torch = torch_cuda()
    wl = synth.WORKLOADS["tiny"]
    keep, ptr, arr = store_buffer(wl)
    R = torch.from_numpy(synth.router(wl)[0]).cuda()
    x = torch.from_numpy(synth.hidden(wl, n_tokens=2)).cuda()
    y = torch.empty_like(x)
    c = make_cache(wl, ptr, wl.budget_slots)
    from paper_2607_09686_amd import moecache
    rc = moecache.lib().moe_layer_forward_static(c.handle, x.data_ptr(), 2, R.data_ptr(), 0,
                                                 y.data_ptr(), None)
    assert rc == moecache.MOE_EINVAL
    c.close()
    side = make_cache(wl, ptr, wl.budget_slots, copy_mode="side")
    with pytest.raises(MoeError):
        side.layer_forward_static(x[0].contiguous(), R, 0, y[0].contiguous())
    side.close()
    keep.free()
