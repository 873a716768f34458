"""GPU parity of a multi-token call past the wide grouped GEMMs' 32-bit element offsets.

The wide-tile kernels address both activation planes ([2][T][H] and [2][T*k][I] bf16)
with 32-bit element offsets; a call whose planes hold more than 2^32 elements
(T*H > 2^31) runs the 256-thread grouped GEMMs instead (Q8_0 / Q4_0: `pf_gateup_kernel`,
`pf_down_kernel`; K-quant: `gm_gateup_kernel`, `gm_down_kernel`), which index 16-byte
units with 32 bits.  The call here is 4096 distinct seeded tokens repeated 2049 times
(T = 8 392 704, H = 256: 2.15e9 elements per plane, 4.3 GB of x), so that

* every copy of a token must come out bit-identical to its first copy (each row's
  arithmetic does not depend on where the row sits in a tile or a launch), and
* the first copies are compared with the bf16-weight oracle (routes, y), the trace and
  counters with the oracle LRU.

About 62 GB of device memory per case (x, y, the library's activation planes and its
per-pair down rows)."""
import numpy as np
import pytest

import synth
from gpu_common import log, make_cache, store_buffer, torch_cuda
from oracle.lru import LayerLRU
from test_gpu_prefill import check_call

pytestmark = pytest.mark.gpu

DISTINCT = 4096
REPS = 2049          # T = 8 392 704 tokens
HIDDEN = INTER = 256


@pytest.mark.parametrize("qtype", ["q8_0", "q4_0", "q4_k_m"])
def test_prefill_past_32bit_activation_offsets(qtype):
    torch = torch_cuda()
    wl = synth.WORKLOADS["tiny"].with_(qtype=qtype, n_layers=1, hidden=HIDDEN, inter=INTER,
                                       n_experts=16, top_k=2, name=f"maxsize_{qtype}")
    T, H, k = DISTINCT * REPS, wl.hidden, wl.top_k
    assert T * H > 2**31 and 2 * T * H // 8 <= 2**32 - 1
    assert T * max(H, k * wl.inter) <= 2**34          # the library's limit for one call
    budget = 8
    log(f"maxsize {qtype}: T={T} H={H} I={wl.inter} E={wl.n_experts} k={k} C={budget}")
    keep, ptr, arr = store_buffer(wl)
    R = synth.router(wl)
    X = synth.hidden(wl.with_(hidden_seed=wl.hidden_seed + 5), rho=-1.0, n_tokens=DISTINCT)
    cache = make_cache(wl, ptr, budget, trace=True, residual=True, prenorm=True)
    x = torch.from_numpy(X).cuda().repeat(REPS, 1)
    y = torch.empty_like(x)
    delta, idx, w = cache.layer_forward(x, torch.from_numpy(R[0]).cuda(), 0, y, n_tokens=T,
                                        routes=True)
    torch.cuda.synchronize()
    log("  call done")
    # every copy's routes and outputs equal the first copy's, bit for bit
    assert (idx.reshape(REPS, DISTINCT, k) == idx[None, :DISTINCT]).all()
    assert (w.reshape(REPS, DISTINCT, k).view(np.uint32) == w[None, :DISTINCT].view(np.uint32)).all()
    yv = y.view(REPS, DISTINCT, H)
    y0 = yv[0]
    for r0 in range(1, REPS, 256):
        bad = int((yv[r0:r0 + 256] != y0).sum())
        assert bad == 0, f"copies {r0}..{min(REPS, r0 + 256) - 1}: {bad} outputs differ from the first copy"
    log("  copies identical")
    # the first copies against the oracle
    y_first = y0.cpu().numpy()
    del x, y, yv, y0
    flips, err = check_call(X, R[0], arr, wl, 0, idx[:DISTINCT], w[:DISTINCT], y_first,
                            prenorm=True, residual=True)
    lru = LayerLRU(wl.n_experts, budget, wl.payload_bytes, 0)
    want = lru.step(np.unique(idx))
    assert cache.read_trace() == want
    assert cache.counters().as_tuple() == lru.counters.as_tuple()
    assert delta.materialized_bytes == delta.misses * wl.payload_bytes
    log(f"  ok: err/rms {err:.2e}, {flips} near-tie flips, counters {cache.counters()}")
    cache.close()
    torch.cuda.empty_cache()
