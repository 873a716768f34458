"""A GGUF MoE model through the whole path: split-packed by the library (moe_pack_gguf),
the pack loaded into pinned memory as the expert store, the packed routers as router_w,
then decoded on the GPU through a residual + pre-norm stack; routes, the slot trace,
counters and outputs against the oracle on the same pack (the oracle's own reading of the
GGUF file gives the same bytes, checked on the CPU)."""
import numpy as np
import pytest

import gguf_writer
import synth
from gpu_common import check_routes, check_y, decode_chain, log, make_cache, oracle_layer_y, \
    replay_trace, torch_cuda

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("qcode,router_type", [(8, 0), (2, 1)])
def test_packed_gguf_decodes(tmp_path, qcode, router_type):
    torch = torch_cuda()
    from paper_2607_09686_amd import HostBuffer, pack_gguf
    src = tmp_path / "m.gguf"
    gguf_writer.moe_model(src, n_layers=3, n_experts=16, hidden=256, inter=128, qcode=qcode,
                          top_k=2, seed=11 + qcode, router_type=router_type)
    info = pack_gguf(src, tmp_path / "e.pack", tmp_path / "e.index", tmp_path / "r.bin")
    wl = synth.WORKLOADS["tiny"].with_(name="gguf", n_layers=info["n_layers"],
                                       n_experts=info["n_experts"], top_k=info["top_k"],
                                       hidden=info["hidden"], inter=info["inter"],
                                       qtype="q8_0" if info["qtype"] == 8 else "q4_0", n_tokens=16)
    assert wl.payload_bytes == info["payload_bytes"] and wl.store_bytes == info["pack_bytes"]
    hb = HostBuffer(wl.store_bytes)
    hb.array[:] = np.fromfile(tmp_path / "e.pack", np.uint8)
    R = np.fromfile(tmp_path / "r.bin", np.float32).reshape(wl.n_layers, wl.hidden, wl.n_experts)
    X = synth.hidden(wl)
    cache = make_cache(wl, hb.ptr, 5, trace=True, residual=True, prenorm=True)
    hfin, inputs, idx, w = decode_chain(cache, wl, X, torch.from_numpy(R).cuda())
    flips = {}
    for t in range(wl.n_tokens):
        for l in range(wl.n_layers):
            io, wo, z, fl = check_routes(inputs[t, l][None], R[l], wl.top_k, idx[t, l][None],
                                         w[t, l][None], prenorm=True)
            flips[(t, l)] = (io, wo, z, fl)
    recs, cnt = replay_trace([[idx[t, l] for t in range(wl.n_tokens)] for l in range(wl.n_layers)],
                             wl, 5)
    assert sorted(cache.read_trace()) == sorted(recs)
    assert cache.counters().as_tuple() == cnt.as_tuple()
    worst = 0.0
    for t in range(wl.n_tokens):
        for l in range(wl.n_layers):
            xin = inputs[t, l][None]
            xout = inputs[t, l + 1] if l + 1 < wl.n_layers else hfin[t]
            io, wo, z, fl = flips[(t, l)]
            yo = oracle_layer_y(xin, R[l], hb.array, wl, l, io, wo, z, idx[t, l][None], fl,
                                prenorm=True)
            worst = max(worst, check_y((xout.astype(np.float64) - xin[0])[None], yo, f"{t},{l}"))
    log(f"packed GGUF q{qcode}: worst err/rms {worst:.2e}, counters {cache.counters()}")
    cache.close()
    hb.free()
