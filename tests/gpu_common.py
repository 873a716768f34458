"""Shared helpers of the GPU parity tests: inputs from the seeded generator, the GPU
path through the C ABI, the oracle on the same inputs, and the comparison rules.

Comparison rules (the oracle is fp64; the GPU computes in fp32):
* top-k sets bit-exact, except where the oracle's gap between the k-th and
  (k+1)-th logit is below 1e-5 (then either set is accepted, and the oracle
  recomputes y with the set the GPU chose);
* the slot trace and counters bit-exact against the oracle LRU replayed on the
  GPU's own routes (and against the oracle's own routes when no near-tie flipped);
* max |y_gpu - y_oracle| <= 2e-3 * RMS(y_oracle) per layer call, y being the
  MoE output (without the residual).
"""
import sys
import time

import numpy as np

import synth
from oracle import router as oracle_router
from oracle.layer import Shape, moe_layer, moe_layer_bf16
from oracle.lru import LayerLRU

TIE_GAP = 1e-5
Y_TOL = 2e-3


def log(msg):
    print(f"[{time.strftime('%H:%M:%S')}] {msg}", file=sys.stderr, flush=True)


def torch_cuda():
    import torch
    assert torch.cuda.is_available(), "GPU test needs a visible GPU"
    return torch


def store_buffer(wl, device=False):
    """Expert store of a workload in pinned host memory (HostBuffer), or a device tensor."""
    from paper_2607_09686_amd import HostBuffer
    hb = HostBuffer(wl.store_bytes)
    t0 = time.time()
    synth.expert_store(wl, out=hb.array)
    log(f"generated {wl.name} store: {wl.store_bytes / 2**30:.2f} GiB in {time.time() - t0:.1f} s")
    if not device:
        return hb, hb.ptr, hb.array
    torch = torch_cuda()
    dev = torch.empty(wl.store_bytes, dtype=torch.uint8, device="cuda")
    dev.copy_(torch.from_numpy(hb.array))
    return (hb, dev), dev.data_ptr(), hb.array


def make_cache(wl, store_ptr, budget, **kw):
    from paper_2607_09686_amd import MoeCache
    return MoeCache(wl.n_layers, wl.n_experts, wl.top_k, wl.hidden, wl.inter, wl.qtype, store_ptr,
                    wl.store_bytes, budget, **kw)


def softmax_of(z, ids):
    zs = z[ids]
    e = np.exp(zs - zs.max())
    return e / e.sum()


def check_routes(x, wr, k, idx_gpu, w_gpu, prenorm=False):
    """Compare one call's routes. Returns (oracle_idx, oracle_w, z, flipped_tokens)."""
    from oracle.layer import rms_normalize
    z = oracle_router.logits(rms_normalize(x) if prenorm else x, wr)
    idx, w, gap = oracle_router.topk(z, k)
    flipped = []
    for t in range(idx.shape[0]):
        same = set(idx[t].tolist()) == set(idx_gpu[t].tolist())
        if not same:
            assert gap[t] < TIE_GAP, f"top-k differs at token {t} with gap {gap[t]}"
            flipped.append(t)
            continue
        # weights of the same set, matched by expert id
        ow = dict(zip(idx[t].tolist(), w[t].tolist()))
        for e, wg in zip(idx_gpu[t].tolist(), w_gpu[t].tolist()):
            assert abs(wg - ow[e]) <= 1e-5 * max(1.0, abs(ow[e])), (t, e, wg, ow[e])
    return idx, w, z, flipped


def check_y(y_gpu, y_ref, what="", slack=None):
    """max |y_gpu - y_ref| <= 2e-3 * RMS(y_ref).  slack (nullable, per element): what the
    output format itself cannot hold, added to the bound -- with the residual flag the GPU
    returns fp32(x + y), whose rounding is not the MoE output's error."""
    y_ref = np.asarray(y_ref, np.float64)
    rms = float(np.sqrt(np.mean(y_ref ** 2)))
    diff = np.abs(np.asarray(y_gpu, np.float64) - y_ref)
    if slack is not None:
        diff = np.maximum(diff - np.asarray(slack, np.float64), 0.0)
    err = float(np.max(diff))
    assert err <= Y_TOL * rms, f"{what}: max err {err:.3e} > {Y_TOL} * rms {rms:.3e}"
    return err / rms if rms > 0 else 0.0


def residual_slack(y_stored):
    """One fp32 ulp of each stored output value: the kernels add the residual (or an earlier
    launch's sum) to the MoE sum in one fp32 addition, at most two such roundings per call
    (the host-table copy modes run the hit and the missed experts in two launches)."""
    y = np.abs(np.asarray(y_stored, np.float32))
    return np.spacing(y).astype(np.float64)


def replay_trace(calls_by_layer, wl, budget):
    """Oracle LRU over per-layer lists of routed-id arrays; returns (records, counters)."""
    recs, cnt = [], None
    for l, calls in enumerate(calls_by_layer):
        lru = LayerLRU(wl.n_experts, budget, wl.payload_bytes, l)
        for ids in calls:
            recs.extend(lru.step(np.unique(ids)))
        cnt = lru.counters if cnt is None else cnt + lru.counters
    return recs, cnt


def union_gemv_fits(H, I, T):
    """Whether the library's union GEMVs take a call of T tokens at this shape (their token
    images and activation digits fit the LDS budgets): mirrors mt_ffn_fits in kernels.hip."""
    pair_pitch = 80
    gateup_lds = T * (3 * (H // 64) * pair_pitch + 16 * (H // 32)) + 8 * 256 * 4
    down_lds = T * (3 * (I // 64) * pair_pitch + I)
    return 1 <= T <= 8 and 3 * T * I // 16 <= 9 * 256 and gateup_lds <= 65536 and down_lds <= 65536


def small_call_exact(T, H, I, n_union, budget, qtype="q8_0"):
    """Whether a multi-token call runs the fp32-accurate GEMVs (exact oracle) rather than the
    bf16 MFMA GEMMs: at most 8 tokens, and either the routed experts fit the slots (decode or
    union GEMVs) or the union GEMVs take the shape (run per chunk of the host-table path; the
    union GEMVs read Q8_0 / Q4_0 only)."""
    union = qtype in ("q8_0", "q4_0") and union_gemv_fits(H, I, T)
    return T <= 8 and (n_union <= budget or union)


def oracle_layer_y(x, wr, store, wl, layer, idx_or, w_or, z, idx_gpu, flipped, bf16=False,
                   tokens=None, prenorm=False):
    """Oracle y of one layer call; for tokens whose top-k flipped at a near-tie the
    GPU's set is used, weighted by the oracle's softmax over that set."""
    idx_use = idx_or.copy()
    w_use = w_or.copy()
    for t in flipped:
        idx_use[t] = idx_gpu[t]
        w_use[t] = softmax_of(z[t], idx_gpu[t])
    fn = moe_layer_bf16 if bf16 else moe_layer
    return fn(x, wr, store, Shape.of(wl), layer, routes=(idx_use, w_use), tokens=tokens,
              prenorm=prenorm)["y"]


def decode_chain(cache, wl, X, routers_dev, record_inputs=True):
    """Decode every token through every layer on the GPU with the library's residual
    flag (h_{l+1} = h_l + moe(h_l)), as the benchmark does.  Returns
    (final h [T,H], inputs [T,L,H] fp32 or None, idx [T,L,k], w [T,L,k])."""
    torch = torch_cuda()
    T, H = X.shape
    L, k = wl.n_layers, wl.top_k
    inputs = np.empty((T, L, H), np.float32) if record_inputs else None
    idx_all = np.empty((T, L, k), np.int32)
    w_all = np.empty((T, L, k), np.float32)
    h = torch.empty(H, dtype=torch.float32, device="cuda")
    y = torch.empty(H, dtype=torch.float32, device="cuda")
    out = np.empty_like(X)
    for t in range(T):
        h.copy_(torch.from_numpy(X[t]))
        for l in range(L):
            if record_inputs:
                inputs[t, l] = h.cpu().numpy()
            _, idx, w = cache.layer_forward(h, routers_dev[l], l, y, n_tokens=1, routes=True)
            idx_all[t, l], w_all[t, l] = idx[0], w[0]
            h, y = y, h
        out[t] = h.cpu().numpy()
    return out, inputs, idx_all, w_all


__all__ = ["log", "store_buffer", "make_cache", "check_routes", "check_y", "residual_slack",
           "replay_trace",
           "softmax_of", "decode_chain", "oracle_layer_y", "union_gemv_fits", "small_call_exact",
           "Shape", "moe_layer", "moe_layer_bf16", "TIE_GAP", "Y_TOL"]
