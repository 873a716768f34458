"""One MoE layer call over the slot cache, and the residual stack (oracle; test infrastructure only).

A layer call (the paper's Native Serving Path section; its throughput model,
the generated-tokens over compute-plus-materialisation relation, is what the
GPU path is timed against):

1. route every token (``router.route``);
2. look the distinct routed experts up in the layer's slot table, counting
   hits, misses, evictions and materialised bytes (``lru.LayerLRU.step``);
3. y_t = sum over the token's routed experts of w_{t,e} f_e(x_t)
   (``ffn``).  Where an expert's weights came from (a hit or a fresh copy)
   does not change y: the cache only moves bytes.

The stack feeds each layer the previous layer's output plus its input
(h_{l+1} = h_l + y_l, rounded to fp32 at the layer boundary, since a layer
takes fp32 hidden states); this reading keeps the true layer-to-layer
dependency of decoding.  With ``prenorm`` a layer routes and runs its experts
on the RMS-normalised input x / sqrt(mean(x^2) + 1e-6) (unit gain), the
pre-norm residual block of MoE transformers without attention; without it a
deep stack of SwiGLU experts grows its activations without bound.

``moe_layer_bf16`` is the prefill variant: the dequantised weights d*q are
rounded to bfloat16 (nearest, ties to even), as the MFMA weight tiles hold
them; inputs, activations and all sums stay exact (fp64).  (The MFMA path
carries its activations as two bf16 terms, hi + lo, about 16 significant bits,
so it is compared against exact activations.)
"""
from dataclasses import dataclass

import numpy as np

from . import ffn, quant, router
from .lru import LayerLRU
from .numerics import bf16_round


@dataclass(frozen=True)
class Shape:
    """The sizes a layer call needs (duck-types any object with these fields)."""
    qtype: str
    n_experts: int
    hidden: int
    inter: int
    top_k: int

    @staticmethod
    def of(obj):
        return Shape(obj.qtype, obj.n_experts, obj.hidden, obj.inter, obj.top_k)

    @property
    def payload_bytes(self):
        return quant.payload_bytes(self.qtype, self.hidden, self.inter)


EPS = 1e-6


def rms_normalize(x):
    """x / sqrt(mean(x^2) + 1e-6) per row, in fp64."""
    x = np.asarray(x, dtype=np.float64)
    return x / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + EPS)


def _experts(store, shape, layer, ids, bf16=False):
    out = {}
    for e in ids:
        w = quant.expert_weights(store, shape.qtype, shape.n_experts, shape.hidden, shape.inter,
                                 layer, int(e))
        out[int(e)] = tuple(bf16_round(m) for m in w) if bf16 else w
    return out


def moe_layer(x, router_w, store, shape, layer, lru=None, routes=None, tokens=None, prenorm=False):
    """One layer call.

    x [T, H] fp32; router_w [H, E] fp32; store: the whole uint8 expert store.
    ``lru``: the layer's LayerLRU (updated in place) or None.
    ``routes``: optional (idx, w) to use instead of the oracle's own routing
    (used when the GPU took the other side of a near-tie).
    ``tokens``: optional subset of token indices whose y is computed (the
    routing and the cache step always cover all tokens).
    ``prenorm``: route and run the experts on rms_normalize(x).
    Returns dict(y [T,H] fp64 (rows outside ``tokens`` are nan), idx, w, gap, records).
    """
    shape = Shape.of(shape)
    x = np.atleast_2d(np.asarray(x, dtype=np.float32))
    x = rms_normalize(x) if prenorm else x.astype(np.float64)
    idx, w, gap = router.route(x, router_w, shape.top_k)
    if routes is not None:
        idx, w = routes
    records = lru.step(np.unique(idx)) if lru is not None else None
    T = x.shape[0]
    tokens = range(T) if tokens is None else tokens
    need = sorted({int(e) for t in tokens for e in idx[t]})
    ex = _experts(store, shape, layer, need)
    y = np.full((T, shape.hidden), np.nan)
    for t in tokens:
        y[t] = ffn.combine(x[t], [ex[int(e)] for e in idx[t]], w[t])
    return dict(y=y, idx=idx, w=w, gap=gap, records=records)


def moe_layer_bf16(x, router_w, store, shape, layer, lru=None, routes=None, tokens=None,
                   prenorm=False):
    """Prefill variant of ``moe_layer``: the dequantised weights rounded to bf16."""
    shape = Shape.of(shape)
    x = np.atleast_2d(np.asarray(x, dtype=np.float32))
    x = rms_normalize(x) if prenorm else x.astype(np.float64)
    idx, w, gap = router.route(x, router_w, shape.top_k)
    if routes is not None:
        idx, w = routes
    records = lru.step(np.unique(idx)) if lru is not None else None
    T = x.shape[0]
    tokens = list(range(T) if tokens is None else tokens)
    need = sorted({int(e) for t in tokens for e in idx[t]})
    ex = _experts(store, shape, layer, need, bf16=True)
    y = np.full((T, shape.hidden), np.nan)
    for t in tokens:
        y[t] = ffn.combine(x[t], [ex[int(e)] for e in idx[t]], w[t])
    return dict(y=y, idx=idx, w=w, gap=gap, records=records)


def run_stack(x_tokens, routers, store, shape, n_slots, decode=True, bf16=False, prenorm=False):
    """Decode (one token per layer call) or prefill (all tokens per call) through
    every layer from a cold cache.

    x_tokens [T, H] fp32; routers [L, H, E] fp32.  Returns dict with the final
    hidden states, per-(token,layer) inputs, routes, records and per-layer
    counters.
    """
    shape = Shape.of(shape)
    L = routers.shape[0]
    lrus = [LayerLRU(shape.n_experts, n_slots, shape.payload_bytes, l) for l in range(L)]
    fn = moe_layer_bf16 if bf16 else moe_layer
    records, inputs, routes = [], {}, {}
    calls = [[t] for t in range(x_tokens.shape[0])] if decode else [list(range(x_tokens.shape[0]))]
    h_final = np.empty_like(x_tokens, dtype=np.float32)
    for toks in calls:
        h = np.asarray(x_tokens[toks], dtype=np.float32)
        for l in range(L):
            out = fn(h, routers[l], store, shape, l, lrus[l], prenorm=prenorm)
            inputs[(toks[0], l)] = h.copy()
            routes[(toks[0], l)] = (out["idx"], out["w"], out["gap"])
            records.extend(out["records"])
            h = (h.astype(np.float64) + out["y"]).astype(np.float32)
        h_final[toks] = h
    return dict(h=h_final, inputs=inputs, routes=routes, records=records,
                counters=[lr.counters for lr in lrus])
