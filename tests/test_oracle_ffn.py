"""Pins of the oracle's SwiGLU expert FFN, combine and layer call: closed forms, scaling,
degenerate weights, invariances."""
import numpy as np
import torch
from scipy.special import expit

import synth
from oracle import ffn, layer, quant
from oracle.layer import Shape


def _q8_matrix(rows, cols, entries, scales):
    """Q8_0 bytes of a matrix with q=1 at the (row, col) entries and per-row fp16 scale."""
    raw = np.zeros((rows, cols // 32, 34), np.uint8)
    for r in range(rows):
        d = int(np.float16(scales[r]).view(np.uint16))
        raw[r, :, 0], raw[r, :, 1] = d & 0xFF, d >> 8
    for r, c in entries:
        raw[r, c // 32, 2 + c % 32] = 1
    return raw.ravel()


def _closed_form_store(H=64, I=32):
    # gate row r reads x[2r], up row r reads x[2r+1], down row j reads a[j % I] with scale s_j
    wg = _q8_matrix(I, H, [(r, 2 * r) for r in range(I)], [1.0] * I)
    wu = _q8_matrix(I, H, [(r, 2 * r + 1) for r in range(I)], [1.0] * I)
    s = np.where(np.arange(H) < I, 1.0, -0.5)
    wd = _q8_matrix(H, I, [(j, j % I) for j in range(H)], s)
    return np.concatenate([wg, wu, wd]), s


def test_silu_matches_torch():
    s = np.concatenate([np.linspace(-50, 50, 10001), [-800.0, 800.0, 0.0]])
    ref = torch.nn.functional.silu(torch.from_numpy(s)).numpy()
    np.testing.assert_allclose(ffn.silu(s), ref, rtol=1e-15, atol=1e-300)
    assert ffn.silu(0.0) == 0.0


def test_closed_form_single_expert():
    H, I = 64, 32
    store, s = _closed_form_store(H, I)
    wg, wu, wd = quant.expert_weights(store, "q8_0", 1, H, I, 0, 0)
    rng = np.random.default_rng(0)
    x = rng.standard_normal(H) * 2
    y = ffn.expert_ffn(x, wg, wu, wd)
    j = np.arange(H)
    g, u = x[2 * (j % I)], x[2 * (j % I) + 1]
    np.testing.assert_allclose(y, s * g * expit(g) * u, rtol=1e-14, atol=1e-15)


def test_closed_form_bf16_variant():
    # weights that are not bf16-representable: d = 1 + 2^-9 (exact in fp16) times q = 1
    # rounds to 1 (ties to even) in bf16; the activation path stays exact
    H, I, E = 64, 32, 1
    store, s = _closed_form_store(H, I)
    st = store.copy()
    d = int(np.float16(1 + 2.0 ** -9).view(np.uint16))
    mb = quant.matrix_bytes("q8_0", I, H)
    gate = st[:mb].reshape(-1, 34)                      # gate matrix blocks only
    gate[:, 0], gate[:, 1] = d & 0xFF, d >> 8
    shape = Shape("q8_0", E, H, I, 1)
    rng = np.random.default_rng(1)
    x = rng.standard_normal((3, H)).astype(np.float32)
    wr = np.zeros((H, E), np.float32)
    exact = layer.moe_layer(x, wr, st, shape, 0)["y"]
    out = layer.moe_layer_bf16(x, wr, st, shape, 0)
    j = np.arange(H)
    for t in range(3):
        g = x[t, 2 * (j % I)].astype(np.float64)          # bf16(1 + 2^-9) = 1
        u = x[t, 2 * (j % I) + 1].astype(np.float64)
        np.testing.assert_allclose(out["y"][t], s * g * expit(g) * u, rtol=1e-14, atol=1e-15)
        assert not np.allclose(exact[t], out["y"][t], rtol=1e-5, atol=0)  # the rounding matters
    # weights already bf16-exact: the variant equals the exact layer
    np.testing.assert_allclose(layer.moe_layer_bf16(x, wr, store, shape, 0)["y"],
                               layer.moe_layer(x, wr, store, shape, 0)["y"], rtol=1e-14, atol=1e-15)


def _random_store(wl):
    return synth.expert_store(wl, threads=2)


def test_identical_experts_all_routed_is_dense_ffn():
    wl = synth.WORKLOADS["tiny"].with_(n_experts=6, top_k=6)
    one = _random_store(wl.with_(n_experts=1))
    store = np.tile(one, 6)
    shape = Shape.of(wl)
    x = synth.hidden(wl, n_tokens=4)
    wr = synth.router(wl)[0]
    out = layer.moe_layer(x, wr, store, shape, 0)
    wg, wu, wd = quant.expert_weights(one, "q8_0", 1, wl.hidden, wl.inter, 0, 0)
    for t in range(4):
        dense = ffn.expert_ffn(x[t].astype(np.float64), wg, wu, wd)
        np.testing.assert_allclose(out["y"][t], dense, rtol=1e-12, atol=1e-14)


def _scale_matrix(store, shape, which, factor_bits):
    """Return a copy of the store with every block scale of matrix `which` modified."""
    st = store.copy()
    mb = quant.matrix_bytes(shape.qtype, shape.inter, shape.hidden)
    P = shape.payload_bytes
    bb = quant.BLOCK_BYTES[shape.qtype]
    for e in range(shape.n_experts):
        base = e * P + which * mb
        blocks = st[base: base + mb].reshape(-1, bb)
        d = blocks[:, 0].astype(np.uint16) | (blocks[:, 1].astype(np.uint16) << 8)
        d = factor_bits(d)
        blocks[:, 0], blocks[:, 1] = d & 0xFF, d >> 8
    return st


def test_down_scale_doubling_doubles_output_and_zero_gate_or_up_gives_zero():
    for qt in ("q8_0", "q4_0"):
        wl = synth.WORKLOADS["tiny"].with_(qtype=qt)
        store = _random_store(wl)
        shape = Shape.of(wl)
        x = synth.hidden(wl, n_tokens=3)
        wr = synth.router(wl)[0]
        base = layer.moe_layer(x, wr, store, shape, 0)["y"]
        # exponent field + 1 doubles every (normal, non-zero) fp16 scale exactly
        dbl = _scale_matrix(store, shape, 2, lambda d: np.where(d & 0x7C00, d + 0x400, d).astype(np.uint16))
        np.testing.assert_array_equal(layer.moe_layer(x, wr, dbl, shape, 0)["y"], 2 * base)
        for which in (0, 1):
            z = _scale_matrix(store, shape, which, lambda d: np.zeros_like(d))
            assert np.all(layer.moe_layer(x, wr, z, shape, 0)["y"] == 0)


def test_output_does_not_depend_on_cache_state():
    wl = synth.WORKLOADS["tiny"]
    store = _random_store(wl)
    shape = Shape.of(wl)
    x = synth.hidden(wl, n_tokens=2)
    wr = synth.router(wl)[0]
    from oracle.lru import LayerLRU
    warm = LayerLRU(16, 4, shape.payload_bytes)
    warm.step([0, 1, 2, 3])
    cold = LayerLRU(16, 4, shape.payload_bytes)
    a = layer.moe_layer(x, wr, store, shape, 0, lru=warm)
    b = layer.moe_layer(x, wr, store, shape, 0, lru=cold)
    np.testing.assert_array_equal(a["y"], b["y"])


def test_stack_counters_agree_with_records():
    wl = synth.WORKLOADS["tiny"]
    store = _random_store(wl)
    out = layer.run_stack(synth.hidden(wl), synth.router(wl), store, wl, wl.budget_slots)
    recs = out["records"]
    c = out["counters"][0]
    assert c.hits == sum(r[3] for r in recs)
    assert c.misses == sum(1 - r[3] for r in recs)
    assert c.evictions == sum(r[5] >= 0 for r in recs)
    assert c.materialized_bytes == c.misses * wl.payload_bytes
    assert len({r[1] for r in recs}) == wl.n_tokens
    assert np.all(np.isfinite(out["h"]))


def test_stack_is_residual_chain():
    # with every gate scale zero each layer adds nothing: the stack is the identity
    wl = synth.WORKLOADS["tiny"].with_(n_layers=2)
    store = _random_store(wl)
    shape = Shape.of(wl)
    zero = store.copy()
    mb = quant.matrix_bytes("q8_0", wl.inter, wl.hidden)
    for le in range(wl.n_layers * wl.n_experts):
        blocks = zero[le * wl.payload_bytes: le * wl.payload_bytes + mb].reshape(-1, 34)
        blocks[:, :2] = 0
    x = synth.hidden(wl, n_tokens=3)
    R = synth.router(wl)
    out = layer.run_stack(x, R, zero, wl, 4)
    np.testing.assert_array_equal(out["h"], x)
    # a real two-layer stack equals two single layer calls with the sum in between
    out = layer.run_stack(x, R, store, wl, 4)
    for t in range(3):
        y0 = layer.moe_layer(x[t:t + 1], R[0], store, shape, 0)["y"]
        h1 = (x[t:t + 1].astype(np.float64) + y0).astype(np.float32)
        y1 = layer.moe_layer(h1, R[1], store, shape, 1)["y"]
        np.testing.assert_array_equal(out["h"][t], (h1.astype(np.float64) + y1).astype(np.float32)[0])
        assert not np.array_equal(out["h"][t], x[t])


def test_prenorm_definition_and_scale_invariance():
    from oracle.layer import rms_normalize
    # a vector of +-c has mean square c^2, so it normalises to +-1/sqrt(1 + 1e-6/c^2)
    for c in (1.0, 3.0, 1e-2):
        v = np.array([c, -c, c, c, -c, -c, c, -c])
        np.testing.assert_allclose(rms_normalize(v), np.sign(v) / np.sqrt(1 + 1e-6 / c ** 2),
                                   rtol=1e-15)
    wl = synth.WORKLOADS["tiny"]
    store = _random_store(wl)
    shape = Shape.of(wl)
    x = synth.hidden(wl, n_tokens=3)
    wr = synth.router(wl)[0]
    a = layer.moe_layer(x, wr, store, shape, 0, prenorm=True)
    b = layer.moe_layer((4 * x).astype(np.float32), wr, store, shape, 0, prenorm=True)
    np.testing.assert_array_equal(a["idx"], b["idx"])
    np.testing.assert_allclose(a["y"], b["y"], rtol=1e-5, atol=1e-9)
    # a stack with pre-norm stays bounded over many layers
    wl48 = synth.WORKLOADS["tiny"].with_(n_layers=24)
    st = _random_store(wl48)
    out = layer.run_stack(synth.hidden(wl48, n_tokens=2), synth.router(wl48), st, wl48, 4,
                          prenorm=True)
    assert np.all(np.isfinite(out["h"])) and np.abs(out["h"]).max() < 100
