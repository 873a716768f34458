"""The seeded input generator: Philox against numpy's, normals, fp16 encoding, determinism."""
import numpy as np
import pytest

import synth


def test_philox_matches_numpy():
    # numpy's Philox bit generator is Philox4x64-10; it advances its counter
    # before each 4-word output, so its k-th block equals our counter k+1.
    for key in ([5, 7], [0, 0], [2**64 - 1, 12345]):
        bg = np.random.Philox(key=np.array(key, np.uint64), counter=np.zeros(4, np.uint64))
        raw = bg.random_raw(12)
        for blk in range(3):
            assert synth.philox4x64([blk + 1, 0, 0, 0], key) == [int(v) for v in raw[4 * blk: 4 * blk + 4]]


def test_normals_moments_and_random_access():
    k0 = synth.key(1, 9, 3, 4, 0)
    z = synth.normal_f32(k0, 0, 1 << 20).astype(np.float64)
    n = z.size
    assert abs(z.mean()) < 5 / np.sqrt(n)
    assert abs(z.std() - 1) < 5e-3
    kurt = ((z - z.mean()) ** 4).mean() / z.var() ** 2
    assert abs(kurt - 3) < 0.05
    assert abs((z < 0).mean() - 0.5) < 3e-3
    # any sub-range equals the same elements of the full draw
    for start, cnt in ((0, 1), (3, 5), (7, 9), (1000, 4097), (12345, 31)):
        np.testing.assert_array_equal(synth.normal_f32(k0, start, cnt), z[start:start + cnt].astype(np.float32))
    # different keys give different streams
    assert not np.array_equal(synth.normal_f32(k0 + 1, 0, 64), z[:64].astype(np.float32))


def test_f16_encoder_matches_numpy():
    rng = np.random.default_rng(0)
    vals = np.concatenate([
        rng.standard_normal(20000).astype(np.float32) * np.float32(1e-3),
        rng.standard_normal(20000).astype(np.float32) * np.float32(1e3),
        (rng.standard_normal(5000) * 1e-6).astype(np.float32),      # subnormal halves
        np.array([0.0, -0.0, 65504.0, 65519.0, 65520.0, 1e9, 2.0**-24, 2.0**-25, 3 * 2.0**-26,
                  1 + 2.0**-11, 1 + 3 * 2.0**-11], np.float32),         # ties and edges
    ])
    ours = np.array([synth.f32_to_f16_bits(v) for v in vals], np.uint16)
    np.testing.assert_array_equal(ours, vals.astype(np.float16).view(np.uint16))


def test_q8_0_encoding_error_bound():
    rng = np.random.default_rng(1)
    w = (rng.standard_normal(32 * 64) * 0.02).astype(np.float32)
    raw = synth.encode_blocks(8, w).reshape(-1, 34)
    d = raw[:, :2].copy().view(np.float16).astype(np.float64).ravel()
    q = raw[:, 2:].view(np.int8).astype(np.float64)
    amax = np.abs(w.reshape(-1, 32)).max(1)
    np.testing.assert_array_equal(d, (amax / 127).astype(np.float32).astype(np.float16).astype(np.float64))
    assert np.all(np.abs(q) <= 127)
    err = np.abs(d[:, None] * q - w.reshape(-1, 32))
    assert np.all(err <= d[:, None] * 0.5 + 1e-12 + np.abs(w.reshape(-1, 32)) * 2e-3)


def test_q4_0_encoding_error_bound():
    rng = np.random.default_rng(2)
    w = (rng.standard_normal(32 * 64) * 0.02).astype(np.float32)
    raw = synth.encode_blocks(2, w).reshape(-1, 18)
    d = raw[:, :2].copy().view(np.float16).astype(np.float64).ravel()
    n = np.concatenate([raw[:, 2:] & 0xF, raw[:, 2:] >> 4], axis=1).astype(np.float64)
    assert np.all((n >= 0) & (n <= 15))
    err = np.abs(d[:, None] * (n - 8) - w.reshape(-1, 32))
    assert np.all(err <= d[:, None] * 0.5 + 1e-12 + np.abs(w.reshape(-1, 32)) * 2e-3)


def test_store_is_thread_count_and_range_invariant():
    wl = synth.WORKLOADS["tiny"].with_(n_layers=3, n_experts=5)
    a = synth.expert_store(wl, threads=1)
    b = synth.expert_store(wl, threads=4)
    np.testing.assert_array_equal(a, b)
    c = synth.expert_store(wl, layer0=1, n_layers=2, threads=3)
    np.testing.assert_array_equal(a[wl.n_experts * wl.payload_bytes:], c)


def test_hidden_ar1_and_iid():
    wl = synth.WORKLOADS["tiny"].with_(hidden=2048, n_tokens=40)
    x = synth.hidden(wl, rho=0.8).astype(np.float64)
    assert abs(x.std() - 1) < 0.05
    corr = np.mean([np.corrcoef(x[t], x[t + 1])[0, 1] for t in range(39)])
    assert abs(corr - 0.8) < 0.03
    y = synth.hidden(wl, rho=-1.0).astype(np.float64)
    corr = np.mean([np.corrcoef(y[t], y[t + 1])[0, 1] for t in range(39)])
    assert abs(corr) < 0.03


@pytest.mark.parametrize("name", sorted(synth.WORKLOADS))
def test_workload_sizes(name):
    wl = synth.WORKLOADS[name]
    expect_p = {"tiny": 104448, "a3b_decode": 5013504, "a3b_sweep": 5013504,
                "q4_decode": 6690816, "a3b_prefill": 5013504, "a3b_verify": 5013504,
                "q4km_decode": 3059712, "q4km_prefill": 3059712}[name]
    assert wl.payload_bytes == expect_p
    assert wl.payload_bytes % 16 == 0


@pytest.mark.parametrize("qtype", ["q4_k", "q6_k", "q4_k_m"])
def test_kquant_store_decodes_near_the_drawn_weights(qtype):
    """The K-quant encoders (generation only) keep the drawn N(0, 0.02) weights: the oracle's
    decoding of the store is within the formats' quantisation error of them."""
    from oracle import quant
    wl = synth.WORKLOADS["tiny"].with_(qtype=qtype, inter=256)
    arr = synth.expert_store(wl)
    assert arr.size == wl.store_bytes
    gu, dn = wl.formats
    for m, fmt in enumerate((gu, gu, dn)):
        w = quant.expert_weights(arr, qtype, wl.n_experts, wl.hidden, wl.inter, 0, 5)[m]
        drawn = synth.normal_f32(synth.key(1, wl.model_seed, 0, 5, m), 0, w.size, wl.weight_sigma)
        rel = np.sqrt(np.mean((w.ravel() - drawn) ** 2)) / np.sqrt(np.mean(drawn.astype(np.float64) ** 2))
        assert rel < {"q4_k": 0.1, "q6_k": 0.03}[fmt], (m, fmt, rel)
