"""Pins of the oracle's number-format decoding against library routines and known bit patterns."""
import numpy as np
import torch

from oracle.numerics import bf16_round, fp16_decode


def test_fp16_decode_all_patterns_match_numpy():
    bits = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)
    ours = fp16_decode(bits)
    ref = bits.view(np.float16).astype(np.float64)
    nan = np.isnan(ref)
    np.testing.assert_array_equal(np.isnan(ours), nan)
    np.testing.assert_array_equal(ours[~nan], ref[~nan])
    np.testing.assert_array_equal(np.signbit(ours[~nan]), np.signbit(ref[~nan]))


def test_fp16_decode_named_patterns():
    assert fp16_decode(0x3C00) == 1.0
    assert fp16_decode(0x0001) == 2.0 ** -24
    assert fp16_decode(0x7BFF) == 65504.0
    assert fp16_decode(0x8000) == 0.0 and np.signbit(fp16_decode(0x8000))
    assert fp16_decode(0xC000) == -2.0
    assert fp16_decode(0x03FF) == 1023 * 2.0 ** -24
    assert fp16_decode(0x7C00) == np.inf


def test_bf16_round_matches_torch_on_fp32_inputs():
    rng = np.random.default_rng(0)
    base = rng.standard_normal(200000).astype(np.float32)
    scales = np.float32(10.0) ** rng.integers(-40, 39, base.size).astype(np.float32)
    with np.errstate(over="ignore"):
        x = (base * scales).astype(np.float32)
    # exact ties: bf16 value plus half an ulp, both parities of the kept bit
    ties = (np.arange(1, 4097, dtype=np.uint32) << 16 | 0x8000).view(np.float32)
    edges = np.array([0.0, -0.0, 1e-45, -1e-45, 1e-40, 3.4e38, -3.4e38, 3.3e38, 1.0, 2.0 ** -126,
                      2.0 ** -127], np.float32)
    x = np.concatenate([x, ties, -ties, edges])
    ours = bf16_round(x.astype(np.float64))
    ref = torch.from_numpy(x).to(torch.bfloat16).to(torch.float64).numpy()
    np.testing.assert_array_equal(ours, ref)
    np.testing.assert_array_equal(np.signbit(ours), np.signbit(ref))


def test_bf16_round_fixed_points():
    # values already representable in bf16 are unchanged
    v = np.array([1.0, -3.5, 2.0 ** -130, 255.0 * 2.0 ** 100, 0.0078125])
    np.testing.assert_array_equal(bf16_round(v), v)
    # 1 + 2^-8 is halfway between 1 and 1 + 2^-7: ties to even -> 1
    assert bf16_round(np.array([1 + 2.0 ** -8]))[0] == 1.0
    assert bf16_round(np.array([1 + 3 * 2.0 ** -8]))[0] == 1 + 2 * 2.0 ** -7
