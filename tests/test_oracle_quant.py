"""Pins of the oracle's Q8_0 / Q4_0 decoding and payload addressing against hand-built blocks."""
import numpy as np
import pytest

from conftest import golden_path
from oracle import quant


def _golden_blocks():
    rows = []
    for line in open(golden_path("quant_hand_blocks.txt")):
        line = line.split("#")[0].strip()
        if not line:
            continue
        lhs, rhs = line.split("=>")
        kind, scale, *payload = lhs.split()
        want = [float(v) for v in rhs.split()]
        assert len(want) == 32, line
        s = int(scale, 16)
        head = bytes([s & 0xFF, s >> 8])
        if kind == "q8":
            assert len(payload) == 32, line
            body = bytes(int(v) & 0xFF for v in payload)
        else:
            assert len(payload) == 16, line
            body = bytes(int(v, 16) for v in payload)
        rows.append((kind, np.frombuffer(head + body, np.uint8), np.array(want)))
    return rows


@pytest.mark.parametrize("row", range(12))
def test_hand_blocks(row):
    kind, raw, want = _golden_blocks()[row]
    got = quant.dequant_q8_0(raw) if kind == "q8" else quant.dequant_q4_0(raw)
    np.testing.assert_array_equal(got, want)


def test_golden_file_has_all_rows():
    assert len(_golden_blocks()) == 12


def test_multi_block_rows_and_matrix_layout():
    # a 3 x 64 Q8_0 matrix whose block (r, c) has scale 2^(r) and q_j = 10*c + j - 16
    raw = bytearray()
    for r in range(3):
        for c in range(2):
            d = np.float16(2.0 ** r).view(np.uint16)
            raw += bytes([int(d) & 0xFF, int(d) >> 8])
            raw += bytes((10 * c + j - 16) & 0xFF for j in range(32))
    m = quant.dequant_matrix(np.frombuffer(bytes(raw), np.uint8), "q8_0", 3, 64)
    for r in range(3):
        for col in range(64):
            c, j = divmod(col, 32)
            assert m[r, col] == 2.0 ** r * (10 * c + j - 16)


def test_payload_offsets():
    # every (layer, expert, matrix) gets a distinct scale; check the slicing picks it
    qt, E, H, I = "q4_0", 3, 64, 32
    mb = quant.matrix_bytes(qt, I, H)
    P = quant.payload_bytes(qt, H, I)
    assert P == 3 * mb == 3 * 32 * 2 * 18
    L = 2
    store = np.zeros(L * E * P, np.uint8)
    for l in range(L):
        for e in range(E):
            for m in range(3):
                tag = 1 + (l * E + e) * 3 + m                      # 1..18, exact in fp16
                d = int(np.float16(tag).view(np.uint16))
                base = (l * E + e) * P + m * mb
                for b in range(mb // 18):
                    store[base + 18 * b] = d & 0xFF
                    store[base + 18 * b + 1] = d >> 8
                    store[base + 18 * b + 2: base + 18 * b + 18] = 0x99   # n = 9 -> weight d
    for l in range(L):
        for e in range(E):
            wg, wu, wd = quant.expert_weights(store, qt, E, H, I, l, e)
            assert wg.shape == (I, H) and wu.shape == (I, H) and wd.shape == (H, I)
            for m, w in enumerate((wg, wu, wd)):
                assert np.all(w == 1 + (l * E + e) * 3 + m)


def test_sizes_match_format_arithmetic():
    assert quant.payload_bytes("q8_0", 2048, 768) == 5013504
    assert quant.payload_bytes("q4_0", 2816, 1408) == 6690816
    assert quant.payload_bytes("q8_0", 256, 128) == 104448
