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


def _expand(tokens):
    """Tokens with "x*n" repetitions expanded."""
    out = []
    for t in tokens:
        if "*" in t:
            v, n = t.split("*")
            out.extend([v] * int(n))
        else:
            out.append(t)
    return out


def _kquant_golden():
    rows = []
    for line in open(golden_path("kquant_hand_blocks.txt")):
        line = line.split("#")[0].strip()
        if not line:
            continue
        lhs, rhs = line.split("=>")
        want = np.array([float(v) for v in _expand(rhs.split())])
        assert want.size == 256, line[:40]
        groups = [g.split() for g in lhs.split("|")]
        kind = groups[0][0]
        if kind == "q4_k":
            d, dmin = int(groups[0][1], 16), int(groups[0][2], 16)
            sc = [int(v, 16) for v in _expand(groups[0][3:])]
            qs = [int(v, 16) for v in _expand(groups[1])]
            assert len(sc) == 12 and len(qs) == 128
            raw = bytes([d & 0xFF, d >> 8, dmin & 0xFF, dmin >> 8] + sc + qs)
        else:
            d = int(groups[0][1], 16)
            ql = [int(v, 16) for v in _expand(groups[0][2:])]
            qh = [int(v, 16) for v in _expand(groups[1])]
            scales = [int(v) & 0xFF for v in _expand(groups[2])]
            assert len(ql) == 128 and len(qh) == 64 and len(scales) == 16
            raw = bytes(ql + qh + scales + [d & 0xFF, d >> 8])
        rows.append((kind, np.frombuffer(raw, np.uint8), want))
    return rows


@pytest.mark.parametrize("row", range(8))
def test_kquant_hand_blocks(row):
    kind, raw, want = _kquant_golden()[row]
    assert raw.size == quant.FORMATS[kind][0]
    np.testing.assert_array_equal(quant.dequant(raw, kind), want)


def test_kquant_golden_has_all_blocks_and_consecutive_blocks_decode_alike():
    rows = _kquant_golden()
    assert [r[0] for r in rows] == ["q4_k"] * 3 + ["q6_k"] * 3 + ["q4_k", "q6_k"]
    for kind in ("q4_k", "q6_k"):
        mine = [r for r in rows if r[0] == kind]
        raw = np.concatenate([r[1] for r in mine])
        np.testing.assert_array_equal(quant.dequant(raw, kind), np.concatenate([r[2] for r in mine]))


def test_q4_k_scale_packing_round_trip():
    # every (scale, min) pair 0..63 in every position survives the 6-bit packing rule
    rng = np.random.default_rng(3)
    for _ in range(200):
        sc, mn = rng.integers(0, 64, size=8), rng.integers(0, 64, size=8)
        b = np.zeros(12, np.int64)
        b[0:4] = sc[0:4] | ((sc[4:8] >> 4) << 6)
        b[4:8] = mn[0:4] | ((mn[4:8] >> 4) << 6)
        b[8:12] = (sc[4:8] & 15) | ((mn[4:8] & 15) << 4)
        got_sc, got_mn = quant.q4_k_scales_mins(b.astype(np.uint8)[None])
        assert got_sc[0].tolist() == sc.tolist() and got_mn[0].tolist() == mn.tolist()


def test_mixed_payload_offsets_and_sizes():
    # Q4_K_M: gate and up Q4_K, down Q6_K; every matrix tagged by its scale
    qt, E, H, I, L = "q4_k_m", 2, 256, 256, 2
    mg = quant.matrix_bytes("q4_k", I, H)
    md = quant.matrix_bytes("q6_k", H, I)
    P = quant.payload_bytes(qt, H, I)
    assert (mg, md, P) == (256 * 144, 256 * 210, 2 * 256 * 144 + 256 * 210)
    store = np.zeros(L * E * P, np.uint8)
    for l in range(L):
        for e in range(E):
            base = (l * E + e) * P
            for m in range(3):
                tag = 1 + (l * E + e) * 3 + m
                dbits = int(np.float16(tag).view(np.uint16))
                if m < 2:   # Q4_K: d = tag, dmin = 0, sc_0..7 = 1, mins 0, every q = 1
                    for b in range(mg // 144):
                        o = base + m * mg + 144 * b
                        store[o:o + 2] = [dbits & 0xFF, dbits >> 8]
                        store[o + 4:o + 8] = 1
                        store[o + 12:o + 16] = 0x01
                        store[o + 16:o + 144] = 0x11
                else:       # Q6_K: scales 1, q = 33 everywhere (ql low nibbles 1, qh bits 0b10)
                    for b in range(md // 210):
                        o = base + 2 * mg + 210 * b
                        store[o:o + 128] = 0x11
                        store[o + 128:o + 192] = 0xAA
                        store[o + 192:o + 208] = 1
                        store[o + 208:o + 210] = [dbits & 0xFF, dbits >> 8]
    for l in range(L):
        for e in range(E):
            wg, wu, wd = quant.expert_weights(store, qt, E, H, I, l, e)
            assert wg.shape == (I, H) and wu.shape == (I, H) and wd.shape == (H, I)
            for m, w in enumerate((wg, wu, wd)):
                assert np.all(w == 1 + (l * E + e) * 3 + m), (l, e, m)


def test_kquant_sizes_match_format_arithmetic():
    assert quant.payload_bytes("q4_k_m", 2048, 768) == 2 * 768 * 8 * 144 + 2048 * 3 * 210 == 3059712
    assert quant.payload_bytes("q4_k", 2048, 768) == 3 * 768 * 8 * 144
    assert quant.payload_bytes("q6_k", 2048, 768) == 3 * 768 * 8 * 210
