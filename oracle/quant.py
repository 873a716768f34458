"""GGUF-style block formats and the expert payload layout (oracle; test infrastructure only).

Block formats (GGUF, the llama.cpp model format the paper serves from; the
paper's model-profile table names Q8_0 profiles and a Q4_K_M profile; Q4_0
stands in for a plain 4-bit format):

* Q8_0, 34 bytes per 32 weights: bytes 0-1 scale d (binary16, little-endian),
  bytes 2-33 signed 8-bit q_j.  Weight j is d * q_j.
* Q4_0, 18 bytes per 32 weights: bytes 0-1 scale d; byte 2+j (j < 16) holds
  n_j in its low nibble and n_{j+16} in its high nibble.  Weight is d*(n-8).
* Q4_K, 144 bytes per super-block of 256 weights: d (binary16), dmin
  (binary16), 12 bytes holding eight 6-bit sub-block scales sc_j and eight 6-bit
  mins m_j, then 128 bytes of 4-bit q.  The 12 bytes b: for j < 4, sc_j is the
  low 6 bits of b[j] and m_j the low 6 bits of b[j+4]; for j >= 4, sc_j is the
  low nibble of b[j+4] with the top two bits of b[j-4] above it, and m_j the high
  nibble of b[j+4] with the top two bits of b[j] above it.  The 256 weights are
  four 64-weight chunks; chunk c reads q bytes 32c..32c+31, whose low nibbles
  are sub-block 2c (32 weights, in byte order) and high nibbles sub-block 2c+1.
  Weight = d * sc_j * q - dmin * m_j.
* Q6_K, 210 bytes per super-block of 256 weights: 128 bytes ql (low 4 bits of
  q), 64 bytes qh (high 2 bits), 16 signed 8-bit scales, d (binary16).  The
  super-block is two halves of 128 weights; weight 32g + l of half h (g < 4,
  l < 32) takes its low 4 bits from ql[64h + 32(g mod 2) + l] (low nibble for
  g < 2, high nibble for g >= 2) and its high 2 bits from bits 2g, 2g+1 of
  qh[32h + l].  Scale i covers weights 16i..16i+15.  Weight = d * scale * (q - 32).

"Q4_K_M" here names the mix of the paper's 4-bit model profile as this path
stores it: Q4_K gate and up matrices and a Q6_K down matrix (the one format per
matrix role that a uniform slot size needs).

Expert payload (the paper's Split-Pack section: one block per layer and expert;
its Native Serving Path section: separate gate, up and down tensors): one
contiguous byte range per (layer l, expert e) at offset (l*E + e)*P, laid out
as [W_gate (inter x hidden) | W_up (inter x hidden) | W_down (hidden x inter)].
Each matrix is row-major, one row per output; a row is its inputs split into
consecutive blocks (or super-blocks) of its format.
"""
import numpy as np

from .numerics import fp16_decode

# format: (bytes per block, weights per block)
FORMATS = {"q8_0": (34, 32), "q4_0": (18, 32), "q4_k": (144, 256), "q6_k": (210, 256)}
# model qtype -> (gate/up format, down format)
MIXES = {"q4_k_m": ("q4_k", "q6_k")}
BLOCK_BYTES = {k: v[0] for k, v in FORMATS.items()}


def roles(qtype):
    """(gate/up format, down format) of a model qtype."""
    return MIXES.get(qtype, (qtype, qtype))


def _fp16(lo, hi):
    return np.asarray(fp16_decode(lo.astype(np.uint16) | (hi.astype(np.uint16) << 8)))


def dequant_q8_0(raw):
    """fp64 weights of consecutive Q8_0 blocks (raw: uint8 bytes, multiple of 34)."""
    b = np.frombuffer(np.ascontiguousarray(raw, dtype=np.uint8), dtype=np.uint8).reshape(-1, 34)
    d = _fp16(b[:, 0], b[:, 1])
    q = b[:, 2:].view(np.int8).astype(np.float64)
    return (d[:, None] * q).ravel()


def dequant_q4_0(raw):
    """fp64 weights of consecutive Q4_0 blocks (raw: uint8 bytes, multiple of 18)."""
    b = np.frombuffer(np.ascontiguousarray(raw, dtype=np.uint8), dtype=np.uint8).reshape(-1, 18)
    d = _fp16(b[:, 0], b[:, 1])
    packed = b[:, 2:].astype(np.int64)
    n = np.concatenate([packed & 0xF, packed >> 4], axis=1)  # elements 0..15, then 16..31
    return (d[:, None] * (n - 8).astype(np.float64)).ravel()


def q4_k_scales_mins(b12):
    """The eight 6-bit (scale, min) pairs of Q4_K super-blocks; b12 [n, 12] uint8 -> two [n, 8]."""
    b = b12.astype(np.int64)
    sc = np.empty((b.shape[0], 8), np.int64)
    mn = np.empty((b.shape[0], 8), np.int64)
    for j in range(4):
        sc[:, j] = b[:, j] & 63
        mn[:, j] = b[:, j + 4] & 63
    for j in range(4, 8):
        sc[:, j] = (b[:, j + 4] & 0xF) | ((b[:, j - 4] >> 6) << 4)
        mn[:, j] = (b[:, j + 4] >> 4) | ((b[:, j] >> 6) << 4)
    return sc, mn


def dequant_q4_k(raw):
    """fp64 weights of consecutive Q4_K super-blocks (raw: multiple of 144 bytes)."""
    b = np.frombuffer(np.ascontiguousarray(raw, dtype=np.uint8), dtype=np.uint8).reshape(-1, 144)
    d = _fp16(b[:, 0], b[:, 1])
    dmin = _fp16(b[:, 2], b[:, 3])
    sc, mn = q4_k_scales_mins(b[:, 4:16])
    qs = b[:, 16:].astype(np.int64)
    out = np.empty((b.shape[0], 256), np.float64)
    for c in range(4):
        chunk = qs[:, 32 * c:32 * c + 32]
        for half, q in ((0, chunk & 0xF), (1, chunk >> 4)):
            j = 2 * c + half
            out[:, 32 * j:32 * j + 32] = (d * sc[:, j])[:, None] * q - (dmin * mn[:, j])[:, None]
    return out.ravel()


def dequant_q6_k(raw):
    """fp64 weights of consecutive Q6_K super-blocks (raw: multiple of 210 bytes)."""
    b = np.frombuffer(np.ascontiguousarray(raw, dtype=np.uint8), dtype=np.uint8).reshape(-1, 210)
    ql = b[:, 0:128].astype(np.int64)
    qh = b[:, 128:192].astype(np.int64)
    scale = b[:, 192:208].view(np.int8).astype(np.float64)
    d = _fp16(b[:, 208], b[:, 209])
    q = np.empty((b.shape[0], 256), np.int64)
    for h in range(2):
        for g in range(4):
            low = ql[:, 64 * h + 32 * (g % 2): 64 * h + 32 * (g % 2) + 32]
            low = (low & 0xF) if g < 2 else (low >> 4)
            high = (qh[:, 32 * h: 32 * h + 32] >> (2 * g)) & 3
            q[:, 128 * h + 32 * g: 128 * h + 32 * g + 32] = low | (high << 4)
    per16 = np.repeat(scale, 16, axis=1)  # scale i over weights 16i .. 16i+15
    return (d[:, None] * per16 * (q - 32).astype(np.float64)).ravel()


DEQUANT = {"q8_0": dequant_q8_0, "q4_0": dequant_q4_0, "q4_k": dequant_q4_k, "q6_k": dequant_q6_k}


def dequant(raw, fmt):
    return DEQUANT[fmt](raw)


def matrix_bytes(fmt, rows, cols):
    bb, wpb = FORMATS[fmt]
    assert cols % wpb == 0, (fmt, cols)
    return rows * (cols // wpb) * bb


def payload_bytes(qtype, hidden, inter):
    gu, dn = roles(qtype)
    return 2 * matrix_bytes(gu, inter, hidden) + matrix_bytes(dn, hidden, inter)


def dequant_matrix(raw, fmt, rows, cols):
    """[rows, cols] fp64 matrix from its row-major block bytes."""
    return dequant(raw[: matrix_bytes(fmt, rows, cols)], fmt).reshape(rows, cols)


def expert_weights(store, qtype, n_experts, hidden, inter, layer, expert):
    """(W_gate [inter,hidden], W_up [inter,hidden], W_down [hidden,inter]) in fp64."""
    gu, dn = roles(qtype)
    P = payload_bytes(qtype, hidden, inter)
    m = matrix_bytes(gu, inter, hidden)
    off = (layer * n_experts + expert) * P
    blob = np.asarray(store[off: off + P], dtype=np.uint8)
    wg = dequant_matrix(blob[0:m], gu, inter, hidden)
    wu = dequant_matrix(blob[m:2 * m], gu, inter, hidden)
    wd = dequant_matrix(blob[2 * m:P], dn, hidden, inter)
    return wg, wu, wd
