"""GGUF-style block formats and the expert payload layout (oracle; test infrastructure only).

Block formats (GGUF, the llama.cpp model format the paper serves from; the
paper names the types through its Q8_0 model profiles; Q4_0 stands in here
for its 4-bit profile):

* Q8_0, 34 bytes per 32 weights: bytes 0-1 scale d (binary16, little-endian),
  bytes 2-33 signed 8-bit q_j.  Weight j is d * q_j.
* Q4_0, 18 bytes per 32 weights: bytes 0-1 scale d; byte 2+j (j < 16) holds
  n_j in its low nibble and n_{j+16} in its high nibble.  Weight is d*(n-8).

Expert payload (the paper's Split-Pack section: one block per layer and expert;
its Native Serving Path section: separate gate, up and down tensors): one
contiguous byte range per (layer l, expert e) at offset (l*E + e)*P, laid out
as [W_gate (inter x hidden) | W_up (inter x hidden) | W_down (hidden x inter)].
Each matrix is row-major, one row per output; a row is its inputs split into
consecutive 32-wide blocks.
"""
import numpy as np

from .numerics import fp16_decode

BLOCK_BYTES = {"q8_0": 34, "q4_0": 18}


def dequant_q8_0(raw):
    """fp64 weights of consecutive Q8_0 blocks (raw: uint8 bytes, multiple of 34)."""
    b = np.frombuffer(np.ascontiguousarray(raw, dtype=np.uint8), dtype=np.uint8).reshape(-1, 34)
    d = fp16_decode(b[:, 0].astype(np.uint16) | (b[:, 1].astype(np.uint16) << 8))
    q = b[:, 2:].view(np.int8).astype(np.float64)
    return (np.asarray(d)[:, None] * q).ravel()


def dequant_q4_0(raw):
    """fp64 weights of consecutive Q4_0 blocks (raw: uint8 bytes, multiple of 18)."""
    b = np.frombuffer(np.ascontiguousarray(raw, dtype=np.uint8), dtype=np.uint8).reshape(-1, 18)
    d = fp16_decode(b[:, 0].astype(np.uint16) | (b[:, 1].astype(np.uint16) << 8))
    packed = b[:, 2:].astype(np.int64)
    n = np.concatenate([packed & 0xF, packed >> 4], axis=1)  # elements 0..15, then 16..31
    return (np.asarray(d)[:, None] * (n - 8).astype(np.float64)).ravel()


def dequant(raw, qtype):
    return dequant_q8_0(raw) if qtype == "q8_0" else dequant_q4_0(raw)


def matrix_bytes(qtype, rows, cols):
    assert cols % 32 == 0
    return rows * (cols // 32) * BLOCK_BYTES[qtype]


def payload_bytes(qtype, hidden, inter):
    return 2 * matrix_bytes(qtype, inter, hidden) + matrix_bytes(qtype, hidden, inter)


def dequant_matrix(raw, qtype, rows, cols):
    """[rows, cols] fp64 matrix from its row-major block bytes."""
    return dequant(raw[: matrix_bytes(qtype, rows, cols)], qtype).reshape(rows, cols)


def expert_weights(store, qtype, n_experts, hidden, inter, layer, expert):
    """(W_gate [inter,hidden], W_up [inter,hidden], W_down [hidden,inter]) in fp64."""
    P = payload_bytes(qtype, hidden, inter)
    m = matrix_bytes(qtype, inter, hidden)
    off = (layer * n_experts + expert) * P
    blob = np.asarray(store[off: off + P], dtype=np.uint8)
    wg = dequant_matrix(blob[0:m], qtype, inter, hidden)
    wu = dequant_matrix(blob[m:2 * m], qtype, inter, hidden)
    wd = dequant_matrix(blob[2 * m:3 * m], qtype, hidden, inter)
    return wg, wu, wd
