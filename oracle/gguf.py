"""GGUF reader and the expected split-pack of a GGUF MoE model (oracle; test infrastructure only).

The paper's Split-Pack Representation section: routed expert tensors are cut, in a
fixed order, into one block per layer and expert.  Here the expected pack is built by the
plainest route: read the whole file, find each expert's three matrices as slices of the
layer's three expert tensors, and concatenate them per (layer, expert).

GGUF as read here (versions 2 and 3): little-endian; magic b"GGUF"; u32 version; u64
tensor count; u64 metadata count; each metadata entry a string key (u64 length +
bytes), a u32 value type and the value (scalars; strings; arrays as u32 element type,
u64 count, elements); each tensor info a string name, u32 dim count, u64 dims
(innermost first), u32 ggml type, u64 offset into the data section; the data section
starts at the next multiple of general.alignment (default 32).
"""
import struct

import numpy as np

SCALAR = {0: "<B", 1: "<b", 2: "<H", 3: "<h", 4: "<I", 5: "<i", 6: "<f", 7: "<?", 10: "<Q",
          11: "<q", 12: "<d"}
# (bytes, elements) per block of the block types (ggml type codes: Q8_0 8, Q4_0 2, Q4_K 12,
# Q6_K 14); bytes per element of the float types
BLOCK = {8: (34, 32), 2: (18, 32), 12: (144, 256), 14: (210, 256)}
ELEM = {0: 4, 1: 2, 30: 2}
# the pack's qtype code for a (gate/up type, down type) pair: the type alone when both
# matrices share it, else gate/up | down << 8


class _Cursor:
    def __init__(self, buf):
        self.buf, self.pos = buf, 0

    def take(self, fmt):
        v = struct.unpack_from(fmt, self.buf, self.pos)[0]
        self.pos += struct.calcsize(fmt)
        return v

    def string(self):
        n = self.take("<Q")
        s = self.buf[self.pos:self.pos + n].decode("utf-8")
        self.pos += n
        return s

    def value(self, t):
        if t == 8:
            return self.string()
        if t == 9:
            et, n = self.take("<I"), self.take("<Q")
            return [self.value(et) for _ in range(n)]
        return self.take(SCALAR[t])


def tensor_bytes(dims, ggml_type):
    n = int(np.prod(dims, dtype=np.int64))
    if ggml_type in BLOCK:
        bb, wpb = BLOCK[ggml_type]
        return n // wpb * bb
    return n * ELEM[ggml_type]


def read(path):
    """(metadata dict, {name: (dims, type, absolute offset, bytes)}, whole file as bytes)."""
    buf = open(path, "rb").read()
    c = _Cursor(buf)
    if buf[:4] != b"GGUF":
        raise ValueError("not a GGUF file")
    c.pos = 4
    version = c.take("<I")
    if version not in (2, 3):
        raise ValueError("unsupported version")
    n_t, n_kv = c.take("<Q"), c.take("<Q")
    meta = {}
    for _ in range(n_kv):
        k = c.string()
        meta[k] = c.value(c.take("<I"))
    infos = []
    for _ in range(n_t):
        name = c.string()
        nd = c.take("<I")
        dims = [c.take("<Q") for _ in range(nd)]
        infos.append((name, dims, c.take("<I"), c.take("<Q")))
    align = meta.get("general.alignment", 32)
    data0 = (c.pos + align - 1) // align * align
    tensors = {n: (d, t, data0 + o, tensor_bytes(d, t)) for n, d, t, o in infos}
    return meta, tensors, buf


def _f32(raw, ggml_type):
    if ggml_type == 0:
        return np.frombuffer(raw, "<f4").astype(np.float32)
    if ggml_type == 1:
        return np.frombuffer(raw, "<f2").astype(np.float32)
    b = np.frombuffer(raw, "<u2").astype(np.uint32) << 16   # bf16: the high half of an fp32
    return b.view(np.float32)


def expected_pack(path):
    """(pack bytes uint8 [L*E*P], routers fp32 [L, H, E], topology dict)."""
    meta, tensors, buf = read(path)
    L = 0
    while f"blk.{L}.ffn_gate_exps.weight" in tensors:
        L += 1
    (H, I, E), qt, _, _ = tensors["blk.0.ffn_gate_exps.weight"]
    qd = tensors["blk.0.ffn_down_exps.weight"][1]
    M = tensor_bytes([H, I], qt)       # one expert's gate (or up) matrix
    Md = tensor_bytes([I, H], qd)      # one expert's down matrix
    blocks, routers = [], np.empty((L, H, E), np.float32)
    for l in range(L):
        mats = []
        for kind, want_t, m in (("gate", qt, M), ("up", qt, M), ("down", qd, Md)):
            d, t, off, nb = tensors[f"blk.{l}.ffn_{kind}_exps.weight"]
            assert t == want_t and nb == E * m
            mats.append(np.frombuffer(buf, np.uint8, count=nb, offset=off).reshape(E, m))
        for e in range(E):
            blocks.append(np.concatenate([mats[0][e], mats[1][e], mats[2][e]]))
        d, t, off, nb = tensors[f"blk.{l}.ffn_gate_inp.weight"]
        w = _f32(buf[off:off + nb], t).reshape(E, H)   # E rows of H
        routers[l] = w.T
    used = [v for k, v in meta.items() if k.endswith(".expert_used_count")]
    topo = {"n_layers": L, "n_experts": E, "hidden": H, "inter": I,
            "qtype": qt if qd == qt else qt | (qd << 8),
            "top_k": used[0] if used else 0, "payload_bytes": 2 * M + Md}
    return np.concatenate(blocks), routers, topo


def fnv1a64(data):
    """FNV-1a, 64 bits (Fowler, Noll, Vo), of a byte string."""
    h = 0xcbf29ce484222325
    for b in bytes(data):
        h = ((h ^ b) * 0x100000001b3) & 0xFFFFFFFFFFFFFFFF
    return h
