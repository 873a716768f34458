"""Writes small GGUF files for the split-pack tests (layout as the oracle's reader describes)."""
import struct

import numpy as np


def _str(s):
    b = s.encode("utf-8")
    return struct.pack("<Q", len(b)) + b


def _value(t, v):
    if t == 8:
        return _str(v)
    if t == 9:
        et, items = v
        return struct.pack("<IQ", et, len(items)) + b"".join(_value(et, x) for x in items)
    fmt = {0: "<B", 1: "<b", 2: "<H", 3: "<h", 4: "<I", 5: "<i", 6: "<f", 7: "<?", 10: "<Q",
           11: "<q", 12: "<d"}[t]
    return struct.pack(fmt, v)


def write(path, metadata, tensors, alignment=32, version=3):
    """metadata: list of (key, type, value); tensors: list of (name, dims, ggml_type, raw bytes)."""
    meta = list(metadata)
    if alignment != 32:
        meta.append(("general.alignment", 4, alignment))
    head = b"GGUF" + struct.pack("<IQQ", version, len(tensors), len(meta))
    head += b"".join(_str(k) + struct.pack("<I", t) + _value(t, v) for k, t, v in meta)
    offs, off = [], 0
    for _, _, _, raw in tensors:
        offs.append(off)
        off = (off + len(raw) + alignment - 1) // alignment * alignment
    for (name, dims, t, _), o in zip(tensors, offs):
        head += _str(name) + struct.pack("<I", len(dims)) + b"".join(struct.pack("<Q", d) for d in dims)
        head += struct.pack("<IQ", t, o)
    data0 = (len(head) + alignment - 1) // alignment * alignment
    out = bytearray(head + b"\0" * (data0 - len(head)))
    for (_, _, _, raw), o in zip(tensors, offs):
        out += b"\0" * (data0 + o - len(out))
        out += raw
    open(path, "wb").write(bytes(out))


def moe_model(path, n_layers, n_experts, hidden, inter, qcode, top_k, seed, router_type=0,
              alignment=32):
    """A GGUF MoE model with random expert blocks (by synth's encoders), routers of the given
    float type, and a few other tensors and metadata entries around them.  qcode: the block
    type of every expert tensor (8 Q8_0, 2 Q4_0, 12 Q4_K, 14 Q6_K), or gate/up | down << 8."""
    import synth
    rng = np.random.default_rng(seed)
    meta = [("general.architecture", 8, "testmoe"), ("general.name", 8, "tiny test moe"),
            ("testmoe.block_count", 4, n_layers), ("testmoe.expert_count", 4, n_experts),
            ("testmoe.expert_used_count", 4, top_k), ("testmoe.rope.freq_base", 6, 10000.0),
            ("tokenizer.ggml.tokens", 9, (8, ["<s>", "</s>", "a", "b"])),
            ("tokenizer.ggml.scores", 9, (6, [0.0, -1.0, -2.0, -3.0])),
            ("testmoe.flag", 7, True), ("testmoe.neg", 5, -3), ("testmoe.big", 10, 1 << 40)]
    tensors = [("token_embd.weight", [hidden, 4], 0,
                rng.normal(size=4 * hidden).astype("<f4").tobytes())]
    for l in range(n_layers):
        tensors.append((f"blk.{l}.attn_norm.weight", [hidden], 0,
                        rng.normal(size=hidden).astype("<f4").tobytes()))
        gu, dn = qcode & 0xFF, (qcode >> 8) or (qcode & 0xFF)
        for kind, dims, code in (("gate", [hidden, inter, n_experts], gu),
                                 ("up", [hidden, inter, n_experts], gu),
                                 ("down", [inter, hidden, n_experts], dn)):
            w = (rng.normal(size=int(np.prod(dims))) * 0.02).astype(np.float32)
            tensors.append((f"blk.{l}.ffn_{kind}_exps.weight", dims, code,
                            synth.encode_blocks(code, w).tobytes()))
        r = rng.normal(size=n_experts * hidden) * 0.1
        raw = {0: r.astype("<f4").tobytes(), 1: r.astype("<f2").tobytes(),
               30: (r.astype(np.float32).view(np.uint32) >> 16).astype("<u2").tobytes()}[router_type]
        tensors.append((f"blk.{l}.ffn_gate_inp.weight", [hidden, n_experts], router_type, raw))
    tensors.append(("output_norm.weight", [hidden], 0, np.ones(hidden, "<f4").tobytes()))
    write(path, meta, tensors, alignment=alignment)
