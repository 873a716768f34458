"""Split-pack of GGUF MoE models: the oracle's GGUF reader pinned to a hand-assembled file;
the library's packer (moe_pack_gguf) against the oracle on synthetic models -- pack bytes
identical, index records and digests, routers transposed to [hidden][n_experts] fp32;
malformed and unsupported files rejected."""
import json
import os
import struct

import numpy as np
import pytest

import gguf_writer
from conftest import golden_path
from oracle import gguf


@pytest.fixture(scope="module")
def mc():
    from paper_2607_09686_amd import build, moecache
    if not os.path.exists(moecache.LIB_PATH):
        build.build()
    moecache.lib()
    return moecache


def hand_file(tmp_path):
    raw = bytearray()
    for line in open(golden_path("tiny_gguf.txt")):
        line = line.split("#", 1)[0].split()
        raw += bytes(int(b, 16) for b in line)
    p = tmp_path / "hand.gguf"
    p.write_bytes(bytes(raw))
    return p, raw


def test_reader_on_hand_assembled_file(tmp_path):
    p, raw = hand_file(tmp_path)
    assert len(raw) == 112
    meta, tensors, _ = gguf.read(p)
    assert meta == {"general.alignment": 32}
    assert tensors == {"t": ([4], 0, 96, 16)}
    assert np.frombuffer(raw[96:112], "<f4").tolist() == [1.0, 2.0, 3.0, 4.0]


def test_fnv1a_reference_values():
    # published FNV-1a 64-bit test vectors: "" and "a"
    assert gguf.fnv1a64(b"") == 0xcbf29ce484222325
    assert gguf.fnv1a64(b"a") == 0xaf63dc4c8601ec8c
    assert gguf.fnv1a64(b"foobar") == 0x85944171f73967e8


@pytest.mark.parametrize("qcode,router_type,alignment", [(8, 0, 32), (2, 1, 64), (8, 30, 128),
                                                        (12, 0, 32), (14, 1, 32),
                                                        (12 | 14 << 8, 30, 64)])
def test_pack_matches_oracle(mc, tmp_path, qcode, router_type, alignment):
    src = tmp_path / "m.gguf"
    gguf_writer.moe_model(src, n_layers=3, n_experts=8, hidden=256,
                          inter=128 if qcode in (8, 2) else 256, qcode=qcode,
                          top_k=2, seed=qcode + router_type, router_type=router_type,
                          alignment=alignment)
    info = mc.pack_gguf(src, tmp_path / "e.pack", tmp_path / "e.index", tmp_path / "r.bin")
    want, routers, topo = gguf.expected_pack(src)
    got = np.fromfile(tmp_path / "e.pack", np.uint8)
    assert np.array_equal(got, want)
    assert info["pack_bytes"] == want.size
    for k in ("n_layers", "n_experts", "hidden", "inter", "top_k", "payload_bytes"):
        assert info[k] == topo[k], k
    assert info["qtype"] == qcode
    r = np.fromfile(tmp_path / "r.bin", np.float32).reshape(routers.shape)
    assert np.array_equal(r, routers)
    lines = [json.loads(x) for x in open(tmp_path / "e.index")]
    head, blocks, tail = lines[0], lines[1:-1], lines[-1]
    assert head["n_layers"] == 3 and head["n_experts"] == 8 and head["payload_bytes"] == topo["payload_bytes"]
    assert len(blocks) == 24 and tail["blocks"] == 24 and tail["pack_bytes"] == want.size
    digests = b"".join(struct.pack("<Q", int(b["fnv1a64"], 16)) for b in blocks)
    assert int(tail["fnv1a64_of_digests"], 16) == gguf.fnv1a64(digests)
    P = topo["payload_bytes"]
    _, tensors, buf = gguf.read(src)
    for i, b in enumerate(blocks):
        assert (b["layer"], b["expert"], b["offset"], b["bytes"]) == (i // 8, i % 8, i * P, P)
        assert int(b["fnv1a64"], 16) == gguf.fnv1a64(want[i * P:(i + 1) * P].tobytes())
        m_gu = tensors["blk.0.ffn_gate_exps.weight"][3] // 8
        for kind, start in (("gate", 0), ("up", m_gu), ("down", 2 * m_gu)):
            off, nb = b[kind]
            assert nb == (m_gu if kind != "down" else P - 2 * m_gu)
            assert bytes(buf[off:off + nb]) == want[i * P + start:i * P + start + nb].tobytes()
            _, _, toff, tnb = tensors[f"blk.{b['layer']}.ffn_{kind}_exps.weight"]
            assert toff + b["expert"] * nb == off


def test_rejects_bad_files(mc, tmp_path):
    p, _ = hand_file(tmp_path)
    with pytest.raises(mc.MoeError) as e:          # a GGUF file without routed experts
        mc.pack_gguf(p, tmp_path / "x.pack", tmp_path / "x.index")
    assert e.value.code == mc.MOE_EINVAL
    bad = tmp_path / "bad.gguf"
    bad.write_bytes(b"GGML" + bytes(100))
    with pytest.raises(mc.MoeError) as e:
        mc.pack_gguf(bad, tmp_path / "x.pack", tmp_path / "x.index")
    assert e.value.code == mc.MOE_EINVAL
    with pytest.raises(mc.MoeError) as e:
        mc.pack_gguf(tmp_path / "missing.gguf", tmp_path / "x.pack", tmp_path / "x.index")
    assert e.value.code == mc.MOE_EIO
    # expert tensors of a block type the kernels do not read (Q4_1 = 3)
    src = tmp_path / "q41.gguf"
    rng = np.random.default_rng(0)
    gguf_writer.write(src, [], [("blk.0.ffn_gate_exps.weight", [64, 64, 2], 3, rng.bytes(64 * 64 * 2 // 32 * 20))])
    with pytest.raises(mc.MoeError) as e:
        mc.pack_gguf(src, tmp_path / "x.pack", tmp_path / "x.index")
    assert e.value.code == mc.MOE_EINVAL and "type 3" in str(e.value)
    # a layer whose down tensor has the wrong shape
    src = tmp_path / "shape.gguf"
    gguf_writer.moe_model(src, 2, 4, 64, 64, 8, 2, 1)
    _, tensors, buf = gguf.read(src)
    items = []
    for name, (dims, t, off, nb) in tensors.items():
        if name == "blk.1.ffn_down_exps.weight":
            dims = [dims[0], dims[1], 3]
            nb = nb // 4 * 3
        items.append((name, dims, t, bytes(buf[off:off + nb])))
    gguf_writer.write(src, [], items)
    with pytest.raises(mc.MoeError) as e:
        mc.pack_gguf(src, tmp_path / "x.pack", tmp_path / "x.index")
    assert e.value.code == mc.MOE_EINVAL and "blk.1.ffn_down_exps" in str(e.value)


def test_rejects_types_that_change_between_layers(mc, tmp_path):
    """Every slot holds P bytes, so the down matrices must share one block type in all
    layers (a file mixing Q6_K and Q4_K down tensors is refused)."""
    src = tmp_path / "mixed_layers.gguf"
    gguf_writer.moe_model(src, 2, 4, 256, 256, 12 | 14 << 8, 2, 1)
    _, tensors, buf = gguf.read(src)
    items = []
    rng = np.random.default_rng(2)
    for name, (dims, t, off, nb) in tensors.items():
        raw = bytes(buf[off:off + nb])
        if name == "blk.1.ffn_down_exps.weight":
            import synth
            t = 12
            raw = synth.encode_blocks(12, (rng.normal(size=int(np.prod(dims))) * 0.02)
                                      .astype(np.float32)).tobytes()
        items.append((name, dims, t, raw))
    gguf_writer.write(src, [], items)
    with pytest.raises(mc.MoeError) as e:
        mc.pack_gguf(src, tmp_path / "x.pack", tmp_path / "x.index")
    assert e.value.code == mc.MOE_EINVAL and "blk.1.ffn_down_exps" in str(e.value)


@pytest.mark.skipif(__import__("shutil").which("g++") is None, reason="g++ not available")
def test_packer_under_sanitizers_on_damaged_files(tmp_path):
    """The GGUF reader and packer built with AddressSanitizer + UndefinedBehaviorSanitizer
    (g++, host code only) on truncated, bit-flipped and field-overwritten copies of valid
    files: every call returns a code of the interface, nothing faults or overflows."""
    import subprocess
    from conftest import ROOT
    seeds = []
    for i, (qcode, inter) in enumerate(((8, 128), (12 | 14 << 8, 256))):
        p = tmp_path / f"seed{i}.gguf"
        gguf_writer.moe_model(p, 2, 4, 256, inter, qcode, 2, i, router_type=i)
        seeds.append(str(p))
    exe = tmp_path / "pack_fuzz"
    cmd = ["g++", "-std=c++17", "-O1", "-g", "-fsanitize=address,undefined",
           "-fno-sanitize-recover=all", os.path.join(ROOT, "tests", "pack_fuzz.cpp"),
           os.path.join(ROOT, "paper_2607_09686_amd", "csrc", "pack.cpp"), "-o", str(exe)]
    subprocess.run(cmd, check=True)
    r = subprocess.run([str(exe), str(tmp_path), *seeds], capture_output=True, text=True,
                       timeout=600)
    assert r.returncode == 0, r.stdout[-2000:] + r.stderr[-4000:]
    assert r.stdout.startswith("ok"), r.stdout
