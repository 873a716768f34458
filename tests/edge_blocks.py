"""Expert stores whose blocks exercise the corners of the Q8_0 / Q4_0 formats (test input
generation only: nothing here decodes a block or computes anything of the method).

The seeded generator's encoders only produce positive, normal fp16 scales, |q| <= 127 and
Q4_0 nibbles chosen by a symmetric quantiser.  A real GGUF file holds more: negative scales
(the usual Q4_0 quantiser divides the signed extreme by -8, so nibble 0 carries the largest
magnitude), subnormal and zero scales, the Q8_0 byte 0x80 (-128) and both Q4_0 nibble
extremes.  ``edge_store`` rewrites a generated store in place under one of three regimes:

* ``mixed``: block by block, a seeded choice among: unchanged; scale sign flipped;
  scale +-0; extremes written into the quantised bytes (Q8_0 -128 / +127, Q4_0 nibbles 0 /
  15); the quantised bytes of a hand-worked block from ``tests/golden/quant_hand_blocks.txt``
  under the block's own scale; a Q4_0 block re-encoded from fresh weights with the scale
  taken as the signed extreme over -8 (so the scale's sign follows the data);
* ``subnormal``: every scale replaced by a random subnormal binary16 pattern of random sign
  (0x0001-0x03ff, or with 0x8000 set), so that outputs are dominated by subnormal scales;
* ``golden``: every block replaced by a hand-worked block of its type, scale included.

Hidden-state rows with edge values: ``edge_tokens`` sets one row to all zeros and one to
values whose magnitudes span 1e-6 .. 1e3 inside every 32-wide block.
"""
import numpy as np

from conftest import golden_path

REGIMES = ("mixed", "subnormal", "golden")


def golden_blocks(kind):
    """Raw bytes of the hand-worked blocks of one type ("q8" or "q4"), in file order."""
    out = []
    for line in open(golden_path("quant_hand_blocks.txt")):
        line = line.split("#")[0].strip()
        if not line:
            continue
        lhs = line.split("=>")[0].split()
        if lhs[0] != kind:
            continue
        s = int(lhs[1], 16)
        head = bytes([s & 0xFF, s >> 8])
        body = bytes(int(v) & 0xFF for v in lhs[2:]) if kind == "q8" else \
            bytes(int(v, 16) for v in lhs[2:])
        out.append(np.frombuffer(head + body, np.uint8))
    return out


def _signed_max_q4(rng, n):
    """n Q4_0 blocks encoded from fresh N(0, 0.02) weights with d = (signed extreme) / -8."""
    w = rng.normal(0.0, 0.02, size=(n, 32))
    ext = w[np.arange(n), np.argmax(np.abs(w), axis=1)]
    d16 = (ext / -8.0).astype(np.float16)
    d = d16.astype(np.float64)
    with np.errstate(divide="ignore", invalid="ignore"):
        q = np.where(d[:, None] != 0, np.rint(w / d[:, None]) + 8, 8)
    nib = np.clip(q, 0, 15).astype(np.uint8)
    out = np.empty((n, 18), np.uint8)
    out[:, 0:2] = d16.view(np.uint8).reshape(n, 2)
    out[:, 2:] = nib[:, :16] | (nib[:, 16:] << 4)
    return out


def edge_store(arr, wl, regime, seed=0):
    """Rewrite the store bytes ``arr`` (flat uint8, the whole store of workload ``wl``)."""
    bb = wl.block_bytes
    kind = "q8" if wl.qtype == "q8_0" else "q4"
    blocks = arr.reshape(-1, bb)
    n = blocks.shape[0]
    rng = np.random.default_rng(1000 + 17 * seed + REGIMES.index(regime))
    gold = golden_blocks(kind)
    if regime == "subnormal":
        bits = rng.integers(1, 0x400, size=n, dtype=np.uint16)
        bits |= (rng.integers(0, 2, size=n, dtype=np.uint16) << 15)
        blocks[:, 0] = bits & 0xFF
        blocks[:, 1] = bits >> 8
        return arr
    if regime == "golden":
        pick = rng.integers(0, len(gold), size=n)
        for g, raw in enumerate(gold):
            blocks[pick == g] = raw
        return arr
    assert regime == "mixed"
    cat = rng.choice(6, size=n, p=[0.40, 0.15, 0.05, 0.15, 0.15, 0.10])
    # 1: scale sign flipped
    blocks[cat == 1, 1] ^= 0x80
    # 2: +0 or -0 scale
    z = np.nonzero(cat == 2)[0]
    blocks[z, 0] = 0
    blocks[z, 1] = np.where(rng.integers(0, 2, size=z.size) == 1, 0x80, 0).astype(np.uint8)
    # 3: extremes in the quantised bytes
    x = np.nonzero(cat == 3)[0]
    if kind == "q8":
        vals = np.where(rng.integers(0, 2, size=(x.size, 32)) == 1, 0x80, 0x7F).astype(np.uint8)
        keep = rng.integers(0, 2, size=(x.size, 32)) == 1
        blocks[x, 2:] = np.where(keep, blocks[x, 2:], vals)
    else:
        lo = np.where(rng.integers(0, 2, size=(x.size, 16)) == 1, 0x0, 0xF).astype(np.uint8)
        hi = np.where(rng.integers(0, 2, size=(x.size, 16)) == 1, 0x0, 0xF).astype(np.uint8)
        blocks[x, 2:] = lo | (hi << 4)
    # 4: a hand-worked block's quantised bytes under the block's own scale
    h = np.nonzero(cat == 4)[0]
    pick = rng.integers(0, len(gold), size=h.size)
    for g, raw in enumerate(gold):
        blocks[h[pick == g], 2:] = raw[2:]
    # 5: Q4_0 signed-extreme encoding (Q8_0: scale sign flipped and extremes together)
    s = np.nonzero(cat == 5)[0]
    if kind == "q4":
        blocks[s] = _signed_max_q4(rng, s.size)
    else:
        blocks[s, 1] ^= 0x80
        blocks[s, 2] = 0x80
        blocks[s, 33] = 0x7F
    return arr


def edge_tokens(X, zero_row=1, wide_row=3, seed=0):
    """X with one all-zero row and one row spanning magnitudes 1e-6 .. 1e3 (random signs)."""
    X = np.array(X, np.float32, copy=True)
    rng = np.random.default_rng(77 + seed)
    if zero_row is not None and zero_row < X.shape[0]:
        X[zero_row] = 0.0
    if wide_row is not None and wide_row < X.shape[0]:
        H = X.shape[1]
        mag = 10.0 ** rng.uniform(-6.0, 3.0, size=H)
        mag[::32] = 1e3          # every 32-wide block holds both ends of the range
        mag[1::32] = 1e-6
        X[wide_row] = (mag * np.where(rng.integers(0, 2, size=H) == 1, 1.0, -1.0)).astype(np.float32)
    return X


def kquant_golden_blocks(kind):
    """Raw bytes of the hand-worked K-quant super-blocks of one format ("q4_k" or "q6_k")."""
    from test_oracle_quant import _kquant_golden
    return [raw for k, raw, _ in _kquant_golden() if k == kind]


def kquant_golden_store(arr, wl, seed=0):
    """Rewrite a K-quant store: every super-block of every matrix replaced by a hand-worked
    super-block of that matrix's format (seeded choice), scales, mins and signs included."""
    rng = np.random.default_rng(500 + seed)
    gu, dn = wl.formats
    P, M = wl.payload_bytes, wl.matrix_bytes
    n_payloads = arr.size // P
    pay = arr.reshape(n_payloads, P)
    for fmt, lo, hi in ((gu, 0, 2 * M), (dn, 2 * M, P)):
        gold = kquant_golden_blocks(fmt)
        sb = len(gold[0])
        view = pay[:, lo:hi].reshape(n_payloads, (hi - lo) // sb, sb)
        pick = rng.integers(0, len(gold), size=view.shape[:2])
        for g, raw in enumerate(gold):
            view[pick == g] = raw
        pay[:, lo:hi] = view.reshape(n_payloads, hi - lo)
    return arr
