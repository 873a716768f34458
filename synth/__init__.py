"""Seeded synthetic inputs shared by the oracle tests and the GPU path.

This package draws random numbers and encodes weights into GGUF-style
blocks; it holds none of the MoE layer's arithmetic (no dequantisation,
routing, caching or FFN).  The work is done by ``libsynth.so`` (C, OpenMP),
built from ``synth.c`` by ``build.py``.
"""
import ctypes
import os

import numpy as np

from .configs import WORKLOADS, Workload  # noqa: F401

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB = None


def _lib():
    global _LIB
    if _LIB is None:
        path = os.path.join(_HERE, "libsynth.so")
        if not os.path.exists(path):
            raise RuntimeError(f"{path} is not built; run synth.build.build()")
        lib = ctypes.CDLL(path)
        u64, i32, i64, u32 = ctypes.c_uint64, ctypes.c_int32, ctypes.c_int64, ctypes.c_uint32
        vp = ctypes.c_void_p
        lib.synth_philox4x64.argtypes = [u64] * 6 + [vp]
        lib.synth_philox4x64.restype = None
        lib.synth_normal_f32.argtypes = [u64, u64, u64, u64, ctypes.c_float, vp]
        lib.synth_normal_f32.restype = None
        lib.synth_f32_to_f16.argtypes = [ctypes.c_float]
        lib.synth_f32_to_f16.restype = ctypes.c_uint16
        lib.synth_encode_blocks.argtypes = [i32, vp, i64, vp]
        lib.synth_encode_blocks.restype = None
        lib.synth_key.argtypes = [u32] * 5
        lib.synth_key.restype = u64
        lib.synth_expert_store.argtypes = [i32] * 6 + [ctypes.c_float, u32, vp, i32]
        lib.synth_expert_store.restype = ctypes.c_int
        lib.synth_router.argtypes = [i32] * 4 + [ctypes.c_float, u32, vp]
        lib.synth_router.restype = ctypes.c_int
        lib.synth_hidden.argtypes = [i32, i32, ctypes.c_double, u32, u32, vp]
        lib.synth_hidden.restype = ctypes.c_int
        _LIB = lib
    return _LIB


def philox4x64(counter, key):
    """Philox4x64-10 of a 4-word counter under a 2-word key (4 uint64)."""
    out = (ctypes.c_uint64 * 4)()
    _lib().synth_philox4x64(*[int(c) for c in counter], int(key[0]), int(key[1]), out)
    return [int(v) for v in out]


def key(kind, seed, layer, expert, matrix):
    return int(_lib().synth_key(kind, seed, layer, expert, matrix))


def normal_f32(k0, start, n, sigma=1.0):
    out = np.empty(n, np.float32)
    _lib().synth_normal_f32(k0, 0, start, n, sigma, out.ctypes.data)
    return out


def f32_to_f16_bits(x):
    return int(_lib().synth_f32_to_f16(float(x)))


def encode_blocks(qcode, w):
    """Encode fp32 weights into blocks of format code qcode: Q8_0 (8) / Q4_0 (2), 32 weights
    per block, or Q4_K (12) / Q6_K (14), 256 weights per super-block."""
    from .configs import FORMATS
    bb, wpb = {code: (b, n) for b, n, code in FORMATS.values()}[qcode]
    w = np.ascontiguousarray(w, np.float32).ravel()
    assert w.size % wpb == 0
    out = np.empty(w.size // wpb * bb, np.uint8)
    _lib().synth_encode_blocks(qcode, w.ctypes.data, w.size // wpb, out.ctypes.data)
    return out


def default_threads():
    try:
        return max(1, min(16, len(os.sched_getaffinity(0))))
    except AttributeError:  # pragma: no cover
        return max(1, min(16, os.cpu_count() or 1))


def expert_store(wl: Workload, out=None, layer0=0, n_layers=None, threads=None):
    """Fill (or allocate) the expert store of layers layer0.. as uint8.

    ``out`` may be any writable buffer of the right size (e.g. a numpy view of
    pinned host memory); it is returned as a flat uint8 numpy array.
    """
    n_layers = wl.n_layers - layer0 if n_layers is None else n_layers
    nbytes = n_layers * wl.n_experts * wl.payload_bytes
    if out is None:
        out = np.empty(nbytes, np.uint8)
    arr = np.frombuffer(out, np.uint8) if not isinstance(out, np.ndarray) else out
    assert arr.nbytes >= nbytes and arr.flags.c_contiguous and arr.flags.writeable
    rc = _lib().synth_expert_store(wl.qcode, layer0, n_layers, wl.n_experts, wl.hidden, wl.inter,
                                   wl.weight_sigma, wl.model_seed, arr.ctypes.data,
                                   threads or default_threads())
    if rc != 0:
        raise ValueError("synth_expert_store rejected the workload")
    return arr[:nbytes]


def router(wl: Workload, layer0=0, n_layers=None):
    """Router matrices [n_layers, hidden, n_experts] fp32."""
    n_layers = wl.n_layers - layer0 if n_layers is None else n_layers
    out = np.empty((n_layers, wl.hidden, wl.n_experts), np.float32)
    _lib().synth_router(layer0, n_layers, wl.hidden, wl.n_experts, wl.router_sigma,
                        wl.model_seed, out.ctypes.data)
    return out


def hidden(wl: Workload, rho=None, n_tokens=None):
    """Hidden states [n_tokens, hidden] fp32 (AR(1) drift, or iid when rho < 0)."""
    rho = wl.rho if rho is None else rho
    n_tokens = wl.n_tokens if n_tokens is None else n_tokens
    out = np.empty((n_tokens, wl.hidden), np.float32)
    rc = _lib().synth_hidden(n_tokens, wl.hidden, rho, wl.hidden_seed, wl.hidden_stream(rho),
                             out.ctypes.data)
    if rc != 0:
        raise ValueError("synth_hidden rejected the shape")
    return out


def acceptance(n_steps, horizon, q, seed):
    """Verification outcomes [n_steps, horizon] (bool) of draft tokens: draft j of step s
    passes when u < q, u the uniform in [0, 1) made of the top 53 bits of word j % 4 of
    Philox4x64-10 at counter (s, j // 4, 0, 0) under key(5, seed, 0, 0, 0)."""
    k0 = key(5, seed, 0, 0, 0)
    out = np.zeros((n_steps, horizon), bool)
    for s in range(n_steps):
        for c in range((horizon + 3) // 4):
            words = philox4x64((s, c, 0, 0), (k0, 0))
            for i, wv in enumerate(words):
                j = 4 * c + i
                if j < horizon:
                    out[s, j] = (wv >> 11) * (1.0 / (1 << 53)) < q
    return out
