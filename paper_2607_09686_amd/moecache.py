"""ctypes binding of libmoecache (include/moecache.h): argument marshalling only.

Every step of a layer call (routing, the slot table, the copies, the FFN)
runs inside the library; this module converts torch tensors and numpy arrays
to pointers and raises on non-zero status codes.  PyTorch provides device
memory and streams.  There is no fallback: if the library is missing or
cannot be loaded, every entry point raises.
"""
import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
# MOECACHE_LIB: an alternative build of the library to load instead of the in-tree one
LIB_PATH = os.environ.get("MOECACHE_LIB") or os.path.join(_HERE, "libmoecache.so")

MOE_OK, MOE_EINVAL, MOE_ENOMEM, MOE_EHIP, MOE_ESTATE, MOE_EIO = 0, -1, -2, -3, -4, -5
MOE_Q8_0, MOE_Q4_0 = 8, 2
MOE_F_RESIDUAL, MOE_F_TRACE, MOE_F_TIMING, MOE_F_PRENORM = 1, 2, 4, 8
MOE_F_SIDE_COPY, MOE_F_SDMA_COPY, MOE_F_SPLIT_COPY, MOE_F_SCORE_EVICT = 16, 32, 64, 128
COPY_MODES = {"kernel": 0, "split": MOE_F_SPLIT_COPY, "side": MOE_F_SIDE_COPY, "sdma": MOE_F_SDMA_COPY}
KIND_ROUTER, KIND_GATEUP, KIND_DOWN, KIND_COPY = 0, 1, 2, 3
KIND_NAMES = {KIND_ROUTER: "router", KIND_GATEUP: "gateup", KIND_DOWN: "down", KIND_COPY: "copy"}
MOE_Q4_K, MOE_Q6_K = 12, 14
# model type: the gate/up format's code, the down format's in the next byte when it differs
QTYPES = {"q8_0": MOE_Q8_0, "q4_0": MOE_Q4_0, "q4_k": MOE_Q4_K, "q6_k": MOE_Q6_K,
          "q4_k_m": MOE_Q4_K | (MOE_Q6_K << 8)}


class MoeError(RuntimeError):
    def __init__(self, code, msg):
        super().__init__(f"moecache error {code}: {msg}")
        self.code = code


class ModelDesc(ctypes.Structure):
    _fields_ = [("n_layers", ctypes.c_int32), ("n_experts", ctypes.c_int32),
                ("top_k", ctypes.c_int32), ("hidden", ctypes.c_int32), ("inter", ctypes.c_int32),
                ("qtype", ctypes.c_int32), ("host_store", ctypes.c_void_p),
                ("store_bytes", ctypes.c_uint64), ("hip_stream", ctypes.c_void_p),
                ("flags", ctypes.c_uint32)]


class Counters(ctypes.Structure):
    _fields_ = [("hits", ctypes.c_uint64), ("misses", ctypes.c_uint64),
                ("evictions", ctypes.c_uint64), ("materialized_bytes", ctypes.c_uint64)]

    def as_tuple(self):
        return (self.hits, self.misses, self.evictions, self.materialized_bytes)

    def __repr__(self):
        return "Counters(hits=%d, misses=%d, evictions=%d, materialized_bytes=%d)" % self.as_tuple()


class StepRec(ctypes.Structure):
    _fields_ = [("layer", ctypes.c_int32), ("step", ctypes.c_int32), ("expert", ctypes.c_int32),
                ("hit", ctypes.c_int32), ("slot", ctypes.c_int32), ("evicted", ctypes.c_int32)]


class KernelStats(ctypes.Structure):
    _fields_ = [("launches", ctypes.c_uint64), ("total_ms", ctypes.c_double),
                ("bytes", ctypes.c_uint64), ("flops", ctypes.c_uint64)]


class PlanIn(ctypes.Structure):
    _fields_ = [("n_layers", ctypes.c_int32), ("n_experts", ctypes.c_int32),
                ("top_k", ctypes.c_int32), ("pad", ctypes.c_int32),
                ("payload_bytes", ctypes.c_uint64), ("common_bytes", ctypes.c_uint64),
                ("kv_bytes_per_token", ctypes.c_uint64), ("overhead_bytes", ctypes.c_uint64),
                ("target_bytes", ctypes.c_uint64)]


class PlanOut(ctypes.Structure):
    _fields_ = [("slots_per_layer", ctypes.c_int32), ("clamped", ctypes.c_int32),
                ("expert_cache_bytes", ctypes.c_uint64), ("kv_bytes", ctypes.c_uint64),
                ("lower_bound_bytes", ctypes.c_uint64), ("footprint_bytes", ctypes.c_uint64),
                ("feasible", ctypes.c_int32), ("pad", ctypes.c_int32)]

    def as_dict(self):
        return {f: getattr(self, f) for f, _ in self._fields_ if f != "pad"}


class PackInfo(ctypes.Structure):
    _fields_ = [("n_layers", ctypes.c_int32), ("n_experts", ctypes.c_int32),
                ("top_k", ctypes.c_int32), ("hidden", ctypes.c_int32), ("inter", ctypes.c_int32),
                ("qtype", ctypes.c_int32), ("payload_bytes", ctypes.c_uint64),
                ("pack_bytes", ctypes.c_uint64)]


_lib = None


def _check_one_hip_runtime():
    """Raise if more than one copy of the HIP runtime is mapped in this process."""
    try:
        with open("/proc/self/maps") as f:
            paths = {ln.split()[-1] for ln in f if "libamdhip64.so" in ln}
    except OSError:
        return
    real = {os.path.realpath(p) for p in paths}
    if len(real) > 1:
        raise RuntimeError("two HIP runtimes are loaded (%s); import torch before the "
                           "library is first loaded" % ", ".join(sorted(real)))


def lib():
    """Load libmoecache.so (raises if it is not built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is not built; run paper_2607_09686_amd.build.build()")
    # torch ships its own HIP runtime (soname libamdhip64.so.7).  Loading torch
    # first makes the library bind to that same runtime, so device pointers and
    # streams from torch are valid in it; loaded the other way round, the process
    # would hold two HIP runtimes and torch's would fail to see the GPU.
    import torch  # noqa: F401
    L = ctypes.CDLL(LIB_PATH)
    _check_one_hip_runtime()
    vp, i32, i64, u64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_uint64
    P = ctypes.POINTER
    sig = {
        "moe_cache_create": ([P(ModelDesc), i32, P(vp)], ctypes.c_int),
        "moe_layer_forward": ([vp, vp, i32, vp, i32, vp, P(Counters)], ctypes.c_int),
        "moe_layer_forward_dbg": ([vp, vp, i32, vp, i32, vp, P(Counters), vp, vp], ctypes.c_int),
        "moe_layer_forward_static": ([vp, vp, i32, vp, i32, vp, P(Counters)], ctypes.c_int),
        "moe_cache_counters": ([vp, i32, P(Counters)], ctypes.c_int),
        "moe_cache_read_trace": ([vp, P(StepRec), i64, P(i64)], ctypes.c_int),
        "moe_cache_reset": ([vp], ctypes.c_int),
        "moe_cache_kernel_stats": ([vp, i32, P(KernelStats)], ctypes.c_int),
        "moe_cache_destroy": ([vp], None),
        "moe_cache_set_timing_stride": ([vp, i32], ctypes.c_int),
        "moe_cache_last_logits": ([vp, vp], ctypes.c_int),
        "moe_cache_fill_slots": ([vp, i32], ctypes.c_int),
        "moe_last_error": ([], ctypes.c_char_p),
        "moe_host_alloc": ([u64, P(vp)], ctypes.c_int),
        "moe_host_free": ([vp], ctypes.c_int),
        "moe_probe_h2d": ([vp, u64, i32, i32, P(ctypes.c_double)], ctypes.c_int),
        "moe_probe_hbm_read": ([u64, i32, P(ctypes.c_double), P(ctypes.c_double)], ctypes.c_int),
        "moe_lru_create": ([i32, i32, u64, i32, P(vp)], ctypes.c_int),
        "moe_lru_step": ([vp, P(i32), i32, P(StepRec), P(i32)], ctypes.c_int),
        "moe_lru_counters": ([vp, P(Counters)], ctypes.c_int),
        "moe_lru_destroy": ([vp], None),
        "moe_plan_percent": ([P(PlanIn), ctypes.c_double, i64, P(PlanOut)], ctypes.c_int),
        "moe_plan_bytes": ([P(PlanIn), u64, i64, P(PlanOut)], ctypes.c_int),
        "moe_policy_min": ([P(i32), P(i64), i64, i32, i32, P(u64)], ctypes.c_int),
        "moe_pack_gguf": ([ctypes.c_char_p] * 4 + [P(PackInfo)], ctypes.c_int),
    }
    for name, (args, res) in sig.items():
        f = getattr(L, name)
        f.argtypes = args
        f.restype = res
    _lib = L
    return L


def _check(rc):
    if rc != MOE_OK:
        msg = lib().moe_last_error()
        raise MoeError(rc, msg.decode() if msg else "")


def _stream_handle(stream):
    if stream is None:
        return None
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream  # torch.cuda.Stream


def _dev_ptr(t, dtype_name, numel, what):
    import torch
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{what} must be a torch tensor")
    if not t.is_cuda:
        raise ValueError(f"{what} must live on the GPU")
    if str(t.dtype) != f"torch.{dtype_name}":
        raise TypeError(f"{what} must be {dtype_name}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{what} must be contiguous")
    if t.numel() != numel:
        raise ValueError(f"{what} has {t.numel()} elements, expected {numel}")
    return t.data_ptr()


class HostBuffer:
    """Pinned host memory from moe_host_alloc, exposed as a numpy uint8 array."""

    def __init__(self, nbytes):
        p = ctypes.c_void_p()
        _check(lib().moe_host_alloc(nbytes, ctypes.byref(p)))
        self.ptr = p.value
        self.nbytes = nbytes
        self.array = np.ctypeslib.as_array((ctypes.c_uint8 * nbytes).from_address(self.ptr))

    def free(self):
        if self.ptr:
            self.array = None
            _check(lib().moe_host_free(self.ptr))
            self.ptr = None

    def __del__(self):
        try:
            self.free()
        except Exception:
            pass


class MoeCache:
    """A per-layer expert-slot cache over an expert store (moe_cache_create)."""

    def __init__(self, n_layers, n_experts, top_k, hidden, inter, qtype, store_ptr, store_bytes,
                 budget_slots, stream=None, residual=False, trace=False, timing=False,
                 prenorm=False, copy_mode="kernel", score_evict=False):
        self.hidden, self.n_experts, self.top_k = hidden, n_experts, top_k
        flags = (MOE_F_RESIDUAL if residual else 0) | (MOE_F_TRACE if trace else 0) | \
                (MOE_F_TIMING if timing else 0) | (MOE_F_PRENORM if prenorm else 0) | \
                COPY_MODES[copy_mode] | (MOE_F_SCORE_EVICT if score_evict else 0)
        q = QTYPES[qtype] if isinstance(qtype, str) else int(qtype)
        self._desc = ModelDesc(n_layers, n_experts, top_k, hidden, inter, q, store_ptr, store_bytes,
                               _stream_handle(stream), flags)
        h = ctypes.c_void_p()
        _check(lib().moe_cache_create(ctypes.byref(self._desc), budget_slots, ctypes.byref(h)))
        self._h = h.value

    @property
    def handle(self):
        if not self._h:
            raise RuntimeError("cache is closed")
        return self._h

    def layer_forward(self, x, router_w, layer, y, n_tokens=None, routes=False, counters=False):
        """y <- MoE layer(x).

        Returns None, or the call's counter delta if counters=True, or
        (delta, idx, w) if routes=True.  Asking for either makes the call wait
        for its own completion; without them a decode call only queues work.
        """
        T = (x.numel() // self.hidden) if n_tokens is None else n_tokens
        xp = _dev_ptr(x, "float32", T * self.hidden, "x")
        wp = _dev_ptr(router_w, "float32", self.hidden * self.n_experts, "router_w")
        yp = _dev_ptr(y, "float32", T * self.hidden, "y")
        delta = Counters()
        if not routes:
            _check(lib().moe_layer_forward(self.handle, xp, T, wp, layer, yp,
                                           ctypes.byref(delta) if counters else None))
            return delta if counters else None
        idx = np.empty((T, self.top_k), np.int32)
        w = np.empty((T, self.top_k), np.float32)
        _check(lib().moe_layer_forward_dbg(self.handle, xp, T, wp, layer, yp, ctypes.byref(delta),
                                           idx.ctypes.data, w.ctypes.data))
        return delta, idx, w

    def layer_forward_static(self, x, router_w, layer, y, counters=False):
        """One-token call through moe_layer_forward_static (scratch in the library's static
        device array, no allocation).  Returns the counter delta if counters=True."""
        xp = _dev_ptr(x, "float32", self.hidden, "x")
        wp = _dev_ptr(router_w, "float32", self.hidden * self.n_experts, "router_w")
        yp = _dev_ptr(y, "float32", self.hidden, "y")
        delta = Counters()
        _check(lib().moe_layer_forward_static(self.handle, xp, 1, wp, layer, yp,
                                              ctypes.byref(delta) if counters else None))
        return delta if counters else None

    def counters(self, layer=-1):
        c = Counters()
        _check(lib().moe_cache_counters(self.handle, layer, ctypes.byref(c)))
        return c

    def read_trace(self, cap=1 << 20):
        out = []
        buf = (StepRec * 65536)()
        n = ctypes.c_int64()
        while len(out) < cap:
            _check(lib().moe_cache_read_trace(self.handle, buf, min(65536, cap - len(out)),
                                              ctypes.byref(n)))
            out.extend((r.layer, r.step, r.expert, r.hit, r.slot, r.evicted) for r in buf[:n.value])
            if n.value == 0:
                break
        return out

    def reset(self):
        _check(lib().moe_cache_reset(self.handle))

    def fill_slots(self, byte):
        """Overwrite every slot byte with `byte` (moe_cache_fill_slots; tests)."""
        _check(lib().moe_cache_fill_slots(self.handle, byte))

    def last_logits(self):
        """Router logits [n_experts] of the last one-token call (moe_cache_last_logits)."""
        z = np.empty(self.n_experts, np.float32)
        _check(lib().moe_cache_last_logits(self.handle, z.ctypes.data))
        return z

    def set_timing_stride(self, every):
        _check(lib().moe_cache_set_timing_stride(self.handle, every))

    def kernel_stats(self, kind):
        s = KernelStats()
        _check(lib().moe_cache_kernel_stats(self.handle, kind, ctypes.byref(s)))
        return s

    def close(self):
        if getattr(self, "_h", None):
            lib().moe_cache_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def probe_hbm_read(nbytes, iters=50):
    """(read_us, empty_us): one plain streaming read of nbytes from HBM per launch, and an empty
    launch, average kernel durations (moe_probe_hbm_read)."""
    r, e = ctypes.c_double(0.0), ctypes.c_double(0.0)
    _check(lib().moe_probe_hbm_read(nbytes, iters, ctypes.byref(r), ctypes.byref(e)))
    return r.value, e.value


def probe_h2d(host_ptr, chunk_bytes, n_chunks, n_streams=1):
    """GB/s of host-to-device copies from pinned memory (moe_probe_h2d)."""
    g = ctypes.c_double()
    _check(lib().moe_probe_h2d(host_ptr, chunk_bytes, n_chunks, n_streams, ctypes.byref(g)))
    return g.value


class SlotTable:
    """The library's LRU slot table alone (moe_lru_*), usable without a GPU."""

    def __init__(self, n_experts, n_slots, payload_bytes, layer=0):
        h = ctypes.c_void_p()
        _check(lib().moe_lru_create(n_experts, n_slots, payload_bytes, layer, ctypes.byref(h)))
        self._h = h.value

    def step(self, ids):
        ids = np.ascontiguousarray(ids, np.int32)
        out = (StepRec * max(1, ids.size))()
        n = ctypes.c_int32()
        _check(lib().moe_lru_step(self._h, ids.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)),
                                  ids.size, out, ctypes.byref(n)))
        return [(r.layer, r.step, r.expert, r.hit, r.slot, r.evicted) for r in out[:n.value]]

    def counters(self):
        c = Counters()
        _check(lib().moe_lru_counters(self._h, ctypes.byref(c)))
        return c

    def close(self):
        if getattr(self, "_h", None):
            lib().moe_lru_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def _plan_in(m):
    return PlanIn(m["n_layers"], m["n_experts"], m["top_k"], 0, m["payload_bytes"],
                  m.get("common_bytes", 0), m.get("kv_bytes_per_token", 0),
                  m.get("overhead_bytes", 0), m.get("target_bytes", 0))


def plan_percent(model, percent, context_tokens=0):
    """Static budget plan for a cache percentage (moe_plan_percent); model is a dict with
    n_layers, n_experts, top_k, payload_bytes and optionally common_bytes,
    kv_bytes_per_token, overhead_bytes, target_bytes.  Returns the plan as a dict."""
    out = PlanOut()
    rc = lib().moe_plan_percent(ctypes.byref(_plan_in(model)), float(percent), int(context_tokens),
                                ctypes.byref(out))
    if rc != MOE_OK:
        raise MoeError(rc, "moe_plan_percent: bad argument or size overflow")
    return out.as_dict()


def plan_bytes(model, cache_bytes, context_tokens=0):
    """Static budget plan for a cache byte budget over all routed layers (moe_plan_bytes)."""
    out = PlanOut()
    rc = lib().moe_plan_bytes(ctypes.byref(_plan_in(model)), int(cache_bytes), int(context_tokens),
                              ctypes.byref(out))
    if rc != MOE_OK:
        raise MoeError(rc, "moe_plan_bytes: bad argument or size overflow")
    return out.as_dict()


def min_misses(calls, n_experts, n_slots):
    """Fewest misses any slot policy can have on one layer's calls (moe_policy_min); calls is a
    sequence of id arrays, one per layer call."""
    calls = [np.asarray(c, np.int32).ravel() for c in calls]
    off = np.zeros(len(calls) + 1, np.int64)
    off[1:] = np.cumsum([c.size for c in calls])
    ids = np.concatenate(calls) if calls else np.zeros(1, np.int32)
    ids = np.ascontiguousarray(ids, np.int32)
    m = ctypes.c_uint64()
    rc = lib().moe_policy_min(ids.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)),
                              off.ctypes.data_as(ctypes.POINTER(ctypes.c_int64)), len(calls),
                              n_experts, n_slots, ctypes.byref(m))
    if rc != MOE_OK:
        raise MoeError(rc, "moe_policy_min: bad argument or a call with more experts than slots")
    return m.value


def pack_gguf(gguf_path, pack_path, index_path, router_path=None):
    """Split-pack a GGUF MoE model (moe_pack_gguf).  Returns the topology as a dict."""
    info = PackInfo()
    enc = lambda p: None if p is None else os.fsencode(p)
    _check(lib().moe_pack_gguf(enc(gguf_path), enc(pack_path), enc(index_path), enc(router_path),
                               ctypes.byref(info)))
    return {f: getattr(info, f) for f, _ in info._fields_}
