// Host side of libmoecache: the C ABI declared in include/moecache.h.
//
// One handle = one model's expert store (pinned host memory, caller-owned),
// per-layer HBM slot slabs, per-layer LRU slot tables, a side stream for the
// miss copies, and small scratch buffers.
//
// Decode with the default copy kernel keeps the slot tables in device memory:
// a layer call is four launches on the caller's stream (router partials;
// router finish + slot-table step, which writes the call's work list; the
// misses' copies fused with gate/up for all routed experts; down) and the host
// never waits.  The other
// copy modes and prefill run the slot table on the host, after waiting for
// the routes; around a prefill call the layer's table moves to the host and back.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <new>
#include <string>
#include <vector>

#include "../../include/moecache.h"
#include "kernels.h"
#include "slot_lru.h"

using namespace moecache;

// Per-call scratch of moe_layer_forward_static (router partials, routes, digit
// staging, work list of one decode call), held by every GPU the library runs on
// until the process ends.  Host code never uses this name as an address: each
// device's copy is reached through the pointer hipGetSymbolAddress returns for
// it (static_scratch_ptr).
constexpr size_t kStaticScratchBytes = size_t(1) << 20;
static __device__ __align__(256) uint8_t scratch[kStaticScratchBytes];

namespace {
thread_local std::string g_err;
}  // namespace

// The message moe_last_error returns, set by the library's other translation units.
void moecache_set_last_error(const char *msg) { g_err = msg; }

namespace {

int fail(int code, const char *fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return code;
}

constexpr int kCopyGrid = 64;  // copy-kernel blocks: enough requests in flight to fill PCIe
// Multi-token calls of at most this many tokens whose routed experts all fit the
// slots run the decode GEMVs once per token instead of the MFMA grouped GEMMs
// (whose 128-row tiles would hold a handful of rows).
constexpr int kSmallTokens = kMtTokens;

struct TimedSpan {
  int kind;
  hipEvent_t start, stop;
  uint64_t launches, bytes, flops;
};

}  // namespace

struct moe_cache {
  moe_model_desc d{};
  int32_t C = 0;
  int64_t M = 0;   // bytes of one W_gate (or W_up) matrix
  int64_t Md = 0;  // bytes of one W_down matrix (the same as M unless the formats differ)
  int64_t P = 0;   // payload bytes: 2 M + Md
  hipStream_t main = nullptr, side = nullptr;
  int device = 0;
  bool poisoned = false;
  const uint8_t *store = nullptr;

  uint8_t *slots = nullptr;  // [L][C][P]
  float *partial = nullptr;  // router split partials [grid][E], then 1/rms
  int8_t *xq = nullptr;         // decode: digits of the scaled token [3][H]
  float *xsc = nullptr;         //   and their block scales [H/32]
  int32_t *topk_idx = nullptr;  // device [cap_tokens][k]
  float *topk_w = nullptr;
  float *zbuf = nullptr;  // prefill logits [cap_tokens][E]
  int64_t cap_tokens = 0;
  // prefill buffers (grown on demand)
  int64_t pf_cap = 0;
  float *pf_inv = nullptr;      // [T]
  __bf16 *pf_xb = nullptr;      // [2][T][H] (hi, lo)
  int32_t *pf_counts = nullptr; // grouping scratch, group_counts_ints(E)
  int32_t *pf_off = nullptr;    // [E+1]
  int32_t *pf_perm = nullptr;   // [T*k]
  __bf16 *pf_ab = nullptr;      // [2][T*k][I] (hi, lo)
  float *pf_P = nullptr;        // [T*k][H]
  int32_t *pf_host_off = nullptr;  // pinned [E+1]
  // multi-token calls small enough for the decode GEMVs (one token at a time)
  int8_t *st_xq = nullptr;          // [kSmallTokens][3][H] digits of each token
  float *st_xsc = nullptr;          // [kSmallTokens][H/32]
  int32_t *st_host_idx = nullptr;   // pinned [kSmallTokens][top_k] routes
  std::vector<hipEvent_t> pf_ev;   // per-chunk events (copy done, compute done)
  int8_t *hq = nullptr;   // decode: digits of the SwiGLU activations [3][k*I]
  float *hsc = nullptr;   //   their 16-wide block scales [k*I/16]
  int32_t *hds = nullptr; //   and digit sums [3][k*I/16]
  // device-resident slot tables (decode with the copy kernel)
  bool dev_lru = false;
  int32_t *dl_slot_of = nullptr;    // [L][E]
  int32_t *dl_expert_in = nullptr;  // [L][C]
  int64_t *dl_stamp = nullptr;      // [L][E]
  int64_t *dl_meta = nullptr;       // [L][3] clock, step, used
  uint64_t *dl_cnt = nullptr;       // [L][4]
  int32_t *dl_trace = nullptr;      // [dl_trace_cap][6]
  uint64_t *dl_trace_n = nullptr;
  int32_t *dl_err = nullptr;
  float *dl_zlast = nullptr;  // [E] logits of the last decode call
  uint64_t *dl_copy_acc = nullptr;  // [2] copies and bytes of the timed copy launches
  WorkList *dl_work = nullptr;
  // small multi-token calls stepped on the device
  float *mt_partial = nullptr;  // [kMtTokens][router grid * E + 1]
  MtWork *mt_work = nullptr;    // [kMtMaxChunks] work lists, one per chunk of a call
  int32_t *mt_flag = nullptr;   // pinned [3]: verdict (0 done, 1 left to the host table, 2
                                //   routing failure), union size, chunks
  int8_t *mt_hq = nullptr;      // [3][kMtTokens * k * I] activation digits by (token, rank)
  float *mt_hsc = nullptr;      // [kMtTokens * k * I / 16]
  int32_t *mt_hds = nullptr;    // [3][kMtTokens * k * I / 16]
  float *mt_R = nullptr;        // [kMtTokens * k][H] unweighted down rows
  // per-chunk work lists of small calls on the host-table path (device, pinned staging)
  MtWork *pf_mt_dev = nullptr, *pf_mt_host = nullptr;
  int pf_mt_cap = 0;
  int64_t dl_trace_cap = 0, dl_trace_pending = 0;
  uint8_t *dl_stage = nullptr;      // pinned staging of one layer's table
  bool table_pulled = false;        // a multi-token call holds the layer's table on the host
  int32_t *host_idx = nullptr;  // host mirrors [k] (decode)
  float *host_w = nullptr;
  hipEvent_t ev_route = nullptr, ev_copy = nullptr;

  std::vector<SlotLru> lru;
  // per layer: the last call of at most kSmallTokens tokens routed more experts
  // than the slots (the next such call goes straight to the host-table path)
  std::vector<uint8_t> small_overflow;
  std::vector<moe_step_rec> trace;
  size_t trace_head = 0;
  std::vector<moe_step_rec> recs;  // scratch for one call

  // timing (MOE_F_TIMING)
  std::vector<hipEvent_t> ev_pool;
  std::vector<TimedSpan> pending;
  moe_kernel_stats stats[MOE_KIND_COUNT]{};
  int32_t timing_every = 1;
  uint64_t n_calls = 0;
  bool timing_now = false;  // this call is bracketed

  uint8_t *static_scratch = nullptr;  // this device's copy of `scratch` (moe_layer_forward_static)

  uint8_t *slot_ptr(int32_t layer, int32_t s) const { return slots + ((int64_t)layer * C + s) * P; }
  DecodeScratch scratch() const { return DecodeScratch{xq, xsc, hq, hsc, hds}; }
};

namespace {

#define HIP_TRY(c, expr)                                                                   \
  do {                                                                                     \
    hipError_t e_ = (expr);                                                                \
    if (e_ != hipSuccess) {                                                                \
      if (c) (c)->poisoned = true;                                                         \
      return fail(MOE_EHIP, "%s failed: %s (%s:%d)", #expr, hipGetErrorString(e_), __FILE__, \
                  __LINE__);                                                               \
    }                                                                                      \
  } while (0)

hipEvent_t get_event(moe_cache *c) {
  if (!c->ev_pool.empty()) {
    hipEvent_t e = c->ev_pool.back();
    c->ev_pool.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}

// Fold completed timing spans into the totals; spans whose stop event has not
// completed yet stay pending (wait = true synchronises them first).
int drain_timing(moe_cache *c, bool wait = false) {
  std::vector<TimedSpan> keep;
  for (auto &sp : c->pending) {
    if (wait) HIP_TRY(c, hipEventSynchronize(sp.stop));
    const hipError_t q = hipEventQuery(sp.stop);
    if (q == hipErrorNotReady) {
      keep.push_back(sp);
      continue;
    }
    HIP_TRY(c, q);
    float ms = 0.f;
    HIP_TRY(c, hipEventElapsedTime(&ms, sp.start, sp.stop));
    auto &st = c->stats[sp.kind];
    st.launches += sp.launches;
    st.total_ms += ms;
    st.bytes += sp.bytes;
    st.flops += sp.flops;
    c->ev_pool.push_back(sp.start);
    c->ev_pool.push_back(sp.stop);
  }
  c->pending.swap(keep);
  return MOE_OK;
}

// Events of one timed launch wrapper.  Kernel launches take them through
// hipExtLaunchKernelGGL (the runtime stamps the kernels' own start and end);
// host-side copies record them on the stream around the copies.
struct Span {
  moe_cache *c;
  hipStream_t s;
  TimedSpan sp{};
  bool on = false;
  Span(moe_cache *c_, hipStream_t s_, int kind, uint64_t launches, uint64_t bytes, uint64_t flops)
      : c(c_), s(s_) {
    if (!c->timing_now) return;
    sp = TimedSpan{kind, get_event(c), get_event(c), launches, bytes, flops};
    on = sp.start && sp.stop;
  }
  Timing timing() const { return on ? Timing{sp.start, sp.stop} : Timing{}; }
  void record_start() {
    if (on && hipEventRecord(sp.start, s) != hipSuccess) on = false;
  }
  void record_stop() {
    if (on && hipEventRecord(sp.stop, s) != hipSuccess) on = false;
  }
  void end() {  // the launch (or the stop record) succeeded: keep the span
    if (on) c->pending.push_back(sp);
    on = false;
  }
  void discard() {  // not kept: the events go back to the pool
    if (on) {
      c->ev_pool.push_back(sp.start);
      c->ev_pool.push_back(sp.stop);
    }
    on = false;
  }
};

int check_desc(const moe_model_desc *d, int32_t budget) {
  if (!d) return fail(MOE_EINVAL, "desc is NULL");
  if (d->n_layers < 1 || d->n_experts < 1 || d->n_experts > 256)
    return fail(MOE_EINVAL, "n_layers must be >= 1 and n_experts in [1, 256]");
  if (d->top_k < 1 || d->top_k > d->n_experts || d->top_k > kMaxRouted)
    return fail(MOE_EINVAL, "top_k must be in [1, min(n_experts, %d)]", kMaxRouted);
  if (d->hidden < 64 || d->hidden % 64 || d->hidden > 8192 || d->inter < 64 || d->inter % 64 ||
      d->inter > 8192)
    return fail(MOE_EINVAL, "hidden and inter must be multiples of 64 in [64, 8192]");
  if ((int64_t)d->top_k * d->inter > 12288)
    return fail(MOE_EINVAL, "top_k * inter must be <= 12288 (decode activations are staged in LDS)");
  {
    const int gu = fmt_gate_up(d->qtype), dn = fmt_down(d->qtype);
    if (d->qtype < 0 || d->qtype > 0xffff || !fmt_known(gu) || !fmt_known(dn) ||
        (gu != dn && !(fmt_kquant(gu) && fmt_kquant(dn))))
      return fail(MOE_EINVAL, "qtype must be MOE_Q8_0, MOE_Q4_0, MOE_Q4_K, MOE_Q6_K or a mix of the two "
                  "K-quant formats (MOE_QTYPE_MIX)");
    if ((fmt_kquant(gu) && d->hidden % 256) || (fmt_kquant(dn) && d->inter % 256))
      return fail(MOE_EINVAL, "K-quant formats need hidden (gate/up) and inter (down) multiples of 256");
  }
  if (budget < d->top_k || budget > d->n_experts)
    return fail(MOE_EINVAL, "budget_slots %d outside [top_k=%d, n_experts=%d]", budget, d->top_k,
                d->n_experts);
  if (!d->host_store) return fail(MOE_EINVAL, "host_store is NULL");
  if ((d->flags & MOE_F_SCORE_EVICT) && (d->flags & (MOE_F_SIDE_COPY | MOE_F_SDMA_COPY)))
    return fail(MOE_EINVAL, "MOE_F_SCORE_EVICT needs the default copy modes (device slot tables)");
  return MOE_OK;
}

void free_all(moe_cache *c) {
  if (!c) return;
  if (c->main || c->side) {
    if (c->side) (void)hipStreamSynchronize(c->side);
    (void)hipStreamSynchronize(c->main);
  }
  (void)hipFree(c->slots);
  (void)hipFree(c->partial);
  (void)hipFree(c->topk_idx);
  (void)hipFree(c->topk_w);
  (void)hipFree(c->zbuf);
  (void)hipFree(c->hq);
  (void)hipFree(c->hsc);
  (void)hipFree(c->hds);
  (void)hipFree(c->pf_inv);
  (void)hipFree(c->pf_xb);
  (void)hipFree(c->pf_counts);
  (void)hipFree(c->pf_off);
  (void)hipFree(c->pf_perm);
  (void)hipFree(c->pf_ab);
  (void)hipFree(c->pf_P);
  if (c->pf_host_off) (void)hipHostFree(c->pf_host_off);
  if (c->st_host_idx) (void)hipHostFree(c->st_host_idx);
  (void)hipFree(c->st_xq);
  (void)hipFree(c->st_xsc);
  for (auto e : c->pf_ev) (void)hipEventDestroy(e);
  (void)hipFree(c->xq);
  (void)hipFree(c->xsc);
  (void)hipFree(c->dl_slot_of);
  (void)hipFree(c->dl_expert_in);
  (void)hipFree(c->dl_stamp);
  (void)hipFree(c->dl_meta);
  (void)hipFree(c->dl_cnt);
  (void)hipFree(c->dl_trace);
  (void)hipFree(c->dl_trace_n);
  (void)hipFree(c->dl_err);
  (void)hipFree(c->dl_zlast);
  (void)hipFree(c->dl_copy_acc);
  (void)hipFree(c->dl_work);
  (void)hipFree(c->mt_partial);
  (void)hipFree(c->mt_work);
  (void)hipFree(c->mt_hq);
  (void)hipFree(c->mt_hsc);
  (void)hipFree(c->mt_hds);
  (void)hipFree(c->mt_R);
  (void)hipFree(c->pf_mt_dev);
  if (c->pf_mt_host) (void)hipHostFree(c->pf_mt_host);
  if (c->mt_flag) (void)hipHostFree(c->mt_flag);
  if (c->dl_stage) (void)hipHostFree(c->dl_stage);
  if (c->host_idx) (void)hipHostFree(c->host_idx);
  if (c->host_w) (void)hipHostFree(c->host_w);
  if (c->ev_route) (void)hipEventDestroy(c->ev_route);
  if (c->ev_copy) (void)hipEventDestroy(c->ev_copy);
  for (auto &sp : c->pending) {
    (void)hipEventDestroy(sp.start);
    (void)hipEventDestroy(sp.stop);
  }
  for (auto e : c->ev_pool) (void)hipEventDestroy(e);
  if (c->side) (void)hipStreamDestroy(c->side);
  delete c;
}

int ensure_tokens(moe_cache *c, int64_t T) {
  if (T <= c->cap_tokens) return MOE_OK;
  HIP_TRY(c, hipStreamSynchronize(c->main));
  (void)hipFree(c->topk_idx);
  (void)hipFree(c->topk_w);
  (void)hipFree(c->zbuf);
  c->topk_idx = nullptr;
  c->topk_w = nullptr;
  c->zbuf = nullptr;
  c->cap_tokens = 0;
  const int64_t k = c->d.top_k, E = c->d.n_experts;
  if (hipMalloc(&c->topk_idx, T * k * sizeof(int32_t)) != hipSuccess ||
      hipMalloc(&c->topk_w, T * k * sizeof(float)) != hipSuccess ||
      hipMalloc(&c->zbuf, router_zbuf_floats(T, (int)E) * sizeof(float)) != hipSuccess)
    return fail(MOE_ENOMEM, "cannot allocate routing buffers for %lld tokens", (long long)T);
  c->cap_tokens = T;
  return MOE_OK;
}

// ---- device-resident slot tables ----

constexpr int64_t kTraceCap = 1 << 16;  // device trace records kept between drains


// The union GEMVs' activations and down rows for calls of up to kMtTokens
// tokens (every copy mode: the host-table path uses them too).
int alloc_mt_buffers(moe_cache *c) {
  const size_t mtKI = (size_t)kMtTokens * c->d.top_k * c->d.inter;
  if (hipMalloc(&c->mt_hq, 3 * mtKI) != hipSuccess ||
      hipMalloc(&c->mt_hsc, mtKI / 16 * sizeof(float)) != hipSuccess ||
      hipMalloc(&c->mt_hds, 3 * mtKI / 16 * sizeof(int32_t)) != hipSuccess ||
      hipMalloc(&c->mt_R, (size_t)kMtTokens * c->d.top_k * c->d.hidden * sizeof(float)) != hipSuccess) {
    (void)hipGetLastError();
    return fail(MOE_ENOMEM, "cannot allocate the multi-token activation buffers");
  }
  return MOE_OK;
}

int alloc_dev_tables(moe_cache *c) {
  const int64_t L = c->d.n_layers, E = c->d.n_experts, C = c->C;
  if (hipMalloc(&c->dl_slot_of, L * E * 4) != hipSuccess ||
      hipMalloc(&c->dl_expert_in, L * C * 4) != hipSuccess ||
      hipMalloc(&c->dl_stamp, L * E * 8) != hipSuccess || hipMalloc(&c->dl_meta, L * 3 * 8) != hipSuccess ||
      hipMalloc(&c->dl_cnt, L * 4 * 8) != hipSuccess || hipMalloc(&c->dl_trace_n, 8) != hipSuccess ||
      hipMalloc(&c->dl_err, 4) != hipSuccess || hipMalloc(&c->dl_copy_acc, 16) != hipSuccess ||
      hipMalloc(&c->dl_zlast, E * 4) != hipSuccess ||
      hipMalloc(&c->dl_work, sizeof(WorkList)) != hipSuccess ||
      hipMalloc(&c->mt_partial, ((size_t)router_decode_grid(c->d.hidden) * E + 1) * kMtTokens *
                                    sizeof(float)) != hipSuccess ||
      hipMalloc(&c->mt_work, kMtMaxChunks * sizeof(MtWork)) != hipSuccess ||
      hipHostMalloc(&c->mt_flag, 3 * sizeof(int32_t), hipHostMallocCoherent) != hipSuccess ||
      hipHostMalloc(&c->dl_stage, table_stage_bytes((int)E, (int)C), hipHostMallocDefault) !=
          hipSuccess) {
    (void)hipGetLastError();
    return fail(MOE_ENOMEM, "cannot allocate the device slot tables");
  }
  if (c->d.flags & MOE_F_TRACE) {
    if (hipMalloc(&c->dl_trace, kTraceCap * 6 * 4) != hipSuccess) {
      (void)hipGetLastError();
      return fail(MOE_ENOMEM, "cannot allocate the device trace");
    }
    c->dl_trace_cap = kTraceCap;
  }
  return MOE_OK;
}

// Empty tables, zero counters (queued on the caller's stream).
int clear_dev_tables(moe_cache *c) {
  const int64_t L = c->d.n_layers, E = c->d.n_experts, C = c->C;
  HIP_TRY(c, hipMemsetAsync(c->dl_slot_of, 0xff, L * E * 4, c->main));
  HIP_TRY(c, hipMemsetAsync(c->dl_expert_in, 0xff, L * C * 4, c->main));
  HIP_TRY(c, hipMemsetAsync(c->dl_stamp, 0, L * E * 8, c->main));
  HIP_TRY(c, hipMemsetAsync(c->dl_meta, 0, L * 3 * 8, c->main));
  HIP_TRY(c, hipMemsetAsync(c->dl_cnt, 0, L * 4 * 8, c->main));
  HIP_TRY(c, hipMemsetAsync(c->dl_trace_n, 0, 8, c->main));
  HIP_TRY(c, hipMemsetAsync(c->dl_err, 0, 4, c->main));
  HIP_TRY(c, hipMemsetAsync(c->dl_zlast, 0, E * 4, c->main));
  HIP_TRY(c, hipMemsetAsync(c->dl_copy_acc, 0, 16, c->main));
  HIP_TRY(c, hipMemsetAsync(c->dl_work, 0, sizeof(WorkList), c->main));
  HIP_TRY(c, hipMemsetAsync(c->mt_work, 0, kMtMaxChunks * sizeof(MtWork), c->main));
  c->dl_trace_pending = 0;
  return MOE_OK;
}

// After a synchronisation: report a routing error the device recorded.
int check_dev_error(moe_cache *c) {
  if (!c->dev_lru) return MOE_OK;
  int32_t err = 0;
  HIP_TRY(c, hipMemcpy(&err, c->dl_err, 4, hipMemcpyDeviceToHost));
  if (err) {
    c->poisoned = true;
    return fail(MOE_EHIP, "router produced expert id %d (non-finite logits?)", (int16_t)(err - 1));
  }
  return MOE_OK;
}

// Synchronise with the caller's stream and check for a recorded error.
int sync_dev(moe_cache *c) {
  HIP_TRY(c, hipStreamSynchronize(c->main));
  return check_dev_error(c);
}

// Move the device trace records into the host trace (synchronises).
int drain_dev_trace(moe_cache *c) {
  if (!c->dev_lru || !c->dl_trace) return MOE_OK;
  int rc = sync_dev(c);
  if (rc) return rc;
  uint64_t n = 0;
  HIP_TRY(c, hipMemcpy(&n, c->dl_trace_n, 8, hipMemcpyDeviceToHost));
  if ((int64_t)n > c->dl_trace_cap) {
    c->poisoned = true;
    return fail(MOE_EHIP, "device trace overflow (%llu records)", (unsigned long long)n);
  }
  if (n) {
    const size_t at = c->trace.size();
    c->trace.resize(at + n);
    static_assert(sizeof(moe_step_rec) == 24, "moe_step_rec is six int32");
    HIP_TRY(c, hipMemcpy(c->trace.data() + at, c->dl_trace, n * sizeof(moe_step_rec),
                         hipMemcpyDeviceToHost));
    HIP_TRY(c, hipMemsetAsync(c->dl_trace_n, 0, 8, c->main));
    HIP_TRY(c, hipStreamSynchronize(c->main));
  }
  c->dl_trace_pending = 0;
  return MOE_OK;
}

LruDev dev_table(moe_cache *c, int32_t layer) {
  const int64_t E = c->d.n_experts, C = c->C;
  LruDev L{};
  L.slot_of = c->dl_slot_of + layer * E;
  L.expert_in = c->dl_expert_in + layer * C;
  L.stamp = c->dl_stamp + layer * E;
  L.meta = c->dl_meta + layer * 3;
  L.cnt = c->dl_cnt + layer * 4;
  L.trace = c->dl_trace;
  L.trace_n = c->dl_trace_n;
  L.err = c->dl_err;
  L.store = c->store + (int64_t)layer * E * c->P;
  L.slots = c->slot_ptr(layer, 0);
  L.work = c->dl_work;
  L.P = c->P;
  L.C = (int32_t)C;
  L.layer = layer;
  L.zlast = c->dl_zlast;
  L.policy = (c->d.flags & MOE_F_SCORE_EVICT) ? 1 : 0;
  return L;
}

// Where one decode call keeps its per-call scratch (router partials, routes,
// digit staging, work list): the handle's own buffers, or the library's static
// per-device array (moe_layer_forward_static).
struct DecodeBufs {
  float *partial;
  int32_t *idx;
  float *w;
  DecodeScratch s;
  WorkList *work;
};

DecodeBufs handle_bufs(moe_cache *c) {
  return DecodeBufs{c->partial, c->topk_idx, c->topk_w, c->scratch(), c->dl_work};
}

// The address of `scratch` on each device, resolved once per device with that
// device current.
std::mutex g_static_mu;
std::vector<uint8_t *> g_static_ptr;

int static_scratch_ptr(int device, uint8_t **out) {
  std::lock_guard<std::mutex> lock(g_static_mu);
  if (device < 0) return fail(MOE_EINVAL, "bad device %d", device);
  if ((int)g_static_ptr.size() <= device) g_static_ptr.resize(device + 1, nullptr);
  if (!g_static_ptr[device]) {
    void *p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p)
      return fail(MOE_EHIP, "hipGetSymbolAddress(scratch) failed: %s", hipGetErrorString(e));
    g_static_ptr[device] = static_cast<uint8_t *>(p);
  }
  *out = g_static_ptr[device];
  return MOE_OK;
}

// One decode call's buffers carved out of the static array (each 256-byte
// aligned); *bytes gets the total.  Nothing in it needs to start at zero: each
// call's router writes the partials, routes, digits and the whole work list
// (count included) before any kernel of the call reads them.
DecodeBufs static_bufs(const moe_cache *c, uint8_t *base, size_t *bytes) {
  const moe_model_desc &d = c->d;
  size_t off = 0;
  auto take = [&](size_t n) {
    uint8_t *p = base + off;
    off += (n + 255) / 256 * 256;
    return p;
  };
  const size_t kI = (size_t)d.top_k * d.inter;
  DecodeBufs b{};
  b.partial = reinterpret_cast<float *>(take(((size_t)router_decode_grid(d.hidden) * d.n_experts + 1) * 4));
  b.idx = reinterpret_cast<int32_t *>(take((size_t)d.top_k * 4));
  b.w = reinterpret_cast<float *>(take((size_t)d.top_k * 4));
  b.s.xq = reinterpret_cast<int8_t *>(take(3 * (size_t)d.hidden));
  b.s.xsc = reinterpret_cast<float *>(take((size_t)d.hidden / 32 * 4));
  b.s.hq = reinterpret_cast<int8_t *>(take(3 * kI));
  b.s.hsc = reinterpret_cast<float *>(take(kI / 16 * 4));
  b.s.hds = reinterpret_cast<int32_t *>(take(3 * kI / 16 * 4));
  b.work = reinterpret_cast<WorkList *>(take(sizeof(WorkList)));
  *bytes = off;
  return b;
}

// A multi-token call steps the layer's table on the host.  The pull is queued
// behind the call's routing (one kernel writes the table and the device error
// word into the pinned staging) and read once the routing has been waited for;
// the push writes the staging and queues one kernel that copies it back.
int pull_table_queue(moe_cache *c, int32_t layer) {
  HIP_TRY(c, launch_table_pack(dev_table(c, layer), c->d.n_experts, c->C, c->dl_err, c->dl_stage,
                               c->main));
  return MOE_OK;
}

// After the caller's stream has passed the pack: the staging into the host table.
int pull_table_load(moe_cache *c, int32_t layer) {
  const int64_t E = c->d.n_experts, C = c->C;
  const uint8_t *p = c->dl_stage;
  const int64_t *stamp = reinterpret_cast<const int64_t *>(p), *meta = stamp + E;
  const uint64_t *cnt = reinterpret_cast<const uint64_t *>(meta + 3);
  const int32_t *err = reinterpret_cast<const int32_t *>(cnt + 4), *so = err + 2, *ei = so + E;
  if (*err) {
    c->poisoned = true;
    return fail(MOE_EHIP, "router produced expert id %d (non-finite logits?)", (int16_t)(*err - 1));
  }
  SlotLru::State st;
  st.slot_of.assign(so, so + E);
  st.expert_in.assign(ei, ei + C);
  st.stamp.assign(stamp, stamp + E);
  st.clock = (uint64_t)meta[0];
  st.step = (int32_t)meta[1];
  st.used = (int32_t)meta[2];
  st.cnt = moe_counters{cnt[0], cnt[1], cnt[2], cnt[3]};
  c->lru[layer].set_state(st);
  return MOE_OK;
}

int push_table(moe_cache *c, int32_t layer) {
  const int64_t E = c->d.n_experts, C = c->C;
  const SlotLru::State st = c->lru[layer].state();
  uint8_t *p = c->dl_stage;
  int64_t *stamp = reinterpret_cast<int64_t *>(p), *meta = stamp + E;
  uint64_t *cnt = reinterpret_cast<uint64_t *>(meta + 3);
  int32_t *so = reinterpret_cast<int32_t *>(cnt + 4) + 2, *ei = so + E;
  for (int64_t e = 0; e < E; ++e) stamp[e] = (int64_t)st.stamp[e];
  meta[0] = (int64_t)st.clock;
  meta[1] = st.step;
  meta[2] = st.used;
  cnt[0] = st.cnt.hits;
  cnt[1] = st.cnt.misses;
  cnt[2] = st.cnt.evictions;
  cnt[3] = st.cnt.materialized_bytes;
  std::copy(st.slot_of.begin(), st.slot_of.end(), so);
  std::copy(st.expert_in.begin(), st.expert_in.end(), ei);
  (void)C;
  HIP_TRY(c, launch_table_unpack(dev_table(c, layer), (int)E, c->C, c->dl_stage, c->main));
  return MOE_OK;
}

// Decode call with the slot table on the device: four launches, no host wait
// (unless the caller asks for the counter delta or the routes).
int forward_decode_dev(moe_cache *c, const float *x, const float *wr, int32_t layer, float *y,
                       moe_counters *delta, int32_t *dbg_idx, float *dbg_w, const DecodeBufs &b) {
  const moe_model_desc &d = c->d;
  const int k = d.top_k;
  c->timing_now = (d.flags & MOE_F_TIMING) && c->n_calls++ % c->timing_every == 0;
  uint64_t before[4] = {0, 0, 0, 0};
  int rc = MOE_OK;
  if (delta) {
    if ((rc = sync_dev(c))) return rc;
    HIP_TRY(c, hipMemcpy(before, c->dl_cnt + 4 * layer, 32, hipMemcpyDeviceToHost));
  }
  if (c->dl_trace && c->dl_trace_pending + k > c->dl_trace_cap && (rc = drain_dev_trace(c)))
    return rc;
  LruDev L = dev_table(c, layer);
  L.work = b.work;
  {
    Span sp(c, c->main, MOE_KIND_ROUTER, 1, (uint64_t)d.hidden * d.n_experts * 4 + d.hidden * 4,
            2ull * d.hidden * d.n_experts);
    HIP_TRY(c, launch_router_decode(x, wr, d.hidden, d.n_experts, k, b.partial, b.idx, b.w,
                                    nullptr, nullptr, b.s.xq, b.s.xsc,
                                    (d.flags & MOE_F_PRENORM) != 0, &L, c->main, sp.timing()));
    sp.end();
  }
  if (c->dl_trace) c->dl_trace_pending += k;
  ExpertList shape{};
  shape.n = k;
  uint64_t *acc = c->timing_now ? c->dl_copy_acc : nullptr;
  if (!(d.flags & MOE_F_SPLIT_COPY) && fusable_copy_gateup(d.qtype, d.hidden, d.inter)) {
    // one launch: the misses' copies, their gate/up on the fly, the hits' gate/up alongside
    Span sp(c, c->main, MOE_KIND_COPY, 0, 0, 0);  // copies and bytes come from the device
    HIP_TRY(c, launch_copy_gateup(d.qtype, b.s, d.hidden, d.inter, k, b.work, c->P,
                                  kCopyGrid, acc, c->main, sp.timing()));
    sp.end();
  } else {
    {
      Span sp(c, c->main, MOE_KIND_COPY, 0, 0, 0);
      HIP_TRY(c, launch_materialize_list(b.work, c->P, kCopyGrid, acc, c->main, sp.timing()));
      sp.end();
    }
    Span sp(c, c->main, MOE_KIND_GATEUP, 1, (uint64_t)k * 2 * c->M, 4ull * k * d.hidden * d.inter);
    HIP_TRY(c, launch_gateup(d.qtype, b.s, d.hidden, d.inter, k, shape, &b.work->list,
                             c->main, sp.timing()));
    sp.end();
  }
  {
    Span sp(c, c->main, MOE_KIND_DOWN, 1, (uint64_t)k * c->Md, 2ull * k * d.hidden * d.inter);
    HIP_TRY(c, launch_down(d.qtype, b.s, d.hidden, d.inter, k, shape, &b.work->list,
                           b.w, x, y, (d.flags & MOE_F_RESIDUAL) ? 1 : 0, c->main, sp.timing()));
    sp.end();
  }
  if ((d.flags & MOE_F_TIMING) && (rc = drain_timing(c))) return rc;
  if (delta || dbg_idx || dbg_w) {
    if ((rc = sync_dev(c))) return rc;
    if (dbg_idx) HIP_TRY(c, hipMemcpy(dbg_idx, b.idx, k * sizeof(int32_t), hipMemcpyDeviceToHost));
    if (dbg_w) HIP_TRY(c, hipMemcpy(dbg_w, b.w, k * sizeof(float), hipMemcpyDeviceToHost));
    if (delta) {
      uint64_t after[4];
      HIP_TRY(c, hipMemcpy(after, c->dl_cnt + 4 * layer, 32, hipMemcpyDeviceToHost));
      *delta = moe_counters{after[0] - before[0], after[1] - before[1], after[2] - before[2],
                            after[3] - before[3]};
    }
  }
  return MOE_OK;
}

int forward_decode(moe_cache *c, const float *x, const float *wr, int32_t layer, float *y,
                   moe_counters *delta, int32_t *dbg_idx, float *dbg_w) {
  if (c->dev_lru) return forward_decode_dev(c, x, wr, layer, y, delta, dbg_idx, dbg_w, handle_bufs(c));
  const moe_model_desc &d = c->d;
  const int k = d.top_k;
  c->timing_now = (d.flags & MOE_F_TIMING) && c->n_calls++ % c->timing_every == 0;
  for (int i = 0; i < k; ++i) reinterpret_cast<volatile int32_t *>(c->host_idx)[i] = -1;
  {
    Span sp(c, c->main, MOE_KIND_ROUTER, 1, (uint64_t)d.hidden * d.n_experts * 4 + d.hidden * 4,
            2ull * d.hidden * d.n_experts);
    HIP_TRY(c, launch_router_decode(x, wr, d.hidden, d.n_experts, k, c->partial, c->topk_idx,
                                    c->topk_w, c->host_idx, c->host_w, c->xq, c->xsc,
                                    (d.flags & MOE_F_PRENORM) != 0, nullptr, c->main, sp.timing()));
    sp.end();
  }
  HIP_TRY(c, hipEventRecord(c->ev_route, c->main));
  // Wait for the routes: spin on the host-mapped ids the router writes (each
  // was set to -1 before the launch); this wakes the host sooner than an
  // event wait.  After a while without them, fall back to the event, which
  // also reports a failed launch.
  {
    volatile int32_t *hid = c->host_idx;
    bool ready = false;
    for (long spin = 0; !ready; ++spin) {
      ready = true;
      for (int i = 0; i < k; ++i) ready = ready && hid[i] >= 0;
      if (!ready && (spin & 0xfff) == 0xfff && hipEventQuery(c->ev_route) != hipErrorNotReady) {
        HIP_TRY(c, hipEventSynchronize(c->ev_route));
        ready = true;
      }
    }
  }
  if (dbg_w) HIP_TRY(c, hipEventSynchronize(c->ev_route));
  if (c->d.flags & MOE_F_TIMING) {
    int rc = drain_timing(c);
    if (rc) return rc;
  }

  int32_t ids[kMaxRouted];
  for (int i = 0; i < k; ++i) {
    ids[i] = c->host_idx[i];
    if (ids[i] < 0 || ids[i] >= d.n_experts) {
      c->poisoned = true;
      return fail(MOE_EHIP, "router produced expert id %d", ids[i]);
    }
  }
  if (dbg_idx) std::memcpy(dbg_idx, ids, sizeof(int32_t) * k);
  if (dbg_w) std::memcpy(dbg_w, c->host_w, sizeof(float) * k);

  SlotLru &t = c->lru[layer];
  const moe_counters before = t.counters();
  c->recs.clear();
  t.step(ids, k, c->recs);

  // hit/miss per routed position (top-k order)
  ExpertList hits{}, misses{}, all{};
  int n_copy = 0;
  for (const auto &r : c->recs) n_copy += r.hit ? 0 : 1;
  for (int i = 0; i < k; ++i) {
    const int32_t e = ids[i];
    bool hit = false;
    for (const auto &r : c->recs)
      if (r.expert == e) hit = r.hit;
    ExpertList &L = hit ? hits : misses;
    L.payload[L.n] = all.payload[all.n] = c->slot_ptr(layer, t.slot_of(e));
    L.pos[L.n++] = all.pos[all.n++] = i;
  }
  const bool resid = d.flags & MOE_F_RESIDUAL;
  const uint64_t gu_bytes = 2ull * c->M, dn_bytes = (uint64_t)c->Md;
  const uint64_t gu_flops = 4ull * d.hidden * d.inter, dn_flops = 2ull * d.hidden * d.inter;
  auto gateup = [&](const ExpertList &L) -> int {
    Span sp(c, c->main, MOE_KIND_GATEUP, 1, L.n * gu_bytes, L.n * gu_flops);
    HIP_TRY(c, launch_gateup(d.qtype, c->scratch(), d.hidden, d.inter, d.top_k, L, nullptr, c->main,
                             sp.timing()));
    sp.end();
    return MOE_OK;
  };
  auto down = [&](const ExpertList &L, int mode) -> int {
    Span sp(c, c->main, MOE_KIND_DOWN, 1, L.n * dn_bytes, L.n * dn_flops);
    HIP_TRY(c, launch_down(d.qtype, c->scratch(), d.hidden, d.inter, d.top_k, L, nullptr, c->topk_w, x,
                           y, mode, c->main, sp.timing()));
    sp.end();
    return MOE_OK;
  };
  // misses in ascending expert order (the records' order)
  auto copy_misses = [&](hipStream_t s) -> int {
    Span sp(c, s, MOE_KIND_COPY, n_copy, (uint64_t)n_copy * c->P, 0);
    sp.record_start();
    for (const auto &r : c->recs) {
      if (r.hit) continue;
      const uint8_t *src = c->store + ((int64_t)layer * d.n_experts + r.expert) * c->P;
      HIP_TRY(c, hipMemcpyAsync(c->slot_ptr(layer, r.slot), src, c->P, hipMemcpyDefault, s));
    }
    sp.record_stop();
    sp.end();
    return MOE_OK;
  };
  int rc = MOE_OK;
  if (d.flags & MOE_F_SIDE_COPY) {
    // copies on the side stream, overlapped with the hit experts on the caller's stream
    if (n_copy) {
      if ((rc = copy_misses(c->side))) return rc;
      HIP_TRY(c, hipEventRecord(c->ev_copy, c->side));
    }
    bool wrote = false;
    if (hits.n) {
      if ((rc = gateup(hits)) || (rc = down(hits, resid ? 1 : 0))) return rc;
      wrote = true;
    }
    if (misses.n) {
      HIP_TRY(c, hipStreamWaitEvent(c->main, c->ev_copy, 0));
      if ((rc = gateup(misses)) || (rc = down(misses, wrote ? 2 : (resid ? 1 : 0)))) return rc;
    }
  } else {
    // everything on the caller's stream: the miss copies first (the critical
    // path), then gate/up and down over all routed experts in top-k order
    if (n_copy) {
      if (d.flags & MOE_F_SDMA_COPY) {
        if ((rc = copy_misses(c->main))) return rc;
      } else {
        const uint8_t *src[kMaxRouted];
        uint8_t *dst[kMaxRouted];
        int n = 0;
        for (const auto &r : c->recs) {
          if (r.hit) continue;
          src[n] = c->store + ((int64_t)layer * d.n_experts + r.expert) * c->P;
          dst[n++] = c->slot_ptr(layer, r.slot);
        }
        Span sp(c, c->main, MOE_KIND_COPY, n, (uint64_t)n * c->P, 0);
        HIP_TRY(c, launch_materialize(src, dst, n, c->P, kCopyGrid, c->main, sp.timing()));
        sp.end();
      }
    }
    if ((rc = gateup(all)) || (rc = down(all, resid ? 1 : 0))) return rc;
  }

  if (d.flags & MOE_F_TRACE) c->trace.insert(c->trace.end(), c->recs.begin(), c->recs.end());
  if (delta) {
    const moe_counters &a = t.counters();
    *delta = moe_counters{a.hits - before.hits, a.misses - before.misses,
                          a.evictions - before.evictions,
                          a.materialized_bytes - before.materialized_bytes};
  }
  return MOE_OK;
}

int forward_prefill(moe_cache *c, const float *x, int32_t T, const float *wr, int32_t layer,
                    float *y, moe_counters *delta, int32_t *dbg_idx, float *dbg_w);

// A multi-token call of at most kMtTokens tokens with the layer's table on
// the device: per token the decode router's partials and digits, then one
// block routes every token, steps the table over the union of their experts
// and writes the work lists (two launches); the misses' copies and the
// union's GEMVs of the first chunk follow, all queued on the caller's stream.
// The host then waits for the table step to learn the number of chunks (more
// than one when the union exceeds the slots and slots are reused inside the
// call), queues the other chunks' copies and GEMVs behind the first one's and
// the combination.  With more chunks than kMtMaxChunks, or for shapes the
// union GEMVs do not take when the union exceeds the slots, the table is left
// untouched, the queued kernels find an empty list and the call is run by
// the multi-token path with the table on the host.
int forward_small_dev(moe_cache *c, const float *x, int32_t T, const float *wr, int32_t layer, float *y,
                      moe_counters *delta, int32_t *dbg_idx, float *dbg_w) {
  const moe_model_desc &d = c->d;
  const int k = d.top_k, E = d.n_experts, H = d.hidden, I = d.inter;
  int rc = ensure_tokens(c, T);
  if (rc) return rc;
  c->timing_now = (d.flags & MOE_F_TIMING) && c->n_calls++ % c->timing_every == 0;
  uint64_t before[4] = {0, 0, 0, 0};
  if (delta) {
    if ((rc = sync_dev(c))) return rc;
    HIP_TRY(c, hipMemcpy(before, c->dl_cnt + 4 * layer, 32, hipMemcpyDeviceToHost));
  }
  if (c->dl_trace && c->dl_trace_pending + (int64_t)T * k > c->dl_trace_cap && (rc = drain_dev_trace(c)))
    return rc;
  const LruDev L = dev_table(c, layer);
  // the union's GEMVs (each expert's weights read once; their byte counts are
  // set once the union's size is known) or, for shapes those kernels do not
  // take, the decode GEMVs once per token (then one chunk only).  By default
  // the union's gate/up runs inside the copy launch (misses from the rows
  // being copied, hits alongside), as in decode.
  const bool union_ffn = mt_ffn_fits(d.qtype, H, I, T);
  const bool fused = union_ffn && !(d.flags & MOE_F_SPLIT_COPY) && fusable_copy_gateup_mt(d.qtype, H, I, T);
  volatile int32_t *flag = c->mt_flag;
  flag[0] = -1;
  {
    Span sp(c, c->main, MOE_KIND_ROUTER, 1, (uint64_t)H * E * 4 + (uint64_t)T * H * 4,
            2ull * T * H * E);
    HIP_TRY(c, launch_router_small(x, wr, T, H, E, k, c->mt_partial, c->topk_idx, c->topk_w, c->st_xq,
                                   c->st_xsc, (d.flags & MOE_F_PRENORM) != 0, L, c->mt_work, c->mt_flag,
                                   union_ffn ? kMtMaxChunks : 1, c->main, sp.timing()));
    sp.end();
  }
  HIP_TRY(c, hipEventRecord(c->ev_route, c->main));
  if (c->dl_trace) c->dl_trace_pending += (int64_t)T * k;
  const int umax = std::min(T * k, (int)c->C);
  uint64_t *acc = c->timing_now ? c->dl_copy_acc : nullptr;
  // one chunk's copies and union GEMVs (gu / dn: the spans of its GEMVs)
  auto chunk_ffn = [&](const MtWork *W, Span &gu, Span &dn) -> int {
    {
      Span sp(c, c->main, MOE_KIND_COPY, 0, 0, 0);  // copies and bytes come from the device
      if (fused)
        HIP_TRY(c, launch_copy_gateup_mt(d.qtype, W, c->st_xq, c->st_xsc, c->mt_hq, c->mt_hsc, c->mt_hds, H,
                                         I, k, T, umax, c->P, kCopyGrid, acc, c->main, sp.timing()));
      else
        HIP_TRY(c, launch_materialize_list(W, c->P, kCopyGrid, acc, c->main, sp.timing()));
      sp.end();
    }
    if (union_ffn) {
      if (!fused)
        HIP_TRY(c, launch_gateup_mt(d.qtype, W, c->st_xq, c->st_xsc, c->mt_hq, c->mt_hsc, c->mt_hds, H, I,
                                    k, T, umax, c->main, gu.timing()));
      HIP_TRY(c, launch_down_mt(d.qtype, W, c->mt_hq, c->mt_hsc, c->mt_hds, c->mt_R, H, I, k, T, umax,
                                c->main, dn.timing()));
    }
    return MOE_OK;
  };
  const int mode = (d.flags & MOE_F_RESIDUAL) ? 1 : 0;
  Span gu(c, c->main, MOE_KIND_GATEUP, 1, 0, 4ull * T * k * H * I);
  Span dn(c, c->main, MOE_KIND_DOWN, 1, 0, 2ull * T * k * H * I);
  if ((rc = chunk_ffn(c->mt_work, gu, dn))) return rc;
  if (!union_ffn) {
    ExpertList shape{};
    shape.n = k;
    for (int32_t tk = 0; tk < T; ++tk) {
      DecodeScratch St = c->scratch();
      St.xq = c->st_xq + (int64_t)tk * 3 * H;
      St.xsc = c->st_xsc + (int64_t)tk * (H / 32);
      {
        Span sp(c, c->main, MOE_KIND_GATEUP, 1, (uint64_t)k * 2 * c->M, 4ull * k * H * I);
        HIP_TRY(c, launch_gateup(d.qtype, St, H, I, k, shape, &c->mt_work->list[tk], c->main, sp.timing()));
        sp.end();
      }
      {
        Span sp(c, c->main, MOE_KIND_DOWN, 1, (uint64_t)k * c->Md, 2ull * k * H * I);
        HIP_TRY(c, launch_down(d.qtype, St, H, I, k, shape, &c->mt_work->list[tk],
                               c->topk_w + (int64_t)tk * k, x + (int64_t)tk * H, y + (int64_t)tk * H, mode,
                               c->main, sp.timing()));
        sp.end();
      }
    }
  }
  // the table step's verdict: spin on the flag the finishing block writes to
  // host memory; now and then ask the event, which also reports a failed launch
  for (long spin = 0; flag[0] < 0; ++spin) {
    if ((spin & 0xfff) == 0xfff && hipEventQuery(c->ev_route) != hipErrorNotReady) {
      HIP_TRY(c, hipEventSynchronize(c->ev_route));
      break;
    }
  }
  const int32_t verdict = flag[0];
  const int32_t n_chunks = flag[2];
  if (union_ffn && verdict == 0) {
    if (n_chunks < 1 || n_chunks > kMtMaxChunks) {
      c->poisoned = true;
      return fail(MOE_EHIP, "multi-token table step reported %d chunks", n_chunks);
    }
    gu.sp.bytes = (uint64_t)flag[1] * 2 * c->M;
    dn.sp.bytes = (uint64_t)flag[1] * c->Md;
    if (fused)
      gu.discard();  // timed with the copies
    else
      gu.end();
    dn.end();
    // the other chunks, each after the previous one (their copies overwrite
    // slots of experts computed in an earlier chunk), then the combination
    for (int ch = 1; ch < n_chunks; ++ch) {
      Span gu2(c, c->main, MOE_KIND_GATEUP, 1, 0, 0);
      Span dn2(c, c->main, MOE_KIND_DOWN, 1, 0, 0);
      if ((rc = chunk_ffn(c->mt_work + ch, gu2, dn2))) return rc;
      if (fused)
        gu2.discard();
      else
        gu2.end();
      dn2.end();
    }
    HIP_TRY(c, launch_combine_mt(c->mt_R, c->topk_w, x, y, H, k, T, mode, c->mt_work, c->main));
  } else {
    gu.discard();
    dn.discard();
  }
  if (verdict == 2) {
    c->poisoned = true;
    return fail(MOE_EHIP, "router of a multi-token call produced non-finite logits");
  }
  if (verdict != 0 && verdict != 1) {
    c->poisoned = true;
    return fail(MOE_EHIP, "multi-token table step did not report (flag %d)", verdict);
  }
  if ((d.flags & MOE_F_TIMING) && (rc = drain_timing(c))) return rc;
  if (verdict == 1) {
    c->small_overflow[layer] = 1;
    // one API call: the host-table path counts it again for the timing stride
    if (d.flags & MOE_F_TIMING) --c->n_calls;
    return forward_prefill(c, x, T, wr, layer, y, delta, dbg_idx, dbg_w);
  }
  if (delta || dbg_idx || dbg_w) {
    if ((rc = sync_dev(c))) return rc;
    if (dbg_idx)
      HIP_TRY(c, hipMemcpy(dbg_idx, c->topk_idx, (size_t)T * k * sizeof(int32_t), hipMemcpyDeviceToHost));
    if (dbg_w) HIP_TRY(c, hipMemcpy(dbg_w, c->topk_w, (size_t)T * k * sizeof(float), hipMemcpyDeviceToHost));
    if (delta) {
      uint64_t after[4];
      HIP_TRY(c, hipMemcpy(after, c->dl_cnt + 4 * layer, 32, hipMemcpyDeviceToHost));
      *delta = moe_counters{after[0] - before[0], after[1] - before[1], after[2] - before[2],
                            after[3] - before[3]};
    }
  }
  return MOE_OK;
}

}  // namespace

extern "C" {

const char *moe_last_error(void) { return g_err.c_str(); }

int moe_host_alloc(uint64_t bytes, void **out) {
  if (!out || bytes == 0) return fail(MOE_EINVAL, "moe_host_alloc: bad arguments");
  *out = nullptr;
  if (hipHostMalloc(out, bytes, hipHostMallocDefault) != hipSuccess || !*out)
    return fail(MOE_ENOMEM, "hipHostMalloc of %llu bytes failed", (unsigned long long)bytes);
  return MOE_OK;
}

int moe_host_free(void *p) {
  if (!p) return MOE_OK;
  hipError_t e = hipHostFree(p);
  return e == hipSuccess ? MOE_OK : fail(MOE_EHIP, "hipHostFree: %s", hipGetErrorString(e));
}

int moe_cache_create(const moe_model_desc *desc, int32_t budget_slots, moe_cache **out) {
  if (!out) return fail(MOE_EINVAL, "out is NULL");
  *out = nullptr;
  int rc = check_desc(desc, budget_slots);
  if (rc) return rc;
  moe_cache *c = new (std::nothrow) moe_cache;
  if (!c) return fail(MOE_ENOMEM, "out of host memory");
  c->d = *desc;
  c->C = budget_slots;
  c->M = fmt_matrix_bytes(fmt_gate_up(desc->qtype), desc->inter, desc->hidden);
  c->Md = fmt_matrix_bytes(fmt_down(desc->qtype), desc->hidden, desc->inter);
  c->P = 2 * c->M + c->Md;
  c->store = static_cast<const uint8_t *>(desc->host_store);
  c->main = static_cast<hipStream_t>(desc->hip_stream);
  const uint64_t want = (uint64_t)desc->n_layers * desc->n_experts * c->P;
  if (desc->store_bytes != want) {
    delete c;
    return fail(MOE_EINVAL, "store_bytes %llu != n_layers*n_experts*P = %llu",
                (unsigned long long)desc->store_bytes, (unsigned long long)want);
  }
  hipPointerAttribute_t attr{};
  if (hipPointerGetAttributes(&attr, desc->host_store) != hipSuccess ||
      (attr.type != hipMemoryTypeHost && attr.type != hipMemoryTypeDevice)) {
    (void)hipGetLastError();
    delete c;
    return fail(MOE_EINVAL, "host_store must be pinned host memory (hipHostMalloc) or device memory");
  }
  if (hipGetDevice(&c->device) != hipSuccess) {
    delete c;
    return fail(MOE_EHIP, "no HIP device");
  }
  if ((rc = static_scratch_ptr(c->device, &c->static_scratch))) {
    delete c;
    return rc;
  }
  for (int32_t l = 0; l < desc->n_layers; ++l) c->lru.emplace_back(desc->n_experts, budget_slots, c->P, l);
  c->small_overflow.assign(desc->n_layers, 0);

  const int64_t slot_bytes = (int64_t)desc->n_layers * budget_slots * c->P;
  if (hipMalloc(&c->slots, slot_bytes) != hipSuccess) {
    (void)hipGetLastError();
    free_all(c);
    return fail(MOE_ENOMEM, "cannot allocate %lld bytes of expert slots", (long long)slot_bytes);
  }
  const int grid = router_decode_grid(desc->hidden);
  if (hipMalloc(&c->partial, ((size_t)grid * desc->n_experts + 1) * sizeof(float)) != hipSuccess ||
      hipMalloc(&c->hq, 3 * (size_t)desc->top_k * desc->inter) != hipSuccess ||
      hipMalloc(&c->hsc, (size_t)desc->top_k * desc->inter / 16 * sizeof(float)) != hipSuccess ||
      hipMalloc(&c->hds, 3 * (size_t)desc->top_k * desc->inter / 16 * sizeof(int32_t)) != hipSuccess ||
      hipMalloc(&c->xq, 3 * (size_t)desc->hidden) != hipSuccess ||
      hipMalloc(&c->xsc, (size_t)desc->hidden / 32 * sizeof(float)) != hipSuccess ||
      hipMalloc(&c->st_xq, (size_t)kSmallTokens * 3 * desc->hidden) != hipSuccess ||
      hipMalloc(&c->st_xsc, (size_t)kSmallTokens * desc->hidden / 32 * sizeof(float)) != hipSuccess ||
      hipHostMalloc(&c->st_host_idx, (size_t)kSmallTokens * desc->top_k * sizeof(int32_t),
                    hipHostMallocDefault) != hipSuccess ||
      hipHostMalloc(&c->host_idx, kMaxRouted * sizeof(int32_t), hipHostMallocCoherent) != hipSuccess ||
      hipHostMalloc(&c->host_w, kMaxRouted * sizeof(float), hipHostMallocCoherent) != hipSuccess) {
    (void)hipGetLastError();
    free_all(c);
    return fail(MOE_ENOMEM, "cannot allocate scratch buffers");
  }
  if (hipStreamCreateWithFlags(&c->side, hipStreamNonBlocking) != hipSuccess ||
      hipEventCreateWithFlags(&c->ev_route, hipEventDisableTiming) != hipSuccess ||
      hipEventCreateWithFlags(&c->ev_copy, hipEventDisableTiming) != hipSuccess) {
    free_all(c);
    return fail(MOE_EHIP, "HIP setup failed");
  }
  rc = ensure_tokens(c, 1);
  if (!rc) rc = alloc_mt_buffers(c);
  c->dev_lru = !(desc->flags & (MOE_F_SIDE_COPY | MOE_F_SDMA_COPY));
  if (!rc && c->dev_lru) {
    rc = alloc_dev_tables(c);
    if (!rc) rc = clear_dev_tables(c);
    if (!rc && hipStreamSynchronize(c->main) != hipSuccess) rc = fail(MOE_EHIP, "stream synchronisation failed");
  }
  if (rc) {
    free_all(c);
    return rc;
  }
  *out = c;
  return MOE_OK;
}

int moe_layer_forward_dbg(moe_cache *c, const float *x, int32_t n_tokens, const float *router_w,
                          int32_t layer, float *y, moe_counters *delta, int32_t *topk_idx,
                          float *topk_w) {
  if (!c) return fail(MOE_EINVAL, "handle is NULL");
  if (c->poisoned) return fail(MOE_ESTATE, "handle poisoned by an earlier HIP error");
  if (!x || !router_w || !y) return fail(MOE_EINVAL, "x, router_w and y must be non-NULL");
  if (n_tokens < 1) return fail(MOE_EINVAL, "n_tokens must be >= 1");
  if (layer < 0 || layer >= c->d.n_layers)
    return fail(MOE_EINVAL, "layer %d outside [0, %d)", layer, c->d.n_layers);
  const int64_t bytes = (int64_t)n_tokens * c->d.hidden * 4;
  const char *xb = (const char *)x, *yb = (const char *)y;
  if (xb < yb + bytes && yb < xb + bytes) return fail(MOE_EINVAL, "y overlaps x");
  if (hipSetDevice(c->device) != hipSuccess) return fail(MOE_EHIP, "hipSetDevice failed");
  if (n_tokens == 1) return forward_decode(c, x, router_w, layer, y, delta, topk_idx, topk_w);
  // the grouped GEMMs index their bf16 hi/lo activation planes in 16-byte units with 32 bits
  if ((int64_t)n_tokens * std::max<int64_t>(c->d.hidden, (int64_t)c->d.top_k * c->d.inter) > (1ll << 34))
    return fail(MOE_EINVAL, "n_tokens * max(hidden, top_k * inter) must be <= 2^34");
  if (c->d.flags & MOE_F_SCORE_EVICT)
    return fail(MOE_EINVAL, "MOE_F_SCORE_EVICT takes one token per layer call");
  // a small call tries the device path, which also takes unions larger than
  // the slots (in chunks) where the union GEMVs take the shape; for other
  // shapes unless the layer's last small call did not fit the slots (then the
  // device step would only report that again).  The two paths step the table
  // by the same rule.
  if (c->dev_lru && n_tokens <= kSmallTokens &&
      (!c->small_overflow[layer] || mt_ffn_fits(c->d.qtype, c->d.hidden, c->d.inter, n_tokens)))
    return forward_small_dev(c, x, n_tokens, router_w, layer, y, delta, topk_idx, topk_w);
  return forward_prefill(c, x, n_tokens, router_w, layer, y, delta, topk_idx, topk_w);
}

int moe_layer_forward(moe_cache *c, const float *x, int32_t n_tokens, const float *router_w,
                      int32_t layer, float *y, moe_counters *delta) {
  return moe_layer_forward_dbg(c, x, n_tokens, router_w, layer, y, delta, nullptr, nullptr);
}

int moe_layer_forward_static(moe_cache *c, const float *x, int32_t n_tokens, const float *router_w,
                             int32_t layer, float *y, moe_counters *delta) {
  if (!c) return fail(MOE_EINVAL, "handle is NULL");
  if (c->poisoned) return fail(MOE_ESTATE, "handle poisoned by an earlier HIP error");
  if (!x || !router_w || !y) return fail(MOE_EINVAL, "x, router_w and y must be non-NULL");
  if (n_tokens != 1) return fail(MOE_EINVAL, "moe_layer_forward_static takes one token (n_tokens = 1)");
  if (layer < 0 || layer >= c->d.n_layers)
    return fail(MOE_EINVAL, "layer %d outside [0, %d)", layer, c->d.n_layers);
  if (!c->dev_lru)
    return fail(MOE_EINVAL, "moe_layer_forward_static needs the device slot tables (not the "
                "MOE_F_SIDE_COPY / MOE_F_SDMA_COPY modes)");
  const int64_t bytes = (int64_t)c->d.hidden * 4;
  const char *xb = (const char *)x, *yb = (const char *)y;
  if (xb < yb + bytes && yb < xb + bytes) return fail(MOE_EINVAL, "y overlaps x");
  size_t need = 0;
  const DecodeBufs b = static_bufs(c, c->static_scratch, &need);
  if (need > kStaticScratchBytes)
    return fail(MOE_EINVAL, "this shape needs %zu bytes of call scratch, more than the static %zu",
                need, kStaticScratchBytes);
  if (hipSetDevice(c->device) != hipSuccess) return fail(MOE_EHIP, "hipSetDevice failed");
  return forward_decode_dev(c, x, router_w, layer, y, delta, nullptr, nullptr, b);
}

int moe_cache_counters(const moe_cache *cc, int32_t layer, moe_counters *out) {
  if (!cc || !out) return fail(MOE_EINVAL, "NULL argument");
  if (layer < -1 || layer >= cc->d.n_layers) return fail(MOE_EINVAL, "layer out of range");
  moe_cache *c = const_cast<moe_cache *>(cc);  // synchronises, reads device tables
  std::vector<uint64_t> dev;
  if (c->dev_lru) {
    if (c->poisoned) return fail(MOE_ESTATE, "handle poisoned by an earlier HIP error");
    int rc = sync_dev(c);
    if (rc) return rc;
    dev.resize(4 * (size_t)c->d.n_layers);
    HIP_TRY(c, hipMemcpy(dev.data(), c->dl_cnt, dev.size() * 8, hipMemcpyDeviceToHost));
  }
  moe_counters s{};
  for (int32_t l = 0; l < c->d.n_layers; ++l) {
    if (layer >= 0 && l != layer) continue;
    const moe_counters a = c->dev_lru ? moe_counters{dev[4 * l], dev[4 * l + 1], dev[4 * l + 2],
                                                     dev[4 * l + 3]}
                                      : c->lru[l].counters();
    s.hits += a.hits;
    s.misses += a.misses;
    s.evictions += a.evictions;
    s.materialized_bytes += a.materialized_bytes;
  }
  *out = s;
  return MOE_OK;
}

int moe_cache_read_trace(moe_cache *c, moe_step_rec *buf, int64_t cap, int64_t *n_out) {
  if (!c || !n_out || cap < 0 || (cap > 0 && !buf)) return fail(MOE_EINVAL, "bad arguments");
  if (c->dev_lru) {
    if (c->poisoned) return fail(MOE_ESTATE, "handle poisoned by an earlier HIP error");
    int rc = drain_dev_trace(c);
    if (rc) return rc;
  }
  const int64_t avail = (int64_t)(c->trace.size() - c->trace_head);
  const int64_t n = std::min(avail, cap);
  if (n > 0) std::memcpy(buf, c->trace.data() + c->trace_head, n * sizeof(moe_step_rec));
  c->trace_head += n;
  if (c->trace_head == c->trace.size()) {
    c->trace.clear();
    c->trace_head = 0;
  }
  *n_out = n;
  return MOE_OK;
}

int moe_cache_reset(moe_cache *c) {
  if (!c) return fail(MOE_EINVAL, "handle is NULL");
  if (c->poisoned) return fail(MOE_ESTATE, "handle poisoned by an earlier HIP error");
  HIP_TRY(c, hipStreamSynchronize(c->side));
  HIP_TRY(c, hipStreamSynchronize(c->main));
  int rc = drain_timing(c, true);
  if (!rc) rc = check_dev_error(c);
  if (rc) return rc;
  for (auto &t : c->lru) t.reset();
  std::fill(c->small_overflow.begin(), c->small_overflow.end(), 0);
  if (c->dev_lru) {
    rc = clear_dev_tables(c);
    if (rc) return rc;
    HIP_TRY(c, hipStreamSynchronize(c->main));
  }
  c->n_calls = 0;
  c->trace.clear();
  c->trace_head = 0;
  for (auto &s : c->stats) s = moe_kernel_stats{};
  return MOE_OK;
}

int moe_cache_fill_slots(moe_cache *c, int32_t byte) {
  if (!c || byte < 0 || byte > 255) return fail(MOE_EINVAL, "bad arguments");
  if (c->poisoned) return fail(MOE_ESTATE, "handle poisoned by an earlier HIP error");
  HIP_TRY(c, hipStreamSynchronize(c->side));
  HIP_TRY(c, hipStreamSynchronize(c->main));
  const size_t bytes = (size_t)c->d.n_layers * c->C * c->P;
  HIP_TRY(c, hipMemsetAsync(c->slots, byte, bytes, c->main));
  HIP_TRY(c, hipStreamSynchronize(c->main));
  return MOE_OK;
}

int moe_cache_kernel_stats(moe_cache *c, int32_t kind, moe_kernel_stats *out) {
  if (!c || !out || kind < 0 || kind >= MOE_KIND_COUNT) return fail(MOE_EINVAL, "bad arguments");
  if (c->poisoned) return fail(MOE_ESTATE, "handle poisoned by an earlier HIP error");
  HIP_TRY(c, hipStreamSynchronize(c->side));
  HIP_TRY(c, hipStreamSynchronize(c->main));
  int rc = drain_timing(c, true);
  if (!rc) rc = check_dev_error(c);
  if (rc) return rc;
  *out = c->stats[kind];
  if (c->dev_lru && kind == MOE_KIND_COPY) {
    // decode copies are counted by the copy kernel itself (their spans carry no
    // count); prefill copies by their spans
    uint64_t acc[2];
    HIP_TRY(c, hipMemcpy(acc, c->dl_copy_acc, 16, hipMemcpyDeviceToHost));
    out->launches += acc[0];
    out->bytes += acc[1];
  }
  return MOE_OK;
}

int moe_cache_last_logits(moe_cache *c, float *z) {
  if (!c || !z) return fail(MOE_EINVAL, "NULL argument");
  if (!c->dev_lru) return fail(MOE_EINVAL, "logits are kept by the device slot tables only");
  if (c->poisoned) return fail(MOE_ESTATE, "handle poisoned by an earlier HIP error");
  int rc = sync_dev(c);
  if (rc) return rc;
  HIP_TRY(c, hipMemcpy(z, c->dl_zlast, (size_t)c->d.n_experts * 4, hipMemcpyDeviceToHost));
  return MOE_OK;
}

void moe_cache_destroy(moe_cache *c) { free_all(c); }

int moe_cache_set_timing_stride(moe_cache *c, int32_t every) {
  if (!c || every < 1) return fail(MOE_EINVAL, "timing stride must be >= 1");
  c->timing_every = every;
  c->n_calls = 0;
  return MOE_OK;
}

int moe_probe_h2d(const void *host_src, uint64_t chunk_bytes, int32_t n_chunks, int32_t n_streams,
                  double *gb_per_s) {
  if (!host_src || !gb_per_s || chunk_bytes == 0 || n_chunks < 1 || n_streams < 1 || n_streams > 16)
    return fail(MOE_EINVAL, "moe_probe_h2d: bad arguments");
  uint8_t *dst = nullptr;
  const uint64_t dst_bytes = chunk_bytes * (uint64_t)std::min(n_chunks, n_streams);
  if (hipMalloc(&dst, dst_bytes) != hipSuccess) return fail(MOE_ENOMEM, "probe buffer");
  std::vector<hipStream_t> st(n_streams, nullptr);
  hipEvent_t start = nullptr, stop = nullptr;
  std::vector<hipEvent_t> done(n_streams, nullptr);
  int rc = MOE_OK;
  float ms = 0.f;
  auto cleanup = [&]() {
    for (auto s_ : st)
      if (s_) (void)hipStreamDestroy(s_);
    for (auto e_ : done)
      if (e_) (void)hipEventDestroy(e_);
    if (start) (void)hipEventDestroy(start);
    if (stop) (void)hipEventDestroy(stop);
    (void)hipFree(dst);
  };
  const uint8_t *src = static_cast<const uint8_t *>(host_src);
  bool ok = hipEventCreate(&start) == hipSuccess && hipEventCreate(&stop) == hipSuccess;
  for (int i = 0; ok && i < n_streams; ++i)
    ok = hipStreamCreateWithFlags(&st[i], hipStreamNonBlocking) == hipSuccess &&
         hipEventCreateWithFlags(&done[i], hipEventDisableTiming) == hipSuccess;
  ok = ok && hipDeviceSynchronize() == hipSuccess && hipEventRecord(start, st[0]) == hipSuccess;
  for (int i = 1; ok && i < n_streams; ++i) ok = hipStreamWaitEvent(st[i], start, 0) == hipSuccess;
  for (int j = 0; ok && j < n_chunks; ++j) {
    int s_ = j % n_streams;
    ok = hipMemcpyAsync(dst + (uint64_t)s_ * chunk_bytes, src + (uint64_t)j * chunk_bytes, chunk_bytes,
                        hipMemcpyDefault, st[s_]) == hipSuccess;
  }
  for (int i = 1; ok && i < n_streams; ++i)
    ok = hipEventRecord(done[i], st[i]) == hipSuccess && hipStreamWaitEvent(st[0], done[i], 0) == hipSuccess;
  ok = ok && hipEventRecord(stop, st[0]) == hipSuccess && hipEventSynchronize(stop) == hipSuccess &&
       hipEventElapsedTime(&ms, start, stop) == hipSuccess;
  if (!ok) rc = fail(MOE_EHIP, "moe_probe_h2d: HIP call failed");
  else *gb_per_s = (double)chunk_bytes * n_chunks / (ms * 1e6);
  cleanup();
  return rc;
}

int moe_probe_hbm_read(uint64_t bytes, int32_t iters, double *read_us, double *empty_us) {
  if (!read_us || !empty_us || bytes == 0 || bytes % 16 || bytes > (1ull << 30) || iters < 1 ||
      iters > 10000)
    return fail(MOE_EINVAL, "moe_probe_hbm_read: bad arguments");
  // read consecutive regions of a buffer four times the size of the 256 MiB
  // last-level cache (or of 4 regions), so that no launch finds its bytes cached
  const uint64_t span = std::max<uint64_t>(1ull << 30, 4 * bytes);
  const uint64_t regions = span / bytes;
  constexpr int kGrids[] = {256, 512, 2048};
  uint8_t *buf = nullptr;
  uint32_t *out = nullptr;
  hipEvent_t start = nullptr, stop = nullptr;
  hipStream_t s = nullptr;
  auto cleanup = [&]() {
    if (s) (void)hipStreamDestroy(s);
    if (start) (void)hipEventDestroy(start);
    if (stop) (void)hipEventDestroy(stop);
    (void)hipFree(buf);
    (void)hipFree(out);
  };
  if (hipMalloc(&buf, span) != hipSuccess || hipMalloc(&out, 2048 * sizeof(uint32_t)) != hipSuccess) {
    cleanup();
    return fail(MOE_ENOMEM, "moe_probe_hbm_read: %llu-byte buffer", (unsigned long long)span);
  }
  bool ok = hipEventCreate(&start) == hipSuccess && hipEventCreate(&stop) == hipSuccess &&
            hipStreamCreateWithFlags(&s, hipStreamNonBlocking) == hipSuccess &&
            hipMemsetAsync(buf, 0x5a, span, s) == hipSuccess && hipStreamSynchronize(s) == hipSuccess;
  // average duration of `n` single launches, each timed by its own kernel events
  auto time = [&](uint64_t nbytes, int grid, int n, uint64_t &region, double &avg_us) {
    double tot = 0.0;
    for (int j = -2; ok && j < n; ++j) {  // two untimed warm-up launches
      const uint8_t *src = buf + (region++ % regions) * nbytes;
      float ms = 0.f;
      ok = launch_read_probe(src, (int64_t)nbytes, grid, out, s, Timing{start, stop}) == hipSuccess &&
           hipEventSynchronize(stop) == hipSuccess && hipEventElapsedTime(&ms, start, stop) == hipSuccess;
      if (j >= 0) tot += ms;
    }
    avg_us = 1e3 * tot / n;
  };
  uint64_t region = 0;
  double best = 0.0, empty = 0.0;
  for (int g : kGrids) {
    double us = 0.0;
    time(bytes, g, iters, region, us);
    if (ok && (best == 0.0 || us < best)) best = us;
  }
  time(0, kGrids[0], iters, region, empty);
  if (!ok) {
    cleanup();
    return fail(MOE_EHIP, "moe_probe_hbm_read: HIP call failed");
  }
  *read_us = best;
  *empty_us = empty;
  cleanup();
  return MOE_OK;
}

}  // extern "C"

namespace {

int ensure_prefill(moe_cache *c, int64_t T) {
  if (T <= c->pf_cap) return MOE_OK;
  HIP_TRY(c, hipStreamSynchronize(c->main));
  void *ptrs[] = {c->pf_inv, c->pf_xb, c->pf_counts, c->pf_off, c->pf_perm, c->pf_ab, c->pf_P};
  for (void *q : ptrs) (void)hipFree(q);
  c->pf_inv = nullptr;
  c->pf_xb = nullptr;
  c->pf_counts = c->pf_off = c->pf_perm = nullptr;
  c->pf_ab = nullptr;
  c->pf_P = nullptr;
  c->pf_cap = 0;
  const int64_t H = c->d.hidden, I = c->d.inter, E = c->d.n_experts, k = c->d.top_k;
  if (hipMalloc(&c->pf_inv, T * sizeof(float)) != hipSuccess ||
      hipMalloc(&c->pf_xb, 2 * T * H * sizeof(__bf16)) != hipSuccess ||
      hipMalloc(&c->pf_counts, group_counts_ints((int)E) * sizeof(int32_t)) != hipSuccess ||
      hipMalloc(&c->pf_off, (E + 1) * sizeof(int32_t)) != hipSuccess ||
      hipMalloc(&c->pf_perm, T * k * sizeof(int32_t)) != hipSuccess ||
      hipMalloc(&c->pf_ab, 2 * T * k * I * sizeof(__bf16)) != hipSuccess ||
      hipMalloc(&c->pf_P, T * k * H * sizeof(float)) != hipSuccess ||
      (!c->pf_host_off &&
       hipHostMalloc(&c->pf_host_off, 257 * sizeof(int32_t), hipHostMallocDefault) != hipSuccess)) {
    (void)hipGetLastError();
    return fail(MOE_ENOMEM, "cannot allocate prefill buffers for %lld tokens", (long long)T);
  }
  c->pf_cap = T;
  return MOE_OK;
}

// End of a multi-token call: routes out (debug), trace records, counter delta.
int finish_multi(moe_cache *c, int32_t T, int32_t layer, const moe_counters &before,
                 moe_counters *delta, int32_t *dbg_idx, float *dbg_w) {
  const int k = c->d.top_k;
  if (dbg_idx || dbg_w) {
    if (dbg_idx)
      HIP_TRY(c, hipMemcpyAsync(dbg_idx, c->topk_idx, (size_t)T * k * sizeof(int32_t),
                                hipMemcpyDeviceToHost, c->main));
    if (dbg_w)
      HIP_TRY(c, hipMemcpyAsync(dbg_w, c->topk_w, (size_t)T * k * sizeof(float), hipMemcpyDeviceToHost,
                                c->main));
    HIP_TRY(c, hipStreamSynchronize(c->main));
  }
  if (c->d.flags & MOE_F_TRACE) c->trace.insert(c->trace.end(), c->recs.begin(), c->recs.end());
  if (delta) {
    const moe_counters &a = c->lru[layer].counters();
    *delta = moe_counters{a.hits - before.hits, a.misses - before.misses, a.evictions - before.evictions,
                          a.materialized_bytes - before.materialized_bytes};
  }
  return MOE_OK;
}

// The FFN of a multi-token call of at most kSmallTokens tokens whose routed
// experts all hold slots after this call's table step (so no slot is reused
// inside the call): the misses' copies, then per token the decode GEMVs over
// its own top_k experts (the digits of every token formed by one kernel), all
// on the caller's stream; each token's output row is written by its down
// launch (with the residual when asked), so no combine is needed.
int small_call_ffn(moe_cache *c, const float *x, int32_t T, int32_t layer, float *y) {
  const moe_model_desc &d = c->d;
  const int k = d.top_k, E = d.n_experts, H = d.hidden, I = d.inter;
  std::vector<int32_t> slot_of(E, -1);
  std::vector<int> miss;
  for (size_t i = 0; i < c->recs.size(); ++i) {
    slot_of[c->recs[i].expert] = c->recs[i].slot;
    if (!c->recs[i].hit) miss.push_back((int)i);
  }
  const int copy_cap = max_copy();
  for (size_t m0 = 0; m0 < miss.size(); m0 += copy_cap) {
    const int n = (int)std::min<size_t>(copy_cap, miss.size() - m0);
    const uint8_t *src[256];
    uint8_t *dst[256];
    for (int q = 0; q < n; ++q) {
      const moe_step_rec &r = c->recs[miss[m0 + q]];
      src[q] = c->store + ((int64_t)layer * E + r.expert) * c->P;
      dst[q] = c->slot_ptr(layer, r.slot);
    }
    Span sp(c, c->main, MOE_KIND_COPY, n, (uint64_t)n * c->P, 0);
    if (d.flags & (MOE_F_SDMA_COPY | MOE_F_SIDE_COPY)) {
      sp.record_start();
      for (int q = 0; q < n; ++q)
        HIP_TRY(c, hipMemcpyAsync(dst[q], src[q], c->P, hipMemcpyDefault, c->main));
      sp.record_stop();
    } else {
      HIP_TRY(c, launch_materialize(src, dst, n, c->P, kCopyGrid, c->main, sp.timing()));
    }
    sp.end();
  }
  HIP_TRY(c, launch_token_digits(x, T, H, (d.flags & MOE_F_PRENORM) != 0, c->st_xq, c->st_xsc, c->main));
  const int mode = (d.flags & MOE_F_RESIDUAL) ? 1 : 0;
  for (int32_t tk = 0; tk < T; ++tk) {
    ExpertList L{};
    for (int j = 0; j < k; ++j) {
      const int32_t e = c->st_host_idx[tk * k + j];
      if (e < 0 || e >= E || slot_of[e] < 0) {
        c->poisoned = true;
        return fail(MOE_EHIP, "routes of a multi-token call name expert %d outside the table step", e);
      }
      L.payload[j] = c->slot_ptr(layer, slot_of[e]);
      L.pos[j] = j;
    }
    L.n = k;
    DecodeScratch St = c->scratch();
    St.xq = c->st_xq + (int64_t)tk * 3 * H;
    St.xsc = c->st_xsc + (int64_t)tk * (H / 32);
    {
      Span sp(c, c->main, MOE_KIND_GATEUP, 1, (uint64_t)k * 2 * c->M, 4ull * k * H * I);
      HIP_TRY(c, launch_gateup(d.qtype, St, H, I, k, L, nullptr, c->main, sp.timing()));
      sp.end();
    }
    {
      Span sp(c, c->main, MOE_KIND_DOWN, 1, (uint64_t)k * c->Md, 2ull * k * H * I);
      HIP_TRY(c, launch_down(d.qtype, St, H, I, k, L, nullptr, c->topk_w + (int64_t)tk * k,
                             x + (int64_t)tk * H, y + (int64_t)tk * H, mode, c->main, sp.timing()));
      sp.end();
    }
  }
  return MOE_OK;
}

// A multi-token layer call.  The routed experts S of all tokens go through the
// slot table once.  The experts are then processed in chunks: the copy kernel
// of a chunk's misses runs on the caller's stream while the MFMA GEMMs of
// earlier chunks run on the side stream.  A copy overwrites a slot only after
// the expert that held it (if it is routed in this call) has been computed:
// the copy stream waits for that expert's chunk, and a chunk is closed early
// when one of its own experts would be evicted by the next miss.
// Room for n per-chunk work lists.  Called after the call's routing has been
// waited for, so no earlier call's copies of these lists are still pending.
int ensure_mt_chunks(moe_cache *c, int n) {
  if (n <= c->pf_mt_cap) return MOE_OK;
  (void)hipFree(c->pf_mt_dev);
  if (c->pf_mt_host) (void)hipHostFree(c->pf_mt_host);
  c->pf_mt_dev = c->pf_mt_host = nullptr;
  c->pf_mt_cap = 0;
  if (hipMalloc(&c->pf_mt_dev, (size_t)n * sizeof(MtWork)) != hipSuccess ||
      hipHostMalloc(&c->pf_mt_host, (size_t)n * sizeof(MtWork), hipHostMallocDefault) != hipSuccess) {
    (void)hipGetLastError();
    return fail(MOE_ENOMEM, "cannot allocate %d chunk work lists", n);
  }
  c->pf_mt_cap = n;
  return MOE_OK;
}

int forward_prefill_impl(moe_cache *c, const float *x, int32_t T, const float *wr, int32_t layer,
                         float *y, moe_counters *delta, int32_t *dbg_idx, float *dbg_w) {
  const moe_model_desc &d = c->d;
  const int k = d.top_k, E = d.n_experts, H = d.hidden, I = d.inter;
  int rc = ensure_tokens(c, T);
  if (!rc) rc = ensure_prefill(c, T);
  if (rc) return rc;
  c->timing_now = (d.flags & MOE_F_TIMING) && c->n_calls++ % c->timing_every == 0;
  const bool prenorm = d.flags & MOE_F_PRENORM;
  {
    Span sp(c, c->main, MOE_KIND_ROUTER, 1, (uint64_t)H * E * 4 + (uint64_t)T * H * 4,
            2ull * T * H * E);
    sp.record_start();
    HIP_TRY(c, launch_prefill_prep(x, T, H, prenorm, c->pf_inv, c->pf_xb, c->main));
    HIP_TRY(c, launch_router_prefill(x, wr, T, H, E, k, prenorm ? c->pf_inv : nullptr, c->zbuf,
                                     c->topk_idx, c->topk_w, c->main));
    HIP_TRY(c, launch_group(c->topk_idx, T * k, E, c->pf_counts, c->pf_off, c->pf_perm, c->main));
    sp.record_stop();
    sp.end();
  }
  HIP_TRY(c, hipMemcpyAsync(c->pf_host_off, c->pf_off, (E + 1) * sizeof(int32_t), hipMemcpyDeviceToHost,
                            c->main));
  if (T <= kSmallTokens)
    HIP_TRY(c, hipMemcpyAsync(c->st_host_idx, c->topk_idx, (size_t)T * k * sizeof(int32_t),
                              hipMemcpyDeviceToHost, c->main));
  if (c->dev_lru && (rc = pull_table_queue(c, layer))) return rc;
  HIP_TRY(c, hipEventRecord(c->ev_route, c->main));
  HIP_TRY(c, hipEventSynchronize(c->ev_route));
  if (c->dev_lru) {
    if ((rc = pull_table_load(c, layer))) return rc;
    c->table_pulled = true;
  }
  if (d.flags & MOE_F_TIMING) {
    rc = drain_timing(c);
    if (rc) return rc;
  }
  const int32_t *off = c->pf_host_off;
  if (off[0] != 0 || off[E] != T * k) {
    c->poisoned = true;
    return fail(MOE_EHIP, "grouping produced offsets [%d, %d] for %d pairs", off[0], off[E], T * k);
  }
  std::vector<int32_t> S;
  for (int e = 0; e < E; ++e) {
    if (off[e + 1] < off[e]) {
      c->poisoned = true;
      return fail(MOE_EHIP, "grouping produced decreasing offsets");
    }
    if (off[e + 1] > off[e]) S.push_back(e);
  }
  SlotLru &t = c->lru[layer];
  const moe_counters before = t.counters();
  c->recs.clear();
  t.step(S.data(), (int32_t)S.size(), c->recs);
  if (T <= kSmallTokens) c->small_overflow[layer] = (int)S.size() > c->C;
  if (T <= kSmallTokens && (int)S.size() <= c->C) {
    rc = small_call_ffn(c, x, T, layer, y);
    if (rc) return rc;
    return finish_multi(c, T, layer, before, delta, dbg_idx, dbg_w);
  }

  // chunks of record indices: the hits first (no copy), then the misses in order
  struct Chunk {
    std::vector<int> recs;
    int copy_dep = -1;  // chunk whose computation must finish before this chunk's copies
  };
  const int per_chunk = std::max(1, std::min(c->C / 3, pf_max_experts()));
  std::vector<Chunk> chunks(1);
  std::vector<int> chunk_of(E, -1);
  for (size_t i = 0; i < c->recs.size(); ++i)
    if (c->recs[i].hit) {
      if ((int)chunks.back().recs.size() == pf_max_experts()) chunks.emplace_back();
      chunks.back().recs.push_back((int)i);
      chunk_of[c->recs[i].expert] = (int)chunks.size() - 1;
    }
  if (!chunks.back().recs.empty()) chunks.emplace_back();
  // miss chunks of per_chunk, the last one split so that a short chunk ends the
  // call: its GEMMs are the only ones no later copy hides
  std::vector<int> caps;
  {
    int left = 0;
    for (const auto &r : c->recs) left += r.hit ? 0 : 1;
    for (; left > 0; left -= std::min(left, per_chunk)) caps.push_back(std::min(left, per_chunk));
    const int tail = std::max(1, per_chunk / 4);
    if (!caps.empty() && caps.back() > tail) {
      caps.back() -= tail;
      caps.push_back(tail);
    }
  }
  size_t cap_i = 0;
  int misses_in_cur = 0;
  for (size_t i = 0; i < c->recs.size(); ++i) {
    const moe_step_rec &r = c->recs[i];
    if (r.hit) continue;
    const int dep = r.evicted >= 0 ? chunk_of[r.evicted] : -1;  // -1: not routed in this call
    const int cap = cap_i < caps.size() ? caps[cap_i] : per_chunk;
    if ((dep >= 0 && dep == (int)chunks.size() - 1) || misses_in_cur == cap) {
      chunks.emplace_back();
      misses_in_cur = 0;
      ++cap_i;
    }
    Chunk &ch = chunks.back();
    ch.recs.push_back((int)i);
    ch.copy_dep = std::max(ch.copy_dep, dep);
    chunk_of[r.expert] = (int)chunks.size() - 1;
    ++misses_in_cur;
  }
  while (!chunks.empty() && chunks.back().recs.empty()) chunks.pop_back();
  while (c->pf_ev.size() < 2 * chunks.size()) {
    hipEvent_t e = nullptr;
    HIP_TRY(c, hipEventCreateWithFlags(&e, hipEventDisableTiming));
    c->pf_ev.push_back(e);
  }
  // chunk i: pf_ev[2i] = its copies done (caller's stream), pf_ev[2i+1] = computed (side)
  HIP_TRY(c, hipStreamWaitEvent(c->side, c->ev_route, 0));
  // a call of at most kMtTokens tokens (here: more routed experts than slots)
  // runs each chunk's experts through the union GEMVs, fp32-accurate like the
  // decode path, instead of the bf16 GEMMs sized for many tokens: one work
  // list per chunk (its experts, their slots and the (token, rank) positions
  // routed to each), all uploaded at once, and the token digits once
  const bool mt = T <= kSmallTokens && mt_ffn_fits(d.qtype, H, I, T);
  int mt_positions = 0;
  if (mt) {
    if ((rc = ensure_mt_chunks(c, (int)chunks.size()))) return rc;
    for (size_t ci = 0; ci < chunks.size(); ++ci) {
      const Chunk &ch = chunks[ci];
      MtWork &h = c->pf_mt_host[ci];
      h.n_copy = 0;
      h.n_union = (int32_t)ch.recs.size();
      for (size_t u = 0; u < ch.recs.size(); ++u) {
        const moe_step_rec &r = c->recs[ch.recs[u]];
        h.upay[u] = c->slot_ptr(layer, r.slot);
        h.uhit[u] = 1;
        int n = 0;
        for (int q = 0; q < T * k; ++q)
          if (c->st_host_idx[q] == r.expert && n < kMtTokens) h.uq[u][n++] = (uint8_t)q;
        h.unt[u] = (uint8_t)n;
        mt_positions += n;
      }
    }
    // every (token, rank) belongs to one routed expert
    if (mt_positions != T * k) {
      c->poisoned = true;
      return fail(MOE_EHIP, "routes of a multi-token call do not match its grouping");
    }
    HIP_TRY(c, hipMemcpyAsync(c->pf_mt_dev, c->pf_mt_host, chunks.size() * sizeof(MtWork),
                              hipMemcpyHostToDevice, c->side));
    HIP_TRY(c, launch_token_digits(x, T, H, prenorm, c->st_xq, c->st_xsc, c->side));
  }
  const int copy_cap = max_copy();
  const uint64_t M = (uint64_t)c->M, Md = (uint64_t)c->Md;
  int waited = -1;
  for (size_t ci = 0; ci < chunks.size(); ++ci) {
    const Chunk &ch = chunks[ci];
    std::vector<int> miss;
    for (int q : ch.recs)
      if (!c->recs[q].hit) miss.push_back(q);
    if (!miss.empty()) {
      if (ch.copy_dep > waited) {
        HIP_TRY(c, hipStreamWaitEvent(c->main, c->pf_ev[2 * ch.copy_dep + 1], 0));
        waited = ch.copy_dep;
      }
      for (size_t m0 = 0; m0 < miss.size(); m0 += copy_cap) {
        const int n = (int)std::min<size_t>(copy_cap, miss.size() - m0);
        const uint8_t *src[256];
        uint8_t *dst[256];
        for (int q = 0; q < n; ++q) {
          const moe_step_rec &r = c->recs[miss[m0 + q]];
          src[q] = c->store + ((int64_t)layer * E + r.expert) * c->P;
          dst[q] = c->slot_ptr(layer, r.slot);
        }
        Span sp(c, c->main, MOE_KIND_COPY, n, (uint64_t)n * c->P, 0);
        if (d.flags & (MOE_F_SDMA_COPY | MOE_F_SIDE_COPY)) {
          sp.record_start();
          for (int q = 0; q < n; ++q)
            HIP_TRY(c, hipMemcpyAsync(dst[q], src[q], c->P, hipMemcpyDefault, c->main));
          sp.record_stop();
        } else {
          HIP_TRY(c, launch_materialize(src, dst, n, c->P, kCopyGrid, c->main, sp.timing()));
        }
        sp.end();
      }
      HIP_TRY(c, hipEventRecord(c->pf_ev[2 * ci], c->main));
      HIP_TRY(c, hipStreamWaitEvent(c->side, c->pf_ev[2 * ci], 0));
    }
    if (mt) {
      const MtWork &h = c->pf_mt_host[ci];
      uint64_t pos = 0;
      for (int u = 0; u < h.n_union; ++u) pos += h.unt[u];
      const int umax = h.n_union;
      {
        Span sp(c, c->side, MOE_KIND_GATEUP, 1, umax * 2 * M, pos * 4ull * H * I);
        HIP_TRY(c, launch_gateup_mt(d.qtype, c->pf_mt_dev + ci, c->st_xq, c->st_xsc, c->mt_hq, c->mt_hsc,
                                    c->mt_hds, H, I, k, T, umax, c->side, sp.timing()));
        sp.end();
      }
      {
        Span sp(c, c->side, MOE_KIND_DOWN, 1, umax * Md, pos * 2ull * H * I);
        HIP_TRY(c, launch_down_mt(d.qtype, c->pf_mt_dev + ci, c->mt_hq, c->mt_hsc, c->mt_hds, c->mt_R, H,
                                  I, k, T, umax, c->side, sp.timing()));
        sp.end();
      }
      HIP_TRY(c, hipEventRecord(c->pf_ev[2 * ci + 1], c->side));
      continue;
    }
    PfWave W{};
    uint64_t rows = 0;
    for (int q : ch.recs) {
      const moe_step_rec &r = c->recs[q];
      W.payload[W.count] = c->slot_ptr(layer, r.slot);
      W.row0[W.count] = off[r.expert];
      W.n[W.count] = off[r.expert + 1] - off[r.expert];
      rows += W.n[W.count];
      ++W.count;
    }
    {
      Span sp(c, c->side, MOE_KIND_GATEUP, 1, W.count * 2 * M, rows * 4ull * H * I);
      HIP_TRY(c, launch_pf_gateup(d.qtype, W, c->pf_perm, c->pf_xb, c->pf_ab, T, H, I, k, c->side,
                                  sp.timing()));
      sp.end();
    }
    {
      Span sp(c, c->side, MOE_KIND_DOWN, 1, W.count * Md, rows * 2ull * H * I);
      HIP_TRY(c, launch_pf_down(d.qtype, W, c->pf_perm, c->pf_ab, c->topk_w, c->pf_P, T * k, H, I,
                                c->side, sp.timing()));
      sp.end();
    }
    HIP_TRY(c, hipEventRecord(c->pf_ev[2 * ci + 1], c->side));
  }
  if (!chunks.empty()) HIP_TRY(c, hipStreamWaitEvent(c->main, c->pf_ev[2 * chunks.size() - 1], 0));
  if (mt) {
    HIP_TRY(c, launch_combine_mt(c->mt_R, c->topk_w, x, y, H, k, T, (d.flags & MOE_F_RESIDUAL) ? 1 : 0,
                                 nullptr, c->main));
  } else {
    HIP_TRY(c, launch_pf_combine(c->pf_P, x, y, T, H, k, (d.flags & MOE_F_RESIDUAL) != 0, c->main));
  }
  return finish_multi(c, T, layer, before, delta, dbg_idx, dbg_w);
}

// Prefill runs the layer's slot table on the host: with device tables, move
// the table to the host for the call and queue it back afterwards.
int forward_prefill(moe_cache *c, const float *x, int32_t T, const float *wr, int32_t layer, float *y,
                    moe_counters *delta, int32_t *dbg_idx, float *dbg_w) {
  // the trace kept on the device is moved out before the host table adds records;
  // the table itself is pulled behind the call's routing (forward_prefill_impl) and
  // pushed back only if it was pulled
  int rc = c->dev_lru ? drain_dev_trace(c) : MOE_OK;
  if (rc) return rc;
  c->table_pulled = false;
  rc = forward_prefill_impl(c, x, T, wr, layer, y, delta, dbg_idx, dbg_w);
  if (c->dev_lru && c->table_pulled) {
    const int rc2 = push_table(c, layer);
    if (!rc) rc = rc2;
  }
  return rc;
}

}  // namespace
