/*
 * moecache: routed-expert MoE FFN over a bounded per-layer expert-slot cache,
 * for AMD Instinct MI355X (gfx950).  C ABI.
 *
 * The method is MawForge's bounded expert materialisation (arXiv 2607.09686):
 * the full set of routed-expert weights stays in a large backing store; each
 * MoE layer owns a fixed number of slots for expert weight blocks; the router
 * decides which experts a token needs; a needed expert that holds no slot is
 * copied ("materialised") into one, and the expert-to-slot map is updated
 * (the paper's Native Serving Path section; the store layout follows its
 * Split-Pack section: one block of bytes per layer and expert).
 *
 * Here the backing store is pinned host memory, the slots are HBM, and a
 * layer call does, in order:
 *   1. router logits z = x W_r, top-k by (-z, id), softmax over the chosen k;
 *   2. LRU slot-table lookup with hit / miss / eviction counters (decode: in
 *      device memory, stepped by the router's last kernel; prefill and the
 *      SIDE/SDMA copy modes: on the host);
 *   3. the misses' copies host -> slot (decode: one copy kernel, fused with the
 *      gate/up of every routed expert; or hipMemcpyAsync per miss);
 *   4. fused dequantise + SwiGLU gate/up, then down projection with the
 *      routing-weighted combine (and optional residual add).
 *
 * Conventions for every function below:
 *   - returns MOE_OK (0) or a negative MOE_E* code; moe_last_error() then
 *     holds a message for the calling thread;
 *   - no C++ exception crosses this boundary;
 *   - after MOE_EHIP the handle is poisoned: every later call on it returns
 *     MOE_ESTATE, and only moe_cache_destroy is meaningful;
 *   - one handle must not be used from two threads at once.
 */
#ifndef MOECACHE_H
#define MOECACHE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define MOE_OK 0
#define MOE_EINVAL (-1) /* bad argument: shape, pointer, range */
#define MOE_ENOMEM (-2) /* device or pinned-host allocation failed */
#define MOE_EHIP (-3)   /* a HIP runtime call failed (text in moe_last_error) */
#define MOE_ESTATE (-4) /* handle poisoned by an earlier MOE_EHIP */
#define MOE_EIO (-5)    /* a file could not be opened, read or written */

/* Block formats of the expert weights (GGUF; the paper's model profiles are
 * Q8_0 and Q4_K_M GGUF files, its Model Profiles section).
 * Q8_0: 34 bytes per 32 weights = fp16 scale d (little-endian) + 32 int8 q;
 *       weight d*q.
 * Q4_0: 18 bytes per 32 weights = fp16 scale d + 16 bytes, byte j holding
 *       element j in its low nibble and element j+16 in its high nibble;
 *       weight d*(n-8).
 * Q4_K: 144 bytes per super-block of 256 weights = fp16 d, fp16 dmin, 12
 *       bytes of eight 6-bit sub-block scales sc_j and mins m_j, 128 bytes of
 *       4-bit q (chunk c of 64 weights: 32 bytes, low nibbles sub-block 2c,
 *       high nibbles 2c+1); weight d*sc_j*q - dmin*m_j.
 * Q6_K: 210 bytes per super-block of 256 weights = 128 bytes of low 4 bits,
 *       64 bytes of high 2 bits, 16 int8 scales (one per 16 weights), fp16 d;
 *       weight d*scale*(q-32).
 * desc.qtype names the format of W_gate and W_up in its low byte and that of
 * W_down in the next byte, 0 meaning the same (MOE_QTYPE_MIX).  The K-quant
 * formats need hidden (their gate/up rows) or inter (their down rows) to be a
 * multiple of 256. */
#define MOE_Q8_0 8
#define MOE_Q4_0 2
#define MOE_Q4_K 12
#define MOE_Q6_K 14
#define MOE_QTYPE_MIX(gate_up, down) ((gate_up) | ((down) << 8))
/* the paper's 4-bit profile as stored here: Q4_K gate/up, Q6_K down */
#define MOE_Q4_K_M MOE_QTYPE_MIX(MOE_Q4_K, MOE_Q6_K)

/* desc.flags */
#define MOE_F_RESIDUAL 1u /* y = x + moe(x) instead of y = moe(x) */
#define MOE_F_TRACE 2u    /* keep one moe_step_rec per routed expert per call */
#define MOE_F_TIMING 4u   /* bracket router, FFN kernels and copies with HIP events */
#define MOE_F_PRENORM 8u  /* route and run the experts on x / sqrt(mean(x^2) + 1e-6) (per
                             token, unit gain); the residual of MOE_F_RESIDUAL adds raw x */
/* How decode copies the missed experts into their slots (default: one copy
 * kernel for all of a call's misses on the caller's stream, then gate/up and
 * down over all routed experts; nothing crosses streams): */
#define MOE_F_SIDE_COPY 16u /* hipMemcpyAsync per miss on a library side stream while the
                               hit experts run on the caller's stream, which then waits
                               for the copies before the missed experts */
#define MOE_F_SDMA_COPY 32u /* hipMemcpyAsync per miss on the caller's stream (copy
                               engine instead of the copy kernel) */
#define MOE_F_SPLIT_COPY 64u /* decode, default copy mode: the copy kernel and gate/up as
                                two launches instead of one launch that copies the misses
                                and runs gate/up for every routed expert (results equal) */
/* Slot policy (default: least recently used, the rule of moe_lru_step): */
#define MOE_F_SCORE_EVICT 128u /* a miss with every slot taken evicts the resident, outside
                                  the call, whose router logit for the call's token is lowest
                                  (ties: the higher id): the expert the current token wants
                                  least, as a guess at the next token's routes.  Decode with
                                  the default copy modes only: moe_cache_create rejects it with
                                  MOE_F_SIDE_COPY / MOE_F_SDMA_COPY, and a multi-token call on
                                  such a handle returns MOE_EINVAL */

typedef struct moe_cache moe_cache; /* opaque, owned by the library */

typedef struct {
  int32_t n_layers;  /* MoE layers, >= 1 */
  int32_t n_experts; /* routed experts per layer, 1..256 */
  int32_t top_k;     /* experts per token, 1..min(n_experts, 16) */
  int32_t hidden;    /* H, model width, multiple of 64, <= 8192 */
  int32_t inter;     /* I, expert intermediate width, multiple of 64, <= 8192;
                        top_k * inter <= 12288 (decode activations live in LDS) */
  int32_t qtype;     /* MOE_Q8_0, MOE_Q4_0, MOE_Q4_K, MOE_Q6_K, or MOE_QTYPE_MIX of the two
                        K-quant formats (MOE_Q4_K_M); K-quants: hidden (gate/up) and inter
                        (down) multiples of 256 */
  /* Expert store, caller-owned, must outlive the handle and stay unchanged.
   * Layout: for layer l and expert e a payload of P bytes at offset
   * (l*n_experts + e)*P, P = 2*M + Md with M = inter*(hidden/w)*block_bytes
   * and Md = hidden*(inter/w_d)*block_bytes_d (w = 32 or 256 weights per block
   * of the matrix's format):
   *   [W_gate: inter rows x hidden | W_up: inter x hidden | W_down: hidden x inter]
   * each row-major, one row per output, a row = its inputs as consecutive
   * blocks (or super-blocks).  Must be pinned host memory from hipHostMalloc (e.g.
   * moe_host_alloc); device memory is accepted too.  Pageable memory is
   * rejected with MOE_EINVAL. */
  const void *host_store;
  uint64_t store_bytes; /* must equal n_layers*n_experts*P */
  void *hip_stream;     /* caller's hipStream_t for all compute; NULL = null stream */
  uint32_t flags;       /* MOE_F_* */
} moe_model_desc;

typedef struct {
  uint64_t hits;               /* routed distinct experts found in a slot */
  uint64_t misses;             /* routed distinct experts copied into a slot */
  uint64_t evictions;          /* misses that displaced a resident expert */
  uint64_t materialized_bytes; /* always misses * P */
} moe_counters;

/* One slot-table decision.  Within a layer call, records come in ascending
 * expert id; step counts that layer's calls from 0 (reset by moe_cache_reset). */
typedef struct {
  int32_t layer, step, expert;
  int32_t hit;     /* 1 hit, 0 miss */
  int32_t slot;    /* slot the expert occupies after the call, 0..budget_slots-1 */
  int32_t evicted; /* expert displaced by this miss, or -1 */
} moe_step_rec;

/* Per-kind totals of the MOE_F_TIMING events (kinds below). */
typedef struct {
  uint64_t launches; /* kernel launches, or copies for MOE_KIND_COPY */
  double total_ms;   /* sum of event-bracketed durations */
  uint64_t bytes;    /* algorithmic bytes moved by those launches / copies */
  uint64_t flops;    /* algorithmic floating-point operations */
} moe_kernel_stats;
#define MOE_KIND_ROUTER 0 /* router logits + top-k kernel(s) */
#define MOE_KIND_GATEUP 1 /* fused dequant + gate/up + SwiGLU */
#define MOE_KIND_DOWN 2   /* dequant + down projection + weighted combine */
#define MOE_KIND_COPY 3   /* miss materialisation copies (host to device) */
#define MOE_KIND_COUNT 4

/* Create a cache with budget_slots slots per layer (top_k <= budget_slots <=
 * n_experts), all empty: the fixed per-layer slot tensors of the paper's
 * Native Serving Path section, one slot holding one expert's whole block
 * (gate, up and down), sized once from the budget and never grown.  Allocates n_layers*budget_slots*P bytes of HBM for
 * the slots plus small scratch, on the current HIP device.  MOE_EINVAL on a
 * bad descriptor, MOE_ENOMEM if the slots do not fit. */
int moe_cache_create(const moe_model_desc *desc, int32_t budget_slots, moe_cache **out);

/* One MoE layer call for n_tokens tokens (the Native Serving Path section's
 * per-layer work).
 *   x        device, [n_tokens][hidden] fp32, read only
 *   router_w device, [hidden][n_experts] fp32 row-major (z = x W_r)
 *   layer    0..n_layers-1
 *   y        device, [n_tokens][hidden] fp32, written; must not overlap x
 *   delta    host, nullable: this call's counter increments
 * n_tokens == 1 takes the decode path (GEMV kernels on fp32 activations held
 * as three int8 digits per value).  n_tokens > 1: the routed experts of all
 * tokens go through the slot table once; then a call of at most 8 tokens whose
 * distinct experts fit the slots runs the decode GEMVs once per token (same
 * numerics as decode), and any other call the prefill path (bf16 MFMA grouped
 * GEMM: weights rounded to bf16, x and the SwiGLU activations carried as two
 * bf16 terms, fp32 accumulation); there n_tokens * max(hidden, top_k * inter)
 * must be <= 2^34 (MOE_EINVAL otherwise).
 * Work is queued on desc.hip_stream and y is ready when that stream passes
 * this call.  Decode with the default copy kernel does not block the host:
 * the layer's slot table lives in device memory and is stepped by the
 * router's last kernel.  A routing failure there (no finite logit among the
 * top_k) makes the call do no work and is returned by the next call that
 * synchronises (a call with delta or routes, counters, trace, stats, reset or
 * a prefill call), which poisons the handle.  The SIDE/SDMA copy modes and
 * prefill block until the routes are known.  A non-NULL delta makes the call
 * wait for its own completion.  Routing reads x, so x must be ready on that
 * stream. */
int moe_layer_forward(moe_cache *c, const float *x, int32_t n_tokens, const float *router_w,
                      int32_t layer, float *y, moe_counters *delta);

/* For callers that cannot allocate device memory during a call (code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc):
 * moe_layer_forward for one token (n_tokens must be 1; MOE_EINVAL otherwise)
 * with the same arguments, results, counters and trace, whose per-call
 * scratch -- router partials, routes, the token's and the activations' digit
 * staging, the call's work list -- lives in a static device array of the
 * library (1 MiB per GPU, held until the process ends) instead of the
 * handle's buffers.  It calls no hipMalloc, hipFree or other allocating
 * routine; with delta NULL it queues its kernels on desc.hip_stream and
 * returns without waiting.  Needs the device slot tables (the default copy
 * modes: MOE_EINVAL with MOE_F_SIDE_COPY / MOE_F_SDMA_COPY) and a shape whose
 * scratch fits the array (MOE_EINVAL otherwise; every shape moe_cache_create
 * accepts does).  Every call on one GPU shares that GPU's array, whichever
 * handle and stream it comes from: calls that overlap in time on one GPU race
 * (the array keeps the last call's contents; nothing in it needs clearing,
 * each call writes what it reads first). */
int moe_layer_forward_static(moe_cache *c, const float *x, int32_t n_tokens, const float *router_w,
                             int32_t layer, float *y, moe_counters *delta);

/* As moe_layer_forward, also copying the routes out (host, nullable):
 * topk_idx [n_tokens][top_k] int32 in rank order, topk_w [n_tokens][top_k] fp32. */
int moe_layer_forward_dbg(moe_cache *c, const float *x, int32_t n_tokens, const float *router_w,
                          int32_t layer, float *y, moe_counters *delta, int32_t *topk_idx,
                          float *topk_w);

/* Counters since creation or the last reset: one layer, or layer = -1 for the sum.
 * These are the cache figures the paper's serving telemetry reports (hit rate
 * and materialised expert bytes; its Native Serving Path and Measurements
 * sections): hit rate = hits / (hits + misses), one lookup per distinct routed
 * expert of a layer call. */
int moe_cache_counters(const moe_cache *c, int32_t layer, moe_counters *out);

/* Move up to cap kept records (MOE_F_TRACE) into buf, oldest first; *n_out
 * gets the number moved.  Records not moved stay for the next read.  A record
 * is one decision of the route-to-slot update the paper's Native Serving Path
 * section describes (hit, or the slot a miss was copied into and the expert it
 * displaced), so a run's cache behaviour can be replayed and checked. */
int moe_cache_read_trace(moe_cache *c, moe_step_rec *buf, int64_t cap, int64_t *n_out);

/* Empty every slot, zero counters, drop the trace and timing totals: the cold
 * cache every run of the paper's validation matrix starts from (its
 * Experimental Method section).  Synchronises with the handle's streams first. */
int moe_cache_reset(moe_cache *c);

/* Overwrite every byte of every slot of every layer with `byte` (0..255),
 * leaving the slot tables as they are.  For tests: after moe_cache_reset (all
 * slots empty) with byte 0xFF, every block scale in a slot reads as a NaN
 * until the slot's expert has been copied in, so a kernel that reads a slot
 * before its copy has landed, or a slot it was not given, shows up as a
 * non-finite output.  Synchronises with the handle's streams first.
 * MOE_EINVAL for byte outside 0..255. */
int moe_cache_fill_slots(moe_cache *c, int32_t byte);

/* Totals of one MOE_KIND_* since creation or reset (needs MOE_F_TIMING).
 * Synchronises with the handle's streams first. */
int moe_cache_kernel_stats(moe_cache *c, int32_t kind, moe_kernel_stats *out);

/* With MOE_F_TIMING, bracket only one layer call in every `every` (>= 1,
 * default 1) with events, so the timing itself barely perturbs the run. */
int moe_cache_set_timing_stride(moe_cache *c, int32_t every);

/* Router logits of the last one-token call, z [n_experts] fp32 (host), as the
 * slot-table step saw them (scaled by the MOE_F_PRENORM factor when set; zeros
 * before the first call).  Decode with the default copy modes only, else
 * MOE_EINVAL.  Synchronises with the handle's streams first. */
int moe_cache_last_logits(moe_cache *c, float *z);

/* Waits for the handle's work, frees everything the library allocated. NULL-safe. */
void moe_cache_destroy(moe_cache *c);

/* Message of the last failed call on this thread ("" if none). */
const char *moe_last_error(void);

/* Pinned (page-locked) host memory suitable as desc.host_store, via
 * hipHostMalloc.  MOE_ENOMEM if it cannot be pinned. */
int moe_host_alloc(uint64_t bytes, void **out);
int moe_host_free(void *p);

/* Host-to-device bandwidth of the copy path used for misses: n_chunks copies
 * of chunk_bytes each, read consecutively from host_src (pinned), spread
 * round-robin over n_streams new streams into one device buffer, timed with
 * HIP events from the first copy to the last.  *gb_per_s = bytes / time. */
int moe_probe_h2d(const void *host_src, uint64_t chunk_bytes, int32_t n_chunks, int32_t n_streams,
                  double *gb_per_s);

/* Reference durations for the short HBM-bound kernels (the decode down
 * GEMV reads 13 MB per launch, where a launch's fixed cost is a large part of
 * its duration): *read_us = the average duration of a plain streaming read of
 * `bytes` (multiple of 16, at most 1 GiB) from device memory in one launch,
 * best of three grid sizes, each launch reading a different region of a
 * buffer at least four times the last-level cache so that its bytes come from
 * HBM; *empty_us = the same for an empty kernel.  Durations come from the
 * runtime's kernel start/end stamps, as the library's own span timings do;
 * `iters` launches per measurement (1..10000).  The probe allocates and frees
 * its own buffer (max(1 GiB, 4 * bytes)) and stream on the current device.
 * MOE_EINVAL on a bad argument, MOE_ENOMEM if the buffer cannot be had,
 * MOE_EHIP on a HIP failure. */
int moe_probe_hbm_read(uint64_t bytes, int32_t iters, double *read_us, double *empty_us);

/* Static budget plan (no HIP dependency, no allocation).  The paper's Native
 * Serving Path section derives the slot count of the routed layers from the
 * requested cache bytes, the routed layer count, the bytes of one expert block,
 * the active experts per token and the experts per layer; its Static Budget
 * Check section bounds the serving footprint from below,
 *   L(p, n) = C + E(p) + K(n)          F(p, n) = L(p, n) + O
 * (C resident common tensors, E(p) the expert cache at cache percentage p,
 * K(n) the KV cache at context n, O runtime overhead) and rejects a
 * configuration whose L already exceeds the serving target.  Here every layer
 * gets the same slot count s, clamped to [top_k, n_experts], so
 * E = n_layers * s * payload_bytes, and K(n) = n * kv_bytes_per_token.
 * All sizes in bytes.  Both functions return MOE_EINVAL (no message) on a bad
 * argument or when a size overflows 64 bits, MOE_OK otherwise. */
typedef struct {
  int32_t n_layers;            /* routed MoE layers, >= 1 */
  int32_t n_experts;           /* experts per layer, >= 1 */
  int32_t top_k;               /* active experts per token, 1..n_experts: the fewest slots
                                  a layer can work with */
  int32_t pad;
  uint64_t payload_bytes;      /* one expert block = one slot, >= 1 */
  uint64_t common_bytes;       /* C */
  uint64_t kv_bytes_per_token; /* K(n) / n */
  uint64_t overhead_bytes;     /* O */
  uint64_t target_bytes;       /* serving target the lower bound is checked against */
} moe_plan_in;

typedef struct {
  int32_t slots_per_layer;     /* s */
  int32_t clamped;             /* 1 if the budget asked for fewer than top_k or more than
                                  n_experts slots and s was clamped */
  uint64_t expert_cache_bytes; /* E = n_layers * s * payload_bytes */
  uint64_t kv_bytes;           /* K(n) */
  uint64_t lower_bound_bytes;  /* L = C + E + K(n) */
  uint64_t footprint_bytes;    /* F = L + O */
  int32_t feasible;            /* 1 if L <= target_bytes, 0 if the plan is rejected */
  int32_t pad;
} moe_plan_out;

/* Cache as a percentage of each layer's experts, 0 < percent <= 100:
 * s = nearest integer to percent/100 * n_experts, halves rounding up
 * (computed in double as floor((2 * percent * n_experts + 100) / 200));
 * 15, 35 and 75 % of 128 experts give 19, 45 and 96 slots. */
int moe_plan_percent(const moe_plan_in *in, double percent, int64_t context_tokens,
                     moe_plan_out *out);

/* Cache as a byte budget for all routed layers: s = floor(cache_bytes /
 * (n_layers * payload_bytes)). */
int moe_plan_bytes(const moe_plan_in *in, uint64_t cache_bytes, int64_t context_tokens,
                   moe_plan_out *out);

/* Offline bound on misses (no HIP dependency): Belady's MIN for per-call expert
 * sets.  For one layer's recorded calls -- call i routes ids[offsets[i] ..
 * offsets[i+1]) (any order, duplicates allowed, each id in [0, n_experts);
 * offsets[0] = 0, n_calls + 1 entries) -- *misses gets the fewest misses any
 * slot policy with n_slots slots can have from a cold cache, each call's
 * distinct experts being resident together: on a miss with every slot taken,
 * evict the resident outside the call whose next use is farthest ahead.  The
 * paper asks for a policy that minimises latency under a memory budget (its
 * Discussion); with slots that do not compete with host memory the latency
 * of a call follows the bytes it materialises, which this bounds.  MOE_EINVAL
 * on a bad argument or a call routing more than n_slots distinct experts. */
int moe_policy_min(const int32_t *ids, const int64_t *offsets, int64_t n_calls, int32_t n_experts,
                   int32_t n_slots, uint64_t *misses);

/* Split-pack of a GGUF MoE model (no HIP dependency; the paper's Split-Pack
 * Representation section): the routed expert tensors of every layer l,
 * blk.l.ffn_{gate,up,down}_exps.weight (Q8_0, Q4_0, Q4_K or Q6_K, gate and up of
 * one type and down of one type in every layer; dims (H, I, E), (H, I, E),
 * (I, H, E), innermost first), are cut into one block per (layer, expert) and
 * written to pack_path in the store layout of moe_model_desc.host_store:
 * payload (l, e) at (l * n_experts + e) * P, [W_gate | W_up | W_down], bytes
 * unchanged.  index_path gets one JSON line with the topology, one per block
 * (layer, expert, offset and bytes in the pack, the source offset and bytes of
 * each of the three matrices, an FNV-1a 64-bit digest of the block) and a last
 * line with the block count, the pack size and a digest of the block digests.
 * info->qtype is the desc.qtype of the pack (MOE_QTYPE_MIX when the down type
 * differs).  router_path (nullable) gets the routers, blk.l.ffn_gate_inp.weight (F32, F16
 * or BF16, dims (H, E)), as fp32 [n_layers][hidden][n_experts], the router_w
 * form of moe_layer_forward.  info gets the topology (top_k from the metadata
 * key *.expert_used_count, 0 if absent).  GGUF versions 2 and 3.  MOE_EINVAL
 * on a malformed file, missing or inconsistent tensors, another block type, a
 * block type that changes between layers, or widths above 65536; MOE_EIO when
 * a file cannot be opened, read or written; MOE_ENOMEM when host memory runs
 * out. */
typedef struct {
  int32_t n_layers, n_experts, top_k, hidden, inter, qtype;
  uint64_t payload_bytes; /* P */
  uint64_t pack_bytes;    /* n_layers * n_experts * P */
} moe_pack_info;
int moe_pack_gguf(const char *gguf_path, const char *pack_path, const char *index_path,
                  const char *router_path, moe_pack_info *info);

/* The slot table alone, with no HIP dependency (used to check it on the CPU):
 * the route-to-slot map of the paper's Native Serving Path section, whose
 * eviction choice the paper leaves open (here least recently used per layer).
 * Same rule as inside moe_layer_forward: for one call with routed experts ids
 * (any order, duplicates allowed), stamp the distinct ids in ascending order,
 * count hits, then give each miss (ascending) the lowest free slot or the slot
 * of the resident expert with the smallest stamp. */
typedef struct moe_lru moe_lru;
int moe_lru_create(int32_t n_experts, int32_t n_slots, uint64_t payload_bytes, int32_t layer,
                   moe_lru **out);
/* out: room for n records (one per distinct id is written); *n_out = records written. */
int moe_lru_step(moe_lru *lru, const int32_t *ids, int32_t n, moe_step_rec *out, int32_t *n_out);
int moe_lru_counters(const moe_lru *lru, moe_counters *out);
void moe_lru_destroy(moe_lru *lru);

#ifdef __cplusplus
}
#endif

#endif /* MOECACHE_H */
