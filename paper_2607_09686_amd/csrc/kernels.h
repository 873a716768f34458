// Launch wrappers of the HIP kernels (internal to libmoecache).
#pragma once

#include <hip/hip_bf16.h>
#include <hip/hip_runtime.h>

#include <cstdint>

namespace moecache {

constexpr int kMaxRouted = 16;  // experts per FFN launch (top_k <= 16 in decode)

// Model type codes (desc.qtype): the format of W_gate / W_up in the low byte,
// that of W_down in the next byte (0: the same).  Formats: 8 Q8_0, 2 Q4_0
// (32 weights per block), 12 Q4_K, 14 Q6_K (256 per super-block).
inline int fmt_gate_up(int qtype) { return qtype & 0xff; }
inline int fmt_down(int qtype) { return (qtype >> 8) & 0xff ? (qtype >> 8) & 0xff : qtype & 0xff; }
inline bool fmt_known(int f) { return f == 8 || f == 2 || f == 12 || f == 14; }
inline bool fmt_kquant(int f) { return f == 12 || f == 14; }
inline int fmt_block_bytes(int f) { return f == 8 ? 34 : f == 2 ? 18 : f == 12 ? 144 : f == 14 ? 210 : 0; }
inline int fmt_block_weights(int f) { return fmt_kquant(f) ? 256 : 32; }
// the activations' digit sums are needed by a down format with a min term (Q4_K); Q4_0's offset
// is taken into its weights as signed nibbles
inline bool fmt_needs_sums(int f) { return f == 12; }
// bytes of a rows x cols matrix (rows of cols inputs) in format f
inline int64_t fmt_matrix_bytes(int f, int64_t rows, int64_t cols) {
  return rows * (cols / fmt_block_weights(f)) * fmt_block_bytes(f);
}

// Optional events recorded by the runtime right at the start of the first
// kernel and the end of the last kernel of a launch wrapper (null: none).
struct Timing {
  hipEvent_t start = nullptr, stop = nullptr;
};

struct ExpertList {
  const uint8_t *payload[kMaxRouted];  // slot holding the expert's [gate|up|down] payload
  int32_t pos[kMaxRouted];             // top-k position of the expert for token 0
  int32_t n;
};

// Work of one decode call written on the device by the slot-table step and
// read by the copy, gate/up and down kernels.
struct WorkList {
  int32_t n_copy, pad;
  const uint8_t *src[kMaxRouted];  // misses in ascending expert order
  uint8_t *dst[kMaxRouted];
  int32_t miss_pos[kMaxRouted];    // top-k position of each miss
  int32_t hit[kMaxRouted];         // per top-k position: 1 hit, 0 miss
  ExpertList list;  // the k routed experts in rank order (n = 0 after a routing error)
};

// Work of a small multi-token call (T <= kMtTokens tokens whose routed
// experts all fit the slots), written on the device by the slot-table step:
// the misses' copies in ascending expert order and, per token, the slots of
// its k experts in rank order.
constexpr int kMtTokens = 8;
constexpr int kMtMaxCopy = kMtTokens * kMaxRouted;
constexpr int kMtParts = 16;  // router partial blocks per token of such a call
constexpr int kMtMaxChunks = 8;  // chunks of a small call whose union exceeds the slots
struct MtWork {
  int32_t n_copy, n_union;
  const uint8_t *src[kMtMaxCopy];
  uint8_t *dst[kMtMaxCopy];
  ExpertList list[kMtTokens];
  // the union's experts in ascending id: slot, the number of tokens routing
  // to it and their positions q = t * k + j (token t, rank j), ascending t
  const uint8_t *upay[kMtMaxCopy];
  uint8_t unt[kMtMaxCopy];
  uint8_t uq[kMtMaxCopy][kMtTokens];
  uint8_t uhit[kMtMaxCopy];  // 1: the expert was resident before the call
  uint8_t mu[kMtMaxCopy];    // per miss (copy order): its index in the union
};

// Device-resident slot table of one layer (the rule of slot_lru.h) and where
// a call's results go.  trace: 6 int32 per record (moe_step_rec), nullable.
struct LruDev {
  int32_t *slot_of;    // [E], -1 if not resident
  int32_t *expert_in;  // [C], -1 if free
  int64_t *stamp;      // [E]
  int64_t *meta;       // [3]: clock, step number, slots in use
  uint64_t *cnt;       // [4]: hits, misses, evictions, materialised bytes
  int32_t *trace;
  uint64_t *trace_n;   // records written so far
  int32_t *err;        // set to 1 + (bad id & 0xffff) when a routed id is out of range
  const uint8_t *store;  // the layer's E payloads in the store
  uint8_t *slots;        // the layer's C slots
  WorkList *work;
  int64_t P;
  int32_t C, layer;
  float *zlast;    // [E], nullable: the call's logits are written here
  int32_t policy;  // 0 least recently used, 1 lowest logit (MOE_F_SCORE_EVICT)
};

// Decode router: one token, two launches.  partial: [grid * E + 1] fp32 scratch.
// Writes idx/w [k] to device and, if non-null, to host-mapped mirrors.
int router_decode_grid(int H);
// Also writes the digits xq [3][H] and block scales xsc [H/32] of x * s,
// s = 1/sqrt(mean(x^2)+1e-6) when prenorm else 1; the logits are scaled by s.
// With lru non-null the finishing block also runs the layer's slot-table
// step and writes lru->work (E <= 256, C <= E).
hipError_t launch_router_decode(const float *x, const float *wr, int H, int E, int k, float *partial,
                                int32_t *idx, float *w, int32_t *host_idx, float *host_w, int8_t *xq,
                                float *xsc, bool prenorm, const LruDev *lru, hipStream_t s,
                                const Timing &t = {});

// Router of a small multi-token call with the layer's table on the device
// (lru.slot_of set, 1 <= T <= kMtTokens): per token, the decode router's
// partials over at most kMtParts blocks of rows, s and digits (partial: T
// regions of at most kMtParts * E + 1 floats; xq [T][3][H], xsc [T][H/32])
// and routes idx / w [T][k]; then one
// table step over the union of the routed experts, written to mw, unless
// that union exceeds the slots.  flag[0] (host memory) becomes 0 (done), 1
// (union too large: table untouched, mw empty) or 2 (routing failure);
// flag[1] the union's size.
// mw: max_chunks work lists (1 <= max_chunks <= kMtMaxChunks); flag: host
// memory [3] (verdict, union size, chunks).
hipError_t launch_router_small(const float *x, const float *wr, int T, int H, int E, int k, float *partial,
                               int32_t *idx, float *w, int8_t *xq, float *xsc, bool prenorm,
                               const LruDev &lru, MtWork *mw, int32_t *flag, int max_chunks, hipStream_t s,
                               const Timing &t = {});

// The FFN of a small multi-token call from its work list, each union expert's
// weights read once: gate/up for all the tokens routing to an expert
// (activations at position q = t*k + j of hq [3][T*k*I], hsc [T*k*I/16], hds
// [3][T*k*I/16]), down into R [T*k][H] (unweighted rows), then y_t =
// (x_t if mode 1) + sum over j in rank order of w[t*k+j] R[t*k+j].  The
// numerics are those of the decode GEMVs (launch_gateup / launch_down per
// token); combine does nothing when W (nullable) is a device list left empty
// by the table step.  umax: an upper bound on the union size (the grids); false from
// mt_ffn_fits: a shape these kernels do not take.
bool mt_ffn_fits(int qtype, int H, int I, int T);
size_t mt_gateup_lds(int H, int T);
hipError_t launch_gateup_mt(int qtype, const MtWork *W, const int8_t *xq, const float *xsc, int8_t *hq,
                            float *hsc, int32_t *hds, int H, int I, int k, int T, int umax,
                            hipStream_t s, const Timing &t = {});
hipError_t launch_down_mt(int qtype, const MtWork *W, const int8_t *hq, const float *hsc,
                          const int32_t *hds, float *R, int H, int I, int k, int T, int umax,
                          hipStream_t s, const Timing &t = {});
hipError_t launch_combine_mt(const float *R, const float *w, const float *x, float *y, int H, int k,
                             int T, int mode, const MtWork *W, hipStream_t s, const Timing &t = {});

// Prefill router: partial logits over router_slices(T) slices of H into
// z [slices][T][E] (router_zbuf_floats(T, E) floats cover any call of at most
// T tokens), then per token z = tscale[t] * (sum of slices) (tscale
// nullable) and top-k rows into idx/w [T][k].
int router_slices(int T);
int64_t router_zbuf_floats(int64_t T, int E);
hipError_t launch_router_prefill(const float *x, const float *wr, int T, int H, int E, int k,
                                 const float *tscale, float *z, int32_t *idx, float *w, hipStream_t s);

// The decode GEMVs' input form for T tokens: digits xq [T][3][H] and block
// scales xsc [T][H/32] of x_t * s_t (s_t = 1/rms of x_t when prenorm, else 1),
// formed exactly as the decode router forms one token's.
hipError_t launch_token_digits(const float *x, int T, int H, bool prenorm, int8_t *xq, float *xsc,
                               hipStream_t s);

// Prefill.  inv[t] = 1/rms (or 1) and xb [2][T][H] = x * inv as bf16 hi and lo terms.
hipError_t launch_prefill_prep(const float *x, int T, int H, bool prenorm, float *inv, __bf16 *xb,
                               hipStream_t s);
// Stable grouping of the T*k (token, expert) pairs by expert: counts (scratch of
// group_counts_ints(E) ints), offsets [E+1], perm [T*k] (pair ids t*k + j).
int group_counts_ints(int E);
hipError_t launch_group(const int32_t *idx, int npairs, int E, int32_t *counts, int32_t *offsets,
                        int32_t *perm, hipStream_t s);
// The experts of one wave (count <= pf_max_experts()).
struct PfWave {
  const uint8_t *payload[256];
  int32_t row0[256], n[256];
  int32_t count;
};
int pf_max_experts();
int max_copy();  // payloads per launch_materialize call
// ab: [2][T*k][I] activations as bf16 hi and lo terms (rows in perm order).
hipError_t launch_pf_gateup(int qtype, const PfWave &W, const int32_t *perm, const __bf16 *xb,
                            __bf16 *ab, int T, int H, int I, int k, hipStream_t s,
                            const Timing &t = {});
hipError_t launch_pf_down(int qtype, const PfWave &W, const int32_t *perm, const __bf16 *ab,
                          const float *w, float *P, int pairs, int H, int I, hipStream_t s,
                          const Timing &t = {});
hipError_t launch_pf_combine(const float *P, const float *x, float *y, int T, int H, int k,
                             bool residual, hipStream_t s);

// Device scratch of the decode FFN (owned by the cache handle).
struct DecodeScratch {
  int8_t *xq;   // [3][H] digits of the (scaled) token, written by the router
  float *xsc;   // [H/32]
  int8_t *hq;   // [3][k*I] digits of the SwiGLU activations, written by gate/up
  float *hsc;   // [k*I/16] their 16-wide block scales
  int32_t *hds; // [3][k*I/16] digit sums of those blocks (down format Q4_K)
};

// Decode FFN.  Gate/up writes the activations of its rows, as digits of
// 16-wide blocks, at each listed expert's top-k position; down stages them
// (n * I <= 12288).  mode of down: 0 y = sum, 1 y = x + sum, 2 y += sum.
// With Ld non-null the kernels read the list from device memory (L.n is then
// only the launch size; a device list with n = 0 makes them do nothing).
hipError_t launch_gateup(int qtype, const DecodeScratch &S, int H, int I, int k, const ExpertList &L,
                         const ExpertList *Ld, hipStream_t s, const Timing &t = {});
hipError_t launch_down(int qtype, const DecodeScratch &S, int H, int I, int k, const ExpertList &L,
                       const ExpertList *Ld, const float *w, const float *x, float *y, int mode,
                       hipStream_t s, const Timing &t = {});

// Decode copy + gate/up in one launch (device work list): `copy_blocks` blocks
// stream the misses' payloads host -> slot and form the SwiGLU activations of
// the missed experts from the gate/up rows they carry; further blocks run
// gate/up for the hit experts from their slots meanwhile.  Writes the same
// activation digits as launch_gateup.  Returns hipErrorInvalidValue for a
// shape it does not take (fusable_copy_gateup false).
bool fusable_copy_gateup(int qtype, int H, int I);
hipError_t launch_copy_gateup(int qtype, const DecodeScratch &S, int H, int I, int k,
                              const WorkList *w, int64_t payload_bytes, int copy_blocks,
                              uint64_t *acc, hipStream_t s, const Timing &t = {});

// The same for a small multi-token call (device work list MtWork): the
// misses' copies with their tokens' activations formed from the copied
// rows, and gate/up of the union's hit experts alongside.  Writes the same
// activation digits as launch_gateup_mt.  Returns hipErrorInvalidValue for a
// shape it does not take (fusable_copy_gateup_mt false).
bool fusable_copy_gateup_mt(int qtype, int H, int I, int T);
hipError_t launch_copy_gateup_mt(int qtype, const MtWork *W, const int8_t *xq, const float *xsc,
                                 int8_t *hq, float *hsc, int32_t *hds, int H, int I, int k, int T,
                                 int umax, int64_t payload_bytes, int copy_blocks, uint64_t *acc,
                                 hipStream_t s, const Timing &t = {});

// Copy n <= max_copy() payloads of `bytes` (multiple of 16, 16-byte aligned)
// src[i] -> dst[i] with a copy kernel of `grid` blocks (host-pinned or device sources).
hipError_t launch_materialize(const uint8_t *const *src, uint8_t *const *dst, int n, int64_t bytes,
                              int grid, hipStream_t s, const Timing &t = {});
// The copies a device work list names (n_copy of them); acc (nullable) gets
// += copies, += bytes.
hipError_t launch_materialize_list(const WorkList *w, int64_t bytes, int grid, uint64_t *acc,
                                   hipStream_t s, const Timing &t = {});
hipError_t launch_materialize_list(const MtWork *w, int64_t bytes, int grid, uint64_t *acc,
                                   hipStream_t s, const Timing &t = {});

// Reference launch (probe.hip): a plain streaming read of `bytes` (multiple of
// 16) from device memory src by `grid` blocks of 256 threads, one word per
// block to out [grid]; bytes == 0 launches an empty kernel instead.
hipError_t launch_read_probe(const uint8_t *src, int64_t bytes, int grid, uint32_t *out, hipStream_t s,
                             const Timing &t = {});

// One layer's slot table to / from a pinned host staging buffer of
// table_stage_bytes(E, C) bytes (stamp [E] i64 | meta [3] i64 | cnt [4] u64 |
// err i32 | pad | slot_of [E] i32 | expert_in [C] i32), one kernel each way;
// the pack also copies the device error word.
size_t table_stage_bytes(int E, int C);
hipError_t launch_table_pack(const LruDev &L, int E, int C, const int32_t *err, uint8_t *stage,
                             hipStream_t s);
hipError_t launch_table_unpack(const LruDev &L, int E, int C, const uint8_t *stage, hipStream_t s);

}  // namespace moecache
