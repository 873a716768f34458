// HIP kernels of the expert-slot-cache MoE layer for gfx950 (CDNA4, wave64).
//
// Router: z = x W_r (fp32), top-k by (-z, id) with wave shuffles, softmax over
// the chosen k.  Decode FFN: block-dequant GEMV straight from the GGUF-style
// Q8_0 / Q4_0 blocks in the slots.  The fp32 input vector of a GEMV is first
// split, per 32-wide block b with scale s_b = max|v|/127, into three int8
// "digits" v = s_b (D1 + D2/254 + D3/254^2) + O(6e-8 max|v|); each block's
// dot product with the int8 (or 4-bit) weights is then three exact int32
// dot4 sums, recombined in fp32 and scaled by d * s_b.  Fixed summation
// order throughout: results do not depend on scheduling.
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdint>

#include "kernels.h"

namespace moecache {
namespace {

constexpr int kThreads = 256;
constexpr int kWave = 64;

// MFMA operand and accumulator vectors.
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ float half_bits_to_float(uint32_t bits16) {
  _Float16 h;
  uint16_t b = (uint16_t)bits16;
  __builtin_memcpy(&h, &b, 2);
  return (float)h;
}

// (value, id) order used for routing: larger value first, lower id on ties.
__device__ __forceinline__ bool better(float v, int id, float bv, int bid) {
  return v > bv || (v == bv && id < bid);
}

// Top-k over z[0..E) by one wave (E <= 256).  Writes ids in rank order and the
// softmax over the chosen logits (idx2/w2: optional further copies of them).
// Must be called by all 64 lanes of a wave.
__device__ void wave_topk(const float *z, int E, int k, int32_t *idx, float *w, int32_t *idx2,
                          float *w2) {
  const int lane = threadIdx.x & (kWave - 1);
  float v[4];
  int taken = 0;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    int e = lane + kWave * j;
    v[j] = e < E ? z[e] : -INFINITY;
  }
  float sel_z = 0.f;
  int sel_id = 0;
  float my_z = 0.f;
  int my_id = 0;
  for (int r = 0; r < k; ++r) {
    float bv = -INFINITY;
    int bid = 0x7fffffff;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      int e = lane + kWave * j;
      if (e < E && !(taken >> j & 1) && better(v[j], e, bv, bid)) {
        bv = v[j];
        bid = e;
      }
    }
#pragma unroll
    for (int off = kWave / 2; off >= 1; off >>= 1) {
      float ov = __shfl_xor(bv, off, kWave);
      int oid = __shfl_xor(bid, off, kWave);
      if (better(ov, oid, bv, bid)) {
        bv = ov;
        bid = oid;
      }
    }
    if ((bid & (kWave - 1)) == lane) taken |= 1 << (bid / kWave);
    if (r == 0) sel_z = bv;  // the largest chosen logit
    if (lane == r) {
      my_z = bv;
      my_id = bid;
    }
    sel_id = bid;
  }
  (void)sel_id;
  float ex = lane < k ? expf(my_z - sel_z) : 0.f;
  float sum = ex;
#pragma unroll
  for (int off = kWave / 2; off >= 1; off >>= 1) sum += __shfl_xor(sum, off, kWave);
  if (lane < k) {
    float wi = ex / sum;
    idx[lane] = my_id;
    w[lane] = wi;
    if (idx2) idx2[lane] = my_id;
    if (w2) w2[lane] = wi;
  }
}

// The three int8 digits of v in a block of scale s, given rs = 1/s (0 for an
// all-zero block): with t = v rs, D1 = rint(t), D2 = rint(254 (t - D1)),
// D3 = rint(254 (254 (t - D1) - D2)).
__device__ __forceinline__ void digits_of(float v, float rs, int &d1, int &d2, int &d3) {
  const float t = v * rs;
  const float a = __builtin_rintf(t);
  const float r1 = (t - a) * 254.f;
  const float b = __builtin_rintf(r1);
  const float c = __builtin_rintf((r1 - b) * 254.f);
  d1 = (int)fminf(127.f, fmaxf(-127.f, a));
  d2 = (int)fminf(127.f, fmaxf(-127.f, b));
  d3 = (int)fminf(127.f, fmaxf(-127.f, c));
}

// Digits of a 32-wide block held by an aligned group of 8 lanes, four
// consecutive values per lane: s = max|v|/127 over the block (three xor
// shuffles; a max is exact in any order), then the digits of the lane's four
// values packed into one dword per plane (byte j = value j).  Returns s
// (0 for an all-zero block, digits 0).  All 8 lanes of the group call it.
__device__ __forceinline__ float octet_digits(float4 v, uint32_t (&dw)[3]) {
  float m = fmaxf(fmaxf(fabsf(v.x), fabsf(v.y)), fmaxf(fabsf(v.z), fabsf(v.w)));
  m = fmaxf(m, __shfl_xor(m, 1, kWave));
  m = fmaxf(m, __shfl_xor(m, 2, kWave));
  m = fmaxf(m, __shfl_xor(m, 4, kWave));
  const float s = m * (1.f / 127.f);
  const float rs = m > 0.f ? 127.f * __builtin_amdgcn_rcpf(m) : 0.f;
  const float vv[4] = {v.x, v.y, v.z, v.w};
  dw[0] = dw[1] = dw[2] = 0u;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    int d1, d2, d3;
    digits_of(vv[j], rs, d1, d2, d3);
    dw[0] |= ((uint32_t)d1 & 0xffu) << (8 * j);
    dw[1] |= ((uint32_t)d2 & 0xffu) << (8 * j);
    dw[2] |= ((uint32_t)d3 & 0xffu) << (8 * j);
  }
  return s;
}

// Dot product of four signed byte pairs plus c.  Where c is a known zero (the
// first term of a chain) the saturating form is used: it takes the zero as an
// inline constant, while the accumulating form the compiler picks otherwise
// needs the zero moved into its destination register first.  Four products
// of bytes stay far inside int32, so the saturation never acts.
__device__ __forceinline__ int sdot4(uint32_t a, uint32_t b, int c) {
  if (__builtin_constant_p(c) && c == 0) return __builtin_amdgcn_sdot4((int)a, (int)b, 0, true);
  return __builtin_amdgcn_sdot4((int)a, (int)b, c, false);
}

// ---------------------------------------------------------------- router ---

constexpr int kRouterRowsPerBlock = 32;

constexpr int kMaxX4 = 8;  // H <= 8192

// Decode router, first kernel: block (b, t) accumulates token t's z over rows [rpb b, rpb b + rpb)
// of W_r into partial[b][E] (no cross-block communication inside a launch:
// on a multi-XCD GPU a device-scope fence costs more than a second launch).
// Every block also forms s = 1/sqrt(mean(x^2) + 1e-6) (or 1) from the whole x,
// in the same order, so all blocks hold the same s; block b writes the digits
// of its 32-wide blocks of x * s, and block 0 writes s at partial[nb * E].
// Thread (c, ph) takes column c and rows r0 + ph + phases j in order.  MULTI:
// blocks of rpb rows (a multiple of 32) for multi-token calls, 32 rows per
// thread per round trip; else 32 rows per block, J of them per thread (J =
// 32 for E > 128, else 16 >= ceil(32 / phases)).  Every load is issued
// unconditionally at a clamped, valid address and the values outside the
// block's rows are zeroed afterwards (a guarded load becomes a branch), so
// the sums are those of the rows in order.
template <bool MULTI, int J>
__global__ __launch_bounds__(kThreads) void router_partial_kernel(
    const float *__restrict__ x, const float *__restrict__ wr, int H, int E, int prenorm, int rpb,
    float *__restrict__ partial, int8_t *__restrict__ xq, float *__restrict__ xsc) {
  __shared__ float red[kThreads];
  __shared__ float wsum[kThreads / kWave];
  {  // token blockIdx.y of a multi-token call: its own x row, partials, s and digits
    const int t = blockIdx.y;
    x += (int64_t)t * H;
    partial += (int64_t)t * ((int64_t)gridDim.x * E + 1);
    xq += (int64_t)t * 3 * H;
    xsc += (int64_t)t * (H / 32);
  }
  const int tid = threadIdx.x;
  const int phases = kThreads / E;  // E <= 256
  const int c = tid % E, ph = tid / E;
  const int rows = MULTI ? rpb : kRouterRowsPerBlock;
  const int r0 = blockIdx.x * rows;
  const int r1 = min(H, r0 + rows);
  const int H4 = H / 4;
  const float4 *x4 = reinterpret_cast<const float4 *>(x);
  float acc = 0.f;
  float xv[J], wv[J];
  auto load_rows = [&](int j0) {
#pragma unroll
    for (int j = 0; j < J; ++j) {
      const int r = r0 + ph + phases * (j0 + j);
      const int rc = min(r, r1 - 1);
      xv[j] = x[rc];
      wv[j] = wr[(int64_t)rc * E + c];
    }
  };
  auto add_rows = [&](int j0) {
#pragma unroll
    for (int j = 0; j < J; ++j) {
      const uint32_t keep = ph < phases && r0 + ph + phases * (j0 + j) < r1 ? ~0u : 0u;
      acc = fmaf(__uint_as_float(__float_as_uint(xv[j]) & keep), __uint_as_float(__float_as_uint(wv[j]) & keep),
                 acc);
    }
  };
  if constexpr (MULTI) {
    for (int j0 = 0; j0 * phases < rows; j0 += J) {
      load_rows(j0);
      add_rows(j0);
    }
  } else {
    load_rows(0);  // all loads first
  }
  float4 xa[kMaxX4];  // (zeroed where unused only at the use: overwriting a load's
                      // destination register would wait for the load)
#pragma unroll
  for (int m = 0; m < kMaxX4; ++m) xa[m] = x4[min(tid + m * kThreads, H4 - 1)];
  const int oct = MULTI ? (r1 - r0) / 32 : 1;  // the block's 32-wide blocks of x, an octet of lanes each
  const float4 mine = x4[min(r0 / 4 + tid, H4 - 1)];
  if constexpr (!MULTI) add_rows(0);
  float ss = 0.f;
#pragma unroll
  for (int m = 0; m < kMaxX4; ++m) {
    const uint32_t keep = prenorm && tid + m * kThreads < H4 ? ~0u : 0u;  // a mask, not a branch
    const float4 v = make_float4(__uint_as_float(__float_as_uint(xa[m].x) & keep),
                                 __uint_as_float(__float_as_uint(xa[m].y) & keep),
                                 __uint_as_float(__float_as_uint(xa[m].z) & keep),
                                 __uint_as_float(__float_as_uint(xa[m].w) & keep));
    ss = fmaf(v.x, v.x, ss);
    ss = fmaf(v.y, v.y, ss);
    ss = fmaf(v.z, v.z, ss);
    ss = fmaf(v.w, v.w, ss);
  }
#pragma unroll
  for (int off = kWave / 2; off >= 1; off >>= 1) ss += __shfl_xor(ss, off, kWave);
  if ((tid & (kWave - 1)) == 0) wsum[tid / kWave] = ss;
  red[tid] = acc;
  __syncthreads();
  float tot = 0.f;
#pragma unroll
  for (int i = 0; i < kThreads / kWave; ++i) tot += wsum[i];
  const float inv = prenorm ? 1.f / sqrtf(tot / (float)H + 1e-6f) : 1.f;
  if (tid < E) {
    float sum = 0.f;
    for (int p = 0; p < phases; ++p) sum += red[p * E + tid];
    partial[blockIdx.x * E + tid] = sum;
  }
  if (tid < 8 * oct) {  // octet o: values r0 + 32 o .. + 31
    const float4 v = make_float4(mine.x * inv, mine.y * inv, mine.z * inv, mine.w * inv);
    uint32_t dw[3];
    const float sc = octet_digits(v, dw);
#pragma unroll
    for (int p = 0; p < 3; ++p) reinterpret_cast<uint32_t *>(xq + (int64_t)p * H + r0)[tid] = dw[p];
    if ((tid & 7) == 0) xsc[r0 / 32 + tid / 8] = sc;
  }
  if (blockIdx.x == 0 && tid == 0) partial[(int64_t)gridDim.x * E] = inv;
}

// The decode GEMVs' input for each of T tokens: s = 1/sqrt(mean(x_t^2) + 1e-6)
// (or 1), formed as in router_partial_kernel, and the digits of x_t * s in
// 32-wide blocks: xq [T][3][H], xsc [T][H/32].  Block (bx, t): token t's
// values [1024 bx, 1024 bx + 1024), one octet of lanes per 32-wide block.
__global__ __launch_bounds__(kThreads) void token_digits_kernel(const float *__restrict__ x, int H,
                                                                int prenorm, int8_t *__restrict__ xq,
                                                                float *__restrict__ xsc) {
  __shared__ float wsum[kThreads / kWave];
  const int tid = threadIdx.x, t = blockIdx.y;
  const int H4 = H / 4;
  const float4 *x4 = reinterpret_cast<const float4 *>(x + (int64_t)t * H);
  float4 xa[kMaxX4];
#pragma unroll
  for (int m = 0; m < kMaxX4; ++m) {
    const int i = tid + m * kThreads;
    xa[m] = prenorm && i < H4 ? x4[i] : make_float4(0.f, 0.f, 0.f, 0.f);
  }
  const int q = blockIdx.x * kThreads + tid;  // this lane's float4
  const float4 mine = q < H4 ? x4[q] : make_float4(0.f, 0.f, 0.f, 0.f);
  float ss = 0.f;
#pragma unroll
  for (int m = 0; m < kMaxX4; ++m) {
    ss = fmaf(xa[m].x, xa[m].x, ss);
    ss = fmaf(xa[m].y, xa[m].y, ss);
    ss = fmaf(xa[m].z, xa[m].z, ss);
    ss = fmaf(xa[m].w, xa[m].w, ss);
  }
#pragma unroll
  for (int off = kWave / 2; off >= 1; off >>= 1) ss += __shfl_xor(ss, off, kWave);
  if ((tid & (kWave - 1)) == 0) wsum[tid / kWave] = ss;
  __syncthreads();
  float tot = 0.f;
#pragma unroll
  for (int i = 0; i < kThreads / kWave; ++i) tot += wsum[i];
  const float inv = prenorm ? 1.f / sqrtf(tot / (float)H + 1e-6f) : 1.f;
  const float4 v = make_float4(mine.x * inv, mine.y * inv, mine.z * inv, mine.w * inv);
  uint32_t dw[3];
  const float sc = octet_digits(v, dw);  // all lanes (an octet never straddles the end: H % 32 == 0)
  if (q < H4) {
    int8_t *row = xq + (int64_t)t * 3 * H;
#pragma unroll
    for (int p = 0; p < 3; ++p) reinterpret_cast<uint32_t *>(row + (int64_t)p * H)[q] = dw[p];
    if ((tid & 7) == 0) xsc[(int64_t)t * (H / 32) + q / 8] = sc;
  }
}

// Order-preserving bits of a routing logit: a larger value means a larger
// logit (NaN taken as -inf, -0 as +0).  Never 0: the bits of -inf are
// 0x007fffff, the smallest.
__device__ __forceinline__ uint32_t logit_bits(float z) {
  z = z != z ? -INFINITY : z + 0.f;
  const uint32_t u = __float_as_uint(z);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// 64-bit rank key of expert e with logit z: its logit bits above 255 - e, so
// that a larger key means a larger logit, then a lower id.
__device__ __forceinline__ uint64_t rank_key(float z, int e) {
  return ((uint64_t)logit_bits(z) << 8) | (uint64_t)(255 - e);
}

// Largest x over a full wave (all 64 lanes active): DPP lane swaps xor 1 and
// xor 2, then the mirrors inside each 8 and each 16 lanes, which leave every
// row of 16 lanes holding its maximum; the four row maxima are read out.
__device__ __forceinline__ uint32_t wave_max_u32(uint32_t x) {
  x = max(x, (uint32_t)__builtin_amdgcn_update_dpp((int)x, (int)x, 0xb1, 0xf, 0xf, false));
  x = max(x, (uint32_t)__builtin_amdgcn_update_dpp((int)x, (int)x, 0x4e, 0xf, 0xf, false));
  x = max(x, (uint32_t)__builtin_amdgcn_update_dpp((int)x, (int)x, 0x141, 0xf, 0xf, false));
  x = max(x, (uint32_t)__builtin_amdgcn_update_dpp((int)x, (int)x, 0x140, 0xf, 0xf, false));
  const uint32_t a = (uint32_t)__builtin_amdgcn_readlane((int)x, 15);
  const uint32_t b = (uint32_t)__builtin_amdgcn_readlane((int)x, 31);
  const uint32_t c = (uint32_t)__builtin_amdgcn_readlane((int)x, 47);
  const uint32_t d = (uint32_t)__builtin_amdgcn_readlane((int)x, 63);
  return max(max(a, b), max(c, d));
}

// Top-k of one token by one full wave over its logits z[0..E) and their bits
// zb = logit_bits(z) (E <= 256, 1 <= k <= 16, k <= E): k rounds of a wave
// maximum of the bits, the lowest expert id among equal bits (so the order of
// rank_key: larger logit first, lower id on a tie), then the softmax over the
// chosen logits (the first is the largest; the sum in butterfly order).  Lane
// r < k returns the expert of rank r in sel and its id and weight in id / wt
// (id 0x7fffffff and weight 0 in every lane if a chosen logit is not finite,
// which *bad records).
__device__ __forceinline__ void wave_topk_bits(const uint32_t *zb, const float *z, int E, int k, int32_t &sel,
                                               int32_t &id, float &wt, int32_t *bad) {
  const int lane = threadIdx.x & (kWave - 1);
  uint32_t h[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) h[j] = lane + kWave * j < E ? zb[lane + kWave * j] : 0u;
  int mine = 0, first = 0;
  for (int r = 0; r < k; ++r) {
    const uint32_t m = wave_max_u32(max(max(h[0], h[1]), max(h[2], h[3])));
    int e = 0;
#pragma unroll
    for (int j = 3; j >= 0; --j) {  // the lowest id holding m
      const uint64_t b = __ballot(h[j] == m);
      if (b) e = kWave * j + __builtin_ctzll(b);
    }
    if (lane == r) mine = e;
    if (r == 0) first = e;
#pragma unroll
    for (int j = 0; j < 4; ++j) h[j] = e == kWave * j + lane ? 0u : h[j];  // taken
  }
  const float z0 = z[first], zl = lane < k ? z[mine] : 0.f;
  const bool ok = __ballot(lane < k && !isfinite(zl)) == 0;
  const float ex = lane < k && ok ? expf(zl - z0) : 0.f;
  float sum = ex;
#pragma unroll
  for (int off = kWave / 2; off >= 1; off >>= 1) sum += __shfl_xor(sum, off, kWave);
  sel = mine;
  id = ok ? mine : 0x7fffffff;
  wt = ok ? ex / sum : 0.f;
  if (lane == 0 && !ok) *bad = 1;
}

// The slot table's words that a step reads and rewrites: clock, step, slots
// in use, trace records written, and the four counters.  Lane i < 8 of a
// finishing block loads word i (a vector load at a valid address for every
// lane, so that nothing waits for it before the call's other loads are out);
// table_word_keep() drops the word of lanes that hold none, at the use.
__device__ __forceinline__ int64_t table_word_load(const LruDev &lru) {
  const int i = threadIdx.x;
  const int64_t *p = i < 3 ? lru.meta + i
                     : i == 3 ? (lru.trace ? reinterpret_cast<const int64_t *>(lru.trace_n) : lru.meta)
                     : i < 8 ? reinterpret_cast<const int64_t *>(lru.cnt) + (i - 4)
                             : lru.meta;
  return *p;
}
__device__ __forceinline__ void table_word_keep(const LruDev &lru, int64_t v, int64_t *words) {
  const int i = threadIdx.x;
  if (i < 8) words[i] = i == 3 && !lru.trace ? 0 : v;
}

// Slot-table step of one layer call inside a one-block kernel (all threads;
// thread tid < E is expert tid, inS marks the call's routed set S).  The rule
// of the host table: stamp S in ascending order; a routed expert holding a
// slot is a hit; misses in ascending order take the lowest free slot, else
// the slot of the resident outside S with the smallest eviction key (the
// stamp: least recently used first; or, with lru.policy, the current rank key
// zkey: lowest logit first, the higher id on a tie).  Stamps are unique and S
// is stamped after every other resident, so the victims are the residents
// outside S in key order, for the misses beyond the free slots in expert
// order.  Writes the table, the counters, the clock and the trace records;
// returns this expert's miss flag, final slot, rank among the misses and the
// number of misses.  |S| <= C.  In two parts: step_publish (every thread,
// before a block barrier: the per-wave counts of S and of the misses, and
// the eviction keys cleared), then table_step after that barrier.
struct StepLds {
  int32_t cnt[2][kThreads / kWave];
  uint64_t key[256];  // eviction key of each slot's resident (candidates only)
  int32_t vic[256], vsl[256];
};
struct StepResult {
  bool miss;
  int fs, rS, rM, nM;
};
__device__ __forceinline__ void step_publish(const LruDev &lru, bool inS, int so, StepLds &sh) {
  const int tid = threadIdx.x, lane = tid & (kWave - 1), wv = tid / kWave;
  const uint64_t bS = __ballot(inS), bM = __ballot(inS && so < 0);
  if (lane == 0) {
    sh.cnt[0][wv] = __popcll(bS);
    sh.cnt[1][wv] = __popcll(bM);
  }
  for (int sl = tid; sl < lru.C; sl += kThreads) sh.key[sl] = UINT64_MAX;
}
__device__ __forceinline__ StepResult table_step(const LruDev &lru, int E, bool inS, int so, int64_t st,
                                                 uint64_t zkey, const int64_t *words, StepLds &sh) {
  const int tid = threadIdx.x, lane = tid & (kWave - 1), wv = tid / kWave;
  const int64_t clock0 = words[0], step = words[1], used = words[2];
  const uint64_t tn = (uint64_t)words[3];
  const bool miss = inS && so < 0;
  const bool cand = tid < E && so >= 0 && !inS;
  const uint64_t bS = __ballot(inS), bM = __ballot(miss), lt = (1ull << lane) - 1ull;
  int rS = __popcll(bS & lt), rM = __popcll(bM & lt), nM = 0, nS = 0;
#pragma unroll
  for (int v = 0; v < kThreads / kWave; ++v) {
    if (v < wv) {
      rS += sh.cnt[0][v];
      rM += sh.cnt[1][v];
    }
    nS += sh.cnt[0][v];
    nM += sh.cnt[1][v];
  }
  const uint64_t vkey = !cand ? 0ull : lru.policy ? zkey : (uint64_t)st;
  if (cand) sh.key[so] = vkey;
  const int nfree = lru.C - (int)used;
  const int nev = max(0, nM - nfree);
  __syncthreads();
  bool evicted = false;
  if (cand && nev > 0) {
    int cr = 0;  // residents outside S evicted before this one
    int sl = 0;
    for (; sl + 8 <= lru.C; sl += 8) {  // eight independent LDS reads per step
      uint64_t v[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) v[j] = sh.key[sl + j];
#pragma unroll
      for (int j = 0; j < 8; ++j) cr += v[j] < vkey ? 1 : 0;
    }
    for (; sl < lru.C; ++sl) cr += sh.key[sl] < vkey ? 1 : 0;
    if (cr < nev) {
      evicted = true;
      sh.vic[cr] = tid;
      sh.vsl[cr] = so;
    }
  }
  __syncthreads();
  int fs = so, fev = -1;
  if (miss) {
    if (rM < nfree) {
      fs = (int)used + rM;
    } else {
      fs = sh.vsl[rM - nfree];
      fev = sh.vic[rM - nfree];
    }
  }
  if (evicted) lru.slot_of[tid] = -1;
  if (inS) {
    lru.stamp[tid] = clock0 + rS + 1;
    if (miss) {
      lru.slot_of[tid] = fs;
      lru.expert_in[fs] = tid;
    }
    if (lru.trace) {
      int32_t *r = lru.trace + 6 * (int64_t)(tn + rS);
      r[0] = lru.layer;
      r[1] = (int32_t)step;
      r[2] = tid;
      r[3] = miss ? 0 : 1;
      r[4] = fs;
      r[5] = fev;
    }
  }
  if (tid == 0) {  // (the counters as read at the kernel's start: no load here, at the end)
    lru.cnt[0] = (uint64_t)words[4] + (uint64_t)(nS - nM);
    lru.cnt[1] = (uint64_t)words[5] + (uint64_t)nM;
    lru.cnt[2] = (uint64_t)words[6] + (uint64_t)nev;
    lru.cnt[3] = (uint64_t)words[7] + (uint64_t)nM * (uint64_t)lru.P;
    lru.meta[0] = clock0 + nS;
    lru.meta[1] = step + 1;
    lru.meta[2] = used + min(nM, nfree);
    if (lru.trace) *lru.trace_n = tn + (uint64_t)nS;
  }
  return StepResult{miss, fs, rS, rM, nM};
}

// Decode router, second kernel (one block): the token's logits z = s * (the
// partial sums in block order; s at partial[nb * E]), its top-k by rank (an
// expert's rank is the number of experts with a larger rank key, counted by
// all threads at once) and the softmax over the chosen logits, and with
// lru.slot_of set the layer's slot-table step and the work list.  Every
// global load is issued first, unconditionally at valid addresses (a guarded
// load becomes a branch with its own wait), the table's words as vector
// loads (a scalar load would be waited for before the partials' loads go
// out); the softmax and every global store but the step's come after the
// step.  A non-finite chosen logit is a routing failure: the error word is
// set and the work list left empty.
__global__ __launch_bounds__(kThreads) void router_finish_kernel(
    const float *__restrict__ partial, int nb, int E, int k, int32_t *idx, float *w,
    int32_t *host_idx, float *host_w, LruDev lru) {
  __shared__ float redL[kThreads];
  __shared__ int32_t cntL[kThreads];
  __shared__ float zL[256];
  __shared__ uint64_t keyL[256];
  __shared__ int32_t selL[kMaxRouted];
  __shared__ int64_t wordsL[8];
  __shared__ StepLds sl;
  __shared__ int32_t badL;
  const int tid = threadIdx.x, lane = tid & (kWave - 1);
  const bool dev = lru.slot_of != nullptr;
  // (without a table the state loads read the partials and are dropped)
  const int ce = min(tid, E - 1);
  const int64_t *p64 = reinterpret_cast<const int64_t *>(partial);
  int so = *(dev ? lru.slot_of + ce : reinterpret_cast<const int32_t *>(partial));
  int64_t st = *(dev ? lru.stamp + ce : p64);
  const int64_t word = dev ? table_word_load(lru) : *p64;
  const float inv = partial[(int64_t)nb * E];
  // thread (c, ph) adds blocks [ph * per, ph * per + per) of expert c in block order
  const int phases = kThreads / E;
  const int c = tid % E, ph = tid / E;
  const int per = (nb + phases - 1) / phases;
  const int b0 = ph * per, b1 = ph < phases ? min(nb, b0 + per) : b0;
  float sacc = 0.f;
  for (int b = b0; b < b1; b += 48) {  // one round trip for up to 48 partials per lane
    float v[48];
#pragma unroll
    for (int j = 0; j < 48; ++j) v[j] = partial[(int64_t)min(b + j, nb - 1) * E + c];
#pragma unroll
    for (int j = 0; j < 48; ++j) sacc += b + j < b1 ? v[j] : 0.f;
  }
  if (!dev || tid >= E) {
    so = -1;
    st = 0;
  }
  if (dev) table_word_keep(lru, word, wordsL);
  redL[tid] = sacc;
  if (tid == 0) badL = 0;
  __syncthreads();
  float z = 0.f;
  if (tid < E) {
    for (int p = 0; p < phases; ++p) z += redL[p * E + tid];
    z *= inv;
    zL[tid] = z;
    keyL[tid] = rank_key(z, tid);
  }
  __syncthreads();
  {  // thread (c, ph): experts in [ph E / phases, (ph + 1) E / phases) with a larger key than c's
    int r = 0;
    if (ph < phases) {
      const uint64_t kc = keyL[c];
      const int f0 = ph * E / phases, f1 = (ph + 1) * E / phases;
      int f = f0;
      for (; f + 16 <= f1; f += 16) {  // sixteen independent LDS reads per step
        uint64_t v[16];
#pragma unroll
        for (int j = 0; j < 16; ++j) v[j] = keyL[f + j];
#pragma unroll
        for (int j = 0; j < 16; ++j) r += v[j] > kc ? 1 : 0;
      }
      for (; f < f1; ++f) r += keyL[f] > kc ? 1 : 0;
    }
    cntL[tid] = r;
  }
  __syncthreads();
  int rank = E;
  if (tid < E) {
    rank = 0;
    for (int p = 0; p < phases; ++p) rank += cntL[p * E + tid];
  }
  const bool inS = rank < k;
  if (inS) {
    selL[rank] = tid;
    if (!isfinite(z)) badL = 1;
  }
  if (dev) step_publish(lru, inS, so, sl);
  __syncthreads();
  const bool bad = badL != 0;
  StepResult o{false, -1, 0, 0, 0};
  if (dev && !bad) {  // uniform
    o = table_step(lru, E, inS, so, st, tid < E ? keyL[tid] : 0ull, wordsL, sl);
    if (inS) {
      lru.work->hit[rank] = o.miss ? 0 : 1;
      if (o.miss) {
        lru.work->src[o.rM] = lru.store + (int64_t)tid * lru.P;
        lru.work->dst[o.rM] = lru.slots + (int64_t)o.fs * lru.P;
        lru.work->miss_pos[o.rM] = rank;
      }
      lru.work->list.payload[rank] = lru.slots + (int64_t)o.fs * lru.P;
      lru.work->list.pos[rank] = rank;
    }
  }
  if (tid < kWave) {
    // the softmax over the chosen logits (the first is the largest), the sum
    // in the order of a butterfly over lanes xor 32, 16, 8, 4, 2, 1 where
    // lanes >= k add zeros: with k <= 16 the steps 32 and 16 add +0, and the
    // rotations by 8, 4, 2, 1 inside each row of 16 lanes pair every lane
    // with one holding the same value as its xor partner
    const int e = lane < k ? selL[lane] : 0;
    const float ex = lane < k && !bad ? expf(zL[e] - zL[selL[0]]) : 0.f;
    float sum = ex;
    sum += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(sum), 0x128, 0xf, 0xf, false));
    sum += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(sum), 0x124, 0xf, 0xf, false));
    sum += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(sum), 0x122, 0xf, 0xf, false));
    sum += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(sum), 0x121, 0xf, 0xf, false));
    if (lane < k) {
      const int32_t id = bad ? 0x7fffffff : e;
      const float wt = bad ? 0.f : ex / sum;
      idx[lane] = id;
      w[lane] = wt;
      if (host_idx) host_idx[lane] = id;
      if (host_w) host_w[lane] = wt;
    }
  }
  if (lru.zlast && tid < E) lru.zlast[tid] = z;
  if (dev && tid == 0) {
    if (bad) {  // no work for this call; reported at the next synchronisation
      *lru.err = 1;
      lru.work->n_copy = 0;
      lru.work->list.n = 0;
    } else {
      lru.work->list.n = k;
      lru.work->n_copy = o.nM;
    }
  }
}

// Router of a small multi-token call (T <= kMtTokens), second kernel (one
// block): every token's logits (the decode router's sums), top-k and softmax
// by one wave per token, then one slot-table step for the union S of the
// tokens' routed experts (the rule of slot_lru.h) and the work lists.
//
// When |S| exceeds the slots, misses beyond the free slots and the slots of
// the residents outside S take, in ascending order, the slot of the resident
// member of S with the smallest stamp, i.e. the lowest id among the members
// holding a slot at that point (stamps follow the ids): slots are reused
// inside the call.  The experts are then computed in chunks, each chunk's
// copies, gate/up and down after the previous chunk's: a miss goes into the
// chunk after the one of the expert whose slot it takes (and not before the
// previous miss), every other expert into chunk 0.  mw[c] holds chunk c's
// copies and union experts.  With more than max_chunks chunks the table is
// left untouched and mw[0] empty.  flag (host memory) gets [0] 0 (done), 1
// (left to the caller: too many chunks) or 2 (routing failure, also in the
// error word), [1] the union's size and [2] the number of chunks.
__global__ __launch_bounds__(kThreads) void router_finish_mt_kernel(
    const float *__restrict__ partial, int nb, int T, int E, int k, int32_t *idx, float *w, LruDev lru,
    MtWork *mw, int32_t *flag, int max_chunks) {
  __shared__ float redL[kThreads * kMtTokens];  // [phase][token][expert] partial sums (phases * E <= 256)
  __shared__ float zL[kMtTokens][256];
  __shared__ uint32_t zbL[kMtTokens][256];
  __shared__ StepLds sl;
  __shared__ int32_t selL[kMtTokens][kMaxRouted];
  __shared__ uint32_t tokL[256];   // bit t: token t routes the expert
  __shared__ int32_t slotL[256], uL[256];  // per expert: slot at placement, index in its chunk's union
  __shared__ int32_t chunkL[256];           // per expert: chunk
  __shared__ uint8_t goneL[256];            // member of S whose slot a later miss takes
  __shared__ int32_t missL[kMtMaxCopy], mslotL[kMtMaxCopy], mevL[kMtMaxCopy];  // per miss, in order
  __shared__ uint64_t resL[kThreads / kWave];  // members of S holding a slot once the free and
                                              // outside residents' slots are taken
  __shared__ int32_t ccntL[kThreads / kWave][kMtMaxChunks];  // per wave and chunk: experts
  __shared__ int32_t rfirstL[kMtMaxChunks + 1];              // first miss of each chunk
  __shared__ int32_t nchunkL;
  __shared__ int64_t wordsL[8];
  __shared__ int32_t badL;
  const int tid = threadIdx.x, lane = tid & (kWave - 1), wv = tid / kWave;
  // the table state and words first (vector loads at clamped addresses,
  // as in router_finish_kernel)
  const int ce = min(tid, E - 1);
  int so = lru.slot_of[ce];
  int64_t st = lru.stamp[ce];
  const int64_t word = table_word_load(lru);
  if (tid == 0) badL = 0;
  tokL[tid] = 0u;
  goneL[tid] = 0;
  chunkL[tid] = 0;
  // every token's partials in one round trip (nb <= kMtParts): thread (c, ph)
  // adds, per token, blocks [ph * per, ph * per + per) of expert c in block
  // order (unconditional loads at clamped, valid addresses, selected
  // afterwards: a guarded load becomes a branch with its own wait)
  const int64_t pstride = (int64_t)nb * E + 1;
  const int phases = kThreads / E;
  const int c = tid % E, ph = tid / E;
  const int per = (nb + phases - 1) / phases, b0 = ph * per, b1 = min(nb, b0 + per);
  float v[kMtTokens][kMtParts], iv[kMtTokens];
#pragma unroll
  for (int t = 0; t < kMtTokens; ++t) {
    const int64_t tb = (int64_t)min(t, T - 1) * pstride;
#pragma unroll
    for (int j = 0; j < kMtParts; ++j) v[t][j] = partial[tb + (int64_t)min(b0 + j, nb - 1) * E + c];
    iv[t] = partial[tb + (int64_t)nb * E];
  }
#pragma unroll
  for (int t = 0; t < kMtTokens; ++t) {
    float a = 0.f;
#pragma unroll
    for (int j = 0; j < kMtParts; ++j) a += t < T && ph < phases && b0 + j < b1 ? v[t][j] : 0.f;
    if (t < T && ph < phases) redL[(ph * kMtTokens + t) * E + c] = a;
  }
  if (tid >= E) {
    so = -1;
    st = 0;
  }
  table_word_keep(lru, word, wordsL);
  __syncthreads();
  // z = s * (sum over the phases in order), as the decode router forms it
  if (tid < E) {
#pragma unroll
    for (int t = 0; t < kMtTokens; ++t) {
      if (t < T) {
        float z = 0.f;
        for (int p = 0; p < phases; ++p) z += redL[(p * kMtTokens + t) * E + tid];
        z *= iv[t];
        zL[t][tid] = z;
        zbL[t][tid] = logit_bits(z);
      }
    }
  }
  __syncthreads();
  for (int t = wv; t < T; t += kThreads / kWave) {
    int32_t sel, id;
    float wt;
    wave_topk_bits(zbL[t], zL[t], E, k, sel, id, wt, &badL);
    if (lane < k) {
      idx[t * k + lane] = id;
      w[t * k + lane] = wt;
      selL[t][lane] = id;
      if (id >= 0 && id < E) atomicOr(&tokL[id], 1u << t);
    }
  }
  __syncthreads();
  const bool inS = tid < E && tokL[tid] != 0u;
  step_publish(lru, inS, so, sl);
  const int nS = __syncthreads_count(inS);
  if (badL) {  // uniform
    if (tid < T) mw->list[tid].n = 0;
    if (tid == 0) {
      mw->n_copy = 0;
      mw->n_union = 0;
      *lru.err = 1;
      flag[1] = nS;
      flag[2] = 0;
      __threadfence_system();
      flag[0] = 2;
    }
    return;
  }
  // the step's counts (as table_step): rank in S, rank among the misses
  const int64_t clock0 = wordsL[0], step = wordsL[1], used = wordsL[2];
  const uint64_t tn = (uint64_t)wordsL[3];
  const int C = lru.C;
  const bool miss = inS && so < 0;
  const bool res = tid < E && so >= 0 && !inS;  // residents outside S
  const uint64_t lt = (1ull << lane) - 1ull;
  int rS = __popcll(__ballot(inS) & lt), rM = __popcll(__ballot(miss) & lt), nM = 0;
#pragma unroll
  for (int v = 0; v < kThreads / kWave; ++v) {
    if (v < wv) {
      rS += sl.cnt[0][v];
      rM += sl.cnt[1][v];
    }
    nM += sl.cnt[1][v];
  }
  const int nfree = C - (int)used;
  const int q = C - (nS - nM);                  // misses placed without taking a slot of S
  const int nev = max(0, min(nM, q) - nfree);   // residents outside S evicted
  const uint64_t vkey = res ? (uint64_t)st : 0ull;
  if (res) sl.key[so] = vkey;
  __syncthreads();
  bool evicted = false;
  if (res && nev > 0) {
    int cr = 0;
    int i = 0;
    for (; i + 8 <= C; i += 8) {
      uint64_t v[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) v[j] = sl.key[i + j];
#pragma unroll
      for (int j = 0; j < 8; ++j) cr += v[j] < vkey ? 1 : 0;
    }
    for (; i < C; ++i) cr += sl.key[i] < vkey ? 1 : 0;
    if (cr < nev) {
      evicted = true;
      sl.vic[cr] = tid;
      sl.vsl[cr] = so;
    }
  }
  __syncthreads();
  // placements that take a free slot or an outside resident's; the members of
  // S holding a slot after them
  if (inS) slotL[tid] = so;
  if (miss) {
    missL[rM] = tid;
    if (rM < q) {
      const int fs = rM < nfree ? (int)used + rM : sl.vsl[rM - nfree];
      slotL[tid] = fs;
      mslotL[rM] = fs;
      mevL[rM] = rM < nfree ? -1 : sl.vic[rM - nfree];
    }
  }
  {
    const uint64_t m = __ballot(inS && (!miss || rM < q));
    if (lane == 0) resL[wv] = m;
  }
  if (tid == 0) {
    rfirstL[0] = 0;
    nchunkL = 1;
  }
  __syncthreads();
  if (nM > q && wv == 0) {  // uniform: the misses that take a slot of S, in order (one wave)
    uint64_t r[kThreads / kWave];
#pragma unroll
    for (int j = 0; j < kThreads / kWave; ++j) r[j] = resL[j];
    int cur = 0;
    for (int i = q; i < nM; ++i) {
      int v = 0;
#pragma unroll
      for (int j = kThreads / kWave - 1; j >= 0; --j)  // the lowest id holding a slot
        if (r[j]) v = kWave * j + __builtin_ctzll(r[j]);
      const int sv = slotL[v], cv = chunkL[v], mi = missL[i];
      const int cm = max(cur, cv + 1);
      if (cm != cur && lane == 0 && cm <= kMtMaxChunks) rfirstL[cm] = i;
      cur = cm;
      r[v / kWave] &= ~(1ull << (v % kWave));
      r[mi / kWave] |= 1ull << (mi % kWave);
      if (lane == 0) {
        slotL[mi] = sv;
        chunkL[mi] = cm;
        mslotL[i] = sv;
        mevL[i] = v;
        goneL[v] = 1;
      }
    }
    if (lane == 0) nchunkL = cur + 1;
  }
  __syncthreads();
  const int nchunk = nchunkL;
  if (nchunk > max_chunks) {  // uniform: left to the caller, the table untouched
    if (tid < T) mw->list[tid].n = 0;
    if (tid == 0) {
      mw->n_copy = 0;
      mw->n_union = 0;
      flag[1] = nS;
      flag[2] = nchunk;
      __threadfence_system();
      flag[0] = 1;
    }
    return;
  }
  if (tid == 0) rfirstL[nchunk] = nM;
  // each expert's index in its chunk's union (ascending id)
  const int ch = chunkL[tid];
  int uidx = 0;
  for (int c2 = 0; c2 < nchunk; ++c2) {
    const uint64_t m = __ballot(inS && ch == c2);
    if (ch == c2) uidx = __popcll(m & lt);
    if (lane == 0) ccntL[wv][c2] = __popcll(m);
  }
  __syncthreads();
#pragma unroll
  for (int v = 0; v < kThreads / kWave; ++v)
    if (v < wv) uidx += ccntL[v][ch];
  // the table: stamps, final slots and occupants, evictions, trace
  if (evicted) lru.slot_of[tid] = -1;
  if (inS) {
    const int fs = slotL[tid];
    const bool gone = goneL[tid] != 0;
    lru.stamp[tid] = clock0 + rS + 1;
    if (gone) lru.slot_of[tid] = -1;
    else if (miss) lru.slot_of[tid] = fs;
    if (!gone) lru.expert_in[fs] = tid;
    if (lru.trace) {
      int32_t *r = lru.trace + 6 * (int64_t)(tn + rS);
      r[0] = lru.layer;
      r[1] = (int32_t)step;
      r[2] = tid;
      r[3] = miss ? 0 : 1;
      r[4] = miss ? mslotL[rM] : so;
      r[5] = miss ? mevL[rM] : -1;
    }
    // chunk ch's work: this expert in its union; a miss in its copies
    MtWork &W = mw[ch];
    if (miss) {
      const int mi = rM - rfirstL[ch];
      W.src[mi] = lru.store + (int64_t)tid * lru.P;
      W.dst[mi] = lru.slots + (int64_t)fs * lru.P;
      W.mu[mi] = (uint8_t)uidx;
    }
    W.upay[uidx] = lru.slots + (int64_t)fs * lru.P;
    W.unt[uidx] = (uint8_t)__popc(tokL[tid]);
    W.uhit[uidx] = (uint8_t)!miss;
    uL[tid] = uidx;
  }
  if (tid == 0) {
    lru.cnt[0] = (uint64_t)wordsL[4] + (uint64_t)(nS - nM);
    lru.cnt[1] = (uint64_t)wordsL[5] + (uint64_t)nM;
    lru.cnt[2] = (uint64_t)wordsL[6] + (uint64_t)max(0, nM - nfree);
    lru.cnt[3] = (uint64_t)wordsL[7] + (uint64_t)nM * (uint64_t)lru.P;
    lru.meta[0] = clock0 + nS;
    lru.meta[1] = step + 1;
    lru.meta[2] = used + min(nM, nfree);
    if (lru.trace) *lru.trace_n = tn + (uint64_t)nS;
  }
  __syncthreads();
  // (token t, rank j): its expert's place among the expert's tokens; with one
  // chunk also its slot in the token's list (read by the per-token GEMVs)
  for (int i = tid; i < T * k; i += kThreads) {
    const int t = i / k, j = i - t * k;
    const int e = selL[t][j];
    mw[chunkL[e]].uq[uL[e]][__popc(tokL[e] & ((1u << t) - 1u))] = (uint8_t)i;
    if (nchunk == 1) {
      mw->list[t].payload[j] = lru.slots + (int64_t)slotL[e] * lru.P;
      mw->list[t].pos[j] = j;
    }
  }
  if (tid < T) mw->list[tid].n = nchunk == 1 ? k : 0;
  if (tid < nchunk) {
    mw[tid].n_copy = rfirstL[tid + 1] - rfirstL[tid];
    int nu = 0;
#pragma unroll
    for (int v = 0; v < kThreads / kWave; ++v) nu += ccntL[v][tid];
    mw[tid].n_union = nu;
  }
  if (tid == 0) {
    flag[1] = nS;
    flag[2] = nchunk;
    __threadfence_system();
    flag[0] = 0;
  }
}

// Partial logits zp[s][T][E] = x[T][rows of slice s] W_r[rows of slice s][E]
// on the fp32 matrix cores (v_mfma_f32_16x16x4_f32, fp32 products and sums):
// a block owns 64 tokens, 128 expert columns (blockIdx.y) and one of `slices`
// slices of H (blockIdx.z); its eight waves (two per SIMD, to cover each
// other's waits) each own tokens 32 (w & 1) .. +31 (two 16-row subtiles) and
// experts 32 (w >> 1) .. +31 (two 16-column subtiles).  K runs
// over the slice in 32-row chunks staged through LDS (x as float4, W_r as
// coalesced scalars: E need not be a multiple of 4), the next chunk loaded
// into registers while the current one is multiplied.  The top-k kernel adds
// the slices in order.  Few tokens get many slices (a 5-token call would
// otherwise read all of W_r with 4 blocks).
constexpr int kPfTok = 32;  // token granularity of router_slices
constexpr int kRtTok = 64, kRtCols = 128, kRtK = 32, kRtThreads = 512;
constexpr int kRtXPitch = 34;   // floats: 16 rows x 2 k of one read on distinct banks
constexpr int kRtWPitch = 144;  // floats: consecutive k rows 16 banks apart

__global__ __launch_bounds__(kRtThreads) void router_logits_kernel(const float *__restrict__ x,
                                                                 const float *__restrict__ wr,
                                                                 int T, int H, int E, int slices,
                                                                 float *__restrict__ zp) {
  __shared__ __align__(16) float xs[2][kRtTok][kRtXPitch];
  __shared__ __align__(16) float ws[2][kRtK][kRtWPitch];
  const int tid = threadIdx.x, lane = tid & (kWave - 1), wv = tid / kWave;
  const int t0 = blockIdx.x * kRtTok, c0 = blockIdx.y * kRtCols;
  const int per = ((H + slices - 1) / slices + kRtK - 1) / kRtK * kRtK;
  const int rbeg = blockIdx.z * per, rend = min(H, rbeg + per);  // multiples of 32
  // loads of one chunk: x rows as float4 (thread i: row i / 8, k 4 (i % 8)),
  // W_r elements (i = tid + 512 m: k i / 128, column i % 128); clamped, selected on store
  float4 xv[1];
  float wvv[8];
  auto gload = [&](int r0) {
#pragma unroll
    for (int m = 0; m < 1; ++m) {
      const int i = tid + m * kRtThreads, row = i >> 3, k4 = (i & 7) * 4;
      const int t = min(t0 + row, T - 1);
      xv[m] = *reinterpret_cast<const float4 *>(x + (int64_t)t * H + r0 + k4);
    }
#pragma unroll
    for (int m = 0; m < 8; ++m) {
      const int i = tid + m * kRtThreads, kk = i >> 7, col = i & (kRtCols - 1);
      wvv[m] = wr[(int64_t)(r0 + kk) * E + min(c0 + col, E - 1)];
    }
  };
  auto lstore = [&](int buf) {
#pragma unroll
    for (int m = 0; m < 1; ++m) {
      const int i = tid + m * kRtThreads, row = i >> 3, k4 = (i & 7) * 4;
      const bool ok = t0 + row < T;
      float2 *d = reinterpret_cast<float2 *>(&xs[buf][row][k4]);
      d[0] = ok ? make_float2(xv[m].x, xv[m].y) : make_float2(0.f, 0.f);
      d[1] = ok ? make_float2(xv[m].z, xv[m].w) : make_float2(0.f, 0.f);
    }
#pragma unroll
    for (int m = 0; m < 8; ++m) {
      const int i = tid + m * kRtThreads, kk = i >> 7, col = i & (kRtCols - 1);
      ws[buf][kk][col] = c0 + col < E ? wvv[m] : 0.f;
    }
  };
  f32x4 acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int q = 0; q < 2; ++q) acc[i][q] = f32x4{0.f, 0.f, 0.f, 0.f};
  const int wrow = 32 * (wv & 1), wcol = 32 * (wv >> 1);
  int buf = 0;
  if (rbeg < rend) {
    gload(rbeg);
    lstore(0);
  }
  __syncthreads();
  for (int r0 = rbeg; r0 < rend; r0 += kRtK) {
    const bool more = r0 + kRtK < rend;  // uniform
    if (more) gload(r0 + kRtK);
#pragma unroll
    for (int s4 = 0; s4 < kRtK / 4; ++s4) {
      const int kk = 4 * s4 + (lane >> 4);
      float av[2], bv[2];
#pragma unroll
      for (int i = 0; i < 2; ++i) av[i] = xs[buf][wrow + 16 * i + (lane & 15)][kk];
#pragma unroll
      for (int q = 0; q < 2; ++q) bv[q] = ws[buf][kk][wcol + 16 * q + (lane & 15)];
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int q = 0; q < 2; ++q)
          acc[i][q] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[i], bv[q], acc[i][q], 0, 0, 0);
    }
    if (more) lstore(buf ^ 1);
    __syncthreads();
    buf ^= 1;
  }
  // C layout (16x16): lane holds rows 4 (lane / 16) + r, column lane % 16
  float *z = zp + (int64_t)blockIdx.z * T * E;
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int t = t0 + wrow + 16 * i + 4 * (lane >> 4) + r;
      if (t >= T) continue;
#pragma unroll
      for (int q = 0; q < 2; ++q) {
        const int col = c0 + wcol + 16 * q + (lane & 15);
        if (col < E) z[(int64_t)t * E + col] = acc[i][q][r];
      }
    }
}

// z[t] = tscale[t] * sum of the slices in order; top-k of each token row.
__global__ __launch_bounds__(kThreads) void topk_rows_kernel(const float *__restrict__ zp, int T,
                                                             int E, int k, int slices,
                                                             const float *__restrict__ tscale,
                                                             int32_t *idx, float *w) {
  __shared__ float zs[kThreads / kWave][256];
  const int wave = threadIdx.x / kWave, lane = threadIdx.x & (kWave - 1);
  const int t = blockIdx.x * (kThreads / kWave) + wave;
  if (t >= T) return;
  const float sc = tscale ? tscale[t] : 1.f;
  for (int e = lane; e < E; e += kWave) {
    float v = 0.f;
    for (int s0 = 0; s0 < slices; s0 += 16) {  // 16 slices in flight, added in slice order
      float p[16];
#pragma unroll
      for (int j = 0; j < 16; ++j)
        p[j] = s0 + j < slices ? zp[((int64_t)(s0 + j) * T + t) * E + e] : 0.f;
#pragma unroll
      for (int j = 0; j < 16; ++j) v += p[j];
    }
    zs[wave][e] = v * sc;
  }
  wave_topk(zs[wave], E, k, idx + (int64_t)t * k, w + (int64_t)t * k, nullptr, nullptr);
}

// ------------------------------------------------------------ decode FFN ---
//
// A "pair" is two consecutive 32-weight blocks of one row (64 weights): 68
// bytes for Q8_0, 36 for Q4_0, always 4-byte aligned because rows hold an
// even number of blocks.  A lane turns a pair into a partial dot product with
// the matching 64 inputs, given as three planes of int8 digits (16 dwords per
// plane per pair) and two block scales.

template <int QT>
struct Fmt;
// kGateUpFlight / kDownFlight: pairs per lane loading at once in the gate/up
// kernel (per matrix) and in the down kernel, about 270 and 210 bytes.
template <>
struct Fmt<8> {
  static constexpr int kBlockBytes = 34, kPairDwords = 17, kGateUpFlight = 2, kDownFlight = 3;
};
template <>
struct Fmt<2> {
  static constexpr int kBlockBytes = 18, kPairDwords = 9, kGateUpFlight = 4, kDownFlight = 6;
};

// LDS image of a digit vector of n values: three planes of n/64 pairs, each
// pair's 64 digit bytes at a pitch of 80 bytes, so that the 16-byte reads of
// eight lanes taking consecutive pairs fall on distinct banks.
constexpr int kPairPitch = 80;
__device__ __forceinline__ int plane_bytes(int n) { return (n / 64) * kPairPitch; }
// Offset in a plane of the value at index i (any i; a 4-aligned i starts a dword).
__device__ __forceinline__ int pad_off(int i) { return (i >> 6) * kPairPitch + (i & 63); }

// A pair is only 4-byte aligned; the 16-byte loads below rely on the
// unaligned global access that gfx9 runtimes enable (one dwordx4 instead of
// four dword loads: a quarter of the address work per byte).
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef u32x4 u32x4_a4 __attribute__((aligned(4)));
// Weight pointers come out of the work lists as generic pointers; loads
// through them would be flat loads, which also count against the LDS wait
// counter (every LDS wait would then wait for the weights as well).  Slots
// are device memory: the weights are read through global-address-space
// pointers.
typedef __attribute__((address_space(1))) const u32x4_a4 g_u32x4_a4;
typedef __attribute__((address_space(1))) const uint32_t g_u32;

template <int QT>
__device__ __forceinline__ void load_pair(const uint8_t *p, uint32_t (&wd)[Fmt<QT>::kPairDwords]) {
  constexpr int PD = Fmt<QT>::kPairDwords;
  g_u32x4_a4 *q = (g_u32x4_a4 *)p;
#pragma unroll
  for (int i = 0; i < PD / 4; ++i) {
    const u32x4 v = q[i];
    wd[4 * i] = v.x;
    wd[4 * i + 1] = v.y;
    wd[4 * i + 2] = v.z;
    wd[4 * i + 3] = v.w;
  }
  wd[PD - 1] = ((g_u32 *)p)[PD - 1];
}

// fp32 value of a block's digit dot products I1 + I2/254 + I3/254^2.
__device__ __forceinline__ float recombine(int i1, int i2, int i3) {
  return fmaf((float)i3, 1.f / 64516.f, fmaf((float)i2, 1.f / 254.f, (float)i1));
}

// Four Q4_0 nibbles of a dword as signed bytes 16 (n - 8): bit 3 of the nibble
// flipped makes it the 4-bit two's complement of n - 8, and at the top of its
// byte (the other nibble cleared) the byte is 16 (n - 8).  q4_lo takes the low
// nibble of each byte, q4_hi the high one; the flip of bit 7 after the shift
// is the flip of bit 3 before it.
__device__ __forceinline__ uint32_t q4_lo(uint32_t w) { return ((w << 4) & 0xf0f0f0f0u) ^ 0x80808080u; }
__device__ __forceinline__ uint32_t q4_hi(uint32_t w) { return (w & 0xf0f0f0f0u) ^ 0x80808080u; }

// Partial dot of one pair with the inputs: D[c][j] = digit plane c, dword j of
// the pair's 64 inputs; sc0/sc1 the two input block scales.
template <int QT>
__device__ __forceinline__ float pair_dot(const uint32_t (&wd)[Fmt<QT>::kPairDwords],
                                          const uint32_t *D, const float sc0, const float sc1) {
  if constexpr (QT == 8) {
    // bytes 0-1 d0 | 2-33 q0 | 34-35 d1 | 36-67 q1
    const float d0 = half_bits_to_float(wd[0] & 0xffffu), d1 = half_bits_to_float(wd[8] >> 16);
    int a1 = 0, a2 = 0, a3 = 0, b1 = 0, b2 = 0, b3 = 0;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const uint32_t q = __builtin_amdgcn_alignbyte(wd[j + 1], wd[j], 2);
      a1 = sdot4(q, D[j], a1);
      a2 = sdot4(q, D[16 + j], a2);
      a3 = sdot4(q, D[32 + j], a3);
    }
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const uint32_t q = wd[9 + j];
      b1 = sdot4(q, D[8 + j], b1);
      b2 = sdot4(q, D[24 + j], b2);
      b3 = sdot4(q, D[40 + j], b3);
    }
    return fmaf(d0 * sc0, recombine(a1, a2, a3), d1 * sc1 * recombine(b1, b2, b3));
  } else {
    // bytes 0-1 d0 | 2-17 nibbles of block 0 | 18-19 d1 | 20-35 block 1;
    // nibble byte j: low -> element j, high -> element j+16; weight d*(n-8).
    // With bit 3 of every nibble flipped, a nibble is the 4-bit two's
    // complement of n - 8; moved to the top of its byte (and the other
    // nibble cleared) the byte is the signed int8 16 (n - 8).  So every dot4
    // sum is exactly 16 times the offset weights' sum, and so is each step of
    // the fp32 combination below (scaling by a power of two is exact): the
    // result, scaled back by 1/16, equals d (sum of (n - 8) D) as combined
    // from exact integer sums, with no digit sums needed.
    const float d0 = half_bits_to_float(wd[0] & 0xffffu), d1 = half_bits_to_float(wd[4] >> 16);
    int a1 = 0, a2 = 0, a3 = 0, b1 = 0, b2 = 0, b3 = 0;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const uint32_t v = __builtin_amdgcn_alignbyte(wd[j + 1], wd[j], 2);
      const uint32_t lo = q4_lo(v), hi = q4_hi(v);
      a1 = sdot4(hi, D[4 + j], sdot4(lo, D[j], a1));
      a2 = sdot4(hi, D[20 + j], sdot4(lo, D[16 + j], a2));
      a3 = sdot4(hi, D[36 + j], sdot4(lo, D[32 + j], a3));
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const uint32_t v = wd[5 + j];
      const uint32_t lo = q4_lo(v), hi = q4_hi(v);
      b1 = sdot4(hi, D[12 + j], sdot4(lo, D[8 + j], b1));
      b2 = sdot4(hi, D[28 + j], sdot4(lo, D[24 + j], b2));
      b3 = sdot4(hi, D[44 + j], sdot4(lo, D[40 + j], b3));
    }
    return 0.0625f * fmaf(d0 * sc0, recombine(a1, a2, a3), d1 * sc1 * recombine(b1, b2, b3));
  }
}

// As pair_dot, with inputs in 16-wide digit blocks: sc[0..3] the scales of
// the pair's four 16-value quarters.  A Q4_0 block's low nibbles are its
// first 16 values and its high nibbles the last 16, so each nibble half meets
// one input block.
template <int QT>
__device__ __forceinline__ float pair_dot16(const uint32_t (&wd)[Fmt<QT>::kPairDwords],
                                            const uint32_t *D, const float *sc) {
  int A[4][3] = {};  // [quarter][digit plane]
  float d0, d1;
  if constexpr (QT == 8) {
    d0 = half_bits_to_float(wd[0] & 0xffffu);
    d1 = half_bits_to_float(wd[8] >> 16);
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const uint32_t q = __builtin_amdgcn_alignbyte(wd[j + 1], wd[j], 2);
#pragma unroll
      for (int c = 0; c < 3; ++c) A[j >> 2][c] = sdot4(q, D[16 * c + j], A[j >> 2][c]);
    }
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const uint32_t q = wd[9 + j];
#pragma unroll
      for (int c = 0; c < 3; ++c) A[2 + (j >> 2)][c] = sdot4(q, D[16 * c + 8 + j], A[2 + (j >> 2)][c]);
    }
  } else {
    // the nibbles as signed bytes 16 (n - 8), as in pair_dot: sums 16 times the
    // offset weights' ones, scaled back exactly at the end
    d0 = half_bits_to_float(wd[0] & 0xffffu);
    d1 = half_bits_to_float(wd[4] >> 16);
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const uint32_t v0 = __builtin_amdgcn_alignbyte(wd[j + 1], wd[j], 2), v1 = wd[5 + j];
      const uint32_t lo0 = q4_lo(v0), hi0 = q4_hi(v0), lo1 = q4_lo(v1), hi1 = q4_hi(v1);
#pragma unroll
      for (int c = 0; c < 3; ++c) {
        A[0][c] = sdot4(lo0, D[16 * c + j], A[0][c]);
        A[1][c] = sdot4(hi0, D[16 * c + 4 + j], A[1][c]);
        A[2][c] = sdot4(lo1, D[16 * c + 8 + j], A[2][c]);
        A[3][c] = sdot4(hi1, D[16 * c + 12 + j], A[3][c]);
      }
    }
  }
  const float r0 = fmaf(sc[0], recombine(A[0][0], A[0][1], A[0][2]),
                        sc[1] * recombine(A[1][0], A[1][1], A[1][2]));
  const float r1 = fmaf(sc[2], recombine(A[2][0], A[2][1], A[2][2]),
                        sc[3] * recombine(A[3][0], A[3][1], A[3][2]));
  const float r = fmaf(d0, r0, d1 * r1);
  return QT == 2 ? 0.0625f * r : r;
}

// The 48 digit dwords of pair p from an LDS digit image (plane stride pb bytes).
__device__ __forceinline__ void load_digits(const uint8_t *planes, int pb, int p,
                                            uint32_t (&D)[48]) {
#pragma unroll
  for (int c = 0; c < 3; ++c) {
    const uint4 *src = reinterpret_cast<const uint4 *>(planes + c * pb + kPairPitch * p);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const uint4 v = src[i];
      D[16 * c + 4 * i] = v.x;
      D[16 * c + 4 * i + 1] = v.y;
      D[16 * c + 4 * i + 2] = v.z;
      D[16 * c + 4 * i + 3] = v.w;
    }
  }
}

__device__ __forceinline__ float silu(float s) { return s / (1.f + expf(-s)); }

// Sum over the `lanes` consecutive lanes of a group (power of 2), butterfly
// order: the same on every run.
__device__ __forceinline__ float group_sum(float v, int lanes) {
  for (int off = lanes >> 1; off >= 1; off >>= 1) v += __shfl_xor(v, off, kWave);
  return v;
}

// Stage the token's digit planes ([3][H] bytes, contiguous) into an LDS digit
// image, and the block scales.  Split in two so that a caller can issue these
// loads ahead of its weight loads and store them afterwards: every lane of a
// used 256-piece round loads (indices past the end clamped to the last piece)
// and stores (pieces past the end to the 16-byte dummyL), so the compiler
// keeps the loads where they are issued.
constexpr int kMaxTok16 = 6;  // 3 * 8192 / 16 / 256
struct TokStage {
  u32x4 v[kMaxTok16];
  float s;
};
__device__ __forceinline__ void stage_token_load(const int8_t *__restrict__ q,
                                                 const float *__restrict__ sc, int H, TokStage &t) {
  const int n16 = 3 * H / 16, nsc = H / 32;
  const u32x4 *src = reinterpret_cast<const u32x4 *>(q);
#pragma unroll
  for (int m = 0; m < kMaxTok16; ++m)
    if (m * kThreads < n16) t.v[m] = src[min((int)threadIdx.x + m * kThreads, n16 - 1)];
  t.s = sc[min((int)threadIdx.x, nsc - 1)];
}
__device__ __forceinline__ void stage_token_store(const TokStage &t, int H, uint8_t *qL, float *scL,
                                                  uint8_t *dummyL) {
  const int n16 = 3 * H / 16, nsc = H / 32, per = H / 16, pb = plane_bytes(H);
#pragma unroll
  for (int m = 0; m < kMaxTok16; ++m) {
    if (m * kThreads < n16) {
      const int i = threadIdx.x + m * kThreads;
      const int c = (i >= per) + (i >= 2 * per);
      uint8_t *dst = i < n16 ? qL + c * pb + pad_off(16 * (i - c * per)) : dummyL;
      *reinterpret_cast<u32x4 *>(dst) = t.v[m];
    }
  }
  float *dsc = (int)threadIdx.x < nsc ? scL + threadIdx.x : reinterpret_cast<float *>(dummyL);
  *dsc = t.s;
}
__device__ __forceinline__ void stage_token(const int8_t *__restrict__ q,
                                            const float *__restrict__ sc, int H, uint8_t *qL,
                                            float *scL, uint8_t *dummyL) {
  TokStage t;
  stage_token_load(q, sc, H, t);
  stage_token_store(t, H, qL, scL, dummyL);
}

// Digit sums of every 32-wide block of a staged digit image of n values
// (the Q4_K min term): dsL[c][b] = sum of the 32 digits of block b in plane c.
__device__ __forceinline__ void digit_sums(const uint8_t *qL, int n, int *dsL) {
  const int nb = n / 32, pb = plane_bytes(n);
  for (int i = threadIdx.x; i < 3 * nb; i += kThreads) {
    const int c = i / nb, b = i - c * nb;
    const uint4 *v = reinterpret_cast<const uint4 *>(qL + c * pb + pad_off(32 * b));
    const uint4 u0 = v[0], u1 = v[1];
    int t = sdot4(u0.x, 0x01010101u, 0);
    t = sdot4(u0.y, 0x01010101u, t);
    t = sdot4(u0.z, 0x01010101u, t);
    t = sdot4(u0.w, 0x01010101u, t);
    t = sdot4(u1.x, 0x01010101u, t);
    t = sdot4(u1.y, 0x01010101u, t);
    t = sdot4(u1.z, 0x01010101u, t);
    dsL[i] = sdot4(u1.w, 0x01010101u, t);
  }
}

struct GateUpParams {
  ExpertList L;
  const ExpertList *Ld;  // device list (nullable): read instead of L
  const int8_t *xq;  // input digits [3][H]
  const float *xsc;  // input block scales [H/32]
  int8_t *hq;        // activation digits [3][k*I]
  float *hsc;        // their 16-wide block scales [k*I/16]
  int32_t *hds;      // their digit sums [3][k*I/16] (down format Q4_K)
  int H, I, k;
  int lanes, mpairs;  // lanes per row (power of 2, <= 16), pairs (K-quants: items) per lane
  int lanes_log2;
  int h_sums;  // K-quant gate/up: also write the activations' digit sums (down format Q4_K)
};

// Digits of SwiGLU activations in 16-wide blocks, called by 16 consecutive
// lanes holding the values of rows row0 .. row0+15 of the expert at top-k
// position pos (one value each, lane l has row row0 + l).
// sums: also the blocks' digit sums (the down formats with an offset or a
// min term, Q4_0 and Q4_K, need them).  Uniform over the 16 lanes.
__device__ __forceinline__ void store_h_digits_rt(float v, int pos, int row, int I, int k, int8_t *hq,
                                                  float *hsc, int32_t *hds, bool sums) {
  float m = fabsf(v);
#pragma unroll
  for (int off = 1; off < 16; off <<= 1) m = fmaxf(m, __shfl_xor(m, off, kWave));
  const float rs = m > 0.f ? 127.f * __builtin_amdgcn_rcpf(m) : 0.f;
  int d1, d2, d3;
  digits_of(v, rs, d1, d2, d3);
  int t1 = d1, t2 = d2, t3 = d3;
  if (sums) {
#pragma unroll
    for (int off = 1; off < 16; off <<= 1) {
      t1 += __shfl_xor(t1, off, kWave);
      t2 += __shfl_xor(t2, off, kWave);
      t3 += __shfl_xor(t3, off, kWave);
    }
  }
  if (row < I) {
    const int64_t i = (int64_t)pos * I + row, KI = (int64_t)k * I;
    hq[i] = (int8_t)d1;
    hq[KI + i] = (int8_t)d2;
    hq[2 * KI + i] = (int8_t)d3;
    if ((row & 15) == 0) {
      hsc[i / 16] = m * (1.f / 127.f);
      if (sums) {
        hds[i / 16] = t1;
        hds[KI / 16 + i / 16] = t2;
        hds[2 * (KI / 16) + i / 16] = t3;
      }
    }
  }
}
template <int QT>
__device__ __forceinline__ void store_h_digits(float v, int pos, int row, int I, int k, int8_t *hq,
                                               float *hsc, int32_t *hds) {
  store_h_digits_rt(v, pos, row, I, k, hq, hsc, hds, false);
}

// One unit = row r of W_gate and row r of W_up; lane l of the unit's `lanes`
// lanes handles pairs l, l+lanes, ... of both rows (F of each in flight).
// A block covers 256 / lanes >= 16 consecutive rows, so it also forms the
// digits of its whole 16-wide blocks of h.  Block blk of the launch: expert
// blk / bpe, rows from (blk % bpe) * (256 / lanes).
// hit (nullable): per list position, 0 = skip this expert (its rows come from elsewhere).
template <int QT>
__device__ __forceinline__ void gateup_body(const GateUpParams &a, const ExpertList &L,
                                            const int32_t *hit, int blk, uint8_t *smem8) {
  constexpr int BB = Fmt<QT>::kBlockBytes, PD = Fmt<QT>::kPairDwords, F = Fmt<QT>::kGateUpFlight;
  const int H = a.H, nb = H / 32, np = nb / 2, pb = plane_bytes(H);
  uint8_t *qL = smem8;                                     // digit image of the token
  float *scL = reinterpret_cast<float *>(smem8 + 3 * pb);  // [H/32]
  int *dsL = reinterpret_cast<int *>(scL + nb);            // [3][H/32]
  float *hL = reinterpret_cast<float *>(dsL + 3 * nb);     // [256 / lanes]
  const int upb = kThreads / a.lanes;
  const int bpe = (a.I + upb - 1) / upb;
  const int ei = blk / bpe;
  // the list's count, slot and position are read together (one round trip);
  // ei < kMaxRouted always (the grid covers at most kMaxRouted experts)
  const int n = L.n, pos = L.pos[ei], use = hit ? hit[ei] : 1;
  const uint8_t *const payload = L.payload[ei];
  // (the slot pointer is part of the test so that its load is issued with the count's)
  if (ei >= n || !use || payload == nullptr) return;  // uniform over the block
  const int r0 = (blk - ei * bpe) * upb;
  const int r = r0 + (threadIdx.x >> a.lanes_log2);
  const int l = threadIdx.x & (a.lanes - 1);
  const bool active = r < a.I;
  const int64_t rowb = (int64_t)nb * BB, mat = (int64_t)a.I * rowb;
  const uint8_t *gate = payload + (int64_t)r * rowb, *up = gate + mat;
  // the token's digits first, then the first round of weight pairs
  // (unconditional: an idle slot reloads its row's first pair), then the
  // digits into LDS while the weights are in flight
  __shared__ __align__(16) uint8_t dummyL[16];
  TokStage ts;
  stage_token_load(a.xq, a.xsc, H, ts);
  __builtin_amdgcn_sched_barrier(0);
  const uint8_t *gatev = payload + (int64_t)min(r, a.I - 1) * rowb, *upv = gatev + mat;
  uint32_t wg[F][PD], wu[F][PD];
#pragma unroll
  for (int m = 0; m < F; ++m) {
    const int p = l + m * a.lanes;
    const bool ok = active && m < a.mpairs && p < np;
    load_pair<QT>(ok ? gate + (int64_t)p * 2 * BB : gatev, wg[m]);
    load_pair<QT>(ok ? up + (int64_t)p * 2 * BB : upv, wu[m]);
  }
  __builtin_amdgcn_sched_barrier(0);
  stage_token_store(ts, H, qL, scL, dummyL);
  __syncthreads();
  float g = 0.f, u = 0.f;
  for (int m0 = 0; m0 < a.mpairs; m0 += F) {
    if (m0 > 0) {
#pragma unroll
      for (int m = 0; m < F; ++m) {
        const int p = l + (m0 + m) * a.lanes;
        if (active && m0 + m < a.mpairs && p < np) {
          load_pair<QT>(gate + (int64_t)p * 2 * BB, wg[m]);
          load_pair<QT>(up + (int64_t)p * 2 * BB, wu[m]);
        }
      }
    }
#pragma unroll
    for (int m = 0; m < F; ++m) {
      const int p = l + (m0 + m) * a.lanes;
      if (active && m0 + m < a.mpairs && p < np) {
        uint32_t D[48];
        load_digits(qL, pb, p, D);
        const float s0 = scL[2 * p], s1 = scL[2 * p + 1];
        g += pair_dot<QT>(wg[m], D, s0, s1);
        u += pair_dot<QT>(wu[m], D, s0, s1);
      }
    }
  }
  g = group_sum(g, a.lanes);
  u = group_sum(u, a.lanes);
  if (l == 0) hL[threadIdx.x >> a.lanes_log2] = active ? silu(g) * u : 0.f;
  __syncthreads();
  // digits of the block's rows: one value per thread, 16-lane groups
  if ((int)threadIdx.x < upb)
    store_h_digits<QT>(hL[threadIdx.x], pos, r0 + threadIdx.x, a.I, a.k, a.hq, a.hsc, a.hds);
}

// DEV: the list is read from device memory (a.Ld), else from the arguments.
template <int QT, bool DEV>
__global__ __launch_bounds__(kThreads) void gateup_kernel(GateUpParams a) {
  extern __shared__ __align__(16) uint8_t smem8[];
  gateup_body<QT>(a, DEV ? *a.Ld : a.L, nullptr, blockIdx.x, smem8);
}


// ---------------------------------------------------- copy + gate/up fused ---
//
// Blocks [0, copy_blocks) move the misses' payloads in "chunks": two spans of
// R rows (R * rowb bytes each) -- the same rows of W_gate and W_up for the
// first I/16 "units" of a miss (one unit = one 16-row block of h, 16/R
// chunks), then the down matrix in units of the same byte size.  A chunk is
// loaded with coalesced 16-byte loads (the copy kernel's pattern), stored to
// the slot and, for gate/up rows, to LDS, where the block computes its R rows
// of h while the next chunk is in flight.  Unit u of the launch goes to
// block u % copy_blocks.  Blocks from copy_blocks on are the gate/up blocks of
// the hit experts (gateup_body); those of missed positions exit.
constexpr int kChunkSlots = 9;  // 16-byte loads per lane per chunk: 2 * R * rowb <= 9 * 4096

// Payload byte offsets of the two spans of chunk c of unit j of a miss:
// gate/up units (j < I/16) hold rows 16 j + c R .. +R-1 of W_gate and of
// W_up; the down matrix follows in pieces of the same size.  True for a
// gate/up unit.
__device__ __forceinline__ bool chunk_spans(int j, int c, int I, int R, int64_t rowb, int64_t &o0,
                                            int64_t &o1) {
  const int64_t M = (int64_t)I * rowb, half = R * rowb;
  if (j < I / 16) {
    o0 = (int64_t)(16 * j + c * R) * rowb;
    o1 = M + o0;
    return true;
  }
  o0 = 2 * M + ((int64_t)(j - I / 16) * (16 / R) + c) * 2 * half;
  o1 = o0 + half;
  return false;
}

// One chunk (h16 16-byte pieces of each span) into registers: piece
// threadIdx.x + 256 m; pieces past the chunk read as zero.
__device__ __forceinline__ void load_chunk(const uint8_t *s0, const uint8_t *s1, int h16,
                                           uint4 (&buf)[kChunkSlots]) {
#pragma unroll
  for (int m = 0; m < kChunkSlots; ++m) {
    const int q = threadIdx.x + m * kThreads;
    const uint8_t *p = q < h16 ? s0 + 16 * (int64_t)q : s1 + 16 * (int64_t)(q - h16);
    buf[m] = q < 2 * h16 ? *reinterpret_cast<const uint4 *>(p) : make_uint4(0u, 0u, 0u, 0u);
  }
}

// The chunk in registers to its slot and, with to_lds, to the LDS chunk image cL.
__device__ __forceinline__ void store_chunk(const uint4 (&buf)[kChunkSlots], uint8_t *d0, uint8_t *d1,
                                            int h16, bool to_lds, uint8_t *cL) {
#pragma unroll
  for (int m = 0; m < kChunkSlots; ++m) {
    const int q = threadIdx.x + m * kThreads;
    if (q < 2 * h16) {
      uint8_t *p = q < h16 ? d0 + 16 * (int64_t)q : d1 + 16 * (int64_t)(q - h16);
      *reinterpret_cast<uint4 *>(p) = buf[m];
      if (to_lds) reinterpret_cast<uint4 *>(cL)[q] = buf[m];
    }
  }
}

// This lane's share of the gate and up dot products of chunk row ri (cL: R
// rows of W_gate, then R of W_up, `half` bytes apart) with a staged token
// image: pairs l, l + L, ... in order, none if !act (the gate/up kernels'
// lanes and order, so the group sums equal theirs bit for bit).
template <int QT>
__device__ __forceinline__ void chunk_row_dots(const uint8_t *cL, int ri, int64_t rowb, int64_t half,
                                               const uint8_t *qL, int pb, const float *scL,
                                               const int *dsL, int nb, int l, int L, bool act,
                                               float &gs, float &us) {
  constexpr int BB = Fmt<QT>::kBlockBytes, PD = Fmt<QT>::kPairDwords;
  const int np = nb / 2;
  const uint8_t *grow = cL + (int64_t)ri * rowb, *urow = grow + half;
  gs = 0.f;
  us = 0.f;
  for (int p = act ? l : np; p < np; p += L) {
    uint32_t wg[PD], wu[PD];
    const uint32_t *gp = reinterpret_cast<const uint32_t *>(grow + (int64_t)p * 2 * BB);
    const uint32_t *up = reinterpret_cast<const uint32_t *>(urow + (int64_t)p * 2 * BB);
#pragma unroll
    for (int e = 0; e < PD; ++e) {
      wg[e] = gp[e];
      wu[e] = up[e];
    }
    uint32_t D[48];
    load_digits(qL, pb, p, D);
    const float sc0 = scL[2 * p], sc1 = scL[2 * p + 1];
    gs += pair_dot<QT>(wg, D, sc0, sc1);
    us += pair_dot<QT>(wu, D, sc0, sc1);
  }
}

struct CopyGateUpParams {
  GateUpParams g;     // token digits, activation outputs, shape, hit-block lanes
  const WorkList *W;
  int64_t P;
  int copy_blocks, R;  // rows per chunk
  uint64_t *acc;      // nullable: += copies, += bytes
};

template <int QT>
__global__ __launch_bounds__(kThreads) void copy_gateup_kernel(CopyGateUpParams a) {
  extern __shared__ __align__(16) uint8_t smem8[];
  const WorkList &W = *a.W;
  if ((int)blockIdx.x >= a.copy_blocks) {  // gate/up of a hit expert
    gateup_body<QT>(a.g, W.list, W.hit, blockIdx.x - a.copy_blocks, smem8);
    return;
  }
  const int n = W.n_copy;
  if (n == 0) return;
  if (a.acc && blockIdx.x == 0 && threadIdx.x == 0) {
    atomicAdd(reinterpret_cast<unsigned long long *>(a.acc), (unsigned long long)n);
    atomicAdd(reinterpret_cast<unsigned long long *>(a.acc + 1), (unsigned long long)(n * a.P));
  }
  constexpr int BB = Fmt<QT>::kBlockBytes;
  const int H = a.g.H, I = a.g.I, nb = H / 32, pb = plane_bytes(H);
  uint8_t *qL = smem8;
  float *scL = reinterpret_cast<float *>(smem8 + 3 * pb);
  int *dsL = reinterpret_cast<int *>(scL + nb);
  float *hL = reinterpret_cast<float *>(dsL + 3 * nb);  // [16]
  uint8_t *cL = reinterpret_cast<uint8_t *>(hL + 16);    // one chunk: 2 spans
  const int R = a.R, cpu = 16 / R;                        // chunks per unit
  const int64_t rowb = (int64_t)nb * BB, half = R * rowb;
  const int h16 = (int)(half / 16);                       // 16-byte pieces per span
  const int upm = I / 16 + I / 32;                         // units per miss
  const int n_units = n * upm;
  int u = blockIdx.x;
  if (u >= n_units) return;  // uniform
  __shared__ __align__(16) uint8_t dummyL[16];
  stage_token(a.g.xq, a.g.xsc, H, qL, scL, dummyL);
  // the two spans of chunk c of unit u (source and slot), and whether it holds gate/up rows
  auto spans = [&](int uu, int c, const uint8_t *&s0, const uint8_t *&s1, uint8_t *&d0, uint8_t *&d1,
                   int &miss, int &g) -> bool {
    miss = uu / upm;
    const int j = uu - miss * upm;
    int64_t o0, o1;
    const bool gu = chunk_spans(j, c, I, R, rowb, o0, o1);
    g = gu ? j : -1;
    s0 = W.src[miss] + o0;
    s1 = W.src[miss] + o1;
    d0 = W.dst[miss] + o0;
    d1 = W.dst[miss] + o1;
    return gu;
  };
  uint4 buf[kChunkSlots];
  const uint8_t *s0, *s1;
  uint8_t *d0, *d1;
  int miss, g, c = 0;
  bool gu = spans(u, 0, s0, s1, d0, d1, miss, g);
  load_chunk(s0, s1, h16, buf);
  // the gate/up kernel's lanes and pair order, so h is bit-identical to its result
  const int L = a.g.lanes, rr = threadIdx.x >> a.g.lanes_log2, l = threadIdx.x & (L - 1);
  for (;;) {
    store_chunk(buf, d0, d1, h16, gu, cL);  // to its slot, and (gate/up rows) to LDS
    const bool cur_gu = gu;
    const int cur_c = c, cur_miss = miss, cur_g = g;
    // next chunk of this block, loads issued before the compute below
    if (++c == cpu) {
      c = 0;
      u += a.copy_blocks;
    }
    const bool more = u < n_units;
    if (more) {
      gu = spans(u, c, s0, s1, d0, d1, miss, g);
      load_chunk(s0, s1, h16, buf);
    }
    __syncthreads();  // chunk in LDS
    if (cur_gu) {
      // R rows of h from the chunk: L lanes per row
      float gs, us;
      chunk_row_dots<QT>(cL, rr < R ? rr : 0, rowb, half, qL, pb, scL, dsL, nb, l, L, rr < R, gs, us);
      gs = group_sum(gs, L);
      us = group_sum(us, L);
      if (l == 0 && rr < R) hL[cur_c * R + rr] = silu(gs) * us;
      if (cur_c == cpu - 1) {
        __syncthreads();
        if (threadIdx.x < 16)
          store_h_digits<QT>(hL[threadIdx.x], W.miss_pos[cur_miss], 16 * cur_g + threadIdx.x, I,
                             a.g.k, a.g.hq, a.g.hsc, a.g.hds);
      }
    }
    __syncthreads();  // LDS free for the next chunk
    if (!more) break;
  }
}

// Stage the activation digits of the listed experts into LDS: digit images
// qL [n] (three planes of plane_bytes(I) each), scales scL [n][I/16] and
// (Q4_K) digit sums dsL [n][3][I/16].  Split in two so that the caller can
// issue these loads ahead of its weight loads and store them afterwards.
constexpr int kMaxDig16 = 9;  // 3 * 12288 / 16 / 256
constexpr int kMaxSc4 = 1;    // 12288 / 16 / 4 / 256
constexpr int kMaxDs4 = 3;    // 3 * 12288 / 16 / 4 / 256
// (16-byte pieces held as native vectors: HIP's uint4 / float4 structs are
// copied through a stack object by the compiler)
struct HStage {
  u32x4 d[kMaxDig16];
  u32x4 s[kMaxSc4];
  u32x4 q[kMaxDs4];
};

// Unit u of n groups of `per` units -> (group, index) by floor((u + 0.5) / per)
// in fp32: exact here (u < 2^12, so the rounding error stays far below the
// 0.5/per margin).
__device__ __forceinline__ int split_unit(int u, float rper, int per, int &j) {
  const int g = (int)(((float)u + 0.5f) * rper);
  j = u - g * per;
  return g;
}

// posL: the listed experts' top-k positions (LDS, n of them).
__device__ __forceinline__ void stage_h_load(const int8_t *__restrict__ hq,
                                             const float *__restrict__ hsc,
                                             const int32_t *__restrict__ hds, const int *posL, int n,
                                             int I, int k, bool sums, HStage &st) {
  // Straight-line code: every lane loads (indices past the end are clamped to
  // the last expert, so each address is inside the buffers) and only the
  // in-range pieces are stored by stage_h_store.  Branch-free, the loads are
  // issued back to back, with no wait between them.
  const int64_t KI = (int64_t)k * I;
  const int u16 = I / 16, u64 = I / 64;
  const float r16 = 1.f / (float)u16, r64 = 1.f / (float)u64;
  const u32x4 *pd[kMaxDig16];
  const u32x4 *ps[kMaxSc4];
  const u32x4 *pq[kMaxDs4];
#pragma unroll
  for (int m = 0; m < kMaxDig16; ++m) {
    const int u = threadIdx.x + m * kThreads;  // (expert, plane, unit)
    int j;
    const int ec = split_unit(u, r16, u16, j);
    const int e = min(ec / 3, n - 1), c = ec - 3 * (ec / 3);
    pd[m] = reinterpret_cast<const u32x4 *>(hq + c * KI + (int64_t)posL[e] * I + 16 * j);
  }
#pragma unroll
  for (int m = 0; m < kMaxSc4; ++m) {
    const int u = threadIdx.x + m * kThreads;  // (expert, 4 scales)
    int j;
    const int e = min(split_unit(u, r64, u64, j), n - 1);
    ps[m] = reinterpret_cast<const u32x4 *>(hsc + (int64_t)posL[e] * u16 + 4 * j);
  }
#pragma unroll
  for (int m = 0; m < kMaxDs4; ++m) {
    const int u = threadIdx.x + m * kThreads;  // (expert, plane, 4 sums)
    int j;
    const int ec = split_unit(u, r64, u64, j);
    const int e = min(ec / 3, n - 1), c = ec - 3 * (ec / 3);
    pq[m] = reinterpret_cast<const u32x4 *>(hds + c * (KI / 16) + (int64_t)posL[e] * u16 + 4 * j);
  }
#pragma unroll
  for (int m = 0; m < kMaxDig16; ++m) st.d[m] = *pd[m];
#pragma unroll
  for (int m = 0; m < kMaxSc4; ++m) st.s[m] = *ps[m];
  if (sums) {
#pragma unroll
    for (int m = 0; m < kMaxDs4; ++m) st.q[m] = *pq[m];
  }
}

// Every lane stores each piece (no branches, so the compiler keeps the loads
// where they were issued); pieces past the end go to the 16-byte dummyL.
__device__ __forceinline__ void stage_h_store(const HStage &st, int n, int I, bool sums, uint8_t *qL,
                                              float *scL, int *dsL, uint8_t *dummyL) {
  const int u16 = I / 16, u64 = I / 64, pb = plane_bytes(I);
  const float r16 = 1.f / (float)u16;
#pragma unroll
  for (int m = 0; m < kMaxDig16; ++m) {
    const int u = threadIdx.x + m * kThreads;
    int j;
    const int ec = split_unit(u, r16, u16, j);
    uint8_t *dst = u < 3 * n * u16 ? qL + ec * pb + pad_off(16 * j) : dummyL;
    *reinterpret_cast<u32x4 *>(dst) = st.d[m];
  }
#pragma unroll
  for (int m = 0; m < kMaxSc4; ++m) {
    const int u = threadIdx.x + m * kThreads;
    u32x4 *dst = u < n * u64 ? reinterpret_cast<u32x4 *>(scL) + u
                             : reinterpret_cast<u32x4 *>(dummyL);
    *dst = st.s[m];
  }
  if (sums) {
#pragma unroll
    for (int m = 0; m < kMaxDs4; ++m) {
      const int u = threadIdx.x + m * kThreads;
      u32x4 *dst = u < 3 * n * u64 ? reinterpret_cast<u32x4 *>(dsL) + u
                                   : reinterpret_cast<u32x4 *>(dummyL);
      *dst = st.q[m];
    }
  }
}

struct DownParams {
  ExpertList L;
  const ExpertList *Ld;  // device list (nullable): read instead of L
  const int8_t *hq;   // activation digits [3][k*I]
  const float *hsc;   // their 16-wide block scales [k*I/16]
  const int32_t *hds; // their digit sums [3][k*I/16] (Q4_K)
  const float *w, *x;
  float *y;
  int H, I, k, mode;
  int lanes, mpairs;  // as in the gate/up kernel
  int rows;           // output rows per block: rows * n * lanes <= 256
  int lanes_log2;
  int64_t down_off;   // K-quant down: bytes from a payload's start to its W_down
};

// One unit = (output row j, expert i), `lanes` lanes, lane l handling pairs
// l, l+lanes, ... (F in flight).  grid: ceil(H / rows).
// y[j] (+)= sum over the listed experts, in list order, of w[pos_i] (W_down,i h_i)_j.
// DEV: the list is read from device memory (a.Ld), else from the arguments.
// Memory round trips: the list; then the activation digits, the routing
// weights and the weight rows, all in flight together.
// NT: threads per block, 256 or 512 (more rows per block, so that the grid
// fits the compute units once; the first 256 threads stage the activations).
template <int QT, bool DEV, int NT>
__global__ __launch_bounds__(NT, 1) void down_kernel(DownParams a) {
  extern __shared__ __align__(16) uint8_t smem8[];
  __shared__ int posL[kMaxRouted];
  __shared__ float wL[kMaxRouted];
  __shared__ __align__(16) uint8_t dummyL[16];  // target of the idle lanes' staging stores
  constexpr int BB = Fmt<QT>::kBlockBytes, PD = Fmt<QT>::kPairDwords, F = Fmt<QT>::kDownFlight;
  const ExpertList &L = DEV ? *a.Ld : a.L;
  const int I = a.I, nb = I / 32, np = nb / 2, n = a.L.n, pb = plane_bytes(I);
  uint8_t *qL = smem8;                                         // n digit images
  float *scL = reinterpret_cast<float *>(smem8 + 3 * n * pb);  // [n][I/16]
  int *dsL = reinterpret_cast<int *>(scL + n * (I / 16));      // [n][3][I/16]
  float *res = reinterpret_cast<float *>(dsL + 3 * n * (I / 16));  // [rows][n]
  const int j0 = blockIdx.x * a.rows;
  // consecutive units take consecutive rows of one expert, so the lanes of a
  // wave that handle the same pair read the same activation digits from LDS
  // (one broadcast read instead of one per expert); ic: i clamped to the list
  const int unit = threadIdx.x >> a.lanes_log2, l = threadIdx.x & (a.lanes - 1);
  const int i = unit / a.rows, rr = unit - i * a.rows, j = j0 + rr, ic = min(i, n - 1);
  const bool active = i < n && j < a.H;
  const int64_t rowb = (int64_t)nb * BB;
  const int64_t mat = (int64_t)I * ((int64_t)(a.H / 32) * BB);
  // the list: count, this unit's slot, the positions (one round trip)
  const int ndev = L.n;
  const uint8_t *const payload = L.payload[ic];
  const int pos_t = (int)threadIdx.x < n ? L.pos[threadIdx.x] : 0;
  if (ndev != n) return;  // a device list emptied by a routing error (uniform)
  if ((int)threadIdx.x < n) posL[threadIdx.x] = pos_t;
  __syncthreads();
  const uint8_t *row = payload + 2 * mat + (int64_t)j * rowb;
  const uint8_t *rowv = payload + 2 * mat + (int64_t)min(j, a.H - 1) * rowb;
  HStage st;
  const bool stager = NT == kThreads || (int)threadIdx.x < kThreads;  // uniform per wave
  if (stager) stage_h_load(a.hq, a.hsc, a.hds, posL, n, I, a.k, false, st);  // ahead of the weights
  // keeps the staging loads here, ahead of the weight loads (the compiler
  // would otherwise sink each load to its LDS store and wait for it there)
  __builtin_amdgcn_sched_barrier(0);
  // unconditional loads at clamped (valid) indices, results selected after
  const float w_t = a.w[posL[min((int)threadIdx.x, n - 1)]];
  // the residual / accumulated output of row j0 + threadIdx.x (rows <= 256)
  const int jt = j0 + (int)threadIdx.x;
  const bool out_t = (int)threadIdx.x < a.rows && jt < a.H;
  const float base_ld = (a.mode == 1 ? a.x : a.y)[min(jt, a.H - 1)];
  const float base_t = a.mode == 0 ? 0.f : base_ld;
  // first round of weight pairs, unconditional: an idle slot (inactive row,
  // pair past the row's end) reloads the unit's first pair, which is valid
  uint32_t wd[F][PD];
#pragma unroll
  for (int m = 0; m < F; ++m) {
    const int p = l + m * a.lanes;
    const bool ok = active && m < a.mpairs && p < np;
    load_pair<QT>(ok ? row + (int64_t)p * 2 * BB : rowv, wd[m]);
  }
  __builtin_amdgcn_sched_barrier(0);
  if (stager) stage_h_store(st, n, I, false, qL, scL, dsL, dummyL);
  __syncthreads();
  float acc = 0.f;
  for (int m0 = 0; m0 < a.mpairs; m0 += F) {
    if (m0 > 0) {
#pragma unroll
      for (int m = 0; m < F; ++m) {
        const int p = l + (m0 + m) * a.lanes;
        if (active && m0 + m < a.mpairs && p < np) load_pair<QT>(row + (int64_t)p * 2 * BB, wd[m]);
      }
    }
#pragma unroll
    for (int m = 0; m < F; ++m) {
      const int p = l + (m0 + m) * a.lanes;
      if (active && m0 + m < a.mpairs && p < np) {
        uint32_t D[48];
        load_digits(qL + 3 * i * pb, pb, p, D);
        acc += pair_dot16<QT>(wd[m], D, scL + i * (I / 16) + 4 * p);
      }
    }
  }
  acc = group_sum(acc, a.lanes);
  if (active && l == 0) res[rr * n + i] = acc;
  if ((int)threadIdx.x < n) wL[threadIdx.x] = w_t;
  __syncthreads();
  if (out_t) {
    // the weighted rows first, then the residual / earlier sum in one addition,
    // so that a small MoE output on a large residual is rounded once
    float v = 0.f;
    for (int ii = 0; ii < n; ++ii) v = fmaf(wL[ii], res[threadIdx.x * n + ii], v);
    a.y[jt] = base_t + v;
  }
}

// ------------------------------------------------------ K-quant decode FFN ---
//
// Q4_K and Q6_K store weights in super-blocks of 256.  A lane's unit of work
// (an "item") is half a super-block: 128 consecutive weights of a row, which
// meet the input digit images of pairs 2 it and 2 it + 1.
//   Q4_K (144-byte super-blocks, 16-byte aligned): the item loads the
//   super-block's 16-byte header (d, dmin, the 12 bytes of 6-bit scales and
//   mins) and its 64 bytes of 4-bit q (chunks 2h and 2h+1: sub-blocks 4h ..
//   4h+3, low nibbles the even sub-block of a chunk, high nibbles the odd).
//   Weight d sc q - dmin m: the min term meets the inputs' digit sums.
//   Q6_K (210-byte super-blocks, so only 2-byte aligned): ql[64h .. +64),
//   qh[32h .. +32), the 8 scales of the half and d, loaded from the 4-byte
//   aligned address below (never outside the payload: a payload starts and
//   ends 16-byte aligned, so its first super-block has offset 0 and its last
//   one ends on a dword) and realigned with alignbyte.  Each q - 32 is formed
//   as a signed byte, so no digit sums are needed.
template <int QT>
struct KFmt;
// kDw: dwords an item holds; flights: items per lane loading at once
template <>
struct KFmt<12> {
  static constexpr int kSB = 144, kDw = 20, kGateUpFlight = 2, kDownFlight = 2;
};
template <>
struct KFmt<14> {
  static constexpr int kSB = 210, kDw = 30, kGateUpFlight = 1, kDownFlight = 2;
};

// Item it of a row into w; returns the byte shift that realigns a Q6_K item (0 or 2).
template <int QT>
__device__ __forceinline__ int load_item(const uint8_t *row, int it, uint32_t (&w)[KFmt<QT>::kDw]) {
  const int sb = it >> 1, h = it & 1;
  if constexpr (QT == 12) {
    const uint8_t *b = row + (int64_t)sb * 144;
    const u32x4 hd = *(g_u32x4_a4 *)b;
    w[0] = hd.x;
    w[1] = hd.y;
    w[2] = hd.z;
    w[3] = hd.w;
    g_u32x4_a4 *q = (g_u32x4_a4 *)(b + 16 + 64 * h);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const u32x4 v = q[i];
      w[4 + 4 * i] = v.x;
      w[5 + 4 * i] = v.y;
      w[6 + 4 * i] = v.z;
      w[7 + 4 * i] = v.w;
    }
    return 0;
  } else {
    const uint8_t *b = row + (int64_t)sb * 210;
    const int sh = (int)((uintptr_t)b & 3);
    const uint8_t *a = b - sh;
    const uint8_t *ql = a + 64 * h, *qh = a + 128 + 32 * h;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const u32x4 v = ((g_u32x4_a4 *)ql)[i];
      w[4 * i] = v.x;
      w[4 * i + 1] = v.y;
      w[4 * i + 2] = v.z;
      w[4 * i + 3] = v.w;
    }
    w[16] = ((g_u32 *)ql)[16];
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const u32x4 v = ((g_u32x4_a4 *)qh)[i];
      w[17 + 4 * i] = v.x;
      w[18 + 4 * i] = v.y;
      w[19 + 4 * i] = v.z;
      w[20 + 4 * i] = v.w;
    }
    w[25] = ((g_u32 *)qh)[8];
    const g_u32 *sc = (g_u32 *)(a + 192 + 8 * h);
    w[26] = sc[0];
    w[27] = sc[1];
    w[28] = sc[2];
    w[29] = ((g_u32 *)(a + 208))[0];
    return sh;
  }
}

// Partial dot of a Q4_K item with 128 inputs given as digit images (pairs 2it,
// 2it+1 of qL).  B16 false: the inputs' 32-wide blocks (scales scL[b], digit
// sums dsL[b + c dstride]); true: 16-wide blocks (scL[q], dsL[q + c dstride]).
template <bool B16>
__device__ __forceinline__ float q4k_item_dot(const uint32_t (&w)[20], const uint8_t *qL, int pb, int it,
                                              const float *scL, const int *dsL, int dstride) {
  const int h = it & 1;
  const float d = half_bits_to_float(w[0] & 0xffffu), dmin = half_bits_to_float(w[0] >> 16);
  const uint32_t B0 = w[1], B1 = w[2], B2 = w[3];  // the 12 scale bytes
  // byte j of SC / MN: scale / min of sub-block 4h + j
  const uint32_t SC = h ? ((B2 & 0x0f0f0f0fu) | ((B0 >> 2) & 0x30303030u)) : (B0 & 0x3f3f3f3fu);
  const uint32_t MN = h ? (((B2 >> 4) & 0x0f0f0f0fu) | ((B1 >> 2) & 0x30303030u)) : (B1 & 0x3f3f3f3fu);
  float acc = 0.f;
#pragma unroll
  for (int t = 0; t < 2; ++t) {
    const int p = 2 * it + t;
    uint32_t D[48];
    load_digits(qL, pb, p, D);
    int A[4][3] = {};
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const uint32_t q = w[4 + 8 * t + i];
      const uint32_t lo = q & 0x0f0f0f0fu, hi = (q >> 4) & 0x0f0f0f0fu;
#pragma unroll
      for (int c = 0; c < 3; ++c) {
        const int ql = B16 ? (i >> 2) : 0, qh = B16 ? 2 + (i >> 2) : 1;
        A[ql][c] = sdot4(lo, D[16 * c + i], A[ql][c]);
        A[qh][c] = sdot4(hi, D[16 * c + 8 + i], A[qh][c]);
      }
    }
    const float sc_lo = (float)((SC >> (16 * t)) & 0xffu), sc_hi = (float)((SC >> (16 * t + 8)) & 0xffu);
    const float m_lo = (float)((MN >> (16 * t)) & 0xffu), m_hi = (float)((MN >> (16 * t + 8)) & 0xffu);
    if constexpr (B16) {
      const float *s = scL + 4 * p;
      const int *ds = dsL + 4 * p;
      float x[4], nsum[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        x[q] = s[q] * recombine(A[q][0], A[q][1], A[q][2]);
        nsum[q] = s[q] * recombine(ds[q], ds[q + dstride], ds[q + 2 * dstride]);
      }
      acc += fmaf(d, fmaf(sc_lo, x[0] + x[1], sc_hi * (x[2] + x[3])),
                  -dmin * fmaf(m_lo, nsum[0] + nsum[1], m_hi * (nsum[2] + nsum[3])));
    } else {
      const float s0 = scL[2 * p], s1 = scL[2 * p + 1];
      const int *ds = dsL + 2 * p;
      const float n0 = s0 * recombine(ds[0], ds[dstride], ds[2 * dstride]);
      const float n1 = s1 * recombine(ds[1], ds[1 + dstride], ds[1 + 2 * dstride]);
      const float x0 = s0 * recombine(A[0][0], A[0][1], A[0][2]);
      const float x1 = s1 * recombine(A[1][0], A[1][1], A[1][2]);
      acc += fmaf(d, fmaf(sc_lo, x0, sc_hi * x1), -dmin * fmaf(m_lo, n0, m_hi * n1));
    }
  }
  return acc;
}

// Partial dot of a Q6_K item (realigned by sh bytes) with 128 inputs as digit
// images.  B16 false: 32-wide input blocks (scales scL[b]); true: 16-wide (scL[q]).
template <bool B16>
__device__ __forceinline__ float q6k_item_dot(const uint32_t (&w)[30], int sh, const uint8_t *qL, int pb,
                                              int it, const float *scL) {
  uint32_t QL[16], QH[8];
#pragma unroll
  for (int i = 0; i < 16; ++i) QL[i] = __builtin_amdgcn_alignbyte(w[i + 1], w[i], sh);
#pragma unroll
  for (int i = 0; i < 8; ++i) QH[i] = __builtin_amdgcn_alignbyte(w[18 + i], w[17 + i], sh);
  const uint32_t S[2] = {__builtin_amdgcn_alignbyte(w[27], w[26], sh),
                         __builtin_amdgcn_alignbyte(w[28], w[27], sh)};
  const float d = half_bits_to_float((w[29] >> (8 * sh)) & 0xffffu);
  float acc = 0.f;
#pragma unroll
  for (int pp = 0; pp < 2; ++pp) {
    uint32_t D[48];
    load_digits(qL, pb, 2 * it + pp, D);
#pragma unroll
    for (int gg = 0; gg < 2; ++gg) {
      const int g = 2 * pp + gg;  // weights 32g .. 32g+31 of the item
      int A[2][3] = {};
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const uint32_t lo4 = (QL[8 * (g & 1) + i] >> (4 * (g >> 1))) & 0x0f0f0f0fu;
        const uint32_t hi2 = (QH[i] >> (2 * g)) & 0x03030303u;
        // q - 32 as signed bytes: flip bit 5, then copy it into bits 6 and 7
        const uint32_t v = (lo4 | (hi2 << 4)) ^ 0x20202020u, sg = v & 0x20202020u;
        const uint32_t q = v | (sg << 1) | (sg << 2);
#pragma unroll
        for (int c = 0; c < 3; ++c) A[i >> 2][c] = sdot4(q, D[16 * c + 8 * gg + i], A[i >> 2][c]);
      }
      const float s_a = (float)(int8_t)((S[g >> 1] >> (16 * (g & 1))) & 0xffu);
      const float s_b = (float)(int8_t)((S[g >> 1] >> (16 * (g & 1) + 8)) & 0xffu);
      const float ra = recombine(A[0][0], A[0][1], A[0][2]), rb = recombine(A[1][0], A[1][1], A[1][2]);
      if constexpr (B16) {
        const int q0 = 8 * it + 2 * g;
        acc += d * fmaf(s_a * scL[q0], ra, s_b * scL[q0 + 1] * rb);
      } else {
        acc += d * scL[4 * it + g] * fmaf(s_a, ra, s_b * rb);
      }
    }
  }
  return acc;
}

template <int QT, bool B16>
__device__ __forceinline__ float item_dot(const uint32_t (&w)[KFmt<QT>::kDw], int sh, const uint8_t *qL,
                                          int pb, int it, const float *scL, const int *dsL, int dstride) {
  if constexpr (QT == 12)
    return q4k_item_dot<B16>(w, qL, pb, it, scL, dsL, dstride);
  else
    return q6k_item_dot<B16>(w, sh, qL, pb, it, scL);
}

// gateup_body for the K-quant formats: one unit = row r of W_gate and of W_up,
// lane l of the unit's lanes handles items l, l+lanes, ... (F of each in flight).
template <int QT>
__device__ __forceinline__ void kgateup_body(const GateUpParams &a, const ExpertList &L,
                                             const int32_t *hit, int blk, uint8_t *smem8) {
  constexpr int DW = KFmt<QT>::kDw, F = KFmt<QT>::kGateUpFlight, SB = KFmt<QT>::kSB;
  const int H = a.H, nb = H / 32, ni = H / 128, pb = plane_bytes(H);
  uint8_t *qL = smem8;
  float *scL = reinterpret_cast<float *>(smem8 + 3 * pb);
  int *dsL = reinterpret_cast<int *>(scL + nb);
  float *hL = reinterpret_cast<float *>(dsL + 3 * nb);
  const int upb = kThreads / a.lanes;
  const int bpe = (a.I + upb - 1) / upb;
  const int ei = blk / bpe;
  const int n = L.n, pos = L.pos[ei], use = hit ? hit[ei] : 1;
  const uint8_t *const payload = L.payload[ei];
  if (ei >= n || !use || payload == nullptr) return;  // uniform over the block
  const int r0 = (blk - ei * bpe) * upb;
  const int r = r0 + (threadIdx.x >> a.lanes_log2);
  const int l = threadIdx.x & (a.lanes - 1);
  const bool active = r < a.I;
  const int64_t rowb = (int64_t)(H / 256) * SB, mat = (int64_t)a.I * rowb;
  const uint8_t *gate = payload + (int64_t)min(r, a.I - 1) * rowb, *up = gate + mat;
  __shared__ __align__(16) uint8_t dummyL[16];
  TokStage ts;
  stage_token_load(a.xq, a.xsc, H, ts);
  __builtin_amdgcn_sched_barrier(0);
  uint32_t wg[F][DW], wu[F][DW];
  int shg[F], shu[F];
#pragma unroll
  for (int m = 0; m < F; ++m) {  // unconditional: an idle slot reloads item 0 of its (clamped) row
    const int it = l + m * a.lanes;
    const int itc = (active && m < a.mpairs && it < ni) ? it : 0;
    shg[m] = load_item<QT>(gate, itc, wg[m]);
    shu[m] = load_item<QT>(up, itc, wu[m]);
  }
  __builtin_amdgcn_sched_barrier(0);
  stage_token_store(ts, H, qL, scL, dummyL);
  __syncthreads();
  if constexpr (QT == 12) {
    digit_sums(qL, H, dsL);
    __syncthreads();
  }
  float g = 0.f, u = 0.f;
  for (int m0 = 0; m0 < a.mpairs; m0 += F) {
    if (m0 > 0) {
#pragma unroll
      for (int m = 0; m < F; ++m) {
        const int it = l + (m0 + m) * a.lanes;
        if (active && m0 + m < a.mpairs && it < ni) {
          shg[m] = load_item<QT>(gate, it, wg[m]);
          shu[m] = load_item<QT>(up, it, wu[m]);
        }
      }
    }
#pragma unroll
    for (int m = 0; m < F; ++m) {
      const int it = l + (m0 + m) * a.lanes;
      if (active && m0 + m < a.mpairs && it < ni) {
        g += item_dot<QT, false>(wg[m], shg[m], qL, pb, it, scL, dsL, nb);
        u += item_dot<QT, false>(wu[m], shu[m], qL, pb, it, scL, dsL, nb);
      }
    }
  }
  g = group_sum(g, a.lanes);
  u = group_sum(u, a.lanes);
  if (l == 0) hL[threadIdx.x >> a.lanes_log2] = active ? silu(g) * u : 0.f;
  __syncthreads();
  if ((int)threadIdx.x < upb)
    store_h_digits_rt(hL[threadIdx.x], pos, r0 + threadIdx.x, a.I, a.k, a.hq, a.hsc, a.hds, a.h_sums != 0);
}

template <int QT, bool DEV>
__global__ __launch_bounds__(kThreads) void kgateup_kernel(GateUpParams a) {
  extern __shared__ __align__(16) uint8_t smem8[];
  kgateup_body<QT>(a, DEV ? *a.Ld : a.L, nullptr, blockIdx.x, smem8);
}

// down_kernel for the K-quant formats: one unit = (output row j, expert i),
// lanes l handling items l, l+lanes, ... (F in flight); W_down at a.down_off.
template <int QT, bool DEV>
__global__ __launch_bounds__(kThreads, 1) void kdown_kernel(DownParams a) {
  extern __shared__ __align__(16) uint8_t smem8[];
  __shared__ int posL[kMaxRouted];
  __shared__ float wL[kMaxRouted];
  __shared__ __align__(16) uint8_t dummyL[16];
  constexpr int DW = KFmt<QT>::kDw, F = KFmt<QT>::kDownFlight, SB = KFmt<QT>::kSB;
  const ExpertList &L = DEV ? *a.Ld : a.L;
  const int I = a.I, ni = I / 128, n = a.L.n, pb = plane_bytes(I);
  uint8_t *qL = smem8;
  float *scL = reinterpret_cast<float *>(smem8 + 3 * n * pb);
  int *dsL = reinterpret_cast<int *>(scL + n * (I / 16));
  float *res = reinterpret_cast<float *>(dsL + 3 * n * (I / 16));
  const int j0 = blockIdx.x * a.rows;
  const int unit = threadIdx.x >> a.lanes_log2, l = threadIdx.x & (a.lanes - 1);
  const int i = unit / a.rows, rr = unit - i * a.rows, j = j0 + rr, ic = min(i, n - 1);
  const bool active = i < n && j < a.H;
  const int64_t rowb = (int64_t)(I / 256) * SB;
  const int ndev = L.n;
  const uint8_t *const payload = L.payload[ic];
  const int pos_t = (int)threadIdx.x < n ? L.pos[threadIdx.x] : 0;
  if (ndev != n) return;  // a device list emptied by a routing error (uniform)
  if ((int)threadIdx.x < n) posL[threadIdx.x] = pos_t;
  __syncthreads();
  const uint8_t *row = payload + a.down_off + (int64_t)min(j, a.H - 1) * rowb;
  HStage st;
  stage_h_load(a.hq, a.hsc, a.hds, posL, n, I, a.k, QT == 12, st);
  __builtin_amdgcn_sched_barrier(0);
  const float w_t = a.w[posL[min((int)threadIdx.x, n - 1)]];
  const int jt = j0 + (int)threadIdx.x;
  const bool out_t = (int)threadIdx.x < a.rows && jt < a.H;
  const float base_ld = (a.mode == 1 ? a.x : a.y)[min(jt, a.H - 1)];
  const float base_t = a.mode == 0 ? 0.f : base_ld;
  uint32_t wd[F][DW];
  int sh[F];
#pragma unroll
  for (int m = 0; m < F; ++m) {
    const int it = l + m * a.lanes;
    sh[m] = load_item<QT>(row, (active && m < a.mpairs && it < ni) ? it : 0, wd[m]);
  }
  __builtin_amdgcn_sched_barrier(0);
  stage_h_store(st, n, I, QT == 12, qL, scL, dsL, dummyL);
  __syncthreads();
  float acc = 0.f;
  for (int m0 = 0; m0 < a.mpairs; m0 += F) {
    if (m0 > 0) {
#pragma unroll
      for (int m = 0; m < F; ++m) {
        const int it = l + (m0 + m) * a.lanes;
        if (active && m0 + m < a.mpairs && it < ni) sh[m] = load_item<QT>(row, it, wd[m]);
      }
    }
#pragma unroll
    for (int m = 0; m < F; ++m) {
      const int it = l + (m0 + m) * a.lanes;
      if (active && m0 + m < a.mpairs && it < ni)
        acc += item_dot<QT, true>(wd[m], sh[m], qL + 3 * i * pb, pb, it, scL + i * (I / 16),
                                  dsL + 3 * i * (I / 16), I / 16);
    }
  }
  acc = group_sum(acc, a.lanes);
  if (active && l == 0) res[rr * n + i] = acc;
  if ((int)threadIdx.x < n) wL[threadIdx.x] = w_t;
  __syncthreads();
  if (out_t) {
    float v = 0.f;  // rows first, then the residual / earlier sum (as down_kernel)
    for (int ii = 0; ii < n; ++ii) v = fmaf(wL[ii], res[threadIdx.x * n + ii], v);
    a.y[jt] = base_t + v;
  }
}

// Copy the payloads of the listed misses (P bytes each, 16-byte aligned) from
// the store into their slots: 16-byte loads and stores, four in flight per
// thread, grid-strided over all misses' bytes.
constexpr int kMaxCopy = 64;
// ------------------------------------------- small multi-token calls ---
//
// The decode GEMVs over the union of a small call's experts: a block takes
// one union expert's rows, holds each lane's weight pairs in registers and
// forms the dot products with every token routing to that expert, in the
// same lane, pair and summation order as the per-token kernels, so each
// token's activations and output rows are those of gateup_kernel /
// down_kernel.

struct GateUpMtParams {
  const MtWork *W;
  const int8_t *xq;  // [T][3][H] token digits
  const float *xsc;  // [T][H/32]
  int8_t *hq;        // [3][T*k*I]
  float *hsc;        // [T*k*I/16]
  int32_t *hds;      // [3][T*k*I/16] (unused: no union format needs digit sums)
  int H, I, k, T;
  int lanes, mpairs, lanes_log2;
};

// One token's LDS image for the gate/up GEMV: digit planes, block scales, digit sums.
__device__ __forceinline__ int mt_image_bytes(int H) { return 3 * plane_bytes(H) + 16 * (H / 32); }

// Block blk: union expert blk / bpe, rows from (blk % bpe) * (256 / lanes).
// Dynamic LDS: T images, then [kMtTokens][256 / lanes] floats.  hits_only:
// the experts copied in by the same launch are left to its copy blocks.
template <int QT>
__device__ __forceinline__ void gateup_mt_body(const GateUpMtParams &a, bool hits_only, int blk,
                                               uint8_t *smem8) {
  __shared__ __align__(16) uint8_t dummyL[16];
  __shared__ int qL[kMtTokens];
  constexpr int BB = Fmt<QT>::kBlockBytes, PD = Fmt<QT>::kPairDwords, F = Fmt<QT>::kGateUpFlight;
  const int H = a.H, nb = H / 32, np = nb / 2, pb = plane_bytes(H), img = mt_image_bytes(H);
  const int upb = kThreads / a.lanes;
  const int bpe = (a.I + upb - 1) / upb;
  const int u = blk / bpe;  // < kMtMaxCopy (the launch bounds the grid)
  // the union's size, this expert's slot, token count and positions (one round trip)
  const int nu = a.W->n_union;
  const uint8_t *const payload = a.W->upay[u];
  const int nt = a.W->unt[u], hit = a.W->uhit[u];
  const int q_t = (int)threadIdx.x < kMtTokens ? a.W->uq[u][threadIdx.x] : 0;
  if (u >= nu || payload == nullptr || (hits_only && !hit)) return;  // uniform over the block
  if ((int)threadIdx.x < kMtTokens) qL[threadIdx.x] = q_t;
  const int r0 = (blk - u * bpe) * upb;
  const int r = r0 + (threadIdx.x >> a.lanes_log2);
  const int l = threadIdx.x & (a.lanes - 1);
  const bool active = r < a.I;
  const int64_t rowb = (int64_t)nb * BB, mat = (int64_t)a.I * rowb;
  const uint8_t *gate = payload + (int64_t)r * rowb, *up = gate + mat;
  const uint8_t *gatev = payload + (int64_t)min(r, a.I - 1) * rowb, *upv = gatev + mat;
  uint32_t wg[F][PD], wu[F][PD];
#pragma unroll
  for (int m = 0; m < F; ++m) {
    const int p = l + m * a.lanes;
    const bool ok = active && m < a.mpairs && p < np;
    load_pair<QT>(ok ? gate + (int64_t)p * 2 * BB : gatev, wg[m]);
    load_pair<QT>(ok ? up + (int64_t)p * 2 * BB : upv, wu[m]);
  }
  __syncthreads();
  // the digits of the tokens routing here while the weights are in flight
  for (int i = 0; i < nt; ++i) {
    const int t = qL[i] / a.k;
    uint8_t *im = smem8 + i * img;
    stage_token(a.xq + (int64_t)t * 3 * H, a.xsc + (int64_t)t * nb, H, im,
                reinterpret_cast<float *>(im + 3 * pb), dummyL);
  }
  __syncthreads();
  float g[kMtTokens], v[kMtTokens];
#pragma unroll
  for (int i = 0; i < kMtTokens; ++i) g[i] = v[i] = 0.f;
  for (int m0 = 0; m0 < a.mpairs; m0 += F) {
    if (m0 > 0) {
#pragma unroll
      for (int m = 0; m < F; ++m) {
        const int p = l + (m0 + m) * a.lanes;
        if (active && m0 + m < a.mpairs && p < np) {
          load_pair<QT>(gate + (int64_t)p * 2 * BB, wg[m]);
          load_pair<QT>(up + (int64_t)p * 2 * BB, wu[m]);
        }
      }
    }
#pragma unroll
    for (int m = 0; m < F; ++m) {
      const int p = l + (m0 + m) * a.lanes;
      if (active && m0 + m < a.mpairs && p < np) {
#pragma unroll
        for (int i = 0; i < kMtTokens; ++i) {
          if (i < nt) {
            const uint8_t *im = smem8 + i * img;
            const float *scL = reinterpret_cast<const float *>(im + 3 * pb);
            uint32_t D[48];
            load_digits(im, pb, p, D);
            const float s0 = scL[2 * p], s1 = scL[2 * p + 1];
            g[i] += pair_dot<QT>(wg[m], D, s0, s1);
            v[i] += pair_dot<QT>(wu[m], D, s0, s1);
          }
        }
      }
    }
  }
  float *hL = reinterpret_cast<float *>(smem8 + a.T * img);  // [kMtTokens][upb]
#pragma unroll
  for (int i = 0; i < kMtTokens; ++i) {
    if (i < nt) {  // uniform
      const float gs = group_sum(g[i], a.lanes), us = group_sum(v[i], a.lanes);
      if (l == 0) hL[i * upb + (threadIdx.x >> a.lanes_log2)] = active ? silu(gs) * us : 0.f;
    }
  }
  __syncthreads();
  if ((int)threadIdx.x < upb)
    for (int i = 0; i < nt; ++i)
      store_h_digits<QT>(hL[i * upb + threadIdx.x], qL[i], r0 + threadIdx.x, a.I, a.T * a.k, a.hq,
                         a.hsc, a.hds);
}

// grid: umax * bpe blocks (gateup_mt_body).
template <int QT>
__global__ __launch_bounds__(kThreads) void gateup_mt_kernel(GateUpMtParams a) {
  extern __shared__ __align__(16) uint8_t smem8[];
  gateup_mt_body<QT>(a, false, blockIdx.x, smem8);
}

// Copy + gate/up of a small multi-token call in one launch, as
// copy_gateup_kernel does for one token: blocks [0, copy_blocks) move the
// misses' payloads in chunks of R rows of W_gate and W_up (then the down
// matrix) and form, from the rows in LDS, the activations of every token
// routing to the copied expert; the blocks after them run gateup_mt_body for
// the union's hit experts.  Per (token, row) the lanes, pair order and sums
// are gateup_mt_body's, so the activations are bit-identical to its result.
struct CopyGateUpMtParams {
  GateUpMtParams g;  // token digits, activation outputs, shape, hit-block lanes
  int64_t P;
  int copy_blocks, R;  // rows per chunk (R divides 16 and 256 / lanes)
  uint64_t *acc;       // nullable: += copies, += bytes
};

// Dynamic LDS: the T token images, hL [kMtTokens][16] floats, one chunk (2 R
// rows); at least what gateup_mt_body takes.
template <int QT>
__global__ __launch_bounds__(kThreads) void copy_gateup_mt_kernel(CopyGateUpMtParams a) {
  extern __shared__ __align__(16) uint8_t smem8[];
  const MtWork &W = *a.g.W;
  if ((int)blockIdx.x >= a.copy_blocks) {  // gate/up of a hit expert
    gateup_mt_body<QT>(a.g, true, blockIdx.x - a.copy_blocks, smem8);
    return;
  }
  const int n = W.n_copy;
  if (n == 0) return;
  if (a.acc && blockIdx.x == 0 && threadIdx.x == 0) {
    atomicAdd(reinterpret_cast<unsigned long long *>(a.acc), (unsigned long long)n);
    atomicAdd(reinterpret_cast<unsigned long long *>(a.acc + 1), (unsigned long long)(n * a.P));
  }
  constexpr int BB = Fmt<QT>::kBlockBytes;
  const int H = a.g.H, I = a.g.I, T = a.g.T, k = a.g.k;
  const int nb = H / 32, pb = plane_bytes(H), img = mt_image_bytes(H);
  float *hL = reinterpret_cast<float *>(smem8 + T * img);  // [kMtTokens][16]
  uint8_t *cL = reinterpret_cast<uint8_t *>(hL + kMtTokens * 16);
  __shared__ int qL[kMtTokens];  // positions of the tokens of the chunk's expert
  const int R = a.R, cpu = 16 / R;
  const int64_t rowb = (int64_t)nb * BB, half = R * rowb;
  const int h16 = (int)(half / 16);
  const int upm = I / 16 + I / 32;
  const int n_units = n * upm;
  int u = blockIdx.x;
  if (u >= n_units) return;  // uniform
  __shared__ __align__(16) uint8_t dummyL[16];
  for (int t = 0; t < T; ++t) {
    uint8_t *im = smem8 + t * img;
    stage_token(a.g.xq + (int64_t)t * 3 * H, a.g.xsc + (int64_t)t * nb, H, im,
                reinterpret_cast<float *>(im + 3 * pb), dummyL);
  }
  // chunk c of unit uu: its two spans, the miss's union index, token count
  // and (threads < kMtTokens) token positions
  auto spans = [&](int uu, int c, const uint8_t *&s0, const uint8_t *&s1, uint8_t *&d0, uint8_t *&d1,
                   int &g, int &nt, int &q) -> bool {
    const int miss = uu / upm;
    const int j = uu - miss * upm;
    int64_t o0, o1;
    const bool gu = chunk_spans(j, c, I, R, rowb, o0, o1);
    g = gu ? j : -1;
    s0 = W.src[miss] + o0;
    s1 = W.src[miss] + o1;
    d0 = W.dst[miss] + o0;
    d1 = W.dst[miss] + o1;
    const int um = W.mu[miss];
    nt = W.unt[um];
    q = W.uq[um][threadIdx.x & (kMtTokens - 1)];
    return gu;
  };
  uint4 buf[kChunkSlots];
  const uint8_t *s0, *s1;
  uint8_t *d0, *d1;
  int g, nt, q, c = 0;
  bool gu = spans(u, 0, s0, s1, d0, d1, g, nt, q);
  load_chunk(s0, s1, h16, buf);
  const int L = a.g.lanes, rr = threadIdx.x >> a.g.lanes_log2, l = threadIdx.x & (L - 1);
  const int tpp = (kThreads / L) / R;  // tokens per pass: row slot rr -> token rr / R, row rr % R
  const int ri = rr % R;
  for (;;) {
    store_chunk(buf, d0, d1, h16, gu, cL);
    if (gu && (int)threadIdx.x < kMtTokens) qL[threadIdx.x] = q;
    const bool cur_gu = gu;
    const int cur_c = c, cur_g = g, cur_nt = nt;
    if (++c == cpu) {
      c = 0;
      u += a.copy_blocks;
    }
    const bool more = u < n_units;
    if (more) {
      gu = spans(u, c, s0, s1, d0, d1, g, nt, q);
      load_chunk(s0, s1, h16, buf);
    }
    __syncthreads();  // chunk and positions in LDS
    if (cur_gu) {
      for (int i0 = 0; i0 < cur_nt; i0 += tpp) {
        const int i = i0 + rr / R;
        const bool act = i < cur_nt;
        const uint8_t *im = smem8 + (act ? qL[i] / k : 0) * img;
        float gs, us;
        chunk_row_dots<QT>(cL, ri, rowb, half, im, pb, reinterpret_cast<const float *>(im + 3 * pb),
                           reinterpret_cast<const int *>(im + 3 * pb + 4 * nb), nb, l, L, act, gs, us);
        gs = group_sum(gs, L);
        us = group_sum(us, L);
        if (l == 0 && act) hL[i * 16 + cur_c * R + ri] = silu(gs) * us;
      }
      if (cur_c == cpu - 1) {
        __syncthreads();
        if ((int)threadIdx.x < 16 * cur_nt) {
          const int i = threadIdx.x >> 4, row = threadIdx.x & 15;
          store_h_digits<QT>(hL[threadIdx.x], qL[i], 16 * cur_g + row, I, T * k, a.g.hq, a.g.hsc,
                             a.g.hds);
        }
      }
    }
    __syncthreads();  // LDS free for the next chunk
    if (!more) break;
  }
}

struct DownMtParams {
  const MtWork *W;
  const int8_t *hq;  // [3][T*k*I]
  const float *hsc;
  const int32_t *hds;
  float *R;  // [T*k][H]
  int H, I, k, T;
  int lanes, mpairs, lanes_log2, rows;  // rows = 256 / lanes
};

// grid: umax * ceil(H / rows) blocks; block b: union expert b / bpe, output
// rows from (b % bpe) * rows.  Dynamic LDS: the h digit images of T positions.
template <int QT>
__global__ __launch_bounds__(kThreads) void down_mt_kernel(DownMtParams a) {
  extern __shared__ __align__(16) uint8_t smem8[];
  __shared__ int posL[kMtTokens];
  __shared__ __align__(16) uint8_t dummyL[16];
  constexpr int BB = Fmt<QT>::kBlockBytes, PD = Fmt<QT>::kPairDwords, F = Fmt<QT>::kDownFlight;
  const int I = a.I, nb = I / 32, np = nb / 2, pb = plane_bytes(I);
  const int bpe = (a.H + a.rows - 1) / a.rows;
  const int u = blockIdx.x / bpe;
  const int nu = a.W->n_union;
  const uint8_t *const payload = a.W->upay[u];
  const int nt = a.W->unt[u];
  const int q_t = (int)threadIdx.x < kMtTokens ? a.W->uq[u][threadIdx.x] : 0;
  if (u >= nu || payload == nullptr) return;  // uniform
  if ((int)threadIdx.x < kMtTokens) posL[threadIdx.x] = q_t;
  __syncthreads();
  uint8_t *qL = smem8;                                          // nt digit images
  float *scL = reinterpret_cast<float *>(smem8 + 3 * a.T * pb);  // [nt][I/16]
  int *dsL = reinterpret_cast<int *>(scL + a.T * (I / 16));      // [nt][3][I/16]
  const int j = (blockIdx.x - u * bpe) * a.rows + (threadIdx.x >> a.lanes_log2);
  const int l = threadIdx.x & (a.lanes - 1);
  const bool active = j < a.H;
  const int64_t rowb = (int64_t)nb * BB;
  const int64_t mat = (int64_t)I * ((int64_t)(a.H / 32) * BB);
  const uint8_t *row = payload + 2 * mat + (int64_t)j * rowb;
  const uint8_t *rowv = payload + 2 * mat + (int64_t)min(j, a.H - 1) * rowb;
  HStage st;
  stage_h_load(a.hq, a.hsc, a.hds, posL, nt, I, a.T * a.k, false, st);  // ahead of the weights
  __builtin_amdgcn_sched_barrier(0);
  uint32_t wd[F][PD];
#pragma unroll
  for (int m = 0; m < F; ++m) {
    const int p = l + m * a.lanes;
    const bool ok = active && m < a.mpairs && p < np;
    load_pair<QT>(ok ? row + (int64_t)p * 2 * BB : rowv, wd[m]);
  }
  __builtin_amdgcn_sched_barrier(0);
  stage_h_store(st, nt, I, false, qL, scL, dsL, dummyL);
  __syncthreads();
  float acc[kMtTokens];
#pragma unroll
  for (int i = 0; i < kMtTokens; ++i) acc[i] = 0.f;
  for (int m0 = 0; m0 < a.mpairs; m0 += F) {
    if (m0 > 0) {
#pragma unroll
      for (int m = 0; m < F; ++m) {
        const int p = l + (m0 + m) * a.lanes;
        if (active && m0 + m < a.mpairs && p < np) load_pair<QT>(row + (int64_t)p * 2 * BB, wd[m]);
      }
    }
#pragma unroll
    for (int m = 0; m < F; ++m) {
      const int p = l + (m0 + m) * a.lanes;
      if (active && m0 + m < a.mpairs && p < np) {
#pragma unroll
        for (int i = 0; i < kMtTokens; ++i) {
          if (i < nt) {
            uint32_t D[48];
            load_digits(qL + 3 * i * pb, pb, p, D);
            acc[i] += pair_dot16<QT>(wd[m], D, scL + i * (I / 16) + 4 * p);
          }
        }
      }
    }
  }
#pragma unroll
  for (int i = 0; i < kMtTokens; ++i) {
    if (i < nt) {  // uniform
      const float s = group_sum(acc[i], a.lanes);
      if (active && l == 0) a.R[(int64_t)posL[i] * a.H + j] = s;
    }
  }
}

// y_t[j] = (x_t[j] if mode 1) + sum over ranks r of w[t*k+r] R[t*k+r][j], in rank order.
// W (nullable): the device work list of the call; an empty one (the union
// did not fit the slots, or routing failed) leaves y untouched.
__global__ __launch_bounds__(kThreads) void combine_mt_kernel(const float *__restrict__ R,
                                                              const float *__restrict__ w,
                                                              const float *__restrict__ x,
                                                              float *__restrict__ y, int H, int k,
                                                              int mode, const MtWork *W) {
  const int t = blockIdx.y, j = blockIdx.x * kThreads + threadIdx.x;
  if (j >= H || (W && W->n_union == 0)) return;
  float v = 0.f;  // rows first, then the residual (one rounding at its scale)
  for (int r = 0; r < k; ++r) v = fmaf(w[t * k + r], R[((int64_t)t * k + r) * H + j], v);
  y[(int64_t)t * H + j] = mode == 1 ? x[(int64_t)t * H + j] + v : v;
}

struct CopyParams {
  const uint4 *src[kMaxCopy];
  uint4 *dst[kMaxCopy];
  int n;
  int64_t p16;  // payload size in 16-byte units
};

__global__ __launch_bounds__(kThreads) void materialize_kernel(CopyParams a) {
  const int64_t total = a.p16 * a.n;
  const int64_t st = (int64_t)gridDim.x * kThreads;
  int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  for (; i + 3 * st < total; i += 4 * st) {
    uint4 v[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int64_t g = i + j * st, e = g / a.p16;
      v[j] = a.src[e][g - e * a.p16];
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int64_t g = i + j * st, e = g / a.p16;
      a.dst[e][g - e * a.p16] = v[j];
    }
  }
  for (; i < total; i += st) {
    const int64_t e = i / a.p16;
    a.dst[e][i - e * a.p16] = a.src[e][i - e * a.p16];
  }
}

// The same copy for the misses a device work list names.
template <class Work>
__global__ __launch_bounds__(kThreads) void materialize_list_kernel(const Work *w, int64_t p16,
                                                                    uint64_t *acc) {
  const int n = w->n_copy;
  if (acc && blockIdx.x == 0 && threadIdx.x == 0) {
    atomicAdd(reinterpret_cast<unsigned long long *>(acc), (unsigned long long)n);
    atomicAdd(reinterpret_cast<unsigned long long *>(acc + 1), (unsigned long long)(n * p16 * 16));
  }
  const int64_t total = p16 * n;
  const int64_t st = (int64_t)gridDim.x * kThreads;
  int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  const uint4 *const *src = reinterpret_cast<const uint4 *const *>(w->src);
  uint4 *const *dst = reinterpret_cast<uint4 *const *>(w->dst);
  for (; i + 3 * st < total; i += 4 * st) {
    uint4 v[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int64_t g = i + j * st, e = g / p16;
      v[j] = src[e][g - e * p16];
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int64_t g = i + j * st, e = g / p16;
      dst[e][g - e * p16] = v[j];
    }
  }
  for (; i < total; i += st) {
    const int64_t e = i / p16;
    dst[e][i - e * p16] = src[e][i - e * p16];
  }
}

// ---------------------------------------------------------------- prefill ---
//
// A multi-token layer call: per-token RMS scale and the scaled input as two
// bf16 terms (hi = bf16(v), lo = bf16(v - hi): about 16 significant bits),
// router logits + top-k, grouping of the (token, expert) pairs by expert (a
// stable counting sort: pairs keep token order), then, wave by wave of at
// most C experts, the copy kernel for the wave's misses and two MFMA grouped
// GEMMs with the weights dequantised to bf16 on the fly (each activation tile
// is multiplied as hi and lo, both into the same fp32 accumulators):
//   gate/up:  A_e = silu(X_e W_gate^T) * (X_e W_up^T)   [n_e, I], kept as hi + lo
//   down:     P[pair] = w_pair * (A_e W_down^T)[row]     [n_e, H]
// and finally y[t] = (x[t] +) sum over the token's k pairs, in rank order.


// inv[t] = 1/sqrt(mean(x_t^2) + 1e-6) (or 1); v = x_t * inv[t] as
// xb[t] = bf16(v) and xb[T*H + t] = bf16(v - bf16(v)).
__global__ __launch_bounds__(kThreads) void prefill_prep_kernel(const float *__restrict__ x, int T,
                                                                int H, int prenorm,
                                                                float *__restrict__ inv,
                                                                __bf16 *__restrict__ xb) {
  __shared__ float wsum[kThreads / kWave];
  const int t = blockIdx.x;
  const float *xt = x + (int64_t)t * H;
  float ss = 0.f;
  if (prenorm)
    for (int i = threadIdx.x; i < H; i += kThreads) ss = fmaf(xt[i], xt[i], ss);
#pragma unroll
  for (int off = kWave / 2; off >= 1; off >>= 1) ss += __shfl_xor(ss, off, kWave);
  if ((threadIdx.x & (kWave - 1)) == 0) wsum[threadIdx.x / kWave] = ss;
  __syncthreads();
  float tot = 0.f;
#pragma unroll
  for (int i = 0; i < kThreads / kWave; ++i) tot += wsum[i];
  const float s = prenorm ? 1.f / sqrtf(tot / (float)H + 1e-6f) : 1.f;
  if (threadIdx.x == 0) inv[t] = s;
  // eight consecutive values per thread (H % 64 == 0): two 16-byte loads, one
  // 16-byte store to each plane
  __bf16 *hi8 = xb + (int64_t)t * H, *lo8 = xb + (int64_t)T * H + (int64_t)t * H;
  for (int i = 8 * threadIdx.x; i < H; i += 8 * kThreads) {
    const float4 a = *reinterpret_cast<const float4 *>(xt + i), b = *reinterpret_cast<const float4 *>(xt + i + 4);
    const float v[8] = {a.x * s, a.y * s, a.z * s, a.w * s, b.x * s, b.y * s, b.z * s, b.w * s};
    __bf16 h[8], l[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      h[j] = (__bf16)v[j];
      l[j] = (__bf16)(v[j] - (float)h[j]);
    }
    *reinterpret_cast<uint4 *>(hi8 + i) = *reinterpret_cast<const uint4 *>(h);
    *reinterpret_cast<uint4 *>(lo8 + i) = *reinterpret_cast<const uint4 *>(l);
  }
}

// Grouping of the (token, rank) pairs by expert (a stable counting sort) in two
// launches over chunks of the pair list: group_hist_kernel counts each chunk's
// pairs per expert, group_place_kernel gives every pair its place.  The pairs
// of expert e are perm[offsets[e] .. offsets[e+1]) in pair order: those of
// earlier chunks first, and inside a chunk by rank (earlier rounds of 256
// pairs, earlier waves of the round, earlier lanes of the wave).
constexpr int kGroupChunks = 512;  // most chunks per call (rows of the count table)

// counts[c][e] = pairs of chunk c (pairs c*chunk .. +chunk) routed to e.
__global__ __launch_bounds__(kThreads) void group_hist_kernel(const int32_t *__restrict__ idx, int npairs,
                                                              int E, int chunk, int32_t *__restrict__ counts) {
  __shared__ int h[kThreads];  // E <= 256
  if ((int)threadIdx.x < E) h[threadIdx.x] = 0;
  __syncthreads();
  const int p0 = blockIdx.x * chunk, p1 = min(npairs, p0 + chunk);
#pragma unroll 4
  for (int p = p0 + (int)threadIdx.x; p < p1; p += kThreads) {
    const int e = idx[p];
    if ((unsigned)e < (unsigned)E) atomicAdd(&h[e], 1);  // an invalid id is left out (the host
  }                                                       // then sees offsets[E] != npairs)
  __syncthreads();
  if ((int)threadIdx.x < E) counts[(int64_t)blockIdx.x * E + threadIdx.x] = h[threadIdx.x];
}

// Exclusive prefix sum of v over the block's threads (all threads call it).
__device__ __forceinline__ int block_exclusive_scan(int v, int *wsum, int &total) {
  const int lane = threadIdx.x & (kWave - 1), wv = threadIdx.x / kWave;
  int inc = v;
#pragma unroll
  for (int off = 1; off < kWave; off <<= 1) {
    const int o = __shfl_up(inc, off, kWave);
    if (lane >= off) inc += o;
  }
  if (lane == kWave - 1) wsum[wv] = inc;
  __syncthreads();
  int before = 0;
  total = 0;
#pragma unroll
  for (int w = 0; w < kThreads / kWave; ++w) {
    if (w < wv) before += wsum[w];
    total += wsum[w];
  }
  return before + inc - v;
}

// Block c: the first place of its pairs of each expert (offsets[e] plus the
// pairs of e in earlier chunks), then its pairs round by round: a pair's rank
// among the round's pairs of its expert is the count in earlier waves plus the
// lanes before it in its wave with the same expert (eight ballots on the id's
// bits).  Block 0 also writes offsets [E + 1].
__global__ __launch_bounds__(kThreads) void group_place_kernel(const int32_t *__restrict__ idx, int npairs,
                                                               int E, int chunk, int nchunks,
                                                               const int32_t *__restrict__ counts,
                                                               int32_t *__restrict__ offsets,
                                                               int32_t *__restrict__ perm) {
  constexpr int NW = kThreads / kWave;
  __shared__ int base[kThreads];
  __shared__ int wc[NW][kThreads];  // pairs of each expert in each wave of the round
  __shared__ int wsum[NW];
  const int tid = threadIdx.x, lane = tid & (kWave - 1), wv = tid / kWave, c = blockIdx.x;
  int tot = 0, before = 0;
  if (tid < E)
    for (int q0 = 0; q0 < nchunks; q0 += 16) {  // 16 loads in flight
      int v[16];
#pragma unroll
      for (int u = 0; u < 16; ++u) v[u] = counts[(int64_t)min(q0 + u, nchunks - 1) * E + tid];
#pragma unroll
      for (int u = 0; u < 16; ++u) {
        const int q = q0 + u;
        tot += q < nchunks ? v[u] : 0;
        before += q < c ? v[u] : 0;
      }
    }
  int total = 0;
  const int first = block_exclusive_scan(tid < E ? tot : 0, wsum, total);
  if (tid < E) {
    base[tid] = first + before;
#pragma unroll
    for (int w = 0; w < NW; ++w) wc[w][tid] = 0;
    if (c == 0) offsets[tid] = first;
  }
  if (c == 0 && tid == 0) offsets[E] = total;
  __syncthreads();
  const int p0 = c * chunk, p1 = min(npairs, p0 + chunk);
  for (int r0 = p0; r0 < p1; r0 += kThreads) {  // uniform
    const int p = r0 + tid;
    const int ep = idx[min(p, p1 - 1)];
    const bool ok = p < p1 && (unsigned)ep < (unsigned)E;
    const int e = ok ? ep : 0;
    uint64_t peers = __ballot(ok);
#pragma unroll
    for (int b = 0; b < 8; ++b) {
      const bool bit = (e >> b) & 1;
      const uint64_t m = __ballot(ok && bit);
      peers &= bit ? m : ~m;
    }
    const uint64_t below = peers & ((1ull << lane) - 1ull);
    if (ok && below == 0) wc[wv][e] = __popcll(peers);
    __syncthreads();
    if (ok) {
      int pos = base[e] + __popcll(below);
      for (int w = 0; w < wv; ++w) pos += wc[w][e];
      perm[pos] = p;
    }
    __syncthreads();
    if (tid < E) {
      int add = 0;
#pragma unroll
      for (int w = 0; w < NW; ++w) {
        add += wc[w][tid];
        wc[w][tid] = 0;
      }
      base[tid] += add;
    }
    __syncthreads();
  }
}

// One wave's experts for the grouped GEMMs (kernel argument, about 3 KB).
constexpr int kPfMaxExperts = 128;
constexpr int kPfMaxTiles = 512;
struct PfExperts {
  const uint8_t *payload[kPfMaxExperts];
  int32_t row0[kPfMaxExperts];  // first row of the expert's pairs in perm / Ab
  int32_t n[kPfMaxExperts];     // pairs (tokens) routed to it
  int32_t count;
  // flat M-tile t (128 rows): expert in the low byte, the expert's M-tile in the
  // high byte; ntiles == 0 when the launch's tiles do not fit (then a scan)
  int32_t ntiles;
  uint16_t tile[kPfMaxTiles];
};

constexpr int kPfBM = 128;  // tokens per tile
constexpr int kPfBK = 64;   // one pair of weight blocks per row
constexpr int kPfLd = kPfBK + 8;  // LDS row stride in bf16 (padding against bank conflicts)

// (expert, M-tile) of a flat M-tile index; returns false past the end.  One
// lookup in the launch's tile table (a scan over the experts, one dependent
// scalar load each, took microseconds for the last tiles of a launch).
__device__ __forceinline__ bool pf_tile(const PfExperts &X, int mt, int &j, int &m0) {
  if (X.ntiles > 0) {
    if (mt >= X.ntiles) return false;
    const uint32_t v = X.tile[mt];
    j = (int)(v & 0xffu);
    m0 = (int)(v >> 8) * kPfBM;
    return true;
  }
  for (j = 0; j < X.count; ++j) {
    const int tiles = (X.n[j] + kPfBM - 1) / kPfBM;
    if (mt < tiles) {
      m0 = mt * kPfBM;
      return true;
    }
    mt -= tiles;
  }
  return false;
}

// Dequantise one 32-weight block (half a pair) of a weight row to bf16.  The
// thread loads the 9 dwords of its half of the pair: half 0 = bytes 0..35,
// half 1 = bytes 32..67 (Q8_0) / half 0 = bytes 0..19, half 1 = 16..35 (Q4_0).
template <int QT>
__device__ __forceinline__ void load_half(const uint8_t *pair, int half, uint32_t (&v)[9]) {
  const uint32_t *q = reinterpret_cast<const uint32_t *>(pair) + (QT == 8 ? 8 * half : 4 * half);
  constexpr int n = QT == 8 ? 9 : 5;
#pragma unroll
  for (int i = 0; i < n; ++i) v[i] = q[i];
}

// The 32 bf16 weights of one block (as loaded by load_half) into dst (16-byte
// aligned), rounded to nearest even from the exact fp32 value d*q.
template <int QT>
__device__ __forceinline__ void dequant_half(const uint32_t (&v)[9], int half, __bf16 *dst) {
  __bf16 o[32];
  if constexpr (QT == 8) {
    // half 0 holds bytes 0..35: d = bytes 0-1, q = bytes 2..33;
    // half 1 holds bytes 32..67: d = bytes 34-35, q = bytes 36..67
    const float d = half_bits_to_float(half == 0 ? (v[0] & 0xffffu) : (v[0] >> 16));
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const uint32_t w = half == 0 ? __builtin_amdgcn_alignbyte(v[j + 1], v[j], 2) : v[j + 1];
#pragma unroll
      for (int b = 0; b < 4; ++b) o[4 * j + b] = (__bf16)(d * (float)(int8_t)((w >> (8 * b)) & 0xff));
    }
  } else {
    // half 0 holds bytes 0..19: d = bytes 0-1, nibble bytes 2..17;
    // half 1 holds bytes 16..35: d = bytes 18-19, nibble bytes 20..35
    const float d = half_bits_to_float(half == 0 ? (v[0] & 0xffffu) : (v[0] >> 16));
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const uint32_t w = half == 0 ? __builtin_amdgcn_alignbyte(v[j + 1], v[j], 2) : v[j + 1];
#pragma unroll
      for (int b = 0; b < 4; ++b) {
        const uint32_t byte = (w >> (8 * b)) & 0xff;
        o[4 * j + b] = (__bf16)(d * (float)((int)(byte & 0xf) - 8));
        o[16 + 4 * j + b] = (__bf16)(d * (float)((int)(byte >> 4) - 8));
      }
    }
  }
#pragma unroll
  for (int i = 0; i < 4; ++i)
    *reinterpret_cast<uint4 *>(dst + 8 * i) = *reinterpret_cast<const uint4 *>(o + 8 * i);
}

struct PfGateUpParams {
  PfExperts X;
  const int32_t *perm;
  const __bf16 *xb;  // [2][T][H]: hi then lo
  __bf16 *ab;        // [2][pairs][I]: hi then lo
  int T, pairs, H, I, k;
};

// MFMA operand of v_mfma_f32_16x16x32_bf16 read straight from global memory:
// lane l holds row l % 16 of a 16-row subtile and k = 8 * (l / 16) .. +7 of a
// 32-wide k slice (16 bytes).  Activation rows are private to the wave that
// multiplies them, so they skip LDS; only the dequantised weight tile, which
// all four waves read, is staged there (three 18 KB buffers, two blocks per CU).
typedef __attribute__((address_space(1))) const bf16x8 g_bf16x8;

// The K loop of both grouped GEMMs (K steps of 64) with two steps of
// prefetch: three register sets (A: activation fragments, B: the raw weight
// blocks of a step) rotate with three LDS weight buffers.  Step kt multiplies
// set kt % 3 from Bs[kt % 3], dequantises the weights of step kt + 1 into
// Bs[(kt + 1) % 3] and loads step kt + 2 (clamped to KT - 1) into set
// (kt + 2) % 3.  Loads are issued unconditionally so that the wait counts the
// compiler places are exact; the scheduling barriers keep the loads ahead of
// the MFMAs and the dequantisation after them.  Two steps in flight cover the
// global loads' latency also while the host-copy kernel runs beside the GEMMs
// (which inflates it): there the one-step loop took 1.3-1.9x as long.
#define PF_STEP(S, KT, kt, GLOAD, MMA, DEQ)                             \
  do {                                                                  \
    GLOAD(min((kt) + 2, (KT) - 1), A[((S) + 2) % 3], B[((S) + 2) % 3]); \
    __builtin_amdgcn_sched_barrier(0);                                  \
    MMA(A[(S)], (S));                                                   \
    __builtin_amdgcn_sched_barrier(0);                                  \
    DEQ(B[((S) + 1) % 3], ((S) + 1) % 3);                               \
    __syncthreads();                                                    \
  } while (0)
// GM_K_LOOP: as PF_K_LOOP for the 256-row tiles, whose dequantiser also takes
// the K step (the K-quant formats locate a step's scales from it).
#define GM_STEP(S, KT, kt, GLOAD, MMA, DEQ)                             \
  do {                                                                  \
    GLOAD(min((kt) + 2, (KT) - 1), A[((S) + 2) % 3], B[((S) + 2) % 3]); \
    __builtin_amdgcn_sched_barrier(0);                                  \
    MMA(A[(S)], (S));                                                   \
    __builtin_amdgcn_sched_barrier(0);                                  \
    DEQ(B[((S) + 1) % 3], ((S) + 1) % 3, min((kt) + 1, (KT) - 1));      \
    __syncthreads();                                                    \
  } while (0)
#define GM_K_LOOP(KT, GLOAD, MMA, DEQ)                                  \
  do {                                                                  \
    GLOAD(0, A[0], B[0]);                                               \
    GLOAD(min(1, (KT) - 1), A[1], B[1]);                                \
    DEQ(B[0], 0, 0);                                                    \
    __syncthreads();                                                    \
    int kt_ = 0;                                                        \
    for (; kt_ + 3 <= (KT); kt_ += 3) {                                 \
      GM_STEP(0, KT, kt_, GLOAD, MMA, DEQ);                             \
      GM_STEP(1, KT, kt_ + 1, GLOAD, MMA, DEQ);                         \
      GM_STEP(2, KT, kt_ + 2, GLOAD, MMA, DEQ);                         \
    }                                                                   \
    if (kt_ < (KT)) GM_STEP(0, KT, kt_, GLOAD, MMA, DEQ);               \
    if (kt_ + 1 < (KT)) GM_STEP(1, KT, kt_ + 1, GLOAD, MMA, DEQ);       \
  } while (0)
#define PF_K_LOOP(KT, GLOAD, MMA, DEQ)                                  \
  do {                                                                  \
    GLOAD(0, A[0], B[0]);                                               \
    GLOAD(min(1, (KT) - 1), A[1], B[1]);                                \
    DEQ(B[0], 0);                                                       \
    __syncthreads();                                                    \
    int kt_ = 0;                                                        \
    for (; kt_ + 3 <= (KT); kt_ += 3) {                                 \
      PF_STEP(0, KT, kt_, GLOAD, MMA, DEQ);                             \
      PF_STEP(1, KT, kt_ + 1, GLOAD, MMA, DEQ);                         \
      PF_STEP(2, KT, kt_ + 2, GLOAD, MMA, DEQ);                         \
    }                                                                   \
    if (kt_ < (KT)) PF_STEP(0, KT, kt_, GLOAD, MMA, DEQ);               \
    if (kt_ + 1 < (KT)) PF_STEP(1, KT, kt_ + 1, GLOAD, MMA, DEQ);       \
  } while (0)

// grid: (M-tiles of the wave's experts, I / 64).  256 threads = 4 waves; wave w
// owns tile rows [32w, 32w+32) (two 16-row MFMA subtiles) and all 4+4
// 16-column subtiles of gate and up.  K loop over H in steps of 64 (one
// weight pair per row).  Rows past the expert's count read its last row and
// are not stored.
template <int QT>
__global__ __launch_bounds__(kThreads, 2) void pf_gateup_kernel(PfGateUpParams a) {
  __shared__ __align__(16) __bf16 Bs[3][128][kPfLd];  // rows 0..63 gate, 64..127 up
  constexpr int BB = Fmt<QT>::kBlockBytes;
  int j, m0;
  if (!pf_tile(a.X, blockIdx.x, j, m0)) return;
  const int n0 = blockIdx.y * 64;
  const int n = a.X.n[j], row0 = a.X.row0[j];
  const int tid = threadIdx.x, lane = tid & (kWave - 1), wv = tid / kWave;
  const int64_t rowb = (int64_t)(a.H / 32) * BB, mat = (int64_t)a.I * rowb;
  const int brow = tid >> 1, bhalf = tid & 1;
  const uint8_t *bptr = a.X.payload[j] + (brow >= 64 ? mat : 0) + (int64_t)(n0 + (brow & 63)) * rowb;
  // activations in 16-byte units (the launch checks that 32 bits index them)
  g_bf16x8 *xb = (g_bf16x8 *)a.xb;
  const uint32_t lo16 = (uint32_t)((int64_t)a.T * a.H / 8);
  uint32_t arow[2];
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int m = min(m0 + 32 * wv + 16 * i + (lane & 15), n - 1);
    arow[i] = (uint32_t)(a.perm[row0 + m] / a.k) * (uint32_t)(a.H / 8) + (lane >> 4);
  }
  bf16x8 A[3][2][2][2];  // [set][plane][i][ks]
  uint32_t B[3][9];
  f32x4 accg[2][4], accu[2][4];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      accg[i][q] = f32x4{0.f, 0.f, 0.f, 0.f};
      accu[i][q] = f32x4{0.f, 0.f, 0.f, 0.f};
    }
  auto gload = [&](int kt, bf16x8 (&Ar)[2][2][2], uint32_t (&Bv)[9]) {
    load_half<QT>(bptr + (int64_t)kt * 2 * BB, bhalf, Bv);
#pragma unroll
    for (int pl = 0; pl < 2; ++pl)
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int ks = 0; ks < 2; ++ks)
          Ar[pl][i][ks] = xb[arow[i] + pl * lo16 + (uint32_t)(kt * kPfBK / 8 + 4 * ks)];
  };
  // for each k slice and column subtile: hi then lo plane, both row subtiles
  auto mma = [&](const bf16x8 (&Ar)[2][2][2], int buf) {
#pragma unroll
    for (int ks = 0; ks < 2; ++ks)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int c = 32 * ks + 8 * (lane >> 4);
        const bf16x8 bg = *reinterpret_cast<const bf16x8 *>(&Bs[buf][16 * q + (lane & 15)][c]);
        const bf16x8 bu = *reinterpret_cast<const bf16x8 *>(&Bs[buf][64 + 16 * q + (lane & 15)][c]);
#pragma unroll
        for (int pl = 0; pl < 2; ++pl)
#pragma unroll
          for (int i = 0; i < 2; ++i) {
            accg[i][q] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(Ar[pl][i][ks], bg, accg[i][q], 0, 0, 0);
            accu[i][q] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(Ar[pl][i][ks], bu, accu[i][q], 0, 0, 0);
          }
      }
  };
  auto deq = [&](const uint32_t (&Bv)[9], int buf) { dequant_half<QT>(Bv, bhalf, &Bs[buf][brow][32 * bhalf]); };
  PF_K_LOOP(a.H / kPfBK, gload, mma, deq);
  // C layout (16x16): lane holds rows 4*(lane/16) + r, column lane % 16
  const int64_t plane = (int64_t)a.pairs * a.I;
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int q = 0; q < 4; ++q)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int m = m0 + 32 * wv + 16 * i + 4 * (lane >> 4) + r;
        if (m < n) {
          const float v = silu(accg[i][q][r]) * accu[i][q][r];
          const __bf16 hi = (__bf16)v;
          const int64_t o = (int64_t)(row0 + m) * a.I + n0 + 16 * q + (lane & 15);
          a.ab[o] = hi;
          a.ab[plane + o] = (__bf16)(v - (float)hi);
        }
      }
}

// SiLU for the grouped GEMMs' epilogue: the hardware base-2 exponential and
// reciprocal (about 1 ulp each) instead of the library exp and an IEEE divide,
// which took a fifth of a tile's time there.
__device__ __forceinline__ float silu_fast(float s) {
  return s * __builtin_amdgcn_rcpf(1.f + __builtin_amdgcn_exp2f(-1.4426950408889634f * s));
}

typedef __attribute__((address_space(3))) void lds_void;
typedef __attribute__((address_space(1))) const void g_void;

// Direct global -> LDS load of 16 bytes per lane: lane l's bytes land at
// dst + 16 l (dst wave-uniform).
__device__ __forceinline__ void dma16(const void *g, void *dst) {
  __builtin_amdgcn_global_load_lds((g_void *)g, (lds_void *)dst, 16, 0, 0);
}

constexpr int kPfWideThreads = 512;

struct PfDownParams {
  PfExperts X;
  const int32_t *perm;
  const __bf16 *ab;  // [2][pairs][I]: hi then lo
  const float *w;    // [pairs] routing weights (pair = t*k + j)
  float *P;          // [pairs][H]
  int pairs, H, I;
};

// grid: (M-tiles, ceil(H / 128)).  Wave w owns rows [32w, 32w+32) and the 8
// 16-column subtiles; K loop over I in steps of 64.  A last tile of 64
// columns (H an odd multiple of 64) reads weight row H-1 for the missing
// rows and stores only its first 64 columns.
template <int QT>
__global__ __launch_bounds__(kThreads, 2) void pf_down_kernel(PfDownParams a) {
  __shared__ __align__(16) __bf16 Bs[3][128][kPfLd];
  constexpr int BB = Fmt<QT>::kBlockBytes;
  int j, m0;
  if (!pf_tile(a.X, blockIdx.x, j, m0)) return;
  const int n0 = blockIdx.y * 128;
  const int n = a.X.n[j], row0 = a.X.row0[j];
  const int tid = threadIdx.x, lane = tid & (kWave - 1), wv = tid / kWave;
  const int64_t rowb = (int64_t)(a.I / 32) * BB;
  const int64_t mat = (int64_t)a.I * ((int64_t)(a.H / 32) * BB);
  const int brow = tid >> 1, bhalf = tid & 1;
  const uint8_t *bptr = a.X.payload[j] + 2 * mat + (int64_t)min(n0 + brow, a.H - 1) * rowb;
  g_bf16x8 *ab = (g_bf16x8 *)a.ab;
  const uint32_t pl16 = (uint32_t)((int64_t)a.pairs * a.I / 8);
  uint32_t arow[2];
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int m = min(m0 + 32 * wv + 16 * i + (lane & 15), n - 1);
    arow[i] = (uint32_t)(row0 + m) * (uint32_t)(a.I / 8) + (lane >> 4);
  }
  bf16x8 A[3][2][2][2];
  uint32_t B[3][9];
  f32x4 acc[2][8];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int q = 0; q < 8; ++q) acc[i][q] = f32x4{0.f, 0.f, 0.f, 0.f};
  auto gload = [&](int kt, bf16x8 (&Ar)[2][2][2], uint32_t (&Bv)[9]) {
    load_half<QT>(bptr + (int64_t)kt * 2 * BB, bhalf, Bv);
#pragma unroll
    for (int pl = 0; pl < 2; ++pl)
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int ks = 0; ks < 2; ++ks)
          Ar[pl][i][ks] = ab[arow[i] + pl * pl16 + (uint32_t)(kt * kPfBK / 8 + 4 * ks)];
  };
  auto mma = [&](const bf16x8 (&Ar)[2][2][2], int buf) {
#pragma unroll
    for (int ks = 0; ks < 2; ++ks)
#pragma unroll
      for (int q = 0; q < 8; ++q) {
        const bf16x8 bf =
            *reinterpret_cast<const bf16x8 *>(&Bs[buf][16 * q + (lane & 15)][32 * ks + 8 * (lane >> 4)]);
#pragma unroll
        for (int pl = 0; pl < 2; ++pl)
#pragma unroll
          for (int i = 0; i < 2; ++i)
            acc[i][q] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(Ar[pl][i][ks], bf, acc[i][q], 0, 0, 0);
      }
  };
  auto deq = [&](const uint32_t (&Bv)[9], int buf) { dequant_half<QT>(Bv, bhalf, &Bs[buf][brow][32 * bhalf]); };
  PF_K_LOOP(a.I / kPfBK, gload, mma, deq);
  // the lane's 8 output rows: pair ids, then their weights (two round trips)
  int pair[2][4];
  float wt[2][4];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int r = 0; r < 4; ++r)
      pair[i][r] = a.perm[row0 + min(m0 + 32 * wv + 16 * i + 4 * (lane >> 4) + r, n - 1)];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int r = 0; r < 4; ++r) wt[i][r] = a.w[pair[i][r]];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int m = m0 + 32 * wv + 16 * i + 4 * (lane >> 4) + r;
      if (m < n) {
        float *dst = a.P + (int64_t)pair[i][r] * a.H + n0 + (lane & 15);
#pragma unroll
        for (int q = 0; q < 8; ++q)
          if (n0 + 16 * q < a.H) dst[16 * q] = wt[i][r] * acc[i][q][r];
      }
    }
}
// ------------------------------------------- grouped GEMMs, K-quant formats ---
//
// The same tiling as pf_gateup_kernel / pf_down_kernel (128-row M-tiles, four
// waves of 32 rows, K steps of 64 with PF_K_LOOP's two steps of prefetch) with
// a dequantiser for any of the four formats: thread t takes weight row t % 128
// of the tile and, per K step, the quarters (t / 128) and (t / 128) + 2 of its
// 64 weights (16 each).  Used for Q4_K / Q6_K; the 32-weight block formats run
// the kernels above, whose one-block-per-thread dequantiser measured faster for
// them (a 256-row, eight-wave variant of this kernel, dequantising each tile
// once per 256 rows, ran no faster: the loop is bound by latency, not by the
// dequantisation).
constexpr int kGmThreads = 256;
constexpr int kGmBM = 128;
constexpr int kGmQ = 512 / kGmThreads;  // dequantised quarters per thread and step

// (expert, M-tile) of a flat M-tile index with kGmBM-row tiles.
__device__ __forceinline__ bool gm_tile(const PfExperts &X, int mt, int &j, int &m0) {
  static_assert(kGmBM == kPfBM, "the tile table is built for 128-row tiles");
  if (X.ntiles > 0) {
    if (mt >= X.ntiles) return false;
    const uint32_t v = X.tile[mt];
    j = (int)(v & 0xffu);
    m0 = (int)(v >> 8) * kGmBM;
    return true;
  }
  for (j = 0; j < X.count; ++j) {
    const int tiles = (X.n[j] + kGmBM - 1) / kGmBM;
    if (mt < tiles) {
      m0 = mt * kGmBM;
      return true;
    }
    mt -= tiles;
  }
  return false;
}

// The raw bytes thread quarter bq (0..3) needs for K step kt of a weight row:
//   Q8_0 (pair of blocks at 68 kt): the 9 dwords of block bq / 2 (load_half);
//   Q4_0 (pair at 36 kt): the 5 dwords of block bq / 2 (load_half);
//   Q4_K (chunk kt % 4 of super-block kt / 4): the 16-byte header and the 16
//     bytes of q holding weights 16 (bq % 2) .. +15 of the chunk's two sub-blocks;
//   Q6_K (weights 64 (kt % 4) .. +63 of super-block kt / 4): 20 bytes around the
//     16 ql bytes and 20 around the 16 qh bytes of the quarter, the dword holding
//     its scale and the one holding d (addresses rounded down to a dword).
template <int FMT>
__device__ __forceinline__ void gm_load_raw(const uint8_t *row, int kt, int bq, uint32_t (&v)[12]) {
  if constexpr (FMT == 8) {
    // dwords of the 68-byte pair: v[0] = the one holding block b's d (dword 8b), v[1..5] =
    // dwords 8b + 4 part .. +4, which hold the 16 q bytes of the quarter (block b = bq / 2,
    // q bytes 2 + 16 part .. of the block)
    const g_u32 *pw = (const g_u32 *)(row + (int64_t)kt * 68);
    const int b = bq >> 1, w0 = 8 * b + 4 * (bq & 1);
    v[0] = pw[8 * b];
#pragma unroll
    for (int i = 0; i < 5; ++i) v[1 + i] = pw[w0 + i];
  } else if constexpr (FMT == 2) {
    uint32_t t[9];
    load_half<FMT>(row + (int64_t)kt * 36, bq >> 1, t);
#pragma unroll
    for (int i = 0; i < 5; ++i) v[i] = t[i];
  } else if constexpr (FMT == 12) {
    const uint8_t *b = row + (int64_t)(kt >> 2) * 144;
    const u32x4 hd = *(g_u32x4_a4 *)b;
    const u32x4 q = *(g_u32x4_a4 *)(b + 16 + 32 * (kt & 3) + 16 * (bq & 1));
    v[0] = hd.x;
    v[1] = hd.y;
    v[2] = hd.z;
    v[3] = hd.w;
    v[4] = q.x;
    v[5] = q.y;
    v[6] = q.z;
    v[7] = q.w;
  } else {
    const uint8_t *b = row + (int64_t)(kt >> 2) * 210;
    const int sh = (int)((uintptr_t)b & 3), h = (kt & 3) >> 1, g = 2 * (kt & 1) + (bq >> 1);
    const int l0 = 16 * (bq & 1);
    const uint8_t *a = b - sh;
    const g_u32 *ql = (const g_u32 *)(a + 64 * h + 32 * (g & 1) + l0);
    const g_u32 *qh = (const g_u32 *)(a + 128 + 32 * h + l0);
#pragma unroll
    for (int i = 0; i < 5; ++i) {
      v[i] = ql[i];
      v[5 + i] = qh[i];
    }
    const uintptr_t sa = (uintptr_t)(b + 192 + 8 * h + 2 * g + (bq & 1));
    v[10] = *(const g_u32 *)(sa & ~(uintptr_t)3);
    v[11] = *(const g_u32 *)(a + 208);
  }
}

// The 16 weights of the quarter as bf16 (nearest, ties to even, from the fp32
// value) into dst (16-byte aligned).
template <int FMT>
__device__ __forceinline__ void gm_dequant(const uint32_t (&v)[12], const uint8_t *row, int kt, int bq,
                                           __bf16 *dst) {
  __bf16 o[16];
  const int part = bq & 1;
  if constexpr (FMT == 8) {
    // block 0: d = bytes 0-1, its q from byte 2 (2 bytes into the window); block 1: d =
    // bytes 34-35, its q from byte 36 (one dword into the window)
    const int half = bq >> 1;
    const float d = half_bits_to_float(half == 0 ? (v[0] & 0xffffu) : (v[0] >> 16));
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const uint32_t w = half == 0 ? __builtin_amdgcn_alignbyte(v[2 + j], v[1 + j], 2) : v[2 + j];
#pragma unroll
      for (int b = 0; b < 4; ++b) o[4 * j + b] = (__bf16)(d * (float)(int8_t)((w >> (8 * b)) & 0xffu));
    }
  } else if constexpr (FMT == 2) {
    // block 0: bytes 0..19 (d = 0-1, nibbles 2..17); block 1: bytes 16..35 (d = 18-19, 20..35);
    // part 0: the low nibbles (weights 0..15 of the block), part 1: the high ones
    const int half = bq >> 1;
    const float d = half_bits_to_float(half == 0 ? (v[0] & 0xffffu) : (v[0] >> 16));
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const uint32_t w = half == 0 ? __builtin_amdgcn_alignbyte(v[j + 1], v[j], 2) : v[j + 1];
#pragma unroll
      for (int b = 0; b < 4; ++b) {
        const uint32_t byte = (w >> (8 * b)) & 0xffu;
        o[4 * j + b] = (__bf16)(d * (float)((int)(part ? byte >> 4 : byte & 0xfu) - 8));
      }
    }
  } else if constexpr (FMT == 12) {
    // sub-block 2c + (bq >> 1): low nibbles for bq < 2, high for bq >= 2
    const int j = 2 * (kt & 3) + (bq >> 1), jj = j & 3;
    const uint32_t B0 = v[1], B1 = v[2], B2 = v[3];
    const uint32_t SC = j >= 4 ? ((B2 & 0x0f0f0f0fu) | ((B0 >> 2) & 0x30303030u)) : (B0 & 0x3f3f3f3fu);
    const uint32_t MN = j >= 4 ? (((B2 >> 4) & 0x0f0f0f0fu) | ((B1 >> 2) & 0x30303030u)) : (B1 & 0x3f3f3f3fu);
    const float d = half_bits_to_float(v[0] & 0xffffu), dmin = half_bits_to_float(v[0] >> 16);
    const float ds = d * (float)((SC >> (8 * jj)) & 0xffu), dm = dmin * (float)((MN >> (8 * jj)) & 0xffu);
    const int nib = 4 * (bq >> 1);
#pragma unroll
    for (int j4 = 0; j4 < 4; ++j4)
#pragma unroll
      for (int b = 0; b < 4; ++b) {
        const float q = (float)((v[4 + j4] >> (8 * b + nib)) & 0xfu);
        o[4 * j4 + b] = (__bf16)fmaf(ds, q, -dm);
      }
  } else {
    const uint8_t *bb = row + (int64_t)(kt >> 2) * 210;
    const int sh = (int)((uintptr_t)bb & 3), g = 2 * (kt & 1) + (bq >> 1);
    const uintptr_t sa = (uintptr_t)(bb + 192 + 8 * ((kt & 3) >> 1) + 2 * g + (bq & 1));
    const float d = half_bits_to_float((v[11] >> (8 * sh)) & 0xffffu);
    const float ds = d * (float)(int8_t)((v[10] >> (8 * (sa & 3))) & 0xffu);
#pragma unroll
    for (int j4 = 0; j4 < 4; ++j4) {
      const uint32_t lq = __builtin_amdgcn_alignbyte(v[j4 + 1], v[j4], sh);
      const uint32_t hq = __builtin_amdgcn_alignbyte(v[6 + j4], v[5 + j4], sh);
#pragma unroll
      for (int b = 0; b < 4; ++b) {
        const int q = (int)(((lq >> (8 * b + 4 * (g >> 1))) & 0xfu) | (((hq >> (8 * b + 2 * g)) & 3u) << 4));
        o[4 * j4 + b] = (__bf16)(ds * (float)(q - 32));
      }
    }
  }
  *reinterpret_cast<uint4 *>(dst) = *reinterpret_cast<const uint4 *>(o);
  *reinterpret_cast<uint4 *>(dst + 8) = *reinterpret_cast<const uint4 *>(o + 8);
}

struct GmParams {
  PfExperts X;
  const int32_t *perm;
  const __bf16 *A;  // gate/up: xb [2][T][H]; down: ab [2][pairs][I] (hi then lo planes)
  __bf16 *ab;       // gate/up output [2][pairs][I]
  const float *w;   // down: routing weights [pairs]
  float *P;         // down output [pairs][H]
  int T, pairs, H, I, k;
  int64_t mat, down_off;  // bytes of W_gate; offset of W_down in a payload
  int64_t rowb;           // bytes of a weight row of the format (gate/up: H inputs; down: I)
};
// kernel arguments stay within 4 KB
static_assert(sizeof(GmParams) <= 4096 && sizeof(PfGateUpParams) <= 4096 && sizeof(PfDownParams) <= 4096,
              "grouped-GEMM kernel arguments exceed 4 KB");

// grid: (M-tiles of the wave's experts, I / 64).  B rows 0..63: W_gate rows
// n0 .. n0+63, rows 64..127: the same rows of W_up; h = silu(g) u written as
// bf16 hi and lo terms at the pair's grouped row.
template <int FMT>
__global__ __launch_bounds__(kGmThreads, 512 / kGmThreads) void gm_gateup_kernel(GmParams a) {
  __shared__ __align__(16) __bf16 Bs[3][128][kPfLd];
  int j, m0;
  if (!gm_tile(a.X, blockIdx.x, j, m0)) return;
  const int n0 = blockIdx.y * 64;
  const int n = a.X.n[j], row0 = a.X.row0[j];
  const int tid = threadIdx.x, lane = tid & (kWave - 1), wv = tid / kWave;
  const bool live = m0 + 32 * wv < n;  // uniform over the wave
  const int br = tid & 127, bq = tid >> 7;  // consecutive lanes: consecutive LDS rows; quarters bq + 2 qi
  const uint8_t *brow = a.X.payload[j] + (br >= 64 ? a.mat : 0) + (int64_t)(n0 + (br & 63)) * a.rowb;
  g_bf16x8 *xb = (g_bf16x8 *)a.A;
  const uint32_t lo16 = (uint32_t)((int64_t)a.T * a.H / 8);
  uint32_t arow[2];
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int m = min(m0 + 32 * wv + 16 * i + (lane & 15), n - 1);
    arow[i] = (uint32_t)(a.perm[row0 + m] / a.k) * (uint32_t)(a.H / 8) + (lane >> 4);
  }
  bf16x8 A[3][2][2][2];  // [set][plane][i][ks]
  uint32_t B[3][kGmQ][12];
  f32x4 accg[2][4], accu[2][4];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      accg[i][q] = f32x4{0.f, 0.f, 0.f, 0.f};
      accu[i][q] = f32x4{0.f, 0.f, 0.f, 0.f};
    }
  auto gload = [&](int kt, bf16x8 (&Ar)[2][2][2], uint32_t (&Bv)[kGmQ][12]) {
#pragma unroll
    for (int qi = 0; qi < kGmQ; ++qi) gm_load_raw<FMT>(brow, kt, bq + 2 * qi, Bv[qi]);
#pragma unroll
    for (int pl = 0; pl < 2; ++pl)
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int ks = 0; ks < 2; ++ks)
          Ar[pl][i][ks] = xb[arow[i] + pl * lo16 + (uint32_t)(kt * kPfBK / 8 + 4 * ks)];
  };
  auto mma = [&](const bf16x8 (&Ar)[2][2][2], int buf) {
#pragma unroll
    for (int ks = 0; ks < 2; ++ks)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int c = 32 * ks + 8 * (lane >> 4);
        const bf16x8 bg = *reinterpret_cast<const bf16x8 *>(&Bs[buf][16 * q + (lane & 15)][c]);
        const bf16x8 bu = *reinterpret_cast<const bf16x8 *>(&Bs[buf][64 + 16 * q + (lane & 15)][c]);
#pragma unroll
        for (int pl = 0; pl < 2; ++pl)
#pragma unroll
          for (int i = 0; i < 2; ++i) {
            accg[i][q] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(Ar[pl][i][ks], bg, accg[i][q], 0, 0, 0);
            accu[i][q] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(Ar[pl][i][ks], bu, accu[i][q], 0, 0, 0);
          }
      }
  };
  auto deq = [&](const uint32_t (&Bv)[kGmQ][12], int buf, int kt) {
#pragma unroll
    for (int qi = 0; qi < kGmQ; ++qi)
      gm_dequant<FMT>(Bv[qi], brow, kt, bq + 2 * qi, &Bs[buf][br][16 * (bq + 2 * qi)]);
  };
  GM_K_LOOP(a.H / kPfBK, gload, mma, deq);
  if (!live) return;
  const int64_t plane = (int64_t)a.pairs * a.I;
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int q = 0; q < 4; ++q)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int m = m0 + 32 * wv + 16 * i + 4 * (lane >> 4) + r;
        if (m < n) {
          const float v = silu(accg[i][q][r]) * accu[i][q][r];
          const __bf16 hi = (__bf16)v;
          const int64_t o = (int64_t)(row0 + m) * a.I + n0 + 16 * q + (lane & 15);
          a.ab[o] = hi;
          a.ab[plane + o] = (__bf16)(v - (float)hi);
        }
      }
}

// grid: (M-tiles, ceil(H / 128)).  B rows: W_down rows n0 .. n0+127 (a last
// tile of 64 columns, H an odd multiple of 64, reads row H-1 for the missing
// rows and stores only its first 64 columns); K over I.  P[pair] = w * row.
template <int FMT>
__global__ __launch_bounds__(kGmThreads, 512 / kGmThreads) void gm_down_kernel(GmParams a) {
  __shared__ __align__(16) __bf16 Bs[3][128][kPfLd];
  int j, m0;
  if (!gm_tile(a.X, blockIdx.x, j, m0)) return;
  const int n0 = blockIdx.y * 128;
  const int n = a.X.n[j], row0 = a.X.row0[j];
  const int tid = threadIdx.x, lane = tid & (kWave - 1), wv = tid / kWave;
  const bool live = m0 + 32 * wv < n;
  const int br = tid & 127, bq = tid >> 7;
  const uint8_t *brow = a.X.payload[j] + a.down_off + (int64_t)min(n0 + br, a.H - 1) * a.rowb;
  g_bf16x8 *ab = (g_bf16x8 *)a.A;
  const uint32_t pl16 = (uint32_t)((int64_t)a.pairs * a.I / 8);
  uint32_t arow[2];
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int m = min(m0 + 32 * wv + 16 * i + (lane & 15), n - 1);
    arow[i] = (uint32_t)(row0 + m) * (uint32_t)(a.I / 8) + (lane >> 4);
  }
  bf16x8 A[3][2][2][2];
  uint32_t B[3][kGmQ][12];
  f32x4 acc[2][8];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int q = 0; q < 8; ++q) acc[i][q] = f32x4{0.f, 0.f, 0.f, 0.f};
  auto gload = [&](int kt, bf16x8 (&Ar)[2][2][2], uint32_t (&Bv)[kGmQ][12]) {
#pragma unroll
    for (int qi = 0; qi < kGmQ; ++qi) gm_load_raw<FMT>(brow, kt, bq + 2 * qi, Bv[qi]);
#pragma unroll
    for (int pl = 0; pl < 2; ++pl)
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int ks = 0; ks < 2; ++ks)
          Ar[pl][i][ks] = ab[arow[i] + pl * pl16 + (uint32_t)(kt * kPfBK / 8 + 4 * ks)];
  };
  auto mma = [&](const bf16x8 (&Ar)[2][2][2], int buf) {
#pragma unroll
    for (int ks = 0; ks < 2; ++ks)
#pragma unroll
      for (int q = 0; q < 8; ++q) {
        const bf16x8 bf =
            *reinterpret_cast<const bf16x8 *>(&Bs[buf][16 * q + (lane & 15)][32 * ks + 8 * (lane >> 4)]);
#pragma unroll
        for (int pl = 0; pl < 2; ++pl)
#pragma unroll
          for (int i = 0; i < 2; ++i)
            acc[i][q] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(Ar[pl][i][ks], bf, acc[i][q], 0, 0, 0);
      }
  };
  auto deq = [&](const uint32_t (&Bv)[kGmQ][12], int buf, int kt) {
#pragma unroll
    for (int qi = 0; qi < kGmQ; ++qi)
      gm_dequant<FMT>(Bv[qi], brow, kt, bq + 2 * qi, &Bs[buf][br][16 * (bq + 2 * qi)]);
  };
  GM_K_LOOP(a.I / kPfBK, gload, mma, deq);
  if (!live) return;
  int pair[2][4];
  float wt[2][4];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int r = 0; r < 4; ++r)
      pair[i][r] = a.perm[row0 + min(m0 + 32 * wv + 16 * i + 4 * (lane >> 4) + r, n - 1)];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int r = 0; r < 4; ++r) wt[i][r] = a.w[pair[i][r]];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int m = m0 + 32 * wv + 16 * i + 4 * (lane >> 4) + r;
      if (m < n) {
        float *dst = a.P + (int64_t)pair[i][r] * a.H + n0 + (lane & 15);
#pragma unroll
        for (int q = 0; q < 8; ++q)
          if (n0 + 16 * q < a.H) dst[16 * q] = wt[i][r] * acc[i][q][r];
      }
    }
}

#undef PF_K_LOOP
#undef PF_STEP
#undef GM_K_LOOP
#undef GM_STEP

// y[t] = (x[t] if residual) + (sum_j P[t*k + j], j = 0..k-1 in rank order).
// One block per token, four values per thread and step (H % 4 == 0), the k
// rows' loads all issued before the sums.
__global__ __launch_bounds__(kThreads) void pf_combine_kernel(const float *__restrict__ P,
                                                              const float *__restrict__ x,
                                                              float *__restrict__ y, int H, int k,
                                                              int residual) {
  const int t = blockIdx.x;
  const int H4 = H / 4;
  const float4 *x4 = reinterpret_cast<const float4 *>(x + (int64_t)t * H);
  const float4 *P4 = reinterpret_cast<const float4 *>(P + (int64_t)t * k * H);
  float4 *y4 = reinterpret_cast<float4 *>(y + (int64_t)t * H);
  for (int i = threadIdx.x; i < H4; i += kThreads) {
    float4 v = make_float4(0.f, 0.f, 0.f, 0.f);  // rows first, then the residual
    for (int j0 = 0; j0 < k; j0 += 8) {  // eight rows in flight (clamped to the last row)
      float4 p[8];
#pragma unroll
      for (int jj = 0; jj < 8; ++jj) p[jj] = P4[(int64_t)min(j0 + jj, k - 1) * H4 + i];
#pragma unroll
      for (int jj = 0; jj < 8; ++jj) {
        if (j0 + jj < k) {
          v.x += p[jj].x;
          v.y += p[jj].y;
          v.z += p[jj].z;
          v.w += p[jj].w;
        }
      }
    }
    if (residual) {
      const float4 r = x4[i];
      v = make_float4(r.x + v.x, r.y + v.y, r.z + v.z, r.w + v.w);
    }
    y4[i] = v;
  }
}

// Lanes per row (a power of two) and pairs per lane for rows of np pairs,
// when a lane keeps `in_flight` pairs of a row loading at once: few load
// rounds first, then few idle lanes, then fewer lanes.
#ifndef MOE_GATEUP_MAX_LANES
#define MOE_GATEUP_MAX_LANES 16
#endif
#ifndef MOE_DOWN_MAX_LANES
#define MOE_DOWN_MAX_LANES 64
#endif
constexpr int kGateUpMaxLanes = MOE_GATEUP_MAX_LANES, kDownMaxLanes = MOE_DOWN_MAX_LANES;

// Compute units of the current device (cached per device; 0 if unknown).
int device_compute_units() {
  static int cache[64] = {0};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 0;
  if (cache[dev] == 0) {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return 0;
    cache[dev] = n;
  }
  return cache[dev];
}

void pick_lanes(int np, int in_flight, int max_lanes, int &lanes, int &mpairs) {
  double best = -1e9;
  lanes = max_lanes;
  mpairs = (np + max_lanes - 1) / max_lanes;
  for (int L = 1; L <= max_lanes; L <<= 1) {
    const int M = (np + L - 1) / L;
    const int rounds = (M + in_flight - 1) / in_flight;
    const double score = (double)np / (L * M) - 0.25 * (rounds - 1) - 0.001 * L;
    if (score > best) {
      best = score;
      lanes = L;
      mpairs = M;
    }
  }
}

}  // namespace

int router_decode_grid(int H) { return (H + kRouterRowsPerBlock - 1) / kRouterRowsPerBlock; }

hipError_t launch_router_decode(const float *x, const float *wr, int H, int E, int k, float *partial,
                                int32_t *idx, float *w, int32_t *host_idx, float *host_w, int8_t *xq,
                                float *xsc, bool prenorm, const LruDev *lru, hipStream_t s,
                                const Timing &t) {
  const LruDev none{};
  const int nb = router_decode_grid(H);
  if (E > 128)
    hipExtLaunchKernelGGL(router_partial_kernel<false, 32>, dim3(nb), dim3(kThreads), 0, s, t.start, nullptr, 0,
                          x, wr, H, E, (int)prenorm, kRouterRowsPerBlock, partial, xq, xsc);
  else
    hipExtLaunchKernelGGL(router_partial_kernel<false, 16>, dim3(nb), dim3(kThreads), 0, s, t.start, nullptr, 0,
                          x, wr, H, E, (int)prenorm, kRouterRowsPerBlock, partial, xq, xsc);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipExtLaunchKernelGGL(router_finish_kernel, dim3(1), dim3(kThreads), 0, s, nullptr, t.stop, 0, partial,
                        nb, E, k, idx, w, host_idx, host_w, lru ? *lru : none);
  return hipGetLastError();
}

hipError_t launch_router_small(const float *x, const float *wr, int T, int H, int E, int k, float *partial,
                               int32_t *idx, float *w, int8_t *xq, float *xsc, bool prenorm,
                               const LruDev &lru, MtWork *mw, int32_t *flag, int max_chunks, hipStream_t s,
                               const Timing &t) {
  if (T < 1 || T > kMtTokens || !lru.slot_of || max_chunks < 1 || max_chunks > kMtMaxChunks)
    return hipErrorInvalidValue;
  // at most kMtParts blocks per token, so the finishing block loads every
  // token's partials in one round trip
  const int pieces = (H + kRouterRowsPerBlock - 1) / kRouterRowsPerBlock;
  const int rpb = kRouterRowsPerBlock * ((pieces + kMtParts - 1) / kMtParts);
  const int nb = (H + rpb - 1) / rpb;
  hipExtLaunchKernelGGL(router_partial_kernel<true, 32>, dim3(nb, T), dim3(kThreads), 0, s, t.start, nullptr, 0,
                        x, wr, H, E, (int)prenorm, rpb, partial, xq, xsc);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipExtLaunchKernelGGL(router_finish_mt_kernel, dim3(1), dim3(kThreads), 0, s, nullptr, t.stop, 0,
                        partial, nb, T, E, k, idx, w, lru, mw, flag, max_chunks);
  return hipGetLastError();
}

hipError_t launch_router_prefill(const float *x, const float *wr, int T, int H, int E, int k,
                                 const float *tscale, float *z, int32_t *idx, float *w, hipStream_t s) {
  const int slices = router_slices(T);
  hipLaunchKernelGGL(router_logits_kernel,
                     dim3((T + kRtTok - 1) / kRtTok, (E + kRtCols - 1) / kRtCols, slices),
                     dim3(kRtThreads), 0, s, x, wr, T, H, E, slices, z);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int wpb = kThreads / kWave;
  hipLaunchKernelGGL(topk_rows_kernel, dim3((T + wpb - 1) / wpb), dim3(kThreads), 0, s, z, T, E, k,
                     slices, tscale, idx, w);
  return hipGetLastError();
}

hipError_t launch_gateup(int qtype, const DecodeScratch &S, int H, int I, int k, const ExpertList &L,
                         const ExpertList *Ld, hipStream_t s, const Timing &t) {
  const int gu = fmt_gate_up(qtype), dn = fmt_down(qtype);
  if (gu == 12 || gu == 14) {
    if (H % 256 || L.n > kMaxRouted) return hipErrorInvalidValue;
    GateUpParams a{L, Ld, S.xq, S.xsc, S.hq, S.hsc, S.hds, H, I, k, 0, 0, 0, fmt_needs_sums(dn) ? 1 : 0};
    pick_lanes(H / 128, gu == 12 ? KFmt<12>::kGateUpFlight : KFmt<14>::kGateUpFlight, kGateUpMaxLanes,
               a.lanes, a.mpairs);
    while ((1 << a.lanes_log2) < a.lanes) ++a.lanes_log2;
    const int upb = kThreads / a.lanes;
    const size_t lds = 3 * (size_t)(H / 64) * kPairPitch + 4 * (size_t)(H / 32) * 4 + 4 * (size_t)upb;
    dim3 grid(L.n * ((I + upb - 1) / upb));
    if (gu == 12 && Ld)
      hipExtLaunchKernelGGL(kgateup_kernel<12, true>, grid, dim3(kThreads), lds, s, t.start, t.stop, 0, a);
    else if (gu == 12)
      hipExtLaunchKernelGGL(kgateup_kernel<12, false>, grid, dim3(kThreads), lds, s, t.start, t.stop, 0, a);
    else if (Ld)
      hipExtLaunchKernelGGL(kgateup_kernel<14, true>, grid, dim3(kThreads), lds, s, t.start, t.stop, 0, a);
    else
      hipExtLaunchKernelGGL(kgateup_kernel<14, false>, grid, dim3(kThreads), lds, s, t.start, t.stop, 0, a);
    return hipGetLastError();
  }
  if (dn != gu) return hipErrorInvalidValue;  // Q8_0 / Q4_0 models use one format throughout
  const int np = H / 64;
  GateUpParams a{L, Ld, S.xq, S.xsc, S.hq, S.hsc, S.hds, H, I, k, 0, 0, 0, 0};
  pick_lanes(np, qtype == 8 ? Fmt<8>::kGateUpFlight : Fmt<2>::kGateUpFlight, kGateUpMaxLanes,
             a.lanes, a.mpairs);
  while ((1 << a.lanes_log2) < a.lanes) ++a.lanes_log2;
  const int upb = kThreads / a.lanes;
  const size_t lds = 3 * (size_t)np * kPairPitch + 4 * (size_t)(H / 32) * 4 + 4 * (size_t)upb;
  dim3 grid(L.n * ((I + upb - 1) / upb));
  if (L.n > kMaxRouted) return hipErrorInvalidValue;
  if (qtype == 8 && Ld)
    hipExtLaunchKernelGGL(gateup_kernel<8, true>, grid, dim3(kThreads), lds, s, t.start, t.stop, 0, a);
  else if (qtype == 8)
    hipExtLaunchKernelGGL(gateup_kernel<8, false>, grid, dim3(kThreads), lds, s, t.start, t.stop, 0, a);
  else if (Ld)
    hipExtLaunchKernelGGL(gateup_kernel<2, true>, grid, dim3(kThreads), lds, s, t.start, t.stop, 0, a);
  else
    hipExtLaunchKernelGGL(gateup_kernel<2, false>, grid, dim3(kThreads), lds, s, t.start, t.stop, 0, a);
  return hipGetLastError();
}

hipError_t launch_down(int qtype, const DecodeScratch &S, int H, int I, int k, const ExpertList &L,
                       const ExpertList *Ld, const float *w, const float *x, float *y, int mode,
                       hipStream_t s, const Timing &t) {
  if (3 * L.n * I / 16 > kMaxDig16 * kThreads) return hipErrorInvalidValue;
  const int dn = fmt_down(qtype);
  if (dn == 12 || dn == 14) {
    if (I % 256 || L.n > kMaxRouted) return hipErrorInvalidValue;
    DownParams a{L, Ld, S.hq, S.hsc, S.hds, w, x, y, H, I, k, mode, 0, 0, 0, 0,
                 2 * fmt_matrix_bytes(fmt_gate_up(qtype), I, H)};
    pick_lanes(I / 128, dn == 12 ? KFmt<12>::kDownFlight : KFmt<14>::kDownFlight, kDownMaxLanes, a.lanes,
               a.mpairs);
    while ((1 << a.lanes_log2) < a.lanes) ++a.lanes_log2;
    a.rows = kThreads / (a.lanes * L.n);
    if (a.rows < 1) return hipErrorInvalidValue;
    const size_t lds = 3 * (size_t)L.n * (I / 64) * kPairPitch + 4 * (size_t)L.n * (I / 16) * 4 +
                       4 * (size_t)a.rows * L.n;
    dim3 grid((H + a.rows - 1) / a.rows);
    if (dn == 12 && Ld)
      hipExtLaunchKernelGGL(kdown_kernel<12, true>, grid, dim3(kThreads), lds, s, t.start, t.stop, 0, a);
    else if (dn == 12)
      hipExtLaunchKernelGGL(kdown_kernel<12, false>, grid, dim3(kThreads), lds, s, t.start, t.stop, 0, a);
    else if (Ld)
      hipExtLaunchKernelGGL(kdown_kernel<14, true>, grid, dim3(kThreads), lds, s, t.start, t.stop, 0, a);
    else
      hipExtLaunchKernelGGL(kdown_kernel<14, false>, grid, dim3(kThreads), lds, s, t.start, t.stop, 0, a);
    return hipGetLastError();
  }
  if (dn != fmt_gate_up(qtype)) return hipErrorInvalidValue;
  const int np = I / 64;
  DownParams a{L, Ld, S.hq, S.hsc, S.hds, w, x, y, H, I, k, mode, 0, 0, 0, 0, 0};
  pick_lanes(np, qtype == 8 ? Fmt<8>::kDownFlight : Fmt<2>::kDownFlight, kDownMaxLanes, a.lanes,
             a.mpairs);
  while ((1 << a.lanes_log2) < a.lanes) ++a.lanes_log2;
  if (L.n < 1 || L.n > kMaxRouted) return hipErrorInvalidValue;
  // rows per block: 256 threads' worth, or, where that would need more blocks
  // than there are compute units, up to 512 threads' worth so that one round
  // of blocks covers H (each block stages all experts' activations once)
  const int per_row = a.lanes * L.n;
  int nt = kThreads;
  a.rows = kThreads / per_row;
  const int cus = device_compute_units();
  if (a.rows >= 1 && cus > 0 && (H + a.rows - 1) / a.rows > cus) {
    const int want = (H + cus - 1) / cus;
    if (want * per_row <= 2 * kThreads) {
      nt = 2 * kThreads;
      a.rows = want;
    }
  }
  if (a.rows < 1) return hipErrorInvalidValue;
  const size_t lds = 3 * (size_t)L.n * np * kPairPitch + 4 * (size_t)L.n * (I / 16) * 4 +
                     4 * (size_t)a.rows * L.n;
  dim3 grid((H + a.rows - 1) / a.rows);
#define MOE_DOWN_LAUNCH(Q, D, N) \
  hipExtLaunchKernelGGL(down_kernel<Q, D, N>, grid, dim3(N), lds, s, t.start, t.stop, 0, a)
  if (nt == kThreads) {
    if (qtype == 8 && Ld) MOE_DOWN_LAUNCH(8, true, kThreads);
    else if (qtype == 8) MOE_DOWN_LAUNCH(8, false, kThreads);
    else if (Ld) MOE_DOWN_LAUNCH(2, true, kThreads);
    else MOE_DOWN_LAUNCH(2, false, kThreads);
  } else {
    if (qtype == 8 && Ld) MOE_DOWN_LAUNCH(8, true, 2 * kThreads);
    else if (qtype == 8) MOE_DOWN_LAUNCH(8, false, 2 * kThreads);
    else if (Ld) MOE_DOWN_LAUNCH(2, true, 2 * kThreads);
    else MOE_DOWN_LAUNCH(2, false, 2 * kThreads);
  }
#undef MOE_DOWN_LAUNCH
  return hipGetLastError();
}

size_t mt_gateup_lds(int H, int T) {
  return (size_t)T * (3 * (size_t)(H / 64) * kPairPitch + 16 * (size_t)(H / 32)) +
         (size_t)kMtTokens * kThreads * sizeof(float);
}
static size_t mt_down_lds(int I, int T) { return (size_t)T * (3 * (size_t)(I / 64) * kPairPitch + I); }

bool mt_ffn_fits(int qtype, int H, int I, int T) {
  return (qtype == 8 || qtype == 2) && T >= 1 && T <= kMtTokens && 3 * T * I / 16 <= kMaxDig16 * kThreads &&
         mt_gateup_lds(H, T) <= 64 * 1024 && mt_down_lds(I, T) <= 64 * 1024;
}

hipError_t launch_gateup_mt(int qtype, const MtWork *W, const int8_t *xq, const float *xsc, int8_t *hq,
                            float *hsc, int32_t *hds, int H, int I, int k, int T, int umax,
                            hipStream_t s, const Timing &t) {
  if (!mt_ffn_fits(qtype, H, I, T) || umax < 1 || umax > kMtMaxCopy) return hipErrorInvalidValue;
  GateUpMtParams a{W, xq, xsc, hq, hsc, hds, H, I, k, T, 0, 0, 0};
  pick_lanes(H / 64, qtype == 8 ? Fmt<8>::kGateUpFlight : Fmt<2>::kGateUpFlight, kGateUpMaxLanes, a.lanes,
             a.mpairs);
  while ((1 << a.lanes_log2) < a.lanes) ++a.lanes_log2;
  const int upb = kThreads / a.lanes;
  dim3 grid(umax * ((I + upb - 1) / upb));
  const size_t lds = mt_gateup_lds(H, T);
  if (qtype == 8)
    hipExtLaunchKernelGGL(gateup_mt_kernel<8>, grid, dim3(kThreads), lds, s, t.start, t.stop, 0, a);
  else
    hipExtLaunchKernelGGL(gateup_mt_kernel<2>, grid, dim3(kThreads), lds, s, t.start, t.stop, 0, a);
  return hipGetLastError();
}

hipError_t launch_down_mt(int qtype, const MtWork *W, const int8_t *hq, const float *hsc,
                          const int32_t *hds, float *R, int H, int I, int k, int T, int umax,
                          hipStream_t s, const Timing &t) {
  if (!mt_ffn_fits(qtype, H, I, T) || umax < 1 || umax > kMtMaxCopy) return hipErrorInvalidValue;
  DownMtParams a{W, hq, hsc, hds, R, H, I, k, T, 0, 0, 0, 0};
  pick_lanes(I / 64, qtype == 8 ? Fmt<8>::kDownFlight : Fmt<2>::kDownFlight, kDownMaxLanes, a.lanes,
             a.mpairs);
  while ((1 << a.lanes_log2) < a.lanes) ++a.lanes_log2;
  a.rows = kThreads / a.lanes;
  dim3 grid(umax * ((H + a.rows - 1) / a.rows));
  const size_t lds = mt_down_lds(I, T);
  if (qtype == 8)
    hipExtLaunchKernelGGL(down_mt_kernel<8>, grid, dim3(kThreads), lds, s, t.start, t.stop, 0, a);
  else
    hipExtLaunchKernelGGL(down_mt_kernel<2>, grid, dim3(kThreads), lds, s, t.start, t.stop, 0, a);
  return hipGetLastError();
}

hipError_t launch_combine_mt(const float *R, const float *w, const float *x, float *y, int H, int k,
                             int T, int mode, const MtWork *W, hipStream_t s, const Timing &t) {
  hipExtLaunchKernelGGL(combine_mt_kernel, dim3((H + kThreads - 1) / kThreads, T), dim3(kThreads), 0, s,
                        t.start, t.stop, 0, R, w, x, y, H, k, mode, W);
  return hipGetLastError();
}

bool fusable_copy_gateup(int qtype, int H, int I) {
  if (qtype != 8 && qtype != 2) return false;  // Q8_0 / Q4_0 models (one format, 32-weight blocks)
  const int64_t rowb = (int64_t)(H / 32) * (qtype == 8 ? 34 : 18);
  return 2 * 4 * rowb <= (int64_t)kChunkSlots * kThreads * 16 && I % 32 == 0;
}

hipError_t launch_copy_gateup(int qtype, const DecodeScratch &S, int H, int I, int k,
                              const WorkList *w, int64_t payload_bytes, int copy_blocks,
                              uint64_t *acc, hipStream_t s, const Timing &t) {
  if (!fusable_copy_gateup(qtype, H, I) || copy_blocks < 1) return hipErrorInvalidValue;
  const int64_t rowb = (int64_t)(H / 32) * (qtype == 8 ? 34 : 18);
  const int R = 2 * 8 * rowb <= (int64_t)kChunkSlots * kThreads * 16 ? 8 : 4;
  CopyGateUpParams a{};
  a.g = GateUpParams{ExpertList{}, nullptr, S.xq, S.xsc, S.hq, S.hsc, S.hds, H, I, k, 0, 0, 0};
  pick_lanes(H / 64, qtype == 8 ? Fmt<8>::kGateUpFlight : Fmt<2>::kGateUpFlight, kGateUpMaxLanes,
             a.g.lanes, a.g.mpairs);
  while ((1 << a.g.lanes_log2) < a.g.lanes) ++a.g.lanes_log2;
  a.W = w;
  a.P = payload_bytes;
  a.copy_blocks = copy_blocks;
  a.R = R;
  a.acc = acc;
  const int upb = kThreads / a.g.lanes;
  const size_t image = 3 * (size_t)(H / 64) * kPairPitch + 16 * (size_t)(H / 32);
  const size_t lds = std::max(image + 4 * (size_t)upb, image + 64 + 2 * (size_t)R * rowb);
  dim3 grid(copy_blocks + k * ((I + upb - 1) / upb));
  if (qtype == 8)
    hipExtLaunchKernelGGL(copy_gateup_kernel<8>, grid, dim3(kThreads), lds, s, t.start, t.stop, 0, a);
  else
    hipExtLaunchKernelGGL(copy_gateup_kernel<2>, grid, dim3(kThreads), lds, s, t.start, t.stop, 0, a);
  return hipGetLastError();
}

constexpr size_t kMtCopyLds = 160 * 1024;  // LDS one workgroup may take on gfx950

// Rows per chunk of the multi-token fused launch: the largest of 8, 4, 2
// whose chunk fits the copy slots and whose LDS (T images, hL, the chunk)
// fits a workgroup; 0 if none does.
static int mt_copy_rows(int qtype, int H, int I, int T, size_t *lds) {
  if (!mt_ffn_fits(qtype, H, I, T) || I % 32 != 0) return 0;
  const int64_t rowb = (int64_t)(H / 32) * (qtype == 8 ? 34 : 18);
  const size_t images = (size_t)T * (3 * (size_t)(H / 64) * kPairPitch + 16 * (size_t)(H / 32));
  for (int R = 8; R >= 2; R /= 2) {
    const size_t need = images + kMtTokens * 16 * sizeof(float) + 2 * (size_t)R * rowb;
    if (2 * R * rowb <= (int64_t)kChunkSlots * kThreads * 16 && need <= kMtCopyLds) {
      if (lds) *lds = std::max(need, mt_gateup_lds(H, T));
      return R;
    }
  }
  return 0;
}

bool fusable_copy_gateup_mt(int qtype, int H, int I, int T) {
  return mt_copy_rows(qtype, H, I, T, nullptr) > 0;
}

hipError_t launch_copy_gateup_mt(int qtype, const MtWork *W, const int8_t *xq, const float *xsc,
                                 int8_t *hq, float *hsc, int32_t *hds, int H, int I, int k, int T,
                                 int umax, int64_t payload_bytes, int copy_blocks, uint64_t *acc,
                                 hipStream_t s, const Timing &t) {
  size_t lds = 0;
  const int R = mt_copy_rows(qtype, H, I, T, &lds);
  if (R == 0 || copy_blocks < 1 || umax < 1 || umax > kMtMaxCopy) return hipErrorInvalidValue;
  CopyGateUpMtParams a{};
  a.g = GateUpMtParams{W, xq, xsc, hq, hsc, hds, H, I, k, T, 0, 0, 0};
  pick_lanes(H / 64, qtype == 8 ? Fmt<8>::kGateUpFlight : Fmt<2>::kGateUpFlight, kGateUpMaxLanes,
             a.g.lanes, a.g.mpairs);
  while ((1 << a.g.lanes_log2) < a.g.lanes) ++a.g.lanes_log2;
  const int upb = kThreads / a.g.lanes;
  if (upb % R != 0) return hipErrorInvalidValue;  // a pass covers whole tokens of R rows
  a.P = payload_bytes;
  a.copy_blocks = copy_blocks;
  a.R = R;
  a.acc = acc;
  dim3 grid(copy_blocks + umax * ((I + upb - 1) / upb));
  const void *fn = qtype == 8 ? reinterpret_cast<const void *>(&copy_gateup_mt_kernel<8>)
                              : reinterpret_cast<const void *>(&copy_gateup_mt_kernel<2>);
  if (lds > 64 * 1024) {
    const hipError_t e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
  }
  if (qtype == 8)
    hipExtLaunchKernelGGL(copy_gateup_mt_kernel<8>, grid, dim3(kThreads), lds, s, t.start, t.stop, 0, a);
  else
    hipExtLaunchKernelGGL(copy_gateup_mt_kernel<2>, grid, dim3(kThreads), lds, s, t.start, t.stop, 0, a);
  return hipGetLastError();
}

hipError_t launch_materialize_list(const WorkList *w, int64_t bytes, int grid, uint64_t *acc,
                                   hipStream_t s, const Timing &t) {
  hipExtLaunchKernelGGL(materialize_list_kernel<WorkList>, dim3(grid), dim3(kThreads), 0, s, t.start,
                        t.stop, 0, w, bytes / 16, acc);
  return hipGetLastError();
}

hipError_t launch_materialize_list(const MtWork *w, int64_t bytes, int grid, uint64_t *acc,
                                   hipStream_t s, const Timing &t) {
  hipExtLaunchKernelGGL(materialize_list_kernel<MtWork>, dim3(grid), dim3(kThreads), 0, s, t.start,
                        t.stop, 0, w, bytes / 16, acc);
  return hipGetLastError();
}

hipError_t launch_materialize(const uint8_t *const *src, uint8_t *const *dst, int n, int64_t bytes,
                              int grid, hipStream_t s, const Timing &t) {
  CopyParams a{};
  for (int i = 0; i < n; ++i) {
    a.src[i] = reinterpret_cast<const uint4 *>(src[i]);
    a.dst[i] = reinterpret_cast<uint4 *>(dst[i]);
  }
  a.n = n;
  a.p16 = bytes / 16;
  hipExtLaunchKernelGGL(materialize_kernel, dim3(grid), dim3(kThreads), 0, s, t.start, t.stop, 0, a);
  return hipGetLastError();
}

hipError_t launch_prefill_prep(const float *x, int T, int H, bool prenorm, float *inv, __bf16 *xb,
                               hipStream_t s) {
  hipLaunchKernelGGL(prefill_prep_kernel, dim3(T), dim3(kThreads), 0, s, x, T, H, (int)prenorm, inv, xb);
  return hipGetLastError();
}

int group_counts_ints(int E) { return kGroupChunks * E; }

hipError_t launch_group(const int32_t *idx, int npairs, int E, int32_t *counts, int32_t *offsets,
                        int32_t *perm, hipStream_t s) {
  if (npairs < 1 || E < 1 || E > kThreads) return hipErrorInvalidValue;
  // chunks of a multiple of 256 pairs, at least 1024 and at most kGroupChunks of them
  const int per = std::max(1024, (npairs + kGroupChunks - 1) / kGroupChunks);
  const int chunk = (per + kThreads - 1) / kThreads * kThreads;
  const int nchunks = (npairs + chunk - 1) / chunk;
  hipLaunchKernelGGL(group_hist_kernel, dim3(nchunks), dim3(kThreads), 0, s, idx, npairs, E, chunk, counts);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(group_place_kernel, dim3(nchunks), dim3(kThreads), 0, s, idx, npairs, E, chunk, nchunks,
                     counts, offsets, perm);
  return hipGetLastError();
}

// The wave's experts and the M-tile count of 256-row tiles.
// ------------------------------------------------ wide-tile grouped GEMMs ---
//
// One block per (M-tile of 128 rows, 256 columns), 512 threads: waves 0-3
// multiply (wave c: tile rows 32c..32c+31 against all 256 weight columns, the
// MFMA sequence per accumulator of pf_gateup_kernel / pf_down_kernel), waves
// 4-7 stage the next K step of 64: the activation tile (both planes) by direct
// global -> LDS loads, each 8 lanes one full 128-byte row segment with its
// 16-byte chunks XOR-swizzled by row (so the MFMA operand reads hit distinct
// banks), and the weight tile dequantised from the raw bytes of one weight row
// per thread, loaded a step ahead.  Each LDS stage is its own array, so that
// the compiler sees the reads of one stage not alias the loads into the other.
// The 1-D grid runs the column tiles of an M-tile, then an expert's M-tiles, one
// after the other on the same XCD (block L runs on XCD L % 8), so that their
// shared activation rows and weights come from that XCD's L2.
//
// A producer thread's raw bytes of one K step (64 weights of its row):
//   Q8_0 / Q4_0: the pair of blocks (17 / 9 dwords);
//   Q4_K / Q6_K: the four 16-weight quarters as gm_load_raw takes them.
//   Q6_K: the 64 bytes of ql, 32 of qh, the 4 scales and d that the step's 64
//     weights use, as aligned dwords around them (see wide_dequant).
template <int FMT>
struct WideRaw {
  static constexpr int kDw = FMT == 8 ? 17 : FMT == 2 ? 9 : FMT == 14 ? 19 : 48;
};

// K order of the wide kernels' steps.  A step multiplies 64 inputs; the sum
// over K does not depend on the order in which they are visited, so a format
// may visit them in the order its bytes hold them, as long as the activation
// tile and the weight tile use the same one.  Step kt, 16-byte chunk c of the
// step (eight inputs) covers K indices wide_kbase(kt) + wide_kchunk(c) + 0..7.
// Q6_K: a step is one quarter (n, j) of a super-block, n = the half (128
// weights), j = which 16 of each of its four 32-weight groups: the weights
// 128 n + 32 g + 16 j + l (g < 4, l < 16), whose low bits sit in 16 bytes of
// ql for g = 0, 2 (low and high nibbles), 16 bytes for g = 1, 3, and whose high
// bits sit in 16 bytes of qh (two bits per group).  So every loaded byte is
// used, once.  Tile position 16 g + l holds weight 128 n + 32 g + 16 j + l.
template <int FMT>
__device__ __forceinline__ uint32_t wide_kbase(int kt) {
  if constexpr (FMT == 14) return 256u * (uint32_t)(kt >> 2) + 128u * (uint32_t)((kt >> 1) & 1) + 16u * (uint32_t)(kt & 1);
  return (uint32_t)(kt * kPfBK);
}
template <int FMT>
__device__ __forceinline__ uint32_t wide_kchunk(int c) {
  if constexpr (FMT == 14) return 32u * (uint32_t)(c >> 1) + 8u * (uint32_t)(c & 1);
  return 8u * (uint32_t)c;
}
template <int FMT>
__device__ __forceinline__ void wide_load(const uint8_t *row, int kt, uint32_t (&v)[WideRaw<FMT>::kDw]) {
  if constexpr (FMT == 8 || FMT == 2) {
    const uint32_t *q = reinterpret_cast<const uint32_t *>(row + (int64_t)kt * 2 * Fmt<FMT>::kBlockBytes);
#pragma unroll
    for (int i = 0; i < WideRaw<FMT>::kDw; ++i) v[i] = q[i];
  } else if constexpr (FMT == 14) {
    // step kt: quarter (n, j) = ((kt / 2) % 2, kt % 2) of super-block kt / 4
    // (210 bytes, 2-byte aligned; a: its address rounded down to a dword).  Its
    // bytes: ql[64 n + 16 j, +16), ql[64 n + 32 + 16 j, +16), qh[32 n + 16 j, +16),
    // scales 8 n + j + 2 g, d.  Loaded: five dwords from each of a + 64 n + 16 j,
    // a + 64 n + 32 + 16 j and a + 128 + 32 n + 16 j (16 bytes plus the 2 of a
    // misaligned start), three from a + 192 + 8 n, the one at a + 208 (d).  The
    // furthest byte is a + 211, inside the payload: a payload ends 16-byte
    // aligned, so its last super-block starts at an address 2 mod 4 and ends at
    // a + 212.
    const uint8_t *b = row + (int64_t)(kt >> 2) * 210;
    const uint8_t *a = b - ((uintptr_t)b & 3);
    const int n = (kt >> 1) & 1, j = kt & 1;
    const uint8_t *run[3] = {a + 64 * n + 16 * j, a + 64 * n + 32 + 16 * j, a + 128 + 32 * n + 16 * j};
#pragma unroll
    for (int r = 0; r < 3; ++r) {
      const u32x4 q = *(g_u32x4_a4 *)run[r];
      v[5 * r] = q.x;
      v[5 * r + 1] = q.y;
      v[5 * r + 2] = q.z;
      v[5 * r + 3] = q.w;
      v[5 * r + 4] = ((const g_u32 *)run[r])[4];
    }
    const g_u32 *sc = (const g_u32 *)(a + 192 + 8 * n);
    v[15] = sc[0];
    v[16] = sc[1];
    v[17] = sc[2];
    v[18] = *(const g_u32 *)(a + 208);
  } else {
#pragma unroll
    for (int bq = 0; bq < 4; ++bq) {
      uint32_t t[12];
      gm_load_raw<FMT>(row, kt, bq, t);
#pragma unroll
      for (int i = 0; i < 12; ++i) v[12 * bq + i] = t[i];
    }
  }
}
// The row's 64 weights of step kt as bf16 into dst (16-byte aligned).
template <int FMT>
__device__ __forceinline__ void wide_dequant(const uint32_t (&v)[WideRaw<FMT>::kDw], const uint8_t *row,
                                             int kt, __bf16 *dst) {
  if constexpr (FMT == 8 || FMT == 2) {
    constexpr int PW = WideRaw<FMT>::kDw, o1 = FMT == 8 ? 8 : 4;
    uint32_t h0[9], h1[9];
#pragma unroll
    for (int i = 0; i < 9; ++i) {
      h0[i] = i < PW ? v[i] : 0u;
      h1[i] = i + o1 < PW ? v[i + o1] : 0u;
    }
    dequant_half<FMT>(h0, 0, dst);
    dequant_half<FMT>(h1, 1, dst + 32);
  } else if constexpr (FMT == 14) {
    // Q6_K weight 128 n + 32 g + 16 j + l of the step (tile position 16 g + l):
    // low four bits from ql run g % 2 (low nibbles for g < 2, high for g >= 2),
    // high two bits from bits 2 g, 2 g + 1 of qh byte l, scale 8 n + 2 g + j.
    // Four 6-bit q are assembled per dword (one per byte); each weight is
    // ds (q - 32) = fma(ds, q, -32 ds) rounded once (32 ds is exact), as the
    // quarter dequantiser forms it.
    const int sh = (int)((uintptr_t)(row + (int64_t)(kt >> 2) * 210) & 3), j = kt & 1;
    const uint64_t sc8 = (uint64_t)__builtin_amdgcn_alignbyte(v[17], v[16], sh) << 32 |
                         __builtin_amdgcn_alignbyte(v[16], v[15], sh);
    const float d = half_bits_to_float((v[18] >> (8 * sh)) & 0xffffu);
    float ds[4];
#pragma unroll
    for (int g = 0; g < 4; ++g) ds[g] = d * (float)(int8_t)((sc8 >> (8 * (2 * g + j))) & 0xffu);
    __bf16 o[64];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const uint32_t lA = __builtin_amdgcn_alignbyte(v[i + 1], v[i], sh);
      const uint32_t lB = __builtin_amdgcn_alignbyte(v[6 + i], v[5 + i], sh);
      const uint32_t hq = __builtin_amdgcn_alignbyte(v[11 + i], v[10 + i], sh);
      const uint32_t q[4] = {(lA & 0x0f0f0f0fu) | ((hq << 4) & 0x30303030u),
                             (lB & 0x0f0f0f0fu) | ((hq << 2) & 0x30303030u),
                             ((lA >> 4) & 0x0f0f0f0fu) | (hq & 0x30303030u),
                             ((lB >> 4) & 0x0f0f0f0fu) | ((hq >> 2) & 0x30303030u)};
#pragma unroll
      for (int g = 0; g < 4; ++g)
#pragma unroll
        for (int b = 0; b < 4; ++b)
          o[16 * g + 4 * i + b] = (__bf16)fmaf(ds[g], (float)((q[g] >> (8 * b)) & 0xffu), -32.f * ds[g]);
    }
#pragma unroll
    for (int i = 0; i < 8; ++i)
      *reinterpret_cast<uint4 *>(dst + 8 * i) = *reinterpret_cast<const uint4 *>(o + 8 * i);
  } else {
#pragma unroll
    for (int bq = 0; bq < 4; ++bq) {
      uint32_t t[12];
#pragma unroll
      for (int i = 0; i < 12; ++i) t[i] = v[12 * bq + i];
      gm_dequant<FMT>(t, row, kt, bq, dst + 16 * bq);
    }
  }
}

// The (M-tile, column tile) of this block in the XCD-grouped order.
__device__ __forceinline__ void wide_tile(int NT, int &mt, int &nt) {
  const int total = gridDim.x, L = blockIdx.x, x = L % 8, idx = L / 8, per = total / 8, rem = total % 8;
  const int w = x * per + min(x, rem) + idx;
  mt = w / NT;
  nt = w % NT;
}

// Producer waves' K loop: stage kt + 1 while the consumers multiply kt.
// asrc[u]: element offset (into the activation planes) of this lane's 16 bytes
// in DMA instruction u; row: the thread's weight row.
template <int FMT>
__device__ __forceinline__ void wide_produce(const __bf16 *Abase, const uint32_t (&asrc)[8], const uint8_t *row,
                                            int KT, int pw, int pt, __bf16 (*As0)[128][64],
                                            __bf16 (*As1)[128][64], __bf16 (*Bs0)[kPfLd],
                                            __bf16 (*Bs1)[kPfLd]) {
  auto aload = [&](int kt, __bf16 (*As)[128][64]) {
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int g = 8 * pw + u;
      dma16(Abase + (asrc[u] + wide_kbase<FMT>(kt)), &As[g >> 4][8 * (g & 15)][0]);
    }
  };
  uint32_t B0[WideRaw<FMT>::kDw], B1[WideRaw<FMT>::kDw];
  aload(0, As0);
  wide_load<FMT>(row, 0, B0);
  wide_load<FMT>(row, min(1, KT - 1), B1);
  wide_dequant<FMT>(B0, row, 0, &Bs0[pt][0]);
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  // step kt: stage kt + 1 into the other arrays; the raw weights of kt + 1 are
  // in BO, BS takes those of kt + 2
#define WIDE_PROD(BS, BO, AN, BN, kt)                          \
  do {                                                         \
    if ((kt) + 1 < KT) {                                       \
      aload((kt) + 1, AN);                                     \
      wide_load<FMT>(row, min((kt) + 2, KT - 1), BS);          \
      wide_dequant<FMT>(BO, row, (kt) + 1, &BN[pt][0]);        \
    }                                                          \
    __builtin_amdgcn_s_waitcnt(0);                             \
    __syncthreads();                                           \
  } while (0)
  int kt = 0;
  for (; kt + 2 <= KT; kt += 2) {
    WIDE_PROD(B0, B1, As1, Bs1, kt);
    WIDE_PROD(B1, B0, As0, Bs0, kt + 1);
  }
  if (kt < KT) WIDE_PROD(B0, B1, As1, Bs1, kt);
#undef WIDE_PROD
}

// Consumer MFMAs of one K step: wave wv's 32 rows against NQ 16-column subtiles
// of each of the NB weight groups (gate/up: NB 2 groups of 8; down: 1 of 16).
template <int NB, int NQ>
__device__ __forceinline__ void wide_mma(f32x4 (&acc)[NB][2][NQ], __bf16 (*As)[128][64], __bf16 (*Bs)[kPfLd],
                                         int wv, int lane) {
#pragma unroll
  for (int ks = 0; ks < 2; ++ks) {
    bf16x8 Ar[2][2];
#pragma unroll
    for (int pl = 0; pl < 2; ++pl)
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        const int r = 32 * wv + 16 * i + (lane & 15);
        const int c = (4 * ks + (lane >> 4)) ^ (r & 7);
        Ar[pl][i] = *reinterpret_cast<const bf16x8 *>(&As[pl][r][8 * c]);
      }
#pragma unroll
    for (int q = 0; q < NQ; ++q) {
      const int c = 32 * ks + 8 * (lane >> 4);
      bf16x8 bf[NB];
#pragma unroll
      for (int b = 0; b < NB; ++b)
        bf[b] = *reinterpret_cast<const bf16x8 *>(&Bs[128 * b + 16 * q + (lane & 15)][c]);
#pragma unroll
      for (int pl = 0; pl < 2; ++pl)
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
          for (int b = 0; b < NB; ++b)
            acc[b][i][q] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(Ar[pl][i], bf[b], acc[b][i][q], 0, 0, 0);
    }
  }
}

// Gate/up (I a multiple of 128): weight rows 0..127 of the tile are W_gate rows
// n0 .. n0+127, rows 128..255 the same rows of W_up; h = silu(g) u written as bf16
// hi and lo terms at the pair's grouped row.
template <int FMT>
__global__ __launch_bounds__(kPfWideThreads, 1) void pf_gateup_wide_kernel(GmParams a) {
  __shared__ __align__(16) __bf16 As0[2][128][64], As1[2][128][64];  // [plane][row][k], swizzled
  __shared__ __align__(16) __bf16 Bs0[256][kPfLd], Bs1[256][kPfLd];
  int mt, nt, j, m0;
  wide_tile(a.I / 128, mt, nt);
  if (!gm_tile(a.X, mt, j, m0)) return;
  const int n0 = nt * 128;
  const int n = a.X.n[j], row0 = a.X.row0[j];
  const int tid = threadIdx.x, lane = tid & (kWave - 1), wv = tid / kWave;
  const int KT = a.H / kPfBK;
  if (wv >= 4) {
    const int pw = wv - 4, pt = tid - 256;
    const uint8_t *row = a.X.payload[j] + (pt >= 128 ? a.mat : 0) + (int64_t)(n0 + (pt & 127)) * a.rowb;
    // DMA instruction g = 8 pw + u: plane g / 16, tile rows 8 (g % 16) .. +7;
    // element offsets into xb (32 bits, checked at launch)
    uint32_t asrc[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int g = 8 * pw + u, p = g >> 4, r = 8 * (g & 15) + (lane >> 3);
      const int m = min(m0 + r, n - 1);
      const int c = (lane & 7) ^ (lane >> 3);
      asrc[u] = (uint32_t)p * (uint32_t)(a.T * a.H) + (uint32_t)(a.perm[row0 + m] / a.k) * (uint32_t)a.H +
                wide_kchunk<FMT>(c);
    }
    wide_produce<FMT>(a.A, asrc, row, KT, pw, pt, As0, As1, Bs0, Bs1);
    return;
  }
  f32x4 acc[2][2][8];  // [gate, up][i][q]
#pragma unroll
  for (int b = 0; b < 2; ++b)
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int q = 0; q < 8; ++q) acc[b][i][q] = f32x4{0.f, 0.f, 0.f, 0.f};
  __syncthreads();
  int kt = 0;
  for (; kt + 2 <= KT; kt += 2) {
    wide_mma<2, 8>(acc, As0, Bs0, wv, lane);
    __syncthreads();
    wide_mma<2, 8>(acc, As1, Bs1, wv, lane);
    __syncthreads();
  }
  if (kt < KT) {
    wide_mma<2, 8>(acc, As0, Bs0, wv, lane);
    __syncthreads();
  }
  const int64_t plane = (int64_t)a.pairs * a.I;
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int q = 0; q < 8; ++q)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int m = m0 + 32 * wv + 16 * i + 4 * (lane >> 4) + r;
        if (m < n) {
          const float v = silu_fast(acc[0][i][q][r]) * acc[1][i][q][r];
          const __bf16 hi = (__bf16)v;
          const int64_t o = (int64_t)(row0 + m) * a.I + n0 + 16 * q + (lane & 15);
          a.ab[o] = hi;
          a.ab[plane + o] = (__bf16)(v - (float)hi);
        }
      }
}

// Down (H a multiple of 256): weight rows are W_down rows n0 .. n0+255; the
// activation rows are the expert's, contiguous in perm order; P[pair] = w * row.
template <int FMT>
__global__ __launch_bounds__(kPfWideThreads, 1) void pf_down_wide_kernel(GmParams a) {
  __shared__ __align__(16) __bf16 As0[2][128][64], As1[2][128][64];
  __shared__ __align__(16) __bf16 Bs0[256][kPfLd], Bs1[256][kPfLd];
  int mt, nt, j, m0;
  wide_tile(a.H / 256, mt, nt);
  if (!gm_tile(a.X, mt, j, m0)) return;
  const int n0 = nt * 256;
  const int n = a.X.n[j], row0 = a.X.row0[j];
  const int tid = threadIdx.x, lane = tid & (kWave - 1), wv = tid / kWave;
  const int KT = a.I / kPfBK;
  if (wv >= 4) {
    const int pw = wv - 4, pt = tid - 256;
    const uint8_t *row = a.X.payload[j] + a.down_off + (int64_t)(n0 + pt) * a.rowb;
    uint32_t asrc[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int g = 8 * pw + u, p = g >> 4, r = 8 * (g & 15) + (lane >> 3);
      const int m = min(m0 + r, n - 1);
      const int c = (lane & 7) ^ (lane >> 3);
      asrc[u] = (uint32_t)p * (uint32_t)(a.pairs * a.I) + (uint32_t)(row0 + m) * (uint32_t)a.I +
                wide_kchunk<FMT>(c);
    }
    wide_produce<FMT>(a.A, asrc, row, KT, pw, pt, As0, As1, Bs0, Bs1);
    return;
  }
  f32x4 acc[1][2][16];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int q = 0; q < 16; ++q) acc[0][i][q] = f32x4{0.f, 0.f, 0.f, 0.f};
  __syncthreads();
  int kt = 0;
  for (; kt + 2 <= KT; kt += 2) {
    wide_mma<1, 16>(acc, As0, Bs0, wv, lane);
    __syncthreads();
    wide_mma<1, 16>(acc, As1, Bs1, wv, lane);
    __syncthreads();
  }
  if (kt < KT) {
    wide_mma<1, 16>(acc, As0, Bs0, wv, lane);
    __syncthreads();
  }
  // the lane's 8 output rows: pair ids, then their weights
  int pair[2][4];
  float wt[2][4];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int r = 0; r < 4; ++r)
      pair[i][r] = a.perm[row0 + min(m0 + 32 * wv + 16 * i + 4 * (lane >> 4) + r, n - 1)];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int r = 0; r < 4; ++r) wt[i][r] = a.w[pair[i][r]];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int m = m0 + 32 * wv + 16 * i + 4 * (lane >> 4) + r;
      if (m < n) {
        float *dst = a.P + (int64_t)pair[i][r] * a.H + n0 + (lane & 15);
#pragma unroll
        for (int q = 0; q < 16; ++q) dst[16 * q] = wt[i][r] * acc[0][i][q][r];
      }
    }
}

static int gm_experts(const PfWave &W, PfExperts &X) {
  X.count = W.count;
  int tiles = 0;
  bool table = true;
  for (int i = 0; i < W.count; ++i) {
    X.payload[i] = W.payload[i];
    X.row0[i] = W.row0[i];
    X.n[i] = W.n[i];
    const int ti = (W.n[i] + kGmBM - 1) / kGmBM;
    if (ti > 256 || tiles + ti > kPfMaxTiles) table = false;
    for (int m = 0; table && m < ti; ++m) X.tile[tiles + m] = (uint16_t)(i | (m << 8));
    tiles += ti;
  }
  X.ntiles = table ? tiles : 0;
  return tiles;
}

// kAll: a kernel for every format; otherwise for the K-quant formats only (the
// 32-weight formats' 256-thread grouped GEMMs are pf_gateup_kernel / pf_down_kernel).
template <template <int> class K, bool kAll = true>
static hipError_t gm_launch(int fmt, dim3 grid, const GmParams &a, hipStream_t s, const Timing &t,
                            int threads = kGmThreads) {
  switch (fmt) {
    case 8:
      if constexpr (!kAll) return hipErrorInvalidValue;
      else hipExtLaunchKernelGGL(K<8>::fn(), grid, dim3(threads), 0, s, t.start, t.stop, 0, a);
      break;
    case 2:
      if constexpr (!kAll) return hipErrorInvalidValue;
      else hipExtLaunchKernelGGL(K<2>::fn(), grid, dim3(threads), 0, s, t.start, t.stop, 0, a);
      break;
    case 12:
      hipExtLaunchKernelGGL(K<12>::fn(), grid, dim3(threads), 0, s, t.start, t.stop, 0, a);
      break;
    case 14:
      hipExtLaunchKernelGGL(K<14>::fn(), grid, dim3(threads), 0, s, t.start, t.stop, 0, a);
      break;
    default:
      return hipErrorInvalidValue;
  }
  return hipGetLastError();
}
template <int F>
struct GmGateUp {
  static auto fn() { return gm_gateup_kernel<F>; }
};
template <int F>
struct GmDown {
  static auto fn() { return gm_down_kernel<F>; }
};
template <int F>
struct WideGateUp {
  static auto fn() { return pf_gateup_wide_kernel<F>; }
};
template <int F>
struct WideDown {
  static auto fn() { return pf_down_wide_kernel<F>; }
};

hipError_t launch_pf_gateup(int qtype, const PfWave &W, const int32_t *perm, const __bf16 *xb,
                            __bf16 *ab, int T, int H, int I, int k, hipStream_t s, const Timing &t) {
  if (W.count < 0 || W.count > kPfMaxExperts) return hipErrorInvalidValue;
  GmParams a{};
  const int tiles = gm_experts(W, a.X);
  const int fmt = fmt_gate_up(qtype);
  a.perm = perm;
  a.A = xb;
  a.ab = ab;
  a.T = T;
  a.pairs = T * k;
  a.H = H;
  a.I = I;
  a.k = k;
  a.rowb = fmt_matrix_bytes(fmt, 1, H);
  a.mat = (int64_t)I * a.rowb;
  if (tiles == 0) return hipSuccess;
  // the kernel indexes the activation planes in 16-byte units with 32 bits
  if (2 * (int64_t)T * H / 8 > (int64_t)UINT32_MAX || I % 64 || H % 64) return hipErrorInvalidValue;
  if (I % 128 == 0 && 2 * (int64_t)T * H <= (int64_t)UINT32_MAX) {
    // wide tiles, every format; element offsets into both activation planes fit 32 bits
    const dim3 g((unsigned)tiles * (unsigned)(I / 128));
    return gm_launch<WideGateUp>(fmt, g, a, s, t, kPfWideThreads);
  }
  if (fmt == 8 || fmt == 2) {  // the 32-weight block formats: pf_gateup_kernel (measured faster)
    PfGateUpParams b{};
    b.X = a.X;
    int tl = 0;
    for (int i = 0; i < W.count; ++i) tl += (W.n[i] + kPfBM - 1) / kPfBM;
    b.perm = perm;
    b.xb = xb;
    b.ab = ab;
    b.T = T;
    b.pairs = T * k;
    b.H = H;
    b.I = I;
    b.k = k;
    if (fmt == 8)
      hipExtLaunchKernelGGL(pf_gateup_kernel<8>, dim3(tl, I / 64), dim3(kThreads), 0, s, t.start, t.stop, 0, b);
    else
      hipExtLaunchKernelGGL(pf_gateup_kernel<2>, dim3(tl, I / 64), dim3(kThreads), 0, s, t.start, t.stop, 0, b);
    return hipGetLastError();
  }
  return gm_launch<GmGateUp, false>(fmt, dim3(tiles, I / 64), a, s, t);
}

hipError_t launch_pf_down(int qtype, const PfWave &W, const int32_t *perm, const __bf16 *ab,
                          const float *w, float *P, int pairs, int H, int I, hipStream_t s,
                          const Timing &t) {
  if (W.count < 0 || W.count > kPfMaxExperts) return hipErrorInvalidValue;
  GmParams a{};
  const int tiles = gm_experts(W, a.X);
  const int fmt = fmt_down(qtype);
  a.perm = perm;
  a.A = ab;
  a.w = w;
  a.P = P;
  a.pairs = pairs;
  a.H = H;
  a.I = I;
  a.rowb = fmt_matrix_bytes(fmt, 1, I);
  a.down_off = 2 * fmt_matrix_bytes(fmt_gate_up(qtype), I, H);
  if (tiles == 0) return hipSuccess;
  if (2 * (int64_t)pairs * I / 8 > (int64_t)UINT32_MAX || I % 64 || H % 64) return hipErrorInvalidValue;
  if (H % 256 == 0 && 2 * (int64_t)pairs * I <= (int64_t)UINT32_MAX) {
    // wide tiles, every format; element offsets into both activation planes fit 32 bits
    const dim3 g((unsigned)tiles * (unsigned)(H / 256));
    return gm_launch<WideDown>(fmt, g, a, s, t, kPfWideThreads);
  }
  if (fmt == 8 || fmt == 2) {
    PfDownParams b{};
    b.X = a.X;
    int tl = 0;
    for (int i = 0; i < W.count; ++i) tl += (W.n[i] + kPfBM - 1) / kPfBM;
    b.perm = perm;
    b.ab = ab;
    b.w = w;
    b.P = P;
    b.pairs = pairs;
    b.H = H;
    b.I = I;
    if (fmt == 8)
      hipExtLaunchKernelGGL(pf_down_kernel<8>, dim3(tl, (H + 127) / 128), dim3(kThreads), 0, s, t.start, t.stop, 0, b);
    else
      hipExtLaunchKernelGGL(pf_down_kernel<2>, dim3(tl, (H + 127) / 128), dim3(kThreads), 0, s, t.start, t.stop, 0, b);
    return hipGetLastError();
  }
  return gm_launch<GmDown, false>(fmt, dim3(tiles, (H + 127) / 128), a, s, t);
}

hipError_t launch_pf_combine(const float *P, const float *x, float *y, int T, int H, int k,
                             bool residual, hipStream_t s) {
  hipLaunchKernelGGL(pf_combine_kernel, dim3(T), dim3(kThreads), 0, s, P, x, y, H, k, (int)residual);
  return hipGetLastError();
}

int pf_max_experts() { return kPfMaxExperts; }
hipError_t launch_token_digits(const float *x, int T, int H, bool prenorm, int8_t *xq, float *xsc,
                               hipStream_t s) {
  if (H % 64 || H > 4 * kMaxX4 * kThreads) return hipErrorInvalidValue;
  hipLaunchKernelGGL(token_digits_kernel, dim3((H / 4 + kThreads - 1) / kThreads, T), dim3(kThreads), 0,
                     s, x, H, (int)prenorm, xq, xsc);
  return hipGetLastError();
}
int router_slices(int T) { return T <= kPfTok ? 64 : (T <= 8 * kPfTok ? 16 : 4); }
int64_t router_zbuf_floats(int64_t T, int E) {
  // the most any call of at most T tokens needs (slices * tokens is not monotonic in T)
  return (int64_t)E * std::max({64 * std::min<int64_t>(T, kPfTok), 16 * std::min<int64_t>(T, 8 * kPfTok),
                                4 * T});
}
int max_copy() { return kMaxCopy; }

}  // namespace moecache
