// HIP kernels of the expert-slot-cache MoE layer for gfx950 (CDNA4, wave64).
//
// Router: z = x W_r (fp32), top-k by (-z, id) with wave shuffles, softmax over
// the chosen k.  Decode FFN: block-dequant GEMV straight from the GGUF-style
// Q8_0 / Q4_0 blocks in the slots, x staged in LDS, fp32 accumulation, fixed
// summation order (results do not depend on scheduling).
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>

#include "kernels.h"

namespace moecache {
namespace {

constexpr int kThreads = 256;
constexpr int kWave = 64;

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
// softmax over the chosen logits.  Must be called by all 64 lanes of a wave.
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

// ---------------------------------------------------------------- router ---

constexpr int kRouterRowsPerBlock = 64;

__global__ __launch_bounds__(kThreads) void router_decode_kernel(
    const float *__restrict__ x, const float *__restrict__ wr, int H, int E, int k,
    float *__restrict__ partial, uint32_t *counter, int32_t *idx, float *w, int32_t *host_idx,
    float *host_w, float *inv_rms, int prenorm) {
  __shared__ float red[kThreads];
  __shared__ float zs[256];
  __shared__ int is_last;
  const int tid = threadIdx.x;
  const int phases = kThreads / E;  // E <= 256
  const int c = tid % E, ph = tid / E;
  const int r0 = blockIdx.x * kRouterRowsPerBlock;
  const int r1 = min(H, r0 + kRouterRowsPerBlock);
  float acc = 0.f;
  if (ph < phases)
    for (int r = r0 + ph; r < r1; r += phases) acc = fmaf(x[r], wr[(int64_t)r * E + c], acc);
  red[tid] = acc;
  __syncthreads();
  if (tid < E) {
    float s = 0.f;
    for (int p = 0; p < phases; ++p) s += red[p * E + tid];
    partial[blockIdx.x * E + tid] = s;
  }
  __threadfence();
  __syncthreads();
  if (tid == 0) {
    uint32_t prev = atomicAdd(counter, 1u);
    is_last = prev == gridDim.x - 1;
  }
  __syncthreads();
  if (!is_last) return;
  __threadfence();
  // RMS scale of the token (pre-norm): z(x / rms) = z(x) / rms
  float ss = 0.f;
  if (prenorm)
    for (int i = tid; i < H; i += kThreads) ss = fmaf(x[i], x[i], ss);
  red[tid] = ss;
  __syncthreads();
  for (int off = kThreads / 2; off >= 1; off >>= 1) {
    if (tid < off) red[tid] += red[tid + off];
    __syncthreads();
  }
  const float inv = prenorm ? 1.f / sqrtf(red[0] / (float)H + 1e-6f) : 1.f;
  if (tid == 0) *inv_rms = inv;
  if (tid < E) {
    float s = 0.f;
    for (int b = 0; b < (int)gridDim.x; ++b)
      s += __hip_atomic_load(partial + b * E + tid, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    zs[tid] = s * inv;
  }
  __syncthreads();
  if (tid == 0) __hip_atomic_store(counter, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  if (tid < kWave) wave_topk(zs, E, k, idx, w, host_idx, host_w);
}

// z[T][E] = x[T][H] W_r[H][E]: a block owns 32 tokens and all E columns.
constexpr int kPfTok = 32, kPfRows = 32;

__global__ __launch_bounds__(kThreads) void router_logits_kernel(const float *__restrict__ x,
                                                                 const float *__restrict__ wr,
                                                                 int T, int H, int E,
                                                                 float *__restrict__ z) {
  __shared__ float xs[kPfTok][kPfRows + 1];
  __shared__ float ws[kPfRows][256];
  const int tid = threadIdx.x;
  const int t0 = blockIdx.x * kPfTok;
  const int phases = kThreads / E;
  const int c = tid % E, ph = tid / E;
  const int per = (kPfTok + phases - 1) / phases;  // tokens per thread
  float acc[kPfTok];
#pragma unroll
  for (int i = 0; i < kPfTok; ++i) acc[i] = 0.f;
  for (int r0 = 0; r0 < H; r0 += kPfRows) {
    for (int i = tid; i < kPfTok * kPfRows; i += kThreads) {
      int tt = i / kPfRows, rr = i % kPfRows;
      xs[tt][rr] = (t0 + tt < T && r0 + rr < H) ? x[(int64_t)(t0 + tt) * H + r0 + rr] : 0.f;
    }
    for (int i = tid; i < kPfRows * E; i += kThreads) {
      int rr = i / E, cc = i % E;
      ws[rr][cc] = r0 + rr < H ? wr[(int64_t)(r0 + rr) * E + cc] : 0.f;
    }
    __syncthreads();
    if (ph < phases) {
#pragma unroll
      for (int i = 0; i < kPfTok; ++i) {
        int tt = ph * per + i;
        if (i < per && tt < kPfTok) {
          float a = acc[i];
          for (int rr = 0; rr < kPfRows; ++rr) a = fmaf(xs[tt][rr], ws[rr][c], a);
          acc[i] = a;
        }
      }
    }
    __syncthreads();
  }
  if (ph < phases)
    for (int i = 0; i < per && i < kPfTok; ++i) {
      int tt = ph * per + i;
      if (tt < kPfTok && t0 + tt < T) z[(int64_t)(t0 + tt) * E + c] = acc[i];
    }
}

__global__ __launch_bounds__(kThreads) void topk_rows_kernel(const float *__restrict__ z, int T,
                                                             int E, int k, int32_t *idx, float *w) {
  const int wave = threadIdx.x / kWave;
  const int t = blockIdx.x * (kThreads / kWave) + wave;
  if (t >= T) return;
  wave_topk(z + (int64_t)t * E, E, k, idx + (int64_t)t * k, w + (int64_t)t * k, nullptr, nullptr);
}

// ------------------------------------------------------------ decode FFN ---
//
// A "pair" is two consecutive 32-weight blocks of one row (64 weights): 68
// bytes for Q8_0, 36 for Q4_0, always 4-byte aligned because rows hold an
// even number of blocks.  One thread turns one pair into one partial dot
// product; partials of a row are then summed in pair order.

template <int QT>
struct Fmt;
template <>
struct Fmt<8> {
  static constexpr int kBlockBytes = 34, kPairDwords = 17;
};
template <>
struct Fmt<2> {
  static constexpr int kBlockBytes = 18, kPairDwords = 9;
};

template <int QT>
__device__ __forceinline__ void load_pair(const uint8_t *p, uint32_t (&wd)[Fmt<QT>::kPairDwords]) {
  const uint32_t *q = reinterpret_cast<const uint32_t *>(p);
#pragma unroll
  for (int i = 0; i < Fmt<QT>::kPairDwords; ++i) wd[i] = __builtin_nontemporal_load(q + i);
}

// sum_j u_j * xs[j] over the four unsigned bytes of v.
__device__ __forceinline__ float dot_u8x4(uint32_t v, const float *xs, float acc) {
  acc = fmaf((float)(v & 0xffu), xs[0], acc);
  acc = fmaf((float)((v >> 8) & 0xffu), xs[1], acc);
  acc = fmaf((float)((v >> 16) & 0xffu), xs[2], acc);
  acc = fmaf((float)(v >> 24), xs[3], acc);
  return acc;
}

// Q8_0 pair: bytes 0-1 d0 | 2-33 q0[0..31] | 34-35 d1 | 36-67 q1[0..31].
// q is signed; with u = q ^ 0x80 (= q + 128), sum q x = sum u x - 128 sum x.
__device__ __forceinline__ float pair_dot_q8(const uint32_t (&wd)[17], const float *xs,
                                             float xsum0, float xsum1) {
  const uint32_t f = 0x80808080u;
  float d0 = half_bits_to_float(wd[0] & 0xffffu);
  float d1 = half_bits_to_float(wd[8] >> 16);
  uint32_t u0 = wd[0] ^ f;
  float a0 = 0.f;
  a0 = fmaf((float)((u0 >> 16) & 0xffu), xs[0], a0);
  a0 = fmaf((float)(u0 >> 24), xs[1], a0);
#pragma unroll
  for (int i = 1; i < 8; ++i) a0 = dot_u8x4(wd[i] ^ f, xs + 2 + 4 * (i - 1), a0);
  uint32_t u8 = wd[8] ^ f;
  a0 = fmaf((float)(u8 & 0xffu), xs[30], a0);
  a0 = fmaf((float)((u8 >> 8) & 0xffu), xs[31], a0);
  float a1 = 0.f;
#pragma unroll
  for (int i = 9; i < 17; ++i) a1 = dot_u8x4(wd[i] ^ f, xs + 32 + 4 * (i - 9), a1);
  return d0 * (a0 - 128.f * xsum0) + d1 * (a1 - 128.f * xsum1);
}

// Q4_0 pair: bytes 0-1 d0 | 2-17 nibbles of block 0 | 18-19 d1 | 20-35 block 1.
// Nibble byte j: low -> element j, high -> element j+16; weight d*(n-8).
__device__ __forceinline__ float nib_dot(uint32_t v, const float *xs, float acc) {
  // v holds nibble bytes j..j+3; xs points at x[j] of the block
  uint32_t lo = v & 0x0f0f0f0fu, hi = (v >> 4) & 0x0f0f0f0fu;
  acc = dot_u8x4(lo, xs, acc);
  acc = dot_u8x4(hi, xs + 16, acc);
  return acc;
}

__device__ __forceinline__ float pair_dot_q4(const uint32_t (&wd)[9], const float *xs,
                                             float xsum0, float xsum1) {
  float d0 = half_bits_to_float(wd[0] & 0xffffu);
  float d1 = half_bits_to_float(wd[4] >> 16);
  float a0 = 0.f;
  {  // nibble bytes 0,1 are the high half of dword 0
    uint32_t v = wd[0] >> 16;
    a0 = fmaf((float)(v & 0xfu), xs[0], a0);
    a0 = fmaf((float)((v >> 4) & 0xfu), xs[16], a0);
    a0 = fmaf((float)((v >> 8) & 0xfu), xs[1], a0);
    a0 = fmaf((float)((v >> 12) & 0xfu), xs[17], a0);
  }
#pragma unroll
  for (int i = 1; i < 4; ++i) a0 = nib_dot(wd[i], xs + 2 + 4 * (i - 1), a0);
  {  // nibble bytes 14,15 are the low half of dword 4
    uint32_t v = wd[4] & 0xffffu;
    a0 = fmaf((float)(v & 0xfu), xs[14], a0);
    a0 = fmaf((float)((v >> 4) & 0xfu), xs[30], a0);
    a0 = fmaf((float)((v >> 8) & 0xfu), xs[15], a0);
    a0 = fmaf((float)((v >> 12) & 0xfu), xs[31], a0);
  }
  float a1 = 0.f;
#pragma unroll
  for (int i = 5; i < 9; ++i) a1 = nib_dot(wd[i], xs + 32 + 4 * (i - 5), a1);
  return d0 * (a0 - 8.f * xsum0) + d1 * (a1 - 8.f * xsum1);
}

template <int QT>
__device__ __forceinline__ float pair_dot(const uint8_t *p, const float *xs, float xsum0,
                                          float xsum1) {
  uint32_t wd[Fmt<QT>::kPairDwords];
  load_pair<QT>(p, wd);
  if constexpr (QT == 8)
    return pair_dot_q8(wd, xs, xsum0, xsum1);
  else
    return pair_dot_q4(wd, xs, xsum0, xsum1);
}

__device__ __forceinline__ float silu(float s) { return s / (1.f + expf(-s)); }

// Stage scale*v (K floats) in LDS plus the sum of each 32-wide block of it.
__device__ __forceinline__ void stage_vec(const float *__restrict__ v, float scale, int K, float *xs,
                                          float *xsum) {
  for (int i = threadIdx.x; i < K; i += kThreads) xs[i] = v[i] * scale;
  __syncthreads();
  for (int b = threadIdx.x; b < K / 32; b += kThreads) {
    float s = 0.f;
    for (int j = 0; j < 32; ++j) s += xs[32 * b + j];
    xsum[b] = s;
  }
}

struct GateUpParams {
  ExpertList L;
  const float *x, *inv_rms;
  float *h;
  int H, I, rows;  // rows of gate (and of up) per block
};

// grid: n experts x (I / rows).  h[pos][r] = silu(g_r) * u_r.
template <int QT>
__global__ __launch_bounds__(kThreads) void gateup_kernel(GateUpParams a) {
  extern __shared__ float smem[];
  const int H = a.H, nb = H / 32, np = nb / 2;
  float *xs = smem, *xsum = xs + H, *part = xsum + nb;  // part[2][rows][np]
  const int tiles = a.I / a.rows;
  const int ei = blockIdx.x / tiles, r0 = (blockIdx.x % tiles) * a.rows;
  const int64_t rowb = (int64_t)nb * Fmt<QT>::kBlockBytes;
  const int64_t mat = (int64_t)a.I * rowb;
  const uint8_t *base = a.L.payload[ei];
  stage_vec(a.x, *a.inv_rms, H, xs, xsum);
  __syncthreads();
  const int items = 2 * a.rows * np;
  for (int it = threadIdx.x; it < items; it += kThreads) {
    int m = it / (a.rows * np), rem = it % (a.rows * np);
    int r = rem / np, p = rem % np;
    const uint8_t *ptr = base + m * mat + (int64_t)(r0 + r) * rowb + (int64_t)p * 2 * Fmt<QT>::kBlockBytes;
    part[it] = pair_dot<QT>(ptr, xs + 64 * p, xsum[2 * p], xsum[2 * p + 1]);
  }
  __syncthreads();
  for (int r = threadIdx.x; r < a.rows; r += kThreads) {
    float g = 0.f, u = 0.f;
    for (int p = 0; p < np; ++p) {
      g += part[r * np + p];
      u += part[(a.rows + r) * np + p];
    }
    a.h[(int64_t)a.L.pos[ei] * a.I + r0 + r] = silu(g) * u;
  }
}

struct DownParams {
  ExpertList L;
  const float *h, *w, *x;
  float *y;
  int H, I, rows, mode;
};

// grid: H / rows.  y[j] (+)= sum_i w[pos_i] * (W_down,i h_i)_j, experts in list order.
template <int QT>
__global__ __launch_bounds__(kThreads) void down_kernel(DownParams a) {
  extern __shared__ float smem[];
  const int I = a.I, nb = I / 32, np = nb / 2, n = a.L.n;
  float *hs = smem, *hsum = hs + n * I, *part = hsum + n * nb;  // part[n][rows][np]
  const int j0 = blockIdx.x * a.rows;
  const int64_t rowb = (int64_t)nb * Fmt<QT>::kBlockBytes;
  const int64_t mat = (int64_t)I * ((int64_t)(a.H / 32) * Fmt<QT>::kBlockBytes);
  for (int i = 0; i < n; ++i) {
    for (int c = threadIdx.x; c < I; c += kThreads) hs[i * I + c] = a.h[(int64_t)a.L.pos[i] * I + c];
  }
  __syncthreads();
  for (int b = threadIdx.x; b < n * nb; b += kThreads) {
    float s = 0.f;
    for (int j = 0; j < 32; ++j) s += hs[32 * b + j];
    hsum[b] = s;
  }
  __syncthreads();
  const int items = n * a.rows * np;
  for (int it = threadIdx.x; it < items; it += kThreads) {
    int i = it / (a.rows * np), rem = it % (a.rows * np);
    int r = rem / np, p = rem % np;
    const uint8_t *ptr = a.L.payload[i] + 2 * mat + (int64_t)(j0 + r) * rowb +
                         (int64_t)p * 2 * Fmt<QT>::kBlockBytes;
    part[it] = pair_dot<QT>(ptr, hs + i * I + 64 * p, hsum[i * nb + 2 * p], hsum[i * nb + 2 * p + 1]);
  }
  __syncthreads();
  for (int r = threadIdx.x; r < a.rows; r += kThreads) {
    const int j = j0 + r;
    float acc = a.mode == 2 ? a.y[j] : (a.mode == 1 ? a.x[j] : 0.f);
    for (int i = 0; i < n; ++i) {
      float s = 0.f;
      for (int p = 0; p < np; ++p) s += part[(i * a.rows + r) * np + p];
      acc = fmaf(a.w[a.L.pos[i]], s, acc);
    }
    a.y[j] = acc;
  }
}

int pick_rows(int total, int per_tile_blocks, int max_rows) {
  // largest power-of-two row count <= max_rows dividing total that still
  // gives at least 512 blocks, else the smallest that divides
  int best = 0;
  for (int r = 1; r <= max_rows; r <<= 1)
    if (total % r == 0) {
      if (best == 0) best = r;
      if ((int64_t)per_tile_blocks * (total / r) >= 512) best = r;
    }
  return best;
}

}  // namespace

int router_decode_grid(int H) { return (H + kRouterRowsPerBlock - 1) / kRouterRowsPerBlock; }

hipError_t launch_router_decode(const float *x, const float *wr, int H, int E, int k, float *partial,
                                uint32_t *counter, int32_t *idx, float *w, int32_t *host_idx,
                                float *host_w, float *inv_rms, bool prenorm, hipStream_t s) {
  hipLaunchKernelGGL(router_decode_kernel, dim3(router_decode_grid(H)), dim3(kThreads), 0, s, x, wr,
                     H, E, k, partial, counter, idx, w, host_idx, host_w, inv_rms, (int)prenorm);
  return hipGetLastError();
}

hipError_t launch_router_prefill(const float *x, const float *wr, int T, int H, int E, int k, float *z,
                                 int32_t *idx, float *w, hipStream_t s) {
  hipLaunchKernelGGL(router_logits_kernel, dim3((T + kPfTok - 1) / kPfTok), dim3(kThreads), 0, s, x,
                     wr, T, H, E, z);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int wpb = kThreads / kWave;
  hipLaunchKernelGGL(topk_rows_kernel, dim3((T + wpb - 1) / wpb), dim3(kThreads), 0, s, z, T, E, k,
                     idx, w);
  return hipGetLastError();
}

hipError_t launch_gateup(int qtype, const float *x, const float *inv_rms, int H, int I,
                         const ExpertList &L, float *h, hipStream_t s) {
  GateUpParams a{L, x, inv_rms, h, H, I, 0};
  a.rows = pick_rows(I, L.n, 16);
  const int np = H / 64;
  size_t lds = sizeof(float) * ((size_t)H + H / 32 + 2 * (size_t)a.rows * np);
  dim3 grid(L.n * (I / a.rows));
  if (qtype == 8)
    hipLaunchKernelGGL(gateup_kernel<8>, grid, dim3(kThreads), lds, s, a);
  else
    hipLaunchKernelGGL(gateup_kernel<2>, grid, dim3(kThreads), lds, s, a);
  return hipGetLastError();
}

hipError_t launch_down(int qtype, const float *h, int H, int I, const ExpertList &L, const float *w,
                       const float *x, float *y, int mode, hipStream_t s) {
  DownParams a{L, h, w, x, y, H, I, 0, mode};
  a.rows = pick_rows(H, 1, 16);
  const int np = I / 64, nb = I / 32;
  size_t lds = sizeof(float) * ((size_t)L.n * I + (size_t)L.n * nb + (size_t)L.n * a.rows * np);
  dim3 grid(H / a.rows);
  if (qtype == 8)
    hipLaunchKernelGGL(down_kernel<8>, grid, dim3(kThreads), lds, s, a);
  else
    hipLaunchKernelGGL(down_kernel<2>, grid, dim3(kThreads), lds, s, a);
  return hipGetLastError();
}

}  // namespace moecache
