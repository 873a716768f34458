/*
 * Seeded synthetic inputs for the expert-slot-cache MoE FFN: expert weights
 * (quantised to GGUF-style Q8_0 / Q4_0 blocks or Q4_K / Q6_K super-blocks),
 * router matrices and hidden
 * states.  This module holds none of the MoE layer's arithmetic: it only
 * draws numbers and encodes them into the block format the store uses.
 *
 * Random bits: Philox4x64-10 (Salmon, Moraes, Dror, Shaw, "Parallel random
 * numbers: as easy as 1, 2, 3", SC 2011), a counter-based generator, so any
 * element of any tensor is computed independently and the store can be
 * filled by many threads in any order with identical bytes.
 *
 * Normals: one Philox call at counter c gives four 64-bit words = eight
 * 32-bit halves; halves (2p, 2p+1) feed one Box-Muller pair, giving the
 * eight normals with element indices 8c .. 8c+7.  The logarithm and the
 * sine/cosine are short polynomials evaluated with IEEE fp32 operations
 * only (no libm, no FMA contraction), so the bytes are the same on every
 * x86-64 host and with any vector width the compiler picks.
 *
 * Build (see build.py): gcc -O3 -mavx2 -ffp-contract=off -fno-math-errno
 *   -fno-trapping-math -fopenmp -shared -fPIC synth.c -o libsynth.so
 */
#include <stdint.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#define PHILOX_M0 0xD2E7470EE14C6C93ULL
#define PHILOX_M1 0xCA5A826395121157ULL
#define PHILOX_W0 0x9E3779B97F4A7C15ULL
#define PHILOX_W1 0xBB67AE8584CAA73BULL

/* Philox4x64 with 10 rounds on counter (c0,c1,c2,c3) and key (k0,k1). */
void synth_philox4x64(uint64_t c0, uint64_t c1, uint64_t c2, uint64_t c3,
                      uint64_t k0, uint64_t k1, uint64_t out[4]) {
  uint64_t c[4] = {c0, c1, c2, c3};
  for (int r = 0; r < 10; ++r) {
    unsigned __int128 p0 = (unsigned __int128)PHILOX_M0 * c[0];
    unsigned __int128 p1 = (unsigned __int128)PHILOX_M1 * c[2];
    uint64_t hi0 = (uint64_t)(p0 >> 64), lo0 = (uint64_t)p0;
    uint64_t hi1 = (uint64_t)(p1 >> 64), lo1 = (uint64_t)p1;
    uint64_t n0 = hi1 ^ c[1] ^ k0, n2 = hi0 ^ c[3] ^ k1;
    c[0] = n0; c[1] = lo1; c[2] = n2; c[3] = lo0;
    k0 += PHILOX_W0; k1 += PHILOX_W1;
  }
  memcpy(out, c, sizeof(c));
}

/* Box-Muller on n pairs of 32-bit words (a[i], b[i]) -> z[2i], z[2i+1].
 * Branch-free so the compiler can vectorise it. */
static void box_muller(const uint32_t *restrict a, const uint32_t *restrict b, int n,
                       float *restrict z) {
  float z0[64], z1[64];
#pragma omp simd
  for (int i = 0; i < n; ++i) {
    /* u1 in (0,1], 24-bit; ln u1 = e ln2 + ln m with m in [sqrt(.5), sqrt(2)) */
    float u1 = (float)(int32_t)((a[i] >> 8) + 1u) * 0x1.0p-24f;
    union { float f; int32_t i; } cv;
    cv.f = u1;
    int32_t e = ((cv.i >> 23) & 0xff) - 127;
    cv.i = (cv.i & 0x7fffff) | 0x3f800000;
    float m = cv.f;
    int32_t big = m > 1.41421356f;
    m = big ? m * 0.5f : m;
    e += big;
    float s = (m - 1.0f) / (m + 1.0f), s2 = s * s;
    float lnm = 2.0f * s * (1.0f + s2 * (1.0f / 3 + s2 * (1.0f / 5 + s2 * (1.0f / 7 + s2 * (1.0f / 9)))));
    float ln = (float)e * 0.693147180559945f + lnm;
    ln = ln < 0.0f ? ln : 0.0f;
    float r = __builtin_sqrtf(-2.0f * ln);
    /* angle 2 pi u2 = (q + f) pi/2 with q = round(4 u2), f in [-1/2, 1/2] */
    float t = (float)(int32_t)(b[i] >> 8) * 0x1.0p-22f; /* 4 u2 in [0,4) */
    int32_t q = (int32_t)(t + 0.5f);
    float x = (t - (float)q) * 1.57079632679f, x2 = x * x;
    float sn = x * (1.0f - x2 * (1.0f / 6 - x2 * (1.0f / 120 - x2 * (1.0f / 5040 - x2 * (1.0f / 362880)))));
    float cs = 1.0f - x2 * (0.5f - x2 * (1.0f / 24 - x2 * (1.0f / 720 - x2 * (1.0f / 40320 - x2 * (1.0f / 3628800)))));
    int32_t odd = q & 1, neg_c = ((q + 1) >> 1) & 1, neg_s = (q >> 1) & 1;
    float c0 = odd ? sn : cs, s0 = odd ? cs : sn;
    c0 = neg_c ? -c0 : c0;
    s0 = neg_s ? -s0 : s0;
    z0[i] = r * c0;
    z1[i] = r * s0;
  }
  for (int i = 0; i < n; ++i) {
    z[2 * i] = z0[i];
    z[2 * i + 1] = z1[i];
  }
}

/* Normals with element indices 8c .. 8c+8*n_calls-1 into z (fp32). */
static void normals_block(uint64_t c, int n_calls, uint64_t k0, uint64_t k1, float *z) {
  uint32_t a[64], b[64];
  for (int j = 0; j < n_calls; ++j) {
    uint64_t r[4];
    synth_philox4x64(c + (uint64_t)j, 0, 0, 0, k0, k1, r);
    for (int p = 0; p < 4; ++p) {
      a[4 * j + p] = (uint32_t)(r[p] & 0xffffffffu);
      b[4 * j + p] = (uint32_t)(r[p] >> 32);
    }
  }
  box_muller(a, b, 4 * n_calls, z);
}

/* out[i] = sigma * N(start + i), fp32, for i < n. */
void synth_normal_f32(uint64_t k0, uint64_t k1, uint64_t start, uint64_t n,
                      float sigma, float *out) {
  float z[128];
  uint64_t i = 0;
  while (i < n) {
    uint64_t e = start + i, c = e >> 3;
    uint64_t want = (n - i) + (e & 7);
    int calls = want >= 128 ? 16 : (int)((want + 7) >> 3);
    normals_block(c, calls, k0, k1, z);
    for (uint64_t j = e & 7; j < (uint64_t)calls * 8 && i < n; ++j, ++i) out[i] = sigma * z[j];
  }
}

/* fp32 -> IEEE binary16 bits, round to nearest even (subnormals, overflow to inf). */
uint16_t synth_f32_to_f16(float f) {
  uint32_t x;
  memcpy(&x, &f, 4);
  uint32_t sign = (x >> 16) & 0x8000u;
  uint32_t absx = x & 0x7fffffffu;
  if (absx >= 0x7f800000u) return (uint16_t)(sign | 0x7c00u | (absx > 0x7f800000u ? 0x200u : 0));
  if (absx >= 0x477ff000u) return (uint16_t)(sign | 0x7c00u);
  if (absx < 0x38800000u) {
    if (absx < 0x33000000u) return (uint16_t)sign;
    uint32_t e = absx >> 23;
    uint32_t m = (absx & 0x7fffffu) | 0x800000u;
    uint32_t shift = 126 - e;
    uint32_t q = m >> shift, rem = m & ((1u << shift) - 1), half = 1u << (shift - 1);
    if (rem > half || (rem == half && (q & 1))) ++q;
    return (uint16_t)(sign | q);
  }
  uint32_t e = (absx >> 23) - 127 + 15;
  uint32_t m = absx & 0x7fffffu;
  uint32_t q = (e << 10) | (m >> 13), rem = m & 0x1fffu;
  if (rem > 0x1000u || (rem == 0x1000u && (q & 1))) ++q;
  return (uint16_t)(sign | q);
}

float synth_f16_to_f32(uint16_t h) {
  uint32_t sign = (uint32_t)(h & 0x8000u) << 16, e = (h >> 10) & 0x1f, m = h & 0x3ff, x;
  if (e == 0) {
    if (m == 0) x = sign;
    else {
      int s = 0;
      while (!(m & 0x400)) { m <<= 1; ++s; }
      x = sign | ((uint32_t)(113 - s) << 23) | ((m & 0x3ff) << 13);
    }
  } else if (e == 31) x = sign | 0x7f800000u | (m << 13);
  else x = sign | ((e + 112) << 23) | (m << 13);
  float f;
  memcpy(&f, &x, 4);
  return f;
}

/* Q8_0: d = fp16(max|w|/127), q = clamp(rint(w/d), -127, 127), all in fp32. */
static void encode_q8_0(const float *w, int64_t n_blocks, uint8_t *dst) {
  for (int64_t blk = 0; blk < n_blocks; ++blk, w += 32, dst += 34) {
    float amax = 0.f;
    for (int j = 0; j < 32; ++j) {
      float a = w[j] < 0 ? -w[j] : w[j];
      amax = a > amax ? a : amax;
    }
    uint16_t dh = synth_f32_to_f16(amax / 127.f);
    float d = synth_f16_to_f32(dh);
    dst[0] = (uint8_t)(dh & 0xff);
    dst[1] = (uint8_t)(dh >> 8);
    float inv_ok = d != 0.f ? 1.f : 0.f, dd = d != 0.f ? d : 1.f;
    int8_t q[32];
    for (int j = 0; j < 32; ++j) {
      float v = __builtin_rintf(w[j] / dd) * inv_ok;
      v = v > 127.f ? 127.f : v < -127.f ? -127.f : v;
      q[j] = (int8_t)v;
    }
    memcpy(dst + 2, q, 32);
  }
}

/* Q4_0: d = fp16(max|w|/7), n = clamp(rint(w/d) + 8, 0, 15); byte j holds
 * element j in its low nibble and element j+16 in its high nibble. */
static void encode_q4_0(const float *w, int64_t n_blocks, uint8_t *dst) {
  for (int64_t blk = 0; blk < n_blocks; ++blk, w += 32, dst += 18) {
    float amax = 0.f;
    for (int j = 0; j < 32; ++j) {
      float a = w[j] < 0 ? -w[j] : w[j];
      amax = a > amax ? a : amax;
    }
    uint16_t dh = synth_f32_to_f16(amax / 7.f);
    float d = synth_f16_to_f32(dh);
    dst[0] = (uint8_t)(dh & 0xff);
    dst[1] = (uint8_t)(dh >> 8);
    float inv_ok = d != 0.f ? 1.f : 0.f, dd = d != 0.f ? d : 1.f;
    uint8_t n[32];
    for (int j = 0; j < 32; ++j) {
      float v = __builtin_rintf(w[j] / dd) * inv_ok + 8.f;
      v = v > 15.f ? 15.f : v < 0.f ? 0.f : v;
      n[j] = (uint8_t)v;
    }
    for (int j = 0; j < 16; ++j) dst[2 + j] = (uint8_t)(n[j] | (n[j + 16] << 4));
  }
}

static float clampf(float v, float lo, float hi) { return v < lo ? lo : v > hi ? hi : v; }

/* Q4_K (generation only): per 32-weight sub-block j an offset o_j = max(0, -min w)
 * and a step s_j = (max w + o_j) / 15, so w ~ s_j q - o_j with q in 0..15; the
 * super-block scales d = fp16(max s_j / 63), dmin = fp16(max o_j / 63); the 6-bit
 * sc_j = rint(s_j / d), m_j = rint(o_j / dmin); q = clamp(rint((w + dmin m_j) /
 * (d sc_j)), 0, 15).  Packed as the format prescribes: d, dmin, the 12 scale
 * bytes (sc_0..3 and m_0..3 in the low 6 bits of bytes 0..7, their top two bits
 * holding the high bits of sc_4..7 / m_4..7, whose low nibbles fill bytes
 * 8..11), then chunk c's 32 bytes with sub-block 2c in the low nibbles and 2c+1
 * in the high ones. */
static void encode_q4_k(const float *w, int64_t n_blocks, uint8_t *dst) {
  for (int64_t blk = 0; blk < n_blocks; ++blk, w += 256, dst += 144) {
    float step[8], off[8], smax = 0.f, omax = 0.f;
    for (int j = 0; j < 8; ++j) {
      float mn = w[32 * j], mx = w[32 * j];
      for (int l = 1; l < 32; ++l) {
        mn = w[32 * j + l] < mn ? w[32 * j + l] : mn;
        mx = w[32 * j + l] > mx ? w[32 * j + l] : mx;
      }
      off[j] = mn < 0.f ? -mn : 0.f;
      step[j] = (mx + off[j]) / 15.f;
      smax = step[j] > smax ? step[j] : smax;
      omax = off[j] > omax ? off[j] : omax;
    }
    const uint16_t dh = synth_f32_to_f16(smax / 63.f), mh = synth_f32_to_f16(omax / 63.f);
    const float d = synth_f16_to_f32(dh), dmin = synth_f16_to_f32(mh);
    int sc[8], m[8];
    for (int j = 0; j < 8; ++j) {
      sc[j] = d > 0.f ? (int)clampf(__builtin_rintf(step[j] / d), 0.f, 63.f) : 0;
      m[j] = dmin > 0.f ? (int)clampf(__builtin_rintf(off[j] / dmin), 0.f, 63.f) : 0;
    }
    dst[0] = (uint8_t)(dh & 0xff);
    dst[1] = (uint8_t)(dh >> 8);
    dst[2] = (uint8_t)(mh & 0xff);
    dst[3] = (uint8_t)(mh >> 8);
    for (int j = 0; j < 4; ++j) {
      dst[4 + j] = (uint8_t)(sc[j] | ((sc[j + 4] >> 4) << 6));
      dst[8 + j] = (uint8_t)(m[j] | ((m[j + 4] >> 4) << 6));
      dst[12 + j] = (uint8_t)((sc[j + 4] & 15) | ((m[j + 4] & 15) << 4));
    }
    for (int c = 0; c < 4; ++c)
      for (int l = 0; l < 32; ++l) {
        int q2[2];
        for (int h = 0; h < 2; ++h) {
          const int j = 2 * c + h;
          const float st = d * (float)sc[j], o = dmin * (float)m[j];
          q2[h] = st > 0.f ? (int)clampf(__builtin_rintf((w[32 * j + l] + o) / st), 0.f, 15.f) : 0;
        }
        dst[16 + 32 * c + l] = (uint8_t)(q2[0] | (q2[1] << 4));
      }
  }
}

/* Q6_K (generation only): per 16-weight group i a step t_i = (max |w|) / 31 with
 * the sign of the group's extreme; d = fp16(max |t_i| / 127), scale_i =
 * rint(t_i / d) (signed 8-bit), q = clamp(rint(w / (d scale_i)) + 32, 0, 63).
 * Packed as the format prescribes: weight 32g + l of half h keeps its low 4 bits
 * in ql[64h + 32(g mod 2) + l] (low nibble for g < 2, high for g >= 2) and its
 * high 2 bits in bits 2g, 2g+1 of qh[32h + l]; then the 16 scales and d. */
static void encode_q6_k(const float *w, int64_t n_blocks, uint8_t *dst) {
  for (int64_t blk = 0; blk < n_blocks; ++blk, w += 256, dst += 210) {
    float t[16], tmax = 0.f;
    for (int i = 0; i < 16; ++i) {
      float ext = 0.f;
      for (int l = 0; l < 16; ++l) {
        const float v = w[16 * i + l], a = v < 0.f ? -v : v, ea = ext < 0.f ? -ext : ext;
        ext = a > ea ? v : ext;
      }
      t[i] = ext / -32.f;  /* q = 0 carries the extreme: |q - 32| reaches 32 on its side */
      const float at = t[i] < 0.f ? -t[i] : t[i];
      tmax = at > tmax ? at : tmax;
    }
    const uint16_t dh = synth_f32_to_f16(tmax / 127.f);
    const float d = synth_f16_to_f32(dh);
    int8_t scale[16];
    for (int i = 0; i < 16; ++i)
      scale[i] = d > 0.f ? (int8_t)clampf(__builtin_rintf(t[i] / d), -127.f, 127.f) : 0;
    memset(dst, 0, 192);
    for (int n = 0; n < 256; ++n) {
      const float st = d * (float)scale[n / 16];
      const int q = st != 0.f ? (int)clampf(__builtin_rintf(w[n] / st) + 32.f, 0.f, 63.f) : 32;
      const int h = n / 128, g = (n % 128) / 32, l = n % 32;
      uint8_t *lo = dst + 64 * h + 32 * (g % 2) + l;
      *lo |= (uint8_t)((q & 15) << (g < 2 ? 0 : 4));
      dst[128 + 32 * h + l] |= (uint8_t)((q >> 4) << (2 * g));
    }
    memcpy(dst + 192, scale, 16);
    dst[208] = (uint8_t)(dh & 0xff);
    dst[209] = (uint8_t)(dh >> 8);
  }
}

/* Bytes and weights per block of a format code: 8 Q8_0, 2 Q4_0, 12 Q4_K, 14 Q6_K. */
static int format_of(int32_t fmt, int64_t *bytes, int64_t *weights) {
  switch (fmt) {
    case 8: *bytes = 34; *weights = 32; return 0;
    case 2: *bytes = 18; *weights = 32; return 0;
    case 12: *bytes = 144; *weights = 256; return 0;
    case 14: *bytes = 210; *weights = 256; return 0;
    default: return -1;
  }
}

/* Encode n_blocks blocks of fp32 weights (consecutive) in format fmt: 8 (Q8_0,
 * 34-byte blocks of 32), 2 (Q4_0, 18 of 32), 12 (Q4_K, 144 of 256), 14 (Q6_K,
 * 210 of 256). */
void synth_encode_blocks(int32_t fmt, const float *w, int64_t n_blocks, uint8_t *dst) {
  if (fmt == 8) encode_q8_0(w, n_blocks, dst);
  else if (fmt == 2) encode_q4_0(w, n_blocks, dst);
  else if (fmt == 12) encode_q4_k(w, n_blocks, dst);
  else if (fmt == 14) encode_q6_k(w, n_blocks, dst);
}

/* Stream key for one tensor: kind (1 expert, 2 router, 3 hidden), model
 * seed, layer (or token) l, expert e, matrix m (0 gate, 1 up, 2 down). */
uint64_t synth_key(uint32_t kind, uint32_t seed, uint32_t l, uint32_t e, uint32_t m) {
  return ((uint64_t)kind << 56) | ((uint64_t)(seed & 0xff) << 48) |
         ((uint64_t)(l & 0xffff) << 32) | ((uint64_t)(e & 0xffffff) << 8) | (m & 0xff);
}

/*
 * Fill the expert store for layers layer0 .. layer0+n_layers-1 (store points
 * at layer layer0).  Per (layer l, expert e) a contiguous payload
 * [gate (inter x hidden) | up (inter x hidden) | down (hidden x inter)], each
 * matrix row-major with every row split into blocks along the input
 * dimension.  qtype: the format of gate and up in its low byte and that of
 * down in the next byte (0: the same).  Weights ~ N(0, sigma) from key
 * (1, seed, l, e, m), drawn in row-major element order.  Returns 0, or -1 on
 * bad arguments.
 */
int synth_expert_store(int32_t qtype, int32_t layer0, int32_t n_layers, int32_t n_experts,
                       int32_t hidden, int32_t inter, float sigma, uint32_t seed,
                       uint8_t *store, int32_t n_threads) {
  const int32_t fgu = qtype & 0xff, fdn = (qtype >> 8) & 0xff ? (qtype >> 8) & 0xff : qtype & 0xff;
  int64_t bgu, wgu, bdn, wdn;
  if (format_of(fgu, &bgu, &wgu) || format_of(fdn, &bdn, &wdn) || hidden % wgu || inter % wdn ||
      n_layers < 0)
    return -1;
  const int64_t gu_bytes = (int64_t)inter * hidden / wgu * bgu;
  const int64_t dn_bytes = (int64_t)inter * hidden / wdn * bdn;
  const int64_t payload = 2 * gu_bytes + dn_bytes;
  const int64_t n_mats = (int64_t)n_layers * n_experts * 3;
#ifdef _OPENMP
  if (n_threads > 0) omp_set_num_threads(n_threads);
#endif
#pragma omp parallel
  {
    float buf[4096];
#pragma omp for schedule(dynamic, 1)
    for (int64_t mi = 0; mi < n_mats; ++mi) {
      int64_t le = mi / 3;
      int32_t m = (int32_t)(mi % 3);
      int32_t l = (int32_t)(le / n_experts), e = (int32_t)(le % n_experts);
      uint64_t k0 = synth_key(1, seed, (uint32_t)(layer0 + l), (uint32_t)e, (uint32_t)m);
      uint8_t *dst = store + le * payload + m * gu_bytes;
      const int32_t f = m < 2 ? fgu : fdn;
      const int64_t bb = m < 2 ? bgu : bdn, wpb = m < 2 ? wgu : wdn;
      const int64_t n_w = (int64_t)inter * hidden;
      for (int64_t s = 0; s < n_w; s += 4096) {  /* 4096 is a whole number of blocks */
        int64_t n = n_w - s < 4096 ? n_w - s : 4096;
        synth_normal_f32(k0, 0, (uint64_t)s, (uint64_t)n, sigma, buf);
        synth_encode_blocks(f, buf, n / wpb, dst + s / wpb * bb);
      }
    }
  }
  return 0;
}

/* Router matrices [n_layers][hidden][n_experts] fp32, N(0, sigma) from key
 * (2, seed, l, 0, 0), row-major. */
int synth_router(int32_t layer0, int32_t n_layers, int32_t hidden, int32_t n_experts,
                 float sigma, uint32_t seed, float *out) {
  for (int32_t l = 0; l < n_layers; ++l)
    synth_normal_f32(synth_key(2, seed, (uint32_t)(layer0 + l), 0, 0), 0, 0,
                     (uint64_t)hidden * n_experts, sigma, out + (int64_t)l * hidden * n_experts);
  return 0;
}

/*
 * Hidden states [n_tokens][hidden] fp32.  rho < 0: iid N(0,1) rows.  Else an
 * AR(1) drift x_0 = eps_0, x_t = rho x_{t-1} + sqrt(1-rho^2) eps_t, carried
 * in fp64 and rounded to fp32 once; eps_t ~ N(0,1) from key
 * (3, seed, t, stream, 0).
 */
int synth_hidden(int32_t n_tokens, int32_t hidden, double rho, uint32_t seed, uint32_t stream,
                 float *out) {
  static __thread double state[16384];
  static __thread float eps[16384];
  if (hidden > 16384 || hidden < 0) return -1;
  double a = rho < 0 ? 0.0 : rho, b = rho < 0 ? 1.0 : __builtin_sqrt(1.0 - rho * rho);
  for (int32_t t = 0; t < n_tokens; ++t) {
    synth_normal_f32(synth_key(3, seed, (uint32_t)t, stream, 0), 0, 0, (uint64_t)hidden, 1.0f, eps);
    for (int32_t i = 0; i < hidden; ++i) {
      state[i] = (t == 0 || rho < 0) ? (double)eps[i] : a * state[i] + b * (double)eps[i];
      out[(int64_t)t * hidden + i] = (float)state[i];
    }
  }
  return 0;
}
