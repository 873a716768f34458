// Launch wrappers of the HIP kernels (internal to libmoecache).
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace moecache {

constexpr int kMaxRouted = 16;  // experts per FFN launch (top_k <= 16 in decode)

struct ExpertList {
  const uint8_t *payload[kMaxRouted];  // slot holding the expert's [gate|up|down] payload
  int32_t pos[kMaxRouted];             // top-k position of the expert for token 0
  int32_t n;
};

// Decode router: one token.  partial: [grid][E] fp32 scratch; counter: one
// uint32, zero on entry (left zero on exit).  Writes idx/w [k] to device and,
// if non-null, to host-mapped mirrors.
int router_decode_grid(int H);
// inv_rms: device scalar written with 1/sqrt(mean(x^2)+1e-6) when prenorm,
// else 1; the logits are scaled by it before top-k.
hipError_t launch_router_decode(const float *x, const float *wr, int H, int E, int k, float *partial,
                                uint32_t *counter, int32_t *idx, float *w, int32_t *host_idx,
                                float *host_w, float *inv_rms, bool prenorm, hipStream_t s);

// Prefill router: z = x W_r for T tokens into z [T][E], then top-k rows.
hipError_t launch_router_prefill(const float *x, const float *wr, int T, int H, int E, int k, float *z,
                                 int32_t *idx, float *w, hipStream_t s);

// Decode FFN.  h: [k][I] fp32 scratch (row pos of each listed expert written
// by gate/up, read by down).  mode of down: 0 y = sum, 1 y = x + sum, 2 y += sum.
// x is scaled by *inv_rms (written by the router) when staged.
hipError_t launch_gateup(int qtype, const float *x, const float *inv_rms, int H, int I,
                         const ExpertList &L, float *h, hipStream_t s);
hipError_t launch_down(int qtype, const float *h, int H, int I, const ExpertList &L, const float *w,
                       const float *x, float *y, int mode, hipStream_t s);

}  // namespace moecache
