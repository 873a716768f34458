// Static budget planner (no HIP dependency): slots per layer from a cache
// budget, and the static check of the paper's Static Budget Check section,
//   L(p, n) = C + E(p) + K(n),  F(p, n) = L(p, n) + O,
// rejecting a configuration whose lower bound L exceeds the serving target.
// The slot count follows the inputs the Native Serving Path section lists
// (cache bytes, routed layers, slot block size, active experts per token,
// experts per layer): equal slots in every layer, clamped to
// [top_k, n_experts].
#include <cmath>
#include <cstdint>

#include "../../include/moecache.h"

namespace {

bool valid(const moe_plan_in *in) {
  return in && in->n_layers >= 1 && in->n_experts >= 1 && in->top_k >= 1 &&
         in->top_k <= in->n_experts && in->payload_bytes >= 1;
}

int finish(const moe_plan_in *in, int64_t want, int64_t context_tokens, moe_plan_out *out) {
  const int64_t s = want < in->top_k ? in->top_k : (want > in->n_experts ? in->n_experts : want);
  uint64_t e, k, lower, foot;
  if (__builtin_mul_overflow((uint64_t)in->n_layers * (uint64_t)s, in->payload_bytes, &e) ||
      __builtin_mul_overflow((uint64_t)context_tokens, in->kv_bytes_per_token, &k) ||
      __builtin_add_overflow(in->common_bytes, e, &lower) ||
      __builtin_add_overflow(lower, k, &lower) ||
      __builtin_add_overflow(lower, in->overhead_bytes, &foot))
    return MOE_EINVAL;
  out->slots_per_layer = (int32_t)s;
  out->clamped = s != want;
  out->expert_cache_bytes = e;
  out->kv_bytes = k;
  out->lower_bound_bytes = lower;
  out->footprint_bytes = foot;
  out->feasible = lower <= in->target_bytes;
  return MOE_OK;
}

}  // namespace

extern "C" {

int moe_plan_percent(const moe_plan_in *in, double percent, int64_t context_tokens,
                     moe_plan_out *out) {
  if (!valid(in) || !out || context_tokens < 0 || !std::isfinite(percent) || percent <= 0.0 ||
      percent > 100.0)
    return MOE_EINVAL;
  // nearest integer to percent/100 * n_experts, halves up: floor((2 p E + 100) / 200)
  const double want = std::floor((2.0 * percent * in->n_experts + 100.0) / 200.0);
  return finish(in, (int64_t)want, context_tokens, out);
}

int moe_plan_bytes(const moe_plan_in *in, uint64_t cache_bytes, int64_t context_tokens,
                   moe_plan_out *out) {
  if (!valid(in) || !out || context_tokens < 0) return MOE_EINVAL;
  const uint64_t per_slot = (uint64_t)in->n_layers * in->payload_bytes;  // one slot in every layer
  if (per_slot / in->payload_bytes != (uint64_t)in->n_layers) return MOE_EINVAL;
  const uint64_t want = cache_bytes / per_slot;
  return finish(in, want > (uint64_t)INT32_MAX ? (int64_t)INT32_MAX : (int64_t)want,
                context_tokens, out);
}

}  // extern "C"
