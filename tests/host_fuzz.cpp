// Randomised self-check of the HIP-free planner and offline miss bound, built
// with AddressSanitizer and UndefinedBehaviorSanitizer by
// tests/test_lru_sanitize.py.  Checks: plans stay consistent (slots clamped to
// [top_k, n_experts], E = layers * slots * P, L = C + E + K, F = L + O, the
// feasibility flag) or the call reports an overflow; the bound never exceeds
// the routed count, never falls below the distinct count, and never grows
// with more slots; bad arguments are rejected.
#include <cstdint>
#include <cstdio>
#include <random>
#include <set>
#include <vector>

#include "../include/moecache.h"

int main() {
  std::mt19937_64 rng(777);
  long plans = 0, traces = 0;
  for (int i = 0; i < 200000; ++i) {
    moe_plan_in in{};
    in.n_layers = 1 + (int32_t)(rng() % 200);
    in.n_experts = 1 + (int32_t)(rng() % 512);
    in.top_k = 1 + (int32_t)(rng() % in.n_experts);
    in.payload_bytes = 1 + (rng() >> (rng() % 64));
    in.common_bytes = rng() >> (rng() % 64);
    in.kv_bytes_per_token = rng() >> (rng() % 64);
    in.overhead_bytes = rng() >> (rng() % 64);
    in.target_bytes = rng();
    const int64_t ctx = (int64_t)(rng() >> (1 + rng() % 63));
    moe_plan_out o{};
    const int rc = (i & 1) ? moe_plan_bytes(&in, rng() >> (rng() % 64), ctx, &o)
                           : moe_plan_percent(&in, 0.01 + (rng() % 10000) / 100.0, ctx, &o);
    if (rc == MOE_OK) {
      ++plans;
      if (o.slots_per_layer < in.top_k || o.slots_per_layer > in.n_experts) return 1;
      if (o.expert_cache_bytes != (uint64_t)in.n_layers * o.slots_per_layer * in.payload_bytes) return 2;
      if (o.kv_bytes != (uint64_t)ctx * in.kv_bytes_per_token) return 3;
      if (o.lower_bound_bytes != in.common_bytes + o.expert_cache_bytes + o.kv_bytes) return 4;
      if (o.footprint_bytes != o.lower_bound_bytes + in.overhead_bytes) return 5;
      if (o.feasible != (o.lower_bound_bytes <= in.target_bytes)) return 6;
    } else if (rc != MOE_EINVAL) {
      return 7;
    }
  }
  moe_plan_out o{};
  if (moe_plan_percent(nullptr, 10, 0, &o) != MOE_EINVAL) return 8;
  for (int t = 0; t < 3000; ++t) {
    const int E = 1 + (int)(rng() % 200), C = 1 + (int)(rng() % E), k = 1 + (int)(rng() % C);
    const int n = (int)(rng() % 120);
    std::vector<int32_t> ids;
    std::vector<int64_t> off(1, 0);
    std::set<int32_t> distinct;
    uint64_t routed = 0;
    for (int c = 0; c < n; ++c) {
      std::set<int32_t> S;
      const int m = 1 + (int)(rng() % (2 * k));
      for (int j = 0; j < m; ++j) {
        const int32_t e = (int32_t)(rng() % E);
        if ((int)S.size() < k || S.count(e)) {
          S.insert(e);
          ids.push_back(e);
        }
      }
      routed += S.size();
      distinct.insert(S.begin(), S.end());
      off.push_back((int64_t)ids.size());
    }
    uint64_t m1 = 0, m2 = 0;
    if (moe_policy_min(ids.data(), off.data(), n, E, C, &m1) != MOE_OK) return 9;
    if (m1 > routed || m1 < distinct.size()) return 10;
    if (C < E && moe_policy_min(ids.data(), off.data(), n, E, C + 1, &m2) == MOE_OK && m2 > m1) return 11;
    ++traces;
  }
  int32_t bad[3] = {0, 1, 2};
  int64_t boff[2] = {0, 3};
  uint64_t m = 0;
  if (moe_policy_min(bad, boff, 1, 4, 2, &m) != MOE_EINVAL) return 12;  // 3 experts, 2 slots
  if (moe_policy_min(bad, boff, 1, 2, 3, &m) != MOE_EINVAL) return 13;  // id out of range
  std::printf("ok %ld plans %ld traces\n", plans, traces);
  return 0;
}
