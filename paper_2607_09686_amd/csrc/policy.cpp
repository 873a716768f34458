// Offline bound on misses for a recorded sequence of layer calls (no HIP
// dependency): Belady's MIN with per-call expert sets.  Each call's distinct
// experts must be resident together; on a miss with every slot taken the
// victim is the resident outside the call whose next use lies farthest ahead
// (never again = infinitely far; ties: the higher id).  No slot policy can
// have fewer misses on the same calls, so this bounds the materialised bytes
// of the cache from below.
#include <algorithm>
#include <cstdint>
#include <vector>

#include "../../include/moecache.h"

extern "C" int moe_policy_min(const int32_t *ids, const int64_t *offsets, int64_t n_calls,
                              int32_t n_experts, int32_t n_slots, uint64_t *misses) {
  if (!misses || n_calls < 0 || n_experts < 1 || n_slots < 1 || (n_calls > 0 && (!ids || !offsets)))
    return MOE_EINVAL;
  if (n_calls > 0 && offsets[0] != 0) return MOE_EINVAL;
  // distinct sorted experts of every call
  std::vector<int64_t> beg(n_calls + 1, 0);
  std::vector<int32_t> req;
  std::vector<char> seen(n_experts, 0);
  for (int64_t i = 0; i < n_calls; ++i) {
    if (offsets[i + 1] < offsets[i]) return MOE_EINVAL;
    const size_t b = req.size();
    for (int64_t j = offsets[i]; j < offsets[i + 1]; ++j) {
      const int32_t e = ids[j];
      if (e < 0 || e >= n_experts) return MOE_EINVAL;
      if (!seen[e]) {
        seen[e] = 1;
        req.push_back(e);
      }
    }
    for (size_t j = b; j < req.size(); ++j) seen[req[j]] = 0;
    std::sort(req.begin() + b, req.end());
    if ((int64_t)(req.size() - b) > n_slots) return MOE_EINVAL;
    beg[i + 1] = (int64_t)req.size();
  }
  // next call that uses the expert of each request (backward pass)
  const int64_t kNever = INT64_MAX;
  std::vector<int64_t> nxt(req.size()), last(n_experts, kNever);
  for (int64_t i = n_calls - 1; i >= 0; --i)
    for (int64_t j = beg[i]; j < beg[i + 1]; ++j) {
      nxt[j] = last[req[j]];
      last[req[j]] = i;
    }
  std::vector<int64_t> next_of(n_experts, kNever), pinned(n_experts, -1);
  std::vector<char> in(n_experts, 0);
  std::vector<int32_t> res;  // resident experts
  res.reserve(n_slots);
  uint64_t m = 0;
  for (int64_t i = 0; i < n_calls; ++i) {
    for (int64_t j = beg[i]; j < beg[i + 1]; ++j) pinned[req[j]] = i;
    for (int64_t j = beg[i]; j < beg[i + 1]; ++j) {
      const int32_t e = req[j];
      if (!in[e]) {
        ++m;
        if ((int32_t)res.size() == n_slots) {
          size_t best = res.size();
          for (size_t r = 0; r < res.size(); ++r) {
            const int32_t v = res[r];
            if (pinned[v] == i) continue;
            if (best == res.size() || next_of[v] > next_of[res[best]] ||
                (next_of[v] == next_of[res[best]] && v > res[best]))
              best = r;
          }
          in[res[best]] = 0;
          res[best] = e;
        } else {
          res.push_back(e);
        }
        in[e] = 1;
      }
      next_of[e] = nxt[j];
    }
  }
  *misses = m;
  return MOE_OK;
}
