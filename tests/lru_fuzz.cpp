// Randomised self-check of the HIP-free slot table, built with AddressSanitizer
// and UndefinedBehaviorSanitizer by tests/test_lru_sanitize.py.  Checks after
// every call: slot_of / expert_in stay a bijection on resident experts, the
// records are ascending and cover the routed set, counters add up.
#include <cstdio>
#include <cstdlib>
#include <random>
#include <set>
#include <vector>

#include "../paper_2607_09686_amd/csrc/slot_lru.h"

int main() {
  std::mt19937_64 rng(12345);
  long calls = 0;
  for (int trial = 0; trial < 300; ++trial) {
    int E = 1 + rng() % 256, k = 1 + rng() % std::min(E, 16), C = 1 + rng() % E;
    moecache::SlotLru t(E, C, 1 + rng() % 1000000, trial);
    std::vector<moe_step_rec> recs;
    uint64_t seen = 0;
    for (int s = 0; s < 200; ++s, ++calls) {
      int n = k * (1 + rng() % 3);
      std::vector<int32_t> ids(n);
      for (auto &v : ids) v = rng() % E;
      recs.clear();
      t.step(ids.data(), n, recs);
      std::set<int32_t> S(ids.begin(), ids.end());
      if (recs.size() != S.size()) return 1;
      size_t i = 0;
      for (int32_t e : S) {
        if (recs[i].expert != e || recs[i].slot < 0 || recs[i].slot >= C) return 2;
        ++i;
      }
      seen += S.size();
      std::vector<int> owner(C, -1);
      int resident = 0;
      for (int e = 0; e < E; ++e) {
        int sl = t.slot_of(e);
        if (sl < 0) continue;
        if (sl >= C || owner[sl] >= 0) return 3;
        owner[sl] = e;
        ++resident;
      }
      if (resident > C) return 4;
      const moe_counters &c = t.counters();
      if (c.hits + c.misses != seen || c.evictions > c.misses) return 5;
    }
  }
  std::printf("ok %ld calls\n", calls);
  return 0;
}
