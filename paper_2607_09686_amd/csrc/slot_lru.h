// Per-layer LRU expert-slot table (no HIP dependency).
//
// Each MoE layer owns n_slots slots; the table maps expert ids to slots (the
// expert-to-slot map of the paper's Native Serving Path section) and picks
// the slot a missed expert is materialised into.  Rule for one layer call with
// routed set S (distinct ids, ascending):
//   1. stamp[e] = ++clock for every e in S, ascending;
//   2. e in S holding a slot is a hit;
//   3. misses, ascending, take the lowest free slot, else evict the resident
//      expert with the smallest stamp and take its slot.
// One record per e in S, ascending.
#pragma once

#include <cstdint>
#include <vector>

#include "../../include/moecache.h"

namespace moecache {

class SlotLru {
 public:
  SlotLru(int32_t n_experts, int32_t n_slots, uint64_t payload_bytes, int32_t layer);

  // ids: routed experts of one call (any order, duplicates allowed, all in
  // [0, n_experts)).  Appends one record per distinct id to out.
  void step(const int32_t *ids, int32_t n, std::vector<moe_step_rec> &out);
  void reset();

  // Whole state of the table, for moving it to and from device memory.
  struct State {
    std::vector<int32_t> slot_of, expert_in;
    std::vector<uint64_t> stamp;
    uint64_t clock = 0;
    int32_t step = 0, used = 0;
    moe_counters cnt{};
  };
  State state() const;
  void set_state(const State &s);  // sizes must match n_experts / n_slots

  const moe_counters &counters() const { return cnt_; }
  int32_t slot_of(int32_t e) const { return slot_of_[e]; }
  int32_t n_slots() const { return n_slots_; }
  int32_t n_experts() const { return n_experts_; }

 private:
  int32_t n_experts_, n_slots_, layer_;
  uint64_t payload_;
  std::vector<int32_t> slot_of_, expert_in_;
  std::vector<uint64_t> stamp_;
  std::vector<uint8_t> mark_;
  uint64_t clock_ = 0;
  int32_t step_no_ = 0, used_ = 0;
  moe_counters cnt_{};
};

}  // namespace moecache
