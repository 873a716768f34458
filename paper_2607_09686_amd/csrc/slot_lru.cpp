// Per-layer LRU expert-slot table; see slot_lru.h for the rule.
#include "slot_lru.h"

#include <cstddef>
#include <new>

namespace moecache {

SlotLru::SlotLru(int32_t n_experts, int32_t n_slots, uint64_t payload_bytes, int32_t layer)
    : n_experts_(n_experts), n_slots_(n_slots), layer_(layer), payload_(payload_bytes) {
  reset();
}

void SlotLru::reset() {
  slot_of_.assign(n_experts_, -1);
  expert_in_.assign(n_slots_, -1);
  stamp_.assign(n_experts_, 0);
  mark_.assign(n_experts_, 0);
  clock_ = 0;
  step_no_ = 0;
  used_ = 0;
  cnt_ = moe_counters{};
}

SlotLru::State SlotLru::state() const {
  State s;
  s.slot_of = slot_of_;
  s.expert_in = expert_in_;
  s.stamp = stamp_;
  s.clock = clock_;
  s.step = step_no_;
  s.used = used_;
  s.cnt = cnt_;
  return s;
}

void SlotLru::set_state(const State &s) {
  slot_of_ = s.slot_of;
  expert_in_ = s.expert_in;
  stamp_ = s.stamp;
  clock_ = s.clock;
  step_no_ = s.step;
  used_ = s.used;
  cnt_ = s.cnt;
}

void SlotLru::step(const int32_t *ids, int32_t n, std::vector<moe_step_rec> &out) {
  // distinct ids, ascending (bitmap over the expert range)
  for (int32_t i = 0; i < n; ++i) mark_[ids[i]] = 1;
  const size_t first = out.size();
  for (int32_t e = 0; e < n_experts_; ++e) {
    if (!mark_[e]) continue;
    mark_[e] = 0;
    stamp_[e] = ++clock_;  // rule 1
    moe_step_rec r{layer_, step_no_, e, slot_of_[e] >= 0 ? 1 : 0, slot_of_[e], -1};
    out.push_back(r);
  }
  // rule 2: hit flags were taken above, before any miss moves a slot
  for (size_t i = first; i < out.size(); ++i) {
    if (out[i].hit) {
      ++cnt_.hits;
      continue;
    }
    moe_step_rec &r = out[i];  // rule 3, ascending misses
    ++cnt_.misses;
    cnt_.materialized_bytes += payload_;
    int32_t s = -1;
    if (used_ < n_slots_) {
      for (int32_t k = 0; k < n_slots_; ++k)
        if (expert_in_[k] < 0) {
          s = k;
          break;
        }
      ++used_;
    } else {
      int32_t victim = expert_in_[0];
      for (int32_t k = 1; k < n_slots_; ++k)
        if (stamp_[expert_in_[k]] < stamp_[victim]) victim = expert_in_[k];
      s = slot_of_[victim];
      slot_of_[victim] = -1;
      r.evicted = victim;
      ++cnt_.evictions;
    }
    expert_in_[s] = r.expert;
    slot_of_[r.expert] = s;
    r.slot = s;
  }
  ++step_no_;
}

}  // namespace moecache

struct moe_lru {
  moecache::SlotLru t;
  std::vector<moe_step_rec> buf;
};

extern "C" {

int moe_lru_create(int32_t n_experts, int32_t n_slots, uint64_t payload_bytes, int32_t layer,
                   moe_lru **out) {
  if (!out || n_experts < 1 || n_slots < 1 || n_slots > n_experts) return MOE_EINVAL;
  *out = new (std::nothrow) moe_lru{moecache::SlotLru(n_experts, n_slots, payload_bytes, layer), {}};
  return *out ? MOE_OK : MOE_ENOMEM;
}

int moe_lru_step(moe_lru *lru, const int32_t *ids, int32_t n, moe_step_rec *out, int32_t *n_out) {
  if (!lru || (n > 0 && (!ids || !out)) || n < 0 || !n_out) return MOE_EINVAL;
  for (int32_t i = 0; i < n; ++i)
    if (ids[i] < 0 || ids[i] >= lru->t.n_experts()) return MOE_EINVAL;
  lru->buf.clear();
  lru->t.step(ids, n, lru->buf);
  for (size_t i = 0; i < lru->buf.size(); ++i) out[i] = lru->buf[i];
  *n_out = (int32_t)lru->buf.size();
  return MOE_OK;
}

int moe_lru_counters(const moe_lru *lru, moe_counters *out) {
  if (!lru || !out) return MOE_EINVAL;
  *out = lru->t.counters();
  return MOE_OK;
}

void moe_lru_destroy(moe_lru *lru) { delete lru; }

}  // extern "C"
