#include "cache_state.h"

#include <algorithm>

namespace oled {

CacheState::CacheState(int n_layers, int n_experts, int capacity, int n_slots)
    : L_(n_layers), E_(n_experts), C_(capacity), n_slots_(n_slots) {
  reset();
}

void CacheState::reset() {
  const size_t n = static_cast<size_t>(L_) * E_;
  slot_.assign(n, -1);
  res_.assign(n, 0);
  staged_.assign(n, 0);
  free_.clear();
  free_.reserve(n_slots_);
  // lowest slot index on top of the stack
  for (int s = n_slots_ - 1; s >= 0; --s) free_.push_back(s);
}

int CacheState::resident_count(int l) const {
  int n = 0;
  for (int e = 0; e < E_; ++e) n += resident(l)[e] ? 1 : 0;
  return n;
}

int CacheState::staged_count(int l) const {
  int n = 0;
  for (int e = 0; e < E_; ++e) n += staged(l)[e] ? 1 : 0;
  return n;
}

void CacheState::launch_slots(int l, int32_t* out) const {
  for (int e = 0; e < E_; ++e) out[e] = slot_of(l)[e];
}

void CacheState::classify(int l, const int32_t* counts, uint8_t* hit, uint8_t* miss,
                          int* n_active, int* n_hits, int* n_misses) const {
  int na = 0, nh = 0, nm = 0;
  const uint8_t* r = resident(l);
  for (int e = 0; e < E_; ++e) {
    const bool a = counts[e] > 0;
    hit[e] = (a && r[e]) ? 1 : 0;
    miss[e] = (a && !r[e]) ? 1 : 0;
    na += a;
    nh += hit[e];
    nm += miss[e];
  }
  *n_active = na;
  *n_hits = nh;
  *n_misses = nm;
}

bool CacheState::stage_misses(int l, const uint8_t* miss, std::vector<int32_t>* experts,
                              std::vector<int32_t>* slots) {
  if (staged_count(l) != 0) return false;
  int need = 0;
  for (int e = 0; e < E_; ++e) {
    if (miss[e] && resident(l)[e]) return false;  // a miss is never resident
    need += miss[e] ? 1 : 0;
  }
  if (need > free_slots()) return false;
  experts->clear();
  slots->clear();
  const size_t base = static_cast<size_t>(l) * E_;
  for (int e = 0; e < E_; ++e) {
    if (!miss[e]) continue;
    const int32_t s = free_.back();
    free_.pop_back();
    slot_[base + e] = s;
    staged_[base + e] = 1;
    experts->push_back(e);
    slots->push_back(s);
  }
  return true;
}

void CacheState::drop_staged(int l) {
  const size_t base = static_cast<size_t>(l) * E_;
  for (int e = 0; e < E_; ++e) {
    if (!staged_[base + e]) continue;
    free_.push_back(slot_[base + e]);
    slot_[base + e] = -1;
    staged_[base + e] = 0;
  }
}

bool CacheState::commit(int l, const uint8_t* retained) {
  const size_t base = static_cast<size_t>(l) * E_;
  int kept = 0;
  for (int e = 0; e < E_; ++e) {
    if (!retained[e]) continue;
    if (!res_[base + e] && !staged_[base + e]) return false;
    ++kept;
  }
  if (kept > C_) return false;
  for (int e = 0; e < E_; ++e) {
    const bool held = res_[base + e] || staged_[base + e];
    if (held && !retained[e]) {
      free_.push_back(slot_[base + e]);
      slot_[base + e] = -1;
    }
    res_[base + e] = retained[e] ? 1 : 0;
    staged_[base + e] = 0;
  }
  return true;
}

bool CacheState::check() const {
  std::vector<int> owner(n_slots_, 0);
  for (int32_t s : free_) {
    if (s < 0 || s >= n_slots_) return false;
    owner[s]++;
  }
  for (int l = 0; l < L_; ++l) {
    int nres = 0;
    for (int e = 0; e < E_; ++e) {
      const size_t i = static_cast<size_t>(l) * E_ + e;
      const bool held = res_[i] || staged_[i];
      if (res_[i] && staged_[i]) return false;
      if (held != (slot_[i] >= 0)) return false;
      if (held) {
        if (slot_[i] >= n_slots_) return false;
        owner[slot_[i]]++;
      }
      nres += res_[i] ? 1 : 0;
    }
    if (nres > C_) return false;
  }
  for (int s = 0; s < n_slots_; ++s)
    if (owner[s] != 1) return false;
  return true;
}

}  // namespace oled
