// Host-side bookkeeping of the per-layer GPU expert caches (OLED-MoE Sec. 4.1:
// one independent cache pool per MoE layer). Pure C++, no HIP: the slot pool,
// each layer's committed resident set R and slot table, the staging of misses
// (Sec. 4.2: M = A \ R, all transferred) and the commit of a retention result.
//
// Slots: one global pool of n_slots expert-sized slots. A layer owns at most C
// slots for committed residents; misses are staged in free slots and, when
// retained, keep their slot (no device-to-device move); evicted experts
// return their slot to the free list.
#pragma once

#include <cstddef>
#include <cstdint>
#include <vector>

namespace oled {

class CacheState {
 public:
  CacheState() = default;
  CacheState(int n_layers, int n_experts, int capacity, int n_slots);

  int n_layers() const { return L_; }
  int n_experts() const { return E_; }
  int capacity() const { return C_; }
  int n_slots() const { return n_slots_; }
  int free_slots() const { return static_cast<int>(free_.size()); }

  // committed state of layer l
  const int32_t* slot_of(int l) const { return &slot_[static_cast<size_t>(l) * E_]; }
  const uint8_t* resident(int l) const { return &res_[static_cast<size_t>(l) * E_]; }
  int resident_count(int l) const;
  // staged misses of layer l (nonzero while a layer has misses in flight)
  const uint8_t* staged(int l) const { return &staged_[static_cast<size_t>(l) * E_]; }
  int staged_count(int l) const;
  // slot table a kernel should read for layer l: residents and staged misses
  void launch_slots(int l, int32_t* out) const;

  // hit/miss classification of layer l from the per-expert route counts
  void classify(int l, const int32_t* counts, uint8_t* hit, uint8_t* miss, int* n_active,
                int* n_hits, int* n_misses) const;

  // Gives each miss of layer l a free slot. Fails (false, nothing changed) if
  // the layer already has staged misses or too few slots are free.
  // assigned receives (expert, slot) pairs in expert order.
  bool stage_misses(int l, const uint8_t* miss, std::vector<int32_t>* assigned_experts,
                    std::vector<int32_t>* assigned_slots);
  // Releases the staged slots of layer l (failed copy, invalid retention).
  void drop_staged(int l);

  // Commits a retention result of layer l: retained[e] != 0 keeps expert e.
  // Valid only if every retained expert is resident or staged and at most C
  // are retained; otherwise returns false and changes nothing.
  bool commit(int l, const uint8_t* retained);

  // Empties every layer (R := {} and no staged misses).
  void reset();

  // Slot conservation and capacity invariants; false if violated.
  bool check() const;

 private:
  int L_ = 0, E_ = 0, C_ = 0, n_slots_ = 0;
  std::vector<int32_t> slot_;    // [L][E] slot of a resident or staged expert, -1 otherwise
  std::vector<uint8_t> res_;     // [L][E] committed residents
  std::vector<uint8_t> staged_;  // [L][E] staged misses
  std::vector<int32_t> free_;    // free slot stack
};

}  // namespace oled
