// C entry points over oled::CacheState for host-only tests (built with g++
// into a separate library; no HIP). Not part of the public ABI.
#include <cstdint>
#include <vector>

#include "cache_state.h"

extern "C" {

void* oled_cs_create(int L, int E, int C, int n_slots) {
  if (L <= 0 || E <= 0 || C < 0 || n_slots < 0) return nullptr;
  return new oled::CacheState(L, E, C, n_slots);
}

void oled_cs_destroy(void* p) { delete static_cast<oled::CacheState*>(p); }

void oled_cs_reset(void* p) { static_cast<oled::CacheState*>(p)->reset(); }

int oled_cs_check(const void* p) { return static_cast<const oled::CacheState*>(p)->check() ? 1 : 0; }

int oled_cs_free_slots(const void* p) { return static_cast<const oled::CacheState*>(p)->free_slots(); }

void oled_cs_classify(const void* p, int l, const int32_t* counts, uint8_t* hit, uint8_t* miss,
                      int32_t* n3) {
  int a = 0, h = 0, m = 0;
  static_cast<const oled::CacheState*>(p)->classify(l, counts, hit, miss, &a, &h, &m);
  n3[0] = a;
  n3[1] = h;
  n3[2] = m;
}

// Returns the number of staged misses, or -1 if staging was refused.
int oled_cs_stage(void* p, int l, const uint8_t* miss, int32_t* experts, int32_t* slots) {
  std::vector<int32_t> ex, sl;
  if (!static_cast<oled::CacheState*>(p)->stage_misses(l, miss, &ex, &sl)) return -1;
  for (size_t i = 0; i < ex.size(); ++i) {
    experts[i] = ex[i];
    slots[i] = sl[i];
  }
  return static_cast<int>(ex.size());
}

void oled_cs_drop(void* p, int l) { static_cast<oled::CacheState*>(p)->drop_staged(l); }

int oled_cs_commit(void* p, int l, const uint8_t* retained) {
  return static_cast<oled::CacheState*>(p)->commit(l, retained) ? 1 : 0;
}

void oled_cs_resident(const void* p, int l, uint8_t* out) {
  const auto* cs = static_cast<const oled::CacheState*>(p);
  for (int e = 0; e < cs->n_experts(); ++e) out[e] = cs->resident(l)[e];
}

void oled_cs_slots(const void* p, int l, int32_t* out) {
  const auto* cs = static_cast<const oled::CacheState*>(p);
  for (int e = 0; e < cs->n_experts(); ++e) out[e] = cs->slot_of(l)[e];
}

}  // extern "C"
