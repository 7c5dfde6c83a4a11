// Randomised self-test of the host cache bookkeeping, built with
// AddressSanitizer and UndefinedBehaviorSanitizer by the CPU test suite.
// Drives stage / commit / drop sequences and checks slot conservation and the
// capacity bound after every step.
#include <cstdio>
#include <random>
#include <vector>

#include "cache_state.h"

static int fail(const char* what, int step) {
  std::fprintf(stderr, "FAIL %s at step %d\n", what, step);
  return 1;
}

int main() {
  std::mt19937 rng(12345);
  for (int trial = 0; trial < 200; ++trial) {
    const int L = 1 + rng() % 4, E = 1 + rng() % 40, C = rng() % (E + 3);
    const int cap = C < E ? C : E;
    const int n_slots = L * cap + E;
    oled::CacheState cs(L, E, C, n_slots);
    if (!cs.check()) return fail("initial check", 0);
    std::vector<uint8_t> hit(E), miss(E), keep(E);
    std::vector<int32_t> counts(E), ex, sl;
    for (int step = 0; step < 60; ++step) {
      const int l = rng() % L;
      for (int e = 0; e < E; ++e) counts[e] = (rng() % 3 == 0) ? 1 + rng() % 5 : 0;
      int na, nh, nm;
      cs.classify(l, counts.data(), hit.data(), miss.data(), &na, &nh, &nm);
      if (na != nh + nm) return fail("classify", step);
      if (!cs.stage_misses(l, miss.data(), &ex, &sl)) return fail("stage refused", step);
      if (static_cast<int>(ex.size()) != nm) return fail("staged count", step);
      if (!cs.check()) return fail("check after stage", step);
      if (rng() % 7 == 0) {  // a failed copy or a rejected retention
        cs.drop_staged(l);
        if (cs.staged_count(l) != 0 || !cs.check()) return fail("drop", step);
        continue;
      }
      // keep a random subset of the candidates, at most C
      int kept = 0;
      for (int e = 0; e < E; ++e) {
        const bool cand = cs.resident(l)[e] || cs.staged(l)[e];
        keep[e] = (cand && kept < C && rng() % 2) ? 1 : 0;
        kept += keep[e];
      }
      if (!cs.commit(l, keep.data())) return fail("commit refused", step);
      if (!cs.check()) return fail("check after commit", step);
      for (int e = 0; e < E; ++e)
        if (cs.resident(l)[e] != keep[e]) return fail("resident != retained", step);
      // an invalid commit (a non-candidate) is refused without change
      for (int e = 0; e < E; ++e) {
        if (!cs.resident(l)[e] && !cs.staged(l)[e]) {
          std::vector<uint8_t> badk(E, 0);
          badk[e] = 1;
          if (cs.commit(l, badk.data())) return fail("invalid commit accepted", step);
          if (!cs.check()) return fail("check after invalid commit", step);
          break;
        }
      }
    }
    cs.reset();
    if (cs.free_slots() != n_slots || !cs.check()) return fail("reset", 0);
  }
  std::printf("cache_state selftest ok\n");
  return 0;
}
