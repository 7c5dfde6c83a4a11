// Drives the runtime's C ABI on the host (linked with fake_hip.cpp) so that a
// sanitizer build sees its argument checks, its per-layer state machine, the
// draining of records, the rollback after a miss copy that cannot be
// enqueued, the wait deadline, resets and teardown. Prints one line per
// check; exits non-zero on the first unexpected status.
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <vector>

#include "oled.h"

extern "C" void fake_hip_stall_events(int on);
extern "C" void fake_hip_stage_misses(int n);

static int g_fail = 0;
#define EXPECT(expr, want)                                                                  \
  do {                                                                                      \
    const int got_ = static_cast<int>(expr);                                                \
    std::printf("%-72s -> %d\n", #expr, got_);                                              \
    if (got_ != static_cast<int>(want)) {                                                   \
      std::printf("  expected %d: %s\n", static_cast<int>(want), oled_last_error(nullptr)); \
      g_fail = 1;                                                                           \
    }                                                                                       \
  } while (0)

static oled_config base_config(void* pool, const int64_t* hbo) {
  oled_config c;
  std::memset(&c, 0, sizeof(c));
  c.hidden = 128;
  c.inter = 128;
  c.n_experts = 8;
  c.top_k = 2;
  c.n_layers = 2;
  c.capacity = 3;
  c.max_tokens = 64;
  c.dtype = OLED_F32;
  c.host_pool = pool;
  c.host_pool_blocks = 16;
  c.host_block_of = hbo;
  return c;
}

// one layer-iteration through the four calls, every status as expected
static void layer(void* ctx, int l, const float* lg, int T, const float* conf, const void* x,
                  void* y) {
  EXPECT(route_block(ctx, l, lg, T, nullptr), OLED_OK);
  if (x) EXPECT(moe_forward_cached(ctx, l, x, y, nullptr), OLED_OK);
  oled_miss_report rep;
  EXPECT(apply_misses(ctx, l, nullptr, &rep), OLED_OK);
  EXPECT(score_and_retain(ctx, l, conf, nullptr), OLED_OK);
}

int main() {
  const int64_t eb = 3 * 128 * 128 * 4;
  void* pool = nullptr;
  EXPECT(oled_host_alloc(16 * eb, &pool), OLED_OK);
  std::vector<int64_t> hbo(16);
  for (int i = 0; i < 16; ++i) hbo[i] = i;
  std::vector<float> dev_lg(64 * 8, 0.f), conf(64, 0.5f), x(64 * 128, 0.f), y(64 * 128, 0.f);
  void* ctx = nullptr;

  // oled_create: argument checks
  oled_config c = base_config(pool, hbo.data());
  EXPECT(oled_create(nullptr, &ctx), OLED_ERR_INVALID_ARG);
  c.hidden = 100;
  EXPECT(oled_create(&c, &ctx), OLED_ERR_UNSUPPORTED);
  c = base_config(pool, hbo.data());
  c.n_experts = 300;
  c.top_k = 2;
  EXPECT(oled_create(&c, &ctx), OLED_ERR_UNSUPPORTED);
  c = base_config(pool, hbo.data());
  c.top_k = 9;
  EXPECT(oled_create(&c, &ctx), OLED_ERR_INVALID_ARG);
  c = base_config(pool, hbo.data());
  c.max_tokens = 70000;
  EXPECT(oled_create(&c, &ctx), OLED_ERR_UNSUPPORTED);
  c = base_config(pool, hbo.data());
  c.capacity = -1;
  EXPECT(oled_create(&c, &ctx), OLED_ERR_INVALID_ARG);
  c = base_config(pool, hbo.data());
  hbo[3] = 16;
  EXPECT(oled_create(&c, &ctx), OLED_ERR_INVALID_ARG);
  hbo[3] = 3;
  c = base_config(pool, hbo.data());
  std::vector<char> unpinned(16 * eb);
  c.host_pool = unpinned.data();
  EXPECT(oled_create(&c, &ctx), OLED_ERR_INVALID_ARG);
  c = base_config(pool, hbo.data());
  c.coop = 1;
  c.copy_mode = OLED_COPY_SDMA;
  c.coop_threads = 2;
  EXPECT(oled_create(&c, &ctx), OLED_ERR_UNSUPPORTED);
  c = base_config(pool, hbo.data());
  c.adapt_period = -2;
  EXPECT(oled_create(&c, &ctx), OLED_ERR_INVALID_ARG);
  if (ctx) g_fail = 1;

  // the per-layer state machine (shader transfer)
  c = base_config(pool, hbo.data());
  c.profile_ops = 0x7FF;
  EXPECT(oled_create(&c, &ctx), OLED_OK);
  EXPECT(apply_misses(ctx, 0, nullptr, nullptr), OLED_ERR_STATE);
  EXPECT(score_and_retain(ctx, 0, conf.data(), nullptr), OLED_ERR_STATE);
  EXPECT(moe_forward_cached(ctx, 0, x.data(), y.data(), nullptr), OLED_ERR_STATE);
  EXPECT(route_block(ctx, 0, dev_lg.data(), 0, nullptr), OLED_ERR_INVALID_ARG);
  EXPECT(route_block(ctx, 0, dev_lg.data(), 65, nullptr), OLED_ERR_INVALID_ARG);
  EXPECT(route_block(ctx, 2, dev_lg.data(), 8, nullptr), OLED_ERR_INVALID_ARG);
  EXPECT(route_block(ctx, 0, nullptr, 8, nullptr), OLED_ERR_INVALID_ARG);
  EXPECT(route_block(ctx, 0, dev_lg.data(), 8, nullptr), OLED_OK);
  EXPECT(route_block(ctx, 1, dev_lg.data(), 8, nullptr), OLED_ERR_STATE);
  EXPECT(apply_misses(ctx, 1, nullptr, nullptr), OLED_ERR_STATE);
  EXPECT(moe_forward_cached(ctx, 0, nullptr, y.data(), nullptr), OLED_ERR_INVALID_ARG);
  EXPECT(moe_forward_cached(ctx, 0, x.data(), y.data(), nullptr), OLED_OK);
  EXPECT(apply_misses(ctx, 0, nullptr, nullptr), OLED_OK);
  EXPECT(score_and_retain(ctx, 0, nullptr, nullptr), OLED_ERR_INVALID_ARG);
  EXPECT(score_and_retain(ctx, 0, conf.data(), nullptr), OLED_OK);
  for (int it = 0; it < 3; ++it)
    for (int l = 0; l < 2; ++l) layer(ctx, l, dev_lg.data(), 40, conf.data(), x.data(), y.data());
  layer(ctx, 1, dev_lg.data(), 64, conf.data(), nullptr, nullptr);   // control path only
  oled_stats stats;
  EXPECT(oled_collect_stats(ctx, &stats), OLED_OK);
  EXPECT(stats.layer_iters, 8);
  std::vector<oled_op_time> ops(4096);
  int32_t n_ops = 0;
  EXPECT(oled_profile_collect(ctx, ops.data(), 4096, &n_ops), OLED_OK);
  std::vector<int32_t> idx(64 * 2), counts(8), offsets(9), perm(64 * 2), inv(64 * 2), slot(8);
  std::vector<float> gates(64 * 2);
  std::vector<uint64_t> sq(8), key(8);
  std::vector<uint8_t> rb(8), ra(8), kept(8);
  oled_layer_state st;
  std::memset(&st, 0, sizeof(st));
  st.topk_idx = idx.data();
  st.gates = gates.data();
  st.counts = counts.data();
  st.offsets = offsets.data();
  st.perm = perm.data();
  st.inv_perm = inv.data();
  st.score_q = sq.data();
  st.resident_before = rb.data();
  st.resident_after = ra.data();
  st.slot_of = slot.data();
  st.retain_key = key.data();
  st.retained = kept.data();
  EXPECT(oled_read_layer_state(ctx, 1, &st), OLED_OK);
  EXPECT(st.tokens, 64);
  EXPECT(oled_read_layer_state(ctx, 5, &st), OLED_ERR_INVALID_ARG);
  EXPECT(oled_set_fault_injection(ctx, -1, 0), OLED_ERR_INVALID_ARG);
  EXPECT(oled_reset_cache(ctx), OLED_OK);
  layer(ctx, 0, dev_lg.data(), 16, conf.data(), x.data(), y.data());
  oled_destroy(ctx);
  ctx = nullptr;

  // copy-engine transfer: a miss copy that cannot be enqueued, then a wait
  // past its deadline
  c = base_config(pool, hbo.data());
  c.copy_mode = OLED_COPY_SDMA;
  EXPECT(oled_create(&c, &ctx), OLED_OK);
  fake_hip_stage_misses(2);
  layer(ctx, 0, dev_lg.data(), 32, conf.data(), x.data(), y.data());
  EXPECT(oled_set_fault_injection(ctx, 3, 0), OLED_OK);
  EXPECT(route_block(ctx, 1, dev_lg.data(), 32, nullptr), OLED_OK);
  EXPECT(moe_forward_cached(ctx, 1, x.data(), y.data(), nullptr), OLED_OK);
  EXPECT(apply_misses(ctx, 1, nullptr, nullptr), OLED_ERR_HIP);
  std::printf("  %s\n", oled_last_error(ctx));
  EXPECT(score_and_retain(ctx, 1, conf.data(), nullptr), OLED_ERR_STATE);
  layer(ctx, 1, dev_lg.data(), 32, conf.data(), x.data(), y.data());   // the context goes on
  EXPECT(oled_set_fault_injection(ctx, 0, 5), OLED_OK);
  fake_hip_stall_events(1);
  EXPECT(route_block(ctx, 0, dev_lg.data(), 32, nullptr), OLED_OK);
  EXPECT(moe_forward_cached(ctx, 0, x.data(), y.data(), nullptr), OLED_OK);
  EXPECT(apply_misses(ctx, 0, nullptr, nullptr), OLED_ERR_HIP);
  std::printf("  %s\n", oled_last_error(ctx));
  EXPECT(route_block(ctx, 0, dev_lg.data(), 32, nullptr), OLED_ERR_STATE);
  fake_hip_stall_events(0);
  EXPECT(oled_reset_cache(ctx), OLED_OK);
  EXPECT(oled_set_fault_injection(ctx, 0, 0), OLED_OK);
  layer(ctx, 0, dev_lg.data(), 32, conf.data(), x.data(), y.data());
  oled_destroy(ctx);
  fake_hip_stage_misses(0);

  // layer-adaptive sizing and the comparison policies: create, a few steps, destroy
  for (int policy = 0; policy < 3; ++policy) {
    c = base_config(pool, hbo.data());
    c.adapt_period = policy == 0 ? 1 : 0;
    c.policy = policy;
    EXPECT(oled_create(&c, &ctx), OLED_OK);
    for (int it = 0; it < 2; ++it)
      for (int l = 0; l < 2; ++l) layer(ctx, l, dev_lg.data(), 24, conf.data(), x.data(), y.data());
    oled_destroy(ctx);
  }
  oled_destroy(nullptr);
  oled_host_free(pool);
  std::printf(g_fail ? "FAILED\n" : "ALL OK\n");
  return g_fail;
}
