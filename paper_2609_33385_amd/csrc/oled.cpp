// Host runtime of the C ABI declared in include/oled.h: the context, the call
// state machine, the per-layer cache bookkeeping, the host-to-device miss
// copies on a side stream and the kernel launches.
#include "oled.h"

#include <hip/hip_runtime.h>

#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <string>
#include <vector>

#include "cache_state.h"
#include "kernels.h"

namespace {

using oled::ExpertMask;
using oled::RetainOut;
using oled::RouteSummary;
using oled::SlotTable;
using oled::WorkItem;

thread_local std::string g_create_error;

enum class Stage { kIdle, kRouted, kApplied, kForwarded };

struct OpRec {
  int kind, layer;
  int64_t bytes, flops;
  hipEvent_t a, b;
};

struct Ctx {
  // shape
  int H = 0, I = 0, E = 0, K = 0, L = 0, C = 0, Tmax = 0, dtype = 0, esz = 0, device = 0, flags = 0;
  int64_t eb = 0;   // bytes of one expert block
  int n_slots = 0;
  int max_items = 0;
  const char* host_pool = nullptr;
  int64_t P = 0;
  std::vector<int64_t> host_block_of;
  // device memory
  char* d_pool = nullptr;
  int32_t* d_topk = nullptr;
  float* d_gates = nullptr;
  int32_t* d_counts = nullptr;
  int32_t* d_offsets = nullptr;
  int32_t* d_perm = nullptr;
  int32_t* d_inv = nullptr;
  int32_t* d_flag = nullptr;
  WorkItem* d_items = nullptr;
  void* d_h = nullptr;
  float* d_O = nullptr;
  uint64_t* d_score = nullptr;  // [L][E]
  // pinned host memory written by kernels
  RouteSummary* h_sum = nullptr;
  RetainOut* h_ret = nullptr;  // [L]
  // streams and events
  hipStream_t own_copy = nullptr;
  hipEvent_t ev_route = nullptr, ev_copy = nullptr, ev_order = nullptr;
  std::vector<hipEvent_t> ev_retain;
  // cache state
  oled::CacheState cs;
  std::vector<uint8_t> pending;     // [L] retention result not yet committed
  std::vector<int> ret_seq;         // [L] sequence number of that result
  std::vector<uint8_t> rejected;    // [L] last retention rejected (bad confidence)
  std::vector<uint8_t> res_before;  // [L][E] R before the layer's last execution
  std::vector<int> last_counts;     // [L][3] n_active, n_hits, n_misses of the last apply
  // the layer in flight
  Stage stage = Stage::kIdle;
  int cur_layer = -1, cur_T = 0;
  hipStream_t cur_stream = nullptr;
  bool have_stream = false;
  int last_routed_layer = -1, last_routed_T = 0;
  std::vector<int32_t> counts;      // [E] route counts of the layer in flight
  std::vector<uint8_t> hit, miss;
  int n_active = 0, n_hits = 0, n_misses = 0, n_hit_items = 0, n_miss_items = 0;
  int64_t hit_rows = 0, miss_rows = 0;
  bool copies_outstanding = false;
  int seq = 0, route_seq = 0;
  int rejected_layer = -1;          // reported by the next apply_misses
  std::string err;
  // profiling
  std::vector<OpRec> ops;
  std::vector<hipEvent_t> ev_free;
};

oled_status fail(Ctx* c, oled_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  c->err = buf;
  return st;
}

oled_status hip_fail(Ctx* c, hipError_t e, const char* what) {
  return fail(c, OLED_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

#define HIP_TRY(c, expr)                                 \
  do {                                                   \
    hipError_t e_ = (expr);                              \
    if (e_ != hipSuccess) return hip_fail((c), e_, #expr); \
  } while (0)

hipEvent_t take_event(Ctx* c) {
  if (!c->ev_free.empty()) {
    hipEvent_t e = c->ev_free.back();
    c->ev_free.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}

// Event pair around one operation when profiling is on.
struct OpTimer {
  Ctx* c;
  hipStream_t s;
  hipEvent_t a = nullptr;
  OpTimer(Ctx* c_, hipStream_t s_) : c(c_), s(s_) {
    if (c->flags & OLED_FLAG_PROFILE) {
      a = take_event(c);
      if (a) hipEventRecord(a, s);
    }
  }
  void done(int kind, int layer, int64_t bytes, int64_t flops) {
    if (!a) return;
    hipEvent_t b = take_event(c);
    if (!b) return;
    hipEventRecord(b, s);
    c->ops.push_back(OpRec{kind, layer, bytes, flops, a, b});
    a = nullptr;
  }
};

ExpertMask mask_of(const uint8_t* m, int E) {
  ExpertMask x;
  std::memset(&x, 0, sizeof(x));
  for (int e = 0; e < E; ++e)
    if (m[e]) x.bits[e >> 5] |= 1u << (e & 31);
  return x;
}

// Commits the retention result of layer l (waits for its event).
oled_status consume_layer(Ctx* c, int l) {
  if (!c->pending[l]) return OLED_OK;
  HIP_TRY(c, hipEventSynchronize(c->ev_retain[l]));
  const RetainOut& o = c->h_ret[l];
  c->pending[l] = 0;
  if (o.seq != c->ret_seq[l]) {
    c->cs.drop_staged(l);
    return fail(c, OLED_ERR_HIP, "stale retention result for layer %d", l);
  }
  if (o.bad_conf) {
    c->cs.drop_staged(l);
    c->rejected[l] = 1;
    c->rejected_layer = l;
    return fail(c, OLED_ERR_INVALID_ARG, "confidence outside [0,1] at layer %d: retention skipped", l);
  }
  c->rejected[l] = 0;
  if (!c->cs.commit(l, o.retained)) {
    c->cs.drop_staged(l);
    return fail(c, OLED_ERR_HIP, "inconsistent retention result for layer %d", l);
  }
  return OLED_OK;
}

oled_status consume_all(Ctx* c) {
  oled_status worst = OLED_OK;
  for (int l = 0; l < c->L; ++l) {
    const oled_status st = consume_layer(c, l);
    if (st == OLED_ERR_HIP) return st;
    if (st != OLED_OK) worst = st;
  }
  return worst;
}

void free_ctx(Ctx* c) {
  if (!c) return;
  hipSetDevice(c->device);
  hipDeviceSynchronize();
  for (auto& op : c->ops) {
    hipEventDestroy(op.a);
    hipEventDestroy(op.b);
  }
  for (auto e : c->ev_free) hipEventDestroy(e);
  for (auto e : c->ev_retain)
    if (e) hipEventDestroy(e);
  if (c->ev_route) hipEventDestroy(c->ev_route);
  if (c->ev_copy) hipEventDestroy(c->ev_copy);
  if (c->ev_order) hipEventDestroy(c->ev_order);
  if (c->own_copy) hipStreamDestroy(c->own_copy);
  hipFree(c->d_pool);
  hipFree(c->d_topk);
  hipFree(c->d_gates);
  hipFree(c->d_counts);
  hipFree(c->d_offsets);
  hipFree(c->d_perm);
  hipFree(c->d_inv);
  hipFree(c->d_flag);
  hipFree(c->d_items);
  hipFree(c->d_h);
  hipFree(c->d_O);
  hipFree(c->d_score);
  if (c->h_sum) hipHostFree(c->h_sum);
  if (c->h_ret) hipHostFree(c->h_ret);
  delete c;
}

template <class T>
hipError_t dev_alloc(T** p, size_t n) {
  return hipMalloc(reinterpret_cast<void**>(p), n * sizeof(T) > 0 ? n * sizeof(T) : 16);
}

oled_status check_call(Ctx* c, int layer, Stage want) {
  if (layer < 0 || layer >= c->L)
    return fail(c, OLED_ERR_INVALID_ARG, "layer %d outside [0,%d)", layer, c->L);
  if (c->stage != want)
    return fail(c, OLED_ERR_STATE, "call out of order (layer %d, stage %d)", layer,
                static_cast<int>(c->stage));
  if (want != Stage::kIdle && layer != c->cur_layer)
    return fail(c, OLED_ERR_STATE, "layer %d is not the layer in flight (%d)", layer, c->cur_layer);
  return OLED_OK;
}

}  // namespace

extern "C" {

oled_status oled_create(const oled_config* cfg, void** ctx_out) {
  if (ctx_out) *ctx_out = nullptr;
  auto bad = [](oled_status st, const char* m) {
    g_create_error = m;
    return st;
  };
  if (!cfg || !ctx_out) return bad(OLED_ERR_INVALID_ARG, "NULL config or output pointer");
  if (cfg->hidden <= 0 || cfg->inter <= 0 || cfg->n_experts <= 0 || cfg->top_k <= 0 ||
      cfg->n_layers <= 0 || cfg->capacity < 0 || cfg->max_tokens <= 0)
    return bad(OLED_ERR_INVALID_ARG, "non-positive shape field");
  if (cfg->dtype != OLED_F32 && cfg->dtype != OLED_BF16)
    return bad(OLED_ERR_INVALID_ARG, "dtype must be OLED_F32 or OLED_BF16");
  if (cfg->top_k > cfg->n_experts) return bad(OLED_ERR_INVALID_ARG, "top_k > n_experts");
  if (cfg->hidden % 128 || cfg->inter % 128)
    return bad(OLED_ERR_UNSUPPORTED, "hidden and inter must be multiples of 128");
  if (cfg->n_experts > oled::kMaxExperts) return bad(OLED_ERR_UNSUPPORTED, "n_experts > 256");
  if (cfg->top_k > oled::kMaxTopK) return bad(OLED_ERR_UNSUPPORTED, "top_k > 16");
  if (cfg->max_tokens > 65535) return bad(OLED_ERR_UNSUPPORTED, "max_tokens > 65535");
  if (!cfg->host_pool || cfg->host_pool_blocks <= 0 || !cfg->host_block_of)
    return bad(OLED_ERR_INVALID_ARG, "host pool, block count and block table are required");
  const int64_t nb = static_cast<int64_t>(cfg->n_layers) * cfg->n_experts;
  for (int64_t i = 0; i < nb; ++i)
    if (cfg->host_block_of[i] < 0 || cfg->host_block_of[i] >= cfg->host_pool_blocks)
      return bad(OLED_ERR_INVALID_ARG, "host_block_of entry outside [0, host_pool_blocks)");

  int ndev = 0;
  if (hipGetDeviceCount(&ndev) != hipSuccess || ndev <= 0)
    return bad(OLED_ERR_HIP, "no HIP device");
  if (cfg->device < 0 || cfg->device >= ndev) return bad(OLED_ERR_INVALID_ARG, "bad device ordinal");
  if (hipSetDevice(cfg->device) != hipSuccess) return bad(OLED_ERR_HIP, "hipSetDevice failed");

  hipPointerAttribute_t attr;
  std::memset(&attr, 0, sizeof(attr));
  if (hipPointerGetAttributes(&attr, cfg->host_pool) != hipSuccess || attr.type != hipMemoryTypeHost) {
    (void)hipGetLastError();
    return bad(OLED_ERR_INVALID_ARG, "host_pool is not pinned host memory");
  }

  Ctx* c = new Ctx();
  c->H = cfg->hidden;
  c->I = cfg->inter;
  c->E = cfg->n_experts;
  c->K = cfg->top_k;
  c->L = cfg->n_layers;
  c->C = cfg->capacity;
  c->Tmax = cfg->max_tokens;
  c->dtype = cfg->dtype;
  c->esz = cfg->dtype == OLED_F32 ? 4 : 2;
  c->device = cfg->device;
  c->flags = cfg->flags;
  c->eb = static_cast<int64_t>(3) * c->H * c->I * c->esz;
  const int cap = c->C < c->E ? c->C : c->E;
  const int64_t routes = static_cast<int64_t>(c->Tmax) * c->K;
  const int staging = routes < c->E ? static_cast<int>(routes) : c->E;
  c->n_slots = c->L * cap + staging;
  c->max_items = static_cast<int>(routes / oled::kItemRows) + c->E + 1;
  c->host_pool = static_cast<const char*>(cfg->host_pool);
  c->P = cfg->host_pool_blocks;
  c->host_block_of.assign(cfg->host_block_of, cfg->host_block_of + nb);

  auto oom = [&](const char* what) {
    (void)hipGetLastError();
    g_create_error = std::string("device allocation failed: ") + what;
    free_ctx(c);
    return OLED_ERR_OUT_OF_MEMORY;
  };
  if (hipMalloc(reinterpret_cast<void**>(&c->d_pool), static_cast<size_t>(c->n_slots) * c->eb) !=
      hipSuccess)
    return oom("slot pool");
  if (dev_alloc(&c->d_topk, routes) || dev_alloc(&c->d_gates, routes) ||
      dev_alloc(&c->d_counts, c->E) || dev_alloc(&c->d_offsets, c->E + 1) ||
      dev_alloc(&c->d_perm, routes) || dev_alloc(&c->d_inv, routes) || dev_alloc(&c->d_flag, 1) ||
      dev_alloc(&c->d_items, c->max_items) ||
      dev_alloc(reinterpret_cast<char**>(&c->d_h), routes * c->I * c->esz) ||
      dev_alloc(&c->d_O, routes * c->H) ||
      dev_alloc(&c->d_score, static_cast<size_t>(c->L) * c->E))
    return oom("routing scratch");
  if (hipMemset(c->d_flag, 0, sizeof(int32_t)) != hipSuccess ||
      hipMemset(c->d_score, 0, sizeof(uint64_t) * c->L * c->E) != hipSuccess)
    return oom("scratch init");
  if (hipHostMalloc(reinterpret_cast<void**>(&c->h_sum), sizeof(RouteSummary), hipHostMallocDefault) ||
      hipHostMalloc(reinterpret_cast<void**>(&c->h_ret), sizeof(RetainOut) * c->L, hipHostMallocDefault))
    return oom("pinned summaries");
  std::memset(c->h_sum, 0, sizeof(RouteSummary));
  std::memset(c->h_ret, 0, sizeof(RetainOut) * c->L);
  if (hipStreamCreateWithFlags(&c->own_copy, hipStreamNonBlocking) != hipSuccess ||
      hipEventCreateWithFlags(&c->ev_route, hipEventDisableTiming) != hipSuccess ||
      hipEventCreateWithFlags(&c->ev_copy, hipEventDisableTiming) != hipSuccess ||
      hipEventCreateWithFlags(&c->ev_order, hipEventDisableTiming) != hipSuccess) {
    g_create_error = "stream/event creation failed";
    free_ctx(c);
    return OLED_ERR_HIP;
  }
  c->ev_retain.assign(c->L, nullptr);
  for (int l = 0; l < c->L; ++l)
    if (hipEventCreateWithFlags(&c->ev_retain[l], hipEventDisableTiming) != hipSuccess) {
      g_create_error = "event creation failed";
      free_ctx(c);
      return OLED_ERR_HIP;
    }
  c->cs = oled::CacheState(c->L, c->E, c->C, c->n_slots);
  c->pending.assign(c->L, 0);
  c->ret_seq.assign(c->L, 0);
  c->rejected.assign(c->L, 0);
  c->res_before.assign(static_cast<size_t>(c->L) * c->E, 0);
  c->last_counts.assign(static_cast<size_t>(c->L) * 3, 0);
  c->counts.assign(c->E, 0);
  c->hit.assign(c->E, 0);
  c->miss.assign(c->E, 0);
  if (hipDeviceSynchronize() != hipSuccess) {
    g_create_error = "device synchronisation failed";
    free_ctx(c);
    return OLED_ERR_HIP;
  }
  g_create_error.clear();
  *ctx_out = c;
  return OLED_OK;
}

void oled_destroy(void* ctx) { free_ctx(static_cast<Ctx*>(ctx)); }

const char* oled_last_error(const void* ctx) {
  if (!ctx) return g_create_error.c_str();
  return static_cast<const Ctx*>(ctx)->err.c_str();
}

oled_status oled_reset_cache(void* ctx) {
  Ctx* c = static_cast<Ctx*>(ctx);
  if (!c) return OLED_ERR_INVALID_ARG;
  if (c->stage != Stage::kIdle) return fail(c, OLED_ERR_STATE, "reset while a layer is in flight");
  HIP_TRY(c, hipSetDevice(c->device));
  HIP_TRY(c, hipDeviceSynchronize());
  for (int l = 0; l < c->L; ++l) c->pending[l] = 0;
  c->cs.reset();
  std::fill(c->rejected.begin(), c->rejected.end(), 0);
  std::fill(c->res_before.begin(), c->res_before.end(), 0);
  c->rejected_layer = -1;
  return OLED_OK;
}

oled_status route_block(void* ctx, int32_t layer, const float* logits_dev, int32_t T, void* stream) {
  Ctx* c = static_cast<Ctx*>(ctx);
  if (!c) return OLED_ERR_INVALID_ARG;
  oled_status st = check_call(c, layer, Stage::kIdle);
  if (st != OLED_OK) return st;
  if (!logits_dev) return fail(c, OLED_ERR_INVALID_ARG, "NULL logits");
  if (T < 1 || T > c->Tmax) return fail(c, OLED_ERR_INVALID_ARG, "T=%d outside [1,%d]", T, c->Tmax);
  HIP_TRY(c, hipSetDevice(c->device));
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (c->have_stream && s != c->cur_stream) {  // order the new stream after the old one
    HIP_TRY(c, hipEventRecord(c->ev_order, c->cur_stream));
    HIP_TRY(c, hipStreamWaitEvent(s, c->ev_order, 0));
  }
  if (c->pending[layer]) {  // the hit/miss split needs this layer's committed R
    st = consume_layer(c, layer);
    if (st == OLED_ERR_HIP) return st;
  }
  const ExpertMask res = mask_of(c->cs.resident(layer), c->E);
  const int seq = ++c->seq;
  {
    OpTimer tm(c, s);
    HIP_TRY(c, oled::launch_route_topk(logits_dev, T, c->E, c->K, c->d_topk, c->d_gates, c->d_flag, s));
    tm.done(OLED_OP_ROUTE_TOPK, layer, static_cast<int64_t>(T) * c->E * 4 + static_cast<int64_t>(T) * c->K * 8, 0);
  }
  {
    OpTimer tm(c, s);
    HIP_TRY(c, oled::launch_permute(c->d_topk, T, c->K, c->E, res, c->d_counts, c->d_offsets,
                                    c->d_perm, c->d_inv, c->d_items, c->d_flag, c->h_sum, seq, s));
    tm.done(OLED_OP_PERMUTE, layer, static_cast<int64_t>(T) * c->K * 12 + static_cast<int64_t>(c->E) * 8, 0);
  }
  HIP_TRY(c, hipEventRecord(c->ev_route, s));
  c->route_seq = seq;
  c->stage = Stage::kRouted;
  c->cur_layer = layer;
  c->cur_T = T;
  c->cur_stream = s;
  c->have_stream = true;
  c->last_routed_layer = layer;
  c->last_routed_T = T;
  return OLED_OK;
}

oled_status apply_misses(void* ctx, int32_t layer, void* copy_stream, oled_miss_report* out) {
  Ctx* c = static_cast<Ctx*>(ctx);
  if (!c) return OLED_ERR_INVALID_ARG;
  oled_status st = check_call(c, layer, Stage::kRouted);
  if (st != OLED_OK) return st;
  HIP_TRY(c, hipSetDevice(c->device));
  HIP_TRY(c, hipEventSynchronize(c->ev_route));
  if (c->h_sum->seq != c->route_seq) {
    c->stage = Stage::kIdle;
    return fail(c, OLED_ERR_HIP, "stale route summary");
  }
  // every retention enqueued before this route has completed: commit them
  st = consume_all(c);
  if (st == OLED_ERR_HIP) {
    c->stage = Stage::kIdle;
    return st;
  }
  if (c->h_sum->bad_logits) {
    c->stage = Stage::kIdle;
    return fail(c, OLED_ERR_INVALID_ARG, "non-finite router logit at layer %d", layer);
  }
  std::memcpy(c->counts.data(), c->h_sum->counts, sizeof(int32_t) * c->E);
  c->cs.classify(layer, c->counts.data(), c->hit.data(), c->miss.data(), &c->n_active, &c->n_hits,
                 &c->n_misses);
  int nhi = 0, nmi = 0;
  c->hit_rows = c->miss_rows = 0;
  for (int e = 0; e < c->E; ++e) {
    const int ni = (c->counts[e] + oled::kItemRows - 1) / oled::kItemRows;
    if (c->hit[e]) {
      nhi += ni;
      c->hit_rows += c->counts[e];
    }
    if (c->miss[e]) {
      nmi += ni;
      c->miss_rows += c->counts[e];
    }
  }
  if (nhi != c->h_sum->n_hit_items || nmi != c->h_sum->n_miss_items) {
    c->stage = Stage::kIdle;
    return fail(c, OLED_ERR_HIP, "work list disagrees with the host cache state");
  }
  c->n_hit_items = nhi;
  c->n_miss_items = nmi;
  std::memcpy(&c->res_before[static_cast<size_t>(layer) * c->E], c->cs.resident(layer), c->E);
  const int n_res = c->cs.resident_count(layer);

  std::vector<int32_t> exps, slots;
  if (!c->cs.stage_misses(layer, c->miss.data(), &exps, &slots)) {
    c->stage = Stage::kIdle;
    return fail(c, OLED_ERR_HIP, "no free staging slots (internal accounting error)");
  }
  hipStream_t cs = copy_stream ? static_cast<hipStream_t>(copy_stream) : c->own_copy;
  int64_t bytes = 0;
  if (!exps.empty()) {
    OpTimer tm(c, cs);
    for (size_t i = 0; i < exps.size(); ++i) {
      const int64_t blk = c->host_block_of[static_cast<size_t>(layer) * c->E + exps[i]];
      const hipError_t e = hipMemcpyAsync(c->d_pool + static_cast<int64_t>(slots[i]) * c->eb,
                                          c->host_pool + blk * c->eb, c->eb,
                                          hipMemcpyHostToDevice, cs);
      if (e != hipSuccess) {
        hipStreamSynchronize(cs);
        c->cs.drop_staged(layer);
        c->stage = Stage::kIdle;
        return hip_fail(c, e, "hipMemcpyAsync of a missed expert");
      }
      bytes += c->eb;
    }
    tm.done(OLED_OP_H2D, layer, bytes, 0);
    const hipError_t e = hipEventRecord(c->ev_copy, cs);
    if (e != hipSuccess) {
      hipStreamSynchronize(cs);
      c->cs.drop_staged(layer);
      c->stage = Stage::kIdle;
      return hip_fail(c, e, "hipEventRecord after the miss copies");
    }
    c->copies_outstanding = true;
  }
  int* lc = &c->last_counts[static_cast<size_t>(layer) * 3];
  lc[0] = c->n_active;
  lc[1] = c->n_hits;
  lc[2] = c->n_misses;
  if (out) {
    out->n_active = c->n_active;
    out->n_hits = c->n_hits;
    out->n_misses = c->n_misses;
    out->n_resident = n_res;
    out->rejected_layer = c->rejected_layer;
    out->reserved = 0;
    out->h2d_bytes = bytes;
  }
  c->rejected_layer = -1;
  c->stage = Stage::kApplied;
  return OLED_OK;
}

oled_status moe_forward_cached(void* ctx, int32_t layer, const void* x_dev, void* y_dev, void* stream) {
  Ctx* c = static_cast<Ctx*>(ctx);
  if (!c) return OLED_ERR_INVALID_ARG;
  oled_status st = check_call(c, layer, Stage::kApplied);
  if (st != OLED_OK) return st;
  if (!x_dev || !y_dev) return fail(c, OLED_ERR_INVALID_ARG, "NULL x or y");
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (s != c->cur_stream) return fail(c, OLED_ERR_INVALID_ARG, "stream differs from route_block's");
  HIP_TRY(c, hipSetDevice(c->device));
  SlotTable tab;
  std::memset(&tab, 0xff, sizeof(tab));
  c->cs.launch_slots(layer, tab.slot);
  for (int e = 0; e < c->E; ++e)
    if (c->counts[e] > 0 && (tab.slot[e] < 0 || tab.slot[e] >= c->n_slots))
      return fail(c, OLED_ERR_HIP, "active expert %d has no slot (internal accounting error)", e);
  const bool bf16 = c->dtype == OLED_BF16;
  const int T = c->cur_T;
  const int64_t e13 = static_cast<int64_t>(2) * c->I * c->H * c->esz;
  const int64_t e2 = static_cast<int64_t>(c->H) * c->I * c->esz;
  auto run = [&](int base, int n, int n_exp, int64_t rows) -> oled_status {
    if (n <= 0) return OLED_OK;
    {
      OpTimer tm(c, s);
      HIP_TRY(c, oled::launch_ffn_up(bf16, c->d_pool, c->eb, tab, c->d_items, base, n, x_dev,
                                     c->d_perm, c->K, c->H, c->I, c->d_h, s));
      tm.done(OLED_OP_FFN_UP, layer,
              n_exp * e13 + rows * c->H * c->esz + rows * c->I * c->esz,
              rows * 2 * 2 * static_cast<int64_t>(c->H) * c->I);
    }
    {
      OpTimer tm(c, s);
      HIP_TRY(c, oled::launch_ffn_down(bf16, c->d_pool, c->eb, tab, c->d_items, base, n, c->d_h,
                                       c->H, c->I, c->d_O, s));
      tm.done(OLED_OP_FFN_DOWN, layer, n_exp * e2 + rows * c->I * c->esz + rows * c->H * 4,
              rows * 2 * static_cast<int64_t>(c->H) * c->I);
    }
    return OLED_OK;
  };
  st = run(0, c->n_hit_items, c->n_hits, c->hit_rows);
  if (st != OLED_OK) return st;
  if (c->copies_outstanding) {
    HIP_TRY(c, hipStreamWaitEvent(s, c->ev_copy, 0));
    c->copies_outstanding = false;
  }
  st = run(c->n_hit_items, c->n_miss_items, c->n_misses, c->miss_rows);
  if (st != OLED_OK) return st;
  {
    OpTimer tm(c, s);
    HIP_TRY(c, oled::launch_combine(bf16, c->d_O, c->d_gates, c->d_inv, T, c->K, c->H, y_dev, s));
    tm.done(OLED_OP_COMBINE, layer,
            static_cast<int64_t>(T) * c->K * (c->H * 4 + 8) + static_cast<int64_t>(T) * c->H * c->esz, 0);
  }
  c->stage = Stage::kForwarded;
  return OLED_OK;
}

oled_status score_and_retain(void* ctx, int32_t layer, const float* conf_dev, void* stream) {
  Ctx* c = static_cast<Ctx*>(ctx);
  if (!c) return OLED_ERR_INVALID_ARG;
  if (layer < 0 || layer >= c->L)
    return fail(c, OLED_ERR_INVALID_ARG, "layer %d outside [0,%d)", layer, c->L);
  // the forward pass is optional: the cache state does not depend on outputs
  if ((c->stage != Stage::kApplied && c->stage != Stage::kForwarded) || layer != c->cur_layer)
    return fail(c, OLED_ERR_STATE, "score_and_retain out of order (layer %d)", layer);
  if (!conf_dev) return fail(c, OLED_ERR_INVALID_ARG, "NULL confidence");
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (s != c->cur_stream) return fail(c, OLED_ERR_INVALID_ARG, "stream differs from route_block's");
  HIP_TRY(c, hipSetDevice(c->device));
  if (c->copies_outstanding) {  // later reads of these slots must see the copies
    HIP_TRY(c, hipStreamWaitEvent(s, c->ev_copy, 0));
    c->copies_outstanding = false;
  }
  const ExpertMask res = mask_of(c->cs.resident(layer), c->E);
  const int seq = ++c->seq;
  {
    OpTimer tm(c, s);
    HIP_TRY(c, oled::launch_score_retain(c->d_gates, static_cast<const float*>(conf_dev), c->d_perm,
                                         c->d_offsets, c->d_counts, c->cur_T, c->K, c->E, c->C, res,
                                         c->d_score + static_cast<size_t>(layer) * c->E,
                                         &c->h_ret[layer], seq, s));
    tm.done(OLED_OP_SCORE_RETAIN, layer,
            static_cast<int64_t>(c->cur_T) * c->K * 12 + static_cast<int64_t>(c->cur_T) * 4 +
                static_cast<int64_t>(c->E) * 16,
            0);
  }
  HIP_TRY(c, hipEventRecord(c->ev_retain[layer], s));
  c->pending[layer] = 1;
  c->ret_seq[layer] = seq;
  c->stage = Stage::kIdle;
  c->cur_layer = -1;
  return OLED_OK;
}

oled_status oled_read_layer_state(void* ctx, int32_t layer, oled_layer_state* out) {
  Ctx* c = static_cast<Ctx*>(ctx);
  if (!c || !out) return OLED_ERR_INVALID_ARG;
  if (layer < 0 || layer >= c->L) return fail(c, OLED_ERR_INVALID_ARG, "layer out of range");
  HIP_TRY(c, hipSetDevice(c->device));
  HIP_TRY(c, hipDeviceSynchronize());
  oled_status st = OLED_OK;
  if (c->stage == Stage::kIdle) {
    st = consume_all(c);
    if (st == OLED_ERR_HIP) return st;
  }
  const int T = (c->last_routed_layer == layer) ? c->last_routed_T : 0;
  const size_t R = static_cast<size_t>(T) * c->K;
  out->tokens = T;
  if (T > 0) {
    if (out->topk_idx) HIP_TRY(c, hipMemcpy(out->topk_idx, c->d_topk, R * 4, hipMemcpyDeviceToHost));
    if (out->gates) HIP_TRY(c, hipMemcpy(out->gates, c->d_gates, R * 4, hipMemcpyDeviceToHost));
    if (out->counts) HIP_TRY(c, hipMemcpy(out->counts, c->d_counts, c->E * 4, hipMemcpyDeviceToHost));
    if (out->offsets)
      HIP_TRY(c, hipMemcpy(out->offsets, c->d_offsets, (c->E + 1) * 4, hipMemcpyDeviceToHost));
    if (out->perm) HIP_TRY(c, hipMemcpy(out->perm, c->d_perm, R * 4, hipMemcpyDeviceToHost));
    if (out->inv_perm) HIP_TRY(c, hipMemcpy(out->inv_perm, c->d_inv, R * 4, hipMemcpyDeviceToHost));
  }
  if (out->score_q)
    HIP_TRY(c, hipMemcpy(out->score_q, c->d_score + static_cast<size_t>(layer) * c->E, c->E * 8,
                         hipMemcpyDeviceToHost));
  if (out->resident_before)
    std::memcpy(out->resident_before, &c->res_before[static_cast<size_t>(layer) * c->E], c->E);
  if (out->resident_after) std::memcpy(out->resident_after, c->cs.resident(layer), c->E);
  if (out->slot_of) {
    for (int e = 0; e < c->E; ++e)
      out->slot_of[e] = c->cs.resident(layer)[e] ? c->cs.slot_of(layer)[e] : -1;
  }
  const int* lc = &c->last_counts[static_cast<size_t>(layer) * 3];
  out->n_active = lc[0];
  out->n_hits = lc[1];
  out->n_misses = lc[2];
  if (c->rejected[layer])
    return fail(c, OLED_ERR_INVALID_ARG, "the last retention of layer %d was rejected", layer);
  return OLED_OK;
}

oled_status oled_profile_collect(void* ctx, oled_op_time* out, int32_t cap, int32_t* n_out) {
  Ctx* c = static_cast<Ctx*>(ctx);
  if (!c || !n_out || (cap > 0 && !out)) return OLED_ERR_INVALID_ARG;
  HIP_TRY(c, hipSetDevice(c->device));
  HIP_TRY(c, hipDeviceSynchronize());
  int n = 0;
  for (auto& op : c->ops) {
    float ms = 0.f;
    const hipError_t e = hipEventElapsedTime(&ms, op.a, op.b);
    if (n < cap) {
      out[n].kind = op.kind;
      out[n].layer = op.layer;
      out[n].ms = e == hipSuccess ? ms : -1.f;
      out[n].bytes = op.bytes;
      out[n].flops = op.flops;
      ++n;
    }
    c->ev_free.push_back(op.a);
    c->ev_free.push_back(op.b);
  }
  c->ops.clear();
  *n_out = n;
  return OLED_OK;
}

oled_status oled_host_alloc(int64_t bytes, void** ptr_out) {
  if (!ptr_out) return OLED_ERR_INVALID_ARG;
  *ptr_out = nullptr;
  if (bytes <= 0) return OLED_ERR_INVALID_ARG;
  if (hipHostMalloc(ptr_out, static_cast<size_t>(bytes), hipHostMallocDefault) != hipSuccess) {
    *ptr_out = nullptr;
    return OLED_ERR_OUT_OF_MEMORY;
  }
  return OLED_OK;
}

void oled_host_free(void* ptr) {
  if (ptr) hipHostFree(ptr);
}

}  // extern "C"
