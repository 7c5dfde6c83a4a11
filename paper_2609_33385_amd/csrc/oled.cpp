// Host runtime of the C ABI declared in include/oled.h: the context, the call
// state machine, the per-layer cache bookkeeping, the host-to-device miss
// copies on a side stream and the kernel launches.
//
// Per layer: route_block enqueues the gate kernels; moe_forward_cached
// enqueues the hit experts at once (their work list and count stay on the
// device); apply_misses is the one host synchronisation of the layer - it
// polls the routing summary the permute kernel publishes in coherent pinned
// memory, commits earlier retentions, stages and copies the misses and
// enqueues their GEMMs behind the copies, then the combine; score_and_retain
// enqueues the priority/retention kernel, whose result is committed at the
// next synchronising call.
#include "oled.h"

#include <hip/hip_runtime.h>
#include <immintrin.h>

#include <algorithm>
#include <atomic>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <string>
#include <vector>

#include "cache_state.h"
#include "kernels.h"

namespace {

using oled::ExpertMask;
using oled::FfnLaunch;
using oled::RetainOut;
using oled::RouteSummary;
using oled::SlotTable;
using oled::WorkItem;

thread_local std::string g_create_error;

enum class Stage { kIdle, kRouted, kHitsQueued, kApplied };

struct OpRec {
  int kind, layer;
  int64_t bytes, flops;
  hipEvent_t a, b;
};

struct Ctx {
  // shape
  int H = 0, I = 0, E = 0, K = 0, L = 0, C = 0, Tmax = 0, dtype = 0, esz = 0, device = 0;
  uint32_t profile_ops = 0;
  int64_t eb = 0;    // bytes of one expert block
  int64_t e13 = 0;   // bytes of its w13 part
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
  int32_t* d_item_counts = nullptr;
  int32_t* d_sync = nullptr;       // completion counter + bad-logit flag of the routing launch
  WorkItem* d_items = nullptr;
  void* d_h = nullptr;
  float* d_O = nullptr;
  uint64_t* d_score = nullptr;  // [L][E]
  // coherent pinned host memory written by kernels
  RouteSummary* h_sum = nullptr;
  RetainOut* h_ret = nullptr;   // [L]
  // streams and events
  hipStream_t own_copy = nullptr;
  hipEvent_t ev_up = nullptr, ev_down = nullptr, ev_order = nullptr;
  // cache state
  oled::CacheState cs;
  std::vector<uint8_t> pending;     // [L] retention result not yet committed
  std::vector<int> ret_seq;         // [L] sequence number of that result
  std::vector<hipStream_t> ret_stream;
  std::vector<uint8_t> rejected;    // [L] last retention rejected (bad confidence)
  std::vector<uint8_t> res_before;  // [L][E] R before the layer's last execution
  std::vector<int> last_counts;     // [L][3] n_active, n_hits, n_misses of the last apply
  // the layer in flight
  Stage stage = Stage::kIdle;
  int cur_layer = -1, cur_T = 0, cur_res = 0;
  hipStream_t cur_stream = nullptr;
  bool have_stream = false;
  const void* fwd_x = nullptr;
  void* fwd_y = nullptr;
  int last_routed_layer = -1, last_routed_T = 0;
  std::vector<int32_t> counts;      // [E] route counts of the layer in flight
  std::vector<uint8_t> hit, miss;
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

#define HIP_TRY(c, expr)                                   \
  do {                                                     \
    hipError_t e_ = (expr);                                \
    if (e_ != hipSuccess) return hip_fail((c), e_, #expr); \
  } while (0)

hipEvent_t take_event(Ctx* c) {
  if (!c->ev_free.empty()) {
    hipEvent_t e = c->ev_free.back();
    c->ev_free.pop_back();
    return e;
  }
  // timing only: no system-scope fence, so the event adds no cache flush
  hipEvent_t e = nullptr;
  if (hipEventCreateWithFlags(&e, hipEventDisableSystemFence) != hipSuccess) return nullptr;
  return e;
}

// Timing events of one operation when its kind is profiled (else null).
struct OpEvents {
  hipEvent_t a = nullptr, b = nullptr;
};

OpEvents op_begin(Ctx* c, int kind) {
  OpEvents ev;
  if (!(c->profile_ops & (1u << kind))) return ev;
  ev.a = take_event(c);
  ev.b = take_event(c);
  if (!ev.a || !ev.b) {
    if (ev.a) c->ev_free.push_back(ev.a);
    if (ev.b) c->ev_free.push_back(ev.b);
    return OpEvents{};
  }
  return ev;
}

void op_end(Ctx* c, const OpEvents& ev, int kind, int layer, int64_t bytes, int64_t flops) {
  if (ev.a) c->ops.push_back(OpRec{kind, layer, bytes, flops, ev.a, ev.b});
}

ExpertMask mask_of(const uint8_t* m, int E) {
  ExpertMask x;
  std::memset(&x, 0, sizeof(x));
  for (int e = 0; e < E; ++e)
    if (m[e]) x.bits[e >> 5] |= 1u << (e & 31);
  return x;
}

// Waits until a kernel has published `want` into *flag (coherent pinned
// memory). Checks the stream now and then so a failed launch cannot hang.
oled_status wait_published(Ctx* c, const int32_t* flag, int want, hipStream_t s, const char* what) {
  const volatile int32_t* p = flag;
  for (uint64_t spin = 1;; ++spin) {
    if (*p == want) {
      std::atomic_thread_fence(std::memory_order_acquire);
      return OLED_OK;
    }
    if ((spin & 255) == 0) {
      const hipError_t e = hipStreamQuery(s);
      if (e == hipSuccess) {  // the stream is idle: the value must be visible now
        if (*p == want) {
          std::atomic_thread_fence(std::memory_order_acquire);
          return OLED_OK;
        }
        return fail(c, OLED_ERR_HIP, "%s: result was not published", what);
      }
      if (e != hipErrorNotReady) return hip_fail(c, e, what);
    }
    _mm_pause();
  }
}

// Waits on the host for an event recorded on the copy stream. Launching the
// dependent kernel after the host has seen the copy complete starts it within
// a few microseconds; a GPU-side stream wait on a copy-engine event has been
// measured to add tens of microseconds on this path.
oled_status wait_event_spin(Ctx* c, hipEvent_t ev, const char* what) {
  for (;;) {
    const hipError_t e = hipEventQuery(ev);
    if (e == hipSuccess) return OLED_OK;
    if (e != hipErrorNotReady) return hip_fail(c, e, what);
    _mm_pause();
  }
}

// Commits the retention result of layer l.
oled_status consume_layer(Ctx* c, int l) {
  if (!c->pending[l]) return OLED_OK;
  oled_status st = wait_published(c, &c->h_ret[l].seq, c->ret_seq[l], c->ret_stream[l], "retention");
  c->pending[l] = 0;
  if (st != OLED_OK) {
    c->cs.drop_staged(l);
    return st;
  }
  const RetainOut& o = c->h_ret[l];
  if (o.bad_conf) {
    c->cs.drop_staged(l);
    c->rejected[l] = 1;
    c->rejected_layer = l;
    return fail(c, OLED_ERR_INVALID_ARG, "confidence outside [0,1] at layer %d: retention skipped", l);
  }
  c->rejected[l] = 0;
  uint8_t keep[oled::kMaxExperts];
  for (int e = 0; e < c->E; ++e) keep[e] = (o.retained[e >> 5] >> (e & 31)) & 1u;
  if (!c->cs.commit(l, keep)) {
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
  if (c->ev_up) hipEventDestroy(c->ev_up);
  if (c->ev_down) hipEventDestroy(c->ev_down);
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
  hipFree(c->d_item_counts);
  hipFree(c->d_sync);
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

oled_status check_layer(Ctx* c, int layer) {
  if (layer < 0 || layer >= c->L)
    return fail(c, OLED_ERR_INVALID_ARG, "layer %d outside [0,%d)", layer, c->L);
  return OLED_OK;
}

oled_status check_in_flight(Ctx* c, int layer, hipStream_t s, const char* call) {
  if (layer != c->cur_layer)
    return fail(c, OLED_ERR_STATE, "%s: layer %d is not the layer in flight (%d)", call, layer,
                c->cur_layer);
  if (s != c->cur_stream)
    return fail(c, OLED_ERR_INVALID_ARG, "%s: stream differs from route_block's", call);
  return OLED_OK;
}

FfnLaunch ffn_args(Ctx* c, const SlotTable* tab, int base, int n_host, int max_items) {
  FfnLaunch a;
  a.pool = c->d_pool;
  a.slot_bytes = c->eb;
  a.slots = tab;
  a.items = c->d_items;
  a.n_items_dev = c->d_item_counts;
  a.item_base = base;
  a.n_items_host = n_host;
  a.max_items = max_items;
  a.src = nullptr;
  a.perm = c->d_perm;
  a.k = c->K;
  a.H = c->H;
  a.I = c->I;
  a.hout = c->d_h;
  a.oout = c->d_O;
  return a;
}

int64_t up_bytes(const Ctx* c, int64_t n_exp, int64_t rows) {
  return n_exp * c->e13 + rows * c->H * c->esz + rows * c->I * c->esz;
}
int64_t down_bytes(const Ctx* c, int64_t n_exp, int64_t rows) {
  return n_exp * (c->eb - c->e13) + rows * c->I * c->esz + rows * c->H * 4;
}
int64_t up_flops(const Ctx* c, int64_t rows) { return rows * 4 * static_cast<int64_t>(c->H) * c->I; }
int64_t down_flops(const Ctx* c, int64_t rows) { return rows * 2 * static_cast<int64_t>(c->H) * c->I; }

// Expert block packing (see oled_pack_expert): fragment f holds 16 rows x SPAN
// columns, element l*V + i <- (row 16q + l%16, column SPAN*s + V*(l/16) + i).
template <class T, int SPAN>
void pack_expert_t(int H, int I, const T* w13, const T* w2, T* out) {
  constexpr int V = SPAN / 4;
  constexpr int FRAG = 16 * SPAN;
  const int S = H / SPAN, S2 = I / SPAN;
  for (int q = 0; q < I / 16; ++q)
    for (int s = 0; s < S; ++s)
      for (int m = 0; m < 2; ++m) {
        T* frag = out + (static_cast<size_t>(q * S + s) * 2 + m) * FRAG;
        for (int l = 0; l < 64; ++l)
          for (int i = 0; i < V; ++i) {
            const size_t row = static_cast<size_t>(m) * I + 16 * q + (l & 15);
            frag[l * V + i] = w13[row * H + SPAN * s + V * (l >> 4) + i];
          }
      }
  T* down = out + static_cast<size_t>(2) * I * H;
  for (int q = 0; q < H / 16; ++q)
    for (int s = 0; s < S2; ++s) {
      T* frag = down + static_cast<size_t>(q * S2 + s) * FRAG;
      for (int l = 0; l < 64; ++l)
        for (int i = 0; i < V; ++i) {
          const size_t row = 16 * q + (l & 15);
          frag[l * V + i] = w2[row * I + SPAN * s + V * (l >> 4) + i];
        }
    }
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
  c->profile_ops = static_cast<uint32_t>(cfg->profile_ops);
  c->eb = static_cast<int64_t>(3) * c->H * c->I * c->esz;
  c->e13 = static_cast<int64_t>(2) * c->H * c->I * c->esz;
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
      dev_alloc(&c->d_item_counts, 2) || dev_alloc(&c->d_sync, 2) ||
      dev_alloc(&c->d_items, c->max_items) ||
      dev_alloc(reinterpret_cast<char**>(&c->d_h), routes * c->I * c->esz) ||
      dev_alloc(&c->d_O, routes * c->H) ||
      dev_alloc(&c->d_score, static_cast<size_t>(c->L) * c->E))
    return oom("routing scratch");
  if (hipMemset(c->d_flag, 0, sizeof(int32_t)) != hipSuccess ||
      hipMemset(c->d_item_counts, 0, 2 * sizeof(int32_t)) != hipSuccess ||
      hipMemset(c->d_sync, 0, 2 * sizeof(int32_t)) != hipSuccess ||
      hipMemset(c->d_score, 0, sizeof(uint64_t) * c->L * c->E) != hipSuccess)
    return oom("scratch init");
  if (hipHostMalloc(reinterpret_cast<void**>(&c->h_sum), sizeof(RouteSummary), hipHostMallocCoherent) ||
      hipHostMalloc(reinterpret_cast<void**>(&c->h_ret), sizeof(RetainOut) * c->L, hipHostMallocCoherent))
    return oom("pinned summaries");
  std::memset(c->h_sum, 0, sizeof(RouteSummary));
  std::memset(c->h_ret, 0, sizeof(RetainOut) * c->L);
  if (hipStreamCreateWithFlags(&c->own_copy, hipStreamNonBlocking) != hipSuccess ||
      hipEventCreateWithFlags(&c->ev_up, hipEventDisableTiming) != hipSuccess ||
      hipEventCreateWithFlags(&c->ev_down, hipEventDisableTiming) != hipSuccess ||
      hipEventCreateWithFlags(&c->ev_order, hipEventDisableTiming) != hipSuccess) {
    g_create_error = "stream/event creation failed";
    free_ctx(c);
    return OLED_ERR_HIP;
  }
  c->cs = oled::CacheState(c->L, c->E, c->C, c->n_slots);
  c->pending.assign(c->L, 0);
  c->ret_seq.assign(c->L, 0);
  c->ret_stream.assign(c->L, nullptr);
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
  std::fill(c->pending.begin(), c->pending.end(), 0);
  c->cs.reset();
  std::fill(c->rejected.begin(), c->rejected.end(), 0);
  std::fill(c->res_before.begin(), c->res_before.end(), 0);
  c->rejected_layer = -1;
  return OLED_OK;
}

oled_status route_block(void* ctx, int32_t layer, const float* logits_dev, int32_t T, void* stream) {
  Ctx* c = static_cast<Ctx*>(ctx);
  if (!c) return OLED_ERR_INVALID_ARG;
  oled_status st = check_layer(c, layer);
  if (st != OLED_OK) return st;
  if (c->stage != Stage::kIdle)
    return fail(c, OLED_ERR_STATE, "route_block while layer %d is in flight", c->cur_layer);
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
  const int64_t route_bytes = static_cast<int64_t>(T) * c->E * 4 + static_cast<int64_t>(T) * c->K * 8;
  const int64_t perm_bytes = static_cast<int64_t>(T) * c->K * 12 + static_cast<int64_t>(c->E) * 8;
  if (oled::route_fused(T, c->K)) {
    OpEvents ev = op_begin(c, OLED_OP_ROUTE_TOPK);
    HIP_TRY(c, oled::launch_route_fused(logits_dev, T, c->E, c->K, res, c->d_topk, c->d_gates,
                                        c->d_counts, c->d_offsets, c->d_perm, c->d_inv, c->d_items,
                                        c->d_item_counts, c->d_sync, c->h_sum, seq, ev.a, ev.b, s));
    op_end(c, ev, OLED_OP_ROUTE_TOPK, layer, route_bytes + perm_bytes, 0);
  } else {
    {
      OpEvents ev = op_begin(c, OLED_OP_ROUTE_TOPK);
      HIP_TRY(c, oled::launch_route_topk(logits_dev, T, c->E, c->K, c->d_topk, c->d_gates,
                                         c->d_flag, ev.a, ev.b, s));
      op_end(c, ev, OLED_OP_ROUTE_TOPK, layer, route_bytes, 0);
    }
    OpEvents ev = op_begin(c, OLED_OP_PERMUTE);
    HIP_TRY(c, oled::launch_permute(c->d_topk, T, c->K, c->E, res, c->d_counts, c->d_offsets,
                                    c->d_perm, c->d_inv, c->d_items, c->d_item_counts, c->d_flag,
                                    c->h_sum, seq, ev.a, ev.b, s));
    op_end(c, ev, OLED_OP_PERMUTE, layer, perm_bytes, 0);
  }
  c->route_seq = seq;
  c->stage = Stage::kRouted;
  c->cur_layer = layer;
  c->cur_T = T;
  c->cur_res = c->cs.resident_count(layer);
  c->cur_stream = s;
  c->have_stream = true;
  c->fwd_x = nullptr;
  c->fwd_y = nullptr;
  c->last_routed_layer = layer;
  c->last_routed_T = T;
  return OLED_OK;
}

oled_status moe_forward_cached(void* ctx, int32_t layer, const void* x_dev, void* y_dev, void* stream) {
  Ctx* c = static_cast<Ctx*>(ctx);
  if (!c) return OLED_ERR_INVALID_ARG;
  oled_status st = check_layer(c, layer);
  if (st != OLED_OK) return st;
  if (c->stage != Stage::kRouted)
    return fail(c, OLED_ERR_STATE, "moe_forward_cached must follow route_block");
  hipStream_t s = static_cast<hipStream_t>(stream);
  st = check_in_flight(c, layer, s, "moe_forward_cached");
  if (st != OLED_OK) return st;
  if (!x_dev || !y_dev) return fail(c, OLED_ERR_INVALID_ARG, "NULL x or y");
  HIP_TRY(c, hipSetDevice(c->device));
  if (c->cur_res > 0) {
    // hits: the active residents; the item count stays on the device, the
    // byte and flop accounting is completed in apply_misses
    SlotTable tab;
    std::memset(&tab, 0xff, sizeof(tab));
    c->cs.launch_slots(layer, tab.slot);
    const int64_t routes = static_cast<int64_t>(c->cur_T) * c->K;
    const int max_hit_items =
        static_cast<int>(std::min<int64_t>(c->cur_res, routes) + routes / oled::kItemRows);
    const bool bf16 = c->dtype == OLED_BF16;
    FfnLaunch a = ffn_args(c, &tab, 0, -1, max_hit_items);
    a.src = x_dev;
    {
      OpEvents ev = op_begin(c, OLED_OP_FFN_UP);
      HIP_TRY(c, oled::launch_ffn_up(bf16, a, ev.a, ev.b, s));
      op_end(c, ev, OLED_OP_FFN_UP, layer, -1, -1);
    }
    a.src = c->d_h;
    {
      OpEvents ev = op_begin(c, OLED_OP_FFN_DOWN);
      HIP_TRY(c, oled::launch_ffn_down(bf16, a, ev.a, ev.b, s));
      op_end(c, ev, OLED_OP_FFN_DOWN, layer, -1, -1);
    }
  }
  c->fwd_x = x_dev;
  c->fwd_y = y_dev;
  c->stage = Stage::kHitsQueued;
  return OLED_OK;
}

oled_status apply_misses(void* ctx, int32_t layer, void* copy_stream, oled_miss_report* out) {
  Ctx* c = static_cast<Ctx*>(ctx);
  if (!c) return OLED_ERR_INVALID_ARG;
  oled_status st = check_layer(c, layer);
  if (st != OLED_OK) return st;
  if (c->stage != Stage::kRouted && c->stage != Stage::kHitsQueued)
    return fail(c, OLED_ERR_STATE, "apply_misses must follow route_block or moe_forward_cached");
  if (layer != c->cur_layer)
    return fail(c, OLED_ERR_STATE, "apply_misses: layer %d is not the layer in flight (%d)", layer,
                c->cur_layer);
  HIP_TRY(c, hipSetDevice(c->device));
  st = wait_published(c, &c->h_sum->seq, c->route_seq, c->cur_stream, "routing summary");
  if (st != OLED_OK) {
    c->stage = Stage::kIdle;
    return st;
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
  int n_active = 0, n_hits = 0, n_misses = 0;
  c->cs.classify(layer, c->counts.data(), c->hit.data(), c->miss.data(), &n_active, &n_hits,
                 &n_misses);
  int nhi = 0, nmi = 0;
  int64_t hit_rows = 0, miss_rows = 0;
  for (int e = 0; e < c->E; ++e) {
    const int ni = (c->counts[e] + oled::kItemRows - 1) / oled::kItemRows;
    if (c->hit[e]) {
      nhi += ni;
      hit_rows += c->counts[e];
    }
    if (c->miss[e]) {
      nmi += ni;
      miss_rows += c->counts[e];
    }
  }
  if (nhi != c->h_sum->n_hit_items || nmi != c->h_sum->n_miss_items) {
    c->stage = Stage::kIdle;
    return fail(c, OLED_ERR_HIP, "work list disagrees with the host cache state");
  }
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
    // gate/up weights of every miss first, then the down weights, so the miss
    // gate/up GEMM can run while the down weights are still in flight
    OpEvents ev = op_begin(c, OLED_OP_H2D);
    hipError_t e = hipSuccess;
    if (ev.a) e = hipEventRecord(ev.a, cs);
    for (int part = 0; part < 2 && e == hipSuccess; ++part) {
      const int64_t off = part == 0 ? 0 : c->e13;
      const int64_t len = part == 0 ? c->e13 : c->eb - c->e13;
      for (size_t i = 0; i < exps.size() && e == hipSuccess; ++i) {
        const int64_t blk = c->host_block_of[static_cast<size_t>(layer) * c->E + exps[i]];
        e = hipMemcpyAsync(c->d_pool + static_cast<int64_t>(slots[i]) * c->eb + off,
                           c->host_pool + blk * c->eb + off, len, hipMemcpyHostToDevice, cs);
        bytes += len;
      }
      if (e == hipSuccess) e = hipEventRecord(part == 0 ? c->ev_up : c->ev_down, cs);
    }
    if (e == hipSuccess && ev.b) e = hipEventRecord(ev.b, cs);
    if (e != hipSuccess) {
      hipStreamSynchronize(cs);
      c->cs.drop_staged(layer);
      c->stage = Stage::kIdle;
      if (ev.a) c->ev_free.push_back(ev.a);
      if (ev.b) c->ev_free.push_back(ev.b);
      return hip_fail(c, e, "enqueueing the miss copies");
    }
    op_end(c, ev, OLED_OP_H2D, layer, bytes, 0);
    c->copies_outstanding = true;
  }
  // complete the accounting of this layer's hit launches
  for (auto it = c->ops.rbegin(); it != c->ops.rend() && it->layer == layer; ++it) {
    if (it->kind == OLED_OP_FFN_UP && it->bytes < 0) {
      it->bytes = up_bytes(c, n_hits, hit_rows);
      it->flops = up_flops(c, hit_rows);
    } else if (it->kind == OLED_OP_FFN_DOWN && it->bytes < 0) {
      it->bytes = down_bytes(c, n_hits, hit_rows);
      it->flops = down_flops(c, hit_rows);
    }
  }
  if (c->stage == Stage::kHitsQueued) {
    hipStream_t s = c->cur_stream;
    const bool bf16 = c->dtype == OLED_BF16;
    if (nmi > 0) {
      SlotTable tab;
      std::memset(&tab, 0xff, sizeof(tab));
      c->cs.launch_slots(layer, tab.slot);
      for (int e = 0; e < c->E; ++e)
        if (c->miss[e] && (tab.slot[e] < 0 || tab.slot[e] >= c->n_slots))
          return fail(c, OLED_ERR_HIP, "missed expert %d has no slot (internal accounting error)", e);
      FfnLaunch a = ffn_args(c, &tab, nhi, nmi, nmi);
      a.src = c->fwd_x;
      st = wait_event_spin(c, c->ev_up, "gate/up weight copies");
      if (st != OLED_OK) return st;
      {
        OpEvents ev = op_begin(c, OLED_OP_FFN_UP);
        HIP_TRY(c, oled::launch_ffn_up(bf16, a, ev.a, ev.b, s));
        op_end(c, ev, OLED_OP_FFN_UP, layer, up_bytes(c, n_misses, miss_rows), up_flops(c, miss_rows));
      }
      a.src = c->d_h;
      st = wait_event_spin(c, c->ev_down, "down weight copies");
      if (st != OLED_OK) return st;
      c->copies_outstanding = false;
      {
        OpEvents ev = op_begin(c, OLED_OP_FFN_DOWN);
        HIP_TRY(c, oled::launch_ffn_down(bf16, a, ev.a, ev.b, s));
        op_end(c, ev, OLED_OP_FFN_DOWN, layer, down_bytes(c, n_misses, miss_rows),
               down_flops(c, miss_rows));
      }
    }
    {
      OpEvents ev = op_begin(c, OLED_OP_COMBINE);
      const int T = c->cur_T;
      HIP_TRY(c, oled::launch_combine(bf16, c->d_O, c->d_gates, c->d_inv, T, c->K, c->H, c->fwd_y,
                                      ev.a, ev.b, s));
      op_end(c, ev, OLED_OP_COMBINE, layer,
             static_cast<int64_t>(T) * c->K * (c->H * 4 + 8) + static_cast<int64_t>(T) * c->H * c->esz,
             0);
    }
  }
  int* lc = &c->last_counts[static_cast<size_t>(layer) * 3];
  lc[0] = n_active;
  lc[1] = n_hits;
  lc[2] = n_misses;
  if (out) {
    out->n_active = n_active;
    out->n_hits = n_hits;
    out->n_misses = n_misses;
    out->n_resident = n_res;
    out->rejected_layer = c->rejected_layer;
    out->reserved = 0;
    out->h2d_bytes = bytes;
  }
  c->rejected_layer = -1;
  c->stage = Stage::kApplied;
  return OLED_OK;
}

oled_status score_and_retain(void* ctx, int32_t layer, const float* conf_dev, void* stream) {
  Ctx* c = static_cast<Ctx*>(ctx);
  if (!c) return OLED_ERR_INVALID_ARG;
  oled_status st = check_layer(c, layer);
  if (st != OLED_OK) return st;
  if (c->stage != Stage::kApplied)
    return fail(c, OLED_ERR_STATE, "score_and_retain must follow apply_misses");
  hipStream_t s = static_cast<hipStream_t>(stream);
  st = check_in_flight(c, layer, s, "score_and_retain");
  if (st != OLED_OK) return st;
  if (!conf_dev) return fail(c, OLED_ERR_INVALID_ARG, "NULL confidence");
  HIP_TRY(c, hipSetDevice(c->device));
  if (c->copies_outstanding) {  // later reads of these slots must see the copies
    HIP_TRY(c, hipStreamWaitEvent(s, c->ev_down, 0));
    c->copies_outstanding = false;
  }
  const ExpertMask res = mask_of(c->cs.resident(layer), c->E);
  const int seq = ++c->seq;
  {
    OpEvents ev = op_begin(c, OLED_OP_SCORE_RETAIN);
    HIP_TRY(c, oled::launch_score_retain(c->d_gates, static_cast<const float*>(conf_dev),
                                         c->d_topk, c->d_counts, c->cur_T, c->K, c->E, c->C, res,
                                         c->d_score + static_cast<size_t>(layer) * c->E,
                                         &c->h_ret[layer], seq, ev.a, ev.b, s));
    op_end(c, ev, OLED_OP_SCORE_RETAIN, layer,
           static_cast<int64_t>(c->cur_T) * c->K * 12 + static_cast<int64_t>(c->cur_T) * 4 +
               static_cast<int64_t>(c->E) * 16,
           0);
  }
  c->pending[layer] = 1;
  c->ret_seq[layer] = seq;
  c->ret_stream[layer] = s;
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
  if (c->stage == Stage::kIdle) {
    const oled_status st = consume_all(c);
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

oled_status oled_pack_expert(int32_t dtype, int32_t hidden, int32_t inter, const void* w13,
                             const void* w2, void* block_out) {
  if (!w13 || !w2 || !block_out) return OLED_ERR_INVALID_ARG;
  if (dtype != OLED_F32 && dtype != OLED_BF16) return OLED_ERR_INVALID_ARG;
  if (hidden <= 0 || inter <= 0 || hidden % 128 || inter % 128) return OLED_ERR_UNSUPPORTED;
  if (dtype == OLED_BF16)
    pack_expert_t<uint16_t, 32>(hidden, inter, static_cast<const uint16_t*>(w13),
                                static_cast<const uint16_t*>(w2), static_cast<uint16_t*>(block_out));
  else
    pack_expert_t<uint32_t, 16>(hidden, inter, static_cast<const uint32_t*>(w13),
                                static_cast<const uint32_t*>(w2), static_cast<uint32_t*>(block_out));
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
