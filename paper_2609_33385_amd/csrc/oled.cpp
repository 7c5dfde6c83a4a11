// Host runtime of the C ABI declared in include/oled.h: the context, the call
// state machine, the device-resident cache state, the transfer of the misses
// and the kernel launches.
//
// The cache state of every layer (resident sets, slot tables, the free-slot
// list, the staged misses of the layer in flight) lives in device memory and
// only kernels change it: the routing kernel stages the misses into free
// slots, the retention kernel commits. With the default shader transfer a
// layer needs no host synchronisation at all: route_block enqueues the
// routing kernel; moe_forward_cached the hit experts' gate/up GEMM, whose
// first workgroups copy the staged misses' gate/up weights from the pinned
// host pool over PCIe meanwhile; apply_misses one launch with the hit
// experts' down GEMM, the copy of the misses' down weights and the misses'
// gate/up GEMM, then the misses' down GEMM; score_and_retain one launch with
// the combine and the priority / retention / commit. The host reads the
// pinned routing records only when a caller asks for counts.
//
// With the copy-engine transfer (OLED_COPY_SDMA) apply_misses waits for the
// routing record, copies the staged misses with hipMemcpyAsync on a side
// stream and launches their GEMMs once the host has seen the copies land.
#include "oled.h"

#include <hip/hip_runtime.h>
#include <immintrin.h>

#include <algorithm>
#include <atomic>
#include <chrono>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <map>
#include <memory>
#include <mutex>
#include <string>
#include <vector>

#include "cpu_ffn.h"
#include "kernels.h"

namespace {

using oled::CacheHdr;
using oled::CacheView;
using oled::ExpertMask;
using oled::FetchArgs;
using oled::FfnLaunch;
using oled::LayerStat;
using oled::PermuteOut;
using oled::RetainOut;
using oled::RouteStats;
using oled::StagedList;
using oled::WorkItem;

thread_local std::string g_create_error;

constexpr int kFetchBlocks = 64;    // workgroups of a launch that copy misses (multiple of 8)
constexpr int kMissGridCap = 256;   // GEMM workgroups of a miss launch (they loop over tiles)

enum class Stage { kIdle, kRouted, kHitsQueued, kApplied };

struct OpRec {
  int kind, layer;
  int route_seq;          // routing record that completes the accounting (0: complete)
  int part;               // 0 gate/up, 1 down, 2 hit down + miss gate/up, 3 dense gate/up,
                          // 4 dense down, -1 other
  bool hits;              // hit-expert launch (else miss launch)
  int64_t bytes, flops, h2d;
  hipEvent_t a, b;
};

constexpr int64_t kDefaultWaitDeadlineMs = 60000;

struct Ctx {
  // shape
  int H = 0, I = 0, E = 0, K = 0, L = 0, C = 0, Tmax = 0, dtype = 0, esz = 0, device = 0;
  int copy_mode = OLED_COPY_SHADER;
  int adapt_period = 0;    // layer-adaptive sizing after every adapt_period-th iteration (0: off)
  int policy = OLED_POLICY_PRIORITY;
  int64_t iters_done = 0;  // iterations of the whole stack completed since the last reset
  uint32_t profile_ops = 0;
  int64_t eb = 0;    // bytes of one expert block
  int64_t e13 = 0;   // bytes of its gate/up part
  int n_slots = 0;
  int cap = 0;       // min(C, E)
  int max_items = 0;
  bool dense_ok = false;  // shapes the dense-tile GEMM takes (bf16, H and I multiples of 256)
  int max_dense = 0;
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
  int32_t* d_sync = nullptr;       // completion counter + bad-logit flag of the fused routing
  int32_t* d_chunk = nullptr;      // [Tmax/512 chunks][E] per-chunk counts / bases (large blocks)
  float* d_logits = nullptr;       // [Tmax][E] logits of route_block_gate's gate GEMM
  int logits_layer = -1;           // the layer they belong to (-1: none)
  unsigned long long* d_sacc = nullptr;  // [E] priority numerators of a many-part scoring
  int32_t* d_ssync = nullptr;      // [2] its completion counter and bad-confidence flag
  WorkItem* d_items = nullptr;
  WorkItem* d_dense_items = nullptr;
  int32_t* d_dense_counts = nullptr;
  void* d_h = nullptr;
  float* d_O = nullptr;
  uint64_t* d_score = nullptr;     // [L][E]
  // device-resident cache state
  CacheHdr* d_hdr = nullptr;
  int32_t* d_slot_of = nullptr;    // [L][E]
  ExpertMask* d_res = nullptr;     // [L]
  ExpertMask* d_res_before = nullptr;
  int32_t* d_last_counts = nullptr;  // [L][kCountsPerLayer]
  int32_t* d_iters = nullptr;      // [L] iterations of each layer (LRU / LFU history)
  int32_t* d_last_use = nullptr;   // [L][E]
  uint64_t* d_freq = nullptr;      // [L][E]
  ExpertMask* d_prev_miss = nullptr;  // [L]
  uint64_t* d_key = nullptr;       // [L][E] keys of each layer's last retention
  int32_t* d_free = nullptr;       // [n_slots]
  int32_t* d_cap = nullptr;        // [L] capacity of each layer
  LayerStat* d_stat = nullptr;     // [L] smoothed statistics of the adaptive sizing
  uint64_t* d_host_addr = nullptr; // [L][E]
  // records written by kernels: device memory, copied out at synchronisation
  // points into pinned mirrors; the staged list for host-issued copies is
  // published straight into coherent pinned memory
  RouteStats* d_ring = nullptr;    // [kStatsRing]
  RetainOut* d_ret = nullptr;      // [L]
  RouteStats* h_ring = nullptr;    // [kStatsRing] pinned mirror
  RetainOut* h_ret = nullptr;      // [L] pinned mirror
  StagedList* h_staged = nullptr;
  // streams and events
  hipStream_t own_copy = nullptr;
  hipEvent_t ev_up = nullptr, ev_down = nullptr, ev_order = nullptr;
  // routing records consumed by the host
  int route_n = 0;                 // sequence number of the last routing call
  int next_stat = 1;               // first record not yet consumed
  std::vector<RouteStats> recs;    // consumed records kept for the profile accounting
  oled_stats acc{};                // accumulated since the last oled_collect_stats
  int bad_route_layer = -1;        // a bad block seen in a record, not yet reported
  int reported_bad_route = 0;      // routing call whose bad block apply_misses reported
  // retention results
  int seq = 0;
  std::vector<int> ret_seq;        // [L] sequence number of the last retention (0: none)
  std::vector<uint8_t> ret_seen;   // [L] that result has been read
  std::vector<uint8_t> rejected;   // [L] the last retention read was rejected
  int rejected_layer = -1;         // reported by the next report
  // the layer in flight
  Stage stage = Stage::kIdle;
  int cur_layer = -1, cur_T = 0, cur_route = 0;
  bool cur_dense = false;          // the layer in flight has dense items
  hipStream_t cur_stream = nullptr;
  bool have_stream = false;
  const void* fwd_x = nullptr;
  void* fwd_y = nullptr;
  int last_routed_layer = -1, last_routed_T = 0;
  bool copies_outstanding = false;
  bool broken = false;             // a HIP failure left the device state unknown
  // host waits give up after this long (oled_set_fault_injection may shorten it)
  int64_t wait_deadline_ms = kDefaultWaitDeadlineMs;
  int copy_fail_at = 0;            // injection: the n-th miss copy enqueue from now fails
  int copy_count = 0;
  std::string err;
  // profiling
  std::vector<OpRec> ops;
  std::vector<hipEvent_t> ev_free;
  // cooperative compensation (coop contexts)
  bool coop = false;
  double coop_t = 0.0, coop_tau = 0.0, coop_nbar = 0.0, coop_lambda = 0.0;
  std::unique_ptr<oled::ThreadPool> pool;
  std::vector<float> cpu_scratch;
  ExpertMask* d_cpu = nullptr;     // [L] CPU-executed misses of the layer in flight
  int32_t* h_ctopk = nullptr;      // pinned copies of the layer's routing, confidence, x
  float* h_cgates = nullptr;
  float* h_cconf = nullptr;
  char* h_cx = nullptr;
  float* h_cout[2] = {nullptr, nullptr};  // CPU expert outputs, alternating per layer
  hipEvent_t ev_cout[2] = {nullptr, nullptr};
  bool cout_used[2] = {false, false};
  int cout_buf = 0;
  hipEvent_t ev_coop = nullptr;    // the confidence copy
  hipEvent_t ev_x = nullptr;       // the copy of x to the host
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
  c->broken = true;
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

void op_end(Ctx* c, const OpEvents& ev, OpRec r) {
  if (!ev.a) return;
  r.a = ev.a;
  r.b = ev.b;
  c->ops.push_back(r);
}

OpRec rec(int kind, int layer, int64_t bytes, int64_t flops = 0) {
  OpRec r{};
  r.kind = kind;
  r.layer = layer;
  r.part = -1;
  r.bytes = bytes;
  r.flops = flops;
  return r;
}

bool past_deadline(const Ctx* c, std::chrono::steady_clock::time_point t0) {
  return std::chrono::steady_clock::now() - t0 > std::chrono::milliseconds(c->wait_deadline_ms);
}

// Spins until a kernel has published `want` into *flag (coherent pinned
// memory). Checks the stream now and then so a failed launch cannot hang.
oled_status wait_published(Ctx* c, const int32_t* flag, int want, hipStream_t s, const char* what) {
  const volatile int32_t* p = flag;
  const auto t0 = std::chrono::steady_clock::now();
  for (uint64_t spin = 1;; ++spin) {
    if (*p == want) {
      std::atomic_thread_fence(std::memory_order_acquire);
      return OLED_OK;
    }
    if ((spin & 255) == 0) {
      if (past_deadline(c, t0)) {
        c->broken = true;
        return fail(c, OLED_ERR_HIP, "%s: not published within %lld ms", what,
                    static_cast<long long>(c->wait_deadline_ms));
      }
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
  const auto t0 = std::chrono::steady_clock::now();
  for (uint64_t spin = 1;; ++spin) {
    const hipError_t e = hipEventQuery(ev);
    if (e == hipSuccess) return OLED_OK;
    if (e != hipErrorNotReady) return hip_fail(c, e, what);
    if ((spin & 63) == 0 && past_deadline(c, t0)) {   // copies still in flight: state unknown
      c->broken = true;
      return fail(c, OLED_ERR_HIP, "%s: not complete within %lld ms", what,
                  static_cast<long long>(c->wait_deadline_ms));
    }
    _mm_pause();
  }
}

// Copies the routing records up to `until` and every layer's retention
// result out of device memory (one synchronisation of the compute stream,
// skipped when there is nothing new to read) and consumes the records in
// order.
oled_status drain_records(Ctx* c, int until, bool retentions = true) {
  if (until > c->route_n) until = c->route_n;
  bool pending_ret = false;
  for (int l = 0; retentions && l < c->L; ++l) pending_ret |= c->ret_seq[l] != 0 && !c->ret_seen[l];
  if ((c->next_stat > until && !pending_ret) || !c->have_stream) return OLED_OK;
  hipStream_t s = c->cur_stream;
  const int first = c->next_stat;
  const int n = until >= first ? until - first + 1 : 0;
  int idx = first % oled::kStatsRing;
  int left = n;
  while (left > 0) {
    const int len = std::min(left, oled::kStatsRing - idx);
    HIP_TRY(c, hipMemcpyAsync(c->h_ring + idx, c->d_ring + idx, sizeof(RouteStats) * len,
                              hipMemcpyDeviceToHost, s));
    left -= len;
    idx = 0;
  }
  HIP_TRY(c, hipMemcpyAsync(c->h_ret, c->d_ret, sizeof(RetainOut) * c->L, hipMemcpyDeviceToHost, s));
  HIP_TRY(c, hipStreamSynchronize(s));
  for (int q = first; q <= until; ++q) {
    const RouteStats& v = c->h_ring[q % oled::kStatsRing];
    if (v.seq != q) return fail(c, OLED_ERR_HIP, "routing record %d missing (found %d)", q, v.seq);
    c->acc.layer_iters += 1;
    c->acc.n_active += v.n_active;
    c->acc.n_hits += v.n_hits;
    c->acc.n_misses += v.n_misses;
    c->acc.n_transferred += v.n_staged;
    c->acc.h2d_bytes += static_cast<int64_t>(v.n_staged) * c->eb;
    c->acc.n_prev_transferred += v.prev_xfer;
    c->acc.n_transfers_reused += v.reused_xfer;
    c->acc.n_ideal_hits += v.ideal_hits;
    c->acc.n_miss_rows += v.miss_rows;
    if (v.bad) {
      c->acc.n_bad_blocks += 1;
      if (v.seq != c->reported_bad_route) c->bad_route_layer = v.layer;
    }
    if (c->profile_ops) c->recs.push_back(v);
  }
  if (n > 0) c->next_stat = until + 1;
  // retentions: every one enqueued before the last consumed routing has run
  for (int l = 0; l < c->L; ++l) {
    if (c->ret_seq[l] == 0 || c->ret_seen[l] || c->h_ret[l].seq != c->ret_seq[l]) continue;
    c->ret_seen[l] = 1;
    if (c->h_ret[l].bad_conf) {
      c->rejected[l] = 1;
      c->rejected_layer = l;
    } else {
      c->rejected[l] = 0;
    }
  }
  return OLED_OK;
}

const RouteStats* find_record(const Ctx* c, int seq) {
  for (auto it = c->recs.rbegin(); it != c->recs.rend(); ++it)
    if (it->seq == seq) return &*it;
  return nullptr;
}

void free_ctx(Ctx* c) {
  if (!c) return;
  (void)hipSetDevice(c->device);
  (void)hipDeviceSynchronize();
  for (auto& op : c->ops) {
    (void)hipEventDestroy(op.a);
    (void)hipEventDestroy(op.b);
  }
  for (auto e : c->ev_free) (void)hipEventDestroy(e);
  if (c->ev_up) (void)hipEventDestroy(c->ev_up);
  if (c->ev_down) (void)hipEventDestroy(c->ev_down);
  if (c->ev_order) (void)hipEventDestroy(c->ev_order);
  if (c->ev_coop) (void)hipEventDestroy(c->ev_coop);
  if (c->ev_x) (void)hipEventDestroy(c->ev_x);
  for (int b = 0; b < 2; ++b) {
    if (c->ev_cout[b]) (void)hipEventDestroy(c->ev_cout[b]);
    if (c->h_cout[b]) (void)hipHostFree(c->h_cout[b]);
  }
  void* pinned[] = {c->h_ctopk, c->h_cgates, c->h_cconf, c->h_cx};
  for (void* p : pinned)
    if (p) (void)hipHostFree(p);
  if (c->d_cpu) (void)hipFree(c->d_cpu);
  c->pool.reset();
  if (c->own_copy) (void)hipStreamDestroy(c->own_copy);
  void* dev[] = {c->d_pool, c->d_topk, c->d_gates, c->d_counts, c->d_offsets, c->d_perm,
                 c->d_inv, c->d_flag, c->d_item_counts, c->d_sync, c->d_items, c->d_dense_items,
                 c->d_dense_counts, c->d_h, c->d_O,
                 c->d_score, c->d_hdr, c->d_slot_of, c->d_res, c->d_res_before,
                 c->d_last_counts, c->d_free, c->d_host_addr, c->d_cap, c->d_stat,
                 c->d_chunk, c->d_sacc, c->d_ssync, c->d_iters, c->d_last_use,
                 c->d_logits,
                 c->d_freq, c->d_prev_miss, c->d_key};
  for (void* p : dev)
    if (p) (void)hipFree(p);
  if (c->h_ring) (void)hipHostFree(c->h_ring);
  if (c->h_staged) (void)hipHostFree(c->h_staged);
  if (c->h_ret) (void)hipHostFree(c->h_ret);
  if (c->d_ring) (void)hipFree(c->d_ring);
  if (c->d_ret) (void)hipFree(c->d_ret);
  delete c;
}

template <class T>
hipError_t dev_alloc(T** p, size_t n) {
  return hipMalloc(reinterpret_cast<void**>(p), n * sizeof(T) > 0 ? n * sizeof(T) : 16);
}

// Empty caches: every slot free, no expert resident or staged.
oled_status init_cache_state(Ctx* c) {
  CacheHdr hdr;
  std::memset(&hdr, 0, sizeof(hdr));
  hdr.free_top = c->n_slots;
  std::vector<int32_t> free_list(c->n_slots);
  for (int i = 0; i < c->n_slots; ++i) free_list[i] = c->n_slots - 1 - i;  // slot 0 taken first
  std::vector<int32_t> slots(static_cast<size_t>(c->L) * c->E, -1);
  HIP_TRY(c, hipMemcpy(c->d_hdr, &hdr, sizeof(hdr), hipMemcpyHostToDevice));
  HIP_TRY(c, hipMemcpy(c->d_free, free_list.data(), sizeof(int32_t) * c->n_slots,
                       hipMemcpyHostToDevice));
  HIP_TRY(c, hipMemcpy(c->d_slot_of, slots.data(), sizeof(int32_t) * slots.size(),
                       hipMemcpyHostToDevice));
  HIP_TRY(c, hipMemset(c->d_res, 0, sizeof(ExpertMask) * c->L));
  HIP_TRY(c, hipMemset(c->d_res_before, 0, sizeof(ExpertMask) * c->L));
  HIP_TRY(c, hipMemset(c->d_last_counts, 0, sizeof(int32_t) * oled::kCountsPerLayer * c->L));
  HIP_TRY(c, hipMemset(c->d_iters, 0, sizeof(int32_t) * c->L));
  HIP_TRY(c, hipMemset(c->d_last_use, 0, sizeof(int32_t) * c->L * c->E));
  HIP_TRY(c, hipMemset(c->d_freq, 0, sizeof(uint64_t) * c->L * c->E));
  HIP_TRY(c, hipMemset(c->d_prev_miss, 0, sizeof(ExpertMask) * c->L));
  HIP_TRY(c, hipMemset(c->d_key, 0, sizeof(uint64_t) * c->L * c->E));
  if (c->d_cpu) HIP_TRY(c, hipMemset(c->d_cpu, 0, sizeof(ExpertMask) * c->L));
  HIP_TRY(c, hipMemset(c->d_score, 0, sizeof(uint64_t) * c->L * c->E));
  std::vector<int32_t> caps(c->L, c->cap);
  HIP_TRY(c, hipMemcpy(c->d_cap, caps.data(), sizeof(int32_t) * c->L, hipMemcpyHostToDevice));
  HIP_TRY(c, hipMemset(c->d_stat, 0, sizeof(LayerStat) * c->L));
  // counters and accumulators that kernels leave at zero
  HIP_TRY(c, hipMemset(c->d_flag, 0, sizeof(int32_t)));
  HIP_TRY(c, hipMemset(c->d_sync, 0, 2 * sizeof(int32_t)));
  HIP_TRY(c, hipMemset(c->d_sacc, 0, sizeof(unsigned long long) * c->E));
  HIP_TRY(c, hipMemset(c->d_ssync, 0, 2 * sizeof(int32_t)));
  HIP_TRY(c, hipDeviceSynchronize());
  c->iters_done = 0;
  return OLED_OK;
}

CacheView view(const Ctx* c) {
  CacheView v;
  v.hdr = c->d_hdr;
  v.slot_of = c->d_slot_of;
  v.res = c->d_res;
  v.res_before = c->d_res_before;
  v.last_counts = c->d_last_counts;
  v.free_list = c->d_free;
  v.cap = c->d_cap;
  v.stat = c->d_stat;
  v.adapt = c->adapt_period > 0;
  v.policy = c->policy;
  v.iters = c->d_iters;
  v.last_use = c->d_last_use;
  v.freq = c->d_freq;
  v.prev_miss = c->d_prev_miss;
  v.cpu_exec = c->d_cpu;
  v.n_slots = c->n_slots;
  return v;
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

FfnLaunch ffn_args(Ctx* c, int layer, int which, int max_items, int max_grid) {
  FfnLaunch a;
  std::memset(&a, 0, sizeof(a));
  a.pool = c->d_pool;
  a.slot_bytes = c->eb;
  a.slot_of = c->d_slot_of + static_cast<size_t>(layer) * c->E;
  a.n_slots = c->n_slots;
  a.items = c->d_items;
  a.item_counts = c->d_item_counts;
  a.which = which;
  a.item_base = 0;
  a.n_items_host = -1;
  a.max_items = max_items;
  a.max_grid = max_grid;
  a.perm = c->d_perm;
  a.k = c->K;
  a.H = c->H;
  a.I = c->I;
  a.hout = c->d_h;
  a.oout = c->d_O;
  a.fetch.host_addr = c->d_host_addr + static_cast<size_t>(layer) * c->E;
  a.fetch.hdr = c->d_hdr;
  a.fetch.nblk = 0;
  a.fetch.E = c->E;
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

// Experts and rows of the streaming launches (the dense experts excluded).
struct Part {
  int64_t n, rows;
};
Part streamed(const RouteStats& r, bool hits) {
  if (hits) return {r.n_hits - r.n_dense_hits, r.hit_rows - r.dense_hit_rows};
  return {r.n_misses - (r.n_dense - r.n_dense_hits), r.miss_rows - (r.dense_rows - r.dense_hit_rows)};
}

// Completes the byte / flop accounting of a launch from its routing record.
void complete_op(const Ctx* c, OpRec& op, const RouteStats& r) {
  if (op.kind == OLED_OP_H2D) {  // transfer-only launch (no GEMM tiles)
    op.bytes = static_cast<int64_t>(r.n_staged) * c->eb;
    op.h2d = op.bytes;
    op.flops = 0;
    return;
  }
  if (op.part == 2) {
    const Part h = streamed(r, true), m = streamed(r, false);
    op.bytes = down_bytes(c, h.n, h.rows) + up_bytes(c, m.n, m.rows);
    op.flops = down_flops(c, h.rows) + up_flops(c, m.rows);
    if (op.h2d < 0) op.h2d = static_cast<int64_t>(r.n_staged) * (c->eb - c->e13);
    return;
  }
  if (op.part == 3 || op.part == 4) {  // dense tiles
    const bool up = op.part == 3;
    op.bytes = up ? up_bytes(c, r.n_dense, r.dense_rows) : down_bytes(c, r.n_dense, r.dense_rows);
    op.flops = up ? up_flops(c, r.dense_rows) : down_flops(c, r.dense_rows);
    op.h2d = 0;
    return;
  }
  const Part pr = streamed(r, op.hits);
  const int64_t n = pr.n;
  const int64_t rows = pr.rows;
  if (op.part == 0) {
    op.bytes = up_bytes(c, n, rows);
    op.flops = up_flops(c, rows);
    if (op.h2d < 0) op.h2d = static_cast<int64_t>(r.n_staged) * c->e13;
  } else {
    op.bytes = down_bytes(c, n, rows);
    op.flops = down_flops(c, rows);
    if (op.h2d < 0) op.h2d = static_cast<int64_t>(r.n_staged) * (c->eb - c->e13);
  }
}

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

// Slot conservation over the device cache state (no layer in flight): every
// slot is free or held by exactly one resident expert, and no layer holds
// more than C experts.
oled_status check_slots(Ctx* c) {
  CacheHdr hdr;
  std::vector<int32_t> slots(static_cast<size_t>(c->L) * c->E), free_list(c->n_slots);
  std::vector<ExpertMask> res(c->L);
  std::vector<int32_t> caps(c->L);
  HIP_TRY(c, hipMemcpy(&hdr, c->d_hdr, sizeof(hdr), hipMemcpyDeviceToHost));
  HIP_TRY(c, hipMemcpy(caps.data(), c->d_cap, sizeof(int32_t) * c->L, hipMemcpyDeviceToHost));
  HIP_TRY(c, hipMemcpy(slots.data(), c->d_slot_of, sizeof(int32_t) * slots.size(),
                       hipMemcpyDeviceToHost));
  HIP_TRY(c, hipMemcpy(free_list.data(), c->d_free, sizeof(int32_t) * c->n_slots,
                       hipMemcpyDeviceToHost));
  HIP_TRY(c, hipMemcpy(res.data(), c->d_res, sizeof(ExpertMask) * c->L, hipMemcpyDeviceToHost));
  if (hdr.fault) return fail(c, OLED_ERR_HIP, "device cache state fault %d", hdr.fault);
  if (hdr.free_top < 0 || hdr.free_top > c->n_slots)
    return fail(c, OLED_ERR_HIP, "free list top %d outside [0,%d]", hdr.free_top, c->n_slots);
  int64_t cap_sum = 0;
  for (int l = 0; l < c->L; ++l) {
    if (caps[l] < 0 || caps[l] > c->E)
      return fail(c, OLED_ERR_HIP, "layer %d capacity %d outside [0,%d]", l, caps[l], c->E);
    cap_sum += caps[l];
  }
  if (cap_sum > static_cast<int64_t>(c->L) * c->cap)
    return fail(c, OLED_ERR_HIP, "capacities sum to %lld > C_total", static_cast<long long>(cap_sum));
  std::vector<int> owner(c->n_slots, 0);
  for (int i = 0; i < hdr.free_top; ++i) {
    const int s = free_list[i];
    if (s < 0 || s >= c->n_slots || owner[s]++)
      return fail(c, OLED_ERR_HIP, "free slot %d listed twice or out of range", s);
  }
  for (int l = 0; l < c->L; ++l) {
    int n_res = 0;
    for (int e = 0; e < c->E; ++e) {
      const int s = slots[static_cast<size_t>(l) * c->E + e];
      const bool r = res[l].test(e);
      n_res += r;
      if (r != (s >= 0))
        return fail(c, OLED_ERR_HIP, "expert %d of layer %d: resident %d but slot %d", e, l, r, s);
      if (s < 0) continue;
      if (s >= c->n_slots || owner[s]++) return fail(c, OLED_ERR_HIP, "slot %d held twice", s);
    }
    if (n_res > caps[l])
      return fail(c, OLED_ERR_HIP, "layer %d holds %d > C_l = %d experts", l, n_res, caps[l]);
  }
  for (int s = 0; s < c->n_slots; ++s)
    if (!owner[s]) return fail(c, OLED_ERR_HIP, "slot %d lost", s);
  return OLED_OK;
}


// The hits' GEMMs: the active residents, at most min(C, E) experts; their
// item count stays on the device. With the shader transfer the first
// workgroups of the gate/up launch copy the staged misses' gate/up weights
// (h2d: their bytes, or -1 to take them from the routing record; 0: the
// launch copies nothing), and the hits' down GEMM is enqueued later (sharing
// a launch with the misses' gate/up); with the copy engine it follows at once.
oled_status launch_hits(Ctx* c, int layer, hipStream_t s, int64_t h2d) {
  const void* x_dev = c->fwd_x;
  const int64_t routes = static_cast<int64_t>(c->cur_T) * c->K;
  const int max_hit_items =
      c->cap > 0 ? static_cast<int>(std::min<int64_t>(c->cap, routes) + routes / oled::kItemRows) : 0;
  const bool shader = c->copy_mode == OLED_COPY_SHADER;
  const bool bf16 = c->dtype == OLED_BF16;
  FfnLaunch a = ffn_args(c, layer, 0, max_hit_items, 0);
  a.src = x_dev;
  if (shader && h2d != 0) {
    a.fetch.nblk = kFetchBlocks;
    a.fetch.off = 0;
    a.fetch.len = c->e13;
  }
  {
    OpEvents ev = op_begin(c, OLED_OP_FFN_UP);
    HIP_TRY(c, oled::launch_ffn_up(bf16, a, ev.a, ev.b, s));
    OpRec r = rec(OLED_OP_FFN_UP, layer, -1);
    r.route_seq = c->cur_route;
    r.part = 0;
    r.hits = true;
    r.h2d = shader ? (h2d >= 0 ? h2d * c->e13 / c->eb : -1) : 0;
    op_end(c, ev, r);
  }
  if (!shader) {
    a.src = c->d_h;
    OpEvents ev = op_begin(c, OLED_OP_FFN_DOWN);
    HIP_TRY(c, oled::launch_ffn_down(bf16, a, ev.a, ev.b, s));
    OpRec r = rec(OLED_OP_FFN_DOWN, layer, -1);
    r.route_seq = c->cur_route;
    r.part = 1;
    r.hits = true;
    op_end(c, ev, r);
  }
  return OLED_OK;
}


// The dense experts (at least kDenseMinRows routes; hits and misses alike,
// every weight already in its slot): gate/up tiles, then down tiles. Their
// item counts are on the device.
oled_status launch_dense(Ctx* c, int layer, hipStream_t s) {
  const int64_t routes = static_cast<int64_t>(c->cur_T) * c->K;
  const int max_items = static_cast<int>(
      routes / oled::kDenseRows + std::min<int64_t>(c->E, routes / oled::kDenseMinRows));
  FfnLaunch a = ffn_args(c, layer, 0, max_items, 0);
  a.items = c->d_dense_items;
  a.item_counts = c->d_dense_counts;
  a.src = c->fwd_x;
  a.src_bytes = static_cast<int64_t>(c->cur_T) * c->H * 2;
  for (int part = 3; part <= 4; ++part) {
    const bool up = part == 3;
    if (!up) {
      a.src = c->d_h;
      a.src_bytes = routes * c->I * 2;
    }
    const int kind = up ? OLED_OP_FFN_DENSE_UP : OLED_OP_FFN_DENSE_DOWN;
    OpEvents ev = op_begin(c, kind);
    HIP_TRY(c, oled::launch_ffn_dense(up, a, ev.a, ev.b, s));
    OpRec o = rec(kind, layer, -1);
    o.route_seq = c->cur_route;
    o.part = part;
    op_end(c, ev, o);
  }
  return OLED_OK;
}

// hipMemcpyAsync of a miss copy on the copy stream, or the injected failure
// of the n-th enqueue (oled_set_fault_injection).
hipError_t enqueue_miss_copy(Ctx* c, void* dst, const void* src, size_t n, hipStream_t cs) {
  if (c->copy_fail_at > 0 && ++c->copy_count >= c->copy_fail_at) {
    c->copy_fail_at = 0;
    c->copy_count = 0;
    return hipErrorInvalidValue;
  }
  return hipMemcpyAsync(dst, src, n, hipMemcpyHostToDevice, cs);
}

// After a miss copy could not be enqueued: waits for the copies already
// enqueued, then a retention launch that commits nothing returns the staged
// misses' slots to the free list and keeps the layer's resident set, slot
// table and last retention keys, so the layer is left as its last retention
// left it. Device work stays in stream order, so the context stays usable.
oled_status rollback_layer(Ctx* c, int layer, hipStream_t s, hipStream_t cs) {
  HIP_TRY(c, hipStreamSynchronize(cs));
  c->copies_outstanding = false;
  const int seq = ++c->seq;
  oled::ScoreArgs a;
  a.gates = c->d_gates;
  a.conf = nullptr;
  a.topk_idx = c->d_topk;
  a.counts = c->d_counts;
  a.T = 0;                  // no route or confidence is read
  a.k = c->K;
  a.E = c->E;
  a.layer = layer;
  a.seq = seq;
  a.cv = view(c);
  a.score_out = c->d_score + static_cast<size_t>(layer) * c->E;
  a.out = c->d_ret + layer;
  a.key_out = c->d_key + static_cast<size_t>(layer) * c->E;
  a.parts = oled::score_parts(0, c->K);
  a.acc = c->d_sacc;
  a.acc_sync = c->d_ssync;
  a.reject = 1;
  HIP_TRY(c, oled::launch_score_retain(a, nullptr, nullptr, s));
  c->ret_seq[layer] = seq;
  c->ret_seen[layer] = 0;
  return OLED_OK;
}

// Copy-engine transfer: the staged misses (from the routing kernel's list)
// are copied with hipMemcpyAsync on the copy stream, gate/up parts of all
// first, then the down parts; if the hits were queued, the misses' GEMMs are
// launched as the host sees their copies land.
oled_status apply_misses_sdma(Ctx* c, int layer, hipStream_t cs, const RouteStats& r,
                              int64_t* bytes_out) {
  hipStream_t s = c->cur_stream;
  oled_status st = OLED_OK;
  const int n = c->h_staged->rec.n_staged;
  if (n < 0 || n > c->E) return fail(c, OLED_ERR_HIP, "staged list out of range");
  int64_t bytes = 0;
  if (n > 0) {
    OpEvents ev = op_begin(c, OLED_OP_H2D);
    hipError_t e = hipSuccess;
    if (ev.a) e = hipEventRecord(ev.a, cs);
    for (int part = 0; part < 2 && e == hipSuccess; ++part) {
      const int64_t off = part == 0 ? 0 : c->e13;
      const int64_t len = part == 0 ? c->e13 : c->eb - c->e13;
      for (int i = 0; i < n && e == hipSuccess; ++i) {
        const int ex = c->h_staged->exp[i], sl = c->h_staged->slot[i];
        if (ex < 0 || ex >= c->E || sl < 0 || sl >= c->n_slots) {
          e = hipErrorInvalidValue;
          break;
        }
        const int64_t blk = c->host_block_of[static_cast<size_t>(layer) * c->E + ex];
        e = enqueue_miss_copy(c, c->d_pool + static_cast<int64_t>(sl) * c->eb + off,
                              c->host_pool + blk * c->eb + off, len, cs);
        bytes += len;
      }
      if (e == hipSuccess) e = hipEventRecord(part == 0 ? c->ev_up : c->ev_down, cs);
    }
    if (e == hipSuccess && ev.b) e = hipEventRecord(ev.b, cs);
    if (e != hipSuccess) {
      if (ev.a) c->ev_free.push_back(ev.a);
      if (ev.b) c->ev_free.push_back(ev.b);
      st = rollback_layer(c, layer, s, cs);
      if (st != OLED_OK) return st;
      return fail(c, OLED_ERR_HIP,
                  "layer %d: a miss copy could not be enqueued (%s); its misses were not "
                  "installed, its cache is unchanged and its output was not computed",
                  layer, hipGetErrorString(e));
    }
    OpRec o = rec(OLED_OP_H2D, layer, bytes);
    o.h2d = bytes;
    op_end(c, ev, o);
    c->copies_outstanding = true;
  }
  *bytes_out = bytes;
  if (c->stage != Stage::kHitsQueued) return OLED_OK;
  if (r.n_miss_items <= 0) {
    if (!c->cur_dense) return OLED_OK;
    if (n > 0) {  // misses with dense items only
      st = wait_event_spin(c, c->ev_down, "weight copies");
      if (st != OLED_OK) return st;
      c->copies_outstanding = false;
    }
    return launch_dense(c, layer, s);
  }
  const bool bf16 = c->dtype == OLED_BF16;
  const Part mp = streamed(r, false);
  FfnLaunch a = ffn_args(c, layer, 1, r.n_miss_items, 0);
  a.item_base = r.n_hit_items;
  a.n_items_host = r.n_miss_items;
  a.src = c->fwd_x;
  st = wait_event_spin(c, c->ev_up, "gate/up weight copies");
  if (st != OLED_OK) return st;
  {
    OpEvents ev = op_begin(c, OLED_OP_FFN_UP);
    HIP_TRY(c, oled::launch_ffn_up(bf16, a, ev.a, ev.b, s));
    op_end(c, ev, rec(OLED_OP_FFN_UP, layer, up_bytes(c, mp.n, mp.rows), up_flops(c, mp.rows)));
  }
  a.src = c->d_h;
  st = wait_event_spin(c, c->ev_down, "down weight copies");
  if (st != OLED_OK) return st;
  c->copies_outstanding = false;
  {
    OpEvents ev = op_begin(c, OLED_OP_FFN_DOWN);
    HIP_TRY(c, oled::launch_ffn_down(bf16, a, ev.a, ev.b, s));
    op_end(c, ev, rec(OLED_OP_FFN_DOWN, layer, down_bytes(c, mp.n, mp.rows),
                      down_flops(c, mp.rows)));
  }
  return c->cur_dense ? launch_dense(c, layer, s) : OLED_OK;
}

// Cooperative compensation, Sec. 4.4: the objective J(G) = T_comp(G) -
// lambda * sum_{e in G} p_e with T_comp = max(T_H2D |G|, tau_CPU * tokens left
// to the CPU) and sum_G p = (sum_G S) / (sum S). float64, no contraction.
double coop_objective(const std::vector<int>& misses, const std::vector<uint8_t>& in_g, int n_g,
                      const int32_t* n_tok, const uint64_t* S, uint64_t S_total, double t_h2d,
                      double tau, double lam) {
  int64_t cpu_tokens = 0;
  uint64_t mass = 0;
  for (int e : misses) {
    if (in_g[e]) mass += S[e];
    else cpu_tokens += n_tok[e];
  }
  const double t_gpu = t_h2d * static_cast<double>(n_g);
  const double t_cpu = tau * static_cast<double>(cpu_tokens);
  const double t_comp = t_gpu >= t_cpu ? t_gpu : t_cpu;
  const double share = S_total > 0 ? static_cast<double>(mass) / static_cast<double>(S_total) : 0.0;
  return t_comp - lam * share;
}

// The two-stage dispatch: rho = nbar tau / (nbar tau + T_H2D); stage 1 takes
// the round_half_up(rho |M|) misses of highest (S desc, id asc); stage 2 makes
// at most |M| swaps, each the best by J (the first in (transferred id, CPU id)
// order among equals) and only if it lowers J.
void coop_dispatch(int E, const uint8_t* miss, const int32_t* n_tok, const uint64_t* S,
                   double t_h2d, double tau, double nbar, double lam, uint8_t* transfer) {
  std::vector<int> misses;
  uint64_t S_total = 0;
  for (int e = 0; e < E; ++e) {
    if (miss[e]) misses.push_back(e);
    S_total += S[e];
  }
  const double cpu = nbar * tau;
  const double den = cpu + t_h2d;
  const double rho = den > 0.0 ? cpu / den : 1.0;
  const int m = static_cast<int>(misses.size());
  const int n_g = static_cast<int>(std::floor(rho * static_cast<double>(m) + 0.5));
  std::vector<int> order = misses;
  std::sort(order.begin(), order.end(), [&](int a, int b) { return S[a] != S[b] ? S[a] > S[b] : a < b; });
  std::vector<uint8_t> in_g(E, 0);
  for (int i = 0; i < n_g && i < m; ++i) in_g[order[i]] = 1;
  double J = coop_objective(misses, in_g, n_g, n_tok, S, S_total, t_h2d, tau, lam);
  for (int round = 0; round < m; ++round) {
    bool found = false;
    double best = 0.0;
    int bg = -1, bc = -1;
    for (int g : misses) {
      if (!in_g[g]) continue;
      for (int c2 : misses) {
        if (in_g[c2]) continue;
        in_g[g] = 0;
        in_g[c2] = 1;
        const double j = coop_objective(misses, in_g, n_g, n_tok, S, S_total, t_h2d, tau, lam);
        in_g[g] = 1;
        in_g[c2] = 0;
        if (!found || j < best) {
          found = true;
          best = j;
          bg = g;
          bc = c2;
        }
      }
    }
    if (!found || !(best < J)) break;
    in_g[bg] = 0;
    in_g[bc] = 1;
    J = best;
  }
  for (int e = 0; e < E; ++e) transfer[e] = in_g[e];
}

// Cooperative compensation, after the hits' gate/up launch (which copied no
// misses): the hits' down GEMM whose first workgroups copy the whole blocks
// of the transferred misses, then the transferred misses' gate/up and down
// GEMMs, then the dense experts. h2d: bytes of the transferred misses.
oled_status launch_coop_rest(Ctx* c, int layer, hipStream_t s, int64_t h2d) {
  const bool bf16 = c->dtype == OLED_BF16;
  const int64_t routes = static_cast<int64_t>(c->cur_T) * c->K;
  const int max_hit_items =
      c->cap > 0 ? static_cast<int>(std::min<int64_t>(c->cap, routes) + routes / oled::kItemRows)
                 : 0;
  const int max_miss_items =
      static_cast<int>(std::min<int64_t>(c->E, routes) + routes / oled::kItemRows);
  FfnLaunch d = ffn_args(c, layer, 0, max_hit_items, 0);
  d.src = c->d_h;
  if (h2d > 0) {
    d.fetch.nblk = kFetchBlocks;
    d.fetch.off = 0;
    d.fetch.len = c->eb;
  }
  {
    OpEvents ev = op_begin(c, OLED_OP_FFN_DOWN);
    HIP_TRY(c, oled::launch_ffn_down(bf16, d, ev.a, ev.b, s));
    OpRec o = rec(OLED_OP_FFN_DOWN, layer, -1);
    o.route_seq = c->cur_route;
    o.part = 1;
    o.hits = true;
    o.h2d = h2d;
    op_end(c, ev, o);
  }
  for (int part = 0; part <= 1; ++part) {
    FfnLaunch a = ffn_args(c, layer, 1, max_miss_items, kMissGridCap);
    a.src = part == 0 ? c->fwd_x : c->d_h;
    const int kind = part == 0 ? OLED_OP_FFN_UP : OLED_OP_FFN_DOWN;
    OpEvents ev = op_begin(c, kind);
    HIP_TRY(c, part == 0 ? oled::launch_ffn_up(bf16, a, ev.a, ev.b, s)
                         : oled::launch_ffn_down(bf16, a, ev.a, ev.b, s));
    OpRec o = rec(kind, layer, -1);
    o.route_seq = c->cur_route;
    o.part = part;
    o.h2d = 0;
    op_end(c, ev, o);
  }
  return c->cur_dense ? launch_dense(c, layer, s) : OLED_OK;
}

// Shader transfer, after the hits' gate/up launch: one launch with the hits'
// down GEMM, the transfer of the misses' down weights and the misses' gate/up
// GEMM (their gate/up weights landed with the previous launch); then the
// misses' down GEMM and the dense experts. Miss items are bounded by the
// staging capacity; their count is on the device. h2d: bytes of the staged
// misses, or -1 to take them from the routing record.
oled_status launch_shader_rest(Ctx* c, int layer, hipStream_t s, int64_t h2d) {
  const bool bf16 = c->dtype == OLED_BF16;
  const int64_t routes = static_cast<int64_t>(c->cur_T) * c->K;
  const int max_hit_items =
      c->cap > 0 ? static_cast<int>(std::min<int64_t>(c->cap, routes) + routes / oled::kItemRows)
                 : 0;
  const int max_miss_items =
      static_cast<int>(std::min<int64_t>(c->E, routes) + routes / oled::kItemRows);
  FfnLaunch d = ffn_args(c, layer, 0, max_hit_items, 0);
  d.src = c->d_h;
  d.fetch.nblk = kFetchBlocks;
  d.fetch.off = c->e13;
  d.fetch.len = c->eb - c->e13;
  FfnLaunch u = ffn_args(c, layer, 1, max_miss_items, kMissGridCap);
  u.src = c->fwd_x;
  {
    OpEvents ev = op_begin(c, OLED_OP_FFN_DOWN);
    HIP_TRY(c, oled::launch_ffn_mix(bf16, d, u, ev.a, ev.b, s));
    OpRec o = rec(OLED_OP_FFN_DOWN, layer, -1);
    o.route_seq = c->cur_route;
    o.part = 2;
    o.h2d = h2d >= 0 ? h2d - h2d * c->e13 / c->eb : -1;
    op_end(c, ev, o);
  }
  FfnLaunch a = ffn_args(c, layer, 1, max_miss_items, kMissGridCap);
  a.src = c->d_h;
  {
    OpEvents ev = op_begin(c, OLED_OP_FFN_DOWN);
    HIP_TRY(c, oled::launch_ffn_down(bf16, a, ev.a, ev.b, s));
    OpRec o = rec(OLED_OP_FFN_DOWN, layer, -1);
    o.route_seq = c->cur_route;
    o.part = 1;
    op_end(c, ev, o);
  }
  return c->cur_dense ? launch_dense(c, layer, s) : OLED_OK;
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
  if (cfg->copy_mode != OLED_COPY_SHADER && cfg->copy_mode != OLED_COPY_SDMA)
    return bad(OLED_ERR_INVALID_ARG, "copy_mode must be OLED_COPY_SHADER or OLED_COPY_SDMA");
  if (cfg->adapt_period < 0) return bad(OLED_ERR_INVALID_ARG, "adapt_period < 0");
  if (cfg->coop != 0 && cfg->coop != 1) return bad(OLED_ERR_INVALID_ARG, "coop must be 0 or 1");
  if (cfg->coop) {
    if (cfg->copy_mode != OLED_COPY_SHADER)
      return bad(OLED_ERR_UNSUPPORTED, "coop needs OLED_COPY_SHADER");
    if (cfg->coop_threads < 1) return bad(OLED_ERR_INVALID_ARG, "coop_threads < 1");
    if (!(cfg->coop_t_h2d_us >= 0.0) || !(cfg->coop_tau_cpu_us >= 0.0) ||
        !(cfg->coop_nbar >= 0.0) || !(cfg->coop_lambda_us >= 0.0) ||
        !std::isfinite(cfg->coop_t_h2d_us) || !std::isfinite(cfg->coop_tau_cpu_us) ||
        !std::isfinite(cfg->coop_nbar) || !std::isfinite(cfg->coop_lambda_us))
      return bad(OLED_ERR_INVALID_ARG, "coop times and weights must be finite and >= 0");
    if (!oled::cpu_ffn_supported())
      return bad(OLED_ERR_UNSUPPORTED, "coop needs a CPU with AVX2 and FMA");
  }
  if (cfg->policy != OLED_POLICY_PRIORITY && cfg->policy != OLED_POLICY_LRU &&
      cfg->policy != OLED_POLICY_LFU)
    return bad(OLED_ERR_INVALID_ARG, "policy must be OLED_POLICY_PRIORITY, _LRU or _LFU");
  if (cfg->adapt_period > 0 && cfg->n_layers > oled::kMaxAdaptLayers)
    return bad(OLED_ERR_UNSUPPORTED, "adapt_period > 0 needs n_layers <= 1024");
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
  // the address kernels use to read the pool (same allocation, device view)
  void* dev_view = nullptr;
  if (hipHostGetDevicePointer(&dev_view, const_cast<void*>(cfg->host_pool), 0) != hipSuccess ||
      !dev_view) {
    (void)hipGetLastError();
    return bad(OLED_ERR_INVALID_ARG, "host_pool is not mapped for device access");
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
  c->copy_mode = cfg->copy_mode;
  c->adapt_period = cfg->adapt_period;
  c->policy = cfg->policy;
  c->coop = cfg->coop != 0;
  c->coop_t = cfg->coop_t_h2d_us;
  c->coop_tau = cfg->coop_tau_cpu_us;
  c->coop_nbar = cfg->coop_nbar;
  c->coop_lambda = cfg->coop_lambda_us;
  c->esz = cfg->dtype == OLED_F32 ? 4 : 2;
  c->device = cfg->device;
  c->profile_ops = static_cast<uint32_t>(cfg->profile_ops);
  c->eb = static_cast<int64_t>(3) * c->H * c->I * c->esz;
  c->e13 = static_cast<int64_t>(2) * c->H * c->I * c->esz;
  c->cap = c->C < c->E ? c->C : c->E;
  const int64_t routes = static_cast<int64_t>(c->Tmax) * c->K;
  const int staging = routes < c->E ? static_cast<int>(routes) : c->E;
  c->n_slots = c->L * c->cap + staging;
  c->max_items = static_cast<int>(routes / oled::kItemRows) + c->E + 1;
  c->dense_ok = c->dtype == OLED_BF16 && c->H % 256 == 0 && c->I % 256 == 0 &&
                c->Tmax >= oled::kDenseMinRows && routes * c->I * 2 <= INT32_MAX &&
                static_cast<int64_t>(c->Tmax) * c->H * 2 <= INT32_MAX;
  c->max_dense = c->dense_ok ? static_cast<int>(routes / oled::kDenseRows) + c->E + 1 : 0;
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
      dev_alloc(&c->d_chunk, static_cast<size_t>(oled::permute_chunks(c->Tmax)) * c->E) ||
      dev_alloc(&c->d_sacc, c->E) || dev_alloc(&c->d_ssync, 2) ||
      dev_alloc(&c->d_logits, static_cast<size_t>(c->Tmax) * c->E) ||
      dev_alloc(&c->d_items, c->max_items) ||
      (c->dense_ok && (dev_alloc(&c->d_dense_items, c->max_dense) ||
                       dev_alloc(&c->d_dense_counts, 2))) ||
      dev_alloc(reinterpret_cast<char**>(&c->d_h), routes * c->I * c->esz) ||
      dev_alloc(&c->d_O, routes * c->H) ||
      dev_alloc(&c->d_score, static_cast<size_t>(c->L) * c->E))
    return oom("routing scratch");
  if (dev_alloc(&c->d_hdr, 1) || dev_alloc(&c->d_slot_of, nb) || dev_alloc(&c->d_res, c->L) ||
      dev_alloc(&c->d_res_before, c->L) ||
      dev_alloc(&c->d_last_counts, oled::kCountsPerLayer * c->L) ||
      dev_alloc(&c->d_iters, c->L) || dev_alloc(&c->d_last_use, nb) || dev_alloc(&c->d_freq, nb) ||
      dev_alloc(&c->d_prev_miss, c->L) || dev_alloc(&c->d_key, nb) ||
      dev_alloc(&c->d_free, c->n_slots) || dev_alloc(&c->d_host_addr, nb) ||
      dev_alloc(&c->d_cap, c->L) || dev_alloc(&c->d_stat, c->L))
    return oom("cache state");
  if (hipMemset(c->d_flag, 0, sizeof(int32_t)) != hipSuccess ||
      hipMemset(c->d_item_counts, 0, 2 * sizeof(int32_t)) != hipSuccess ||
      hipMemset(c->d_sync, 0, 2 * sizeof(int32_t)) != hipSuccess ||
      hipMemset(c->d_sacc, 0, sizeof(unsigned long long) * c->E) != hipSuccess ||
      hipMemset(c->d_ssync, 0, 2 * sizeof(int32_t)) != hipSuccess)
    return oom("scratch init");
  {
    std::vector<uint64_t> addr(nb);
    for (int64_t i = 0; i < nb; ++i)
      addr[i] = reinterpret_cast<uint64_t>(dev_view) +
                static_cast<uint64_t>(c->host_block_of[i]) * static_cast<uint64_t>(c->eb);
    if (hipMemcpy(c->d_host_addr, addr.data(), sizeof(uint64_t) * nb, hipMemcpyHostToDevice) !=
        hipSuccess)
      return oom("host block table");
  }
  if (hipHostMalloc(reinterpret_cast<void**>(&c->h_ring), sizeof(RouteStats) * oled::kStatsRing,
                    hipHostMallocDefault) ||
      hipHostMalloc(reinterpret_cast<void**>(&c->h_staged), sizeof(StagedList), hipHostMallocCoherent) ||
      hipHostMalloc(reinterpret_cast<void**>(&c->h_ret), sizeof(RetainOut) * c->L, hipHostMallocDefault))
    return oom("pinned records");
  if (dev_alloc(&c->d_ring, oled::kStatsRing) || dev_alloc(&c->d_ret, c->L) ||
      hipMemset(c->d_ring, 0, sizeof(RouteStats) * oled::kStatsRing) != hipSuccess ||
      hipMemset(c->d_ret, 0, sizeof(RetainOut) * c->L) != hipSuccess)
    return oom("record rings");
  std::memset(c->h_ring, 0, sizeof(RouteStats) * oled::kStatsRing);
  std::memset(c->h_staged, 0, sizeof(StagedList));
  std::memset(c->h_ret, 0, sizeof(RetainOut) * c->L);
  if (hipStreamCreateWithFlags(&c->own_copy, hipStreamNonBlocking) != hipSuccess ||
      hipEventCreateWithFlags(&c->ev_up, hipEventDisableTiming) != hipSuccess ||
      hipEventCreateWithFlags(&c->ev_down, hipEventDisableTiming) != hipSuccess ||
      hipEventCreateWithFlags(&c->ev_order, hipEventDisableTiming) != hipSuccess) {
    g_create_error = "stream/event creation failed";
    free_ctx(c);
    return OLED_ERR_HIP;
  }
  if (c->coop) {
    const size_t rmax = static_cast<size_t>(routes);
    if (dev_alloc(&c->d_cpu, c->L) ||
        hipHostMalloc(reinterpret_cast<void**>(&c->h_ctopk), rmax * 4, hipHostMallocDefault) ||
        hipHostMalloc(reinterpret_cast<void**>(&c->h_cgates), rmax * 4, hipHostMallocDefault) ||
        hipHostMalloc(reinterpret_cast<void**>(&c->h_cconf), static_cast<size_t>(c->Tmax) * 4,
                      hipHostMallocDefault) ||
        hipHostMalloc(reinterpret_cast<void**>(&c->h_cx),
                      static_cast<size_t>(c->Tmax) * c->H * c->esz, hipHostMallocDefault) ||
        hipHostMalloc(reinterpret_cast<void**>(&c->h_cout[0]), rmax * c->H * 4,
                      hipHostMallocDefault) ||
        hipHostMalloc(reinterpret_cast<void**>(&c->h_cout[1]), rmax * c->H * 4,
                      hipHostMallocDefault))
      return oom("cooperative compensation buffers");
    if (hipEventCreateWithFlags(&c->ev_coop, hipEventDisableTiming) != hipSuccess ||
        hipEventCreateWithFlags(&c->ev_x, hipEventDisableTiming) != hipSuccess ||
        hipEventCreateWithFlags(&c->ev_cout[0], hipEventDisableTiming) != hipSuccess ||
        hipEventCreateWithFlags(&c->ev_cout[1], hipEventDisableTiming) != hipSuccess) {
      g_create_error = "coop event creation failed";
      free_ctx(c);
      return OLED_ERR_HIP;
    }
    c->pool.reset(new oled::ThreadPool(cfg->coop_threads));
  }
  c->ret_seq.assign(c->L, 0);
  c->ret_seen.assign(c->L, 0);
  c->rejected.assign(c->L, 0);
  if (init_cache_state(c) != OLED_OK) {
    g_create_error = c->err;
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

oled_status oled_set_fault_injection(void* ctx, int32_t copy_fail_at, int32_t wait_deadline_ms) {
  Ctx* c = static_cast<Ctx*>(ctx);
  if (!c || copy_fail_at < 0 || wait_deadline_ms < 0) return OLED_ERR_INVALID_ARG;
  c->copy_fail_at = copy_fail_at;
  c->copy_count = 0;
  c->wait_deadline_ms = wait_deadline_ms > 0 ? wait_deadline_ms : kDefaultWaitDeadlineMs;
  return OLED_OK;
}

oled_status oled_reset_cache(void* ctx) {
  Ctx* c = static_cast<Ctx*>(ctx);
  if (!c) return OLED_ERR_INVALID_ARG;
  if (c->stage != Stage::kIdle) return fail(c, OLED_ERR_STATE, "reset while a layer is in flight");
  HIP_TRY(c, hipSetDevice(c->device));
  HIP_TRY(c, hipDeviceSynchronize());
  oled_status st = drain_records(c, c->route_n);
  if (st != OLED_OK) return st;
  st = init_cache_state(c);
  if (st != OLED_OK) return st;
  HIP_TRY(c, hipMemset(c->d_ret, 0, sizeof(RetainOut) * c->L));
  c->broken = false;
  std::fill(c->ret_seq.begin(), c->ret_seq.end(), 0);
  std::fill(c->ret_seen.begin(), c->ret_seen.end(), 0);
  std::fill(c->rejected.begin(), c->rejected.end(), 0);
  c->rejected_layer = -1;
  c->bad_route_layer = -1;
  c->reported_bad_route = 0;
  return OLED_OK;
}

}  // extern "C"

namespace {

// Checks shared by route_block and route_block_gate, and the ordering of a
// new stream after the previous one.
oled_status route_begin(Ctx* c, int32_t layer, int32_t T, hipStream_t s, const char* call) {
  oled_status st = check_layer(c, layer);
  if (st != OLED_OK) return st;
  if (c->broken)
    return fail(c, OLED_ERR_STATE, "an earlier HIP failure left the cache state unknown: "
                                   "call oled_reset_cache");
  if (c->stage != Stage::kIdle)
    return fail(c, OLED_ERR_STATE, "%s while layer %d is in flight", call, c->cur_layer);
  if (T < 1 || T > c->Tmax) return fail(c, OLED_ERR_INVALID_ARG, "T=%d outside [1,%d]", T, c->Tmax);
  HIP_TRY(c, hipSetDevice(c->device));
  if (c->have_stream && s != c->cur_stream) {  // order the new stream after the old one
    HIP_TRY(c, hipEventRecord(c->ev_order, c->cur_stream));
    HIP_TRY(c, hipStreamWaitEvent(s, c->ev_order, 0));
    c->cur_stream = s;
  }
  return OLED_OK;
}

// Routing, permutation and staging of the layer from logits on the device.
oled_status route_impl(Ctx* c, int32_t layer, const float* logits_dev, int32_t T, hipStream_t s) {
  // consume what has been published; this call's ring entry must be free
  const int n = c->route_n + 1;
  oled_status st = drain_records(c, n - oled::kStatsRing, false);
  if (st != OLED_OK) return st;

  PermuteOut o;
  o.counts = c->d_counts;
  o.offsets = c->d_offsets;
  o.perm = c->d_perm;
  o.inv_perm = c->d_inv;
  o.items = c->d_items;
  o.item_counts = c->d_item_counts;
  // experts with many rows go to the dense-tile GEMM; a token picks an expert
  // at most once, so no expert of a block of fewer tokens can have that many
  o.dense_min = c->dense_ok && T >= oled::kDenseMinRows ? oled::kDenseMinRows : 0;
  o.dense_items = c->d_dense_items;
  o.dense_counts = c->d_dense_counts;
  o.ring = c->d_ring;
  o.staged = (c->copy_mode == OLED_COPY_SDMA || c->coop) ? c->h_staged : nullptr;
  o.gates = c->d_gates;
  o.pub_topk = c->coop ? c->h_ctopk : nullptr;
  o.pub_gates = c->coop ? c->h_cgates : nullptr;
  o.layer = layer;
  o.E = c->E;
  o.seq = n;
  o.cv = view(c);
  const int64_t route_bytes = static_cast<int64_t>(T) * c->E * 4 + static_cast<int64_t>(T) * c->K * 8;
  const int64_t perm_bytes = static_cast<int64_t>(T) * c->K * 12 + static_cast<int64_t>(c->E) * 8;
  if (oled::route_fused(T, c->K)) {
    OpEvents ev = op_begin(c, OLED_OP_ROUTE_TOPK);
    HIP_TRY(c, oled::launch_route_fused(logits_dev, T, c->K, c->d_topk, c->d_gates, c->d_sync, o,
                                        ev.a, ev.b, s));
    op_end(c, ev, rec(OLED_OP_ROUTE_TOPK, layer, route_bytes + perm_bytes));
  } else {
    {
      OpEvents ev = op_begin(c, OLED_OP_ROUTE_TOPK);
      HIP_TRY(c, oled::launch_route_topk(logits_dev, T, c->E, c->K, c->d_topk, c->d_gates,
                                         c->d_flag, ev.a, ev.b, s));
      op_end(c, ev, rec(OLED_OP_ROUTE_TOPK, layer, route_bytes));
    }
    OpEvents ev = op_begin(c, OLED_OP_PERMUTE);
    if (oled::permute_chunked(T))
      HIP_TRY(c, oled::launch_permute_chunked(c->d_topk, T, c->K, c->d_flag, c->d_chunk, o, ev.a,
                                              ev.b, s));
    else
      HIP_TRY(c, oled::launch_permute(c->d_topk, T, c->K, c->d_flag, o, ev.a, ev.b, s));
    op_end(c, ev, rec(OLED_OP_PERMUTE, layer, perm_bytes));
  }
  c->route_n = n;
  c->cur_route = n;
  c->stage = Stage::kRouted;
  c->cur_layer = layer;
  c->cur_T = T;
  c->cur_dense = o.dense_min > 0;
  c->cur_stream = s;
  c->have_stream = true;
  c->fwd_x = nullptr;
  c->fwd_y = nullptr;
  c->last_routed_layer = layer;
  c->last_routed_T = T;
  return OLED_OK;
}

}  // namespace

extern "C" {

oled_status route_block(void* ctx, int32_t layer, const float* logits_dev, int32_t T, void* stream) {
  Ctx* c = static_cast<Ctx*>(ctx);
  if (!c) return OLED_ERR_INVALID_ARG;
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (!logits_dev && layer >= 0 && layer < c->L && c->stage == Stage::kIdle)
    return fail(c, OLED_ERR_INVALID_ARG, "NULL logits");
  oled_status st = route_begin(c, layer, T, s, "route_block");
  if (st != OLED_OK) return st;
  return route_impl(c, layer, logits_dev, T, s);
}

oled_status route_block_gate(void* ctx, int32_t layer, const void* x_dev, const void* w_gate_dev,
                             int32_t T, void* stream) {
  Ctx* c = static_cast<Ctx*>(ctx);
  if (!c) return OLED_ERR_INVALID_ARG;
  hipStream_t s = static_cast<hipStream_t>(stream);
  if ((!x_dev || !w_gate_dev) && layer >= 0 && layer < c->L && c->stage == Stage::kIdle)
    return fail(c, OLED_ERR_INVALID_ARG, "NULL x or gate weights");
  oled_status st = route_begin(c, layer, T, s, "route_block_gate");
  if (st != OLED_OK) return st;
  OpEvents ev = op_begin(c, OLED_OP_ROUTE_GEMM);
  HIP_TRY(c, oled::launch_router_logits(c->dtype == OLED_BF16, x_dev, w_gate_dev, T, c->E, c->H,
                                        c->d_logits, ev.a, ev.b, s));
  op_end(c, ev, rec(OLED_OP_ROUTE_GEMM, layer,
                    static_cast<int64_t>(T) * c->H * c->esz +
                        static_cast<int64_t>(c->E) * c->H * c->esz +
                        static_cast<int64_t>(T) * c->E * 4,
                    static_cast<int64_t>(2) * T * c->E * c->H));
  c->logits_layer = layer;
  return route_impl(c, layer, c->d_logits, T, s);
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
  c->fwd_x = x_dev;
  c->fwd_y = y_dev;
  c->stage = Stage::kHitsQueued;
  if (c->coop) {
    // x to the host for CPU-executed experts (copy stream; x is an input);
    // the hits' gate/up GEMM at once, without copying misses: which misses
    // are transferred is decided in apply_misses_coop
    HIP_TRY(c, hipMemcpyAsync(c->h_cx, x_dev, static_cast<size_t>(c->cur_T) * c->H * c->esz,
                              hipMemcpyDeviceToHost, c->own_copy));
    HIP_TRY(c, hipEventRecord(c->ev_x, c->own_copy));
    st = launch_hits(c, layer, s, 0);
    if (st != OLED_OK) c->stage = Stage::kRouted;
    return st;
  }
  st = launch_hits(c, layer, s, -1);
  if (st != OLED_OK) c->stage = Stage::kRouted;
  return st;
}


oled_status apply_misses(void* ctx, int32_t layer, void* copy_stream, oled_miss_report* out) {
  Ctx* c = static_cast<Ctx*>(ctx);
  if (!c) return OLED_ERR_INVALID_ARG;
  oled_status st = check_layer(c, layer);
  if (st != OLED_OK) return st;
  if (c->coop) return fail(c, OLED_ERR_STATE, "a coop context compensates with apply_misses_coop");
  if (c->stage != Stage::kRouted && c->stage != Stage::kHitsQueued)
    return fail(c, OLED_ERR_STATE, "apply_misses must follow route_block or moe_forward_cached");
  if (layer != c->cur_layer)
    return fail(c, OLED_ERR_STATE, "apply_misses: layer %d is not the layer in flight (%d)", layer,
                c->cur_layer);
  HIP_TRY(c, hipSetDevice(c->device));
  hipStream_t s = c->cur_stream;
  const bool shader = c->copy_mode == OLED_COPY_SHADER;
  const bool bf16 = c->dtype == OLED_BF16;
  RouteStats r{};
  if (!shader) {  // copy engine: staged list and record, published by the routing kernel
    st = wait_published(c, &c->h_staged->seq, c->cur_route, s, "staged misses");
    if (st != OLED_OK) {
      c->stage = Stage::kIdle;
      return st;
    }
    r = c->h_staged->rec;
  } else if (out) {  // a report synchronises the compute stream
    st = drain_records(c, c->cur_route);
    if (st != OLED_OK) {
      c->stage = Stage::kIdle;
      return st;
    }
    r = c->h_ring[c->cur_route % oled::kStatsRing];
  }
  if ((out || !shader) && r.bad) {
    c->reported_bad_route = c->cur_route;
    if (c->bad_route_layer == layer) c->bad_route_layer = -1;  // reported here
    c->stage = Stage::kIdle;
    return fail(c, OLED_ERR_INVALID_ARG,
                "bad block at layer %d (non-finite router logit): nothing staged, cache "
                "unchanged", layer);
  }
  int64_t bytes = 0;
  if (shader) {
    if (c->stage == Stage::kHitsQueued) {
      st = launch_shader_rest(c, layer, s, -1);
      if (st != OLED_OK) return st;
    } else {
      // control path: transfer the whole blocks of the staged misses
      FetchArgs f;
      f.host_addr = c->d_host_addr + static_cast<size_t>(layer) * c->E;
      f.hdr = c->d_hdr;
      f.off = 0;
      f.len = c->eb;
      f.nblk = kFetchBlocks;
      f.E = c->E;
      OpEvents ev = op_begin(c, OLED_OP_H2D);
      HIP_TRY(c, oled::launch_fetch(c->d_pool, c->eb, c->n_slots, f, ev.a, ev.b, s));
      OpRec o = rec(OLED_OP_H2D, layer, -1);
      o.route_seq = c->cur_route;
      op_end(c, ev, o);
    }
    bytes = static_cast<int64_t>(r.n_staged) * c->eb;
  } else {
    hipStream_t cs = copy_stream ? static_cast<hipStream_t>(copy_stream) : c->own_copy;
    st = apply_misses_sdma(c, layer, cs, r, &bytes);
    if (st != OLED_OK) {
      c->stage = Stage::kIdle;
      return st;
    }
  }
  if (out) {
    out->n_active = r.n_active;
    out->n_hits = r.n_hits;
    out->n_misses = r.n_misses;
    out->n_resident = r.n_resident;
    out->rejected_layer = c->rejected_layer;
    out->n_cpu = 0;
    out->h2d_bytes = bytes;
    c->rejected_layer = -1;
  }
  c->stage = Stage::kApplied;
  return OLED_OK;
}

oled_status apply_misses_coop(void* ctx, int32_t layer, const float* conf_dev,
                              oled_miss_report* out) {
  Ctx* c = static_cast<Ctx*>(ctx);
  if (!c) return OLED_ERR_INVALID_ARG;
  oled_status st = check_layer(c, layer);
  if (st != OLED_OK) return st;
  if (!c->coop) return fail(c, OLED_ERR_STATE, "apply_misses_coop needs a context with coop = 1");
  if (c->stage != Stage::kRouted && c->stage != Stage::kHitsQueued)
    return fail(c, OLED_ERR_STATE, "apply_misses_coop must follow route_block or moe_forward_cached");
  if (layer != c->cur_layer)
    return fail(c, OLED_ERR_STATE, "apply_misses_coop: layer %d is not the layer in flight (%d)",
                layer, c->cur_layer);
  if (!conf_dev) return fail(c, OLED_ERR_INVALID_ARG, "NULL confidence");
  HIP_TRY(c, hipSetDevice(c->device));
  hipStream_t s = c->cur_stream;
  st = wait_published(c, &c->h_staged->seq, c->cur_route, s, "staged misses");
  if (st != OLED_OK) {
    c->stage = Stage::kIdle;
    return st;
  }
  const RouteStats r = c->h_staged->rec;
  if (r.bad) {
    c->reported_bad_route = c->cur_route;
    if (c->bad_route_layer == layer) c->bad_route_layer = -1;
    c->stage = Stage::kIdle;
    return fail(c, OLED_ERR_INVALID_ARG,
                "bad block at layer %d (non-finite router logit): nothing staged, cache "
                "unchanged", layer);
  }
  const int n = r.n_staged, E = c->E, T = c->cur_T, k = c->K;
  if (n < 0 || n > E) return fail(c, OLED_ERR_HIP, "staged list out of range");
  const bool fwd = c->stage == Stage::kHitsQueued;
  std::vector<uint8_t> cpu(E, 0);
  std::vector<int32_t> cnt(E, 0);
  int n_cpu = 0;
  if (n > 0) {
    // the routes came with the staged list; the confidence over the copy stream
    HIP_TRY(c, hipMemcpyAsync(c->h_cconf, conf_dev, static_cast<size_t>(T) * 4,
                              hipMemcpyDeviceToHost, c->own_copy));
    HIP_TRY(c, hipEventRecord(c->ev_coop, c->own_copy));
    st = wait_event_spin(c, c->ev_coop, "confidence copy");
    if (st != OLED_OK) return st;
    // routes per expert and priority numerators, as the retention computes them
    const size_t R = static_cast<size_t>(T) * k;
    std::vector<uint64_t> S(E, 0);
    for (size_t q = 0; q < R; ++q) {
      const int e = c->h_ctopk[q];
      if (e < 0 || e >= E) return fail(c, OLED_ERR_HIP, "published routes out of range");
      ++cnt[e];
      const float cf = c->h_cconf[q / k];
      if (cf >= 0.f && cf <= 1.f)
        S[e] += static_cast<uint64_t>(
            std::floor(static_cast<double>(c->h_cgates[q]) * static_cast<double>(cf) * 0x1p48));
    }
    std::vector<uint8_t> miss(E, 0), transfer(E, 0);
    for (int j = 0; j < n; ++j) {
      const int e = c->h_staged->exp[j];
      if (e < 0 || e >= E) return fail(c, OLED_ERR_HIP, "staged list out of range");
      miss[e] = 1;
    }
    coop_dispatch(E, miss.data(), cnt.data(), S.data(), c->coop_t, c->coop_tau, c->coop_nbar,
                  c->coop_lambda, transfer.data());
    for (int e = 0; e < E; ++e) {
      cpu[e] = miss[e] && !transfer[e];
      n_cpu += cpu[e];
    }
  }
  ExpertMask cm;
  std::memset(&cm, 0, sizeof(cm));
  for (int e = 0; e < E; ++e)
    if (cpu[e]) cm.bits[e >> 5] |= 1u << (e & 31);
  if (n_cpu > 0) HIP_TRY(c, oled::launch_coop_unstage(view(c), layer, E, cm, s));
  const int64_t g_bytes = static_cast<int64_t>(n - n_cpu) * c->eb;
  if (fwd) {
    st = n == 0 ? launch_shader_rest(c, layer, s, 0) : launch_coop_rest(c, layer, s, g_bytes);
    if (st != OLED_OK) return st;
  } else if (n - n_cpu > 0) {  // control path: whole blocks of the transferred misses
    FetchArgs f;
    f.host_addr = c->d_host_addr + static_cast<size_t>(layer) * E;
    f.hdr = c->d_hdr;
    f.off = 0;
    f.len = c->eb;
    f.nblk = kFetchBlocks;
    f.E = E;
    OpEvents ev = op_begin(c, OLED_OP_H2D);
    HIP_TRY(c, oled::launch_fetch(c->d_pool, c->eb, c->n_slots, f, ev.a, ev.b, s));
    OpRec o = rec(OLED_OP_H2D, layer, g_bytes);
    o.h2d = g_bytes;
    op_end(c, ev, o);
  }
  if (fwd && n_cpu > 0) {
    // the CPU experts' rows, in the expert-sorted route order (offsets of the
    // stable permutation: an expert's routes in token order)
    std::vector<int32_t> off(E + 1, 0);
    for (int e = 0; e < E; ++e) off[e + 1] = off[e] + cnt[e];
    std::vector<std::vector<int32_t>> toks(E);
    const size_t R = static_cast<size_t>(T) * k;
    for (size_t q = 0; q < R; ++q)
      if (cpu[c->h_ctopk[q]]) toks[c->h_ctopk[q]].push_back(static_cast<int32_t>(q / k));
    const int b = c->cout_buf;
    if (c->cout_used[b]) {  // its previous rows have been copied out
      st = wait_event_spin(c, c->ev_cout[b], "CPU output copy");
      if (st != OLED_OK) return st;
    }
    st = wait_event_spin(c, c->ev_x, "copy of x");
    if (st != OLED_OK) return st;
    float* hout = c->h_cout[b];
    std::vector<oled::CpuExpertJob> jobs;
    for (int e = 0; e < E; ++e) {
      if (!cpu[e]) continue;
      const int64_t blk = c->host_block_of[static_cast<size_t>(layer) * E + e];
      jobs.push_back({c->host_pool + blk * c->eb, toks[e].data(), cnt[e],
                      hout + static_cast<size_t>(off[e]) * c->H});
    }
    oled::cpu_ffn_run(*c->pool, c->dtype == OLED_BF16, c->H, c->I, c->h_cx, jobs.data(),
                      static_cast<int>(jobs.size()), c->cpu_scratch);
    for (int e = 0; e < E; ++e) {
      if (!cpu[e]) continue;
      const size_t o0 = static_cast<size_t>(off[e]) * c->H;
      HIP_TRY(c, hipMemcpyAsync(c->d_O + o0, hout + o0, static_cast<size_t>(cnt[e]) * c->H * 4,
                                hipMemcpyHostToDevice, s));
    }
    HIP_TRY(c, hipEventRecord(c->ev_cout[b], s));
    c->cout_used[b] = true;
    c->cout_buf = b ^ 1;
  }
  c->acc.n_cpu_executed += n_cpu;
  c->acc.n_transferred -= n_cpu;
  c->acc.h2d_bytes -= static_cast<int64_t>(n_cpu) * c->eb;
  if (out) {
    out->n_active = r.n_active;
    out->n_hits = r.n_hits;
    out->n_misses = r.n_misses;
    out->n_resident = r.n_resident;
    out->rejected_layer = c->rejected_layer;
    out->n_cpu = n_cpu;
    out->h2d_bytes = g_bytes;
    c->rejected_layer = -1;
  }
  c->stage = Stage::kApplied;
  return OLED_OK;
}

oled_status oled_coop_dispatch(int32_t n_experts, const uint8_t* miss, const int32_t* n_tok,
                               const uint64_t* score, double t_h2d_us, double tau_cpu_us,
                               double nbar, double lambda_us, uint8_t* transfer_out) {
  if (!miss || !n_tok || !score || !transfer_out) return OLED_ERR_INVALID_ARG;
  if (n_experts < 1 || n_experts > oled::kMaxExperts) return OLED_ERR_INVALID_ARG;
  if (!(t_h2d_us >= 0.0) || !(tau_cpu_us >= 0.0) || !(nbar >= 0.0) || !(lambda_us >= 0.0))
    return OLED_ERR_INVALID_ARG;
  coop_dispatch(n_experts, miss, n_tok, score, t_h2d_us, tau_cpu_us, nbar, lambda_us,
                transfer_out);
  return OLED_OK;
}

oled_status oled_cpu_ffn(int32_t dtype, int32_t hidden, int32_t inter, const void* block,
                         const void* x, int32_t n, float* out, int32_t threads) {
  if (!block || !x || !out || n < 0 || threads < 1) return OLED_ERR_INVALID_ARG;
  if (dtype != OLED_F32 && dtype != OLED_BF16) return OLED_ERR_INVALID_ARG;
  if (hidden <= 0 || inter <= 0 || hidden % 128 || inter % 128) return OLED_ERR_UNSUPPORTED;
  if (!oled::cpu_ffn_supported()) return OLED_ERR_UNSUPPORTED;
  if (n == 0) return OLED_OK;
  std::vector<int32_t> rows(n);
  for (int i = 0; i < n; ++i) rows[i] = i;
  oled::CpuExpertJob job{block, rows.data(), n, out};
  // thread pools live until the process ends, one per thread count
  static std::mutex mu;
  static std::map<int, std::unique_ptr<oled::ThreadPool>> pools;
  std::lock_guard<std::mutex> lk(mu);
  std::unique_ptr<oled::ThreadPool>& pool = pools[threads];
  if (!pool) pool.reset(new oled::ThreadPool(threads));
  std::vector<float> scratch;
  oled::cpu_ffn_run(*pool, dtype == OLED_BF16, hidden, inter, x, &job, 1, scratch);
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
  const int seq = ++c->seq;
  oled::ScoreArgs a;
  a.gates = c->d_gates;
  a.conf = static_cast<const float*>(conf_dev);
  a.topk_idx = c->d_topk;
  a.counts = c->d_counts;
  a.T = c->cur_T;
  a.k = c->K;
  a.E = c->E;
  a.layer = layer;
  a.seq = seq;
  a.cv = view(c);
  a.score_out = c->d_score + static_cast<size_t>(layer) * c->E;
  a.out = c->d_ret + layer;
  a.key_out = c->d_key + static_cast<size_t>(layer) * c->E;
  a.parts = oled::score_parts(c->cur_T, c->K);
  a.acc = c->d_sacc;
  a.acc_sync = c->d_ssync;
  const int64_t score_bytes = static_cast<int64_t>(c->cur_T) * c->K * 12 +
                              static_cast<int64_t>(c->cur_T) * 4 + static_cast<int64_t>(c->E) * 16;
  if (c->fwd_y) {  // the forward ran: the combine shares the launch
    oled::CombineArgs cb;
    cb.O = c->d_O;
    cb.gates = c->d_gates;
    cb.inv_perm = c->d_inv;
    cb.T = c->cur_T;
    cb.k = c->K;
    cb.H = c->H;
    cb.y = c->fwd_y;
    OpEvents ev = op_begin(c, OLED_OP_COMBINE);
    HIP_TRY(c, oled::launch_combine_score(c->dtype == OLED_BF16, cb, a, ev.a, ev.b, s));
    op_end(c, ev, rec(OLED_OP_COMBINE, layer,
                      static_cast<int64_t>(c->cur_T) * c->K * (c->H * 4 + 8) +
                          static_cast<int64_t>(c->cur_T) * c->H * c->esz + score_bytes));
  } else {
    OpEvents ev = op_begin(c, OLED_OP_SCORE_RETAIN);
    HIP_TRY(c, oled::launch_score_retain(a, ev.a, ev.b, s));
    op_end(c, ev, rec(OLED_OP_SCORE_RETAIN, layer, score_bytes));
  }
  c->ret_seq[layer] = seq;
  c->ret_seen[layer] = 0;
  c->stage = Stage::kIdle;
  c->cur_layer = -1;
  if (c->adapt_period > 0 && layer == c->L - 1 && ++c->iters_done % c->adapt_period == 0) {
    oled::AdaptArgs ad;
    ad.cv = view(c);
    ad.score = c->d_key;
    ad.L = c->L;
    ad.E = c->E;
    ad.c_total = c->L * c->cap;
    OpEvents ev = op_begin(c, OLED_OP_LAYER_ADAPT);
    HIP_TRY(c, oled::launch_layer_adapt(ad, ev.a, ev.b, s));
    op_end(c, ev, rec(OLED_OP_LAYER_ADAPT, layer,
                      static_cast<int64_t>(c->L) * (c->E * 8 + 64)));
  }
  return OLED_OK;
}

oled_status oled_read_layer_state(void* ctx, int32_t layer, oled_layer_state* out) {
  Ctx* c = static_cast<Ctx*>(ctx);
  if (!c || !out) return OLED_ERR_INVALID_ARG;
  if (layer < 0 || layer >= c->L) return fail(c, OLED_ERR_INVALID_ARG, "layer out of range");
  HIP_TRY(c, hipSetDevice(c->device));
  HIP_TRY(c, hipDeviceSynchronize());
  oled_status st = drain_records(c, c->route_n);
  if (st != OLED_OK) return st;
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
  ExpertMask before, after;
  int32_t lc[oled::kCountsPerLayer];
  std::vector<int32_t> slots(c->E);
  HIP_TRY(c, hipMemcpy(&before, c->d_res_before + layer, sizeof(ExpertMask), hipMemcpyDeviceToHost));
  HIP_TRY(c, hipMemcpy(&after, c->d_res + layer, sizeof(ExpertMask), hipMemcpyDeviceToHost));
  HIP_TRY(c, hipMemcpy(lc, c->d_last_counts + oled::kCountsPerLayer * layer, sizeof(lc),
                       hipMemcpyDeviceToHost));
  HIP_TRY(c, hipMemcpy(slots.data(), c->d_slot_of + static_cast<size_t>(layer) * c->E,
                       sizeof(int32_t) * c->E, hipMemcpyDeviceToHost));
  for (int e = 0; e < c->E; ++e) {
    if (out->resident_before) out->resident_before[e] = before.test(e);
    if (out->resident_after) out->resident_after[e] = after.test(e);
    if (out->slot_of) out->slot_of[e] = after.test(e) ? slots[e] : -1;
  }
  out->n_active = lc[0];
  out->n_hits = lc[1];
  out->n_misses = lc[2];
  int32_t cap_now = 0;
  HIP_TRY(c, hipMemcpy(&cap_now, c->d_cap + layer, sizeof(int32_t), hipMemcpyDeviceToHost));
  out->capacity = cap_now;
  out->reserved = 0;
  out->prev_transferred = lc[4];
  out->reused_transfers = lc[5];
  if (out->logits && T > 0 && c->logits_layer == layer)
    HIP_TRY(c, hipMemcpy(out->logits, c->d_logits, static_cast<size_t>(T) * c->E * 4,
                         hipMemcpyDeviceToHost));
  if (out->retain_key)
    HIP_TRY(c, hipMemcpy(out->retain_key, c->d_key + static_cast<size_t>(layer) * c->E, c->E * 8,
                         hipMemcpyDeviceToHost));
  if (out->retained) {
    RetainOut ro;
    HIP_TRY(c, hipMemcpy(&ro, c->d_ret + layer, sizeof(RetainOut), hipMemcpyDeviceToHost));
    for (int e = 0; e < c->E; ++e) out->retained[e] = (ro.retained[e >> 5] >> (e & 31)) & 1u;
  }
  if (c->stage == Stage::kIdle) {
    st = check_slots(c);
    if (st != OLED_OK) return st;
  }
  if (c->rejected[layer])
    return fail(c, OLED_ERR_INVALID_ARG, "the last retention of layer %d was rejected", layer);
  if (c->bad_route_layer == layer) {
    c->bad_route_layer = -1;
    return fail(c, OLED_ERR_INVALID_ARG, "a bad block (non-finite router logit) was seen at layer %d",
                layer);
  }
  return OLED_OK;
}

oled_status oled_collect_stats(void* ctx, oled_stats* out) {
  Ctx* c = static_cast<Ctx*>(ctx);
  if (!c || !out) return OLED_ERR_INVALID_ARG;
  HIP_TRY(c, hipSetDevice(c->device));
  HIP_TRY(c, hipDeviceSynchronize());
  const oled_status st = drain_records(c, c->route_n);
  if (st != OLED_OK) return st;
  *out = c->acc;
  c->acc = oled_stats{};
  return OLED_OK;
}

oled_status oled_profile_collect(void* ctx, oled_op_time* out, int32_t cap, int32_t* n_out) {
  Ctx* c = static_cast<Ctx*>(ctx);
  if (!c || !n_out || (cap > 0 && !out)) return OLED_ERR_INVALID_ARG;
  HIP_TRY(c, hipSetDevice(c->device));
  HIP_TRY(c, hipDeviceSynchronize());
  const oled_status st = drain_records(c, c->route_n);
  if (st != OLED_OK) return st;
  int n = 0;
  for (auto& op : c->ops) {
    if (op.route_seq > 0) {
      const RouteStats* r = find_record(c, op.route_seq);
      if (r) complete_op(c, op, *r);
    }
    float ms = 0.f;
    const hipError_t e = hipEventElapsedTime(&ms, op.a, op.b);
    if (n < cap) {
      out[n].kind = op.kind;
      out[n].layer = op.layer;
      out[n].ms = e == hipSuccess ? ms : -1.f;
      out[n].bytes = op.bytes;
      out[n].flops = op.flops;
      out[n].h2d_bytes = op.h2d;
      ++n;
    }
    c->ev_free.push_back(op.a);
    c->ev_free.push_back(op.b);
  }
  c->ops.clear();
  c->recs.clear();
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
  if (ptr) (void)hipHostFree(ptr);
}

}  // extern "C"

namespace oled {
void set_noctx_error(const char* msg) { g_create_error = msg; }
}  // namespace oled
