// A host-only stand-in for the HIP runtime and for the library's kernel
// launchers, so that the runtime (oled.cpp) can be built with g++ under
// AddressSanitizer / UndefinedBehaviorSanitizer and driven through its C ABI
// on a machine without a GPU. "Device" memory is host memory, copies are
// memcpy, streams and events complete at once (unless fake_hip_stall_events
// holds them back, to drive the runtime's wait deadline). The launcher stubs
// compute nothing: they publish the records the runtime reads back (routing
// record, staged list, retention result) so that its state machine, argument
// checks, record draining and failure paths run as they do on the GPU.
#include <hip/hip_runtime.h>

#include <cstdlib>
#include <cstring>
#include <mutex>
#include <set>

#include "kernels.h"

namespace {
std::mutex g_mu;
std::set<const void*> g_pinned;   // fake hipHostMalloc allocations
int g_stall_events = 0;           // 1: hipEventQuery reports hipErrorNotReady
struct FakeEvent { int id; };
struct FakeStream { int id; };
int g_staged = 0;                 // misses the routing stub stages (expert i -> slot i)
}  // namespace

extern "C" {

void fake_hip_stall_events(int on) { g_stall_events = on; }
void fake_hip_stage_misses(int n) { g_staged = n; }

hipError_t hipMalloc(void** ptr, size_t size) {
  if (!ptr) return hipErrorInvalidValue;
  *ptr = std::calloc(1, size ? size : 1);
  return *ptr ? hipSuccess : hipErrorOutOfMemory;
}
hipError_t hipFree(void* ptr) {
  std::free(ptr);
  return hipSuccess;
}
hipError_t hipHostMalloc(void** ptr, size_t size, unsigned int) {
  if (!ptr) return hipErrorInvalidValue;
  *ptr = std::calloc(1, size ? size : 1);
  if (!*ptr) return hipErrorOutOfMemory;
  std::lock_guard<std::mutex> lk(g_mu);
  g_pinned.insert(*ptr);
  return hipSuccess;
}
hipError_t hipHostFree(void* ptr) {
  {
    std::lock_guard<std::mutex> lk(g_mu);
    g_pinned.erase(ptr);
  }
  std::free(ptr);
  return hipSuccess;
}
hipError_t hipMemcpy(void* dst, const void* src, size_t n, hipMemcpyKind) {
  if (n) std::memmove(dst, src, n);
  return hipSuccess;
}
hipError_t hipMemcpyAsync(void* dst, const void* src, size_t n, hipMemcpyKind, hipStream_t) {
  if (n) std::memmove(dst, src, n);
  return hipSuccess;
}
hipError_t hipMemset(void* dst, int value, size_t n) {
  std::memset(dst, value, n);
  return hipSuccess;
}
hipError_t hipSetDevice(int d) { return d == 0 ? hipSuccess : hipErrorInvalidDevice; }
hipError_t hipGetDeviceCount(int* n) {
  *n = 1;
  return hipSuccess;
}
hipError_t hipDeviceSynchronize(void) { return hipSuccess; }
hipError_t hipStreamCreateWithFlags(hipStream_t* s, unsigned int) {
  *s = reinterpret_cast<hipStream_t>(new FakeStream{1});
  return hipSuccess;
}
hipError_t hipStreamDestroy(hipStream_t s) {
  delete reinterpret_cast<FakeStream*>(s);
  return hipSuccess;
}
hipError_t hipStreamSynchronize(hipStream_t) { return hipSuccess; }
hipError_t hipStreamQuery(hipStream_t) { return hipSuccess; }
hipError_t hipStreamWaitEvent(hipStream_t, hipEvent_t, unsigned int) { return hipSuccess; }
hipError_t hipEventCreateWithFlags(hipEvent_t* e, unsigned) {
  *e = reinterpret_cast<hipEvent_t>(new FakeEvent{1});
  return hipSuccess;
}
hipError_t hipEventDestroy(hipEvent_t e) {
  delete reinterpret_cast<FakeEvent*>(e);
  return hipSuccess;
}
hipError_t hipEventRecord(hipEvent_t, hipStream_t) { return hipSuccess; }
hipError_t hipEventQuery(hipEvent_t) { return g_stall_events ? hipErrorNotReady : hipSuccess; }
hipError_t hipEventElapsedTime(float* ms, hipEvent_t, hipEvent_t) {
  *ms = 0.01f;
  return hipSuccess;
}
hipError_t hipGetLastError(void) { return hipSuccess; }
const char* hipGetErrorString(hipError_t e) {
  return e == hipSuccess ? "hipSuccess" : "fake HIP error";
}
hipError_t hipHostGetDevicePointer(void** dev, void* host, unsigned int) {
  *dev = host;
  return hipSuccess;
}
hipError_t hipPointerGetAttributes(hipPointerAttribute_t* attr, const void* ptr) {
  std::memset(attr, 0, sizeof(*attr));
  std::lock_guard<std::mutex> lk(g_mu);
  attr->type = g_pinned.count(ptr) ? hipMemoryTypeHost : hipMemoryTypeUnregistered;
  return hipSuccess;
}

}  // extern "C"

namespace oled {

bool route_fused(int T, int k) { return T * k <= 1024; }
bool permute_chunked(int T) { return T > 1024; }
int permute_chunks(int T) { return (T + 511) / 512; }
int score_parts(int T, int k) {
  const long R = static_cast<long>(T) * k;
  return R <= 8192 ? 1 : static_cast<int>((R + 8191) / 8192);
}

namespace {
// The routing record (and, when asked, the staged list and the routes) as
// the permute kernels leave them: nothing active unless misses are staged.
void publish_route(int T, int k, const PermuteOut& o) {
  RouteStats rs{};
  rs.layer = o.layer;
  rs.n_staged = rs.n_misses = rs.n_active = rs.n_miss_items = rs.miss_rows = g_staged;
  rs.seq = o.seq;
  if (o.ring) o.ring[o.seq % kStatsRing] = rs;
  if (o.item_counts) o.item_counts[0] = o.item_counts[1] = 0;
  if (o.staged) {
    for (int i = 0; i < g_staged; ++i) {
      o.staged->exp[i] = i;
      o.staged->slot[i] = i;
    }
    if (o.pub_topk)
      for (int r = 0; r < T * k; ++r) {
        o.pub_topk[r] = r % o.E;
        o.pub_gates[r] = 1.0f / static_cast<float>(k);
      }
    o.staged->rec = rs;
    o.staged->seq = o.seq;
  }
}
}  // namespace

hipError_t launch_router_logits(bool, const void*, const void*, int, int, int, float*, hipEvent_t,
                                hipEvent_t, hipStream_t) {
  return hipSuccess;
}
hipError_t launch_route_topk(const float*, int, int, int, int32_t*, float*, int32_t*, hipEvent_t,
                             hipEvent_t, hipStream_t, int) {
  return hipSuccess;
}
hipError_t launch_permute(const int32_t*, int T, int k, int32_t*, const PermuteOut& o, hipEvent_t,
                          hipEvent_t, hipStream_t) {
  publish_route(T, k, o);
  return hipSuccess;
}
hipError_t launch_permute_chunked(const int32_t*, int T, int k, int32_t*, int32_t*,
                                  const PermuteOut& o, hipEvent_t, hipEvent_t, hipStream_t) {
  publish_route(T, k, o);
  return hipSuccess;
}
hipError_t launch_route_fused(const float*, int T, int k, int32_t*, float*, int32_t*,
                              const PermuteOut& o, hipEvent_t, hipEvent_t, hipStream_t) {
  publish_route(T, k, o);
  return hipSuccess;
}
hipError_t launch_ffn_up(bool, const FfnLaunch&, hipEvent_t, hipEvent_t, hipStream_t) {
  return hipSuccess;
}
hipError_t launch_ffn_down(bool, const FfnLaunch&, hipEvent_t, hipEvent_t, hipStream_t) {
  return hipSuccess;
}
hipError_t launch_ffn_mix(bool, const FfnLaunch&, const FfnLaunch&, hipEvent_t, hipEvent_t,
                          hipStream_t) {
  return hipSuccess;
}
hipError_t launch_ffn_dense(bool, const FfnLaunch&, hipEvent_t, hipEvent_t, hipStream_t) {
  return hipSuccess;
}
hipError_t launch_fetch(const void*, int64_t, int, const FetchArgs&, hipEvent_t, hipEvent_t,
                        hipStream_t) {
  return hipSuccess;
}
hipError_t launch_score_retain(const ScoreArgs& a, hipEvent_t, hipEvent_t, hipStream_t) {
  if (a.parts != score_parts(a.T, a.k)) return hipErrorInvalidValue;
  if (!a.reject && !a.conf) return hipErrorInvalidValue;   // the kernel would read it
  a.out->seq = a.seq;
  a.out->bad_conf = 0;
  return hipSuccess;
}
hipError_t launch_combine_score(bool, const CombineArgs&, const ScoreArgs& a, hipEvent_t ev0,
                                hipEvent_t ev1, hipStream_t s) {
  return launch_score_retain(a, ev0, ev1, s);
}
hipError_t launch_layer_adapt(const AdaptArgs&, hipEvent_t, hipEvent_t, hipStream_t) {
  return hipSuccess;
}
hipError_t launch_coop_unstage(const CacheView&, int, int, const ExpertMask&, hipStream_t) {
  return hipSuccess;
}

}  // namespace oled
