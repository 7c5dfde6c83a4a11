// Launchers of the gfx950 kernels of the block-MoE layer, and the small
// structs that travel between host and device (pinned summaries, kernel
// argument tables). Internal to the library.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace oled {

constexpr int kMaxExperts = 256;
constexpr int kMaxTopK = 16;
constexpr int kItemRows = 64;   // routes (token rows) per grouped-GEMM work item
constexpr int kScoreShift = 48; // priority numerators are floor(g * c * 2^48)

// Written by the permute kernel into coherent pinned host memory (seq last,
// after a system-scope fence); the host polls seq.
struct RouteSummary {
  int32_t counts[kMaxExperts];
  int32_t n_hit_items;
  int32_t n_miss_items;
  int32_t bad_logits;  // a non-finite router logit was seen
  int32_t seq;         // call sequence number, for freshness checks
};

// Written by the score/retain kernel into coherent pinned host memory, one
// per layer (seq last, after a system-scope fence).
struct RetainOut {
  uint32_t retained[kMaxExperts / 32];  // bit e: expert e stays cached
  int32_t bad_conf;    // a confidence outside [0, 1] was seen
  int32_t n_retained;
  int32_t seq;
  int32_t pad;
};

// Expert mask passed by value as a kernel argument.
struct ExpertMask {
  uint32_t bits[kMaxExperts / 32];
  __host__ __device__ bool test(int e) const { return (bits[e >> 5] >> (e & 31)) & 1u; }
};

// Cache slot of every expert of the layer (-1: not on the device), by value.
struct SlotTable {
  int32_t slot[kMaxExperts];
};

// One grouped-GEMM work item: rows [row_begin, row_begin + rows) of the
// expert-sorted route order, all routed to `expert`.
struct WorkItem {
  int32_t expert;
  int32_t row_begin;
  int32_t rows;
  int32_t pad;
};

// Arguments of a grouped-GEMM launch over work items [item_base, item_base + n).
// n = n_items_host if >= 0, else read from n_items_dev on the device (the
// launch may then be enqueued before the host knows the routing result);
// max_items bounds n and sizes the persistent grid.
struct FfnLaunch {
  const void* pool;
  int64_t slot_bytes;
  const SlotTable* slots;
  const WorkItem* items;
  const int32_t* n_items_dev;
  int item_base;
  int n_items_host;
  int max_items;
  const void* src;        // up: x [T][H]; down: h [T*k][I]
  const int32_t* perm;    // up: route of each sorted position (token = route / k)
  int k, H, I;
  void* hout;             // up: h [T*k][I]
  float* oout;            // down: O [T*k][H]
};

// Every launcher takes optional (ev0, ev1): if non-null they record the
// kernel's start and end on the dispatch itself (no extra stream packets).

// K1: top-k + fp64 gates, one wavefront per token.
hipError_t launch_route_topk(const float* logits, int T, int E, int k, int32_t* topk_idx,
                             float* gates, int32_t* bad_flag, hipEvent_t ev0, hipEvent_t ev1,
                             hipStream_t s);

// K2: histogram, offsets, stable permutation, hit-first work list, item counts
// (device: item_counts[0] hits, [1] misses) and the pinned host summary.
hipError_t launch_permute(const int32_t* topk_idx, int T, int k, int E, const ExpertMask& resident,
                          int32_t* counts, int32_t* offsets, int32_t* perm, int32_t* inv_perm,
                          WorkItem* items, int32_t* item_counts, int32_t* bad_flag,
                          RouteSummary* summary, int seq, hipEvent_t ev0, hipEvent_t ev1,
                          hipStream_t s);

// K1+K2 as one launch for blocks with T*k <= 1024 (route_fused true): the
// last workgroup to finish routing permutes. sync: 2 device ints, zero
// before the first launch; the kernel leaves them zero.
bool route_fused(int T, int k);
hipError_t launch_route_fused(const float* logits, int T, int E, int k, const ExpertMask& resident,
                              int32_t* topk_idx, float* gates, int32_t* counts, int32_t* offsets,
                              int32_t* perm, int32_t* inv_perm, WorkItem* items,
                              int32_t* item_counts, int32_t* sync, RouteSummary* summary, int seq,
                              hipEvent_t ev0, hipEvent_t ev1, hipStream_t s);

// K4a: grouped gate/up GEMM with SiLU*up epilogue (h = silu(W1 x) * (W3 x)).
hipError_t launch_ffn_up(bool bf16, const FfnLaunch& a, hipEvent_t ev0, hipEvent_t ev1,
                         hipStream_t s);

// K4b: grouped down GEMM (O = W2 h, fp32).
hipError_t launch_ffn_down(bool bf16, const FfnLaunch& a, hipEvent_t ev0, hipEvent_t ev1,
                           hipStream_t s);

// K5: y[t] = sum_j gate[t][j] * O[inv_perm[t*k + j]], fp32, rounded once to dtype.
hipError_t launch_combine(bool bf16, const float* O, const float* gates, const int32_t* inv_perm,
                          int T, int k, int H, void* y, hipEvent_t ev0, hipEvent_t ev1,
                          hipStream_t s);

// K6: priority numerators (per-expert segment sums) + Top-C retention.
hipError_t launch_score_retain(const float* gates, const float* conf, const int32_t* topk_idx,
                               const int32_t* counts, int T, int k, int E, int C,
                               const ExpertMask& resident, uint64_t* score_out, RetainOut* out,
                               int seq, hipEvent_t ev0, hipEvent_t ev1, hipStream_t s);

}  // namespace oled
