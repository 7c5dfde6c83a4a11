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
constexpr int kFeatTile = 64;   // output features per grouped-GEMM workgroup
constexpr int kScoreShift = 48; // priority numerators are floor(g * c * 2^48)

// Written by the permute kernel into pinned host memory; read by the host
// after the route event has completed.
struct RouteSummary {
  int32_t counts[kMaxExperts];
  int32_t n_hit_items;
  int32_t n_miss_items;
  int32_t bad_logits;  // a non-finite router logit was seen
  int32_t seq;         // call sequence number, for freshness checks
};

// Written by the score/retain kernel into pinned host memory, one per layer.
struct RetainOut {
  uint8_t retained[kMaxExperts];
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

// K1: top-k + fp64 gates, one wavefront per token.
hipError_t launch_route_topk(const float* logits, int T, int E, int k, int32_t* topk_idx,
                             float* gates, int32_t* bad_flag, hipStream_t s);

// K2: histogram, offsets, stable permutation, hit-first work list, summary.
hipError_t launch_permute(const int32_t* topk_idx, int T, int k, int E, const ExpertMask& resident,
                          int32_t* counts, int32_t* offsets, int32_t* perm, int32_t* inv_perm,
                          WorkItem* items, int32_t* bad_flag, RouteSummary* summary, int seq,
                          hipStream_t s);

// K4a: grouped gate/up GEMM with SiLU*up epilogue over items [item_base, +n_items).
// x: [T][H] (gathered through perm[row] / k); h: [T*k][I]. bf16 or f32 by `bf16`.
hipError_t launch_ffn_up(bool bf16, const void* pool, int64_t slot_bytes, const SlotTable& slots,
                         const WorkItem* items, int item_base, int n_items, const void* x,
                         const int32_t* perm, int k, int H, int I, void* h, hipStream_t s);

// K4b: grouped down GEMM over the same items: O [T*k][H] fp32.
hipError_t launch_ffn_down(bool bf16, const void* pool, int64_t slot_bytes, const SlotTable& slots,
                           const WorkItem* items, int item_base, int n_items, const void* h,
                           int H, int I, float* O, hipStream_t s);

// K5: y[t] = sum_j gate[t][j] * O[inv_perm[t*k + j]], fp32, rounded once to dtype.
hipError_t launch_combine(bool bf16, const float* O, const float* gates, const int32_t* inv_perm,
                          int T, int k, int H, void* y, hipStream_t s);

// K6: priority numerators (segmented reduction) + Top-C retention.
hipError_t launch_score_retain(const float* gates, const float* conf, const int32_t* perm,
                               const int32_t* offsets, const int32_t* counts, int T, int k, int E,
                               int C, const ExpertMask& resident, uint64_t* score_out,
                               RetainOut* out, int seq, hipStream_t s);

}  // namespace oled
