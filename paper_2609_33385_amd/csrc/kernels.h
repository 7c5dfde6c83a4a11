// Launchers of the gfx950 kernels of the block-MoE layer, and the small
// structs that travel between host and device (device-resident cache state,
// pinned summaries, kernel argument tables). Internal to the library.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace oled {

constexpr int kMaxExperts = 256;
constexpr int kMaxTopK = 16;
constexpr int kItemRows = 64;    // routes (token rows) per grouped-GEMM work item
constexpr int kScoreShift = 48;  // priority numerators are floor(g * c * 2^48)
constexpr int kStatsRing = 4096; // routing records kept in pinned memory

// Expert mask (one bit per expert).
struct ExpertMask {
  uint32_t bits[kMaxExperts / 32];
  __host__ __device__ bool test(int e) const { return (bits[e >> 5] >> (e & 31)) & 1u; }
};

// Device-resident cache state of a layer stack. Only the routing kernel
// (staging) and the retention kernel (commit) change it, both on the compute
// stream, so every layer sees the previous layer's result in stream order.
struct CacheHdr {
  int32_t free_top;    // free slots: free_list[0, free_top)
  int32_t staged_n;    // misses of the layer in flight, each given a free slot
  int32_t route_bad;   // the layer in flight staged nothing and commits nothing
  int32_t fault;       // sticky: 1 no free slot for a miss, 2 free list overflow,
                       // 4 retained expert without a slot
  int32_t staged_exp[kMaxExperts];
  int32_t staged_slot[kMaxExperts];
};

// Smoothed statistics of a layer for the layer-adaptive sizing: activation
// ratio a and cache utilisation u (float64 moving averages).
struct LayerStat {
  double a, u;
  int32_t has_a, has_u;
};

struct CacheView {
  CacheHdr* hdr;
  int32_t* slot_of;        // [L][E] slot of a resident or staged expert, else -1
  ExpertMask* res;         // [L] committed resident set R
  ExpertMask* res_before;  // [L] R when the layer was last routed
  int32_t* last_counts;    // [L][kCountsPerLayer] n_active, n_hits, n_misses, |R|, experts
                           // transferred at the previous iteration, of them reused now
  int32_t* free_list;      // [n_slots]
  int32_t* cap;            // [L] capacity of each layer now
  LayerStat* stat;         // [L] smoothed statistics (updated only when adapt != 0)
  int adapt;
  int n_slots;
  int policy;              // retention key: 0 priority, 1 LRU, 2 LFU
  int32_t* iters;          // [L] iterations of each layer (LRU / LFU history)
  int32_t* last_use;       // [L][E] layer iteration of the last activation (0: never)
  uint64_t* freq;          // [L][E] routes so far
  ExpertMask* prev_miss;   // [L] misses transferred at the layer's previous iteration
  ExpertMask* cpu_exec;    // [L] misses of the layer in flight executed on the CPU (not
                           // retention candidates); cleared by the retention
};

constexpr int kCountsPerLayer = 8;

constexpr int kMaxAdaptLayers = 1024;

// One routing call, written by the permute stage into a device ring at
// seq % kStatsRing; the host copies records out at its synchronisation points.
struct RouteStats {
  int32_t layer;
  int32_t n_active;
  int32_t n_hits;
  int32_t n_misses;
  int32_t n_resident;
  int32_t hit_rows;
  int32_t miss_rows;
  int32_t n_staged;
  int32_t bad;         // non-finite logit, or no free slot: nothing staged
  int32_t n_hit_items;
  int32_t n_miss_items;
  int32_t n_dense;     // experts with dense items (at least kDenseMinRows rows)
  int32_t n_dense_hits;
  int32_t dense_rows;
  int32_t dense_hit_rows;
  int32_t n_dense_items;
  int32_t prev_xfer;   // experts transferred at the layer's previous iteration
  int32_t reused_xfer; // of them retained and activated now
  int32_t ideal_hits;  // the clairvoyant bound min(C_l, |A|)
  int32_t seq;
};

// Staged misses and the record of the last routing call, for host-issued
// copies: written by the permute stage into coherent pinned host memory when
// asked (fields, system-scope fence, then seq).
struct StagedList {
  RouteStats rec;
  int32_t exp[kMaxExperts];
  int32_t slot[kMaxExperts];
  int32_t seq;
};

// Written by the retention kernel into device memory, one per layer.
struct RetainOut {
  uint32_t retained[kMaxExperts / 32];  // bit e: expert e stays cached
  int32_t bad_conf;    // a confidence outside [0, 1] was seen: nothing changed
  int32_t n_retained;
  int32_t seq;
  int32_t pad;
};

// One grouped-GEMM work item: rows [row_begin, row_begin + rows) of the
// expert-sorted route order, all routed to `expert`.
struct WorkItem {
  int32_t expert;
  int32_t row_begin;
  int32_t rows;
  int32_t pad;   // a hit's cache slot (fixed until the layer's retention), -1 for a miss
};

// Host-to-device transfer of the staged misses done by workgroups of a GEMM
// launch: bytes [off, off + len) of every staged expert's host block into its
// slot. Workgroups [0, nblk) of the launch copy; the GEMM tiles follow.
struct FetchArgs {
  const uint64_t* host_addr;  // [E] device-visible address of each expert's host block
  const CacheHdr* hdr;        // staged list
  int64_t off, len;
  int nblk;
  int E;
};

// Arguments of a grouped-GEMM launch. Work items: hits are items
// [0, c0), misses [c0, c0 + c1) with (c0, c1) = item_counts on the device;
// `which` selects them. With n_items_host >= 0 the host's (item_base,
// n_items_host) are used instead. max_items bounds the count and sizes the
// grid (capped at max_grid workgroups; tiles beyond are looped over).
struct FfnLaunch {
  const void* pool;
  int64_t slot_bytes;
  const int32_t* slot_of;  // [E] of the layer
  int n_slots;
  const WorkItem* items;
  const int32_t* item_counts;
  int which;
  int item_base;
  int n_items_host;
  int max_items;
  int max_grid;
  const void* src;        // up: x [T][H]; down: h [T*k][I]
  const int32_t* perm;    // up: route of each sorted position (token = route / k)
  int k, H, I;
  void* hout;             // up: h [T*k][I]
  float* oout;            // down: O [T*k][H]
  FetchArgs fetch;
  int64_t src_bytes;      // dense launches: bytes of src (below 2^31)
};

// Every launcher takes optional (ev0, ev1): if non-null they record the
// kernel's start and end on the dispatch itself (no extra stream packets).

// The gate GEMM in front of K1: logits [T][E] fp32 = x [T][H] . wg [E][H]^T
// (bf16 or fp32 inputs, fp32 accumulation in a fixed order).
hipError_t launch_router_logits(bool bf16, const void* x, const void* wg, int T, int E, int H,
                                float* logits, hipEvent_t ev0, hipEvent_t ev1, hipStream_t s);

// K1: top-k + fp64 gates: one wavefront per token, or for large blocks one
// token per lane.
// block_tokens > 0: the T tokens are blocks of that many, and a non-finite
// logit of token t sets bad_flag[t / block_tokens] (else bad_flag[0]).
hipError_t launch_route_topk(const float* logits, int T, int E, int k, int32_t* topk_idx,
                             float* gates, int32_t* bad_flag, hipEvent_t ev0, hipEvent_t ev1,
                             hipStream_t s, int block_tokens = 0);

// Outputs of the permute stage for one layer.
struct PermuteOut {
  int32_t* counts;
  int32_t* offsets;
  int32_t* perm;
  int32_t* inv_perm;
  WorkItem* items;
  int32_t* item_counts;   // [2] hit items, miss items
  WorkItem* dense_items;  // experts with at least dense_min rows (0: none)
  int32_t* dense_counts;  // [2] items of kDenseRows rows, shorter items
  int dense_min;
  RouteStats* ring;       // device ring of routing records
  StagedList* staged;     // pinned, or null
  const float* gates;     // the layer's gates (read when routes are published)
  int32_t* pub_topk;      // pinned [T*k]: with `staged`, the routes are published too
  float* pub_gates;       //   (cooperative compensation), or null
  int layer, E, seq;
  CacheView cv;           // cv.hdr null: no expert cache (routing and permutation only:
                          // no staging, work items, records or cache-state writes)
  int32_t* bad_out = nullptr;  // without a cache: 1 if a logit was non-finite, else 0
};

// K2: histogram, offsets, stable permutation, hit-first work list, and the
// staging of the misses into free slots (device cache state); one workgroup.
hipError_t launch_permute(const int32_t* topk_idx, int T, int k, int32_t* bad_flag,
                          const PermuteOut& o, hipEvent_t ev0, hipEvent_t ev1, hipStream_t s);

// K2 over many workgroups for large blocks (permute_chunked true): a counting
// launch over chunks of 512 tokens, a planning launch of one workgroup, then a
// ranking launch over the chunks. chunk_base: [permute_chunks(T)][E] ints of
// scratch.
bool permute_chunked(int T);
int permute_chunks(int T);
hipError_t launch_permute_chunked(const int32_t* topk_idx, int T, int k, int32_t* bad_flag,
                                  int32_t* chunk_base, const PermuteOut& o, hipEvent_t ev0,
                                  hipEvent_t ev1, hipStream_t s);

// K2 over B independent blocks of T tokens without a cache (o.cv.hdr null):
// a counting launch over (chunk, block), a planning launch of one workgroup
// per block and a ranking launch over (chunk, block); o's outputs advance per
// block (routes by T*k, counts by E, offsets by E+1, bad_out by 1).
// bad_flag: [B] non-finite flags of the top-k launch; chunk_base:
// [B][permute_chunks(T)][E] scratch.
hipError_t launch_permute_batch(const int32_t* topk_idx, int B, int T, int k,
                                const int32_t* bad_flag, int32_t* chunk_base, const PermuteOut& o,
                                hipStream_t s);

// K1+K2 as one launch for blocks with T*k <= 1024 (route_fused true): the
// last workgroup to finish routing permutes. sync: 2 device ints, zero
// before the first launch; the kernel leaves them zero.
bool route_fused(int T, int k);
hipError_t launch_route_fused(const float* logits, int T, int k, int32_t* topk_idx, float* gates,
                              int32_t* sync, const PermuteOut& o, hipEvent_t ev0, hipEvent_t ev1,
                              hipStream_t s);

// K4a: grouped gate/up GEMM with SiLU*up epilogue (h = silu(W1 x) * (W3 x)).
hipError_t launch_ffn_up(bool bf16, const FfnLaunch& a, hipEvent_t ev0, hipEvent_t ev1,
                         hipStream_t s);

// K4b: grouped down GEMM (O = W2 h, fp32).
hipError_t launch_ffn_down(bool bf16, const FfnLaunch& a, hipEvent_t ev0, hipEvent_t ev1,
                           hipStream_t s);

// The hit experts' down GEMM with the transfer of the misses' down weights
// (d.fetch), and the misses' gate/up GEMM (u), in one launch.
hipError_t launch_ffn_mix(bool bf16, const FfnLaunch& d, const FfnLaunch& u, hipEvent_t ev0,
                          hipEvent_t ev1, hipStream_t s);

// Dense tiles (bf16; H and I multiples of 256; src below 2 GiB) for experts
// with at least kDenseMinRows routed rows, hits and misses alike, once all
// their weights are in their slots. Items of kDenseRows rows first
// (item_counts[0] of them), then one shorter item per expert
// (item_counts[1]); up: 128 features x 256 rows per workgroup, down: 256 x
// 256. Those experts have no items in the streaming lists. The threshold is
// one row above a streaming work item: an expert the streaming kernels would
// split into two items (each reading all of its weights) runs as one dense
// item instead.
constexpr int kDenseMinRows = kItemRows + 1;
constexpr int kDenseRows = 256;
hipError_t launch_ffn_dense(bool up, const FfnLaunch& a, hipEvent_t ev0, hipEvent_t ev1,
                            hipStream_t s);

// Transfer of the staged misses alone (no GEMM tiles).
hipError_t launch_fetch(const void* pool, int64_t slot_bytes, int n_slots, const FetchArgs& f,
                        hipEvent_t ev0, hipEvent_t ev1, hipStream_t s);

// K6 arguments: priority numerators (per-expert segment sums), Top-C
// retention and the commit into the device cache state of `layer`.
struct ScoreArgs {
  const float* gates;
  const float* conf;
  const int32_t* topk_idx;
  const int32_t* counts;
  int T, k, E, layer, seq;     // the capacity is cv.cap[layer]
  CacheView cv;
  uint64_t* score_out;
  RetainOut* out;         // device, one per layer
  uint64_t* key_out;      // [E] retention key of each expert (S under the priority policy)
  int parts;              // scoring workgroups: score_parts(T, k)
  unsigned long long* acc;  // [E] zero between launches (several parts only)
  int32_t* acc_sync;        // [2]: unused, non-finite confidence flag; zero between layers
  int reject = 0;         // 1: commit nothing (R stays, staged misses return their slots);
                          // with T = 0 no route or confidence is read
};

// Workgroups that score a block of T tokens (one up to 8192 routes).
int score_parts(int T, int k);

// K5 arguments: y[t] = sum_j gate[t][j] * O[inv_perm[t*k + j]], fp32, rounded
// once to dtype.
struct CombineArgs {
  const float* O;
  const float* gates;
  const int32_t* inv_perm;
  int T, k, H;
  void* y;
};

// K6; blocks of more than 8192 routes (a.parts > 1) take a second, one-workgroup
// commit launch (ev1 is recorded after it).
hipError_t launch_score_retain(const ScoreArgs& a, hipEvent_t ev0, hipEvent_t ev1, hipStream_t s);

// Layer-adaptive re-sizing of every layer's capacity from the smoothed
// statistics, and the eviction of the lowest-priority residents of layers
// left over their new capacity (L <= kMaxAdaptLayers).
struct AdaptArgs {
  CacheView cv;
  const uint64_t* score;  // [L][E] keys of each layer's last retention
  int L, E, c_total;
};
hipError_t launch_layer_adapt(const AdaptArgs& a, hipEvent_t ev0, hipEvent_t ev1, hipStream_t s);

// Cooperative compensation: the staged misses in `cpu` run on the host CPU.
// Their staging slots return to the free list, they leave the staged list
// (so only the transferred ones are copied) and the previous-transfer mask,
// and the retention of the layer skips them as candidates.
// Text of oled_last_error(NULL): errors of calls without a context.
void set_noctx_error(const char* msg);

hipError_t launch_coop_unstage(const CacheView& cv, int layer, int E, const ExpertMask& cpu,
                               hipStream_t s);

// K5 and K6 in one launch (the layer's last), plus the commit launch when a.parts > 1.
hipError_t launch_combine_score(bool bf16, const CombineArgs& c, const ScoreArgs& a,
                                hipEvent_t ev0, hipEvent_t ev1, hipStream_t s);

}  // namespace oled
