// K6 reuse priority and retention of one layer (OLED-MoE Sec. 4.3 priority
// p_e = sum_t g_te psi(c_t) / normaliser with psi(c) = c, stale residents at
// zero; Sec. 4.2 retention R' = Top_C(R u G, p) with G = M), committed into
// the device-resident cache state: slots of evicted residents and of misses
// not retained return to the free list, retained misses keep their slot.
//
// Priority numerators are exact integers: g and c are fp32, so g*c is exact
// in fp64, scaling by 2^48 is exact and the floor is exact; the per-expert
// segment sums are accumulated with integer LDS atomics, so any order gives
// the same bits. Ranking by the numerator equals ranking by p_e (one
// normaliser per layer).
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include "kernels.h"

namespace oled {
namespace {

constexpr int kThreads = 256;

__device__ __forceinline__ bool ranks_above(unsigned long long sa, bool ra, int a,
                                            unsigned long long sb, bool rb, int b) {
  return sa > sb || (sa == sb && (ra > rb || (ra == rb && a < b)));
}

__global__ __launch_bounds__(kThreads) void k_score_retain(
    const float* __restrict__ gates, const float* __restrict__ conf,
    const int32_t* __restrict__ topk_idx, const int32_t* __restrict__ counts, int T, int k, int E,
    int C, int layer, CacheView cv, uint64_t* __restrict__ score_out, RetainOut* __restrict__ out,
    int seq) {
  __shared__ unsigned long long s_S[kMaxExperts];
  __shared__ uint32_t s_rc[kMaxExperts];  // bit 1: previously resident, bit 0: candidate
  __shared__ int32_t s_rank[kMaxExperts];
  __shared__ uint32_t s_res[kMaxExperts / 32];
  __shared__ int32_t s_bad;
  const int tid = threadIdx.x;
  if (tid < kMaxExperts / 32) s_res[tid] = cv.res[layer].bits[tid];
  if (tid == 0) s_bad = 0;
  __syncthreads();
  for (int e = tid; e < kMaxExperts; e += kThreads) {
    s_S[e] = 0ull;
    s_rank[e] = 0;
    const bool r = e < E && ((s_res[e >> 5] >> (e & 31)) & 1u);
    const bool c = e < E && (r || counts[e] > 0);
    s_rc[e] = (r ? 2u : 0u) | (c ? 1u : 0u);
  }
  __syncthreads();

  // Segment sums per expert: each route's term is added to its expert's
  // segment with an integer LDS atomic. The routes are read in token order,
  // so the expert id, gate and confidence loads of a route are independent.
  int bad = 0;
  const int R = T * k;
  for (int r = tid; r < R; r += kThreads) {
    const int e = topk_idx[r];
    const float g = gates[r];
    const float c = conf[r / k];
    if (!(c >= 0.f && c <= 1.f)) {
      bad = 1;
      continue;
    }
    const double prod = static_cast<double>(g) * static_cast<double>(c);
    atomicAdd(&s_S[e], static_cast<unsigned long long>(floor(prod * 0x1p48)));
  }
  if (bad) atomicOr(&s_bad, 1);
  __syncthreads();

  // Top-C over candidates R u A by (S desc, previously resident first, id
  // asc): rank[e] = number of candidates above e. Thread pairs (e, quarter of
  // the candidates) count with broadcast LDS reads; LDS atomics sum the parts.
  const int fq = (E + 3) >> 2;
  for (int idx = tid; idx < 4 * E; idx += kThreads) {
    const int e = idx % E, part = idx / E;
    const unsigned long long se = s_S[e];
    const bool re = s_rc[e] & 2u;
    int cnt = 0;
    const int f1 = min(E, (part + 1) * fq);
    for (int f = part * fq; f < f1; ++f) {
      const uint32_t rcf = s_rc[f];
      cnt += ((rcf & 1u) && ranks_above(s_S[f], rcf & 2u, f, se, re, e)) ? 1 : 0;
    }
    atomicAdd(&s_rank[e], cnt);
  }
  __syncthreads();
  if (tid >= 64) return;

  // One wavefront commits: the retained set becomes R (or, if the confidence
  // or the routing was bad, R stays and the staged misses are dropped); every
  // slot no longer held returns to the free list, in expert order.
  const int lane = tid;
  constexpr int Q = kMaxExperts / 64;
  CacheHdr* hdr = cv.hdr;
  const bool commit = !s_bad && !hdr->route_bad;
  int32_t* slot_row = cv.slot_of + static_cast<size_t>(layer) * E;
  int top = hdr->free_top;
  int fault = 0;
  uint32_t word[kMaxExperts / 32];
#pragma unroll
  for (int w = 0; w < kMaxExperts / 32; ++w) word[w] = 0u;
  int kept = 0;
#pragma unroll
  for (int q = 0; q < Q; ++q) {
    const int e = lane + 64 * q;
    const bool was = e < E && (s_rc[e] & 2u);
    bool keep = commit ? (e < E && (s_rc[e] & 1u) && s_rank[e] < C) : was;
    const int sl = e < E ? slot_row[e] : -1;
    if (keep && sl < 0) {
      fault |= 4;
      keep = false;
    }
    if (e < E) score_out[e] = s_S[e];
    const bool release = sl >= 0 && !keep;
    const uint64_t rel = __ballot(release);
    const int pos = top + __popcll(rel & ((1ull << lane) - 1ull));
    if (release) {
      if (pos < cv.n_slots) cv.free_list[pos] = sl;
      slot_row[e] = -1;
    }
    top += __popcll(rel);
    const uint64_t ballot = __ballot(keep);
    word[2 * q] = static_cast<uint32_t>(ballot);
    word[2 * q + 1] = static_cast<uint32_t>(ballot >> 32);
    kept += __popcll(ballot);
  }
  if (top > cv.n_slots) {
    fault |= 2;
    top = cv.n_slots;
  }
  fault = (__ballot(fault & 4) ? 4 : 0) | (fault & 2);
  uint32_t my_word = 0u;
#pragma unroll
  for (int w = 0; w < kMaxExperts / 32; ++w)
    if (lane == w) my_word = word[w];
  if (lane < kMaxExperts / 32) {
    cv.res[layer].bits[lane] = my_word;
    out->retained[lane] = my_word;
  }
  if (lane == 0) {
    hdr->free_top = top;
    hdr->staged_n = 0;
    hdr->route_bad = 0;
    if (fault) hdr->fault |= fault;
    out->bad_conf = s_bad;
    out->n_retained = kept;
  }
  // publish: fields, system-scope fence, then seq
  __threadfence_system();
  if (lane == 0) *reinterpret_cast<volatile int32_t*>(&out->seq) = seq;
}

}  // namespace

hipError_t launch_score_retain(const float* gates, const float* conf, const int32_t* topk_idx,
                               const int32_t* counts, int T, int k, int E, int C, int layer,
                               const CacheView& cv, uint64_t* score_out, RetainOut* out, int seq,
                               hipEvent_t ev0, hipEvent_t ev1, hipStream_t s) {
  hipExtLaunchKernelGGL(k_score_retain, dim3(1), dim3(kThreads), 0, s, ev0, ev1, 0, gates, conf,
                        topk_idx, counts, T, k, E, C, layer, cv, score_out, out, seq);
  return hipGetLastError();
}

}  // namespace oled
