// K5 the gate-weighted combine of the layer output and K6 the reuse priority
// and retention of one layer (OLED-MoE Sec. 4.3 priority
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

__device__ __forceinline__ void score_body(const ScoreArgs& a) {
  const float* __restrict__ gates = a.gates;
  const float* __restrict__ conf = a.conf;
  const int32_t* __restrict__ topk_idx = a.topk_idx;
  const int32_t* __restrict__ counts = a.counts;
  const int T = a.T, k = a.k, E = a.E, C = a.C, layer = a.layer;
  const CacheView& cv = a.cv;
  uint64_t* __restrict__ score_out = a.score_out;
  RetainOut* __restrict__ out = a.out;
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
    out->seq = a.seq;
  }
}

__device__ __forceinline__ uint16_t f32_to_bf16_rne(float f) {
  const uint32_t u = __float_as_uint(f);
  return static_cast<uint16_t>((u + 0x7FFFu + ((u >> 16) & 1u)) >> 16);
}

// K5 for 1024 outputs of token t: one thread per 4 consecutive outputs sums
// the token's k routes in slot order in fp32 and rounds once.
template <bool BF16>
__device__ __forceinline__ void combine_body(const CombineArgs& c, int t, int hb) {
  const int h = (hb * 256 + static_cast<int>(threadIdx.x)) * 4;
  if (h >= c.H) return;
  const int k = c.k, H = c.H;
  float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
  for (int j = 0; j < k; ++j) {
    const float gj = c.gates[static_cast<size_t>(t) * k + j];
    const int pos = c.inv_perm[static_cast<size_t>(t) * k + j];
    const float4 o = *reinterpret_cast<const float4*>(c.O + static_cast<size_t>(pos) * H + h);
    acc.x = fmaf(gj, o.x, acc.x);
    acc.y = fmaf(gj, o.y, acc.y);
    acc.z = fmaf(gj, o.z, acc.z);
    acc.w = fmaf(gj, o.w, acc.w);
  }
  if (BF16) {
    uint2 packed;
    packed.x = f32_to_bf16_rne(acc.x) | (static_cast<uint32_t>(f32_to_bf16_rne(acc.y)) << 16);
    packed.y = f32_to_bf16_rne(acc.z) | (static_cast<uint32_t>(f32_to_bf16_rne(acc.w)) << 16);
    *reinterpret_cast<uint2*>(static_cast<uint16_t*>(c.y) + static_cast<size_t>(t) * H + h) = packed;
  } else {
    *reinterpret_cast<float4*>(static_cast<float*>(c.y) + static_cast<size_t>(t) * H + h) = acc;
  }
}

__global__ __launch_bounds__(kThreads) void k_score_retain(ScoreArgs a) { score_body(a); }

// The layer's last launch: workgroup 0 scores and commits the retention,
// workgroups 1.. combine (the two parts touch disjoint data).
template <bool BF16>
__global__ __launch_bounds__(kThreads) void k_combine_score(CombineArgs c, ScoreArgs a) {
  const int b = blockIdx.x;
  if (b == 0) {
    score_body(a);
    return;
  }
  const int hx = (c.H + 1023) / 1024;
  combine_body<BF16>(c, (b - 1) / hx, (b - 1) % hx);
}

}  // namespace

hipError_t launch_score_retain(const ScoreArgs& a, hipEvent_t ev0, hipEvent_t ev1, hipStream_t s) {
  hipExtLaunchKernelGGL(k_score_retain, dim3(1), dim3(kThreads), 0, s, ev0, ev1, 0, a);
  return hipGetLastError();
}

hipError_t launch_combine_score(bool bf16, const CombineArgs& c, const ScoreArgs& a,
                                hipEvent_t ev0, hipEvent_t ev1, hipStream_t s) {
  const int grid = 1 + c.T * ((c.H + 1023) / 1024);
  if (bf16)
    hipExtLaunchKernelGGL(k_combine_score<true>, dim3(grid), dim3(kThreads), 0, s, ev0, ev1, 0, c, a);
  else
    hipExtLaunchKernelGGL(k_combine_score<false>, dim3(grid), dim3(kThreads), 0, s, ev0, ev1, 0, c, a);
  return hipGetLastError();
}

}  // namespace oled
