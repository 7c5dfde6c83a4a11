// K6 reuse priority and retention of one layer (OLED-MoE Sec. 4.3 priority
// p_e = sum_t g_te psi(c_t) / normaliser with psi(c) = c, stale residents at
// zero; Sec. 4.2 retention R' = Top_C(R u G, p) with G = M).
//
// Priority numerators are exact integers: g and c are fp32, so g*c is exact
// in fp64, scaling by 2^48 is exact and the floor is exact; the per-expert sum
// is a segmented reduction over the expert-sorted route order with integer
// LDS atomics between segments, so any order gives the same bits. Ranking by
// the numerator equals ranking by p_e (one normaliser per layer).
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
    const int32_t* __restrict__ perm, const int32_t* __restrict__ offsets,
    const int32_t* __restrict__ counts, int T, int k, int E, int C, ExpertMask resident,
    uint64_t* __restrict__ score_out, RetainOut* __restrict__ out, int seq) {
  __shared__ unsigned long long s_S[kMaxExperts];
  __shared__ int32_t s_off[kMaxExperts + 1];
  __shared__ int32_t s_bad;
  const int tid = threadIdx.x;
  for (int e = tid; e < kMaxExperts; e += kThreads) s_S[e] = 0ull;
  for (int e = tid; e <= E; e += kThreads) s_off[e] = offsets[e];
  if (tid == 0) s_bad = 0;
  __syncthreads();

  // segmented reduction: thread tid owns sorted positions [p0, p1)
  const int R = T * k;
  const int per = (R + kThreads - 1) / kThreads;
  const int p0 = tid * per;
  const int p1 = min(R, p0 + per);
  if (p0 < p1) {
    int lo = 0, hi = E - 1;  // last expert whose segment starts at or before p0
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (s_off[mid] <= p0) lo = mid; else hi = mid - 1;
    }
    int e = lo;
    unsigned long long acc = 0ull;
    int bad = 0;
    for (int p = p0; p < p1; ++p) {
      while (p >= s_off[e + 1]) {
        if (acc) atomicAdd(&s_S[e], acc);
        acc = 0ull;
        ++e;
      }
      const int r = perm[p];
      const float c = conf[r / k];
      if (!(c >= 0.f && c <= 1.f)) {
        bad = 1;
        continue;
      }
      const double prod = static_cast<double>(gates[r]) * static_cast<double>(c);
      acc += static_cast<unsigned long long>(floor(prod * 0x1p48));
    }
    if (acc) atomicAdd(&s_S[e], acc);
    if (bad) atomicOr(&s_bad, 1);
  }
  __syncthreads();
  if (tid >= 64) return;

  // Top-C over candidates R u A by (S desc, previously resident first, id
  // asc): one wavefront, lane l holds experts l, l+64, ...; a candidate's rank
  // counts the candidates above it, broadcast from registers lane by lane.
  const int lane = tid;
  constexpr int Q = kMaxExperts / 64;
  unsigned long long key_s[Q];
  uint32_t key_rc[Q];  // bit 1: previously resident, bit 0: candidate
  int rank[Q];
#pragma unroll
  for (int q = 0; q < Q; ++q) {
    const int e = lane + 64 * q;
    key_s[q] = s_S[e];
    const bool r = e < E && resident.test(e);
    const bool c = e < E && (r || counts[e] > 0);
    key_rc[q] = (r ? 2u : 0u) | (c ? 1u : 0u);
    rank[q] = 0;
  }
  const int nq = (E + 63) >> 6;
  for (int qf = 0; qf < Q; ++qf) {
    if (qf >= nq) break;
    for (int src = 0; src < 64; ++src) {
      const uint32_t rcf = __builtin_amdgcn_readlane(key_rc[qf], src);
      if (!(rcf & 1u)) continue;  // not a candidate (uniform branch)
      const uint32_t lo = __builtin_amdgcn_readlane(static_cast<uint32_t>(key_s[qf]), src);
      const uint32_t hi = __builtin_amdgcn_readlane(static_cast<uint32_t>(key_s[qf] >> 32), src);
      const unsigned long long sf = (static_cast<unsigned long long>(hi) << 32) | lo;
      const int f = src + 64 * qf;
#pragma unroll
      for (int q = 0; q < Q; ++q)
        rank[q] += ranks_above(sf, rcf & 2u, f, key_s[q], key_rc[q] & 2u, lane + 64 * q) ? 1 : 0;
    }
  }
  uint32_t word[kMaxExperts / 32];
#pragma unroll
  for (int w = 0; w < kMaxExperts / 32; ++w) word[w] = 0u;
  int kept = 0;
#pragma unroll
  for (int q = 0; q < Q; ++q) {
    const int e = lane + 64 * q;
    const bool keep = (key_rc[q] & 1u) && rank[q] < C;
    if (e < E) score_out[e] = key_s[q];
    const uint64_t ballot = __ballot(keep);
    word[2 * q] = static_cast<uint32_t>(ballot);
    word[2 * q + 1] = static_cast<uint32_t>(ballot >> 32);
    kept += __popcll(ballot);
  }
  // one wavefront publishes the result: fields, system-scope fence, then seq
  uint32_t my_word = 0u;
#pragma unroll
  for (int w = 0; w < kMaxExperts / 32; ++w)
    if (lane == w) my_word = word[w];
  if (lane < kMaxExperts / 32) out->retained[lane] = my_word;
  if (lane == 0) {
    out->bad_conf = s_bad;
    out->n_retained = kept;
  }
  __threadfence_system();
  if (lane == 0) *reinterpret_cast<volatile int32_t*>(&out->seq) = seq;
}

}  // namespace

hipError_t launch_score_retain(const float* gates, const float* conf, const int32_t* perm,
                               const int32_t* offsets, const int32_t* counts, int T, int k, int E,
                               int C, const ExpertMask& resident, uint64_t* score_out,
                               RetainOut* out, int seq, hipEvent_t ev0, hipEvent_t ev1,
                               hipStream_t s) {
  hipExtLaunchKernelGGL(k_score_retain, dim3(1), dim3(kThreads), 0, s, ev0, ev1, 0, gates, conf,
                        perm, offsets, counts, T, k, E, C, resident, score_out, out, seq);
  return hipGetLastError();
}

}  // namespace oled
