// K6 reuse priority and retention of one layer (OLED-MoE Sec. 4.3 priority
// p_e = sum_t g_te psi(c_t) / normaliser with psi(c) = c, stale residents at
// zero; Sec. 4.2 retention R' = Top_C(R u G, p) with G = M).
//
// Priority numerators are exact integers: g and c are fp32, so g*c is exact
// in fp64, scaling by 2^48 is exact and the floor is exact; the per-expert sum
// is a segmented reduction over the expert-sorted route order with integer
// LDS atomics between segments, so any order gives the same bits. Ranking by
// the numerator equals ranking by p_e (one normaliser per layer).
#include <hip/hip_runtime.h>

#include "kernels.h"

namespace oled {
namespace {

constexpr int kThreads = 256;

__global__ __launch_bounds__(kThreads) void k_score_retain(
    const float* __restrict__ gates, const float* __restrict__ conf,
    const int32_t* __restrict__ perm, const int32_t* __restrict__ offsets,
    const int32_t* __restrict__ counts, int T, int k, int E, int C, ExpertMask resident,
    uint64_t* __restrict__ score_out, RetainOut* __restrict__ out, int seq) {
  __shared__ unsigned long long s_S[kMaxExperts];
  __shared__ int32_t s_off[kMaxExperts + 1];
  __shared__ int32_t s_bad;
  __shared__ int32_t s_kept;
  const int tid = threadIdx.x;
  for (int e = tid; e < kMaxExperts; e += kThreads) s_S[e] = 0ull;
  for (int e = tid; e <= E; e += kThreads) s_off[e] = offsets[e];
  if (tid == 0) {
    s_bad = 0;
    s_kept = 0;
  }
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

  // Top-C over candidates R u A by (S desc, previously resident first, id asc)
  for (int e = tid; e < E; e += kThreads) {
    const bool res_e = resident.test(e);
    const bool cand = res_e || counts[e] > 0;
    const unsigned long long se = s_S[e];
    int rank = 0;
    for (int f = 0; f < E; ++f) {
      const bool res_f = resident.test(f);
      if (!(res_f || counts[f] > 0)) continue;
      const unsigned long long sf = s_S[f];
      const bool better = sf > se || (sf == se && (res_f && !res_e)) ||
                          (sf == se && res_f == res_e && f < e);
      rank += better ? 1 : 0;
    }
    const bool keep = cand && rank < C;
    out->retained[e] = keep ? 1 : 0;
    score_out[e] = se;
    if (keep) atomicAdd(&s_kept, 1);
  }
  __syncthreads();
  if (tid == 0) {
    out->bad_conf = s_bad;
    out->n_retained = s_kept;
    __threadfence_system();
    out->seq = seq;
  }
}

}  // namespace

hipError_t launch_score_retain(const float* gates, const float* conf, const int32_t* perm,
                               const int32_t* offsets, const int32_t* counts, int T, int k, int E,
                               int C, const ExpertMask& resident, uint64_t* score_out,
                               RetainOut* out, int seq, hipStream_t s) {
  hipLaunchKernelGGL(k_score_retain, dim3(1), dim3(kThreads), 0, s, gates, conf, perm, offsets,
                     counts, T, k, E, C, resident, score_out, out, seq);
  return hipGetLastError();
}

}  // namespace oled
