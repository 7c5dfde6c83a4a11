// K1 top-k routing and K2 histogram / prefix-sum / stable permutation for one
// denoising block (OLED-MoE Sec. 4.1: the gate yields routed expert ids and
// gate scores for every token of the block; Sec. 4.2: the active set A).
#include <hip/hip_runtime.h>

#include "kernels.h"

namespace oled {
namespace {

__device__ __forceinline__ uint64_t wave_max_u64(uint64_t v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    const uint32_t lo = __shfl_xor(static_cast<uint32_t>(v), off);
    const uint32_t hi = __shfl_xor(static_cast<uint32_t>(v >> 32), off);
    const uint64_t o = (static_cast<uint64_t>(hi) << 32) | lo;
    v = o > v ? o : v;
  }
  return v;
}

// Orderable 64-bit key: (logit as an order-preserving uint32, ~expert id).
// The larger key is the larger logit, and on equal logits the lower id.
__device__ __forceinline__ uint64_t route_key(float v, int e) {
  uint32_t b = __float_as_uint(v);
  if ((b << 1) == 0u) b = 0u;  // -0.0 ranks equal to +0.0
  const uint32_t ord = (b & 0x80000000u) ? ~b : (b | 0x80000000u);
  return (static_cast<uint64_t>(ord) << 32) | (0xFFFFFFFFu - static_cast<uint32_t>(e));
}

__device__ __forceinline__ float key_value(uint64_t key) {
  const uint32_t ord = static_cast<uint32_t>(key >> 32);
  return __uint_as_float((ord & 0x80000000u) ? (ord & 0x7FFFFFFFu) : ~ord);
}

// One wavefront per token; lane l holds logits l, l+64, ... (EPL per lane).
// k rounds of a wavefront arg-max over the keys, then the gates in fp64:
// e_j = exp(l_j - l_0), s = e_0 + ... + e_{k-1} in slot order, g_j = fl32(e_j / s).
template <int EPL>
__global__ __launch_bounds__(256) void k_route_topk(const float* __restrict__ logits, int T, int E,
                                                    int k, int32_t* __restrict__ topk_idx,
                                                    float* __restrict__ gates,
                                                    int32_t* __restrict__ bad_flag) {
  const int lane = threadIdx.x & 63;
  const int nwaves = gridDim.x * 4;
  for (int t = blockIdx.x * 4 + (threadIdx.x >> 6); t < T; t += nwaves) {
    const float* row = logits + static_cast<size_t>(t) * E;
    uint64_t key[EPL];
    int bad = 0;
#pragma unroll
    for (int q = 0; q < EPL; ++q) {
      const int e = lane + 64 * q;
      key[q] = 0;
      if (e < E) {
        const float v = row[e];
        bad |= !__builtin_isfinite(v);
        key[q] = route_key(v, e);
      }
    }
    if (__any(bad) && lane == 0) atomicOr(bad_flag, 1);

    float sel_v[kMaxTopK];
    int32_t sel_e[kMaxTopK];
#pragma unroll
    for (int j = 0; j < kMaxTopK; ++j) {
      sel_v[j] = 0.f;
      sel_e[j] = 0;
      if (j < k) {
        uint64_t best = 0;
#pragma unroll
        for (int q = 0; q < EPL; ++q) best = key[q] > best ? key[q] : best;
        const uint64_t m = wave_max_u64(best);
#pragma unroll
        for (int q = 0; q < EPL; ++q)
          if (key[q] == m) key[q] = 0;  // keys are unique: exactly one owner
        sel_v[j] = key_value(m);
        sel_e[j] = static_cast<int32_t>(0xFFFFFFFFu - static_cast<uint32_t>(m));
      }
    }
    double ex[kMaxTopK];
    double s = 0.0;
#pragma unroll
    for (int j = 0; j < kMaxTopK; ++j) {
      ex[j] = 0.0;
      if (j < k) {
        ex[j] = exp(static_cast<double>(sel_v[j]) - static_cast<double>(sel_v[0]));
        s += ex[j];
      }
    }
#pragma unroll
    for (int j = 0; j < kMaxTopK; ++j) {
      if (j < k && lane == j) {
        topk_idx[static_cast<size_t>(t) * k + j] = sel_e[j];
        gates[static_cast<size_t>(t) * k + j] = static_cast<float>(ex[j] / s);
      }
    }
  }
}

constexpr int kPermThreads = 1024;
constexpr int kChunkWords = 16;               // bitmask words per expert per chunk
constexpr int kChunkTokens = kChunkWords * 32;

// Single workgroup. Pass 1: per-expert counts (LDS atomics). Scan: offsets
// and the work list, hit experts first. Pass 2, chunk by chunk of 512 tokens:
// a per-expert token bitmask (the ballot of the tokens that chose the
// expert), a running popcount prefix per 32-token word, and each route's
// stable position = offsets[e] + tokens before it that chose e.
__global__ __launch_bounds__(kPermThreads) void k_permute(
    const int32_t* __restrict__ topk_idx, int T, int k, int E, ExpertMask resident,
    int32_t* __restrict__ counts, int32_t* __restrict__ offsets, int32_t* __restrict__ perm,
    int32_t* __restrict__ inv_perm, WorkItem* __restrict__ items, int32_t* __restrict__ bad_flag,
    RouteSummary* __restrict__ summary, int seq) {
  __shared__ int32_t s_cnt[kMaxExperts];
  __shared__ int32_t s_off[kMaxExperts + 1];
  __shared__ int32_t s_item_base[kMaxExperts];
  __shared__ int32_t s_run[kMaxExperts];
  __shared__ int32_t s_tot[2];
  __shared__ uint32_t s_mask[kMaxExperts * kChunkWords];
  __shared__ int32_t s_pre[kMaxExperts * kChunkWords];

  const int tid = threadIdx.x;
  const int R = T * k;
  for (int e = tid; e < kMaxExperts; e += kPermThreads) s_cnt[e] = 0;
  __syncthreads();
  for (int r = tid; r < R; r += kPermThreads) atomicAdd(&s_cnt[topk_idx[r]], 1);
  __syncthreads();

  if (tid < 64) {  // wave 0: scans over experts, 4 per lane
    const int lane = tid;
    int c[4], nh[4], nm[4];
    int sc = 0, sh = 0, sm = 0;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int e = 4 * lane + q;
      c[q] = e < E ? s_cnt[e] : 0;
      const int ni = (c[q] + kItemRows - 1) / kItemRows;
      const bool res = e < E && resident.test(e);
      nh[q] = res ? ni : 0;
      nm[q] = res ? 0 : ni;
      sc += c[q];
      sh += nh[q];
      sm += nm[q];
    }
    int ic = sc, ih = sh, im = sm;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
      const int tc = __shfl_up(ic, off), th = __shfl_up(ih, off), tm = __shfl_up(im, off);
      if (lane >= off) {
        ic += tc;
        ih += th;
        im += tm;
      }
    }
    const int tot_hit = __shfl(ih, 63);
    int xc = ic - sc, xh = ih - sh, xm = im - sm;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int e = 4 * lane + q;
      if (e < E) {
        s_off[e] = xc;
        s_item_base[e] = (nh[q] > 0) ? xh : tot_hit + xm;
      }
      xc += c[q];
      xh += nh[q];
      xm += nm[q];
    }
    if (lane == 63) {
      s_off[E] = ic;
      s_tot[0] = ih;
      s_tot[1] = im;
    }
  }
  __syncthreads();

  for (int e = tid; e < E; e += kPermThreads) {
    const int c = s_cnt[e];
    counts[e] = c;
    offsets[e] = s_off[e];
    summary->counts[e] = c;
    s_run[e] = s_off[e];
    const int base = s_item_base[e];
    for (int m = 0; m * kItemRows < c; ++m) {
      WorkItem it;
      it.expert = e;
      it.row_begin = s_off[e] + m * kItemRows;
      it.rows = min(kItemRows, c - m * kItemRows);
      it.pad = 0;
      items[base + m] = it;
    }
  }
  if (tid == 0) offsets[E] = s_off[E];

  for (int t0 = 0; t0 < T; t0 += kChunkTokens) {
    const int t1 = min(T, t0 + kChunkTokens);
    for (int i = tid; i < E * kChunkWords; i += kPermThreads) s_mask[i] = 0u;
    __syncthreads();
    for (int r = t0 * k + tid; r < t1 * k; r += kPermThreads) {
      const int e = topk_idx[r];
      const int lt = r / k - t0;
      atomicOr(&s_mask[e * kChunkWords + (lt >> 5)], 1u << (lt & 31));
    }
    __syncthreads();
    for (int e = tid; e < E; e += kPermThreads) {
      int run = s_run[e];
#pragma unroll
      for (int w = 0; w < kChunkWords; ++w) {
        s_pre[e * kChunkWords + w] = run;
        run += __popc(s_mask[e * kChunkWords + w]);
      }
      s_run[e] = run;
    }
    __syncthreads();
    for (int r = t0 * k + tid; r < t1 * k; r += kPermThreads) {
      const int e = topk_idx[r];
      const int lt = r / k - t0;
      const int w = lt >> 5;
      const uint32_t below = s_mask[e * kChunkWords + w] & ((1u << (lt & 31)) - 1u);
      const int pos = s_pre[e * kChunkWords + w] + __popc(below);
      perm[pos] = r;
      inv_perm[r] = pos;
    }
    __syncthreads();
  }

  if (tid == 0) {
    summary->n_hit_items = s_tot[0];
    summary->n_miss_items = s_tot[1];
    summary->bad_logits = *bad_flag;
    *bad_flag = 0;
    __threadfence_system();
    summary->seq = seq;
  }
}

}  // namespace

hipError_t launch_route_topk(const float* logits, int T, int E, int k, int32_t* topk_idx,
                             float* gates, int32_t* bad_flag, hipStream_t s) {
  const int blocks = (T + 3) / 4 < 4096 ? (T + 3) / 4 : 4096;
  if (E <= 64)
    hipLaunchKernelGGL(k_route_topk<1>, dim3(blocks), dim3(256), 0, s, logits, T, E, k, topk_idx,
                       gates, bad_flag);
  else if (E <= 128)
    hipLaunchKernelGGL(k_route_topk<2>, dim3(blocks), dim3(256), 0, s, logits, T, E, k, topk_idx,
                       gates, bad_flag);
  else
    hipLaunchKernelGGL(k_route_topk<4>, dim3(blocks), dim3(256), 0, s, logits, T, E, k, topk_idx,
                       gates, bad_flag);
  return hipGetLastError();
}

hipError_t launch_permute(const int32_t* topk_idx, int T, int k, int E, const ExpertMask& resident,
                          int32_t* counts, int32_t* offsets, int32_t* perm, int32_t* inv_perm,
                          WorkItem* items, int32_t* bad_flag, RouteSummary* summary, int seq,
                          hipStream_t s) {
  hipLaunchKernelGGL(k_permute, dim3(1), dim3(kPermThreads), 0, s, topk_idx, T, k, E, resident,
                     counts, offsets, perm, inv_perm, items, bad_flag, summary, seq);
  return hipGetLastError();
}

}  // namespace oled
