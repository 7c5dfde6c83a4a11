// K1 top-k routing and K2 histogram / prefix-sum / stable permutation for one
// denoising block (OLED-MoE Sec. 4.1: the gate yields routed expert ids and
// gate scores for every token of the block; Sec. 4.2: the active set A, the
// misses M = A \ R, each given a staging slot in the device cache state).
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include "kernels.h"

namespace oled {
namespace {

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

__device__ __forceinline__ uint64_t bcast_u64(uint64_t v, int lane) {
  const uint32_t lo = __builtin_amdgcn_readlane(static_cast<int>(static_cast<uint32_t>(v)), lane);
  const uint32_t hi = __builtin_amdgcn_readlane(static_cast<int>(static_cast<uint32_t>(v >> 32)), lane);
  return (static_cast<uint64_t>(hi) << 32) | lo;
}

// Routes one token with one wavefront; lane l holds logits l, l+64, ... (EPL
// per lane). Each key's rank is the number of keys above it (all E keys are
// broadcast lane by lane); the keys of rank j < k fill slot j, so the slots
// are ordered by (logit desc, id asc). Slot j's expert and logit pass through
// LDS (s_e, s_v: this wavefront's k entries); lane j < k takes
// e_j = exp(l_j - l_0) in fp64, every lane sums e_0 + ... + e_{k-1} in slot
// order (through s_x), and lane j returns g_j = fl32(e_j / s) and its expert
// (else -1). `bad` collects non-finite logits.
template <int EPL>
__device__ __forceinline__ int route_token(const float* __restrict__ row, int E, int k,
                                           int32_t* s_e, float* s_v, double* s_x,
                                           float* __restrict__ gate_out, int* bad) {
  const int lane = threadIdx.x & 63;
  uint64_t key[EPL];
  int rank[EPL];
  int nonfinite = 0;
#pragma unroll
  for (int q = 0; q < EPL; ++q) {
    const int e = lane + 64 * q;
    key[q] = 0;
    rank[q] = 0;
    if (e < E) {
      const float v = row[e];
      nonfinite |= !__builtin_isfinite(v);
      key[q] = route_key(v, e);
    }
  }
  *bad |= __any(nonfinite);
#pragma unroll
  for (int qs = 0; qs < EPL; ++qs) {
    if (64 * qs >= E) break;
#pragma unroll 8
    for (int src = 0; src < 64; ++src) {
      const uint64_t other = bcast_u64(key[qs], src);
#pragma unroll
      for (int q = 0; q < EPL; ++q) rank[q] += other > key[q] ? 1 : 0;
    }
  }
#pragma unroll
  for (int q = 0; q < EPL; ++q) {
    if (key[q] != 0 && rank[q] < k) {
      s_e[rank[q]] = static_cast<int32_t>(0xFFFFFFFFu - static_cast<uint32_t>(key[q]));
      s_v[rank[q]] = key_value(key[q]);
    }
  }
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
  const float v0 = s_v[0];
  const int my_e = lane < k ? s_e[lane] : -1;
  const double ex = lane < k ? exp(static_cast<double>(s_v[lane]) - static_cast<double>(v0)) : 0.0;
  if (lane < k) s_x[lane] = ex;
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
  double s = 0.0;
  for (int j = 0; j < k; ++j) s += s_x[j];
  *gate_out = static_cast<float>(ex / s);
  __builtin_amdgcn_wave_barrier();  // s_* are reused by this wavefront's next token
  return my_e;
}

template <int EPL>
__global__ __launch_bounds__(256) void k_route_topk(const float* __restrict__ logits, int T, int E,
                                                    int k, int32_t* __restrict__ topk_idx,
                                                    float* __restrict__ gates,
                                                    int32_t* __restrict__ bad_flag) {
  __shared__ int32_t s_e[4][kMaxTopK];
  __shared__ float s_v[4][kMaxTopK];
  __shared__ double s_x[4][kMaxTopK];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int nwaves = gridDim.x * 4;
  int bad = 0;
  for (int t = blockIdx.x * 4 + wave; t < T; t += nwaves) {
    float g;
    const int e = route_token<EPL>(logits + static_cast<size_t>(t) * E, E, k, s_e[wave], s_v[wave],
                                   s_x[wave], &g, &bad);
    if (lane < k) {
      topk_idx[static_cast<size_t>(t) * k + lane] = e;
      gates[static_cast<size_t>(t) * k + lane] = g;
    }
  }
  if (bad && lane == 0) atomicOr(bad_flag, 1);
}

constexpr int kPermThreads = 1024;
constexpr int kChunkWords = 16;               // bitmask words per expert per chunk
constexpr int kChunkTokens = kChunkWords * 32;

constexpr int kFusedMaxRoutes = 1024;       // fused routing path: T * k routes kept in LDS

// Histogram, offsets, work list and stable permutation of the T*k routes in
// `idx` (global or LDS), by one workgroup, plus the staging of the layer's
// misses. Pass 1: per-expert counts (LDS atomics). Wave 0 then scans the
// experts (4 per lane): offsets, the work list (hit experts first), the hit /
// miss split against the layer's resident set, and the staging: miss j (in
// expert order) takes the free slot free_list[free_top - 1 - j]. Pass 2,
// chunk by chunk of 512 tokens: a per-expert token bitmask (the ballot of
// the tokens that chose the expert), a running popcount prefix per 32-token
// word, and each route's stable position = offsets[e] + tokens before it
// that chose e. Finally one wavefront publishes the routing record (fields,
// system-scope fence, seq).
__device__ __forceinline__ void permute_body(const int32_t* idx, int T, int k, int bad,
                                             const PermuteOut& o) {
  __shared__ int32_t s_cnt[kMaxExperts];
  __shared__ int32_t s_off[kMaxExperts + 1];
  __shared__ int32_t s_item_base[kMaxExperts];
  __shared__ int32_t s_run[kMaxExperts];
  __shared__ int32_t s_stat[12];
  __shared__ int32_t s_sexp[kMaxExperts];
  __shared__ int32_t s_sslot[kMaxExperts];
  __shared__ uint32_t s_res[kMaxExperts / 32];
  __shared__ uint32_t s_mask[kMaxExperts * kChunkWords];
  __shared__ int32_t s_pre[kMaxExperts * kChunkWords];

  const int tid = threadIdx.x;
  const int nthr = blockDim.x;
  const int E = o.E, layer = o.layer;
  const int R = T * k;
  for (int e = tid; e < kMaxExperts; e += nthr) s_cnt[e] = 0;
  if (tid < kMaxExperts / 32) s_res[tid] = o.cv.res[layer].bits[tid];
  __syncthreads();
  for (int r = tid; r < R; r += nthr) atomicAdd(&s_cnt[idx[r]], 1);
  __syncthreads();

  if (tid < 64) {  // wave 0: scans over experts, 4 per lane
    const int lane = tid;
    int c[4], nh[4], nm[4];
    bool hit[4], miss[4];
    int sc = 0, sh = 0, sm = 0, sx = 0;
    int n_act = 0, n_hit = 0, n_res = 0, hrows = 0, mrows = 0;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int e = 4 * lane + q;
      c[q] = e < E ? s_cnt[e] : 0;
      const int ni = (c[q] + kItemRows - 1) / kItemRows;
      const bool res = e < E && ((s_res[e >> 5] >> (e & 31)) & 1u);
      hit[q] = res && c[q] > 0;
      miss[q] = !res && c[q] > 0;
      nh[q] = hit[q] ? ni : 0;
      nm[q] = miss[q] ? ni : 0;
      sc += c[q];
      sh += nh[q];
      sm += nm[q];
      sx += miss[q] ? 1 : 0;
      n_act += c[q] > 0 ? 1 : 0;
      n_hit += hit[q] ? 1 : 0;
      n_res += res ? 1 : 0;
      hrows += hit[q] ? c[q] : 0;
      mrows += miss[q] ? c[q] : 0;
    }
    int ic = sc, ih = sh, im = sm, ix = sx;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
      const int tc = __shfl_up(ic, off), th = __shfl_up(ih, off), tm = __shfl_up(im, off),
                tx = __shfl_up(ix, off);
      if (lane >= off) {
        ic += tc;
        ih += th;
        im += tm;
        ix += tx;
      }
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
      n_act += __shfl_xor(n_act, off);
      n_hit += __shfl_xor(n_hit, off);
      n_res += __shfl_xor(n_res, off);
      hrows += __shfl_xor(hrows, off);
      mrows += __shfl_xor(mrows, off);
    }
    const int tot_hit = __shfl(ih, 63);
    const int n_miss = __shfl(ix, 63);
    // staging: every miss takes a free slot, unless the block is bad
    CacheHdr* hdr = o.cv.hdr;
    const int free_top = hdr->free_top;
    const bool stage = !bad && free_top >= 0 && free_top <= o.cv.n_slots && n_miss <= free_top;
    int xc = ic - sc, xh = ih - sh, xm = im - sm, xx = ix - sx;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int e = 4 * lane + q;
      if (e < E) {
        s_off[e] = xc;
        s_item_base[e] = (nh[q] > 0) ? xh : tot_hit + xm;
        if (stage && miss[q]) {
          const int slot = o.cv.free_list[free_top - 1 - xx];
          o.cv.slot_of[static_cast<size_t>(layer) * E + e] = slot;
          hdr->staged_exp[xx] = e;
          hdr->staged_slot[xx] = slot;
          s_sexp[xx] = e;
          s_sslot[xx] = slot;
        }
      }
      xc += c[q];
      xh += nh[q];
      xm += nm[q];
      xx += miss[q] ? 1 : 0;
    }
    if (lane == 0) {
      hdr->free_top = stage ? free_top - n_miss : free_top;
      hdr->staged_n = stage ? n_miss : 0;
      hdr->route_bad = stage ? 0 : 1;
      if (!bad && !stage) hdr->fault |= 1;
      int32_t* lc = o.cv.last_counts + 4 * layer;
      lc[0] = n_act;
      lc[1] = n_hit;
      lc[2] = n_miss;
      lc[3] = n_res;
      s_stat[0] = n_act;
      s_stat[1] = n_hit;
      s_stat[2] = n_miss;
      s_stat[3] = n_res;
      s_stat[4] = hrows;
      s_stat[5] = mrows;
      s_stat[6] = stage ? n_miss : 0;
      s_stat[7] = stage ? 0 : 1;
    }
    if (lane < kMaxExperts / 32) o.cv.res_before[layer].bits[lane] = s_res[lane];
    if (lane == 63) {
      s_off[E] = ic;
      s_stat[8] = ih;
      s_stat[9] = im;
    }
  }
  __syncthreads();

  for (int e = tid; e < E; e += nthr) {
    const int c = s_cnt[e];
    o.counts[e] = c;
    o.offsets[e] = s_off[e];
    s_run[e] = s_off[e];
    const int base = s_item_base[e];
    for (int m = 0; m * kItemRows < c; ++m) {
      WorkItem it;
      it.expert = e;
      it.row_begin = s_off[e] + m * kItemRows;
      it.rows = min(kItemRows, c - m * kItemRows);
      it.pad = 0;
      o.items[base + m] = it;
    }
  }
  if (tid == 0) o.offsets[E] = s_off[E];

  for (int t0 = 0; t0 < T; t0 += kChunkTokens) {
    const int t1 = min(T, t0 + kChunkTokens);
    for (int i = tid; i < E * kChunkWords; i += nthr) s_mask[i] = 0u;
    __syncthreads();
    for (int r = t0 * k + tid; r < t1 * k; r += nthr) {
      const int e = idx[r];
      const int lt = r / k - t0;
      atomicOr(&s_mask[e * kChunkWords + (lt >> 5)], 1u << (lt & 31));
    }
    __syncthreads();
    for (int e = tid; e < E; e += nthr) {
      int run = s_run[e];
#pragma unroll
      for (int w = 0; w < kChunkWords; ++w) {
        s_pre[e * kChunkWords + w] = run;
        run += __popc(s_mask[e * kChunkWords + w]);
      }
      s_run[e] = run;
    }
    __syncthreads();
    for (int r = t0 * k + tid; r < t1 * k; r += nthr) {
      const int e = idx[r];
      const int lt = r / k - t0;
      const int w = lt >> 5;
      const uint32_t below = s_mask[e * kChunkWords + w] & ((1u << (lt & 31)) - 1u);
      const int pos = s_pre[e * kChunkWords + w] + __popc(below);
      o.perm[pos] = r;
      o.inv_perm[r] = pos;
    }
    __syncthreads();
  }

  if (tid < 64) {
    const int n_staged = s_stat[6];
    if (o.staged) {
      for (int j = tid; j < n_staged; j += 64) {
        o.staged->exp[j] = s_sexp[j];
        o.staged->slot[j] = s_sslot[j];
      }
    }
    RouteStats* rs = o.ring + (o.seq % kStatsRing);
    if (tid == 0) {
      o.item_counts[0] = s_stat[8];
      o.item_counts[1] = s_stat[9];
      rs->layer = layer;
      rs->n_active = s_stat[0];
      rs->n_hits = s_stat[1];
      rs->n_misses = s_stat[2];
      rs->n_resident = s_stat[3];
      rs->hit_rows = s_stat[4];
      rs->miss_rows = s_stat[5];
      rs->n_staged = n_staged;
      rs->bad = bad ? 1 : s_stat[7];
      rs->n_hit_items = s_stat[8];
      rs->n_miss_items = s_stat[9];
      if (o.staged) o.staged->n = n_staged;
    }
    __threadfence_system();
    if (tid == 0) {
      *reinterpret_cast<volatile int32_t*>(&rs->seq) = o.seq;
      if (o.staged) *reinterpret_cast<volatile int32_t*>(&o.staged->seq) = o.seq;
    }
  }
}

__global__ __launch_bounds__(kPermThreads) void k_permute(const int32_t* __restrict__ topk_idx,
                                                          int T, int k,
                                                          int32_t* __restrict__ bad_flag,
                                                          PermuteOut o) {
  const int bad = *bad_flag;
  __syncthreads();
  if (threadIdx.x == 0) *bad_flag = 0;
  permute_body(topk_idx, T, k, bad, o);
}

// Small blocks (T*k <= 1024): routing on many CUs, one token per wavefront,
// then the last workgroup to finish (a fenced counter; no workgroup ever
// waits for another) permutes all routes. Workgroups hold 256 threads and
// the permutation above is written for any workgroup size.
template <int EPL>
__global__ __launch_bounds__(256) void k_route_fused(const float* __restrict__ logits, int T,
                                                     int k, int32_t* __restrict__ topk_idx,
                                                     float* __restrict__ gates,
                                                     int32_t* __restrict__ sync, PermuteOut o) {
  __shared__ int32_t s_e[4][kMaxTopK];
  __shared__ float s_v[4][kMaxTopK];
  __shared__ double s_x[4][kMaxTopK];
  __shared__ int32_t s_idx[kFusedMaxRoutes];
  __shared__ int32_t s_last;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int E = o.E;
  int bad = 0;
  for (int t = blockIdx.x * 4 + wave; t < T; t += gridDim.x * 4) {
    float g;
    const int e = route_token<EPL>(logits + static_cast<size_t>(t) * E, E, k, s_e[wave], s_v[wave],
                                   s_x[wave], &g, &bad);
    if (lane < k) {
      topk_idx[static_cast<size_t>(t) * k + lane] = e;
      gates[static_cast<size_t>(t) * k + lane] = g;
    }
  }
  if (bad && lane == 0) atomicOr(&sync[1], 1);
  __threadfence();   // this workgroup's routes are visible device-wide
  __syncthreads();
  if (threadIdx.x == 0) s_last = atomicAdd(&sync[0], 1) == static_cast<int>(gridDim.x) - 1;
  __syncthreads();
  if (!s_last) return;
  __threadfence();   // see every other workgroup's routes
  for (int r = threadIdx.x; r < T * k; r += blockDim.x) s_idx[r] = __hip_atomic_load(
      &topk_idx[r], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  const int any_bad = __hip_atomic_load(&sync[1], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  __syncthreads();
  if (threadIdx.x == 0) {  // re-arm for the next launch (stream order)
    sync[0] = 0;
    sync[1] = 0;
  }
  permute_body(s_idx, T, k, any_bad, o);
}

}  // namespace

bool route_fused(int T, int k) { return T * k <= kFusedMaxRoutes; }

hipError_t launch_route_topk(const float* logits, int T, int E, int k, int32_t* topk_idx,
                             float* gates, int32_t* bad_flag, hipEvent_t ev0, hipEvent_t ev1,
                             hipStream_t s) {
  const int blocks = (T + 3) / 4 < 4096 ? (T + 3) / 4 : 4096;
  if (E <= 64)
    hipExtLaunchKernelGGL(k_route_topk<1>, dim3(blocks), dim3(256), 0, s, ev0, ev1, 0, logits, T,
                          E, k, topk_idx, gates, bad_flag);
  else if (E <= 128)
    hipExtLaunchKernelGGL(k_route_topk<2>, dim3(blocks), dim3(256), 0, s, ev0, ev1, 0, logits, T,
                          E, k, topk_idx, gates, bad_flag);
  else
    hipExtLaunchKernelGGL(k_route_topk<4>, dim3(blocks), dim3(256), 0, s, ev0, ev1, 0, logits, T,
                          E, k, topk_idx, gates, bad_flag);
  return hipGetLastError();
}

hipError_t launch_permute(const int32_t* topk_idx, int T, int k, int32_t* bad_flag,
                          const PermuteOut& o, hipEvent_t ev0, hipEvent_t ev1, hipStream_t s) {
  hipExtLaunchKernelGGL(k_permute, dim3(1), dim3(kPermThreads), 0, s, ev0, ev1, 0, topk_idx, T, k,
                        bad_flag, o);
  return hipGetLastError();
}

hipError_t launch_route_fused(const float* logits, int T, int k, int32_t* topk_idx, float* gates,
                              int32_t* sync, const PermuteOut& o, hipEvent_t ev0, hipEvent_t ev1,
                              hipStream_t s) {
  const int blocks = (T + 3) / 4;
  if (o.E <= 64)
    hipExtLaunchKernelGGL(k_route_fused<1>, dim3(blocks), dim3(256), 0, s, ev0, ev1, 0, logits, T,
                          k, topk_idx, gates, sync, o);
  else if (o.E <= 128)
    hipExtLaunchKernelGGL(k_route_fused<2>, dim3(blocks), dim3(256), 0, s, ev0, ev1, 0, logits, T,
                          k, topk_idx, gates, sync, o);
  else
    hipExtLaunchKernelGGL(k_route_fused<4>, dim3(blocks), dim3(256), 0, s, ev0, ev1, 0, logits, T,
                          k, topk_idx, gates, sync, o);
  return hipGetLastError();
}

}  // namespace oled
