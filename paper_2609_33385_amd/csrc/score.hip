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
constexpr int kScoreRoutes = 8192;         // routes per scoring workgroup of a large block
constexpr int kScoreRoutesSingle = 8192;   // up to this many routes one workgroup scores

__device__ __forceinline__ bool ranks_above(unsigned long long sa, bool ra, int a,
                                            unsigned long long sb, bool rb, int b) {
  return sa > sb || (sa == sb && (ra > rb || (ra == rb && a < b)));
}

// Folds the layer's last routing into its smoothed statistics (Sec. 4.3):
// activation ratio |A| / E and utilisation hits / C, moving averages with
// weight 1/2 on the newest value (float64; halving is exact, so a fused
// multiply-add rounds the same as the separate operations).
__device__ __forceinline__ void observe_layer(const CacheView& cv, int layer, int E, int C) {
  const int32_t* lc = cv.last_counts + kCountsPerLayer * layer;
  LayerStat st = cv.stat[layer];
  const double a_obs = static_cast<double>(lc[0]) / static_cast<double>(E);
  st.a = st.has_a ? 0.5 * a_obs + 0.5 * st.a : a_obs;
  st.has_a = 1;
  if (C > 0) {
    const double u_obs = static_cast<double>(lc[1]) / static_cast<double>(C);
    st.u = st.has_u ? 0.5 * u_obs + 0.5 * st.u : u_obs;
    st.has_u = 1;
  }
  cv.stat[layer] = st;
}

// Segment sums of routes [r0, r1) into s_S (zeroed by the caller): each
// route's term floor(g * c * 2^48) is added to its expert's segment with an
// integer LDS atomic. The routes are read in token order, so the expert id,
// gate and confidence loads of a route are independent. Sets *s_bad for a
// confidence outside [0, 1].
__device__ __forceinline__ void score_sums(const ScoreArgs& a, int r0, int r1,
                                           unsigned long long* s_S, int32_t* s_bad) {
  const float* __restrict__ gates = a.gates;
  const float* __restrict__ conf = a.conf;
  const int32_t* __restrict__ topk_idx = a.topk_idx;
  const int k = a.k;
  // kSumBatch routes per thread are loaded before any of them is added, so
  // their loads are in flight together (integer adds: any order, same bits)
  constexpr int kSumBatch = 8;
  int bad = 0;
  for (int r = r0 + static_cast<int>(threadIdx.x); r < r1; r += kThreads * kSumBatch) {
    int e[kSumBatch];
    float g[kSumBatch], c[kSumBatch];
#pragma unroll
    for (int u = 0; u < kSumBatch; ++u) {
      const int ru = r + u * kThreads;
      e[u] = -1;
      if (ru < r1) {
        e[u] = topk_idx[ru];
        g[u] = gates[ru];
        c[u] = conf[ru / k];
      }
    }
#pragma unroll
    for (int u = 0; u < kSumBatch; ++u) {
      if (e[u] < 0) continue;
      if (!(c[u] >= 0.f && c[u] <= 1.f)) {
        bad = 1;
        continue;
      }
      const double prod = static_cast<double>(g[u]) * static_cast<double>(c[u]);
      atomicAdd(&s_S[e[u]], static_cast<unsigned long long>(floor(prod * 0x1p48)));
    }
  }
  if (bad) atomicOr(s_bad, 1);
}

// The cache state a commit reads, loaded into LDS by the committing workgroup
// (before it sums the routes, when it is the only part), so that its global
// reads overlap the sums instead of following one another. Nothing else in
// the launch writes it.
struct ScoreState {
  uint32_t res[kMaxExperts / 32];
  uint32_t cpu[kMaxExperts / 32];   // CPU-executed misses: no candidates
  int32_t cnt[kMaxExperts];         // routes per expert
  int32_t slot[kMaxExperts];        // the layer's slot table
  int32_t cap, iters, free_top, route_bad;
};

__device__ __forceinline__ void score_prefetch(const ScoreArgs& a, ScoreState& st) {
  const CacheView& cv = a.cv;
  const int tid = threadIdx.x, E = a.E, layer = a.layer;
  for (int e = tid; e < E; e += kThreads) {
    st.cnt[e] = a.counts[e];
    st.slot[e] = cv.slot_of[static_cast<size_t>(layer) * E + e];
  }
  if (tid < kMaxExperts / 32) {
    st.res[tid] = cv.res[layer].bits[tid];
    st.cpu[tid] = cv.cpu_exec ? cv.cpu_exec[layer].bits[tid] : 0u;
  } else if (tid == kMaxExperts / 32) {
    st.cap = cv.cap[layer];
    st.iters = cv.iters[layer];
    st.free_top = cv.hdr->free_top;
    st.route_bad = cv.hdr->route_bad;
  }
}

// Ranking, retention and commit of one layer from its numerators in s_S (and
// *s_bad) and the prefetched state st, by one workgroup.
__device__ __forceinline__ void score_commit(const ScoreArgs& a, unsigned long long* s_S,
                                             int32_t* p_bad, const ScoreState& st) {
  const int32_t* __restrict__ counts = st.cnt;
  const int E = a.E, layer = a.layer;
  const CacheView& cv = a.cv;
  const int C = st.cap;
  uint64_t* __restrict__ score_out = a.score_out;
  RetainOut* __restrict__ out = a.out;
  __shared__ uint32_t s_rc[kMaxExperts];  // bit 1: previously resident, bit 0: candidate
  __shared__ int32_t s_rank[kMaxExperts];
  const uint32_t* s_res = st.res;
  const uint32_t* s_cpu = st.cpu;
  const int tid = threadIdx.x;
  for (int e = tid; e < kMaxExperts; e += kThreads) {
    s_rank[e] = 0;
    const bool r = e < E && ((s_res[e >> 5] >> (e & 31)) & 1u);
    const bool cpu = e < E && ((s_cpu[e >> 5] >> (e & 31)) & 1u);
    const bool c = e < E && (r || (counts[e] > 0 && !cpu));
    s_rc[e] = (r ? 2u : 0u) | (c ? 1u : 0u);
  }
  // (s_rc and s_rank are next read after the barrier that follows the keys)
  const int s_bad = *p_bad;
  CacheHdr* hdr = cv.hdr;
  const bool commit = !s_bad && !st.route_bad && !a.reject;

  // The retention key: S under the paper's priority; under LRU / LFU the
  // layer's history, advanced by this iteration's routing when it commits
  // (the iteration of the last activation, or the routes so far).
  __shared__ unsigned long long s_K[kMaxExperts];
  const int it_now = st.iters + 1;
  for (int e = tid; e < E; e += kThreads) {
    if (cv.policy == 0) {
      s_K[e] = s_S[e];
      continue;
    }
    int32_t* lu = cv.last_use + static_cast<size_t>(layer) * E + e;
    uint64_t* fr = cv.freq + static_cast<size_t>(layer) * E + e;
    int32_t u = *lu;
    uint64_t f = *fr;
    if (commit && counts[e] > 0) {
      u = it_now;
      f += static_cast<uint64_t>(counts[e]);
      *lu = u;
      *fr = f;
    }
    s_K[e] = cv.policy == 1 ? static_cast<unsigned long long>(u) : f;
  }
  __syncthreads();
  if (tid == 0 && commit && cv.policy != 0) cv.iters[layer] = it_now;

  // Top-C over candidates R u A by (key desc, previously resident first, id
  // asc): rank[e] = number of candidates above e. Thread pairs (e, quarter of
  // the candidates) count with broadcast LDS reads; LDS atomics sum the parts.
  const int fq = (E + 3) >> 2;
  for (int idx = tid; idx < 4 * E; idx += kThreads) {
    const int e = idx % E, part = idx / E;
    const unsigned long long se = s_K[e];
    const bool re = s_rc[e] & 2u;
    int cnt = 0;
    const int f1 = min(E, (part + 1) * fq);
    for (int f = part * fq; f < f1; ++f) {
      const uint32_t rcf = s_rc[f];
      cnt += ((rcf & 1u) && ranks_above(s_K[f], rcf & 2u, f, se, re, e)) ? 1 : 0;
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
  int32_t* slot_row = cv.slot_of + static_cast<size_t>(layer) * E;
  int top = st.free_top;
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
    const int sl = e < E ? st.slot[e] : -1;
    if (keep && sl < 0) {
      fault |= 4;
      keep = false;
    }
    if (e < E && !a.reject) {   // a rejected layer keeps its last retention's keys
      score_out[e] = s_S[e];
      a.key_out[e] = s_K[e];
    }
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
    if (cv.cpu_exec) cv.cpu_exec[layer].bits[lane] = 0u;
  }
  if (lane == 0) {
    hdr->free_top = top;
    hdr->staged_n = 0;
    hdr->route_bad = 0;
    if (fault) hdr->fault |= fault;
    out->bad_conf = s_bad;
    out->n_retained = kept;
    out->seq = a.seq;
    if (cv.adapt && commit) observe_layer(cv, layer, E, C);
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
  // every route's gate and row position, then every row, are loaded before
  // the sum, so the loads of all k routes are in flight together
  float gj[kMaxTopK];
  int pos[kMaxTopK];
#pragma unroll
  for (int j = 0; j < kMaxTopK; ++j)
    if (j < k) {
      gj[j] = c.gates[static_cast<size_t>(t) * k + j];
      pos[j] = c.inv_perm[static_cast<size_t>(t) * k + j];
    }
  float4 o[kMaxTopK];
#pragma unroll
  for (int j = 0; j < kMaxTopK; ++j)
    if (j < k) o[j] = *reinterpret_cast<const float4*>(c.O + static_cast<size_t>(pos[j]) * H + h);
  float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
  for (int j = 0; j < kMaxTopK; ++j)
    if (j < k) {
      acc.x = fmaf(gj[j], o[j].x, acc.x);
      acc.y = fmaf(gj[j], o[j].y, acc.y);
      acc.z = fmaf(gj[j], o[j].z, acc.z);
      acc.w = fmaf(gj[j], o[j].w, acc.w);
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

// Priority numerators and retention of one layer by the first a.parts
// workgroups of a launch. One part: that workgroup sums every route and
// commits. Several parts (large blocks): part p sums routes [p*n, (p+1)*n)
// (n = kScoreRoutes) into LDS and adds its nonzero numerators to the device
// accumulators with integer atomics (any order, same bits); a second launch
// of one workgroup (k_score_commit) reads the totals, re-arms the
// accumulators and commits. Two launches in stream order: no workgroup waits
// on another and no device-scope fence orders the sums.
__device__ __forceinline__ void score_part(const ScoreArgs& a, int part) {
  __shared__ unsigned long long s_S[kMaxExperts];
  __shared__ int32_t s_bad;
  __shared__ ScoreState st;
  const int tid = threadIdx.x, E = a.E;
  const int R = a.T * a.k;
  for (int e = tid; e < kMaxExperts; e += kThreads) s_S[e] = 0ull;
  if (tid == 0) s_bad = 0;
  if (a.parts <= 1) score_prefetch(a, st);
  __syncthreads();
  if (a.parts <= 1) {
    score_sums(a, 0, R, s_S, &s_bad);
    __syncthreads();
    score_commit(a, s_S, &s_bad, st);
    return;
  }
  const int r0 = part * kScoreRoutes;
  score_sums(a, r0, min(R, r0 + kScoreRoutes), s_S, &s_bad);
  __syncthreads();
  for (int e = tid; e < E; e += kThreads)
    if (s_S[e]) atomicAdd(&a.acc[e], s_S[e]);
  if (tid == 0 && s_bad) atomicOr(&a.acc_sync[1], 1);
}

// Several parts, second launch: the totals of every part, the accumulators
// re-armed for the next layer (stream order), the commit.
__global__ __launch_bounds__(kThreads) void k_score_commit(ScoreArgs a) {
  __shared__ unsigned long long s_S[kMaxExperts];
  __shared__ int32_t s_bad;
  __shared__ ScoreState st;
  const int tid = threadIdx.x, E = a.E;
  for (int e = tid; e < kMaxExperts; e += kThreads) {
    s_S[e] = e < E ? a.acc[e] : 0ull;
    if (e < E) a.acc[e] = 0ull;
  }
  if (tid == 0) {
    s_bad = a.acc_sync[1];
    a.acc_sync[1] = 0;
  }
  score_prefetch(a, st);
  __syncthreads();
  score_commit(a, s_S, &s_bad, st);
}

__global__ __launch_bounds__(kThreads) void k_score_retain(ScoreArgs a) {
  score_part(a, blockIdx.x);
}

// The layer's last launch: workgroups [0, a.parts) score and commit the
// retention, the rest combine (the two parts touch disjoint data).
template <bool BF16>
__global__ __launch_bounds__(kThreads) void k_combine_score(CombineArgs c, ScoreArgs a) {
  const int b = blockIdx.x;
  const int np = a.parts < 1 ? 1 : a.parts;
  if (b < np) {
    score_part(a, b);
    return;
  }
  const int hx = (c.H + 1023) / 1024;
  combine_body<BF16>(c, (b - np) / hx, (b - np) % hx);
}

// Layer-adaptive sizing (Sec. 4.3): w_l = a_l * u_l, C_l = C_total * w_l /
// sum_j w_j in integers, then the eviction of the lowest-priority residents of
// every layer left over its new capacity. One workgroup; the shares are
// computed by one thread in layer order, so every sum has a fixed order.
//  * shares: q_l = (C_avail * w_l) / W over the open layers (W their sum in
//    layer order); layers with q_l > E are closed at E and the rest re-shared;
//  * integers: floor(q_l); the units left go one each to the open layers below
//    E by (q_l - floor(q_l) desc, layer asc); should the rounded shares
//    overshoot, the layers with the smallest remainders (ties: higher layer)
//    give one back;
//  * eviction: a layer with more residents than C_l keeps those of highest
//    (S desc, id asc); released slots go back to the free list in expert order.
// If every w_l is 0 nothing changes.
__global__ __launch_bounds__(kThreads) void k_layer_adapt(AdaptArgs a) {
#pragma clang fp contract(off)
  __shared__ double s_w[kMaxAdaptLayers];
  __shared__ double s_q[kMaxAdaptLayers];   // share, then its fractional part
  __shared__ int32_t s_cap[kMaxAdaptLayers];
  __shared__ uint8_t s_open[kMaxAdaptLayers];
  __shared__ int32_t s_left, s_skip;
  __shared__ int32_t s_rank[kMaxExperts];
  const CacheView& cv = a.cv;
  const int L = a.L, E = a.E, tid = threadIdx.x;
  for (int l = tid; l < L; l += kThreads) {
    const LayerStat st = cv.stat[l];
    s_w[l] = (st.has_a && st.has_u) ? st.a * st.u : 0.0;
  }
  __syncthreads();
  if (tid == 0) {
    double total = 0.0;
    for (int l = 0; l < L; ++l) total += s_w[l];
    s_skip = total == 0.0;
    if (!s_skip) {
      int avail = a.c_total;
      for (int l = 0; l < L; ++l) {
        s_open[l] = 1;
        s_cap[l] = 0;
      }
      for (;;) {
        double W = 0.0;
        for (int l = 0; l < L; ++l)
          if (s_open[l]) W += s_w[l];
        if (W == 0.0) {
          for (int l = 0; l < L; ++l)
            if (s_open[l]) s_q[l] = 0.0;
          break;
        }
        int n_over = 0;
        for (int l = 0; l < L; ++l)
          if (s_open[l]) {
            const double num = static_cast<double>(avail) * s_w[l];
            s_q[l] = num / W;
            n_over += s_q[l] > static_cast<double>(E);
          }
        if (n_over == 0) break;
        for (int l = 0; l < L; ++l)
          if (s_open[l] && s_q[l] > static_cast<double>(E)) {
            s_cap[l] = E;
            s_open[l] = 0;
            avail -= E;
          }
      }
      int given = 0;
      for (int l = 0; l < L; ++l)
        if (s_open[l]) {
          const double f = floor(s_q[l]);
          s_cap[l] = static_cast<int>(f);
          s_q[l] = s_q[l] - f;
          given += s_cap[l];
        }
      s_left = avail - given;
    }
  }
  __syncthreads();
  if (s_skip) return;
  const int left = s_left;
  for (int l = tid; l < L; l += kThreads) {
    if (!s_open[l]) continue;
    const double fl = s_q[l];
    if (left > 0 && s_cap[l] < E) {
      int rank = 0;
      for (int j = 0; j < L; ++j)
        if (s_open[j] && s_cap[j] < E && (s_q[j] > fl || (s_q[j] == fl && j < l))) ++rank;
      if (rank < left) ++s_cap[l];
    } else if (left < 0 && s_cap[l] > 0) {
      int rank = 0;
      for (int j = 0; j < L; ++j)
        if (s_open[j] && s_cap[j] > 0 && (s_q[j] < fl || (s_q[j] == fl && j > l))) ++rank;
      if (rank < -left) --s_cap[l];
    }
  }
  __syncthreads();
  for (int l = tid; l < L; l += kThreads) cv.cap[l] = s_cap[l];

  // eviction, layer by layer
  CacheHdr* hdr = cv.hdr;
  for (int l = 0; l < L; ++l) {
    const ExpertMask held = cv.res[l];
    int n_held = 0;
#pragma unroll
    for (int w = 0; w < kMaxExperts / 32; ++w) n_held += __popc(held.bits[w]);
    const int cap = s_cap[l];
    if (n_held <= cap) continue;   // uniform across the workgroup
    const uint64_t* S = a.score + static_cast<size_t>(l) * E;
    for (int e = tid; e < E; e += kThreads) {
      int rank = 0;
      if (held.test(e)) {
        const uint64_t se = S[e];
        for (int f = 0; f < E; ++f)
          if (held.test(f) && (S[f] > se || (S[f] == se && f < e))) ++rank;
      }
      s_rank[e] = rank;
    }
    __syncthreads();
    if (tid < 64) {
      const int lane = tid;
      int32_t* slot_row = cv.slot_of + static_cast<size_t>(l) * E;
      int top = hdr->free_top;
      int fault = 0;
      uint32_t word[kMaxExperts / 32];
#pragma unroll
      for (int q = 0; q < kMaxExperts / 64; ++q) {
        const int e = lane + 64 * q;
        const bool h = e < E && held.test(e);
        const bool drop = h && s_rank[e] >= cap;
        const int sl = drop ? slot_row[e] : -1;
        const bool release = drop && sl >= 0;
        const uint64_t rel = __ballot(release);
        const int pos = top + __popcll(rel & ((1ull << lane) - 1ull));
        if (release) {
          if (pos < cv.n_slots) cv.free_list[pos] = sl;
          else fault = 2;
        }
        if (drop) slot_row[e] = -1;
        top += __popcll(rel);
        const uint64_t keep = __ballot(h && !drop);
        word[2 * q] = static_cast<uint32_t>(keep);
        word[2 * q + 1] = static_cast<uint32_t>(keep >> 32);
      }
      fault = __ballot(fault) ? 2 : 0;
      uint32_t my_word = 0u;
#pragma unroll
      for (int w = 0; w < kMaxExperts / 32; ++w)
        if (lane == w) my_word = word[w];
      if (lane < kMaxExperts / 32) cv.res[l].bits[lane] = my_word;
      if (lane == 0) {
        hdr->free_top = top > cv.n_slots ? cv.n_slots : top;
        if (fault) hdr->fault |= fault;
      }
    }
    __syncthreads();
  }
}

// See launch_coop_unstage. One thread walks the staged list in order.
__global__ __launch_bounds__(64) void k_coop_unstage(CacheView cv, int layer, int E,
                                                     ExpertMask cpu) {
  if (threadIdx.x != 0) return;
  CacheHdr* hdr = cv.hdr;
  int32_t* slot_row = cv.slot_of + static_cast<size_t>(layer) * E;
  int top = hdr->free_top;
  const int n = min(hdr->staged_n, kMaxExperts);
  int m = 0;
  for (int j = 0; j < n; ++j) {
    const int e = hdr->staged_exp[j], sl = hdr->staged_slot[j];
    if (e >= 0 && e < E && cpu.test(e)) {
      if (sl >= 0 && sl < cv.n_slots && top < cv.n_slots) cv.free_list[top++] = sl;
      else hdr->fault |= 2;
      slot_row[e] = -1;
    } else {
      hdr->staged_exp[m] = e;
      hdr->staged_slot[m] = sl;
      ++m;
    }
  }
  hdr->staged_n = m;
  hdr->free_top = top;
  for (int w = 0; w < kMaxExperts / 32; ++w) {
    cv.prev_miss[layer].bits[w] &= ~cpu.bits[w];
    cv.cpu_exec[layer].bits[w] = cpu.bits[w];
  }
}

}  // namespace

hipError_t launch_coop_unstage(const CacheView& cv, int layer, int E, const ExpertMask& cpu,
                               hipStream_t s) {
  if (!cv.cpu_exec) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_coop_unstage, dim3(1), dim3(64), 0, s, cv, layer, E, cpu);
  return hipGetLastError();
}

hipError_t launch_layer_adapt(const AdaptArgs& a, hipEvent_t ev0, hipEvent_t ev1, hipStream_t s) {
  if (a.L <= 0 || a.L > kMaxAdaptLayers) return hipErrorInvalidValue;
  hipExtLaunchKernelGGL(k_layer_adapt, dim3(1), dim3(kThreads), 0, s, ev0, ev1, 0, a);
  return hipGetLastError();
}

int score_parts(int T, int k) {
  const int64_t R = static_cast<int64_t>(T) * k;
  return R <= kScoreRoutesSingle ? 1 : static_cast<int>((R + kScoreRoutes - 1) / kScoreRoutes);
}

hipError_t launch_score_retain(const ScoreArgs& a, hipEvent_t ev0, hipEvent_t ev1, hipStream_t s) {
  if (a.parts != score_parts(a.T, a.k)) return hipErrorInvalidValue;
  const bool split = a.parts > 1;
  hipExtLaunchKernelGGL(k_score_retain, dim3(a.parts), dim3(kThreads), 0, s, ev0,
                        split ? nullptr : ev1, 0, a);
  if (!split) return hipGetLastError();
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipExtLaunchKernelGGL(k_score_commit, dim3(1), dim3(kThreads), 0, s, nullptr, ev1, 0, a);
  return hipGetLastError();
}

hipError_t launch_combine_score(bool bf16, const CombineArgs& c, const ScoreArgs& a,
                                hipEvent_t ev0, hipEvent_t ev1, hipStream_t s) {
  if (a.parts != score_parts(a.T, a.k)) return hipErrorInvalidValue;
  const int grid = a.parts + c.T * ((c.H + 1023) / 1024);
  const bool split = a.parts > 1;
  if (bf16)
    hipExtLaunchKernelGGL(k_combine_score<true>, dim3(grid), dim3(kThreads), 0, s, ev0,
                          split ? nullptr : ev1, 0, c, a);
  else
    hipExtLaunchKernelGGL(k_combine_score<false>, dim3(grid), dim3(kThreads), 0, s, ev0,
                          split ? nullptr : ev1, 0, c, a);
  if (!split) return hipGetLastError();
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipExtLaunchKernelGGL(k_score_commit, dim3(1), dim3(kThreads), 0, s, nullptr, ev1, 0, a);
  return hipGetLastError();
}

}  // namespace oled

// ---------------------------------------------------------------------------
// Priority numerators of many independent blocks in one pass (no retention):
// workgroup (p, b) sums routes [p n, (p + 1) n) of block b (n = kScoreRoutes)
// into LDS and adds its nonzero numerators to S[b][*] with integer atomics
// (any order, same bits); S and the flags are cleared by a first launch.
#include "oled.h"

namespace oled {
namespace {

__global__ __launch_bounds__(kThreads) void k_priority_clear(unsigned long long* S, int n,
                                                             int32_t* bad, int B) {
  const int i = blockIdx.x * kThreads + static_cast<int>(threadIdx.x);
  if (i < n) S[i] = 0ull;
  if (bad && i < B) bad[i] = 0;
}

__global__ __launch_bounds__(kThreads) void k_priority_batch(const int32_t* __restrict__ topk_idx,
                                                             const float* __restrict__ gates,
                                                             const float* __restrict__ conf,
                                                             int T, int k, int E,
                                                             unsigned long long* __restrict__ S,
                                                             int32_t* __restrict__ bad) {
  __shared__ unsigned long long s_S[kMaxExperts];
  __shared__ int32_t s_bad;
  const int tid = threadIdx.x, b = blockIdx.y;
  const size_t R = static_cast<size_t>(T) * k;
  for (int e = tid; e < kMaxExperts; e += kThreads) s_S[e] = 0ull;
  if (tid == 0) s_bad = 0;
  __syncthreads();
  ScoreArgs a{};
  a.gates = gates + b * R;
  a.conf = conf + static_cast<size_t>(b) * T;
  a.topk_idx = topk_idx + b * R;
  a.k = k;
  const int r0 = blockIdx.x * kScoreRoutes;
  score_sums(a, r0, min(static_cast<int>(R), r0 + kScoreRoutes), s_S, &s_bad);
  __syncthreads();
  for (int e = tid; e < E; e += kThreads)
    if (s_S[e]) atomicAdd(&S[static_cast<size_t>(b) * E + e], s_S[e]);
  if (tid == 0 && s_bad && bad) atomicOr(&bad[b], 1);
}

}  // namespace
}  // namespace oled

extern "C" oled_status oled_priority_batch(const int32_t* topk_idx_dev, const float* gates_dev,
                                           const float* conf_dev, int32_t B, int32_t T, int32_t E,
                                           int32_t k, uint64_t* score_q_dev,
                                           int32_t* bad_conf_dev, void* stream) {
  if (!topk_idx_dev || !gates_dev || !conf_dev || !score_q_dev) {
    oled::set_noctx_error("oled_priority_batch: NULL input or output");
    return OLED_ERR_INVALID_ARG;
  }
  if (B < 1 || T < 1 || E < 1 || k < 1 || k > E) {
    oled::set_noctx_error("oled_priority_batch: B, T, E and k must be >= 1 and k <= E");
    return OLED_ERR_INVALID_ARG;
  }
  if (T > 65535 || E > oled::kMaxExperts || k > oled::kMaxTopK ||
      static_cast<int64_t>(B) * T * k > INT32_MAX || static_cast<int64_t>(B) * E > INT32_MAX) {
    oled::set_noctx_error("oled_priority_batch: T above 65535, E above 256, k above 16 or "
                          "B*T*k above 2^31-1");
    return OLED_ERR_UNSUPPORTED;
  }
  hipStream_t s = static_cast<hipStream_t>(stream);
  const int n = B * E;
  const int clear = (n > B ? n : B);
  hipLaunchKernelGGL(oled::k_priority_clear, dim3((clear + oled::kThreads - 1) / oled::kThreads),
                     dim3(oled::kThreads), 0, s,
                     reinterpret_cast<unsigned long long*>(score_q_dev), n, bad_conf_dev, B);
  hipError_t e = hipGetLastError();
  if (e == hipSuccess) {
    const int parts = static_cast<int>((static_cast<int64_t>(T) * k + oled::kScoreRoutes - 1) /
                                       oled::kScoreRoutes);
    hipLaunchKernelGGL(oled::k_priority_batch, dim3(parts, B), dim3(oled::kThreads), 0, s,
                       topk_idx_dev, gates_dev, conf_dev, T, k, E,
                       reinterpret_cast<unsigned long long*>(score_q_dev), bad_conf_dev);
    e = hipGetLastError();
  }
  if (e != hipSuccess) {
    oled::set_noctx_error("oled_priority_batch: launch failed");
    return OLED_ERR_HIP;
  }
  return OLED_OK;
}
