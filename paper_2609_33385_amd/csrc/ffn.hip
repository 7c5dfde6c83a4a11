// K4 grouped SwiGLU expert FFN over the experts of one layer (hits from their
// cache slots, transferred misses from their staging slots) and the transfer
// of the misses (OLED-MoE Sec. 4.1: cache-hit experts execute on the
// GPU; the output does not depend on where an expert's weights came from).
//
// The GEMMs are weight-streaming: a layer iteration routes few tokens to each
// expert (tens of rows), so every weight byte should be read from HBM once
// while enough wavefronts are in flight to cover HBM latency.
//
// Tile = one work item (up to 64 expert-sorted routes of one expert) x
// 16 * 4 / KS output features. The 4 wavefronts of a workgroup form 4 / KS
// feature groups of 16 and split K in KS contiguous parts (KS = 4, 2 or 1 by
// the size of K); each streams its 16 (gate/up: 2 x 16) weight rows from HBM
// straight into registers (A operand, M = features) and the token rows of its
// K part from L2 (B operand, N = 16 tokens per MFMA tile); the KS partial
// tiles are summed in LDS in a fixed order (deterministic). Expert weights are
// stored packed (see oled_pack_expert): the A fragment of one MFMA step is
// 1 KiB of contiguous memory in lane order, so each wavefront streams one
// contiguous range of its expert's block.
// MFMA: v_mfma_f32_16x16x32_bf16 (bf16) or v_mfma_f32_16x16x4_f32 (fp32).
//
// One tile per workgroup over a grid sized for every possible tile (capped;
// workgroups then loop over tiles); tiles past the live count exit at once,
// and the hardware dispatcher balances the rest over the CUs. Workgroup b runs
// on XCD b % 8; tiles are renumbered so that each XCD takes a contiguous range
// (consecutive feature tiles of the same expert share its token rows in that
// XCD's L2). The number of items comes from device memory, so the launches
// are enqueued before the host has seen the routing result.
//
// A launch may also carry the host-to-device transfer of the layer's misses
// (Sec. 4.2, every miss is transferred): its first workgroups copy a byte
// range of each staged expert's pinned host block into the expert's staging
// slot over PCIe while the other workgroups compute the hit experts' tiles.
//
// Results for an expert depend only on its own rows, never on the other
// experts of the launch, so hit and miss launches give identical bits.
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include "kernels.h"

namespace oled {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float floatx4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

__device__ __forceinline__ uint16_t f32_to_bf16_rne(float f) {
  const uint32_t u = __float_as_uint(f);
  return static_cast<uint16_t>((u + 0x7FFFu + ((u >> 16) & 1u)) >> 16);
}

// bf16: a 16-byte vector holds 8 consecutive k; lane group g (= lane / 16)
// supplies k 8g..8g+7 of a 32-wide MFMA step.
struct TrBF16 {
  using T = uint16_t;
  static constexpr int EPV = 8;    // elements per 16-byte vector
  static constexpr int SPAN = 32;  // k covered by one vector across the 4 lane groups
  __device__ static void mma(floatx4_t& acc, const u32x4_t& a, const u32x4_t& b) {
    acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, a),
                                                  __builtin_bit_cast(bf16x8_t, b), acc, 0, 0, 0);
  }
  __device__ static float silu(float a) { return a / (1.f + __expf(-a)); }
};

// fp32: a 16-byte vector holds 4 consecutive k (16v + 4g + q); MFMA q of the
// vector takes element q from every lane group.
struct TrF32 {
  using T = float;
  static constexpr int EPV = 4;
  static constexpr int SPAN = 16;
  __device__ static void mma(floatx4_t& acc, const u32x4_t& a, const u32x4_t& b) {
#pragma unroll
    for (int q = 0; q < 4; ++q)
      acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a[q]), __uint_as_float(b[q]), acc,
                                                 0, 0, 0);
  }
  __device__ static float silu(float a) { return a / (1.f + expf(-a)); }
};

constexpr int kThreads = 256;
constexpr int kWaves = 4;
constexpr int kFeat = 16;                  // output features per tile
constexpr int kMaxNT = kItemRows / 16;     // token tiles per item

__device__ __forceinline__ u32x4_t ldg16(const void* p) {
  return *reinterpret_cast<const u32x4_t*>(p);
}

// Expert weights are read once per work item: stream them past the caches.
__device__ __forceinline__ u32x4_t ldw16(const void* p) {
  return __builtin_nontemporal_load(reinterpret_cast<const u32x4_t*>(p));
}

// Bijection on [0, total): tile t (XCD t % 8) -> contiguous range per XCD.
__device__ __forceinline__ int xcd_order(int t, int total) {
  const int x = t & 7, local = t >> 3;
  const int q = total >> 3, r = total & 7;
  return x * q + (x < r ? x : r) + local;
}

// Streams one K range of a tile: NT token tiles, groups of U MFMA steps with
// the next group's loads in flight while the current group multiplies (U is
// smaller for more token tiles to keep registers, and so occupancy, in check).
template <class TR, bool UP, int NT>
__device__ __forceinline__ void stream_k(const typename TR::T* a1, const typename TR::T* a3,
                                         const typename TR::T* const* b, int steps,
                                         floatx4_t* acc1, floatx4_t* acc3) {
  constexpr int SPAN = TR::SPAN;
  constexpr int U = NT == 1 ? 4 : 2;
  const int groups = steps / U;
  u32x4_t ra1[2][U], ra3[2][U], rb[2][U][NT];
  constexpr int ASTEP = (UP ? 2 : 1) * 16 * SPAN;  // packed weights per MFMA step
  auto load = [&](int buf, int g0) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int kk = (g0 * U + u) * SPAN;
      ra1[buf][u] = ldw16(a1 + (g0 * U + u) * ASTEP);
      if (UP) ra3[buf][u] = ldw16(a3 + (g0 * U + u) * ASTEP);
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) rb[buf][u][nt] = ldg16(b[nt] + kk);
    }
  };
  auto mult = [&](int buf) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) {
        TR::mma(acc1[nt], ra1[buf][u], rb[buf][u][nt]);
        if (UP) TR::mma(acc3[nt], ra3[buf][u], rb[buf][u][nt]);
      }
    }
  };
  if (groups > 0) load(0, 0);
  int gi = 0;
  for (; gi + 2 <= groups; gi += 2) {
    load(1, gi + 1);
    mult(0);
    if (gi + 2 < groups) load(0, gi + 2);
    mult(1);
  }
  if (gi < groups) mult(0);
  // remaining steps (K range not a multiple of U steps)
  for (int st = groups * U; st < steps; ++st) {
    const int kk = st * SPAN;
    const u32x4_t x1 = ldw16(a1 + st * ASTEP);
    u32x4_t x3;
    if (UP) x3 = ldw16(a3 + st * ASTEP);
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      const u32x4_t bv = ldg16(b[nt] + kk);
      TR::mma(acc1[nt], x1, bv);
      if (UP) TR::mma(acc3[nt], x3, bv);
    }
  }
}

// Epilogue of one 16x16 output tile held in D layout: lane (lr, g), register
// r -> feature f0 + 4g + r, token row 16 nt + lr of the item.
template <class TR, bool UP>
__device__ __forceinline__ void store_tile(const WorkItem& it, int nt, int f0, const floatx4_t& s1,
                                           const floatx4_t& s3, int H, int I,
                                           typename TR::T* __restrict__ hout,
                                           float* __restrict__ oout) {
  using T = typename TR::T;
  const int lane = threadIdx.x & 63;
  const int lr = lane & 15, g = lane >> 4;
  const int row = 16 * nt + lr;
  if (row >= it.rows) return;
  const size_t pos = static_cast<size_t>(it.row_begin + row);
  if (UP) {
    float hv[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) hv[r] = TR::silu(s1[r]) * s3[r];
    if constexpr (sizeof(T) == 2) {
      uint2 packed;
      packed.x = f32_to_bf16_rne(hv[0]) | (static_cast<uint32_t>(f32_to_bf16_rne(hv[1])) << 16);
      packed.y = f32_to_bf16_rne(hv[2]) | (static_cast<uint32_t>(f32_to_bf16_rne(hv[3])) << 16);
      *reinterpret_cast<uint2*>(hout + pos * I + f0 + 4 * g) = packed;
    } else {
      *reinterpret_cast<float4*>(hout + pos * I + f0 + 4 * g) = make_float4(hv[0], hv[1], hv[2], hv[3]);
    }
  } else {
    *reinterpret_cast<float4*>(oout + pos * H + f0 + 4 * g) = make_float4(s1[0], s1[1], s1[2], s1[3]);
  }
}

// One tile of 16 * (4 / KS) output features. Wavefront w takes feature group
// w / KS and K part w % KS; with KS > 1 the KS partial tiles of a feature
// group are summed in LDS in a fixed order and the parts share the epilogue.
template <class TR, bool UP, int KS, int NT>
__device__ __forceinline__ void run_tile(const WorkItem& it, int tile_f0, const typename TR::T* W,
                                         const typename TR::T* __restrict__ src,
                                         const int32_t* __restrict__ perm, int k, int H, int I,
                                         typename TR::T* __restrict__ hout,
                                         float* __restrict__ oout,
                                         floatx4_t (*s_red)[(UP ? 2 : 1) * kMaxNT][64]) {
  using T = typename TR::T;
  constexpr int EPV = TR::EPV;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int lr = lane & 15, g = lane >> 4;
  const int fg = wave / KS, kp = wave % KS;
  const int f0 = tile_f0 + kFeat * fg;
  const int Kdim = UP ? H : I;
  const int kw = Kdim / KS;
  const int kbeg = kp * kw;
  const int rows = it.rows;

  // packed expert block: one 16-row x SPAN-k fragment per MFMA step, stored in
  // the order the lanes consume it, so a wavefront load reads 1 KiB contiguously
  constexpr int FRAG = 16 * TR::SPAN;
  const T* a1;
  const T* a3;
  if (UP) {
    a1 = W + (static_cast<size_t>(f0 / 16) * (H / TR::SPAN) + kbeg / TR::SPAN) * 2 * FRAG + lane * EPV;
    a3 = a1 + FRAG;
  } else {
    a1 = W + static_cast<size_t>(2) * I * H +
         (static_cast<size_t>(f0 / 16) * (I / TR::SPAN) + kbeg / TR::SPAN) * FRAG + lane * EPV;
    a3 = a1;
  }
  // token rows past the item's end read its last row; their results are dropped
  const T* b[NT];
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) {
    const int r = min(16 * nt + lr, rows - 1);
    const int pos = it.row_begin + r;
    b[nt] = (UP ? src + static_cast<size_t>(perm[pos] / k) * H : src + static_cast<size_t>(pos) * I) +
            kbeg + EPV * g;
  }
  floatx4_t acc1[NT], acc3[NT];
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) {
    acc1[nt] = floatx4_t{0.f, 0.f, 0.f, 0.f};
    acc3[nt] = floatx4_t{0.f, 0.f, 0.f, 0.f};
  }
  stream_k<TR, UP, NT>(a1, a3, b, kw / TR::SPAN, acc1, acc3);

  if constexpr (KS == 1) {
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) store_tile<TR, UP>(it, nt, f0, acc1[nt], acc3[nt], H, I, hout, oout);
  } else {
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      s_red[wave][nt][lane] = acc1[nt];
      if (UP) s_red[wave][kMaxNT + nt][lane] = acc3[nt];
    }
    __syncthreads();
    for (int nt = kp; nt < NT; nt += KS) {
      floatx4_t s1 = s_red[fg * KS][nt][lane];
      floatx4_t s3 = UP ? s_red[fg * KS][kMaxNT + nt][lane] : floatx4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int j = 1; j < KS; ++j) {
        s1 += s_red[fg * KS + j][nt][lane];
        if (UP) s3 += s_red[fg * KS + j][kMaxNT + nt][lane];
      }
      store_tile<TR, UP>(it, nt, f0, s1, s3, H, I, hout, oout);
    }
    __syncthreads();  // s_red is reused by the next tile
  }
}

// Copies bytes [off, off + len) of every staged expert's host block into its
// slot: workgroup b of nblk takes 16-byte vectors b*256 + tid + m*nblk*256,
// four loads in flight per thread. The loads cross PCIe; the stores bypass
// the caches.
__device__ __forceinline__ void fetch_blocks(const FetchArgs& f, char* pool, int64_t slot_bytes,
                                             int n_slots, int b) {
  const int n = min(f.hdr->staged_n, kMaxExperts);
  if (n <= 0) return;
  const int64_t per = f.len >> 4;
  const int64_t total = static_cast<int64_t>(n) * per;
  const int64_t stride = static_cast<int64_t>(f.nblk) * kThreads;
  for (int64_t i0 = static_cast<int64_t>(b) * kThreads + threadIdx.x; i0 < total; i0 += 4 * stride) {
    u32x4_t v[4];
    char* dst[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int64_t i = i0 + u * stride;
      dst[u] = nullptr;
      if (i < total) {
        const int j = static_cast<int>(i / per);
        const int64_t o = f.off + ((i - j * per) << 4);
        const int slot = f.hdr->staged_slot[j];
        const int e = f.hdr->staged_exp[j];
        if (slot >= 0 && slot < n_slots && e >= 0 && e < f.E) {
          v[u] = ldw16(reinterpret_cast<const char*>(f.host_addr[e]) + o);
          dst[u] = pool + static_cast<int64_t>(slot) * slot_bytes + o;
        }
      }
    }
#pragma unroll
    for (int u = 0; u < 4; ++u)
      if (dst[u]) __builtin_nontemporal_store(v[u], reinterpret_cast<u32x4_t*>(dst[u]));
  }
}

// The GEMM tiles of one launch part: tiles t0, t0 + stride, ... of the live
// tile count (stride a multiple of 8, so a workgroup keeps its XCD).
template <class TR, bool UP, int KS>
__device__ __forceinline__ void gemm_tiles(const FfnLaunch& a, int t0, int stride,
                                           floatx4_t (*s_red)[(UP ? 2 : 1) * kMaxNT][64]) {
  using T = typename TR::T;
  constexpr int FEAT = kFeat * (kWaves / KS);  // output features per tile
  int base, n_items;
  if (a.n_items_host >= 0) {
    base = a.item_base;
    n_items = a.n_items_host;
  } else {
    const int c0 = a.item_counts[0];
    base = a.which ? c0 : 0;
    n_items = a.which ? a.item_counts[1] : c0;
  }
  const int nf = (UP ? a.I : a.H) / FEAT;
  const int total = n_items * nf;
  const T* src = static_cast<const T*>(a.src);
  T* hout = static_cast<T*>(a.hout);
  for (int t = t0; t < total; t += stride) {
    const int v = xcd_order(t, total);
    const int ii = v / nf;
    const int f0 = (v - ii * nf) * FEAT;
    const WorkItem it = a.items[base + ii];
    const int slot = a.slot_of[it.expert];
    if (slot < 0 || slot >= a.n_slots) continue;  // no weights on the device (bad block)
    const T* W = reinterpret_cast<const T*>(static_cast<const char*>(a.pool) +
                                            static_cast<int64_t>(slot) * a.slot_bytes);
    switch ((it.rows + 15) >> 4) {
      case 1: run_tile<TR, UP, KS, 1>(it, f0, W, src, a.perm, a.k, a.H, a.I, hout, a.oout, s_red); break;
      case 2: run_tile<TR, UP, KS, 2>(it, f0, W, src, a.perm, a.k, a.H, a.I, hout, a.oout, s_red); break;
      case 3: run_tile<TR, UP, KS, 3>(it, f0, W, src, a.perm, a.k, a.H, a.I, hout, a.oout, s_red); break;
      default: run_tile<TR, UP, KS, 4>(it, f0, W, src, a.perm, a.k, a.H, a.I, hout, a.oout, s_red); break;
    }
  }
}

template <class TR, bool UP, int KS>
__global__ __launch_bounds__(kThreads) void k_ffn(FfnLaunch a) {
  __shared__ floatx4_t s_red[KS > 1 ? kWaves : 1][(UP ? 2 : 1) * kMaxNT][64];
  const int nfetch = a.fetch.nblk;
  const int b = blockIdx.x;
  if (b < nfetch) {
    fetch_blocks(a.fetch, static_cast<char*>(const_cast<void*>(a.pool)), a.slot_bytes, a.n_slots, b);
    return;
  }
  gemm_tiles<TR, UP, KS>(a, b - nfetch, static_cast<int>(gridDim.x) - nfetch, s_red);
}

// One launch for three independent parts: the transfer of the misses' down
// weights (workgroups [0, nfetch)), the hit experts' down GEMM (the next gd
// workgroups) and the misses' gate/up GEMM, whose weights the previous launch
// transferred (the rest).
template <class TR, int KSD, int KSU>
__global__ __launch_bounds__(kThreads) void k_ffn_mix(FfnLaunch d, FfnLaunch u, int gd) {
  __shared__ floatx4_t s_buf[kWaves][2 * kMaxNT][64];
  const int nfetch = d.fetch.nblk;
  const int b = blockIdx.x;
  if (b < nfetch) {
    fetch_blocks(d.fetch, static_cast<char*>(const_cast<void*>(d.pool)), d.slot_bytes, d.n_slots, b);
    return;
  }
  if (b < nfetch + gd) {
    gemm_tiles<TR, false, KSD>(d, b - nfetch, gd,
                               reinterpret_cast<floatx4_t (*)[kMaxNT][64]>(&s_buf[0][0][0]));
    return;
  }
  gemm_tiles<TR, true, KSU>(u, b - nfetch - gd, static_cast<int>(gridDim.x) - nfetch - gd, s_buf);
}

__global__ __launch_bounds__(kThreads) void k_fetch(char* pool, int64_t slot_bytes, int n_slots,
                                                    FetchArgs f) {
  fetch_blocks(f, pool, slot_bytes, n_slots, blockIdx.x);
}

// K split of the wavefronts of a tile: a function of the GEMM and its K
// alone, so every launch over an expert reduces in the same order. Gate/up
// (K = H) keeps a K range of at least 256 per wavefront; down (K = I) splits
// only from 2048 on, so a tile streams longer weight rows.
inline int k_split_up(int K) { return K >= 1024 ? 4 : (K >= 512 ? 2 : 1); }
inline int k_split_down(int K) { return K >= 4096 ? 4 : (K >= 2048 ? 2 : 1); }

int part_grid(const FfnLaunch& a, int nf);

template <class TR, bool UP, int KS>
hipError_t launch_ffn_ks(const FfnLaunch& a, hipEvent_t ev0, hipEvent_t ev1, hipStream_t s) {
  if (a.fetch.nblk % 8) return hipErrorInvalidValue;
  const int64_t grid = static_cast<int64_t>(a.fetch.nblk) +
                       part_grid(a, (UP ? a.I : a.H) / (kFeat * (kWaves / KS)));
  if (grid <= 0) return hipSuccess;
  hipExtLaunchKernelGGL(k_ffn<TR, UP, KS>, dim3(static_cast<unsigned>(grid)), dim3(kThreads), 0, s,
                        ev0, ev1, 0, a);
  return hipGetLastError();
}

// Workgroups of one GEMM part: max_items * tiles per item, capped at
// max_grid, rounded up to a multiple of 8.
int part_grid(const FfnLaunch& a, int nf) {
  int64_t tiles = static_cast<int64_t>(a.max_items) * nf;
  if (a.max_grid > 0 && tiles > a.max_grid) tiles = a.max_grid;
  return static_cast<int>((tiles + 7) & ~static_cast<int64_t>(7));
}

template <class TR, int KSD, int KSU>
hipError_t launch_mix_ks(const FfnLaunch& d, const FfnLaunch& u, hipEvent_t ev0, hipEvent_t ev1,
                         hipStream_t s) {
  if (d.fetch.nblk % 8) return hipErrorInvalidValue;
  const int gd = part_grid(d, d.H / (kFeat * (kWaves / KSD)));
  const int gu = part_grid(u, u.I / (kFeat * (kWaves / KSU)));
  const int64_t grid = static_cast<int64_t>(d.fetch.nblk) + gd + gu;
  if (grid <= 0) return hipSuccess;
  hipExtLaunchKernelGGL(k_ffn_mix<TR, KSD, KSU>, dim3(static_cast<unsigned>(grid)), dim3(kThreads),
                        0, s, ev0, ev1, 0, d, u, gd);
  return hipGetLastError();
}

template <class TR, int KSD>
hipError_t launch_mix_d(const FfnLaunch& d, const FfnLaunch& u, hipEvent_t ev0, hipEvent_t ev1,
                        hipStream_t s) {
  switch (k_split_up(u.H)) {
    case 4: return launch_mix_ks<TR, KSD, 4>(d, u, ev0, ev1, s);
    case 2: return launch_mix_ks<TR, KSD, 2>(d, u, ev0, ev1, s);
    default: return launch_mix_ks<TR, KSD, 1>(d, u, ev0, ev1, s);
  }
}

template <class TR>
hipError_t launch_mix_t(const FfnLaunch& d, const FfnLaunch& u, hipEvent_t ev0, hipEvent_t ev1,
                        hipStream_t s) {
  switch (k_split_down(d.I)) {
    case 4: return launch_mix_d<TR, 4>(d, u, ev0, ev1, s);
    case 2: return launch_mix_d<TR, 2>(d, u, ev0, ev1, s);
    default: return launch_mix_d<TR, 1>(d, u, ev0, ev1, s);
  }
}

template <class TR, bool UP>
hipError_t launch_ffn_t(const FfnLaunch& a, hipEvent_t ev0, hipEvent_t ev1, hipStream_t s) {
  switch (UP ? k_split_up(a.H) : k_split_down(a.I)) {
    case 4: return launch_ffn_ks<TR, UP, 4>(a, ev0, ev1, s);
    case 2: return launch_ffn_ks<TR, UP, 2>(a, ev0, ev1, s);
    default: return launch_ffn_ks<TR, UP, 1>(a, ev0, ev1, s);
  }
}

}  // namespace

hipError_t launch_ffn_up(bool bf16, const FfnLaunch& a, hipEvent_t ev0, hipEvent_t ev1,
                         hipStream_t s) {
  return bf16 ? launch_ffn_t<TrBF16, true>(a, ev0, ev1, s) : launch_ffn_t<TrF32, true>(a, ev0, ev1, s);
}

hipError_t launch_ffn_down(bool bf16, const FfnLaunch& a, hipEvent_t ev0, hipEvent_t ev1,
                           hipStream_t s) {
  return bf16 ? launch_ffn_t<TrBF16, false>(a, ev0, ev1, s)
              : launch_ffn_t<TrF32, false>(a, ev0, ev1, s);
}

hipError_t launch_ffn_mix(bool bf16, const FfnLaunch& d, const FfnLaunch& u, hipEvent_t ev0,
                          hipEvent_t ev1, hipStream_t s) {
  return bf16 ? launch_mix_t<TrBF16>(d, u, ev0, ev1, s) : launch_mix_t<TrF32>(d, u, ev0, ev1, s);
}

hipError_t launch_fetch(const void* pool, int64_t slot_bytes, int n_slots, const FetchArgs& f,
                        hipEvent_t ev0, hipEvent_t ev1, hipStream_t s) {
  if (f.nblk <= 0) return hipSuccess;
  hipExtLaunchKernelGGL(k_fetch, dim3(f.nblk), dim3(kThreads), 0, s, ev0, ev1, 0,
                        static_cast<char*>(const_cast<void*>(pool)), slot_bytes, n_slots, f);
  return hipGetLastError();
}

}  // namespace oled
