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
// 32 * 4 / KS output features. The 4 wavefronts of a workgroup form 4 / KS
// feature groups of 2 x 16 and split K in KS contiguous parts (KS = 4, 2 or 1
// by the size of K); each streams its 2 x 16 (gate/up: 2 x 2 x 16) weight rows
// from HBM straight into registers (A operand, M = features) and the token
// rows of its K part from L2 (B operand, N = 16 tokens per MFMA tile), each
// token load feeding both runs of 16 features (half the L2 reads of the token
// rows of one run per wavefront); the KS partial tiles are summed in LDS in a
// fixed order (deterministic). Expert weights are
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

#include <type_traits>

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
constexpr int kFeat = 16;                  // output features per 16-row weight fragment
constexpr int kFG = 2;                     // runs of 16 features per wavefront (share token loads)
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

// Streams one K range of a tile: F groups of 16 weight rows (gate and up rows
// for gate/up) against NT token tiles; every token load feeds all F groups.
// Groups of U MFMA steps, the next group's loads in flight while the current
// group multiplies (U shrinks as the loads per step grow, to keep registers,
// and so occupancy, in check).
template <class TR, bool UP, int NT, int F>
__device__ __forceinline__ void stream_k(const typename TR::T* const* a1,
                                         const typename TR::T* const* a3,
                                         const typename TR::T* const* b, int steps,
                                         floatx4_t (*acc1)[NT], floatx4_t (*acc3)[NT]) {
  constexpr int SPAN = TR::SPAN;
  constexpr int VEC = F * (UP ? 2 : 1) + NT;        // 16-byte loads per lane per step
  constexpr int U = VEC <= 3 ? 4 : (VEC <= 6 ? 2 : 1);
  const int groups = steps / U;
  u32x4_t ra1[2][U][F], ra3[2][U][F], rb[2][U][NT];
  constexpr int ASTEP = (UP ? 2 : 1) * 16 * SPAN;  // packed weights per MFMA step
  auto load = [&](int buf, int g0) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int kk = (g0 * U + u) * SPAN;
#pragma unroll
      for (int j = 0; j < F; ++j) {
        ra1[buf][u][j] = ldw16(a1[j] + (g0 * U + u) * ASTEP);
        if (UP) ra3[buf][u][j] = ldw16(a3[j] + (g0 * U + u) * ASTEP);
      }
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) rb[buf][u][nt] = ldg16(b[nt] + kk);
    }
  };
  auto mult = [&](int buf) {
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int j = 0; j < F; ++j)
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) {
          TR::mma(acc1[j][nt], ra1[buf][u][j], rb[buf][u][nt]);
          if (UP) TR::mma(acc3[j][nt], ra3[buf][u][j], rb[buf][u][nt]);
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
    u32x4_t x1[F], x3[F];
#pragma unroll
    for (int j = 0; j < F; ++j) {
      x1[j] = ldw16(a1[j] + st * ASTEP);
      if (UP) x3[j] = ldw16(a3[j] + st * ASTEP);
    }
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      const u32x4_t bv = ldg16(b[nt] + kk);
#pragma unroll
      for (int j = 0; j < F; ++j) {
        TR::mma(acc1[j][nt], x1[j], bv);
        if (UP) TR::mma(acc3[j][nt], x3[j], bv);
      }
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

// One tile of 16 * F * (4 / KS) output features. Wavefront w takes feature
// group w / KS (F runs of 16 features) and K part w % KS; with KS > 1 the KS
// partial tiles of each run of 16 features are summed in LDS in a fixed order
// and the parts share the epilogue. Which workgroup computes a feature does not
// change its arithmetic: the K split is a function of the GEMM alone.
template <class TR, bool UP, int KS, int NT, int F>
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
  const int f0 = tile_f0 + kFeat * F * fg;
  const int Kdim = UP ? H : I;
  const int kw = Kdim / KS;
  const int kbeg = kp * kw;
  const int rows = it.rows;

  // packed expert block: one 16-row x SPAN-k fragment per MFMA step, stored in
  // the order the lanes consume it, so a wavefront load reads 1 KiB contiguously
  constexpr int FRAG = 16 * TR::SPAN;
  const T* a1[F];
  const T* a3[F];
#pragma unroll
  for (int j = 0; j < F; ++j) {
    const int fj = f0 + kFeat * j;
    if (UP) {
      a1[j] = W + (static_cast<size_t>(fj / 16) * (H / TR::SPAN) + kbeg / TR::SPAN) * 2 * FRAG +
              lane * EPV;
      a3[j] = a1[j] + FRAG;
    } else {
      a1[j] = W + static_cast<size_t>(2) * I * H +
              (static_cast<size_t>(fj / 16) * (I / TR::SPAN) + kbeg / TR::SPAN) * FRAG + lane * EPV;
      a3[j] = a1[j];
    }
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
  floatx4_t acc1[F][NT], acc3[F][NT];
#pragma unroll
  for (int j = 0; j < F; ++j)
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      acc1[j][nt] = floatx4_t{0.f, 0.f, 0.f, 0.f};
      acc3[j][nt] = floatx4_t{0.f, 0.f, 0.f, 0.f};
    }
  stream_k<TR, UP, NT, F>(a1, a3, b, kw / TR::SPAN, acc1, acc3);

  if constexpr (KS == 1) {
#pragma unroll
    for (int j = 0; j < F; ++j)
#pragma unroll
      for (int nt = 0; nt < NT; ++nt)
        store_tile<TR, UP>(it, nt, f0 + kFeat * j, acc1[j][nt], acc3[j][nt], H, I, hout, oout);
  } else {
#pragma unroll
    for (int j = 0; j < F; ++j) {
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) {
        s_red[wave][nt][lane] = acc1[j][nt];
        if (UP) s_red[wave][kMaxNT + nt][lane] = acc3[j][nt];
      }
      __syncthreads();
      for (int nt = kp; nt < NT; nt += KS) {
        floatx4_t s1 = s_red[fg * KS][nt][lane];
        floatx4_t s3 = UP ? s_red[fg * KS][kMaxNT + nt][lane] : floatx4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int q = 1; q < KS; ++q) {
          s1 += s_red[fg * KS + q][nt][lane];
          if (UP) s3 += s_red[fg * KS + q][kMaxNT + nt][lane];
        }
        store_tile<TR, UP>(it, nt, f0 + kFeat * j, s1, s3, H, I, hout, oout);
      }
      __syncthreads();  // s_red is reused by the next run of features / tile
    }
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
  constexpr int FEAT = kFeat * kFG * (kWaves / KS);  // output features per tile
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
    const int slot = it.pad >= 0 ? it.pad : a.slot_of[it.expert];
    if (slot < 0 || slot >= a.n_slots) continue;  // no weights on the device (bad block)
    const T* W = reinterpret_cast<const T*>(static_cast<const char*>(a.pool) +
                                            static_cast<int64_t>(slot) * a.slot_bytes);
    switch ((it.rows + 15) >> 4) {
      case 1: run_tile<TR, UP, KS, 1, kFG>(it, f0, W, src, a.perm, a.k, a.H, a.I, hout, a.oout, s_red); break;
      case 2: run_tile<TR, UP, KS, 2, kFG>(it, f0, W, src, a.perm, a.k, a.H, a.I, hout, a.oout, s_red); break;
      case 3: run_tile<TR, UP, KS, 3, kFG>(it, f0, W, src, a.perm, a.k, a.H, a.I, hout, a.oout, s_red); break;
      default: run_tile<TR, UP, KS, 4, kFG>(it, f0, W, src, a.perm, a.k, a.H, a.I, hout, a.oout, s_red); break;
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

// ---------------------------------------------------------------------------
// Dense tiles for experts with many routed rows (bf16). A workgroup computes
// up to 256 rows of one expert against 256 weight rows: gate/up 128 features
// (each with its W1 and W3 row), down 256 features. Wavefront w owns 64 of
// the weight rows and multiplies them by all of the tile's token rows with
// v_mfma_f32_32x32x16_bf16 (the 16x16x32 form runs at less than half its
// rate on this part), accumulators in registers.
//  * Weights are private to a wavefront: it loads them from the packed
//    fragments straight into registers, about two stages of 64 of K ahead.
//  * Token rows are shared by the four wavefronts: they are copied from
//    memory into a 4-stage LDS ring (32 KiB per stage of 64 of K, three
//    stages in flight) by LDS DMA (buffer loads with an LDS destination,
//    lane l's 16 bytes at lane slot l), 8 rows of 128 bytes per instruction:
//    whole 128-byte lines per 8 lanes run at the full L2-to-LDS rate, where
//    16-byte pieces of 16 rows per instruction run at a third of it.
//  * With one wavefront per SIMD, the matrix core idles whenever the
//    wavefront stops issuing MFMAs (a run of other instructions, a wait), so
//    the loop is software-pipelined by hand: each quarter of a stage (16 of
//    K) is 8 groups of two MFMAs (token tile n against the two weight tiles)
//    plus the LDS read of token tile n for the next quarter, with the weight
//    loads and the ring's DMA spread over the groups; scheduling barriers
//    keep the groups in order. Each MFMA pair waits only for its own token
//    fragment.
//  * Down multiplies token rows (A) by weight rows (B), so that lane l holds
//    output feature l % 32: every store writes 128 contiguous bytes of an
//    output row. (Gate/up keeps weights as A: a lane then holds four
//    consecutive features of a row for its gate and up products.)
// Every output sums its K range in ascending order in one accumulator (the
// same products and order either way round). Tiles are ordered feature tile
// major, so the row tiles of one expert that share weights run next to each
// other on one XCD (its L2).
constexpr int kDenseRing = 4;     // token stages in LDS
constexpr int kDenseGroup = 4;    // items per tile group

// Word 3 of a raw buffer resource (32-bit data format) on this part.
constexpr int kBufferFlags = 0x00020000;

// s_waitcnt immediate: wait until at most N vector-memory operations are
// outstanding (other counters left at their maximum).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  __builtin_amdgcn_s_waitcnt((N & 0xF) | ((N >> 4) << 14) | (0x7 << 4) | (0xF << 8));
}

// Workgroup barrier without a memory fence: __syncthreads() would also wait
// for every outstanding load of the wavefront, draining the ring. Each
// wavefront has already waited for its own loads of the stage it needs; LDS
// is coherent inside the CU. The empty asm statements keep the compiler from
// moving memory accesses across the barrier.
__device__ __forceinline__ void ring_barrier() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

typedef float floatx16_t __attribute__((ext_vector_type(16)));

// One 32x32 output tile over 16 of K: v_mfma_f32_32x32x16_bf16. A: lane l
// holds row l%32, k 8*(l/32)..+7; B: lane l holds column l%32, the same k;
// D: lane l, register r -> row 8*(r/4) + 4*(l/32) + r%4, column l%32.
__device__ __forceinline__ void mma32(floatx16_t& acc, const u32x4_t& a, const u32x4_t& b) {
  acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, a),
                                               __builtin_bit_cast(bf16x8_t, b), acc, 0, 0, 0);
}

// Reads of the token ring are inline assembly, with explicit waits: the
// compiler cannot tell which stage a read touches, so for its own LDS reads it
// would wait for every LDS DMA in flight (vmcnt(0)) and drain the ring.
__device__ __forceinline__ u32x4_t lds_read16(uint32_t addr) {
  u32x4_t v;
  asm volatile("ds_read_b128 %0, %1" : "=v"(v) : "v"(addr));
  return v;
}

__device__ __forceinline__ uint32_t lds_addr(const void* p) {
  return static_cast<uint32_t>(reinterpret_cast<uintptr_t>(p));
}

// Token stage layout: instruction j of a stage holds rows 8j..8j+7, row r's
// 16-byte chunk c (8 of K) at lane 8 (r%8) + (c ^ tok_swz(r)). The rotation
// makes the operand reads of 8 or 16 consecutive rows hit distinct banks.
__device__ __forceinline__ int tok_swz(int r) { return (r ^ (r >> 3)) & 7; }

// Wait until at most N LDS operations are outstanding; the operand is tied
// through the wait so that nothing reads it before.
template <int N>
__device__ __forceinline__ void wait_lgkm1(u32x4_t& b) {
  asm volatile("s_waitcnt lgkmcnt(%1)" : "+v"(b) : "n"(N));
}

// Wait for token fragment n of the last quarter of a tile, when no reads of
// a next quarter follow it (NT - 1 - n reads issued after it).
template <int NT>
__device__ __forceinline__ void wait_last(u32x4_t& b, int n) {
  if constexpr (NT == 8) {
    switch (n) {
      case 0: wait_lgkm1<7>(b); break;
      case 1: wait_lgkm1<6>(b); break;
      case 2: wait_lgkm1<5>(b); break;
      case 3: wait_lgkm1<4>(b); break;
      case 4: wait_lgkm1<3>(b); break;
      case 5: wait_lgkm1<2>(b); break;
      case 6: wait_lgkm1<1>(b); break;
      default: wait_lgkm1<0>(b); break;
    }
  } else {
    wait_lgkm1<0>(b);
  }
}

template <int V>
using ic_t = std::integral_constant<int, V>;

// One tile: NT token tiles of 32 rows (item rows <= 32 NT).
//
// Issue order. Stage s of 64 of K has quarters q0..q3; group n of quarter q
// issues { MFMA pair of token tile n, LDS read n of the next quarter }, and
// group 0 also two weight loads: in q0 W(s+1) quarter 3, in q1..q3 W(s+2)
// quarter q-1 (each into registers freed by the quarter before). Barrier
// B(s+1) sits between q2 and q3 (stage s+1 landed for every wavefront, stage
// s-1's slot free); q3 also issues DMA instruction n of DMA(s+3) into that
// slot, after its weight loads. The prologue issues the same sequence for
// stages -3..-1: DMA(0); W(0) q0..q2, DMA(1); W(0) q3, W(1) q0..q2, DMA(2).
// Vector-memory operations complete in issue order, so the wait before
// B(s+1) may leave outstanding what was issued after DMA(s+1): all of stage
// s-1 and q0..q2 of stage s, 14 + NT in steady state (10 two stages from the
// end, where no DMA and only the last weight quarter remain).
template <bool UP, int NT>
__device__ __forceinline__ void dense_tile(const FfnLaunch& a, const WorkItem& it, int f0,
                                           const uint16_t* W, u32x4_t (*ring)[32][64]) {
  constexpr int FRAG = 512;               // packed fragment: 16 rows x 32 of K
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);  // uniform: scalar LDS bases
  const int H = a.H, I = a.I;
  const int K = UP ? H : I;
  const int NS = K / 64;                  // stages (a multiple of 4)
  const int S32 = K / 32;                 // packed fragments per 16 weight rows
  const uint16_t* src = static_cast<const uint16_t*>(a.src);

  // token rows: NT DMA instructions per wavefront per stage, through a
  // buffer resource over the source (reads past src_bytes return zeros).
  // The per-lane byte offsets stay in registers for the whole tile; a stage
  // adds 128 bytes through the scalar offset.
  int toff[NT];
#pragma unroll
  for (int i = 0; i < NT; ++i) {
    const int r = 8 * (wave * NT + i) + (lane >> 3);
    const int rr = min(r, it.rows - 1);   // rows past the item read its last
    const int pos = it.row_begin + rr;
    const int c = (lane & 7) ^ tok_swz(r);
    toff[i] = (UP ? (a.perm[pos] / a.k) * H : pos * I) * 2 + 16 * c;
  }
  const __amdgpu_buffer_rsrc_t trs = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint16_t*>(src), 0, static_cast<int>(a.src_bytes), kBufferFlags);
  auto dma1 = [&](int s, int i) {
    u32x4_t (*stage)[64] = ring[s % kDenseRing];
    __builtin_amdgcn_raw_ptr_buffer_load_lds(
        trs, (__attribute__((address_space(3))) void*)(stage[wave * NT + i]), 16, toff[i],
        128 * s, 0, 0);
  };
  auto dma_all = [&](int s) {
#pragma unroll
    for (int i = 0; i < NT; ++i) dma1(s, i);
  };

  // weights: two 32-row tiles per wavefront (gate and up of 32 features, or
  // 64 down features). Lane l holds row l%32 (16-row fragment (l/16)%2) and
  // the 8 of K at fragment lane l%16 + 16 (2 q + l/32) for the half q of a
  // 32 step.
  const uint16_t* wp[2];
  size_t wstep;
  {
    const int m16 = (lane & 15) + 16 * (lane >> 5);
    const int q0 = f0 / 16;
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      if (UP) {
        const int q = q0 + 2 * wave + ((lane >> 4) & 1);
        wp[t] = W + ((static_cast<size_t>(q) * S32) * 2 + t) * FRAG + 8 * m16;
      } else {
        const int q = q0 + 4 * wave + 2 * t + ((lane >> 4) & 1);
        wp[t] = W + static_cast<size_t>(2) * I * H + static_cast<size_t>(q) * S32 * FRAG + 8 * m16;
      }
    }
    wstep = (UP ? 2 : 1) * FRAG;
  }
  // weight quarter h (16 of K) of stage s: one 16-byte load per weight tile
  auto load_wq = [&](int s, int h, u32x4_t (&w)[2][4]) {
#pragma unroll
    for (int t = 0; t < 2; ++t) w[t][h] = ldg16(wp[t] + (2 * s + (h >> 1)) * wstep + 256 * (h & 1));
  };

  floatx16_t acc[2][NT];
#pragma unroll
  for (int t = 0; t < 2; ++t)
#pragma unroll
    for (int n = 0; n < NT; ++n)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[t][n][r] = 0.f;

  // operand position of token tile n for this lane (chunk c added later)
  uint32_t brow_off[NT];
  int bsw[NT];
#pragma unroll
  for (int n = 0; n < NT; ++n) {
    const int r = 32 * n + (lane & 31);
    brow_off[n] = static_cast<uint32_t>((r >> 3) * 1024 + 128 * (lane & 7));
    bsw[n] = tok_swz(r);
  }
  const uint32_t ring_base = lds_addr(&ring[0][0][0]);
  auto read1 = [&](int s, int h, int n) {
    const uint32_t sbase = ring_base + static_cast<uint32_t>(s % kDenseRing) * (32 * 64 * 16);
    const int c = 2 * h + (lane >> 5);
    return lds_read16(sbase + brow_off[n] + 16 * (c ^ bsw[n]));
  };

  u32x4_t wr[2][2][4];   // weights of stages of even / odd index
  dma_all(0);
  asm volatile("" ::: "memory");
  load_wq(0, 0, wr[0]);
  load_wq(0, 1, wr[0]);
  load_wq(0, 2, wr[0]);
  asm volatile("" ::: "memory");
  dma_all(1);
  asm volatile("" ::: "memory");
  load_wq(0, 3, wr[0]);
  load_wq(1, 0, wr[1]);
  load_wq(1, 1, wr[1]);
  load_wq(1, 2, wr[1]);
  asm volatile("" ::: "memory");
  dma_all(2);
  asm volatile("" ::: "memory");
  wait_vmcnt<14 + 2 * NT>();   // DMA(0) landed
  ring_barrier();              // B(0)
  u32x4_t bq[2][NT];           // token fragments of the current / next quarter
#pragma unroll
  for (int n = 0; n < NT; ++n) bq[0][n] = read1(0, 0, n);

  // NX: a next stage exists; DMA: issue DMA(s+3); W1: load W(s+1) quarter 3;
  // W2: load W(s+2); CNT: the wait before B(s+1)
  auto stage_body = [&](auto nx, auto dma, auto w1, auto w2, auto cnt, int s,
                        u32x4_t (&w)[2][4], u32x4_t (&wn)[2][4]) {
    constexpr bool NX = decltype(nx)::value, DM = decltype(dma)::value;
    constexpr bool W1 = decltype(w1)::value, W2 = decltype(w2)::value;
#pragma unroll
    for (int h = 0; h < 4; ++h) {
      if (h == 3) {
        if constexpr (NX) {
          asm volatile("" ::: "memory");
          wait_vmcnt<decltype(cnt)::value>();
          ring_barrier();  // B(s+1)
        }
      }
      u32x4_t (&cur)[NT] = bq[h & 1];
      u32x4_t (&nxt)[NT] = bq[(h + 1) & 1];
      const bool reads_next = h < 3 || NX;
#pragma unroll
      for (int n = 0; n < NT; ++n) {
        // reads in flight after fragment n: the rest of this quarter and
        // the next quarter's reads issued so far, NT - 1 in all
        if (reads_next) wait_lgkm1<NT - 1>(cur[n]);
        else wait_last<NT>(cur[n], n);
        if (UP) {
          mma32(acc[0][n], w[0][h], cur[n]);
          mma32(acc[1][n], w[1][h], cur[n]);
        } else {
          mma32(acc[0][n], cur[n], w[0][h]);
          mma32(acc[1][n], cur[n], w[1][h]);
        }
        if (h < 3) nxt[n] = read1(s, h + 1, n);
        else if constexpr (NX) nxt[n] = read1(s + 1, 0, n);
        if (n == 0) {
          asm volatile("" ::: "memory");
          if (h == 0) {
            if constexpr (W1) load_wq(s + 1, 3, wn);
          } else {
            if constexpr (W2) load_wq(s + 2, h - 1, w);
          }
          asm volatile("" ::: "memory");
        }
        if (h == 3) {
          if constexpr (DM) dma1(s + 3, n);
        }
        __builtin_amdgcn_sched_barrier(0);
      }
    }
  };
  using T_ = std::true_type;
  using F_ = std::false_type;
  constexpr int STEADY = 14 + NT;
  int s = 0;
  for (; s + 4 < NS; s += 2) {
    stage_body(T_{}, T_{}, T_{}, T_{}, ic_t<STEADY>{}, s, wr[0], wr[1]);
    stage_body(T_{}, T_{}, T_{}, T_{}, ic_t<STEADY>{}, s + 1, wr[1], wr[0]);
  }
  // the last four stages (NS - 4 is even)
  stage_body(T_{}, T_{}, T_{}, T_{}, ic_t<STEADY>{}, s, wr[0], wr[1]);
  stage_body(T_{}, F_{}, T_{}, T_{}, ic_t<STEADY>{}, s + 1, wr[1], wr[0]);
  stage_body(T_{}, F_{}, T_{}, F_{}, ic_t<10>{}, s + 2, wr[0], wr[1]);
  stage_body(F_{}, F_{}, F_{}, F_{}, ic_t<0>{}, s + 3, wr[1], wr[0]);

  const int col = lane & 31, hi = lane >> 5;
  if constexpr (UP) {
    // lane l holds token row 32 n + l%32 and, for register r, weight row
    // 8 (r/4) + 4 (l/32) + r%4 of each weight tile
#pragma unroll
    for (int n = 0; n < NT; ++n) {
      const int row = 32 * n + col;
      if (row >= it.rows) continue;
      const size_t pos = static_cast<size_t>(it.row_begin + row);
#pragma unroll
      for (int r4 = 0; r4 < 4; ++r4) {
        const int f = f0 + 32 * wave + 8 * r4 + 4 * hi;
        float hv[4];
#pragma unroll
        for (int r = 0; r < 4; ++r)
          hv[r] = TrBF16::silu(acc[0][n][4 * r4 + r]) * acc[1][n][4 * r4 + r];
        uint2 packed;
        packed.x = f32_to_bf16_rne(hv[0]) | (static_cast<uint32_t>(f32_to_bf16_rne(hv[1])) << 16);
        packed.y = f32_to_bf16_rne(hv[2]) | (static_cast<uint32_t>(f32_to_bf16_rne(hv[3])) << 16);
        *reinterpret_cast<uint2*>(static_cast<uint16_t*>(a.hout) + pos * I + f) = packed;
      }
    }
  } else {
    // lane l holds feature 32 t + l%32 of the wavefront's 64 and, for
    // register r, token row 8 (r/4) + 4 (l/32) + r%4 of token tile n
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      float* o = a.oout + f0 + 64 * wave + 32 * t + col;
#pragma unroll
      for (int n = 0; n < NT; ++n)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int row = 32 * n + 8 * (r >> 2) + 4 * hi + (r & 3);
          if (row < it.rows) o[static_cast<size_t>(it.row_begin + row) * H] = acc[t][n][r];
        }
    }
  }
}

// Dense launch: one tile per workgroup. Items [0, c0) hold 256 rows each
// and [c0, c0 + c1) fewer ((c0, c1) = item_counts on the device); full tiles
// come first in dispatch order and the short ones last, so the hardware's
// in-order dispatch balances the CUs. Within each class the tiles are spread
// over the XCDs in contiguous ranges.
template <bool UP>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(1, 1)))
void k_ffn_dense(FfnLaunch a) {
  __shared__ u32x4_t s_ring[kDenseRing][32][64];
  constexpr int DF = UP ? 128 : 256;
  const int n_full = a.item_counts[0], n_short = a.item_counts[1];
  const int nf = (UP ? a.I : a.H) / DF;
  const int t = blockIdx.x;
  int v, n, first;
  if (t < n_full * nf) {
    v = xcd_order(t, n_full * nf);
    n = n_full;
    first = 0;
  } else {
    const int u = t - n_full * nf;
    if (u >= n_short * nf) return;
    v = xcd_order(u, n_short * nf);
    n = n_short;
    first = n_full;
  }
  // groups of kDenseGroup items, feature tile major inside a group: the
  // tiles running at once on an XCD share a few token row blocks and a few
  // weight slices through its L2
  const int gsz = kDenseGroup * nf;
  const int g = v / gsz, rem = v - g * gsz;
  const int gi = min(kDenseGroup, n - g * kDenseGroup);
  const int ft = rem / gi;
  const WorkItem it = a.items[a.item_base + first + g * kDenseGroup + (rem - ft * gi)];
  const int slot = it.pad >= 0 ? it.pad : a.slot_of[it.expert];
  if (slot < 0 || slot >= a.n_slots || it.rows <= 0 || it.rows > kDenseRows) return;
  const uint16_t* W = reinterpret_cast<const uint16_t*>(static_cast<const char*>(a.pool) +
                                                        static_cast<int64_t>(slot) * a.slot_bytes);
  if (it.rows > 128) dense_tile<UP, 8>(a, it, ft * DF, W, s_ring);
  else if (it.rows > 64) dense_tile<UP, 4>(a, it, ft * DF, W, s_ring);
  else if (it.rows > 32) dense_tile<UP, 2>(a, it, ft * DF, W, s_ring);
  else dense_tile<UP, 1>(a, it, ft * DF, W, s_ring);
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
                       part_grid(a, (UP ? a.I : a.H) / (kFeat * kFG * (kWaves / KS)));
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
  const int gd = part_grid(d, d.H / (kFeat * kFG * (kWaves / KSD)));
  const int gu = part_grid(u, u.I / (kFeat * kFG * (kWaves / KSU)));
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

hipError_t launch_ffn_dense(bool up, const FfnLaunch& a, hipEvent_t ev0, hipEvent_t ev1,
                            hipStream_t s) {
  if (a.H % 256 || a.I % 256 || a.src_bytes <= 0 || a.src_bytes > INT32_MAX) return hipErrorInvalidValue;
  const int64_t grid = static_cast<int64_t>(a.max_items) * (up ? a.I / 128 : a.H / 256);
  if (grid <= 0) return hipSuccess;
  if (grid > INT32_MAX) return hipErrorInvalidValue;
  if (up)
    hipExtLaunchKernelGGL(k_ffn_dense<true>, dim3(static_cast<unsigned>(grid)), dim3(kThreads), 0, s,
                          ev0, ev1, 0, a);
  else
    hipExtLaunchKernelGGL(k_ffn_dense<false>, dim3(static_cast<unsigned>(grid)), dim3(kThreads), 0,
                          s, ev0, ev1, 0, a);
  return hipGetLastError();
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
