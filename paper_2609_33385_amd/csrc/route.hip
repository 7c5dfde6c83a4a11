// K1 top-k routing and K2 histogram / prefix-sum / stable permutation for one
// denoising block (OLED-MoE Sec. 4.1: the gate yields routed expert ids and
// gate scores for every token of the block; Sec. 4.2: the active set A, the
// misses M = A \ R, each given a staging slot in the device cache state), and
// the gate GEMM that can precede them (logits = x W_gate^T, Sec. 2.1).
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include <type_traits>

#include "kernels.h"

namespace oled {
namespace {

// Order-preserving 32-bit key of a logit (-0.0 ranks equal to +0.0).
__device__ __forceinline__ uint32_t ord_key(float v) {
  uint32_t b = __float_as_uint(v);
  if ((b << 1) == 0u) b = 0u;
  return (b & 0x80000000u) ? ~b : (b | 0x80000000u);
}

// Median of three (the compiler emits one v_med3_u32 for this form).
__device__ __forceinline__ uint32_t med3u(uint32_t a, uint32_t b, uint32_t c) {
  return max(min(a, b), min(max(a, b), c));
}

__device__ __forceinline__ float ord_value(uint32_t o) {
  return __uint_as_float((o & 0x80000000u) ? (o & 0x7FFFFFFFu) : ~o);
}

// Maximum over the 64 lanes of a wavefront of values >= 0 (DPP row shifts
// and row broadcasts as in an inclusive scan; lane 63 ends with the maximum).
__device__ __forceinline__ uint32_t wave_max(uint32_t v) {
  v = max(v, static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, static_cast<int>(v), 0x111, 0xf, 0xf, true)));
  v = max(v, static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, static_cast<int>(v), 0x112, 0xf, 0xf, true)));
  v = max(v, static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, static_cast<int>(v), 0x114, 0xf, 0xf, true)));
  v = max(v, static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, static_cast<int>(v), 0x118, 0xf, 0xf, true)));
  v = max(v, static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, static_cast<int>(v), 0x142, 0xa, 0xf, false)));
  v = max(v, static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, static_cast<int>(v), 0x143, 0xc, 0xf, false)));
  return static_cast<uint32_t>(__builtin_amdgcn_readlane(static_cast<int>(v), 63));
}

__device__ __forceinline__ double readlane_f64(double x, int lane) {
  const uint64_t b = __double_as_longlong(x);
  const uint32_t lo = __builtin_amdgcn_readlane(static_cast<int>(static_cast<uint32_t>(b)), lane);
  const uint32_t hi = __builtin_amdgcn_readlane(static_cast<int>(static_cast<uint32_t>(b >> 32)), lane);
  return __longlong_as_double(static_cast<long long>((static_cast<uint64_t>(hi) << 32) | lo));
}

// Routes one token with one wavefront; lane l owns experts l, l+64, ... (EPL
// per lane) of the logit row (global memory or LDS). Slot j takes the largest
// remaining key in the order (logit desc, id asc): a wavefront maximum of the
// ordered keys, then the lowest expert id holding it (ballots in expert
// order), which leaves the candidates. Keys of valid experts are >= 1, so a
// taken or absent expert (key 0) is never chosen again. Lane j < k keeps slot
// j's expert and logit, takes e_j = exp(l_j - l_0) in fp64; every lane sums
// e_0 + ... + e_{k-1} in slot order, and lane j returns g_j = fl32(e_j / s)
// and its expert (else -1). *bad is set if a logit is non-finite.
template <int EPL>
__device__ __forceinline__ int route_token(const float* row, int E, int k,
                                           float* __restrict__ gate_out, int* bad) {
  const int lane = threadIdx.x & 63;
  uint32_t ok[EPL];
  int nonfinite = 0;
#pragma unroll
  for (int q = 0; q < EPL; ++q) {
    const int e = lane + 64 * q;
    ok[q] = 0u;
    if (e < E) {
      const float v = row[e];
      nonfinite |= !__builtin_isfinite(v);
      ok[q] = max(ord_key(v), 1u);
    }
  }
  *bad |= __any(nonfinite);
  int my_e = -1;
  uint32_t my_key = 0u, key0 = 0u;
  for (int j = 0; j < k; ++j) {
    uint32_t lm = ok[0];
#pragma unroll
    for (int q = 1; q < EPL; ++q) lm = max(lm, ok[q]);
    const uint32_t m = wave_max(lm);
    int id = -1;
#pragma unroll
    for (int q = 0; q < EPL; ++q) {
      const uint64_t b = __ballot(ok[q] == m);
      if (id < 0 && b != 0ull) id = 64 * q + __builtin_ctzll(b);
    }
#pragma unroll
    for (int q = 0; q < EPL; ++q)
      if (lane + 64 * q == id) ok[q] = 0u;
    if (lane == j) {
      my_e = id;
      my_key = m;
    }
    if (j == 0) key0 = m;
  }
  const double v0 = static_cast<double>(ord_value(key0));
  const double ex = lane < k ? exp(static_cast<double>(ord_value(my_key)) - v0) : 0.0;
  double s = 0.0;
  for (int j = 0; j < k; ++j) s += readlane_f64(ex, j);
  *gate_out = static_cast<float>(ex / s);
  return lane < k ? my_e : -1;
}

// Inclusive prefix sum over the 64 lanes of a wavefront: shifts by 1, 2, 4
// and 8 within each row of 16 lanes, then the row totals carried to the rows
// above (DPP row_shr and row_bcast; lanes without a source add zero).
__device__ __forceinline__ int wave_incl_scan(int v) {
  v += __builtin_amdgcn_update_dpp(0, v, 0x111, 0xf, 0xf, true);
  v += __builtin_amdgcn_update_dpp(0, v, 0x112, 0xf, 0xf, true);
  v += __builtin_amdgcn_update_dpp(0, v, 0x114, 0xf, 0xf, true);
  v += __builtin_amdgcn_update_dpp(0, v, 0x118, 0xf, 0xf, true);
  v += __builtin_amdgcn_update_dpp(0, v, 0x142, 0xa, 0xf, false);
  v += __builtin_amdgcn_update_dpp(0, v, 0x143, 0xc, 0xf, false);
  return v;
}

__device__ __forceinline__ int wave_total(int incl) { return __builtin_amdgcn_readlane(incl, 63); }

// Inclusive prefix sum within each row of 16 lanes (the first four steps of
// wave_incl_scan).
__device__ __forceinline__ int row16_incl_scan(int v) {
  v += __builtin_amdgcn_update_dpp(0, v, 0x111, 0xf, 0xf, true);
  v += __builtin_amdgcn_update_dpp(0, v, 0x112, 0xf, 0xf, true);
  v += __builtin_amdgcn_update_dpp(0, v, 0x114, 0xf, 0xf, true);
  v += __builtin_amdgcn_update_dpp(0, v, 0x118, 0xf, 0xf, true);
  return v;
}

// T tokens in blocks of Tb: a non-finite logit of token t sets bad_flag[t / Tb].
template <int EPL>
__global__ __launch_bounds__(256) void k_route_topk(const float* __restrict__ logits, int T, int E,
                                                    int k, int32_t* __restrict__ topk_idx,
                                                    float* __restrict__ gates,
                                                    int32_t* __restrict__ bad_flag, int Tb) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int nwaves = gridDim.x * 4;
  for (int t = blockIdx.x * 4 + wave; t < T; t += nwaves) {
    float g;
    int bad = 0;
    const int e = route_token<EPL>(logits + static_cast<size_t>(t) * E, E, k, &g, &bad);
    if (lane < k) {
      topk_idx[static_cast<size_t>(t) * k + lane] = e;
      gates[static_cast<size_t>(t) * k + lane] = g;
    }
    if (bad && lane == 0) atomicOr(&bad_flag[t / Tb], 1);
  }
}

// Large blocks: one token per lane. A wavefront takes 64 tokens; their
// logits pass through LDS 32 experts at a time (coalesced row loads, one
// padded row per token), the next 32 already in flight while the current ones
// are ranked. Each lane ranks its token's experts by a packed 32-bit key: the
// top 24 bits of the order-preserving logit key, then 255 - id, so that one
// max / min pair per list position inserts (a bubble network over KP >= k + 1
// positions). Where the k + 1 best packed keys differ in their top 24 bits,
// their order is the exact (logit desc, id asc) order and the first k are the
// routes; where two of them share those bits the whole wavefront ranks that
// token again from memory with full keys (wave_topk_ids). Gates as in route_token (fp64 exp of
// l_j - l_0, sum in slot order, one rounding to fp32), from the logits re-read
// by expert id.
constexpr int kLaneChunk = 32;
constexpr int kLaneRow = kLaneChunk + 1;   // padded LDS row (floats): conflict-free lane reads
constexpr int kLaneRowsPerLoad = 64 / kLaneChunk;

// The whole wavefront ranks one row with full keys (E <= 256): k rounds of a
// wavefront maximum, the lowest id holding it taken by ballot, as in
// route_token; the lane that owns the token keeps the ids.
template <int KM>
__device__ __forceinline__ void wave_topk_ids(const float* row, int E, int k, bool mine,
                                              int32_t (&ids)[KM]) {
  const int lane = threadIdx.x & 63;
  uint32_t ok[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int e = lane + 64 * q;
    ok[q] = e < E ? max(ord_key(row[e]), 1u) : 0u;
  }
#pragma unroll
  for (int j = 0; j < KM; ++j) {
    if (j < k) {
      const uint32_t m = wave_max(max(max(ok[0], ok[1]), max(ok[2], ok[3])));
      int id = -1;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const uint64_t bq = __ballot(ok[q] == m);
        if (id < 0 && bq != 0ull) id = 64 * q + __builtin_ctzll(bq);
      }
#pragma unroll
      for (int q = 0; q < 4; ++q)
        if (lane + 64 * q == id) ok[q] = 0u;
      if (mine) ids[j] = id;
    }
  }
}

// Word 3 of a raw buffer resource (32-bit data format) on this part.
constexpr int kRouteBufferFlags = 0x00020000;

// s_waitcnt immediate: at most N vector-memory operations outstanding.
template <int N>
__device__ __forceinline__ void route_wait_vmcnt() {
  __builtin_amdgcn_s_waitcnt((N & 0xF) | ((N >> 4) << 14) | (0x7 << 4) | (0xF << 8));
}

typedef uint32_t u32x4r_t __attribute__((ext_vector_type(4)));

__device__ __forceinline__ u32x4r_t lds_read16r(uint32_t addr) {
  u32x4r_t v;
  asm volatile("ds_read_b128 %0, %1" : "=v"(v) : "v"(addr));
  return v;
}

// 4-byte LDS accesses as inline assembly, ordered with explicit lgkmcnt
// waits: the compiler's own LDS accesses would wait for every LDS DMA in
// flight.
__device__ __forceinline__ void lds_write4r(uint32_t addr, uint32_t v) {
  asm volatile("ds_write_b32 %0, %1" ::"v"(addr), "v"(v) : "memory");
}
__device__ __forceinline__ uint32_t lds_read4r(uint32_t addr) {
  uint32_t v;
  asm volatile("ds_read_b32 %0, %1" : "=v"(v) : "v"(addr) : "memory");
  return v;
}
template <int N>
__device__ __forceinline__ void lds_wait_all(uint32_t (&v)[N]) {
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
#pragma unroll
  for (int i = 0; i < N; ++i) asm volatile("" : "+v"(v[i]));
}

// DMA streaming (E % 32 == 0, the rows within a 32-bit byte offset): each
// wavefront ranks several blocks of 64 tokens in turn, its logits copied into
// LDS 32 experts (128 bytes per row) at a time by LDS DMA, two chunks in
// flight across block boundaries; no staging registers. DMA instruction i of
// a chunk moves rows 8 i .. 8 i + 7: lane l = 8 r + s loads the 16-byte slot
// s ^ r of row 8 i + r into LDS slot l, so that token t's slot c sits at
// 8 t + (c ^ (t % 8)) and the 8 lanes of each LDS access group read 8
// distinct bank groups. A block's ids are written when its ranking ends; the
// logits of its routes for the gates are loaded then and the gates computed
// after the next block, so the wavefront does not wait for those loads.
// Otherwise (register staging) one block per wavefront, one 4-byte load per
// lane through registers and a padded LDS row.
template <int KP, int KM, bool DMA>
__global__ __launch_bounds__(256) void k_route_lanes(const float* __restrict__ logits, int T, int E,
                                                     int k, int32_t* __restrict__ topk_idx,
                                                     float* __restrict__ gates,
                                                     int32_t* __restrict__ bad_flag, int Tb) {
  static_assert(KP > KM, "the packed list holds the k-th and the (k+1)-th key");
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  uint32_t key[KP];
  int nonfinite = 0;
  auto reset = [&]() {
#pragma unroll
    for (int j = 0; j < KP; ++j) key[j] = 0u;
    nonfinite = 0;
  };
  auto insert = [&](float x, int e) {
    nonfinite |= !__builtin_isfinite(x);
    const uint32_t c = (max(ord_key(x), 1u) & 0xFFFFFF00u) | static_cast<uint32_t>(255 - e);
    // insertion into the descending list: new[q] = max(old[q], min(old[q-1], c)),
    // the median of (old[q-1], old[q], c) since old[q-1] >= old[q]: one
    // v_med3_u32 per position, every position from the old list
#pragma unroll
    for (int q = KP - 1; q >= 1; --q) key[q] = med3u(key[q - 1], key[q], c);
    key[0] = max(key[0], c);
  };
  // ids of the block at t0 from the lanes' keys: where two of the k + 1 best
  // share their top 24 bits, the whole wavefront ranks that token again from
  // memory with full keys
  auto block_ids = [&](int t0, int32_t (&id)[KM]) {
    const int t = t0 + lane;
    bool amb = false;
    if (t < T) {
#pragma unroll
      for (int j = 0; j + 1 < KP; ++j)
        if (j < k) amb |= (key[j] >> 8) == (key[j + 1] >> 8);
    }
#pragma unroll
    for (int j = 0; j < KM; ++j) id[j] = 255 - static_cast<int>(key[j] & 0xFFu);
    for (uint64_t todo = __ballot(amb); todo != 0ull; todo &= todo - 1) {
      const int owner = __builtin_ctzll(todo);
      wave_topk_ids<KM>(logits + static_cast<size_t>(t0 + owner) * E, E, k, lane == owner, id);
    }
  };
  // gates of token t from the logits of its routes: fp64 exp of l_j - l_0,
  // summed in slot order, one rounding to fp32
  auto write_gates = [&](const float (&lvf)[KM], int t) {
    double ex[KM];
    double sum = 0.0;
#pragma unroll
    for (int j = 0; j < KM; ++j) {
      ex[j] = j < k ? exp(static_cast<double>(lvf[j]) - static_cast<double>(lvf[0])) : 0.0;
      if (j < k) sum += ex[j];
    }
#pragma unroll
    for (int j = 0; j < KM; ++j)
      if (j < k) gates[static_cast<size_t>(t) * k + j] = static_cast<float>(ex[j] / sum);
  };
  if constexpr (DMA) {
    __shared__ u32x4r_t s_dma[4][2][64 * 8];   // [wavefront][buffer][token][slot]: 64 KiB
    const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<float*>(logits), 0, T * E * 4, kRouteBufferFlags);   // rows past T read 0
    const int r8 = lane >> 3, s8 = lane & 7;
    const int nch = E / 32;
    const int stride = static_cast<int>(gridDim.x) * 4;   // blocks per grid step
    const int blk0 = static_cast<int>(blockIdx.x) * 4 + wave;
    const int nblk = (T + 63) >> 6;
    const int my_n = blk0 < nblk ? (nblk - 1 - blk0) / stride + 1 : 0;
    const int total = my_n * nch;   // chunks of this wavefront
    auto dma = [&](int g) {
      const int bi = g / nch, c = g - bi * nch;
      const int voff = ((blk0 + bi * stride) * 64 + r8) * E * 4 + 16 * (s8 ^ r8);
#pragma unroll
      for (int i = 0; i < 8; ++i)
        __builtin_amdgcn_raw_ptr_buffer_load_lds(
            rs, (__attribute__((address_space(3))) void*)(&s_dma[wave][g & 1][64 * i]), 16,
            voff + i * 8 * E * 4, 128 * c, 0, 0);
    };
    if (total > 0) dma(0);
    if (total > 1) dma(1);
    const uint32_t rbase = static_cast<uint32_t>(reinterpret_cast<uintptr_t>(&s_dma[wave][0][0])) +
                           16u * 8u * static_cast<uint32_t>(lane);
    const int sw = lane & 7;
    bool pend = false;   // a block whose gates are still to be written
    int pt = 0;
    float gv[KM];        // its route logits: token (64 m + lane) / KM, slot lane % KM
    uint32_t gon = 0u;   // bit m: gv[m] is a route's logit
#pragma unroll
    for (int j = 0; j < KM; ++j) gv[j] = 0.f;
    __shared__ uint32_t s_tbl[4][64 * KM];   // per wavefront: [token][slot] ids, then logits
    const uint32_t tbl = static_cast<uint32_t>(reinterpret_cast<uintptr_t>(&s_tbl[wave][0]));
    // gates of the pending block: its logits back to one token per lane
    auto finish = [&]() {
#pragma unroll
      for (int m = 0; m < KM; ++m)
        lds_write4r(tbl + 4u * (64 * m + lane), ((gon >> m) & 1u) ? __float_as_uint(gv[m]) : 0u);
      asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
      uint32_t lvu[KM];
#pragma unroll
      for (int j = 0; j < KM; ++j) lvu[j] = lds_read4r(tbl + 4u * (KM * lane + j));
      lds_wait_all(lvu);
      float lvf[KM];
#pragma unroll
      for (int j = 0; j < KM; ++j) lvf[j] = __uint_as_float(lvu[j]);
      if (pt < T) write_gates(lvf, pt);
    };
    for (int g = 0; g < total; ++g) {
      const int bi = g / nch, c = g - bi * nch;
      if (c == 0) reset();
      // wait for DMA(g): issued after it are DMA(g + 1) (8 loads) and, in the
      // first two chunks of every block but the first, the last block's KM
      // gate loads (issued by every lane, so exactly KM; with one chunk per
      // block two blocks' loads, of which counting one only waits longer)
      const bool more = g + 1 < total, loads = c <= 1 && bi >= 1;
      if (more) {
        if (loads) route_wait_vmcnt<8 + KM>();
        else route_wait_vmcnt<8>();
      } else {
        if (loads) route_wait_vmcnt<KM>();
        else route_wait_vmcnt<0>();
      }
      asm volatile("" ::: "memory");
      const uint32_t base = rbase + static_cast<uint32_t>(g & 1) * (64u * 8u * 16u);
      u32x4r_t x[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) x[j] = lds_read16r(base + 16u * static_cast<uint32_t>(j ^ sw));
      asm volatile("s_waitcnt lgkmcnt(0)"
                   : "+v"(x[0]), "+v"(x[1]), "+v"(x[2]), "+v"(x[3]), "+v"(x[4]), "+v"(x[5]),
                     "+v"(x[6]), "+v"(x[7])::"memory");
      if (g + 2 < total) dma(g + 2);   // into the buffer just read
#pragma unroll
      for (int j = 0; j < 8; ++j)
#pragma unroll
        for (int q = 0; q < 4; ++q) insert(__uint_as_float(x[j][q]), 32 * c + 4 * j + q);
      if (c == nch - 1) {   // the block is ranked
        const int t0 = (blk0 + bi * stride) * 64;
        int32_t id[KM];
        block_ids(t0, id);
        const int t = t0 + lane;
        if (t < T) {
#pragma unroll
          for (int j = 0; j < KM; ++j)
            if (j < k) topk_idx[static_cast<size_t>(t) * k + j] = id[j];
          if (nonfinite) atomicOr(&bad_flag[t / Tb], 1);   // token t's block
        }
        if (pend) finish();   // the last block's logits have landed
        // this block's route logits for its gates, loaded with KM lanes per
        // token (through the table) so that one load's lanes share a row
        uint32_t idx[KM];
#pragma unroll
        for (int j = 0; j < KM; ++j) lds_write4r(tbl + 4u * (KM * lane + j), static_cast<uint32_t>(id[j]));
        asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
#pragma unroll
        for (int m = 0; m < KM; ++m) idx[m] = lds_read4r(tbl + 4u * (64 * m + lane));
        lds_wait_all(idx);
        // every lane loads (row t0, expert 0 when inactive); the values are
        // first used after the next block, so nothing waits for them here
        gon = 0u;
#pragma unroll
        for (int m = 0; m < KM; ++m) {
          const int q = 64 * m + lane, jj = q % KM;
          const bool on = t0 + q / KM < T && jj < k;
          const int tok = on ? t0 + q / KM : t0;
          gv[m] = logits[static_cast<size_t>(tok) * E + (on ? static_cast<int>(idx[m]) : 0)];
          gon |= (on ? 1u : 0u) << m;
        }
        asm volatile("" ::: "memory");
        pend = true;
        pt = t;
      }
    }
    if (pend) finish();   // the last block
  } else {
    __shared__ float s_buf[4][64 * kLaneRow];
    float* buf = s_buf[wave];
    const int t0 = (blockIdx.x * 4 + wave) * 64;
    // lane l loads column l % C of rows l / C + (64 / C) i, i < C, of a chunk
    // of C = kLaneChunk experts
    const int lc = lane % kLaneChunk, lr = lane / kLaneChunk;
    float v[kLaneChunk];
    auto load = [&](int e0) {
      const int e = e0 + lc;
#pragma unroll
      for (int i = 0; i < kLaneChunk; ++i) {
        const int t = t0 + lr + kLaneRowsPerLoad * i;
        v[i] = (t < T && e < E) ? logits[static_cast<size_t>(t) * E + e] : 0.f;
      }
    };
    reset();
    load(0);
    // Each wavefront stages its own rows: ordering its LDS writes and reads
    // needs no workgroup barrier, only that the compiler keep them in program
    // order (a wavefront's LDS operations complete in issue order).
    for (int e0 = 0; e0 < E; e0 += kLaneChunk) {
      asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");   // the previous chunk's reads are done
#pragma unroll
      for (int i = 0; i < kLaneChunk; ++i) buf[(lr + kLaneRowsPerLoad * i) * kLaneRow + lc] = v[i];
      if (e0 + kLaneChunk < E) load(e0 + kLaneChunk);
      asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
      const int ne = min(kLaneChunk, E - e0);
      for (int j = 0; j < ne; ++j) insert(buf[lane * kLaneRow + j], e0 + j);
    }
    int32_t id[KM];
    block_ids(t0, id);
    const int t = t0 + lane;
    if (t < T) {
      const float* row = logits + static_cast<size_t>(t) * E;
      float lv[KM];
#pragma unroll
      for (int j = 0; j < KM; ++j) lv[j] = j < k ? row[id[j]] : 0.f;
#pragma unroll
      for (int j = 0; j < KM; ++j)
        if (j < k) topk_idx[static_cast<size_t>(t) * k + j] = id[j];
      write_gates(lv, t);
      if (nonfinite) atomicOr(&bad_flag[t / Tb], 1);   // token t's block
    }
  }
}

constexpr int kPermThreads = 1024;
constexpr int kChunkWords = 16;               // bitmask words per expert per chunk
static_assert(kChunkWords == 16, "the ranking's per-expert prefix is a 16-lane row scan");
constexpr int kChunkTokens = kChunkWords * 32;
// Per-expert token bitmasks of a chunk: rows of kMaskStride = 17 words (16
// words of 32 tokens, one pad word). The lanes of a wavefront share a 32-token
// word and scatter over experts; with 17-word rows they fall in distinct LDS
// banks (with 16-word rows every expert's row began in one of two banks).
constexpr int kMaskStride = kChunkWords + 1;
constexpr int kMaskRows = kMaxExperts + 1;     // + a row that missing routes target
constexpr int kMaskSpare = kMaxExperts * kMaskStride;
constexpr int kRouteBits = 13;                 // chunk-local route index
static_assert(kChunkTokens * kMaxTopK <= 1 << kRouteBits, "chunk-local routes fit 13 bits");
static_assert(kPermThreads == 2 * kChunkTokens, "two threads per token of a chunk");

constexpr int kFusedMaxRoutes = 1024;       // fused routing path: T * k routes kept in LDS
constexpr int kLaneTokensMin = 1024;        // blocks of more tokens route one token per lane
constexpr int kRouteStreamGrid = 512;       // DMA-streamed top-k: two workgroups per CU
constexpr int kGateFullGrid = 256;          // gate GEMM workgroups that fill the compute units
constexpr int kChunkedMinTokens = 1024;     // and permute over many workgroups
constexpr int kMaxChunks = 128;             // chunked permutation: T <= 65535 tokens
// chunks per planning thread: kMaxChunks over the fewest groups (E = 256 at kPermThreads)
constexpr int kPlanPer = kMaxChunks / (kPermThreads / kMaxExperts);

// Stable positions of the routes of tokens [t0, t1) (at most kChunkTokens):
// a per-expert bitmask of the chunk's tokens that chose the expert (LDS
// atomics into kMaskStride-word rows), a running popcount prefix per 32-token
// word from the expert's base s_run[e], and each route's position = that
// prefix + the tokens of its word below it (positions outside [0, n_routes)
// are dropped). Advances s_run past the chunk. Every thread of the workgroup
// takes part (any workgroup size).
__device__ __forceinline__ void rank_chunk(const int32_t* idx, int t0, int t1, int k, int E,
                                           int n_routes,
                                           uint32_t* s_mask, int32_t* s_pre, int32_t* s_run,
                                           int32_t* __restrict__ perm,
                                           int32_t* __restrict__ inv_perm) {
  const int tid = threadIdx.x, nthr = blockDim.x;
  for (int i = tid; i < E * kMaskStride; i += nthr) s_mask[i] = 0u;
  __syncthreads();
  for (int r = t0 * k + tid; r < t1 * k; r += nthr) {
    const int e = idx[r];
    const int lt = r / k - t0;
    atomicOr(&s_mask[e * kMaskStride + (lt >> 5)], 1u << (lt & 31));
  }
  __syncthreads();
  for (int i = tid; i < ((E * kChunkWords + 63) & ~63); i += nthr) {
    const int e = i / kChunkWords, w = i & (kChunkWords - 1);
    const int c = e < E ? __popc(s_mask[e * kMaskStride + w]) : 0;
    const int incl = row16_incl_scan(c);
    if (e < E) {
      const int run = s_run[e];
      s_pre[e * kMaskStride + w] = run + incl - c;
      if (w == kChunkWords - 1) s_run[e] = run + incl;
    }
  }
  __syncthreads();
  for (int r = t0 * k + tid; r < t1 * k; r += nthr) {
    const int e = idx[r];
    const int lt = r / k - t0;
    const int w = e * kMaskStride + (lt >> 5);
    const uint32_t below = s_mask[w] & ((1u << (lt & 31)) - 1u);
    const int pos = s_pre[w] + __popc(below);
    if (pos >= 0 && pos < n_routes) {
      perm[pos] = r;
      inv_perm[r] = pos;
    }
  }
  __syncthreads();
}

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
                                             const PermuteOut& o, const int32_t* s_free,
                                             const int32_t* s_ftop, const uint32_t* s_res,
                                             const uint32_t* s_pm, const int32_t* s_slot,
                                             int32_t* __restrict__ chunk_base = nullptr,
                                             int n_chunks = 0) {
  __shared__ int32_t s_cnt[kMaxExperts];
  __shared__ int32_t s_off[kMaxExperts + 1];
  __shared__ int32_t s_item_base[kMaxExperts];
  __shared__ int32_t s_run[kMaxExperts];
  __shared__ int32_t s_stat[18];
  __shared__ int32_t s_dfull[kMaxExperts];   // first full dense item of the expert, or -1
  __shared__ int32_t s_dshort[kMaxExperts];  // its short dense item, or -1
  __shared__ int32_t s_sexp[kMaxExperts];
  __shared__ int32_t s_sslot[kMaxExperts];
  __shared__ uint32_t s_mask[kMaskRows * kMaskStride];
  __shared__ int32_t s_pre[kMaskRows * kMaskStride];

  const int tid = threadIdx.x;
  const int nthr = blockDim.x;
  const int E = o.E, layer = o.layer;
  const int R = T * k;
  const bool cache = o.cv.hdr != nullptr;   // else routing and permutation only
  for (int e = tid; e < kMaxExperts; e += nthr) s_cnt[e] = 0;
  __syncthreads();
  // Chunked: counts per chunk in chunk_base [n_chunks][E], from an earlier
  // launch. G threads per expert each take a contiguous run of at most
  // kPlanPer chunks, loaded at once into registers (kept for the per-chunk
  // bases at the end); their partial sums stay in s_pre (g * E + e), which the
  // chunked path does not otherwise use.
  const int G = chunk_base ? max(1, min(nthr / E, n_chunks)) : 1;
  const int per = chunk_base ? (n_chunks + G - 1) / G : 0;
  const int my_g = chunk_base && tid < G * E ? tid / E : -1;
  const int my_e = my_g >= 0 ? tid - my_g * E : 0;
  const int ch_lo = my_g >= 0 ? my_g * per : 0;
  const int ch_hi = my_g >= 0 ? min(n_chunks, ch_lo + per) : 0;
  int cc[kPlanPer];
  if (chunk_base) {
    int c = 0;
#pragma unroll
    for (int q = 0; q < kPlanPer; ++q) {
      cc[q] = ch_lo + q < ch_hi ? chunk_base[static_cast<size_t>(ch_lo + q) * E + my_e] : 0;
      c += cc[q];
    }
    if (my_g >= 0) s_pre[tid] = c;
    __syncthreads();
    for (int e = tid; e < E; e += nthr) {
      int c = 0;
      for (int g = 0; g < G; ++g) c += s_pre[g * E + e];
      s_cnt[e] = c;
    }
  } else {
    for (int r = tid; r < R; r += nthr) atomicAdd(&s_cnt[idx[r]], 1);
  }
  __syncthreads();

  if (tid < 64) {  // wave 0: scans over experts, 4 per lane (DPP scans)
    const int lane = tid;
    int c[4], nh[4], nm[4];
    bool hit[4], miss[4], dn[4];
    int sc = 0, sh = 0, sm = 0, sx = 0, sdf = 0, sds = 0;
    int n_act = 0, n_hit = 0, n_res = 0, hrows = 0, mrows = 0, n_px = 0, n_rx = 0;
    int n_dense = 0, n_dhit = 0, drows = 0, dhrows = 0;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int e = 4 * lane + q;
      c[q] = e < E ? s_cnt[e] : 0;
      const int ni = (c[q] + kItemRows - 1) / kItemRows;
      const bool res = e < E && ((s_res[e >> 5] >> (e & 31)) & 1u);
      hit[q] = res && c[q] > 0;
      miss[q] = !res && c[q] > 0;
      dn[q] = o.dense_min > 0 && c[q] >= o.dense_min;
      nh[q] = hit[q] && !dn[q] ? ni : 0;
      nm[q] = miss[q] && !dn[q] ? ni : 0;
      sdf += dn[q] ? c[q] / kDenseRows : 0;
      sds += dn[q] && c[q] % kDenseRows ? 1 : 0;
      n_dense += dn[q] ? 1 : 0;
      n_dhit += dn[q] && hit[q] ? 1 : 0;
      drows += dn[q] ? c[q] : 0;
      dhrows += dn[q] && hit[q] ? c[q] : 0;
      sc += c[q];
      sh += nh[q];
      sm += nm[q];
      sx += miss[q] ? 1 : 0;
      n_act += c[q] > 0 ? 1 : 0;
      n_hit += hit[q] ? 1 : 0;
      n_res += res ? 1 : 0;
      const bool pm = e < E && ((s_pm[e >> 5] >> (e & 31)) & 1u);   // transferred last time
      n_px += pm ? 1 : 0;
      n_rx += pm && hit[q] ? 1 : 0;   // retained (resident now) and activated again
      hrows += hit[q] ? c[q] : 0;
      mrows += miss[q] ? c[q] : 0;
    }
    const int ic = wave_incl_scan(sc), ih = wave_incl_scan(sh), im = wave_incl_scan(sm),
              ix = wave_incl_scan(sx);
    n_act = wave_total(wave_incl_scan(n_act));
    n_hit = wave_total(wave_incl_scan(n_hit));
    n_res = wave_total(wave_incl_scan(n_res));
    n_px = wave_total(wave_incl_scan(n_px));
    n_rx = wave_total(wave_incl_scan(n_rx));
    hrows = wave_total(wave_incl_scan(hrows));
    mrows = wave_total(wave_incl_scan(mrows));
    const int tot_hit = wave_total(ih);
    const int n_miss = wave_total(ix);
    const int tot_routes = wave_total(ic);
    const int tot_miss_items = wave_total(im);
    int idf = 0, ids = 0, tot_full = 0, tot_short = 0;
    if (o.dense_min > 0) {
      idf = wave_incl_scan(sdf);
      ids = wave_incl_scan(sds);
      tot_full = wave_total(idf);
      tot_short = wave_total(ids);
      n_dense = wave_total(wave_incl_scan(n_dense));
      n_dhit = wave_total(wave_incl_scan(n_dhit));
      drows = wave_total(wave_incl_scan(drows));
      dhrows = wave_total(wave_incl_scan(dhrows));
    }
    // staging: every miss takes a free slot, unless the block is bad
    CacheHdr* hdr = o.cv.hdr;
    const int free_top = *s_ftop;
    const bool stage = cache && !bad && free_top >= 0 && free_top <= o.cv.n_slots &&
                       n_miss <= free_top;
    int xc = ic - sc, xh = ih - sh, xm = im - sm, xx = ix - sx, xdf = idf - sdf,
        xds = tot_full + ids - sds;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int e = 4 * lane + q;
      if (e < E) {
        s_off[e] = xc;
        s_item_base[e] = (nh[q] > 0) ? xh : tot_hit + xm;
        s_dfull[e] = dn[q] ? xdf : -1;
        s_dshort[e] = dn[q] && c[q] % kDenseRows ? xds : -1;
        if (stage && miss[q]) {
          const int slot = s_free[xx];
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
      xdf += dn[q] ? c[q] / kDenseRows : 0;
      xds += dn[q] && c[q] % kDenseRows ? 1 : 0;
    }
    // this iteration's transferred misses, for the next one: expert e = 4 lane + q
    // is bit 4 (lane % 8) + q of word lane / 8
    uint64_t mb[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) mb[q] = __ballot(stage && miss[q]);
    if (cache && lane < kMaxExperts / 32) {
      uint32_t word = 0u;
#pragma unroll
      for (int j = 0; j < 8; ++j)
#pragma unroll
        for (int q = 0; q < 4; ++q)
          word |= static_cast<uint32_t>((mb[q] >> (8 * lane + j)) & 1ull) << (4 * j + q);
      o.cv.prev_miss[layer].bits[lane] = word;
    }
    if (lane == 0) {
      if (cache) {
        hdr->free_top = stage ? free_top - n_miss : free_top;
        hdr->staged_n = stage ? n_miss : 0;
        hdr->route_bad = stage ? 0 : 1;
        if (!bad && !stage) hdr->fault |= 1;
        int32_t* lc = o.cv.last_counts + kCountsPerLayer * layer;
        lc[0] = n_act;
        lc[1] = n_hit;
        lc[2] = n_miss;
        lc[3] = n_res;
        lc[4] = n_px;
        lc[5] = n_rx;
      } else if (o.bad_out) {
        *o.bad_out = bad ? 1 : 0;
      }
      s_stat[16] = n_px;
      s_stat[17] = n_rx;
      s_stat[0] = n_act;
      s_stat[1] = n_hit;
      s_stat[2] = n_miss;
      s_stat[3] = n_res;
      s_stat[4] = hrows;
      s_stat[5] = mrows;
      s_stat[6] = stage ? n_miss : 0;
      s_stat[7] = stage ? 0 : 1;
      s_off[E] = tot_routes;
      s_stat[8] = tot_hit;
      s_stat[9] = tot_miss_items;
      s_stat[10] = n_dense;
      s_stat[11] = n_dhit;
      s_stat[12] = drows;
      s_stat[13] = dhrows;
      s_stat[14] = tot_full;
      s_stat[15] = tot_short;
    }
    if (cache && lane < kMaxExperts / 32) o.cv.res_before[layer].bits[lane] = s_res[lane];
  }
  __syncthreads();

  for (int e = tid; e < E; e += nthr) {
    const int c = s_cnt[e];
    o.counts[e] = c;
    o.offsets[e] = s_off[e];
    s_run[e] = s_off[e];
    if (!o.items) continue;   // no work lists without a cache
    // a hit's slot cannot change before the layer's retention: the GEMMs take
    // it from the item; a miss's slot is looked up when its GEMM runs
    const int hslot = ((s_res[e >> 5] >> (e & 31)) & 1u) ? s_slot[e] : -1;
    if (s_dfull[e] >= 0) {  // dense: full items, then the expert's short item
      const int full = c / kDenseRows;
      for (int m = 0; m < full; ++m)
        o.dense_items[s_dfull[e] + m] = WorkItem{e, s_off[e] + m * kDenseRows, kDenseRows, hslot};
      if (s_dshort[e] >= 0)
        o.dense_items[s_dshort[e]] = WorkItem{e, s_off[e] + full * kDenseRows, c - full * kDenseRows, hslot};
      continue;
    }
    const int base = s_item_base[e];
    for (int m = 0; m * kItemRows < c; ++m) {
      WorkItem it;
      it.expert = e;
      it.row_begin = s_off[e] + m * kItemRows;
      it.rows = min(kItemRows, c - m * kItemRows);
      it.pad = hslot;
      o.items[base + m] = it;
    }
  }
  if (tid == 0) o.offsets[E] = s_off[E];

  if (chunk_base) {   // per-chunk bases for the ranking launch: exclusive scan over chunks
    if (my_g >= 0) {
      int run = s_off[my_e];
      for (int h = 0; h < my_g; ++h) run += s_pre[h * E + my_e];
#pragma unroll
      for (int q = 0; q < kPlanPer; ++q)
        if (ch_lo + q < ch_hi) {
          chunk_base[static_cast<size_t>(ch_lo + q) * E + my_e] = run;
          run += cc[q];
        }
    }
  } else {
    for (int t0 = 0; t0 < T; t0 += kChunkTokens)
      rank_chunk(idx, t0, min(T, t0 + kChunkTokens), k, E, T * k, s_mask, s_pre, s_run, o.perm,
                 o.inv_perm);
  }
  __syncthreads();

  // the routing record: device ring (read by the host at its synchronisation
  // points), and for host-issued copies the staged list in pinned memory
  if (cache && tid < 64) {
    const int n_staged = s_stat[6];
    RouteStats rs;
    rs.layer = layer;
    rs.n_active = s_stat[0];
    rs.n_hits = s_stat[1];
    rs.n_misses = s_stat[2];
    rs.n_resident = s_stat[3];
    rs.hit_rows = s_stat[4];
    rs.miss_rows = s_stat[5];
    rs.n_staged = n_staged;
    rs.bad = bad ? 1 : s_stat[7];
    rs.n_hit_items = s_stat[8];
    rs.n_miss_items = s_stat[9];
    const bool dense = o.dense_min > 0;
    rs.n_dense = dense ? s_stat[10] : 0;
    rs.n_dense_hits = dense ? s_stat[11] : 0;
    rs.dense_rows = dense ? s_stat[12] : 0;
    rs.dense_hit_rows = dense ? s_stat[13] : 0;
    rs.n_dense_items = dense ? s_stat[14] + s_stat[15] : 0;
    rs.prev_xfer = s_stat[16];
    rs.reused_xfer = s_stat[17];
    rs.ideal_hits = min(o.cv.cap[layer], s_stat[0]);
    rs.seq = o.seq;
    if (tid == 0) {
      o.item_counts[0] = s_stat[8];
      o.item_counts[1] = s_stat[9];
      if (dense) {
        o.dense_counts[0] = s_stat[14];
        o.dense_counts[1] = s_stat[15];
      }
      o.ring[o.seq % kStatsRing] = rs;
    }
    if (o.staged) {
      for (int j = tid; j < n_staged; j += 64) {
        o.staged->exp[j] = s_sexp[j];
        o.staged->slot[j] = s_sslot[j];
      }
      if (o.pub_topk && n_staged > 0) {   // the routes, for the host's dispatch of the misses
        for (int r = tid; r < T * k; r += 64) {
          o.pub_topk[r] = idx[r];
          o.pub_gates[r] = __hip_atomic_load(o.gates + r, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
      }
      if (tid == 0) o.staged->rec = rs;
      __threadfence_system();
      if (tid == 0) *reinterpret_cast<volatile int32_t*>(&o.staged->seq) = o.seq;
    }
  }
}

// One wavefront reads the cache state the planning step needs into LDS: the
// layer's resident set and the experts transferred at its previous iteration
// (words), and the top of the free-slot list.
__device__ __forceinline__ void prefetch_state(const CacheView& cv, int E, int layer,
                                               int32_t* s_free, int32_t* s_ftop, uint32_t* s_res,
                                               uint32_t* s_pm, int32_t* s_slot) {
  const int lane = threadIdx.x & 63;
  if (!cv.hdr) {   // no expert cache: nothing resident, nothing to stage into
#pragma unroll
    for (int q = 0; q < kMaxExperts / 64; ++q)
      if (lane + 64 * q < E) s_slot[lane + 64 * q] = -1;
    if (lane < kMaxExperts / 32) s_res[lane] = 0u;
    else if (lane < kMaxExperts / 16) s_pm[lane - kMaxExperts / 32] = 0u;
    if (lane == 0) *s_ftop = 0;
    return;
  }
#pragma unroll
  for (int q = 0; q < kMaxExperts / 64; ++q) {
    const int e = lane + 64 * q;
    if (e < E) s_slot[e] = cv.slot_of[static_cast<size_t>(layer) * E + e];
  }
  if (lane < kMaxExperts / 32) s_res[lane] = cv.res[layer].bits[lane];
  else if (lane < kMaxExperts / 16) s_pm[lane - kMaxExperts / 32] = cv.prev_miss[layer].bits[lane - kMaxExperts / 32];
  const int ft = cv.hdr->free_top;
  if (ft >= 0 && ft <= cv.n_slots) {
#pragma unroll
    for (int q = 0; q < kMaxExperts / 64; ++q) {
      const int j = lane + 64 * q;
      if (j < E && j < ft) s_free[j] = cv.free_list[ft - 1 - j];
    }
  }
  if (lane == 0) *s_ftop = ft;
}

__global__ __launch_bounds__(kPermThreads) void k_permute(const int32_t* __restrict__ topk_idx,
                                                          int T, int k,
                                                          int32_t* __restrict__ bad_flag,
                                                          PermuteOut o) {
  __shared__ int32_t s_free[kMaxExperts];
  __shared__ int32_t s_ftop;
  __shared__ uint32_t s_res[kMaxExperts / 32], s_pm[kMaxExperts / 32];
  __shared__ int32_t s_slot[kMaxExperts];
  const int bad = *bad_flag;
  if ((threadIdx.x >> 6) == 1) prefetch_state(o.cv, o.E, o.layer, s_free, &s_ftop, s_res, s_pm, s_slot);
  __syncthreads();
  if (threadIdx.x == 0) *bad_flag = 0;
  permute_body(topk_idx, T, k, bad, o, s_free, &s_ftop, s_res, s_pm, s_slot);
}

// Large blocks: the routes of chunk c (tokens [512 c, 512 c + 512)) are
// counted per expert by the counting launch below (k_perm_count_batch over a
// single block), then one workgroup plans the layer from the per-chunk counts
// as permute_body does (totals, offsets, work lists, staging, records) and
// turns the counts into each chunk's first position per expert, then the
// ranking launch. Three launches in stream order, so no workgroup waits on
// another and no device-scope fence is needed between them (with the
// planning done by the last counting workgroup, the fences that ordered the
// counts cost more than the whole permutation).
__global__ __launch_bounds__(kPermThreads) void k_perm_plan(const int32_t* __restrict__ topk_idx,
                                                            int T, int k, int n_chunks,
                                                            int32_t* __restrict__ bad_flag,
                                                            int32_t* __restrict__ chunk_base,
                                                            PermuteOut o) {
  __shared__ int32_t s_free[kMaxExperts];
  __shared__ int32_t s_ftop;
  __shared__ uint32_t s_res[kMaxExperts / 32], s_pm[kMaxExperts / 32];
  __shared__ int32_t s_slot[kMaxExperts];
  const int bad = *bad_flag;
  if ((threadIdx.x >> 6) == 1) prefetch_state(o.cv, o.E, o.layer, s_free, &s_ftop, s_res, s_pm, s_slot);
  __syncthreads();
  if (threadIdx.x == 0) *bad_flag = 0;   // re-armed for the next top-k launch (stream order)
  permute_body(topk_idx, T, k, bad, o, s_free, &s_ftop, s_res, s_pm, s_slot, chunk_base, n_chunks);
}

// Large blocks, third launch: workgroup c ranks the routes of chunk c from
// its first positions per expert (chunk_base[c][e]). Thread i takes token
// i / 2 of the chunk and half (i % 2) of its routes (at most KH), loaded once
// into registers, so the lanes of a wavefront share one 32-token word; the
// per-expert token bitmasks sit in kMaskStride-word rows. Each route's rank
// among the chunk's routes to its expert also places it in a counting sort of
// the chunk by expert in LDS, so perm is written in contiguous runs per expert
// (positions s_run[e] + rank) by consecutive lanes instead of one scattered
// store per lane. perm (and inv_perm, except on the 16-byte path) is stored
// through buffer resources of T*k entries: positions outside are dropped.
template <int KH>
__device__ __forceinline__ void perm_rank_body(const int32_t* __restrict__ topk_idx, int T, int k,
                                               int E, const int32_t* __restrict__ chunk_base,
                                               int32_t* __restrict__ perm,
                                               int32_t* __restrict__ inv_perm, int ch) {
  static_assert(2 * KH <= kMaxTopK && 2 * KH >= 4, "routes per thread");
  __shared__ uint32_t s_mask[kMaskRows * kMaskStride];
  __shared__ int32_t s_pre[kMaskRows * kMaskStride];
  __shared__ int32_t s_run[kMaxExperts];
  __shared__ int32_t s_first[kMaxExperts];
  __shared__ int32_t s_sorted[kChunkTokens * kMaxTopK];
  const int tid = threadIdx.x, lt = tid >> 1;
  const int kh = (k + 1) >> 1, j0 = (tid & 1) * kh, nj = min(kh, k - j0);
  const int t0 = ch * kChunkTokens, t = t0 + lt;
  const bool tok = t < T;
  const int nr = (min(T, t0 + kChunkTokens) - t0) * k;
  const int rl = lt * k + j0;                  // chunk-local route of this thread's first slot
  const size_t r0 = static_cast<size_t>(t0) * k;
  // the common case, k = 8 on 16-byte aligned arrays: one 16-byte load and store per thread
  const bool vec = KH == 4 && k == 8 &&
                   ((reinterpret_cast<uintptr_t>(topk_idx) | reinterpret_cast<uintptr_t>(inv_perm)) &
                    15) == 0;
  int ev[KH];
  if (vec) {
    const int4 v = tok ? *reinterpret_cast<const int4*>(topk_idx + r0 + rl) : make_int4(-1, -1, -1, -1);
    ev[0] = v.x;
    ev[1] = v.y;
    ev[2] = v.z;
    ev[3] = v.w;
  } else {
#pragma unroll
    for (int u = 0; u < KH; ++u) ev[u] = tok && u < nj ? topk_idx[r0 + rl + u] : -1;
  }
  const int run = tid < E ? chunk_base[static_cast<size_t>(ch) * E + tid] : 0;
  const uint32_t bit = 1u << (lt & 31);
  const int wofs = lt >> 5;
  int a[KH];
#pragma unroll
  for (int u = 0; u < KH; ++u) a[u] = ev[u] >= 0 && ev[u] < E ? ev[u] * kMaskStride + wofs : kMaskSpare;

  for (int i = tid; i < E * kMaskStride; i += kPermThreads) s_mask[i] = 0u;
  if (tid < kMaskStride) s_mask[kMaskSpare + tid] = 0u;
  __syncthreads();
  // token t takes its slots in the order (u + t) mod KH: the tokens of a
  // 32-token word (one wavefront) often share their best experts, and an LDS
  // atomic serialises the lanes that hit one address
#pragma unroll
  for (int u = 0; u < KH; ++u) {
    const int q = (u + lt) & (KH - 1);
    int aq = a[0];
#pragma unroll
    for (int v = 1; v < KH; ++v) aq = q == v ? a[v] : aq;
    atomicOr(&s_mask[aq], bit);
  }
  if (tid < E) s_run[tid] = run;
  __syncthreads();
  // word w of expert e is lane w of a 16-lane row: the chunk-local prefix of
  // the expert's words, and its chunk total at the row's last lane
  for (int i = tid; i < ((E * kChunkWords + 63) & ~63); i += kPermThreads) {
    const int e = i / kChunkWords, w = i & (kChunkWords - 1);
    const int cnt = e < E ? __popc(s_mask[e * kMaskStride + w]) : 0;
    const int incl = row16_incl_scan(cnt);
    if (e < E) {
      s_pre[e * kMaskStride + w] = incl - cnt;
      if (w == kChunkWords - 1) s_first[e] = incl;
    }
  }
  __syncthreads();
  if (tid < 64) {   // the experts' first chunk-local positions: one wavefront, 4 experts a lane
    int c[4], sum = 0;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int e = 4 * tid + q;
      c[q] = e < E ? s_first[e] : 0;
      sum += c[q];
    }
    int first = wave_incl_scan(sum) - sum;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int e = 4 * tid + q;
      if (e < E) s_first[e] = first;
      first += c[q];
    }
  }
  __syncthreads();
  const int n_routes = T * k;
  int pv[KH];
  uint32_t mv[KH];
#pragma unroll
  for (int u = 0; u < KH; ++u) {
    pv[u] = s_pre[a[u]];
    mv[u] = s_mask[a[u]];
  }
  const __amdgpu_buffer_rsrc_t rinv =
      __builtin_amdgcn_make_buffer_rsrc(inv_perm, 0, n_routes * 4, kRouteBufferFlags);
#pragma unroll
  for (int u = 0; u < KH; ++u) {
    const bool ok = a[u] != kMaskSpare;
    const int e = ok ? ev[u] : 0;
    const int local = pv[u] + __popc(mv[u] & (bit - 1u));
    pv[u] = s_run[e] + local;
    if (ok) s_sorted[s_first[e] + local] = (e << kRouteBits) | (rl + u);
    if (!vec && ok)
      __builtin_amdgcn_raw_buffer_store_b32(pv[u], rinv, static_cast<int>(r0 + rl + u) * 4, 0, 0);
  }
  if (vec && tok)
    *reinterpret_cast<int4*>(inv_perm + r0 + rl) = make_int4(pv[0], pv[1], pv[2], pv[3]);
  __syncthreads();
  const __amdgpu_buffer_rsrc_t rperm =
      __builtin_amdgcn_make_buffer_rsrc(perm, 0, n_routes * 4, kRouteBufferFlags);
  for (int p = tid; p < nr; p += kPermThreads) {
    const int v = s_sorted[p];
    const int e = (v >> kRouteBits) & (kMaxExperts - 1);
    __builtin_amdgcn_raw_buffer_store_b32(static_cast<int>(r0) + (v & ((1 << kRouteBits) - 1)),
                                          rperm, (s_run[e] + p - s_first[e]) * 4, 0, 0);
  }
}

template <int KH>
__global__ __launch_bounds__(kPermThreads) void k_perm_rank(const int32_t* __restrict__ topk_idx,
                                                            int T, int k, int E,
                                                            const int32_t* __restrict__ chunk_base,
                                                            int32_t* __restrict__ perm,
                                                            int32_t* __restrict__ inv_perm) {
  perm_rank_body<KH>(topk_idx, T, k, E, chunk_base, perm, inv_perm, blockIdx.x);
}

// Many independent blocks of T tokens (no cache), in three launches with no
// workgroup waiting on another. First: workgroup (c, b) counts chunk c of
// block b per expert into chunk_base[b][c][*].
__global__ __launch_bounds__(256) void k_perm_count_batch(const int32_t* __restrict__ topk_idx,
                                                         int T, int k, int E,
                                                         int32_t* __restrict__ chunk_base) {
  __shared__ int32_t s_h[kMaxExperts];
  const int b = blockIdx.y, ch = blockIdx.x, tid = threadIdx.x;
  const int32_t* idx = topk_idx + static_cast<size_t>(b) * T * k;
  for (int e = tid; e < kMaxExperts; e += 256) s_h[e] = 0;
  __syncthreads();
  const int t0 = ch * kChunkTokens, t1 = min(T, t0 + kChunkTokens);
  for (int r = t0 * k + tid; r < t1 * k; r += 4 * 256) {   // 4 loads in flight per thread
    int e[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) e[u] = r + u * 256 < t1 * k ? idx[r + u * 256] : -1;
#pragma unroll
    for (int u = 0; u < 4; ++u)
      if (e[u] >= 0) atomicAdd(&s_h[e[u]], 1);
  }
  __syncthreads();
  int32_t* out = chunk_base + (static_cast<size_t>(b) * gridDim.x + ch) * E;
  for (int e = tid; e < E; e += 256) out[e] = s_h[e];
}

// Second: one workgroup per block turns its per-chunk counts into the
// block's counts, offsets and per-chunk first positions. Per block b: counts
// at b*E, offsets at b*(E+1), non-finite flag at b. G threads per expert each
// keep a contiguous run of at most kPlanPer chunk counts in registers: their
// partial sums give the expert totals and the offsets (a DPP scan over the
// experts, 4 per lane), then each run's first positions are written from the
// registers. (The planning of permute_body without its cache, work-list and
// record steps.)
__global__ __launch_bounds__(kPermThreads) void k_perm_plan_batch(
    const int32_t* __restrict__ bad_flag, int n_chunks, int32_t* __restrict__ chunk_base,
    PermuteOut o) {
  __shared__ int32_t s_part[kPermThreads];
  __shared__ int32_t s_cnt[kMaxExperts];
  __shared__ int32_t s_off[kMaxExperts];
  const int b = blockIdx.x, E = o.E, tid = threadIdx.x;
  int32_t* cb = chunk_base + static_cast<size_t>(b) * n_chunks * E;
  const int G = max(1, min(kPermThreads / E, n_chunks));
  const int per = (n_chunks + G - 1) / G;
  const int my_g = tid < G * E ? tid / E : -1;
  const int my_e = my_g >= 0 ? tid - my_g * E : 0;
  const int ch_lo = my_g >= 0 ? my_g * per : 0;
  const int ch_hi = my_g >= 0 ? min(n_chunks, ch_lo + per) : 0;
  int cc[kPlanPer];
  int sum = 0;
#pragma unroll
  for (int q = 0; q < kPlanPer; ++q) {
    cc[q] = ch_lo + q < ch_hi ? cb[static_cast<size_t>(ch_lo + q) * E + my_e] : 0;
    sum += cc[q];
  }
  if (my_g >= 0) s_part[tid] = sum;
  __syncthreads();
  for (int e = tid; e < E; e += kPermThreads) {
    int c = 0;
    for (int g = 0; g < G; ++g) c += s_part[g * E + e];
    s_cnt[e] = c;
  }
  __syncthreads();
  if (tid < 64) {
    int c[4], tot = 0;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int e = 4 * tid + q;
      c[q] = e < E ? s_cnt[e] : 0;
      tot += c[q];
    }
    const int incl = wave_incl_scan(tot);
    int run = incl - tot;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int e = 4 * tid + q;
      if (e < E) {
        s_off[e] = run;
        o.counts[static_cast<size_t>(b) * E + e] = c[q];
        o.offsets[static_cast<size_t>(b) * (E + 1) + e] = run;
      }
      run += c[q];
    }
    if (tid == 63) o.offsets[static_cast<size_t>(b) * (E + 1) + E] = incl;
    if (tid == 0 && o.bad_out) o.bad_out[b] = bad_flag[b] ? 1 : 0;
  }
  __syncthreads();
  if (my_g >= 0) {
    int run = s_off[my_e];
    for (int h = 0; h < my_g; ++h) run += s_part[h * E + my_e];
#pragma unroll
    for (int q = 0; q < kPlanPer; ++q)
      if (ch_lo + q < ch_hi) {
        cb[static_cast<size_t>(ch_lo + q) * E + my_e] = run;
        run += cc[q];
      }
  }
}

// Third: workgroup (c, b) ranks chunk c of block b from its first positions.
template <int KH>
__global__ __launch_bounds__(kPermThreads) void k_perm_rank_batch(
    const int32_t* __restrict__ topk_idx, int T, int k, int E,
    const int32_t* __restrict__ chunk_base, int32_t* __restrict__ perm,
    int32_t* __restrict__ inv_perm) {
  const int b = blockIdx.y;
  const size_t R = static_cast<size_t>(T) * k;
  perm_rank_body<KH>(topk_idx + b * R, T, k, E,
                     chunk_base + static_cast<size_t>(b) * gridDim.x * E, perm + b * R,
                     inv_perm + b * R, blockIdx.x);
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
  __shared__ int32_t s_idx[kFusedMaxRoutes];
  __shared__ int32_t s_free[kMaxExperts];
  __shared__ int32_t s_ftop;
  __shared__ int32_t s_last;
  __shared__ uint32_t s_res[kMaxExperts / 32], s_pm[kMaxExperts / 32];
  __shared__ int32_t s_slot[kMaxExperts];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int E = o.E;
  // the cache state the last workgroup plans with, read while the tokens are
  // routed (no kernel of this launch changes it before the planning step)
  if (wave == 3) prefetch_state(o.cv, E, o.layer, s_free, &s_ftop, s_res, s_pm, s_slot);
  int bad = 0;
  for (int t = blockIdx.x * 4 + wave; t < T; t += gridDim.x * 4) {
    float g;
    const int e = route_token<EPL>(logits + static_cast<size_t>(t) * E, E, k, &g, &bad);
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
  for (int r = threadIdx.x; r < T * k; r += 256) s_idx[r] = __hip_atomic_load(
      &topk_idx[r], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  const int any_bad = __hip_atomic_load(&sync[1], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  __syncthreads();
  if (threadIdx.x == 0) {  // re-arm for the next launch (stream order)
    sync[0] = 0;
    sync[1] = 0;
  }
  permute_body(s_idx, T, k, any_bad, o, s_free, &s_ftop, s_res, s_pm, s_slot);
}

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float floatx4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

// Bijection on [0, total): workgroup b (XCD b % 8) -> contiguous tile range
// per XCD, so the tiles of one token range share an L2.
__device__ __forceinline__ int xcd_tile(int b, int total) {
  const int x = b & 7, local = b >> 3;
  const int q = total >> 3, r = total & 7;
  return x * q + (x < r ? x : r) + local;
}

// The gate: logits[t][e] = sum_h x[t][h] * wg[e][h] in fp32. A workgroup
// owns a tile of 16*TA tokens x 16*NB experts; its KS wavefronts split the
// hidden dimension into KS contiguous ranges, each accumulating every 16 x 16
// fragment of the tile over its range (A = token rows, B = gate rows, both
// read straight from memory; the next step's operands in flight while the
// current one multiplies, or the loads of G steps issued together). The partial tiles meet in LDS and are summed in
// wavefront order, so the result does not depend on timing. A step covers 64
// hidden elements in bf16 (lane group g holds elements 16g..16g+15, 32
// contiguous bytes of its row: two MFMAs of 8) or 32 in fp32 (elements
// 8g..8g+7: eight 16x16x4 MFMAs); the hidden size is a multiple of 128, so
// the steps tile it exactly. D lane (c, g) register
// i -> token 4g + i, expert c. Tokens and experts past the end read the last
// row; their results are not stored. Tiles are numbered token-major and laid
// out over the XCDs in contiguous ranges.
template <bool BF16, int TA, int NB, int KS, int G>
__global__ __launch_bounds__(64 * KS) void k_router_logits(const void* __restrict__ x,
                                                          const void* __restrict__ wg, int T,
                                                          int E, int H,
                                                          float* __restrict__ logits) {
  constexpr int NF = TA * NB;
  constexpr int kStep = BF16 ? 64 : 32;          // hidden elements per step
  constexpr int kEsz = BF16 ? 2 : 4;
  __shared__ floatx4_t s_part[KS][NF][64];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int c = lane & 15, g = lane >> 4;
  const int tiles_e = (E + 16 * NB - 1) / (16 * NB);
  const int tile = xcd_tile(blockIdx.x, gridDim.x);
  const int tt = tile / tiles_e, te = tile - tt * tiles_e;
  const int t0 = tt * 16 * TA, e0 = te * 16 * NB;
  const int n_steps = H / kStep;
  const int s0 = wave * n_steps / KS, s1 = (wave + 1) * n_steps / KS;
  const char* pa[TA];
  const char* pb[NB];
#pragma unroll
  for (int a = 0; a < TA; ++a)
    pa[a] = static_cast<const char*>(x) +
            (static_cast<size_t>(min(t0 + 16 * a + c, T - 1)) * H) * kEsz + 32 * g;
#pragma unroll
  for (int b = 0; b < NB; ++b)
    pb[b] = static_cast<const char*>(wg) +
            (static_cast<size_t>(min(e0 + 16 * b + c, E - 1)) * H) * kEsz + 32 * g;
  floatx4_t acc[TA][NB];
#pragma unroll
  for (int a = 0; a < TA; ++a)
#pragma unroll
    for (int b = 0; b < NB; ++b) acc[a][b] = floatx4_t{0.f, 0.f, 0.f, 0.f};

  auto mma = [&](const u32x4_t (&va)[TA][2], const u32x4_t (&vb)[NB][2]) {
#pragma unroll
    for (int a = 0; a < TA; ++a)
#pragma unroll
      for (int b = 0; b < NB; ++b) {
        if constexpr (BF16) {
#pragma unroll
          for (int v = 0; v < 2; ++v)
            acc[a][b] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                __builtin_bit_cast(bf16x8_t, va[a][v]), __builtin_bit_cast(bf16x8_t, vb[b][v]),
                acc[a][b], 0, 0, 0);
        } else {
#pragma unroll
          for (int v = 0; v < 2; ++v) {
            const floatx4_t fa = __builtin_bit_cast(floatx4_t, va[a][v]);
            const floatx4_t fb = __builtin_bit_cast(floatx4_t, vb[b][v]);
#pragma unroll
            for (int q = 0; q < 4; ++q)
              acc[a][b] = __builtin_amdgcn_mfma_f32_16x16x4f32(fa[q], fb[q], acc[a][b], 0, 0, 0);
          }
        }
      }
  };
  const int n = s1 - s0;
  auto offset = [&](int j) { return static_cast<size_t>(s0 + j) * kStep * kEsz; };
  auto load_a = [&](int j, u32x4_t (&va)[TA][2]) {
    const size_t off = offset(j);
#pragma unroll
    for (int a = 0; a < TA; ++a) {
      va[a][0] = *reinterpret_cast<const u32x4_t*>(pa[a] + off);
      va[a][1] = *reinterpret_cast<const u32x4_t*>(pa[a] + off + 16);
    }
  };
  auto load_b = [&](int j, u32x4_t (&vb)[NB][2]) {
    const size_t off = offset(j);
#pragma unroll
    for (int b = 0; b < NB; ++b) {
      vb[b][0] = *reinterpret_cast<const u32x4_t*>(pb[b] + off);
      vb[b][1] = *reinterpret_cast<const u32x4_t*>(pb[b] + off + 16);
    }
  };
  auto load = [&](int j, u32x4_t (&va)[TA][2], u32x4_t (&vb)[NB][2]) {
    load_a(j, va);
    load_b(j, vb);
  };

  if constexpr (G > 1) {
    // short ranges: the loads of G steps at once, then their products
    for (int j0 = 0; j0 < n; j0 += G) {
      u32x4_t va[G][TA][2], vb[G][NB][2];
#pragma unroll
      for (int j = 0; j < G; ++j)
        if (j0 + j < n) load(j0 + j, va[j], vb[j]);
#pragma unroll
      for (int j = 0; j < G; ++j)
        if (j0 + j < n) mma(va[j], vb[j]);
    }
  } else {
    u32x4_t ca[TA][2], cb[NB][2], na[TA][2], nb[NB][2];
    if (n > 0) load(0, ca, cb);
    int j = 0;
    for (; j + 1 < n; j += 2) {
      load(j + 1, na, nb);
      mma(ca, cb);
      if (j + 2 < n) load(j + 2, ca, cb);
      mma(na, nb);
    }
    if (j < n) mma(ca, cb);
  }
#pragma unroll
  for (int a = 0; a < TA; ++a)
#pragma unroll
    for (int b = 0; b < NB; ++b) s_part[wave][a * NB + b][lane] = acc[a][b];
  __syncthreads();
  for (int f = wave; f < NF; f += KS) {   // fragment f is summed by wavefront f mod KS
    floatx4_t sum = s_part[0][f][lane];
#pragma unroll
    for (int w = 1; w < KS; ++w) sum += s_part[w][f][lane];
    const int a = f / NB, b = f - a * NB;
    const int ec = e0 + 16 * b + c;
    if (ec < E) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int tr = t0 + 16 * a + 4 * g + i;
        if (tr < T) logits[static_cast<size_t>(tr) * E + ec] = sum[i];
      }
    }
  }
}

// The wide tiles (64 tokens x 16*NB experts, 4 wavefronts splitting the
// hidden dimension) with the gate rows staged through LDS: each step a
// wavefront loads its 16*NB rows' next 128 bytes as whole lines (8 rows of
// 128 bytes per instruction; chunk q of row r kept at q ^ (r mod 8), so the
// fragment reads of 8 consecutive rows hit distinct banks), then reads its B
// fragments from LDS. Token rows come straight from memory as in
// k_router_logits. Each wavefront stages only its own range (double-buffered;
// LDS operations of one wavefront complete in order), and the buffer is
// reused for the partial tiles once every wavefront is done.
template <bool BF16, int NB>
__global__ __launch_bounds__(256) void k_router_logits_staged(const void* __restrict__ x,
                                                             const void* __restrict__ wg,
                                                             int T, int E, int H,
                                                             float* __restrict__ logits) {
  constexpr int TA = 4, KS = 4, NF = TA * NB;
  constexpr int kStep = BF16 ? 64 : 32;          // hidden elements per 128-byte step
  constexpr int kEsz = BF16 ? 2 : 4;
  constexpr int kRows = 16 * NB;                 // gate rows of the tile
  constexpr int kStage = kRows * 8;              // 16-byte chunks per stage
  constexpr int kPart = KS * NF * 64;            // 16-byte slots of the partial tiles
  constexpr int kLds = kPart > KS * 2 * kStage ? kPart : KS * 2 * kStage;
  __shared__ u32x4_t s_lds[kLds];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int c = lane & 15, g = lane >> 4;
  const int tiles_e = (E + kRows - 1) / kRows;
  const int tile = xcd_tile(blockIdx.x, gridDim.x);
  const int tt = tile / tiles_e, te = tile - tt * tiles_e;
  const int t0 = tt * 16 * TA, e0 = te * kRows;
  const int n_steps = H / kStep;
  const int s0 = wave * n_steps / KS, s1 = (wave + 1) * n_steps / KS;
  const int n = s1 - s0;
  const char* pa[TA];
#pragma unroll
  for (int a = 0; a < TA; ++a)
    pa[a] = static_cast<const char*>(x) +
            (static_cast<size_t>(min(t0 + 16 * a + c, T - 1)) * H) * kEsz + 32 * g;
  // staging: instruction i loads rows 8i + lane / 8, chunk lane % 8
  const char* ps[2 * NB];
  int slot_w[2 * NB];
#pragma unroll
  for (int i = 0; i < 2 * NB; ++i) {
    const int r = 8 * i + (lane >> 3), q = lane & 7;
    ps[i] = static_cast<const char*>(wg) +
            (static_cast<size_t>(min(e0 + r, E - 1)) * H) * kEsz + 16 * q;
    slot_w[i] = r * 8 + (q ^ (r & 7));
  }
  int slot_r[NB][2];
#pragma unroll
  for (int b = 0; b < NB; ++b) {
    const int r = 16 * b + c;
    slot_r[b][0] = r * 8 + ((2 * g) ^ (r & 7));
    slot_r[b][1] = r * 8 + ((2 * g + 1) ^ (r & 7));
  }
  u32x4_t* stage = s_lds + wave * 2 * kStage;
  floatx4_t acc[TA][NB];
#pragma unroll
  for (int a = 0; a < TA; ++a)
#pragma unroll
    for (int b = 0; b < NB; ++b) acc[a][b] = floatx4_t{0.f, 0.f, 0.f, 0.f};

  auto off = [&](int j) { return static_cast<size_t>(s0 + j) * kStep * kEsz; };
  auto load_a = [&](int j, u32x4_t (&va)[TA][2]) {
#pragma unroll
    for (int a = 0; a < TA; ++a) {
      va[a][0] = *reinterpret_cast<const u32x4_t*>(pa[a] + off(j));
      va[a][1] = *reinterpret_cast<const u32x4_t*>(pa[a] + off(j) + 16);
    }
  };
  auto load_s = [&](int j, u32x4_t (&vs)[2 * NB]) {
#pragma unroll
    for (int i = 0; i < 2 * NB; ++i) vs[i] = *reinterpret_cast<const u32x4_t*>(ps[i] + off(j));
  };
  auto put_s = [&](int buf, const u32x4_t (&vs)[2 * NB]) {
#pragma unroll
    for (int i = 0; i < 2 * NB; ++i) stage[buf * kStage + slot_w[i]] = vs[i];
  };
  auto mma = [&](int buf, const u32x4_t (&va)[TA][2]) {
#pragma unroll
    for (int b = 0; b < NB; ++b) {
      const u32x4_t vb0 = stage[buf * kStage + slot_r[b][0]];
      const u32x4_t vb1 = stage[buf * kStage + slot_r[b][1]];
#pragma unroll
      for (int a = 0; a < TA; ++a) {
        if constexpr (BF16) {
          acc[a][b] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, va[a][0]),
                                                              __builtin_bit_cast(bf16x8_t, vb0),
                                                              acc[a][b], 0, 0, 0);
          acc[a][b] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, va[a][1]),
                                                              __builtin_bit_cast(bf16x8_t, vb1),
                                                              acc[a][b], 0, 0, 0);
        } else {
          const floatx4_t fa0 = __builtin_bit_cast(floatx4_t, va[a][0]);
          const floatx4_t fa1 = __builtin_bit_cast(floatx4_t, va[a][1]);
          const floatx4_t fb0 = __builtin_bit_cast(floatx4_t, vb0);
          const floatx4_t fb1 = __builtin_bit_cast(floatx4_t, vb1);
#pragma unroll
          for (int q = 0; q < 4; ++q)
            acc[a][b] = __builtin_amdgcn_mfma_f32_16x16x4f32(fa0[q], fb0[q], acc[a][b], 0, 0, 0);
#pragma unroll
          for (int q = 0; q < 4; ++q)
            acc[a][b] = __builtin_amdgcn_mfma_f32_16x16x4f32(fa1[q], fb1[q], acc[a][b], 0, 0, 0);
        }
      }
    }
  };

  if (n > 0) {
    u32x4_t ca[TA][2], na[TA][2], vs[2 * NB];
    load_s(0, vs);
    load_a(0, ca);
    put_s(0, vs);
    for (int j = 0; j < n; ++j) {
      const bool more = j + 1 < n;
      if (more) {
        load_s(j + 1, vs);
        load_a(j + 1, na);
      }
      mma(j & 1, ca);
      if (more) {
        put_s((j + 1) & 1, vs);
#pragma unroll
        for (int a = 0; a < TA; ++a) {
          ca[a][0] = na[a][0];
          ca[a][1] = na[a][1];
        }
      }
    }
  }
  __syncthreads();   // every wavefront is done with its stages: the LDS holds partials now
  floatx4_t (*s_part)[NF][64] = reinterpret_cast<floatx4_t (*)[NF][64]>(s_lds);
#pragma unroll
  for (int a = 0; a < TA; ++a)
#pragma unroll
    for (int b = 0; b < NB; ++b) s_part[wave][a * NB + b][lane] = acc[a][b];
  __syncthreads();
  for (int f = wave; f < NF; f += KS) {   // fragment f is summed by wavefront f mod KS
    floatx4_t sum = s_part[0][f][lane];
#pragma unroll
    for (int w = 1; w < KS; ++w) sum += s_part[w][f][lane];
    const int a = f / NB, b = f - a * NB;
    const int ec = e0 + 16 * b + c;
    if (ec < E) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int tr = t0 + 16 * a + 4 * g + i;
        if (tr < T) logits[static_cast<size_t>(tr) * E + ec] = sum[i];
      }
    }
  }
}

template <bool BF16, int NB>
void launch_logits_staged(const void* x, const void* wg, int T, int E, int H, float* logits,
                          hipEvent_t ev0, hipEvent_t ev1, hipStream_t s) {
  const int64_t blocks =
      static_cast<int64_t>((T + 63) / 64) * ((E + 16 * NB - 1) / (16 * NB));
  hipExtLaunchKernelGGL(k_router_logits_staged<BF16, NB>, dim3(static_cast<unsigned>(blocks)),
                        dim3(256), 0, s, ev0, ev1, 0, x, wg, T, E, H, logits);
}

template <bool BF16, int TA, int NB, int KS, int G>
void launch_logits_cfg(const void* x, const void* wg, int T, int E, int H, float* logits,
                       hipEvent_t ev0, hipEvent_t ev1, hipStream_t s) {
  const int64_t blocks =
      static_cast<int64_t>((T + 16 * TA - 1) / (16 * TA)) * ((E + 16 * NB - 1) / (16 * NB));
  hipExtLaunchKernelGGL(k_router_logits<BF16, TA, NB, KS, G>, dim3(static_cast<unsigned>(blocks)),
                        dim3(64 * KS), 0, s, ev0, ev1, 0, x, wg, T, E, H, logits);
}

// Tile shape of the gate GEMM: the largest tile that still gives every
// compute unit a workgroup (64 tokens x all of up to 128 experts reads x
// once, its gate rows staged through LDS; 32 x 64 and 16 x 32 for mid-sized
// blocks). The re-reads of the gate rows by every tile, not HBM, bound the
// larger blocks: with each wavefront load spread over 16 rows (64 bytes of
// each), the operands come in at about 8 TB/s for every tile shape measured
// (a coalesced read of L2-resident data runs at about 25 TB/s), so the tile
// that reads the fewest bytes wins. Small blocks take 16 x 16 tiles whose 4
// wavefronts issue the loads of 4 steps at once.
template <bool BF16>
void launch_logits(const void* x, const void* wg, int T, int E, int H, float* logits,
                   hipEvent_t ev0, hipEvent_t ev1, hipStream_t s) {
  auto wgs = [&](int ta, int nb) {
    return static_cast<int64_t>((T + 16 * ta - 1) / (16 * ta)) * ((E + 16 * nb - 1) / (16 * nb));
  };
  if (E <= 64 && wgs(4, 4) >= kGateFullGrid)
    launch_logits_staged<BF16, 4>(x, wg, T, E, H, logits, ev0, ev1, s);
  else if (E > 64 && wgs(4, 8) >= kGateFullGrid)
    launch_logits_staged<BF16, 8>(x, wg, T, E, H, logits, ev0, ev1, s);
  else if (wgs(2, 4) >= kGateFullGrid)
    launch_logits_cfg<BF16, 2, 4, 8, 1>(x, wg, T, E, H, logits, ev0, ev1, s);
  else if (wgs(1, 2) >= kGateFullGrid)
    launch_logits_cfg<BF16, 1, 2, 16, 2>(x, wg, T, E, H, logits, ev0, ev1, s);
  else
    launch_logits_cfg<BF16, 1, 1, 4, 4>(x, wg, T, E, H, logits, ev0, ev1, s);
}

}  // namespace

hipError_t launch_router_logits(bool bf16, const void* x, const void* wg, int T, int E, int H,
                                float* logits, hipEvent_t ev0, hipEvent_t ev1, hipStream_t s) {
  if (T <= 0 || E <= 0 || H <= 0 || H % 64) return hipErrorInvalidValue;
  if (static_cast<int64_t>((T + 15) / 16) * ((E + 15) / 16) > INT32_MAX) return hipErrorInvalidValue;
  if (bf16)
    launch_logits<true>(x, wg, T, E, H, logits, ev0, ev1, s);
  else
    launch_logits<false>(x, wg, T, E, H, logits, ev0, ev1, s);
  return hipGetLastError();
}

bool route_fused(int T, int k) { return T * k <= kFusedMaxRoutes; }

bool route_lanes(int T) { return T > kLaneTokensMin; }
bool permute_chunked(int T) { return T > kChunkedMinTokens; }
int permute_chunks(int T) { return (T + kChunkTokens - 1) / kChunkTokens; }

hipError_t launch_route_topk(const float* logits, int T, int E, int k, int32_t* topk_idx,
                             float* gates, int32_t* bad_flag, hipEvent_t ev0, hipEvent_t ev1,
                             hipStream_t s, int block_tokens) {
  const int Tb = block_tokens > 0 ? block_tokens : T;
  if (route_lanes(T)) {
    const int blocks = (T + 255) / 256;
    // DMA streaming: whole 32-expert chunks, byte offsets of every row the
    // wavefronts touch within a 32-bit buffer offset; one grid of two
    // workgroups per CU whose wavefronts take blocks of 64 tokens in turn.
    // Up to k = 8 (the streamed form's gathers for k = 16 hold 179 VGPRs and
    // take the compiler minutes; k = 16 stages through registers)
    const bool dma = k <= 8 && E % 32 == 0 && E <= 256 &&
                     static_cast<int64_t>((T + 63) / 64) * 64 * E * 4 <= INT32_MAX;
    const int grid = dma ? (blocks < kRouteStreamGrid ? blocks : kRouteStreamGrid) : blocks;
    auto go = [&](auto kp, auto km) {
      constexpr int KP = decltype(kp)::value, KM = decltype(km)::value;
      if constexpr (KM <= 8) {
        if (dma) {
          hipExtLaunchKernelGGL(k_route_lanes<KP, KM, true>, dim3(grid), dim3(256), 0, s, ev0,
                                ev1, 0, logits, T, E, k, topk_idx, gates, bad_flag, Tb);
          return;
        }
      }
      hipExtLaunchKernelGGL(k_route_lanes<KP, KM, false>, dim3(blocks), dim3(256), 0, s, ev0, ev1,
                            0, logits, T, E, k, topk_idx, gates, bad_flag, Tb);
    };
    using std::integral_constant;
    if (k <= 2) go(integral_constant<int, 3>{}, integral_constant<int, 2>{});
    else if (k <= 4) go(integral_constant<int, 5>{}, integral_constant<int, 4>{});
    else if (k <= 8) go(integral_constant<int, 9>{}, integral_constant<int, 8>{});
    else go(integral_constant<int, 17>{}, integral_constant<int, 16>{});
    return hipGetLastError();
  }
  const int blocks = (T + 3) / 4 < 4096 ? (T + 3) / 4 : 4096;
  if (E <= 64)
    hipExtLaunchKernelGGL(k_route_topk<1>, dim3(blocks), dim3(256), 0, s, ev0, ev1, 0, logits, T,
                          E, k, topk_idx, gates, bad_flag, Tb);
  else if (E <= 128)
    hipExtLaunchKernelGGL(k_route_topk<2>, dim3(blocks), dim3(256), 0, s, ev0, ev1, 0, logits, T,
                          E, k, topk_idx, gates, bad_flag, Tb);
  else
    hipExtLaunchKernelGGL(k_route_topk<4>, dim3(blocks), dim3(256), 0, s, ev0, ev1, 0, logits, T,
                          E, k, topk_idx, gates, bad_flag, Tb);
  return hipGetLastError();
}

hipError_t launch_permute(const int32_t* topk_idx, int T, int k, int32_t* bad_flag,
                          const PermuteOut& o, hipEvent_t ev0, hipEvent_t ev1, hipStream_t s) {
  hipExtLaunchKernelGGL(k_permute, dim3(1), dim3(kPermThreads), 0, s, ev0, ev1, 0, topk_idx, T, k,
                        bad_flag, o);
  return hipGetLastError();
}

hipError_t launch_permute_chunked(const int32_t* topk_idx, int T, int k, int32_t* bad_flag,
                                  int32_t* chunk_base, const PermuteOut& o, hipEvent_t ev0,
                                  hipEvent_t ev1, hipStream_t s) {
  const int n = permute_chunks(T);
  if (n > kMaxChunks) return hipErrorInvalidValue;   // the planning keeps kPlanPer counts a thread
  hipExtLaunchKernelGGL(k_perm_count_batch, dim3(n, 1), dim3(256), 0, s, ev0, nullptr, 0, topk_idx,
                        T, k, o.E, chunk_base);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_perm_plan, dim3(1), dim3(kPermThreads), 0, s, topk_idx, T, k, n, bad_flag,
                     chunk_base, o);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (k <= 8)
    hipExtLaunchKernelGGL(k_perm_rank<4>, dim3(n), dim3(kPermThreads), 0, s, nullptr, ev1, 0,
                          topk_idx, T, k, o.E, chunk_base, o.perm, o.inv_perm);
  else
    hipExtLaunchKernelGGL(k_perm_rank<8>, dim3(n), dim3(kPermThreads), 0, s, nullptr, ev1, 0,
                          topk_idx, T, k, o.E, chunk_base, o.perm, o.inv_perm);
  return hipGetLastError();
}

hipError_t launch_permute_batch(const int32_t* topk_idx, int B, int T, int k,
                                const int32_t* bad_flag, int32_t* chunk_base, const PermuteOut& o,
                                hipStream_t s) {
  const int n = permute_chunks(T);
  if (n > kMaxChunks) return hipErrorInvalidValue;   // the planning keeps kPlanPer counts a thread
  hipLaunchKernelGGL(k_perm_count_batch, dim3(n, B), dim3(256), 0, s, topk_idx, T, k, o.E,
                     chunk_base);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_perm_plan_batch, dim3(B), dim3(kPermThreads), 0, s, bad_flag, n,
                     chunk_base, o);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (k <= 8)
    hipLaunchKernelGGL(k_perm_rank_batch<4>, dim3(n, B), dim3(kPermThreads), 0, s, topk_idx, T, k,
                       o.E, chunk_base, o.perm, o.inv_perm);
  else
    hipLaunchKernelGGL(k_perm_rank_batch<8>, dim3(n, B), dim3(kPermThreads), 0, s, topk_idx, T, k,
                       o.E, chunk_base, o.perm, o.inv_perm);
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

// ---------------------------------------------------------------------------
// Routing and permutation without a context and without allocation: the
// scratch of the routing launches lives in one file-scope device array.
#include <mutex>

#include "oled.h"

namespace {

constexpr int kNoAllocMaxTokens = 65535;
constexpr int kNoAllocChunks = (kNoAllocMaxTokens + oled::kChunkTokens - 1) / oled::kChunkTokens;
// int32 layout: [0] non-finite flag of the top-k launch, [1] unused, [2..3]
// completion counter and flag of the fused launch, [64, 64 + kNoAllocChunks *
// kMaxExperts) per-chunk counts.
constexpr int kScratchHead = 64;
constexpr int kScratchInts = kScratchHead + kNoAllocChunks * oled::kMaxExperts;
constexpr int kMaxDevices = 64;

__device__ __align__(256) int32_t scratch[kScratchInts];

int32_t* g_scratch_dev[kMaxDevices];   // device address of `scratch` on each GPU
std::mutex g_scratch_mu;

__global__ __launch_bounds__(64) void k_clear_head(int32_t* head) {
  head[threadIdx.x] = 0;
}

// Address of this GPU's copy of the array (looked up once per device, with
// that device current).
hipError_t scratch_on(int dev, int32_t** out) {
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_dev[dev]) {
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    g_scratch_dev[dev] = static_cast<int32_t*>(p);
  }
  *out = g_scratch_dev[dev];
  return hipSuccess;
}

}  // namespace

extern "C" size_t oled_route_noalloc_scratch_bytes(void) {
  return sizeof(int32_t) * static_cast<size_t>(kScratchInts);
}

extern "C" oled_status oled_route_noalloc(const float* logits_dev, int32_t T, int32_t E,
                                          int32_t k, int32_t* topk_idx_dev, float* gates_dev,
                                          int32_t* counts_dev, int32_t* offsets_dev,
                                          int32_t* perm_dev, int32_t* inv_perm_dev,
                                          int32_t* nonfinite_dev, void* stream) {
  if (!logits_dev || !topk_idx_dev || !gates_dev || !counts_dev || !offsets_dev || !perm_dev ||
      !inv_perm_dev) {
    oled::set_noctx_error("oled_route_noalloc: NULL input or output");
    return OLED_ERR_INVALID_ARG;
  }
  if (T < 1 || E < 1 || k < 1 || k > E) {
    oled::set_noctx_error("oled_route_noalloc: T, E and k must be >= 1 and k <= E");
    return OLED_ERR_INVALID_ARG;
  }
  if (T > kNoAllocMaxTokens || E > oled::kMaxExperts || k > oled::kMaxTopK) {
    oled::set_noctx_error("oled_route_noalloc: T above 65535, E above 256 or k above 16 "
                          "exceeds the fixed scratch array");
    return OLED_ERR_UNSUPPORTED;
  }
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) {
    oled::set_noctx_error("oled_route_noalloc: no current device");
    return OLED_ERR_HIP;
  }
  int32_t* sc = nullptr;
  if (scratch_on(dev, &sc) != hipSuccess) {
    oled::set_noctx_error("oled_route_noalloc: hipGetSymbolAddress of the scratch array failed");
    return OLED_ERR_HIP;
  }
  hipStream_t s = static_cast<hipStream_t>(stream);

  oled::PermuteOut o{};
  o.counts = counts_dev;
  o.offsets = offsets_dev;
  o.perm = perm_dev;
  o.inv_perm = inv_perm_dev;
  o.gates = gates_dev;
  o.E = E;
  o.bad_out = nonfinite_dev;   // written by the planning workgroup (cv.hdr null: no cache)

  // the counters and flags start at zero (the launches also leave them zero)
  hipLaunchKernelGGL(k_clear_head, dim3(1), dim3(kScratchHead), 0, s, sc);
  if (hipGetLastError() != hipSuccess) {
    oled::set_noctx_error("oled_route_noalloc: launch failed");
    return OLED_ERR_HIP;
  }
  hipError_t e;
  if (oled::route_fused(T, k)) {
    e = oled::launch_route_fused(logits_dev, T, k, topk_idx_dev, gates_dev, sc + 2, o, nullptr,
                                 nullptr, s);
  } else {
    e = oled::launch_route_topk(logits_dev, T, E, k, topk_idx_dev, gates_dev, sc, nullptr,
                                nullptr, s);
    if (e == hipSuccess) {
      if (oled::permute_chunked(T))
        e = oled::launch_permute_chunked(topk_idx_dev, T, k, sc, sc + kScratchHead, o,
                                         nullptr, nullptr, s);
      else
        e = oled::launch_permute(topk_idx_dev, T, k, sc, o, nullptr, nullptr, s);
    }
  }
  if (e != hipSuccess) {
    oled::set_noctx_error("oled_route_noalloc: launch failed");
    return OLED_ERR_HIP;
  }
  return OLED_OK;
}

// ---------------------------------------------------------------------------
// Routing and permutation of many independent blocks in one pass (no cache):
// one top-k launch over every token of the batch, then the counting and
// ranking launches over (chunk, block).
namespace {

__global__ __launch_bounds__(256) void k_clear_ints(int32_t* p, int n) {
  const int i = blockIdx.x * 256 + static_cast<int>(threadIdx.x);
  if (i < n) p[i] = 0;
}

size_t batch_head_ints(int32_t B) { return ((2 * static_cast<size_t>(B) + 63) / 64) * 64; }

}  // namespace

extern "C" size_t oled_route_batch_workspace(int32_t B, int32_t T, int32_t E) {
  if (B < 1 || T < 1 || E < 1) return 0;
  return sizeof(int32_t) * (batch_head_ints(B) + static_cast<size_t>(B) *
                                                      oled::permute_chunks(T) * E);
}

extern "C" oled_status oled_route_batch(const float* logits_dev, int32_t B, int32_t T, int32_t E,
                                        int32_t k, int32_t* topk_idx_dev, float* gates_dev,
                                        int32_t* counts_dev, int32_t* offsets_dev,
                                        int32_t* perm_dev, int32_t* inv_perm_dev,
                                        int32_t* nonfinite_dev, void* workspace_dev,
                                        size_t workspace_bytes, void* stream) {
  if (!logits_dev || !topk_idx_dev || !gates_dev || !counts_dev || !offsets_dev || !perm_dev ||
      !inv_perm_dev || !workspace_dev) {
    oled::set_noctx_error("oled_route_batch: NULL input, output or workspace");
    return OLED_ERR_INVALID_ARG;
  }
  if (B < 1 || T < 1 || E < 1 || k < 1 || k > E) {
    oled::set_noctx_error("oled_route_batch: B, T, E and k must be >= 1 and k <= E");
    return OLED_ERR_INVALID_ARG;
  }
  if (T > kNoAllocMaxTokens || E > oled::kMaxExperts || k > oled::kMaxTopK ||
      static_cast<int64_t>(B) * T * k > INT32_MAX) {
    oled::set_noctx_error("oled_route_batch: T above 65535, E above 256, k above 16 or "
                          "B*T*k above 2^31-1");
    return OLED_ERR_UNSUPPORTED;
  }
  if (workspace_bytes < oled_route_batch_workspace(B, T, E)) {
    oled::set_noctx_error("oled_route_batch: workspace smaller than "
                          "oled_route_batch_workspace(B, T, E)");
    return OLED_ERR_INVALID_ARG;
  }
  hipStream_t s = static_cast<hipStream_t>(stream);
  int32_t* ws = static_cast<int32_t*>(workspace_dev);
  int32_t* bad = ws;                                  // [B] non-finite flags of the top-k launch
  int32_t* chunk_base = ws + batch_head_ints(B);      // [B][chunks][E]
  const int n_head = B;
  hipLaunchKernelGGL(k_clear_ints, dim3((n_head + 255) / 256), dim3(256), 0, s, ws, n_head);
  hipError_t e = hipGetLastError();
  if (e == hipSuccess)
    e = oled::launch_route_topk(logits_dev, B * T, E, k, topk_idx_dev, gates_dev, bad, nullptr,
                                nullptr, s, T);
  if (e == hipSuccess) {
    oled::PermuteOut o{};
    o.counts = counts_dev;
    o.offsets = offsets_dev;
    o.perm = perm_dev;
    o.inv_perm = inv_perm_dev;
    o.gates = gates_dev;
    o.E = E;
    o.bad_out = nonfinite_dev;
    e = oled::launch_permute_batch(topk_idx_dev, B, T, k, bad, chunk_base, o, s);
  }
  if (e != hipSuccess) {
    oled::set_noctx_error("oled_route_batch: launch failed");
    return OLED_ERR_HIP;
  }
  return OLED_OK;
}
