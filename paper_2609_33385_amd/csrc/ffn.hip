// K4 grouped SwiGLU expert FFN over the experts of one layer (hits from their
// cache slots, transferred misses from their staging slots) and K5 the
// gate-weighted combine (OLED-MoE Sec. 4.1: cache-hit experts execute on the
// GPU; the output does not depend on where an expert's weights came from).
//
// Work decomposition: a work item is up to 64 routes (rows of the
// expert-sorted order) of one expert; grid = (feature tiles of 64, items).
// Each of the 4 wavefronts owns 16 output features and multiplies its 16
// weight rows, streamed straight from HBM into registers, with up to four
// 16-row token tiles staged per 128-wide K chunk in LDS. The weights are the
// A operand (M = features) and the tokens the B operand (N = tokens) of
// v_mfma_f32_16x16x32_bf16 (v_mfma_f32_16x16x4_f32 for fp32), so each weight
// byte is read once per item and reused across the token tiles in registers.
// Results per expert depend only on that expert's rows, never on the other
// experts of the launch, so hit and miss launches give identical bits.
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

// fp32: a 16-byte vector holds 4 consecutive k (16g + 4g' + q); MFMA q of the
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
constexpr int kKC = 128;  // K elements per chunk

template <class TR, bool UP>
__global__ __launch_bounds__(kThreads) void k_ffn(
    const char* __restrict__ pool, int64_t slot_bytes, SlotTable st,
    const WorkItem* __restrict__ items, int item_base, const typename TR::T* __restrict__ src,
    const int32_t* __restrict__ perm, int k, int H, int I, typename TR::T* __restrict__ hout,
    float* __restrict__ oout) {
  using T = typename TR::T;
  constexpr int EPV = TR::EPV;
  constexpr int SPAN = TR::SPAN;
  constexpr int NV = kKC / SPAN;          // vectors per lane per chunk
  constexpr int VPR = kKC / EPV;          // vectors per LDS row
  constexpr int NQ = 64 * VPR / kThreads; // B vectors loaded per thread per chunk
  constexpr int RS = kKC + EPV;           // LDS row stride (elements), +16 bytes
  __shared__ __attribute__((aligned(16))) T s_b[64 * RS];

  const WorkItem it = items[item_base + blockIdx.y];
  const int rows = it.rows;
  const T* W = reinterpret_cast<const T*>(pool + static_cast<int64_t>(st.slot[it.expert]) * slot_bytes);
  const int Kdim = UP ? H : I;
  const int lane = threadIdx.x & 63;
  const int lr = lane & 15, g = lane >> 4;
  const int fw = blockIdx.x * kFeatTile + (threadIdx.x >> 6) * 16;

  const T* a1;
  const T* a3;
  if (UP) {
    a1 = W + static_cast<size_t>(fw + lr) * H + EPV * g;
    a3 = W + static_cast<size_t>(I + fw + lr) * H + EPV * g;
  } else {
    a1 = W + static_cast<size_t>(2) * I * H + static_cast<size_t>(fw + lr) * I + EPV * g;
    a3 = a1;
  }

  const int bcol = threadIdx.x % VPR;
  const T* bsrc[NQ];
  int brow[NQ];
#pragma unroll
  for (int q = 0; q < NQ; ++q) {
    brow[q] = threadIdx.x / VPR + q * (kThreads / VPR);
    bsrc[q] = nullptr;
    if (brow[q] < rows) {
      const int pos = it.row_begin + brow[q];
      bsrc[q] = (UP ? src + static_cast<size_t>(perm[pos] / k) * H : src + static_cast<size_t>(pos) * I) +
                bcol * EPV;
    }
  }
  const int NT = (rows + 15) >> 4;

  floatx4_t acc1[4], acc3[4];
#pragma unroll
  for (int nt = 0; nt < 4; ++nt) {
    acc1[nt] = floatx4_t{0.f, 0.f, 0.f, 0.f};
    acc3[nt] = floatx4_t{0.f, 0.f, 0.f, 0.f};
  }

  for (int kc = 0; kc < Kdim; kc += kKC) {
    u32x4_t av1[NV], av3[NV];
#pragma unroll
    for (int v = 0; v < NV; ++v) {
      av1[v] = *reinterpret_cast<const u32x4_t*>(a1 + kc + SPAN * v);
      if (UP) av3[v] = *reinterpret_cast<const u32x4_t*>(a3 + kc + SPAN * v);
    }
    u32x4_t bv[NQ];
#pragma unroll
    for (int q = 0; q < NQ; ++q)
      bv[q] = bsrc[q] ? *reinterpret_cast<const u32x4_t*>(bsrc[q] + kc) : u32x4_t{0u, 0u, 0u, 0u};
    __syncthreads();
#pragma unroll
    for (int q = 0; q < NQ; ++q)
      *reinterpret_cast<u32x4_t*>(&s_b[brow[q] * RS + bcol * EPV]) = bv[q];
    __syncthreads();
#pragma unroll
    for (int v = 0; v < NV; ++v) {
#pragma unroll
      for (int nt = 0; nt < 4; ++nt) {
        if (nt < NT) {
          const u32x4_t b =
              *reinterpret_cast<const u32x4_t*>(&s_b[(16 * nt + lr) * RS + SPAN * v + EPV * g]);
          TR::mma(acc1[nt], av1[v], b);
          if (UP) TR::mma(acc3[nt], av3[v], b);
        }
      }
    }
  }

  // D layout: lane (lr, g), register r -> feature fw + 4g + r, token row 16 nt + lr.
#pragma unroll
  for (int nt = 0; nt < 4; ++nt) {
    const int row = 16 * nt + lr;
    if (nt < NT && row < rows) {
      const size_t pos = static_cast<size_t>(it.row_begin + row);
      if (UP) {
        float hv[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) hv[r] = TR::silu(acc1[nt][r]) * acc3[nt][r];
        if constexpr (sizeof(T) == 2) {
          uint2 packed;
          packed.x = f32_to_bf16_rne(hv[0]) | (static_cast<uint32_t>(f32_to_bf16_rne(hv[1])) << 16);
          packed.y = f32_to_bf16_rne(hv[2]) | (static_cast<uint32_t>(f32_to_bf16_rne(hv[3])) << 16);
          *reinterpret_cast<uint2*>(hout + pos * I + fw + 4 * g) = packed;
        } else {
          *reinterpret_cast<float4*>(hout + pos * I + fw + 4 * g) =
              make_float4(hv[0], hv[1], hv[2], hv[3]);
        }
      } else {
        *reinterpret_cast<float4*>(oout + pos * H + fw + 4 * g) =
            make_float4(acc1[nt][0], acc1[nt][1], acc1[nt][2], acc1[nt][3]);
      }
    }
  }
}

// One thread per 4 consecutive outputs of a token; sums its k routes in slot
// order in fp32 and rounds once.
template <bool BF16>
__global__ __launch_bounds__(256) void k_combine(const float* __restrict__ O,
                                                 const float* __restrict__ gates,
                                                 const int32_t* __restrict__ inv_perm, int k, int H,
                                                 void* __restrict__ y) {
  const int t = blockIdx.y;
  const int h = (blockIdx.x * 256 + threadIdx.x) * 4;
  if (h >= H) return;
  float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
  for (int j = 0; j < k; ++j) {
    const float gj = gates[static_cast<size_t>(t) * k + j];
    const int pos = inv_perm[static_cast<size_t>(t) * k + j];
    const float4 o = *reinterpret_cast<const float4*>(O + static_cast<size_t>(pos) * H + h);
    acc.x = fmaf(gj, o.x, acc.x);
    acc.y = fmaf(gj, o.y, acc.y);
    acc.z = fmaf(gj, o.z, acc.z);
    acc.w = fmaf(gj, o.w, acc.w);
  }
  if (BF16) {
    uint2 packed;
    packed.x = f32_to_bf16_rne(acc.x) | (static_cast<uint32_t>(f32_to_bf16_rne(acc.y)) << 16);
    packed.y = f32_to_bf16_rne(acc.z) | (static_cast<uint32_t>(f32_to_bf16_rne(acc.w)) << 16);
    *reinterpret_cast<uint2*>(static_cast<uint16_t*>(y) + static_cast<size_t>(t) * H + h) = packed;
  } else {
    *reinterpret_cast<float4*>(static_cast<float*>(y) + static_cast<size_t>(t) * H + h) = acc;
  }
}

}  // namespace

hipError_t launch_ffn_up(bool bf16, const void* pool, int64_t slot_bytes, const SlotTable& slots,
                         const WorkItem* items, int item_base, int n_items, const void* x,
                         const int32_t* perm, int k, int H, int I, void* h, hipStream_t s) {
  if (n_items <= 0) return hipSuccess;
  const dim3 grid(I / kFeatTile, n_items);
  const char* p = static_cast<const char*>(pool);
  if (bf16)
    hipLaunchKernelGGL((k_ffn<TrBF16, true>), grid, dim3(kThreads), 0, s, p, slot_bytes, slots,
                       items, item_base, static_cast<const uint16_t*>(x), perm, k, H, I,
                       static_cast<uint16_t*>(h), nullptr);
  else
    hipLaunchKernelGGL((k_ffn<TrF32, true>), grid, dim3(kThreads), 0, s, p, slot_bytes, slots,
                       items, item_base, static_cast<const float*>(x), perm, k, H, I,
                       static_cast<float*>(h), nullptr);
  return hipGetLastError();
}

hipError_t launch_ffn_down(bool bf16, const void* pool, int64_t slot_bytes, const SlotTable& slots,
                           const WorkItem* items, int item_base, int n_items, const void* h,
                           int H, int I, float* O, hipStream_t s) {
  if (n_items <= 0) return hipSuccess;
  const dim3 grid(H / kFeatTile, n_items);
  const char* p = static_cast<const char*>(pool);
  if (bf16)
    hipLaunchKernelGGL((k_ffn<TrBF16, false>), grid, dim3(kThreads), 0, s, p, slot_bytes, slots,
                       items, item_base, static_cast<const uint16_t*>(h), nullptr, 1, H, I,
                       nullptr, O);
  else
    hipLaunchKernelGGL((k_ffn<TrF32, false>), grid, dim3(kThreads), 0, s, p, slot_bytes, slots,
                       items, item_base, static_cast<const float*>(h), nullptr, 1, H, I, nullptr,
                       O);
  return hipGetLastError();
}

hipError_t launch_combine(bool bf16, const float* O, const float* gates, const int32_t* inv_perm,
                          int T, int k, int H, void* y, hipStream_t s) {
  const dim3 grid((H + 1023) / 1024, T);
  if (bf16)
    hipLaunchKernelGGL(k_combine<true>, grid, dim3(256), 0, s, O, gates, inv_perm, k, H, y);
  else
    hipLaunchKernelGGL(k_combine<false>, grid, dim3(256), 0, s, O, gates, inv_perm, k, H, y);
  return hipGetLastError();
}

}  // namespace oled
