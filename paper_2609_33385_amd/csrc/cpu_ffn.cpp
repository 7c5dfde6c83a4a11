// Host CPU execution of missed experts (OLED-MoE Sec. 4.4): the SwiGLU
// expert FFN on a few token rows, read straight from the packed expert block
// in the pinned host pool, so a CPU-executed miss moves no weights over PCIe.
//
// The packed block holds fragments of 16 weight rows x SPAN columns (SPAN =
// 32 for bf16, 16 for fp32) with element l*V + i (V = SPAN/4) at row 16q +
// l%16, column SPAN*s + V*(l/16) + i. A 16-row feature block is therefore a
// run of fragments over s; every lane's V contiguous weights meet V
// contiguous inputs: each weight row accumulates, for a few tokens at a
// time, V-wide vector multiply-adds in registers over its pieces, summed
// across the vector at the end. fp32 accumulation; the intermediate
// silu(W1 x) * (W3 x) is rounded to the layer dtype as the GPU kernels store
// it.
#include "cpu_ffn.h"

#include <immintrin.h>

#include <atomic>
#include <cmath>
#include <cstdlib>
#include <cstring>

namespace oled {

ThreadPool::ThreadPool(int n_threads) : n_(n_threads < 1 ? 1 : n_threads) {
  for (int t = 1; t < n_; ++t) workers_.emplace_back(&ThreadPool::worker, this, t);
}

ThreadPool::~ThreadPool() {
  {
    std::lock_guard<std::mutex> lk(m_);
    stop_ = true;
    gen_.fetch_add(1, std::memory_order_release);
  }
  wake_.notify_all();
  for (auto& w : workers_) w.join();
}

void ThreadPool::worker(int tid) {
  uint64_t seen = 0;
  for (;;) {
    // poll for a new job, then sleep until one is posted
    for (int spin = 0; spin < (1 << 16) && gen_.load(std::memory_order_acquire) == seen; ++spin)
      _mm_pause();
    if (gen_.load(std::memory_order_acquire) == seen) {
      std::unique_lock<std::mutex> lk(m_);
      wake_.wait(lk, [&] { return stop_ || gen_.load(std::memory_order_acquire) != seen; });
    }
    {
      std::lock_guard<std::mutex> lk(m_);
      if (stop_) return;
    }
    seen = gen_.load(std::memory_order_acquire);
    (*fn_)(tid);
    pending_.fetch_sub(1, std::memory_order_acq_rel);
  }
}

void ThreadPool::run(const std::function<void(int)>& fn) {
  if (n_ == 1) {
    fn(0);
    return;
  }
  fn_ = &fn;
  pending_.store(n_ - 1, std::memory_order_relaxed);
  {
    std::lock_guard<std::mutex> lk(m_);
    gen_.fetch_add(1, std::memory_order_release);
  }
  wake_.notify_all();
  fn(0);
  while (pending_.load(std::memory_order_acquire) != 0) _mm_pause();
  fn_ = nullptr;
}

bool cpu_ffn_supported() {
  return __builtin_cpu_supports("avx2") && __builtin_cpu_supports("fma");
}

namespace {

inline float bf16_to_f32(uint16_t b) {
  const uint32_t u = static_cast<uint32_t>(b) << 16;
  float f;
  std::memcpy(&f, &u, 4);
  return f;
}

inline float round_bf16(float f) {
  uint32_t u;
  std::memcpy(&u, &f, 4);
  u = (u + 0x7FFFu + ((u >> 16) & 1u)) & 0xFFFF0000u;
  float r;
  std::memcpy(&r, &u, 4);
  return r;
}

// Dot products of one weight row r of a 16-row block with NT token rows:
// out1[t] (and out3[t] for the second matrix of a gate/up step) = sum over
// the fragments s of the row's SPAN columns times the token's. The row's
// V-element pieces sit at lanes r + 16 g, g < 4, of each fragment; every piece
// meets V contiguous inputs in one vector multiply-add per token.
__attribute__((target("avx2,fma"))) inline __m256 load_w8(const uint16_t* p) {
  const __m256i w = _mm256_cvtepu16_epi32(_mm_loadu_si128(reinterpret_cast<const __m128i*>(p)));
  return _mm256_castsi256_ps(_mm256_slli_epi32(w, 16));
}

__attribute__((target("avx2,fma"))) inline float hsum8(__m256 v) {
  const __m128 s = _mm_add_ps(_mm256_castps256_ps128(v), _mm256_extractf128_ps(v, 1));
  const __m128 t = _mm_add_ps(s, _mm_movehl_ps(s, s));
  return _mm_cvtss_f32(_mm_add_ss(t, _mm_shuffle_ps(t, t, 1)));
}

__attribute__((target("avx2,fma"))) inline float hsum4(__m128 s) {
  const __m128 t = _mm_add_ps(s, _mm_movehl_ps(s, s));
  return _mm_cvtss_f32(_mm_add_ss(t, _mm_shuffle_ps(t, t, 1)));
}

template <int NT, int NM>
__attribute__((target("avx2,fma"))) void row_bf16(const uint16_t* blk, size_t first, size_t step,
                                                  int steps, const float* xs, int K, int nt, int r,
                                                  float* out1, float* out3) {
  __m256 a1[NT], a3[NT];
  for (int t = 0; t < NT; ++t) a1[t] = a3[t] = _mm256_setzero_ps();
  for (int s = 0; s < steps; ++s) {
    const uint16_t* f = blk + first + static_cast<size_t>(s) * step;
    for (int g = 0; g < 4; ++g) {
      const int l = r + 16 * g;
      const __m256 w1 = load_w8(f + l * 8);
      const __m256 w3 = NM == 2 ? load_w8(f + 512 + l * 8) : _mm256_setzero_ps();
      const float* xc = xs + 32 * s + 8 * g;
#pragma GCC unroll 12
      for (int t = 0; t < NT; ++t) {
        if (t < nt) {
          const __m256 x8 = _mm256_loadu_ps(xc + static_cast<size_t>(t) * K);
          a1[t] = _mm256_fmadd_ps(w1, x8, a1[t]);
          if (NM == 2) a3[t] = _mm256_fmadd_ps(w3, x8, a3[t]);
        }
      }
    }
  }
  for (int t = 0; t < nt; ++t) {
    out1[t] = hsum8(a1[t]);
    if (NM == 2) out3[t] = hsum8(a3[t]);
  }
}

template <int NT, int NM>
__attribute__((target("avx2,fma"))) void row_f32(const float* blk, size_t first, size_t step,
                                                 int steps, const float* xs, int K, int nt, int r,
                                                 float* out1, float* out3) {
  __m128 a1[NT], a3[NT];
  for (int t = 0; t < NT; ++t) a1[t] = a3[t] = _mm_setzero_ps();
  for (int s = 0; s < steps; ++s) {
    const float* f = blk + first + static_cast<size_t>(s) * step;
    for (int g = 0; g < 4; ++g) {
      const int l = r + 16 * g;
      const __m128 w1 = _mm_loadu_ps(f + l * 4);
      const __m128 w3 = NM == 2 ? _mm_loadu_ps(f + 256 + l * 4) : _mm_setzero_ps();
      const float* xc = xs + 16 * s + 4 * g;
#pragma GCC unroll 12
      for (int t = 0; t < NT; ++t) {
        if (t < nt) {
          const __m128 x4 = _mm_loadu_ps(xc + static_cast<size_t>(t) * K);
          a1[t] = _mm_fmadd_ps(w1, x4, a1[t]);
          if (NM == 2) a3[t] = _mm_fmadd_ps(w3, x4, a3[t]);
        }
      }
    }
  }
  for (int t = 0; t < nt; ++t) {
    out1[t] = hsum4(a1[t]);
    if (NM == 2) out3[t] = hsum4(a3[t]);
  }
}

// All 16 rows of a block for n tokens, NT tokens at a time (accumulators in
// registers: 6 per matrix for gate/up, 12 for down).
template <bool BF16, int NM>
void block_rows(const void* blk, size_t first, size_t step, int steps, const float* xs, int K,
                int n, float* out1, float* out3) {
  constexpr int NT = NM == 2 ? 6 : 12;
  for (int t0 = 0; t0 < n; t0 += NT) {
    const int nt = n - t0 < NT ? n - t0 : NT;
    const float* x = xs + static_cast<size_t>(t0) * K;
    for (int r = 0; r < 16; ++r) {
      float* o1 = out1 + static_cast<size_t>(r) * n + t0;
      float* o3 = NM == 2 ? out3 + static_cast<size_t>(r) * n + t0 : nullptr;
      if (BF16)
        row_bf16<NT, NM>(static_cast<const uint16_t*>(blk), first, step, steps, x, K, nt, r, o1, o3);
      else
        row_f32<NT, NM>(static_cast<const float*>(blk), first, step, steps, x, K, nt, r, o1, o3);
    }
  }
}

// bf16 with AVX-512 BF16 (vdpbf16ps: pairs of bf16 products summed into fp32
// lanes). Within a fragment the 16-byte pieces of rows 4m..4m+3 for lane
// group g are 64 contiguous bytes, so one 512-bit load holds 4 rows x 8 k;
// the token's 8 matching inputs, broadcast to the four 128-bit lanes, meet
// them in one instruction, and fp32 lanes 4p..4p+3 collect row 4m + p. Each
// quad of rows streams a quarter of the block's cache lines whole; token
// inputs stay bf16 (the intermediate is rounded to bf16 anyway).
__attribute__((target("avx512f,avx512bw,avx512vl,avx512bf16"))) inline __m512i bcast16(
    const uint16_t* p) {
  return _mm512_broadcast_i32x4(_mm_loadu_si128(reinterpret_cast<const __m128i*>(p)));
}

template <int NT, int NM>
__attribute__((target("avx512f,avx512bw,avx512vl,avx512bf16"))) void quad_bf16(
    const uint16_t* blk, size_t first, size_t step, int steps, const uint16_t* xs, int K, int nt,
    int m, float* out1, float* out3, int ld) {
  __m512 a1[NT], a3[NT];
  for (int t = 0; t < NT; ++t) a1[t] = a3[t] = _mm512_setzero_ps();
  for (int s = 0; s < steps; ++s) {
    const uint16_t* f = blk + first + static_cast<size_t>(s) * step;
    for (int g = 0; g < 4; ++g) {
      const int l = 16 * g + 4 * m;
      const __m512i w1 = _mm512_loadu_si512(f + l * 8);
      const __m512i w3 = NM == 2 ? _mm512_loadu_si512(f + 512 + l * 8) : _mm512_setzero_si512();
      const uint16_t* xc = xs + 32 * s + 8 * g;
#pragma GCC unroll 16
      for (int t = 0; t < NT; ++t) {
        if (t < nt) {
          const __m512i xb = bcast16(xc + static_cast<size_t>(t) * K);
          a1[t] = _mm512_dpbf16_ps(a1[t], (__m512bh)w1, (__m512bh)xb);
          if (NM == 2) a3[t] = _mm512_dpbf16_ps(a3[t], (__m512bh)w3, (__m512bh)xb);
        }
      }
    }
  }
  alignas(64) float v[16];
  for (int t = 0; t < nt; ++t) {
    _mm512_store_ps(v, a1[t]);
    for (int p = 0; p < 4; ++p)
      out1[static_cast<size_t>(4 * m + p) * ld + t] = (v[4 * p] + v[4 * p + 1]) + (v[4 * p + 2] + v[4 * p + 3]);
    if (NM == 2) {
      _mm512_store_ps(v, a3[t]);
      for (int p = 0; p < 4; ++p)
        out3[static_cast<size_t>(4 * m + p) * ld + t] =
            (v[4 * p] + v[4 * p + 1]) + (v[4 * p + 2] + v[4 * p + 3]);
    }
  }
}

// All 16 rows of a block for n tokens (bf16 inputs xs [n][K]), NT tokens at a
// time: out [16][n].
template <int NM>
void block_quads(const uint16_t* blk, size_t first, size_t step, int steps, const uint16_t* xs,
                 int K, int n, float* out1, float* out3) {
  constexpr int NT = NM == 2 ? 12 : 16;
  for (int t0 = 0; t0 < n; t0 += NT) {
    const int nt = n - t0 < NT ? n - t0 : NT;
    const uint16_t* x = xs + static_cast<size_t>(t0) * K;
    for (int m = 0; m < 4; ++m)
      quad_bf16<NT, NM>(blk, first, step, steps, x, K, nt, m, out1 + t0,
                        NM == 2 ? out3 + t0 : nullptr, n);
  }
}

inline uint16_t bf16_bits_rne(float f) {
  uint32_t u;
  std::memcpy(&u, &f, 4);
  return static_cast<uint16_t>((u + 0x7FFFu + ((u >> 16) & 1u)) >> 16);
}

void run_bf16_avx512(ThreadPool& pool, int H, int I, const void* x, const CpuExpertJob* jobs,
                     int n_jobs, std::vector<float>& scratch) {
  constexpr int SPAN = 32;
  constexpr int FRAG = 16 * SPAN;
  // scratch (16-bit words): per job xs [n][H] and h [n][I]
  std::vector<size_t> xs_off(n_jobs), h_off(n_jobs);
  size_t total = 0;
  int max_n = 0;
  for (int j = 0; j < n_jobs; ++j) {
    xs_off[j] = total;
    total += static_cast<size_t>(jobs[j].n) * H;
    h_off[j] = total;
    total += static_cast<size_t>(jobs[j].n) * I;
    if (jobs[j].n > max_n) max_n = jobs[j].n;
  }
  if (scratch.size() * 2 < total) scratch.resize((total + 1) / 2);
  uint16_t* sc = reinterpret_cast<uint16_t*>(scratch.data());
  const int nth = pool.size();
  std::vector<std::vector<float>> part(nth);   // per thread: [16][n] of each matrix
  for (auto& a : part) a.resize(static_cast<size_t>(max_n) * 16 * 2);

  // phase 0: gather the token rows (bf16 as they are)
  for (int j = 0; j < n_jobs; ++j)
    for (int t = 0; t < jobs[j].n; ++t)
      std::memcpy(sc + xs_off[j] + static_cast<size_t>(t) * H,
                  static_cast<const uint16_t*>(x) + static_cast<size_t>(jobs[j].tokens[t]) * H,
                  sizeof(uint16_t) * H);

  // phase 1: gate/up blocks of 16 features, h = silu(W1 x) * (W3 x) in bf16
  const int nq = I / 16, S = H / SPAN;
  std::atomic<int> next{0};
  pool.run([&](int tid) {
    float* pa = part[tid].data();
    for (int i = next.fetch_add(1); i < n_jobs * nq; i = next.fetch_add(1)) {
      const int j = i / nq, q = i % nq;
      const CpuExpertJob& jb = jobs[j];
      float* pb = pa + static_cast<size_t>(jb.n) * 16;
      block_quads<2>(static_cast<const uint16_t*>(jb.block), static_cast<size_t>(q) * S * 2 * FRAG,
                     2 * FRAG, S, sc + xs_off[j], H, jb.n, pa, pb);
      for (int r = 0; r < 16; ++r)
        for (int t = 0; t < jb.n; ++t) {
          const float a = pa[static_cast<size_t>(r) * jb.n + t];
          const float b = pb[static_cast<size_t>(r) * jb.n + t];
          sc[h_off[j] + static_cast<size_t>(t) * I + 16 * q + r] =
              bf16_bits_rne(a / (1.f + std::exp(-a)) * b);
        }
    }
  });

  // phase 2: down blocks of 16 output features
  const int np = H / 16, S2 = I / SPAN;
  const size_t down0 = static_cast<size_t>(2) * I * H;
  next = 0;
  pool.run([&](int tid) {
    float* pa = part[tid].data();
    for (int i = next.fetch_add(1); i < n_jobs * np; i = next.fetch_add(1)) {
      const int j = i / np, p = i % np;
      const CpuExpertJob& jb = jobs[j];
      block_quads<1>(static_cast<const uint16_t*>(jb.block), down0 + static_cast<size_t>(p) * S2 * FRAG,
                     FRAG, S2, sc + h_off[j], I, jb.n, pa, nullptr);
      for (int r = 0; r < 16; ++r)
        for (int t = 0; t < jb.n; ++t)
          jb.out[static_cast<size_t>(t) * H + 16 * p + r] = pa[static_cast<size_t>(r) * jb.n + t];
    }
  });
}

bool has_avx512_bf16() {
  static const bool v = __builtin_cpu_supports("avx512f") && __builtin_cpu_supports("avx512bw") &&
                        __builtin_cpu_supports("avx512vl") && __builtin_cpu_supports("avx512bf16");
  return v;
}

// OLED_CPU_FFN_AVX2=1 keeps bf16 on the AVX2 kernels (read at every call)
bool force_avx2() {
  const char* e = std::getenv("OLED_CPU_FFN_AVX2");
  return e && e[0] == '1';
}

template <bool BF16>
void run_t(ThreadPool& pool, int H, int I, const void* x, const CpuExpertJob* jobs, int n_jobs,
           std::vector<float>& scratch) {
  constexpr int V = BF16 ? 8 : 4;
  constexpr int SPAN = 4 * V;
  constexpr int FRAG = 16 * SPAN;
  // scratch: per job xs [n][H] and h [n][I]
  std::vector<size_t> xs_off(n_jobs), h_off(n_jobs);
  size_t total = 0;
  int max_n = 0;
  for (int j = 0; j < n_jobs; ++j) {
    xs_off[j] = total;
    total += static_cast<size_t>(jobs[j].n) * H;
    h_off[j] = total;
    total += static_cast<size_t>(jobs[j].n) * I;
    if (jobs[j].n > max_n) max_n = jobs[j].n;
  }
  if (scratch.size() < total) scratch.resize(total);
  float* sc = scratch.data();
  const int nth = pool.size();
  std::vector<std::vector<float>> part(nth);   // per thread: [16][n] of each matrix
  for (auto& a : part) a.resize(static_cast<size_t>(max_n) * 16 * 2);

  // phase 0: token rows to fp32
  std::atomic<int> next{0};
  std::vector<int> row_job, row_idx;
  for (int j = 0; j < n_jobs; ++j)
    for (int t = 0; t < jobs[j].n; ++t) {
      row_job.push_back(j);
      row_idx.push_back(t);
    }
  const int rows_total = static_cast<int>(row_job.size());
  pool.run([&](int) {
    for (int i = next.fetch_add(1); i < rows_total; i = next.fetch_add(1)) {
      const CpuExpertJob& jb = jobs[row_job[i]];
      const int t = row_idx[i];
      float* dst = sc + xs_off[row_job[i]] + static_cast<size_t>(t) * H;
      const size_t src = static_cast<size_t>(jb.tokens[t]) * H;
      if (BF16) {
        const uint16_t* xr = static_cast<const uint16_t*>(x) + src;
        for (int h = 0; h < H; ++h) dst[h] = bf16_to_f32(xr[h]);
      } else {
        std::memcpy(dst, static_cast<const float*>(x) + src, sizeof(float) * H);
      }
    }
  });

  // phase 1: gate/up blocks of 16 features, h = silu(W1 x) * (W3 x)
  const int nq = I / 16, S = H / SPAN;
  next = 0;
  pool.run([&](int tid) {
    float* pa = part[tid].data();
    for (int i = next.fetch_add(1); i < n_jobs * nq; i = next.fetch_add(1)) {
      const int j = i / nq, q = i % nq;
      const CpuExpertJob& jb = jobs[j];
      float* pb = pa + static_cast<size_t>(jb.n) * 16;
      block_rows<BF16, 2>(jb.block, static_cast<size_t>(q) * S * 2 * FRAG, 2 * FRAG, S,
                          sc + xs_off[j], H, jb.n, pa, pb);
      for (int r = 0; r < 16; ++r)
        for (int t = 0; t < jb.n; ++t) {
          const float a = pa[static_cast<size_t>(r) * jb.n + t];
          const float b = pb[static_cast<size_t>(r) * jb.n + t];
          float hv = a / (1.f + std::exp(-a)) * b;
          if (BF16) hv = round_bf16(hv);
          sc[h_off[j] + static_cast<size_t>(t) * I + 16 * q + r] = hv;
        }
    }
  });

  // phase 2: down blocks of 16 output features
  const int np = H / 16, S2 = I / SPAN;
  const size_t down0 = static_cast<size_t>(2) * I * H;
  next = 0;
  pool.run([&](int tid) {
    float* pa = part[tid].data();
    for (int i = next.fetch_add(1); i < n_jobs * np; i = next.fetch_add(1)) {
      const int j = i / np, p = i % np;
      const CpuExpertJob& jb = jobs[j];
      block_rows<BF16, 1>(jb.block, down0 + static_cast<size_t>(p) * S2 * FRAG, FRAG, S2,
                          sc + h_off[j], I, jb.n, pa, nullptr);
      for (int r = 0; r < 16; ++r)
        for (int t = 0; t < jb.n; ++t)
          jb.out[static_cast<size_t>(t) * H + 16 * p + r] = pa[static_cast<size_t>(r) * jb.n + t];
    }
  });
}

}  // namespace

void cpu_ffn_run(ThreadPool& pool, bool bf16, int H, int I, const void* x,
                 const CpuExpertJob* jobs, int n_jobs, std::vector<float>& scratch) {
  if (n_jobs <= 0) return;
  if (bf16 && has_avx512_bf16() && !force_avx2())
    run_bf16_avx512(pool, H, I, x, jobs, n_jobs, scratch);
  else if (bf16)
    run_t<true>(pool, H, I, x, jobs, n_jobs, scratch);
  else
    run_t<false>(pool, H, I, x, jobs, n_jobs, scratch);
}

}  // namespace oled
