// Host CPU execution of missed experts for the cooperative compensation
// (OLED-MoE Sec. 4.4: some cache misses run on the CPU instead of being
// transferred). Internal to the library.
#pragma once

#include <atomic>
#include <condition_variable>
#include <cstdint>
#include <functional>
#include <mutex>
#include <thread>
#include <vector>

namespace oled {

// Fixed set of worker threads; run(fn) calls fn(tid) once on every thread
// (the caller is tid 0) and returns when all calls have returned. Between
// jobs a worker polls for the next one for a short while before it sleeps,
// so back-to-back jobs (the phases of a layer) start without a wake-up.
class ThreadPool {
 public:
  explicit ThreadPool(int n_threads);
  ~ThreadPool();
  ThreadPool(const ThreadPool&) = delete;
  ThreadPool& operator=(const ThreadPool&) = delete;
  int size() const { return n_; }
  void run(const std::function<void(int)>& fn);

 private:
  void worker(int tid);
  int n_;
  std::vector<std::thread> workers_;
  std::mutex m_;
  std::condition_variable wake_;
  const std::function<void(int)>* fn_ = nullptr;
  std::atomic<uint64_t> gen_{0};
  std::atomic<int> pending_{0};
  bool stop_ = false;
};

// One expert's share of a layer run on the CPU: `n` token rows of x (row
// indices `tokens`) through the SwiGLU of the packed expert `block`; results
// (fp32, [n][H]) to `out`.
struct CpuExpertJob {
  const void* block;
  const int32_t* tokens;
  int n;
  float* out;
};

// True if this CPU has the vector instructions the kernels are built for.
bool cpu_ffn_supported();

// Runs the jobs on the pool: gate/up with the SiLU * up epilogue (the
// intermediate rounded to the layer dtype, as on the GPU), then the down
// projection, both split over 16-feature blocks of every job. x: [T][H] in
// the layer dtype (bf16 as raw 16-bit patterns). Scratch grows as needed.
void cpu_ffn_run(ThreadPool& pool, bool bf16, int H, int I, const void* x,
                 const CpuExpertJob* jobs, int n_jobs, std::vector<float>& scratch);

}  // namespace oled
