#include "cpu_ffn.h"
#include <cmath>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <random>
#include <vector>
using namespace oled;

// Runs the host expert kernels over ragged shapes (fp32 and bf16 layers, jobs
// of 1..T token rows with repeats) so that a sanitizer build sees every
// access; prints one line per shape with the sum of |y|.
static uint16_t bf(float f) { uint32_t u; memcpy(&u, &f, 4); return (u + 0x7FFF + ((u >> 16) & 1)) >> 16; }
int main() {
  std::mt19937 g(1);
  std::normal_distribution<float> nd(0.f, 0.02f);
  ThreadPool pool(4);
  std::vector<float> scratch;
  int shapes[][4] = {{256, 256, 29, 3}, {128, 64, 7, 2}, {512, 128, 33, 5}, {64, 32, 1, 1}, {256, 512, 100, 4}};
  for (int bf16 = 0; bf16 < 2; ++bf16)
    for (auto& sh : shapes) {
      const int H = sh[0], I = sh[1], T = sh[2], nj = sh[3];
      const size_t es = bf16 ? 2 : 4;
      std::vector<std::vector<uint8_t>> blocks(nj, std::vector<uint8_t>(3ull * H * I * es));
      for (auto& b : blocks)
        for (size_t i = 0; i < 3ull * H * I; ++i) {
          float v = nd(g);
          if (bf16) { uint16_t h = bf(v); memcpy(&b[i * 2], &h, 2); } else memcpy(&b[i * 4], &v, 4);
        }
      std::vector<uint8_t> x(static_cast<size_t>(T) * H * es);
      for (int i = 0; i < T * H; ++i) {
        float v = nd(g) * 50;
        if (bf16) { uint16_t h = bf(v); memcpy(&x[i * 2], &h, 2); } else memcpy(&x[i * 4], &v, 4);
      }
      std::vector<std::vector<int32_t>> toks(nj);
      std::vector<std::vector<float>> outs(nj);
      std::vector<CpuExpertJob> jobs(nj);
      for (int j = 0; j < nj; ++j) {
        int n = 1 + (g() % T);
        for (int r = 0; r < n; ++r) toks[j].push_back(g() % T);
        outs[j].assign(static_cast<size_t>(n) * H, 0.f);
        jobs[j] = {blocks[j].data(), toks[j].data(), n, outs[j].data()};
      }
      cpu_ffn_run(pool, bf16, H, I, x.data(), jobs.data(), nj, scratch);
      double s = 0;
      for (auto& o : outs) for (float v : o) s += std::fabs(v);
      printf("bf16=%d H=%d I=%d T=%d jobs=%d sum|y|=%g\n", bf16, H, I, T, nj, s);
    }
  return 0;
}
