// Measurement hook: the chip's practical bf16 matrix-core rate.
//
// Every wave runs eight independent v_mfma_f32_32x32x16_bf16 accumulator chains on operands held
// in registers (no memory traffic inside the loop), two waves per SIMD on every compute unit.
// With zero operands the rate shows the issue limit; with random operands it shows the rate the
// power limit allows on data like the FFN products' (the clock drops with switching activity).
// The FFN GEMMs are judged against the 2.5 PFLOP/s dense bf16 figure; this loop says how much of
// that a kernel with perfect feeding could reach on this board.
#include "hero.h"
#include "hero_device.h"

namespace hero {
namespace {

constexpr int kPeakThreads = 512;   // 8 waves: two per SIMD
constexpr int kPeakChains = 8;      // independent accumulators per wave

__global__ __launch_bounds__(kPeakThreads) void peak_mfma_kernel(uint32_t seed, int iters, float* sink) {
  const int l = threadIdx.x;
  bf16x8 a[2], b[2];
#pragma unroll
  for (int q = 0; q < 2; ++q)
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      uint32_t h = static_cast<uint32_t>(l * 16 + q * 8 + e + blockIdx.x * 9973) * 2654435761u ^ seed;
      h ^= h >> 13;
      h *= 0x5bd1e995u;
      h ^= h >> 15;
      const float v = seed ? (static_cast<float>(h & 0xffffu) / 65536.0f - 0.5f) : 0.0f;
      a[q][e] = static_cast<__bf16>(v);
      b[q][e] = static_cast<__bf16>(0.5f * v);
    }
  f32x16 acc[kPeakChains];
#pragma unroll
  for (int i = 0; i < kPeakChains; ++i)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[i][r] = 0.0f;
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int i = 0; i < kPeakChains; ++i)
      acc[i] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[i & 1], b[(i >> 1) & 1], acc[i], 0, 0, 0);
  }
  float t = 0.0f;
#pragma unroll
  for (int i = 0; i < kPeakChains; ++i) t += acc[i][0] + acc[i][15];
  // never true for these operands; keeps the loop from being removed
  if (t == 1234.5f) sink[0] = t;
}

}  // namespace
}  // namespace hero

extern "C" int hero_peak_mfma(int random_operands, int iters, int workgroups, float* sink, void* hip_stream,
                              double* flop) {
  if (!sink || !flop) return HERO_E_NULL;
  if (iters < 1 || iters > (1 << 24) || workgroups < 1 || workgroups > 65536) return HERO_E_RANGE;
  const uint32_t seed = random_operands ? 12345u : 0u;
  hipLaunchKernelGGL(hero::peak_mfma_kernel, dim3(workgroups), dim3(hero::kPeakThreads), 0,
                     static_cast<hipStream_t>(hip_stream), seed, iters, sink);
  if (hipGetLastError() != hipSuccess) return HERO_E_LAUNCH;
  *flop = static_cast<double>(workgroups) * (hero::kPeakThreads / 64) * static_cast<double>(iters) *
          hero::kPeakChains * (2.0 * 32 * 32 * 16);
  return HERO_OK;
}
