// Measurement hooks: the chip's practical ceilings.
//
// hero_peak_mfma: every wave runs eight independent bf16 MFMA accumulator chains
// (v_mfma_f32_32x32x16_bf16, or v_mfma_f32_16x16x32_bf16 as in the FFN products) on operands held
// in registers (no memory traffic inside the loop), two waves per SIMD on every compute unit.
// With zero operands the rate shows the issue limit; with random operands it shows the rate the
// power limit allows on data like the FFN products' (the clock drops with switching activity).
// The FFN GEMMs are judged against the 2.5 PFLOP/s dense bf16 figure; this loop says how much of
// that a kernel with perfect feeding could reach on this board.
//
// hero_peak_read: HBM read rates by access pattern.  Contiguous: plain non-temporal 16-byte loads
// into registers, eight in flight per lane, grid-stride.  Row visits: the pattern of a decode
// step's weight stream, a bf16 matrix of 8 KiB rows (d = 4096) read 96 rows per workgroup, one
// workgroup per CU, visit_bytes of every row per step (one 64-deep k-tile is 128 bytes) through
// LDS-DMA into a ring of stages, four loading waves.
#include <stdint.h>

#include <type_traits>

#include "hero.h"
#include "hero_device.h"

namespace hero {
namespace {

constexpr int kPeakThreads = 512;   // 8 waves: two per SIMD
constexpr int kCUsPeak = 256;       // compute units of an MI355X
constexpr int kPeakChains = 8;      // independent accumulators per wave

template <int MI>
__global__ __launch_bounds__(kPeakThreads) void peak_mfma_kernel(uint32_t seed, int iters, float* sink) {
  using Acc = typename std::conditional<MI == 32, f32x16, f32x4>::type;
  constexpr int NA = MI == 32 ? 16 : 4;
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
  Acc acc[kPeakChains];
#pragma unroll
  for (int i = 0; i < kPeakChains; ++i)
#pragma unroll
    for (int r = 0; r < NA; ++r) acc[i][r] = 0.0f;
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int i = 0; i < kPeakChains; ++i) {
      if constexpr (MI == 32)
        acc[i] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[i & 1], b[(i >> 1) & 1], acc[i], 0, 0, 0);
      else
        acc[i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[i & 1], b[(i >> 1) & 1], acc[i], 0, 0, 0);
    }
  }
  float t = 0.0f;
#pragma unroll
  for (int i = 0; i < kPeakChains; ++i) t += acc[i][0] + acc[i][NA - 1];
  // never true for these operands; keeps the loop from being removed
  if (t == 1234.5f) sink[0] = t;
}

// contiguous read: lane loads 16 bytes at a time, UNR in flight, grid-stride over n16 chunks
constexpr int kReadThreads = 256, kReadUnroll = 8;
__global__ __launch_bounds__(kReadThreads) void peak_read_kernel(const u32x4* __restrict__ p, size_t n16,
                                                                 float* sink) {
  u32x4 acc = {0u, 0u, 0u, 0u};
  const size_t stride = static_cast<size_t>(gridDim.x) * kReadThreads * kReadUnroll;
  for (size_t base = static_cast<size_t>(blockIdx.x) * kReadThreads * kReadUnroll + threadIdx.x; base < n16;
       base += stride) {
    u32x4 v[kReadUnroll];
#pragma unroll
    for (int u = 0; u < kReadUnroll; ++u) {
      const size_t i = base + static_cast<size_t>(u) * kReadThreads;
      v[u] = i < n16 ? __builtin_nontemporal_load(p + i) : u32x4{0u, 0u, 0u, 0u};
    }
#pragma unroll
    for (int u = 0; u < kReadUnroll; ++u) acc ^= v[u];
  }
  if ((acc[0] ^ acc[1] ^ acc[2] ^ acc[3]) == 0x9e3779b9u) sink[0] = 1.0f;   // keeps the loads
}

// row visits: workgroup w reads rows [96 w, 96 w + 96) of 8 KiB each, VB bytes of every row per
// step; a step's 96 VB bytes go as 96 VB / 1024 LDS-DMA loads of 1 KiB (1024 / VB rows each) spread
// over the four waves, into a ring of NS stages; one barrier per step
constexpr int kRowBytes = 8192, kRowsPerWg = 96, kRowWaves = 4;
typedef __attribute__((address_space(3))) void peak_lds_void;
template <int N>
__device__ __forceinline__ void peak_wait_vm() {
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}
template <int VB, int NS>
__global__ __launch_bounds__(64 * kRowWaves) void peak_rows_kernel(const unsigned char* __restrict__ p, float* sink) {
  constexpr int LPS = kRowsPerWg * VB / 1024, LW = LPS / kRowWaves, RPL = 1024 / VB;
  static_assert(LPS % kRowWaves == 0 && (NS - 1) * LW < 64, "load split");
  __shared__ __attribute__((aligned(1024))) unsigned char smem[NS * LPS * 1024];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  // load i of a step covers rows (wave + 4 i) RPL .. + RPL - 1; lane: row + lane / (VB / 16),
  // bytes 16 (lane % (VB / 16))
  const unsigned char* src0 = p + static_cast<size_t>(blockIdx.x) * kRowsPerWg * kRowBytes +
                              static_cast<size_t>(wave * RPL + lane / (VB / 16)) * kRowBytes + (lane % (VB / 16)) * 16;
  const size_t istride = static_cast<size_t>(kRowWaves) * RPL * kRowBytes;
  constexpr int nv = kRowBytes / VB;
  auto issue = [&](int v) {
#pragma unroll
    for (int i = 0; i < LW; ++i)
      __builtin_amdgcn_global_load_lds(src0 + i * istride + static_cast<size_t>(v) * VB,
                                       (peak_lds_void*)(smem + ((v % NS) * LPS + wave + kRowWaves * i) * 1024), 16, 0, 0);
  };
  for (int v = 0; v < NS && v < nv; ++v) issue(v);
  uint32_t acc = 0;
  for (int v = 0; v < nv; ++v) {
    if (v + NS <= nv) peak_wait_vm<(NS - 1) * LW>(); else peak_wait_vm<0>();
    __syncthreads();
    acc ^= *reinterpret_cast<const volatile uint32_t*>(smem + ((v % NS) * LPS) * 1024 + threadIdx.x * 4);
    __syncthreads();
    if (v + NS < nv) issue(v + NS);
  }
  if (acc == 0x9e3779b9u) sink[0] = 1.0f;
}

}  // namespace
}  // namespace hero

extern "C" int hero_peak_mfma(int mode, int iters, int workgroups, float* sink, void* hip_stream, double* flop) {
  if (!sink || !flop) return HERO_E_NULL;
  if (mode < 0 || mode > 3 || iters < 1 || iters > (1 << 24) || workgroups < 1 || workgroups > 65536)
    return HERO_E_RANGE;
  const uint32_t seed = (mode & 1) ? 12345u : 0u;
  const hipStream_t s = static_cast<hipStream_t>(hip_stream);
  if (mode & 2)
    hipLaunchKernelGGL(hero::peak_mfma_kernel<16>, dim3(workgroups), dim3(hero::kPeakThreads), 0, s, seed, iters, sink);
  else
    hipLaunchKernelGGL(hero::peak_mfma_kernel<32>, dim3(workgroups), dim3(hero::kPeakThreads), 0, s, seed, iters, sink);
  if (hipGetLastError() != hipSuccess) return HERO_E_LAUNCH;
  // both instructions do 2 * 16384 FLOP per lane-group issue: 32 x 32 x 16 or 16 x 16 x 32 multiply-adds
  *flop = static_cast<double>(workgroups) * (hero::kPeakThreads / 64) * static_cast<double>(iters) *
          hero::kPeakChains * (mode & 2 ? 2.0 * 16 * 16 * 32 : 2.0 * 32 * 32 * 16);
  return HERO_OK;
}

extern "C" int hero_peak_read(const void* src, size_t bytes, int visit_bytes, float* sink, void* hip_stream) {
  if (!src || !sink) return HERO_E_NULL;
  if ((reinterpret_cast<uintptr_t>(src) & 15u) != 0) return HERO_E_ALIGN;
  const hipStream_t s = static_cast<hipStream_t>(hip_stream);
  if (visit_bytes == 0) {
    if (bytes < 16 || bytes % 16 != 0) return HERO_E_DIM;
    hipLaunchKernelGGL(hero::peak_read_kernel, dim3(hero::kCUsPeak), dim3(hero::kReadThreads), 0, s,
                       static_cast<const hero::u32x4*>(src), bytes / 16, sink);
  } else {
    const size_t per = static_cast<size_t>(hero::kRowsPerWg) * hero::kRowBytes;
    if (bytes < per || bytes % per != 0 || bytes / per > 65536) return HERO_E_DIM;
    const dim3 grid(static_cast<unsigned>(bytes / per)), block(64 * hero::kRowWaves);
    const unsigned char* p = static_cast<const unsigned char*>(src);
    switch (visit_bytes) {
      case 128: hipLaunchKernelGGL((hero::peak_rows_kernel<128, 7>), grid, block, 0, s, p, sink); break;
      case 256: hipLaunchKernelGGL((hero::peak_rows_kernel<256, 4>), grid, block, 0, s, p, sink); break;
      case 512: hipLaunchKernelGGL((hero::peak_rows_kernel<512, 2>), grid, block, 0, s, p, sink); break;
      default: return HERO_E_RANGE;
    }
  }
  return hipGetLastError() == hipSuccess ? HERO_OK : HERO_E_LAUNCH;
}
