// Row pass over the post-attention states of a routed layer.
//
// For every token t (one workgroup per token row, HBM-streaming):
//   inv_rms = 1 / sqrt(mean(hbar^2) + eps_norm)            RMSNorm of the FFN input and of
//                                                           the router's hidden encoder
//                                                           (Sec. 3.1 eq:dense_attention, Sec. 3.2)
//   |delta_j|^2, <delta_j, delta_{j-1}>, |delta_{j-1}|^2    residual transitions
//     with delta_j = hbar_j - hbar_{j-1}                     (Sec. 3.2, eq:transition_features)
//   u = bf16/fp32(hbar * inv_rms * w)                        the FFN / adapter input
// The transition sums are only formed where the paper defines them (j >= 2, j >= 3).
#include "hero_device.h"
#include "hero_kernels.h"

namespace hero {

// Eight consecutive elements as loaded (bf16 stays packed: 4 registers per chunk).
template <typename T> struct Raw8;
template <> struct Raw8<bf16_t> {
  u32x4 v;
  __device__ __forceinline__ void load(const bf16_t* p) { v = *reinterpret_cast<const u32x4*>(p); }
  __device__ __forceinline__ float operator[](int i) const {
    const uint32_t w = v[i >> 1];
    return __uint_as_float((i & 1) ? (w & 0xffff0000u) : (w << 16));
  }
};
template <> struct Raw8<float> {
  f32x4 a, b;
  __device__ __forceinline__ void load(const float* p) {
    a = *reinterpret_cast<const f32x4*>(p);
    b = *reinterpret_cast<const f32x4*>(p + 4);
  }
  __device__ __forceinline__ float operator[](int i) const { return i < 4 ? a[i] : b[i - 4]; }
};

// One workgroup per token, its row split over the 4 waves (8 elements per lane per pass, up to
// four passes kept in registers for the normalisation), the four sums reduced across the waves
// through LDS.  Measured against four tokens per workgroup (one per wave): 26.8 against 28.4 us at
// 4096 tokens of d = 4096, 7.2 against 13.6 us at 256 tokens, where a wave per row left most CUs idle.
template <typename T>
__global__ __launch_bounds__(256) void rowstats_row_kernel(const T* __restrict__ hbar,
                                                           const T* __restrict__ prev1,
                                                           const T* __restrict__ prev2,
                                                           const T* __restrict__ norm_w, int d, int j,
                                                           float eps_norm, float* __restrict__ rowstat,
                                                           T* __restrict__ u) {
  __shared__ f32x4 part[4];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const size_t row = static_cast<size_t>(blockIdx.x) * d;
  constexpr int RC = 4;   // 8-element chunks per thread kept in registers (rows up to 8192)
  Raw8<T> h[RC];
  float ss = 0.f, dd = 0.f, dp = 0.f, pp = 0.f;
  const bool resident = d <= RC * 8 * 256;
  for (int c0 = 0; c0 < d; c0 += RC * 8 * 256) {
    Raw8<T> a[RC], b[RC];
#pragma unroll
    for (int c = 0; c < RC; ++c) {
      const int col = c0 + 8 * (tid + 256 * c);
      if (col < d) {
        h[c].load(hbar + row + col);
        if (j >= 2) a[c].load(prev1 + row + col);
        if (j >= 3) b[c].load(prev2 + row + col);
      }
    }
#pragma unroll
    for (int c = 0; c < RC; ++c) {
      const int col = c0 + 8 * (tid + 256 * c);
      if (col >= d) continue;
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const float hv = h[c][i];
        ss += hv * hv;
        if (j >= 2) {
          const float av = a[c][i];
          const float dj = hv - av;
          dd += dj * dj;
          if (j >= 3) {
            const float dq = av - b[c][i];
            dp += dj * dq;
            pp += dq * dq;
          }
        }
      }
    }
  }
  ss = wave_sum(ss);
  dd = wave_sum(dd);
  dp = wave_sum(dp);
  pp = wave_sum(pp);
  if (lane == 0) part[wave] = f32x4{ss, dd, dp, pp};
  __syncthreads();
  const f32x4 tot = part[0] + part[1] + part[2] + part[3];
  const float inv_rms = 1.0f / sqrtf(tot[0] / static_cast<float>(d) + eps_norm);
  if (tid == 0) {
    f32x4 r = {inv_rms, tot[1], tot[2], tot[3]};
    *reinterpret_cast<f32x4*>(rowstat + 4 * static_cast<size_t>(blockIdx.x)) = r;
  }
  for (int c0 = 0; c0 < d; c0 += RC * 8 * 256) {
#pragma unroll
    for (int c = 0; c < RC; ++c) {
      const int col = c0 + 8 * (tid + 256 * c);
      if (col >= d) continue;
      if (!resident) h[c].load(hbar + row + col);
      Raw8<T> w;
      w.load(norm_w + col);
      float o[8];
#pragma unroll
      for (int i = 0; i < 8; ++i) o[i] = h[c][i] * inv_rms * w[i];
      st8(u + row + col, o);
    }
  }
}

hipError_t launch_rowstats(int dtype, const void* hbar, const void* prev1, const void* prev2,
                           const void* norm_w, int T, int d, int j, float eps_norm,
                           float* rowstat, void* u, hipStream_t s) {
  if (T <= 0) return hipSuccess;
  if (dtype == 1)
    rowstats_row_kernel<bf16_t><<<T, 256, 0, s>>>(
        static_cast<const bf16_t*>(hbar), static_cast<const bf16_t*>(prev1), static_cast<const bf16_t*>(prev2),
        static_cast<const bf16_t*>(norm_w), d, j, eps_norm, rowstat, static_cast<bf16_t*>(u));
  else
    rowstats_row_kernel<float><<<T, 256, 0, s>>>(
        static_cast<const float*>(hbar), static_cast<const float*>(prev1), static_cast<const float*>(prev2),
        static_cast<const float*>(norm_w), d, j, eps_norm, rowstat, static_cast<float*>(u));
  return hipGetLastError();
}

}  // namespace hero
