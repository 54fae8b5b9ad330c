// Row pass over the post-attention states of a routed layer.
//
// For every token t (one wave per token row, HBM-streaming):
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

template <typename T>
__global__ __launch_bounds__(256) void rowstats_kernel(const T* __restrict__ hbar,
                                                       const T* __restrict__ prev1,
                                                       const T* __restrict__ prev2,
                                                       const T* __restrict__ norm_w, int ntok,
                                                       int d, int j, float eps_norm,
                                                       float* __restrict__ rowstat,
                                                       T* __restrict__ u) {
  const int lane = threadIdx.x & 63;
  const int t = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (t >= ntok) return;
  const size_t row = static_cast<size_t>(t) * d;
  float ss = 0.f, dd = 0.f, dp = 0.f, pp = 0.f;
  for (int c = lane * 8; c < d; c += 64 * 8) {
    float h[8];
    ld8(hbar + row + c, h);
#pragma unroll
    for (int i = 0; i < 8; ++i) ss += h[i] * h[i];
    if (j >= 2) {
      float a[8];
      ld8(prev1 + row + c, a);
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const float dj = h[i] - a[i];
        dd += dj * dj;
      }
      if (j >= 3) {
        float b[8];
        ld8(prev2 + row + c, b);
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          const float dj = h[i] - a[i];
          const float dq = a[i] - b[i];
          dp += dj * dq;
          pp += dq * dq;
        }
      }
    }
  }
  ss = wave_sum(ss);
  dd = wave_sum(dd);
  dp = wave_sum(dp);
  pp = wave_sum(pp);
  const float inv_rms = 1.0f / sqrtf(ss / static_cast<float>(d) + eps_norm);
  if (lane == 0) {
    f32x4 r = {inv_rms, dd, dp, pp};
    *reinterpret_cast<f32x4*>(rowstat + 4 * static_cast<size_t>(t)) = r;
  }
  for (int c = lane * 8; c < d; c += 64 * 8) {
    float h[8], w[8], o[8];
    ld8(hbar + row + c, h);
    ld8(norm_w + c, w);
#pragma unroll
    for (int i = 0; i < 8; ++i) o[i] = h[i] * inv_rms * w[i];
    st8(u + row + c, o);
  }
}

hipError_t launch_rowstats(int dtype, const void* hbar, const void* prev1, const void* prev2,
                           const void* norm_w, int T, int d, int j, float eps_norm,
                           float* rowstat, void* u, hipStream_t s) {
  dim3 grid((T + 3) / 4), block(256);
  if (dtype == 1) {
    rowstats_kernel<bf16_t><<<grid, block, 0, s>>>(
        static_cast<const bf16_t*>(hbar), static_cast<const bf16_t*>(prev1),
        static_cast<const bf16_t*>(prev2), static_cast<const bf16_t*>(norm_w), T, d, j, eps_norm,
        rowstat, static_cast<bf16_t*>(u));
  } else {
    rowstats_kernel<float><<<grid, block, 0, s>>>(
        static_cast<const float*>(hbar), static_cast<const float*>(prev1),
        static_cast<const float*>(prev2), static_cast<const float*>(norm_w), T, d, j, eps_norm,
        rowstat, static_cast<float*>(u));
  }
  return hipGetLastError();
}

}  // namespace hero
