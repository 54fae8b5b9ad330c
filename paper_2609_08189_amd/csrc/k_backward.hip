// Training side of the routed block: the row and reduction passes of its backward, and the
// gate-utilisation penalty.
//
// The block is h = hbar + g FFN(u) on the FFN branch and h = hbar + (1 - g) Adapter(u) on the
// adapter branch, u = RMSNorm_w(hbar) (Sec. 3.1, eq:ffn_route).  The threshold that picks the
// branch is not differentiated; the gradient reaches the router through the scaling by g or
// 1 - g (the remark after eq:ffn_route), as dL/dlogit = dL/dg g (1 - g).  The backbone is
// frozen (Sec. 3.3): its FFN passes a gradient to hbar but takes none.  The adapter's weights
// take theirs here.  The products (FFN and adapter) run on the GEMM core; this file holds
//   * a tiled transpose (the frozen weights' K-contiguous copies, the adapter's per call);
//   * the adapter's middle step: a = SiLU(z), dz = (1 - g) e_a SiLU'(z), dL/dg = -<e_a, a>;
//   * the adapter weight gradients, summed over token chunks in a fixed order;
//   * the row pass: dL/dhbar = dL/dh + the RMSNorm backward of du, and dL/dg, dL/dlogit;
//   * alpha L_skip (Sec. 3.3, Eq. 18): the squared per-token sum of the gates over the routed
//     blocks, averaged over the positions with a next token, and its gradient.
// Every reduction runs in a fixed order, so results do not depend on scheduling.
#include <algorithm>

#include "hero_device.h"
#include "hero_kernels.h"

namespace hero {
namespace {

template <typename T>
__global__ __launch_bounds__(256) void transpose_kernel(const T* __restrict__ in, int R, int C, int ld_in,
                                                        T* __restrict__ out, int ld_out, int R_pad) {
  __shared__ T tile[64][65];
  const int c0 = blockIdx.x * 64, r0 = blockIdx.y * 64;
  const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;
  for (int i = ty; i < 64; i += 4) {
    const int r = r0 + i, c = c0 + tx;
    tile[i][tx] = (r < R && c < C) ? in[static_cast<size_t>(r) * ld_in + c] : T(0);
  }
  __syncthreads();
  for (int i = ty; i < 64; i += 4) {
    const int c = c0 + i, r = r0 + tx;   // output row c, column r
    if (c < C && r < R_pad) out[static_cast<size_t>(c) * ld_out + r] = tile[tx][i];
  }
}

// One wave per adapter row m < counts[1]; the K-slice partials of z and e_a are added in order.
template <typename T>
__global__ __launch_bounds__(256) void adapter_bwd_mid_kernel(BlockBwdArgs a) {
  const int lane = threadIdx.x & 63;
  const int m = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (m >= a.counts[1]) return;
  const int t = a.idx_ad[m];
  const float om = 1.0f - a.gate[t];
  const size_t slice = static_cast<size_t>(a.T) * a.d_r;
  const size_t row = static_cast<size_t>(m) * a.d_r;
  T* dzk = static_cast<T*>(a.dzk) + static_cast<size_t>(m) * a.rpad;
  float acc = 0.f;
  for (int r = lane; r < a.rpad; r += kWave) {
    if (r >= a.d_r) {
      stf(dzk + r, 0.0f);
      continue;
    }
    float z = 0.f, e = 0.f;
    for (int g = 0; g < a.splits; ++g) {
      z += a.part_z[g * slice + row + r];
      e += a.part_e[g * slice + row + r];
    }
    const float sg = 1.0f / (1.0f + expf(-z));
    const float act = z * sg;
    const float dz = om * e * sg * (1.0f + z * (1.0f - sg));
    acc += e * act;
    a.dz32[row + r] = dz;
    a.a32[row + r] = act;
    stf(dzk + r, dz);
  }
  acc = wave_sum(acc);
  if (lane == 0) a.dg_ad[m] = -acc;
}

// Weight-gradient partials of one chunk of adapter rows: thread = one column i of d, RB ranks.
//   pw1[c][r][i] = sum_m dz[m][r] u[t_m][i],  pw2[c][i][r] = sum_m a[m][r] (1 - g_t) dh[t_m][i]
constexpr int WG_RB = 32, WG_TB = 64;

template <typename T>
__global__ __launch_bounds__(256) void adapter_wgrad_kernel(BlockBwdArgs a) {
  __shared__ float sdz[WG_TB][WG_RB];
  __shared__ float sa[WG_TB][WG_RB];
  __shared__ int st[WG_TB];
  __shared__ float sg[WG_TB];
  const int n = a.counts[1];
  const int mb = blockIdx.z * a.chunk;
  if (mb >= n) return;
  const int me = min(n, mb + a.chunk);
  const int i = blockIdx.x * 256 + threadIdx.x;
  const int r0 = blockIdx.y * WG_RB;
  const bool col_ok = i < a.d;
  const T* U = static_cast<const T*>(a.u);
  const T* DH = static_cast<const T*>(a.dh);
  float g1[WG_RB], g2[WG_RB];
#pragma unroll
  for (int rr = 0; rr < WG_RB; ++rr) g1[rr] = g2[rr] = 0.f;
  for (int m0 = mb; m0 < me; m0 += WG_TB) {
    const int nb = min(WG_TB, me - m0);
    __syncthreads();
    for (int e = threadIdx.x; e < WG_TB * WG_RB; e += 256) {
      const int k = e / WG_RB, rr = e % WG_RB, r = r0 + rr;
      const bool ok = k < nb && r < a.d_r;
      sdz[k][rr] = ok ? a.dz32[static_cast<size_t>(m0 + k) * a.d_r + r] : 0.f;
      sa[k][rr] = ok ? a.a32[static_cast<size_t>(m0 + k) * a.d_r + r] : 0.f;
    }
    if (threadIdx.x < WG_TB) {
      const int k = threadIdx.x;
      const int t = k < nb ? a.idx_ad[m0 + k] : 0;
      st[k] = t;
      sg[k] = k < nb ? 1.0f - a.gate[t] : 0.f;
    }
    __syncthreads();
    if (!col_ok) continue;
#pragma unroll 4
    for (int k = 0; k < nb; ++k) {
      const size_t row = static_cast<size_t>(st[k]) * a.d + i;
      const float uu = ldf(U + row), dy = sg[k] * ldf(DH + row);
#pragma unroll
      for (int rr = 0; rr < WG_RB; ++rr) {
        g1[rr] = fmaf(sdz[k][rr], uu, g1[rr]);
        g2[rr] = fmaf(sa[k][rr], dy, g2[rr]);
      }
    }
  }
  if (!col_ok) return;
  const size_t c = blockIdx.z;
#pragma unroll
  for (int rr = 0; rr < WG_RB; ++rr) {
    const int r = r0 + rr;
    if (r >= a.d_r) break;
    a.pw1[(c * a.d_r + r) * a.d + i] = g1[rr];
    a.pw2[(c * a.d + i) * a.d_r + r] = g2[rr];
  }
}

// dW = the sum of the chunks' partials, chunk 0 first (zero when no token took the adapter)
__global__ __launch_bounds__(256) void adapter_wgrad_reduce(BlockBwdArgs a) {
  const int n = a.counts[1];
  const int nc = (n + a.chunk - 1) / a.chunk;
  const size_t E = static_cast<size_t>(a.d_r) * a.d;
  for (size_t e = blockIdx.x * static_cast<size_t>(256) + threadIdx.x; e < E;
       e += static_cast<size_t>(gridDim.x) * 256) {
    float s1 = 0.f, s2 = 0.f;
    for (int c = 0; c < nc; ++c) {
      s1 += a.pw1[c * E + e];
      s2 += a.pw2[c * E + e];
    }
    a.dw1[e] = s1;
    a.dw2[e] = s2;
  }
}

// One wave per token: virtual row v < counts[0] is FFN row v, the rest adapter row v - counts[0].
template <typename T>
__global__ __launch_bounds__(256) void block_bwd_rows_kernel(BlockBwdArgs a) {
  const int lane = threadIdx.x & 63;
  const int v = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (v >= a.T) return;
  const int nf = a.counts[0];
  int t;
  const float* du;
  float dg;
  if (v < nf) {
    t = a.idx_ffn[v];
    du = a.du_f + static_cast<size_t>(v) * a.d;
    float s = 0.f;
    for (int p = lane; p < a.n_parts; p += kWave) s += a.dgpart[static_cast<size_t>(v) * a.n_parts + p];
    dg = wave_sum(s);
  } else {
    const int m = v - nf;
    if (m >= a.counts[1]) return;
    t = a.idx_ad[m];
    du = a.du_a + static_cast<size_t>(m) * a.d;
    dg = a.dg_ad[m];
  }
  const T* hb = static_cast<const T*>(a.hbar) + static_cast<size_t>(t) * a.d;
  const T* dh = static_cast<const T*>(a.dh) + static_cast<size_t>(t) * a.d;
  const T* w = static_cast<const T*>(a.norm_w);
  float s1 = 0.f;
  for (int c = 8 * lane; c < a.d; c += 8 * kWave) {
    float x[8], y[8], z[8];
    ld8(hb + c, x);
    ld8(w + c, y);
    ld8(du + c, z);
#pragma unroll
    for (int k = 0; k < 8; ++k) s1 += y[k] * z[k] * x[k];
  }
  s1 = wave_sum(s1);
  const float r = a.rowstat[4 * static_cast<size_t>(t)];
  const float k3 = r * r * r * s1 / static_cast<float>(a.d);
  T* out = static_cast<T*>(a.dhbar) + static_cast<size_t>(t) * a.d;
  for (int c = 8 * lane; c < a.d; c += 8 * kWave) {
    float x[8], y[8], z[8], g[8], o[8];
    ld8(hb + c, x);
    ld8(w + c, y);
    ld8(du + c, z);
    ld8(dh + c, g);
#pragma unroll
    for (int k = 0; k < 8; ++k) o[k] = g[k] + r * y[k] * z[k] - k3 * x[k];
    st8(out + c, o);
  }
  if (lane == 0) {
    if (a.dgate_in) dg += a.dgate_in[t];
    const float g = a.gate[t];
    a.dgate[t] = dg;
    a.dlogit[t] = dg * g * (1.0f - g);
  }
}

// One workgroup: thread k takes tokens k, k + 1024, ...; the loss is a fixed tree over the
// threads' sums.
__global__ __launch_bounds__(1024) void skip_penalty_kernel(const float* __restrict__ gates, int L_R, int batch,
                                                            int seq, float alpha, float* __restrict__ loss,
                                                            float* __restrict__ dgates) {
  __shared__ float red[1024];
  const int T = batch * seq;
  const float npos = static_cast<float>(batch) * static_cast<float>(seq - 1);
  const float k = seq > 1 ? 2.0f * alpha / npos : 0.0f;
  float acc = 0.f;
  for (int t = threadIdx.x; t < T; t += 1024) {
    const bool has_next = (t % seq) != seq - 1;
    float tot = 0.f;
    for (int j = 0; j < L_R; ++j) tot += gates[static_cast<size_t>(j) * T + t];
    if (has_next) acc += tot * tot;
    const float gd = has_next ? k * tot : 0.0f;
    for (int j = 0; j < L_R; ++j) dgates[static_cast<size_t>(j) * T + t] = gd;
  }
  red[threadIdx.x] = acc;
  __syncthreads();
  for (int w = 512; w > 0; w >>= 1) {
    if (static_cast<int>(threadIdx.x) < w) red[threadIdx.x] += red[threadIdx.x + w];
    __syncthreads();
  }
  if (threadIdx.x == 0) loss[0] = seq > 1 ? alpha * red[0] / npos : 0.0f;
}

// The caller's branch lists, copied with every count and index clamped into range, so that a
// malformed list gives wrong numbers but no access outside the buffers.
__global__ __launch_bounds__(256) void bwd_lists_kernel(int T, const int* __restrict__ idx_ffn,
                                                        const int* __restrict__ idx_ad,
                                                        const int* __restrict__ counts, int* __restrict__ f,
                                                        int* __restrict__ ad, int* __restrict__ c) {
  const int nf = min(max(counts[0], 0), T);
  const int na = min(max(counts[1], 0), T - nf);
  const int i = blockIdx.x * 256 + threadIdx.x;
  if (i == 0) {
    c[0] = nf;
    c[1] = na;
  }
  if (i < nf) f[i] = min(max(idx_ffn[i], 0), T - 1);
  if (i < na) ad[i] = min(max(idx_ad[i], 0), T - 1);
}

}  // namespace

hipError_t launch_bwd_lists(int T, const int* idx_ffn, const int* idx_ad, const int* counts, int* f, int* ad,
                            int* c, hipStream_t s) {
  bwd_lists_kernel<<<(T + 255) / 256, 256, 0, s>>>(T, idx_ffn, idx_ad, counts, f, ad, c);
  return hipGetLastError();
}

hipError_t launch_transpose(int dtype, const void* in, int R, int C, int ld_in, void* out, int ld_out,
                            int R_pad, hipStream_t s) {
  if (R <= 0 || C <= 0) return hipSuccess;
  R_pad = R_pad > R ? R_pad : R;
  const dim3 grid((C + 63) / 64, (R_pad + 63) / 64);
  if (dtype == 1)
    transpose_kernel<bf16_t><<<grid, 256, 0, s>>>(static_cast<const bf16_t*>(in), R, C, ld_in,
                                                  static_cast<bf16_t*>(out), ld_out, R_pad);
  else
    transpose_kernel<float><<<grid, 256, 0, s>>>(static_cast<const float*>(in), R, C, ld_in,
                                                 static_cast<float*>(out), ld_out, R_pad);
  return hipGetLastError();
}

hipError_t launch_adapter_bwd_mid(const BlockBwdArgs& a, hipStream_t s) {
  const dim3 grid((a.T + 3) / 4);
  if (a.dtype == 1)
    adapter_bwd_mid_kernel<bf16_t><<<grid, 256, 0, s>>>(a);
  else
    adapter_bwd_mid_kernel<float><<<grid, 256, 0, s>>>(a);
  return hipGetLastError();
}

hipError_t launch_adapter_wgrad(const BlockBwdArgs& a, hipStream_t s) {
  const dim3 grid((a.d + 255) / 256, (a.d_r + WG_RB - 1) / WG_RB, (a.T + a.chunk - 1) / a.chunk);
  if (a.dtype == 1)
    adapter_wgrad_kernel<bf16_t><<<grid, 256, 0, s>>>(a);
  else
    adapter_wgrad_kernel<float><<<grid, 256, 0, s>>>(a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const size_t E = static_cast<size_t>(a.d_r) * a.d;
  const int blocks = static_cast<int>(std::min<size_t>((E + 255) / 256, 4096));
  adapter_wgrad_reduce<<<blocks, 256, 0, s>>>(a);
  return hipGetLastError();
}

hipError_t launch_block_bwd_rows(const BlockBwdArgs& a, hipStream_t s) {
  const dim3 grid((a.T + 3) / 4);
  if (a.dtype == 1)
    block_bwd_rows_kernel<bf16_t><<<grid, 256, 0, s>>>(a);
  else
    block_bwd_rows_kernel<float><<<grid, 256, 0, s>>>(a);
  return hipGetLastError();
}

hipError_t launch_skip_penalty(const float* gates, int L_R, int batch, int seq, float alpha, float* loss,
                               float* dgates, hipStream_t s) {
  skip_penalty_kernel<<<1, 1024, 0, s>>>(gates, L_R, batch, seq, alpha, loss, dgates);
  return hipGetLastError();
}

}  // namespace hero
