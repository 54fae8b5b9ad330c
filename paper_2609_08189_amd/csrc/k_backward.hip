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
//   * the adapter weight gradients, summed over token chunks in a fixed order (for wide ranks,
//     tokens-contiguous copies of the adapter rows, which the GEMM core then contracts);
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
__device__ __forceinline__ void transpose_tile(const T* __restrict__ in, int R, int C, int ld_in,
                                               T* __restrict__ out, int ld_out, int R_pad, int c0, int r0) {
  __shared__ T tile[64][65];
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

template <typename T>
__global__ __launch_bounds__(256) void transpose_kernel(const T* __restrict__ in, int R, int C, int ld_in,
                                                        T* __restrict__ out, int ld_out, int R_pad) {
  transpose_tile(in, R, C, ld_in, out, ld_out, R_pad, blockIdx.x * 64, blockIdx.y * 64);
}

// W_2^T [d_r][d] and W_1^T [d][rpad] (zero columns past d_r) in one launch: the first tiles of
// the 1-D grid cover W_2, the rest W_1
template <typename T>
__global__ __launch_bounds__(256) void adapter_transpose_kernel(const T* __restrict__ w1, const T* __restrict__ w2,
                                                                T* __restrict__ w1t, T* __restrict__ w2t, int d,
                                                                int d_r, int rpad) {
  const int tx2 = (d_r + 63) / 64;             // W_2 [d][d_r]: column tiles x row tiles
  const int n2 = tx2 * ((d + 63) / 64);
  const int b = blockIdx.x;
  if (b < n2)
    transpose_tile(w2, d, d_r, d_r, w2t, d, d, (b % tx2) * 64, (b / tx2) * 64);
  else {
    const int b1 = b - n2, tx1 = (d + 63) / 64;  // W_1 [d_r][d], rows padded to rpad
    transpose_tile(w1, d_r, d, d, w1t, rpad, rpad, (b1 % tx1) * 64, (b1 / tx1) * 64);
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
  const size_t slice = static_cast<size_t>(a.na_max) * a.d_r;
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

// Weight-gradient partials of one chunk of adapter rows,
//   pw1[c][r][i] = sum_m dz[m][r] u[t_m][i],  pw2[c][i][r] = sum_m a[m][r] (1 - g_t) dh[t_m][i].
// A workgroup covers 128 columns i and 64 ranks r; a thread owns an 8-rank x 4-column block of
// both (rank group tid % 8, column group tid / 8), so each staged
// value read from LDS feeds 4 or 8 FMAs.  Rows are staged WG_TB at a time (u and
// (1 - g) dh as fp32, dz, a), zero past the chunk's end.  The rows split into gridDim.z chunks
// of equal size (whole batches) from the device count.
constexpr int WG_TB = 32, WG_C = 128, WG_R = 64;

__device__ __forceinline__ int wgrad_chunk(int n, int slices) {
  return ((n + slices - 1) / slices + WG_TB - 1) / WG_TB * WG_TB;
}

template <typename T>
__global__ __launch_bounds__(256) void adapter_wgrad_kernel(BlockBwdArgs a) {
  __shared__ __attribute__((aligned(16))) float su[WG_TB][WG_C];
  __shared__ __attribute__((aligned(16))) float sdy[WG_TB][WG_C];
  __shared__ __attribute__((aligned(16))) float sdz[WG_TB][WG_R];
  __shared__ __attribute__((aligned(16))) float sa[WG_TB][WG_R];
  const int n = a.counts[1];
  const int chunk = wgrad_chunk(n, gridDim.z);
  const int mb = blockIdx.z * chunk;
  if (mb >= n) return;
  const int me = min(n, mb + chunk);
  const int tid = threadIdx.x;
  const int rg = tid & 7, cg = tid >> 3;            // 8 ranks, 4 columns
  const int c0 = blockIdx.x * WG_C, r0 = blockIdx.y * WG_R;
  const T* U = static_cast<const T*>(a.u);
  const T* DH = static_cast<const T*>(a.dh);
  float g1[8][4], g2[4][8];
#pragma unroll
  for (int x = 0; x < 8; ++x)
#pragma unroll
    for (int y = 0; y < 4; ++y) g1[x][y] = g2[y][x] = 0.f;
  for (int m0 = mb; m0 < me; m0 += WG_TB) {
    const int nb = min(WG_TB, me - m0);
    __syncthreads();
    // u and (1 - g) dh: WG_TB rows x 128 columns in 8-column pieces, two per thread
#pragma unroll
    for (int q = 0; q < 2; ++q) {
      const int e = tid + 256 * q;
      const int k = e >> 4, c8 = (e & 15) * 8;
      float uv[8], dv[8];
      if (k < nb && c0 + c8 < a.d) {
        const int t = a.idx_ad[m0 + k];
        const float om = 1.0f - a.gate[t];
        const size_t row = static_cast<size_t>(t) * a.d + c0 + c8;
        ld8(U + row, uv);
        ld8(DH + row, dv);
#pragma unroll
        for (int x = 0; x < 8; ++x) dv[x] *= om;
      } else {
#pragma unroll
        for (int x = 0; x < 8; ++x) uv[x] = dv[x] = 0.f;
      }
#pragma unroll
      for (int x = 0; x < 8; ++x) {
        su[k][c8 + x] = uv[x];
        sdy[k][c8 + x] = dv[x];
      }
    }
    for (int e = tid; e < WG_TB * WG_R; e += 256) {
      const int k = e / WG_R, rr = e % WG_R, r = r0 + rr;
      const bool ok = k < nb && r < a.d_r;
      sdz[k][rr] = ok ? a.dz32[static_cast<size_t>(m0 + k) * a.d_r + r] : 0.f;
      sa[k][rr] = ok ? a.a32[static_cast<size_t>(m0 + k) * a.d_r + r] : 0.f;
    }
    __syncthreads();
#pragma unroll 4
    for (int k = 0; k < WG_TB; ++k) {
      const f32x4 u4 = *reinterpret_cast<const f32x4*>(&su[k][cg * 4]);
      const f32x4 y4 = *reinterpret_cast<const f32x4*>(&sdy[k][cg * 4]);
      const f32x4 z0 = *reinterpret_cast<const f32x4*>(&sdz[k][rg * 8]);
      const f32x4 z1 = *reinterpret_cast<const f32x4*>(&sdz[k][rg * 8 + 4]);
      const f32x4 a0 = *reinterpret_cast<const f32x4*>(&sa[k][rg * 8]);
      const f32x4 a1 = *reinterpret_cast<const f32x4*>(&sa[k][rg * 8 + 4]);
#pragma unroll
      for (int x = 0; x < 8; ++x) {
        const float zv = x < 4 ? z0[x] : z1[x - 4];
        const float av = x < 4 ? a0[x] : a1[x - 4];
#pragma unroll
        for (int y = 0; y < 4; ++y) {
          g1[x][y] = fmaf(zv, u4[y], g1[x][y]);
          g2[y][x] = fmaf(av, y4[y], g2[y][x]);
        }
      }
    }
  }
  const size_t c = blockIdx.z;
  const int i = c0 + cg * 4;
  if (i >= a.d) return;
#pragma unroll
  for (int x = 0; x < 8; ++x) {
    const int r = r0 + rg * 8 + x;
    if (r < a.d_r) {
      f32x4 v = {g1[x][0], g1[x][1], g1[x][2], g1[x][3]};
      *reinterpret_cast<f32x4*>(a.pw1 + (c * a.d_r + r) * a.d + i) = v;
    }
  }
#pragma unroll
  for (int y = 0; y < 4; ++y) {
    float* o = a.pw2 + (c * a.d + i + y) * a.d_r + r0 + rg * 8;
#pragma unroll
    for (int x = 0; x < 8; ++x)
      if (r0 + rg * 8 + x < a.d_r) o[x] = g2[y][x];
  }
}

// The same partials on the matrix cores (bf16): the tokens are the K of two products,
//   dW_1 block [64 r][128 i] = dz^T [r][m] (u [m][i]),  dW_2 block [128 i][64 r] = dy^T [i][m] (a [m][r]),
// with dy = (1 - g) dh.  A batch of 32 rows is staged transposed in LDS as bf16 (K contiguous, row
// pitch 40 elements, so the 16-byte fragment reads of 32 rows spread over the banks); the next
// batch's global loads are in flight while the current one is multiplied.  Wave w owns column
// block i = 32 w of both products: 2 + 2 tiles of v_mfma_f32_32x32x16_bf16 per 16 rows.
// RT: 32-rank tiles per workgroup (2: 128-rank blocks at rank 896 measured no faster, the
// kernel being bound by each batch's load latency rather than by re-staging u and dh).
constexpr int WM_TB = 32, WM_PT = 40;

template <int RT>
__global__ __launch_bounds__(256) void adapter_wgrad_mfma(BlockBwdArgs a) {
  constexpr int WR = 32 * RT;
  __shared__ __attribute__((aligned(16))) bf16_t suT[WG_C][WM_PT];
  __shared__ __attribute__((aligned(16))) bf16_t sdyT[WG_C][WM_PT];
  __shared__ __attribute__((aligned(16))) bf16_t sdzT[WR][WM_PT];
  __shared__ __attribute__((aligned(16))) bf16_t saT[WR][WM_PT];
  const int n = a.counts[1];
  const int chunk = wgrad_chunk(n, gridDim.z);
  const int mb = blockIdx.z * chunk;
  if (mb >= n) return;
  const int me = min(n, mb + chunk);
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int c0 = blockIdx.x * WG_C, r0 = blockIdx.y * WR;
  const bf16_t* U = static_cast<const bf16_t*>(a.u);
  const bf16_t* DH = static_cast<const bf16_t*>(a.dh);
  // this thread's staging work per batch: two 8-column pieces of u and dh (token k = e / 16),
  // 4 RT (token, rank) entries of dz and a; fetched into registers one batch ahead
  constexpr int NZ = WM_TB * WR / 256;
  u32x4 pu0, pu1, pd0, pd1;
  float om0, om1, pz[NZ], pa[NZ];
  const int k0 = tid >> 4, k1 = (tid + 256) >> 4, c8 = (tid & 15) * 8;
#define HERO_WG_FETCH(m0_)                                                                          \
  {                                                                                               \
    const int nb_ = min(WM_TB, me - (m0_));                                                       \
    om0 = om1 = 0.f;                                                                              \
    pu0 = pu1 = pd0 = pd1 = u32x4{0, 0, 0, 0};                                                    \
    if (k0 < nb_) {                                                                               \
      const int t_ = a.idx_ad[(m0_) + k0];                                                        \
      om0 = 1.0f - a.gate[t_];                                                                    \
      const size_t row_ = static_cast<size_t>(t_) * a.d + c0 + c8;                                \
      pu0 = *reinterpret_cast<const u32x4*>(U + row_);                                            \
      pd0 = *reinterpret_cast<const u32x4*>(DH + row_);                                           \
    }                                                                                             \
    if (k1 < nb_) {                                                                               \
      const int t_ = a.idx_ad[(m0_) + k1];                                                        \
      om1 = 1.0f - a.gate[t_];                                                                    \
      const size_t row_ = static_cast<size_t>(t_) * a.d + c0 + c8;                                \
      pu1 = *reinterpret_cast<const u32x4*>(U + row_);                                            \
      pd1 = *reinterpret_cast<const u32x4*>(DH + row_);                                           \
    }                                                                                             \
    _Pragma("unroll") for (int q = 0; q < NZ; ++q) {                                              \
      const int e_ = tid + 256 * q;                                                               \
      const int k_ = e_ / WR, r_ = r0 + e_ % WR;                                                  \
      const bool ok_ = k_ < nb_ && r_ < a.d_r;                                                    \
      pz[q] = ok_ ? a.dz32[static_cast<size_t>((m0_) + k_) * a.d_r + r_] : 0.f;                   \
      pa[q] = ok_ ? a.a32[static_cast<size_t>((m0_) + k_) * a.d_r + r_] : 0.f;                    \
    }                                                                                             \
  }
  auto put8 = [&](int k, u32x4 wu, u32x4 wd, float om) {
#pragma unroll
    for (int x = 0; x < 8; ++x) {
      const uint32_t u2 = wu[x >> 1], d2 = wd[x >> 1];
      suT[c8 + x][k] = static_cast<bf16_t>((x & 1) ? (u2 >> 16) : (u2 & 0xffffu));
      sdyT[c8 + x][k] = f32_to_bf16(__uint_as_float((x & 1) ? (d2 & 0xffff0000u) : (d2 << 16)) * om);
    }
  };
  f32x16 acc1[RT], acc2[RT];
#pragma unroll
  for (int b = 0; b < RT; ++b)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc1[b][r] = acc2[b][r] = 0.f;
  const int fr = lane & 31, kh = 8 * (lane >> 5);
  HERO_WG_FETCH(mb)
  for (int m0 = mb; m0 < me; m0 += WM_TB) {
    __syncthreads();
    put8(k0, pu0, pd0, om0);
    put8(k1, pu1, pd1, om1);
#pragma unroll
    for (int q = 0; q < NZ; ++q) {
      const int e = tid + 256 * q;
      const int k = e / WR, rr = e % WR;
      sdzT[rr][k] = f32_to_bf16(pz[q]);
      saT[rr][k] = f32_to_bf16(pa[q]);
    }
    __syncthreads();
    if (m0 + WM_TB < me) HERO_WG_FETCH(m0 + WM_TB)
#pragma unroll
    for (int ks = 0; ks < WM_TB / 16; ++ks) {
      const int ko = 16 * ks + kh;
      const bf16x8 fu = *reinterpret_cast<const bf16x8*>(&suT[32 * wave + fr][ko]);
      const bf16x8 fy = *reinterpret_cast<const bf16x8*>(&sdyT[32 * wave + fr][ko]);
#pragma unroll
      for (int b = 0; b < RT; ++b) {
        const bf16x8 fz = *reinterpret_cast<const bf16x8*>(&sdzT[32 * b + fr][ko]);
        const bf16x8 fa = *reinterpret_cast<const bf16x8*>(&saT[32 * b + fr][ko]);
        acc1[b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fz, fu, acc1[b], 0, 0, 0);
        acc2[b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fy, fa, acc2[b], 0, 0, 0);
      }
    }
  }
#undef HERO_WG_FETCH
  const size_t c = blockIdx.z;
#pragma unroll
  for (int b = 0; b < RT; ++b)
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int row = 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
      // dW_1: row = rank 32 b + row, column i = 32 wave + fr
      const int rk = r0 + 32 * b + row;
      if (rk < a.d_r) a.pw1[(c * a.d_r + rk) * a.d + c0 + 32 * wave + fr] = acc1[b][r];
      // dW_2: row = column i = 32 wave + row, column = rank 32 b + fr
      const int rk2 = r0 + 32 * b + fr;
      if (rk2 < a.d_r) a.pw2[(c * a.d + c0 + 32 * wave + row) * a.d_r + rk2] = acc2[b][r];
    }
}

// Tokens-contiguous copies of the adapter rows for the wide-rank weight gradients.  A workgroup
// takes 64 tokens x 64 features of one of the four outputs (blockIdx.z): it reads the token-major
// rows with loads contiguous along the features, and writes the transposed tile with stores
// contiguous along the tokens; tokens past counts[1] (up to kp) are written as zero.
__global__ __launch_bounds__(256) void adapter_wgrad_stage_kernel(BlockBwdArgs a, int kp, bf16_t* __restrict__ uaT,
                                                                  bf16_t* __restrict__ dyT, bf16_t* __restrict__ dzT,
                                                                  bf16_t* __restrict__ aT) {
  __shared__ float tile[64][65];
  const int n = a.counts[1];
  const int which = blockIdx.z;                      // 0 u, 1 dy, 2 dz, 3 a
  const int F = which < 2 ? a.d : a.d_r;             // features of this output
  const int f0 = blockIdx.y * 64, m0 = blockIdx.x * 64;
  if (f0 >= F) return;
  const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;
  const bf16_t* U = static_cast<const bf16_t*>(a.u);
  const bf16_t* DH = static_cast<const bf16_t*>(a.dh);
  for (int k = ty; k < 64; k += 4) {
    const int m = m0 + k, f = f0 + tx;
    float v = 0.f;
    if (m < n && f < F) {
      if (which < 2) {
        const int t = a.idx_ad[m];
        const size_t o = static_cast<size_t>(t) * a.d + f;
        v = which == 0 ? bf16_to_f32(U[o]) : (1.0f - a.gate[t]) * bf16_to_f32(DH[o]);
      } else {
        v = (which == 2 ? a.dz32 : a.a32)[static_cast<size_t>(m) * a.d_r + f];
      }
    }
    tile[k][tx] = v;
  }
  __syncthreads();
  bf16_t* out = which == 0 ? uaT : which == 1 ? dyT : which == 2 ? dzT : aT;
  for (int k = ty; k < 64; k += 4) {
    const int f = f0 + k, m = m0 + tx;
    if (f < F && m < kp) out[static_cast<size_t>(f) * kp + m] = f32_to_bf16(tile[tx][k]);
  }
}

// dW = the sum of the chunks' partials, chunk 0 first (zero when no token took the adapter)
__global__ __launch_bounds__(256) void adapter_wgrad_reduce(BlockBwdArgs a) {
  const int n = a.counts[1];
  const int chunk = wgrad_chunk(n, a.n_slices);
  const int nc = n > 0 ? (n + chunk - 1) / chunk : 0;
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
__global__ __launch_bounds__(256) void bwd_lists_kernel(int T, int nf_max, int na_max,
                                                        const int* __restrict__ idx_ffn,
                                                        const int* __restrict__ idx_ad,
                                                        const int* __restrict__ counts, int* __restrict__ f,
                                                        int* __restrict__ ad, int* __restrict__ c) {
  const int nf = min(max(counts[0], 0), nf_max);
  const int na = min(min(max(counts[1], 0), T - nf), na_max);
  const int i = blockIdx.x * 256 + threadIdx.x;
  if (i == 0) {
    c[0] = nf;
    c[1] = na;
  }
  if (i < nf) f[i] = min(max(idx_ffn[i], 0), T - 1);
  if (i < na) ad[i] = min(max(idx_ad[i], 0), T - 1);
}

}  // namespace

hipError_t launch_bwd_lists(int T, int nf_max, int na_max, const int* idx_ffn, const int* idx_ad, const int* counts,
                            int* f, int* ad, int* c, hipStream_t s) {
  bwd_lists_kernel<<<(T + 255) / 256, 256, 0, s>>>(T, nf_max, na_max, idx_ffn, idx_ad, counts, f, ad, c);
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

hipError_t launch_adapter_transpose(int dtype, const void* w1, const void* w2, void* w1t, void* w2t, int d, int d_r,
                                    int rpad, hipStream_t s) {
  const int blocks = (d_r + 63) / 64 * ((d + 63) / 64) + (d + 63) / 64 * ((rpad + 63) / 64);
  if (dtype == 1)
    adapter_transpose_kernel<bf16_t><<<blocks, 256, 0, s>>>(static_cast<const bf16_t*>(w1),
                                                            static_cast<const bf16_t*>(w2), static_cast<bf16_t*>(w1t),
                                                            static_cast<bf16_t*>(w2t), d, d_r, rpad);
  else
    adapter_transpose_kernel<float><<<blocks, 256, 0, s>>>(static_cast<const float*>(w1),
                                                           static_cast<const float*>(w2), static_cast<float*>(w1t),
                                                           static_cast<float*>(w2t), d, d_r, rpad);
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
  if (a.dtype == 1) {
    adapter_wgrad_mfma<2><<<dim3((a.d + WG_C - 1) / WG_C, (a.d_r + 63) / 64, a.n_slices), 256, 0, s>>>(a);
  } else {
    adapter_wgrad_kernel<float><<<dim3((a.d + WG_C - 1) / WG_C, (a.d_r + WG_R - 1) / WG_R, a.n_slices), 256, 0, s>>>(a);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const size_t E = static_cast<size_t>(a.d_r) * a.d;
  const int blocks = static_cast<int>(std::min<size_t>((E + 255) / 256, 4096));
  adapter_wgrad_reduce<<<blocks, 256, 0, s>>>(a);
  return hipGetLastError();
}

hipError_t launch_adapter_wgrad_stage(const BlockBwdArgs& a, int kp, void* uaT, void* dyT, void* dzT, void* aT,
                                      hipStream_t s) {
  const int fmax = a.d > a.d_r ? a.d : a.d_r;
  const dim3 grid((kp + 63) / 64, (fmax + 63) / 64, 4);
  adapter_wgrad_stage_kernel<<<grid, 256, 0, s>>>(a, kp, static_cast<bf16_t*>(uaT), static_cast<bf16_t*>(dyT),
                                                  static_cast<bf16_t*>(dzT), static_cast<bf16_t*>(aT));
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
