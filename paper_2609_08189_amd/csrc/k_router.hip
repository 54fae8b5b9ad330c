// Fused router tail with the depth-memory read-modify-write (Sec. 3.2).
//
// One workgroup of 256 threads takes TB consecutive tokens.  From the router
// pre-activations P = [W_hd hbar; psi_1 hbar] and the row statistics it forms,
// per token and in the paper's order:
//   z^h = W_hu SiLU(inv_rms * W_hd hbar)                         (hidden encoder, unit-gain RMSNorm)
//   x^path = [j/L_R, (L_R-j)/L_R, |delta_j|, gamma_j, p_{j-1}, m_{j-1}]   (eq:path_vector)
//   z^a = W_p2 SiLU(W_p1 x^path),  s = [z^h; z^a]                (eq:router_state)
//   q, k, v = W_q s, W_k s, W_v s
//   one streaming pass over S (fp32, d_m x d_m per token):
//     c = phi(q)^T S / (phi(q)^T zeta + eps)                     (eq:memory_read, read first)
//     S <- rho S + phi(k) v^T,  zeta <- rho zeta + phi(k)         (eq:memory_update, same pass)
//   nu = 1 - cos(W_n s, W_c c) (0 at j = 1)
//   a = th2 . SiLU(th1 [s; c; nu]),  p = sigma(a / T_hist),  m = m_{j-1} p
//   b = ps2 . SiLU(psi_1 hbar),  logit = a + b (+ bias),  g = sigma(logit)   (eq:final_gate)
// At j = 1 the state is the paper's initial value: S and zeta are not read (taken
// as zero) and p_{0} = m_{0} = 1.
// The S pass is the HBM-bound part (2 * 4 * d_m^2 bytes per token); the small
// matrix-vector products reuse each weight element across the TB tokens.
#include "hero_device.h"
#include "hero_kernels.h"

namespace hero {
namespace {

constexpr int TB = 8;     // tokens per workgroup
constexpr int NT = 256;   // threads per workgroup
constexpr int MAXE = 512; // max(d_e, d_head)
constexpr int MAXS = 128; // max d_s
constexpr int MAXP = 128; // max d_p

struct Ident {
  __device__ __forceinline__ float operator()(float x) const { return x; }
};
struct SiLU {
  __device__ __forceinline__ float operator()(float x) const { return siluf_(x); }
};

// out[t*os + o] = act(sum_i W[o*ldw + i] * in[t*is + i]) for o < O and all TB tokens.
// P lanes share one output row (power of two, within a wave) and reduce by shuffles.
template <typename W, class Act>
__device__ __forceinline__ void matvec(const W* __restrict__ w, int ldw, int O, int I,
                                       const float* in, int is, float* out, int os, Act act) {
  int P = 64;
  while (P > 1 && P * O > NT) P >>= 1;
  const int rows_per_pass = NT / P;
  const int slice = threadIdx.x % P;
  for (int o0 = 0; o0 < O; o0 += rows_per_pass) {
    const int o = o0 + static_cast<int>(threadIdx.x) / P;
    float acc[TB];
#pragma unroll
    for (int t = 0; t < TB; ++t) acc[t] = 0.f;
    if (o < O) {
      const W* wr = w + static_cast<size_t>(o) * ldw;
      for (int i = slice; i < I; i += P) {
        const float wv = ldf(wr + i);
#pragma unroll
        for (int t = 0; t < TB; ++t) acc[t] = fmaf(wv, in[t * is + i], acc[t]);
      }
    }
    for (int off = P >> 1; off > 0; off >>= 1)
#pragma unroll
      for (int t = 0; t < TB; ++t) acc[t] += __shfl_xor(acc[t], off, kWave);
    if (o < O && slice == 0)
#pragma unroll
      for (int t = 0; t < TB; ++t) out[t * os + o] = act(acc[t]);
  }
}

template <typename W, int DM>
__global__ __launch_bounds__(NT) void router_tail_kernel(RouterTailArgs a) {
  constexpr int C4 = DM / 4;        // float4 columns of one S row
  constexpr int RP = NT / C4;       // S rows per pass
  constexpr int NR = DM / RP;       // S rows per thread
  constexpr int XIN = MAXS + DM + 1;
#define LDS16 __shared__ __attribute__((aligned(16)))
  LDS16 float bufA[TB][MAXE];       // SiLU(inv_rms W_hd hbar), later the f_theta hidden
  LDS16 float bufB[TB][MAXE];       // SiLU(psi_1 hbar)
  LDS16 float x[TB][XIN];           // [s; c; nu]
  LDS16 float xp[TB][8];            // path vector
  LDS16 float zp[TB][MAXP];         // path-encoder hidden
  LDS16 float qkvn[4][TB][DM];      // phi(q), phi(k), v, W_n s
  LDS16 float wc[TB][DM];           // W_c c
  LDS16 f32x4 red[RP][C4];          // partial memory reads
  LDS16 float sc[8][TB];            // per-token scalars
#undef LDS16

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int t0 = blockIdx.x * TB;
  const int j = a.j;
  const int d_s = a.d_s, d_e = a.d_e, d_head = a.d_head, NP = a.d_e + a.d_head;
  const float rho = 1.0f / (1.0f + expf(-a.eta));
  const W* w_hu = static_cast<const W*>(a.w_hu);

  // per-token scalars and the path vector
  if (tid < TB) {
    const int t = t0 + tid;
    float inv_rms = 0.f, dd = 0.f, dp = 0.f, pp = 0.f, pprev = 1.f, mprev = 1.f, beta = 0.f;
    if (t < a.T) {
      const f32x4 rs = *reinterpret_cast<const f32x4*>(a.rowstat + 4 * static_cast<size_t>(t));
      inv_rms = rs[0];
      dd = rs[1];
      dp = rs[2];
      pp = rs[3];
      if (j > 1) {
        pprev = a.p_hist[t];
        mprev = a.m_hist[t];
      }
      if (a.beta) beta = a.beta[t];
    }
    const float dj = j >= 2 ? sqrtf(dd) : 0.f;
    const float gam = j >= 3 ? dp / (dj * sqrtf(pp) + a.eps) : 0.f;
    xp[tid][0] = static_cast<float>(j) / static_cast<float>(a.L_R);
    xp[tid][1] = static_cast<float>(a.L_R - j) / static_cast<float>(a.L_R);
    xp[tid][2] = dj;
    xp[tid][3] = gam;
    xp[tid][4] = pprev;
    xp[tid][5] = mprev;
    sc[0][tid] = inv_rms;
    sc[1][tid] = mprev;
    sc[2][tid] = beta;
  }
  __syncthreads();

  // SiLU of the encoder and local-head pre-activations
  for (int e = tid; e < TB * NP; e += NT) {
    const int tt = e / NP, i = e % NP;
    const int t = min(t0 + tt, a.T - 1);
    const float pv = a.P[static_cast<size_t>(t) * NP + i];
    if (i < d_e)
      bufA[tt][i] = siluf_(sc[0][tt] * pv);
    else
      bufB[tt][i - d_e] = siluf_(pv);
  }
  __syncthreads();

  // z^h into s[0:d_h), path-encoder hidden, local head b
  matvec(w_hu, d_e, a.d_h, d_e, &bufA[0][0], MAXE, &x[0][0], XIN, Ident());
  matvec(static_cast<const W*>(a.w_p1), 6, a.d_p, 6, &xp[0][0], 8, &zp[0][0], MAXP, SiLU());
  matvec(static_cast<const W*>(a.ps2), d_head, 1, d_head, &bufB[0][0], MAXE, &sc[3][0], 1, Ident());
  __syncthreads();
  // z^a into s[d_h:d_s)
  matvec(static_cast<const W*>(a.w_p2), a.d_p, a.d_a, a.d_p, &zp[0][0], MAXP, &x[0][a.d_h], XIN, Ident());
  __syncthreads();
  // q, k, v, W_n s
  matvec(static_cast<const W*>(a.w_q), d_s, DM, d_s, &x[0][0], XIN, &qkvn[0][0][0], DM, Ident());
  matvec(static_cast<const W*>(a.w_k), d_s, DM, d_s, &x[0][0], XIN, &qkvn[1][0][0], DM, Ident());
  matvec(static_cast<const W*>(a.w_v), d_s, DM, d_s, &x[0][0], XIN, &qkvn[2][0][0], DM, Ident());
  matvec(static_cast<const W*>(a.w_n), d_s, DM, d_s, &x[0][0], XIN, &qkvn[3][0][0], DM, Ident());
  __syncthreads();
  for (int e = tid; e < 2 * TB * DM; e += NT) {
    float* p = &qkvn[0][0][0] + e;
    *p = phif_(*p);
  }
  __syncthreads();

  // normaliser: den = phi(q).zeta (before the update), zeta <- rho zeta + phi(k)
  for (int tt = wave; tt < TB; tt += NT / 64) {
    const int t = t0 + tt;
    float part = 0.f;
    if (t < a.T) {
      float* z = a.zeta + static_cast<size_t>(t) * DM;
      for (int k = lane; k < DM; k += 64) {
        const float zv = j > 1 ? z[k] : 0.f;
        part = fmaf(qkvn[0][tt][k], zv, part);
        z[k] = fmaf(rho, zv, qkvn[1][tt][k]);
      }
    }
    part = wave_sum(part);
    if (lane == 0) sc[4][tt] = part;
  }

  // memory read-modify-write, one token at a time, all threads streaming its S
  const int cq = tid % C4, rg = tid / C4;
  for (int tt = 0; tt < TB; ++tt) {
    const int t = t0 + tt;
    f32x4 cacc = {0.f, 0.f, 0.f, 0.f};
    if (t < a.T) {
      float* Sp = a.S + static_cast<size_t>(t) * DM * DM + 4 * cq;
      const f32x4 v4 = *reinterpret_cast<const f32x4*>(&qkvn[2][tt][4 * cq]);
      if (j == 1) {
#pragma unroll 16
        for (int i = 0; i < NR; ++i) {
          const int r = rg + RP * i;
          *reinterpret_cast<f32x4*>(Sp + r * DM) = qkvn[1][tt][r] * v4;
        }
      } else {
        constexpr int CH = NR < 16 ? NR : 16;
        for (int i0 = 0; i0 < NR; i0 += CH) {
          f32x4 sv[CH];
#pragma unroll
          for (int c = 0; c < CH; ++c) sv[c] = *reinterpret_cast<const f32x4*>(Sp + (rg + RP * (i0 + c)) * DM);
#pragma unroll
          for (int c = 0; c < CH; ++c) {
            const int r = rg + RP * (i0 + c);
            const float fq = qkvn[0][tt][r], fk = qkvn[1][tt][r];
            f32x4 o;
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              cacc[e] = fmaf(fq, sv[c][e], cacc[e]);
              o[e] = fmaf(rho, sv[c][e], fk * v4[e]);
            }
            *reinterpret_cast<f32x4*>(Sp + r * DM) = o;
          }
        }
      }
    }
    red[rg][cq] = cacc;
    __syncthreads();
    if (tid < DM) {
      float cs = 0.f;
      for (int g = 0; g < RP; ++g) cs += red[g][tid >> 2][tid & 3];
      x[tt][d_s + tid] = j > 1 ? cs / (sc[4][tt] + a.eps) : 0.f;
    }
    __syncthreads();
  }

  // nu = 1 - cos(W_n s, W_c c)
  matvec(static_cast<const W*>(a.w_c), DM, DM, DM, &x[0][d_s], XIN, &wc[0][0], DM, Ident());
  __syncthreads();
  for (int tt = wave; tt < TB; tt += NT / 64) {
    float nn = 0.f, cc = 0.f, nc = 0.f;
    for (int k = lane; k < DM; k += 64) {
      const float n = qkvn[3][tt][k], c = wc[tt][k];
      nn = fmaf(n, n, nn);
      cc = fmaf(c, c, cc);
      nc = fmaf(n, c, nc);
    }
    nn = wave_sum(nn);
    cc = wave_sum(cc);
    nc = wave_sum(nc);
    if (lane == 0) x[tt][d_s + DM] = j > 1 ? 1.0f - nc / (sqrtf(nn) * sqrtf(cc) + a.eps) : 0.f;
  }
  __syncthreads();

  // history head
  const int XI = d_s + DM + 1;
  matvec(static_cast<const W*>(a.th1), XI, d_head, XI, &x[0][0], XIN, &bufA[0][0], MAXE, SiLU());
  __syncthreads();
  matvec(static_cast<const W*>(a.th2), d_head, 1, d_head, &bufA[0][0], MAXE, &sc[5][0], 1, Ident());
  __syncthreads();

  if (tid < TB) {
    const int t = t0 + tid;
    if (t < a.T) {
      const float av = sc[5][tid], bv = sc[3][tid];
      const float p = sigmoidf_(av / a.T_hist);
      a.p_hist[t] = p;
      a.m_hist[t] = sc[1][tid] * p;
      const float l = av + bv + sc[2][tid];
      a.logit[t] = l;
      a.gate[t] = sigmoidf_(l);
    }
  }
}

template <typename W>
hipError_t launch_dm(const RouterTailArgs& a, hipStream_t s) {
  dim3 grid((a.T + TB - 1) / TB), block(NT);
  switch (a.d_m) {
    case 32: router_tail_kernel<W, 32><<<grid, block, 0, s>>>(a); break;
    case 64: router_tail_kernel<W, 64><<<grid, block, 0, s>>>(a); break;
    case 128: router_tail_kernel<W, 128><<<grid, block, 0, s>>>(a); break;
    case 256: router_tail_kernel<W, 256><<<grid, block, 0, s>>>(a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace

hipError_t launch_router_tail(const RouterTailArgs& a, hipStream_t s) {
  if (a.T <= 0) return hipSuccess;
  return a.dtype == 1 ? launch_dm<bf16_t>(a, s) : launch_dm<float>(a, s);
}

}  // namespace hero
