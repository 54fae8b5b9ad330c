// Router of one routed layer after the two large projections (Sec. 3.2), as three kernels:
//
//   router_pre   (8 tokens per workgroup, reuses each weight across them)
//     z^h = W_hu SiLU(inv_rms * W_hd hbar)                       hidden encoder (unit-gain RMSNorm)
//     x^path = [j/L_R, (L_R-j)/L_R, |delta_j|, gamma_j, p_{j-1}, m_{j-1}]   (eq:path_vector,
//                                                                 eq:transition_features)
//     z^a = W_p2 SiLU(W_p1 x^path),  s = [z^h; z^a]              (eq:router_state)
//     phi(q), phi(k), v, W_n s;  th1[:, :d_s] s (the s part of the history head's input layer)
//     b = ps2 . SiLU(psi_1 hbar)                                  local head (eq:final_gate)
//   router_mem   (one token per workgroup: a streaming read-modify-write of the memory)
//     c = phi(q)^T S / (phi(q)^T zeta + eps)                      (eq:memory_read, read first)
//     S <- rho S + phi(k) v^T,  zeta <- rho zeta + phi(k)          (eq:memory_update, same pass)
//   router_post  (8 tokens per workgroup)
//     nu = 1 - cos(W_n s, W_c c)  (0 at j = 1)
//     a = th2 . SiLU(th1 [s; c; nu]),  p = sigma(a / T_hist),  m = m_{j-1} p
//     logit = a + b (+ bias),  g = sigma(logit)
// At j = 1 the incoming state is the paper's initial value: S and zeta are not read
// (taken as zero) and p_0 = m_0 = 1.
// Router ablations (Table 3): without the position state the first four path features are
// zero; without the auxiliary state z^a = 0; without the memory read (or the whole history
// branch) router_mem is not launched, c = 0 and nu = 0 at every layer; without the history
// branch a = 0, so logit = b (+ bias), and p = m = 1 are written.
// The memory kernel moves 2 * 4 * (d_m^2 + d_m) bytes of state per token (2 * (2 d_m^2 + 4 d_m)
// with S stored in bf16) and is the HBM-bound part; keeping it free of the matrix-vector work lets many workgroups per
// CU keep HBM busy.  All arithmetic is fp32.
#include <algorithm>

#include "hero_device.h"
#include "hero_kernels.h"

namespace hero {
namespace {

constexpr int TB = 16;    // tokens per workgroup (pre / post)
constexpr int NT = 256;   // threads per workgroup
constexpr int MAXE = 256; // max(d_e, d_head)
constexpr int KC = 32;    // weight columns staged per step of block_matmul
constexpr int MAXS = 128; // max d_s
constexpr int MAXP = 128; // max d_p
constexpr int MAXM = 256; // max d_m

struct Ident {
  __device__ __forceinline__ float operator()(float x) const { return x; }
};
struct SiLU {
  __device__ __forceinline__ float operator()(float x) const { return siluf_(x); }
};
struct Phi {
  __device__ __forceinline__ float operator()(float x) const { return phif_(x); }
};

// out[t*os + o] = act(sum_i W[o*ldw + i] * in[t*is + i]) for o < O and tokens t < nvalid.
// P lanes share one output row (power of two, within a wave) and reduce by shuffles;
// each lane takes 8 consecutive inputs per step, loaded as one 16-byte vector when
// the row pitch allows it and as 8 independent loads otherwise.
template <typename W, class Act>
__device__ __forceinline__ void matvec(const W* __restrict__ w, int ldw, int O, int I,
                                       const float* in, int is, float* out, int os, Act act,
                                       int nvalid = TB) {
  int P = 64;
  while (P > 1 && P * O > NT) P >>= 1;
  while (P > 1 && 8 * (P >> 1) >= I) P >>= 1;   // no lane without work
  const int rows_per_pass = NT / P;
  const int slice = threadIdx.x % P;
  const bool vec = (ldw % 8 == 0) && ((reinterpret_cast<uintptr_t>(w) & 15) == 0);
  for (int o0 = 0; o0 < O; o0 += rows_per_pass) {
    const int o = o0 + static_cast<int>(threadIdx.x) / P;
    float acc[TB];
#pragma unroll
    for (int t = 0; t < TB; ++t) acc[t] = 0.f;
    if (o < O) {
      const W* wr = w + static_cast<size_t>(o) * ldw;
      for (int i = 8 * slice; i < I; i += 8 * P) {
        float wv[8];
        if (vec && i + 8 <= I) {
          ld8(wr + i, wv);
        } else {
#pragma unroll
          for (int e = 0; e < 8; ++e) wv[e] = (i + e < I) ? ldf(wr + i + e) : 0.f;
        }
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          if (i + e < I) {
#pragma unroll
            for (int t = 0; t < TB; ++t) acc[t] = fmaf(wv[e], in[t * is + i + e], acc[t]);
          }
        }
      }
    }
    for (int off = P >> 1; off > 0; off >>= 1)
#pragma unroll
      for (int t = 0; t < TB; ++t) acc[t] += __shfl_xor(acc[t], off, kWave);
    if (o < O && slice == 0)
#pragma unroll
      for (int t = 0; t < TB; ++t)
        if (t < nvalid) out[t * os + o] = act(acc[t]);
  }
}

// out[t*os + o] = act(bias[t*bs + o] + sum_i W[o*ldw + i] * X[t*ldx + i]) for o < O (<= 256) and
// tokens t < nvalid, all TB tokens computed.  Weight columns are staged KC at a time into LDS,
// transposed to [k][o] and converted to fp32, with loads that are contiguous along each
// row; each thread then accumulates a tile of RO rows x 4 tokens, reading one RO-wide weight
// vector and four broadcast inputs per k.
template <int RO, typename W, class Act>
__device__ __forceinline__ void block_matmul_ro(const W* __restrict__ w, int ldw, int O, int I,
                                                const float* X, int ldx, const float* bias, int bs,
                                                float* out, int os, Act act, float* wst, int nvalid) {
  constexpr int OPAD = 4 * 64 + 4;   // staged row pitch (floats)
  const int tid = threadIdx.x;
  const int og = tid >> 2, tg = tid & 3;   // rows og*RO.., tokens 4*tg..
  float acc[RO][4];
#pragma unroll
  for (int r = 0; r < RO; ++r)
#pragma unroll
    for (int q = 0; q < 4; ++q) acc[r][q] = 0.f;
  constexpr int U = 4 * 64 * KC / NT;   // staged elements per thread (rows <= 256)
  for (int i0 = 0; i0 < I; i0 += KC) {
    // all of this thread's loads are issued before any is used
    float tmp[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int e = tid + NT * u;
      const int o = e / KC, k = e % KC;
      tmp[u] = (o < O && i0 + k < I) ? ldf(w + static_cast<size_t>(o) * ldw + i0 + k) : 0.f;
    }
    __syncthreads();
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int e = tid + NT * u;
      const int o = e / KC, k = e % KC;
      if (o < O) wst[k * OPAD + o] = tmp[u];
    }
    __syncthreads();
    if (og * RO < O) {
      const int kn = min(KC, I - i0);
      for (int k = 0; k < kn; ++k) {
        float wv[RO];
#pragma unroll
        for (int r = 0; r < RO; ++r) wv[r] = wst[k * OPAD + og * RO + r];
        float xv[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) xv[q] = X[(4 * tg + q) * ldx + i0 + k];
#pragma unroll
        for (int r = 0; r < RO; ++r)
#pragma unroll
          for (int q = 0; q < 4; ++q) acc[r][q] = fmaf(wv[r], xv[q], acc[r][q]);
      }
    }
  }
  if (og * RO < O) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int t = 4 * tg + q;
      if (t >= nvalid) continue;
#pragma unroll
      for (int r = 0; r < RO; ++r) {
        const int o = og * RO + r;
        if (o < O) out[t * os + o] = act(acc[r][q] + (bias ? bias[t * bs + o] : 0.f));
      }
    }
  }
}

template <typename W, class Act>
__device__ __forceinline__ void block_matmul(const W* w, int ldw, int O, int I, const float* X, int ldx,
                                             const float* bias, int bs, float* out, int os, Act act,
                                             float* wst, int nvalid = TB) {
  if (O > 128)
    block_matmul_ro<4>(w, ldw, O, I, X, ldx, bias, bs, out, os, act, wst, nvalid);
  else if (O > 64)
    block_matmul_ro<2>(w, ldw, O, I, X, ldx, bias, bs, out, os, act, wst, nvalid);
  else
    block_matmul_ro<1>(w, ldw, O, I, X, ldx, bias, bs, out, os, act, wst, nvalid);
  __syncthreads();
}

// for (e = tid; e < n; e += NT) f(e, src(e)), with eight loads in flight per thread
template <class Src, class F>
__device__ __forceinline__ void batched(int n, Src src, F f) {
  for (int e0 = threadIdx.x; e0 < n; e0 += 8 * NT) {
    float v[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int e = e0 + NT * u;
      v[u] = e < n ? src(e) : 0.f;
    }
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int e = e0 + NT * u;
      if (e < n) f(e, v[u]);
    }
  }
}

#define LDS16 __shared__ __attribute__((aligned(16)))

// ---------------------------------------------------------------------------
// router_pre
// ---------------------------------------------------------------------------
template <typename W>
__global__ __launch_bounds__(NT) void router_pre_kernel(RouterTailArgs a) {
  constexpr int EP = MAXE + 4;
  LDS16 float bufA[TB][EP];     // SiLU(inv_rms W_hd hbar)
  LDS16 float bufB[TB][EP];     // SiLU(psi_1 hbar)
  LDS16 float s[TB][MAXS + 4];  // router state
  LDS16 float xp[TB][8];        // path vector
  LDS16 float zp[TB][MAXP];     // path-encoder hidden
  LDS16 float wst[KC * (4 * 64 + 4)];
  LDS16 float sc[TB];

  const int tid = threadIdx.x;
  const int t0 = blockIdx.x * TB;
  const int nvalid = min(TB, a.T - t0);
  const int j = a.j;
  const int d_e = a.d_e, d_head = a.d_head, NP = a.d_e + a.d_head, DM = a.d_m;

  if (tid < TB) {
    const int t = t0 + tid;
    float inv_rms = 0.f, dd = 0.f, dp = 0.f, pp = 0.f, pprev = 1.f, mprev = 1.f;
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
    }
    const float dj = j >= 2 ? sqrtf(dd) : 0.f;
    const float gam = j >= 3 ? dp / (dj * sqrtf(pp) + a.eps) : 0.f;
    const bool pos = !(a.abl & ABL_NO_POS);
    xp[tid][0] = pos ? static_cast<float>(j) / static_cast<float>(a.L_R) : 0.f;
    xp[tid][1] = pos ? static_cast<float>(a.L_R - j) / static_cast<float>(a.L_R) : 0.f;
    xp[tid][2] = pos ? dj : 0.f;
    xp[tid][3] = pos ? gam : 0.f;
    xp[tid][4] = pprev;
    xp[tid][5] = mprev;
    sc[tid] = inv_rms;
  }
  __syncthreads();
  batched(
      TB * NP,
      [&](int e) { return a.P[static_cast<size_t>(min(t0 + e / NP, a.T - 1)) * NP + e % NP]; },
      [&](int e, float pv) {
        const int tt = e / NP, i = e % NP;
        if (i < d_e)
          bufA[tt][i] = siluf_(sc[tt] * pv);
        else
          bufB[tt][i - d_e] = siluf_(pv);
      });
  __syncthreads();
  block_matmul(static_cast<const W*>(a.w_hu), d_e, a.d_h, d_e, &bufA[0][0], EP, nullptr, 0, &s[0][0],
               MAXS + 4, Ident(), wst);
  matvec(static_cast<const W*>(a.w_p1), 6, a.d_p, 6, &xp[0][0], 8, &zp[0][0], MAXP, SiLU());
  matvec(static_cast<const W*>(a.ps2), d_head, 1, d_head, &bufB[0][0], EP, a.bvec + t0, 1, Ident(),
         nvalid);
  __syncthreads();
  if (a.abl & ABL_NO_AUX) {
    for (int e = tid; e < TB * a.d_a; e += NT) s[e / a.d_a][a.d_h + e % a.d_a] = 0.f;
  } else {
    matvec(static_cast<const W*>(a.w_p2), a.d_p, a.d_a, a.d_p, &zp[0][0], MAXP, &s[0][a.d_h], MAXS + 4,
           Ident());
  }
  __syncthreads();
  const int d_s = a.d_s;
  float* qkvn = a.qkvn + static_cast<size_t>(t0) * 4 * DM;
  const float* S0 = &s[0][0];
  block_matmul(static_cast<const W*>(a.w_q), d_s, DM, d_s, S0, MAXS + 4, nullptr, 0, qkvn, 4 * DM, Phi(),
               wst, nvalid);
  block_matmul(static_cast<const W*>(a.w_k), d_s, DM, d_s, S0, MAXS + 4, nullptr, 0, qkvn + DM, 4 * DM,
               Phi(), wst, nvalid);
  block_matmul(static_cast<const W*>(a.w_v), d_s, DM, d_s, S0, MAXS + 4, nullptr, 0, qkvn + 2 * DM, 4 * DM,
               Ident(), wst, nvalid);
  block_matmul(static_cast<const W*>(a.w_n), d_s, DM, d_s, S0, MAXS + 4, nullptr, 0, qkvn + 3 * DM, 4 * DM,
               Ident(), wst, nvalid);
  // the s columns of the history head's input layer
  block_matmul(static_cast<const W*>(a.th1), a.ld_th1, d_head, d_s, S0, MAXS + 4, nullptr, 0,
               a.hs + static_cast<size_t>(t0) * d_head, d_head, Ident(), wst, nvalid);
}

// ---------------------------------------------------------------------------
// router_mem: one token per workgroup
// ---------------------------------------------------------------------------
// 16 bytes of the state as fp32 values: four fp32, or eight bf16
template <typename ST>
struct SVec {
  static constexpr int N = 16 / static_cast<int>(sizeof(ST));
  float v[N];
  __device__ __forceinline__ void load(const ST* p) {
    if constexpr (sizeof(ST) == 4) {
      const f32x4 x = *reinterpret_cast<const f32x4*>(p);
#pragma unroll
      for (int e = 0; e < 4; ++e) v[e] = x[e];
    } else {
      const u32x4 x = *reinterpret_cast<const u32x4*>(p);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        v[2 * e] = __uint_as_float(x[e] << 16);
        v[2 * e + 1] = __uint_as_float(x[e] & 0xffff0000u);
      }
    }
  }
  __device__ __forceinline__ void store(ST* p) const {
    if constexpr (sizeof(ST) == 4) {
      f32x4 x;
#pragma unroll
      for (int e = 0; e < 4; ++e) x[e] = v[e];
      *reinterpret_cast<f32x4*>(p) = x;
    } else {
      u32x4 x;
#pragma unroll
      for (int e = 0; e < 4; ++e)
        x[e] = static_cast<uint32_t>(f32_to_bf16(v[2 * e])) |
               (static_cast<uint32_t>(f32_to_bf16(v[2 * e + 1])) << 16);
      *reinterpret_cast<u32x4*>(p) = x;
    }
  }
};

// ST: storage type of S (float, or bf16_t: every written element rounded to nearest even)
template <int DM, typename ST>
__global__ __launch_bounds__(NT) void router_mem_kernel(RouterTailArgs a) {
  constexpr int VE = SVec<ST>::N;  // state elements per 16-byte vector
  constexpr int CV = DM / VE;      // vectors per S row
  constexpr int RP = NT / CV;      // S rows per pass
  constexpr int NR = DM / RP;      // S rows per thread
  static_assert(NR >= 1 && NT % CV == 0, "state layout");
  LDS16 float fq[DM];
  LDS16 float fk[DM];
  LDS16 float vv[DM];
  LDS16 float red[RP][DM];
  __shared__ float sden;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int t = blockIdx.x;
  const int j = a.j;
  const float rho = 1.0f / (1.0f + expf(-a.eta));
  const float* q = a.qkvn + static_cast<size_t>(t) * 4 * DM;
  for (int i = tid; i < 3 * DM; i += NT) {
    const float x = q[i];
    if (i < DM)
      fq[i] = x;
    else if (i < 2 * DM)
      fk[i - DM] = x;
    else
      vv[i - 2 * DM] = x;
  }
  __syncthreads();
  if (wave == 0) {
    float part = 0.f;
    float* z = a.zeta + static_cast<size_t>(t) * DM;
    for (int k = lane; k < DM; k += 64) {
      const float zv = j > 1 ? z[k] : 0.f;
      part = fmaf(fq[k], zv, part);
      z[k] = fmaf(rho, zv, fk[k]);
    }
    part = wave_sum(part);
    if (lane == 0) sden = part;
  }
  const int cq = tid % CV, rg = tid / CV;
  ST* Sp = static_cast<ST*>(a.S) + static_cast<size_t>(t) * DM * DM + VE * cq;
  float vr[VE], cacc[VE];
#pragma unroll
  for (int e = 0; e < VE; ++e) {
    vr[e] = vv[VE * cq + e];
    cacc[e] = 0.f;
  }
  if (j == 1) {
#pragma unroll 16
    for (int i = 0; i < NR; ++i) {
      const int r = rg + RP * i;
      SVec<ST> o;
#pragma unroll
      for (int e = 0; e < VE; ++e) o.v[e] = fk[r] * vr[e];
      o.store(Sp + r * DM);
    }
  } else {
    constexpr int CH = NR < 16 ? NR : 16;
    for (int i0 = 0; i0 < NR; i0 += CH) {
      SVec<ST> sv[CH];
#pragma unroll
      for (int c = 0; c < CH; ++c) sv[c].load(Sp + (rg + RP * (i0 + c)) * DM);
#pragma unroll
      for (int c = 0; c < CH; ++c) {
        const int r = rg + RP * (i0 + c);
        const float qv = fq[r], kv = fk[r];
        SVec<ST> o;
#pragma unroll
        for (int e = 0; e < VE; ++e) {
          cacc[e] = fmaf(qv, sv[c].v[e], cacc[e]);
          o.v[e] = fmaf(rho, sv[c].v[e], kv * vr[e]);
        }
        o.store(Sp + r * DM);
      }
    }
  }
#pragma unroll
  for (int e = 0; e < VE; ++e) red[rg][VE * cq + e] = cacc[e];
  __syncthreads();
  if (tid < DM) {
    float cs = 0.f;
    for (int g = 0; g < RP; ++g) cs += red[g][tid];
    a.cvec[static_cast<size_t>(t) * DM + tid] = j > 1 ? cs / (sden + a.eps) : 0.f;
  }
}

// ---------------------------------------------------------------------------
// router_post
// ---------------------------------------------------------------------------
template <typename W>
__global__ __launch_bounds__(NT) void router_post_kernel(RouterTailArgs a) {
  constexpr int CX = MAXM + 4;
  constexpr int HP = MAXE + 4;
  LDS16 float cx[TB][CX];         // [c; nu]
  LDS16 float ns[TB][MAXM];       // W_n s
  LDS16 float wc[TB][MAXM];       // W_c c
  LDS16 float hh[TB][HP];         // s part of the f_theta pre-activation, then its hidden
  LDS16 float wst[KC * (4 * 64 + 4)];
  LDS16 float sc[TB];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int t0 = blockIdx.x * TB;
  const int nvalid = min(TB, a.T - t0);
  const int j = a.j;
  const int DM = a.d_m, d_head = a.d_head, d_s = a.d_s;
  auto tok = [&](int tt) { return static_cast<size_t>(min(t0 + tt, a.T - 1)); };
  // a memory context exists after the first layer unless an ablation removes the memory
  const bool ctx = j > 1 && !(a.abl & (ABL_NO_MEMREAD | ABL_NO_HISTORY));
  batched(
      TB * DM, [&](int e) { return ctx ? a.cvec[tok(e / DM) * DM + e % DM] : 0.f; },
      [&](int e, float v) { cx[e / DM][e % DM] = v; });
  batched(
      TB * DM, [&](int e) { return a.qkvn[tok(e / DM) * 4 * DM + 3 * DM + e % DM]; },
      [&](int e, float v) { ns[e / DM][e % DM] = v; });
  batched(
      TB * d_head, [&](int e) { return a.hs[tok(e / d_head) * d_head + e % d_head]; },
      [&](int e, float v) { hh[e / d_head][e % d_head] = v; });
  __syncthreads();
  block_matmul(static_cast<const W*>(a.w_c), DM, DM, DM, &cx[0][0], CX, nullptr, 0, &wc[0][0], MAXM,
               Ident(), wst);
  for (int tt = wave; tt < TB; tt += NT / 64) {
    float nn = 0.f, cc = 0.f, nc = 0.f;
    for (int k = lane; k < DM; k += 64) {
      const float n = ns[tt][k], c = wc[tt][k];
      nn = fmaf(n, n, nn);
      cc = fmaf(c, c, cc);
      nc = fmaf(n, c, nc);
    }
    nn = wave_sum(nn);
    cc = wave_sum(cc);
    nc = wave_sum(nc);
    if (lane == 0) cx[tt][DM] = ctx ? 1.0f - nc / (sqrtf(nn) * sqrtf(cc) + a.eps) : 0.f;
  }
  __syncthreads();
  // the [c; nu] columns of the history head's input layer on top of its s part, then SiLU
  block_matmul(static_cast<const W*>(a.th1) + d_s, a.ld_th1, d_head, DM + 1, &cx[0][0], CX, &hh[0][0], HP,
               &hh[0][0], HP, SiLU(), wst);
  matvec(static_cast<const W*>(a.th2), d_head, 1, d_head, &hh[0][0], HP, &sc[0], 1, Ident());
  __syncthreads();
  if (tid < nvalid) {
    const int t = t0 + tid;
    const bool hist = !(a.abl & ABL_NO_HISTORY);
    const float av = hist ? sc[tid] : 0.f;
    const float mprev = j > 1 ? a.m_hist[t] : 1.0f;
    const float p = sigmoidf_(av / a.T_hist);
    a.p_hist[t] = hist ? p : 1.0f;
    a.m_hist[t] = hist ? mprev * p : 1.0f;
    const float l = av + a.bvec[t] + (a.beta ? a.beta[t] : 0.f);
    a.logit[t] = l;
    a.gate[t] = sigmoidf_(l);
  }
}


// ---------------------------------------------------------------------------
// bf16 weights: matrix cores.  Every product above is a contraction over a batch of
// tokens, run here on v_mfma_f32_16x16x32_bf16 with one 16-token row block per
// workgroup.  The fp32 activations are split as x = hi + lo into two bf16 values
// (|x - hi - lo| <= 2^-18 |x|) and the bf16 weights are exact, so each product
// hi*w and lo*w is exact in fp32 and only the fp32 accumulation rounds.
// A fragments live in LDS in MFMA order: entry [k-step s][lane], lane = i + 16 g,
// holds row i at k = 32 s + 8 g .. + 7.  B fragments are 16-byte loads of eight
// consecutive weights of one output row (L2-resident: every workgroup reads the
// same router weights).  Output lane i + 16 g holds rows 4 g .. 4 g + 3 of column i.
// ---------------------------------------------------------------------------
constexpr int MT = 16;            // tokens per workgroup
constexpr int MAXSPLIT = 4;       // K-slice partials of P
constexpr int KS_E = MAXE / 32;   // k-steps over d_e
constexpr int KS_S = MAXS / 32;   // k-steps over d_s
constexpr int KS_M = MAXM / 32;   // k-steps over d_m

__device__ __forceinline__ void split8(const float* x, bf16x8& hi, bf16x8& lo) {
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const __bf16 h = static_cast<__bf16>(x[e]);
    hi[e] = h;
    lo[e] = static_cast<__bf16>(x[e] - static_cast<float>(h));
  }
}

__device__ __forceinline__ f32x4 mfma_split(const bf16x8& ahi, const bf16x8& alo, const bf16x8& b,
                                            f32x4 acc) {
  acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ahi, b, acc, 0, 0, 0);
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(alo, b, acc, 0, 0, 0);
}

// Weights w[r][k0 + 8 g .. + 7] of row r = r0 + (lane & 15), g = lane >> 4, of a [nrows][ld]
// matrix (ld % 8 == 0, 16-byte aligned base); zero past nrows or past kmax (kmax % 8 == 0).
__device__ __forceinline__ bf16x8 bfrag(const bf16_t* __restrict__ w, int ld, int nrows, int r0,
                                        int k0, int kmax, int lane) {
  const int r = r0 + (lane & 15), k = k0 + 8 * (lane >> 4);
  u32x4 v = {0u, 0u, 0u, 0u};
  if (r < nrows && k < kmax) v = *reinterpret_cast<const u32x4*>(w + static_cast<size_t>(r) * ld + k);
  return __builtin_bit_cast(bf16x8, v);
}

// One 16-column output tile of the s-projections: which matrix, its row offset, destination.
struct SProj {
  const bf16_t* w;
  int ld, nrows, r0, os;
  float* out;
  bool phi;
};

// router_pre on 8 waves (16 tokens per workgroup).  Every global load of the kernel is issued
// first: the P partials, the hidden encoder's and the s-projections' weight fragments (up to
// PF2 output tiles per wave), the local head's weights and the path-vector inputs; what follows
// works from registers and LDS between four barriers.
constexpr int NTP = 512;
constexpr unsigned kCUsRouter = 256;   // compute units of an MI355X
constexpr int NWP = NTP / kWave;
constexpr int PF2 = 6;

// KSS: k-steps over d_s (ceil(d_s / 32)).  WPE: waves per SIMD the kernel is compiled for (2: one
// workgroup per CU with every weight fragment loaded up front, for launches of about one round of
// workgroups; 4: two workgroups per CU, each hiding the other's latencies, for many rounds)
// NSPL: the most K-slice partials of P the launch may have (p_splits <= NSPL); PF: output tiles
// of the s-projections per wave whose weight fragments are loaded up front
template <int KSS, int WPE = 2, int NSPL = MAXSPLIT, int PF = PF2>
__global__ __launch_bounds__(NTP, WPE) void router_pre_mfma(RouterTailArgs a) {
  LDS16 bf16x8 ax[2][KS_E][kWave];   // SiLU(inv_rms W_hd hbar): hi, lo
  LDS16 bf16x8 as[2][KS_S][kWave];   // s: hi, lo
  LDS16 float s[MT][MAXS + 4];
  LDS16 float hp[MT][MAXP + 1];      // path-encoder hidden
  __shared__ float xp[MT][8];
  __shared__ float sc[MT];
  __shared__ float bpart[MT][16];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int t0 = blockIdx.x * MT;
  // column groups (few tokens): workgroup y of CS takes the output tiles ct = y + CS i of the
  // s-projections; every group forms s itself
  const int cs = blockIdx.y, CS = gridDim.y;
  const int nvalid = min(MT, a.T - t0);
  const int j = a.j;
  const int d_e = a.d_e, d_head = a.d_head, NP = d_e + d_head, DM = a.d_m, d_s = a.d_s;
  const int d_h = a.d_h, d_a = a.d_a, d_p = a.d_p;
  const int nq = DM / 16, nct = 4 * nq + d_head / 16;
  auto proj = [&](int ct) {
    const int m = ct / nq;
    if (m < 4) {
      const void* ws[4] = {a.w_q, a.w_k, a.w_v, a.w_n};
      return SProj{static_cast<const bf16_t*>(ws[m]), d_s, DM, 16 * (ct - m * nq), 4 * DM, a.qkvn + m * DM,
                   m < 2};
    }
    return SProj{static_cast<const bf16_t*>(a.th1), a.ld_th1, d_head, 16 * (ct - 4 * nq), d_head, a.hs, false};
  };

  // (1) P: token tt, columns [16 pc, 16 pc + 16) (NP <= 512), the K-slice partials
  const int tt = tid >> 5, pc = tid & 31;
  const bool has_p = 16 * pc < NP;
  const bool head = has_p && 16 * pc >= d_e;
  f32x4 pz[NSPL][4];
  if (has_p) {
    const float* src = a.P + static_cast<size_t>(min(t0 + tt, a.T - 1)) * NP + 16 * pc;
    const size_t zs = static_cast<size_t>(a.T) * NP;
#pragma unroll
    for (int z = 0; z < NSPL; ++z)
#pragma unroll
      for (int q = 0; q < 4; ++q)
        pz[z][q] = *reinterpret_cast<const f32x4*>(src + (z < a.p_splits ? z : 0) * zs + 4 * q);
  }
  // (2) the local head's output weights for head columns
  u32x4 wps2[2] = {{0u, 0u, 0u, 0u}, {0u, 0u, 0u, 0u}};
  if (head) {
    const bf16_t* w = static_cast<const bf16_t*>(a.ps2) + 16 * pc - d_e;
    wps2[0] = *reinterpret_cast<const u32x4*>(w);
    wps2[1] = *reinterpret_cast<const u32x4*>(w + 8);
  }
  // (3) hidden encoder: wave w computes z_h columns [16 w, 16 w + 16)
  const int ks1 = d_e / 32;
  const bool st1 = 16 * wave < d_h;
  bf16x8 b1[KS_E];
  if (st1) {
#pragma unroll
    for (int st = 0; st < KS_E; ++st)
      if (st < ks1) b1[st] = bfrag(static_cast<const bf16_t*>(a.w_hu), d_e, d_h, 16 * wave, 32 * st, d_e, lane);
  }
  // (4) s-projections: this wave's first PF output tiles ct = wave + NWP c
  bf16x8 b2[PF][KSS];
#pragma unroll
  for (int c = 0; c < PF; ++c) {
    const int ct = cs + CS * (wave + NWP * c);
    if (ct < nct) {
      const SProj p = proj(ct);
#pragma unroll
      for (int st = 0; st < KSS; ++st) b2[c][st] = bfrag(p.w, p.ld, p.nrows, p.r0, 32 * st, d_s, lane);
    }
  }
  // (5) path vector
  if (tid < MT) {
    const int t = t0 + tid;
    float inv_rms = 0.f, dd = 0.f, dp = 0.f, pp = 0.f, pprev = 1.f, mprev = 1.f;
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
    }
    const float dj = j >= 2 ? sqrtf(dd) : 0.f;
    const float gam = j >= 3 ? dp / (dj * sqrtf(pp) + a.eps) : 0.f;
    const bool pos = !(a.abl & ABL_NO_POS);
    xp[tid][0] = pos ? static_cast<float>(j) / static_cast<float>(a.L_R) : 0.f;
    xp[tid][1] = pos ? static_cast<float>(a.L_R - j) / static_cast<float>(a.L_R) : 0.f;
    xp[tid][2] = pos ? dj : 0.f;
    xp[tid][3] = pos ? gam : 0.f;
    xp[tid][4] = pprev;
    xp[tid][5] = mprev;
    sc[tid] = inv_rms;
  }
  __syncthreads();

  // hidden-encoder A fragments (columns k = 16 pc + e: k-step pc/2, groups 2 (pc&1), +1),
  // local-head partial dot products, path-encoder hidden layer
  if (has_p) {
    float x[16];
#pragma unroll
    for (int q = 0; q < 4; ++q)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        float v = pz[0][q][e];
#pragma unroll
        for (int z = 1; z < NSPL; ++z)
          if (z < a.p_splits) v += pz[z][q][e];
        x[4 * q + e] = v;
      }
    if (!head) {
      const float ir = sc[tt];
#pragma unroll
      for (int e = 0; e < 16; ++e) x[e] = siluf_(ir * x[e]);
      const int st = pc >> 1, g0 = 2 * (pc & 1);
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        bf16x8 hi, lo;
        split8(x + 8 * h, hi, lo);
        ax[0][st][tt + 16 * (g0 + h)] = hi;
        ax[1][st][tt + 16 * (g0 + h)] = lo;
      }
    } else {
      float acc = 0.f;
#pragma unroll
      for (int h = 0; h < 2; ++h)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const uint32_t w = wps2[h][i];
          acc = fmaf(__uint_as_float(w << 16), siluf_(x[8 * h + 2 * i]), acc);
          acc = fmaf(__uint_as_float(w & 0xffff0000u), siluf_(x[8 * h + 2 * i + 1]), acc);
        }
      bpart[tt][pc - d_e / 16] = acc;
    }
  }
  {
    const bf16_t* w1 = static_cast<const bf16_t*>(a.w_p1);
    for (int e = tid; e < MT * d_p; e += NTP) {
      const int t = e / d_p, o = e % d_p;
      float acc = 0.f;
#pragma unroll
      for (int k = 0; k < 6; ++k) acc = fmaf(ldf(w1 + o * 6 + k), xp[t][k], acc);
      hp[t][o] = siluf_(acc);
    }
  }
  __syncthreads();

  // z_h = W_hu x on matrix cores, z_a = W_p2 hp
  if (st1) {
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int st = 0; st < KS_E; ++st)
      if (st < ks1) acc = mfma_split(ax[0][st][lane], ax[1][st][lane], b1[st], acc);
    const int o = 16 * wave + (lane & 15);
    if (o < d_h)
#pragma unroll
      for (int r = 0; r < 4; ++r) s[4 * (lane >> 4) + r][o] = acc[r];
  }
  {
    const bf16_t* w2 = static_cast<const bf16_t*>(a.w_p2);
    for (int e = tid; e < MT * d_a; e += NTP) {
      const int t = e / d_a, o = e % d_a;
      float acc = 0.f;
      if (!(a.abl & ABL_NO_AUX))
        for (int k = 0; k < d_p; ++k) acc = fmaf(ldf(w2 + o * d_p + k), hp[t][k], acc);
      s[t][d_h + o] = acc;
    }
  }
  __syncthreads();

  // s as A fragments (zero past d_s); the local-head logit b
  for (int e = tid; e < MT * 4 * KSS; e += NTP) {
    const int i = e & 15, g = (e >> 4) & 3, st = e >> 6;
    const int k0 = 32 * st + 8 * g;
    float x[8];
#pragma unroll
    for (int q = 0; q < 8; ++q) x[q] = k0 + q < d_s ? s[i][k0 + q] : 0.f;
    split8(x, as[0][st][i + 16 * g], as[1][st][i + 16 * g]);
  }
  if (tid < nvalid && cs == 0) {
    float b = 0.f;
    for (int q = 0; q < d_head / 16; ++q) b += bpart[tid][q];
    a.bvec[t0 + tid] = b;
  }
  __syncthreads();

  // [phi(q); phi(k); v; W_n s; th1[:, :d_s] s]
  auto finish = [&](int ct, const bf16x8* bw) {
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int st = 0; st < KSS; ++st) acc = mfma_split(as[0][st][lane], as[1][st][lane], bw[st], acc);
    const SProj p = proj(ct);
    const int o = p.r0 + (lane & 15);
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int t = t0 + 4 * (lane >> 4) + r;
      if (t < a.T) p.out[static_cast<size_t>(t) * p.os + o] = p.phi ? phif_(acc[r]) : acc[r];
    }
  };
#pragma unroll
  for (int c = 0; c < PF; ++c)
    if (cs + CS * (wave + NWP * c) < nct) finish(cs + CS * (wave + NWP * c), b2[c]);
  for (int ct = cs + CS * (wave + NWP * PF); ct < nct; ct += CS * NWP) {
    const SProj p = proj(ct);
    bf16x8 bw[KSS];
#pragma unroll
    for (int st = 0; st < KSS; ++st) bw[st] = bfrag(p.w, p.ld, p.nrows, p.r0, 32 * st, d_s, lane);
    finish(ct, bw);
  }
}

// router_post on 8 waves (16 tokens per workgroup), every global load issued first:
// c (as split A fragments), W_n s, the s part of f_theta's first layer, and the weight
// fragments of W_c and of f_theta's c columns for this wave's output tiles.
template <int KSM>   // k-steps over d_m (d_m / 32)
__global__ __launch_bounds__(NTP) void router_post_mfma(RouterTailArgs a) {
  constexpr int DM = 32 * KSM;
  constexpr int TWC = (DM / 16 + NWP - 1) / NWP;      // W_c output tiles per wave
  constexpr int TWH = (MAXE / 16 + NWP - 1) / NWP;    // f_theta output tiles per wave (d_head <= 256)
  LDS16 bf16x8 ac[2][KSM][kWave];   // c: hi, lo
  LDS16 float ns[MT][DM + 4];       // W_n s
  LDS16 float wc[MT][DM + 4];       // W_c c
  __shared__ float nu[MT];
  __shared__ float apart[NWP][MT];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int t0 = blockIdx.x * MT;
  const int nvalid = min(MT, a.T - t0);
  const int j = a.j;
  const int d_head = a.d_head, d_s = a.d_s;
  const int g4 = 4 * (lane >> 4);
  auto tok = [&](int i) { return static_cast<size_t>(min(t0 + i, a.T - 1)); };
  const bf16_t* th1 = static_cast<const bf16_t*>(a.th1);
  const bf16_t* th2 = static_cast<const bf16_t*>(a.th2);
  const bf16_t* w_c = static_cast<const bf16_t*>(a.w_c);
  const int ld = a.ld_th1, nct_h = d_head / 16;

  // a memory context exists after the first layer unless an ablation removes the memory
  const bool ctx = j > 1 && !(a.abl & (ABL_NO_MEMREAD | ABL_NO_HISTORY));
  // c rows as split fragments, and W_n s
  for (int e = tid; e < MT * 4 * KSM; e += NTP) {
    const int i = e & 15, g = (e >> 4) & 3, st = e >> 6;
    const float* src = a.cvec + tok(i) * DM + 32 * st + 8 * g;
    const f32x4 zero = {0.f, 0.f, 0.f, 0.f};
    const f32x4 lo4 = ctx ? *reinterpret_cast<const f32x4*>(src) : zero;
    const f32x4 hi4 = ctx ? *reinterpret_cast<const f32x4*>(src + 4) : zero;
    float x[8];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      x[q] = lo4[q];
      x[4 + q] = hi4[q];
    }
    split8(x, ac[0][st][i + 16 * g], ac[1][st][i + 16 * g]);
  }
  for (int e = tid; e < MT * DM / 4; e += NTP) {
    const int i = e / (DM / 4), c4 = e % (DM / 4);
    *reinterpret_cast<f32x4*>(&ns[i][4 * c4]) =
        *reinterpret_cast<const f32x4*>(a.qkvn + tok(i) * 4 * DM + 3 * DM + 4 * c4);
  }
  // weight fragments of this wave's tiles, the s part of the pre-activation, nu and th2 weights
  bf16x8 bc[TWC][KSM], bh[TWH][KSM];
  float hsv[TWH][4], wnu[TWH], w2[TWH];
#pragma unroll
  for (int c = 0; c < TWC; ++c) {
    const int ct = wave + NWP * c;
    if (16 * ct < DM)
#pragma unroll
      for (int st = 0; st < KSM; ++st) bc[c][st] = bfrag(w_c, DM, DM, 16 * ct, 32 * st, DM, lane);
  }
#pragma unroll
  for (int c = 0; c < TWH; ++c) {
    const int ct = wave + NWP * c;
    if (ct < nct_h) {
      const int o = 16 * ct + (lane & 15);
#pragma unroll
      for (int st = 0; st < KSM; ++st) bh[c][st] = bfrag(th1 + d_s, ld, d_head, 16 * ct, 32 * st, DM, lane);
#pragma unroll
      for (int r = 0; r < 4; ++r) hsv[c][r] = a.hs[tok(g4 + r) * d_head + o];
      wnu[c] = bf16_to_f32(th1[static_cast<size_t>(o) * ld + d_s + DM]);
      w2[c] = bf16_to_f32(th2[o]);
    }
  }
  __syncthreads();

  // W_c c
#pragma unroll
  for (int c = 0; c < TWC; ++c) {
    const int ct = wave + NWP * c;
    if (16 * ct < DM) {
      f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int st = 0; st < KSM; ++st) acc = mfma_split(ac[0][st][lane], ac[1][st][lane], bc[c][st], acc);
      const int o = 16 * ct + (lane & 15);
#pragma unroll
      for (int r = 0; r < 4; ++r) wc[g4 + r][o] = acc[r];
    }
  }
  __syncthreads();

  // nu = 1 - cos(W_n s, W_c c); 0 at j = 1
  for (int i = wave; i < MT; i += NWP) {
    float nn = 0.f, cc = 0.f, nc = 0.f;
    for (int k = lane; k < DM; k += kWave) {
      const float n = ns[i][k], c = wc[i][k];
      nn = fmaf(n, n, nn);
      cc = fmaf(c, c, cc);
      nc = fmaf(n, c, nc);
    }
    nn = wave_sum(nn);
    cc = wave_sum(cc);
    nc = wave_sum(nc);
    if (lane == 0) nu[i] = ctx ? 1.0f - nc / (sqrtf(nn) * sqrtf(cc) + a.eps) : 0.f;
  }
  __syncthreads();

  // a = th2 . SiLU(th1 [s; c; nu])
  float ap[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int c = 0; c < TWH; ++c) {
    const int ct = wave + NWP * c;
    if (ct < nct_h) {
      f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int st = 0; st < KSM; ++st) acc = mfma_split(ac[0][st][lane], ac[1][st][lane], bh[c][st], acc);
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const float pre = acc[r] + hsv[c][r] + wnu[c] * nu[g4 + r];
        ap[r] = fmaf(w2[c], siluf_(pre), ap[r]);
      }
    }
  }
#pragma unroll
  for (int r = 0; r < 4; ++r)
#pragma unroll
    for (int off = 1; off < 16; off <<= 1) ap[r] += __shfl_xor(ap[r], off, kWave);
  if ((lane & 15) == 0)
#pragma unroll
    for (int r = 0; r < 4; ++r) apart[wave][g4 + r] = ap[r];
  __syncthreads();
  if (tid < nvalid) {
    const int t = t0 + tid;
    const bool hist = !(a.abl & ABL_NO_HISTORY);
    float av = 0.f;
#pragma unroll
    for (int w = 0; w < NWP; ++w) av += apart[w][tid];
    if (!hist) av = 0.f;
    const float mprev = j > 1 ? a.m_hist[t] : 1.0f;
    const float p = sigmoidf_(av / a.T_hist);
    a.p_hist[t] = hist ? p : 1.0f;
    a.m_hist[t] = hist ? mprev * p : 1.0f;
    const float l = av + a.bvec[t] + (a.beta ? a.beta[t] : 0.f);
    a.logit[t] = l;
    a.gate[t] = sigmoidf_(l);
  }
}

// ---------------------------------------------------------------------------
// router_mem_hist: the memory read in depth-history form, one wave per token.
//   a_i = w_i phi(q) . phi(k_i),  c = sum_i a_i v_i / (sum_i a_i + eps)  over the stored
//   pairs i < j-1 (oldest first), then the layer's own (phi(k), v) stored as entry j-1.
// Each lane owns EPL consecutive elements of the d_m-vectors; the pairs are read in
// batches of HB with all of a batch's loads issued first.
// ---------------------------------------------------------------------------
template <int DM>
__global__ __launch_bounds__(NT) void router_mem_hist_kernel(RouterTailArgs a) {
  constexpr int EPL = DM >= kWave ? DM / kWave : 1;   // elements per lane
  constexpr int LANES = DM >= kWave ? kWave : DM;     // lanes holding elements
  constexpr int HB = 8;
  const int lane = threadIdx.x & 63;
  const int t = blockIdx.x * (NT / kWave) + (threadIdx.x >> 6);
  if (t >= a.T) return;
  const int n = a.j - 1;
  const bool on = lane < LANES;
  const int e0 = lane * EPL;
  const float* q = a.qkvn + static_cast<size_t>(t) * 4 * DM;
  float fq[EPL], fk[EPL], vv[EPL];
#pragma unroll
  for (int x = 0; x < EPL; ++x) {
    fq[x] = on ? q[e0 + x] : 0.f;
    fk[x] = on ? q[DM + e0 + x] : 0.f;
    vv[x] = on ? q[2 * DM + e0 + x] : 0.f;
  }
  float* H = a.kv + static_cast<size_t>(t) * a.L_R * 2 * DM;
  float c[EPL];
#pragma unroll
  for (int x = 0; x < EPL; ++x) c[x] = 0.f;
  float den = 0.f;
  for (int i0 = 0; i0 < n; i0 += HB) {
    float kk[HB][EPL], vh[HB][EPL];
#pragma unroll
    for (int u = 0; u < HB; ++u) {
      const int i = i0 + u;
      const float* hk = H + static_cast<size_t>(min(i, n - 1)) * 2 * DM + e0;
#pragma unroll
      for (int x = 0; x < EPL; ++x) {
        kk[u][x] = on ? hk[x] : 0.f;
        vh[u][x] = on ? hk[DM + x] : 0.f;
      }
    }
    float dots[HB];
#pragma unroll
    for (int u = 0; u < HB; ++u) {
      float s = 0.f;
#pragma unroll
      for (int x = 0; x < EPL; ++x) s = fmaf(fq[x], kk[u][x], s);
      dots[u] = wave_sum(s);
    }
#pragma unroll
    for (int u = 0; u < HB; ++u) {
      if (i0 + u < n) {
        const float al = a.hw[i0 + u] * dots[u];
        den += al;
#pragma unroll
        for (int x = 0; x < EPL; ++x) c[x] = fmaf(al, vh[u][x], c[x]);
      }
    }
  }
  if (on) {
    float* cv = a.cvec + static_cast<size_t>(t) * DM + e0;
    float* hn = H + static_cast<size_t>(n) * 2 * DM + e0;
#pragma unroll
    for (int x = 0; x < EPL; ++x) {
      cv[x] = n > 0 ? c[x] / (den + a.eps) : 0.f;
      hn[x] = fk[x];
      hn[DM + x] = vv[x];
    }
  }
}

// S[t][k][v] = sum_{i<n} w_i phi(k_i)[k] v_i[v], zeta[t][k] = sum_{i<n} w_i phi(k_i)[k];
// one workgroup per token, oldest pair first.
template <int DM>
__global__ __launch_bounds__(NT) void history_state_kernel(const float* __restrict__ kv, int L_R, int n,
                                                           HistWeights hw, float* __restrict__ S,
                                                           float* __restrict__ zeta) {
  const int t = blockIdx.x;
  const float* H = kv + static_cast<size_t>(t) * L_R * 2 * DM;
  float* St = S + static_cast<size_t>(t) * DM * DM;
  for (int e = threadIdx.x; e < DM * DM; e += NT) {
    const int k = e / DM, v = e % DM;
    float acc = 0.f;
    for (int i = 0; i < n; ++i) acc = fmaf(hw.w[i] * H[i * 2 * DM + k], H[i * 2 * DM + DM + v], acc);
    St[e] = acc;
  }
  for (int k = threadIdx.x; k < DM; k += NT) {
    float z = 0.f;
    for (int i = 0; i < n; ++i) z = fmaf(hw.w[i], H[i * 2 * DM + k], z);
    zeta[static_cast<size_t>(t) * DM + k] = z;
  }
}

#undef LDS16

hipError_t launch_pre_post(const RouterTailArgs& a, bool post, hipStream_t s) {
  if (a.dtype == 1) {
    dim3 grid((a.T + MT - 1) / MT);
    if (post) {
      switch (a.d_m) {
        case 32: router_post_mfma<1><<<grid, NTP, 0, s>>>(a); break;
        case 64: router_post_mfma<2><<<grid, NTP, 0, s>>>(a); break;
        case 128: router_post_mfma<4><<<grid, NTP, 0, s>>>(a); break;
        case 256: router_post_mfma<8><<<grid, NTP, 0, s>>>(a); break;
        default: return hipErrorInvalidValue;
      }
    } else {
      // many rounds of workgroups (more than two per CU) with an unsplit P: two resident
      // workgroups per CU, weight fragments loaded as they are needed
      const bool many = grid.x > 2u * kCUsRouter && a.p_splits == 1;
      // few token groups: the s-projections' output tiles split over up to 16 column groups per
      // token group, so that the launch covers the CUs (decode, 256 tokens: 16 x 16 workgroups)
      const int nct = 4 * (a.d_m / 16) + a.d_head / 16;
      grid.y = static_cast<unsigned>(std::max(1, std::min({16, static_cast<int>(kCUsRouter / grid.x), nct})));
      switch ((a.d_s + 31) / 32) {
        case 1: many ? router_pre_mfma<1, 4, 1, 1><<<grid, NTP, 0, s>>>(a) : router_pre_mfma<1><<<grid, NTP, 0, s>>>(a); break;
        case 2: many ? router_pre_mfma<2, 4, 1, 1><<<grid, NTP, 0, s>>>(a) : router_pre_mfma<2><<<grid, NTP, 0, s>>>(a); break;
        case 3: many ? router_pre_mfma<3, 4, 1, 1><<<grid, NTP, 0, s>>>(a) : router_pre_mfma<3><<<grid, NTP, 0, s>>>(a); break;
        case 4: many ? router_pre_mfma<4, 4, 1, 1><<<grid, NTP, 0, s>>>(a) : router_pre_mfma<4><<<grid, NTP, 0, s>>>(a); break;
        default: return hipErrorInvalidValue;
      }
    }
  } else {
    dim3 grid((a.T + TB - 1) / TB), block(NT);
    if (post)
      router_post_kernel<float><<<grid, block, 0, s>>>(a);
    else
      router_pre_kernel<float><<<grid, block, 0, s>>>(a);
  }
  return hipGetLastError();
}

}  // namespace

size_t router_scratch_floats(int d_m, int d_head, int T) {
  return static_cast<size_t>(T) * (4 * d_m + d_head + d_m + 1);
}

hipError_t launch_router_pre(const RouterTailArgs& a, hipStream_t s) {
  if (a.T <= 0) return hipSuccess;
  if (a.p_splits < 1 || a.p_splits > (a.dtype == 1 ? MAXSPLIT : 1)) return hipErrorInvalidValue;
  return launch_pre_post(a, false, s);
}

hipError_t launch_router_mem(const RouterTailArgs& a, hipStream_t s) {
  if (a.T <= 0) return hipSuccess;
  dim3 grid(a.T), block(NT);
  if (a.state_bf16) {
    switch (a.d_m) {
      case 64: router_mem_kernel<64, bf16_t><<<grid, block, 0, s>>>(a); break;
      case 128: router_mem_kernel<128, bf16_t><<<grid, block, 0, s>>>(a); break;
      case 256: router_mem_kernel<256, bf16_t><<<grid, block, 0, s>>>(a); break;
      default: return hipErrorInvalidValue;
    }
  } else {
    switch (a.d_m) {
      case 32: router_mem_kernel<32, float><<<grid, block, 0, s>>>(a); break;
      case 64: router_mem_kernel<64, float><<<grid, block, 0, s>>>(a); break;
      case 128: router_mem_kernel<128, float><<<grid, block, 0, s>>>(a); break;
      case 256: router_mem_kernel<256, float><<<grid, block, 0, s>>>(a); break;
      default: return hipErrorInvalidValue;
    }
  }
  return hipGetLastError();
}

hipError_t launch_router_mem_hist(const RouterTailArgs& a, hipStream_t s) {
  if (a.T <= 0) return hipSuccess;
  if (a.j < 1 || a.j > a.L_R || a.L_R > 64) return hipErrorInvalidValue;
  dim3 grid((a.T + NT / kWave - 1) / (NT / kWave)), block(NT);
  switch (a.d_m) {
    case 32: router_mem_hist_kernel<32><<<grid, block, 0, s>>>(a); break;
    case 64: router_mem_hist_kernel<64><<<grid, block, 0, s>>>(a); break;
    case 128: router_mem_hist_kernel<128><<<grid, block, 0, s>>>(a); break;
    case 256: router_mem_hist_kernel<256><<<grid, block, 0, s>>>(a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_history_state(int d_m, int L_R, int n, int T, const float* kv, const HistWeights& w,
                                float* S, float* zeta, hipStream_t s) {
  if (T <= 0) return hipSuccess;
  if (n < 0 || n > L_R || L_R > 64) return hipErrorInvalidValue;
  dim3 grid(T), block(NT);
  switch (d_m) {
    case 32: history_state_kernel<32><<<grid, block, 0, s>>>(kv, L_R, n, w, S, zeta); break;
    case 64: history_state_kernel<64><<<grid, block, 0, s>>>(kv, L_R, n, w, S, zeta); break;
    case 128: history_state_kernel<128><<<grid, block, 0, s>>>(kv, L_R, n, w, S, zeta); break;
    case 256: history_state_kernel<256><<<grid, block, 0, s>>>(kv, L_R, n, w, S, zeta); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_router_post(const RouterTailArgs& a, hipStream_t s) {
  if (a.T <= 0) return hipSuccess;
  return launch_pre_post(a, true, s);
}

}  // namespace hero
