// Backward of the router at one routed layer (Sec. 3.2 in reverse order): the gradient that
// reaches the router through the gate scaling (Sec. 3.1, the remark after eq:ffn_route) flows
// through the local head, the history head, the history dissimilarity, the memory read and
// write, the projections q, k, v, the router state, the path encoder and the hidden encoder.
//
// The token work (fp32 arithmetic; five passes, described where they are defined below):
//   forward recompute of the layer's router from P = hbar [W_hd; psi_1]^T (recomputed on the
//   GEMM core) and the state entering the layer; then the reverse:
//     dL/da = dL/dlogit + (dL/dp_j + dL/dm_j m_{j-1}) p (1 - p) / T_hist,  dL/db = dL/dlogit,
//     heads, nu (cosine backward), one streaming pass over S_{j-1} and the carried dL/dS_j that
//     forms dL/dphi(k), dL/dv, dL/dphi(q) and dL/drho and writes dL/dS_{j-1} in place,
//     projections, path encoder (dL/dp_{j-1}, dL/dm_{j-1}, and the transition features'
//     gradients as coefficients of delta_j, delta_{j-1}), hidden encoder;
//   writes the gradient over P ([ir dL/dpre_h; dL/dpre_b], row- and token-major), the per-row
//   coefficients of the RMSNorm and transition terms, and every (vector, token) pair the weight
//   gradients need, token-contiguous, so that each weight gradient is one product with the
//   tokens as K (run by the caller with a fixed summation order: small_products_kernel /
//   small_products_reduce below for the eleven small ones, the GEMM core with dP split into bf16 hi + lo
//   for dW_hd, dpsi_1 and dP [W_hd; psi_1]; tn_part / tn_reduce for those three in fp32 storage).
// router_bwd_rows: dL/dhbar_j += c_norm hbar_j + ddelta_j, dL/dhbar_{j-1} += ddelta_{j-1} -
//   ddelta_j, dL/dhbar_{j-2} -= ddelta_{j-1}, with ddelta_j = c1 delta_j + c2 delta_{j-1} and
//   ddelta_{j-1} = c3 delta_j + c4 delta_{j-1}.
// At j = 1 the state entering the layer is the initial one (S = 0, zeta = 0, p = m = 1) whatever
// the buffers hold; the carried gradient written there is rho dL/dS_1 (the state is a constant).
#include <algorithm>
#include <type_traits>

#include "hero_device.h"
#include "hero_kernels.h"

namespace hero {
namespace {

constexpr int RB_NT = 256;
constexpr int RB_NW = RB_NT / kWave;
constexpr int RB_MAXE = 256, RB_MAXH = 256, RB_MAXS = 128, RB_MAXM = 256, RB_MAXP = 128;
constexpr int RB_MAXX = RB_MAXS + RB_MAXM + 1;
constexpr int RB_MAXSPL = 4;                            // K-slice partials of P at most
constexpr int RB_PQ = (RB_MAXE + RB_MAXH) / 4 / 64;     // float4s of a P row per lane

// The activations on the hardware's exp2 and reciprocal (a few ulp each).  The library forms take a
// range-reduced exp and a correctly rounded division, several times the instructions, and the
// elementwise phases of the batched passes are bound by instruction issue.
__device__ __forceinline__ float exp_hw(float x) { return __builtin_amdgcn_exp2f(x * 1.44269504088896341f); }
__device__ __forceinline__ float sigmoid_hw(float x) { return __builtin_amdgcn_rcpf(1.0f + exp_hw(-x)); }
__device__ __forceinline__ float silu_hw(float x) { return x * sigmoid_hw(x); }
__device__ __forceinline__ float silu_grad_hw(float x) {
  const float s = sigmoid_hw(x);
  return s * (1.0f + x * (1.0f - s));
}
__device__ __forceinline__ float phi_hw(float x) { return x > 0.0f ? x + 1.0f : exp_hw(x); }   // ELU(x) + 1
__device__ __forceinline__ float phi_grad_hw(float x) { return x > 0.0f ? 1.0f : exp_hw(x); }

// Sum over the wave's 64 lanes (all active), every lane gets the same bits: within each 16-lane
// row by DPP moves (the two quad swaps, then the half-row and row mirrors, each lane adding the
// same pair), then the four row sums read out and added as (r0 + r1) + (r2 + r3).  A chain of
// LDS permutes would cost several times the latency.
template <int CTRL>
__device__ __forceinline__ float dpp_movf(float x) {
  return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(x), CTRL, 0xf, 0xf, false));
}
__device__ __forceinline__ float wave_sum_dpp(float v) {
  v += dpp_movf<0xB1>(v);    // quad_perm [1, 0, 3, 2]
  v += dpp_movf<0x4E>(v);    // quad_perm [2, 3, 0, 1]
  v += dpp_movf<0x141>(v);   // row_half_mirror
  v += dpp_movf<0x140>(v);   // row_mirror
  const int b = __float_as_int(v);
  auto row = [b](int l) { return __int_as_float(__builtin_amdgcn_readlane(b, l)); };
  return (row(0) + row(16)) + (row(32) + row(48));
}

// sum over the workgroup (every thread calls it; every thread gets the result, the same bits)
__device__ float block_sum(float v, float* red) {
  v = wave_sum_dpp(v);
  __syncthreads();
  if ((threadIdx.x & (kWave - 1)) == 0) red[threadIdx.x / kWave] = v;
  __syncthreads();
  float s = 0.0f;
#pragma unroll
  for (int i = 0; i < RB_NW; ++i) s += red[i];
  return s;
}

// w[i] with i a 32-bit element index from a workgroup-uniform base (the router weights are far below
// 4 GiB), so the load takes the scalar base plus a 32-bit lane offset instead of 64-bit lane addresses
template <typename W>
__device__ __forceinline__ float ldw(const W* w, unsigned i) {
  return ldf(reinterpret_cast<const W*>(reinterpret_cast<const char*>(w) + i * static_cast<unsigned>(sizeof(W))));
}

// ---------------------------------------------------------------------------
// The token work in six passes.  The three on the router's small products take RB_TB tokens per
// workgroup, so that every weight element loaded from L2 serves RB_TB tokens (one token per
// workgroup chained ~100 dependent mat-vec phases, each waiting on its weights); the others stream
// per-token rows: the residual rows for the row statistics, and one token's d_m x d_m state per
// workgroup, as the forward's memory pass does.
//   stats (a wave per token): inv_rms(hbar_j), |delta_j|, |delta_{j-1}|, delta_j . delta_{j-1}, and
//      P's K slices summed;
//   F1 (batched): the P partials of the hidden encoder, the path encoder, s, and q, k, v, W_n s;
//   M1 (per token): the memory read c = phi(q)^T S_{j-1} / (phi(q)^T zeta_{j-1} + eps);
//   F2 (batched): W_c c, nu, the history head, p, and the reverse from dL/dlogit through the
//      heads, f_theta's first layer, nu and the read's normaliser: dL/dc as dL/dnum, dL/dden;
//   M2 (per token): one pass over S_{j-1} and the carried dL/dS_j (dL/dphi(k), dL/dphi(q),
//      dL/dv, dL/drho, dL/dS_{j-1} in place), then zeta;
//   F3 (batched): the projections, path and hidden encoders in reverse, the row coefficients.
// Per-token intermediates go through the scratch named in RouterBwdArgs (token-major).  Loops over
// (token, row) pairs run token-fastest where they write the token-contiguous operands and
// row-fastest where they read or write token-major rows, so that both sides coalesce.
// ---------------------------------------------------------------------------
constexpr int RB_TB = 16;              // tokens per workgroup of the batched passes
constexpr int RB_BT = 512;             // threads of the batched passes
constexpr int RB_BW = RB_BT / kWave;   // their waves
constexpr int RB_RED = RB_BW * RB_TB * 64;   // floats of bmv_cols' partial sums
constexpr int RB_PF = 8;                     // weight loads in flight per lane in the transposed mat-vecs
constexpr int RB_PP = 4;                     // pairs of k-steps in flight per lane in the row mat-vecs

// The batched mat-vecs run on the fp32 matrix cores (v_mfma_f32_16x16x4f32: exact fp32 products,
// so bf16 weights and fp32 activations keep the precision of scalar FMAs).  A product tile is the
// RB_TB = 16 tokens times 16 outputs; lane l supplies operand row l % 16 at k slot l / 16, and
// holds the result rows 4 (l / 16) + q, q < 4, of column l % 16.  Every wave of the workgroup calls
// these; tiles are dealt to the waves round-robin.  Weights come in batches of RB_PF steps, the
// next batch's loads issued before the current batch's products (across tiles too).  A result
// column depends on its own weight column alone and a token row on its own operand row alone, so
// out-of-range outputs read a clamped in-range weight address and are never stored; out-of-range k
// (or rows o in the transposed form) enter the operand as zeros, since the LDS there may hold
// anything; token rows b >= nb are computed from whatever the LDS holds there and never stored.
// the wave's index in the workgroup as a scalar (threadIdx.x / 64 is uniform per wave, but the
// compiler treats it as varying by lane, which turns every loop over tiles into divergent code)
__device__ __forceinline__ int wave_id() { return __builtin_amdgcn_readfirstlane(static_cast<int>(threadIdx.x) / kWave); }
__device__ __forceinline__ f32x4 mfma4(float a, float b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}
// w[i .. i + 3] (i a multiple of 4, the row pitch too) as loaded (raw4), and in fp32 (cvt4), for the
// fp32 weights' transposed products.  The batches hold raw words and convert at their products:
// converting at the load would make the compiler wait for the next batch's loads before the
// current batch's products.
template <typename W>
struct Raw4;
template <>
struct Raw4<float> {
  using type = f32x4;
};
__device__ __forceinline__ f32x4 raw4(const float* w, unsigned i) {
  return *reinterpret_cast<const f32x4*>(reinterpret_cast<const char*>(w) + i * 4u);
}
__device__ __forceinline__ f32x4 cvt4(f32x4 v) { return v; }
// w[i .. i + 7] the same way (i a multiple of 8, the row pitch too): one 16-byte load in bf16
template <typename W>
struct Raw8;
template <>
struct Raw8<bf16_t> {
  using type = u32x4;
};
struct F32x8 {
  f32x4 a, b;
};
template <>
struct Raw8<float> {
  using type = F32x8;
};
__device__ __forceinline__ u32x4 raw8(const bf16_t* w, unsigned i) {
  return *reinterpret_cast<const u32x4*>(reinterpret_cast<const char*>(w) + i * 2u);
}
__device__ __forceinline__ F32x8 raw8(const float* w, unsigned i) {
  const f32x4* p = reinterpret_cast<const f32x4*>(reinterpret_cast<const char*>(w) + i * 4u);
  return F32x8{p[0], p[1]};
}
__device__ __forceinline__ f32x4 cvt8lo(u32x4 u) {
  return f32x4{__uint_as_float(u.x << 16), __uint_as_float(u.x & 0xffff0000u), __uint_as_float(u.y << 16),
               __uint_as_float(u.y & 0xffff0000u)};
}
__device__ __forceinline__ f32x4 cvt8hi(u32x4 u) {
  return f32x4{__uint_as_float(u.z << 16), __uint_as_float(u.z & 0xffff0000u), __uint_as_float(u.w << 16),
               __uint_as_float(u.w & 0xffff0000u)};
}
__device__ __forceinline__ f32x4 cvt8lo(const F32x8& v) { return v.a; }
__device__ __forceinline__ f32x4 cvt8hi(const F32x8& v) { return v.b; }

// Up to four weight matrices of one row pitch stacked by rows: stack row o is row o - m om of
// matrix m (om rows each, a multiple of 16 when there are several; one matrix: om = its rows)
template <typename W>
struct Mats {
  const W *w0, *w1, *w2, *w3;
  int om, ld;
  __device__ __forceinline__ int mat(int o) const { return (o >= om) + (o >= 2 * om) + (o >= 3 * om); }
  __device__ __forceinline__ const W* base(int m) const { return m == 0 ? w0 : m == 1 ? w1 : m == 2 ? w2 : w3; }
};
template <typename W>
__device__ __forceinline__ Mats<W> mats1(const void* w, int rows, int ld) {
  return Mats<W>{static_cast<const W*>(w), nullptr, nullptr, nullptr, rows, ld};
}

// lane's eight weights of stack row ot 16 + r (clamped to the last row) from column k, as loaded
template <typename W>
__device__ __forceinline__ typename Raw8<W>::type rows_w8(const Mats<W>& M, int O, int ot, int r, int k) {
  const int m = M.mat(ot * 16), o = min(ot * 16 + r, O - 1);   // a tile lies in one matrix
  return raw8(M.base(m), static_cast<unsigned>(o - m * M.om) * M.ld + k);
}
// the k >= kb steps of tile ot with scalar loads (the ragged end, or every k when the pitch is not a
// multiple of 4)
template <typename W>
__device__ __forceinline__ f32x4 rows_tail(const Mats<W>& M, int O, int ot, int I, int kb, const float* x, int ldx,
                                           int r, int g, f32x4 acc) {
  const int m = M.mat(ot * 16), o = min(ot * 16 + r, O - 1);
  const W* wb = M.base(m);
  const unsigned wr = static_cast<unsigned>(o - m * M.om) * M.ld;
  for (int k0 = kb; k0 < I; k0 += 16) {
    const int kk = k0 + 4 * g;
    float wa[4], xa[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const bool kv = kk + i < I;
      const int kc = kv ? kk + i : I - 1;
      const float wl = ldw(wb, wr + kc), xl = x[r * ldx + kc];
      wa[i] = kv ? wl : 0.0f;
      xa[i] = kv ? xl : 0.0f;
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) acc = mfma4(xa[i], wa[i], acc);
  }
  return acc;
}
__device__ __forceinline__ void rows_store(f32x4 acc, int O, int ot, int r, int g, float* y, int ldy, int nb) {
  const int o = ot * 16 + r;
  if (o < O)
#pragma unroll
    for (int q = 0; q < 4; ++q)
      if (4 * g + q < nb) y[(4 * g + q) * ldy + o] = acc[q];
}

// y[b][o] = sum_k W[o][k] x[b][k] for b < nb, o < O over a stack W (x in LDS, [RB_TB][ldx]; y in
// LDS or global).  With a row pitch that is a multiple of 8, k goes in pairs of 16-k steps: over the 32
// k of a pair, slot g takes k0 + 8 g + i in the first step's i-th product and k0 + 8 g + 4 + i in the
// second's, so each lane loads its eight k of the pair at once (16 bytes in bf16; four lanes cover 64
// bytes of a weight row per load).  Two accumulators alternate.
template <typename W>
__device__ __forceinline__ void bmv_rows(const Mats<W>& M, int O, int I, const float* x, int ldx, float* y, int ldy,
                                         int nb) {
  const int lane = threadIdx.x & (kWave - 1), r = lane & 15, g = lane >> 4, wv = wave_id();
  const int ntile = (O + 15) / 16;
  const int ntw = wv < ntile ? (ntile - 1 - wv) / RB_BW + 1 : 0;   // this wave's tiles (uniform)
  const int npr = (M.ld & 7) == 0 ? I / 32 : 0, I32 = 32 * npr;   // pairs of steps
  const f32x4 zero = {0.0f, 0.0f, 0.0f, 0.0f};
  if (npr == 0) {
    for (int ti = 0; ti < ntw; ++ti) {
      const int ot = wv + ti * RB_BW;
      rows_store(rows_tail(M, O, ot, I, 0, x, ldx, r, g, zero), O, ot, r, g, y, ldy, nb);
    }
    return;
  }
  // the wave's batches of RB_PP pairs in sequence: batch q is batch q % nbt of its tile q / nbt
  const int nbt = (npr + RB_PP - 1) / RB_PP, total = ntw * nbt;
  const float* xr = x + r * ldx + 8 * g;
  typename Raw8<W>::type cur[RB_PP];
  if (total > 0)
#pragma unroll
    for (int u = 0; u < RB_PP; ++u) cur[u] = rows_w8(M, O, wv, r, 32 * min(u, npr - 1) + 8 * g);
  f32x4 acc0 = zero, acc1 = zero;
  for (int q = 0; q < total; ++q) {
    const int ti = q / nbt, c = q - ti * nbt, ot = wv + ti * RB_BW;
    typename Raw8<W>::type nxt[RB_PP];
    if (q + 1 < total) {   // uniform
      const int t1 = (q + 1) / nbt, c1 = q + 1 - t1 * nbt;
#pragma unroll
      for (int u = 0; u < RB_PP; ++u)
        nxt[u] = rows_w8(M, O, wv + t1 * RB_BW, r, 32 * min(c1 * RB_PP + u, npr - 1) + 8 * g);
    }
#pragma unroll
    for (int u = 0; u < RB_PP; ++u) {
      const int pr = c * RB_PP + u;
      if (pr < npr) {   // uniform
        const float* xk = xr + 32 * pr;
        const f32x4 w0 = cvt8lo(cur[u]), w1 = cvt8hi(cur[u]);
        acc0 = mfma4(xk[0], w0[0], acc0);
        acc1 = mfma4(xk[1], w0[1], acc1);
        acc0 = mfma4(xk[2], w0[2], acc0);
        acc1 = mfma4(xk[3], w0[3], acc1);
        acc0 = mfma4(xk[4], w1[0], acc0);
        acc1 = mfma4(xk[5], w1[1], acc1);
        acc0 = mfma4(xk[6], w1[2], acc0);
        acc1 = mfma4(xk[7], w1[3], acc1);
      }
    }
    if (c == nbt - 1) {   // the tile's last batch
      rows_store(rows_tail(M, O, ot, I, I32, x, ldx, r, g, acc0 + acc1), O, ot, r, g, y, ldy, nb);
      acc0 = acc1 = zero;
    }
#pragma unroll
    for (int u = 0; u < RB_PP; ++u) cur[u] = nxt[u];
  }
}

// One transposed product x[b][k] (+)= sum_o W[o][k] y[b][o], b < nb, k < I, over a stack W of O rows
// (y and x in LDS).  With a row pitch that is a multiple of 4 (and at least I rounded up to 4), a
// tile is 64 columns in four accumulators (lane r of accumulator i: column 64 kt + 4 r + i, so each
// lane loads four adjacent weights per row) and each product takes four rows o (slot g: o0 + g);
// otherwise a tile is 16 columns with scalar loads.  When there are fewer tiles than waves, the o
// range is cut into parts whose partial sums meet in red ([parts][RB_TB][tiles x 64] floats) and
// are added in part order.
template <typename W>
struct Cols {
  Mats<W> M;
  int O, I;
  const float* y;
  int ldy;
  float* x;
  int ldx;
  bool acc;
};
struct ColsPlan {
  int ntile, parts, ocnt, wid, items;
  bool vec;
};
__device__ __forceinline__ ColsPlan cols_plan(int O, int I, int ld, int waves) {
  ColsPlan p;
  p.vec = (ld & 3) == 0;
  p.ntile = p.vec ? (I + 63) / 64 : (I + 15) / 16;
  p.parts = (!p.vec || p.ntile >= waves) ? 1 : waves / p.ntile;   // parts x ntile <= waves
  p.ocnt = ((O + p.parts - 1) / p.parts + 3) & ~3;                  // rows per part, a multiple of 4
  p.wid = p.ntile * 64;
  p.items = p.ntile * p.parts;
  return p;
}
template <typename W>
__device__ __forceinline__ void cols_item(const Cols<W>& J, const ColsPlan& P, int it, int nb, float* red) {
  const int lane = threadIdx.x & (kWave - 1), r = lane & 15, g = lane >> 4;
  const f32x4 zero = {0.0f, 0.0f, 0.0f, 0.0f};
  const int kt = it % P.ntile, pt = it / P.ntile;
  const float* yr = J.y + r * J.ldy;
  if (!P.vec) {
    const int k = kt * 16 + r;
    const bool kv = k < J.I;
    const int kc = kv ? k : J.I - 1;
    f32x4 acc = zero;
    for (int o0 = 0; o0 < J.O; o0 += 16) {
      const int oo = o0 + 4 * g;
      float wa[4], ya[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const bool ov = oo + i < J.O;
        const int oc = ov ? oo + i : J.O - 1, m = J.M.mat(oc);
        wa[i] = ldw(J.M.base(m), static_cast<unsigned>(oc - m * J.M.om) * J.M.ld + kc);
        const float yl = yr[oc];
        ya[i] = ov ? yl : 0.0f;
      }
#pragma unroll
      for (int i = 0; i < 4; ++i) acc = mfma4(ya[i], wa[i], acc);
    }
    if (kv)
#pragma unroll
      for (int q = 0; q < 4; ++q)
        if (4 * g + q < nb) {
          float* xe = J.x + (4 * g + q) * J.ldx + k;
          *xe = J.acc ? *xe + acc[q] : acc[q];
        }
    return;
  }
  const int ob = min(J.O, pt * P.ocnt), oe = min(J.O, ob + P.ocnt);
  const int kc = kt * 64 + 4 * r;
  const unsigned kl = static_cast<unsigned>(kc < J.I ? kc : (J.I - 1) & ~3);   // columns >= I: any in-row chunk
  const int nst = (oe - ob + 3) / 4;   // steps of four rows (of one matrix: om is a multiple of 4)
  f32x4 acc[4] = {zero, zero, zero, zero};
  if (nst > 0) {
    typename Raw4<W>::type bc[RB_PF];
    float ac[RB_PF];
#pragma unroll
    for (int u = 0; u < RB_PF; ++u) {
      const int so = ob + 4 * min(u, nst - 1), m = J.M.mat(so), o = so + g, oc = min(o, oe - 1);
      bc[u] = raw4(J.M.base(m), static_cast<unsigned>(oc - m * J.M.om) * J.M.ld + kl);
      const float yl = yr[oc];
      ac[u] = o < oe ? yl : 0.0f;
    }
    for (int s0 = 0; s0 < nst; s0 += RB_PF) {
      typename Raw4<W>::type bn[RB_PF];
      float an[RB_PF];
      if (s0 + RB_PF < nst) {   // uniform
#pragma unroll
        for (int u = 0; u < RB_PF; ++u) {
          const int so = ob + 4 * min(s0 + RB_PF + u, nst - 1), m = J.M.mat(so), o = so + g, oc = min(o, oe - 1);
          bn[u] = raw4(J.M.base(m), static_cast<unsigned>(oc - m * J.M.om) * J.M.ld + kl);
          const float yl = yr[oc];
          an[u] = o < oe ? yl : 0.0f;
        }
      }
#pragma unroll
      for (int u = 0; u < RB_PF; ++u)
        if (s0 + u < nst) {   // uniform
          const f32x4 bv = cvt4(bc[u]);
#pragma unroll
          for (int i = 0; i < 4; ++i) acc[i] = mfma4(ac[u], bv[i], acc[i]);
        }
#pragma unroll
      for (int u = 0; u < RB_PF; ++u) {
        bc[u] = bn[u];
        ac[u] = an[u];
      }
    }
  }
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int b = 4 * g + q;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      if (P.parts > 1) {
        red[(pt * RB_TB + b) * P.wid + kc + i] = acc[i][q];
      } else if (b < nb && kc + i < J.I) {
        float* xe = J.x + b * J.ldx + kc + i;
        *xe = J.acc ? *xe + acc[i][q] : acc[i][q];
      }
    }
  }
}
template <typename W>
__device__ __forceinline__ void cols_reduce(const Cols<W>& J, const ColsPlan& P, int nb, const float* red) {
  for (int e = threadIdx.x; e < nb * J.I; e += RB_BT) {
    const int b = e / J.I, k = e % J.I;
    float v = J.acc ? J.x[b * J.ldx + k] : 0.0f;
    for (int pt = 0; pt < P.parts; ++pt) v += red[(pt * RB_TB + b) * P.wid + k];
    J.x[b * J.ldx + k] = v;
  }
}
// one or two independent transposed products in one phase (two: half the waves' worth of parts
// each, their partial sums in separate halves of red, at most RB_RED floats); every thread calls
// it, and when partial sums are used it ends on a barrier
template <typename W>
__device__ __forceinline__ void bmv_cols2(const Cols<W>& A, const Cols<W>& B, bool two, int nb, float* red) {
  const int wv = wave_id(), waves = two ? RB_BW / 2 : RB_BW;
  const ColsPlan PA = cols_plan(A.O, A.I, A.M.ld, waves);
  ColsPlan PB = PA;
  PB.items = 0;
  PB.parts = 1;
  if (two) PB = cols_plan(B.O, B.I, B.M.ld, waves);
  float* redB = red + (PA.parts > 1 ? PA.parts * RB_TB * PA.wid : 0);
  for (int it = wv; it < PA.items + PB.items; it += RB_BW) {   // uniform per wave
    if (it < PA.items)
      cols_item(A, PA, it, nb, red);
    else
      cols_item(B, PB, it - PA.items, nb, redB);
  }
  if (PA.parts > 1 || PB.parts > 1) {
    __syncthreads();
    if (PA.parts > 1) cols_reduce(A, PA, nb, red);
    if (PB.parts > 1) cols_reduce(B, PB, nb, redB);
    __syncthreads();
  }
}
template <typename W>
__device__ __forceinline__ void bmv_cols(const Cols<W>& A, int nb, float* red) {
  bmv_cols2(A, A, false, nb, red);
}

// bf16 weights: the batched products on v_mfma_f32_16x16x32_bf16.  An fp32 activation block (LDS,
// [RB_TB][ldx]) is split, where it is produced or once before its product, into x = hi + lo, two bf16
// values with |x - hi - lo| <= 2^-18 |x|, kept in LDS as two [RB_TB][xp] copies; the bf16 weights are exact, so
// the two products of each 32-k step are exact in fp32 and only the accumulation rounds.  The
// transposed products run as row products over transposed copies of the weights.
constexpr int RB_XPAD = 8;   // bf16 entries past a split row's 32-multiple (spreads the rows over LDS banks)
__host__ __device__ constexpr int rb_round(int x, int m) { return (x + m - 1) / m * m; }
__host__ __device__ constexpr int rb_split_pitch(int I) { return rb_round(I, 32) + RB_XPAD; }

// v into its split copies at entry i
__device__ __forceinline__ void put_split(bf16_t* xh, bf16_t* xl, int i, float v) {
  const __bf16 h = static_cast<__bf16>(v);
  xh[i] = __builtin_bit_cast(bf16_t, h);
  xl[i] = __builtin_bit_cast(bf16_t, static_cast<__bf16>(v - static_cast<float>(h)));
}
// x[b][k] (b < nb, k < I) into its split copies, zeros for I <= k < Iz (a product's K past the
// valid entries, where the weights are zero padding); every thread calls it, between barriers
__device__ __forceinline__ void split_x(const float* x, int ldx, int I, int Iz, int nb, bf16_t* xh, bf16_t* xl,
                                        int xp) {
  for (int e = threadIdx.x; e < nb * Iz; e += RB_BT) {
    const int b = e / Iz, k = e - b * Iz;
    put_split(xh, xl, b * xp + k, k < I ? x[b * ldx + k] : 0.0f);
  }
}

constexpr int RB_P16 = 8;   // 32-k steps of weight loads in flight per lane in the split-bf16 products

// Up to four bf16 matrices of one row pitch stacked by rows (as Mats), held as separate values: a
// struct in memory selected by a runtime index gets compiled into an indexed load from scratch
struct Stack16 {
  const bf16_t *w0, *w1, *w2, *w3;
  int om, ld;
};
__device__ __forceinline__ Stack16 stack16(const Mats<bf16_t>& M) { return Stack16{M.w0, M.w1, M.w2, M.w3, M.om, M.ld}; }
__device__ __forceinline__ Stack16 one16(const void* w, int rows, int ld) {
  return Stack16{static_cast<const bf16_t*>(w), nullptr, nullptr, nullptr, rows, ld};
}
// lane's weight row in tile ot (stack row ot 16 + r, clamped to the last row; a tile lies in one
// matrix, so the choice of matrix is uniform)
__device__ __forceinline__ const bf16_t* w_row16(const bf16_t* w0, const bf16_t* w1, const bf16_t* w2,
                                                 const bf16_t* w3, int om, int ld, int O, int ot, int r) {
  const int o0 = ot * 16, m = (o0 >= om) + (o0 >= 2 * om) + (o0 >= 3 * om);
  const bf16_t* w = m == 0 ? w0 : m == 1 ? w1 : m == 2 ? w2 : w3;
  return w + static_cast<unsigned>(min(o0 + r, O - 1) - m * om) * ld;
}

// y[b][o] (+)= sum_{k < I} W[o][k] x[b][k] for b < nb, o < O over a stack W of bf16 rows (pitch a
// multiple of 8; I a multiple of 8), x given by its split copies (pitch xp at least I rounded up to
// 32; entries past I and rows past nb may hold anything).  16-row tiles spread over the waves; a tile's k range goes in 32-k steps
// (slot g: k0 + 8 g .. + 7, one 16-byte weight load a lane), and the wave's steps over all its tiles
// run as one sequence with RB_P16 steps' loads in flight ahead of the products; hi and lo
// accumulate apart.  With oh set, each stored value also goes into split copies (oh, ol, pitch osp).
__device__ __forceinline__ void bmv16(Stack16 M, int O, int I, const bf16_t* xh, const bf16_t* xl, int xp, float* y,
                                      int ldy, int nb, bool acc, bf16_t* oh = nullptr, bf16_t* ol = nullptr,
                                      int osp = 0) {
  const bf16_t *w0 = M.w0, *w1 = M.w1, *w2 = M.w2, *w3 = M.w3;
  const int om = M.om, ld = M.ld;
  const int lane = threadIdx.x & (kWave - 1), r = lane & 15, g = lane >> 4, wv = wave_id();
  const int ntile = (O + 15) / 16;
  const int ntw = wv < ntile ? (ntile - 1 - wv) / RB_BW + 1 : 0;   // this wave's tiles (uniform)
  const int nst = (I + 31) / 32, total = ntw * nst;
  if (total == 0) return;
  const f32x4 zero = {0.0f, 0.0f, 0.0f, 0.0f};
  const bf16x8 zx = __builtin_bit_cast(bf16x8, u32x4{0u, 0u, 0u, 0u});
  const bf16_t* ah = xh + r * xp + 8 * g;
  const bf16_t* al = xl + r * xp + 8 * g;
  // load side: the next step to load, as (tile, step), and that tile's weight row.  Every load is
  // issued unconditionally (columns clamped below I; the products zero the x fragments past I),
  // which keeps the compiler's count of loads in flight exact: a load under a branch makes it wait
  // for all of them.
  int lt = 0, ls = 0;
  const bf16_t* lrow = w_row16(w0, w1, w2, w3, om, ld, O, wv, r);
  u32x4 cur[RB_P16];
#define RB_NEXT_LOAD(dst)                                          \
  do {                                                             \
    dst = raw8(lrow, static_cast<unsigned>(min(32 * ls + 8 * g, I - 8))); \
    if (++ls == nst) {                                             \
      ls = 0;                                                      \
      lt = min(lt + 1, ntw - 1); /* past the end: the last tile again (unused) */ \
      lrow = w_row16(w0, w1, w2, w3, om, ld, O, wv + lt * RB_BW, r);                    \
    }                                                              \
  } while (0)
#pragma unroll
  for (int u = 0; u < RB_P16; ++u) RB_NEXT_LOAD(cur[u]);
  f32x4 acc0 = zero, acc1 = zero;
  int ti = 0, st = 0;   // the step the products are at
  for (int q0 = 0; q0 < total; q0 += RB_P16) {
    u32x4 nxt[RB_P16];
    if (q0 + RB_P16 < total)   // uniform
#pragma unroll
      for (int u = 0; u < RB_P16; ++u) RB_NEXT_LOAD(nxt[u]);
    // the batch's x fragments first (every step's row entries exist, whatever the step), so that
    // their LDS latency is paid once a batch rather than at every step
    bf16x8 xhi[RB_P16], xlo[RB_P16];
    {
      int sx = st;
#pragma unroll
      for (int u = 0; u < RB_P16; ++u) {
        xhi[u] = *reinterpret_cast<const bf16x8*>(ah + 32 * sx);
        xlo[u] = *reinterpret_cast<const bf16x8*>(al + 32 * sx);
        if (32 * sx + 8 * g >= I) xhi[u] = xlo[u] = zx;   // (the split rows hold I rounded up to 32)
        if (++sx == nst) sx = 0;
      }
    }
#pragma unroll
    for (int u = 0; u < RB_P16; ++u) {
      if (q0 + u < total) {   // uniform
        const bf16x8 w = __builtin_bit_cast(bf16x8, cur[u]);
        acc0 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(xhi[u], w, acc0, 0, 0, 0);
        acc1 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(xlo[u], w, acc1, 0, 0, 0);
        if (++st == nst) {   // the tile's last step
          const f32x4 v = acc0 + acc1;
          const int o = (wv + ti * RB_BW) * 16 + r;
          if (o < O)
#pragma unroll
            for (int q2 = 0; q2 < 4; ++q2) {
              const int b = 4 * g + q2;
              if (b < nb) {
                float* ye = y + b * ldy + o;
                const float f = acc ? *ye + v[q2] : v[q2];
                *ye = f;
                if (oh) put_split(oh, ol, b * osp + o, f);
              }
            }
          acc0 = acc1 = zero;
          st = 0;
          ++ti;
        }
      }
    }
#pragma unroll
    for (int u = 0; u < RB_P16; ++u) cur[u] = nxt[u];
  }
#undef RB_NEXT_LOAD
}

// stats: a wave per token over the residual rows (16-byte loads) and P's slices
template <typename T>
__global__ __launch_bounds__(RB_NT) void rbwd_stats(RouterBwdArgs a) {
  constexpr int SB = 4;   // 8-element chunks of each row per lane in flight
  using R8 = typename Raw8<T>::type;
  const int t = a.t_begin + static_cast<int>(blockIdx.x) * RB_NW + static_cast<int>(threadIdx.x) / kWave;
  const int lane = threadIdx.x & (kWave - 1);
  if (t >= a.t_end) return;   // whole waves; no barrier below
  const int j = a.j, d = a.d, NP = a.d_e + a.d_head, T_ = a.T, ns = a.p_splits;
  // P's K slices (float4 rows when NP allows), in flight with the rows' first batch
  const bool v4 = (NP & 3) == 0;
  f32x4 pv[RB_PQ][RB_MAXSPL];
  if (v4) {
#pragma unroll
    for (int u = 0; u < RB_PQ; ++u) {
      const int q = lane + u * kWave;
#pragma unroll
      for (int z = 0; z < RB_MAXSPL; ++z)
        pv[u][z] = 4 * q < NP && z < ns
                       ? *reinterpret_cast<const f32x4*>(a.P + (static_cast<size_t>(z) * T_ + t) * NP + 4 * q)
                       : f32x4{0.0f, 0.0f, 0.0f, 0.0f};
    }
  }
  const T* hb = static_cast<const T*>(a.hbar) + static_cast<size_t>(t) * d;
  const T* h1 = j >= 2 ? static_cast<const T*>(a.prev1) + static_cast<size_t>(t) * d : hb;
  const T* h2 = j >= 3 ? static_cast<const T*>(a.prev2) + static_cast<size_t>(t) * d : hb;
  float s2 = 0.0f, dd = 0.0f, dpv = 0.0f, pp2 = 0.0f;
  for (int i0 = lane * 8; i0 < d; i0 += kWave * 8 * SB) {
    R8 x[SB], y[SB], z[SB];
#pragma unroll
    for (int u = 0; u < SB; ++u) {
      const int i = min(i0 + u * kWave * 8, d - 8);   // a clamped chunk is loaded but not used
      x[u] = raw8(hb, static_cast<unsigned>(i));
      if (j >= 2) y[u] = raw8(h1, static_cast<unsigned>(i));
      if (j >= 3) z[u] = raw8(h2, static_cast<unsigned>(i));
    }
#pragma unroll
    for (int u = 0; u < SB; ++u) {
      if (i0 + u * kWave * 8 >= d) break;
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const f32x4 xv = h ? cvt8hi(x[u]) : cvt8lo(x[u]);
        f32x4 yv = xv, zv = xv;
        if (j >= 2) yv = h ? cvt8hi(y[u]) : cvt8lo(y[u]);
        if (j >= 3) zv = h ? cvt8hi(z[u]) : cvt8lo(z[u]);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          s2 = fmaf(xv[e], xv[e], s2);
          if (j >= 2) {
            const float del = xv[e] - yv[e];
            dd = fmaf(del, del, dd);
            if (j >= 3) {
              const float dp_ = yv[e] - zv[e];
              dpv = fmaf(del, dp_, dpv);
              pp2 = fmaf(dp_, dp_, pp2);
            }
          }
        }
      }
    }
  }
  s2 = wave_sum_dpp(s2);
  dd = wave_sum_dpp(dd);
  dpv = wave_sum_dpp(dpv);
  pp2 = wave_sum_dpp(pp2);
  if (lane == 0) {
    float* rs = a.RS + static_cast<size_t>(t) * 4;
    rs[0] = 1.0f / sqrtf(s2 / static_cast<float>(d) + a.eps_norm);
    rs[1] = j >= 2 ? sqrtf(dd) : 0.0f;
    rs[2] = sqrtf(pp2);
    rs[3] = dpv;
  }
  // P's K slices added in slice order, once for the three batched passes
  if (v4) {
#pragma unroll
    for (int u = 0; u < RB_PQ; ++u) {
      const int q = lane + u * kWave;
      if (4 * q >= NP) break;
      f32x4 v = pv[u][0];
#pragma unroll
      for (int z = 1; z < RB_MAXSPL; ++z)
        if (z < ns) v += pv[u][z];
      *reinterpret_cast<f32x4*>(a.PSUM + static_cast<size_t>(t) * NP + 4 * q) = v;
    }
  } else {
    for (int k = lane; k < NP; k += kWave) {
      float v = 0.0f;
      for (int z = 0; z < ns; ++z) v += a.P[(static_cast<size_t>(z) * T_ + t) * NP + k];
      a.PSUM[static_cast<size_t>(t) * NP + k] = v;
    }
  }
}

// F1
template <typename T>
__global__ __launch_bounds__(RB_BT) void rbwd_f1(RouterBwdArgs a) {
  __shared__ float sh[RB_TB][RB_MAXE + 1];     // SiLU(ir P_h)
  __shared__ float pp[RB_TB][RB_MAXP + 1];     // SiLU of the path encoder's pre-activation
  __shared__ float xs[RB_TB][RB_MAXS + 1];     // s
  __shared__ float xp[RB_TB][8];
  __shared__ float wp1[RB_MAXP * 6];
  __shared__ float irs[RB_TB];
  // bf16: the split copies of SiLU(ir P_h), of the path encoder's SiLU and of s
  constexpr bool kB = std::is_same<T, bf16_t>::value;
  constexpr int XE = kB ? rb_split_pitch(RB_MAXE) : 0, XQ = kB ? rb_split_pitch(RB_MAXP) : 0;
  constexpr int XS = kB ? rb_split_pitch(RB_MAXS) : 0;
  __shared__ __attribute__((aligned(16))) bf16_t xsp[kB ? 2 * RB_TB * (XE + XQ + XS) : 8];
  bf16_t *eh = xsp, *el = eh + RB_TB * XE, *qh = el + RB_TB * XE, *ql = qh + RB_TB * XQ, *sh2 = ql + RB_TB * XQ;
  bf16_t* sl2 = sh2 + RB_TB * XS;
  const int xe = rb_split_pitch(a.d_e), xq = rb_split_pitch(a.d_p), xsx = rb_split_pitch(a.d_s);
  const bool p8 = (a.d_p & 7) == 0;   // W_p2's rows as 16-byte loads
  const int tid = threadIdx.x;
  const int T_ = a.T, j = a.j, DM = a.d_m, d_s = a.d_s, d_h = a.d_h, d_a = a.d_a;
  const int d_e = a.d_e, d_p = a.d_p, NP = d_e + a.d_head;
  const int t0 = a.t_begin + static_cast<int>(blockIdx.x) * RB_TB, nb = min(RB_TB, a.t_end - t0);
  // P's hidden part (loads first, clamped to the last element), W_p1, the path features
  constexpr int UE = (RB_TB * RB_MAXE + RB_BT - 1) / RB_BT;
  const int ne = nb * d_e;
  float ph[UE];
#pragma unroll
  for (int u = 0; u < UE; ++u) {
    const int e = min(tid + u * RB_BT, ne - 1), b = e / d_e, k = e % d_e;
    ph[u] = a.PSUM[static_cast<size_t>(t0 + b) * NP + k];
  }
  for (int e = tid; e < d_p * 6; e += RB_BT) wp1[e] = ldf(static_cast<const T*>(a.w_p1) + e);
  if (tid < nb) {
    const int b = tid, t = t0 + b;
    const float* rs = a.RS + static_cast<size_t>(t) * 4;
    const float dj = rs[1], np_ = rs[2], dpv = rs[3];
    irs[b] = rs[0];
    xp[b][0] = static_cast<float>(j) / static_cast<float>(a.L_R);
    xp[b][1] = static_cast<float>(a.L_R - j) / static_cast<float>(a.L_R);
    xp[b][2] = dj;
    xp[b][3] = j >= 3 ? dpv / (dj * np_ + a.eps) : 0.0f;
    xp[b][4] = j > 1 ? a.p_in[t] : 1.0f;
    xp[b][5] = j > 1 ? a.m_in[t] : 1.0f;
    xp[b][6] = xp[b][7] = 0.0f;
  }
  __syncthreads();
  // SiLU(ir P_h); the path encoder W_p1 x^path (six terms) and its SiLU
#pragma unroll
  for (int u = 0; u < UE; ++u) {
    const int e = tid + u * RB_BT, b = e / d_e, k = e % d_e;
    if (e < ne) {
      const float v = silu_hw(irs[b] * ph[u]);
      sh[b][k] = v;
      if (kB) put_split(eh, el, b * xe + k, v);
    }
  }
  for (int e = tid; e < nb * d_p; e += RB_BT) {
    const int b = e / d_p, o = e % d_p;
    float pre = 0.0f;
#pragma unroll
    for (int k = 0; k < 6; ++k) pre = fmaf(wp1[o * 6 + k], xp[b][k], pre);
    a.PPRE[static_cast<size_t>(t0 + b) * d_p + o] = pre;
    const float v = silu_hw(pre);
    pp[b][o] = v;
    if (kB && p8) put_split(qh, ql, b * xq + o, v);
  }
  __syncthreads();
  for (int e = tid; e < nb * d_p; e += RB_BT) {
    const int o = e / nb, b = e % nb;
    a.SPT[static_cast<size_t>(o) * T_ + t0 + b] = pp[b][o];
  }
  for (int e = tid; e < nb * 6; e += RB_BT) {
    const int o = e / nb, b = e % nb;
    a.XPT[static_cast<size_t>(o) * T_ + t0 + b] = xp[b][o];
  }
  // s = [W_hu SiLU(ir P_h); W_p2 SiLU(W_p1 x^path)]
  if constexpr (kB) {   // s's split copies as it is stored
    bmv16(one16(a.w_hu, d_h, d_e), d_h, d_e, eh, el, xe, &xs[0][0], RB_MAXS + 1, nb, false, sh2, sl2,
          xsx);
    if (p8)
      bmv16(one16(a.w_p2, d_a, d_p), d_a, d_p, qh, ql, xq, &xs[0][d_h], RB_MAXS + 1, nb, false, sh2 + d_h,
            sl2 + d_h, xsx);
    else
      bmv_rows(mats1<T>(a.w_p2, d_a, d_p), d_a, d_p, &pp[0][0], RB_MAXP + 1, &xs[0][d_h], RB_MAXS + 1, nb);
  } else {
    bmv_rows(mats1<T>(a.w_hu, d_h, d_e), d_h, d_e, &sh[0][0], RB_MAXE + 1, &xs[0][0], RB_MAXS + 1, nb);
    bmv_rows(mats1<T>(a.w_p2, d_a, d_p), d_a, d_p, &pp[0][0], RB_MAXP + 1, &xs[0][d_h], RB_MAXS + 1, nb);
  }
  __syncthreads();
  for (int e = tid; e < nb * d_s; e += RB_BT) {
    const int k = e / nb, b = e % nb;
    a.XT[static_cast<size_t>(k) * T_ + t0 + b] = xs[b][k];
  }
  // [q; k; v; W_n s] (pre-activations) in one stacked product, token-major
  const Mats<T> qkvn{static_cast<const T*>(a.w_q), static_cast<const T*>(a.w_k), static_cast<const T*>(a.w_v),
                     static_cast<const T*>(a.w_n), DM, d_s};
  float* qkvu = a.QKVU + static_cast<size_t>(t0) * 4 * DM;
  if constexpr (kB) {
    if (!p8) {   // W_p2's part of s came from the fp32 path
      split_x(&xs[0][d_h], RB_MAXS + 1, d_a, d_a, nb, sh2 + d_h, sl2 + d_h, xsx);
      __syncthreads();
    }
    bmv16(stack16(qkvn), 4 * DM, d_s, sh2, sl2, xsx, qkvu, 4 * DM, nb, false);
  } else {
    bmv_rows(qkvn, 4 * DM, d_s, &xs[0][0], RB_MAXS + 1, qkvu, 4 * DM, nb);
  }
}

// M1: c and the normaliser for one token; thread: 4 columns (a float4) of DM / (RB_NT / (DM / 4))
// rows, partial sums added over the row groups in order.  S is read once, with the non-temporal
// hint, so that the stream does not push the router weights out of L2 between the batched passes.
template <int DM>
__global__ __launch_bounds__(RB_NT) void rbwd_read(RouterBwdArgs a) {
  constexpr int CG = DM / 4, RG = RB_NT / CG;   // column groups, row groups
  constexpr int NR = DM / RG, PF = NR < 16 ? NR : 16;   // rows per thread, rows loaded before phi(q)
  __shared__ float fq[DM];
  __shared__ f32x4 part[RG][CG];
  __shared__ float red[RB_NW];
  const int t = a.t_begin + static_cast<int>(blockIdx.x), tid = threadIdx.x, j = a.j;
  const int cg = tid % CG, rg = tid / CG;
  const f32x4* S = j > 1 ? reinterpret_cast<const f32x4*>(a.S_in + static_cast<size_t>(t) * DM * DM) + cg : nullptr;
  f32x4 pre[PF];
  if (S)
#pragma unroll
    for (int u = 0; u < PF; ++u) pre[u] = __builtin_nontemporal_load(S + static_cast<size_t>(rg + u * RG) * CG);
  for (int k = tid; k < DM; k += RB_NT) fq[k] = phi_hw(a.QKVU[static_cast<size_t>(t) * 4 * DM + k]);
  __syncthreads();
  f32x4 acc = {0.0f, 0.0f, 0.0f, 0.0f};
  float den = 0.0f;
  if (S) {
#pragma unroll
    for (int u = 0; u < PF; ++u) acc += fq[rg + u * RG] * pre[u];
#pragma unroll 16
    for (int u = PF; u < NR; ++u) {
      const int k = rg + u * RG;
      acc += fq[k] * __builtin_nontemporal_load(S + static_cast<size_t>(k) * CG);
    }
    for (int k = tid; k < DM; k += RB_NT) den = fmaf(fq[k], a.zeta_in[static_cast<size_t>(t) * DM + k], den);
  }
  part[rg][cg] = acc;
  den = block_sum(den, red) + a.eps;   // (its barriers also publish part)
  for (int v = tid; v < DM; v += RB_NT) {
    float c = 0.0f;
    for (int r = 0; r < RG; ++r) c += part[r][v / 4][v % 4];
    a.Cv[static_cast<size_t>(t) * DM + v] = c / den;
  }
  if (tid == 0) a.DEN[t] = den;
}

// F2
template <typename T>
__global__ __launch_bounds__(RB_BT) void rbwd_f2(RouterBwdArgs a) {
  constexpr int LX = RB_MAXX + 1, LH = RB_MAXH + 1, LM = RB_MAXM + 1;
  __shared__ float xth[RB_TB][LX];    // [s; c; nu]
  __shared__ float dxth[RB_TB][LX];   // P's head part for a while, then [ds; dc; dnu]
  __shared__ float pa[RB_TB][LH];     // f_theta's hidden pre-activation, then dL/dpre_a
  __shared__ float u1[RB_TB][LM];     // W_n s, then dL/du1
  __shared__ float u2[RB_TB][LM];     // W_c c, then dL/du2
  // bf16: split copies of [s; c], then dL/dpre_a, then dL/du1 and dL/du2, each written where the
  // value is produced (the transposed products as row products over the transposed weights; red
  // then only holds the normaliser's products)
  constexpr bool kB = std::is_same<T, bf16_t>::value;
  constexpr int XW = kB ? std::max(rb_split_pitch(RB_MAXS + RB_MAXM), 2 * rb_split_pitch(RB_MAXM)) : 0;
  __shared__ __attribute__((aligned(16))) bf16_t xsp[kB ? 2 * RB_TB * XW : 8];
  __shared__ float red[kB ? RB_TB * RB_MAXM : RB_RED];
  bf16_t *bh = xsp, *bl = xsp + RB_TB * XW;
  const int xpx = rb_split_pitch(a.d_s + a.d_m), xph = rb_split_pitch(a.d_head), xpu = rb_split_pitch(a.d_m);
  __shared__ float hv[3][RB_MAXH];    // th1's nu column, th2, psi_2
  __shared__ float nrm[RB_TB][4];     // n1, n2, nn, Dc
  __shared__ float dens[RB_TB];       // the memory read's normaliser
  __shared__ float tsc[RB_TB][4];     // dL/dlogit, m_{j-1}, dL/dp, dL/dm
  __shared__ float dab[RB_TB][2];     // dL/da, dL/db
  static_assert(RB_RED >= RB_TB * RB_MAXM, "phi(q) zeta products");
  const int tid = threadIdx.x, lane = tid & (kWave - 1), wv = wave_id();
  const int T_ = a.T, j = a.j, DM = a.d_m, d_s = a.d_s, d_e = a.d_e, d_head = a.d_head;
  const int NP = d_e + d_head, d_x = d_s + DM + 1;
  const int t0 = a.t_begin + static_cast<int>(blockIdx.x) * RB_TB, nb = min(RB_TB, a.t_end - t0);
  // s, c, W_n s, P's head part (loads first, clamped to the last element), the heads' vectors
  {
    constexpr int US = (RB_TB * RB_MAXS + RB_BT - 1) / RB_BT, UM = (RB_TB * RB_MAXM + RB_BT - 1) / RB_BT;
    constexpr int UH = (RB_TB * RB_MAXH + RB_BT - 1) / RB_BT;
    const int ns = nb * d_s, nm = nb * DM, nh = nb * d_head;
    float vs[US], vc[UM], vu[UM], vh[UH], vq[UM], vz[UM], sc[4] = {0.0f, 1.0f, 0.0f, 0.0f};
#pragma unroll
    for (int u = 0; u < US; ++u) {
      const int e = min(tid + u * RB_BT, ns - 1), k = e / nb, b = e % nb;
      vs[u] = a.XT[static_cast<size_t>(k) * T_ + t0 + b];
    }
#pragma unroll
    for (int u = 0; u < UM; ++u) {
      const int e = min(tid + u * RB_BT, nm - 1), b = e / DM, k = e % DM;
      vc[u] = a.Cv[static_cast<size_t>(t0 + b) * DM + k];
      vu[u] = a.QKVU[static_cast<size_t>(t0 + b) * 4 * DM + 3 * DM + k];
      if (a.c_given) {   // for the read's normaliser phi(q)^T zeta_{j-1} + eps
        vq[u] = a.QKVU[static_cast<size_t>(t0 + b) * 4 * DM + k];
        vz[u] = a.zeta_in[static_cast<size_t>(t0 + b) * DM + k];
      }
    }
    if (tid < nb) {
      const int t = t0 + tid;
      sc[0] = a.dlogit[t];
      if (j > 1) sc[1] = a.m_in[t];
      sc[2] = a.dp[t];
      sc[3] = a.dm[t];
      if (!a.c_given) dens[tid] = a.DEN[t];
    }
#pragma unroll
    for (int u = 0; u < UH; ++u) {
      const int e = min(tid + u * RB_BT, nh - 1), b = e / d_head, o = e % d_head;
      vh[u] = a.PSUM[static_cast<size_t>(t0 + b) * NP + d_e + o];
    }
    for (int o = tid; o < d_head; o += RB_BT) {
      hv[0][o] = ldf(static_cast<const T*>(a.th1) + static_cast<size_t>(o) * a.ld_th1 + d_s + DM);
      hv[1][o] = ldf(static_cast<const T*>(a.th2) + o);
      hv[2][o] = ldf(static_cast<const T*>(a.ps2) + o);
    }
#pragma unroll
    for (int u = 0; u < US; ++u) {
      const int e = tid + u * RB_BT, k = e / nb, b = e % nb;
      if (e < ns) {
        xth[b][k] = vs[u];
        if (kB) put_split(bh, bl, b * xpx + k, vs[u]);
      }
    }
#pragma unroll
    for (int u = 0; u < UM; ++u) {
      const int e = tid + u * RB_BT, b = e / DM, k = e % DM;
      if (e < nm) {
        xth[b][d_s + k] = vc[u];
        if (kB) put_split(bh, bl, b * xpx + d_s + k, vc[u]);
        u1[b][k] = vu[u];
        if (a.c_given) red[b * DM + k] = phi_hw(vq[u]) * vz[u];
      }
    }
    if (tid < nb)
      for (int x = 0; x < 4; ++x) tsc[tid][x] = sc[x];
#pragma unroll
    for (int u = 0; u < UH; ++u) {
      const int e = tid + u * RB_BT, b = e / d_head, o = e % d_head;
      if (e < nh) dxth[b][o] = vh[u];
    }
  }
  __syncthreads();
  // W_c c and f_theta's first layer over [s; c] (nu's column is added with the head below)
  for (int e = tid; e < nb * DM; e += RB_BT) {
    const int k = d_s + e / nb, b = e % nb;
    a.XT[static_cast<size_t>(k) * T_ + t0 + b] = xth[b][k];
  }
  if constexpr (kB) {
    bmv16(one16(a.w_c, DM, DM), DM, DM, bh + d_s, bl + d_s, xpx, &u2[0][0], LM, nb, false);
    bmv16(one16(a.th1, d_head, a.ld_th1), d_head, d_s + DM, bh, bl, xpx, &pa[0][0], LH, nb, false);
  } else {
    bmv_rows(mats1<T>(a.w_c, DM, DM), DM, DM, &xth[0][d_s], LX, &u2[0][0], LM, nb);
    bmv_rows(mats1<T>(a.th1, d_head, a.ld_th1), d_head, d_s + DM, &xth[0][0], LX, &pa[0][0], LH, nb);
  }
  __syncthreads();
  // a wave per token: nu = 1 - cos(W_n s, W_c c); the history head a = th2 . SiLU(pre_a),
  // p = sigma(a / T_hist); dL/da, dL/db; dL/dP's head part in its token-major row
  for (int b = wv; b < nb; b += RB_BW) {
    const int t = t0 + b;
    float den = 0.0f;
    if (a.c_given) {
      for (int k = lane; k < DM; k += kWave) den += red[b * DM + k];
      den = wave_sum_dpp(den) + a.eps;
    }
    float n1 = 0.0f, n2 = 0.0f, nn = 0.0f;
    for (int k = lane; k < DM; k += kWave) {
      n1 = fmaf(u1[b][k], u1[b][k], n1);
      n2 = fmaf(u2[b][k], u2[b][k], n2);
      nn = fmaf(u1[b][k], u2[b][k], nn);
    }
    n1 = sqrtf(wave_sum_dpp(n1));
    n2 = sqrtf(wave_sum_dpp(n2));
    nn = wave_sum_dpp(nn);
    const float Dc = n1 * n2 + a.eps;
    const float nu = j > 1 ? 1.0f - nn / Dc : 0.0f;
    float aa = 0.0f;
    for (int o = lane; o < d_head; o += kWave) {
      const float pre = fmaf(hv[0][o], nu, pa[b][o]);
      pa[b][o] = pre;
      aa = fmaf(hv[1][o], silu_hw(pre), aa);
    }
    aa = wave_sum_dpp(aa);
    const float p = sigmoid_hw(aa / a.T_hist);
    const float dl = tsc[b][0], m_prev = tsc[b][1];
    const float da = dl + (tsc[b][2] + tsc[b][3] * m_prev) * p * (1.0f - p) / a.T_hist;
    for (int o = lane; o < d_head; o += kWave)
      a.dP[static_cast<size_t>(t) * NP + d_e + o] = dl * hv[2][o] * silu_grad_hw(dxth[b][o]);
    if (lane == 0) {
      if (a.c_given) dens[b] = den;
      nrm[b][0] = n1;
      nrm[b][1] = n2;
      nrm[b][2] = nn;
      nrm[b][3] = Dc;
      xth[b][d_s + DM] = nu;
      dab[b][0] = da;
      dab[b][1] = dl;
      a.PS[t] = p;
      a.DA[t] = da;
      a.DB[t] = dl;
    }
  }
  __syncthreads();
  // the heads' pre-activation gradients, token-contiguous: dL/dpre_a (over pa, in place), dL/dpre_b
  for (int e = tid; e < nb * d_head; e += RB_BT) {
    const int o = e / nb, b = e % nb, t = t0 + b;
    const float x = pa[b][o];
    a.SAT[static_cast<size_t>(o) * T_ + t] = silu_hw(x);
    const float g = dab[b][0] * hv[1][o] * silu_grad_hw(x);
    a.dPAT[static_cast<size_t>(o) * T_ + t] = g;
    pa[b][o] = g;
    if (kB) put_split(bh, bl, b * xph + o, g);
    const float pb = dxth[b][o];
    a.dPT[static_cast<size_t>(d_e + o) * T_ + t] = dab[b][1] * hv[2][o] * silu_grad_hw(pb);
    a.SBT[static_cast<size_t>(o) * T_ + t] = silu_hw(pb);
  }
  if (tid < nb) a.XT[static_cast<size_t>(d_s + DM) * T_ + t0 + tid] = xth[tid][d_s + DM];
  __syncthreads();
  // [ds; dc; dnu] = th1^T dL/dpre_a
  if constexpr (kB) {
    bmv16(one16(a.th1T, d_x, d_head), d_x, d_head, bh, bl, xph, &dxth[0][0], LX, nb, false);
  } else {
    bmv_cols(Cols<T>{mats1<T>(a.th1, d_head, a.ld_th1), d_head, d_x, &pa[0][0], LH, &dxth[0][0], LX, false}, nb, red);
  }
  __syncthreads();
  // nu's cosine backward (a constant at j = 1)
  for (int e = tid; e < nb * DM; e += RB_BT) {
    const int k = e / nb, b = e % nb, t = t0 + b;
    const float n1 = nrm[b][0], n2 = nrm[b][1], nn = nrm[b][2], Dc = nrm[b][3];
    const float dcos = j > 1 ? -dxth[b][d_s + DM] : 0.0f;
    const float q_ = nn / (Dc * Dc);
    const float a1 = u1[b][k], a2 = u2[b][k];
    const float g1 = dcos * (a2 / Dc - q_ * n2 * (n1 > 0.0f ? a1 / n1 : 0.0f));
    const float g2 = dcos * (a1 / Dc - q_ * n1 * (n2 > 0.0f ? a2 / n2 : 0.0f));
    u1[b][k] = g1;
    u2[b][k] = g2;
    if (kB) {
      put_split(bh, bl, b * xpu + k, g1);
      put_split(bh + RB_TB * xpu, bl + RB_TB * xpu, b * xpu + k, g2);
    }
    a.dU1T[static_cast<size_t>(k) * T_ + t] = g1;
    a.dU2T[static_cast<size_t>(k) * T_ + t] = g2;
  }
  __syncthreads();
  // ds += W_n^T du1, dc += W_c^T du2
  if constexpr (kB) {
    const int h2 = RB_TB * xpu;
    bmv16(one16(a.wnT, d_s, DM), d_s, DM, bh, bl, xpu, &dxth[0][0], LX, nb, true);
    bmv16(one16(a.wcT, DM, DM), DM, DM, bh + h2, bl + h2, xpu, &dxth[0][d_s], LX, nb, true);
  } else {
    bmv_cols2(Cols<T>{mats1<T>(a.w_n, DM, d_s), DM, d_s, &u1[0][0], LM, &dxth[0][0], LX, true},
              Cols<T>{mats1<T>(a.w_c, DM, DM), DM, DM, &u2[0][0], LM, &dxth[0][d_s], LX, true}, true, nb, red);
  }
  __syncthreads();
  // the read's normaliser: dL/dnum = dc / den, dL/dden = -<dc, c> / den (no read at j = 1)
  for (int b = wv; b < nb; b += RB_BW) {
    const int t = t0 + b;
    const float den = dens[b];
    float dden = 0.0f;
    for (int v = lane; v < DM; v += kWave) {
      a.DNUM[static_cast<size_t>(t) * DM + v] = j > 1 ? dxth[b][d_s + v] / den : 0.0f;
      dden += j > 1 ? -dxth[b][d_s + v] * xth[b][d_s + v] / den : 0.0f;
    }
    dden = wave_sum_dpp(dden);
    if (lane == 0) a.DDEN[t] = dden;
  }
  for (int e = tid; e < nb * d_s; e += RB_BT) {
    const int b = e / d_s, k = e % d_s;
    a.DSP[static_cast<size_t>(t0 + b) * d_s + k] = dxth[b][k];
  }
}

// M2: the pass over S_{j-1} and dL/dS_j of one token.  LPR lanes hold a row's DM columns as float4s
// (RPW rows per wave at a time); row sums by shuffles within the LPR lanes, column sums over the
// waves' row sets added in order.  The three state streams carry the non-temporal hint, as in M1.
template <int DM>
__global__ __launch_bounds__(RB_NT) void rbwd_spass(RouterBwdArgs a) {
  constexpr int LPR = DM / 4 < kWave ? DM / 4 : kWave, RPW = kWave / LPR, RSETS = RB_NW * RPW;
  __shared__ float fq[DM], fk[DM], vv[DM], dn[DM], zi[DM];
  __shared__ float sk[DM], sq[DM];
  __shared__ f32x4 dvp[RSETS][LPR];
  __shared__ float red[RB_NW];
  const int t = a.t_begin + static_cast<int>(blockIdx.x), tid = threadIdx.x, lane = tid & (kWave - 1), wv = wave_id();
  const int j = a.j;
  const float* qkv = a.QKVU + static_cast<size_t>(t) * 4 * DM;
  for (int k = tid; k < DM; k += RB_NT) {
    fq[k] = phi_hw(qkv[k]);
    fk[k] = phi_hw(qkv[DM + k]);
    vv[k] = qkv[2 * DM + k];
    dn[k] = a.DNUM[static_cast<size_t>(t) * DM + k];
    zi[k] = j > 1 ? a.zeta_in[static_cast<size_t>(t) * DM + k] : 0.0f;
  }
  __syncthreads();
  const float dden = a.DDEN[t], rho = a.rho;
  const int cg = lane % LPR, rset = wv * RPW + lane / LPR;
  f32x4* dS = reinterpret_cast<f32x4*>(a.dS + static_cast<size_t>(t) * DM * DM) + cg;
  const f32x4* Sin = j > 1 ? reinterpret_cast<const f32x4*>(a.S_in + static_cast<size_t>(t) * DM * DM) + cg : nullptr;
  const f32x4 v4 = {vv[4 * cg], vv[4 * cg + 1], vv[4 * cg + 2], vv[4 * cg + 3]};
  const f32x4 n4 = {dn[4 * cg], dn[4 * cg + 1], dn[4 * cg + 2], dn[4 * cg + 3]};
  f32x4 dva = {0.0f, 0.0f, 0.0f, 0.0f};
  float rho_acc = 0.0f;
#pragma unroll 4
  for (int it = 0; it < DM / RSETS; ++it) {
    const int k = rset + it * RSETS;
    const size_t o = static_cast<size_t>(k) * (DM / 4);
    const f32x4 g = __builtin_nontemporal_load(dS + o);
    const f32x4 sv = Sin ? __builtin_nontemporal_load(Sin + o) : f32x4{0.0f, 0.0f, 0.0f, 0.0f};
    float rk = g[0] * v4[0] + g[1] * v4[1] + g[2] * v4[2] + g[3] * v4[3];
    float rq = sv[0] * n4[0] + sv[1] * n4[1] + sv[2] * n4[2] + sv[3] * n4[3];
    rho_acc += g[0] * sv[0] + g[1] * sv[1] + g[2] * sv[2] + g[3] * sv[3];
    dva += fk[k] * g;
    __builtin_nontemporal_store(rho * g + fq[k] * n4, dS + o);
#pragma unroll
    for (int off = LPR / 2; off > 0; off >>= 1) {
      rk += __shfl_xor(rk, off, kWave);
      rq += __shfl_xor(rq, off, kWave);
    }
    if (cg == 0) {
      sk[k] = rk;
      sq[k] = rq;
    }
  }
  dvp[rset][cg] = dva;
  __syncthreads();
  // zeta: its share of dL/drho and dL/dzeta_{j-1} in place, after dL/dphi(k) read the incoming value
  float* dz = a.dzeta + static_cast<size_t>(t) * DM;
  float* df = a.DF + static_cast<size_t>(t) * 3 * DM;
  for (int k = tid; k < DM; k += RB_NT) {
    const float g = dz[k];
    float dv = 0.0f;
    for (int r = 0; r < RSETS; ++r) dv += dvp[r][k / 4][k % 4];
    df[k] = sk[k] + g;
    df[DM + k] = sq[k] + zi[k] * dden;
    df[2 * DM + k] = dv;
    rho_acc = fmaf(g, zi[k], rho_acc);
    dz[k] = fmaf(rho, g, fq[k] * dden);
  }
  rho_acc = block_sum(rho_acc, red);
  if (tid == 0) a.rho_part[t] = rho_acc;
}

// F3
template <typename T>
__global__ __launch_bounds__(RB_BT) void rbwd_f3(RouterBwdArgs a) {
  constexpr int LQ = 3 * RB_MAXM + 1, LS = RB_MAXS + 1, LP = RB_MAXP + 1, LE = RB_MAXE + 1;
  static_assert(LQ >= RB_MAXE, "dqkv holds P's hidden part at the end");
  __shared__ float dqkv[RB_TB][LQ];   // [dL/dq; dL/dk; dL/dv], later P's hidden part
  __shared__ float ds[RB_TB][LS];
  __shared__ float dpp[RB_TB][LP];
  __shared__ float dxp[RB_TB][8];
  __shared__ float dsh[RB_TB][LE];
  // bf16: split copies of [dq; dk; dv] (written as they are formed), then of dz^a and dz^h (the
  // transposed products as row products over the transposed weights); fp32: red for the
  // transposed products' partial sums
  constexpr bool kB = std::is_same<T, bf16_t>::value;
  constexpr int XW = kB ? rb_split_pitch(3 * RB_MAXM) : 0;
  static_assert(!kB || XW >= 2 * rb_split_pitch(RB_MAXS), "dz^a and dz^h side by side");
  __shared__ __attribute__((aligned(16))) bf16_t xsp[kB ? 2 * RB_TB * XW : 8];
  __shared__ float red[kB ? 1 : RB_RED];
  bf16_t *bh = xsp, *bl = xsp + RB_TB * XW;
  const int xpq = rb_split_pitch(3 * a.d_m);
  __shared__ float wp1[RB_MAXP * 6];
  __shared__ float cnv[RB_TB], irs[RB_TB];
  const int tid = threadIdx.x, lane = tid & (kWave - 1), wv = wave_id();
  const int T_ = a.T, j = a.j, DM = a.d_m, d_s = a.d_s, d_h = a.d_h, d_a = a.d_a, d_e = a.d_e, d_p = a.d_p;
  const int NP = d_e + a.d_head;
  const int t0 = a.t_begin + static_cast<int>(blockIdx.x) * RB_TB, nb = min(RB_TB, a.t_end - t0);
  // dL/dq, dL/dk through phi (phi'(x) = 1 for x > 0, exp(x) otherwise), dL/dv, dL/ds so far; P's
  // hidden part waits in registers (loads first, clamped to the last element)
  constexpr int UE = (RB_TB * RB_MAXE + RB_BT - 1) / RB_BT;
  const int ne = nb * d_e;
  float ph[UE];
  {
    constexpr int UM = (RB_TB * RB_MAXM + RB_BT - 1) / RB_BT, US = (RB_TB * RB_MAXS + RB_BT - 1) / RB_BT;
    const int nm = nb * DM, ns = nb * d_s;
    float fq_[UM], fk_[UM], gq[UM], gk[UM], gv[UM], gs[US];
#pragma unroll
    for (int u = 0; u < UM; ++u) {
      const int e = min(tid + u * RB_BT, nm - 1), b = e / DM, k = e % DM, t = t0 + b;
      const float* qkv = a.QKVU + static_cast<size_t>(t) * 4 * DM;
      const float* df = a.DF + static_cast<size_t>(t) * 3 * DM;
      fq_[u] = qkv[k];
      fk_[u] = qkv[DM + k];
      gk[u] = df[k];
      gq[u] = df[DM + k];
      gv[u] = df[2 * DM + k];
    }
#pragma unroll
    for (int u = 0; u < US; ++u) {
      const int e = min(tid + u * RB_BT, ns - 1), b = e / d_s, k = e % d_s;
      gs[u] = a.DSP[static_cast<size_t>(t0 + b) * d_s + k];
    }
#pragma unroll
    for (int u = 0; u < UE; ++u) {
      const int e = min(tid + u * RB_BT, ne - 1), b = e / d_e, k = e % d_e;
      ph[u] = a.PSUM[static_cast<size_t>(t0 + b) * NP + k];
    }
    for (int e = tid; e < d_p * 6; e += RB_BT) wp1[e] = ldf(static_cast<const T*>(a.w_p1) + e);
    if (tid < nb) irs[tid] = a.RS[static_cast<size_t>(t0 + tid) * 4];
#pragma unroll
    for (int u = 0; u < UM; ++u) {
      const int e = tid + u * RB_BT, b = e / DM, k = e % DM;
      if (e < nm) {
        const float q = gq[u] * phi_grad_hw(fq_[u]), kk = gk[u] * phi_grad_hw(fk_[u]);
        dqkv[b][k] = q;
        dqkv[b][DM + k] = kk;
        dqkv[b][2 * DM + k] = gv[u];
        if (kB) {
          put_split(bh, bl, b * xpq + k, q);
          put_split(bh, bl, b * xpq + DM + k, kk);
          put_split(bh, bl, b * xpq + 2 * DM + k, gv[u]);
        }
      }
    }
#pragma unroll
    for (int u = 0; u < US; ++u) {
      const int e = tid + u * RB_BT, b = e / d_s, k = e % d_s;
      if (e < ns) ds[b][k] = gs[u];
    }
  }
  __syncthreads();
  for (int e = tid; e < nb * DM; e += RB_BT) {
    const int k = e / nb, b = e % nb, t = t0 + b;
    a.dQT[static_cast<size_t>(k) * T_ + t] = dqkv[b][k];
    a.dKT[static_cast<size_t>(k) * T_ + t] = dqkv[b][DM + k];
    a.dVT[static_cast<size_t>(k) * T_ + t] = dqkv[b][2 * DM + k];
  }
  // ds += [W_q; W_k; W_v]^T [dq; dk; dv] in one stacked product
  const Mats<T> qkv{static_cast<const T*>(a.w_q), static_cast<const T*>(a.w_k), static_cast<const T*>(a.w_v), nullptr,
                    DM, d_s};
  if constexpr (kB) {
    bmv16(one16(a.wqkvT, d_s, 3 * DM), d_s, 3 * DM, bh, bl, xpq, &ds[0][0], LS, nb, true);
  } else {
    bmv_cols(Cols<T>{qkv, 3 * DM, d_s, &dqkv[0][0], LQ, &ds[0][0], LS, true}, nb, red);
  }
  __syncthreads();
  for (int e = tid; e < nb * d_s; e += RB_BT) {
    const int k = e / nb, b = e % nb, t = t0 + b;
    if (k < d_h)
      a.dZHT[static_cast<size_t>(k) * T_ + t] = ds[b][k];
    else
      a.dZAT[static_cast<size_t>(k - d_h) * T_ + t] = ds[b][k];
  }
  // dL/dSiLU(pre_p) = W_p2^T dz^a and dL/dSiLU(pre_h) = W_hu^T dz^h
  if constexpr (kB) {
    const int xa = rb_split_pitch(a.ld_ta), xh = rb_split_pitch(a.ld_th), h2 = RB_TB * xa;
    split_x(&ds[0][d_h], LS, d_a, a.ld_ta, nb, bh, bl, xa);   // (the weights' pad columns meet zeros)
    split_x(&ds[0][0], LS, d_h, a.ld_th, nb, bh + h2, bl + h2, xh);
    __syncthreads();
    bmv16(one16(a.wp2T, d_p, a.ld_ta), d_p, a.ld_ta, bh, bl, xa, &dpp[0][0], LP, nb, false);
    bmv16(one16(a.whuT, d_e, a.ld_th), d_e, a.ld_th, bh + h2, bl + h2, xh, &dsh[0][0], LE, nb,
          false);
  } else {
    bmv_cols2(Cols<T>{mats1<T>(a.w_p2, d_a, d_p), d_a, d_p, &ds[0][d_h], LS, &dpp[0][0], LP, false},
              Cols<T>{mats1<T>(a.w_hu, d_h, d_e), d_h, d_e, &ds[0][0], LS, &dsh[0][0], LE, false}, true, nb, red);
  }
  __syncthreads();
  for (int e = tid; e < nb * d_p; e += RB_BT) {
    const int o = e / nb, b = e % nb, t = t0 + b;
    const float g = dpp[b][o] * silu_grad_hw(a.PPRE[static_cast<size_t>(t) * d_p + o]);
    dpp[b][o] = g;
    a.dPPT[static_cast<size_t>(o) * T_ + t] = g;
  }
  // dL/dP's hidden part, ir SiLU'(ir P_h) dL/dSiLU, in the token-major rows (P_h waits in dqkv,
  // dL/dpre_h in dsh, for the token-contiguous writes)
#pragma unroll
  for (int u = 0; u < UE; ++u) {
    const int e = tid + u * RB_BT, b = e / d_e, k = e % d_e, t = t0 + b;
    if (e < ne) {
      const float ir = irs[b];
      const float dph = dsh[b][k] * silu_grad_hw(ir * ph[u]);
      dqkv[b][k] = ph[u];
      dsh[b][k] = dph;
      a.dP[static_cast<size_t>(t) * NP + k] = ir * dph;
    }
  }
  __syncthreads();
  // the six path features' gradients W_p1^T dL/dpre_p and the RMSNorm coefficient's
  // sum_e dph_e P_h,e, a wave per (token, feature) and per token
  for (int idx = wv; idx < nb * 6; idx += RB_BW) {
    const int b = idx / 6, k = idx % 6;
    float sacc = 0.0f;
    for (int o = lane; o < d_p; o += kWave) sacc = fmaf(wp1[o * 6 + k], dpp[b][o], sacc);
    sacc = wave_sum_dpp(sacc);
    if (lane == 0) dxp[b][k] = sacc;
  }
  for (int b = wv; b < nb; b += RB_BW) {
    float cn = 0.0f;
    for (int k = lane; k < d_e; k += kWave) cn = fmaf(dsh[b][k], dqkv[b][k], cn);
    cn = wave_sum_dpp(cn);
    if (lane == 0) cnv[b] = cn;
  }
  for (int e = tid; e < nb * d_e; e += RB_BT) {
    const int k = e / nb, b = e % nb, t = t0 + b;
    const float ir = irs[b];
    a.dPT[static_cast<size_t>(k) * T_ + t] = ir * dsh[b][k];
    a.SHT[static_cast<size_t>(k) * T_ + t] = silu_hw(ir * dqkv[b][k]);
  }
  __syncthreads();
  if (tid < nb) {
    const int b = tid, t = t0 + b;
    const float* rs = a.RS + static_cast<size_t>(t) * 4;
    const float ir = rs[0], nd = rs[1], np_ = rs[2], dpv = rs[3];
    // transitions: d_j = |delta_j| (j >= 2), gamma_j = cos(delta_j, delta_{j-1}) (j >= 3)
    const float ddj = dxp[b][2], dg = dxp[b][3];
    float c1 = 0.0f, c2 = 0.0f, c3 = 0.0f, c4 = 0.0f;
    if (j >= 2 && nd > 0.0f) c1 += ddj / nd;
    if (j >= 3) {
      const float D = nd * np_ + a.eps, q_ = dpv / (D * D);
      c2 += dg / D;
      c3 += dg / D;
      if (nd > 0.0f) c1 -= dg * q_ * np_ / nd;
      if (np_ > 0.0f) c4 -= dg * q_ * nd / np_;
    }
    float* rc = a.rowcoef + static_cast<size_t>(t) * 8;
    rc[0] = -(ir * ir * ir / static_cast<float>(a.d)) * cnv[b];
    rc[1] = c1;
    rc[2] = c2;
    rc[3] = c3;
    rc[4] = c4;
    const float p = a.PS[t];
    a.dm[t] = a.dm[t] * p + dxp[b][5];
    a.dp[t] = dxp[b][4];
  }
}

// the per-row RMSNorm and transition terms of dL/dhbar (one workgroup per token; eight elements a
// thread per step through 16-byte accesses: d is a multiple of 128 and the rows 16-byte aligned)
__device__ __forceinline__ void rows_rmw8(float* p, const float* v) {
  f32x4* q = reinterpret_cast<f32x4*>(p);
  f32x4 u0 = q[0], u1 = q[1];
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    u0[k] += v[k];
    u1[k] += v[4 + k];
  }
  q[0] = u0;
  q[1] = u1;
}
template <typename T>
__global__ __launch_bounds__(256) void router_bwd_rows(RouterBwdArgs a) {
  const int t = blockIdx.x, j = a.j, d = a.d;
  const float* rc = a.rowcoef + static_cast<size_t>(t) * 8;
  const float cnorm = rc[0], c1 = rc[1], c2 = rc[2], c3 = rc[3], c4 = rc[4];
  const size_t row = static_cast<size_t>(t) * d;
  const T* hb = static_cast<const T*>(a.hbar) + row;
  const T* h1 = j >= 2 ? static_cast<const T*>(a.prev1) + row : nullptr;
  const T* h2 = j >= 3 ? static_cast<const T*>(a.prev2) + row : nullptr;
  for (int i = threadIdx.x * 8; i < d; i += 256 * 8) {
    float x[8], y[8], z[8], g0[8], g1[8], g2[8];
    ld8(hb + i, x);
    if (j >= 2) ld8(h1 + i, y);
    if (j >= 3) ld8(h2 + i, z);
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      const float yk = j >= 2 ? y[k] : x[k], zk = j >= 3 ? z[k] : yk;
      const float del = x[k] - yk, delp = yk - zk;
      const float gj = c1 * del + c2 * delp, gp = c3 * del + c4 * delp;
      g0[k] = cnorm * x[k] + gj;
      g1[k] = gp - gj;
      g2[k] = -gp;
    }
    rows_rmw8(a.dhbar + row + i, g0);
    if (j >= 2) rows_rmw8(a.dhbar1 + row + i, g1);
    if (j >= 3) rows_rmw8(a.dhbar2 + row + i, g2);
  }
}

// The transposed bf16 weights of the batched passes (bf16 storage): one element a thread, written
// in order, gathered from the row-major weights (about 0.1 M elements at the 8B shape)
__global__ __launch_bounds__(256) void rbwd_wt(RouterBwdArgs a) {
  const int DM = a.d_m, d_s = a.d_s, d_x = d_s + DM + 1, dh = a.d_head, d_p = a.d_p, d_a = a.d_a, d_h = a.d_h;
  const int d_e = a.d_e, ta = a.ld_ta, th = a.ld_th;
  const int n0 = d_x * dh, n1 = n0 + d_s * DM, n2 = n1 + DM * DM, n3 = n2 + d_s * 3 * DM, n4 = n3 + d_p * ta;
  const int n5 = n4 + d_e * th;
  const bf16_t* th1 = static_cast<const bf16_t*>(a.th1);
  for (int e = static_cast<int>(blockIdx.x * blockDim.x + threadIdx.x); e < n5;
       e += static_cast<int>(gridDim.x * blockDim.x)) {
    if (e < n0) {
      const int k = e / dh, o = e % dh;
      a.th1T[e] = th1[static_cast<size_t>(o) * a.ld_th1 + k];
    } else if (e < n1) {
      const int f = e - n0, k = f / DM, o = f % DM;
      a.wnT[f] = static_cast<const bf16_t*>(a.w_n)[o * d_s + k];
    } else if (e < n2) {
      const int f = e - n1, k = f / DM, o = f % DM;
      a.wcT[f] = static_cast<const bf16_t*>(a.w_c)[o * DM + k];
    } else if (e < n3) {
      const int f = e - n2, k = f / (3 * DM), c = f % (3 * DM), m = c / DM, o = c % DM;
      const void* w = m == 0 ? a.w_q : m == 1 ? a.w_k : a.w_v;
      a.wqkvT[f] = static_cast<const bf16_t*>(w)[o * d_s + k];
    } else if (e < n4) {
      const int f = e - n3, k = f / ta, o = f % ta;
      a.wp2T[f] = o < d_a ? static_cast<const bf16_t*>(a.w_p2)[o * d_p + k] : bf16_t{0};
    } else {
      const int f = e - n4, k = f / th, o = f % th;
      a.whuT[f] = o < d_h ? static_cast<const bf16_t*>(a.w_hu)[o * d_e + k] : bf16_t{0};
    }
  }
}

// dL/deta = rho (1 - rho) sum_t rho_part[t], summed in a fixed order (one workgroup)
constexpr int RB_DETA_NT = 1024;
__global__ __launch_bounds__(RB_DETA_NT) void router_bwd_deta(const float* __restrict__ part, int T, float rho,
                                                             float* __restrict__ deta) {
  constexpr int U = 8;   // loads in flight per thread
  __shared__ float red[RB_DETA_NT / kWave];
  // thread i adds its contiguous run of ceil(T / RB_DETA_NT) entries in order
  const int C = (T + RB_DETA_NT - 1) / RB_DETA_NT, b0 = static_cast<int>(threadIdx.x) * C, b1 = min(b0 + C, T);
  float s = 0.0f;
  for (int t = b0; t < b1; t += U) {
    float v[U];
#pragma unroll
    for (int u = 0; u < U; ++u) v[u] = t + u < b1 ? part[t + u] : 0.0f;
#pragma unroll
    for (int u = 0; u < U; ++u) s += v[u];
  }
  s = wave_sum_dpp(s);
  if ((threadIdx.x & (kWave - 1)) == 0) red[threadIdx.x / kWave] = s;
  __syncthreads();
  if (threadIdx.x == 0) {
    float tot = 0.0f;
    for (int w = 0; w < RB_DETA_NT / kWave; ++w) tot += red[w];
    deta[0] = rho * (1.0f - rho) * tot;
  }
}

// out[c][r] = float(in[r][c]) for r < R, c < C (64 x 64 tiles through LDS)
template <typename T>
__global__ __launch_bounds__(256) void to_f32_transpose(const T* __restrict__ in, int R, int C, int ld_in,
                                                       float* __restrict__ out, int ld_out) {
  __shared__ float tile[64][65];
  const int c0 = blockIdx.x * 64, r0 = blockIdx.y * 64;
  const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;
  for (int i = ty; i < 64; i += 4) {
    const int r = r0 + i, c = c0 + tx;
    tile[i][tx] = (r < R && c < C) ? ldf(in + static_cast<size_t>(r) * ld_in + c) : 0.0f;
  }
  __syncthreads();
  for (int i = ty; i < 64; i += 4) {
    const int c = c0 + i, r = r0 + tx;
    if (c < C && r < R) out[static_cast<size_t>(c) * ld_out + r] = tile[tx][i];
  }
}

// part[z][m][n] = sum_{k in chunk z} A[m][k] B[n][k] (64 x 64 output tiles, 4 x 4 per thread, every
// access bounds-checked; chunk z covers k in [z kc, min(K, (z + 1) kc)))
__global__ __launch_bounds__(256) void tn_part_kernel(const float* __restrict__ A, int lda, int M,
                                                     const float* __restrict__ B, int ldb, int N, int K, int kc,
                                                     float* __restrict__ part) {
  __shared__ float As[16][68];
  __shared__ float Bs[16][68];
  const int m0 = blockIdx.y * 64, n0 = blockIdx.x * 64, z = blockIdx.z;
  const int k_lo = z * kc, k_hi = min(K, k_lo + kc);
  const int tx = threadIdx.x & 15, ty = threadIdx.x >> 4;
  float acc[4][4] = {};
  for (int k0 = k_lo; k0 < k_hi; k0 += 16) {
    for (int e = threadIdx.x; e < 64 * 16; e += 256) {
      const int r = e >> 4, kk = e & 15, k = k0 + kk;
      As[kk][r] = (m0 + r < M && k < k_hi) ? A[static_cast<size_t>(m0 + r) * lda + k] : 0.0f;
      Bs[kk][r] = (n0 + r < N && k < k_hi) ? B[static_cast<size_t>(n0 + r) * ldb + k] : 0.0f;
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < 16; ++kk)
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int jj = 0; jj < 4; ++jj) acc[i][jj] = fmaf(As[kk][ty * 4 + i], Bs[kk][tx * 4 + jj], acc[i][jj]);
    __syncthreads();
  }
  float* P = part + static_cast<size_t>(z) * M * N;
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int jj = 0; jj < 4; ++jj) {
      const int m = m0 + ty * 4 + i, n = n0 + tx * 4 + jj;
      if (m < M && n < N) P[static_cast<size_t>(m) * N + n] = acc[i][jj];
    }
}

// C[m][n] += sum_z part[z][m][n], z in order
__global__ __launch_bounds__(256) void tn_reduce_kernel(const float* __restrict__ part, int nz, int M, int N,
                                                       float* __restrict__ C, int ldc) {
  const size_t e = static_cast<size_t>(blockIdx.x) * 256 + threadIdx.x;
  if (e >= static_cast<size_t>(M) * N) return;
  float v = 0.0f;
  for (int z = 0; z < nz; ++z) v += part[static_cast<size_t>(z) * M * N + e];
  const size_t m = e / N, n = e % N;
  C[m * ldc + n] += v;
}

__global__ __launch_bounds__(256) void split_bf16_kernel(const float* __restrict__ x, int R, int C, int ld_in,
                                                        bf16_t* __restrict__ hi, bf16_t* __restrict__ lo, int C_pad) {
  const size_t n = static_cast<size_t>(R) * C_pad;
  for (size_t e = static_cast<size_t>(blockIdx.x) * 256 + threadIdx.x; e < n;
       e += static_cast<size_t>(gridDim.x) * 256) {
    const size_t r = e / C_pad;
    const int c = static_cast<int>(e % C_pad);
    const float v = c < C ? x[r * ld_in + c] : 0.0f;
    const bf16_t h = f32_to_bf16(v);
    hi[e] = h;
    lo[e] = f32_to_bf16(v - bf16_to_f32(h));
  }
}


// The small weight-gradient products in one launch: C_p[m][n] += sum_t A_p[m][t] B_p[n][t] for every
// product p, on the fp32 matrix cores.  A workgroup takes a 64 x 64 output tile of one product and a
// chunk of kc tokens; each wave a 32 x 32 quarter as 2 x 2 MFMA tiles of 16 x 16.  Lane (r, g)
// supplies operand row r at k slot g, tokens t0 + 4 g + i for the i-th of four products, loaded as one
// float4 per operand row when the token pitch is a multiple of 4.  Rows past M or N read a clamped
// row and are never stored; tokens past the chunk enter as zeros on both sides.  With one chunk the
// tile adds into C; otherwise it writes its partial sums to part[chunk][tile][64 x 64], which
// small_products_reduce adds into C in chunk order.
struct SmallProductsArgs {
  SmallProduct p[kSmallProducts];
  int tile0[kSmallProducts + 1];   // first tile of each product (tile0[n] = tiles in all)
  int ntn[kSmallProducts];         // column tiles of each product
  int el0[kSmallProducts + 1];     // first output element of each product (el0[n] = elements in all)
  int n, T, ldk, kc, nchunks;
  float* part;
};

__device__ __forceinline__ int sp_product(const int* first, int n, int x) {
  int pi = 0;
  while (pi + 1 < n && first[pi + 1] <= x) ++pi;
  return pi;
}

__global__ __launch_bounds__(256) void small_products_kernel(SmallProductsArgs a) {
  const int nt = a.tile0[a.n];
  const int tile = static_cast<int>(blockIdx.x) % nt, c = static_cast<int>(blockIdx.x) / nt;
  const int pi = sp_product(a.tile0, a.n, tile);
  const SmallProduct P = a.p[pi];
  const int lt = tile - a.tile0[pi], tm = lt / a.ntn[pi], tn = lt % a.ntn[pi];
  const int lane = threadIdx.x & (kWave - 1), r = lane & 15, g = lane >> 4, wv = wave_id();
  const int mb = tm * 64 + (wv >> 1) * 32, nbs = tn * 64 + (wv & 1) * 32;
  const int ldk = a.ldk;
  const float* Ar[2];
  const float* Br[2];
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    Ar[h] = P.A + static_cast<size_t>(min(mb + 16 * h + r, P.M - 1)) * ldk;
    Br[h] = P.B + static_cast<size_t>(min(nbs + 16 * h + r, P.N - 1)) * ldk;
  }
  const int tb = c * a.kc, te = min(a.T, tb + a.kc);
  const f32x4 zero = {0.0f, 0.0f, 0.0f, 0.0f};
  f32x4 acc[2][2] = {{zero, zero}, {zero, zero}};
  if ((ldk & 3) == 0) {
    // 16 tokens a step, the next step's operands in flight during the current step's products
    auto load = [&](int t0, f32x4* av, f32x4* bv) {
      const int tt = t0 + 4 * g;
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        if (tt + 3 < te) {
          av[h] = *reinterpret_cast<const f32x4*>(Ar[h] + tt);
          bv[h] = *reinterpret_cast<const f32x4*>(Br[h] + tt);
        } else {
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const bool in = tt + i < te;
            const int tc = in ? tt + i : te - 1;
            const float x = Ar[h][tc], y = Br[h][tc];
            av[h][i] = in ? x : 0.0f;
            bv[h][i] = in ? y : 0.0f;
          }
        }
      }
    };
    f32x4 ac[2], bc[2];
    if (tb < te) load(tb, ac, bc);
    for (int t0 = tb; t0 < te; t0 += 16) {
      f32x4 an[2], bn[2];
      if (t0 + 16 < te) load(t0 + 16, an, bn);
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int h = 0; h < 2; ++h)
#pragma unroll
          for (int w = 0; w < 2; ++w) acc[h][w] = mfma4(ac[h][i], bc[w][i], acc[h][w]);
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        ac[h] = an[h];
        bc[h] = bn[h];
      }
    }
  } else {
    for (int t0 = tb; t0 < te; t0 += 16) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int t = t0 + 4 * g + i;
        const bool in = t < te;
        const int tc = in ? t : te - 1;
        float av[2], bv[2];
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          const float x = Ar[h][tc], y = Br[h][tc];
          av[h] = in ? x : 0.0f;
          bv[h] = in ? y : 0.0f;
        }
#pragma unroll
        for (int h = 0; h < 2; ++h)
#pragma unroll
          for (int w = 0; w < 2; ++w) acc[h][w] = mfma4(av[h], bv[w], acc[h][w]);
      }
    }
  }
  // lane (r, g) holds rows 4 g + q of column r of each 16 x 16 tile
  float* pp = a.nchunks > 1 ? a.part + (static_cast<size_t>(c) * nt + tile) * 4096 : nullptr;
#pragma unroll
  for (int h = 0; h < 2; ++h)
#pragma unroll
    for (int w = 0; w < 2; ++w)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int ml = (wv >> 1) * 32 + 16 * h + 4 * g + q, nl = (wv & 1) * 32 + 16 * w + r;
        if (pp) {
          pp[ml * 64 + nl] = acc[h][w][q];
        } else {
          const int m = tm * 64 + ml, n = tn * 64 + nl;
          if (m < P.M && n < P.N) P.C[static_cast<size_t>(m) * P.ldc + n] += acc[h][w][q];
        }
      }
}

// C_p[m][n] += sum over chunks of part[chunk][tile of (m, n)][local], chunks in order
__global__ __launch_bounds__(256) void small_products_reduce(SmallProductsArgs a) {
  const int e = static_cast<int>(blockIdx.x) * 256 + static_cast<int>(threadIdx.x);
  if (e >= a.el0[a.n]) return;
  const int pi = sp_product(a.el0, a.n, e);
  const SmallProduct P = a.p[pi];
  const int le = e - a.el0[pi], m = le / P.N, n = le % P.N;
  const int tile = a.tile0[pi] + (m / 64) * a.ntn[pi] + n / 64, local = (m % 64) * 64 + n % 64;
  const int nt = a.tile0[a.n];
  float v = 0.0f;
  for (int c = 0; c < a.nchunks; ++c) v += a.part[(static_cast<size_t>(c) * nt + tile) * 4096 + local];
  P.C[static_cast<size_t>(m) * P.ldc + n] += v;
}
}  // namespace

int tn_chunks(int K) { return (K + kTnChunk - 1) / kTnChunk; }

static int small_products_plan(const SmallProduct* p, int n, int T, SmallProductsArgs* a) {
  a->n = n;
  a->T = T;
  int tiles = 0, els = 0;
  for (int i = 0; i < n; ++i) {
    a->p[i] = p[i];
    a->tile0[i] = tiles;
    a->el0[i] = els;
    a->ntn[i] = (p[i].N + 63) / 64;
    tiles += ((p[i].M + 63) / 64) * a->ntn[i];
    els += p[i].M * p[i].N;
  }
  a->tile0[n] = tiles;
  a->el0[n] = els;
  // chunks of at least 256 tokens (a multiple of 16), at most kSmallProductChunks
  a->nchunks = std::max(1, std::min(kSmallProductChunks, T / 256));
  a->kc = ((T + a->nchunks - 1) / a->nchunks + 15) / 16 * 16;
  a->nchunks = (T + a->kc - 1) / a->kc;
  return tiles;
}

size_t small_products_floats(const SmallProduct* p, int n, int T) {
  if (n <= 0 || n > kSmallProducts || T <= 0) return 0;
  SmallProductsArgs a{};
  const int tiles = small_products_plan(p, n, T, &a);
  return a.nchunks > 1 ? static_cast<size_t>(a.nchunks) * tiles * 4096 : 0;
}

hipError_t launch_small_products(const SmallProduct* p, int n, int T, int ldk, float* part, size_t part_floats,
                                 hipStream_t s) {
  if (n <= 0 || T <= 0) return hipSuccess;
  if (n > kSmallProducts) return hipErrorInvalidValue;
  for (int i = 0; i < n; ++i)
    if (p[i].M <= 0 || p[i].N <= 0 || !p[i].A || !p[i].B || !p[i].C) return hipErrorInvalidValue;
  SmallProductsArgs a{};
  const int tiles = small_products_plan(p, n, T, &a);
  a.ldk = ldk;
  a.part = part;
  if (a.nchunks > 1 && (!part || part_floats < static_cast<size_t>(a.nchunks) * tiles * 4096))
    return hipErrorInvalidValue;
  small_products_kernel<<<static_cast<unsigned>(tiles * a.nchunks), 256, 0, s>>>(a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || a.nchunks == 1) return e;
  small_products_reduce<<<static_cast<unsigned>((a.el0[n] + 255) / 256), 256, 0, s>>>(a);
  return hipGetLastError();
}


hipError_t launch_gemm_tn_acc_f32(const float* A, int lda, int M, const float* B, int ldb, int N, int K, float* C,
                                  int ldc, float* part, size_t part_floats, hipStream_t s) {
  if (M <= 0 || N <= 0 || K <= 0) return hipSuccess;
  // as many K chunks of at least kTnChunk as the partial buffer holds for this M x N
  const size_t mn = static_cast<size_t>(M) * N;
  const int nz = static_cast<int>(std::max<size_t>(1, std::min<size_t>(tn_chunks(K), part_floats / mn)));
  const int kc = ((K + nz - 1) / nz + 15) / 16 * 16;
  tn_part_kernel<<<dim3((N + 63) / 64, (M + 63) / 64, nz), 256, 0, s>>>(A, lda, M, B, ldb, N, K, kc, part);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const size_t n = static_cast<size_t>(M) * N;
  tn_reduce_kernel<<<static_cast<unsigned>((n + 255) / 256), 256, 0, s>>>(part, nz, M, N, C, ldc);
  return hipGetLastError();
}

hipError_t launch_split_bf16(const float* x, int R, int C, int ld_in, void* hi, void* lo, int C_pad, hipStream_t s) {
  const size_t n = static_cast<size_t>(R) * C_pad;
  if (n == 0) return hipSuccess;
  const unsigned blocks = static_cast<unsigned>(std::min<size_t>((n + 255) / 256, 8192));
  split_bf16_kernel<<<blocks, 256, 0, s>>>(x, R, C, ld_in, static_cast<bf16_t*>(hi), static_cast<bf16_t*>(lo), C_pad);
  return hipGetLastError();
}

size_t router_bwd_vector_floats(int d_m, int d_s, int d_h, int d_a, int d_e, int d_p, int d_head) {
  // XT, dQT, dKT, dVT, dU1T, dU2T, dPAT, SAT, DA, DB, SBT, dPPT, SPT, XPT, dZAT, dZHT, SHT
  return static_cast<size_t>(d_s + d_m + 1) + 5 * d_m + 3 * d_head + 2 + 2 * d_p + 8 + d_a + d_h + d_e;
}

size_t router_bwd_token_floats(int d_m, int d_s, int d_p, int np) {
  // RS, QKVU, PPRE, Cv, DEN, PS, DSP, DNUM, DDEN, DF, PSUM
  return 4 + 4 * static_cast<size_t>(d_m) + d_p + d_m + 1 + 1 + d_s + d_m + 1 + 3 * static_cast<size_t>(d_m) + np;
}

// the transposed weights' element counts, each rounded up to 8 (16 bytes)
static void router_bwd_wt_counts(int d_m, int d_s, int d_h, int d_a, int d_e, int d_p, int d_head, size_t n[6]) {
  const size_t dx = static_cast<size_t>(d_s) + d_m + 1;
  n[0] = dx * d_head;
  n[1] = static_cast<size_t>(d_s) * d_m;
  n[2] = static_cast<size_t>(d_m) * d_m;
  n[3] = static_cast<size_t>(d_s) * 3 * d_m;
  n[4] = static_cast<size_t>(d_p) * rb_round(d_a, 8);
  n[5] = static_cast<size_t>(d_e) * rb_round(d_h, 8);
  for (int i = 0; i < 6; ++i) n[i] = (n[i] + 7) / 8 * 8;
}

size_t router_bwd_wt_elems(int d_m, int d_s, int d_h, int d_a, int d_e, int d_p, int d_head) {
  size_t n[6], tot = 0;
  router_bwd_wt_counts(d_m, d_s, d_h, d_a, d_e, d_p, d_head, n);
  for (size_t x : n) tot += x;
  return tot;
}

void router_bwd_wt_assign(RouterBwdArgs& a, uint16_t* base) {
  size_t n[6];
  router_bwd_wt_counts(a.d_m, a.d_s, a.d_h, a.d_a, a.d_e, a.d_p, a.d_head, n);
  uint16_t** dst[6] = {&a.th1T, &a.wnT, &a.wcT, &a.wqkvT, &a.wp2T, &a.whuT};
  for (int i = 0; i < 6; ++i) {
    *dst[i] = base;
    base += n[i];
  }
  a.ld_ta = rb_round(a.d_a, 8);
  a.ld_th = rb_round(a.d_h, 8);
}

static bool router_bwd_token_shape_ok(const RouterBwdArgs& a) {
  if (a.d_e > RB_MAXE || a.d_head > RB_MAXH || a.d_s > RB_MAXS || a.d_m > RB_MAXM || a.d_p > RB_MAXP) return false;
  if (a.d_m != 32 && a.d_m != 64 && a.d_m != 128 && a.d_m != 256) return false;
  if (a.p_splits < 1 || a.p_splits > RB_MAXSPL || a.d % 8) return false;
  return 0 <= a.t_begin && a.t_begin <= a.t_end && a.t_end <= a.T;
}

hipError_t launch_router_bwd_wt(const RouterBwdArgs& a, hipStream_t s) {
  if (a.dtype != 1) return hipSuccess;
  if (!router_bwd_token_shape_ok(a) || !a.th1T || !a.wnT || !a.wcT || !a.wqkvT || !a.wp2T || !a.whuT ||
      a.ld_ta != rb_round(a.d_a, 8) || a.ld_th != rb_round(a.d_h, 8))
    return hipErrorInvalidValue;
  const int n = static_cast<int>(router_bwd_wt_elems(a.d_m, a.d_s, a.d_h, a.d_a, a.d_e, a.d_p, a.d_head));
  rbwd_wt<<<static_cast<unsigned>((n + 255) / 256), 256, 0, s>>>(a);
  return hipGetLastError();
}

hipError_t launch_router_bwd_stats(const RouterBwdArgs& a, hipStream_t s) {
  if (!router_bwd_token_shape_ok(a)) return hipErrorInvalidValue;
  const int n = a.t_end - a.t_begin;
  if (n == 0) return hipSuccess;
  const unsigned nst = static_cast<unsigned>((n + RB_NW - 1) / RB_NW);
  if (a.dtype == 1)
    rbwd_stats<bf16_t><<<nst, RB_NT, 0, s>>>(a);
  else
    rbwd_stats<float><<<nst, RB_NT, 0, s>>>(a);
  return hipGetLastError();
}

hipError_t launch_router_bwd_chain(const RouterBwdArgs& a, hipStream_t s) {
  if (!router_bwd_token_shape_ok(a) || (a.t_begin % RB_TB) != 0) return hipErrorInvalidValue;
  if (a.dtype == 1 && (!a.th1T || !a.wnT || !a.wcT || !a.wqkvT || !a.wp2T || !a.whuT)) return hipErrorInvalidValue;
  const int n = a.t_end - a.t_begin;
  if (n == 0) return hipSuccess;
  const unsigned nbat = static_cast<unsigned>((n + RB_TB - 1) / RB_TB), nt = static_cast<unsigned>(n);
  const bool bf = a.dtype == 1;
  hipError_t e;
  if (bf)
    rbwd_f1<bf16_t><<<nbat, RB_BT, 0, s>>>(a);
  else
    rbwd_f1<float><<<nbat, RB_BT, 0, s>>>(a);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  if (!a.c_given) {
    switch (a.d_m) {
      case 32: rbwd_read<32><<<nt, RB_NT, 0, s>>>(a); break;
      case 64: rbwd_read<64><<<nt, RB_NT, 0, s>>>(a); break;
      case 128: rbwd_read<128><<<nt, RB_NT, 0, s>>>(a); break;
      default: rbwd_read<256><<<nt, RB_NT, 0, s>>>(a); break;
    }
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  if (bf)
    rbwd_f2<bf16_t><<<nbat, RB_BT, 0, s>>>(a);
  else
    rbwd_f2<float><<<nbat, RB_BT, 0, s>>>(a);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  switch (a.d_m) {
    case 32: rbwd_spass<32><<<nt, RB_NT, 0, s>>>(a); break;
    case 64: rbwd_spass<64><<<nt, RB_NT, 0, s>>>(a); break;
    case 128: rbwd_spass<128><<<nt, RB_NT, 0, s>>>(a); break;
    default: rbwd_spass<256><<<nt, RB_NT, 0, s>>>(a); break;
  }
  if ((e = hipGetLastError()) != hipSuccess) return e;
  if (bf)
    rbwd_f3<bf16_t><<<nbat, RB_BT, 0, s>>>(a);
  else
    rbwd_f3<float><<<nbat, RB_BT, 0, s>>>(a);
  return hipGetLastError();
}

hipError_t launch_router_bwd_rows(const RouterBwdArgs& a, hipStream_t s) {
  if (a.dtype == 1)
    router_bwd_rows<bf16_t><<<a.T, 256, 0, s>>>(a);
  else
    router_bwd_rows<float><<<a.T, 256, 0, s>>>(a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  router_bwd_deta<<<1, RB_DETA_NT, 0, s>>>(a.rho_part, a.T, a.rho, a.deta);
  return hipGetLastError();
}

hipError_t launch_to_f32_transpose(int dtype, const void* in, int R, int C, int ld_in, float* out, int ld_out,
                                   hipStream_t s) {
  if (R <= 0 || C <= 0) return hipSuccess;
  const dim3 grid((C + 63) / 64, (R + 63) / 64);
  if (dtype == 1)
    to_f32_transpose<bf16_t><<<grid, 256, 0, s>>>(static_cast<const bf16_t*>(in), R, C, ld_in, out, ld_out);
  else
    to_f32_transpose<float><<<grid, 256, 0, s>>>(static_cast<const float*>(in), R, C, ld_in, out, ld_out);
  return hipGetLastError();
}

}  // namespace hero
