// Branch decision and ordered token compaction for one routed layer.
//
// Threshold mode: a token takes the FFN iff its logit >= ln(tau/(1-tau)), which is
// g >= tau_exec of Sec. 3.1 (eq:ffn_route) decided in logit space; ties go to the FFN.
// Budget mode: exactly n_skip tokens take the adapter, those with the smallest
// (logit, token index).  The n_skip-th smallest key is found by an MSB-first radix
// select (4 passes of 8 bits) over order-preserving 32-bit images of the fp32
// logits, then, among tokens whose logit equals that key, by token index.
// Compaction: a wave ballot gives each token its rank within the wave, a
// 16-wave scan its rank within a 1024-token chunk, and a running count across
// chunks keeps both index lists in ascending token order.
// One workgroup of 1024 threads does the whole layer: the work is ~10 bytes per
// token and the cost is latency, so each thread keeps its tokens' logits in registers
// (up to 32 chunks of 1024 tokens) for the six passes instead of reading them again.
#include "hero_device.h"
#include "hero_kernels.h"

namespace hero {
namespace {

constexpr int NT = 1024;
constexpr int NW = NT / 64;

// order-preserving image of an fp32 value (-0 and +0 map to the same key)
__device__ __forceinline__ uint32_t okey(float f) {
  uint32_t b = __float_as_uint(f);
  if (b == 0x80000000u) b = 0u;
  return (b & 0x80000000u) ? ~b : (b | 0x80000000u);
}

__device__ __forceinline__ int lane_prefix(unsigned long long bal, int lane) {
  return __popcll(bal & ((1ull << lane) - 1ull));
}

// R > 0: token t = tid + NT r (r < R) keeps its logit in a register for all passes (T <= NT R);
// R == 0: every pass reads the logits again (any T).
template <int R>
struct Logits {
  float v[R > 0 ? R : 1];
  __device__ __forceinline__ void load(const float* lg, int T) {
#pragma unroll
    for (int r = 0; r < R; ++r) {
      const int t = static_cast<int>(threadIdx.x) + NT * r;
      v[r] = t < T ? lg[t] : 0.f;
    }
  }
  __device__ __forceinline__ float at(const float* lg, int r, int t) const {
    if constexpr (R > 0) {
      return v[r];
    } else {
      return lg[t];
    }
  }
};

// for (r = 0; NT r < T; ++r) f(r, t = tid + NT r), unrolled when the chunk count is static
template <int R, class F>
__device__ __forceinline__ void for_chunks(int T, F&& f) {
  if constexpr (R > 0) {
#pragma unroll
    for (int r = 0; r < R; ++r)
      if (NT * r < T) f(r, static_cast<int>(threadIdx.x) + NT * r);
  } else {
    for (int r = 0; NT * r < T; ++r) f(r, static_cast<int>(threadIdx.x) + NT * r);
  }
}

template <int R>
__global__ __launch_bounds__(NT) void select_kernel(SelectArgs a) {
  __shared__ uint32_t hist[256];
  __shared__ int wcount[NW];
  __shared__ int wcount2[NW];
  __shared__ float wmin[NW];
  __shared__ uint32_t s_prefix;
  __shared__ int s_k;
  __shared__ int s_tstar;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int T = a.T;
  const bool budget = a.mode == 1;
  Logits<R> lg;
  lg.load(a.logit, T);

  // adapter iff key < vstar, or key == vstar and t <= tstar
  uint32_t vstar = 0u;
  int tstar = -1;
  if (budget && a.n_skip > 0) {
    if (tid == 0) {
      s_prefix = 0u;
      s_k = a.n_skip;
    }
    for (int shift = 24; shift >= 0; shift -= 8) {
      for (int i = tid; i < 256; i += NT) hist[i] = 0u;
      __syncthreads();
      const uint32_t prefix = s_prefix;
      for_chunks<R>(T, [&](int r, int t) {
        if (t < T) {
          const uint32_t key = okey(lg.at(a.logit, r, t));
          if (shift == 24 || (key >> (shift + 8)) == (prefix >> (shift + 8)))
            atomicAdd(&hist[(key >> shift) & 255u], 1u);
        }
      });
      __syncthreads();
      if (wave == 0) {
        // lane l owns bins [4l, 4l+4); inclusive scan of their sums across the wave
        uint32_t h[4], sum = 0;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          h[i] = hist[4 * lane + i];
          sum += h[i];
        }
        uint32_t incl = sum;
#pragma unroll
        for (int off = 1; off < 64; off <<= 1) {
          const uint32_t v = __shfl_up(incl, off, 64);
          if (lane >= off) incl += v;
        }
        const int k = s_k;
        uint32_t before = incl - sum;
        if (static_cast<int>(before) < k && k <= static_cast<int>(incl)) {
          int dgt = 4 * lane;
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            if (static_cast<int>(before + h[i]) >= k) break;
            before += h[i];
            ++dgt;
          }
          s_prefix = prefix | (static_cast<uint32_t>(dgt) << shift);
          s_k = k - static_cast<int>(before);
        }
      }
      __syncthreads();
    }
    vstar = s_prefix;
    // the s_k-th token (1-based, by index) whose key equals vstar
    const int k = s_k;
    if (tid == 0) s_tstar = -1;
    int run = 0;
    for_chunks<R>(T, [&](int r, int t) {
      if (run >= k) return;   // uniform: every thread holds the same run
      const bool pred = t < T && okey(lg.at(a.logit, r, t)) == vstar;
      const unsigned long long bal = __ballot(pred);
      if (lane == 0) wcount[wave] = __popcll(bal);
      __syncthreads();
      int wpre = 0, tot = 0;
      for (int w = 0; w < NW; ++w) {
        const int c = wcount[w];
        if (w < wave) wpre += c;
        tot += c;
      }
      if (pred && run + wpre + lane_prefix(bal, lane) + 1 == k) s_tstar = t;
      run += tot;
      __syncthreads();
    });
    __syncthreads();
    tstar = s_tstar;
  }

  // decision and compaction
  int nf = 0, na = 0;
  float lmin = __builtin_inff();
  for_chunks<R>(T, [&](int r, int t) {
    const bool valid = t < T;
    bool ffn = false;
    if (valid) {
      const float l = lg.at(a.logit, r, t);
      if (budget) {
        const uint32_t key = okey(l);
        const bool skip = a.n_skip > 0 && (key < vstar || (key == vstar && t <= tstar));
        ffn = !skip;
      } else {
        ffn = l >= a.thr;
      }
      a.mask[t] = ffn ? 1 : 0;
      if (ffn) lmin = fminf(lmin, l);
    }
    const unsigned long long bal = __ballot(ffn);
    if (lane == 0) wcount2[wave] = __popcll(bal);
    __syncthreads();
    int wpre = 0, tot = 0;
    for (int w = 0; w < NW; ++w) {
      const int c = wcount2[w];
      if (w < wave) wpre += c;
      tot += c;
    }
    if (valid) {
      const int fpos = wpre + lane_prefix(bal, lane);  // FFN tokens before t in this chunk
      if (ffn)
        a.idx_ffn[nf + fpos] = t;
      else
        a.idx_ad[na + (tid - fpos)] = t;
    }
    const int nvalid = min(NT, T - NT * r);
    nf += tot;
    na += nvalid - tot;
    __syncthreads();
  });

  // smallest FFN logit
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) lmin = fminf(lmin, __shfl_xor(lmin, off, 64));
  if (lane == 0) wmin[wave] = lmin;
  __syncthreads();
  if (tid == 0) {
    float m = wmin[0];
    for (int w = 1; w < NW; ++w) m = fminf(m, wmin[w]);
    const float lam = budget ? m : a.thr;
    a.counts[0] = nf;
    a.counts[1] = na;
    a.lambda[0] = lam;
  }
}

// ---------------------------------------------------------------------------
// Large batches: thread i owns the contiguous run of R tokens [i R, (i + 1) R).  The radix
// select takes 11-bit digits (three passes), and each thread adds its run's digits to the LDS
// histogram run-length encoded: the logits of an untrained router cluster, so the leading
// digits of a run are mostly equal and one atomic add covers many tokens.  The tie rank and the
// compaction each need one block-wide scan of per-thread counts (every thread then writes its
// own run in token order), instead of a barrier pair per 1024-token chunk.  Same decisions,
// index lists, counts and lambda as select_kernel (the result is unique).
// ---------------------------------------------------------------------------

// exclusive prefix over the block of one int per thread; *total receives the block sum
__device__ __forceinline__ int block_exclusive_scan(int v, int* wsum, int* total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  int incl = v;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const int u = __shfl_up(incl, off, 64);
    if (lane >= off) incl += u;
  }
  if (lane == 63) wsum[wave] = incl;
  __syncthreads();
  int before = 0, tot = 0;
#pragma unroll
  for (int w = 0; w < NW; ++w) {
    const int c = wsum[w];
    if (w < wave) before += c;
    tot += c;
  }
  __syncthreads();   // wsum may be reused by the caller's next scan
  *total = tot;
  return before + incl - v;
}

template <int R>
__global__ __launch_bounds__(NT) void select_run_kernel(SelectArgs a) {
  static_assert(R % 4 == 0, "runs are read as float4");
  constexpr int DB = 11, NB = 1 << DB;          // digit bits and histogram bins
  __shared__ uint32_t hist[NB];
  __shared__ int wsum[NW];
  __shared__ float wmin[NW];
  __shared__ uint32_t s_prefix;
  __shared__ int s_k;
  __shared__ int s_tstar;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int T = a.T;
  const bool budget = a.mode == 1;
  const int t0 = tid * R;
  // tokens past T get the largest key (the bits 0x7fffffff): in (key, index) order they come
  // after every real token, so the k-th smallest (k <= T) is always a real one and the radix and
  // tie passes need no bounds test; decision and compaction skip them
  const float pad = __uint_as_float(0x7fffffffu);
  float v[R];
#pragma unroll
  for (int q = 0; q < R / 4; ++q) {
    const int t = t0 + 4 * q;
    if (t + 3 < T) {
      const f32x4 x = *reinterpret_cast<const f32x4*>(a.logit + t);
      v[4 * q] = x[0];
      v[4 * q + 1] = x[1];
      v[4 * q + 2] = x[2];
      v[4 * q + 3] = x[3];
    } else {
#pragma unroll
      for (int e = 0; e < 4; ++e) v[4 * q + e] = t + e < T ? a.logit[t + e] : pad;
    }
  }
  const int nmine = max(0, min(R, T - t0));     // valid tokens of this run

  // adapter iff key < vstar, or key == vstar and t <= tstar
  uint32_t vstar = 0u;
  int tstar = -1;
  if (budget && a.n_skip > 0) {
    if (tid == 0) {
      s_prefix = 0u;
      s_k = a.n_skip;
    }
    // digits: bits 21..31, 10..20, 0..9
    for (int pass = 0; pass < 3; ++pass) {
      const int shift = pass == 0 ? 21 : (pass == 1 ? 10 : 0);
      const int width = pass == 2 ? 10 : DB;
      const uint32_t dmask = (1u << width) - 1u;
      for (int i = tid; i < NB; i += NT) hist[i] = 0u;
      __syncthreads();
      const uint32_t prefix = s_prefix;
      const int hi = shift + width;                 // bits above this digit are fixed
      int last = -1;
      uint32_t cnt = 0;
#pragma unroll
      for (int r = 0; r < R; ++r) {
        const uint32_t key = okey(v[r]);
        if (hi >= 32 || (key >> hi) == (prefix >> hi)) {
          const int dgt = static_cast<int>((key >> shift) & dmask);
          if (dgt == last) {
            ++cnt;
          } else {
            if (cnt) atomicAdd(&hist[last], cnt);
            last = dgt;
            cnt = 1;
          }
        }
      }
      if (cnt) atomicAdd(&hist[last], cnt);
      __syncthreads();
      if (wave == 0) {
        // lane l owns bins [32 l, 32 l + 32); inclusive scan of their sums across the wave
        uint32_t sum = 0;
        for (int i = 0; i < NB / 64; ++i) sum += hist[(NB / 64) * lane + i];
        uint32_t incl = sum;
#pragma unroll
        for (int off = 1; off < 64; off <<= 1) {
          const uint32_t u = __shfl_up(incl, off, 64);
          if (lane >= off) incl += u;
        }
        const int k = s_k;
        uint32_t before = incl - sum;
        if (static_cast<int>(before) < k && k <= static_cast<int>(incl)) {
          int dgt = (NB / 64) * lane;
          for (int i = 0; i < NB / 64; ++i) {
            const uint32_t h = hist[dgt];
            if (static_cast<int>(before + h) >= k) break;
            before += h;
            ++dgt;
          }
          s_prefix = prefix | (static_cast<uint32_t>(dgt) << shift);
          s_k = k - static_cast<int>(before);
        }
      }
      __syncthreads();
    }
    vstar = s_prefix;
    // the s_k-th token (1-based, by index) whose key equals vstar
    const int k = s_k;
    int neq = 0;
#pragma unroll
    for (int r = 0; r < R; ++r) neq += okey(v[r]) == vstar ? 1 : 0;
    int tot;
    const int eq_before = block_exclusive_scan(neq, wsum, &tot);
    if (tid == 0) s_tstar = -1;
    __syncthreads();
    if (eq_before < k && k <= eq_before + neq) {
      int seen = eq_before;
#pragma unroll
      for (int r = 0; r < R; ++r) {
        if (okey(v[r]) == vstar) {
          ++seen;
          if (seen == k) s_tstar = t0 + r;
        }
      }
    }
    __syncthreads();
    tstar = s_tstar;
  }

  // decision and compaction
  uint32_t ffn_bits = 0;
  int nf_mine = 0;
  float lmin = __builtin_inff();
#pragma unroll
  for (int r = 0; r < R; ++r) {
    if (r < nmine) {
      const int t = t0 + r;
      bool ffn;
      if (budget) {
        const uint32_t key = okey(v[r]);
        ffn = !(a.n_skip > 0 && (key < vstar || (key == vstar && t <= tstar)));
      } else {
        ffn = v[r] >= a.thr;
      }
      if (ffn) {
        ffn_bits |= 1u << r;
        ++nf_mine;
        lmin = fminf(lmin, v[r]);
      }
    }
  }
  int nf_tot;
  const int f_before = block_exclusive_scan(nf_mine, wsum, &nf_tot);
  if (nmine > 0) {
    const int a_before = t0 - f_before;         // adapter tokens before this run
    int nf = 0, na = 0;
#pragma unroll
    for (int q = 0; q < R / 4; ++q) {
      uint32_t packed = 0;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int r = 4 * q + e;
        if (r < nmine) {
          const bool ffn = (ffn_bits >> r) & 1u;
          packed |= (ffn ? 1u : 0u) << (8 * e);
          if (ffn)
            a.idx_ffn[f_before + nf++] = t0 + r;
          else
            a.idx_ad[a_before + na++] = t0 + r;
        }
      }
      const int t = t0 + 4 * q;
      if (t + 3 < T) {
        *reinterpret_cast<uint32_t*>(a.mask + t) = packed;
      } else {
#pragma unroll
        for (int e = 0; e < 4; ++e)
          if (t + e < T) a.mask[t + e] = static_cast<uint8_t>((packed >> (8 * e)) & 1u);
      }
    }
  }

  // smallest FFN logit
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) lmin = fminf(lmin, __shfl_xor(lmin, off, 64));
  if (lane == 0) wmin[wave] = lmin;
  __syncthreads();
  if (tid == 0) {
    float m = wmin[0];
    for (int w = 1; w < NW; ++w) m = fminf(m, wmin[w]);
    a.counts[0] = nf_tot;
    a.counts[1] = T - nf_tot;
    a.lambda[0] = budget ? m : a.thr;
  }
}

}  // namespace

hipError_t launch_select(const SelectArgs& a, hipStream_t s) {
  const int chunks = (a.T + NT - 1) / NT;
  // large batches: contiguous runs per thread (one scan per phase instead of a barrier pair per
  // chunk; up to 32768 tokens)
  if (a.T > 8 * NT && a.T <= 16 * NT) {
    select_run_kernel<16><<<1, NT, 0, s>>>(a);
    return hipGetLastError();
  }
  if (a.T > 16 * NT && a.T <= 32 * NT) {
    select_run_kernel<32><<<1, NT, 0, s>>>(a);
    return hipGetLastError();
  }
  if (chunks <= 1)
    select_kernel<1><<<1, NT, 0, s>>>(a);
  else if (chunks <= 4)
    select_kernel<4><<<1, NT, 0, s>>>(a);
  else if (chunks <= 8)
    select_kernel<8><<<1, NT, 0, s>>>(a);
  else if (chunks <= 32)
    select_kernel<32><<<1, NT, 0, s>>>(a);
  else
    select_kernel<0><<<1, NT, 0, s>>>(a);
  return hipGetLastError();
}

}  // namespace hero
