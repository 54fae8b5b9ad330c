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

}  // namespace

hipError_t launch_select(const SelectArgs& a, hipStream_t s) {
  const int chunks = (a.T + NT - 1) / NT;
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
