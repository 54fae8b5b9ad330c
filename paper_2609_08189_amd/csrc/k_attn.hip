// Causal grouped-query attention of a decoder block (Sec. 3.1, eq:dense_attention): for every
// sequence, query head h and position t, o_t = sum_{i <= t} softmax_i(q_t . k_i / sqrt(128)) v_i
// with key/value head h / (n_h / n_kv).  Head width 128, bf16 operands, fp32 softmax.
//
// One workgroup (4 waves) takes 128 consecutive queries of one head; wave w owns 32 of them.
// Keys stream through LDS in tiles of 64 (K [64][128] and V^T [128][64], double-buffered,
// filled by global_load_lds_dwordx4), with an online softmax, so the scores never leave
// registers (the V^T positions past the sequence are zeroed first, since the workspace may hold
// anything there):
//   * scores are formed transposed, S^T = K Q^T, on v_mfma_f32_32x32x16_bf16; in the
//     accumulator layout lane l then holds query l % 32, so a query's running max and sum are
//     lane-local (plus one exchange with lane l ^ 32, which holds the other 16 keys);
//   * the output is also formed transposed, O^T = V^T P^T, so the rescaling of a query's
//     partial output by exp(m_old - m_new) is lane-local too;
//   * P^T goes from the score accumulators straight into the B operand of the second product:
//     the contraction over keys takes the keys in the order the accumulator holds them (four
//     consecutive, then four 8 further on), and V^T is stored with its positions in that
//     order (within each group of 16, the blocks 4-7 and 8-11 swapped), so that a lane's 8
//     keys are one 16-byte read.
// The LDS rows are XOR-swizzled in 16-byte chunks, K rows (256 B) by row % 16 and V^T rows
// (128 B) by (row / 2) % 8, which makes both kinds of 32-row fragment reads conflict free.
#include "hero_device.h"
#include "hero_kernels.h"

namespace hero {
namespace {

constexpr int HD = 128;                  // head width
constexpr int QT = 128;                  // queries per workgroup
constexpr int KT = 64;                   // keys per tile
constexpr int NTA = 256;                 // 4 waves
constexpr int K_BYTES = KT * HD * 2;     // K tile [64][128] bf16
constexpr int V_BYTES = HD * KT * 2;     // V^T tile [128][64] bf16
constexpr int STG = K_BYTES + V_BYTES;
constexpr int OPITCH = HD + 8;           // output staging row pitch (bf16 elements)

typedef __attribute__((address_space(3))) void lds_void;

__device__ __forceinline__ void load_lds16(const void* g, unsigned char* l) {
  __builtin_amdgcn_global_load_lds(g, (lds_void*)(l), 16, 0, 0);
}

// instruction classes of __builtin_amdgcn_sched_group_barrier
constexpr int SG_MFMA = 0x008, SG_DS_READ = 0x100;

// Order the 16 fragment reads and 16 MFMAs of a product phase as: 4 reads ahead, then one
// MFMA and one read alternately, then the last 4 MFMAs (bounds the fragments in flight)
__device__ __forceinline__ void pipeline_reads_with_mfmas() {
  __builtin_amdgcn_sched_group_barrier(SG_DS_READ, 4, 0);
#pragma unroll
  for (int i = 0; i < 12; ++i) {
    __builtin_amdgcn_sched_group_barrier(SG_MFMA, 1, 0);
    __builtin_amdgcn_sched_group_barrier(SG_DS_READ, 1, 0);
  }
  __builtin_amdgcn_sched_group_barrier(SG_MFMA, 4, 0);
}

typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

// eight fp32 values to bf16 (nearest even), two per v_cvt_pk_bf16_f32
__device__ __forceinline__ bf16x8 pack8(const float* x) {
  u32x4 w;
#pragma unroll
  for (int i = 0; i < 4; ++i)
    w[i] = __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2{x[2 * i], x[2 * i + 1]}, bf16x2));
  return __builtin_bit_cast(bf16x8, w);
}

__global__ __launch_bounds__(NTA, 2) void attn_fwd_kernel(const bf16_t* __restrict__ q,
                                                      const bf16_t* __restrict__ k,
                                                      const bf16_t* __restrict__ vt,
                                                      bf16_t* __restrict__ o, int batch, int seq,
                                                      int seq_pad, int nh, int nkv, float scale_log2) {
  __shared__ __attribute__((aligned(1024))) unsigned char smem[2 * STG];
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(static_cast<int>(threadIdx.x) >> 6);
  const int hl = lane >> 5, col = lane & 31;
  // Work items (sequence b, kv head, query head of its group, query tile) are laid over the 8
  // XCDs (workgroups go to XCD blockIdx % 8) so that each XCD takes whole kv groups: the K and
  // V^T of a group (2 x 128 x seq_pad bf16) then stay in that XCD's L2.  Within an XCD the
  // longest query tiles come first.
  const int n_qt = seq_pad / QT;
  const int hpg = nh / nkv;                              // query heads per kv head
  const int n_groups = batch * nkv;
  const int gx = (n_groups + 7) / 8;                     // kv groups per XCD
  const int xcd = blockIdx.x & 7, kq = blockIdx.x >> 3;
  const int g = xcd + 8 * (kq % gx);
  if (g >= n_groups) return;
  const int rest = kq / gx;                              // < hpg * n_qt
  const int qt = n_qt - 1 - rest / hpg;
  const int b = g / nkv, kvh = g % nkv, head = kvh * hpg + rest % hpg;
  const int q0 = qt * QT;
  const int wq0 = q0 + 32 * wave;                 // this wave's first query
  const int my_q = wq0 + col;                     // the query this lane's columns hold

  const bf16_t* qb = q + (static_cast<size_t>(b) * nh + head) * seq_pad * HD;
  const bf16_t* kb = k + (static_cast<size_t>(b) * nkv + kvh) * seq_pad * HD;
  const bf16_t* vb = vt + (static_cast<size_t>(b) * nkv + kvh) * HD * seq_pad;

  // keys needed by this workgroup: 0 .. min(q0 + 127, seq - 1)
  const int n_kt = (min(q0 + QT, seq) + KT - 1) / KT;

  // per-lane element offsets of the stage loads (rows and swizzled 16-byte chunks)
  int k_off[4], v_off[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int blk = 4 * wave + i;
    const int rk = 4 * blk + (lane >> 4), rv = 8 * blk + (lane >> 3);
    k_off[i] = rk * HD + 8 * ((lane & 15) ^ (rk & 15));
    v_off[i] = rv * seq_pad + 8 * ((lane & 7) ^ ((rv >> 1) & 7));
  }
  auto issue = [&](int stage, int k0) {
    unsigned char* st = smem + stage * STG;
    const bf16_t* kt0 = kb + static_cast<size_t>(k0) * HD;
    const bf16_t* vt0 = vb + k0;
#pragma unroll
    for (int i = 0; i < 4; ++i) load_lds16(kt0 + k_off[i], st + (4 * wave + i) * 1024);
#pragma unroll
    for (int i = 0; i < 4; ++i) load_lds16(vt0 + v_off[i], st + K_BYTES + (4 * wave + i) * 1024);
  };

  issue(0, 0);

  // this lane's query as the B operand of S^T = K Q^T: hd 16 s + 8 hl .. + 8, s = 0..7
  bf16x8 qf[8];
#pragma unroll
  for (int s = 0; s < 8; ++s)
    qf[s] = *reinterpret_cast<const bf16x8*>(qb + static_cast<size_t>(my_q) * HD + 16 * s + 8 * hl);

  f32x16 acc_o[4];
#pragma unroll
  for (int t4 = 0; t4 < 4; ++t4)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc_o[t4][r] = 0.f;
  float m_run = -INFINITY, l_run = 0.f;

  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  __syncthreads();

  for (int kt = 0; kt < n_kt; ++kt) {
    const int k0 = kt * KT;
    if (kt + 1 < n_kt) issue((kt + 1) & 1, k0 + KT);
    const unsigned char* st = smem + (kt & 1) * STG;
    // keys past this wave's last query are all masked: nothing to add
    if (k0 <= wq0 + 31) {
      // the two 32-key halves are independent accumulation chains: alternate them
      f32x16 sacc[2];
#pragma unroll
      for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int r = 0; r < 16; ++r) sacc[t][r] = 0.f;
#pragma unroll
      for (int s = 0; s < 8; ++s)
#pragma unroll
        for (int t = 0; t < 2; ++t) {
          const int r = 32 * t + col, c = 2 * s + hl;
          const bf16x8 kf = *reinterpret_cast<const bf16x8*>(st + 256 * r + 16 * (c ^ (r & 15)));
          sacc[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[s], sacc[t], 0, 0, 0);
        }
      pipeline_reads_with_mfmas();
      // causal / length mask (keys past the query or the sequence; only tiles that reach the
      // diagonal or the end can hold any) and the running max, in raw score units; the base-2
      // scale enters through the exponent's fma
      const bool edge = k0 + KT - 1 > wq0 || k0 + KT > seq;
      float mx = -INFINITY;
      if (edge) {
        const int lim = min(my_q, seq - 1) - k0;     // last visible key of the tile
#pragma unroll
        for (int t = 0; t < 2; ++t)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int kr = 32 * t + 8 * (r >> 2) + 4 * hl + (r & 3);
            if (kr > lim) sacc[t][r] = -INFINITY;
            mx = fmaxf(mx, sacc[t][r]);
          }
      } else {
#pragma unroll
        for (int t = 0; t < 2; ++t)
#pragma unroll
          for (int r = 0; r < 16; ++r) mx = fmaxf(mx, sacc[t][r]);
      }
      mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
      const float m_new = fmaxf(m_run, mx);
      const float mc = m_new * scale_log2;
      float ps = 0.f;
#pragma unroll
      for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const float p = __builtin_amdgcn_exp2f(fmaf(sacc[t][r], scale_log2, -mc));
          sacc[t][r] = p;
          ps += p;
        }
      ps += __shfl_xor(ps, 32, 64);
      // rescale the partial output only when some query's max moved (exp2(0) = 1 otherwise)
      if (__any(m_new > m_run)) {
        const float alpha = __builtin_amdgcn_exp2f(m_run * scale_log2 - mc);
        l_run *= alpha;
#pragma unroll
        for (int t4 = 0; t4 < 4; ++t4)
#pragma unroll
          for (int r = 0; r < 16; ++r) acc_o[t4][r] *= alpha;
      }
      l_run += ps;
      m_run = m_new;
      // P^T as B operands: k-step (t, u) takes accumulator registers 8u .. 8u + 7 of tile t
      bf16x8 pf[2][2];
#pragma unroll
      for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int u = 0; u < 2; ++u) {
          float x[8];
#pragma unroll
          for (int e = 0; e < 8; ++e) x[e] = sacc[t][8 * u + e];
          pf[t][u] = pack8(x);
        }
      // O^T += V^T P^T; the V^T fragment of k-step (t, u) holds keys 32t + 16u + 4hl + {0..3}
      // and the same + 8; the four 32-row output blocks are independent chains, alternated
#pragma unroll
      for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int u = 0; u < 2; ++u)
#pragma unroll
          for (int t4 = 0; t4 < 4; ++t4) {
            const int r = 32 * t4 + col;
            const unsigned char* vrow = st + K_BYTES + 128 * r;
            const int sw = (r >> 1) & 7;
            const bf16x8 vf = *reinterpret_cast<const bf16x8*>(vrow + 16 * ((4 * t + 2 * u + hl) ^ sw));
            acc_o[t4] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, pf[t][u], acc_o[t4], 0, 0, 0);
          }
      pipeline_reads_with_mfmas();
    }
    // every wave is done with this stage and the next tile has landed
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
  }

  // normalise and stage the wave's [32 queries][128] block, then write 16-byte row pieces
  const float inv_l = 1.0f / l_run;
  bf16_t* stg = reinterpret_cast<bf16_t*>(smem) + wave * 32 * OPITCH;
#pragma unroll
  for (int t4 = 0; t4 < 4; ++t4)
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      const int c = 32 * t4 + 8 * g + 4 * hl;
      uint32_t w0 = static_cast<uint32_t>(f32_to_bf16(acc_o[t4][4 * g + 0] * inv_l)) |
                    (static_cast<uint32_t>(f32_to_bf16(acc_o[t4][4 * g + 1] * inv_l)) << 16);
      uint32_t w1 = static_cast<uint32_t>(f32_to_bf16(acc_o[t4][4 * g + 2] * inv_l)) |
                    (static_cast<uint32_t>(f32_to_bf16(acc_o[t4][4 * g + 3] * inv_l)) << 16);
      uint32_t* dst = reinterpret_cast<uint32_t*>(stg + col * OPITCH + c);
      dst[0] = w0;
      dst[1] = w1;
    }
  __syncthreads();
  const size_t ld_o = static_cast<size_t>(nh) * HD;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const int e = lane + 64 * i;
    const int row = e >> 4, piece = e & 15;
    const int tq = wq0 + row;
    if (tq < seq) {
      const u32x4 v = *reinterpret_cast<const u32x4*>(stg + row * OPITCH + 8 * piece);
      *reinterpret_cast<u32x4*>(o + (static_cast<size_t>(b) * seq + tq) * ld_o + head * HD + 8 * piece) = v;
    }
  }
}

// V^T positions seq .. seq_pad - 1 of every row set to zero: their probabilities are zero, and
// a zero probability must not meet whatever the workspace held there (a NaN)
__global__ void vt_pad_kernel(bf16_t* __restrict__ vt, int rows, int seq, int seq_pad) {
  const int pad = seq_pad - seq;
  const size_t e = static_cast<size_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (e >= static_cast<size_t>(rows) * pad) return;
  const int row = static_cast<int>(e / pad), p = seq + static_cast<int>(e % pad);
  const int slot = (p & ~15) | (p & 3) | ((p & 4) << 1) | ((p & 8) >> 1);
  vt[static_cast<size_t>(row) * seq_pad + slot] = 0;
}

}  // namespace

hipError_t launch_attn_core(const void* q, const void* k, void* vt, void* o, int batch, int seq,
                            int seq_pad, int nh, int nkv, hipStream_t s) {
  if (batch <= 0 || seq <= 0) return hipSuccess;
  if (seq_pad % QT != 0 || seq_pad < seq || nkv <= 0 || nh % nkv != 0) return hipErrorInvalidValue;
  if (seq_pad > seq) {
    const size_t n = static_cast<size_t>(batch) * nkv * HD * (seq_pad - seq);
    vt_pad_kernel<<<static_cast<unsigned>((n + 255) / 256), 256, 0, s>>>(static_cast<bf16_t*>(vt),
                                                                      batch * nkv * HD, seq, seq_pad);
  }
  const int n_groups = batch * nkv, gx = (n_groups + 7) / 8;
  const dim3 grid(8 * gx * (nh / nkv) * (seq_pad / QT));
  const float scale_log2 = 1.4426950408889634f / sqrtf(static_cast<float>(HD));
  attn_fwd_kernel<<<grid, NTA, 0, s>>>(static_cast<const bf16_t*>(q), static_cast<const bf16_t*>(k),
                                       static_cast<const bf16_t*>(vt), static_cast<bf16_t*>(o), batch,
                                       seq, seq_pad, nh, nkv, scale_log2);
  return hipGetLastError();
}

}  // namespace hero
