// Dense contractions of the routed layer.
//
//   router pre-activations   P = hbar [W_hd; psi_1]^T                 (Sec. 3.2, z^h and f_psi)
//   FFN gate/up              act = SiLU(u W_g^T) * (u W_u^T)          (frozen SwiGLU FFN)
//   FFN down + scatter       h_out[t] = hbar[t] + g_t (act W_d^T)     (Sec. 3.1, eq:ffn_route)
//   adapter down             hid = SiLU(u W_1^T)                      (Sec. 3.1, adapter)
//   adapter up + scatter     h_out[t] = hbar[t] + (1 - g_t) (hid W_2^T)
//
// bf16 path: v_mfma_f32_32x32x16_bf16 with fp32 accumulation.  A and B are both
// K-contiguous ("x W^T" with nn.Linear weights).  A k-tile of 64 elements
// (128 bytes per row) of A and B is staged through LDS, double buffered, with
// the 16-byte chunks of each row XOR-swizzled by (row & 7) so that the 32-row
// fragment reads of one MFMA hit distinct banks.  A rows may be gathered through
// an index list whose length lives on the device (tiles past it exit at once).
// Workgroups are mapped to tiles so that each XCD (8 per MI355X, round-robin
// dispatch) owns a contiguous run of a grouped tile order: the tiles it runs at
// once share a few row panels and a few weight panels in its L2.
//
// f32 path: a plain LDS-tiled VALU GEMM with full bounds checks (small shapes).
#include <limits.h>

#include <algorithm>

#include <type_traits>

#include "hero_device.h"
#include "hero_kernels.h"

namespace hero {
namespace {

constexpr int BK = 64;     // k elements per tile
constexpr int ROWB = 128;  // bytes of one row of a bf16 k-tile

template <typename T>
struct ARows {
  const T* base;
  const int* idx;  // null: identity
  int ld;
  __device__ __forceinline__ const T* row(int m) const {
    return base + static_cast<size_t>(idx ? idx[m] : m) * ld;
  }
};

// B rows: [0, split) from b0, [split, ...) from b1 (router: W_hd then psi_1);
// for the gate/up product b0 = W_g, b1 = W_u and rows are addressed by column.
template <typename T>
struct BRows {
  const T* b0;
  const T* b1;
  int split;
  int ld;
  __device__ __forceinline__ const T* row(int n) const {
    return n < split ? b0 + static_cast<size_t>(n) * ld : b1 + static_cast<size_t>(n - split) * ld;
  }
  __device__ __forceinline__ const T* gate_row(int c) const { return b0 + static_cast<size_t>(c) * ld; }
  __device__ __forceinline__ const T* up_row(int c) const { return b1 + static_cast<size_t>(c) * ld; }
};

// ---------------------------------------------------------------------------
// epilogues
// ---------------------------------------------------------------------------

struct EpiStoreF32 {  // P[m][n] = acc; the MFMA path's K-slice z writes out + z * split_stride
  float* out;
  int ld;
  size_t split_stride;
  struct Pre {};
  __device__ __forceinline__ Pre prep(int, int) const { return {}; }
  __device__ __forceinline__ void store(int m, int n, float v) const {
    out[static_cast<size_t>(m) * ld + n] = v;
  }
  __device__ __forceinline__ void emit8(const Pre&, int m, int n, const float* v) const {
    float* o = out + blockIdx.y * split_stride + static_cast<size_t>(m) * ld + n;
    *reinterpret_cast<f32x4*>(o) = *reinterpret_cast<const f32x4*>(v);
    *reinterpret_cast<f32x4*>(o + 4) = *reinterpret_cast<const f32x4*>(v + 4);
  }
};

template <typename T>
struct EpiSwiGLU {  // act[m][c] = SiLU(gate) * up
  T* act;
  int ld;
  __device__ __forceinline__ void store2(int m, int c, float g, float u) const {
    stf(act + static_cast<size_t>(m) * ld + c, siluf_(g) * u);
  }
  // eight finished bf16 values (the MFMA path forms SiLU(gate) * up while staging)
  __device__ __forceinline__ void emit_packed(int m, int c, u32x4 v) const {
    *reinterpret_cast<u32x4*>(act + static_cast<size_t>(m) * ld + c) = v;
  }
};

template <typename T>
struct EpiSiLU {  // hid[m][n] = SiLU(acc)
  T* out;
  int ld;
  __device__ __forceinline__ void store(int m, int n, float v) const {
    stf(out + static_cast<size_t>(m) * ld + n, siluf_(v));
  }
};

template <typename T>
struct EpiStore {  // out[m][n] = acc in the storage dtype
  T* out;
  int ld;
  struct Pre {};
  __device__ __forceinline__ Pre prep(int, int) const { return {}; }
  __device__ __forceinline__ void store(int m, int n, float v) const {
    stf(out + static_cast<size_t>(m) * ld + n, v);
  }
  __device__ __forceinline__ void emit8(const Pre&, int m, int n, const float* v) const {
    st8(out + static_cast<size_t>(m) * ld + n, v);
  }
};

// Backward of the gated SwiGLU branch, on the recomputed gate/up products G = u W_g^T,
// U = u W_u^T of FFN row m (token t = idx[m]), given e = dL/dy W_d at the same (m, c) with
// dL/dy = g_t dL/dh (e itself carries no g):
//   act = SiLU(G) U,  dL/dact = g_t e,
//   dG = g_t e U SiLU'(G),  dU = g_t e SiLU(G)   -> dgu[m][c], dgu[m][d_ff + c]
//   the row's share of dL/dg_t = <dL/dh_t, y_t> = <e_m, act_m> over the tile's columns
//                                                  -> dgpart[m][part]
// The MFMA path hands this epilogue the accumulators of a finished wave tile (dual); the
// fp32 path calls store2 per element with one partial per column.
template <typename T>
struct EpiSwiGLUBwd {
  const T* e;
  int ld_e;
  const int* idx;
  const float* gate;
  T* dgu;
  int ld_dgu;
  int d_ff;
  float* dgpart;
  int n_parts;
  static constexpr bool kDualHook = true;
  __device__ __forceinline__ void store2(int m, int c, float g, float u) const {
    const int t = idx ? idx[m] : m;
    const float gt = gate ? gate[t] : 1.0f;
    const float ev = ldf(e + static_cast<size_t>(m) * ld_e + c);
    const float sg = 1.0f / (1.0f + expf(-g));
    const float act = g * sg * u, dact = gt * ev;
    stf(dgu + static_cast<size_t>(m) * ld_dgu + c, dact * u * sg * (1.0f + g * (1.0f - sg)));
    stf(dgu + static_cast<size_t>(m) * ld_dgu + d_ff + c, dact * g * sg);
    dgpart[static_cast<size_t>(m) * n_parts + c] = ev * act;
  }
};

// h_out[t][n] = hbar[t][n] + scale(g_t) * acc, t = idx[m]; FFN scales by g, adapter by 1 - g.
// Without an index list t = m, and without gates the scale is 1 (a plain residual add: the
// dense FFN of a non-routed block, the attention output projection).
// The MFMA path fetches each 8-column piece of hbar (prep) before it stages the accumulators,
// so that the loads of a whole wave tile are in flight together.
template <typename T, bool ADAPTER>
struct EpiScatter {
  const int* idx;
  const T* hbar;
  const float* gate;
  T* out;
  int ld;
  __device__ __forceinline__ void store(int m, int n, float v) const {
    const int t = idx ? idx[m] : m;
    const float g = gate ? gate[t] : (ADAPTER ? 0.0f : 1.0f);
    const float sc = ADAPTER ? 1.0f - g : g;
    const size_t o = static_cast<size_t>(t) * ld + n;
    stf(out + o, ldf(hbar + o) + sc * v);
  }
  struct Pre {
    u32x4 h;
    uint32_t row;
    float sc;
  };
  __device__ __forceinline__ Pre prep(int m, int n) const {
    const int t = idx ? idx[m] : m;
    const float g = gate ? gate[t] : (ADAPTER ? 0.0f : 1.0f);
    Pre p;
    p.row = static_cast<uint32_t>(t);
    p.sc = ADAPTER ? 1.0f - g : g;
    p.h = *reinterpret_cast<const u32x4*>(hbar + static_cast<size_t>(t) * ld + n);
    return p;
  }
  __device__ __forceinline__ void emit8(const Pre& p, int, int n, const float* v) const {
    u32x4 w;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float lo = __uint_as_float(p.h[i] << 16) + p.sc * v[2 * i];
      const float hi = __uint_as_float(p.h[i] & 0xffff0000u) + p.sc * v[2 * i + 1];
      w[i] = static_cast<uint32_t>(f32_to_bf16(lo)) | (static_cast<uint32_t>(f32_to_bf16(hi)) << 16);
    }
    *reinterpret_cast<u32x4*>(out + static_cast<size_t>(p.row) * ld + n) = w;
  }
};

// ---------------------------------------------------------------------------
// bf16 MFMA GEMM
//
// One workgroup of WM x WN waves computes a BM x BN tile; each wave owns a
// (BM/WM) x (BN/WN) block of 32 x 32 MFMA tiles with fp32 accumulators.  The big
// products run 8 waves (two per SIMD) on a 256 x 256 (or 192 x 256) tile, so that one
// wave's MFMAs cover the other's waits.  K advances in 64-deep tiles through two
// LDS stages:
//   * each stage is filled by wave-wide global_load_lds_dwordx4: one instruction
//     moves 64 x 16 bytes into a contiguous 1 KiB of LDS, i.e. eight 128-byte
//     tile rows; lane L lands in row 8b + L/8 at physical chunk L%8 and so loads
//     logical chunk (L%8) ^ ((row/2)%8) of that row.  The fragment reads undo the
//     XOR; with it, the 16 lanes of one LDS read phase (16 consecutive rows, one
//     logical chunk) hit 16 distinct 16-byte slots of the 256-byte bank window;
//   * within a k-tile the fragments of the next 16-deep k-step are read while the
//     MFMAs of the current one run (two register sets), the reads interleaved one
//     by one with the MFMAs;
//   * the workgroup barrier sits before the last k-step: by then every wave has
//     read the whole stage, so the loads of tile k+2 are issued into it, one per
//     MFMA of that last k-step, together with the first fragment reads of tile k+1.
// A grid with gridDim.y = S > 1 splits K: workgroup y covers k-tiles [y n / S, (y + 1) n / S)
// of the n = K / 64 and its epilogue writes partial sums to a slice of its own (router
// pre-activations; FFN products with few rows).
// Epilogues: the gate/up product stages its finished bf16 tile in LDS at once and
// writes 16-byte row pieces; the others first fetch what they combine with (hbar
// rows) for the whole wave tile, then stage fp32 results in 32-row blocks.
// ---------------------------------------------------------------------------

typedef __attribute__((address_space(3))) void lds_void;

__device__ __forceinline__ void load_lds16(const void* g, unsigned char* l) {
  __builtin_amdgcn_global_load_lds(g, (lds_void*)(l), 16, 0, 0);
}

__device__ __forceinline__ int swz(int row, int ch) { return row * ROWB + ((ch ^ ((row >> 1) & 7)) << 4); }

constexpr int GROUP_M = 8;   // row tiles per group of the tile order
constexpr int kCUs = 256;    // compute units of an MI355X

// instruction classes of __builtin_amdgcn_sched_group_barrier
constexpr int SG_MFMA = 0x008, SG_VMEM_READ = 0x020, SG_DS_READ = 0x100;

// An epilogue with a block() member takes each staged 32-row block of a wave tile whole,
// instead of 8-column row pieces through emit8().
template <class E, class = void>
struct BlockEpilogue : std::false_type {};
template <class E>
struct BlockEpilogue<E, std::void_t<decltype(&E::block)>> : std::true_type {};
// A two-product epilogue with kDualHook takes the gate/up accumulators of a finished wave tile
// itself (the backward of the gated SwiGLU) instead of the forward's SiLU(gate) * up staging.
template <class E, class = void>
struct DualHook : std::false_type {};
template <class E>
struct DualHook<E, std::void_t<decltype(E::kDualHook)>> : std::true_type {};

template <class C, class Epi>
__device__ __forceinline__ void swiglu_bwd_tile(const Epi& epi, f32x16 (&acc)[C::TM][C::TN], unsigned char* smem, int m0,
                                int nt, int wave, int wm, int wn, int M, int lane);

// NS_: LDS stages of the k-loop; the loads of tile k + NS - 1 are in flight while tile k is
// consumed (2 for the big products, more where streaming weights from HBM needs more bytes in
// flight per CU).
// MI_: the matrix instruction, v_mfma_f32_32x32x16_bf16 (32) or v_mfma_f32_16x16x32_bf16 (16).
// Both run at the same nominal rate; on random data the 16 x 16 x 32 form sustains a markedly
// higher clock under the board's power limit (2.20 against 1.83-1.91 PFLOP/s in a register-only
// loop on all CUs), so the FFN products use it.
template <int BM_, int BN_, int WM_, int WN_, bool DUAL_, int NS_ = 2, int MI_ = 32>
struct Tile {
  static constexpr int BM = BM_, BN = BN_, WM = WM_, WN = WN_;
  static constexpr bool DUAL = DUAL_;
  static constexpr int NS = NS_;
  static constexpr int MI = MI_;
  static constexpr int NACC = MI * MI / 64;           // accumulator registers per MFMA tile
  using Acc = typename std::conditional<MI == 32, f32x16, f32x4>::type;
  static constexpr int KSTEP = MI == 32 ? 16 : 32;    // k per MFMA
  static constexpr int NT = 64 * WM * WN;
  static constexpr int NW = WM * WN;
  static constexpr int WTM = BM / WM, WTN = BN / WN;
  static constexpr int TM = WTM / MI, TN = WTN / MI;
  static constexpr int STAGE = (BM + BN) * ROWB;
  static constexpr int OUT_N = DUAL ? BN / 2 : BN;   // output columns per tile
  static constexpr int ON = DUAL ? WTN / 2 : WTN;     // output columns per wave
  static constexpr int OPAD = ON + 4;                 // fp32 staging row pitch (floats)
  static constexpr int SPAD = ON + 8;                 // bf16 staging row pitch (elements)
  static_assert(MI == 32 || MI == 16, "matrix instruction");
  static_assert(WTM % MI == 0 && WTN % MI == 0, "wave tile must be whole MFMA tiles");
  static_assert(!DUAL || TN % 2 == 0, "gate/up tiles come in pairs");
  static_assert(BM % (8 * NW) == 0 && BN % (8 * NW) == 0, "loader split");
  static_assert(DUAL ? NW * WTM * SPAD * 2 <= 2 * STAGE : NW * MI * OPAD * 4 <= 2 * STAGE,
                "epilogue staging must fit in the stages");
  static_assert((MI * (ON / 8)) % 64 == 0, "epilogue pieces split evenly over the lanes");
  static_assert(NS >= 2 && NS * STAGE <= 160 * 1024, "stages fit in LDS");
};

// Lane layout of the two matrix instructions (wave64).  Operands: lane l holds 8 consecutive k of
// row (l mod MI) of its 16 x 32 (MI 16) or 32 x 16 (MI 32) block, at k-chunk l / MI.  Result:
// element r of lane l is row frag_out_row(r, l), column (l mod MI) of the MI x MI tile.
template <int MI>
__device__ __forceinline__ int out_row(int r, int lane) {
  if constexpr (MI == 32)
    return 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
  else
    return 4 * (lane >> 4) + r;
}
template <int MI>
__device__ __forceinline__ int in_chunk(int ks, int lane) {   // 16-byte chunk of a 128-byte row
  if constexpr (MI == 32)
    return 2 * ks + (lane >> 5);
  else
    return 4 * ks + (lane >> 4);
}
__device__ __forceinline__ f32x16 mfma_op(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ f32x4 mfma_op(bf16x8 a, bf16x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

// s_waitcnt vmcnt(N) lgkmcnt(0) for a compile-time N
template <int N>
__device__ __forceinline__ void wait_vm_lgkm() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)" ::"n"(N) : "memory");
}

template <class C, class Epi>
__global__ __launch_bounds__(C::NT) void mfma_gemm(ARows<bf16_t> A, BRows<bf16_t> B, Epi epi,
                                                  const int* __restrict__ m_count, int M_fixed,
                                                  int K, int mt_max, int n_tiles) {
  constexpr int NW = C::NW;
  constexpr int A_LD = C::BM / 8 / NW;  // wave-wide loads per k-tile, A
  constexpr int B_LD = C::BN / 8 / NW;
  constexpr int KS = BK / C::KSTEP;     // k-steps per k-tile
  constexpr int MI = C::MI;
  constexpr int NM = C::TM * C::TN;     // MFMAs per k-step
  constexpr int NR = C::TM + C::TN;     // fragment reads per k-step
  constexpr int NL = A_LD + B_LD;       // stage loads per k-tile
  __shared__ __attribute__((aligned(1024))) unsigned char smem[C::NS * C::STAGE];
  // Workgroups go to the 8 XCDs round-robin; XCD x takes the contiguous range
  // [x per, (x+1) per) of a grouped tile order (GROUP_M row tiles by every column tile),
  // so that the 32 tiles one XCD runs at a time share 8 row panels and 4 column panels
  // in its L2.
  // The grid is sized for M_fixed rows; the order is laid over the rows that exist (the device
  // count), so that every XCD gets an equal share however few rows there are.
  const int M = m_count ? *m_count : M_fixed;
  const int mt_act = min(mt_max, (M + C::BM - 1) / C::BM);
  const int per = (mt_act * n_tiles + 7) >> 3;
  const int q = blockIdx.x >> 3;
  if (q >= per) return;
  const int tile = (blockIdx.x & 7) * per + q;
  if (tile >= mt_act * n_tiles) return;
  const int grp = tile / (GROUP_M * n_tiles), rem = tile % (GROUP_M * n_tiles);
  const int gsz = min(GROUP_M, mt_act - grp * GROUP_M);
  const int mt = grp * GROUP_M + rem % gsz, nt = rem / gsz;
  const int m0 = mt * C::BM;
  // split K: workgroup y covers k-tiles [y nkt / S, (y+1) nkt / S) (S = gridDim.y <= nkt)
  const int nkt = K / BK;
  const int kt0 = static_cast<int>(blockIdx.y) * nkt / static_cast<int>(gridDim.y);
  const int kt1 = (static_cast<int>(blockIdx.y) + 1) * nkt / static_cast<int>(gridDim.y);

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(static_cast<int>(threadIdx.x) >> 6);
  const int wm = wave / C::WN, wn = wave % C::WN;
  const int rsub = lane >> 3;

  const unsigned char* a_base = reinterpret_cast<const unsigned char*>(A.base);
  uint32_t a_off[A_LD];
#pragma unroll
  for (int i = 0; i < A_LD; ++i) {
    const int r = 8 * (i * NW + wave) + rsub;
    const int ch = (lane & 7) ^ ((r >> 1) & 7);
    const int m = min(m0 + r, M - 1);
    const int row = A.idx ? A.idx[m] : m;
    a_off[i] = static_cast<uint32_t>(row) * static_cast<uint32_t>(A.ld * 2) + ch * 16;
  }
  const unsigned char* b_base[B_LD];
  uint32_t b_off[B_LD];
#pragma unroll
  for (int i = 0; i < B_LD; ++i) {
    const int blk = i * NW + wave;  // 8-row block, wave-uniform
    const int r = 8 * blk + rsub;
    const int ch = (lane & 7) ^ ((r >> 1) & 7);
    const bf16_t* base;
    int row;
    if constexpr (C::DUAL) {
      const int wb = (8 * blk) / C::WTN, q0 = (8 * blk) % C::WTN, h = C::WTN / 2;
      const bool up = q0 >= h;
      base = up ? B.b1 : B.b0;
      row = nt * C::OUT_N + wb * h + (r % C::WTN) - (up ? h : 0);
    } else {
      const bool second = nt * C::BN + 8 * blk >= B.split;
      base = second ? B.b1 : B.b0;
      row = nt * C::BN + r - (second ? B.split : 0);
    }
    b_base[i] = reinterpret_cast<const unsigned char*>(base);
    b_off[i] = static_cast<uint32_t>(row) * static_cast<uint32_t>(B.ld * 2) + ch * 16;
  }

  auto issue = [&](int stage, int k0) {
    unsigned char* sa = smem + stage * C::STAGE;
    const uint32_t kb = static_cast<uint32_t>(k0 + kt0 * BK) * 2;
#pragma unroll
    for (int i = 0; i < A_LD; ++i) load_lds16(a_base + a_off[i] + kb, sa + (i * NW + wave) * 1024);
#pragma unroll
    for (int i = 0; i < B_LD; ++i)
      load_lds16(b_base[i] + b_off[i] + kb, sa + C::BM * ROWB + (i * NW + wave) * 1024);
  };

  typename C::Acc acc[C::TM][C::TN];
#pragma unroll
  for (int a = 0; a < C::TM; ++a)
#pragma unroll
    for (int b = 0; b < C::TN; ++b)
#pragma unroll
      for (int r = 0; r < C::NACC; ++r) acc[a][b][r] = 0.f;

  int fa_row[C::TM], fb_row[C::TN];
#pragma unroll
  for (int a = 0; a < C::TM; ++a) fa_row[a] = wm * C::WTM + a * MI + (lane & (MI - 1));
#pragma unroll
  for (int b = 0; b < C::TN; ++b) fb_row[b] = C::BM + wn * C::WTN + b * MI + (lane & (MI - 1));
  bf16x8 fa[2][C::TM], fb[2][C::TN];
  auto read_frags = [&](int buf, const unsigned char* st, int ks) {
    const int c = in_chunk<MI>(ks, lane);
#pragma unroll
    for (int a = 0; a < C::TM; ++a) fa[buf][a] = *reinterpret_cast<const bf16x8*>(st + swz(fa_row[a], c));
#pragma unroll
    for (int b = 0; b < C::TN; ++b) fb[buf][b] = *reinterpret_cast<const bf16x8*>(st + swz(fb_row[b], c));
  };
  auto mfmas = [&](int buf) {
#pragma unroll
    for (int a = 0; a < C::TM; ++a)
#pragma unroll
      for (int b = 0; b < C::TN; ++b)
        acc[a][b] = mfma_op(fa[buf][a], fb[buf][b], acc[a][b]);
  };
  // order within the current scheduling region: MFMA, then (while any remain) one stage load
  // and one fragment read after each
  auto interleave = [&](auto nl_, auto nr_) {
    constexpr int nl = decltype(nl_)::value, nr = decltype(nr_)::value;
#pragma unroll
    for (int i = 0; i < NM; ++i) {
      __builtin_amdgcn_sched_group_barrier(SG_MFMA, 1, 0);
      if (i < nl) __builtin_amdgcn_sched_group_barrier(SG_VMEM_READ, 1, 0);
      if (i < nr) __builtin_amdgcn_sched_group_barrier(SG_DS_READ, 1, 0);
    }
    if constexpr (nl > NM) __builtin_amdgcn_sched_group_barrier(SG_VMEM_READ, nl - NM, 0);
    if constexpr (nr > NM) __builtin_amdgcn_sched_group_barrier(SG_DS_READ, nr - NM, 0);
  };

  const int nk = kt1 - kt0;
  constexpr int NS = C::NS;
  // One k-tile.  MODE 2 (steady state): the loads of tile kt + NS go into the stage just
  // consumed and the first fragments of tile kt + 1 are read, both interleaved with the MFMAs
  // of the last k-step; MODE 1: no tile left to load; MODE 0: the last tile.  Each mode is its
  // own straight-line code, so that the scheduler can interleave the loads with the MFMAs
  // (a load under a run-time condition would sit in a block of its own and issue as a burst).
  auto ktile = [&](int kt, auto mode_) {
    constexpr int mode = decltype(mode_)::value;
    const unsigned char* st = smem + (kt % NS) * C::STAGE;
#pragma unroll
    for (int ks = 0; ks < KS - 1; ++ks) {
      read_frags((ks + 1) & 1, st, ks + 1);
      mfmas(ks & 1);
      interleave(std::integral_constant<int, 0>(), std::integral_constant<int, NR>());
      __builtin_amdgcn_sched_barrier(0);
    }
    // every wave has read all of stage kt and the loads of tile kt+1 have landed (tiles
    // kt+2 .. kt+NS-1 may still be in flight; near the end, fewer were issued)
    if constexpr (mode == 2)
      wait_vm_lgkm<(NS - 2) * NL>();
    else
      wait_vm_lgkm<0>();
    __syncthreads();
    if constexpr (mode == 2) issue(kt % NS, (kt + NS) * BK);
    if constexpr (mode >= 1) read_frags(KS & 1, smem + ((kt + 1) % NS) * C::STAGE, 0);
    mfmas((KS - 1) & 1);
    interleave(std::integral_constant<int, mode == 2 ? NL : 0>(), std::integral_constant<int, mode >= 1 ? NR : 0>());
    __builtin_amdgcn_sched_barrier(0);
  };

  // tiles 0 .. NS-1 into the NS stages; wait for tile 0 (the others may still be landing)
#pragma unroll
  for (int i = 0; i < NS; ++i)
    if (i < nk) issue(i, i * BK);
  if (nk >= NS)
    wait_vm_lgkm<(NS - 1) * NL>();
  else
    wait_vm_lgkm<0>();
  __syncthreads();
  read_frags(0, smem, 0);
  int kt = 0;
  for (; kt + NS < nk; ++kt) ktile(kt, std::integral_constant<int, 2>());
  for (; kt + 1 < nk; ++kt) ktile(kt, std::integral_constant<int, 1>());
  if (kt < nk) ktile(kt, std::integral_constant<int, 0>());

  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  __syncthreads();
  if constexpr (DualHook<Epi>::value) {
    static_assert(MI == 32, "the backward SwiGLU epilogue takes 32 x 32 accumulator tiles");
    swiglu_bwd_tile<C>(epi, acc, smem, m0, nt, wave, wm, wn, M, lane);
  } else if constexpr (C::DUAL) {
    // the wave's finished tile, SiLU(gate) * up in bf16, staged at once
    bf16_t* stg = reinterpret_cast<bf16_t*>(smem) + wave * (C::WTM * C::SPAD);
#pragma unroll
    for (int a = 0; a < C::TM; ++a)
#pragma unroll
      for (int r = 0; r < C::NACC; ++r) {
        const int i = a * MI + out_row<MI>(r, lane);
#pragma unroll
        for (int b = 0; b < C::TN / 2; ++b) {
          const float g = acc[a][b][r], u = acc[a][b + C::TN / 2][r];
          stg[i * C::SPAD + b * MI + (lane & (MI - 1))] =
              f32_to_bf16(g * __builtin_amdgcn_rcpf(1.0f + __expf(-g)) * u);
        }
      }
    constexpr int CPR = C::ON / 8;                 // 8-column pieces per row
    constexpr int PPL = C::WTM * CPR / kWave;      // pieces per lane
#pragma unroll
    for (int q = 0; q < PPL; ++q) {
      const int e = lane + kWave * q;
      const int i = e / CPR, c8 = (e % CPR) * 8;
      const int m = m0 + wm * C::WTM + i;
      const u32x4 v = *reinterpret_cast<const u32x4*>(stg + i * C::SPAD + c8);
      if (m < M) epi.emit_packed(m, nt * C::OUT_N + wn * C::ON + c8, v);
    }
  } else {
    constexpr int CPR = C::ON / 8;                 // 8-column pieces per staged row
    constexpr int PPB = MI * CPR / kWave;          // pieces per lane per MI-row block
    // what the epilogue combines with (hbar rows) is fetched ahead of the staging, so those loads
    // are in flight together: the whole wave tile with 32 x 32 tiles, 64 rows ahead with 16 x 16
    // tiles (whose narrower blocks would otherwise hold twice the registers)
    constexpr int AHEAD = MI == 32 ? C::TM : ((64 / MI) < C::TM ? (64 / MI) : C::TM);
    typename Epi::Pre pre[C::TM][PPB];
    auto fetch = [&](int a) {
#pragma unroll
      for (int q = 0; q < PPB; ++q) {
        const int e = lane + kWave * q;
        const int m = m0 + wm * C::WTM + a * MI + e / CPR;
        pre[a][q] = epi.prep(min(m, M - 1), nt * C::OUT_N + wn * C::ON + (e % CPR) * 8);
      }
    };
#pragma unroll
    for (int a = 0; a < AHEAD; ++a) fetch(a);
    float* stg = reinterpret_cast<float*>(smem) + wave * (MI * C::OPAD);
#pragma unroll
    for (int a = 0; a < C::TM; ++a) {
      if (a + AHEAD < C::TM) fetch(a + AHEAD);
#pragma unroll
      for (int r = 0; r < C::NACC; ++r) {
        const int i = out_row<MI>(r, lane);
#pragma unroll
        for (int b = 0; b < C::TN; ++b) stg[i * C::OPAD + b * MI + (lane & (MI - 1))] = acc[a][b][r];
      }
      if constexpr (BlockEpilogue<Epi>::value) {
        static_assert(MI == 32, "block epilogues take 32-row blocks");
        // the epilogue takes the whole staged 32-row block (any lane may read any element)
        epi.block(stg, C::OPAD, C::ON, m0 + wm * C::WTM + a * 32, nt * C::OUT_N + wn * C::ON, M, lane);
      } else {
#pragma unroll
        for (int q = 0; q < PPB; ++q) {
          const int e = lane + kWave * q;
          const int i = e / CPR, c8 = (e % CPR) * 8;
          const int m = m0 + wm * C::WTM + a * MI + i;
          if (m < M) epi.emit8(pre[a][q], m, nt * C::OUT_N + wn * C::ON + c8, stg + i * C::OPAD + c8);
        }
      }
    }
  }
}

// Backward SwiGLU epilogue of one wave tile (EpiSwiGLUBwd on the MFMA path).  Lane (lane & 31)
// holds column b 32 + (lane & 31) of gate tile b and of up tile b + TN/2, at rows
// a 32 + 8 (r >> 2) + 4 (lane >> 5) + (r & 3) for accumulator element r.  The wave's own LDS
// region (the stages are free once the k-loop has ended) holds in turn the rows' gates, the
// per-lane shares of <e, act> (one lane then sums each row), and the bf16 staging of dG, then
// dU, which leave as 16-byte row pieces.  A wave's LDS operations complete in order, so the
// region needs no barrier between these uses.
template <class C, class Epi>
__device__ __forceinline__ void swiglu_bwd_tile(const Epi& epi, f32x16 (&acc)[C::TM][C::TN], unsigned char* smem, int m0,
                                int nt, int wave, int wm, int wn, int M, int lane) {
  static_assert(C::DUAL, "gate/up tiles");
  constexpr int TM = C::TM, TH = C::TN / 2, WTM = C::WTM;
  constexpr int PP = 33;   // row pitch of the per-lane shares (floats): rows hit distinct banks
  constexpr int RP = (WTM + WTM * PP) * 4, RS = WTM * C::SPAD * 2;
  constexpr int REG = ((RP > RS ? RP : RS) + 15) / 16 * 16;
  static_assert(C::NW * REG <= C::NS * C::STAGE, "backward staging fits in the stages");
  unsigned char* reg = smem + wave * REG;
  float* gl = reinterpret_cast<float*>(reg);
  float* pr = gl + WTM;
  const int rw = m0 + wm * WTM;                   // first row of the wave tile
  const int col0 = nt * C::OUT_N + wn * C::ON;    // first output column of the wave
  for (int i = lane; i < WTM; i += kWave) {
    const int m = min(rw + i, M - 1);
    const int t = epi.idx ? epi.idx[m] : m;
    gl[i] = epi.gate ? epi.gate[t] : 1.0f;
  }
#pragma unroll
  for (int a = 0; a < TM; ++a) {
    // e at this lane's elements of the 32-row block, the loads in flight together: held as the
    // loaded 16-bit words and widened at use (widening at the load let the compiler wait for each
    // load in turn: 694 -> 798 us for the 8B layer's recompute)
    bf16_t ev[16][TH];
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int m = min(rw + a * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3), M - 1);
#pragma unroll
      for (int b = 0; b < TH; ++b) ev[r][b] = epi.e[static_cast<size_t>(m) * epi.ld_e + col0 + b * 32 + (lane & 31)];
    }
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int i = a * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
      const float gt = gl[i];
      float sum = 0.f;
#pragma unroll
      for (int b = 0; b < TH; ++b) {
        const float g = acc[a][b][r], u = acc[a][b + TH][r];
        const float sg = __builtin_amdgcn_rcpf(1.0f + __expf(-g));
        const float ee = bf16_to_f32(ev[r][b]);
        const float dact = gt * ee;
        sum += ee * (g * sg * u);
        acc[a][b][r] = dact * u * sg * (1.0f + g * (1.0f - sg));   // dG
        acc[a][b + TH][r] = dact * g * sg;                          // dU
      }
      pr[i * PP + (lane & 31)] = sum;
    }
  }
  for (int i = lane; i < WTM; i += kWave) {
    float v = 0.f;
#pragma unroll 8
    for (int c = 0; c < 32; ++c) v += pr[i * PP + c];
    if (rw + i < M) epi.dgpart[static_cast<size_t>(rw + i) * epi.n_parts + col0 / C::ON] = v;
  }
  bf16_t* stg = reinterpret_cast<bf16_t*>(reg);
  constexpr int CPR = C::ON / 8, PPL = WTM * CPR / kWave;
  static_assert(WTM * CPR % kWave == 0, "pieces split evenly over the lanes");
#pragma unroll
  for (int h = 0; h < 2; ++h) {
#pragma unroll
    for (int a = 0; a < TM; ++a)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int i = a * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
#pragma unroll
        for (int b = 0; b < TH; ++b) stg[i * C::SPAD + b * 32 + (lane & 31)] = f32_to_bf16(acc[a][b + h * TH][r]);
      }
#pragma unroll
    for (int q = 0; q < PPL; ++q) {
      const int e = lane + kWave * q;
      const int i = e / CPR, c8 = (e % CPR) * 8;
      const u32x4 v = *reinterpret_cast<const u32x4*>(stg + i * C::SPAD + c8);
      if (rw + i < M)
        *reinterpret_cast<u32x4*>(epi.dgu + static_cast<size_t>(rw + i) * epi.ld_dgu + h * epi.d_ff + col0 + c8) = v;
    }
  }
}

// ---------------------------------------------------------------------------
// Persistent gate/up product.  The plain kernel ends every tile with an epilogue during
// which the CU does no MFMA work, and all CUs reach it together, once per round of tiles.
// Here one workgroup per CU walks the tiles its XCD owns (the same grouped order and
// XCD ranges as mfma_gemm, workgroup q of an XCD taking every nq-th tile of the range);
// a finished tile is staged as bf16 SiLU(gate) * up in a third LDS region and written
// out at the start of the next tile's first k-tile, after its loads are in flight, so the
// stores overlap that tile's MFMAs.  Each wave stages and stores only its own block, so the
// staging region needs no barrier.  Results are identical to mfma_gemm's.
// ---------------------------------------------------------------------------
template <class C>
__global__ __launch_bounds__(C::NT) void gateup_persist(ARows<bf16_t> A, BRows<bf16_t> B,
                                                       EpiSwiGLU<bf16_t> epi,
                                                       const int* __restrict__ m_count, int M_fixed,
                                                       int K, int mt_max, int n_tiles) {
  static_assert(C::DUAL, "gate/up only");
  constexpr int NW = C::NW;
  constexpr int A_LD = C::BM / 8 / NW;
  constexpr int B_LD = C::BN / 8 / NW;
  constexpr int KS = BK / C::KSTEP;
  constexpr int MI = C::MI;
  constexpr int NM = C::TM * C::TN;
  constexpr int NR = C::TM + C::TN;
  constexpr int NL = A_LD + B_LD;
  constexpr int OUT_W = C::WTM * C::ON;            // staged bf16 elements per wave
  constexpr int CPR = C::ON / 8;                   // 16-byte pieces per staged row
  constexpr int PPL = C::WTM * CPR / kWave;        // pieces per lane
  __shared__ __attribute__((aligned(1024))) unsigned char smem[2 * C::STAGE + NW * OUT_W * 2];
  const int xcd = blockIdx.x & 7, q = blockIdx.x >> 3, nq = gridDim.x >> 3;
  const int M = m_count ? *m_count : M_fixed;
  const int mt_act = min(mt_max, (M + C::BM - 1) / C::BM);   // row tiles that exist
  const int total = mt_act * n_tiles;
  const int per = (total + 7) >> 3;                           // tiles per XCD
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(static_cast<int>(threadIdx.x) >> 6);
  const int wm = wave / C::WN, wn = wave % C::WN;
  const int rsub = lane >> 3;
  bf16_t* ostg = reinterpret_cast<bf16_t*>(smem + 2 * C::STAGE) + wave * OUT_W;
  const int nk = K / BK;

  int fa_row[C::TM], fb_row[C::TN];
#pragma unroll
  for (int a = 0; a < C::TM; ++a) fa_row[a] = wm * C::WTM + a * MI + (lane & (MI - 1));
#pragma unroll
  for (int b = 0; b < C::TN; ++b) fb_row[b] = C::BM + wn * C::WTN + b * MI + (lane & (MI - 1));
  bf16x8 fa[2][C::TM], fb[2][C::TN];
  typename C::Acc acc[C::TM][C::TN];
  auto read_frags = [&](int buf, const unsigned char* st, int ks) {
    const int c = in_chunk<MI>(ks, lane);
#pragma unroll
    for (int a = 0; a < C::TM; ++a) fa[buf][a] = *reinterpret_cast<const bf16x8*>(st + swz(fa_row[a], c));
#pragma unroll
    for (int b = 0; b < C::TN; ++b) fb[buf][b] = *reinterpret_cast<const bf16x8*>(st + swz(fb_row[b], c));
  };
  auto mfmas = [&](int buf) {
#pragma unroll
    for (int a = 0; a < C::TM; ++a)
#pragma unroll
      for (int b = 0; b < C::TN; ++b)
        acc[a][b] = mfma_op(fa[buf][a], fb[buf][b], acc[a][b]);
  };
  auto interleave = [&](auto nl_, auto nr_) {
    constexpr int nl = decltype(nl_)::value, nr = decltype(nr_)::value;
#pragma unroll
    for (int i = 0; i < NM; ++i) {
      __builtin_amdgcn_sched_group_barrier(SG_MFMA, 1, 0);
      if (i < nl) __builtin_amdgcn_sched_group_barrier(SG_VMEM_READ, 1, 0);
      if (i < nr) __builtin_amdgcn_sched_group_barrier(SG_DS_READ, 1, 0);
    }
    if constexpr (nl > NM) __builtin_amdgcn_sched_group_barrier(SG_VMEM_READ, nl - NM, 0);
    if constexpr (nr > NM) __builtin_amdgcn_sched_group_barrier(SG_DS_READ, nr - NM, 0);
  };
  // write this wave's staged block of the tile at (m0, nt) to act
  auto store_staged = [&](int m0, int nt) {
#pragma unroll
    for (int p = 0; p < PPL; ++p) {
      const int e = lane + kWave * p;
      const int i = e / CPR, c8 = (e % CPR) * 8;
      const int m = m0 + wm * C::WTM + i;
      const u32x4 v = *reinterpret_cast<const u32x4*>(ostg + i * C::ON + c8);
      if (m < M) epi.emit_packed(m, nt * C::OUT_N + wn * C::ON + c8, v);
    }
  };

  int prev_m0 = -1, prev_nt = 0;
  for (int li = q; li < per; li += nq) {
    const int tile = xcd * per + li;
    if (tile >= total) break;
    const int grp = tile / (GROUP_M * n_tiles), rem = tile % (GROUP_M * n_tiles);
    const int gsz = min(GROUP_M, mt_act - grp * GROUP_M);
    const int mt = grp * GROUP_M + rem % gsz, nt = rem / gsz;
    const int m0 = mt * C::BM;

    const unsigned char* a_base = reinterpret_cast<const unsigned char*>(A.base);
    uint32_t a_off[A_LD];
#pragma unroll
    for (int i = 0; i < A_LD; ++i) {
      const int r = 8 * (i * NW + wave) + rsub;
      const int ch = (lane & 7) ^ ((r >> 1) & 7);
      const int m = min(m0 + r, M - 1);
      const int row = A.idx ? A.idx[m] : m;
      a_off[i] = static_cast<uint32_t>(row) * static_cast<uint32_t>(A.ld * 2) + ch * 16;
    }
    const unsigned char* b_base[B_LD];
    uint32_t b_off[B_LD];
#pragma unroll
    for (int i = 0; i < B_LD; ++i) {
      const int blk = i * NW + wave;
      const int r = 8 * blk + rsub;
      const int ch = (lane & 7) ^ ((r >> 1) & 7);
      const int wb = (8 * blk) / C::WTN, q0 = (8 * blk) % C::WTN, h = C::WTN / 2;
      const bool up = q0 >= h;
      b_base[i] = reinterpret_cast<const unsigned char*>(up ? B.b1 : B.b0);
      const int row = nt * C::OUT_N + wb * h + (r % C::WTN) - (up ? h : 0);
      b_off[i] = static_cast<uint32_t>(row) * static_cast<uint32_t>(B.ld * 2) + ch * 16;
    }
    auto issue = [&](int stage, int k0) {
      unsigned char* sa = smem + stage * C::STAGE;
      const uint32_t kb = static_cast<uint32_t>(k0) * 2;
#pragma unroll
      for (int i = 0; i < A_LD; ++i) load_lds16(a_base + a_off[i] + kb, sa + (i * NW + wave) * 1024);
#pragma unroll
      for (int i = 0; i < B_LD; ++i)
        load_lds16(b_base[i] + b_off[i] + kb, sa + C::BM * ROWB + (i * NW + wave) * 1024);
    };

#pragma unroll
    for (int a = 0; a < C::TM; ++a)
#pragma unroll
      for (int b = 0; b < C::TN; ++b)
#pragma unroll
        for (int r = 0; r < C::NACC; ++r) acc[a][b][r] = 0.f;

    // every wave is past the previous tile's last barrier: the stages are free
    issue(0, 0);
    if (nk > 1) issue(1, BK);
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
    // the previous tile's results leave while this tile computes
    if (prev_m0 >= 0) store_staged(prev_m0, prev_nt);
    read_frags(0, smem, 0);
    // one k-tile; the modes are straight-line code as in mfma_gemm (2: the loads of tile kt + 2
    // and the first fragments of tile kt + 1 interleave with the last k-step; 1: no tile left to
    // load; 0: the last tile)
    auto ktile = [&](int kt, auto mode_) {
      constexpr int mode = decltype(mode_)::value;
      const unsigned char* st = smem + (kt & 1) * C::STAGE;
#pragma unroll
      for (int ks = 0; ks < KS - 1; ++ks) {
        read_frags((ks + 1) & 1, st, ks + 1);
        mfmas(ks & 1);
        interleave(std::integral_constant<int, 0>(), std::integral_constant<int, NR>());
        __builtin_amdgcn_sched_barrier(0);
      }
      asm volatile("s_waitcnt vmcnt(0) lgkmcnt(0)" ::: "memory");
      __syncthreads();
      if constexpr (mode == 2) issue(kt & 1, (kt + 2) * BK);
      if constexpr (mode >= 1) read_frags(KS & 1, smem + ((kt + 1) & 1) * C::STAGE, 0);
      mfmas((KS - 1) & 1);
      interleave(std::integral_constant<int, mode == 2 ? NL : 0>(),
                 std::integral_constant<int, mode >= 1 ? NR : 0>());
      __builtin_amdgcn_sched_barrier(0);
    };
    int kt = 0;
    for (; kt + 2 < nk; ++kt) ktile(kt, std::integral_constant<int, 2>());
    for (; kt + 1 < nk; ++kt) ktile(kt, std::integral_constant<int, 1>());
    if (kt < nk) ktile(kt, std::integral_constant<int, 0>());
    // stage SiLU(gate) * up of this wave's block (its previous contents were stored above)
#pragma unroll
    for (int a = 0; a < C::TM; ++a)
#pragma unroll
      for (int r = 0; r < C::NACC; ++r) {
        const int i = a * MI + out_row<MI>(r, lane);
#pragma unroll
        for (int b = 0; b < C::TN / 2; ++b) {
          const float g = acc[a][b][r], u = acc[a][b + C::TN / 2][r];
          ostg[i * C::ON + b * MI + (lane & (MI - 1))] = f32_to_bf16(g * __builtin_amdgcn_rcpf(1.0f + __expf(-g)) * u);
        }
      }
    prev_m0 = m0;
    prev_nt = nt;
  }
  if (prev_m0 >= 0) store_staged(prev_m0, prev_nt);
}

// Persistent launch: one workgroup per CU (a multiple of 8 workgroups so that each XCD holds
// the same number), each XCD owning a contiguous range of the grouped tile order.
template <class C>
hipError_t run_persist(ARows<bf16_t> A, BRows<bf16_t> B, EpiSwiGLU<bf16_t> epi, const int* m_count,
                       int M_max, int N_out, int K, hipStream_t s) {
  const int mt_max = (M_max + C::BM - 1) / C::BM;
  const int n_tiles = N_out / C::OUT_N;
  const int total = mt_max * n_tiles;
  if (total == 0) return hipSuccess;
  const int nq = std::min((total + 7) / 8, kCUs / 8);   // workgroups per XCD
  gateup_persist<C><<<8 * nq, C::NT, 0, s>>>(A, B, epi, m_count, M_max, K, mt_max, n_tiles);
  return hipGetLastError();
}

template <class C, class Epi>
hipError_t run_tile(ARows<bf16_t> A, BRows<bf16_t> B, Epi epi, const int* m_count, int M_max,
                    int N_out, int K, hipStream_t s, int splits = 1) {
  const int mt_max = (M_max + C::BM - 1) / C::BM;
  const int n_tiles = N_out / C::OUT_N;
  const int total = mt_max * n_tiles;
  if (total == 0) return hipSuccess;
  const dim3 grid((total + 7) / 8 * 8, splits);
  mfma_gemm<C, Epi><<<grid, C::NT, 0, s>>>(A, B, epi, m_count, M_max, K, mt_max, n_tiles);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Skinny products: a batch of at most 256 rows (a decode step) against weights streamed once
// from HBM.  The output columns are cut into 16-column blocks spread evenly over the workgroups
// (block group x takes the contiguous blocks [x nb / G, (x + 1) nb / G), and for the gate/up
// product the same blocks of W_u); S K-slices per block group where one workgroup per group
// would pull the activation rows through L2 too many times.
// Eight waves, one workgroup per CU.  Four consumers run the MFMAs (16 x 16 x 32), each on 16 RB
// rows against every weight block of the workgroup; four producers stage tiles into LDS, two the
// activation rows and two the weight rows, each pair into a ring of its own depth (weights come
// from HBM and need more bytes in flight than the L2-resident activations).  A producer's waits
// count only its own loads.  One barrier per k-tile, placed before the consumers' last k-step: by
// then they hold the whole stage in registers, so the producers refill it and the first
// fragments of the next tile are read while the last MFMAs run.
// What bounds it (measured on cold weights): a 64-deep k-tile takes 128 bytes from each weight
// row, and HBM serves such row-strided visits at ~3.5 TB/s (4.5 at 256 bytes, 5.3 at 512); with
// three or more row blocks the per-tile LDS traffic (DMA writes plus every consumer's fragment
// reads, ~108 KiB at 192 x 96) takes longer still, so deeper weight visits (which cost the
// activation ring its stages) and activation loads straight to registers both measured slower.
// ---------------------------------------------------------------------------
template <int NB_, int RB_, int NSA_, int NSB_, bool DUAL_>
struct Skinny {
  static constexpr int NB = NB_, RB = RB_, NSA = NSA_, NSB = NSB_;
  static constexpr bool DUAL = DUAL_;
  static constexpr int SL = DUAL ? 2 * NB : NB;   // 16-row weight blocks per stage
  static constexpr int MP = 64 * RB;              // rows covered (4 consumer waves x 16 RB)
  static constexpr int A_STAGE = MP * ROWB, B_STAGE = SL * 16 * ROWB;
  static constexpr int LDS = NSA * A_STAGE + NSB * B_STAGE;
  static constexpr int AL = MP / 16;              // 1 KiB loads per stage per A producer
  static constexpr int BL = SL;                   // 1 KiB loads per stage per B producer
  static_assert(LDS <= 160 * 1024, "stages fit in LDS");
  static_assert((NSA - 1) * AL < 64 && (NSB - 1) * BL < 64, "loads in flight within vmcnt");
  static_assert(NSA >= 2 && NSB >= 2 && RB >= 1 && RB <= 4 && NB >= 1, "shape");
};

// deepest weight ring that fits beside NSA activation stages
constexpr int skinny_nsb(int NB, int RB, bool dual, int NSA) {
  const int sl = dual ? 2 * NB : NB;
  int n = (160 * 1024 - NSA * 64 * RB * ROWB) / (sl * 16 * ROWB);
  n = n < 8 ? n : 8;
  return n < 63 / sl + 1 ? n : 63 / sl + 1;
}

template <int N>
__device__ __forceinline__ void wait_vm() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

// Epilogue: gate/up writes act[m][c] = bf16(SiLU(g) u) (out = act, ld = d_ff); otherwise the
// K-slice y writes fp32 sums to part + y split_stride (out = part, ld = N).
// tiled != 0: b0 holds the weights in the streaming order of tile_ffn_weights_kernel (16 x 64
// tiles, k-tile by k-tile, each k-tile's row of `tiled` 16-row blocks contiguous; for the
// gate/up product the W_g and W_u tiles of a block alternate) and b1, ldb are unused.  The same
// rows land in the same LDS slots either way, so the results are identical.  In the tiled order
// a workgroup's weights of one k-tile are one contiguous run of 2 KiB tiles, and the workgroups
// running the same k-tile read neighbouring runs, instead of 128-byte visits of rows 8 KiB apart.
template <class C>
__global__ __launch_bounds__(512) void skinny_gemm(ARows<bf16_t> A, const bf16_t* __restrict__ b0,
                                                  const bf16_t* __restrict__ b1, int ldb, int tiled,
                                                  void* __restrict__ out, int ld, size_t split_stride,
                                                  const int* __restrict__ m_count, int n_max, int K,
                                                  int nb, int G, int S) {
  __shared__ __attribute__((aligned(1024))) unsigned char smem[C::LDS];
  unsigned char* const sa = smem;
  unsigned char* const sb = smem + C::NSA * C::A_STAGE;
  // G block groups x S K-slices in slice-major order, laid over the 8 XCDs (round-robin dispatch)
  // in contiguous runs: the workgroups of one XCD share one or two K-slices of the activations
  // in its L2
  const int id = static_cast<int>(blockIdx.x), N = G * S;
  const int L = N % 8 == 0 ? (id & 7) * (N >> 3) + (id >> 3) : id;
  const int x = L % G, y = L / G;
  const int blk0 = x * nb / G;
  const int cnt = (x + 1) * nb / G - blk0;
  const int M = m_count ? min(*m_count, n_max) : n_max;
  if (M <= 0) return;
  const int nkt = K / BK;
  const int kt0 = y * nkt / S;
  const int nk = (y + 1) * nkt / S - kt0;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(static_cast<int>(threadIdx.x) >> 6);
  constexpr int NSA = C::NSA, NSB = C::NSB;

  if (wave >= 6) {
    // weight producer: loads q = 2 i + pw, LDS rows 8q .. 8q + 7 = half (q & 1) of block slot q / 2;
    // a workgroup with fewer than NB blocks reloads its last one into the spare slots
    const int pw = wave - 6;
    const unsigned char* base[C::BL];
    uint32_t off[C::BL];
    constexpr int GU = C::DUAL ? 2 : 1;                       // matrices interleaved in a tiled block
    const uint32_t tstride = tiled ? static_cast<uint32_t>(tiled) * GU * 16 * ROWB : ROWB;  // k-tile to k-tile
#pragma unroll
    for (int i = 0; i < C::BL; ++i) {
      const int q = 2 * i + pw, slot = q >> 1;
      const int j = slot % C::NB;
      const int r = 8 * q + (lane >> 3);
      const int ch = (lane & 7) ^ ((r >> 1) & 7);
      const int blk = blk0 + min(j, cnt - 1), rr = 8 * (q & 1) + (lane >> 3);
      const int second = C::DUAL && slot >= C::NB;
      if (tiled) {
        base[i] = reinterpret_cast<const unsigned char*>(b0);
        off[i] = ((static_cast<uint32_t>(kt0) * tiled + blk) * GU + second) * (16 * ROWB) + rr * ROWB + ch * 16;
      } else {
        base[i] = reinterpret_cast<const unsigned char*>(second ? b1 : b0);
        off[i] = static_cast<uint32_t>(16 * blk + rr) * static_cast<uint32_t>(ldb * 2) + kt0 * ROWB + ch * 16;
      }
    }
    auto issue = [&](int t) {
      unsigned char* st = sb + (t % NSB) * C::B_STAGE;
#pragma unroll
      for (int i = 0; i < C::BL; ++i) load_lds16(base[i] + off[i] + t * tstride, st + (2 * i + pw) * 1024);
    };
    for (int t = 0; t < NSB; ++t)
      if (t < nk) issue(t);
    // before barrier j tile j + 1 has landed; tiles up to j + NSB - 1 may be in flight
    for (int j = -1; j < nk; ++j) {
      if (j < 0) {
        if (nk >= NSB) wait_vm<(NSB - 1) * C::BL>(); else wait_vm<0>();
      } else if (j + NSB <= nk) {
        wait_vm<(NSB - 2) * C::BL>();
      } else {
        wait_vm<0>();
      }
      __syncthreads();
      if (j >= 0 && j + NSB < nk) issue(j + NSB);
    }
    return;
  }
  if (wave >= 4) {
    // activation producer: loads q = 2 i + pw, LDS rows 8q .. 8q + 7; rows past M repeat row M - 1
    const int pw = wave - 4;
    uint32_t off[C::AL];
#pragma unroll
    for (int i = 0; i < C::AL; ++i) {
      const int r = 8 * (2 * i + pw) + (lane >> 3);
      const int ch = (lane & 7) ^ ((r >> 1) & 7);
      const int m = min(r, M - 1);
      const int row = A.idx ? A.idx[m] : m;
      off[i] = static_cast<uint32_t>(row) * static_cast<uint32_t>(A.ld * 2) + kt0 * ROWB + ch * 16;
    }
    const unsigned char* abase = reinterpret_cast<const unsigned char*>(A.base);
    auto issue = [&](int t) {
      unsigned char* st = sa + (t % NSA) * C::A_STAGE;
#pragma unroll
      for (int i = 0; i < C::AL; ++i) load_lds16(abase + off[i] + t * ROWB, st + (2 * i + pw) * 1024);
    };
    for (int t = 0; t < NSA; ++t)
      if (t < nk) issue(t);
    for (int j = -1; j < nk; ++j) {
      if (j < 0) {
        if (nk >= NSA) wait_vm<(NSA - 1) * C::AL>(); else wait_vm<0>();
      } else if (j + NSA <= nk) {
        wait_vm<(NSA - 2) * C::AL>();
      } else {
        wait_vm<0>();
      }
      __syncthreads();
      if (j >= 0 && j + NSA < nk) issue(j + NSA);
    }
    return;
  }

  // consumers
  constexpr int RB = C::RB, SL = C::SL;
  f32x4 acc[RB][SL];
#pragma unroll
  for (int r = 0; r < RB; ++r)
#pragma unroll
    for (int c = 0; c < SL; ++c) acc[r][c] = f32x4{0.f, 0.f, 0.f, 0.f};
  bf16x8 fa[2][RB], fb[2][SL];
  const int arow0 = wave * 16 * RB + (lane & 15), brow0 = lane & 15;
  auto read = [&](int buf, const unsigned char* ast, const unsigned char* bst, int ks) {
    const int c = in_chunk<16>(ks, lane);
#pragma unroll
    for (int r = 0; r < RB; ++r) fa[buf][r] = *reinterpret_cast<const bf16x8*>(ast + swz(arow0 + 16 * r, c));
#pragma unroll
    for (int b = 0; b < SL; ++b) fb[buf][b] = *reinterpret_cast<const bf16x8*>(bst + swz(brow0 + 16 * b, c));
  };
  auto mfmas = [&](int buf) {
#pragma unroll
    for (int r = 0; r < RB; ++r)
#pragma unroll
      for (int b = 0; b < SL; ++b) acc[r][b] = mfma_op(fa[buf][r], fb[buf][b], acc[r][b]);
  };
  // the fragment reads of the other k-step go out one after each MFMA; the reads of tile kt + 1
  // past the last tile hit a stale stage and are never used
  auto interleave = [&]() {
#pragma unroll
    for (int i = 0; i < RB * SL; ++i) {
      __builtin_amdgcn_sched_group_barrier(SG_MFMA, 1, 0);
      if (i < RB + SL) __builtin_amdgcn_sched_group_barrier(SG_DS_READ, 1, 0);
    }
    if constexpr (RB + SL > RB * SL) __builtin_amdgcn_sched_group_barrier(SG_DS_READ, RB + SL - RB * SL, 0);
  };
  __syncthreads();                       // barrier -1: tile 0 has landed
  read(0, sa, sb, 0);
  int ia = 0, ib = 0;                    // stages of tile kt
  for (int kt = 0; kt < nk; ++kt) {
    read(1, sa + ia * C::A_STAGE, sb + ib * C::B_STAGE, 1);
    mfmas(0);
    interleave();
    __builtin_amdgcn_sched_barrier(0);
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
    __syncthreads();                     // barrier kt: stage kt is free, tile kt + 1 has landed
    ia = ia + 1 == NSA ? 0 : ia + 1;
    ib = ib + 1 == NSB ? 0 : ib + 1;
    read(0, sa + ia * C::A_STAGE, sb + ib * C::B_STAGE, 0);
    mfmas(1);
    interleave();
    __builtin_amdgcn_sched_barrier(0);
  }

  // element i of acc[r][b] in lane l: row 16 (wave RB + r) + 4 (l >> 4) + i, column l & 15
  const int col = lane & 15;
#pragma unroll
  for (int r = 0; r < RB; ++r)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int m = 16 * (wave * RB + r) + 4 * (lane >> 4) + i;
      if (m >= M) continue;
      if constexpr (C::DUAL) {
        bf16_t* o = static_cast<bf16_t*>(out) + static_cast<size_t>(m) * ld;
#pragma unroll
        for (int j = 0; j < C::NB; ++j) {
          if (j >= cnt) break;
          const float g = acc[r][j][i], u = acc[r][C::NB + j][i];
          o[16 * (blk0 + j) + col] = f32_to_bf16(g * __builtin_amdgcn_rcpf(1.0f + __expf(-g)) * u);
        }
      } else {
        float* o = static_cast<float*>(out) + y * split_stride + static_cast<size_t>(m) * ld;
#pragma unroll
        for (int j = 0; j < C::NB; ++j) {
          if (j >= cnt) break;
          o[16 * (blk0 + j) + col] = acc[r][j][i];
        }
      }
    }
}

template <class C>
hipError_t run_skinny(ARows<bf16_t> A, const bf16_t* b0, const bf16_t* b1, int ldb, int tiled, void* out, int ld,
                      size_t split_stride, const int* m_count, int n_max, int K, int nb, int G, int S,
                      hipStream_t s) {
  skinny_gemm<C><<<G * S, 512, 0, s>>>(A, b0, b1, ldb, tiled, out, ld, split_stride, m_count, n_max, K, nb, G, S);
  return hipGetLastError();
}

// Time of a launch in units of one round of 192-row tiles: CU rounds times the relative
// duration of a round.  A 256-row tile moves fewer bytes through L2 per FLOP, so its round
// takes ~1.23x (not 256/192 = 1.33x) a 192-row round on the FFN products (measured on the
// Llama-3.1-8B gate/up and down shapes at 3k-20k rows).
double tile_cost(int M, int BM, int n_tiles) {
  const int tiles = (M + BM - 1) / BM * n_tiles;
  return static_cast<double>((tiles + kCUs - 1) / kCUs) * (BM == 256 ? 1.23 : 1.0);
}

// Big-tile launch: 256 or 192 rows per tile, whichever finishes in fewer CU-rounds.  The FFN
// products run the 16 x 16 x 32 instruction (MI = 16); other users keep 32 x 32 x 16 tiles.
template <int BN, bool DUAL, class Epi, int MI = 32>
hipError_t run_big(ARows<bf16_t> A, BRows<bf16_t> B, Epi epi, const int* m_count, int M_max,
                   int N_out, int K, hipStream_t s) {
  using T256 = Tile<256, BN, 2, 4, DUAL, 2, MI>;
  using T192 = Tile<192, BN, 2, 4, DUAL, 2, MI>;
  const int n_tiles = N_out / T256::OUT_N;
  if (tile_cost(M_max, 192, n_tiles) < tile_cost(M_max, 256, n_tiles)) {
    if constexpr (DUAL) {
      // more tiles than CUs: the persistent kernel hides each tile's epilogue behind the next
      if ((M_max + 191) / 192 * n_tiles > kCUs) return run_persist<T192>(A, B, epi, m_count, M_max, N_out, K, s);
    }
    return run_tile<T192>(A, B, epi, m_count, M_max, N_out, K, s);
  }
  return run_tile<T256>(A, B, epi, m_count, M_max, N_out, K, s);
}

// ---------------------------------------------------------------------------
// fp32 VALU GEMM (64 x 64 tile, 4 x 4 outputs per thread, full bounds checks)
// ---------------------------------------------------------------------------

template <bool DUAL, class Epi>
__global__ __launch_bounds__(256) void f32_gemm(ARows<float> A, BRows<float> B, Epi epi,
                                               const int* __restrict__ m_count, int M_fixed,
                                               int N, int K) {
  __shared__ float As[16][68];
  __shared__ float Bs[16][68];
  __shared__ float Us[DUAL ? 16 : 1][68];
  const int M = m_count ? *m_count : M_fixed;
  const int m0 = blockIdx.y * 64, n0 = blockIdx.x * 64;
  if (m0 >= M) return;
  const int tx = threadIdx.x & 15, ty = threadIdx.x >> 4;
  float acc[4][4], acu[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = acu[i][j] = 0.f;
  for (int k0 = 0; k0 < K; k0 += 16) {
    for (int e = threadIdx.x; e < 64 * 16; e += 256) {
      const int r = e >> 4, kk = e & 15, k = k0 + kk;
      const int m = m0 + r, n = n0 + r;
      As[kk][r] = (m < M && k < K) ? A.row(m)[k] : 0.f;
      if (DUAL) {
        Bs[kk][r] = (n < N && k < K) ? B.gate_row(n)[k] : 0.f;
        Us[kk][r] = (n < N && k < K) ? B.up_row(n)[k] : 0.f;
      } else {
        Bs[kk][r] = (n < N && k < K) ? B.row(n)[k] : 0.f;
      }
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < 16; ++kk) {
      float a[4], b[4], u[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        a[i] = As[kk][ty * 4 + i];
        b[i] = Bs[kk][tx * 4 + i];
        if (DUAL) u[i] = Us[kk][tx * 4 + i];
      }
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          acc[i][j] = fmaf(a[i], b[j], acc[i][j]);
          if (DUAL) acu[i][j] = fmaf(a[i], u[j], acu[i][j]);
        }
    }
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int m = m0 + ty * 4 + i;
    if (m >= M) continue;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int n = n0 + tx * 4 + j;
      if (n >= N) continue;
      if constexpr (DUAL) {
        epi.store2(m, n, acc[i][j], acu[i][j]);
      } else {
        epi.store(m, n, acc[i][j]);
      }
    }
  }
}

template <bool DUAL, class Epi>
hipError_t run_f32(ARows<float> A, BRows<float> B, Epi epi, const int* m_count, int M_max, int N,
                   int K, hipStream_t s) {
  if (M_max <= 0 || N <= 0) return hipSuccess;
  dim3 grid((N + 63) / 64, (M_max + 63) / 64);
  f32_gemm<DUAL, Epi><<<grid, 256, 0, s>>>(A, B, epi, m_count, M_max, N, K);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// bf16 adapter: skinny GEMMs with MFMA fragments loaded straight from memory
// ---------------------------------------------------------------------------

// Adapter down-projection partial sums.  Workgroup (row tile of 32, k-group g) has
// 4 waves, each over a quarter of the group's k range; the 4 partial 32 x d_r
// tiles are summed in LDS and written to part[g][m][n] (fp32).
template <int TN, int SB>
__global__ __launch_bounds__(256) void adapter_down_bf16(const bf16_t* __restrict__ u0,
                                                         const int* __restrict__ idx,
                                                         const int* __restrict__ m_count,
                                                         const bf16_t* __restrict__ w0,
                                                         float* __restrict__ part0, int T, int K,
                                                         int k_group, const bf16_t* __restrict__ u_z1,
                                                         const bf16_t* __restrict__ w_z1,
                                                         float* __restrict__ part_z1) {
  // gridDim.z = 2 runs a second product over the same rows (the backward's z and e_a)
  const bf16_t* __restrict__ u = blockIdx.z ? u_z1 : u0;
  const bf16_t* __restrict__ w1 = blockIdx.z ? w_z1 : w0;
  float* __restrict__ part = blockIdx.z ? part_z1 : part0;
  constexpr int R = TN * 32;
  __shared__ float red[4][32][R + 1];
  const int M = *m_count;
  const int m0 = blockIdx.x * 32;
  if (m0 >= M) return;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int g = blockIdx.y;
  const int kw = k_group / 4;
  const int kbeg = g * k_group + wave * kw;
  const int m = min(m0 + (lane & 31), M - 1);
  const bf16_t* arow = u + static_cast<size_t>(idx[m]) * K + 8 * (lane >> 5);
  f32x16 acc[TN];
#pragma unroll
  for (int b = 0; b < TN; ++b)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[b][r] = 0.f;
  // SB 16-deep k-steps per batch, all of a batch's loads issued first (kw % (16 SB) == 0)
  for (int k = kbeg; k < kbeg + kw; k += 16 * SB) {
    bf16x8 fa[SB], fb[SB][TN];
#pragma unroll
    for (int st = 0; st < SB; ++st) {
      fa[st] = *reinterpret_cast<const bf16x8*>(arow + k + 16 * st);
#pragma unroll
      for (int b = 0; b < TN; ++b)
        fb[st][b] = *reinterpret_cast<const bf16x8*>(
            w1 + static_cast<size_t>(b * 32 + (lane & 31)) * K + 8 * (lane >> 5) + k + 16 * st);
    }
    __builtin_amdgcn_sched_barrier(0);   // keep the whole batch of loads ahead of the MFMAs
#pragma unroll
    for (int st = 0; st < SB; ++st)
#pragma unroll
      for (int b = 0; b < TN; ++b)
        acc[b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[st], fb[st][b], acc[b], 0, 0, 0);
  }
#pragma unroll
  for (int b = 0; b < TN; ++b)
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int i = 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
      red[wave][i][b * 32 + (lane & 31)] = acc[b][r];
    }
  __syncthreads();
  for (int e = threadIdx.x; e < 32 * R; e += 256) {
    const int i = e / R, n = e % R;
    if (m0 + i >= M) continue;
    const float v = red[0][i][n] + red[1][i][n] + red[2][i][n] + red[3][i][n];
    part[(static_cast<size_t>(g) * T + m0 + i) * R + n] = v;
  }
}

// Adapter up-projection with scatter, one workgroup per (32 rows, 256 columns):
//   hid = SiLU(sum_g part[g]) for the 32 rows, rounded to bf16 (the MFMA A operand), in LDS;
//   each wave computes 64 columns; results are staged in LDS and every thread then writes
//   8-column pieces h_out[t] = hbar[t] + (1 - g_t) acc with hbar fetched at the start.
template <int KR, int G>
__global__ __launch_bounds__(256) void adapter_up_bf16(const float* __restrict__ part,
                                                       const int* __restrict__ idx,
                                                       const int* __restrict__ m_count,
                                                       const bf16_t* __restrict__ w2,
                                                       const bf16_t* __restrict__ hbar,
                                                       const float* __restrict__ gate,
                                                       bf16_t* __restrict__ out, int T, int d) {
  constexpr int NC = 256;
  constexpr int HP = KR + 8;     // hid row pitch (bf16)
  constexpr int SP = NC + 4;     // staged row pitch (fp32)
  constexpr int PPT = 32 * NC / 8 / 256;   // 8-column output pieces per thread
  __shared__ __attribute__((aligned(16))) bf16_t hid[32 * HP];
  __shared__ __attribute__((aligned(16))) float stg[32 * SP];
  const int M = *m_count;
  const int m0 = blockIdx.x * 32;
  if (m0 >= M) return;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int n0 = blockIdx.y * NC;
  EpiScatter<bf16_t, true> epi{idx, hbar, gate, out, d};
  typename EpiScatter<bf16_t, true>::Pre pre[PPT];
#pragma unroll
  for (int q = 0; q < PPT; ++q) {
    const int e = tid + 256 * q;
    pre[q] = epi.prep(min(m0 + (e >> 5), M - 1), n0 + (e & 31) * 8);
  }
  for (int e = tid; e < 32 * KR / 8; e += 256) {
    const int i = e / (KR / 8), k8 = (e % (KR / 8)) * 8;
    const int mr = min(m0 + i, M - 1);
    f32x4 x[G][2];
#pragma unroll
    for (int g = 0; g < G; ++g) {
      const float* p = part + (static_cast<size_t>(g) * T + mr) * KR + k8;
      x[g][0] = *reinterpret_cast<const f32x4*>(p);
      x[g][1] = *reinterpret_cast<const f32x4*>(p + 4);
    }
    bf16x8 v;
#pragma unroll
    for (int c = 0; c < 8; ++c) {
      float h = 0.f;
#pragma unroll
      for (int g = 0; g < G; ++g) h += x[g][c >> 2][c & 3];
      v[c] = static_cast<__bf16>(siluf_(h));
    }
    *reinterpret_cast<bf16x8*>(hid + i * HP + k8) = v;
  }
  bf16x8 fb[KR / 16][2];
#pragma unroll
  for (int st = 0; st < KR / 16; ++st)
#pragma unroll
    for (int b = 0; b < 2; ++b)
      fb[st][b] = *reinterpret_cast<const bf16x8*>(
          w2 + static_cast<size_t>(n0 + wave * 64 + b * 32 + (lane & 31)) * KR + 16 * st + 8 * (lane >> 5));
  __syncthreads();
  f32x16 acc[2];
#pragma unroll
  for (int b = 0; b < 2; ++b)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[b][r] = 0.f;
#pragma unroll
  for (int st = 0; st < KR / 16; ++st) {
    const bf16x8 fa = *reinterpret_cast<const bf16x8*>(hid + (lane & 31) * HP + 16 * st + 8 * (lane >> 5));
#pragma unroll
    for (int b = 0; b < 2; ++b) acc[b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa, fb[st][b], acc[b], 0, 0, 0);
  }
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    const int i = 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
#pragma unroll
    for (int b = 0; b < 2; ++b) stg[i * SP + wave * 64 + b * 32 + (lane & 31)] = acc[b][r];
  }
  __syncthreads();
#pragma unroll
  for (int q = 0; q < PPT; ++q) {
    const int e = tid + 256 * q;
    const int i = e >> 5, c8 = (e & 31) * 8;
    if (m0 + i < M) epi.emit8(pre[q], m0 + i, n0 + c8, stg + i * SP + c8);
  }
}

template <int KR>
void adapter_up_launch(dim3 g2, hipStream_t s, int G, const float* part, const int* idx, const int* counts,
                       const bf16_t* w2, const bf16_t* hb, const float* gate, bf16_t* ho, int T, int d) {
  switch (G) {
    case 1: adapter_up_bf16<KR, 1><<<g2, 256, 0, s>>>(part, idx, counts, w2, hb, gate, ho, T, d); break;
    case 2: adapter_up_bf16<KR, 2><<<g2, 256, 0, s>>>(part, idx, counts, w2, hb, gate, ho, T, d); break;
    case 4: adapter_up_bf16<KR, 4><<<g2, 256, 0, s>>>(part, idx, counts, w2, hb, gate, ho, T, d); break;
    default: adapter_up_bf16<KR, 8><<<g2, 256, 0, s>>>(part, idx, counts, w2, hb, gate, ho, T, d); break;
  }
}

// K-slices of the adapter down-projection: up to 8, each deep enough for whole batches
// (four waves times SB 16-deep k-steps); eight-step batches where the depth allows.
int adapter_groups(int K) {
  int G = 8;
  while (G > 1 && K % (G * 512) != 0) G >>= 1;
  if (K % (G * 512) != 0) {
    G = 8;
    while (G > 1 && K % (G * 256) != 0) G >>= 1;
  }
  return G;
}
int adapter_batch(int K, int G) { return (K / G) % 512 == 0 ? 8 : 4; }
// The forward's K-slices for a call of up to n_max adapter rows: fewer as the rows alone give
// enough workgroups (the up-projection reads every slice once per 256-column block, so at the
// 8B stack's 12.7k adapter rows eight slices would be read 16 times over for nothing).
int adapter_groups_rows(int K, int n_max) {
  int G = adapter_groups(K);
  const long long row_tiles = (static_cast<long long>(n_max) + 31) / 32;
  while (G > 1 && row_tiles * G > 2048) G >>= 1;
  return G;
}

// router pre-activations: 128-row tiles over all 8 waves, K split four ways
using TileRouter = Tile<128, 256, 2, 4, false>;
using TileRouterNarrow = Tile<128, 128, 2, 4, false>;
// few tokens (a decode batch): 64-row tiles of 4 waves, four times the workgroups; each streams
// a quarter of K, with three k-tiles in flight
using TileRouterSmall = Tile<64, 128, 1, 4, false, 4>;
// many tokens: 256 x 256 tiles on v_mfma_f32_16x16x32_bf16
using TileRouterBig = Tile<256, 256, 2, 4, false, 2, 16>;

}  // namespace

// K split of the router pre-activation product: four slices while the tiles alone would leave
// most CUs idle (a 4096-token layer has 64 tiles of 128 x 256), fewer as the token count grows,
// none from one full round of tiles on (32768 tokens: 512 tiles), where the slices would only add
// fp32 partial traffic for the router's pre pass to read.
int router_gemm_splits(int dtype, int d, int T, int N) {
  if (dtype != 1 || d % (4 * 64) != 0) return 1;
  if (T <= 1024) return 4;
  const long long tiles = static_cast<long long>((T + TileRouter::BM - 1) / TileRouter::BM) *
                          ((N + TileRouter::BN - 1) / TileRouter::BN);
  return static_cast<int>(std::max(1LL, std::min(4LL, kCUs / std::max(1LL, tiles))));
}

hipError_t launch_router_gemm(int dtype, const void* hbar, const void* w_hd, const void* ps1, int T,
                              int d, int d_e, int d_head, float* P, hipStream_t s) {
  const int N = d_e + d_head;
  EpiStoreF32 epi{P, N, static_cast<size_t>(T) * N};
  if (dtype == 1) {
    ARows<bf16_t> A{static_cast<const bf16_t*>(hbar), nullptr, d};
    BRows<bf16_t> B{static_cast<const bf16_t*>(w_hd), static_cast<const bf16_t*>(ps1), d_e, d};
    const int splits = router_gemm_splits(dtype, d, T, N);
    if (T <= 1024 && N % TileRouterSmall::OUT_N == 0)
      return run_tile<TileRouterSmall>(A, B, epi, nullptr, T, N, d, s, splits);
    // a full round or more of tiles: the FFN products' 256 x 256 tiles on the 16 x 16 x 32
    // instruction (32768 tokens: 256 tiles, no K split)
    if (splits == 1 && T >= 16384 && N % TileRouterBig::OUT_N == 0)
      return run_tile<TileRouterBig>(A, B, epi, nullptr, T, N, d, s);
    if (N % TileRouter::OUT_N == 0) return run_tile<TileRouter>(A, B, epi, nullptr, T, N, d, s, splits);
    return run_tile<TileRouterNarrow>(A, B, epi, nullptr, T, N, d, s, splits);
  }
  ARows<float> A{static_cast<const float*>(hbar), nullptr, d};
  BRows<float> B{static_cast<const float*>(w_hd), static_cast<const float*>(ps1), d_e, d};
  return run_f32<false>(A, B, epi, nullptr, T, N, d, s);
}

namespace {

// ---------------------------------------------------------------------------
// FFN products with few rows (a decode batch): the plain launch has fewer output tiles than
// half the CUs, each streaming the whole of K.  K is then split S ways (the most that keeps
// the launch within one round of workgroups), the slices write fp32 partial sums, and a pass
// over them adds the S slices in a fixed order and finishes the epilogue.
// ---------------------------------------------------------------------------
using TileSplitGU = Tile<192, 256, 2, 4, false>;    // [W_g; W_u] as one 2 d_ff-row operand
using TileSplitDown = Tile<192, 128, 2, 4, false, 4>;
constexpr int kMaxSplitGU = 8, kMaxSplitDown = 16;

// At most 256 rows (a decode batch): the skinny products.  Gate/up: one workgroup per CU, each
// with 2-4 blocks of 16 columns of W_g and W_u and the whole of K.  Down: blocks of 8 x 16 output
// columns by kSkinnyDownS K-slices, whose fp32 partial sums a pass adds in a fixed order.
constexpr int kSkinnyRows = 256, kSkinnyDownNB = 8, kSkinnyDownS = 8;
bool skinny_gateup_fits(int n_max, int d, int d_ff) {
  const int nb = d_ff / 16;
  return n_max <= kSkinnyRows && d % BK == 0 && d_ff % 16 == 0 && nb <= 4 * kCUs;
}
int skinny_down_splits(int d, int d_ff) {
  const int G = d / (16 * kSkinnyDownNB), nkt = d_ff / BK;
  return std::max(1, std::min({kSkinnyDownS, kCUs / std::max(G, 1), nkt}));
}
bool skinny_down_fits(int n_max, int d, int d_ff) {
  return n_max <= kSkinnyRows && d % (16 * kSkinnyDownNB) == 0 && d_ff % BK == 0;
}

template <int NB, int RB>
hipError_t skinny_gateup_nb_rb(ARows<bf16_t> A, const bf16_t* wg, const bf16_t* wu, const bf16_t* tiled,
                               bf16_t* act, const int* counts, int n_max, int d, int d_ff, hipStream_t s) {
  using C = Skinny<NB, RB, 3, skinny_nsb(NB, RB, true, 3), true>;
  const int nb = d_ff / 16, G = std::min(kCUs, nb);
  if (tiled) return run_skinny<C>(A, tiled, nullptr, 0, nb, act, d_ff, 0, counts, n_max, d, nb, G, 1, s);
  return run_skinny<C>(A, wg, wu, d, 0, act, d_ff, 0, counts, n_max, d, nb, G, 1, s);
}
template <int NB>
hipError_t skinny_gateup_nb(ARows<bf16_t> A, const bf16_t* wg, const bf16_t* wu, const bf16_t* tiled,
                            bf16_t* act, const int* counts, int n_max, int d, int d_ff, hipStream_t s) {
  switch ((n_max + 63) / 64) {
    case 1: return skinny_gateup_nb_rb<NB, 1>(A, wg, wu, tiled, act, counts, n_max, d, d_ff, s);
    case 2: return skinny_gateup_nb_rb<NB, 2>(A, wg, wu, tiled, act, counts, n_max, d, d_ff, s);
    case 3: return skinny_gateup_nb_rb<NB, 3>(A, wg, wu, tiled, act, counts, n_max, d, d_ff, s);
    default: return skinny_gateup_nb_rb<NB, 4>(A, wg, wu, tiled, act, counts, n_max, d, d_ff, s);
  }
}
hipError_t skinny_gateup(ARows<bf16_t> A, const bf16_t* wg, const bf16_t* wu, const bf16_t* tiled, bf16_t* act,
                         const int* counts, int n_max, int d, int d_ff, hipStream_t s) {
  const int nb = d_ff / 16, G = std::min(kCUs, nb);
  switch ((nb + G - 1) / G) {   // most blocks a workgroup takes
    case 1: return skinny_gateup_nb<1>(A, wg, wu, tiled, act, counts, n_max, d, d_ff, s);
    case 2: return skinny_gateup_nb<2>(A, wg, wu, tiled, act, counts, n_max, d, d_ff, s);
    case 3: return skinny_gateup_nb<3>(A, wg, wu, tiled, act, counts, n_max, d, d_ff, s);
    default: return skinny_gateup_nb<4>(A, wg, wu, tiled, act, counts, n_max, d, d_ff, s);
  }
}
template <int RB>
hipError_t skinny_down_rb(ARows<bf16_t> A, const bf16_t* wd, const bf16_t* tiled, float* part, size_t stride,
                          const int* counts, int n_max, int d, int d_ff, int S, hipStream_t s) {
  using C = Skinny<kSkinnyDownNB, RB, 3, skinny_nsb(kSkinnyDownNB, RB, false, 3), false>;
  const int nb = d / 16;
  if (tiled)
    return run_skinny<C>(A, tiled, nullptr, 0, nb, part, d, stride, counts, n_max, d_ff, nb, nb / kSkinnyDownNB, S, s);
  return run_skinny<C>(A, wd, nullptr, d_ff, 0, part, d, stride, counts, n_max, d_ff, nb, nb / kSkinnyDownNB, S, s);
}
hipError_t skinny_down(ARows<bf16_t> A, const bf16_t* wd, const bf16_t* tiled, float* part, size_t stride,
                       const int* counts, int n_max, int d, int d_ff, int S, hipStream_t s) {
  switch ((n_max + 63) / 64) {
    case 1: return skinny_down_rb<1>(A, wd, tiled, part, stride, counts, n_max, d, d_ff, S, s);
    case 2: return skinny_down_rb<2>(A, wd, tiled, part, stride, counts, n_max, d, d_ff, S, s);
    case 3: return skinny_down_rb<3>(A, wd, tiled, part, stride, counts, n_max, d, d_ff, S, s);
    default: return skinny_down_rb<4>(A, wd, tiled, part, stride, counts, n_max, d, d_ff, S, s);
  }
}

int split_ways(int tiles, int nkt, int cap) {
  if (tiles <= 0 || 2 * tiles > kCUs) return 1;
  return std::max(1, std::min({cap, kCUs / tiles, nkt}));
}
int gateup_split(int n, int d, int d_ff) {
  return split_ways((n + TileSplitGU::BM - 1) / TileSplitGU::BM * (2 * d_ff / TileSplitGU::OUT_N),
                    d / BK, kMaxSplitGU);
}
int down_split(int n, int d, int d_ff) {
  return split_ways((n + TileSplitDown::BM - 1) / TileSplitDown::BM * (d / TileSplitDown::OUT_N),
                    d_ff / BK, kMaxSplitDown);
}

// act[m][c] = bf16(SiLU(g) u) with g, u the sums over z < S of P[z][m][c] and P[z][m][d_ff + c];
// one thread per 8 columns of a row, rows m < *m_count
__global__ __launch_bounds__(256) void swiglu_reduce(const float* __restrict__ P, int S,
                                                    size_t stride, const int* __restrict__ m_count,
                                                    int n_max, int d_ff, bf16_t* __restrict__ act) {
  const int M = m_count ? min(*m_count, n_max) : n_max;
  const int q = d_ff / 8;
  const size_t e = static_cast<size_t>(blockIdx.x) * 256 + threadIdx.x;
  const int m = static_cast<int>(e / q), c = static_cast<int>(e % q) * 8;
  if (m >= M) return;
  const float* p = P + static_cast<size_t>(m) * 2 * d_ff + c;
  f32x4 g0 = *reinterpret_cast<const f32x4*>(p), g1 = *reinterpret_cast<const f32x4*>(p + 4);
  f32x4 u0 = *reinterpret_cast<const f32x4*>(p + d_ff), u1 = *reinterpret_cast<const f32x4*>(p + d_ff + 4);
  for (int z = 1; z < S; ++z) {
    const float* pz = p + z * stride;
    g0 += *reinterpret_cast<const f32x4*>(pz);
    g1 += *reinterpret_cast<const f32x4*>(pz + 4);
    u0 += *reinterpret_cast<const f32x4*>(pz + d_ff);
    u1 += *reinterpret_cast<const f32x4*>(pz + d_ff + 4);
  }
  u32x4 w;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const float ga = i < 2 ? g0[2 * i] : g1[2 * i - 4], gb = i < 2 ? g0[2 * i + 1] : g1[2 * i - 3];
    const float ua = i < 2 ? u0[2 * i] : u1[2 * i - 4], ub = i < 2 ? u0[2 * i + 1] : u1[2 * i - 3];
    const float lo = ga * __builtin_amdgcn_rcpf(1.0f + __expf(-ga)) * ua;
    const float hi = gb * __builtin_amdgcn_rcpf(1.0f + __expf(-gb)) * ub;
    w[i] = static_cast<uint32_t>(f32_to_bf16(lo)) | (static_cast<uint32_t>(f32_to_bf16(hi)) << 16);
  }
  *reinterpret_cast<u32x4*>(act + static_cast<size_t>(m) * d_ff + c) = w;
}

// h_out[t][n] = bf16(hbar[t][n] + g_t y) with y the sum over z < S of P[z][m][n], t = idx[m];
// one thread per 8 columns of a row, rows m < *m_count
__global__ __launch_bounds__(256) void scatter_reduce(const float* __restrict__ P, int S, size_t stride,
                                                     const int* __restrict__ m_count, int n_max,
                                                     const int* __restrict__ idx,
                                                     const bf16_t* __restrict__ hbar,
                                                     const float* __restrict__ gate,
                                                     bf16_t* __restrict__ out, int d) {
  const int M = m_count ? min(*m_count, n_max) : n_max;
  const int q = d / 8;
  const size_t e = static_cast<size_t>(blockIdx.x) * 256 + threadIdx.x;
  const int m = static_cast<int>(e / q), n = static_cast<int>(e % q) * 8;
  if (m >= M) return;
  const float* p = P + static_cast<size_t>(m) * d + n;
  f32x4 y0 = *reinterpret_cast<const f32x4*>(p), y1 = *reinterpret_cast<const f32x4*>(p + 4);
  for (int z = 1; z < S; ++z) {
    y0 += *reinterpret_cast<const f32x4*>(p + z * stride);
    y1 += *reinterpret_cast<const f32x4*>(p + z * stride + 4);
  }
  const int t = idx ? idx[m] : m;
  const float sc = gate ? gate[t] : 1.0f;
  const size_t o = static_cast<size_t>(t) * d + n;
  const u32x4 h = *reinterpret_cast<const u32x4*>(hbar + o);
  u32x4 w;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const float ya = i < 2 ? y0[2 * i] : y1[2 * i - 4], yb = i < 2 ? y0[2 * i + 1] : y1[2 * i - 3];
    const float lo = __uint_as_float(h[i] << 16) + sc * ya;
    const float hi = __uint_as_float(h[i] & 0xffff0000u) + sc * yb;
    w[i] = static_cast<uint32_t>(f32_to_bf16(lo)) | (static_cast<uint32_t>(f32_to_bf16(hi)) << 16);
  }
  *reinterpret_cast<u32x4*>(out + o) = w;
}

// out[((kt NB + b) G + g) 16 + r][c] = W_g[16 b + r][64 kt + c] with NB = N / 16 blocks (w0: g = 0,
// w1: g = 1); one thread per 16-byte piece of the output, so the writes are contiguous and each
// group of eight threads reads one 128-byte run of a source row.
__global__ __launch_bounds__(256) void tile_ffn_weights_kernel(const bf16_t* __restrict__ w0,
                                                              const bf16_t* __restrict__ w1, int G, int K,
                                                              size_t pieces, bf16_t* __restrict__ out) {
  const size_t e = static_cast<size_t>(blockIdx.x) * 256 + threadIdx.x;
  if (e >= pieces) return;
  const int c8 = static_cast<int>(e & 7), r = static_cast<int>((e >> 3) & 15);
  const size_t t = e >> 7;                       // (kt NB + b) G + g
  const int g = static_cast<int>(t % G);
  const size_t bk = t / G;
  const size_t NB = pieces / (static_cast<size_t>(K / BK) * G * 128);
  const size_t b = bk % NB;
  const int kt = static_cast<int>(bk / NB);
  const bf16_t* src = (g ? w1 : w0) + (16 * b + r) * static_cast<size_t>(K) + kt * BK + 8 * c8;
  *reinterpret_cast<u32x4*>(out + 8 * e) = *reinterpret_cast<const u32x4*>(src);
}

}  // namespace

size_t ffn_part_floats(int dtype, int d, int d_ff, int T) {
  if (dtype != 1 || T <= 0) return 0;
  // S is fixed per row-tile count and the slices hold n rows: the largest n of each count
  size_t most = 0;
  const int ns = std::min(T, kSkinnyRows);
  if (skinny_down_fits(ns, d, d_ff)) most = static_cast<size_t>(skinny_down_splits(d, d_ff)) * ns * d;
  for (int mt = 1; (mt - 1) * TileSplitGU::BM < T; ++mt) {
    const int n = std::min(mt * TileSplitGU::BM, T);
    const int sg = gateup_split(n, d, d_ff), sd = down_split(n, d, d_ff);
    if (sg > 1) most = std::max(most, static_cast<size_t>(sg) * n * 2 * d_ff);
    if (sd > 1) most = std::max(most, static_cast<size_t>(sd) * n * d);
    if (sg == 1 && sd == 1) break;   // both counts only grow from here
  }
  return most;
}

hipError_t launch_tile_ffn_weights(const void* w0, const void* w1, int N, int K, void* out, hipStream_t s) {
  if (N <= 0 || K <= 0 || N % 16 != 0 || K % BK != 0) return hipErrorInvalidValue;
  const int G = w1 ? 2 : 1;
  const size_t pieces = static_cast<size_t>(N) * (K / 8) * G;
  tile_ffn_weights_kernel<<<static_cast<unsigned>((pieces + 255) / 256), 256, 0, s>>>(
      static_cast<const bf16_t*>(w0), static_cast<const bf16_t*>(w1), G, K, pieces, static_cast<bf16_t*>(out));
  return hipGetLastError();
}

hipError_t launch_ffn_gateup(int dtype, const void* u, const int* idx_ffn, const int* counts,
                             int n_max, const void* w_gate, const void* w_up, const void* w_gate_up_tiled,
                             void* act, float* part, int d, int d_ff, hipStream_t s) {
  if (n_max <= 0) return hipSuccess;
  if (dtype == 1) {
    ARows<bf16_t> A{static_cast<const bf16_t*>(u), idx_ffn, d};
    if (skinny_gateup_fits(n_max, d, d_ff))
      return skinny_gateup(A, static_cast<const bf16_t*>(w_gate), static_cast<const bf16_t*>(w_up),
                           static_cast<const bf16_t*>(w_gate_up_tiled), static_cast<bf16_t*>(act), counts,
                           n_max, d, d_ff, s);
    const int S = gateup_split(n_max, d, d_ff);
    if (S > 1) {
      BRows<bf16_t> B{static_cast<const bf16_t*>(w_gate), static_cast<const bf16_t*>(w_up), d_ff, d};
      const size_t stride = static_cast<size_t>(n_max) * 2 * d_ff;
      hipError_t e = run_tile<TileSplitGU>(A, B, EpiStoreF32{part, 2 * d_ff, stride}, counts, n_max,
                                           2 * d_ff, d, s, S);
      if (e != hipSuccess) return e;
      const size_t n8 = static_cast<size_t>(n_max) * (d_ff / 8);
      swiglu_reduce<<<static_cast<unsigned>((n8 + 255) / 256), 256, 0, s>>>(
          part, S, stride, counts, n_max, d_ff, static_cast<bf16_t*>(act));
      return hipGetLastError();
    }
    BRows<bf16_t> B{static_cast<const bf16_t*>(w_gate), static_cast<const bf16_t*>(w_up), INT_MAX, d};
    return run_big<256, true, EpiSwiGLU<bf16_t>, 16>(A, B, EpiSwiGLU<bf16_t>{static_cast<bf16_t*>(act), d_ff},
                                                     counts, n_max, d_ff, d, s);
  }
  ARows<float> A{static_cast<const float*>(u), idx_ffn, d};
  BRows<float> B{static_cast<const float*>(w_gate), static_cast<const float*>(w_up), INT_MAX, d};
  return run_f32<true>(A, B, EpiSwiGLU<float>{static_cast<float*>(act), d_ff}, counts, n_max, d_ff,
                       d, s);
}

hipError_t launch_ffn_down(int dtype, const void* act, const int* idx_ffn, const int* counts,
                           int n_max, const void* w_down, const void* w_down_tiled, const void* hbar,
                           const float* gate, void* h_out, float* part, int d, int d_ff, hipStream_t s) {
  if (n_max <= 0) return hipSuccess;
  if (dtype == 1) {
    ARows<bf16_t> A{static_cast<const bf16_t*>(act), nullptr, d_ff};
    BRows<bf16_t> B{static_cast<const bf16_t*>(w_down), nullptr, INT_MAX, d_ff};
    const bool skinny = skinny_down_fits(n_max, d, d_ff);
    const int S = skinny ? skinny_down_splits(d, d_ff) : down_split(n_max, d, d_ff);
    if (S > 1 || skinny) {
      const size_t stride = static_cast<size_t>(n_max) * d;
      hipError_t e = skinny ? skinny_down(A, static_cast<const bf16_t*>(w_down),
                                          static_cast<const bf16_t*>(w_down_tiled), part, stride, counts,
                                          n_max, d, d_ff, S, s)
                            : run_tile<TileSplitDown>(A, B, EpiStoreF32{part, d, stride}, counts, n_max, d,
                                                      d_ff, s, S);
      if (e != hipSuccess) return e;
      const size_t n8 = static_cast<size_t>(n_max) * (d / 8);
      scatter_reduce<<<static_cast<unsigned>((n8 + 255) / 256), 256, 0, s>>>(
          part, S, stride, counts, n_max, idx_ffn, static_cast<const bf16_t*>(hbar), gate,
          static_cast<bf16_t*>(h_out), d);
      return hipGetLastError();
    }
    EpiScatter<bf16_t, false> epi{idx_ffn, static_cast<const bf16_t*>(hbar), gate,
                                  static_cast<bf16_t*>(h_out), d};
    return run_big<256, false, EpiScatter<bf16_t, false>, 16>(A, B, epi, counts, n_max, d, d_ff, s);
  }
  ARows<float> A{static_cast<const float*>(act), nullptr, d_ff};
  BRows<float> B{static_cast<const float*>(w_down), nullptr, INT_MAX, d_ff};
  EpiScatter<float, false> epi{idx_ffn, static_cast<const float*>(hbar), gate,
                               static_cast<float*>(h_out), d};
  return run_f32<false>(A, B, epi, counts, n_max, d, d_ff, s);
}

// ---------------------------------------------------------------------------
// Attention projections of a decoder block (Sec. 3.1, eq:dense_attention).
// [q; k; v] = x [W_q; W_k; W_v]^T runs on the GEMM core with an epilogue that applies the
// rotary embedding to q and k (pair (2i, 2i+1) of a head turned by pos * inv_freq[i]: a
// table of cos and sin for the call's positions, made once in fp32) and writes each head
// where the attention kernel reads it: q [B][n_h][S_pad][128], k [B][n_kv][S_pad][128] and
// v transposed, [B][n_kv][128][S_pad] with positions permuted within groups of 16 (the
// attention kernel's key order), written as 16-byte runs.  The output projection
// adds its product to the block input: hbar = h + o W_o^T.
// ---------------------------------------------------------------------------
namespace {

constexpr int kHeadDim = 128;

struct EpiQKV {
  bf16_t* q;
  bf16_t* k;
  bf16_t* vt;
  const float2* cs;   // [seq][64] (cos, sin) of pos * inv_freq[i]
  int seq, seq_pad, nh, nkv;
  struct Pre {};
  __device__ __forceinline__ Pre prep(int, int) const { return {}; }
  __device__ __forceinline__ void store(int, int, float) const {}
  __device__ __forceinline__ void emit8(const Pre&, int, int, const float*) const {}
  // a staged block of 32 token rows x `on` columns (one head's half: 64 | 128) starting at
  // row mb, column nb
  __device__ __forceinline__ void block(const float* stg, int opad, int on, int mb, int nb, int M,
                                        int lane) const {
    const int head = nb / kHeadDim, c0 = nb % kHeadDim;
    if (head < nh + nkv) {
      // q or k: 8-column row pieces, turned by the rotary table
      const int cpr = on / 8;
      for (int e = lane; e < 32 * cpr; e += kWave) {
        const int i = e / cpr, c8 = (e % cpr) * 8;
        const int m = mb + i;
        if (m >= M) continue;
        const int b = m / seq, pos = m - b * seq;
        const int c = c0 + c8;
        const float* v = stg + i * opad + c8;
        const float2* t = cs + static_cast<size_t>(pos) * (kHeadDim / 2) + c / 2;
        u32x4 w;
#pragma unroll
        for (int x = 0; x < 4; ++x) {
          const float2 r = t[x];
          const float a = v[2 * x], bb = v[2 * x + 1];
          w[x] = static_cast<uint32_t>(f32_to_bf16(a * r.x - bb * r.y)) |
                 (static_cast<uint32_t>(f32_to_bf16(a * r.y + bb * r.x)) << 16);
        }
        bf16_t* dst = head < nh
            ? q + ((static_cast<size_t>(b) * nh + head) * seq_pad + pos) * kHeadDim + c
            : k + ((static_cast<size_t>(b) * nkv + (head - nh)) * seq_pad + pos) * kHeadDim + c;
        *reinterpret_cast<u32x4*>(dst) = w;
      }
    } else {
      // v, transposed, positions permuted within each group of 16 (position p at slot
      // p with bits 2 and 3 swapped: 0-3, 8-11, 4-7, 12-15): a piece is one column over the
      // 8 positions 16G + 4X + {0..3} and 16G + 8 + 4X + {0..3} of the block, one 16-byte run
      const int vh = head - nh - nkv;
      for (int e = lane; e < 4 * on; e += kWave) {
        const int col = e % on, rg = e / on;
        const int G = rg >> 1, X = rg & 1;
        const int m16 = mb + 16 * G;
        if (m16 >= M) continue;
        const int b = m16 / seq, p16 = m16 - b * seq;
        bf16_t* row = vt + ((static_cast<size_t>(b) * nkv + vh) * kHeadDim + c0 + col) * seq_pad;
        if (m16 + 15 < M && p16 + 15 < seq && (p16 & 15) == 0) {
          u32x4 w;
#pragma unroll
          for (int x = 0; x < 4; ++x) {
            const int r0 = 16 * G + (x < 2 ? 4 * X + 2 * x : 8 + 4 * X + 2 * (x - 2));
            w[x] = static_cast<uint32_t>(f32_to_bf16(stg[r0 * opad + col])) |
                   (static_cast<uint32_t>(f32_to_bf16(stg[(r0 + 1) * opad + col])) << 16);
          }
          *reinterpret_cast<u32x4*>(row + p16 + 8 * X) = w;
        } else {
          for (int x = 0; x < 8; ++x) {
            const int r = 16 * G + (x < 4 ? 4 * X + x : 8 + 4 * X + x - 4);
            const int mm = mb + r;
            if (mm >= M) continue;
            const int bx = mm / seq, px = mm - bx * seq;
            const int slot = (px & ~15) | (px & 3) | ((px & 4) << 1) | ((px & 8) >> 1);
            vt[((static_cast<size_t>(bx) * nkv + vh) * kHeadDim + c0 + col) * seq_pad + slot] =
                f32_to_bf16(stg[r * opad + col]);
          }
        }
      }
    }
  }
};

__global__ void rope_table_kernel(float2* __restrict__ cs, int seq, RopeTable rope) {
  const int e = blockIdx.x * blockDim.x + threadIdx.x;
  if (e >= seq * (kHeadDim / 2)) return;
  const int pos = e / (kHeadDim / 2), i = e % (kHeadDim / 2);
  float sn, c;
  sincosf(static_cast<float>(pos) * rope.inv_freq[i], &sn, &c);
  cs[e] = make_float2(c, sn);
}

}  // namespace

hipError_t launch_rope_table(int seq, const RopeTable& rope, float* cs, hipStream_t s) {
  const int n = seq * (kHeadDim / 2);
  if (n <= 0) return hipSuccess;
  rope_table_kernel<<<(n + 255) / 256, 256, 0, s>>>(reinterpret_cast<float2*>(cs), seq, rope);
  return hipGetLastError();
}

hipError_t launch_attn_qkv(const void* x, const void* w_qkv, int T, int d, int seq, int seq_pad, int nh,
                           int nkv, const float* rope_cs, void* q, void* k, void* vt, hipStream_t s) {
  if (T <= 0) return hipSuccess;
  ARows<bf16_t> A{static_cast<const bf16_t*>(x), nullptr, d};
  BRows<bf16_t> B{static_cast<const bf16_t*>(w_qkv), nullptr, INT_MAX, d};
  EpiQKV epi{static_cast<bf16_t*>(q), static_cast<bf16_t*>(k), static_cast<bf16_t*>(vt),
             reinterpret_cast<const float2*>(rope_cs), seq, seq_pad, nh, nkv};
  return run_big<256, false>(A, B, epi, nullptr, T, (nh + 2 * nkv) * kHeadDim, d, s);
}

hipError_t launch_attn_out(const void* o, const void* w_o, const void* h, void* hbar, int T, int d, int nh,
                           hipStream_t s) {
  if (T <= 0) return hipSuccess;
  const int K = nh * kHeadDim;
  ARows<bf16_t> A{static_cast<const bf16_t*>(o), nullptr, K};
  BRows<bf16_t> B{static_cast<const bf16_t*>(w_o), nullptr, INT_MAX, K};
  EpiScatter<bf16_t, false> epi{nullptr, static_cast<const bf16_t*>(h), nullptr, static_cast<bf16_t*>(hbar), d};
  return run_big<256, false>(A, B, epi, nullptr, T, d, K, s);
}

// Wide adapters (ranks above 128, in steps of 128: the paper's d_r = 896).  The down-projection
// runs on the MFMA GEMM core with K split WIDE_SPLIT ways into fp32 partials, a reduction pass forms
// hid = bf16(SiLU(sum of the partials)), and the up-projection is a GEMM whose epilogue scatters
// hbar + (1 - g) (W_2 hid) into the adapter rows.
constexpr int WIDE_SPLIT = 4;
using TileWide = Tile<128, 128, 2, 4, false>;

bool adapter_wide(int d_r) { return d_r > 128; }

size_t adapter_part_floats(int dtype, int d, int d_r, int T) {
  if (dtype == 1 && adapter_wide(d_r))   // partials, then hid (bf16, half a float per element)
    return static_cast<size_t>(WIDE_SPLIT) * T * d_r + static_cast<size_t>(T) * d_r / 2;
  const int G = dtype == 1 ? adapter_groups(d) : 1;
  return static_cast<size_t>(G) * T * d_r;
}

namespace {

// hid[m][n] = bf16(SiLU(sum_z part[z][m][n])) for m < *m_count, eight columns per thread
__global__ __launch_bounds__(256) void adapter_hidden_wide(const float* __restrict__ part, size_t split_stride,
                                                           const int* __restrict__ m_count, int d_r,
                                                           bf16_t* __restrict__ hid) {
  const size_t n8 = static_cast<size_t>(*m_count) * d_r / 8;
  for (size_t e = blockIdx.x * static_cast<size_t>(256) + threadIdx.x; e < n8;
       e += static_cast<size_t>(gridDim.x) * 256) {
    f32x4 x[WIDE_SPLIT][2];
#pragma unroll
    for (int z = 0; z < WIDE_SPLIT; ++z) {
      const float* p = part + z * split_stride + 8 * e;
      x[z][0] = *reinterpret_cast<const f32x4*>(p);
      x[z][1] = *reinterpret_cast<const f32x4*>(p + 4);
    }
    float h[8];
#pragma unroll
    for (int c = 0; c < 8; ++c) {
      float v = 0.f;
#pragma unroll
      for (int z = 0; z < WIDE_SPLIT; ++z) v += x[z][c >> 2][c & 3];
      h[c] = siluf_(v);
    }
    st8(hid + 8 * e, h);
  }
}

}  // namespace

namespace {

// K-sliced partials of rows[idx[m]] W^T for the register-tiled ranks (32 .. 128); with u2 set, a
// second product over the same rows in the same launch (gridDim.z = 2)
hipError_t adapter_down_small(const bf16_t* uu, const int* idx_ad, const int* counts, int n_max, const bf16_t* ww,
                              float* part, int d, int d_r, hipStream_t s, const bf16_t* u2, const bf16_t* w2_,
                              float* p2, int G) {
  dim3 g1((n_max + 31) / 32, G, u2 ? 2 : 1);
  // the adapter rank is a compile-time count of 32-column MFMA tiles
  const bool b8 = adapter_batch(d, G) == 8;
#define HERO_ADAPTER_DOWN(TN_)                                                                       \
  (b8 ? adapter_down_bf16<TN_, 8><<<g1, 256, 0, s>>>(uu, idx_ad, counts, ww, part, n_max, d, d / G, u2, w2_, p2) \
      : adapter_down_bf16<TN_, 4><<<g1, 256, 0, s>>>(uu, idx_ad, counts, ww, part, n_max, d, d / G, u2, w2_, p2))
  switch (d_r) {
    case 32: HERO_ADAPTER_DOWN(1); break;
    case 64: HERO_ADAPTER_DOWN(2); break;
    case 96: HERO_ADAPTER_DOWN(3); break;
    case 128: HERO_ADAPTER_DOWN(4); break;
    default: return hipErrorInvalidValue;
  }
#undef HERO_ADAPTER_DOWN
  return hipGetLastError();
}

}  // namespace

hipError_t launch_adapter_down(int dtype, const void* u, const int* idx_ad, const int* counts,
                               int n_max, const void* w1, float* part, int d, int d_r,
                               hipStream_t s) {
  if (n_max <= 0) return hipSuccess;
  if (dtype == 1 && adapter_wide(d_r)) {
    ARows<bf16_t> A{static_cast<const bf16_t*>(u), idx_ad, d};
    BRows<bf16_t> B{static_cast<const bf16_t*>(w1), nullptr, INT_MAX, d};
    const size_t stride = static_cast<size_t>(n_max) * d_r;
    hipError_t e = run_tile<TileWide>(A, B, EpiStoreF32{part, d_r, stride}, counts, n_max, d_r, d, s, WIDE_SPLIT);
    if (e != hipSuccess) return e;
    bf16_t* hid = reinterpret_cast<bf16_t*>(part + WIDE_SPLIT * stride);
    const int blocks = static_cast<int>(std::min<size_t>((stride / 8 + 255) / 256, 2048));
    adapter_hidden_wide<<<blocks, 256, 0, s>>>(part, stride, counts, d_r, hid);
    return hipGetLastError();
  }
  if (dtype == 1)
    return adapter_down_small(static_cast<const bf16_t*>(u), idx_ad, counts, n_max, static_cast<const bf16_t*>(w1),
                              part, d, d_r, s, nullptr, nullptr, nullptr, adapter_groups_rows(d, n_max));
  // fp32: hid = SiLU(u W_1^T) into part[m][n]
  ARows<float> A{static_cast<const float*>(u), idx_ad, d};
  BRows<float> B{static_cast<const float*>(w1), nullptr, INT_MAX, d};
  return run_f32<false>(A, B, EpiSiLU<float>{part, d_r}, counts, n_max, d_r, d, s);
}

hipError_t launch_adapter_up(int dtype, const float* part, const int* idx_ad, const int* counts,
                             int n_max, const void* w2, const void* hbar, const float* gate,
                             void* h_out, int d, int d_r, hipStream_t s) {
  if (n_max <= 0) return hipSuccess;
  if (dtype == 1 && adapter_wide(d_r)) {
    const bf16_t* hid =
        reinterpret_cast<const bf16_t*>(part + static_cast<size_t>(WIDE_SPLIT) * n_max * d_r);
    ARows<bf16_t> A{hid, nullptr, d_r};
    BRows<bf16_t> B{static_cast<const bf16_t*>(w2), nullptr, INT_MAX, d_r};
    EpiScatter<bf16_t, true> epi{idx_ad, static_cast<const bf16_t*>(hbar), gate, static_cast<bf16_t*>(h_out), d};
    return run_tile<TileWide>(A, B, epi, counts, n_max, d, d_r, s);
  }
  if (dtype == 1) {
    const int G = adapter_groups_rows(d, n_max);
    dim3 g2((n_max + 31) / 32, d / 256);
    const bf16_t* ww = static_cast<const bf16_t*>(w2);
    const bf16_t* hb = static_cast<const bf16_t*>(hbar);
    bf16_t* ho = static_cast<bf16_t*>(h_out);
    switch (d_r) {
      case 32: adapter_up_launch<32>(g2, s, G, part, idx_ad, counts, ww, hb, gate, ho, n_max, d); break;
      case 64: adapter_up_launch<64>(g2, s, G, part, idx_ad, counts, ww, hb, gate, ho, n_max, d); break;
      case 96: adapter_up_launch<96>(g2, s, G, part, idx_ad, counts, ww, hb, gate, ho, n_max, d); break;
      case 128: adapter_up_launch<128>(g2, s, G, part, idx_ad, counts, ww, hb, gate, ho, n_max, d); break;
      default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
  }
  ARows<float> A{part, nullptr, d_r};
  BRows<float> B{static_cast<const float*>(w2), nullptr, INT_MAX, d_r};
  EpiScatter<float, true> epi{idx_ad, static_cast<const float*>(hbar), gate,
                              static_cast<float*>(h_out), d};
  return run_f32<false>(A, B, epi, counts, n_max, d, d_r, s);
}

// ---------------------------------------------------------------------------
// Backward of the routed block (frozen FFN, trained adapter) on the same cores.  The frozen
// weights enter through transposed copies, so every product keeps K contiguous:
//   e    = dL/dh[idx] W_d         B = W_d^T [d_ff][d]          (FFN rows)
//   G, U recomputed from u[idx]   B = W_g, W_u                 epilogue: EpiSwiGLUBwd
//   du   = [dG dU] [W_g; W_u]     B = [W_g; W_u]^T [d][2 d_ff]
// and the adapter's: z = u[idx] W_1^T, e_a = dL/dh[idx] W_2 (B = W_2^T), du = dz W_1 (B = W_1^T).
// ---------------------------------------------------------------------------
namespace {
using TileBwdGU = Tile<192, 256, 2, 4, true>;
}

int swiglu_bwd_parts(int dtype, int d_ff) { return dtype == 1 ? d_ff / TileBwdGU::ON : d_ff; }

hipError_t launch_ffn_bwd_e(int dtype, const void* dh, const int* idx_ffn, const int* counts, int n_max,
                            const void* w_down_t, void* e, int d, int d_ff, hipStream_t s) {
  if (n_max <= 0) return hipSuccess;
  if (dtype == 1) {
    ARows<bf16_t> A{static_cast<const bf16_t*>(dh), idx_ffn, d};
    BRows<bf16_t> B{static_cast<const bf16_t*>(w_down_t), nullptr, INT_MAX, d};
    EpiStore<bf16_t> epi{static_cast<bf16_t*>(e), d_ff};
    return d_ff % 256 == 0 ? run_big<256, false>(A, B, epi, counts, n_max, d_ff, d, s)
                           : run_big<128, false>(A, B, epi, counts, n_max, d_ff, d, s);
  }
  ARows<float> A{static_cast<const float*>(dh), idx_ffn, d};
  BRows<float> B{static_cast<const float*>(w_down_t), nullptr, INT_MAX, d};
  return run_f32<false>(A, B, EpiStore<float>{static_cast<float*>(e), d_ff}, counts, n_max, d_ff, d, s);
}

hipError_t launch_ffn_bwd_gateup(int dtype, const void* u, const int* idx_ffn, const int* counts, int n_max,
                                 const void* w_gate, const void* w_up, const void* e, const float* gate,
                                 void* dgu, float* dgpart, int d, int d_ff, hipStream_t s) {
  if (n_max <= 0) return hipSuccess;
  if (dtype == 1) {
    ARows<bf16_t> A{static_cast<const bf16_t*>(u), idx_ffn, d};
    BRows<bf16_t> B{static_cast<const bf16_t*>(w_gate), static_cast<const bf16_t*>(w_up), INT_MAX, d};
    EpiSwiGLUBwd<bf16_t> epi{static_cast<const bf16_t*>(e), d_ff, idx_ffn, gate, static_cast<bf16_t*>(dgu),
                             2 * d_ff, d_ff, dgpart, swiglu_bwd_parts(1, d_ff)};
    return run_tile<TileBwdGU>(A, B, epi, counts, n_max, d_ff, d, s);
  }
  ARows<float> A{static_cast<const float*>(u), idx_ffn, d};
  BRows<float> B{static_cast<const float*>(w_gate), static_cast<const float*>(w_up), INT_MAX, d};
  EpiSwiGLUBwd<float> epi{static_cast<const float*>(e), d_ff, idx_ffn, gate, static_cast<float*>(dgu),
                          2 * d_ff, d_ff, dgpart, d_ff};
  return run_f32<true>(A, B, epi, counts, n_max, d_ff, d, s);
}

hipError_t launch_ffn_bwd_du(int dtype, const void* dgu, const int* counts, int n_max, const void* w_gate_up_t,
                             float* du, int d, int d_ff, hipStream_t s) {
  if (n_max <= 0) return hipSuccess;
  const int K = 2 * d_ff;
  if (dtype == 1) {
    ARows<bf16_t> A{static_cast<const bf16_t*>(dgu), nullptr, K};
    BRows<bf16_t> B{static_cast<const bf16_t*>(w_gate_up_t), nullptr, INT_MAX, K};
    return run_big<256, false>(A, B, EpiStoreF32{du, d, 0}, counts, n_max, d, K, s);
  }
  ARows<float> A{static_cast<const float*>(dgu), nullptr, K};
  BRows<float> B{static_cast<const float*>(w_gate_up_t), nullptr, INT_MAX, K};
  return run_f32<false>(A, B, EpiStoreF32{du, d, 0}, counts, n_max, d, K, s);
}

int adapter_proj_splits(int dtype, int d, int d_r) {
  if (dtype != 1) return 1;
  return adapter_wide(d_r) ? WIDE_SPLIT : adapter_groups(d);
}

hipError_t launch_adapter_proj2(int dtype, const void* rows0, const void* w0, float* part0, const void* rows1,
                                const void* w1, float* part1, const int* idx_ad, const int* counts, int n_max, int d,
                                int d_r, hipStream_t s) {
  if (n_max <= 0) return hipSuccess;
  if (dtype == 1 && !adapter_wide(d_r))
    return adapter_down_small(static_cast<const bf16_t*>(rows0), idx_ad, counts, n_max, static_cast<const bf16_t*>(w0),
                              part0, d, d_r, s, static_cast<const bf16_t*>(rows1), static_cast<const bf16_t*>(w1),
                              part1, adapter_groups(d));
  hipError_t e = launch_adapter_proj(dtype, rows0, idx_ad, counts, n_max, w0, part0, d, d_r, s);
  if (e != hipSuccess) return e;
  return launch_adapter_proj(dtype, rows1, idx_ad, counts, n_max, w1, part1, d, d_r, s);
}

hipError_t launch_adapter_proj(int dtype, const void* rows, const int* idx_ad, const int* counts, int n_max,
                               const void* w, float* part, int d, int d_r, hipStream_t s) {
  if (n_max <= 0) return hipSuccess;
  if (dtype == 1 && adapter_wide(d_r)) {
    // the K-sliced partials only (the forward's SiLU hidden rows are not needed here)
    ARows<bf16_t> A{static_cast<const bf16_t*>(rows), idx_ad, d};
    BRows<bf16_t> B{static_cast<const bf16_t*>(w), nullptr, INT_MAX, d};
    const size_t stride = static_cast<size_t>(n_max) * d_r;
    return run_tile<TileWide>(A, B, EpiStoreF32{part, d_r, stride}, counts, n_max, d_r, d, s, WIDE_SPLIT);
  }
  // the backward's consumers sum adapter_proj_splits() = adapter_groups(d) slices
  if (dtype == 1)
    return adapter_down_small(static_cast<const bf16_t*>(rows), idx_ad, counts, n_max, static_cast<const bf16_t*>(w),
                              part, d, d_r, s, nullptr, nullptr, nullptr, adapter_groups(d));
  ARows<float> A{static_cast<const float*>(rows), idx_ad, d};
  BRows<float> B{static_cast<const float*>(w), nullptr, INT_MAX, d};
  return run_f32<false>(A, B, EpiStoreF32{part, d_r, 0}, counts, n_max, d_r, d, s);
}

hipError_t launch_adapter_du(int dtype, const void* dz, const int* counts, int n_max, const void* w1t, float* du,
                             int d, int k, hipStream_t s) {
  if (n_max <= 0) return hipSuccess;
  if (dtype == 1) {
    ARows<bf16_t> A{static_cast<const bf16_t*>(dz), nullptr, k};
    BRows<bf16_t> B{static_cast<const bf16_t*>(w1t), nullptr, INT_MAX, k};
    return run_tile<TileWide>(A, B, EpiStoreF32{du, d, 0}, counts, n_max, d, k, s);
  }
  ARows<float> A{static_cast<const float*>(dz), nullptr, k};
  BRows<float> B{static_cast<const float*>(w1t), nullptr, INT_MAX, k};
  return run_f32<false>(A, B, EpiStoreF32{du, d, 0}, counts, n_max, d, k, s);
}

namespace {
struct EpiAccF32 {  // C[m][n] += acc
  float* out;
  int ld;
  __device__ __forceinline__ void store(int m, int n, float v) const { out[static_cast<size_t>(m) * ld + n] += v; }
};
}  // namespace

namespace {
struct EpiAccF32Mfma {  // C[m][n] += acc on the MFMA path (each element owned by one lane)
  float* out;
  int ld;
  struct Pre {};
  __device__ __forceinline__ Pre prep(int, int) const { return {}; }
  __device__ __forceinline__ void emit8(const Pre&, int m, int n, const float* v) const {
    float* o = out + static_cast<size_t>(m) * ld + n;
    f32x4 a = *reinterpret_cast<const f32x4*>(o), b = *reinterpret_cast<const f32x4*>(o + 4);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      a[i] += v[i];
      b[i] += v[4 + i];
    }
    *reinterpret_cast<f32x4*>(o) = a;
    *reinterpret_cast<f32x4*>(o + 4) = b;
  }
};
}  // namespace

hipError_t launch_gemm_nt_acc_bf16(const void* A, int lda, int M, const void* B, int ldb, int N, int K, float* C,
                                   int ldc, hipStream_t s) {
  if (M <= 0 || N <= 0 || K <= 0) return hipSuccess;
  ARows<bf16_t> a{static_cast<const bf16_t*>(A), nullptr, lda};
  BRows<bf16_t> b{static_cast<const bf16_t*>(B), nullptr, INT_MAX, ldb};
  return run_tile<TileWide>(a, b, EpiAccF32Mfma{C, ldc}, nullptr, M, N, K, s);
}

hipError_t launch_gemm_acc_f32(const float* A, int lda, int M, const float* B, int ldb, int N, int K, float* C,
                               int ldc, hipStream_t s) {
  ARows<float> a{A, nullptr, lda};
  BRows<float> b{B, nullptr, INT_MAX, ldb};
  return run_f32<false>(a, b, EpiAccF32{C, ldc}, nullptr, M, N, K, s);
}

hipError_t launch_gemm_nt_f32(const void* A, int M, const void* B, int N, int K, float* C, int ldc, hipStream_t s) {
  if (M <= 0 || N <= 0 || K <= 0) return hipSuccess;
  ARows<bf16_t> a{static_cast<const bf16_t*>(A), nullptr, K};
  BRows<bf16_t> b{static_cast<const bf16_t*>(B), nullptr, INT_MAX, K};
  return run_tile<TileWide>(a, b, EpiStoreF32{C, ldc, 0}, nullptr, M, N, K, s);
}

}  // namespace hero
