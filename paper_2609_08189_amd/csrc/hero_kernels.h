// Host-side launchers of the HeRo kernels (one translation unit per kernel family).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace hero {

// router ablation bits (the values of the C ABI's hero_ablation)
constexpr int ABL_NO_POS = 1, ABL_NO_AUX = 2, ABL_NO_MEMREAD = 4, ABL_NO_HISTORY = 8;

// Row statistics of the post-attention states and the FFN input:
//   rowstat[t] = {1/rms(hbar_t), |delta_j|^2, <delta_j, delta_{j-1}>, |delta_{j-1}|^2}
//   u[t] = RMSNorm_w(hbar_t) in the storage dtype.
hipError_t launch_rowstats(int dtype, const void* hbar, const void* prev1, const void* prev2,
                           const void* norm_w, int T, int d, int j, float eps_norm,
                           float* rowstat, void* u, hipStream_t s);

// Router pre-activations P[t] = [W_hd hbar_t ; psi_1 hbar_t] (fp32, [T][d_e + d_head]),
// written as router_gemm_splits(dtype, d, T, d_e + d_head) partial sums over K slices, slice z at
// P + z T (d_e + d_head).
int router_gemm_splits(int dtype, int d, int T, int N);
hipError_t launch_router_gemm(int dtype, const void* hbar, const void* w_hd, const void* ps1,
                              int T, int d, int d_e, int d_head, float* P, hipStream_t s);

struct RouterTailArgs {
  int dtype;
  int T, j, L_R;
  int d_m, d_s, d_h, d_a, d_e, d_p, d_head;
  float eps, T_hist, eta;
  const float* P;         // [p_splits][T][d_e + d_head] partial sums
  int p_splits;
  const float* rowstat;   // [T][4]
  const void *w_hu, *w_p1, *w_p2, *w_q, *w_k, *w_v, *w_n, *w_c, *th1, *th2, *ps2;
  int ld_th1;             // row pitch of th1 (elements)
  const float* beta;      // [T] or null
  int abl;                // router ablation bits (ABL_*)
  void* S;                // [T][d_m][d_m]   in/out, fp32 or (state_bf16) bf16
  int state_bf16;
  float* zeta;            // [T][d_m]        in/out
  float* p_hist;          // [T]             in/out
  float* m_hist;          // [T]             in/out
  float* logit;           // [T]
  float* gate;            // [T]
  // intermediates between the three router kernels (router_scratch_floats(d_m, d_head, T))
  float* qkvn;            // [T][4][d_m]  phi(q), phi(k), v, W_n s
  float* hs;              // [T][d_head]  th1[:, :d_s] s
  float* cvec;            // [T][d_m]     memory read c
  float* bvec;            // [T]          local-head logit b
  // depth-history form of the memory (router_mem_hist): kv [T][L_R][2][d_m], and the weights
  // w_{j,i} of the j-1 stored pairs (hw[i] for entry i, i.e. routed layer i+1)
  float* kv;
  float hw[64];
};
size_t router_scratch_floats(int d_m, int d_head, int T);
// router state, q/k/v, W_n s, the s part of the history head, local head
hipError_t launch_router_pre(const RouterTailArgs& a, hipStream_t s);
// streaming memory read-modify-write (one token per workgroup)
hipError_t launch_router_mem(const RouterTailArgs& a, hipStream_t s);
// nu, history head, p, m, logit and gate
hipError_t launch_router_post(const RouterTailArgs& a, hipStream_t s);
// memory read as attention over the stored pairs, then the layer's own pair appended
hipError_t launch_router_mem_hist(const RouterTailArgs& a, hipStream_t s);
// matrix-form state S, zeta after n layers from a history (weights w[i] for entry i)
struct HistWeights {
  float w[64];
};
hipError_t launch_history_state(int d_m, int L_R, int n, int T, const float* kv, const HistWeights& w,
                                float* S, float* zeta, hipStream_t s);

// Branch decision and ordered compaction (one workgroup).
struct SelectArgs {
  const float* logit;
  int T;
  int mode;        // 0 threshold, 1 budget
  float thr;       // threshold mode: logit threshold
  int n_skip;      // budget mode
  uint8_t* mask;
  int* idx_ffn;
  int* idx_ad;
  int* counts;     // [2]
  float* lambda;   // [1]
};
hipError_t launch_select(const SelectArgs& a, hipStream_t s);

// FFN branch, gate/up: act[m] = SiLU(W_g u_t) * (W_u u_t), t = idx_ffn[m], m < counts[0].
// part: fp32 scratch of ffn_part_floats(dtype, d, d_ff, T) floats for any n_max <= T (used
// when few rows split K).
size_t ffn_part_floats(int dtype, int d, int d_ff, int T);
// w_gate_up_tiled (may be null): W_g and W_u in the streaming order of launch_tile_ffn_weights,
// read instead of w_gate, w_up by the products of at most 256 rows.
hipError_t launch_ffn_gateup(int dtype, const void* u, const int* idx_ffn, const int* counts,
                             int n_max, const void* w_gate, const void* w_up, const void* w_gate_up_tiled,
                             void* act, float* part, int d, int d_ff, hipStream_t s);
// FFN branch, down + scatter: h_out[t] = hbar[t] + g[t] * (W_d act[m]), t = idx_ffn[m].
// w_down_tiled (may be null): W_d in the streaming order, read instead of w_down by the products
// of at most 256 rows.
hipError_t launch_ffn_down(int dtype, const void* act, const int* idx_ffn, const int* counts,
                           int n_max, const void* w_down, const void* w_down_tiled, const void* hbar,
                           const float* gate, void* h_out, float* part, int d, int d_ff, hipStream_t s);
// The frozen FFN weights in the decode products' streaming order (bf16): W [N][K] becomes
// [K/64][N/16][G][16][64], i.e. 16 x 64 tiles of 2 KiB, k-tile by k-tile, each k-tile's row of
// 16-row blocks contiguous, with G = 2 matrices alternating tile by tile (W_g then W_u) or G = 1 (W_d).
// w1 may be null when G = 1.  Needs N % 16 == 0 and K % 64 == 0.
hipError_t launch_tile_ffn_weights(const void* w0, const void* w1, int N, int K, void* out, hipStream_t s);

// FFN of a non-routed block: the two launchers above with idx_ffn = counts = gate = null
// (every row, t = m, g = 1).

// Attention sub-block of a decoder block (bf16, head width 128).  Token t = b seq + pos.
struct RopeTable {
  float inv_freq[64];   // [head_dim / 2] rotary frequencies
};
// cs[pos][i] = (cos, sin)(pos * inv_freq[i]) in fp32, pos < seq, i < 64 (2 seq 64 floats)
hipError_t launch_rope_table(int seq, const RopeTable& rope, float* cs, hipStream_t s);
// [q; k; v] = x [W_q; W_k; W_v]^T with the rotary embedding on q, k; q [B][nh][seq_pad][128],
// k [B][nkv][seq_pad][128], vt [B][nkv][128][seq_pad] with position p of a row at slot p with
// bits 2 and 3 swapped (rows past seq are not written)
hipError_t launch_attn_qkv(const void* x, const void* w_qkv, int T, int d, int seq, int seq_pad, int nh,
                           int nkv, const float* rope_cs, void* q, void* k, void* vt, hipStream_t s);
// o[t][h 128 + c] = causal softmax(q k^T / sqrt(128)) v, head h reading kv head h / (nh / nkv)
// (zeroes the V^T positions seq .. seq_pad - 1 first)
hipError_t launch_attn_core(const void* q, const void* k, void* vt, void* o, int batch, int seq,
                            int seq_pad, int nh, int nkv, hipStream_t s);
// hbar = h + o W_o^T
hipError_t launch_attn_out(const void* o, const void* w_o, const void* h, void* hbar, int T, int d, int nh,
                           hipStream_t s);

// Adapter branch: h_out[t] = hbar[t] + (1 - g[t]) * W_2 SiLU(W_1 u_t) for t = idx_ad[m].
// part: fp32 scratch of adapter_part_floats(dtype, d, d_r, T) floats.
size_t adapter_part_floats(int dtype, int d, int d_r, int T);
hipError_t launch_adapter_down(int dtype, const void* u, const int* idx_ad, const int* counts,
                               int n_max, const void* w1, float* part, int d, int d_r,
                               hipStream_t s);
hipError_t launch_adapter_up(int dtype, const float* part, const int* idx_ad, const int* counts,
                             int n_max, const void* w2, const void* hbar, const float* gate,
                             void* h_out, int d, int d_r, hipStream_t s);

// ---------------------------------------------------------------------------
// Backward of the routed block (training side; frozen FFN, trained adapter)
// ---------------------------------------------------------------------------
// copies of the branch lists with counts clamped to [0, nf_max] and [0, na_max] (n_ffn + n_ad <= T)
// and indices to [0, T - 1]: f, ad [T], c [2]
hipError_t launch_bwd_lists(int T, int nf_max, int na_max, const int* idx_ffn, const int* idx_ad, const int* counts,
                            int* f, int* ad, int* c, hipStream_t s);
// out[c][r] = in[r][c] for r < R, c < C ([R][C] with row pitch ld_in into rows of pitch
// ld_out); with R_pad > R the columns R .. R_pad - 1 of every output row are written as 0
hipError_t launch_transpose(int dtype, const void* in, int R, int C, int ld_in, void* out, int ld_out,
                            int R_pad, hipStream_t s);
// W_2^T [d_r][d] and W_1^T [d][rpad] (columns d_r .. rpad - 1 zero) of an adapter, one launch
hipError_t launch_adapter_transpose(int dtype, const void* w1, const void* w2, void* w1t, void* w2t, int d, int d_r,
                                    int rpad, hipStream_t s);
// e[m] = dL/dh[idx_ffn[m]] W_d (W_d^T given, [d_ff][d]), storage dtype, [n][d_ff]
hipError_t launch_ffn_bwd_e(int dtype, const void* dh, const int* idx_ffn, const int* counts, int n_max,
                            const void* w_down_t, void* e, int d, int d_ff, hipStream_t s);
// G, U recomputed from u[idx_ffn[m]]; dgu[m] = [dG | dU] (storage dtype, [n][2 d_ff]) and
// dgpart[m][p] = the p-th share of <e_m, act_m> (swiglu_bwd_parts(dtype, d_ff) per row)
int swiglu_bwd_parts(int dtype, int d_ff);
hipError_t launch_ffn_bwd_gateup(int dtype, const void* u, const int* idx_ffn, const int* counts, int n_max,
                                 const void* w_gate, const void* w_up, const void* e, const float* gate,
                                 void* dgu, float* dgpart, int d, int d_ff, hipStream_t s);
// du[m] = dgu[m] [W_g; W_u] (([W_g; W_u])^T given, [d][2 d_ff]), fp32 [n][d]
hipError_t launch_ffn_bwd_du(int dtype, const void* dgu, const int* counts, int n_max, const void* w_gate_up_t,
                             float* du, int d, int d_ff, hipStream_t s);
// part[z][m][n] (z < adapter_proj_splits, slices n_max d_r floats apart): K-slice partial sums
// of rows[idx_ad[m]] W^T for W [d_r][d] (adapter_part_floats(dtype, d, d_r, n_max) floats)
int adapter_proj_splits(int dtype, int d, int d_r);
hipError_t launch_adapter_proj(int dtype, const void* rows, const int* idx_ad, const int* counts, int n_max,
                               const void* w, float* part, int d, int d_r, hipStream_t s);
// two such products over the same rows (one launch where the ranks allow)
hipError_t launch_adapter_proj2(int dtype, const void* rows0, const void* w0, float* part0, const void* rows1,
                                const void* w1, float* part1, const int* idx_ad, const int* counts, int n_max, int d,
                                int d_r, hipStream_t s);
// du[m] = dz[m] W_1 (W_1^T given, [d][k]); dz [n][k] in the storage dtype, k = the rank padded to
// a multiple of 64 (bf16) or d_r (fp32)
hipError_t launch_adapter_du(int dtype, const void* dz, const int* counts, int n_max, const void* w1t, float* du,
                             int d, int k, hipStream_t s);

struct BlockBwdArgs {
  int dtype, T, d, d_r, rpad;
  const void* dh;            // [T][d]    dL/dh_out
  const void* hbar;          // [T][d]
  const void* norm_w;        // [d]
  const float* rowstat;      // [T][4]    1/rms in [0]
  const int* idx_ffn;
  const int* idx_ad;
  const int* counts;         // [2]
  const float* gate;         // [T]
  const float* dgate_in;     // [T] or null
  const float* du_f;         // [T][d]    FFN rows, in idx_ffn order
  const float* du_a;         // [T][d]    adapter rows, in idx_ad order
  const float* dgpart;       // [T][n_parts]
  int n_parts;
  float* dg_ad;              // [T]
  // adapter
  int na_max;                // launch bound of the adapter rows (the partials' slice height)
  const float* part_z;       // [splits][na_max][d_r]
  const float* part_e;
  int splits;
  float* dz32;               // [T][d_r]
  float* a32;                // [T][d_r]
  void* dzk;                 // [T][rpad] storage dtype (the du product's A operand)
  const void* u;             // [T][d]
  int n_slices;              // weight-gradient partials: the adapter rows split this many ways
  float* pw1;                // [n_slices][d_r][d]
  float* pw2;                // [n_slices][d][d_r]
  // outputs
  void* dhbar;               // [T][d]
  float* dgate;              // [T]
  float* dlogit;             // [T]
  float* dw1;                // [d_r][d]
  float* dw2;                // [d][d_r]
};
// a = SiLU(z), dz = (1 - g) e_a SiLU'(z), dL/dg = -<e_a, a> for every adapter row
hipError_t launch_adapter_bwd_mid(const BlockBwdArgs& a, hipStream_t s);
// dW_1 = sum_m dz_m u_m^T, dW_2 = sum_m ((1 - g) dL/dh)_m a_m^T over the adapter rows
hipError_t launch_adapter_wgrad(const BlockBwdArgs& a, hipStream_t s);
// dL/dhbar = dL/dh + RMSNorm backward of du (every token once), dL/dg, dL/dlogit
hipError_t launch_block_bwd_rows(const BlockBwdArgs& a, hipStream_t s);
// Wide adapter ranks: the adapter rows staged transposed in bf16 with the tokens contiguous
// (columns m >= counts[1] up to kp zero): uaT [d][kp] = u rows, dyT [d][kp] = (1 - g) dh rows,
// dzT [d_r][kp], aT [d_r][kp]; then dW_1 = dzT uaT^T and dW_2 = dyT aT^T on the GEMM core.
hipError_t launch_adapter_wgrad_stage(const BlockBwdArgs& a, int kp, void* uaT, void* dyT, void* dzT, void* aT,
                                      hipStream_t s);
// C[m][n] = sum_k A[m][k] B[n][k] (bf16 A [M][K], B [N][K]; fp32 C with row pitch ldc); N % 128 == 0,
// K % 64 == 0
hipError_t launch_gemm_nt_f32(const void* A, int M, const void* B, int N, int K, float* C, int ldc, hipStream_t s);
// C[m][n] += sum_k A[m][k] B[n][k] in fp32 (rows of A and B with leading dims lda, ldb)
hipError_t launch_gemm_acc_f32(const float* A, int lda, int M, const float* B, int ldb, int N, int K, float* C,
                               int ldc, hipStream_t s);

// C[m][n] += sum_k A[m][k] B[n][k] on the bf16 GEMM core (fp32 accumulators; K a multiple of 64,
// N of the tile's 128 columns, C rows 16-byte aligned)
hipError_t launch_gemm_nt_acc_bf16(const void* A, int lda, int M, const void* B, int ldb, int N, int K, float* C,
                                   int ldc, hipStream_t s);
// C[m][n] += sum_k A[m][k] B[n][k] in fp32 for small M x N and long K (the tokens): K split into up to
// tn_chunks(K) chunks of at least kTnChunk (as many as part_floats holds, nz M N), partial sums added
// in chunk order
constexpr int kTnChunk = 64;
int tn_chunks(int K);
hipError_t launch_gemm_tn_acc_f32(const float* A, int lda, int M, const float* B, int ldb, int N, int K, float* C,
                                  int ldc, float* part, size_t part_floats, hipStream_t s);
// C_p[m][n] += sum_t A_p[m][t] B_p[n][t] for up to kSmallProducts products in one launch (A_p [M][T],
// B_p [N][T] fp32 with token pitch ldk; C_p fp32 with row pitch ldc) on the fp32 matrix cores.  The
// tokens are cut into at most kSmallProductChunks chunks of at least 256 whose partial sums (part,
// small_products_floats of them) are added in chunk order.
struct SmallProduct {
  const float* A;
  const float* B;
  float* C;
  int M, N, ldc;
};
constexpr int kSmallProducts = 12;
constexpr int kSmallProductChunks = 16;
size_t small_products_floats(const SmallProduct* p, int n, int T);
hipError_t launch_small_products(const SmallProduct* p, int n, int T, int ldk, float* part, size_t part_floats,
                                 hipStream_t s);
// x [R][C] fp32 (row pitch ld_in) as bf16 hi = bf16(x), lo = bf16(x - hi), [R][C_pad] with zero columns
// from C to C_pad: hi + lo carries x to about 2^-16 relative
hipError_t launch_split_bf16(const float* x, int R, int C, int ld_in, void* hi, void* lo, int C_pad, hipStream_t s);

// Backward of the router at routed layer j (k_router_bwd.hip).
struct RouterBwdArgs {
  int dtype, T, j, L_R, d, d_m, d_s, d_h, d_a, d_e, d_p, d_head, ld_th1;
  float eps_norm, eps, T_hist, rho;
  const void *hbar, *prev1, *prev2;          // [T][d]: hbar_j, hbar_{j-1} (j >= 2), hbar_{j-2} (j >= 3)
  const float* P;                            // [p_splits][T][d_e + d_head] partial pre-activations
  int p_splits;
  const void *w_hu, *w_p1, *w_p2, *w_q, *w_k, *w_v, *w_n, *w_c, *th1, *th2, *ps2;
  const float *S_in, *zeta_in, *p_in, *m_in; // the state entering layer j
  const float* dlogit;                       // [T]
  float *dS, *dzeta, *dp, *dm;               // carried gradient, in place: state leaving -> entering
  float* dP;                                 // [T][d_e + d_head]: [ir dL/dpre_h; dL/dpre_b]
  float* dPT;                                // the same, [d_e + d_head][T]
  float* rowcoef;                            // [T][8]: c_norm, c1, c2, c3, c4
  float* rho_part;                           // [T]
  // token-contiguous ([rows][T]) operands of the weight-gradient products
  float *XT, *dQT, *dKT, *dVT, *dU1T, *dU2T, *dPAT, *SAT, *DA, *DB, *SBT, *dPPT, *SPT, *XPT, *dZAT, *dZHT, *SHT;
  float *dhbar, *dhbar1, *dhbar2;            // [T][d] fp32, accumulated
  float* deta;                               // [1]
  // per-token intermediates handed from one token pass to the next (token-major scratch):
  // row statistics (ir, |delta_j|, |delta_{j-1}|, delta_j . delta_{j-1}), q k v W_n s, the path
  // encoder's pre-activation, c, the read's normaliser, p_j, dL/ds so far, dL/dnum, dL/dden,
  // [dL/dphi(k); dL/dphi(q); dL/dv], P with its K slices summed
  float *RS, *QKVU, *PPRE, *Cv, *DEN, *PS, *DSP, *DNUM, *DDEN, *DF, *PSUM;
  // the tokens the token passes take, [t_begin, t_end) (t_begin a multiple of 16 for the chain);
  // every token-indexed array above keeps its layout over all T tokens
  int t_begin, t_end;
  // nonzero: Cv holds the forward's memory read (j >= 2); the read pass is skipped and F2 forms
  // the normaliser phi(q)^T zeta_{j-1} + eps itself
  int c_given;
  // bf16 storage: the router weights transposed for the batched passes' transposed products, bf16,
  // written by launch_router_bwd_wt (null for fp32 storage): th1^T [d_s + d_m + 1][d_head],
  // W_n^T [d_s][d_m], W_c^T [d_m][d_m], [W_q; W_k; W_v]^T [d_s][3 d_m], W_p2^T [d_p][ld_ta],
  // W_hu^T [d_e][ld_th] (ld_ta, ld_th: d_a, d_h rounded up to 8, the pad columns zero)
  uint16_t *th1T, *wnT, *wcT, *wqkvT, *wp2T, *whuT;
  int ld_ta, ld_th;
};
// bf16 elements of the transposed weights (each array starting on 16 bytes), and their placement
// in a buffer of that many elements
size_t router_bwd_wt_elems(int d_m, int d_s, int d_h, int d_a, int d_e, int d_p, int d_head);
void router_bwd_wt_assign(RouterBwdArgs& a, uint16_t* base);
hipError_t launch_router_bwd_wt(const RouterBwdArgs& a, hipStream_t s);
// rows of the token-contiguous operands above, per token
size_t router_bwd_vector_floats(int d_m, int d_s, int d_h, int d_a, int d_e, int d_p, int d_head);
// floats of the token passes' intermediates, per token
size_t router_bwd_token_floats(int d_m, int d_s, int d_p, int np);
// the token passes over [t_begin, t_end): the row statistics (and P's slice sums), then the chain
// F1, memory read, F2, state pass, F3
hipError_t launch_router_bwd_stats(const RouterBwdArgs& a, hipStream_t s);
hipError_t launch_router_bwd_chain(const RouterBwdArgs& a, hipStream_t s);
// the RMSNorm / transition terms of dL/dhbar, then dL/deta
hipError_t launch_router_bwd_rows(const RouterBwdArgs& a, hipStream_t s);
// out[c][r] = float(in[r][c])
hipError_t launch_to_f32_transpose(int dtype, const void* in, int R, int C, int ld_in, float* out, int ld_out,
                                   hipStream_t s);
// alpha L_skip (Eq. 18) into loss[0] and its gradient over gates [L_R][batch seq]
hipError_t launch_skip_penalty(const float* gates, int L_R, int batch, int seq, float alpha, float* loss,
                               float* dgates, hipStream_t s);

}  // namespace hero
