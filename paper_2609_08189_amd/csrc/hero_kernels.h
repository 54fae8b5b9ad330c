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
// written as router_gemm_splits(dtype, d) partial sums over K slices, slice z at P + z T (d_e + d_head).
int router_gemm_splits(int dtype, int d);
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
hipError_t launch_ffn_gateup(int dtype, const void* u, const int* idx_ffn, const int* counts,
                             int n_max, const void* w_gate, const void* w_up, void* act,
                             float* part, int d, int d_ff, hipStream_t s);
// FFN branch, down + scatter: h_out[t] = hbar[t] + g[t] * (W_d act[m]), t = idx_ffn[m].
hipError_t launch_ffn_down(int dtype, const void* act, const int* idx_ffn, const int* counts,
                           int n_max, const void* w_down, const void* hbar, const float* gate,
                           void* h_out, float* part, int d, int d_ff, hipStream_t s);

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

}  // namespace hero
