/*
 * hero.h -- C ABI of the HeRo routed FFN stack for AMD Instinct MI355X (gfx950).
 *
 * HeRo ("History-Aware Routing", arxiv 2609.08189) routes every token at every
 * routed layer either to the frozen backbone's FFN or to a small adapter
 * (Sec. 3.1, eq:ffn_route).  The router scores the token from its
 * post-attention state and a per-token linear-attention memory over depth
 * (Sec. 3.2), reads that memory before writing the layer's router state into
 * it, and carries four pieces of per-token state to the next routed layer: the
 * memory matrix S, its normaliser zeta, and the history scores p and m.
 *
 * This library runs that hot path on one GPU.  It is a plain C interface:
 *   - every tensor argument is a DEVICE pointer to caller-owned memory unless a
 *     comment says "host"; the calls allocate no device memory (the caller passes
 *     a workspace; hero_routed_layer_noalloc uses a fixed device array of the
 *     library's).  What the library keeps between calls: per calling thread and
 *     device, a second stream and two events, created on the first call (outside
 *     any graph capture that follows) for the work it forks beside the call's
 *     stream; per device, the address of the no-allocation scratch; and the
 *     process-global registry of the measurement hook hero_kernel_timer (empty
 *     unless a caller attaches events).  No data of one call is read by another;
 *   - calls are asynchronous: they validate their arguments on the host, enqueue
 *     kernels on `stream` (a hipStream_t passed as void*, NULL = the null
 *     stream) and return; results are valid once the stream has synchronised;
 *   - calls return a hero_status; they never abort.  Argument checks run before
 *     anything touches the GPU, so a bad argument never launches a kernel.
 *     Device faults surface at the caller's next synchronisation.
 *   - calls on different streams are independent when their buffers are
 *     disjoint; two calls sharing a workspace must be ordered by the caller.
 *
 * Layouts (row-major throughout, token-major for per-token data):
 *   hidden states           [T][d]                 dtype = dims.dtype
 *   weights                 [out][in] (nn.Linear)  dtype = dims.dtype
 *   memory matrix S         [T][d_m][d_m] fp32, key index first, so the read is
 *                           c[v] = sum_k phi(q)[k] S[k][v] / (phi(q).zeta + eps)
 *   normaliser zeta         [T][d_m] fp32
 *   history scores p, m     [T] fp32
 * All device pointers must be 16-byte aligned.
 * Size limit (bf16): the matrix products address operand rows with 32-bit byte
 * offsets, so a call whose token rows (T x max(d, d_ff, d_r), or the attention
 * width n_heads x head_dim in the decoder calls) or weight matrices (d_ff x d,
 * d_r x d, the attention projections) would span 4 GiB or more returns
 * HERO_E_UNSUPPORTED; split such a batch into smaller calls.
 */
#ifndef HERO_H
#define HERO_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define HERO_ABI_VERSION 7

typedef enum hero_status {
  HERO_OK = 0,
  HERO_E_NULL = 1,        /* a required pointer is NULL                               */
  HERO_E_DIM = 2,         /* a size is non-positive or inconsistent (d_s != d_h + d_a) */
  HERO_E_RANGE = 3,       /* j outside 1..L_R, tau outside (0,1), budget outside [0,1] */
  HERO_E_DTYPE = 4,       /* unknown dtype code                                        */
  HERO_E_ALIGN = 5,       /* a device pointer is not 16-byte aligned                  */
  HERO_E_ALIAS = 6,       /* an output buffer overlaps an input it must not overlap   */
  HERO_E_WORKSPACE = 7,   /* workspace NULL or smaller than hero_workspace_size()      */
  HERO_E_UNSUPPORTED = 8, /* valid shape that the kernels do not implement            */
  HERO_E_LAUNCH = 9,      /* a kernel launch was rejected by the runtime              */
  HERO_E_DEVICE = 10,     /* no usable gfx950 device is current                       */
  HERO_E_SCRATCH = 11     /* hero_routed_layer_noalloc: the call needs more scratch than
                             the library's fixed device area (HERO_NOALLOC_SCRATCH_BYTES) */
} hero_status;

typedef enum hero_dtype { HERO_F32 = 0, HERO_BF16 = 1 } hero_dtype;

typedef enum hero_mode {
  HERO_MODE_THRESHOLD = 0, /* FFN iff g >= tau (Sec. 3.1, eq:ffn_route), tau_exec = 0.5 in Sec. 4.1 */
  HERO_MODE_BUDGET = 1     /* per layer, floor(budget*T + 1/2) tokens with the smallest
                              (logit, token index) take the adapter; not in the paper, it
                              fixes the skip fraction of untrained routers              */
} hero_mode;

/*
 * Shapes and constants.  d_s = d_h + d_a is the router-state width (Sec. 4.1:
 * 64 = 48 + 16); d_e is the hidden encoder's inner width, d_p the path
 * encoder's, d_head the history/local heads' hidden width (Sec. 4.1: 256); the
 * comparison space of W_n, W_c has width d_m.
 * Supported: d % 256 == 0 (bf16) or d % 128 == 0 (f32); bf16 also needs
 * d_ff % 128 == 0, d_r in {32, 64, 96, 128} or a multiple of 128 up to 8192
 * (the paper's 896), d_s % 8 == 0, d_e % 64 == 0 and
 * (d_e + d_head) % 128 == 0; d_m in
 * {32, 64, 128, 256}; d_s <= 128; d_e, d_head <= 256; d_p <= 128.
 * state_dtype selects how the memory matrix S is stored between layers: HERO_F32 (0, the
 * default of a zeroed struct) or HERO_BF16, which halves the memory pass's traffic; every
 * element written is rounded to the nearest bf16 (ties to even) and all arithmetic stays
 * fp32.  zeta, p and m are fp32 either way.  A bf16 S needs d_m >= 64 and the matrix form
 * (the depth-history entry points reject it).
 */
typedef struct hero_dims {
  int d, d_ff, d_r, L_R;
  int d_m, d_s, d_h, d_a;
  int d_e, d_p, d_head;
  int dtype;          /* hero_dtype of hidden states and every weight            */
  float eps_norm;     /* RMSNorm epsilon (1e-5)                                   */
  float eps;          /* epsilon of the two cosines and the memory read (1e-6)   */
  float T_hist;       /* history temperature (Sec. 4.1: 0.9)                      */
  int state_dtype;    /* hero_dtype of S                                          */
} hero_dims;

/*
 * Frozen backbone FFN of one routed layer: LN^ffn gain [d], W_g, W_u [d_ff][d], W_d [d][d_ff]
 * (eq:dense_attention, eq:ffn_route).
 * w_gate_up_tiled, w_down_tiled (optional, NULL when absent; bf16 models only): the same weights
 * in the streaming order of the products with few rows, made once per model by
 * hero_ffn_decode_weights_make.  When given, a branch of at most 256 rows (a decode step) reads
 * them instead of w_gate/w_up (resp. w_down); the results are bit-identical either way.
 */
typedef struct hero_ffn_weights {
  const void *norm_w, *w_gate, *w_up, *w_down;
  const void *w_gate_up_tiled, *w_down_tiled;
} hero_ffn_weights;

/* Bottleneck adapter of one routed layer (Sec. 3.1): W_1 [d_r][d], W_2 [d][d_r]. */
typedef struct hero_adapter_weights {
  const void *w1, *w2;
} hero_adapter_weights;

/*
 * Router weights shared by every routed layer (Sec. 3.2), bias-free:
 *   w_hd [d_e][d], w_hu [d_h][d_e]         hidden encoder z_h = W_hu SiLU(W_hd RMSNorm(hbar))
 *   w_p1 [d_p][6], w_p2 [d_a][d_p]         path encoder z_a = FFN_path(x_path)
 *   w_q, w_k, w_v [d_m][d_s]               memory projections
 *   w_n [d_m][d_s], w_c [d_m][d_m]         comparison projections of nu
 *   th1 [d_head][HERO_TH1_PITCH(d_s, d_m)], th2 [d_head]
 *                                          history head f_theta([s; c; nu]): row o holds the
 *                                          d_s + d_m + 1 input weights, then zero padding to a
 *                                          multiple of 8 elements (16-byte rows in bf16); the
 *                                          padding is never read
 *   ps1 [d_head][d], ps2 [d_head]          local head f_psi(hbar)
 */
#define HERO_TH1_PITCH(d_s, d_m) ((((d_s) + (d_m) + 1) + 7) / 8 * 8)

typedef struct hero_router_weights {
  const void *w_hd, *w_hu, *w_p1, *w_p2, *w_q, *w_k, *w_v, *w_n, *w_c;
  const void *th1, *th2, *ps1, *ps2;
} hero_router_weights;

/* Per-token router state (fp32), read and written in place.
 * c_read (optional, NULL when unused): the layer's memory read c_j = phi(q)^T S_{j-1} /
 * (phi(q)^T zeta_{j-1} + eps) (eq:memory_read), [T][d_m] fp32, 16-byte aligned, disjoint from every
 * other buffer of the call.  hero_routed_layer and hero_routed_layer_noalloc write it when set (with
 * the full router; an ablation without the memory read leaves it untouched); the stack and decoder
 * calls do not use it.  hero_router_backward reads it, when set and j >= 2, in place of re-reading
 * S_{j-1} for the read, so a training caller that keeps each layer's c (d_m floats per token) saves
 * the backward one of its four passes over the d_m x d_m state. */
typedef struct hero_state {
  void *S;        /* [T][d_m][d_m], fp32 or bf16 (dims.state_dtype) */
  float *zeta;    /* [T][d_m]      */
  float *p_hist;  /* [T]           */
  float *m_hist;  /* [T]           */
  float *c_read;  /* [T][d_m] or NULL */
} hero_state;

/*
 * Router ablations (Table 3, Sec. 4.3), a bit set in
 * hero_routing.ablation; 0 is the full router.  Readings of the paper's one-line
 * descriptions:
 *   NO_POS_STATE  the path vector loses the routing-progress and residual-transition
 *                 features: r = q_rem = d = gamma = 0, p and m stay;
 *   NO_AUX_STATE  no auxiliary path encoder: z_a = 0, so s = [z_h; 0];
 *   NO_MEMREAD    the history head keeps its inputs but not the memory: c = 0 and
 *                 nu = 0 (as at the first routed block) at every layer; S and zeta are
 *                 neither read nor written (their buffers are left as passed);
 *   NO_HISTORY    no history branch: logit = b (+ bias), a is not formed, p = m = 1 are
 *                 written (the initial scores); S and zeta are left as passed.
 * Bits combine; NO_HISTORY implies NO_MEMREAD's treatment of the memory.
 */
typedef enum hero_ablation {
  HERO_ABL_NO_POS_STATE = 1,
  HERO_ABL_NO_AUX_STATE = 2,
  HERO_ABL_NO_MEMREAD = 4,
  HERO_ABL_NO_HISTORY = 8,
  HERO_ABL_ALL = 15
} hero_ablation;

typedef struct hero_routing {
  int mode;                 /* hero_mode                                                */
  float tau;                /* threshold mode: tau_exec in (0,1)                        */
  double budget;            /* budget mode: skip fraction in [0,1]                      */
  const float *logit_bias;  /* optional device [T] fp32 added to the gate logit only;
                               NULL = none                                               */
  int ablation;             /* hero_ablation bits, 0 = full router; other bits are
                               rejected with HERO_E_RANGE                                */
} hero_routing;

/*
 * Optional per-layer outputs; every field may be NULL.
 *   mask    [T] u8     1 = FFN branch, 0 = adapter
 *   idx_ffn [T] i32    FFN tokens, ascending; entries past counts[0] are undefined
 *   idx_ad  [T] i32    adapter tokens, ascending; entries past counts[1] are undefined
 *   counts  [2] i32    n_ffn, n_adapter
 *   logit   [T] f32    a + b (+ bias)
 *   gate    [T] f32    g = sigma(logit)
 *   lambda  [1] f32    threshold mode: ln(tau/(1-tau)); budget mode: the smallest
 *                      logit on the FFN branch (+inf if none)
 */
typedef struct hero_layer_stats {
  uint8_t *mask;
  int32_t *idx_ffn, *idx_ad, *counts;
  float *logit, *gate, *lambda;
} hero_layer_stats;

/* Kernels of one routed layer, in launch order, then those of the attention sub-block (for
 * hero_kernel_timer).  The pretrained FFN of a non-routed decoder block is timed as
 * HERO_K_ROWSTATS, HERO_K_FFN_GATE_UP and HERO_K_FFN_DOWN. */
typedef enum hero_kernel {
  HERO_K_ROWSTATS = 0,      /* inv_rms, residual-transition sums, u = RMSNorm_w(hbar)          */
  HERO_K_ROUTER_GEMM = 1,   /* [W_hd; psi_1] hbar                                               */
  HERO_K_ROUTER_PRE = 2,    /* router state s, phi(q), phi(k), v, W_n s, local head            */
  HERO_K_ROUTER_MEM = 3,    /* memory read c and write S, zeta (one pass over the state)       */
  HERO_K_ROUTER_POST = 4,   /* nu, history head, p, m, logit, gate                             */
  HERO_K_SELECT = 5,        /* branch decision and ordered compaction                           */
  HERO_K_FFN_GATE_UP = 6,   /* SiLU(W_g u) * (W_u u) over the FFN tokens                        */
  HERO_K_FFN_DOWN = 7,      /* W_d act, scattered as hbar + g y                                 */
  HERO_K_ADAPTER_DOWN = 8,  /* W_1 u over the adapter tokens (partial sums)                     */
  HERO_K_ADAPTER_UP = 9,    /* W_2 SiLU(.), scattered as hbar + (1 - g) y                       */
  /* attention sub-block of a decoder block (hero_attention_block, hero_decoder_stack) */
  HERO_K_ATTN_NORM = 10,    /* x = RMSNorm(h) * norm_w                                          */
  HERO_K_ATTN_QKV = 11,     /* [q; k; v] = x W_qkv^T with the rotary embedding                  */
  HERO_K_ATTN_CORE = 12,    /* causal grouped-query softmax attention                           */
  HERO_K_ATTN_OUT = 13,     /* hbar = h + o W_o^T                                               */
  /* backward of the routed block (hero_routed_block_backward) and the penalty */
  HERO_K_BWD_NORM = 14,     /* branch lists copied in range; u and 1/rms recomputed             */
  HERO_K_BWD_FFN_E = 15,    /* e = dL/dh W_d over the FFN tokens                                */
  HERO_K_BWD_FFN_GATE_UP = 16, /* G, U recomputed; dG, dU and the shares of dL/dg              */
  HERO_K_BWD_FFN_DU = 17,   /* du = [dG dU] [W_g; W_u]                                          */
  HERO_K_BWD_ADAPTER = 18,  /* W_1^T, W_2^T; z, e_a; a, dz, dL/dg; du = dz W_1                 */
  HERO_K_BWD_ADAPTER_WGRAD = 19, /* dW_1, dW_2                                                  */
  HERO_K_BWD_ROWS = 20,     /* dL/dhbar (RMSNorm backward + residual), dL/dg, dL/dlogit          */
  HERO_K_SKIP_PENALTY = 21, /* alpha L_skip and its gradient                                    */
  /* backward of the router at one routed layer (hero_router_backward) */
  HERO_K_ROUTER_BWD_GEMM = 22,     /* P = hbar [W_hd; psi_1]^T recomputed                         */
  HERO_K_ROUTER_BWD_TOKEN = 23,    /* the router's forward recomputed and reversed, per token     */
  HERO_K_ROUTER_BWD_PRODUCTS = 24, /* weight gradients (tokens as K) and dP [W_hd; psi_1]         */
  HERO_K_ROUTER_BWD_ROWS = 25,     /* RMSNorm and transition terms of dL/dhbar; dL/deta           */
  HERO_K_COUNT = 26
} hero_kernel;

/*
 * Measurement hook.  While attached, every launch of `kernel` is bracketed by
 * hipEventRecord(start_events[i]) and hipEventRecord(stop_events[i]) on the
 * call's stream, with i cycling over the n_slots caller-created hipEvent_t
 * handles (passed as void*).  n_slots = 0 detaches.  The registry is process
 * global and must not be changed while routed calls are being enqueued.
 */
int hero_kernel_timer(int kernel, void *const *start_events, void *const *stop_events, int n_slots);

/*
 * Measurement hook, not part of the method: the practical bf16 matrix-core rate of the board.
 * Launches `workgroups` workgroups of 8 waves (two per SIMD; 256 = one per compute unit of an
 * MI355X) on hip_stream, each wave running 8 independent MFMA chains for `iters` iterations on
 * register operands.  mode bit 0: hashed operand values in [-0.5, 0.5) (the power-limited rate on
 * realistic data) instead of zeros (the issue limit); bit 1: v_mfma_f32_16x16x32_bf16 (the FFN
 * products' instruction) instead of v_mfma_f32_32x32x16_bf16.  *flop (host) receives the
 * floating-point operations the launch performs.  sink (device, >= 1 float) is never written in
 * practice.  Time the launch with the caller's events.
 * Errors: HERO_E_NULL, HERO_E_RANGE (mode outside 0..3, iters outside 1..2^24, workgroups outside
 * 1..65536), HERO_E_LAUNCH.
 */
int hero_peak_mfma(int mode, int iters, int workgroups, float *sink, void *hip_stream, double *flop);

/*
 * Measurement hook, not part of the method: HBM read rates by access pattern, reading `bytes` of
 * src (device, 16-byte aligned; its contents are irrelevant) once on hip_stream.
 * visit_bytes = 0: contiguous, plain non-temporal 16-byte loads into registers (256 workgroups of
 * 256 threads, eight loads in flight per lane, grid-stride; bytes a multiple of 16).
 * visit_bytes = 128, 256 or 512: the weight stream of a decode step: src is a bf16 matrix of 8 KiB
 * rows (d = 4096), read by bytes / (96 * 8 KiB) workgroups (bytes a multiple of that, at most
 * 65536 of them) of four waves, each taking 96 rows and visit_bytes of every row per step through
 * LDS-DMA (a 64-deep k-tile of bf16 is 128 bytes a row).  sink (device, >= 1 float) is never
 * written in practice.  Time the launch with the caller's events; use a region that the previous
 * launches did not touch to measure cold reads (the 256 MB MALL keeps recent lines).
 * Errors: HERO_E_NULL, HERO_E_ALIGN, HERO_E_DIM (bytes), HERO_E_RANGE (visit_bytes), HERO_E_LAUNCH.
 */
int hero_peak_read(const void *src, size_t bytes, int visit_bytes, float *sink, void *hip_stream);

/* Static string for a status code (host). */
const char *hero_status_string(int status);

/* ABI version (HERO_ABI_VERSION). */
int hero_abi_version(void);

/*
 * Workspace bytes needed by hero_routed_layer (for_stack = 0) or
 * hero_routed_stack (for_stack = 1) with T tokens.  Host-only; validates dims.
 */
int hero_workspace_size(const hero_dims *dims, int T, int for_stack, size_t *bytes);

/*
 * One routed layer l_j, j in 1..L_R (Sec. 3, overview paragraph, and
 * Sec. 3.1-3.2).  For every token t:
 *   router state s from hbar, (hbar - hbar_prev1), (hbar_prev1 - hbar_prev2), p, m
 *   (eq:path_vector, eq:transition_features, eq:router_state);
 *   memory read c from S, zeta, then memory write S <- rho S + phi(k) v^T,
 *   zeta <- rho zeta + phi(k), rho = sigma(eta) (eq:memory_read, eq:memory_update);
 *   nu, a, p <- sigma(a/T_hist), m <- m p; b; logit = a + b (+bias), g = sigma(logit)
 *   (Sec. 3.2 gate computation, eq:final_gate);
 *   branch decision (threshold or budget mode) and
 *   h_out = hbar + g FFN(u) or hbar + (1 - g) Adapter(u), u = RMSNorm_w(hbar)
 *   (eq:dense_attention, eq:ffn_route).
 * hbar_prev1 is read for j >= 2, hbar_prev2 for j >= 3 (NULL otherwise).  At
 * j = 1 the incoming state is taken as the paper's initial value (S = 0,
 * zeta = 0, p = m = 1) whatever the buffers hold, and is then overwritten.
 * h_out must not overlap hbar, hbar_prev1 or hbar_prev2.
 * Output rounding: h_out is rounded once to dims.dtype; all arithmetic is fp32.
 */
int hero_routed_layer(const hero_dims *dims, int j, int T,
                      const void *hbar, const void *hbar_prev1, const void *hbar_prev2,
                      void *h_out, const hero_state *state,
                      const hero_ffn_weights *ffn, const hero_router_weights *router,
                      const hero_adapter_weights *adapter, float eta,
                      const hero_routing *routing, const hero_layer_stats *stats,
                      void *workspace, size_t workspace_bytes, void *stream);

/*
 * hero_routed_layer for callers that cannot allocate device memory: code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc.  Same arguments, results and
 * errors as hero_routed_layer, without the workspace: the call's scratch (the layer's
 * intermediates: normalised rows, router pre-activations and state, logits, index lists, the FFN
 * activation, partial sums) lives in a fixed device array of HERO_NOALLOC_SCRATCH_BYTES that the
 * library holds on every device it runs on until the process ends.  The call allocates nothing
 * and issues no memset (no region of the scratch must start at zero: every kernel writes what it
 * later reads within the same call).  A call whose workspace (hero_workspace_size with
 * for_stack = 0) exceeds the area returns HERO_E_SCRATCH before any launch; at the
 * Llama-3.1-8B shape (d = 4096, d_ff = 14336, r = 64, d_m = 128) that allows up to 473 tokens,
 * and a 256-token decode batch of the Llama-2-7B shape needs 43.0 MiB of it.  The first call on a device looks the area up on that device (it must be
 * current); later calls reuse it.  Every call on one device shares that device's area: calls that
 * overlap in time on one device (two streams, two threads) race and must be serialised by the
 * caller.
 */
#define HERO_NOALLOC_SCRATCH_BYTES (64u << 20)
int hero_routed_layer_noalloc(const hero_dims *dims, int j, int T,
                              const void *hbar, const void *hbar_prev1, const void *hbar_prev2,
                              void *h_out, const hero_state *state,
                              const hero_ffn_weights *ffn, const hero_router_weights *router,
                              const hero_adapter_weights *adapter, float eta,
                              const hero_routing *routing, const hero_layer_stats *stats, void *stream);

/*
 * The whole routed stack: L_R chained routed layers with no attention between
 * them, hbar_1 = h_in and hbar_{j+1} = h_j; the state starts from the paper's
 * initial value (Sec. 3.2: zero memory at the start of a forward pass) and its
 * final value is left in `state`.  ffn, adapter and eta are HOST arrays of
 * L_R entries (device weight pointers inside); stats is a HOST array of L_R
 * entries or NULL.  The result equals L_R chained hero_routed_layer calls bit
 * for bit.  h_out must not overlap h_in.
 */
int hero_routed_stack(const hero_dims *dims, int T, const void *h_in, void *h_out,
                      const hero_state *state, const hero_ffn_weights *ffn,
                      const hero_router_weights *router, const hero_adapter_weights *adapter,
                      const float *eta, const hero_routing *routing,
                      const hero_layer_stats *stats,
                      void *workspace, size_t workspace_bytes, void *stream);

/*
 * Depth-history form of the router memory.  The memory recursion of Sec. 3.2
 * (eq:memory_update) starts from S_0 = 0, zeta_0 = 0, so it unrolls to
 *   S_{j-1} = sum_{i<j} w_{j,i} phi(k_i) v_i^T,  zeta_{j-1} = sum_{i<j} w_{j,i} phi(k_i),
 *   w_{j,i} = prod_{l=i+1}^{j-1} rho_l,  rho_l = sigma(eta_l),
 * and the read of layer j (eq:memory_read) becomes attention over depth,
 *   c_j = sum_i a_i v_i / (sum_i a_i + eps),  a_i = w_{j,i} phi(q_j) . phi(k_i).
 * This form keeps the pairs (phi(k_i), v_i) instead of S and zeta: 2 d_m floats
 * per token per layer, read j-1 times at layer j, instead of d_m^2 + d_m floats
 * read and written at every layer.  The results equal those of the matrix form
 * up to fp32 rounding order.  Supported for L_R <= 64.
 */
typedef struct hero_history {
  float *kv;      /* [T][L_R][2][d_m] fp32: entry i-1 holds phi(k_i), then v_i, of routed layer i;
                     layer j reads entries 0..j-2 and writes entry j-1 */
  float *p_hist;  /* [T] fp32, in/out (as in hero_state) */
  float *m_hist;  /* [T] fp32, in/out                    */
} hero_history;

/*
 * hero_routed_layer with the memory in depth-history form.  eta is a HOST array
 * of the j values eta_1 .. eta_j (the decays of the earlier layers weight the
 * stored pairs).  Entries j .. L_R-1 of the history are neither read nor written.
 * Everything else, including the workspace, is as for hero_routed_layer.
 */
int hero_routed_layer_hist(const hero_dims *dims, int j, int T,
                           const void *hbar, const void *hbar_prev1, const void *hbar_prev2,
                           void *h_out, const hero_history *history,
                           const hero_ffn_weights *ffn, const hero_router_weights *router,
                           const hero_adapter_weights *adapter, const float *eta,
                           const hero_routing *routing, const hero_layer_stats *stats,
                           void *workspace, size_t workspace_bytes, void *stream);

/*
 * hero_routed_stack with the memory in depth-history form: on return
 * history->kv holds all L_R entries.  The result equals L_R chained
 * hero_routed_layer_hist calls bit for bit.
 */
int hero_routed_stack_hist(const hero_dims *dims, int T, const void *h_in, void *h_out,
                           const hero_history *history, const hero_ffn_weights *ffn,
                           const hero_router_weights *router, const hero_adapter_weights *adapter,
                           const float *eta, const hero_routing *routing,
                           const hero_layer_stats *stats,
                           void *workspace, size_t workspace_bytes, void *stream);

/*
 * The matrix-form state after routed layer n (0 <= n <= L_R) from a history:
 * S[t] = sum_{i<=n} w_{n+1,i} phi(k_i) v_i^T and zeta[t] likewise (see above);
 * n = 0 gives zeros.  eta: HOST array of n values.  S [T][d_m][d_m] and
 * zeta [T][d_m] fp32 must not overlap kv.  Asynchronous on `stream`.
 */
int hero_history_state(const hero_dims *dims, int n, int T, const float *kv, const float *eta,
                       float *S, float *zeta, void *stream);

/*
 * The full decoder (Sec. 3.1): dense attention at every block,
 *   hbar = h + Attn(LN^attn(h))                                        (eq:dense_attention)
 * then the block's FFN: the pretrained one, h = hbar + FFN(LN^ffn(hbar)), at non-routed
 * blocks, and the routed layer at routed blocks.  The routed blocks are the last L_R of the
 * n_layers (the paper routes the latter half, Sec. 4.1).
 *
 * Attn is bias-free grouped-query self-attention of Llama form, causal within each sequence:
 * x = RMSNorm(h) * norm_w; q, k, v = x W_{q,k,v}^T per head of width head_dim; the rotary
 * embedding turns each pair (x_{2i}, x_{2i+1}) of q and k by pos * inv_freq[i], pos the
 * token's index in its sequence; o_h = softmax(q_h k_g^T / sqrt(head_dim)) v_g with
 * g = h / (n_heads / n_kv_heads); hbar = h + [o_1 .. o_{n_heads}] W_o^T.  Tokens are laid out
 * [batch][seq].  bf16 only; supported: head_dim == 128, n_heads % n_kv_heads == 0,
 * n_heads even.  q, k, v and the attention output are rounded to bf16 on their way through
 * HBM; softmax and every sum are fp32.
 */
typedef struct hero_attn_dims {
  int n_heads, n_kv_heads, head_dim;
} hero_attn_dims;

/* One block's attention weights: LN^attn gain [d]; W_q, W_k, W_v stacked as one
 * [(n_heads + 2 n_kv_heads) head_dim][d] matrix (rows: the q heads, then k, then v);
 * W_o [d][n_heads head_dim]. */
typedef struct hero_attn_weights {
  const void *norm_w, *w_qkv, *w_o;
} hero_attn_weights;

/*
 * Workspace bytes for hero_attention_block (n_layers = 0) or hero_decoder_stack with
 * batch x seq tokens.  Host-only; validates both dims structs.
 */
int hero_decoder_workspace_size(const hero_dims *dims, const hero_attn_dims *adims, int n_layers,
                                int batch, int seq, size_t *bytes);

/*
 * The attention sub-block of one decoder block: hbar = h + Attn(LN^attn(h)).  inv_freq is a
 * HOST array of head_dim / 2 rotary frequencies.  hbar must not overlap h.
 */
int hero_attention_block(const hero_dims *dims, const hero_attn_dims *adims, int batch, int seq,
                         const void *h, void *hbar, const hero_attn_weights *attn,
                         const float *inv_freq, void *workspace, size_t workspace_bytes,
                         void *stream);

/*
 * n_layers decoder blocks (L_R <= n_layers): attention at every block; the pretrained FFN at
 * blocks 1 .. n_layers - L_R; routed layers j = 1 .. L_R at the rest, with the router state
 * starting from its initial value at routed layer 1 and left in `state` (as in
 * hero_routed_stack; the residual transitions of the path vector are taken between the
 * post-attention states of consecutive routed blocks).  attn and ffn are HOST arrays of
 * n_layers entries; adapter, eta and stats (or NULL) of L_R entries.  The routing rule
 * applies at every routed block.  h_out must not overlap h_in.
 */
int hero_decoder_stack(const hero_dims *dims, const hero_attn_dims *adims, int n_layers, int batch,
                       int seq, const void *h_in, void *h_out, const hero_state *state,
                       const hero_attn_weights *attn, const hero_ffn_weights *ffn,
                       const hero_router_weights *router, const hero_adapter_weights *adapter,
                       const float *eta, const float *inv_freq, const hero_routing *routing,
                       const hero_layer_stats *stats, void *workspace, size_t workspace_bytes,
                       void *stream);

/* ---------------------------------------------------------------------------------------
 * Training side: the backward of a routed block through the gate scaling (Sec. 3.1,
 * eq:ffn_route and the remark after it) and the gate-utilisation penalty (Sec. 3.3,
 * Eq. 17-18).  The backbone is frozen: its FFN and LN^ffn pass a gradient on to hbar but take
 * none; the adapter's weights take theirs; the router receives dL/dlogit.  The branch
 * decision is a constant of the backward (the threshold is not differentiated).
 * ------------------------------------------------------------------------------------- */

/* Transposed copies of one frozen FFN's weights, which the backward's products read
 * (dims.dtype, caller-owned, made once per model by hero_ffn_backward_weights_make):
 *   w_down_t    [d_ff][d]      W_d^T
 *   w_gate_up_t [d][2 d_ff]    [W_g; W_u]^T: row i holds column i of W_g, then of W_u */
typedef struct hero_ffn_backward_weights {
  const void *w_down_t, *w_gate_up_t;
} hero_ffn_backward_weights;

/* Fill w_down_t and w_gate_up_t (device, dims.dtype, 16-byte aligned, not overlapping the
 * weights or each other) from ffn.  Asynchronous on `stream`. */
int hero_ffn_backward_weights_make(const hero_dims *dims, const hero_ffn_weights *ffn, void *w_down_t,
                                   void *w_gate_up_t, void *stream);

/*
 * The frozen FFN weights in the streaming order of the products with few rows (the FFN of a
 * decode step, eq:ffn_route with at most 256 FFN tokens), made once per model.  Those products
 * stream every weight once per call, 64-deep k-tile by k-tile; read row by row, each k-tile
 * visits 128 bytes of every weight row, a whole row (2 K bytes) apart.  In the tiled order the matrix is cut into
 * 16 x 64 tiles of 2 KiB, stored k-tile by k-tile, so that the weights one k-tile of the products
 * needs are one contiguous range:
 *   w_gate_up_tiled [d/64][d_ff/16][2][16][64]   tile (t, b) of W_g, then tile (t, b) of W_u:
 *                   element [t][b][0][r][c] = W_g[16 b + r][64 t + c], [t][b][1][r][c] = W_u[...]
 *   w_down_tiled    [d_ff/64][d/16][16][64]      element [t][b][r][c] = W_d[16 b + r][64 t + c]
 * Both are bf16 (dims.dtype must be HERO_BF16), 2 d d_ff and d d_ff elements, 16-byte aligned,
 * caller-owned, not overlapping the weights or each other; d_ff % 64 == 0.  Either may be NULL
 * (not made).  Asynchronous on `stream`.  Pass them in hero_ffn_weights.
 * Errors: HERO_E_NULL (dims, ffn or its weights), HERO_E_UNSUPPORTED (fp32 model, d_ff % 64 != 0),
 * HERO_E_ALIGN, HERO_E_ALIAS, HERO_E_DEVICE, HERO_E_LAUNCH.  The layer and stack calls reject
 * tiled pointers that are misaligned (HERO_E_ALIGN) or given for such a model (HERO_E_UNSUPPORTED).
 */
int hero_ffn_decode_weights_make(const hero_dims *dims, const hero_ffn_weights *ffn, void *w_gate_up_tiled,
                                 void *w_down_tiled, void *stream);

/* Outputs of hero_routed_block_backward (all required, device, overwritten):
 *   dhbar  [T][d] dims.dtype   dL/dhbar: dL/dh plus LN^ffn's backward of the branch's du
 *   dgate  [T] fp32            dL/dg (with dgate_in added)
 *   dlogit [T] fp32            dL/dlogit = dL/dg g (1 - g), what the router's backward takes
 *   dw1    [d_r][d] fp32       dL/dW_1
 *   dw2    [d][d_r] fp32       dL/dW_2 */
typedef struct hero_block_grads {
  void *dhbar;
  float *dgate, *dlogit, *dw1, *dw2;
} hero_block_grads;

/* Workspace bytes for hero_routed_block_backward with T tokens.  Host-only; validates dims.
 * The workspace must not overlap any argument of the call (HERO_E_ALIAS). */
int hero_backward_workspace_size(const hero_dims *dims, int T, size_t *bytes);

/*
 * Backward of one routed block (eq:ffn_route with u = RMSNorm_w(hbar)) given dL/dh_out:
 *   FFN token t   (h = hbar + g y, y = W_d (SiLU(W_g u) * (W_u u))):
 *     dL/dg = <dL/dh, y>; du from dL/dy = g dL/dh through the SwiGLU;
 *   adapter token (h = hbar + (1 - g) y, y = W_2 SiLU(W_1 u)):
 *     dL/dg = -<dL/dh, y>; dW_2 += ((1 - g) dL/dh) SiLU(z)^T, dW_1 += dz u^T, du = dz W_1;
 *   dL/dhbar = dL/dh + RMSNorm_w backward of du;  dL/dg += dgate_in (may be NULL: e.g. the
 *   penalty's gradient from hero_skip_penalty);  dL/dlogit = dL/dg g (1 - g).
 * gate, idx_ffn, idx_ad, counts are the forward's (hero_layer_stats of the same layer: every
 * token in exactly one list), and routing is the forward's rule (NULL: taken as threshold mode):
 * in budget mode the branch sizes are known on the host (T - n_skip FFN tokens, n_skip adapter
 * tokens), which sizes the launches; counts are then clamped to those sizes.  The lists are read
 * through copies with counts clamped to [0, T] and indices to [0, T - 1], so malformed lists
 * give wrong values, never an access out of bounds.  The FFN's gate/up products are recomputed from hbar (the forward's activations
 * are not kept).  dhbar must not overlap hbar or dh_out.  All products are bf16 x bf16 with
 * fp32 accumulation for a bf16 model (e and [dG dU] pass through HBM in bf16), fp32 otherwise;
 * every reduction has a fixed order.
 */
int hero_routed_block_backward(const hero_dims *dims, int T, const void *hbar, const void *dh_out,
                               const float *gate, const int32_t *idx_ffn, const int32_t *idx_ad,
                               const int32_t *counts, const hero_routing *routing, const float *dgate_in,
                               const hero_ffn_weights *ffn,
                               const hero_ffn_backward_weights *ffn_t, const hero_adapter_weights *adapter,
                               const hero_block_grads *grads, void *workspace, size_t workspace_bytes,
                               void *stream);

/*
 * alpha L_skip (Eq. 18) and its gradient: gates [L_R][batch seq] fp32 (the routed blocks'
 * g, token t = b seq + pos); L_skip is the mean, over the batch (seq - 1) positions that have
 * a next token, of the square of the token's gate sum over the L_R blocks.  loss[0] = alpha
 * L_skip; dgates [L_R][batch seq] = 2 alpha (sum_j g) / (batch (seq - 1)) at those positions
 * and 0 at each sequence's last (everything 0 when seq = 1).  dgates must not overlap gates.
 */
int hero_skip_penalty(int L_R, int batch, int seq, const float *gates, float alpha, float *loss,
                      float *dgates, void *stream);

/* Gradients of the router weights (fp32, the shapes and row pitches of hero_router_weights,
 * th1 with its padded pitch); hero_router_backward adds into them. */
typedef struct hero_router_grads {
  float *w_hd, *w_hu, *w_p1, *w_p2, *w_q, *w_k, *w_v, *w_n, *w_c, *th1, *th2, *ps1, *ps2;
} hero_router_grads;

/* The gradient over the router state carried backwards across routed layers (fp32, in place):
 * on entry dL/dS_j [T][d_m][d_m], dL/dzeta_j [T][d_m], dL/dp_j [T], dL/dm_j [T] for the state
 * routed layer j hands on (zeros at the last layer); on return the same for the state it
 * received (S_{j-1}, zeta_{j-1}, p_{j-1}, m_{j-1}). */
typedef struct hero_router_carry {
  float *dS, *dzeta, *dp, *dm;
} hero_router_carry;

/* Workspace bytes for hero_router_backward with T tokens.  Host-only; validates dims. */
int hero_router_backward_workspace_size(const hero_dims *dims, int T, size_t *bytes);

/*
 * Backward of the router at routed layer j (Sec. 3.2 in reverse order; the gradient reaches
 * the router through the gate scaling, Sec. 3.1 remark after eq:ffn_route).  Given dL/dlogit
 * (e.g. hero_routed_block_backward's) and the carried state gradient, it
 *   - adds dL/d(router weights) into grads (the weights are shared by every routed layer, so a
 *     caller sums them over layers by calling for j = L_R .. 1 on the same buffers);
 *   - adds the post-attention states' share into dhbar (hbar_j: hidden encoder, local head,
 *     residual transitions), dhbar_prev1 (hbar_{j-1}, j >= 2) and dhbar_prev2 (hbar_{j-2},
 *     j >= 3): fp32 [T][d], three distinct buffers;
 *   - writes dL/deta_j into deta[0] (device fp32; rho_j = sigma(eta));
 *   - turns carry into the gradient over the state the layer received.
 * state_in is the router state entering layer j (fp32 S, zeta, p, m as the forward call read
 * them; not read at j = 1, where the state is the initial one and may be NULL, and carry's
 * return there is rho dL/dS_1).  Its c_read, when set (j >= 2), is the forward's memory read of
 * this layer, used instead of reading S_{j-1} a second time; it must not overlap the workspace or
 * any buffer the call writes.
 * hbar_prev1 / hbar_prev2: as in hero_routed_layer.  The full router with S in fp32
 * (dims->state_dtype HERO_F32, else HERO_E_UNSUPPORTED); branch decisions are constants.
 * Deterministic: every sum runs in a fixed order.
 */
int hero_router_backward(const hero_dims *dims, int j, int T, const void *hbar, const void *hbar_prev1,
                         const void *hbar_prev2, const hero_state *state_in, const hero_router_weights *router,
                         float eta, const float *dlogit, const hero_router_carry *carry, float *dhbar,
                         float *dhbar_prev1, float *dhbar_prev2, const hero_router_grads *grads, float *deta,
                         void *workspace, size_t workspace_bytes, void *stream);

#ifdef __cplusplus
}
#endif

#endif /* HERO_H */
