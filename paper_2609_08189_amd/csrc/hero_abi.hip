// C ABI of the HeRo routed FFN stack: argument validation, workspace layout and
// the per-layer kernel sequence.  Every argument check runs on the host before
// any HIP call, so invalid calls never reach the GPU.
#include <limits.h>
#include <math.h>
#include <stdint.h>
#include <string.h>

#include <algorithm>
#include <atomic>
#include <mutex>
#include <new>

#include "../../include/hero.h"
#include "hero_kernels.h"

static_assert(HERO_ABL_NO_POS_STATE == hero::ABL_NO_POS && HERO_ABL_NO_AUX_STATE == hero::ABL_NO_AUX &&
                  HERO_ABL_NO_MEMREAD == hero::ABL_NO_MEMREAD && HERO_ABL_NO_HISTORY == hero::ABL_NO_HISTORY,
              "ablation bits of the ABI and the kernels agree");

namespace {

constexpr size_t kAlign = 256;
size_t align_up(size_t x) { return (x + kAlign - 1) & ~(kAlign - 1); }

size_t esize(int dtype) { return dtype == HERO_BF16 ? 2 : 4; }

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// a workspace argument that tells check_layer_call the entry point brings its own scratch
void* const kNoWorkspace = reinterpret_cast<void*>(static_cast<uintptr_t>(-256));

bool overlap(const void* a, size_t na, const void* b, size_t nb) {
  if (!a || !b || na == 0 || nb == 0) return false;
  const uintptr_t x = reinterpret_cast<uintptr_t>(a), y = reinterpret_cast<uintptr_t>(b);
  return x < y + nb && y < x + na;
}

struct Layout {
  size_t u, P, rowstat, logit, gate, mask, idx_ffn, idx_ad, counts, lambda, act, part, part_ad, rscr, ring,
      total;
};

// At most this many tokens (a decode batch) the row statistics run beside the router product and
// the adapter branch beside the FFN branch, on a second stream (the adapter with a partial-sum
// region of its own).
constexpr int kOverlapTokens = 256;

Layout layout_of(const hero_dims& d, int T, bool stack) {
  const size_t es = esize(d.dtype), t = static_cast<size_t>(T);
  Layout L{};
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t o = off;
    off = align_up(off + bytes);
    return o;
  };
  L.u = take(t * d.d * es);
  L.P = take(t * (d.d_e + d.d_head) * 4 * hero::router_gemm_splits(d.dtype, d.d, T, d.d_e + d.d_head));
  L.rowstat = take(t * 16);
  L.logit = take(t * 4);
  L.gate = take(t * 4);
  L.mask = take(t);
  L.idx_ffn = take(t * 4);
  L.idx_ad = take(t * 4);
  L.counts = take(16);
  L.lambda = take(16);
  L.act = take(t * d.d_ff * es);
  // the FFN's split-K partials and the adapter's hidden rows: one region used in turn, or two
  // when the branches overlap
  const size_t pa = hero::adapter_part_floats(d.dtype, d.d, d.d_r, T) * 4;
  const size_t pf = hero::ffn_part_floats(d.dtype, d.d, d.d_ff, T) * 4;
  if (T <= kOverlapTokens) {
    L.part = take(pf);
    L.part_ad = take(pa);
  } else {
    L.part = L.part_ad = take(std::max(pa, pf));
  }
  L.rscr = take(hero::router_scratch_floats(d.d_m, d.d_head, T) * 4);
  L.ring = stack ? take(3 * t * d.d * es) : 0;
  L.total = off;
  return L;
}

// The bf16 GEMM core addresses operand rows with 32-bit byte offsets, so every operand it reads
// must span less than 4 GiB: T token rows of width d, d_ff or d_r (or of a given extra width),
// and the d_ff x d and d_r x d weights (the fp32 path uses 64-bit offsets).
constexpr long long kGemmSpan = 1LL << 32;
bool fwd_fits(const hero_dims& d, long long T, long long extra_width = 0) {
  if (d.dtype != HERO_BF16) return true;
  const long long w = std::max({static_cast<long long>(d.d), static_cast<long long>(d.d_ff),
                                static_cast<long long>(d.d_r), extra_width});
  return T * w * 2 < kGemmSpan && 2LL * d.d_ff * d.d < kGemmSpan && 2LL * d.d_r * d.d < kGemmSpan;
}

int check_dims(const hero_dims* d) {
  if (!d) return HERO_E_NULL;
  if (d->dtype != HERO_F32 && d->dtype != HERO_BF16) return HERO_E_DTYPE;
  if (d->d <= 0 || d->d_ff <= 0 || d->d_r <= 0 || d->L_R <= 0 || d->d_m <= 0 || d->d_s <= 0 ||
      d->d_h <= 0 || d->d_a <= 0 || d->d_e <= 0 || d->d_p <= 0 || d->d_head <= 0)
    return HERO_E_DIM;
  if (d->d_s != d->d_h + d->d_a) return HERO_E_DIM;
  if (!(d->eps_norm >= 0.f) || !(d->eps > 0.f) || !(d->T_hist > 0.f)) return HERO_E_RANGE;
  if (d->state_dtype != HERO_F32 && d->state_dtype != HERO_BF16) return HERO_E_DTYPE;
  if (d->state_dtype == HERO_BF16 && d->d_m < 64) return HERO_E_UNSUPPORTED;
  // kernel support
  if (d->d_m != 32 && d->d_m != 64 && d->d_m != 128 && d->d_m != 256) return HERO_E_UNSUPPORTED;
  if (d->d_s > 128 || d->d_e > 256 || d->d_head > 256 || d->d_p > 128) return HERO_E_UNSUPPORTED;
  if (d->dtype == HERO_BF16) {
    if (d->d % 256 || d->d_ff % 128 || d->d_e % 64 || (d->d_e + d->d_head) % 128) return HERO_E_UNSUPPORTED;
    // adapter ranks: 32..128 in steps of 32 (register-tiled kernels) or wider in steps of 128
    // (GEMM path, e.g. the paper's 896)
    const bool small_r = d->d_r % 32 == 0 && d->d_r <= 128;
    const bool wide_r = d->d_r % 128 == 0 && d->d_r > 128 && d->d_r <= 8192;
    if (!(small_r || wide_r) || d->d_s % 8) return HERO_E_UNSUPPORTED;
  } else {
    if (d->d % 128) return HERO_E_UNSUPPORTED;
  }
  return HERO_OK;
}

int check_routing(const hero_routing* r) {
  if (!r) return HERO_E_NULL;
  if (r->mode == HERO_MODE_THRESHOLD) {
    if (!(r->tau > 0.f && r->tau < 1.f)) return HERO_E_RANGE;
  } else if (r->mode == HERO_MODE_BUDGET) {
    if (!(r->budget >= 0.0 && r->budget <= 1.0)) return HERO_E_RANGE;
  } else {
    return HERO_E_RANGE;
  }
  if (r->ablation & ~HERO_ABL_ALL) return HERO_E_RANGE;
  if (r->logit_bias && !aligned16(r->logit_bias)) return HERO_E_ALIGN;
  return HERO_OK;
}

// the optional tiled FFN weights (hero_ffn_decode_weights_make): bf16 models with d_ff % 64 == 0
int check_ffn_tiled(const hero_dims& d, const hero_ffn_weights* f) {
  if (!f->w_gate_up_tiled && !f->w_down_tiled) return HERO_OK;
  if (d.dtype != HERO_BF16 || d.d_ff % 64 != 0) return HERO_E_UNSUPPORTED;
  if ((f->w_gate_up_tiled && !aligned16(f->w_gate_up_tiled)) || (f->w_down_tiled && !aligned16(f->w_down_tiled)))
    return HERO_E_ALIGN;
  return HERO_OK;
}

int check_weights(const hero_ffn_weights* f, const hero_router_weights* r, const hero_adapter_weights* a) {
  if (!f || !r || !a) return HERO_E_NULL;
  const void* ptrs[] = {f->norm_w, f->w_gate, f->w_up, f->w_down, a->w1, a->w2,
                        r->w_hd, r->w_hu, r->w_p1, r->w_p2, r->w_q, r->w_k, r->w_v,
                        r->w_n, r->w_c, r->th1, r->th2, r->ps1, r->ps2};
  for (const void* p : ptrs)
    if (!p) return HERO_E_NULL;
  for (const void* p : ptrs)
    if (!aligned16(p)) return HERO_E_ALIGN;
  return HERO_OK;
}

int check_state(const hero_state* s) {
  if (!s || !s->S || !s->zeta || !s->p_hist || !s->m_hist) return HERO_E_NULL;
  if (!aligned16(s->S) || !aligned16(s->zeta) || !aligned16(s->p_hist) || !aligned16(s->m_hist) ||
      (s->c_read && !aligned16(s->c_read)))
    return HERO_E_ALIGN;
  return HERO_OK;
}

// the optional memory-read output (hero_state.c_read) may not overlap the state, the layer's
// activations or the workspace
int check_c_read(const hero_dims& d, int T, const hero_state* s, const void* hbar, const void* hbar_prev1,
                 const void* hbar_prev2, const void* h_out, const void* ws, size_t ws_bytes) {
  if (!s->c_read) return HERO_OK;
  const size_t t = static_cast<size_t>(T), dm = static_cast<size_t>(d.d_m), cb = t * dm * 4;
  const size_t sb = t * dm * dm * (d.state_dtype == HERO_BF16 ? 2 : 4);
  const size_t hb = t * static_cast<size_t>(d.d) * (d.dtype == HERO_BF16 ? 2 : 4);
  const void* c = s->c_read;
  if (overlap(c, cb, s->S, sb) || overlap(c, cb, s->zeta, t * dm * 4) || overlap(c, cb, s->p_hist, t * 4) ||
      overlap(c, cb, s->m_hist, t * 4) || overlap(c, cb, hbar, hb) || overlap(c, cb, hbar_prev1, hb) ||
      overlap(c, cb, hbar_prev2, hb) || overlap(c, cb, h_out, hb) || overlap(c, cb, ws, ws_bytes))
    return HERO_E_ALIAS;
  return HERO_OK;
}

int check_history(const hero_history* h) {
  if (!h || !h->kv || !h->p_hist || !h->m_hist) return HERO_E_NULL;
  if (!aligned16(h->kv) || !aligned16(h->p_hist) || !aligned16(h->m_hist)) return HERO_E_ALIGN;
  return HERO_OK;
}

int check_stats(const hero_layer_stats* s) {
  if (!s) return HERO_OK;
  const void* ptrs[] = {s->mask, s->idx_ffn, s->idx_ad, s->counts, s->logit, s->gate, s->lambda};
  for (const void* p : ptrs)
    if (p && !aligned16(p)) return HERO_E_ALIGN;
  return HERO_OK;
}

// The current device must be gfx950; checked once per device.
int check_device() {
  static std::atomic<int> known[64];  // 0 unknown, 1 ok, 2 not gfx950
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0) return HERO_E_DEVICE;
  if (dev < 64) {
    const int k = known[dev].load(std::memory_order_acquire);
    if (k != 0) return k == 1 ? HERO_OK : HERO_E_DEVICE;
  }
  hipDeviceProp_t prop;
  if (hipGetDeviceProperties(&prop, dev) != hipSuccess) return HERO_E_DEVICE;
  const bool ok = strncmp(prop.gcnArchName, "gfx950", 6) == 0;
  if (dev < 64) known[dev].store(ok ? 1 : 2, std::memory_order_release);
  return ok ? HERO_OK : HERO_E_DEVICE;
}

// Measurement hook: caller-created events recorded around the launches of one kernel.
struct KernelTimer {
  hipEvent_t* start = nullptr;
  hipEvent_t* stop = nullptr;
  int n = 0;
  int next = 0;
};
KernelTimer g_timer[HERO_K_COUNT];

template <class F>
hipError_t timed(int which, hipStream_t s, F&& launch) {
  KernelTimer& k = g_timer[which];
  if (k.n == 0) return launch();
  const int i = k.next;
  hipError_t e = hipEventRecord(k.start[i], s);
  if (e != hipSuccess) return e;
  e = launch();
  if (e != hipSuccess) return e;
  e = hipEventRecord(k.stop[i], s);
  k.next = (i + 1) % k.n;
  return e;
}

// A second stream of the calling thread on one device, with the events that fork work onto it
// and join it back (thread-local: calls from different host threads never share one).  Created
// on a device's first call from the thread, outside any graph capture that follows (a failure
// leaves the calls on one stream), and kept until the process ends.
struct Side {
  hipStream_t s = nullptr;
  hipEvent_t fork = nullptr, join = nullptr;
  bool tried = false;
};

const Side* side_of_current_device() {
  constexpr int kDevices = 64;
  thread_local Side sides[kDevices];
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kDevices) return nullptr;
  Side& sd = sides[dev];
  if (!sd.tried) {
    sd.tried = true;
    // default priority (work on streams of different priorities has hung on this hardware)
    if (hipStreamCreateWithFlags(&sd.s, hipStreamNonBlocking) != hipSuccess) sd.s = nullptr;
    if (sd.s && (hipEventCreateWithFlags(&sd.fork, hipEventDisableTiming) != hipSuccess ||
                 hipEventCreateWithFlags(&sd.join, hipEventDisableTiming) != hipSuccess))
      sd.s = nullptr;
  }
  return sd.s ? &sd : nullptr;
}

struct LayerCall {
  const hero_dims* dims;
  int j, T;
  const void *hbar, *prev1, *prev2;
  void* h_out;
  const hero_state* st;
  const hero_ffn_weights* ffn;
  const hero_router_weights* rt;
  const hero_adapter_weights* ad;
  float eta;
  const hero_routing* rc;
  const hero_layer_stats* stats;
  unsigned char* ws;
  const Layout* L;
  hipStream_t stream;
  // depth-history form of the memory: the pairs and the weights of the j-1 stored ones
  const hero_history* hist = nullptr;
  const float* hw = nullptr;
  // the second stream (null: every launch on the call's stream)
  const Side* side = nullptr;
  // where the layer's memory read c goes as well (null: nowhere)
  float* c_read = nullptr;
};

// rho_l = sigma(eta_l); w[i] = prod_{l=i+2}^{j-1} rho_l is the weight of entry i (routed layer
// i+1) in the read of layer j, i < j-1 (eta: host, eta_1 .. eta_{j-1} at least)
void history_weights(const float* eta, int j, float* w) {
  double acc = 1.0;
  for (int i = j - 2; i >= 0; --i) {
    w[i] = static_cast<float>(acc);
    const double rho = 1.0 / (1.0 + exp(-static_cast<double>(eta[i])));   // layer i+1
    acc *= rho;
  }
}

int run_layer(const LayerCall& c) {
  using namespace hero;
  const hero_dims& D = *c.dims;
  const int T = c.T;
  unsigned char* ws = c.ws;
  const Layout& L = *c.L;
  const hero_layer_stats* S = c.stats;
  float* logit = (S && S->logit) ? S->logit : reinterpret_cast<float*>(ws + L.logit);
  float* gate = (S && S->gate) ? S->gate : reinterpret_cast<float*>(ws + L.gate);
  uint8_t* mask = (S && S->mask) ? S->mask : reinterpret_cast<uint8_t*>(ws + L.mask);
  int* idx_ffn = (S && S->idx_ffn) ? S->idx_ffn : reinterpret_cast<int*>(ws + L.idx_ffn);
  int* idx_ad = (S && S->idx_ad) ? S->idx_ad : reinterpret_cast<int*>(ws + L.idx_ad);
  int* counts = (S && S->counts) ? S->counts : reinterpret_cast<int*>(ws + L.counts);
  float* lambda = (S && S->lambda) ? S->lambda : reinterpret_cast<float*>(ws + L.lambda);
  void* u = ws + L.u;
  float* P = reinterpret_cast<float*>(ws + L.P);
  float* rowstat = reinterpret_cast<float*>(ws + L.rowstat);

  const hipStream_t st = c.stream;
  // work on the second stream starts after everything issued so far on st, and st waits for it
  const Side* sd = c.side;
  auto fork = [&]() {
    hipError_t x = hipEventRecord(sd->fork, st);
    return x == hipSuccess ? hipStreamWaitEvent(sd->s, sd->fork, 0) : x;
  };
  auto join = [&]() {
    hipError_t x = hipEventRecord(sd->join, sd->s);
    return x == hipSuccess ? hipStreamWaitEvent(st, sd->join, 0) : x;
  };
  // the row statistics (for the router's path vector and the branches' input) and the router's
  // pre-activation product both read only hbar: side by side for a decode batch (with many
  // tokens the product fills every CU and the statistics pass, starved, only stretches)
  const bool ovl_rows = sd && T <= kOverlapTokens;
  const hipStream_t s_rows = ovl_rows ? sd->s : st;
  hipError_t e = ovl_rows ? fork() : hipSuccess;
  if (e != hipSuccess) return HERO_E_LAUNCH;
  e = timed(HERO_K_ROWSTATS, s_rows, [&] {
    return launch_rowstats(D.dtype, c.hbar, c.j >= 2 ? c.prev1 : nullptr, c.j >= 3 ? c.prev2 : nullptr,
                           c.ffn->norm_w, T, D.d, c.j, D.eps_norm, rowstat, u, s_rows);
  });
  if (e != hipSuccess) return HERO_E_LAUNCH;
  e = timed(HERO_K_ROUTER_GEMM, st, [&] {
    return launch_router_gemm(D.dtype, c.hbar, c.rt->w_hd, c.rt->ps1, T, D.d, D.d_e, D.d_head, P, st);
  });
  if (e != hipSuccess) return HERO_E_LAUNCH;
  if (ovl_rows && join() != hipSuccess) return HERO_E_LAUNCH;

  RouterTailArgs ra{};
  ra.dtype = D.dtype;
  ra.T = T;
  ra.j = c.j;
  ra.L_R = D.L_R;
  ra.d_m = D.d_m;
  ra.d_s = D.d_s;
  ra.d_h = D.d_h;
  ra.d_a = D.d_a;
  ra.d_e = D.d_e;
  ra.d_p = D.d_p;
  ra.d_head = D.d_head;
  ra.eps = D.eps;
  ra.T_hist = D.T_hist;
  ra.eta = c.eta;
  ra.P = P;
  ra.p_splits = router_gemm_splits(D.dtype, D.d, c.T, D.d_e + D.d_head);
  ra.rowstat = rowstat;
  ra.w_hu = c.rt->w_hu;
  ra.w_p1 = c.rt->w_p1;
  ra.w_p2 = c.rt->w_p2;
  ra.w_q = c.rt->w_q;
  ra.w_k = c.rt->w_k;
  ra.w_v = c.rt->w_v;
  ra.w_n = c.rt->w_n;
  ra.w_c = c.rt->w_c;
  ra.th1 = c.rt->th1;
  ra.ld_th1 = HERO_TH1_PITCH(D.d_s, D.d_m);
  ra.th2 = c.rt->th2;
  ra.ps2 = c.rt->ps2;
  ra.beta = c.rc->logit_bias;
  ra.abl = c.rc->ablation;
  if (c.hist) {
    ra.kv = c.hist->kv;
    ra.p_hist = c.hist->p_hist;
    ra.m_hist = c.hist->m_hist;
    for (int i = 0; i < c.j - 1; ++i) ra.hw[i] = c.hw[i];
  } else {
    ra.S = c.st->S;
    ra.state_bf16 = D.state_dtype == HERO_BF16;
    ra.zeta = c.st->zeta;
    ra.p_hist = c.st->p_hist;
    ra.m_hist = c.st->m_hist;
  }
  ra.logit = logit;
  ra.gate = gate;
  {
    float* r = reinterpret_cast<float*>(ws + L.rscr);
    const size_t t = static_cast<size_t>(T);
    ra.qkvn = r;
    ra.hs = r + t * 4 * D.d_m;
    ra.cvec = ra.hs + t * D.d_head;
    ra.bvec = ra.cvec + t * D.d_m;
  }
  e = timed(HERO_K_ROUTER_PRE, st, [&] { return launch_router_pre(ra, st); });
  if (e != hipSuccess) return HERO_E_LAUNCH;
  // the ablations without memory access leave S, zeta (or the stored pairs) untouched
  if (!(ra.abl & (HERO_ABL_NO_MEMREAD | HERO_ABL_NO_HISTORY))) {
    e = timed(HERO_K_ROUTER_MEM, st, [&] {
      return c.hist ? launch_router_mem_hist(ra, st) : launch_router_mem(ra, st);
    });
    if (e != hipSuccess) return HERO_E_LAUNCH;
    if (c.c_read &&
        hipMemcpyAsync(c.c_read, ra.cvec, static_cast<size_t>(T) * D.d_m * sizeof(float), hipMemcpyDeviceToDevice,
                       st) != hipSuccess)
      return HERO_E_LAUNCH;
  }
  e = timed(HERO_K_ROUTER_POST, st, [&] { return launch_router_post(ra, st); });
  if (e != hipSuccess) return HERO_E_LAUNCH;

  SelectArgs sa{};
  sa.logit = logit;
  sa.T = T;
  sa.mode = c.rc->mode;
  sa.thr = static_cast<float>(log(static_cast<double>(c.rc->tau) / (1.0 - static_cast<double>(c.rc->tau))));
  const int n_skip = c.rc->mode == HERO_MODE_BUDGET
                         ? static_cast<int>(floor(c.rc->budget * static_cast<double>(T) + 0.5))
                         : 0;
  sa.n_skip = n_skip;
  sa.mask = mask;
  sa.idx_ffn = idx_ffn;
  sa.idx_ad = idx_ad;
  sa.counts = counts;
  sa.lambda = lambda;
  e = timed(HERO_K_SELECT, st, [&] { return launch_select(sa, st); });
  if (e != hipSuccess) return HERO_E_LAUNCH;

  // grid sizes: exact in budget mode, T in threshold mode (tiles past the device count exit)
  const int n_ffn_max = c.rc->mode == HERO_MODE_BUDGET ? T - n_skip : T;
  const int n_ad_max = c.rc->mode == HERO_MODE_BUDGET ? n_skip : T;
  void* act = ws + L.act;
  float* part = reinterpret_cast<float*>(ws + L.part);
  float* part_ad = reinterpret_cast<float*>(ws + L.part_ad);
  // the two branches write disjoint rows of h_out and read only hbar, u, the gates and the lists:
  // for a decode batch the adapter's latency-bound launches run beside the FFN's weight stream
  const bool ovl = sd && T <= kOverlapTokens && n_ffn_max > 0 && n_ad_max > 0;
  const hipStream_t s_ad = ovl ? sd->s : st;
  if (ovl && fork() != hipSuccess) return HERO_E_LAUNCH;
  if (n_ffn_max > 0) {
    e = timed(HERO_K_FFN_GATE_UP, st, [&] {
      return launch_ffn_gateup(D.dtype, u, idx_ffn, counts, n_ffn_max, c.ffn->w_gate, c.ffn->w_up,
                               c.ffn->w_gate_up_tiled, act, part, D.d, D.d_ff, st);
    });
    if (e != hipSuccess) return HERO_E_LAUNCH;
    e = timed(HERO_K_FFN_DOWN, st, [&] {
      return launch_ffn_down(D.dtype, act, idx_ffn, counts, n_ffn_max, c.ffn->w_down, c.ffn->w_down_tiled,
                             c.hbar, gate, c.h_out, part, D.d, D.d_ff, st);
    });
    if (e != hipSuccess) return HERO_E_LAUNCH;
  }
  if (n_ad_max > 0) {
    e = timed(HERO_K_ADAPTER_DOWN, s_ad, [&] {
      return launch_adapter_down(D.dtype, u, idx_ad, counts + 1, n_ad_max, c.ad->w1, part_ad, D.d,
                                 D.d_r, s_ad);
    });
    if (e != hipSuccess) return HERO_E_LAUNCH;
    e = timed(HERO_K_ADAPTER_UP, s_ad, [&] {
      return launch_adapter_up(D.dtype, part_ad, idx_ad, counts + 1, n_ad_max, c.ad->w2, c.hbar, gate,
                               c.h_out, D.d, D.d_r, s_ad);
    });
    if (e != hipSuccess) return HERO_E_LAUNCH;
  }
  if (ovl && join() != hipSuccess) return HERO_E_LAUNCH;
  return HERO_OK;
}

}  // namespace

extern "C" {

const char* hero_status_string(int status) {
  switch (status) {
    case HERO_OK: return "ok";
    case HERO_E_NULL: return "a required pointer is NULL";
    case HERO_E_DIM: return "a size is non-positive or inconsistent";
    case HERO_E_RANGE: return "an argument is out of range";
    case HERO_E_DTYPE: return "unknown dtype";
    case HERO_E_ALIGN: return "a device pointer is not 16-byte aligned";
    case HERO_E_ALIAS: return "an output overlaps an input";
    case HERO_E_WORKSPACE: return "workspace missing or too small";
    case HERO_E_UNSUPPORTED: return "shape not supported by the kernels";
    case HERO_E_LAUNCH: return "kernel launch failed";
    case HERO_E_DEVICE: return "no usable gfx950 device";
    case HERO_E_SCRATCH: return "the call needs more device scratch than the fixed no-alloc area holds";
    default: return "unknown status";
  }
}

int hero_abi_version(void) { return HERO_ABI_VERSION; }

int hero_kernel_timer(int kernel, void* const* start_events, void* const* stop_events, int n_slots) {
  if (kernel < 0 || kernel >= HERO_K_COUNT || n_slots < 0) return HERO_E_RANGE;
  if (n_slots > 0 && (!start_events || !stop_events)) return HERO_E_NULL;
  KernelTimer& k = g_timer[kernel];
  delete[] k.start;
  delete[] k.stop;
  k.start = k.stop = nullptr;
  k.n = k.next = 0;
  if (n_slots == 0) return HERO_OK;
  // no exception may leave the C interface: a registry too large to allocate is out of range
  k.start = new (std::nothrow) hipEvent_t[n_slots];
  k.stop = new (std::nothrow) hipEvent_t[n_slots];
  if (!k.start || !k.stop) {
    delete[] k.start;
    delete[] k.stop;
    k.start = k.stop = nullptr;
    return HERO_E_RANGE;
  }
  for (int i = 0; i < n_slots; ++i) {
    k.start[i] = static_cast<hipEvent_t>(start_events[i]);
    k.stop[i] = static_cast<hipEvent_t>(stop_events[i]);
  }
  k.n = n_slots;
  return HERO_OK;
}

int hero_workspace_size(const hero_dims* dims, int T, int for_stack, size_t* bytes) {
  if (!bytes) return HERO_E_NULL;
  const int st = check_dims(dims);
  if (st != HERO_OK) return st;
  if (T <= 0) return HERO_E_DIM;
  *bytes = layout_of(*dims, T, for_stack != 0).total;
  return HERO_OK;
}

namespace {

// Checks shared by both forms of the layer call; state or history is checked by the caller.
int check_layer_call(const hero_dims* dims, int j, int T, const void* hbar, const void* hbar_prev1,
                     const void* hbar_prev2, const void* h_out, const hero_ffn_weights* ffn,
                     const hero_router_weights* router, const hero_adapter_weights* adapter,
                     const hero_routing* routing, const hero_layer_stats* stats, const void* workspace,
                     size_t workspace_bytes, Layout* L) {
  int st = check_dims(dims);
  if (st != HERO_OK) return st;
  if (T <= 0) return HERO_E_DIM;
  if (!fwd_fits(*dims, T)) return HERO_E_UNSUPPORTED;
  if (j < 1 || j > dims->L_R) return HERO_E_RANGE;
  if (!hbar || !h_out) return HERO_E_NULL;
  if (j >= 2 && !hbar_prev1) return HERO_E_NULL;
  if (j >= 3 && !hbar_prev2) return HERO_E_NULL;
  if (!aligned16(hbar) || !aligned16(h_out) || (j >= 2 && !aligned16(hbar_prev1)) ||
      (j >= 3 && !aligned16(hbar_prev2)))
    return HERO_E_ALIGN;
  if ((st = check_weights(ffn, router, adapter)) != HERO_OK) return st;
  if ((st = check_ffn_tiled(*dims, ffn)) != HERO_OK) return st;
  if ((st = check_routing(routing)) != HERO_OK) return st;
  if ((st = check_stats(stats)) != HERO_OK) return st;
  const size_t hb = static_cast<size_t>(T) * dims->d * esize(dims->dtype);
  if (overlap(h_out, hb, hbar, hb) || (j >= 2 && overlap(h_out, hb, hbar_prev1, hb)) ||
      (j >= 3 && overlap(h_out, hb, hbar_prev2, hb)))
    return HERO_E_ALIAS;
  *L = layout_of(*dims, T, false);
  if (workspace == kNoWorkspace) return HERO_OK;      // the no-alloc entry point brings its own
  if (!workspace) return HERO_E_WORKSPACE;
  if (workspace_bytes < L->total) return HERO_E_WORKSPACE;
  if (!aligned16(workspace)) return HERO_E_ALIGN;
  return HERO_OK;
}

// The no-alloc entry point's scratch: one fixed device array per device, for the life of the
// process.  In host code the name `noalloc_scratch` is only a host-side stand-in for the array;
// the device address comes from hipGetSymbolAddress, looked up once per device with that device
// current, and only that address is ever handed to kernels.
__device__ __align__(256) unsigned char noalloc_scratch[HERO_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices];

int scratch_of_current_device(void** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return HERO_E_DEVICE;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(noalloc_scratch)) != hipSuccess || !p) return HERO_E_DEVICE;
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return HERO_OK;
}

}  // namespace

int hero_routed_layer(const hero_dims* dims, int j, int T, const void* hbar, const void* hbar_prev1,
                      const void* hbar_prev2, void* h_out, const hero_state* state,
                      const hero_ffn_weights* ffn, const hero_router_weights* router,
                      const hero_adapter_weights* adapter, float eta, const hero_routing* routing,
                      const hero_layer_stats* stats, void* workspace, size_t workspace_bytes,
                      void* stream) {
  Layout L;
  int st = check_layer_call(dims, j, T, hbar, hbar_prev1, hbar_prev2, h_out, ffn, router, adapter, routing,
                            stats, workspace, workspace_bytes, &L);
  if (st != HERO_OK) return st;
  if ((st = check_state(state)) != HERO_OK) return st;
  if (!(eta == eta)) return HERO_E_RANGE;
  if ((st = check_c_read(*dims, T, state, hbar, j >= 2 ? hbar_prev1 : nullptr, j >= 3 ? hbar_prev2 : nullptr,
                         h_out, workspace, L.total)) != HERO_OK)
    return st;
  if ((st = check_device()) != HERO_OK) return st;
  LayerCall c{dims, j, T, hbar, hbar_prev1, hbar_prev2, h_out, state, ffn, router, adapter, eta,
              routing, stats, static_cast<unsigned char*>(workspace), &L,
              static_cast<hipStream_t>(stream)};
  c.side = side_of_current_device();
  c.c_read = state->c_read;
  return run_layer(c);
}

int hero_routed_layer_noalloc(const hero_dims* dims, int j, int T, const void* hbar, const void* hbar_prev1,
                              const void* hbar_prev2, void* h_out, const hero_state* state,
                              const hero_ffn_weights* ffn, const hero_router_weights* router,
                              const hero_adapter_weights* adapter, float eta, const hero_routing* routing,
                              const hero_layer_stats* stats, void* stream) {
  Layout L;
  int st = check_layer_call(dims, j, T, hbar, hbar_prev1, hbar_prev2, h_out, ffn, router, adapter, routing,
                            stats, kNoWorkspace, 0, &L);
  if (st != HERO_OK) return st;
  if (L.total > HERO_NOALLOC_SCRATCH_BYTES) return HERO_E_SCRATCH;
  if ((st = check_state(state)) != HERO_OK) return st;
  if (!(eta == eta)) return HERO_E_RANGE;
  if ((st = check_device()) != HERO_OK) return st;
  void* scratch = nullptr;
  if ((st = scratch_of_current_device(&scratch)) != HERO_OK) return st;
  if ((st = check_c_read(*dims, T, state, hbar, j >= 2 ? hbar_prev1 : nullptr, j >= 3 ? hbar_prev2 : nullptr,
                         h_out, scratch, L.total)) != HERO_OK)
    return st;
  LayerCall c{dims, j, T, hbar, hbar_prev1, hbar_prev2, h_out, state, ffn, router, adapter, eta,
              routing, stats, static_cast<unsigned char*>(scratch), &L, static_cast<hipStream_t>(stream)};
  c.c_read = state->c_read;
  return run_layer(c);
}

int hero_routed_layer_hist(const hero_dims* dims, int j, int T, const void* hbar, const void* hbar_prev1,
                           const void* hbar_prev2, void* h_out, const hero_history* history,
                           const hero_ffn_weights* ffn, const hero_router_weights* router,
                           const hero_adapter_weights* adapter, const float* eta,
                           const hero_routing* routing, const hero_layer_stats* stats, void* workspace,
                           size_t workspace_bytes, void* stream) {
  Layout L;
  int st = check_layer_call(dims, j, T, hbar, hbar_prev1, hbar_prev2, h_out, ffn, router, adapter, routing,
                            stats, workspace, workspace_bytes, &L);
  if (st != HERO_OK) return st;
  if (dims->L_R > 64 || dims->state_dtype != HERO_F32) return HERO_E_UNSUPPORTED;
  if ((st = check_history(history)) != HERO_OK) return st;
  if (!eta) return HERO_E_NULL;
  for (int l = 0; l < j; ++l)
    if (!(eta[l] == eta[l])) return HERO_E_RANGE;
  if ((st = check_device()) != HERO_OK) return st;
  float hw[64];
  history_weights(eta, j, hw);
  LayerCall c{dims, j, T, hbar, hbar_prev1, hbar_prev2, h_out, nullptr, ffn, router, adapter, eta[j - 1],
              routing, stats, static_cast<unsigned char*>(workspace), &L,
              static_cast<hipStream_t>(stream), history, hw, side_of_current_device()};
  return run_layer(c);
}

namespace {

// hero_routed_stack and hero_routed_stack_hist: exactly one of state / history is set.
int routed_stack(const hero_dims* dims, int T, const void* h_in, void* h_out, const hero_state* state,
                 const hero_history* history, const hero_ffn_weights* ffn, const hero_router_weights* router,
                 const hero_adapter_weights* adapter, const float* eta, const hero_routing* routing,
                 const hero_layer_stats* stats, void* workspace, size_t workspace_bytes, void* stream) {
  int st = check_dims(dims);
  if (st != HERO_OK) return st;
  if (T <= 0) return HERO_E_DIM;
  if (!fwd_fits(*dims, T)) return HERO_E_UNSUPPORTED;
  if (!h_in || !h_out || !ffn || !adapter || !eta) return HERO_E_NULL;
  if (!aligned16(h_in) || !aligned16(h_out)) return HERO_E_ALIGN;
  if (history) {
    if (dims->L_R > 64 || dims->state_dtype != HERO_F32) return HERO_E_UNSUPPORTED;
    if ((st = check_history(history)) != HERO_OK) return st;
  } else if ((st = check_state(state)) != HERO_OK) {
    return st;
  }
  if ((st = check_routing(routing)) != HERO_OK) return st;
  for (int l = 0; l < dims->L_R; ++l) {
    if ((st = check_weights(&ffn[l], router, &adapter[l])) != HERO_OK) return st;
    if ((st = check_ffn_tiled(*dims, &ffn[l])) != HERO_OK) return st;
    if (!(eta[l] == eta[l])) return HERO_E_RANGE;
    if (stats && (st = check_stats(&stats[l])) != HERO_OK) return st;
  }
  const size_t hb = static_cast<size_t>(T) * dims->d * esize(dims->dtype);
  if (overlap(h_out, hb, h_in, hb)) return HERO_E_ALIAS;
  const Layout L = layout_of(*dims, T, true);
  if (!workspace) return HERO_E_WORKSPACE;
  if (workspace_bytes < L.total) return HERO_E_WORKSPACE;
  if (!aligned16(workspace)) return HERO_E_ALIGN;
  if (overlap(h_out, hb, workspace, L.total)) return HERO_E_ALIAS;
  if ((st = check_device()) != HERO_OK) return st;

  unsigned char* ws = static_cast<unsigned char*>(workspace);
  const void* ring[3] = {ws + L.ring, ws + L.ring + hb, ws + L.ring + 2 * hb};
  auto hbar_of = [&](int jj) -> const void* {  // post-attention state entering routed layer jj
    return jj == 1 ? h_in : ring[(jj - 2) % 3];
  };
  float hw[64];
  const Side* side = side_of_current_device();
  for (int j = 1; j <= dims->L_R; ++j) {
    void* out = j == dims->L_R ? h_out : const_cast<void*>(ring[(j - 1) % 3]);
    if (history) history_weights(eta, j, hw);
    LayerCall c{dims, j, T, hbar_of(j), j >= 2 ? hbar_of(j - 1) : nullptr,
                j >= 3 ? hbar_of(j - 2) : nullptr, out, state, &ffn[j - 1], router,
                &adapter[j - 1], eta[j - 1], routing, stats ? &stats[j - 1] : nullptr, ws, &L,
                static_cast<hipStream_t>(stream), history, history ? hw : nullptr, side};
    if ((st = run_layer(c)) != HERO_OK) return st;
  }
  return HERO_OK;
}

}  // namespace

int hero_routed_stack(const hero_dims* dims, int T, const void* h_in, void* h_out,
                      const hero_state* state, const hero_ffn_weights* ffn,
                      const hero_router_weights* router, const hero_adapter_weights* adapter,
                      const float* eta, const hero_routing* routing, const hero_layer_stats* stats,
                      void* workspace, size_t workspace_bytes, void* stream) {
  return routed_stack(dims, T, h_in, h_out, state, nullptr, ffn, router, adapter, eta, routing, stats,
                      workspace, workspace_bytes, stream);
}

int hero_routed_stack_hist(const hero_dims* dims, int T, const void* h_in, void* h_out,
                           const hero_history* history, const hero_ffn_weights* ffn,
                           const hero_router_weights* router, const hero_adapter_weights* adapter,
                           const float* eta, const hero_routing* routing, const hero_layer_stats* stats,
                           void* workspace, size_t workspace_bytes, void* stream) {
  if (!history) return HERO_E_NULL;
  return routed_stack(dims, T, h_in, h_out, nullptr, history, ffn, router, adapter, eta, routing, stats,
                      workspace, workspace_bytes, stream);
}

int hero_history_state(const hero_dims* dims, int n, int T, const float* kv, const float* eta, float* S,
                       float* zeta, void* stream) {
  int st = check_dims(dims);
  if (st != HERO_OK) return st;
  if (T <= 0) return HERO_E_DIM;
  if (dims->L_R > 64 || dims->state_dtype != HERO_F32) return HERO_E_UNSUPPORTED;
  if (n < 0 || n > dims->L_R) return HERO_E_RANGE;
  if (!kv || !S || !zeta || (n > 0 && !eta)) return HERO_E_NULL;
  if (!aligned16(kv) || !aligned16(S) || !aligned16(zeta)) return HERO_E_ALIGN;
  for (int l = 0; l < n; ++l)
    if (!(eta[l] == eta[l])) return HERO_E_RANGE;
  const size_t dm = static_cast<size_t>(dims->d_m), t = static_cast<size_t>(T);
  const size_t kvb = t * dims->L_R * 2 * dm * 4;
  if (overlap(S, t * dm * dm * 4, kv, kvb) || overlap(zeta, t * dm * 4, kv, kvb) ||
      overlap(S, t * dm * dm * 4, zeta, t * dm * 4))
    return HERO_E_ALIAS;
  if ((st = check_device()) != HERO_OK) return st;
  hero::HistWeights w{};
  history_weights(eta, n + 1, w.w);   // the weights of a read at layer n + 1
  return hero::launch_history_state(dims->d_m, dims->L_R, n, T, kv, w, S, zeta,
                                    static_cast<hipStream_t>(stream)) == hipSuccess
             ? HERO_OK
             : HERO_E_LAUNCH;
}

}  // extern "C"

// ---------------------------------------------------------------------------
// The full decoder: attention sub-block, pretrained FFN of non-routed blocks, decoder stack
// ---------------------------------------------------------------------------
namespace {

constexpr int kAttnHeadDim = 128;
constexpr int kAttnQTile = 128;   // queries per attention workgroup: the q/k/v row padding

int check_attn_dims(const hero_dims* d, const hero_attn_dims* a) {
  if (!a) return HERO_E_NULL;
  if (a->n_heads <= 0 || a->n_kv_heads <= 0 || a->head_dim <= 0) return HERO_E_DIM;
  if (a->n_heads % a->n_kv_heads) return HERO_E_DIM;
  if (d->dtype != HERO_BF16 || a->head_dim != kAttnHeadDim || a->n_heads % 2) return HERO_E_UNSUPPORTED;
  return HERO_OK;
}

// token count and the spans of the attention products' operands (x [T][d], o [T][n_h hd],
// W_qkv [(n_h + 2 n_kv) hd][d], W_o [d][n_h hd]) on the GEMM core
int check_dec_size(const hero_dims& d, const hero_attn_dims& a, int batch, int seq) {
  if (batch <= 0 || seq <= 0) return HERO_E_DIM;
  const long long T = static_cast<long long>(batch) * seq;
  if (T > INT_MAX / 2) return HERO_E_DIM;
  const long long q_width = static_cast<long long>(a.n_heads) * a.head_dim;
  const long long qkv_rows = static_cast<long long>(a.n_heads + 2 * a.n_kv_heads) * a.head_dim;
  if (!fwd_fits(d, T, q_width) || 2 * qkv_rows * d.d >= kGemmSpan || 2 * q_width * d.d >= kGemmSpan)
    return HERO_E_UNSUPPORTED;
  return HERO_OK;
}

int check_attn_weights(const hero_attn_weights* w) {
  if (!w || !w->norm_w || !w->w_qkv || !w->w_o) return HERO_E_NULL;
  if (!aligned16(w->norm_w) || !aligned16(w->w_qkv) || !aligned16(w->w_o)) return HERO_E_ALIGN;
  return HERO_OK;
}

int check_rope(const float* inv_freq, int head_dim, hero::RopeTable* t) {
  if (!inv_freq) return HERO_E_NULL;
  for (int i = 0; i < head_dim / 2; ++i) {
    if (!(inv_freq[i] == inv_freq[i]) || inv_freq[i] - inv_freq[i] != 0.f) return HERO_E_RANGE;
    t->inv_freq[i] = inv_freq[i];
  }
  return HERO_OK;
}

struct DecLayout {
  Layout L;            // the routed layer's workspace (its u region holds LN^attn(h) too)
  int seq_pad;
  size_t q, k, vt, o;  // attention intermediates
  size_t rope;         // [seq][64] (cos, sin) of the rotary angles
  size_t ring, hA, hB, hbar_tmp;
  size_t total;
};

DecLayout dec_layout_of(const hero_dims& d, const hero_attn_dims& a, int n_layers, int batch, int seq) {
  DecLayout D{};
  const size_t T = static_cast<size_t>(batch) * seq;
  D.L = layout_of(d, static_cast<int>(T), false);
  D.seq_pad = (seq + kAttnQTile - 1) / kAttnQTile * kAttnQTile;
  size_t off = D.L.total;
  auto take = [&](size_t bytes) {
    const size_t o = off;
    off = align_up(off + bytes);
    return o;
  };
  const size_t hd = a.head_dim, sp = D.seq_pad, B = batch;
  D.q = take(B * a.n_heads * sp * hd * 2);
  D.k = take(B * a.n_kv_heads * sp * hd * 2);
  D.vt = take(B * a.n_kv_heads * hd * sp * 2);
  D.o = take(T * a.n_heads * hd * 2);
  D.rope = take(static_cast<size_t>(seq) * (hd / 2) * 8);
  if (n_layers > 0) {
    const size_t hb = T * d.d * 2;
    D.ring = take(3 * hb);
    D.hA = take(hb);
    D.hB = take(hb);
    D.hbar_tmp = take(hb);
  }
  D.total = off;
  return D;
}

// hbar = h + Attn(LN^attn(h)) over batch x seq tokens
// the rotary table of the call's positions, made once per call
int make_rope_table(int seq, const hero::RopeTable& rope, unsigned char* ws, const DecLayout& DL, hipStream_t st) {
  return hero::launch_rope_table(seq, rope, reinterpret_cast<float*>(ws + DL.rope), st) == hipSuccess
             ? HERO_OK : HERO_E_LAUNCH;
}

// hbar = h + Attn(LN^attn(h)) over batch x seq tokens (the rotary table already made)
int run_attention(const hero_dims& dm, const hero_attn_dims& a, int batch, int seq, const void* h, void* hbar,
                  const hero_attn_weights& w, unsigned char* ws, const DecLayout& DL, hipStream_t st) {
  using namespace hero;
  const int T = batch * seq;
  void* x = ws + DL.L.u;
  float* rowstat = reinterpret_cast<float*>(ws + DL.L.rowstat);
  void *q = ws + DL.q, *k = ws + DL.k, *vt = ws + DL.vt, *o = ws + DL.o;
  hipError_t e = timed(HERO_K_ATTN_NORM, st, [&] {
    return launch_rowstats(dm.dtype, h, nullptr, nullptr, w.norm_w, T, dm.d, 1, dm.eps_norm, rowstat, x, st);
  });
  if (e != hipSuccess) return HERO_E_LAUNCH;
  e = timed(HERO_K_ATTN_QKV, st, [&] {
    return launch_attn_qkv(x, w.w_qkv, T, dm.d, seq, DL.seq_pad, a.n_heads, a.n_kv_heads,
                           reinterpret_cast<const float*>(ws + DL.rope), q, k, vt, st);
  });
  if (e != hipSuccess) return HERO_E_LAUNCH;
  e = timed(HERO_K_ATTN_CORE, st, [&] {
    return launch_attn_core(q, k, vt, o, batch, seq, DL.seq_pad, a.n_heads, a.n_kv_heads, st);
  });
  if (e != hipSuccess) return HERO_E_LAUNCH;
  e = timed(HERO_K_ATTN_OUT, st, [&] {
    return launch_attn_out(o, w.w_o, h, hbar, T, dm.d, a.n_heads, st);
  });
  return e == hipSuccess ? HERO_OK : HERO_E_LAUNCH;
}

// The pretrained FFN of a non-routed block: h = hbar + FFN(LN^ffn(hbar)), every token
int run_dense_ffn(const hero_dims& dm, int T, const void* hbar, void* h, const hero_ffn_weights& f,
                  unsigned char* ws, const Layout& L, hipStream_t st) {
  using namespace hero;
  void* u = ws + L.u;
  void* act = ws + L.act;
  float* part = reinterpret_cast<float*>(ws + L.part);
  float* rowstat = reinterpret_cast<float*>(ws + L.rowstat);
  hipError_t e = timed(HERO_K_ROWSTATS, st, [&] {
    return launch_rowstats(dm.dtype, hbar, nullptr, nullptr, f.norm_w, T, dm.d, 1, dm.eps_norm, rowstat, u, st);
  });
  if (e != hipSuccess) return HERO_E_LAUNCH;
  e = timed(HERO_K_FFN_GATE_UP, st, [&] {
    return launch_ffn_gateup(dm.dtype, u, nullptr, nullptr, T, f.w_gate, f.w_up, f.w_gate_up_tiled, act, part,
                             dm.d, dm.d_ff, st);
  });
  if (e != hipSuccess) return HERO_E_LAUNCH;
  e = timed(HERO_K_FFN_DOWN, st, [&] {
    return launch_ffn_down(dm.dtype, act, nullptr, nullptr, T, f.w_down, f.w_down_tiled, hbar, nullptr, h, part,
                           dm.d, dm.d_ff, st);
  });
  return e == hipSuccess ? HERO_OK : HERO_E_LAUNCH;
}

}  // namespace

int hero_decoder_workspace_size(const hero_dims* dims, const hero_attn_dims* adims, int n_layers, int batch,
                                int seq, size_t* bytes) {
  if (!bytes) return HERO_E_NULL;
  int st = check_dims(dims);
  if (st != HERO_OK) return st;
  if ((st = check_attn_dims(dims, adims)) != HERO_OK) return st;
  if (n_layers < 0) return HERO_E_DIM;
  if ((st = check_dec_size(*dims, *adims, batch, seq)) != HERO_OK) return st;
  *bytes = dec_layout_of(*dims, *adims, n_layers, batch, seq).total;
  return HERO_OK;
}

int hero_attention_block(const hero_dims* dims, const hero_attn_dims* adims, int batch, int seq, const void* h,
                         void* hbar, const hero_attn_weights* attn, const float* inv_freq, void* workspace,
                         size_t workspace_bytes, void* stream) {
  int st = check_dims(dims);
  if (st != HERO_OK) return st;
  if ((st = check_attn_dims(dims, adims)) != HERO_OK) return st;
  if ((st = check_dec_size(*dims, *adims, batch, seq)) != HERO_OK) return st;
  if (!h || !hbar) return HERO_E_NULL;
  if (!aligned16(h) || !aligned16(hbar)) return HERO_E_ALIGN;
  if ((st = check_attn_weights(attn)) != HERO_OK) return st;
  hero::RopeTable rope{};
  if ((st = check_rope(inv_freq, adims->head_dim, &rope)) != HERO_OK) return st;
  const size_t hb = static_cast<size_t>(batch) * seq * dims->d * 2;
  if (overlap(h, hb, hbar, hb)) return HERO_E_ALIAS;
  const DecLayout DL = dec_layout_of(*dims, *adims, 0, batch, seq);
  if (!workspace || workspace_bytes < DL.total) return HERO_E_WORKSPACE;
  if (!aligned16(workspace)) return HERO_E_ALIGN;
  if (overlap(hbar, hb, workspace, DL.total) || overlap(h, hb, workspace, DL.total)) return HERO_E_ALIAS;
  if ((st = check_device()) != HERO_OK) return st;
  unsigned char* ws = static_cast<unsigned char*>(workspace);
  const hipStream_t s = static_cast<hipStream_t>(stream);
  if ((st = make_rope_table(seq, rope, ws, DL, s)) != HERO_OK) return st;
  return run_attention(*dims, *adims, batch, seq, h, hbar, *attn, ws, DL, s);
}

int hero_decoder_stack(const hero_dims* dims, const hero_attn_dims* adims, int n_layers, int batch, int seq,
                       const void* h_in, void* h_out, const hero_state* state, const hero_attn_weights* attn,
                       const hero_ffn_weights* ffn, const hero_router_weights* router,
                       const hero_adapter_weights* adapter, const float* eta, const float* inv_freq,
                       const hero_routing* routing, const hero_layer_stats* stats, void* workspace,
                       size_t workspace_bytes, void* stream) {
  int st = check_dims(dims);
  if (st != HERO_OK) return st;
  if ((st = check_attn_dims(dims, adims)) != HERO_OK) return st;
  if ((st = check_dec_size(*dims, *adims, batch, seq)) != HERO_OK) return st;
  if (n_layers < dims->L_R) return HERO_E_RANGE;
  if (!h_in || !h_out || !attn || !ffn || !adapter || !eta || !router) return HERO_E_NULL;
  if (!aligned16(h_in) || !aligned16(h_out)) return HERO_E_ALIGN;
  if ((st = check_state(state)) != HERO_OK) return st;
  if ((st = check_routing(routing)) != HERO_OK) return st;
  hero::RopeTable rope{};
  if ((st = check_rope(inv_freq, adims->head_dim, &rope)) != HERO_OK) return st;
  const int first = n_layers - dims->L_R;   // index of the first routed block
  for (int l = 0; l < n_layers; ++l) {
    if ((st = check_attn_weights(&attn[l])) != HERO_OK) return st;
    if (l < first) {
      if (!ffn[l].norm_w || !ffn[l].w_gate || !ffn[l].w_up || !ffn[l].w_down) return HERO_E_NULL;
      if (!aligned16(ffn[l].norm_w) || !aligned16(ffn[l].w_gate) || !aligned16(ffn[l].w_up) ||
          !aligned16(ffn[l].w_down))
        return HERO_E_ALIGN;
      if ((st = check_ffn_tiled(*dims, &ffn[l])) != HERO_OK) return st;
    } else {
      const int j = l - first;
      if ((st = check_weights(&ffn[l], router, &adapter[j])) != HERO_OK) return st;
      if ((st = check_ffn_tiled(*dims, &ffn[l])) != HERO_OK) return st;
      if (!(eta[j] == eta[j])) return HERO_E_RANGE;
      if (stats && (st = check_stats(&stats[j])) != HERO_OK) return st;
    }
  }
  const int T = batch * seq;
  const size_t hb = static_cast<size_t>(T) * dims->d * 2;
  if (overlap(h_out, hb, h_in, hb)) return HERO_E_ALIAS;
  const DecLayout DL = dec_layout_of(*dims, *adims, n_layers, batch, seq);
  if (!workspace || workspace_bytes < DL.total) return HERO_E_WORKSPACE;
  if (!aligned16(workspace)) return HERO_E_ALIGN;
  if (overlap(h_out, hb, workspace, DL.total) || overlap(h_in, hb, workspace, DL.total)) return HERO_E_ALIAS;
  if ((st = check_device()) != HERO_OK) return st;

  unsigned char* ws = static_cast<unsigned char*>(workspace);
  const hipStream_t s = static_cast<hipStream_t>(stream);
  unsigned char* ring[3] = {ws + DL.ring, ws + DL.ring + hb, ws + DL.ring + 2 * hb};
  unsigned char* hbuf[2] = {ws + DL.hA, ws + DL.hB};
  if ((st = make_rope_table(seq, rope, ws, DL, s)) != HERO_OK) return st;
  const void* h = h_in;
  for (int l = 0; l < n_layers; ++l) {
    void* out = l == n_layers - 1 ? h_out : static_cast<void*>(hbuf[l & 1]);
    if (l < first) {
      void* hbar = ws + DL.hbar_tmp;
      if ((st = run_attention(*dims, *adims, batch, seq, h, hbar, attn[l], ws, DL, s)) != HERO_OK) return st;
      if ((st = run_dense_ffn(*dims, T, hbar, out, ffn[l], ws, DL.L, s)) != HERO_OK) return st;
    } else {
      const int j = l - first + 1;
      void* hbar = ring[(j - 1) % 3];
      if ((st = run_attention(*dims, *adims, batch, seq, h, hbar, attn[l], ws, DL, s)) != HERO_OK) return st;
      LayerCall c{dims, j, T, hbar, j >= 2 ? ring[(j - 2) % 3] : nullptr, j >= 3 ? ring[(j - 3) % 3] : nullptr,
                  out, state, &ffn[l], router, &adapter[j - 1], eta[j - 1], routing,
                  stats ? &stats[j - 1] : nullptr, ws, &DL.L, s};
      c.side = side_of_current_device();
      if ((st = run_layer(c)) != HERO_OK) return st;
    }
    h = out;
  }
  return HERO_OK;
}

// ---------------------------------------------------------------------------
// Training side: backward of the routed block, the utilisation penalty
// ---------------------------------------------------------------------------
namespace {

// partials of the adapter weight gradients: the adapter rows split up to 8 ways, in chunks of at
// least 32 rows
int wgrad_slices(int T) { return std::max(1, std::min(8, T / 32)); }

// the adapter rank as the K of the du product: whole 64-deep k-tiles on the MFMA path
int rank_pad(const hero_dims& d) { return d.dtype == HERO_BF16 ? (d.d_r + 63) / 64 * 64 : d.d_r; }

// wide adapter ranks (bf16, above 128): the weight gradients run on the GEMM core over
// tokens-contiguous copies of the adapter rows
bool wgrad_wide(const hero_dims& d) { return d.dtype == HERO_BF16 && d.d_r > 128; }
int wgrad_kp(int n) { return std::max(64, (n + 63) / 64 * 64); }

struct BwdLayout {
  size_t idx_f, idx_a, counts, rowstat, u, e, dgu, dgpart, du_f, du_a, part_z, part_e, dz32, a32, dzk, dg_ad,
      w1t, w2t, pw1, pw2, uaT, dyT, dzT, aT, total;
  int n_parts, n_slices, rpad;
};

BwdLayout bwd_layout_of(const hero_dims& d, int T) {
  const size_t es = esize(d.dtype), t = static_cast<size_t>(T);
  BwdLayout L{};
  L.n_parts = hero::swiglu_bwd_parts(d.dtype, d.d_ff);
  L.n_slices = wgrad_slices(T);
  L.rpad = rank_pad(d);
  const size_t n_chunks = L.n_slices;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t o = off;
    off = align_up(off + bytes);
    return o;
  };
  L.idx_f = take(t * 4);
  L.idx_a = take(t * 4);
  L.counts = take(16);
  L.rowstat = take(t * 16);
  L.u = take(t * d.d * es);
  L.e = take(t * d.d_ff * es);
  L.dgu = take(t * 2 * d.d_ff * es);
  L.dgpart = take(t * L.n_parts * 4);
  L.du_f = take(t * d.d * 4);
  L.du_a = take(t * d.d * 4);
  L.part_z = take(hero::adapter_part_floats(d.dtype, d.d, d.d_r, T) * 4);
  L.part_e = take(hero::adapter_part_floats(d.dtype, d.d, d.d_r, T) * 4);
  L.dz32 = take(t * d.d_r * 4);
  L.a32 = take(t * d.d_r * 4);
  L.dzk = take(t * L.rpad * es);
  L.dg_ad = take(t * 4);
  L.w1t = take(static_cast<size_t>(d.d) * L.rpad * es);
  L.w2t = take(static_cast<size_t>(d.d_r) * d.d * es);
  const bool wide = wgrad_wide(d);
  const size_t kp = static_cast<size_t>(wgrad_kp(T));
  L.pw1 = take(wide ? 0 : n_chunks * d.d_r * d.d * 4);
  L.pw2 = take(wide ? 0 : n_chunks * d.d_r * d.d * 4);
  L.uaT = take(wide ? kp * d.d * 2 : 0);
  L.dyT = take(wide ? kp * d.d * 2 : 0);
  L.dzT = take(wide ? kp * d.d_r * 2 : 0);
  L.aT = take(wide ? kp * d.d_r * 2 : 0);
  L.total = off;
  return L;
}

// the GEMM core addresses operand rows with 32-bit byte offsets
bool bwd_fits(const hero_dims& d, int T) {
  const size_t es = esize(d.dtype);
  return static_cast<size_t>(T) * 2 * d.d_ff * es < (static_cast<size_t>(1) << 32) &&
         static_cast<size_t>(d.d_ff) * d.d * es < (static_cast<size_t>(1) << 32) &&
         static_cast<size_t>(T) * d.d * es < (static_cast<size_t>(1) << 32);
}

int check_ffn(const hero_ffn_weights* f) {
  if (!f || !f->norm_w || !f->w_gate || !f->w_up || !f->w_down) return HERO_E_NULL;
  if (!aligned16(f->norm_w) || !aligned16(f->w_gate) || !aligned16(f->w_up) || !aligned16(f->w_down))
    return HERO_E_ALIGN;
  return HERO_OK;
}

int check_adapter(const hero_adapter_weights* a) {
  if (!a || !a->w1 || !a->w2) return HERO_E_NULL;
  if (!aligned16(a->w1) || !aligned16(a->w2)) return HERO_E_ALIGN;
  return HERO_OK;
}

}  // namespace

int hero_ffn_backward_weights_make(const hero_dims* dims, const hero_ffn_weights* ffn, void* w_down_t,
                                   void* w_gate_up_t, void* stream) {
  int st = check_dims(dims);
  if (st != HERO_OK) return st;
  if ((st = check_ffn(ffn)) != HERO_OK) return st;
  if (!w_down_t || !w_gate_up_t) return HERO_E_NULL;
  if (!aligned16(w_down_t) || !aligned16(w_gate_up_t)) return HERO_E_ALIGN;
  const size_t wb = static_cast<size_t>(dims->d) * dims->d_ff * esize(dims->dtype);
  const void* in[] = {ffn->w_gate, ffn->w_up, ffn->w_down};
  for (const void* p : in)
    if (overlap(w_down_t, wb, p, wb) || overlap(w_gate_up_t, 2 * wb, p, wb)) return HERO_E_ALIAS;
  if (overlap(w_down_t, wb, w_gate_up_t, 2 * wb)) return HERO_E_ALIAS;
  if ((st = check_device()) != HERO_OK) return st;
  const hipStream_t s = static_cast<hipStream_t>(stream);
  const int d = dims->d, f = dims->d_ff, dt = dims->dtype;
  unsigned char* gu = static_cast<unsigned char*>(w_gate_up_t);
  hipError_t e = hero::launch_transpose(dt, ffn->w_down, d, f, f, w_down_t, d, d, s);
  if (e == hipSuccess) e = hero::launch_transpose(dt, ffn->w_gate, f, d, d, gu, 2 * f, f, s);
  if (e == hipSuccess) e = hero::launch_transpose(dt, ffn->w_up, f, d, d, gu + f * esize(dt), 2 * f, f, s);
  return e == hipSuccess ? HERO_OK : HERO_E_LAUNCH;
}

int hero_ffn_decode_weights_make(const hero_dims* dims, const hero_ffn_weights* ffn, void* w_gate_up_tiled,
                                 void* w_down_tiled, void* stream) {
  int st = check_dims(dims);
  if (st != HERO_OK) return st;
  if ((st = check_ffn(ffn)) != HERO_OK) return st;
  if (dims->dtype != HERO_BF16 || dims->d_ff % 64 != 0) return HERO_E_UNSUPPORTED;
  if ((w_gate_up_tiled && !aligned16(w_gate_up_tiled)) || (w_down_tiled && !aligned16(w_down_tiled)))
    return HERO_E_ALIGN;
  const size_t wb = static_cast<size_t>(dims->d) * dims->d_ff * 2;
  const void* in[] = {ffn->w_gate, ffn->w_up, ffn->w_down};
  for (const void* p : in)
    if ((w_gate_up_tiled && overlap(w_gate_up_tiled, 2 * wb, p, wb)) || (w_down_tiled && overlap(w_down_tiled, wb, p, wb)))
      return HERO_E_ALIAS;
  if (w_gate_up_tiled && w_down_tiled && overlap(w_gate_up_tiled, 2 * wb, w_down_tiled, wb)) return HERO_E_ALIAS;
  if ((st = check_device()) != HERO_OK) return st;
  const hipStream_t s = static_cast<hipStream_t>(stream);
  hipError_t e = hipSuccess;
  if (w_gate_up_tiled)
    e = hero::launch_tile_ffn_weights(ffn->w_gate, ffn->w_up, dims->d_ff, dims->d, w_gate_up_tiled, s);
  if (e == hipSuccess && w_down_tiled)
    e = hero::launch_tile_ffn_weights(ffn->w_down, nullptr, dims->d, dims->d_ff, w_down_tiled, s);
  return e == hipSuccess ? HERO_OK : HERO_E_LAUNCH;
}

int hero_backward_workspace_size(const hero_dims* dims, int T, size_t* bytes) {
  if (!bytes) return HERO_E_NULL;
  const int st = check_dims(dims);
  if (st != HERO_OK) return st;
  if (T <= 0) return HERO_E_DIM;
  *bytes = bwd_layout_of(*dims, T).total;
  return HERO_OK;
}

int hero_routed_block_backward(const hero_dims* dims, int T, const void* hbar, const void* dh_out,
                               const float* gate, const int32_t* idx_ffn, const int32_t* idx_ad,
                               const int32_t* counts, const hero_routing* routing, const float* dgate_in,
                               const hero_ffn_weights* ffn, const hero_ffn_backward_weights* ffn_t,
                               const hero_adapter_weights* adapter, const hero_block_grads* grads, void* workspace,
                               size_t workspace_bytes, void* stream) {
  using namespace hero;
  int st = check_dims(dims);
  if (st != HERO_OK) return st;
  if (T <= 0) return HERO_E_DIM;
  if (!bwd_fits(*dims, T)) return HERO_E_UNSUPPORTED;
  if (!hbar || !dh_out || !gate || !idx_ffn || !idx_ad || !counts || !ffn_t || !grads) return HERO_E_NULL;
  if (!ffn_t->w_down_t || !ffn_t->w_gate_up_t || !grads->dhbar || !grads->dgate || !grads->dlogit ||
      !grads->dw1 || !grads->dw2)
    return HERO_E_NULL;
  if ((st = check_ffn(ffn)) != HERO_OK) return st;
  if ((st = check_adapter(adapter)) != HERO_OK) return st;
  if (routing && (st = check_routing(routing)) != HERO_OK) return st;
  const void* al[] = {hbar, dh_out, gate, idx_ffn, idx_ad, counts, dgate_in, ffn_t->w_down_t, ffn_t->w_gate_up_t,
                      grads->dhbar, grads->dgate, grads->dlogit, grads->dw1, grads->dw2, workspace};
  for (const void* p : al)
    if (p && !aligned16(p)) return HERO_E_ALIGN;
  const size_t hb = static_cast<size_t>(T) * dims->d * esize(dims->dtype);
  if (overlap(grads->dhbar, hb, hbar, hb) || overlap(grads->dhbar, hb, dh_out, hb)) return HERO_E_ALIAS;
  const BwdLayout L = bwd_layout_of(*dims, T);
  if (!workspace || workspace_bytes < L.total) return HERO_E_WORKSPACE;
  const size_t tb = static_cast<size_t>(T) * 4, wb = static_cast<size_t>(dims->d) * dims->d_r * 4;
  if (overlap(workspace, L.total, hbar, hb) || overlap(workspace, L.total, dh_out, hb) ||
      overlap(workspace, L.total, grads->dhbar, hb) || overlap(workspace, L.total, grads->dgate, tb) ||
      overlap(workspace, L.total, grads->dlogit, tb) || overlap(workspace, L.total, grads->dw1, wb) ||
      overlap(workspace, L.total, grads->dw2, wb) || overlap(grads->dw1, wb, grads->dw2, wb))
    return HERO_E_ALIAS;
  if ((st = check_device()) != HERO_OK) return st;

  const hero_dims& D = *dims;
  const hipStream_t s = static_cast<hipStream_t>(stream);
  unsigned char* ws = static_cast<unsigned char*>(workspace);
  BlockBwdArgs a{};
  a.dtype = D.dtype;
  a.T = T;
  a.d = D.d;
  a.d_r = D.d_r;
  a.rpad = L.rpad;
  a.dh = dh_out;
  a.hbar = hbar;
  a.norm_w = ffn->norm_w;
  a.rowstat = reinterpret_cast<float*>(ws + L.rowstat);
  int* idx_f = reinterpret_cast<int*>(ws + L.idx_f);
  int* idx_a = reinterpret_cast<int*>(ws + L.idx_a);
  int* cnt = reinterpret_cast<int*>(ws + L.counts);
  a.idx_ffn = idx_f;
  a.idx_ad = idx_a;
  a.counts = cnt;
  a.gate = gate;
  a.dgate_in = dgate_in;
  a.du_f = reinterpret_cast<float*>(ws + L.du_f);
  a.du_a = reinterpret_cast<float*>(ws + L.du_a);
  a.dgpart = reinterpret_cast<float*>(ws + L.dgpart);
  a.n_parts = L.n_parts;
  a.dg_ad = reinterpret_cast<float*>(ws + L.dg_ad);
  a.part_z = reinterpret_cast<float*>(ws + L.part_z);
  a.part_e = reinterpret_cast<float*>(ws + L.part_e);
  a.splits = adapter_proj_splits(D.dtype, D.d, D.d_r);
  a.dz32 = reinterpret_cast<float*>(ws + L.dz32);
  a.a32 = reinterpret_cast<float*>(ws + L.a32);
  a.dzk = ws + L.dzk;
  a.u = ws + L.u;
  a.n_slices = L.n_slices;
  a.pw1 = reinterpret_cast<float*>(ws + L.pw1);
  a.pw2 = reinterpret_cast<float*>(ws + L.pw2);
  a.dhbar = grads->dhbar;
  a.dgate = grads->dgate;
  a.dlogit = grads->dlogit;
  a.dw1 = grads->dw1;
  a.dw2 = grads->dw2;
  void* u = ws + L.u;
  void* e = ws + L.e;
  void* dgu = ws + L.dgu;
  void* w1t = ws + L.w1t;
  void* w2t = ws + L.w2t;

  // launch sizes: exact in budget mode, T otherwise (tiles past the device count exit)
  const bool budget = routing && routing->mode == HERO_MODE_BUDGET;
  const int n_skip = budget ? static_cast<int>(floor(routing->budget * static_cast<double>(T) + 0.5)) : 0;
  const int nf_max = budget ? T - n_skip : T;
  const int na_max = budget ? n_skip : T;
  a.na_max = na_max;
  hipError_t err = timed(HERO_K_BWD_NORM, s, [&] {
    hipError_t x = launch_bwd_lists(T, nf_max, na_max, idx_ffn, idx_ad, counts, idx_f, idx_a, cnt, s);
    if (x != hipSuccess) return x;
    return launch_rowstats(D.dtype, hbar, nullptr, nullptr, ffn->norm_w, T, D.d, 1, D.eps_norm,
                           const_cast<float*>(a.rowstat), u, s);
  });
  if (err != hipSuccess) return HERO_E_LAUNCH;
  err = timed(HERO_K_BWD_FFN_E, s, [&] {
    return launch_ffn_bwd_e(D.dtype, dh_out, idx_f, cnt, nf_max, ffn_t->w_down_t, e, D.d, D.d_ff, s);
  });
  if (err != hipSuccess) return HERO_E_LAUNCH;
  err = timed(HERO_K_BWD_FFN_GATE_UP, s, [&] {
    return launch_ffn_bwd_gateup(D.dtype, u, idx_f, cnt, nf_max, ffn->w_gate, ffn->w_up, e, gate, dgu,
                                 const_cast<float*>(a.dgpart), D.d, D.d_ff, s);
  });
  if (err != hipSuccess) return HERO_E_LAUNCH;
  err = timed(HERO_K_BWD_FFN_DU, s, [&] {
    return launch_ffn_bwd_du(D.dtype, dgu, cnt, nf_max, ffn_t->w_gate_up_t, const_cast<float*>(a.du_f), D.d,
                             D.d_ff, s);
  });
  if (err != hipSuccess) return HERO_E_LAUNCH;
  err = timed(HERO_K_BWD_ADAPTER, s, [&] {
    hipError_t x = launch_adapter_transpose(D.dtype, adapter->w1, adapter->w2, w1t, w2t, D.d, D.d_r, L.rpad, s);
    if (x == hipSuccess)
      x = launch_adapter_proj2(D.dtype, u, adapter->w1, const_cast<float*>(a.part_z), dh_out, w2t,
                               const_cast<float*>(a.part_e), idx_a, cnt + 1, na_max, D.d, D.d_r, s);
    if (x == hipSuccess) x = launch_adapter_bwd_mid(a, s);
    if (x == hipSuccess)
      x = launch_adapter_du(D.dtype, a.dzk, cnt + 1, na_max, w1t, const_cast<float*>(a.du_a), D.d, L.rpad, s);
    return x;
  });
  if (err != hipSuccess) return HERO_E_LAUNCH;
  err = timed(HERO_K_BWD_ADAPTER_WGRAD, s, [&] {
    if (!wgrad_wide(D)) return launch_adapter_wgrad(a, s);
    // dW_1 = dz^T u, dW_2 = dy^T a with the adapter tokens as K (zero columns pad it to kp)
    const int kp = wgrad_kp(na_max);
    hipError_t x = launch_adapter_wgrad_stage(a, kp, ws + L.uaT, ws + L.dyT, ws + L.dzT, ws + L.aT, s);
    if (x == hipSuccess) x = launch_gemm_nt_f32(ws + L.dzT, D.d_r, ws + L.uaT, D.d, kp, grads->dw1, D.d, s);
    if (x == hipSuccess) x = launch_gemm_nt_f32(ws + L.dyT, D.d, ws + L.aT, D.d_r, kp, grads->dw2, D.d_r, s);
    return x;
  });
  if (err != hipSuccess) return HERO_E_LAUNCH;
  err = timed(HERO_K_BWD_ROWS, s, [&] { return launch_block_bwd_rows(a, s); });
  return err == hipSuccess ? HERO_OK : HERO_E_LAUNCH;
}

int hero_skip_penalty(int L_R, int batch, int seq, const float* gates, float alpha, float* loss, float* dgates,
                      void* stream) {
  if (L_R <= 0 || batch <= 0 || seq <= 0) return HERO_E_DIM;
  if (static_cast<long long>(batch) * seq > INT_MAX) return HERO_E_DIM;
  if (!(alpha - alpha == 0.f)) return HERO_E_RANGE;
  if (!gates || !loss || !dgates) return HERO_E_NULL;
  if (!aligned16(gates) || !aligned16(loss) || !aligned16(dgates)) return HERO_E_ALIGN;
  const size_t gb = static_cast<size_t>(L_R) * batch * seq * 4;
  if (overlap(dgates, gb, gates, gb) || overlap(loss, 4, gates, gb) || overlap(loss, 4, dgates, gb))
    return HERO_E_ALIAS;
  int st = check_device();
  if (st != HERO_OK) return st;
  return timed(HERO_K_SKIP_PENALTY, static_cast<hipStream_t>(stream), [&] {
           return hero::launch_skip_penalty(gates, L_R, batch, seq, alpha, loss, dgates,
                                            static_cast<hipStream_t>(stream));
         }) == hipSuccess
             ? HERO_OK
             : HERO_E_LAUNCH;
}

// ---------------------------------------------------------------------------
// Backward of the router at one routed layer
// ---------------------------------------------------------------------------
namespace {

struct RouterBwdLayout {
  size_t P, dP, dPT, rowcoef, rho_part, vec, tok, hbT, wT;
  // bf16: the big products on the GEMM core, dP split into bf16 hi + lo, K padded to kp
  size_t dPT_hi, dPT_lo, dP_hi, dP_lo, hbT16, wT16;
  size_t tn_part, tn_floats;   // K-split partials of the fp32 path's large weight-gradient products
  size_t sp_part, sp_floats;   // chunk partials of the small weight-gradient products
  size_t wt;                   // bf16: the transposed router weights of the batched passes
  int kp;
  size_t total;
};

// the small weight-gradient products (tokens as K): dW_q, dW_k, dW_v, dW_n, dW_c, dth1, dth2, dpsi_2,
// dW_p1, dW_p2, dW_hu.  Pointers come from a (operands) and grads (outputs); either may be null when
// only the shapes are wanted.
int router_small_products(const hero_dims& D, const hero::RouterBwdArgs* a, const hero_router_grads* g,
                          hero::SmallProduct* out) {
  const int T = a ? a->T : 0, dx = D.d_s + D.d_m + 1, ld_th1 = HERO_TH1_PITCH(D.d_s, D.d_m);
  auto A = [&](float* hero::RouterBwdArgs::*f) -> const float* { return a ? a->*f : nullptr; };
  const float* xs = A(&hero::RouterBwdArgs::XT);
  const float* xc = xs ? xs + static_cast<size_t>(D.d_s) * T : nullptr;
  int n = 0;
  auto put = [&](const float* Ao, int M, const float* Bo, int N, float* C, int ldc) {
    out[n++] = hero::SmallProduct{Ao, Bo, C, M, N, ldc};
  };
  put(A(&hero::RouterBwdArgs::dQT), D.d_m, xs, D.d_s, g ? g->w_q : nullptr, D.d_s);
  put(A(&hero::RouterBwdArgs::dKT), D.d_m, xs, D.d_s, g ? g->w_k : nullptr, D.d_s);
  put(A(&hero::RouterBwdArgs::dVT), D.d_m, xs, D.d_s, g ? g->w_v : nullptr, D.d_s);
  put(A(&hero::RouterBwdArgs::dU1T), D.d_m, xs, D.d_s, g ? g->w_n : nullptr, D.d_s);
  put(A(&hero::RouterBwdArgs::dU2T), D.d_m, xc, D.d_m, g ? g->w_c : nullptr, D.d_m);
  put(A(&hero::RouterBwdArgs::dPAT), D.d_head, xs, dx, g ? g->th1 : nullptr, ld_th1);
  put(A(&hero::RouterBwdArgs::SAT), D.d_head, A(&hero::RouterBwdArgs::DA), 1, g ? g->th2 : nullptr, 1);
  put(A(&hero::RouterBwdArgs::SBT), D.d_head, A(&hero::RouterBwdArgs::DB), 1, g ? g->ps2 : nullptr, 1);
  put(A(&hero::RouterBwdArgs::dPPT), D.d_p, A(&hero::RouterBwdArgs::XPT), 6, g ? g->w_p1 : nullptr, 6);
  put(A(&hero::RouterBwdArgs::dZAT), D.d_a, A(&hero::RouterBwdArgs::SPT), D.d_p, g ? g->w_p2 : nullptr, D.d_p);
  put(A(&hero::RouterBwdArgs::dZHT), D.d_h, A(&hero::RouterBwdArgs::SHT), D.d_e, g ? g->w_hu : nullptr, D.d_e);
  return n;
}

RouterBwdLayout router_bwd_layout_of(const hero_dims& d, int T) {
  RouterBwdLayout L{};
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t at = off;
    off += (bytes + 255) & ~static_cast<size_t>(255);
    return at;
  };
  const size_t t = static_cast<size_t>(T), np = static_cast<size_t>(d.d_e + d.d_head);
  L.P = take(t * np * 4 * hero::router_gemm_splits(d.dtype, d.d, T, d.d_e + d.d_head));
  L.dP = take(t * np * 4);
  L.dPT = take(np * t * 4);
  L.rowcoef = take(t * 8 * 4);
  L.rho_part = take(t * 4);
  L.vec = take(hero::router_bwd_vector_floats(d.d_m, d.d_s, d.d_h, d.d_a, d.d_e, d.d_p, d.d_head) * t * 4);
  L.tok = take(hero::router_bwd_token_floats(d.d_m, d.d_s, d.d_p, d.d_e + d.d_head) * t * 4);
  const bool mfma = d.dtype == HERO_BF16;
  L.kp = (T + 63) / 64 * 64;
  const size_t kp = static_cast<size_t>(L.kp);
  L.hbT = take(mfma ? 0 : static_cast<size_t>(d.d) * t * 4);
  L.wT = take(mfma ? 0 : static_cast<size_t>(d.d) * np * 4);
  L.dPT_hi = take(mfma ? np * kp * 2 : 0);
  L.dPT_lo = take(mfma ? np * kp * 2 : 0);
  L.dP_hi = take(mfma ? t * np * 2 : 0);
  L.dP_lo = take(mfma ? t * np * 2 : 0);
  L.hbT16 = take(mfma ? static_cast<size_t>(d.d) * kp * 2 : 0);
  L.wT16 = take(mfma ? static_cast<size_t>(d.d) * np * 2 : 0);
  // K chunks for fp32 storage's dW_hd and dpsi_1 (bf16 runs them on the GEMM core): up to one per 64
  // tokens, at most 16 M floats (64 MB) of partials
  const size_t mn = static_cast<size_t>(std::max(d.d_e, d.d_head)) * d.d;
  L.tn_floats = mfma ? 0 : std::min(static_cast<size_t>(hero::tn_chunks(T)) * mn, std::max<size_t>(mn, 16u << 20));
  L.tn_part = take(L.tn_floats * 4);
  hero::SmallProduct sp[hero::kSmallProducts];
  const int nsp = router_small_products(d, nullptr, nullptr, sp);
  L.sp_floats = hero::small_products_floats(sp, nsp, T);
  L.sp_part = take(L.sp_floats * 4);
  L.wt = take(mfma ? hero::router_bwd_wt_elems(d.d_m, d.d_s, d.d_h, d.d_a, d.d_e, d.d_p, d.d_head) * 2 : 0);
  L.total = off;
  return L;
}

int check_router(const hero_router_weights* r) {
  if (!r) return HERO_E_NULL;
  const void* p[] = {r->w_hd, r->w_hu, r->w_p1, r->w_p2, r->w_q, r->w_k, r->w_v,
                     r->w_n, r->w_c, r->th1, r->th2, r->ps1, r->ps2};
  for (const void* x : p)
    if (!x) return HERO_E_NULL;
  for (const void* x : p)
    if (!aligned16(x)) return HERO_E_ALIGN;
  return HERO_OK;
}

}  // namespace

int hero_router_backward_workspace_size(const hero_dims* dims, int T, size_t* bytes) {
  if (!bytes) return HERO_E_NULL;
  const int st = check_dims(dims);
  if (st != HERO_OK) return st;
  if (T <= 0) return HERO_E_DIM;
  *bytes = router_bwd_layout_of(*dims, T).total;
  return HERO_OK;
}

int hero_router_backward(const hero_dims* dims, int j, int T, const void* hbar, const void* hbar_prev1,
                         const void* hbar_prev2, const hero_state* state_in, const hero_router_weights* router,
                         float eta, const float* dlogit, const hero_router_carry* carry, float* dhbar,
                         float* dhbar_prev1, float* dhbar_prev2, const hero_router_grads* grads, float* deta,
                         void* workspace, size_t workspace_bytes, void* stream) {
  int st = check_dims(dims);
  if (st != HERO_OK) return st;
  if (T <= 0) return HERO_E_DIM;
  if (j < 1 || j > dims->L_R) return HERO_E_RANGE;
  if (dims->state_dtype != HERO_F32 || !fwd_fits(*dims, T)) return HERO_E_UNSUPPORTED;
  if (!(eta == eta)) return HERO_E_RANGE;
  if (!hbar || !dlogit || !carry || !dhbar || !grads || !deta) return HERO_E_NULL;
  if ((j >= 2 && (!hbar_prev1 || !dhbar_prev1)) || (j >= 3 && (!hbar_prev2 || !dhbar_prev2))) return HERO_E_NULL;
  if ((j > 1 || state_in) && (st = check_state(state_in)) != HERO_OK) return st;   // not read at j = 1
  if ((st = check_router(router)) != HERO_OK) return st;
  const float* gp[] = {grads->w_hd, grads->w_hu, grads->w_p1, grads->w_p2, grads->w_q, grads->w_k, grads->w_v,
                       grads->w_n, grads->w_c, grads->th1, grads->th2, grads->ps1, grads->ps2};
  for (const float* x : gp)
    if (!x) return HERO_E_NULL;
  if (!carry->dS || !carry->dzeta || !carry->dp || !carry->dm) return HERO_E_NULL;
  const void* al[] = {hbar, j >= 2 ? hbar_prev1 : nullptr, j >= 3 ? hbar_prev2 : nullptr, dlogit, carry->dS,
                      carry->dzeta, carry->dp, carry->dm, dhbar, j >= 2 ? dhbar_prev1 : nullptr,
                      j >= 3 ? dhbar_prev2 : nullptr, deta, workspace};
  for (const void* x : al)
    if (x && !aligned16(x)) return HERO_E_ALIGN;
  for (const float* x : gp)
    if (!aligned16(x)) return HERO_E_ALIGN;
  const hero_dims& D = *dims;
  const size_t t = static_cast<size_t>(T), dm = static_cast<size_t>(D.d_m);
  const size_t hb = t * D.d * 4, sb = t * dm * dm * 4, zb = t * dm * 4, tb = t * 4;
  float* outs[] = {dhbar, j >= 2 ? dhbar_prev1 : nullptr, j >= 3 ? dhbar_prev2 : nullptr};
  for (int a = 0; a < 3; ++a)
    for (int b = a + 1; b < 3; ++b)
      if (overlap(outs[a], hb, outs[b], hb)) return HERO_E_ALIAS;
  // the memory pass reads S_{j-1} while it writes dL/dS_{j-1} over dL/dS_j
  if (j > 1 && (overlap(carry->dS, sb, state_in->S, sb) || overlap(carry->dzeta, zb, state_in->zeta, zb)))
    return HERO_E_ALIAS;
  const RouterBwdLayout L = router_bwd_layout_of(D, T);
  if (!workspace || workspace_bytes < L.total) return HERO_E_WORKSPACE;
  struct Span {
    const void* p;
    size_t bytes;
  };
  const Span written[] = {{carry->dS, sb}, {carry->dzeta, zb}, {carry->dp, tb}, {carry->dm, tb}, {dhbar, hb},
                          {j >= 2 ? dhbar_prev1 : nullptr, hb}, {j >= 3 ? dhbar_prev2 : nullptr, hb}, {deta, 4}};
  for (const Span& x : written)
    if (overlap(workspace, L.total, x.p, x.bytes)) return HERO_E_ALIAS;
  // the forward's memory read, when given, is read after several of these are written
  const float* c_in = j > 1 && state_in ? state_in->c_read : nullptr;
  if (c_in) {
    if (overlap(c_in, zb, workspace, L.total)) return HERO_E_ALIAS;
    for (const Span& x : written)
      if (overlap(c_in, zb, x.p, x.bytes)) return HERO_E_ALIAS;
  }
  if ((st = check_device()) != HERO_OK) return st;

  const hipStream_t s = static_cast<hipStream_t>(stream);
  unsigned char* ws = static_cast<unsigned char*>(workspace);
  const int NP = D.d_e + D.d_head, dx = D.d_s + D.d_m + 1, ld_th1 = HERO_TH1_PITCH(D.d_s, D.d_m);
  hero::RouterBwdArgs a{};
  a.dtype = D.dtype;
  a.T = T;
  a.j = j;
  a.L_R = D.L_R;
  a.d = D.d;
  a.d_m = D.d_m;
  a.d_s = D.d_s;
  a.d_h = D.d_h;
  a.d_a = D.d_a;
  a.d_e = D.d_e;
  a.d_p = D.d_p;
  a.d_head = D.d_head;
  a.ld_th1 = ld_th1;
  a.eps_norm = D.eps_norm;
  a.eps = D.eps;
  a.T_hist = D.T_hist;
  a.rho = 1.0f / (1.0f + expf(-eta));
  a.hbar = hbar;
  a.prev1 = hbar_prev1;
  a.prev2 = hbar_prev2;
  a.P = reinterpret_cast<float*>(ws + L.P);
  a.p_splits = hero::router_gemm_splits(D.dtype, D.d, T, D.d_e + D.d_head);
  a.w_hu = router->w_hu;
  a.w_p1 = router->w_p1;
  a.w_p2 = router->w_p2;
  a.w_q = router->w_q;
  a.w_k = router->w_k;
  a.w_v = router->w_v;
  a.w_n = router->w_n;
  a.w_c = router->w_c;
  a.th1 = router->th1;
  a.th2 = router->th2;
  a.ps2 = router->ps2;
  a.S_in = state_in ? static_cast<const float*>(state_in->S) : nullptr;
  a.zeta_in = state_in ? state_in->zeta : nullptr;
  a.p_in = state_in ? state_in->p_hist : nullptr;
  a.m_in = state_in ? state_in->m_hist : nullptr;
  a.dlogit = dlogit;
  a.dS = carry->dS;
  a.dzeta = carry->dzeta;
  a.dp = carry->dp;
  a.dm = carry->dm;
  a.dP = reinterpret_cast<float*>(ws + L.dP);
  a.dPT = reinterpret_cast<float*>(ws + L.dPT);
  a.rowcoef = reinterpret_cast<float*>(ws + L.rowcoef);
  a.rho_part = reinterpret_cast<float*>(ws + L.rho_part);
  float* v = reinterpret_cast<float*>(ws + L.vec);
  auto rows = [&](int n) {
    float* at = v;
    v += static_cast<size_t>(n) * T;
    return at;
  };
  a.XT = rows(dx);
  a.dQT = rows(D.d_m);
  a.dKT = rows(D.d_m);
  a.dVT = rows(D.d_m);
  a.dU1T = rows(D.d_m);
  a.dU2T = rows(D.d_m);
  a.dPAT = rows(D.d_head);
  a.SAT = rows(D.d_head);
  a.DA = rows(1);
  a.DB = rows(1);
  a.SBT = rows(D.d_head);
  a.dPPT = rows(D.d_p);
  a.SPT = rows(D.d_p);
  a.XPT = rows(8);
  a.dZAT = rows(D.d_a);
  a.dZHT = rows(D.d_h);
  a.SHT = rows(D.d_e);
  float* tk = reinterpret_cast<float*>(ws + L.tok);
  auto per_token = [&](int n) {
    float* at = tk;
    tk += static_cast<size_t>(n) * T;
    return at;
  };
  a.RS = per_token(4);
  a.QKVU = per_token(4 * D.d_m);
  a.PPRE = per_token(D.d_p);
  a.Cv = per_token(D.d_m);
  a.DEN = per_token(1);
  a.PS = per_token(1);
  a.DSP = per_token(D.d_s);
  a.DNUM = per_token(D.d_m);
  a.DDEN = per_token(1);
  a.DF = per_token(3 * D.d_m);
  a.PSUM = per_token(NP);
  a.t_begin = 0;
  a.t_end = T;
  if (D.dtype == HERO_BF16) hero::router_bwd_wt_assign(a, reinterpret_cast<uint16_t*>(ws + L.wt));
  if (c_in) {
    a.Cv = const_cast<float*>(c_in);   // read only: the memory read pass is skipped
    a.c_given = 1;
  }
  a.dhbar = dhbar;
  a.dhbar1 = dhbar_prev1;
  a.dhbar2 = dhbar_prev2;
  a.deta = deta;
  float* hbT = reinterpret_cast<float*>(ws + L.hbT);
  float* wT = reinterpret_cast<float*>(ws + L.wT);

  hipError_t e = timed(HERO_K_ROUTER_BWD_GEMM, s, [&] {
    return hero::launch_router_gemm(D.dtype, hbar, router->w_hd, router->ps1, T, D.d, D.d_e, D.d_head,
                                     const_cast<float*>(a.P), s);
  });
  if (e == hipSuccess)
    e = timed(HERO_K_ROUTER_BWD_TOKEN, s, [&] {
      // one chain over all tokens (two halves on two streams, each half's batched passes beside the
      // other's state streams, measured 341 against 336 us at the 8B layer: the batched passes slow
      // down under the streams' memory traffic)
      hipError_t x = hero::launch_router_bwd_wt(a, s);
      if (x == hipSuccess) x = hero::launch_router_bwd_stats(a, s);
      return x == hipSuccess ? hero::launch_router_bwd_chain(a, s) : x;
    });
  if (e != hipSuccess) return HERO_E_LAUNCH;
  e = timed(HERO_K_ROUTER_BWD_PRODUCTS, s, [&] {
    // the weight gradients: products with the tokens as K (every operand token-contiguous)
    float* tn_part = reinterpret_cast<float*>(ws + L.tn_part);
    auto acc = [&](const float* A, int M, const float* B, int N, float* C, int ldc) {
      return hero::launch_gemm_tn_acc_f32(A, T, M, B, T, N, T, C, ldc, tn_part, L.tn_floats, s);
    };
    hipError_t x = hipSuccess;
    hero::SmallProduct sp[hero::kSmallProducts];
    const int nsp = router_small_products(D, &a, grads, sp);
    float* sp_part = reinterpret_cast<float*>(ws + L.sp_part);
    if (D.dtype == HERO_BF16) {
      // dW_hd, dpsi_1 = dP^T hbar and dL/dhbar_j += dP [W_hd; psi_1] on the GEMM core: hbar and the
      // weights are exact in bf16, dP enters as bf16 hi + lo (two accumulating products each).
      // dW_hd's pair (64 output tiles a product, a quarter of the CUs) and the small products run on
      // the side stream beside dpsi_1's pair and dL/dhbar's; their outputs are disjoint (measured:
      // 348 -> 261 us for the group at the 8B layer; dpsi_1's pair on the side too measured 298).
      const int kp = L.kp;
      unsigned char *ph = ws + L.dPT_hi, *pl = ws + L.dPT_lo, *qh = ws + L.dP_hi, *ql = ws + L.dP_lo;
      unsigned char *h16 = ws + L.hbT16, *w16 = ws + L.wT16;
      const size_t re = static_cast<size_t>(D.d_e) * kp * 2;
      const Side* sd = side_of_current_device();
      const hipStream_t s2 = sd ? sd->s : s;
      x = hero::launch_split_bf16(a.dPT, NP, T, T, ph, pl, kp, s);
      if (x == hipSuccess) x = hero::launch_transpose(D.dtype, hbar, T, D.d, D.d, h16, kp, kp, s);
      if (x == hipSuccess && sd) {
        x = hipEventRecord(sd->fork, s);
        if (x == hipSuccess) x = hipStreamWaitEvent(s2, sd->fork, 0);
      }
      for (unsigned char* part : {ph, pl})
        if (x == hipSuccess)
          x = hero::launch_gemm_nt_acc_bf16(part, kp, D.d_e, h16, kp, D.d, kp, grads->w_hd, D.d, s2);
      if (x == hipSuccess) x = hero::launch_small_products(sp, nsp, T, T, sp_part, L.sp_floats, s2);
      for (unsigned char* part : {ph, pl})
        if (x == hipSuccess)
          x = hero::launch_gemm_nt_acc_bf16(part + re, kp, D.d_head, h16, kp, D.d, kp, grads->ps1, D.d, s);
      if (x == hipSuccess) x = hero::launch_split_bf16(a.dP, T, NP, NP, qh, ql, NP, s);
      if (x == hipSuccess) x = hero::launch_transpose(D.dtype, router->w_hd, D.d_e, D.d, D.d, w16, NP, D.d_e, s);
      if (x == hipSuccess)
        x = hero::launch_transpose(D.dtype, router->ps1, D.d_head, D.d, D.d, w16 + static_cast<size_t>(D.d_e) * 2, NP,
                                   D.d_head, s);
      for (unsigned char* part : {qh, ql})
        if (x == hipSuccess) x = hero::launch_gemm_nt_acc_bf16(part, NP, T, w16, NP, D.d, NP, dhbar, D.d, s);
      if (sd) {
        // joined even after a failed launch, so that the side stream holds nothing of this call
        const hipError_t y = hipEventRecord(sd->join, s2);
        const hipError_t z = y == hipSuccess ? hipStreamWaitEvent(s, sd->join, 0) : y;
        if (x == hipSuccess) x = z;
      }
    } else {
      x = hero::launch_to_f32_transpose(D.dtype, hbar, T, D.d, D.d, hbT, T, s);
      if (x == hipSuccess) x = acc(a.dPT, D.d_e, hbT, D.d, grads->w_hd, D.d);
      if (x == hipSuccess) x = acc(a.dPT + static_cast<size_t>(D.d_e) * T, D.d_head, hbT, D.d, grads->ps1, D.d);
      if (x == hipSuccess) x = hero::launch_to_f32_transpose(D.dtype, router->w_hd, D.d_e, D.d, D.d, wT, NP, s);
      if (x == hipSuccess)
        x = hero::launch_to_f32_transpose(D.dtype, router->ps1, D.d_head, D.d, D.d, wT + D.d_e, NP, s);
      if (x == hipSuccess) x = hero::launch_gemm_acc_f32(a.dP, NP, T, wT, NP, D.d, NP, dhbar, D.d, s);
      if (x == hipSuccess) x = hero::launch_small_products(sp, nsp, T, T, sp_part, L.sp_floats, s);
    }
    return x;
  });
  if (e != hipSuccess) return HERO_E_LAUNCH;
  e = timed(HERO_K_ROUTER_BWD_ROWS, s, [&] { return hero::launch_router_bwd_rows(a, s); });
  return e == hipSuccess ? HERO_OK : HERO_E_LAUNCH;
}
