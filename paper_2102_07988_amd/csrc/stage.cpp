// Stage engine behind the C ABI of include/terapipe.h: workspace layout, the
// slice state machine (cached length / backward frontier), the per-layer
// launch sequences of a slice's forward and backward, the deferred
// weight-gradient pass, the slice-cost profiler and per-kernel timing.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstring>
#include <new>
#include <string>
#include <vector>

#include "tp_common.hpp"
#include "tp_kernels.hpp"

using namespace tp;

namespace tp {
void* static_scratch(size_t* bytes);  // static_scratch.hip
}

namespace {

struct LayerBufs {
  // per-token activation arena, rows are absolute token positions
  void *x_in, *u, *q, *kc, *vc, *o, *x1, *u2, *z, *g;
  float *mean1, *rstd1, *mean2, *rstd2;
  float* lse;     // [heads][Lmax]
  float *dk, *dv; // fp32 [Lmax][H]: gradient reaching each cached key / value
  // per-token output gradients of the four projections (inputs of dW GEMMs)
  void *dy, *dz, *dx1, *dqkv;
  // per-token LayerNorm output gradients (DEFERRED mode: inputs of the
  // LayerNorm-parameter gradients, reduced once per sequence)
  void *du2, *du;
  // mixed-precision path only: fp16 copy of the LN1 output, bf16 copy of the
  // values (the backward's), fp16 copy of W_qkv (taken at the sequence start)
  void *u16, *vb, *w16;
};

struct Scratch {
  void *du2, *du, *dout;  // [Lmax][H]
  float* D;               // [heads][Lmax]
  void *io_a, *io_b;      // profiler slice buffers [Lmax][H]
  float* splitk;          // split-K partial sums of the slice GEMMs
  size_t splitk_elems;
  float* attn;            // key-split partials of the query-parallel attention kernels
  size_t attn_elems;
  uint16_t* pd;           // stored dS planes of the matrix-core attention backward
  size_t pd_elems;
};

struct Carver {
  char* base;
  size_t off = 0;
  explicit Carver(void* b) : base((char*)b) {}
  void* take(size_t bytes) {
    off = (off + 255) & ~(size_t)255;
    void* p = base ? base + off : nullptr;
    off += bytes;
    return p;
  }
};

enum KClass { K_GEMM_FWD, K_GEMM_DX, K_GEMM_DW, K_ATTN_FWD, K_ATTN_BWD, K_NORM, K_MISC, K_N };
const char* kclass_name[K_N] = {"gemm_fwd_nt", "gemm_bwd_dx_nn", "gemm_bwd_dw_tn", "attn_fwd",
                                "attn_bwd",    "layernorm",      "misc"};

struct PendingTiming {
  int cls;
  hipEvent_t a, b;
  double flops, bytes;
};

}  // namespace

struct tp_stage {
  tp_stage_config cfg;
  // H: residual width; A = heads * d: attention width of this device's heads;
  // F: its FFN width (A = H, F = 4H without operation partitioning)
  int H, A, F, heads, d, L, dt;
  int bsz;  // sequences per batch slice: token t of sequence s is row t * bsz + s
  size_t esz;
  bool mixed;   // mixed-precision path (see mixed_of)
  size_t resz;  // element size of the residual stream (fp32 on the mixed path)
  std::vector<tp_layer_ptrs> P, G;
  std::vector<LayerBufs> lb;
  Scratch sc;
  hipStream_t stream;
  int cached_len = 0, bwd_frontier = 0;
  // a sequence has been started by tp_kv_prefix_reset since the stage was
  // created or last profiled (the dK/dV buffer is zero, the fp16 W_qkv copy taken)
  bool prepared = false;
  // the sequence's next gradient writes store rather than add
  // (TP_SEQ_OVERWRITE_GRADS; cleared once every gradient has been written)
  bool grad_store = false;
  // the fp16 W_qkv copies hold the current weights as of the last snapshot
  bool w16_valid = false;
  bool profiling = false;
  // planning pass (tp_slice_forward_static): no launch, only the largest
  // partial-sum scratch (fp32 elements) the slice's kernels would take
  bool dry = false;
  long dry_need = 0;
  // timing
  bool timing = false;
  std::vector<PendingTiming> pending;
  std::vector<hipEvent_t> free_events;
  int64_t launches[K_N] = {};
  double total_ms[K_N] = {}, flops[K_N] = {}, bytes[K_N] = {};
};

namespace {

bool config_ok(const tp_stage_config* c) {
  if (!c) return false;
  if (c->n_layers < 1 || c->n_layers > 1024 || c->hidden < 1 || c->heads < 1 || c->max_seq < 1)
    return false;
  if (c->hidden % c->heads) return false;
  if (c->dtype != TP_DTYPE_BF16 && c->dtype != TP_DTYPE_FP32) return false;
  if (c->wgrad_mode != TP_WGRAD_PER_SLICE && c->wgrad_mode != TP_WGRAD_DEFERRED) return false;
  if (!(c->ln_eps > 0.f) || !std::isfinite(c->ln_eps)) return false;
  if (c->batch < 0 || c->batch > 64) return false;
  const int p = c->op_parts > 0 ? c->op_parts : 1;
  if (c->op_parts < 0 || c->heads % p || (4 * c->hidden) % p) return false;
  return true;
}

int batch_of(const tp_stage_config* c) { return c->batch > 0 ? c->batch : 1; }
int parts_of(const tp_stage_config* c) { return c->op_parts > 0 ? c->op_parts : 1; }
// The mixed-precision path of bf16 stages whose head width the matrix-core
// attention takes (64, 128): residual stream in fp32, fp16 operands for the
// query/key/value product and the attention scores.
bool mixed_of(const tp_stage_config* c) {
  const int d = c->hidden / c->heads;
  return c->dtype == TP_DTYPE_BF16 && (d == 64 || d == 128);
}

bool config_supported(const tp_stage_config* c) {
  const int d = c->hidden / c->heads;
  if (d != 16 && d != 32 && d != 64 && d != 128) return false;
  if (c->hidden % 8 || c->hidden > 16384) return false;  // LayerNorm rows live in registers
  // the generic attention keeps one score row per block in LDS
  if ((2 * (size_t)c->max_seq + 272) * 4 > 160 * 1024) return false;
  return true;
}

size_t carve(const tp_stage_config* c, void* base, std::vector<LayerBufs>* lbs, Scratch* sc) {
  Carver cv(base);
  const size_t esz = c->dtype == TP_DTYPE_FP32 ? 4 : 2;
  const bool mixed = mixed_of(c);
  const size_t resz = mixed ? 4 : esz;  // residual stream (layer inputs, x1)
  // every per-token arena holds max_seq * batch rows
  const size_t L = (size_t)c->max_seq * batch_of(c), H = c->hidden, pp = parts_of(c);
  const size_t a = c->heads / pp, A = a * (H / c->heads), F = 4 * H / pp;
  for (int i = 0; i < c->n_layers; ++i) {
    LayerBufs b;
    b.x_in = cv.take(L * H * resz);
    b.u = cv.take(L * H * esz);
    b.q = cv.take(L * A * esz);
    b.kc = cv.take(L * A * esz);
    b.vc = cv.take(L * A * esz);
    b.o = cv.take(L * A * esz);
    b.x1 = cv.take(L * H * resz);
    b.u2 = cv.take(L * H * esz);
    b.z = cv.take(L * F * esz);
    b.g = cv.take(L * F * esz);
    b.mean1 = (float*)cv.take(L * 4);
    b.rstd1 = (float*)cv.take(L * 4);
    b.mean2 = (float*)cv.take(L * 4);
    b.rstd2 = (float*)cv.take(L * 4);
    b.lse = (float*)cv.take(a * L * 4);
    b.dk = (float*)cv.take(L * A * 4);
    b.dv = (float*)cv.take(L * A * 4);
    b.dy = cv.take(L * H * esz);
    b.dz = cv.take(L * F * esz);
    b.dx1 = cv.take(L * H * esz);
    b.dqkv = cv.take(L * 3 * A * esz);
    if (c->wgrad_mode == TP_WGRAD_DEFERRED) {
      b.du2 = cv.take(L * H * esz);
      b.du = cv.take(L * H * esz);
    } else {
      b.du2 = b.du = nullptr;
    }
    if (mixed) {
      b.u16 = cv.take(L * H * 2);
      b.vb = cv.take(L * A * 2);
      b.w16 = cv.take(3 * A * H * 2);
    } else {
      b.u16 = b.vb = b.w16 = nullptr;
    }
    if (lbs) lbs->push_back(b);
  }
  Scratch s;
  s.du2 = cv.take(L * H * esz);
  s.du = cv.take(L * H * esz);
  s.dout = cv.take(L * A * esz);
  s.D = (float*)cv.take(a * L * 4);
  s.io_a = cv.take(L * H * esz);
  s.io_b = cv.take(L * H * esz);
  // up to 8 partial [min(L, 256)][widest product output] fp32 products
  s.splitk_elems = 8 * std::min<size_t>(L, 256) * std::max(std::max(F, H), 3 * A);
  s.splitk = (float*)cv.take(s.splitk_elems * 4);
  // attention key splits happen for launches of under 128 blocks of 128 queries
  // (fewer than 16384 query-heads): at most 8 splits of [rows][A] partials and
  // per-query (max, sum) pairs
  {
    const size_t d = H / c->heads, qh = std::min<size_t>(L * a, 16384);
    s.attn_elems = 8 * (qh * d + 2 * qh);
    s.attn = (float*)cv.take(s.attn_elems * 4);
  }
  // the attention backward's stored dS (mixed path: matrix-core attention):
  // 16-bit planes of every key for up to PD_ROWS query rows (whole 256-row
  // blocks) of every head and sequence; longer slices run in query chunks
  {
    constexpr size_t PD_ROWS = 1024;
    const size_t T = (size_t)c->max_seq;
    s.pd_elems = mixed ? (size_t)batch_of(c) * a * T * std::min(PD_ROWS, (T + 255) / 256 * 256) : 0;
    s.pd = s.pd_elems ? (uint16_t*)cv.take(s.pd_elems * 2) : nullptr;
  }
  if (sc) *sc = s;
  return (cv.off + 255) & ~(size_t)255;
}

inline void* rowp(void* p, long t, long width, size_t esz) { return (char*)p + t * width * esz; }
inline const void* rowp(const void* p, long t, long width, size_t esz) {
  return (const char*)p + t * width * esz;
}

hipEvent_t get_event(tp_stage* S) {
  if (!S->free_events.empty()) {
    hipEvent_t e = S->free_events.back();
    S->free_events.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}

// Run one launch, bracketed by events when timing is on.  A failed event call
// fails the launch (its status is returned; the events go back to the pool).
template <typename Fn>
hipError_t launch(tp_stage* S, int cls, double flops, double bytes, Fn&& fn) {
  if (S->dry) return hipSuccess;
  if (!S->timing) return fn();
  hipEvent_t a = get_event(S);
  if (!a) return hipErrorOutOfMemory;
  hipEvent_t b = get_event(S);
  if (!b) {
    S->free_events.push_back(a);
    return hipErrorOutOfMemory;
  }
  hipError_t e = hipEventRecord(a, S->stream);
  if (e == hipSuccess) e = fn();
  if (e == hipSuccess) e = hipEventRecord(b, S->stream);
  if (e != hipSuccess) {
    S->free_events.push_back(a);
    S->free_events.push_back(b);
    return e;
  }
  S->pending.push_back({cls, a, b, flops, bytes});
  return hipSuccess;
}

#define TRY(expr)                             \
  do {                                        \
    hipError_t _e = (expr);                   \
    if (_e != hipSuccess) return TP_ERR_HIP;  \
  } while (0)

double gemm_bytes(const GemmArgs& g, size_t esz) {
  double b = ((double)g.M * g.K + (double)g.K * g.N) * esz;
  if (g.epi == EPI_ACC_F32)
    b += (g.overwrite ? 4.0 : 8.0) * g.M * g.N;
  else
    b += (double)g.M * g.N * esz * (g.epi == EPI_GELU ? 2 : 1) +
         (g.epi == EPI_RESID || g.epi == EPI_DGELU ? (double)g.M * g.N * esz : 0.0);
  return b;
}

hipError_t run_gemm(tp_stage* S, int cls, GemmArgs g) {
  g.ws = S->sc.splitk;
  g.ws_elems = (long)S->sc.splitk_elems;
  if (S->dry) {
    long need = 0;
    g.need = &need;
    const hipError_t e = gemm(S->dt, g, S->stream);
    S->dry_need = std::max(S->dry_need, need);
    return e;
  }
  return launch(S, cls, 2.0 * g.M * g.N * g.K, gemm_bytes(g, S->esz),
                [&] { return gemm(S->dt, g, S->stream); });
}

// A(m,k) row-major [M][K] times weight W [N][K] (B(k,n) = W[n][k]).
GemmArgs nt(int M, int N, int K, const void* A, long lda, const void* W) {
  GemmArgs g;
  g.M = M, g.N = N, g.K = K;
  g.A = A, g.sam = lda, g.sak = 1;
  g.B = W, g.sbk = 1, g.sbn = K;
  return g;
}
// dX = dY [M][K] times W [K][N] (W stored [out = K][in = N]).
GemmArgs nn(int M, int N, int K, const void* A, long lda, const void* W) {
  GemmArgs g;
  g.M = M, g.N = N, g.K = K;
  g.A = A, g.sam = lda, g.sak = 1;
  g.B = W, g.sbk = N, g.sbn = 1;
  return g;
}
// dW [M][N] += sum over K tokens of dY[t][m] X[t][n].
GemmArgs tn(int M, int N, int K, const void* dY, long ldy, const void* X, long ldx, float* dW) {
  GemmArgs g;
  g.M = M, g.N = N, g.K = K;
  g.A = dY, g.sam = 1, g.sak = ldy;
  g.B = X, g.sbk = ldx, g.sbn = 1;
  g.epi = EPI_ACC_F32;
  g.C = dW, g.ldc = N;
  return g;
}

// rows [l, l + n) of the per-token arenas
tp_status wgrad_gemms(tp_stage* S, int li, int l, int n) {
  const int H = S->H, A = S->A, F = S->F;
  const size_t e = S->esz;
  LayerBufs& B = S->lb[li];
  tp_layer_ptrs& G = S->G[li];
  const int ow = S->grad_store;
  GemmArgs g[4] = {
      tn(H, F, n, rowp(B.dy, l, H, e), H, rowp(B.g, l, F, e), F, (float*)G.w_fc2),
      tn(F, H, n, rowp(B.dz, l, F, e), F, rowp(B.u2, l, H, e), H, (float*)G.w_fc1),
      tn(H, A, n, rowp(B.dx1, l, H, e), H, rowp(B.o, l, A, e), A, (float*)G.w_o),
      tn(3 * A, H, n, rowp(B.dqkv, l, 3 * A, e), 3 * A, rowp(B.u, l, H, e), H, (float*)G.w_qkv)};
  for (GemmArgs& gi : g) {
    gi.overwrite = ow;
    TRY(run_gemm(S, K_GEMM_DW, gi));
  }
  return TP_OK;
}

// DEFERRED mode: bias and LayerNorm-parameter gradients of layer li as column
// reductions over all rows [0, rows) of the kept per-token gradients.
tp_status deferred_param_reductions(tp_stage* S, int li, int rows) {
  const int H = S->H, A = S->A, F = S->F, dt = S->dt;
  const size_t e = S->esz;
  const double nb = (double)rows * H * e;
  hipStream_t st = S->stream;
  LayerBufs& B = S->lb[li];
  tp_layer_ptrs& G = S->G[li];
  const int ow = S->grad_store;
  TRY(launch(S, K_MISC, 0, nb,
             [&] { return colsum_acc(dt, rows, H, B.dy, H, (float*)G.b_fc2, ow, st); }));
  TRY(launch(S, K_MISC, 0, (double)rows * F * e,
             [&] { return colsum_acc(dt, rows, F, B.dz, F, (float*)G.b_fc1, ow, st); }));
  TRY(launch(S, K_NORM, 0, 2 * nb, [&] {
    return ln_param_grads(dt, rows, H, B.du2, B.x1, S->mixed, B.mean2, B.rstd2, (float*)G.ln2_g,
                          (float*)G.ln2_b, ow, st);
  }));
  TRY(launch(S, K_MISC, 0, nb,
             [&] { return colsum_acc(dt, rows, H, B.dx1, H, (float*)G.b_o, ow, st); }));
  TRY(launch(S, K_MISC, 0, 3.0 * rows * A * e,
             [&] { return colsum_acc(dt, rows, 3 * A, B.dqkv, 3 * A, (float*)G.b_qkv, ow, st); }));
  TRY(launch(S, K_NORM, 0, 2 * nb, [&] {
    return ln_param_grads(dt, rows, H, B.du, B.x_in, S->mixed, B.mean1, B.rstd1, (float*)G.ln1_g,
                          (float*)G.ln1_b, ow, st);
  }));
  return TP_OK;
}

// Mixed-precision path: fp16 copies of every layer's W_qkv for the
// query/key/value product, taken at the start of a sequence (the parameters
// stay fixed while its slices run).
hipError_t snapshot_wqkv(tp_stage* S) {
  S->w16_valid = false;
  if (!S->mixed) return hipSuccess;
  const size_t n = (size_t)3 * S->A * S->H;
  for (int li = 0; li < S->cfg.n_layers; ++li) {
    const hipError_t e = launch(S, K_MISC, 0, 4.0 * n,
                                [&] { return cvt_bf16_f16(n, S->P[li].w_qkv, S->lb[li].w16, S->stream); });
    if (e != hipSuccess) return e;
  }
  S->w16_valid = true;
  return hipSuccess;
}

tp_status forward_impl(tp_stage* S, int l, int r, const void* x, void* y) {
  const int H = S->H, A = S->A, F = S->F, NL = S->cfg.n_layers, dt = S->dt;
  // batch slice: tokens [l, r) of bsz sequences are rows [lr, lr + n)
  const int ntok = r - l, lr = l * S->bsz, n = ntok * S->bsz;
  const size_t e = S->esz;
  hipStream_t st = S->stream;
  const double nb = (double)n * H * e;
  for (int li = 0; li < NL; ++li) {
    LayerBufs& B = S->lb[li];
    const tp_layer_ptrs& P = S->P[li];
    const bool mx = S->mixed;
    const size_t re = S->resz;
    void* xin = rowp(B.x_in, lr, H, re);
    void* x1 = rowp(B.x1, lr, H, re);
    TRY(launch(S, K_NORM, 0, 2 * nb, [&] {
      return ln_fwd(dt, n, H, li == 0 ? x : xin, li > 0 && mx, li == 0 ? xin : nullptr, mx,
                    P.ln1_g, P.ln1_b, rowp(B.u, lr, H, e), mx ? rowp(B.u16, lr, H, 2) : nullptr,
                    B.mean1 + lr, B.rstd1 + lr, S->cfg.ln_eps, st);
    }));
    GemmArgs g = mx ? nt(n, 3 * A, H, rowp(B.u16, lr, H, 2), H, B.w16)
                    : nt(n, 3 * A, H, rowp(B.u, lr, H, e), H, P.w_qkv);
    g.epi = EPI_QKV;
    g.bias = P.b_qkv;
    g.q = rowp(B.q, lr, A, e), g.k = rowp(B.kc, lr, A, e), g.v = rowp(B.vc, lr, A, e), g.H = A;
    if (mx) g.in_f16 = 1, g.qkv_f16 = 1, g.vb = rowp(B.vb, lr, A, 2);
    TRY(run_gemm(S, K_GEMM_FWD, g));
    AttnArgs a;
    a.l = l, a.r = r, a.H = A, a.heads = S->heads, a.d = S->d, a.Lmax = S->L;
    a.bs = S->bsz, a.ld = S->bsz * A;
    a.ws = S->sc.attn, a.ws_elems = (long)S->sc.attn_elems;
    a.scale = 1.f / std::sqrt((float)S->d);
    a.q = rowp(B.q, lr, A, e), a.kc = B.kc, a.vc = B.vc, a.o = rowp(B.o, lr, A, e), a.lse = B.lse;
    a.f16 = mx;
    if (S->dry) {
      long need = 0;
      a.need = &need;
      TRY(attn_fwd(dt, a, st));
      S->dry_need = std::max(S->dry_need, need);
      a.need = nullptr;
    }
    const double pairs = ((double)ntok * l + (double)ntok * (ntok + 1) / 2) * S->bsz;
    TRY(launch(S, K_ATTN_FWD, 4.0 * A * pairs, (2.0 * ntok + 2.0 * r) * S->bsz * A * e,
               [&] { return attn_fwd(dt, a, st); }));
    g = nt(n, H, A, rowp(B.o, lr, A, e), A, P.w_o);
    g.epi = EPI_RESID, g.bias = P.b_o, g.R = xin, g.ldr = H, g.C = x1, g.ldc = H;
    g.r_f32 = g.c_f32 = mx;
    TRY(run_gemm(S, K_GEMM_FWD, g));
    TRY(launch(S, K_NORM, 0, 2 * nb, [&] {
      return ln_fwd(dt, n, H, x1, mx, nullptr, 0, P.ln2_g, P.ln2_b, rowp(B.u2, lr, H, e), nullptr,
                    B.mean2 + lr, B.rstd2 + lr, S->cfg.ln_eps, st);
    }));
    g = nt(n, F, H, rowp(B.u2, lr, H, e), H, P.w_fc1);
    g.epi = EPI_GELU, g.bias = P.b_fc1, g.C = rowp(B.z, lr, F, e), g.ldc = F;
    g.C2 = rowp(B.g, lr, F, e), g.ldc2 = F;
    TRY(run_gemm(S, K_GEMM_FWD, g));
    g = nt(n, H, F, rowp(B.g, lr, F, e), F, P.w_fc2);
    g.epi = EPI_RESID, g.bias = P.b_fc2, g.R = x1, g.ldr = H, g.r_f32 = mx;
    g.C = li == NL - 1 ? y : rowp(S->lb[li + 1].x_in, lr, H, re), g.ldc = H;
    g.c_f32 = mx && li < NL - 1;
    TRY(run_gemm(S, K_GEMM_FWD, g));
  }
  return TP_OK;
}

tp_status backward_impl(tp_stage* S, int l, int r, const void* dy, void* dx) {
  const int H = S->H, A = S->A, F = S->F, NL = S->cfg.n_layers, dt = S->dt;
  // batch slice: tokens [l, r) of bsz sequences are rows [lr, lr + n)
  const int ntok = r - l, lr = l * S->bsz, n = ntok * S->bsz;
  const size_t e = S->esz;
  hipStream_t st = S->stream;
  const bool per_slice = S->cfg.wgrad_mode == TP_WGRAD_PER_SLICE;
  const double nb = (double)n * H * e;
  const bool mx = S->mixed;
  const int ow = S->grad_store;
  for (int li = NL - 1; li >= 0; --li) {
    LayerBufs& B = S->lb[li];
    const tp_layer_ptrs& P = S->P[li];
    tp_layer_ptrs& G = S->G[li];
    void* dyl = rowp(B.dy, lr, H, e);
    const void* x1 = rowp(B.x1, lr, H, S->resz);
    const void* xin = rowp(B.x_in, lr, H, S->resz);
    if (li == NL - 1)
      TRY(launch(S, K_MISC, 0, 2 * nb, [&] { return copy_rows(dt, n, H, dy, dyl, st); }));
    // FC2 backward (dX fused with GELU'): dz = (dy W2) * GELU'(z)
    GemmArgs g = nn(n, F, H, dyl, H, P.w_fc2);
    g.epi = EPI_DGELU, g.R = rowp(B.z, lr, F, e), g.ldr = F, g.C = rowp(B.dz, lr, F, e), g.ldc = F;
    TRY(run_gemm(S, K_GEMM_DX, g));
    if (per_slice)
      TRY(launch(S, K_MISC, 0, nb, [&] { return colsum_acc(dt, n, H, dyl, H, (float*)G.b_fc2, ow, st); }));
    // LayerNorm output gradients: per-slice scratch, or (deferred mode) rows of
    // per-layer arenas kept for the once-per-sequence parameter reductions
    void* du2 = per_slice ? S->sc.du2 : rowp(B.du2, lr, H, e);
    void* du = per_slice ? S->sc.du : rowp(B.du, lr, H, e);
    // FC1 backward: du2 = dz W1
    g = nn(n, H, F, rowp(B.dz, lr, F, e), F, P.w_fc1);
    g.C = du2, g.ldc = H;
    TRY(run_gemm(S, K_GEMM_DX, g));
    if (per_slice)
      TRY(launch(S, K_MISC, 0, (double)n * F * e, [&] {
        return colsum_acc(dt, n, F, rowp(B.dz, lr, F, e), F, (float*)G.b_fc1, ow, st);
      }));
    // LN2 backward + residual: dx1 = dy + LN2^T(du2)
    TRY(launch(S, K_NORM, 0, 4 * nb, [&] {
      return ln_bwd(dt, n, H, du2, x1, mx, B.mean2 + lr, B.rstd2 + lr, P.ln2_g,
                    dyl, rowp(B.dx1, lr, H, e), st);
    }));
    if (per_slice)
      TRY(launch(S, K_NORM, 0, 2 * nb, [&] {
        return ln_param_grads(dt, n, H, du2, x1, mx, B.mean2 + lr, B.rstd2 + lr,
                              (float*)G.ln2_g, (float*)G.ln2_b, ow, st);
      }));
    // output projection backward: dO = dx1 W_o
    g = nn(n, A, H, rowp(B.dx1, lr, H, e), H, P.w_o);
    g.C = S->sc.dout, g.ldc = A;
    TRY(run_gemm(S, K_GEMM_DX, g));
    if (per_slice)
      TRY(launch(S, K_MISC, 0, nb, [&] {
        return colsum_acc(dt, n, H, rowp(B.dx1, lr, H, e), H, (float*)G.b_o, ow, st);
      }));
    // attention backward: dq rows, dK/dV into the fp32 buffer for keys [0, r)
    AttnArgs a;
    a.l = l, a.r = r, a.H = A, a.heads = S->heads, a.d = S->d, a.Lmax = S->L;
    a.bs = S->bsz, a.ld = S->bsz * A;
    a.ws = S->sc.attn, a.ws_elems = (long)S->sc.attn_elems;
    a.pd = S->sc.pd, a.pd_elems = (long)S->sc.pd_elems;
    a.scale = 1.f / std::sqrt((float)S->d);
    a.q = rowp(B.q, lr, A, e), a.kc = B.kc, a.o = rowp(B.o, lr, A, e), a.lse = B.lse;
    a.vc = mx ? B.vb : B.vc;  // the backward's values are bf16
    a.f16 = mx;
    a.dout = S->sc.dout, a.D = S->sc.D;
    a.dq = rowp(B.dqkv, lr, 3 * A, e), a.ld_dq = (long)S->bsz * 3 * A, a.dq_seq = 3 * A;
    a.dk = B.dk, a.dv = B.dv;
    const double pairs = ((double)ntok * l + (double)ntok * (ntok + 1) / 2) * S->bsz;
    TRY(launch(S, K_ATTN_BWD, 8.0 * A * pairs,
               ((4.0 * ntok + 2.0 * r) * A * e + 16.0 * r * A) * S->bsz,
               [&] { return attn_bwd(dt, a, st); }));
    TRY(launch(S, K_MISC, 0, (8.0 + 4.0 * e) * n * A, [&] {
      return pack_dkv(dt, n, A, B.dk + (long)lr * A, B.dv + (long)lr * A,
                      rowp(B.dqkv, lr, 3 * A, e), st);
    }));
    // QKV backward: du = [dq dk dv] W_qkv
    g = nn(n, H, 3 * A, rowp(B.dqkv, lr, 3 * A, e), 3 * A, P.w_qkv);
    g.C = du, g.ldc = H;
    TRY(run_gemm(S, K_GEMM_DX, g));
    if (per_slice)
      TRY(launch(S, K_MISC, 0, 3.0 * n * A * e, [&] {
        return colsum_acc(dt, n, 3 * A, rowp(B.dqkv, lr, 3 * A, e), 3 * A, (float*)G.b_qkv, ow, st);
      }));
    // LN1 backward + residual: dx = dx1 + LN1^T(du)
    void* out = li == 0 ? dx : rowp(S->lb[li - 1].dy, lr, H, e);
    TRY(launch(S, K_NORM, 0, 4 * nb, [&] {
      return ln_bwd(dt, n, H, du, xin, mx, B.mean1 + lr, B.rstd1 + lr, P.ln1_g,
                    rowp(B.dx1, lr, H, e), out, st);
    }));
    if (per_slice)
      TRY(launch(S, K_NORM, 0, 2 * nb, [&] {
        return ln_param_grads(dt, n, H, du, xin, mx, B.mean1 + lr, B.rstd1 + lr,
                              (float*)G.ln1_g, (float*)G.ln1_b, ow, st);
      }));
    if (per_slice) {
      tp_status s = wgrad_gemms(S, li, lr, n);
      if (s != TP_OK) return s;
    }
  }
  if (!per_slice && l == 0 && !S->profiling) {
    for (int li = NL - 1; li >= 0; --li) {
      tp_status s = deferred_param_reductions(S, li, S->cached_len * S->bsz);
      if (s != TP_OK) return s;
      s = wgrad_gemms(S, li, 0, S->cached_len * S->bsz);
      if (s != TP_OK) return s;
    }
  }
  return TP_OK;
}

}  // namespace

extern "C" {

size_t tp_stage_workspace_bytes(const tp_stage_config* cfg) {
  if (!config_ok(cfg)) return 0;
  return carve(cfg, nullptr, nullptr, nullptr);
}

static bool layer_ptrs_ok(const tp_layer_ptrs& p) {
  const void* a[] = {p.ln1_g, p.ln1_b, p.w_qkv, p.b_qkv, p.w_o,   p.b_o,
                     p.ln2_g, p.ln2_b, p.w_fc1, p.b_fc1, p.w_fc2, p.b_fc2};
  for (const void* v : a)
    if (!v) return false;
  return true;
}

tp_status tp_stage_init(const tp_stage_config* cfg, const tp_layer_ptrs* params,
                        const tp_layer_ptrs* grads, void* workspace, size_t workspace_bytes,
                        void* stream, tp_stage** out) {
  if (!out) return TP_ERR_INVALID;
  *out = nullptr;
  if (!config_ok(cfg) || !params || !grads || !workspace) return TP_ERR_INVALID;
  for (int i = 0; i < cfg->n_layers; ++i)
    if (!layer_ptrs_ok(params[i]) || !layer_ptrs_ok(grads[i])) return TP_ERR_INVALID;
  if (!config_supported(cfg)) return TP_ERR_UNSUPPORTED;
  if (((uintptr_t)workspace & 255) || workspace_bytes < carve(cfg, nullptr, nullptr, nullptr))
    return TP_ERR_WORKSPACE;
  tp_stage* S = new (std::nothrow) tp_stage();
  if (!S) return TP_ERR_INVALID;
  S->cfg = *cfg;
  S->H = cfg->hidden;
  S->heads = cfg->heads / parts_of(cfg);
  S->d = cfg->hidden / cfg->heads;
  S->A = S->heads * S->d;
  S->F = 4 * cfg->hidden / parts_of(cfg);
  S->L = cfg->max_seq;
  S->bsz = batch_of(cfg);
  S->dt = cfg->dtype == TP_DTYPE_FP32 ? DT_FP32 : DT_BF16;
  S->esz = cfg->dtype == TP_DTYPE_FP32 ? 4 : 2;
  S->mixed = mixed_of(cfg);
  S->resz = S->mixed ? 4 : S->esz;
  S->P.assign(params, params + cfg->n_layers);
  S->G.assign(grads, grads + cfg->n_layers);
  carve(cfg, workspace, &S->lb, &S->sc);
  S->stream = (hipStream_t)stream;
  *out = S;
  return TP_OK;
}

void tp_stage_destroy(tp_stage* S) {
  if (!S) return;
  for (auto& p : S->pending) {
    hipEventDestroy(p.a);
    hipEventDestroy(p.b);
  }
  for (auto e : S->free_events) hipEventDestroy(e);
  delete S;
}

tp_status tp_kv_prefix_reset(tp_stage* S) { return tp_kv_prefix_reset_ex(S, 0); }

tp_status tp_kv_prefix_reset_ex(tp_stage* S, unsigned flags) {
  if (!S || (flags & ~(TP_SEQ_OVERWRITE_GRADS | TP_SEQ_REUSE_WQKV_COPY))) return TP_ERR_INVALID;
  const size_t n = (size_t)S->L * S->bsz * S->A;
  for (auto& B : S->lb) {
    TRY(fill_f32(B.dk, n, 0.f, S->stream));
    TRY(fill_f32(B.dv, n, 0.f, S->stream));
  }
  if (!(flags & TP_SEQ_REUSE_WQKV_COPY) || !S->w16_valid) TRY(snapshot_wqkv(S));
  S->cached_len = 0;
  S->bwd_frontier = 0;
  S->prepared = true;
  S->grad_store = (flags & TP_SEQ_OVERWRITE_GRADS) != 0;
  return TP_OK;
}

static bool aligned16(const void* p) { return ((uintptr_t)p & 15) == 0; }

tp_status tp_slice_forward(tp_stage* S, int l, int r, const void* x, void* y) {
  if (!S || !x || !y || !aligned16(x) || !aligned16(y)) return TP_ERR_INVALID;
  if (l < 0 || r <= l || r > S->L) return TP_ERR_INVALID;
  // a sequence starts with tp_kv_prefix_reset; slices arrive in order; once
  // the backward pass has begun (frontier below the cached length) only
  // another reset starts over
  if (!S->prepared || l != S->cached_len || S->bwd_frontier != S->cached_len)
    return TP_ERR_ORDER;
  tp_status s = forward_impl(S, l, r, x, y);
  if (s != TP_OK) return s;
  S->cached_len = r;
  S->bwd_frontier = r;
  return TP_OK;
}

tp_status tp_slice_forward_static(tp_stage* S, int l, int r, const void* x, void* y) {
  if (!S || !x || !y || !aligned16(x) || !aligned16(y)) return TP_ERR_INVALID;
  if (l < 0 || r <= l || r > S->L) return TP_ERR_INVALID;
  if (l != S->cached_len || S->bwd_frontier != S->cached_len) return TP_ERR_ORDER;
  // plan the slice exactly as tp_slice_forward would run it (same split
  // choices), nothing enqueued: the largest partial-sum scratch any of its
  // kernels takes must fit the static array.  The plan reads only the shapes,
  // so it is checked before whether a sequence has been started.
  S->dry = true;
  S->dry_need = 0;
  tp_status s = forward_impl(S, l, r, x, y);
  S->dry = false;
  if (s != TP_OK) return s;
  size_t cap = 0;
  void* p = static_scratch(&cap);
  if ((size_t)S->dry_need * 4 > cap) return TP_ERR_WORKSPACE;
  if (!S->prepared) return TP_ERR_ORDER;
  if (!p) return TP_ERR_HIP;
  // the kernels, split plans included, are those of tp_slice_forward; only the
  // partial sums live in the static array (one launch's partials at a time:
  // every split product is reduced before the next launch on the stream).
  // Timing events are not created here.
  Scratch saved = S->sc;
  const bool was_timing = S->timing;
  S->sc.splitk = (float*)p;
  S->sc.attn = (float*)p;
  S->timing = false;
  s = forward_impl(S, l, r, x, y);
  S->sc = saved;
  S->timing = was_timing;
  if (s != TP_OK) return s;
  S->cached_len = r;
  S->bwd_frontier = r;
  return TP_OK;
}

tp_status tp_slice_backward(tp_stage* S, int l, int r, const void* dy, void* dx) {
  if (!S || !dy || !dx || !aligned16(dy) || !aligned16(dx)) return TP_ERR_INVALID;
  if (l < 0 || r <= l || r > S->L) return TP_ERR_INVALID;
  if (!S->prepared || r != S->bwd_frontier) return TP_ERR_ORDER;
  tp_status s = backward_impl(S, l, r, dy, dx);
  if (s != TP_OK) return s;
  S->bwd_frontier = l;
  // every gradient has now been written once: later writes add
  if (S->cfg.wgrad_mode == TP_WGRAD_PER_SLICE || l == 0) S->grad_store = false;
  return TP_OK;
}

tp_status tp_profile_slice_cost(tp_stage* S, const int* lens, int n_lens, const int* ctxs,
                                int n_ctxs, int warmup, int reps, int64_t* t_fwd_ns,
                                int64_t* t_bwd_ns) {
  if (!S || !lens || !ctxs || !t_fwd_ns || !t_bwd_ns || n_lens < 1 || n_ctxs < 1 || warmup < 0 ||
      reps < 1)
    return TP_ERR_INVALID;
  for (int i = 0; i < n_lens; ++i)
    if (lens[i] < 1) return TP_ERR_INVALID;
  for (int j = 0; j < n_ctxs; ++j)
    if (ctxs[j] < 0) return TP_ERR_INVALID;
  hipEvent_t e0 = nullptr, e1 = nullptr, e2 = nullptr;
  if (hipEventCreate(&e0) != hipSuccess || hipEventCreate(&e1) != hipSuccess ||
      hipEventCreate(&e2) != hipSuccess) {
    for (hipEvent_t e : {e0, e1, e2})
      if (e) hipEventDestroy(e);
    return TP_ERR_HIP;
  }
  const bool was_timing = S->timing;
  S->timing = false;
  S->profiling = true;
  S->grad_store = false;
  tp_status status = snapshot_wqkv(S) == hipSuccess ? TP_OK : TP_ERR_HIP;
  // deterministic, finite slice inputs
  const size_t io = (size_t)S->L * S->bsz * S->H;
  if (S->dt == DT_FP32) {
    if (fill_f32((float*)S->sc.io_a, io, 0.5f, S->stream) != hipSuccess) status = TP_ERR_HIP;
  } else {
    if (fill_f32((float*)S->sc.io_a, io / 2, 0.5f, S->stream) != hipSuccess) status = TP_ERR_HIP;
  }
  std::vector<float> tf, tb;
  for (int i = 0; i < n_lens && status == TP_OK; ++i)
    for (int j = 0; j < n_ctxs && status == TP_OK; ++j) {
      const int len = lens[i], ctx = ctxs[j];
      const size_t idx = (size_t)i * n_ctxs + j;
      if ((long)len + ctx > S->L) {
        t_fwd_ns[idx] = t_bwd_ns[idx] = -1;
        continue;
      }
      tf.clear();
      tb.clear();
      for (int rep = 0; rep < warmup + reps && status == TP_OK; ++rep) {
        S->cached_len = ctx;
        if (hipEventRecord(e0, S->stream) != hipSuccess) {
          status = TP_ERR_HIP;
          break;
        }
        status = forward_impl(S, ctx, ctx + len, S->sc.io_a, S->sc.io_b);
        if (status != TP_OK) break;
        if (hipEventRecord(e1, S->stream) != hipSuccess) {
          status = TP_ERR_HIP;
          break;
        }
        status = backward_impl(S, ctx, ctx + len, S->sc.io_a, S->sc.io_b);
        if (status != TP_OK) break;
        float f = 0, b = 0;
        if (hipEventRecord(e2, S->stream) != hipSuccess || hipEventSynchronize(e2) != hipSuccess ||
            hipEventElapsedTime(&f, e0, e1) != hipSuccess ||
            hipEventElapsedTime(&b, e1, e2) != hipSuccess) {
          status = TP_ERR_HIP;
          break;
        }
        if (rep >= warmup) {
          tf.push_back(f);
          tb.push_back(b);
        }
      }
      if (status != TP_OK) break;
      std::sort(tf.begin(), tf.end());
      std::sort(tb.begin(), tb.end());
      auto med = [](const std::vector<float>& v) {
        const size_t m = v.size();
        return m % 2 ? (double)v[m / 2] : 0.5 * ((double)v[m / 2 - 1] + v[m / 2]);
      };
      t_fwd_ns[idx] = (int64_t)std::llround(med(tf) * 1e6);
      t_bwd_ns[idx] = (int64_t)std::llround(med(tb) * 1e6);
    }
  hipEventDestroy(e0);
  hipEventDestroy(e1);
  hipEventDestroy(e2);
  S->profiling = false;
  S->timing = was_timing;
  // the caches, dK/dV accumulators and slice buffers now hold profiling data
  S->cached_len = 0;
  S->bwd_frontier = 0;
  S->prepared = false;
  return status;
}

const char* tp_status_string(tp_status s) {
  switch (s) {
    case TP_OK: return "ok";
    case TP_ERR_INVALID: return "invalid argument";
    case TP_ERR_ORDER: return "slice out of order";
    case TP_ERR_UNSUPPORTED: return "unsupported configuration";
    case TP_ERR_WORKSPACE: return "workspace too small or misaligned";
    case TP_ERR_HIP: return "HIP runtime error";
  }
  return "unknown status";
}

tp_status tp_stage_enable_kernel_timing(tp_stage* S, int enable) {
  if (!S) return TP_ERR_INVALID;
  S->timing = enable != 0;
  return TP_OK;
}

int tp_stage_kernel_stats(tp_stage* S, tp_kernel_stat* out, int cap) {
  if (!S) return -1;
  if (!S->pending.empty()) {
    bool ok = hipStreamSynchronize(S->stream) == hipSuccess;
    for (auto& p : S->pending) {
      float ms = 0.f;
      if (ok && hipEventElapsedTime(&ms, p.a, p.b) != hipSuccess) ok = false;
      S->free_events.push_back(p.a);
      S->free_events.push_back(p.b);
      if (!ok) continue;
      S->launches[p.cls] += 1;
      S->total_ms[p.cls] += ms;
      S->flops[p.cls] += p.flops;
      S->bytes[p.cls] += p.bytes;
    }
    S->pending.clear();
    if (!ok) {
      // the sums would be wrong: drop them all
      for (int c = 0; c < K_N; ++c) {
        S->launches[c] = 0;
        S->total_ms[c] = S->flops[c] = S->bytes[c] = 0;
      }
      return -1;
    }
  }
  int w = 0;
  for (int c = 0; c < K_N && out && w < cap; ++c) {
    if (!S->launches[c]) continue;
    std::memset(&out[w], 0, sizeof(tp_kernel_stat));
    std::strncpy(out[w].name, kclass_name[c], sizeof(out[w].name) - 1);
    out[w].launches = S->launches[c];
    out[w].total_ms = S->total_ms[c];
    out[w].flops = S->flops[c];
    out[w].bytes = S->bytes[c];
    ++w;
  }
  // reading resets the counters
  for (int c = 0; c < K_N; ++c) {
    S->launches[c] = 0;
    S->total_ms[c] = S->flops[c] = S->bytes[c] = 0;
  }
  return w;
}

}  // extern "C"
