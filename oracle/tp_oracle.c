/*
 * TeraPipe stage oracle -- TEST INFRASTRUCTURE ONLY.
 *
 * A plain, slow, fp64 CPU implementation of what one pipeline stage of the
 * token-level pipeline computes, and of the slicing dynamic program.  Only the
 * test suite, the smoke check and the CPU-baseline leg of the benchmark may load
 * it.  It shares no code with the GPU library.
 *
 * Paper: Li et al., "TeraPipe: Token-Level Pipeline Parallelism for Training
 * Large-Scale Language Models" (ICML 2021, arXiv 2102.07988).
 *
 * Stage model (Sec. 3.1, Eq. 2 self-attention and Eq. 3 feed-forward; cells of
 * consecutive layers, Sec. 3.2).  The paper writes a single-head, bias-free
 * attention with scale 1/sqrt(H) and no layer norm; this oracle uses the GPT-3
 * block the evaluation follows (Sec. 4): pre-LayerNorm, a heads of width
 * d = H/a with scale 1/sqrt(d), biases on all four projections, output
 * projection, residual connections, and sigma = GELU (tanh form).  The causal
 * sum is inclusive (key s <= query t), exactly as the sum in Eq. 2 is written.
 *
 * Per layer, for every token t:
 *   u  = LN1(x)                       (biased variance, eps, affine)
 *   [q,k,v] = W_qkv u + b_qkv         (k, v appended to the per-layer K/V cache)
 *   o_h = sum_{s<=t} softmax_s(q_h . k_{s,h} / sqrt(d)) v_{s,h}
 *   x1 = x + W_o o + b_o
 *   u2 = LN2(x1);  z = W_1 u2 + b_1;  g = GELU(z)
 *   y  = x1 + W_2 g + b_2
 *
 * A stage may also be one device's shard of operation partitioning (the #Op
 * column of Table 1, partitioning inside a layer as in Megatron-LM): heads / p
 * heads and 4H / p FFN units; the partial sums of the output and FC2
 * projections that the all-reduce would add up across devices are taken as this
 * device's whole sum (or_stage_create_ex).
 *
 * Slices (Sec. 3.2): a forward call processes tokens [l, r) with l equal to the
 * number of tokens already cached, attending to the cached K/V of every earlier
 * slice.  Backward calls run slices in reverse order; the gradient flowing into
 * an earlier slice's keys and values is held in a dK/dV buffer.  Every
 * cross-token sum (weight, bias and LayerNorm-parameter gradients, dK, dV) is
 * accumulated in globally descending token order and every per-token sum
 * (dot products, softmax) in ascending index order, so that any slicing of a
 * sequence performs exactly the same floating-point operations as processing
 * it whole: the outputs are bitwise identical for every slicing.
 *
 * Slicing DP (Sec. 3.3, Eq. 5-8, Algorithm 1, and the "Optimization"
 * paragraph that follows it): see or_dp_optimal_slicing below.
 *
 * Parity pins (tests/): the single-slice stage is checked against PyTorch CPU
 * float64 autograd of a textbook pre-LN block, gradients against central finite
 * differences, slicings against each other bitwise, and the DP against
 * exhaustive enumeration and closed forms.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define OR_OK 0
#define OR_ERR_INVALID -1
#define OR_ERR_ORDER -2

typedef struct {
  const double *ln1_g, *ln1_b, *w_qkv, *b_qkv, *w_o, *b_o;
  const double *ln2_g, *ln2_b, *w1, *b1, *w2, *b2;
} or_params;

typedef struct {
  double *ln1_g, *ln1_b, *w_qkv, *b_qkv, *w_o, *b_o;
  double *ln2_g, *ln2_b, *w1, *b1, *w2, *b2;
} or_grads;

/* Per-layer state; every per-token array is indexed by absolute position. */
typedef struct {
  double *x, *mean1, *rstd1, *u, *q, *o, *x1, *mean2, *rstd2, *u2, *z, *g;
  double *kc, *vc;   /* K/V cache [Lmax][A] */
  double *dk, *dv;   /* dK/dV gradient buffer [Lmax][A] */
  double *dx1, *dob; /* backward temporaries [Lmax][H], [Lmax][A] */
} or_layer_state;

typedef struct {
  int n_layers, H, heads, d, A, F, Lmax; /* A = heads * d (attention width), F = FFN width */
  double eps;
  int cached_len, bwd_frontier;
  const or_params *p;
  or_grads *gr;
  or_layer_state *st;
} or_stage;

static double *zalloc(size_t n) { return (double *)calloc(n ? n : 1, sizeof(double)); }

/* ---------------------------------------------------------------- primitives */

/* C[m][n] = bias[n] + sum_k A[m][k] * B[n][k], k ascending. */
static void mm_nt_bias(int M, int N, int K, const double *A, const double *B,
                       const double *bias, double *C) {
#pragma omp parallel for collapse(2) schedule(static) if ((long)M * N * K > 100000)
  for (int m = 0; m < M; ++m)
    for (int n = 0; n < N; ++n) {
      double s = 0.0;
      const double *a = A + (size_t)m * K, *b = B + (size_t)n * K;
      for (int k = 0; k < K; ++k) s += a[k] * b[k];
      C[(size_t)m * N + n] = s + bias[n];
    }
}

/* C[m][n] = sum_k A[m][k] * B[k][n], k ascending for every element. */
static void mm_nn(int M, int N, int K, const double *A, const double *B, double *C) {
#pragma omp parallel for schedule(static) if ((long)M * N * K > 100000)
  for (int m = 0; m < M; ++m) {
    double *c = C + (size_t)m * N;
    for (int n = 0; n < N; ++n) c[n] = 0.0;
    for (int k = 0; k < K; ++k) {
      const double a = A[(size_t)m * K + k];
      const double *b = B + (size_t)k * N;
      for (int n = 0; n < N; ++n) c[n] += a * b[n];
    }
  }
}

/* G[o][i] += sum over tokens t = r-1 down to l of dY[t][o] * X[t][i];
 * gb[o] += sum over the same tokens of dY[t][o].  Rows of dY/X are absolute
 * token positions with strides No / Ni. */
static void acc_wgrad_desc(int l, int r, int No, int Ni, const double *dY, const double *X,
                           double *G, double *gb) {
#pragma omp parallel for schedule(static) if ((long)(r - l) * No * Ni > 100000)
  for (int o = 0; o < No; ++o) {
    double *gr = G + (size_t)o * Ni;
    for (int t = r - 1; t >= l; --t) {
      const double a = dY[(size_t)t * No + o];
      const double *x = X + (size_t)t * Ni;
      for (int i = 0; i < Ni; ++i) gr[i] += a * x[i];
      gb[o] += a;
    }
  }
}

static const double GELU_C = 0.7978845608028654; /* sqrt(2/pi) */
static const double GELU_A = 0.044715;

double or_gelu(double z) { return 0.5 * z * (1.0 + tanh(GELU_C * (z + GELU_A * z * z * z))); }

double or_gelu_grad(double z) {
  const double th = tanh(GELU_C * (z + GELU_A * z * z * z));
  return 0.5 * (1.0 + th) + 0.5 * z * (1.0 - th * th) * GELU_C * (1.0 + 3.0 * GELU_A * z * z);
}

/* LayerNorm of one row: biased variance, eps inside the square root. */
static void ln_row(int H, double eps, const double *x, const double *gam, const double *bet,
                   double *y, double *mean_out, double *rstd_out) {
  double s = 0.0;
  for (int i = 0; i < H; ++i) s += x[i];
  const double mean = s / H;
  double v = 0.0;
  for (int i = 0; i < H; ++i) v += (x[i] - mean) * (x[i] - mean);
  const double rstd = 1.0 / sqrt(v / H + eps);
  for (int i = 0; i < H; ++i) y[i] = gam[i] * ((x[i] - mean) * rstd) + bet[i];
  *mean_out = mean;
  *rstd_out = rstd;
}

/* Exact derivative of one LayerNorm row: given dL/du returns dL/dx. */
static void ln_row_bwd(int H, const double *x, double mean, double rstd, const double *gam,
                       const double *du, double *dx) {
  double a = 0.0, b = 0.0;
  for (int i = 0; i < H; ++i) {
    const double xh = (x[i] - mean) * rstd;
    const double dxh = du[i] * gam[i];
    a += dxh;
    b += dxh * xh;
  }
  a /= H;
  b /= H;
  for (int i = 0; i < H; ++i) {
    const double xh = (x[i] - mean) * rstd;
    dx[i] = rstd * (du[i] * gam[i] - a - xh * b);
  }
}

/* Softmax weights of query t of head h over keys 0..t (Eq. 2): fills P[0..t]. */
static void attn_probs(const or_stage *S, const or_layer_state *L, int t, int h, double *P) {
  const int A = S->A, d = S->d;
  const double scale = 1.0 / sqrt((double)d);
  const double *q = L->q + (size_t)t * A + h * d;
  double mx = -INFINITY;
  for (int s = 0; s <= t; ++s) {
    const double *k = L->kc + (size_t)s * A + h * d;
    double dot = 0.0;
    for (int j = 0; j < d; ++j) dot += q[j] * k[j];
    P[s] = dot * scale;
    if (P[s] > mx) mx = P[s];
  }
  double Z = 0.0;
  for (int s = 0; s <= t; ++s) {
    P[s] = exp(P[s] - mx);
    Z += P[s];
  }
  for (int s = 0; s <= t; ++s) P[s] /= Z;
}

/* ----------------------------------------------------------------- the stage */

/* A stage whose attention has `heads` heads of width d and whose FFN has F
 * units, on a residual stream of width H (the full block: heads * d = H,
 * F = 4H; one GPU's shard of p-way operation partitioning: heads / p heads and
 * 4H / p units, the partial sums of the output and FC2 projections taken as
 * this device's whole sum). */
or_stage *or_stage_create_ex(int n_layers, int H, int heads, int d, int F, int Lmax, double eps,
                             const or_params *p, or_grads *g) {
  if (n_layers < 1 || H < 1 || heads < 1 || d < 1 || F < 1 || Lmax < 1 || !p || !g) return NULL;
  or_stage *S = (or_stage *)calloc(1, sizeof(or_stage));
  S->n_layers = n_layers;
  S->H = H;
  S->heads = heads;
  S->d = d;
  S->A = heads * d;
  S->F = F;
  S->Lmax = Lmax;
  S->eps = eps;
  S->p = p;
  S->gr = g;
  S->st = (or_layer_state *)calloc(n_layers, sizeof(or_layer_state));
  const size_t LH = (size_t)Lmax * H, LF = (size_t)Lmax * S->F, LA = (size_t)Lmax * S->A;
  for (int i = 0; i < n_layers; ++i) {
    or_layer_state *L = &S->st[i];
    L->x = zalloc(LH);
    L->mean1 = zalloc(Lmax);
    L->rstd1 = zalloc(Lmax);
    L->u = zalloc(LH);
    L->q = zalloc(LA);
    L->o = zalloc(LA);
    L->x1 = zalloc(LH);
    L->mean2 = zalloc(Lmax);
    L->rstd2 = zalloc(Lmax);
    L->u2 = zalloc(LH);
    L->z = zalloc(LF);
    L->g = zalloc(LF);
    L->kc = zalloc(LA);
    L->vc = zalloc(LA);
    L->dk = zalloc(LA);
    L->dv = zalloc(LA);
    L->dx1 = zalloc(LH);
    L->dob = zalloc(LA);
  }
  return S;
}

/* The full block: heads of width H / heads, FFN width 4H. */
or_stage *or_stage_create(int n_layers, int H, int heads, int Lmax, double eps,
                          const or_params *p, or_grads *g) {
  if (heads < 1 || H % heads) return NULL;
  return or_stage_create_ex(n_layers, H, heads, H / heads, 4 * H, Lmax, eps, p, g);
}

void or_stage_destroy(or_stage *S) {
  if (!S) return;
  for (int i = 0; i < S->n_layers; ++i) {
    or_layer_state *L = &S->st[i];
    double *ptrs[] = {L->x, L->mean1, L->rstd1, L->u, L->q, L->o, L->x1, L->mean2, L->rstd2,
                      L->u2, L->z, L->g, L->kc, L->vc, L->dk, L->dv, L->dx1, L->dob};
    for (size_t j = 0; j < sizeof(ptrs) / sizeof(ptrs[0]); ++j) free(ptrs[j]);
  }
  free(S->st);
  free(S);
}

/* Start of a new sequence: empty cache, zero dK/dV buffers. */
void or_reset(or_stage *S) {
  S->cached_len = 0;
  S->bwd_frontier = 0;
  const size_t LA = (size_t)S->Lmax * S->A;
  for (int i = 0; i < S->n_layers; ++i) {
    memset(S->st[i].dk, 0, LA * sizeof(double));
    memset(S->st[i].dv, 0, LA * sizeof(double));
  }
}

/* Forward of slice [l, r): x, y are [r-l][H]. */
int or_forward(or_stage *S, int l, int r, const double *x, double *y) {
  if (!S || !x || !y || l < 0 || r <= l || r > S->Lmax) return OR_ERR_INVALID;
  if (l != S->cached_len) return OR_ERR_ORDER;
  const int H = S->H, A = S->A, F = S->F, a = S->heads, d = S->d, n = r - l;
  double *qkv = zalloc((size_t)n * 3 * A);
  double *tmp = zalloc((size_t)n * H);
  for (int li = 0; li < S->n_layers; ++li) {
    const or_params *p = &S->p[li];
    or_layer_state *L = &S->st[li];
    /* layer input rows [l, r): the stage input, or the previous layer's output */
    for (int t = 0; t < n; ++t) {
      const double *src;
      if (li == 0)
        src = x + (size_t)t * H;
      else
        src = tmp + (size_t)t * H; /* previous layer's output, kept in tmp */
      memcpy(L->x + (size_t)(l + t) * H, src, H * sizeof(double));
    }
    for (int t = l; t < r; ++t)
      ln_row(H, S->eps, L->x + (size_t)t * H, p->ln1_g, p->ln1_b, L->u + (size_t)t * H,
             &L->mean1[t], &L->rstd1[t]);
    mm_nt_bias(n, 3 * A, H, L->u + (size_t)l * H, p->w_qkv, p->b_qkv, qkv);
    for (int t = 0; t < n; ++t) {
      memcpy(L->q + (size_t)(l + t) * A, qkv + (size_t)t * 3 * A, A * sizeof(double));
      memcpy(L->kc + (size_t)(l + t) * A, qkv + (size_t)t * 3 * A + A, A * sizeof(double));
      memcpy(L->vc + (size_t)(l + t) * A, qkv + (size_t)t * 3 * A + 2 * A, A * sizeof(double));
    }
    /* attention: each query row of each head over keys 0..t */
#pragma omp parallel if ((long)n * a * r * d > 200000)
    {
      double *Pl = zalloc((size_t)S->Lmax);
#pragma omp for collapse(2) schedule(static)
      for (int t = l; t < r; ++t)
        for (int h = 0; h < a; ++h) {
          attn_probs(S, L, t, h, Pl);
          double *o = L->o + (size_t)t * A + h * d;
          for (int j = 0; j < d; ++j) {
            double acc = 0.0;
            for (int s = 0; s <= t; ++s) acc += Pl[s] * L->vc[(size_t)s * A + h * d + j];
            o[j] = acc;
          }
        }
      free(Pl);
    }
    mm_nt_bias(n, H, A, L->o + (size_t)l * A, p->w_o, p->b_o, L->x1 + (size_t)l * H);
    for (size_t i = 0; i < (size_t)n * H; ++i) L->x1[(size_t)l * H + i] += L->x[(size_t)l * H + i];
    for (int t = l; t < r; ++t)
      ln_row(H, S->eps, L->x1 + (size_t)t * H, p->ln2_g, p->ln2_b, L->u2 + (size_t)t * H,
             &L->mean2[t], &L->rstd2[t]);
    mm_nt_bias(n, F, H, L->u2 + (size_t)l * H, p->w1, p->b1, L->z + (size_t)l * F);
    for (size_t i = 0; i < (size_t)n * F; ++i) L->g[(size_t)l * F + i] = or_gelu(L->z[(size_t)l * F + i]);
    /* y = x1 + W_2 g + b_2 */
    double *out = (li == S->n_layers - 1) ? y : tmp;
    double *f2 = zalloc((size_t)n * H);
    mm_nt_bias(n, H, F, L->g + (size_t)l * F, p->w2, p->b2, f2);
    for (size_t i = 0; i < (size_t)n * H; ++i) out[i] = L->x1[(size_t)l * H + i] + f2[i];
    free(f2);
  }
  free(qkv);
  free(tmp);
  S->cached_len = r;
  S->bwd_frontier = r;
  return OR_OK;
}

/* Backward of slice [l, r): dy, dx are [r-l][H]; slices must arrive in reverse
 * order (r equal to the current backward frontier).  Gradients accumulate (+=). */
int or_backward(or_stage *S, int l, int r, const double *dy, double *dx) {
  if (!S || !dy || !dx || l < 0 || r <= l || r > S->Lmax) return OR_ERR_INVALID;
  if (r != S->bwd_frontier) return OR_ERR_ORDER;
  const int H = S->H, A = S->A, F = S->F, a = S->heads, d = S->d, n = r - l;
  const double scale = 1.0 / sqrt((double)d);
  double *dcur = zalloc((size_t)n * H); /* gradient w.r.t. this layer's output, rows [l,r) */
  memcpy(dcur, dy, (size_t)n * H * sizeof(double));
  double *dg = zalloc((size_t)n * F), *dz = zalloc((size_t)n * F);
  double *du2 = zalloc((size_t)n * H), *dq = zalloc((size_t)n * A);
  double *dqkv = zalloc((size_t)n * 3 * A), *du = zalloc((size_t)n * H);
  double *dyabs = zalloc((size_t)S->Lmax * H);
  double *dzabs = zalloc((size_t)S->Lmax * F);
  double *dqkvabs = zalloc((size_t)S->Lmax * 3 * A);
  for (int li = S->n_layers - 1; li >= 0; --li) {
    const or_params *p = &S->p[li];
    or_grads *G = &S->gr[li];
    or_layer_state *L = &S->st[li];
    memcpy(dyabs + (size_t)l * H, dcur, (size_t)n * H * sizeof(double));
    /* FFN: y = x1 + W2 g + b2 */
    acc_wgrad_desc(l, r, H, F, dyabs, L->g, G->w2, G->b2);
    mm_nn(n, F, H, dcur, p->w2, dg);
    for (size_t i = 0; i < (size_t)n * F; ++i) dz[i] = dg[i] * or_gelu_grad(L->z[(size_t)l * F + i]);
    memcpy(dzabs + (size_t)l * F, dz, (size_t)n * F * sizeof(double));
    acc_wgrad_desc(l, r, F, H, dzabs, L->u2, G->w1, G->b1);
    mm_nn(n, H, F, dz, p->w1, du2);
    /* LN2 and the residual: dx1 = dy + LN2^T(du2) */
    for (int t = r - 1; t >= l; --t) {
      const double *x1 = L->x1 + (size_t)t * H;
      const double *dut = du2 + (size_t)(t - l) * H;
      const double mean = L->mean2[t], rstd = L->rstd2[t];
      for (int i = 0; i < H; ++i) {
        G->ln2_g[i] += dut[i] * ((x1[i] - mean) * rstd);
        G->ln2_b[i] += dut[i];
      }
      double *dx1 = L->dx1 + (size_t)t * H;
      ln_row_bwd(H, x1, mean, rstd, p->ln2_g, dut, dx1);
      for (int i = 0; i < H; ++i) dx1[i] += dcur[(size_t)(t - l) * H + i];
    }
    /* output projection: x1 = x + W_o o + b_o */
    acc_wgrad_desc(l, r, H, A, L->dx1, L->o, G->w_o, G->b_o);
    mm_nn(n, A, H, L->dx1 + (size_t)l * H, p->w_o, L->dob + (size_t)l * A);
    /* attention backward: dq rows; dK/dV buffer for keys 0..t, queries descending */
#pragma omp parallel if ((long)n * a * r * d > 200000)
    {
      double *Pl = zalloc((size_t)S->Lmax), *dP = zalloc((size_t)S->Lmax);
#pragma omp for schedule(static)
      for (int h = 0; h < a; ++h)
        for (int t = r - 1; t >= l; --t) {
          attn_probs(S, L, t, h, Pl);
          const double *dob = L->dob + (size_t)t * A + h * d;
          const double *q = L->q + (size_t)t * A + h * d;
          double D = 0.0;
          for (int s = 0; s <= t; ++s) {
            const double *v = L->vc + (size_t)s * A + h * d;
            double acc = 0.0;
            for (int j = 0; j < d; ++j) acc += dob[j] * v[j];
            dP[s] = acc;
            D += Pl[s] * acc;
          }
          double *dqt = dq + (size_t)(t - l) * A + h * d;
          for (int j = 0; j < d; ++j) dqt[j] = 0.0;
          for (int s = 0; s <= t; ++s) {
            const double dS = Pl[s] * (dP[s] - D);
            const double *k = L->kc + (size_t)s * A + h * d;
            double *dkr = L->dk + (size_t)s * A + h * d;
            double *dvr = L->dv + (size_t)s * A + h * d;
            for (int j = 0; j < d; ++j) {
              dqt[j] += dS * k[j] * scale;
              dkr[j] += dS * q[j] * scale;
              dvr[j] += Pl[s] * dob[j];
            }
          }
        }
      free(Pl);
      free(dP);
    }
    /* QKV projection: keys/values of [l, r) are complete in the buffer now */
    for (int t = 0; t < n; ++t) {
      memcpy(dqkv + (size_t)t * 3 * A, dq + (size_t)t * A, A * sizeof(double));
      memcpy(dqkv + (size_t)t * 3 * A + A, L->dk + (size_t)(l + t) * A, A * sizeof(double));
      memcpy(dqkv + (size_t)t * 3 * A + 2 * A, L->dv + (size_t)(l + t) * A, A * sizeof(double));
    }
    memcpy(dqkvabs + (size_t)l * 3 * A, dqkv, (size_t)n * 3 * A * sizeof(double));
    acc_wgrad_desc(l, r, 3 * A, H, dqkvabs, L->u, G->w_qkv, G->b_qkv);
    mm_nn(n, H, 3 * A, dqkv, p->w_qkv, du);
    /* LN1 and the residual: dx = dx1 + LN1^T(du) */
    for (int t = r - 1; t >= l; --t) {
      const double *xr = L->x + (size_t)t * H;
      const double *dut = du + (size_t)(t - l) * H;
      const double mean = L->mean1[t], rstd = L->rstd1[t];
      for (int i = 0; i < H; ++i) {
        G->ln1_g[i] += dut[i] * ((xr[i] - mean) * rstd);
        G->ln1_b[i] += dut[i];
      }
      double *dxt = dcur + (size_t)(t - l) * H;
      ln_row_bwd(H, xr, mean, rstd, p->ln1_g, dut, dxt);
      for (int i = 0; i < H; ++i) dxt[i] += L->dx1[(size_t)t * H + i];
    }
  }
  memcpy(dx, dcur, (size_t)n * H * sizeof(double));
  free(dcur);
  free(dg);
  free(dz);
  free(du2);
  free(dq);
  free(dqkv);
  free(du);
  free(dyabs);
  free(dzabs);
  free(dqkvabs);
  S->bwd_frontier = l;
  return OR_OK;
}

/* Copy cache rows [0, cached_len) of one layer: which = 0 -> K, 1 -> V,
 * 2 -> dK buffer, 3 -> dV buffer.  Returns the number of rows copied. */
int or_get_cache(const or_stage *S, int layer, int which, double *out) {
  if (!S || layer < 0 || layer >= S->n_layers || which < 0 || which > 3) return OR_ERR_INVALID;
  const or_layer_state *L = &S->st[layer];
  const double *src = which == 0 ? L->kc : which == 1 ? L->vc : which == 2 ? L->dk : L->dv;
  memcpy(out, src, (size_t)S->cached_len * S->A * sizeof(double));
  return S->cached_len;
}

int or_cached_len(const or_stage *S) { return S->cached_len; }
int or_bwd_frontier(const or_stage *S) { return S->bwd_frontier; }

/* ------------------------------------------------------------ slicing DP */

static int cmp_i64(const void *a, const void *b) {
  const int64_t x = *(const int64_t *)a, y = *(const int64_t *)b;
  return (x > y) - (x < y);
}

/*
 * Optimal slicing (Sec. 3.3).  Units: the sequence has U units of `unit`
 * tokens; cost[(k-1)*U + j] is t(k units long, j units of context), used only
 * where k + j <= U (Eq. 4 cost t_i = t(l_i, sum_{j<i} l_j)).
 *
 * For every candidate t_max (the distinct table values, ascending), solve
 * Eq. 8 -- S*(i) = min_k S*(i-k) + t(k, i-k) over t(k, i-k) <= t_max, with
 * S*(0) = 0 -- remembering the minimising k (Algorithm 1 reads the r_{i-k} of
 * its argmin as S*(i-k)), and score the threshold by Eq. 6:
 * S*(U) + (K-1) t_max.  The smallest score over thresholds is T* (Eq. 5-7).
 * Ties: k is scanned ascending and replaced only by a strictly smaller value;
 * thresholds are scanned ascending and the best replaced only by a strictly
 * smaller score.  Enumeration stops once K * t_max exceeds the best score
 * ("Optimization" paragraph after Algorithm 1).  With eps > 0 the thresholds
 * are taken in windows: from the smallest threshold v not yet covered, only the
 * largest threshold <= v + eps is evaluated.  Every threshold then has an
 * evaluated one at most eps above it, which yields the paper's bound of K * eps
 * on the gap to the optimum even where the table values are sparse (skipping
 * every threshold closer than eps to the last evaluated one, read literally,
 * does not).  eps = 0 evaluates every distinct value.
 * The reported T is Eq. 5 evaluated on the chosen slicing.
 *
 * Returns 0, or OR_ERR_INVALID on bad arguments or a negative used cost.
 * out_units receives the slice lengths in units (capacity U).
 */
int or_dp_optimal_slicing(const int64_t *cost, int U, int K, int64_t eps, int *out_units,
                          int *out_M, int64_t *out_T, int64_t *out_tmax, int *out_evaluated) {
  if (!cost || U < 1 || K < 1 || eps < 0 || !out_units || !out_M || !out_T) return OR_ERR_INVALID;
  size_t nvals = 0;
  int64_t *vals = (int64_t *)malloc(sizeof(int64_t) * (size_t)U * (U + 1) / 2);
  for (int k = 1; k <= U; ++k)
    for (int j = 0; j + k <= U; ++j) {
      const int64_t c = cost[(size_t)(k - 1) * U + j];
      if (c < 0) {
        free(vals);
        return OR_ERR_INVALID;
      }
      vals[nvals++] = c;
    }
  qsort(vals, nvals, sizeof(int64_t), cmp_i64);
  size_t nu = 0;
  for (size_t i = 0; i < nvals; ++i)
    if (nu == 0 || vals[i] != vals[nu - 1]) vals[nu++] = vals[i];

  const int64_t INF = INT64_MAX;
  int64_t *Sst = (int64_t *)malloc(sizeof(int64_t) * (U + 1));
  int *qk = (int *)malloc(sizeof(int) * (U + 1));
  int64_t best = INF, best_tmax = -1;
  int best_M = 0, evaluated = 0;
  int *tmp = (int *)malloc(sizeof(int) * (U + 1));
  size_t next = 0;
  while (next < nu) {
    const int64_t v = vals[next];
    /* stop: any slicing whose largest slice costs >= v has T >= K * v */
    if (best != INF && (double)K * (double)v > (double)best) break;
    size_t tj = next;
    while (tj + 1 < nu && vals[tj + 1] <= v + eps) ++tj;
    next = tj + 1;
    const int64_t tmax = vals[tj];
    ++evaluated;
    Sst[0] = 0;
    for (int i = 1; i <= U; ++i) {
      Sst[i] = INF;
      qk[i] = 0;
      for (int k = 1; k <= i; ++k) {
        const int64_t c = cost[(size_t)(k - 1) * U + (i - k)];
        if (c > tmax || Sst[i - k] == INF) continue;
        const int64_t v = Sst[i - k] + c;
        if (v < Sst[i]) {
          Sst[i] = v;
          qk[i] = k;
        }
      }
    }
    if (Sst[U] == INF) continue;
    const int64_t T = Sst[U] + (int64_t)(K - 1) * tmax;
    if (T < best) {
      best = T;
      best_tmax = tmax;
      int m = 0;
      for (int i = U; i > 0; i -= qk[i]) tmp[m++] = qk[i];
      best_M = m;
      for (int i = 0; i < m; ++i) out_units[i] = tmp[m - 1 - i]; /* prepend order */
    }
  }
  free(tmp);
  free(vals);
  free(Sst);
  free(qk);
  if (best == INF) return OR_ERR_INVALID;
  /* Eq. 5 on the chosen slicing */
  int64_t sum = 0, mx = 0;
  int ctx = 0;
  for (int i = 0; i < best_M; ++i) {
    const int64_t c = cost[(size_t)(out_units[i] - 1) * U + ctx];
    sum += c;
    if (c > mx) mx = c;
    ctx += out_units[i];
  }
  *out_M = best_M;
  *out_T = sum + (int64_t)(K - 1) * mx;
  if (out_tmax) *out_tmax = best_tmax;
  if (out_evaluated) *out_evaluated = evaluated;
  return OR_OK;
}
