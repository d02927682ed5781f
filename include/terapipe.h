/*
 * terapipe.h -- C ABI of the TeraPipe stage engine for MI355X (gfx950).
 *
 * Paper: Li et al., "TeraPipe: Token-Level Pipeline Parallelism for Training
 * Large-Scale Language Models", ICML 2021 (arXiv 2102.07988).
 *
 * A pipeline cell ("stage") is a run of consecutive Transformer layers placed
 * on one device (Sec. 3.2).  TeraPipe splits one training sequence of length L
 * into token slices s_1..s_M and runs each cell over the slices in order: slice
 * i's self-attention needs the keys and values of every earlier position of the
 * same sequence (Eq. 2: token t attends to positions s <= t), and its
 * feed-forward part only its own tokens (Eq. 3).  The backward pass runs the
 * slices in reverse.  The cost of a slice depends on its length and on the
 * length of the prefix before it (Eq. 4), and the optimal slicing minimises the
 * pipeline latency of Eq. 5 by the dynamic program of Sec. 3.3 (Eq. 6-8,
 * Algorithm 1).
 *
 * Layer model: a GPT-3 pre-LayerNorm block (the setting of Sec. 4):
 *   u = LN1(x); [q,k,v] = W_qkv u + b_qkv; o = causal multi-head attention
 *   (heads of width d = hidden/heads, scale 1/sqrt(d), key s <= query t);
 *   x1 = x + W_o o + b_o; u2 = LN2(x1); y = x1 + W_2 GELU(W_1 u2 + b_1) + b_2,
 *   GELU in its tanh form, LayerNorm with biased variance and eps.
 *
 * Conventions
 *  - Every device pointer is caller-owned device memory (HBM) on the device
 *    that is current when tp_stage_init is called; the stage keeps pointers
 *    only.  Matrices are row-major; weight matrices are [out][in].
 *  - Activations and parameters use the stage dtype (bf16 or fp32); gradients
 *    are always fp32 and are ACCUMULATED (+=): the caller zeroes them, or
 *    starts the sequence with tp_kv_prefix_reset_ex(TP_SEQ_OVERWRITE_GRADS)
 *    to have its gradients stored in place of the old contents.
 *  - Precision of a bf16 stage whose head width is 64 or 128: matrix products
 *    take bf16 operands with fp32 accumulation, except that (1) the residual
 *    stream inside the stage (the input of every layer but the first, and x1)
 *    is kept in fp32, and (2) the query/key/value product and the attention
 *    scores run on fp16 operands: the LN1 output, a copy of W_qkv converted to
 *    fp16 by tp_kv_prefix_reset (so W_qkv must not change during a sequence,
 *    and its entries must lie within the fp16 range), q, k and the forward's
 *    v; the forward's softmax weights and the backward's dS are fp16 where
 *    they meet those operands.  With bf16 there, the rounding of the LN1 output
 *    and of q and k is amplified by sharp softmax rows (e.g. logits of standard
 *    deviation ~5 at hidden size 12288 with N(0, 0.02) weights) to several
 *    percent of relative error in the gradients; fp16 keeps 3 more mantissa
 *    bits at the same matrix-core rate.  Gradient-side operands stay bf16.
 *    Other bf16 stages (head widths 16, 32) use bf16 throughout.
 *  - Calls are asynchronous on the stage's stream unless stated otherwise; a
 *    HIP launch failure is reported as TP_ERR_HIP.  Argument and ordering
 *    errors are detected on the host before anything is enqueued and leave
 *    the stage unchanged.
 *  - One stage object per stream; calls on one stage must not overlap.
 */
#ifndef TERAPIPE_H
#define TERAPIPE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  TP_OK = 0,
  TP_ERR_INVALID = -1,     /* null pointer, bad size or bad configuration */
  TP_ERR_ORDER = -2,       /* slice out of order (see tp_slice_forward/backward) */
  TP_ERR_UNSUPPORTED = -3, /* valid but unsupported configuration (e.g. head width) */
  TP_ERR_WORKSPACE = -4,   /* workspace too small or not 256-byte aligned */
  TP_ERR_HIP = -5          /* a HIP runtime call or kernel launch failed */
} tp_status;

typedef enum { TP_DTYPE_BF16 = 0, TP_DTYPE_FP32 = 1 } tp_dtype;

/* How weight gradients are formed.  PER_SLICE: every backward slice adds its
 * dW contribution (fp32 read-modify-write of all weight gradients per slice).
 * DEFERRED: backward slices keep the per-token output gradients, and the
 * weight-gradient GEMMs run once over the whole sequence (reduction length =
 * number of cached tokens) when the backward frontier reaches position 0.
 * Both give the same gradients up to fp32 summation order.  Bias and
 * LayerNorm-parameter gradients (column sums over tokens) follow the same
 * mode: per slice, or once per sequence from kept per-token gradients. */
typedef enum { TP_WGRAD_PER_SLICE = 0, TP_WGRAD_DEFERRED = 1 } tp_wgrad_mode;

typedef struct {
  int n_layers;   /* layers in this stage, >= 1 */
  int hidden;     /* H; FFN width is 4H */
  int heads;      /* a; head width d = H / a must be 16, 32, 64 or 128; H % 8 == 0, H <= 16384 */
  int max_seq;    /* largest sequence length L the stage will see */
  int dtype;      /* tp_dtype */
  int wgrad_mode; /* tp_wgrad_mode */
  float ln_eps;   /* LayerNorm epsilon (1e-5 in the GPT-3 setting) */
  int batch;      /* b: sequences that move through the stage together as one batch slice
                     (Sec. 3.4, slicing the batch and token dimensions jointly); 0 means 1,
                     at most 64.  Token t of sequence s is row t * b + s of every
                     slice tensor below, so a slice [l, r) is (r-l) * b consecutive rows. */
  int op_parts;   /* p: the stage is one device's shard of p-way operation partitioning
                     inside each layer (the #Op column of Table 1): heads / p heads and
                     4H / p FFN units on the full residual stream, the output and FC2
                     projections' partial sums taken as this device's whole sum (the
                     all-reduce across the p devices is left out).  0 means 1; heads and
                     4H must be multiples of p.  Weight shapes below use A = H / p and
                     F = 4H / p (A = H, F = 4H for p = 1). */
} tp_stage_config;

/* Parameters (stage dtype) or gradients (fp32) of one layer.  Shapes (A and F
 * as in tp_stage_config.op_parts): ln*_g, ln*_b, b_o, b_fc2: [H]; w_qkv: [3A][H]
 * (rows: q, then k, then v; local head h owns rows h*d..h*d+d-1 of each);
 * b_qkv: [3A]; w_o: [H][A]; w_fc1: [F][H]; b_fc1: [F]; w_fc2: [H][F]. */
typedef struct {
  void *ln1_g, *ln1_b, *w_qkv, *b_qkv, *w_o, *b_o;
  void *ln2_g, *ln2_b, *w_fc1, *b_fc1, *w_fc2, *b_fc2;
} tp_layer_ptrs;

typedef struct tp_stage tp_stage;

/* Bytes of device workspace the stage needs for `cfg` (K/V cache, fp32 dK/dV
 * buffer, per-token activation and gradient arenas, scratch).  0 if cfg is
 * invalid.  Host only. */
size_t tp_stage_workspace_bytes(const tp_stage_config *cfg);

/* Create a stage: one pipeline cell, the run of consecutive layers that one
 * device holds and runs over every slice of a sequence (Sec. 3.2; the cell
 * partition of the layers is the unit of the pipeline in Sec. 3.3).
 * params / grads: arrays of cfg->n_layers entries.
 * workspace: >= tp_stage_workspace_bytes(cfg) bytes of device memory,
 * 256-byte aligned, owned by the caller and used only by this stage until
 * tp_stage_destroy.  stream: a hipStream_t (NULL = default stream) on which
 * all of the stage's device work is enqueued.  Host only: nothing is enqueued.
 * The new stage holds no sequence: its dK/dV buffer holds whatever the
 * workspace held and the fp16 W_qkv copy is not taken, so every slice call
 * returns TP_ERR_ORDER until tp_kv_prefix_reset starts a sequence.
 * Errors: TP_ERR_INVALID, TP_ERR_UNSUPPORTED, TP_ERR_WORKSPACE. */
tp_status tp_stage_init(const tp_stage_config *cfg, const tp_layer_ptrs *params,
                        const tp_layer_ptrs *grads, void *workspace, size_t workspace_bytes,
                        void *stream, tp_stage **out);

/* Free the host-side stage object.  Does not synchronise or free device memory. */
void tp_stage_destroy(tp_stage *stage);

/* Start a new sequence (required before the first slice call after
 * tp_stage_init or tp_profile_slice_cost): no cached tokens, backward frontier 0, and the fp32
 * dK/dV buffer zeroed (enqueued on the stream; a fill kernel, no memset node);
 * on the mixed-precision path (see Conventions) also the fp16 copy of every
 * layer's W_qkv taken.
 * This is the empty prefix state of Eq. 2: the keys and values of positions
 * before the first slice, which every later slice's attention sums over,
 * start out empty (Sec. 3.2: the cell keeps them from slice to slice).
 * Parameter gradients are not touched. */
tp_status tp_kv_prefix_reset(tp_stage *stage);

/* Flags of tp_kv_prefix_reset_ex. */
#define TP_SEQ_OVERWRITE_GRADS 1u
#define TP_SEQ_REUSE_WQKV_COPY 2u

/* tp_kv_prefix_reset, plus per-sequence flags (0 = tp_kv_prefix_reset).
 * TP_SEQ_OVERWRITE_GRADS: the sequence's first write of each parameter
 * gradient stores its value instead of adding it, so the gradients end up as
 * this sequence's alone, exactly as if the caller had zeroed them first (a
 * training iteration's first sequence; later sequences of the same iteration
 * start with flags 0 and add).  The gradient buffers' earlier contents are
 * never read and may be anything, NaN included.  The first write is the
 * first backward slice with TP_WGRAD_PER_SLICE, the backward slice that
 * reaches position 0 with TP_WGRAD_DEFERRED (the only one that writes
 * gradients); a DEFERRED sequence whose backward never reaches 0 writes none.
 * This changes no value the method computes (Sec. 4: TeraPipe trains with
 * the same gradients as whole-sequence processing); it saves the read of
 * every fp32 gradient in the weight-gradient GEMMs' epilogues and the
 * caller's zeroing pass.
 * TP_SEQ_REUSE_WQKV_COPY (mixed-precision path, see Conventions; no effect
 * elsewhere): W_qkv is unchanged since the fp16 copy was last taken (by the
 * previous sequence start or profiling call on this stage), so that copy is
 * kept instead of converting W_qkv again; with no copy taken yet it is taken.
 * For the later sequences or batch slices (Sec. 3.4) of one training
 * iteration, which all use the same weights.  The caller vouches for it: after
 * W_qkv has changed, the forward's query/key/value product would run on the
 * old weights.
 * Errors: TP_ERR_INVALID (null stage, unknown flag bits; nothing enqueued),
 * TP_ERR_HIP. */
tp_status tp_kv_prefix_reset_ex(tp_stage *stage, unsigned flags);

/* Forward of token slice [l, r) through every layer (Sec. 3.2).
 * x: [r-l][b][H] stage input rows, y: [r-l][b][H] stage output rows (stage
 * dtype, device; b = cfg.batch, token-major).  Requires 0 <= l < r <= max_seq
 * (else TP_ERR_INVALID), a sequence started by tp_kv_prefix_reset, l equal
 * to the number of cached tokens and no backward call since that reset
 * (else TP_ERR_ORDER: a
 * slice's backward needs the forward of every later slice, so a forward after
 * backward has begun is misuse).  Appends the slice's keys
 * and values to each layer's cache, saves what backward needs, and sets the
 * cached length and the backward frontier to r.  x and y must not overlap and
 * must be 16-byte aligned (else TP_ERR_INVALID). */
tp_status tp_slice_forward(tp_stage *stage, int l, int r, const void *x, void *y);

/* For callers that cannot allocate (code under stream capture, serving loops,
 * harnesses that forbid allocation): tp_slice_forward with the partial sums of
 * its kernels (split-K GEMM partials, key-split attention partials) in the
 * library's static per-device scratch array of 32 MiB instead of the stage
 * workspace.  Nothing is allocated: no device or host memory, no events (kernel
 * timing is not recorded for this call).  The kernels and their split plans are
 * those tp_slice_forward would use, so the results are the same.  The plan is
 * made on the host first: a slice whose largest partial-sum buffer exceeds
 * 32 MiB is rejected with TP_ERR_WORKSPACE and the stage left unchanged (this
 * check precedes the one for a started sequence).  The
 * array keeps whatever the last call left in it (no contents carry meaning
 * across calls); calls that overlap on one device race on it, as do
 * overlapping calls of different stages on one device.  Other arguments,
 * checks and effects as tp_slice_forward. */
tp_status tp_slice_forward_static(tp_stage *stage, int l, int r, const void *x, void *y);

/* Backward of token slice [l, r) through every layer, in reverse layer order.
 * The backward pass of a cell runs over the slices in the reverse of their
 * forward order (the last paragraph of Sec. 3.3 applies the same slicing
 * analysis to the backward time t_bwd; Sec. 3.2 for the cell pipeline):
 * gradients that a slice's queries send to earlier positions' keys and values
 * must be complete before those positions' own backward runs.
 * dy: [r-l][b][H] gradient of the stage output rows, dx: [r-l][b][H] gradient
 * of the stage input rows (stage dtype, device).  Requires 0 <= l < r and r equal to
 * the backward frontier (slices arrive in reverse order; their boundaries need
 * not match the forward slicing) in a sequence started by tp_kv_prefix_reset,
 * else TP_ERR_ORDER / TP_ERR_INVALID (argument checks come first).  Adds
 * this slice's contributions to the parameter gradients (stores them where
 * the sequence started with TP_SEQ_OVERWRITE_GRADS and this is its first
 * gradient write, see tp_kv_prefix_reset_ex); the gradient that
 * queries in [l, r) send to earlier keys/values is added to the dK/dV buffer.
 * Sets the frontier to l; in DEFERRED mode the weight-gradient GEMMs run when
 * l reaches 0.  dy and dx must not overlap and must be 16-byte aligned. */
tp_status tp_slice_backward(tp_stage *stage, int l, int r, const void *dy, void *dx);

/* Measure the per-slice costs t_fwd(len, ctx) and t_bwd(len, ctx) of Eq. 4 on
 * this device: for every len in lens[0..n_lens) and ctx in ctxs[0..n_ctxs),
 * position the stage after ctx cached tokens, then time `reps` forward and
 * backward runs of slice [ctx, ctx+len) (after `warmup` untimed runs) with HIP
 * events and store the medians in nanoseconds at [i_len * n_ctxs + i_ctx] of
 * t_fwd_ns / t_bwd_ns (host arrays).  Entries with len + ctx > max_seq get -1.
 * In DEFERRED mode t_bwd excludes the once-per-sequence weight-gradient GEMMs
 * and bias / LayerNorm-parameter reductions.
 * Synchronous.  Overwrites the K/V cache, the arenas and the parameter
 * gradients with meaningless values and ends any sequence: slice calls return
 * TP_ERR_ORDER until tp_kv_prefix_reset; zero the gradients afterwards (or
 * start the next sequence with TP_SEQ_OVERWRITE_GRADS). */
tp_status tp_profile_slice_cost(tp_stage *stage, const int *lens, int n_lens, const int *ctxs,
                                int n_ctxs, int warmup, int reps, int64_t *t_fwd_ns,
                                int64_t *t_bwd_ns);

/* Optimal slicing of a sequence of L_units * unit tokens for a pipeline of K
 * cells (Sec. 3.3).  cost (host, int64, [L_units][L_units]):
 * cost[(k-1)*L_units + j] = t(k*unit tokens, j*unit tokens of context) -- the
 * per-slice forward+backward time; entries with k + j > L_units are ignored.
 * For every distinct cost value t_max in ascending order it solves Eq. 8 with
 * Algorithm 1 (smallest S*(i) over slice lengths k with t(k, i-k) <= t_max)
 * and scores S*(L) + (K-1) t_max (Eq. 6-7); enumeration stops once
 * K * t_max exceeds the best score.  eps_ns > 0 evaluates only the largest
 * threshold within eps of each not-yet-covered one (gap to the optimum at most
 * K * eps).  Ties: shortest last slice (k ascending, strict improvement), then
 * smallest t_max.  Outputs: out_lens[0..*out_M) slice lengths in tokens
 * (capacity L_units), *out_T = Eq. 5 latency of that slicing.  Host only,
 * deterministic.  Errors: TP_ERR_INVALID (null pointer, L_units < 1, unit < 1,
 * K < 1, eps_ns < 0, a negative cost among the used entries). */
tp_status tp_dp_optimal_slicing(const int64_t *cost, int L_units, int unit, int K, int64_t eps_ns,
                                int *out_lens, int *out_M, int64_t *out_T);

/* Batch split of Sec. 3.4 (slicing the batch and token dimensions jointly):
 * a batch of B sequences is cut into groups of b_1 + ... + b_D = B sequences,
 * each group pipelined with its own optimal token slicing, minimising
 * T_{b_1} + ... + T_{b_D} (a one-dimensional knapsack).  T_b (host, int64,
 * [B]): T_b[b-1] = the optimal latency of a group of b sequences (e.g. *out_T
 * of tp_dp_optimal_slicing on the cost table of a stage with batch b); a
 * negative entry marks a size that may not be used.  Outputs: out_sizes (capacity
 * B) the group sizes, largest first, *out_D their number, *out_total the
 * minimal sum.  Ties: for each prefix total the last group is the smallest
 * size reaching the minimum.  Host only, deterministic.  Errors:
 * TP_ERR_INVALID (null pointer, B < 1, no combination of usable sizes sums
 * to B, overflow). */
tp_status tp_dp_batch_split(const int64_t *T_b, int B, int *out_sizes, int *out_D,
                            int64_t *out_total);

/* Joint plan of Sec. 3.4: tp_dp_optimal_slicing on the cost table of every
 * group size b = 1..B, then tp_dp_batch_split over the resulting latencies.
 * costs (host, int64, [B][L_units][L_units]): plane b-1 is the table of a batch
 * slice of b sequences, in the layout of tp_dp_optimal_slicing.  Outputs:
 * out_T_b[B] the latency of each size; out_sizes / *out_D / *out_total as
 * tp_dp_batch_split; for group g, out_M[g] slices with token lengths
 * out_lens[g * L_units .. g * L_units + out_M[g]) (capacities: out_sizes,
 * out_M: B; out_lens: B * L_units).  Errors: those of the two calls. */
tp_status tp_dp_joint_slicing(const int64_t *costs, int B, int L_units, int unit, int K,
                              int64_t eps_ns, int *out_sizes, int *out_D, int *out_lens,
                              int *out_M, int64_t *out_T_b, int64_t *out_total);

/* Cost estimate of Sec. 3.3 (Eq. 9): t(i, j) = t(i, 0) + t_ctx(i, j) with the
 * context overhead t_ctx(i, j) = a0 + a1 i + a2 j + a3 i j (i = slice length,
 * j = context length, both in tokens) fitted by least squares.
 *
 * tp_fit_ctx_model: t0_ns (host, [L_units]): t0_ns[k-1] = t(k*unit tokens, 0).
 * Samples s = 0..n_samples-1 (host arrays): a slice of s_len[s] tokens (a
 * multiple of unit) after s_ctx[s] >= 1 tokens of context cost s_t_ns[s]; its
 * overhead is s_t_ns[s] - t0_ns[s_len[s]/unit - 1].  Writes coef[0..3] =
 * a0 (ns), a1, a2 (ns per token), a3 (ns per token^2) minimising the sum of
 * squared overhead residuals.  Host only, deterministic.  Errors:
 * TP_ERR_INVALID (null pointer, n_samples < 4, a sample off the unit grid or
 * past L_units*unit tokens, a negative time, or samples that do not determine
 * the four coefficients, e.g. a single length or a single context). */
tp_status tp_fit_ctx_model(const int64_t *t0_ns, int L_units, int unit, const int *s_len,
                           const int *s_ctx, const int64_t *s_t_ns, int n_samples, double *coef);

/* Cost table for tp_dp_optimal_slicing from the Eq. 9 model: cost (host,
 * [L_units][L_units]) entry (k-1)*L_units + j = t0_ns[k-1] for j = 0, and
 * t0_ns[k-1] + llround(a0 + a1 i + a2 c + a3 i c) at i = k*unit, c = j*unit
 * for j > 0, clamped at 0; entries with k + j > L_units are -1.  Host only.
 * Errors: TP_ERR_INVALID (null pointer, L_units < 1, unit < 1, negative t0). */
tp_status tp_cost_table_from_model(const int64_t *t0_ns, int L_units, int unit, const double *coef,
                                   int64_t *cost);

/* Profile in model mode (Sec. 3.3, Eq. 9): measure t(i, 0) = t_fwd + t_bwd for
 * every length i = unit .. L_units*unit with tp_profile_slice_cost, measure the
 * subset sub_lens x sub_ctxs (lengths multiples of unit, contexts >= 1; pairs
 * past L_units*unit tokens are skipped), fit the overhead model and write the
 * [L_units][L_units] cost table (layout of tp_cost_table_from_model) and the
 * coefficients coef[0..3].  The stage needs max_seq >= L_units*unit.
 * Synchronous; clobbers the K/V cache, arenas and gradients like
 * tp_profile_slice_cost.  Errors: TP_ERR_INVALID (bad arguments, fewer than 4
 * usable subset points, a subset that does not determine the model), TP_ERR_HIP. */
tp_status tp_profile_cost_model(tp_stage *stage, int L_units, int unit, const int *sub_lens,
                                int n_sub_lens, const int *sub_ctxs, int n_sub_ctxs, int warmup,
                                int reps, int64_t *cost, double *coef);

/* Static description of a status code. */
const char *tp_status_string(tp_status status);

/* Per-kernel-class timing of the stage's launches, for measurement.  When
 * enabled, every launch of an instrumented kernel class is bracketed by HIP
 * events on the stage stream; tp_stage_kernel_stats synchronises the stream
 * and returns, per class, the number of launches, their summed duration and
 * their summed algorithmic flop and HBM-byte counts since the last reset of
 * the counters.  Returns the number of classes written (<= cap), or -1 when
 * the stream or an event could not be read (events recorded under stream
 * capture cannot be): the pending timings are then dropped and the counters
 * reset.  Launches captured into a graph are not timed by this mechanism. */
typedef struct {
  char name[48];
  int64_t launches;
  double total_ms;
  double flops;
  double bytes;
} tp_kernel_stat;

tp_status tp_stage_enable_kernel_timing(tp_stage *stage, int enable);
int tp_stage_kernel_stats(tp_stage *stage, tp_kernel_stat *out, int cap);

/* Measurement helper: dense bf16 matrix-core throughput this device sustains.
 * Runs, on the current device and the given stream (a hipStream_t, NULL =
 * default), two workgroups of 4 waves per compute unit, each wave issuing
 * `iters` x 8 independent 32x32x16 bf16 MFMAs with operands in registers (no
 * memory traffic), after one untimed run, and writes the achieved TFLOP/s of
 * the timed run to *tflops.  sink: device memory of >= 4 bytes per workgroup
 * (2 x compute units), never written in practice (it keeps the work live).
 * Synchronous.  Errors: TP_ERR_INVALID, TP_ERR_HIP. */
tp_status tp_measure_mfma_peak(void *stream, int iters, void *sink, double *tflops);

#ifdef __cplusplus
}
#endif

#endif /* TERAPIPE_H */
