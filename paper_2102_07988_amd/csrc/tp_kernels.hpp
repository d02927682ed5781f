// Launchers of the stage's device kernels.  All pointers are device pointers;
// element types follow the stage dtype (0 = bf16, 1 = fp32) unless the name or
// the comment says fp32.  Every launcher enqueues on `s` and returns the launch
// status.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace tp {

enum Dtype { DT_BF16 = 0, DT_FP32 = 1 };

// GEMM epilogues (what happens to acc = sum_k A(m,k) B(k,n), fp32):
enum EpiKind {
  EPI_STORE = 0,  // C[m][n] = acc (+ bias[n])
  EPI_QKV = 1,    // v = acc + bias[n]; n < H -> q[m][n], n < 2H -> k[m][n-H], else v[m][n-2H]
  EPI_RESID = 2,  // C[m][n] = acc + bias[n] + R[m][n]
  EPI_GELU = 3,   // z = acc + bias[n]; C[m][n] = z; C2[m][n] = GELU(z)
  EPI_DGELU = 4,  // C[m][n] = acc * GELU'(R[m][n])
  EPI_ACC_F32 = 5 // Cf[m][n] += acc (fp32 output, read-modify-write; with
                  // GemmArgs::overwrite, Cf[m][n] = acc without the read)
};

struct GemmArgs {
  int M = 0, N = 0, K = 0;
  const void* A = nullptr;  // A(m,k) = A[m*sam + k*sak]
  long sam = 0, sak = 0;
  const void* B = nullptr;  // B(k,n) = B[k*sbk + n*sbn]
  long sbk = 0, sbn = 0;
  int epi = EPI_STORE;
  const void* bias = nullptr;  // [N], stage dtype; may be null
  void* C = nullptr;           // rows of ldc elements (stage dtype; fp32 for EPI_ACC_F32)
  long ldc = 0;
  const void* R = nullptr;  // residual (EPI_RESID) or pre-activation z (EPI_DGELU)
  long ldr = 0;
  void* C2 = nullptr;  // GELU output (EPI_GELU)
  long ldc2 = 0;
  void *q = nullptr, *k = nullptr, *v = nullptr;  // EPI_QKV destinations, row stride H
  int H = 0;
  // Mixed-precision path of a bf16 stage: A and B are fp16 (the query/key/value
  // product of fp16 LayerNorm output and an fp16 copy of W_qkv); EPI_QKV then
  // writes q, k, v as fp16 and v once more as bf16 to vb.  EPI_RESID: r_f32 /
  // c_f32 mark an fp32 residual input / output (the residual stream of a
  // mixed-precision stage).
  int in_f16 = 0;
  int qkv_f16 = 0;
  void* vb = nullptr;
  int r_f32 = 0, c_f32 = 0;
  // EPI_ACC_F32 only: store acc instead of adding it (the destination's old
  // contents are never read)
  int overwrite = 0;
  // fp32 scratch for split-K partial sums (may be null: no split)
  float* ws = nullptr;
  long ws_elems = 0;
  // set by the launcher: reduction range of one split and the split count
  int k_split = 0, splits = 1;
  // set by the launcher for a split product run as two launches over column
  // groups: columns [0, split_cols) leave `splits` partial planes of split_cols
  // columns, columns [split_cols, N) `splits2` planes of N - split_cols
  // columns after them; 0 for one launch over every column
  int split_cols = 0, splits2 = 0;
  // set by the launcher: output-tile order (0 grid order, 1 XCD super-tiles)
  int walk = 0;
  // Host-side planning: when set, the launcher launches nothing and stores
  // the fp32 scratch elements (split-K partials) its plan for this product
  // takes, 0 without a split.  The caller zeroes *need first.
  long* need = nullptr;
};

hipError_t gemm(int dtype, const GemmArgs& a, hipStream_t s);
// host: the 8-column vector epilogues apply (sizes and alignment)
bool vec8_ok(const GemmArgs& a);
// Generic (any strides, any dtype) tiled FMA GEMM; the bf16 fast path falls back
// to it for shapes it does not cover.
hipError_t gemm_generic(int dtype, const GemmArgs& a, hipStream_t s);

// Prefix-causal attention over a slice: queries t in [l, r), keys s in [0, t].
// q, o: rows [r-l][H] (row i = token l+i); kc, vc: cache rows [Lmax][H] from
// token 0; lse: fp32 [heads][Lmax] (absolute token index).
// A batch of bs sequences shares the token positions: row t * bs + s holds
// token t of sequence s (bs = 1: row t).  Every row-indexed tensor below
// (q, o, dout: the slice's rows; kc, vc, dk, dv: absolute rows) has row stride
// ld = bs * H elements and sequence s starts at column s * H; dq has row stride
// ld_dq and sequence s at column s * dq_seq; lse and D hold one [heads][Lmax]
// plane per sequence.  Kernels take the sequence from blockIdx.z.
struct AttnArgs {
  int l = 0, r = 0, H = 0, heads = 0, d = 0, Lmax = 0;
  int bs = 1, ld = 0;
  float scale = 1.f;
  const void* q = nullptr;
  const void* kc = nullptr;
  const void* vc = nullptr;
  void* o = nullptr;
  float* lse = nullptr;
  // backward
  const void* dout = nullptr;  // the slice's rows
  float* D = nullptr;          // fp32 [bs][heads][Lmax] scratch: rowsum(dO * O)
  void* dq = nullptr;          // the slice's rows, ld_dq elements apart
  long ld_dq = 0, dq_seq = 0;
  float* dk = nullptr;  // fp32 accumulation buffers (absolute rows)
  float* dv = nullptr;
  // Key-range split of the query-parallel kernels (forward, dQ) when their
  // grid is small: blockIdx.z = sequence * nsplit + split, split z takes keys
  // [z * kv_chunk, (z + 1) * kv_chunk), and writes fp32 partials that a
  // combine kernel adds up in split order.  part: [nsplit][(r-l) * bs][H]
  // (rows as in q); ml (forward): [nsplit][bs][heads][r-l] pairs of (running
  // maximum in log2 units, sum of weights).  Scratch of ws_elems floats.
  int nsplit = 1, kv_chunk = 0;
  float* ws = nullptr;
  long ws_elems = 0;
  // Mixed-precision path: q and kc hold fp16, and so does vc in the forward;
  // scores (Q K^T) and, in the forward, P V run on fp16 operands, the dS
  // products of the backward on fp16 dS.  The backward's vc is bf16 (dP = dO
  // V^T and dV = P^T dO keep the gradient side in bf16).
  int f16 = 0;
  // Host-side planning, as GemmArgs::need: the key-split partials' fp32
  // elements (forward: with the running maxima and sums), 0 without a split.
  long* need = nullptr;
  // Backward scratch of pd_elems 16-bit elements for the stored dS planes
  // (matrix-core path): the dK kernel writes dS and the dQ kernel streams it
  // instead of recomputing the scores; slices whose planes do not fit run in
  // query chunks.  Null: the recomputing dQ kernel.
  uint16_t* pd = nullptr;
  long pd_elems = 0;
  // set by the launcher: the planes' base and their query columns
  uint16_t* dst = nullptr;
  long pd_ld = 0;
};
// The arguments of sequence blockIdx.z of the batch as a one-sequence view:
// pointers moved to its columns (element type T) and planes; the row stride
// stays a.ld.
template <typename T>
__device__ inline AttnArgs attn_seq_view(AttnArgs a) {
  const int s = blockIdx.z / a.nsplit;
  if (s == 0) return a;
  const long off = (long)s * a.H, plane = (long)s * a.heads * a.Lmax;
  a.q = (const T*)a.q + off;
  a.kc = (const T*)a.kc + off;
  a.vc = (const T*)a.vc + off;
  if (a.o) a.o = (T*)a.o + off;
  if (a.dout) a.dout = (const T*)a.dout + off;
  if (a.dq) a.dq = (T*)a.dq + s * a.dq_seq;
  if (a.dk) a.dk += off;
  if (a.dv) a.dv += off;
  if (a.lse) a.lse += plane;
  if (a.D) a.D += plane;
  return a;
}
hipError_t attn_fwd(int dtype, const AttnArgs& a, hipStream_t s);
hipError_t attn_bwd(int dtype, const AttnArgs& a, hipStream_t s);

// LayerNorm over rows of H: u = g * (x - mean) * rstd + b.  x is fp32 when
// x_f32, else of the stage dtype.  If x_copy is not null, the input rows are
// also copied there (fp32 when copy_f32).  If u16 is not null, u is written
// once more there as fp16 (bf16 stages only).
hipError_t ln_fwd(int dtype, int n, int H, const void* x, int x_f32, void* x_copy, int copy_f32,
                  const void* g, const void* b, void* u, void* u16, float* mean, float* rstd,
                  float eps, hipStream_t s);
// dx = LN^T(du) + resid (resid may be null); x fp32 when x_f32.
hipError_t ln_bwd(int dtype, int n, int H, const void* du, const void* x, int x_f32,
                  const float* mean, const float* rstd, const void* g, const void* resid, void* dx,
                  hipStream_t s);
// dg[i] += sum_t du[t][i] * xhat[t][i];  db[i] += sum_t du[t][i]   (fp32 outputs;
// with store set, = in place of +=)
hipError_t ln_param_grads(int dtype, int n, int H, const void* du, const void* x, int x_f32,
                          const float* mean, const float* rstd, float* dg, float* db, int store,
                          hipStream_t s);
// dst[i] = fp16(src[i]) for n bf16 values (round to nearest even).
hipError_t cvt_bf16_f16(size_t n, const void* src, void* dst, hipStream_t s);
// out[j] += sum_{i<n} A[i*lda + j], j < N (fp32 output; with store set, = in place of +=)
hipError_t colsum_acc(int dtype, int n, int N, const void* A, long lda, float* out, int store,
                      hipStream_t s);
// dqkv[i][H + j] = dk[l+i][j], dqkv[i][2H + j] = dv[l+i][j] (stage dtype <- fp32)
hipError_t pack_dkv(int dtype, int n, int H, const float* dk, const float* dv, void* dqkv,
                    hipStream_t s);
hipError_t fill_f32(float* p, size_t n, float v, hipStream_t s);
hipError_t copy_rows(int dtype, int n, int H, const void* src, void* dst, hipStream_t s);

}  // namespace tp
