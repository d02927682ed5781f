// Generic kernels of the stage: a strided tiled-FMA GEMM with the fused
// epilogues, straightforward prefix-causal attention forward/backward (one
// block per (query, head)), LayerNorm forward/backward, column reductions.
// These carry the fp32 validation mode and every shape the bf16 fast kernels
// do not take.
#include "tp_common.hpp"
#include "tp_epilogue.hpp"
#include "tp_kernels.hpp"

namespace tp {

// ------------------------------------------------------------- generic GEMM

template <typename T, int EPI>
__global__ __launch_bounds__(256) void gemm_generic_kernel(GemmArgs a) {
  __shared__ float As[16][65];
  __shared__ float Bs[16][65];
  const T* A = (const T*)a.A;
  const T* B = (const T*)a.B;
  const int m0 = blockIdx.y * 64, n0 = blockIdx.x * 64;
  const int tx = threadIdx.x & 15, ty = threadIdx.x >> 4;
  // contiguous dimension of each operand decides the load order (coalescing)
  const bool a_k_fast = a.sak == 1;
  const bool b_n_fast = a.sbn == 1;
  float acc[4][4] = {};
  for (int k0 = 0; k0 < a.K; k0 += 16) {
    for (int e = threadIdx.x; e < 1024; e += 256) {
      int kk, mm;
      if (a_k_fast) {
        kk = e & 15;
        mm = e >> 4;
      } else {
        kk = e >> 6;
        mm = e & 63;
      }
      const int gm = m0 + mm, gk = k0 + kk;
      As[kk][mm] = (gm < a.M && gk < a.K) ? ld(A + (long)gm * a.sam + (long)gk * a.sak) : 0.f;
      int kb, nn;
      if (b_n_fast) {
        kb = e >> 6;
        nn = e & 63;
      } else {
        kb = e & 15;
        nn = e >> 4;
      }
      const int gn = n0 + nn, gkb = k0 + kb;
      Bs[kb][nn] = (gn < a.N && gkb < a.K) ? ld(B + (long)gkb * a.sbk + (long)gn * a.sbn) : 0.f;
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < 16; ++kk) {
      float av[4], bv[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) av[i] = As[kk][ty + 16 * i];
#pragma unroll
      for (int j = 0; j < 4; ++j) bv[j] = Bs[kk][tx + 16 * j];
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] += av[i] * bv[j];
    }
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int m = m0 + ty + 16 * i, n = n0 + tx + 16 * j;
      if (m < a.M && n < a.N) epi1<T, EPI>(a, m, n, acc[i][j]);
    }
}

template <typename T>
static hipError_t gemm_generic_t(const GemmArgs& a, hipStream_t s) {
  if (a.need || a.M <= 0 || a.N <= 0) return hipSuccess;  // no scratch
  dim3 grid(cdiv(a.N, 64), cdiv(a.M, 64));
  switch (a.epi) {
    case EPI_STORE: gemm_generic_kernel<T, EPI_STORE><<<grid, 256, 0, s>>>(a); break;
    case EPI_QKV: gemm_generic_kernel<T, EPI_QKV><<<grid, 256, 0, s>>>(a); break;
    case EPI_RESID: gemm_generic_kernel<T, EPI_RESID><<<grid, 256, 0, s>>>(a); break;
    case EPI_GELU: gemm_generic_kernel<T, EPI_GELU><<<grid, 256, 0, s>>>(a); break;
    case EPI_DGELU: gemm_generic_kernel<T, EPI_DGELU><<<grid, 256, 0, s>>>(a); break;
    case EPI_ACC_F32: gemm_generic_kernel<T, EPI_ACC_F32><<<grid, 256, 0, s>>>(a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t gemm_generic(int dtype, const GemmArgs& a, hipStream_t s) {
  return dtype == DT_FP32 ? gemm_generic_t<float>(a, s) : gemm_generic_t<bf16>(a, s);
}

// ------------------------------------------------------- generic attention

// One block per (query row, head).  LDS: scores [Lmax] (+ dP [Lmax] for bwd),
// q and dO rows, reduction scratch.
template <typename T>
__global__ __launch_bounds__(256) void attn_fwd_generic_kernel(AttnArgs a0) {
  extern __shared__ float sm[];
  const AttnArgs a = attn_seq_view<T>(a0);
  const int i = blockIdx.x, t = a.l + i, h = blockIdx.y, d = a.d, H = a.ld;  // H: row stride
  float* S = sm;
  float* qs = sm + a.Lmax;
  float* red = qs + 128;
  const T* q = (const T*)a.q + (long)i * H + h * d;
  for (int j = threadIdx.x; j < d; j += blockDim.x) qs[j] = ld(q + j);
  __syncthreads();
  float mx = -INFINITY;
  for (int s = threadIdx.x; s <= t; s += blockDim.x) {
    const T* k = (const T*)a.kc + (long)s * H + h * d;
    float dot = 0.f;
    for (int j = 0; j < d; ++j) dot += qs[j] * ld(k + j);
    dot *= a.scale;
    S[s] = dot;
    mx = fmaxf(mx, dot);
  }
  mx = block_max(mx, red);
  float sum = 0.f;
  for (int s = threadIdx.x; s <= t; s += blockDim.x) {
    const float e = __expf(S[s] - mx);
    S[s] = e;
    sum += e;
  }
  sum = block_sum(sum, red);
  const float inv = 1.f / sum;
  for (int j = threadIdx.x; j < d; j += blockDim.x) {
    float acc = 0.f;
    for (int s = 0; s <= t; ++s) acc += S[s] * ld((const T*)a.vc + (long)s * H + h * d + j);
    st((T*)a.o + (long)i * H + h * d + j, acc * inv);
  }
  if (threadIdx.x == 0) a.lse[(long)h * a.Lmax + t] = mx + logf(sum);
}

template <typename T>
__global__ __launch_bounds__(256) void attn_bwd_generic_kernel(AttnArgs a0) {
  extern __shared__ float sm[];
  const AttnArgs a = attn_seq_view<T>(a0);
  const int i = blockIdx.x, t = a.l + i, h = blockIdx.y, d = a.d, H = a.ld;  // H: row stride
  float* P = sm;
  float* dS = sm + a.Lmax;
  float* qs = dS + a.Lmax;
  float* ds_ = qs + 128;
  float* red = ds_ + 128;
  for (int j = threadIdx.x; j < d; j += blockDim.x) {
    qs[j] = ld((const T*)a.q + (long)i * H + h * d + j);
    ds_[j] = ld((const T*)a.dout + (long)i * H + h * d + j);
  }
  __syncthreads();
  const float lse = a.lse[(long)h * a.Lmax + t];
  float Dp = 0.f;
  for (int s = threadIdx.x; s <= t; s += blockDim.x) {
    const T* k = (const T*)a.kc + (long)s * H + h * d;
    const T* v = (const T*)a.vc + (long)s * H + h * d;
    float dot = 0.f, dpv = 0.f;
    for (int j = 0; j < d; ++j) {
      dot += qs[j] * ld(k + j);
      dpv += ds_[j] * ld(v + j);
    }
    const float p = __expf(dot * a.scale - lse);
    P[s] = p;
    dS[s] = dpv;
    Dp += p * dpv;
  }
  const float D = block_sum(Dp, red);
  for (int s = threadIdx.x; s <= t; s += blockDim.x) dS[s] = P[s] * (dS[s] - D);
  __syncthreads();
  for (int j = threadIdx.x; j < d; j += blockDim.x) {
    float acc = 0.f;
    for (int s = 0; s <= t; ++s) acc += dS[s] * ld((const T*)a.kc + (long)s * H + h * d + j);
    st((T*)a.dq + (long)i * a.ld_dq + h * d + j, acc * a.scale);
  }
  const long tot = (long)(t + 1) * d;
  for (long e = threadIdx.x; e < tot; e += blockDim.x) {
    const int s = (int)(e / d), j = (int)(e % d);
    atomicAdd(a.dk + (long)s * H + h * d + j, dS[s] * qs[j] * a.scale);
    atomicAdd(a.dv + (long)s * H + h * d + j, P[s] * ds_[j]);
  }
}

template <typename T>
static hipError_t attn_generic_t(const AttnArgs& a, bool bwd, hipStream_t s) {
  if (a.need) return hipSuccess;  // no scratch
  const size_t lds = bwd ? (2 * (size_t)a.Lmax + 256 + 16) * 4 : ((size_t)a.Lmax + 128 + 16) * 4;
  if (lds > 160 * 1024) return hipErrorInvalidValue;
  if (lds > 64 * 1024) {
    const void* fn = bwd ? (const void*)attn_bwd_generic_kernel<T>
                         : (const void*)attn_fwd_generic_kernel<T>;
    hipError_t e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
  }
  dim3 grid(a.r - a.l, a.heads, a.bs);
  if (bwd)
    attn_bwd_generic_kernel<T><<<grid, 256, lds, s>>>(a);
  else
    attn_fwd_generic_kernel<T><<<grid, 256, lds, s>>>(a);
  return hipGetLastError();
}

hipError_t attn_fwd_generic(int dtype, const AttnArgs& a, hipStream_t s) {
  return dtype == DT_FP32 ? attn_generic_t<float>(a, false, s) : attn_generic_t<bf16>(a, false, s);
}
hipError_t attn_bwd_generic(int dtype, const AttnArgs& a, hipStream_t s) {
  return dtype == DT_FP32 ? attn_generic_t<float>(a, true, s) : attn_generic_t<bf16>(a, true, s);
}

// ------------------------------------------------------------- LayerNorm

// 8 consecutive elements <-> 8 floats (16-byte loads for bf16, 2 x 16 for fp32).
__device__ inline void load8(const bf16* p, float* v) {
  const uint4 u = *(const uint4*)p;
  const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    v[2 * i] = __uint_as_float(w[i] << 16);
    v[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
  }
}
__device__ inline void load8(const float* p, float* v) {
  const float4 a = ((const float4*)p)[0], b = ((const float4*)p)[1];
  v[0] = a.x, v[1] = a.y, v[2] = a.z, v[3] = a.w, v[4] = b.x, v[5] = b.y, v[6] = b.z, v[7] = b.w;
}
__device__ inline void store8(bf16* p, const float* v) {
  uint4 u;
  u.x = f32_to_bf16_bits(v[0]) | ((uint32_t)f32_to_bf16_bits(v[1]) << 16);
  u.y = f32_to_bf16_bits(v[2]) | ((uint32_t)f32_to_bf16_bits(v[3]) << 16);
  u.z = f32_to_bf16_bits(v[4]) | ((uint32_t)f32_to_bf16_bits(v[5]) << 16);
  u.w = f32_to_bf16_bits(v[6]) | ((uint32_t)f32_to_bf16_bits(v[7]) << 16);
  *(uint4*)p = u;
}
__device__ inline void store8(float* p, const float* v) {
  ((float4*)p)[0] = make_float4(v[0], v[1], v[2], v[3]);
  ((float4*)p)[1] = make_float4(v[4], v[5], v[6], v[7]);
}

// One block per row; the row stays in registers (H % 8 == 0, H <= 16384).  The
// block has nt threads (a multiple of 64, <= 1024) and thread t owns the
// 8-element chunks t + nt * c, c < CPT; CPT = 2 only when H / 8 > 1024.  Every
// load a thread makes (row, gamma, beta, residual) is issued before the first
// reduction, so a row costs one memory latency instead of several.
struct LnShape {
  int cpt, nt;
};
inline LnShape ln_shape(int H) {
  const int nc = H / 8, cpt = nc > 1024 ? 2 : 1;
  return {cpt, cdiv(cdiv(nc, cpt), 64) * 64};
}

// T: stage dtype (gamma, beta, u); TX: type of the input rows x (fp32 for the
// residual stream of a mixed-precision stage).  x_copy (fp32 when copy_f32, else
// T) and u16 (fp16 copy of u) are optional.
template <typename T, typename TX, int CPT>
__global__ __launch_bounds__(1024) void ln_fwd_kernel(int H, const TX* x, void* x_copy,
                                                      int copy_f32, const T* g, const T* b, T* u,
                                                      f16s* u16, float* mean, float* rstd,
                                                      float eps) {
  __shared__ float red[16];
  const int row = blockIdx.x, nc = H >> 3, nt = blockDim.x;
  const TX* xr = x + (long)row * H;
  float v[CPT][8], gg[CPT][8], bb[CPT][8];
#pragma unroll
  for (int c = 0; c < CPT; ++c) {
    const int ci = threadIdx.x + nt * c;
    if (ci < nc) {
      load8(xr + ci * 8, v[c]);
      load8(g + ci * 8, gg[c]);
      load8(b + ci * 8, bb[c]);
    }
  }
  float s = 0.f;
#pragma unroll
  for (int c = 0; c < CPT; ++c)
    if (threadIdx.x + nt * c < nc)
#pragma unroll
      for (int e = 0; e < 8; ++e) s += v[c][e];
  const float mu = block_sum(s, red) / H;
  float q = 0.f;
#pragma unroll
  for (int c = 0; c < CPT; ++c)
    if (threadIdx.x + nt * c < nc)
#pragma unroll
      for (int e = 0; e < 8; ++e) q += (v[c][e] - mu) * (v[c][e] - mu);
  const float rs = rsqrtf(block_sum(q, red) / H + eps);
#pragma unroll
  for (int c = 0; c < CPT; ++c) {
    const int ci = threadIdx.x + nt * c;
    if (ci < nc) {
      float o[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) o[e] = gg[c][e] * ((v[c][e] - mu) * rs) + bb[c][e];
      store8(u + (long)row * H + ci * 8, o);
      if (u16) st8(u16 + (long)row * H + ci * 8, o);
      if (x_copy) {
        if (copy_f32)
          store8((float*)x_copy + (long)row * H + ci * 8, v[c]);
        else
          store8((T*)x_copy + (long)row * H + ci * 8, v[c]);
      }
    }
  }
  if (threadIdx.x == 0) {
    mean[row] = mu;
    rstd[row] = rs;
  }
}

// Two block-wide sums in one pass (blockDim.x a multiple of 64, <= 1024).
__device__ inline float2 block_sum2(float a, float b, float* red /* >= 32 floats */) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, nw = blockDim.x >> 6;
  a = wave_sum(a);
  b = wave_sum(b);
  if (lane == 0) red[w] = a, red[16 + w] = b;
  __syncthreads();
  float sa = 0.f, sb = 0.f;
  for (int i = 0; i < nw; ++i) sa += red[i], sb += red[16 + i];
  return make_float2(sa, sb);
}

template <typename T, typename TX, int CPT>
__global__ __launch_bounds__(1024) void ln_bwd_kernel(int H, const T* du, const TX* x,
                                                      const float* mean, const float* rstd,
                                                      const T* g, const T* resid, T* dx) {
  __shared__ float red[32];
  const int row = blockIdx.x, nc = H >> 3, nt = blockDim.x;
  const float mu = mean[row], rs = rstd[row];
  float xh[CPT][8], dg[CPT][8], r[CPT][8];
#pragma unroll
  for (int c = 0; c < CPT; ++c) {
    const int ci = threadIdx.x + nt * c;
    if (ci < nc) {
      float gg[8];
      load8(x + (long)row * H + ci * 8, xh[c]);
      load8(du + (long)row * H + ci * 8, dg[c]);
      load8(g + ci * 8, gg);
      if (resid) load8(resid + (long)row * H + ci * 8, r[c]);
#pragma unroll
      for (int e = 0; e < 8; ++e) dg[c][e] *= gg[e];
    }
  }
  float sa = 0.f, sb = 0.f;
#pragma unroll
  for (int c = 0; c < CPT; ++c)
    if (threadIdx.x + nt * c < nc)
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        xh[c][e] = (xh[c][e] - mu) * rs;
        sa += dg[c][e];
        sb += dg[c][e] * xh[c][e];
      }
  const float2 ab = block_sum2(sa, sb, red);
  const float a = ab.x / H, bm = ab.y / H;
#pragma unroll
  for (int c = 0; c < CPT; ++c) {
    const int ci = threadIdx.x + nt * c;
    if (ci < nc) {
      float o[8];
#pragma unroll
      for (int e = 0; e < 8; ++e)
        o[e] = rs * (dg[c][e] - a - xh[c][e] * bm) + (resid ? r[c][e] : 0.f);
      store8(dx + (long)row * H + ci * 8, o);
    }
  }
}

// Column reductions over n rows.  A block owns 32 columns (4 chunks of 8) and
// 64 row groups; row group rg sums rows rg, rg + 64, ... in order, loading four
// rows at a time, then the 64 partial sums of a column are added as 8 in-order
// groups of 8, the group sums in order.  Deterministic.
constexpr int CR_RG = 64, CR_COLS = 32, CR_UNROLL = 4;

// Adds the 64 per-row-group partials of each of the block's 32 columns (in
// p[rg][col]) and returns the column total in threads 0..31.
__device__ inline float col_partials_sum(float (*p)[CR_COLS + 1], float* q /* 8 x 33 */) {
  const int col = threadIdx.x & 31, grp = threadIdx.x >> 5;
  float s = 0.f;
#pragma unroll
  for (int i = 0; i < 8; ++i) s += p[grp * 8 + i][col];
  q[grp * (CR_COLS + 1) + col] = s;
  __syncthreads();
  float t = 0.f;
  if (threadIdx.x < CR_COLS)
#pragma unroll
    for (int i = 0; i < 8; ++i) t += q[i * (CR_COLS + 1) + col];
  return t;
}

template <typename T, typename TX>
__global__ __launch_bounds__(256) void ln_param_grads_kernel(int n, int H, const T* du,
                                                             const TX* x, const float* mean,
                                                             const float* rstd, float* dg,
                                                             float* db, int store) {
  __shared__ float pg[CR_RG][CR_COLS + 1], pb[CR_RG][CR_COLS + 1], q[2][8 * (CR_COLS + 1)];
  const int cc = threadIdx.x & 3, rg = threadIdx.x >> 2;
  const int c0 = blockIdx.x * CR_COLS + cc * 8;
  float sg[8] = {}, sb[8] = {};
  if (c0 < H) {
    for (int t0 = rg; t0 < n; t0 += CR_UNROLL * CR_RG) {
      float d[CR_UNROLL][8], xv[CR_UNROLL][8], mu[CR_UNROLL], rs[CR_UNROLL];
#pragma unroll
      for (int k = 0; k < CR_UNROLL; ++k) {
        const int t = t0 + k * CR_RG;
        if (t < n) {
          load8(du + (long)t * H + c0, d[k]);
          load8(x + (long)t * H + c0, xv[k]);
          mu[k] = mean[t], rs[k] = rstd[t];
        }
      }
#pragma unroll
      for (int k = 0; k < CR_UNROLL; ++k)
        if (t0 + k * CR_RG < n)
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            sg[e] += d[k][e] * ((xv[k][e] - mu[k]) * rs[k]);
            sb[e] += d[k][e];
          }
    }
  }
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    pg[rg][cc * 8 + e] = sg[e];
    pb[rg][cc * 8 + e] = sb[e];
  }
  __syncthreads();
  const float a = col_partials_sum(pg, q[0]);
  const float b = col_partials_sum(pb, q[1]);
  const int col = blockIdx.x * CR_COLS + threadIdx.x;
  if (threadIdx.x < CR_COLS && col < H) {
    dg[col] = store ? a : dg[col] + a;
    db[col] = store ? b : db[col] + b;
  }
}

template <typename T>
__global__ __launch_bounds__(256) void colsum_kernel(int n, int N, const T* A, long lda,
                                                     float* out, int store) {
  __shared__ float ps[CR_RG][CR_COLS + 1], q[8 * (CR_COLS + 1)];
  const int cc = threadIdx.x & 3, rg = threadIdx.x >> 2;
  const int c0 = blockIdx.x * CR_COLS + cc * 8;
  float s[8] = {};
  if (c0 < N) {
    for (int t0 = rg; t0 < n; t0 += CR_UNROLL * CR_RG) {
      float v[CR_UNROLL][8];
#pragma unroll
      for (int k = 0; k < CR_UNROLL; ++k)
        if (t0 + k * CR_RG < n) load8(A + (long)(t0 + k * CR_RG) * lda + c0, v[k]);
#pragma unroll
      for (int k = 0; k < CR_UNROLL; ++k)
        if (t0 + k * CR_RG < n)
#pragma unroll
          for (int e = 0; e < 8; ++e) s[e] += v[k][e];
    }
  }
#pragma unroll
  for (int e = 0; e < 8; ++e) ps[rg][cc * 8 + e] = s[e];
  __syncthreads();
  const float a = col_partials_sum(ps, q);
  const int col = blockIdx.x * CR_COLS + threadIdx.x;
  if (threadIdx.x < CR_COLS && col < N) out[col] = store ? a : out[col] + a;
}

// dK and dV (fp32, [n, H]) into the K and V thirds of the dQKV rows, 8
// consecutive columns per thread (H % 8 == 0; 16-byte aligned pointers).
template <typename T>
__global__ void pack_dkv_kernel(int n, int H, const float* dk, const float* dv, T* dqkv) {
  const int h8 = H >> 3;
  const long e = (long)blockIdx.x * blockDim.x + threadIdx.x;
  if (e >= (long)n * h8) return;
  const long i = e / h8, j = (e - i * h8) * 8;
  float v[8];
  load8(dk + i * H + j, v);
  store8(dqkv + i * 3 * H + H + j, v);
  load8(dv + i * H + j, v);
  store8(dqkv + i * 3 * H + 2 * H + j, v);
}

__global__ void fill_f32_kernel(float* p, size_t n, float v) {
  for (size_t e = (size_t)blockIdx.x * blockDim.x + threadIdx.x; e < n;
       e += (size_t)gridDim.x * blockDim.x)
    p[e] = v;
}

template <typename T>
__global__ void copy_kernel(size_t n, const T* src, T* dst) {
  for (size_t e = (size_t)blockIdx.x * blockDim.x + threadIdx.x; e < n;
       e += (size_t)gridDim.x * blockDim.x)
    dst[e] = src[e];
}

hipError_t ln_fwd(int dtype, int n, int H, const void* x, int x_f32, void* x_copy, int copy_f32,
                  const void* g, const void* b, void* u, void* u16, float* mean, float* rstd,
                  float eps, hipStream_t s) {
  clear_stale_error();
  if (n <= 0) return hipSuccess;
  const LnShape sh = ln_shape(H);
#define TP_LN(TT, TX, C)                                                                   \
  ln_fwd_kernel<TT, TX, C><<<n, sh.nt, 0, s>>>(H, (const TX*)x, x_copy, copy_f32,           \
                                               (const TT*)g, (const TT*)b, (TT*)u,          \
                                               (f16s*)u16, mean, rstd, eps)
  if (dtype == DT_FP32) {
    if (sh.cpt == 1) TP_LN(float, float, 1); else TP_LN(float, float, 2);
  } else if (x_f32) {
    if (sh.cpt == 1) TP_LN(bf16, float, 1); else TP_LN(bf16, float, 2);
  } else {
    if (sh.cpt == 1) TP_LN(bf16, bf16, 1); else TP_LN(bf16, bf16, 2);
  }
#undef TP_LN
  return hipGetLastError();
}

hipError_t ln_bwd(int dtype, int n, int H, const void* du, const void* x, int x_f32,
                  const float* mean, const float* rstd, const void* g, const void* resid, void* dx,
                  hipStream_t s) {
  clear_stale_error();
  if (n <= 0) return hipSuccess;
  const LnShape sh = ln_shape(H);
#define TP_LN(TT, TX, C)                                                                   \
  ln_bwd_kernel<TT, TX, C><<<n, sh.nt, 0, s>>>(H, (const TT*)du, (const TX*)x, mean, rstd,  \
                                               (const TT*)g, (const TT*)resid, (TT*)dx)
  if (dtype == DT_FP32) {
    if (sh.cpt == 1) TP_LN(float, float, 1); else TP_LN(float, float, 2);
  } else if (x_f32) {
    if (sh.cpt == 1) TP_LN(bf16, float, 1); else TP_LN(bf16, float, 2);
  } else {
    if (sh.cpt == 1) TP_LN(bf16, bf16, 1); else TP_LN(bf16, bf16, 2);
  }
#undef TP_LN
  return hipGetLastError();
}

hipError_t ln_param_grads(int dtype, int n, int H, const void* du, const void* x, int x_f32,
                          const float* mean, const float* rstd, float* dg, float* db, int store,
                          hipStream_t s) {
  clear_stale_error();
  if (n <= 0) return hipSuccess;
  const int blocks = cdiv(H, CR_COLS);
  if (dtype == DT_FP32)
    ln_param_grads_kernel<float, float><<<blocks, 256, 0, s>>>(n, H, (const float*)du,
                                                               (const float*)x, mean, rstd, dg, db, store);
  else if (x_f32)
    ln_param_grads_kernel<bf16, float><<<blocks, 256, 0, s>>>(n, H, (const bf16*)du,
                                                              (const float*)x, mean, rstd, dg, db, store);
  else
    ln_param_grads_kernel<bf16, bf16><<<blocks, 256, 0, s>>>(n, H, (const bf16*)du,
                                                             (const bf16*)x, mean, rstd, dg, db, store);
  return hipGetLastError();
}

// 8 bf16 values per thread as fp16 (n % 8 == 0, 16-byte aligned), else one.
__global__ void cvt_bf16_f16_kernel(size_t n, const uint16_t* src, uint16_t* dst, int vec) {
  const size_t stride = (size_t)gridDim.x * blockDim.x;
  if (vec) {
    const size_t n8 = n / 8;
    size_t e = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
    // four independent 16-byte loads in flight per thread
    for (; e + 3 * stride < n8; e += 4 * stride) {
      float v[4][8];
#pragma unroll
      for (int u = 0; u < 4; ++u) ld8((const bf16*)src + 8 * (e + u * stride), v[u]);
#pragma unroll
      for (int u = 0; u < 4; ++u) st8((f16s*)dst + 8 * (e + u * stride), v[u]);
    }
    for (; e < n8; e += stride) {
      float v[8];
      ld8((const bf16*)src + 8 * e, v);
      st8((f16s*)dst + 8 * e, v);
    }
  } else {
    for (size_t e = (size_t)blockIdx.x * blockDim.x + threadIdx.x; e < n; e += stride)
      dst[e] = f32_to_f16_bits(to_f32(bf16{src[e]}));
  }
}

hipError_t cvt_bf16_f16(size_t n, const void* src, void* dst, hipStream_t s) {
  clear_stale_error();
  if (n == 0) return hipSuccess;
  const int vec = n % 8 == 0 && ((uintptr_t)src & 15) == 0 && ((uintptr_t)dst & 15) == 0;
  const size_t work = vec ? n / 8 : n;
  const int blocks = (int)((work + 255) / 256 < 8192 ? (work + 255) / 256 : 8192);
  cvt_bf16_f16_kernel<<<blocks, 256, 0, s>>>(n, (const uint16_t*)src, (uint16_t*)dst, vec);
  return hipGetLastError();
}

hipError_t colsum_acc(int dtype, int n, int N, const void* A, long lda, float* out, int store,
                      hipStream_t s) {
  clear_stale_error();
  if (n <= 0 || N <= 0) return hipSuccess;
  const int blocks = cdiv(N, CR_COLS);
  if (dtype == DT_FP32)
    colsum_kernel<float><<<blocks, 256, 0, s>>>(n, N, (const float*)A, lda, out, store);
  else
    colsum_kernel<bf16><<<blocks, 256, 0, s>>>(n, N, (const bf16*)A, lda, out, store);
  return hipGetLastError();
}

hipError_t pack_dkv(int dtype, int n, int H, const float* dk, const float* dv, void* dqkv,
                    hipStream_t s) {
  clear_stale_error();
  const long tot = (long)n * (H / 8);
  if (tot <= 0) return hipSuccess;
  auto al = [](const void* p) { return ((uintptr_t)p & 15) == 0; };
  if (H % 8 || !al(dk) || !al(dv) || !al(dqkv)) return hipErrorInvalidValue;
  if (dtype == DT_FP32)
    pack_dkv_kernel<float><<<cdiv(tot, 256), 256, 0, s>>>(n, H, dk, dv, (float*)dqkv);
  else
    pack_dkv_kernel<bf16><<<cdiv(tot, 256), 256, 0, s>>>(n, H, dk, dv, (bf16*)dqkv);
  return hipGetLastError();
}

hipError_t fill_f32(float* p, size_t n, float v, hipStream_t s) {
  clear_stale_error();
  if (n == 0) return hipSuccess;
  const int blocks = (int)((n + 255) / 256 < 8192 ? (n + 255) / 256 : 8192);
  fill_f32_kernel<<<blocks, 256, 0, s>>>(p, n, v);
  return hipGetLastError();
}

hipError_t copy_rows(int dtype, int n, int H, const void* src, void* dst, hipStream_t s) {
  clear_stale_error();
  const size_t tot = (size_t)n * H;
  if (tot == 0) return hipSuccess;
  const int blocks = (int)((tot + 255) / 256 < 8192 ? (tot + 255) / 256 : 8192);
  if (dtype == DT_FP32)
    copy_kernel<float><<<blocks, 256, 0, s>>>(tot, (const float*)src, (float*)dst);
  else
    copy_kernel<bf16><<<blocks, 256, 0, s>>>(tot, (const bf16*)src, (bf16*)dst);
  return hipGetLastError();
}

}  // namespace tp
