// Fused GEMM epilogues, shared by every GEMM kernel and the split-K
// reductions: what happens to one accumulator value (epi1) or to 8
// consecutive columns of one output row (epi8, 16-byte accesses, bf16
// stages).  acc = sum_k A(m, k) B(k, n) in fp32; the kinds are listed with
// EpiKind in tp_kernels.hpp.
#pragma once

#include "tp_common.hpp"
#include "tp_kernels.hpp"

namespace tp {

// EPI_QKV destination of output column n: (base pointer, element offset, part
// 0 = q, 1 = k, 2 = v).
__device__ inline void* qkv_dst(const GemmArgs& a, int m, int n, long* off, int* part) {
  const int H = a.H;
  const int p = n < H ? 0 : n < 2 * H ? 1 : 2;
  *off = (long)m * H + (n - p * H);
  *part = p;
  return p == 0 ? a.q : p == 1 ? a.k : a.v;
}

// T: the stage dtype (float or bf16).
template <typename T, int EPI>
__device__ inline void epi1(const GemmArgs& a, int m, int n, float acc) {
  if constexpr (EPI == EPI_ACC_F32) {
    float* C = (float*)a.C + (long)m * a.ldc + n;
    *C = a.overwrite ? acc : *C + acc;
  } else if constexpr (EPI == EPI_DGELU) {
    const float z = ld((const T*)a.R + (long)m * a.ldr + n);
    st((T*)a.C + (long)m * a.ldc + n, acc * gelu_tanh_grad(z));
  } else {
    const float v = acc + (a.bias ? ld((const T*)a.bias + n) : 0.f);
    if constexpr (EPI == EPI_STORE) {
      st((T*)a.C + (long)m * a.ldc + n, v);
    } else if constexpr (EPI == EPI_RESID) {
      const long ro = (long)m * a.ldr + n, co = (long)m * a.ldc + n;
      const float r = a.r_f32 ? ((const float*)a.R)[ro] : ld((const T*)a.R + ro);
      if (a.c_f32)
        ((float*)a.C)[co] = v + r;
      else
        st((T*)a.C + co, v + r);
    } else if constexpr (EPI == EPI_GELU) {
      st((T*)a.C + (long)m * a.ldc + n, v);
      st((T*)a.C2 + (long)m * a.ldc2 + n, gelu_tanh(v));
    } else if constexpr (EPI == EPI_QKV) {
      long off;
      int part;
      void* dst = qkv_dst(a, m, n, &off, &part);
      if (a.qkv_f16) {
        st((f16s*)dst + off, v);
        if (part == 2) st((bf16*)a.vb + off, v);
      } else {
        st((T*)dst + off, v);
      }
    }
  }
}

// The same for columns n .. n+7 of row m of a bf16 stage; x holds the 8
// accumulators and is clobbered.  Sizes and alignment were checked by the
// launcher (vec8_ok).
template <int EPI>
__device__ inline void epi8(const GemmArgs& a, int m, int n, float* x) {
  if constexpr (EPI == EPI_ACC_F32) {
    float* c = (float*)a.C + (long)m * a.ldc + n;
    if (a.overwrite) {
      st8(c, x);
    } else {
      float o[8];
      ld8(c, o);
#pragma unroll
      for (int i = 0; i < 8; ++i) o[i] += x[i];
      st8(c, o);
    }
  } else if constexpr (EPI == EPI_DGELU) {
    float z[8];
    ld8((const bf16*)a.R + (long)m * a.ldr + n, z);
#pragma unroll
    for (int i = 0; i < 8; ++i) x[i] *= gelu_tanh_grad(z[i]);
    st8((bf16*)a.C + (long)m * a.ldc + n, x);
  } else {
    if (a.bias) {
      float b[8];
      ld8((const bf16*)a.bias + n, b);
#pragma unroll
      for (int i = 0; i < 8; ++i) x[i] += b[i];
    }
    if constexpr (EPI == EPI_STORE) {
      st8((bf16*)a.C + (long)m * a.ldc + n, x);
    } else if constexpr (EPI == EPI_RESID) {
      float r[8];
      if (a.r_f32)
        ld8((const float*)a.R + (long)m * a.ldr + n, r);
      else
        ld8((const bf16*)a.R + (long)m * a.ldr + n, r);
#pragma unroll
      for (int i = 0; i < 8; ++i) x[i] += r[i];
      if (a.c_f32)
        st8((float*)a.C + (long)m * a.ldc + n, x);
      else
        st8((bf16*)a.C + (long)m * a.ldc + n, x);
    } else if constexpr (EPI == EPI_GELU) {
      st8((bf16*)a.C + (long)m * a.ldc + n, x);
#pragma unroll
      for (int i = 0; i < 8; ++i) x[i] = gelu_tanh(x[i]);
      st8((bf16*)a.C2 + (long)m * a.ldc2 + n, x);
    } else if constexpr (EPI == EPI_QKV) {
      long off;
      int part;
      void* dst = qkv_dst(a, m, n, &off, &part);
      if (a.qkv_f16) {
        st8((f16s*)dst + off, x);
        if (part == 2) st8((bf16*)a.vb + off, x);
      } else {
        st8((bf16*)dst + off, x);
      }
    }
  }
}

}  // namespace tp
