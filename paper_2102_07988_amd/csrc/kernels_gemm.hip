// bf16 GEMM on the CDNA4 matrix cores: C = sum_k A(m,k) B(k,n) with fp32
// accumulation in v_mfma_f32_32x32x16_bf16, followed by the stage's fused
// epilogues.
//
// Block tile BM x BN x 64 with WGM x WGN waves; each wave owns a
// (BM/WGM) x (BN/WGN) sub-tile made of 32 x 32 MFMA tiles.  Both operands sit
// in LDS k-contiguous (64 k per row, 16-byte chunks XOR-swizzled by row), so
// one ds_read_b128 gives a lane its 8 consecutive k values.  An operand whose global layout is
// k-contiguous (activations; weights [out][in] in the forward) is copied with
// 16-byte loads; an operand that is contiguous along m or n (weights in the
// dX products, token-major activations and gradients in the dW products) is
// read as 4 (k) x 8 (m/n) blocks with 16-byte row loads and transposed in
// registers before it is written.  The next k-tile is fetched into registers
// while the current one is multiplied.
#include "tp_common.hpp"
#include "tp_epilogue.hpp"
#include "tp_kernels.hpp"

#include <algorithm>

namespace tp {

namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef _Float16 f16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

constexpr int BK = 64;

// LDS tile layout: row r holds 64 k values (128 bytes, no padding); its eight
// 16-byte chunks are permuted by chunk ^ swz(r).  With swz(r) = (r ^ r/8) & 7
// the fragment reads of 16 consecutive rows at one chunk hit 16 distinct
// 16-byte bank groups, and the transposed 8-byte writes of one instruction
// spread over all chunks.
__device__ inline int swz(int r) { return (r ^ (r >> 3)) & 7; }
__device__ inline int lds_off(int r, int k) { return r * BK + ((((k >> 3) ^ swz(r))) << 3) + (k & 7); }

__device__ inline uint4 pack8(const uint16_t* t) {
  return make_uint4(t[0] | (uint32_t)t[1] << 16, t[2] | (uint32_t)t[3] << 16,
                    t[4] | (uint32_t)t[5] << 16, t[6] | (uint32_t)t[7] << 16);
}

// Operand tile of R rows (m or n) by BK k values, k-contiguous in global
// memory: X(r, k) = X[r * ld + k].  Chunks of 8 k values (16 bytes).
template <int R, int NTH>
struct TileKC {
  static constexpr int CH = R * (BK / 8) / NTH;  // chunks per thread
  static_assert(CH >= 1, "tile too small");
  uint4 v[CH];
  __device__ void load(const uint16_t* X, long ld, int r0, int rmax, int k0, int kmax) {
#pragma unroll
    for (int i = 0; i < CH; ++i) {
      const int c = threadIdx.x + NTH * i;
      const int r = c >> 3, kc = (c & 7) * 8;
      const int gr = r0 + r, gk = k0 + kc;
      if (gr < rmax && gk + 8 <= kmax) {
        v[i] = *(const uint4*)(X + (long)gr * ld + gk);
      } else {
        uint16_t t[8];
#pragma unroll
        for (int e = 0; e < 8; ++e)
          t[e] = (gr < rmax && gk + e < kmax) ? X[(long)gr * ld + gk + e] : (uint16_t)0;
        v[i] = pack8(t);
      }
    }
  }
  __device__ void store(uint16_t* lds) const {
#pragma unroll
    for (int i = 0; i < CH; ++i) {
      const int c = threadIdx.x + NTH * i;
      const int r = c >> 3, kc = (c & 7) * 8;
      *(uint4*)(lds + lds_off(r, kc)) = v[i];
    }
  }
};

// Operand tile of R rows (m or n) by BK k values, contiguous along r in global
// memory: X(r, k) = X[k * ld + r].  Blocks of 4 k x 8 r, transposed in registers.
template <int R, int NTH>
struct TileMC {
  static constexpr int NB = (BK / 4) * (R / 8);   // blocks per tile
  static constexpr int PER = (NB + NTH - 1) / NTH;  // blocks per thread
  uint4 x[PER][4];  // [block][k row]: 8 r values of one k
  __device__ void load(const uint16_t* X, long ld, int r0, int rmax, int k0, int kmax) {
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int b = threadIdx.x + NTH * i;
      if (NB % NTH != 0 && b >= NB) break;
      const int kb = b / (R / 8), rb = b % (R / 8);
      const int gr = r0 + rb * 8;
#pragma unroll
      for (int kk = 0; kk < 4; ++kk) {
        const int gk = k0 + kb * 4 + kk;
        if (gk < kmax && gr + 8 <= rmax) {
          x[i][kk] = *(const uint4*)(X + (long)gk * ld + gr);
        } else {
          uint16_t t[8];
#pragma unroll
          for (int e = 0; e < 8; ++e)
            t[e] = (gk < kmax && gr + e < rmax) ? X[(long)gk * ld + gr + e] : (uint16_t)0;
          x[i][kk] = pack8(t);
        }
      }
    }
  }
  __device__ static uint32_t word(const uint4& v, int w) {
    return w == 0 ? v.x : w == 1 ? v.y : w == 2 ? v.z : v.w;
  }
  __device__ void store(uint16_t* lds) const {
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int b = threadIdx.x + NTH * i;
      if (NB % NTH != 0 && b >= NB) break;
      const int kb = b / (R / 8), rb = b % (R / 8);
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        // LDS row rb*8 + e receives k = kb*4 .. kb*4+3
        const uint32_t sel = (e & 1) ? 0x07060302u : 0x05040100u;
        const uint32_t p0 = __builtin_amdgcn_perm(word(x[i][1], e >> 1), word(x[i][0], e >> 1), sel);
        const uint32_t p1 = __builtin_amdgcn_perm(word(x[i][3], e >> 1), word(x[i][2], e >> 1), sel);
        *(uint2*)(lds + lds_off(rb * 8 + e, kb * 4)) = make_uint2(p0, p1);
      }
    }
  }
};

template <int R, int NTH, bool KC>
struct TileSel;
template <int R, int NTH>
struct TileSel<R, NTH, true> {
  using type = TileKC<R, NTH>;
};
template <int R, int NTH>
struct TileSel<R, NTH, false> {
  using type = TileMC<R, NTH>;
};

// F16: both operands are fp16 (the mixed-precision query/key/value product).
template <int BM, int BN, int WGM, int WGN, bool A_KC, bool B_KC, int EPI, bool SPLIT, bool F16>
__global__ __launch_bounds__(64 * WGM * WGN) void gemm_mfma_kernel(GemmArgs a) {
  constexpr int NTH = 64 * WGM * WGN;
  constexpr int WM = BM / WGM, WN = BN / WGN, FM = WM / 32, FN = WN / 32;
  static_assert(FM >= 1 && FN >= 1, "wave tile below 32 x 32");
  __shared__ __attribute__((aligned(16))) uint16_t As[BM * BK];
  __shared__ __attribute__((aligned(16))) uint16_t Bs[BN * BK];
  const uint16_t* A = (const uint16_t*)a.A;
  const uint16_t* B = (const uint16_t*)a.B;
  const long lda = A_KC ? a.sam : a.sak;
  const long ldb = B_KC ? a.sbn : a.sbk;
  const int m0 = blockIdx.y * BM, n0 = blockIdx.x * BN;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm0 = (wave / WGN) * WM, wn0 = (wave % WGN) * WN;
  // reduction range of this split
  const int kbeg = SPLIT ? blockIdx.z * a.k_split : 0;
  const int kend = SPLIT ? min(a.K, kbeg + a.k_split) : a.K;

  typename TileSel<BM, NTH, A_KC>::type ta;
  typename TileSel<BN, NTH, B_KC>::type tb;
  f32x16_t acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;

  const int nk = (kend - kbeg + BK - 1) / BK;
  if (nk > 0) {
    ta.load(A, lda, m0, a.M, kbeg, kend);
    tb.load(B, ldb, n0, a.N, kbeg, kend);
    ta.store(As);
    tb.store(Bs);
  }
  __syncthreads();
  const int fr = lane & 31, fk = (lane >> 5) * 8;
  for (int kt = 0; kt < nk; ++kt) {
    if (kt + 1 < nk) {
      ta.load(A, lda, m0, a.M, kbeg + (kt + 1) * BK, kend);
      tb.load(B, ldb, n0, a.N, kbeg + (kt + 1) * BK, kend);
    }
#pragma unroll
    for (int kk = 0; kk < BK; kk += 16) {
      bf16x8_t af[FM], bfr[FN];
#pragma unroll
      for (int i = 0; i < FM; ++i)
        af[i] = __builtin_bit_cast(bf16x8_t,
                                   *(const uint4*)(As + lds_off(wm0 + i * 32 + fr, kk + fk)));
#pragma unroll
      for (int j = 0; j < FN; ++j)
        bfr[j] = __builtin_bit_cast(bf16x8_t,
                                    *(const uint4*)(Bs + lds_off(wn0 + j * 32 + fr, kk + fk)));
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j) {
          if constexpr (F16)
            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(f16x8_t, af[i]),
                                                               __builtin_bit_cast(f16x8_t, bfr[j]),
                                                               acc[i][j], 0, 0, 0);
          else
            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[i], bfr[j], acc[i][j], 0, 0, 0);
        }
    }
    if (kt + 1 < nk) {
      __syncthreads();
      ta.store(As);
      tb.store(Bs);
      __syncthreads();
    }
  }
  // acc[i][j][v] holds D[row][col] of the 32x32 tile with
  // row = 8 (v / 4) + 4 (lane / 32) + v % 4, col = lane % 32
  float* part = SPLIT ? a.ws + (long)blockIdx.z * a.M * a.N : nullptr;
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int m = m0 + wm0 + i * 32 + 8 * (v >> 2) + 4 * (lane >> 5) + (v & 3);
        const int n = n0 + wn0 + j * 32 + (lane & 31);
        if (m < a.M && n < a.N) {
          if constexpr (SPLIT)
            part[(long)m * a.N + n] = acc[i][j][v];
          else
            epi1<bf16, EPI>(a, m, n, acc[i][j][v]);
        }
      }
}

// The partial planes that hold column n: their first element for row 0 and
// column n, the row stride and plane size, and their count (two column groups,
// see GemmArgs::split_cols, or one).
struct SplitPlanes {
  const float* p;
  long ld, plane;
  int count;
};
__device__ inline SplitPlanes split_planes(const GemmArgs& a, int n) {
  if (a.split_cols && n >= a.split_cols) {
    const long ld = a.N - a.split_cols;
    return {a.ws + (long)a.splits * a.M * a.split_cols + (n - a.split_cols), ld, a.M * ld,
            a.splits2};
  }
  const long ld = a.split_cols ? a.split_cols : a.N;
  return {a.ws + n, ld, a.M * ld, a.splits};
}

// Sums the split partials in split order (deterministic) and applies the epilogue.
template <int EPI>
__global__ __launch_bounds__(256) void splitk_reduce_kernel(GemmArgs a) {
  const long tot = (long)a.M * a.N;
  for (long e = (long)blockIdx.x * 256 + threadIdx.x; e < tot; e += (long)gridDim.x * 256) {
    const int m = (int)(e / a.N), n = (int)(e % a.N);
    const SplitPlanes sp = split_planes(a, n);
    float s = 0.f;
    for (int z = 0; z < sp.count; ++z) s += sp.p[z * sp.plane + m * sp.ld];
    epi1<bf16, EPI>(a, m, n, s);
  }
}

// The same reduction, 8 consecutive columns per thread: 16-byte reads of the
// partials and of bf16 operands (bias, residual, z), 16-byte bf16 stores.
// Requires N, every leading dimension and H to be multiples of 8 and every
// pointer 16-byte aligned (checked by the launcher).
template <int EPI>
__global__ __launch_bounds__(256) void splitk_reduce8_kernel(GemmArgs a) {
  const long tot8 = (long)a.M * a.N / 8;
  const int n8 = a.N / 8;
  for (long e = (long)blockIdx.x * 256 + threadIdx.x; e < tot8; e += (long)gridDim.x * 256) {
    const int m = (int)(e / n8), n = (int)(e % n8) * 8;
    // split_cols is a multiple of 8: the 8 columns lie in one group
    const SplitPlanes sp = split_planes(a, n);
    float s[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    // RED planes' loads in flight before the first add (one memory round trip
    // per RED splits, not per split); the adds stay in split order
    constexpr int RED = 4;
    for (int z0 = 0; z0 < sp.count; z0 += RED) {
      float4 u[RED], w[RED];
#pragma unroll
      for (int k = 0; k < RED; ++k) {
        if (z0 + k < sp.count) {
          const float4* p = (const float4*)(sp.p + (z0 + k) * sp.plane + (long)m * sp.ld);
          u[k] = p[0], w[k] = p[1];
        }
      }
#pragma unroll
      for (int k = 0; k < RED; ++k) {
        if (z0 + k < sp.count) {
          s[0] += u[k].x, s[1] += u[k].y, s[2] += u[k].z, s[3] += u[k].w;
          s[4] += w[k].x, s[5] += w[k].y, s[6] += w[k].z, s[7] += w[k].w;
        }
      }
    }
    epi8<EPI>(a, m, n, s);
  }
}

template <int BM, int BN, int WGM, int WGN, bool A_KC, bool B_KC, bool SPLIT>
hipError_t launch_cfg(const GemmArgs& a, hipStream_t s) {
  dim3 grid(cdiv(a.N, BN), cdiv(a.M, BM), SPLIT ? a.splits : 1);
  constexpr int NTH = 64 * WGM * WGN;
  if (a.in_f16) {
    // fp16 operands: the query/key/value product (k-contiguous operands only)
    if constexpr (A_KC && B_KC) {
      if (SPLIT)
        gemm_mfma_kernel<BM, BN, WGM, WGN, true, true, EPI_STORE, true, true><<<grid, NTH, 0, s>>>(a);
      else if (a.epi == EPI_QKV)
        gemm_mfma_kernel<BM, BN, WGM, WGN, true, true, EPI_QKV, false, true><<<grid, NTH, 0, s>>>(a);
      else
        return hipErrorNotSupported;
      return hipGetLastError();
    } else {
      return hipErrorNotSupported;
    }
  }
  if constexpr (SPLIT) {
    gemm_mfma_kernel<BM, BN, WGM, WGN, A_KC, B_KC, EPI_STORE, true, false><<<grid, NTH, 0, s>>>(a);
  } else {
    switch (a.epi) {
#define TP_CASE(E) \
  case E: gemm_mfma_kernel<BM, BN, WGM, WGN, A_KC, B_KC, E, false, false><<<grid, NTH, 0, s>>>(a); break;
      TP_CASE(EPI_STORE)
      TP_CASE(EPI_QKV)
      TP_CASE(EPI_RESID)
      TP_CASE(EPI_GELU)
      TP_CASE(EPI_DGELU)
      TP_CASE(EPI_ACC_F32)
#undef TP_CASE
      default: return hipErrorInvalidValue;
    }
  }
  return hipGetLastError();
}

hipError_t launch_reduce(const GemmArgs& a, hipStream_t s) {
  const long tot = (long)a.M * a.N;
  if (vec8_ok(a)) {
    const int blocks = (int)std::min<long>(cdiv(tot / 8, 256), 4096);
    switch (a.epi) {
#define TP_CASE(E) \
  case E: splitk_reduce8_kernel<E><<<blocks, 256, 0, s>>>(a); break;
      TP_CASE(EPI_STORE)
      TP_CASE(EPI_QKV)
      TP_CASE(EPI_RESID)
      TP_CASE(EPI_GELU)
      TP_CASE(EPI_DGELU)
      TP_CASE(EPI_ACC_F32)
#undef TP_CASE
      default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
  }
  const int blocks = (int)std::min<long>(cdiv(tot, 256), 4096);
  switch (a.epi) {
#define TP_CASE(E) \
  case E: splitk_reduce_kernel<E><<<blocks, 256, 0, s>>>(a); break;
    TP_CASE(EPI_STORE)
    TP_CASE(EPI_QKV)
    TP_CASE(EPI_RESID)
    TP_CASE(EPI_GELU)
    TP_CASE(EPI_DGELU)
    TP_CASE(EPI_ACC_F32)
#undef TP_CASE
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

// Tile choice and split-K.  Slice-shaped products (M <= 256 tokens) take all
// rows in one block so every weight byte is fetched once; products over a
// whole sequence use 128 x 128 blocks.  Split-K raises the workgroup count to
// about three per CU while keeping >= 8 k-tiles per split.
template <int BM, int BN, int WGM, int WGN, bool A_KC, bool B_KC>
hipError_t run_cfg(GemmArgs a, hipStream_t s) {
  constexpr int TARGET_WGS = 768;
  const long tiles = (long)cdiv(a.M, BM) * cdiv(a.N, BN);
  int splits = 1;
  if (tiles < TARGET_WGS && a.ws) {
    splits = (int)std::min<long>(8, cdiv(TARGET_WGS, tiles));
    while (splits > 1 && (a.K / splits < 8 * BK || (long)splits * a.M * a.N > a.ws_elems))
      --splits;
  }
  if (a.need) {
    *a.need = splits > 1 ? (long)cdiv(a.K, cdiv(cdiv(a.K, splits), BK) * BK) * a.M * a.N : 0;
    return hipSuccess;
  }
  if (splits > 1) {
    a.k_split = cdiv(cdiv(a.K, splits), BK) * BK;
    a.splits = cdiv(a.K, a.k_split);
    hipError_t e = launch_cfg<BM, BN, WGM, WGN, A_KC, B_KC, true>(a, s);
    if (e != hipSuccess) return e;
    return launch_reduce(a, s);
  }
  return launch_cfg<BM, BN, WGM, WGN, A_KC, B_KC, false>(a, s);
}

template <bool A_KC, bool B_KC>
hipError_t launch_layout(const GemmArgs& a, hipStream_t s) {
  if (a.M <= 64) return run_cfg<64, 128, 1, 2, A_KC, B_KC>(a, s);
  if (a.M <= 128) return run_cfg<128, 128, 2, 2, A_KC, B_KC>(a, s);
  if (a.M <= 256) return run_cfg<256, 128, 4, 2, A_KC, B_KC>(a, s);
  return run_cfg<128, 128, 2, 2, A_KC, B_KC>(a, s);
}

}  // namespace

// 8-column vector epilogues: N, every leading dimension and H multiples of 8,
// every pointer 16-byte aligned
bool vec8_ok(const GemmArgs& a) {
  auto al = [](const void* p) { return ((uintptr_t)p & 15) == 0; };
  if (a.N % 8 || (a.ws && !al(a.ws)) || !al(a.C) || a.ldc % 8) return false;
  if (a.bias && !al(a.bias)) return false;
  if ((a.epi == EPI_RESID || a.epi == EPI_DGELU) && (!al(a.R) || a.ldr % 8)) return false;
  if (a.epi == EPI_GELU && (!al(a.C2) || a.ldc2 % 8)) return false;
  if (a.epi == EPI_QKV && (a.H % 8 || !al(a.q) || !al(a.k) || !al(a.v))) return false;
  if (a.epi == EPI_QKV && a.qkv_f16 && !al(a.vb)) return false;
  return true;
}

hipError_t gemm_splitk_reduce(const GemmArgs& a, hipStream_t s) { return launch_reduce(a, s); }

namespace {

inline bool al16(const void* p) { return ((uintptr_t)p & 15) == 0; }

}  // namespace

// bf16 operands whose contiguous dimension has unit stride, 16-byte aligned
// bases and leading dimensions that are multiples of 8 elements.  Returns
// hipErrorNotSupported when the shape is not covered (the caller falls back).
hipError_t gemm_mfma_bf16(const GemmArgs& a, hipStream_t s) {
  if (a.M <= 0 || a.N <= 0) return hipSuccess;
  const bool a_kc = a.sak == 1, a_mc = a.sam == 1;
  const bool b_kc = a.sbk == 1, b_nc = a.sbn == 1;
  if (!al16(a.A) || !al16(a.B)) return hipErrorNotSupported;
  const long lda = a_kc ? a.sam : a.sak, ldb = b_kc ? a.sbn : a.sbk;
  if ((lda & 7) || (ldb & 7)) return hipErrorNotSupported;
  if (a_kc && b_kc) return launch_layout<true, true>(a, s);
  if (a_kc && b_nc) return launch_layout<true, false>(a, s);
  if (a_mc && b_nc) return launch_layout<false, false>(a, s);
  return hipErrorNotSupported;
}

}  // namespace tp
