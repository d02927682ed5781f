// bf16 GEMM on the CDNA4 matrix cores: C = sum_k A(m,k) B(k,n) with fp32
// accumulation in v_mfma_f32_32x32x16_bf16, followed by the stage's fused
// epilogues.
//
// Block tile BM x BN x 64 with four waves in a 2 x 2 arrangement; each wave
// owns a (BM/2) x (BN/2) sub-tile made of 32 x 32 MFMA tiles.  Both operands
// sit in LDS k-contiguous ([row][64 k + 8 pad], the pad keeps the 16-byte
// fragment reads of 16 consecutive rows on distinct banks), so one ds_read_b128
// gives a lane its 8 consecutive k values.  An operand whose global layout is
// k-contiguous (activations; weights [out][in] in the forward) is copied with
// 16-byte loads; an operand that is contiguous along m or n (weights in the
// dX products, token-major activations and gradients in the dW products) is
// read as 4 (k) x 8 (m/n) blocks with 16-byte row loads and transposed in
// registers before it is written.  The next k-tile is fetched into registers
// while the current one is multiplied.
#include "tp_common.hpp"
#include "tp_kernels.hpp"

namespace tp {

namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

constexpr int BK = 64;
constexpr int LDK = BK + 8;  // LDS row stride in bf16 elements
constexpr int NT = 256;

template <typename T, int EPI>
__device__ inline void epi_store(const GemmArgs& a, int m, int n, float acc) {
  if constexpr (EPI == EPI_ACC_F32) {
    float* C = (float*)a.C + (long)m * a.ldc + n;
    *C += acc;
  } else if constexpr (EPI == EPI_DGELU) {
    const float z = ld((const T*)a.R + (long)m * a.ldr + n);
    st((T*)a.C + (long)m * a.ldc + n, acc * gelu_tanh_grad(z));
  } else {
    const float v = acc + (a.bias ? ld((const T*)a.bias + n) : 0.f);
    if constexpr (EPI == EPI_STORE) {
      st((T*)a.C + (long)m * a.ldc + n, v);
    } else if constexpr (EPI == EPI_RESID) {
      st((T*)a.C + (long)m * a.ldc + n, v + ld((const T*)a.R + (long)m * a.ldr + n));
    } else if constexpr (EPI == EPI_GELU) {
      st((T*)a.C + (long)m * a.ldc + n, v);
      st((T*)a.C2 + (long)m * a.ldc2 + n, gelu_tanh(v));
    } else if constexpr (EPI == EPI_QKV) {
      const int H = a.H;
      if (n < H)
        st((T*)a.q + (long)m * H + n, v);
      else if (n < 2 * H)
        st((T*)a.k + (long)m * H + (n - H), v);
      else
        st((T*)a.v + (long)m * H + (n - 2 * H), v);
    }
  }
}

// Operand tile of R rows (m or n) by BK k values, k-contiguous in global
// memory: X(r, k) = X[r * ld + k].  Chunks of 8 k values (16 bytes).
template <int R>
struct TileKC {
  static constexpr int CH = R * (BK / 8) / NT;  // chunks per thread
  static_assert(CH >= 1, "tile too small");
  uint4 v[CH];
  __device__ void load(const uint16_t* X, long ld, int r0, int rmax, int k0, int kmax) {
#pragma unroll
    for (int i = 0; i < CH; ++i) {
      const int c = threadIdx.x + NT * i;
      const int r = c >> 3, kc = (c & 7) * 8;
      const int gr = r0 + r, gk = k0 + kc;
      if (gr < rmax && gk + 8 <= kmax) {
        v[i] = *(const uint4*)(X + (long)gr * ld + gk);
      } else {
        uint16_t t[8];
#pragma unroll
        for (int e = 0; e < 8; ++e)
          t[e] = (gr < rmax && gk + e < kmax) ? X[(long)gr * ld + gk + e] : (uint16_t)0;
        v[i] = make_uint4(t[0] | (uint32_t)t[1] << 16, t[2] | (uint32_t)t[3] << 16,
                          t[4] | (uint32_t)t[5] << 16, t[6] | (uint32_t)t[7] << 16);
      }
    }
  }
  __device__ void store(uint16_t* lds) const {
#pragma unroll
    for (int i = 0; i < CH; ++i) {
      const int c = threadIdx.x + NT * i;
      const int r = c >> 3, kc = (c & 7) * 8;
      *(uint4*)(lds + r * LDK + kc) = v[i];
    }
  }
};

// Operand tile of R rows (m or n) by BK k values, contiguous along r in global
// memory: X(r, k) = X[k * ld + r].  Blocks of 4 k x 8 r, transposed in registers.
template <int R>
struct TileMC {
  static constexpr int NB = (BK / 4) * (R / 8);        // blocks per tile
  static constexpr int PER = (NB + NT - 1) / NT;       // blocks per thread
  uint2 v[PER][4];  // [block][k row] : 8 r values of one k (16 bytes as 2 x uint2)
  uint2 w[PER][4];
  __device__ void load(const uint16_t* X, long ld, int r0, int rmax, int k0, int kmax) {
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int b = threadIdx.x + NT * i;
      if (b >= NB) break;
      const int kb = b / (R / 8), rb = b % (R / 8);
      const int gr = r0 + rb * 8;
#pragma unroll
      for (int kk = 0; kk < 4; ++kk) {
        const int gk = k0 + kb * 4 + kk;
        uint4 x;
        if (gk < kmax && gr + 8 <= rmax) {
          x = *(const uint4*)(X + (long)gk * ld + gr);
        } else {
          uint16_t t[8];
#pragma unroll
          for (int e = 0; e < 8; ++e)
            t[e] = (gk < kmax && gr + e < rmax) ? X[(long)gk * ld + gr + e] : (uint16_t)0;
          x = make_uint4(t[0] | (uint32_t)t[1] << 16, t[2] | (uint32_t)t[3] << 16,
                         t[4] | (uint32_t)t[5] << 16, t[6] | (uint32_t)t[7] << 16);
        }
        v[i][kk] = make_uint2(x.x, x.y);
        w[i][kk] = make_uint2(x.z, x.w);
      }
    }
  }
  // element e (0..7) of k row kk
  __device__ static uint32_t half_word(const uint2& lo, const uint2& hi, int e) {
    const uint32_t d = e < 2 ? lo.x : e < 4 ? lo.y : e < 6 ? hi.x : hi.y;
    return d;
  }
  __device__ void store(uint16_t* lds) const {
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int b = threadIdx.x + NT * i;
      if (b >= NB) break;
      const int kb = b / (R / 8), rb = b % (R / 8);
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        // output row r = rb*8 + e holds k = kb*4 + 0..3
        const uint32_t d0 = half_word(v[i][0], w[i][0], e), d1 = half_word(v[i][1], w[i][1], e);
        const uint32_t d2 = half_word(v[i][2], w[i][2], e), d3 = half_word(v[i][3], w[i][3], e);
        const uint32_t sel = (e & 1) ? 0x07060302u : 0x05040100u;
        const uint32_t p0 = __builtin_amdgcn_perm(d1, d0, sel);
        const uint32_t p1 = __builtin_amdgcn_perm(d3, d2, sel);
        *(uint2*)(lds + (rb * 8 + e) * LDK + kb * 4) = make_uint2(p0, p1);
      }
    }
  }
};

template <int R, bool KC>
struct TileSel;
template <int R>
struct TileSel<R, true> {
  using type = TileKC<R>;
};
template <int R>
struct TileSel<R, false> {
  using type = TileMC<R>;
};

template <int BM, int BN, bool A_KC, bool B_KC, int EPI>
__global__ __launch_bounds__(NT) void gemm_mfma_kernel(GemmArgs a) {
  constexpr int WM = BM / 2, WN = BN / 2, FM = WM / 32, FN = WN / 32;
  __shared__ __attribute__((aligned(16))) uint16_t As[BM * LDK];
  __shared__ __attribute__((aligned(16))) uint16_t Bs[BN * LDK];
  const uint16_t* A = (const uint16_t*)a.A;
  const uint16_t* B = (const uint16_t*)a.B;
  const long lda = A_KC ? a.sam : a.sak;
  const long ldb = B_KC ? a.sbn : a.sbk;
  const int m0 = blockIdx.y * BM, n0 = blockIdx.x * BN;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm0 = (wave >> 1) * WM, wn0 = (wave & 1) * WN;

  typename TileSel<BM, A_KC>::type ta;
  typename TileSel<BN, B_KC>::type tb;
  f32x16_t acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;

  const int nk = (a.K + BK - 1) / BK;
  ta.load(A, lda, m0, a.M, 0, a.K);
  tb.load(B, ldb, n0, a.N, 0, a.K);
  ta.store(As);
  tb.store(Bs);
  __syncthreads();
  const int fr = lane & 31, fk = (lane >> 5) * 8;
  for (int kt = 0; kt < nk; ++kt) {
    if (kt + 1 < nk) {
      ta.load(A, lda, m0, a.M, (kt + 1) * BK, a.K);
      tb.load(B, ldb, n0, a.N, (kt + 1) * BK, a.K);
    }
#pragma unroll
    for (int kk = 0; kk < BK; kk += 16) {
      bf16x8_t af[FM], bfr[FN];
#pragma unroll
      for (int i = 0; i < FM; ++i) {
        const uint4 x = *(const uint4*)(As + (wm0 + i * 32 + fr) * LDK + kk + fk);
        af[i] = __builtin_bit_cast(bf16x8_t, x);
      }
#pragma unroll
      for (int j = 0; j < FN; ++j) {
        const uint4 x = *(const uint4*)(Bs + (wn0 + j * 32 + fr) * LDK + kk + fk);
        bfr[j] = __builtin_bit_cast(bf16x8_t, x);
      }
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[i], bfr[j], acc[i][j], 0, 0, 0);
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
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int m = m0 + wm0 + i * 32 + 8 * (v >> 2) + 4 * (lane >> 5) + (v & 3);
        const int n = n0 + wn0 + j * 32 + (lane & 31);
        if (m < a.M && n < a.N) epi_store<bf16, EPI>(a, m, n, acc[i][j][v]);
      }
}

template <int BM, int BN, bool A_KC, bool B_KC>
hipError_t launch_cfg(const GemmArgs& a, hipStream_t s) {
  dim3 grid(cdiv(a.N, BN), cdiv(a.M, BM));
  switch (a.epi) {
    case EPI_STORE: gemm_mfma_kernel<BM, BN, A_KC, B_KC, EPI_STORE><<<grid, NT, 0, s>>>(a); break;
    case EPI_QKV: gemm_mfma_kernel<BM, BN, A_KC, B_KC, EPI_QKV><<<grid, NT, 0, s>>>(a); break;
    case EPI_RESID: gemm_mfma_kernel<BM, BN, A_KC, B_KC, EPI_RESID><<<grid, NT, 0, s>>>(a); break;
    case EPI_GELU: gemm_mfma_kernel<BM, BN, A_KC, B_KC, EPI_GELU><<<grid, NT, 0, s>>>(a); break;
    case EPI_DGELU: gemm_mfma_kernel<BM, BN, A_KC, B_KC, EPI_DGELU><<<grid, NT, 0, s>>>(a); break;
    case EPI_ACC_F32:
      gemm_mfma_kernel<BM, BN, A_KC, B_KC, EPI_ACC_F32><<<grid, NT, 0, s>>>(a);
      break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

template <bool A_KC, bool B_KC>
hipError_t launch_layout(const GemmArgs& a, hipStream_t s) {
  if (a.M <= 64) return launch_cfg<64, 128, A_KC, B_KC>(a, s);
  if (a.M <= 128) return launch_cfg<128, 128, A_KC, B_KC>(a, s);
  return launch_cfg<256, 128, A_KC, B_KC>(a, s);
}

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
