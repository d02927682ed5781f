// Prefix-causal attention of a token slice on the CDNA4 matrix cores (bf16
// operands, fp32 accumulation, v_mfma_f32_32x32x16_bf16), head width 64 or 128.
//
// Queries t in [l, r) attend keys s <= t of the per-layer cache [0, r) (Eq. 2
// with every earlier slice's keys/values cached).
//
// MFMA fragment conventions (32 x 32 x 16): a lane l = 32 G + c supplies row c
// of the left operand and column c of the right operand, 8 values each at the
// lane group's 8 reduction slots; the accumulator element v of lane l is
// D[8 (v / 4) + 4 G + v % 4][c].  A score tile computed by one MFMA therefore
// gives each lane one column and 16 rows; when those 16 values feed the next
// MFMA as an operand, the reduction slot e of group G stands for row
// 16 ks + (e < 4 ? 4 G + e : 8 + 4 G + e - 4) (ks = which half of the 32),
// and the other operand is read from LDS with the same pairing.
//
//  forward  : S^T = K Q^T (lane = one query, so the online softmax is
//             lane-local plus one exchange with lane ^ 32), O^T += V^T P^T.
//  dK/dV    : one block of keys per wave; S = Q K^T and dP = dO V^T (lane =
//             one key), dV += P^T dO, dK += dS^T Q; results are added to the
//             fp32 dK/dV buffer (each element owned by one lane: no atomics).
//  dQ       : one block of queries per wave; S^T = K Q^T, dP^T = V dO^T,
//             dQ^T += K^T dS^T.
// Tiles that must be read along the key/query index are transposed in
// registers on their way into LDS.
#include "tp_common.hpp"
#include "tp_kernels.hpp"

namespace tp {

namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

constexpr float LOG2E = 1.4426950408889634f;
constexpr float LN2 = 0.6931471805599453f;

__device__ inline f32x16_t mfma(bf16x8_t a, bf16x8_t b, f32x16_t c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

__device__ inline f32x16_t zero16() {
  f32x16_t z;
#pragma unroll
  for (int v = 0; v < 16; ++v) z[v] = 0.f;
  return z;
}

__device__ inline uint32_t pack_bf16x2(float lo, float hi) {
  return (uint32_t)f32_to_bf16_bits(lo) | ((uint32_t)f32_to_bf16_bits(hi) << 16);
}

// 8 accumulator values (one reduction half) as a bf16 operand.
__device__ inline bf16x8_t acc_half_bf16(const f32x16_t& x, int ks) {
  uint4 u;
  if (ks == 0)
    u = make_uint4(pack_bf16x2(x[0], x[1]), pack_bf16x2(x[2], x[3]), pack_bf16x2(x[4], x[5]),
                   pack_bf16x2(x[6], x[7]));
  else
    u = make_uint4(pack_bf16x2(x[8], x[9]), pack_bf16x2(x[10], x[11]),
                   pack_bf16x2(x[12], x[13]), pack_bf16x2(x[14], x[15]));
  return __builtin_bit_cast(bf16x8_t, u);
}

// Operand read from a row of an LDS tile that is contiguous along the
// reduction index, in the paired slot order: 4 values at k0 + 4G and 4 at
// k0 + 8 + 4G.
__device__ inline bf16x8_t lds_pair_read(const uint16_t* row, int k0, int G) {
  const uint2 a = *(const uint2*)(row + k0 + 4 * G);
  const uint2 b = *(const uint2*)(row + k0 + 8 + 4 * G);
  return __builtin_bit_cast(bf16x8_t, make_uint4(a.x, a.y, b.x, b.y));
}

__device__ inline bf16x8_t lds_read16(const uint16_t* p) {
  return __builtin_bit_cast(bf16x8_t, *(const uint4*)p);
}

// LDS[r][c] = G[r][c] (row stride ld) for r < ROWS, c < COLS; rows >= rvalid are 0.
template <int ROWS, int COLS, int LDR, int NTH>
__device__ inline void lds_copy(uint16_t* lds, const uint16_t* G, long ld, int rvalid) {
  constexpr int CPR = COLS / 8, TOT = ROWS * CPR;
#pragma unroll
  for (int c = threadIdx.x; c < TOT; c += NTH) {
    const int r = c / CPR, k = (c % CPR) * 8;
    uint4 v = make_uint4(0, 0, 0, 0);
    if (r < rvalid) v = *(const uint4*)(G + (long)r * ld + k);
    *(uint4*)(lds + r * LDR + k) = v;
  }
}

__device__ inline uint32_t word_of(const uint4& x, int w) {
  return w == 0 ? x.x : w == 1 ? x.y : w == 2 ? x.z : x.w;
}

// LDS[c][r] = G[r][c] (transpose; LDS row stride LDR runs over r) for r < ROWS,
// c < COLS; rows r >= rvalid are 0.  Blocks of 4 rows x 8 columns per thread.
template <int ROWS, int COLS, int LDR, int NTH>
__device__ inline void lds_copy_t(uint16_t* lds, const uint16_t* G, long ld, int rvalid) {
  constexpr int CB = COLS / 8, TOT = (ROWS / 4) * CB;
  for (int b = threadIdx.x; b < TOT; b += NTH) {
    const int rb = b / CB, cb = b % CB;
    uint4 x[4];
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) {
      const int r = rb * 4 + kk;
      x[kk] = r < rvalid ? *(const uint4*)(G + (long)r * ld + cb * 8) : make_uint4(0, 0, 0, 0);
    }
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const uint32_t sel = (e & 1) ? 0x07060302u : 0x05040100u;
      const uint32_t p0 = __builtin_amdgcn_perm(word_of(x[1], e >> 1), word_of(x[0], e >> 1), sel);
      const uint32_t p1 = __builtin_amdgcn_perm(word_of(x[3], e >> 1), word_of(x[2], e >> 1), sel);
      *(uint2*)(lds + (cb * 8 + e) * LDR + rb * 4) = make_uint2(p0, p1);
    }
  }
}

// ------------------------------------------------------------------ forward

template <int D, int NW>
__global__ __launch_bounds__(64 * NW) void attn_fwd_mfma(AttnArgs a) {
  constexpr int NTH = 64 * NW, BKV = 64, LDK = D + 8, LDV = BKV + 8, KS = D / 16, JB = D / 32;
  __shared__ __attribute__((aligned(16))) uint16_t Ks[BKV * LDK];
  __shared__ __attribute__((aligned(16))) uint16_t Vt[D * LDV];
  const int h = blockIdx.y, lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int G = lane >> 5, c = lane & 31, H = a.H;
  const int q_lo = a.l + blockIdx.x * 32 * NW;       // first query of the block
  const int t = q_lo + 32 * w + c;                    // this lane's query
  const bool tvalid = t < a.r;
  const int kend_blk = min(a.r, q_lo + 32 * NW);      // keys the block needs
  const int kend_w = min(a.r, q_lo + 32 * w + 32);    // keys this wave needs
  const uint16_t* Q = (const uint16_t*)a.q;
  const uint16_t* Kc = (const uint16_t*)a.kc + h * D;
  const uint16_t* Vc = (const uint16_t*)a.vc + h * D;

  bf16x8_t qf[KS];
#pragma unroll
  for (int kk = 0; kk < KS; ++kk) {
    uint4 v = make_uint4(0, 0, 0, 0);
    if (tvalid) v = *(const uint4*)(Q + (long)(t - a.l) * H + h * D + 16 * kk + 8 * G);
    qf[kk] = __builtin_bit_cast(bf16x8_t, v);
  }
  const float sl2 = a.scale * LOG2E;
  float m = -INFINITY, lsum = 0.f;
  f32x16_t o[JB];
#pragma unroll
  for (int j = 0; j < JB; ++j) o[j] = zero16();

  for (int kb = 0; kb < kend_blk; kb += BKV) {
    const int kval = min(BKV, kend_blk - kb);
    lds_copy<BKV, D, LDK, NTH>(Ks, Kc + (long)kb * H, H, kval);
    lds_copy_t<BKV, D, LDV, NTH>(Vt, Vc + (long)kb * H, H, kval);
    __syncthreads();
    if (kb < kend_w) {
      f32x16_t p[2];
#pragma unroll
      for (int sb = 0; sb < 2; ++sb) {
        f32x16_t s = zero16();
        if (kb + 32 * sb < kend_w) {
#pragma unroll
          for (int kk = 0; kk < KS; ++kk)
            s = mfma(lds_read16(Ks + (32 * sb + c) * LDK + 16 * kk + 8 * G), qf[kk], s);
        }
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const int key = kb + 32 * sb + 8 * (v >> 2) + 4 * G + (v & 3);
          p[sb][v] = (key <= t && key < a.r) ? s[v] * sl2 : -INFINITY;
        }
      }
      float mx = -INFINITY;
#pragma unroll
      for (int v = 0; v < 16; ++v) mx = fmaxf(mx, fmaxf(p[0][v], p[1][v]));
      mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
      const float mnew = fmaxf(m, mx);
      const float alpha = (mnew == -INFINITY) ? 1.f : exp2f(m - mnew);
      float rs = 0.f;
#pragma unroll
      for (int sb = 0; sb < 2; ++sb)
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const float e = (mnew == -INFINITY) ? 0.f : exp2f(p[sb][v] - mnew);
          p[sb][v] = e;
          rs += e;
        }
      rs += __shfl_xor(rs, 32, 64);
      lsum = lsum * alpha + rs;
      m = mnew;
#pragma unroll
      for (int j = 0; j < JB; ++j)
#pragma unroll
        for (int v = 0; v < 16; ++v) o[j][v] *= alpha;
#pragma unroll
      for (int sb = 0; sb < 2; ++sb) {
        if (kb + 32 * sb >= kend_w) break;
#pragma unroll
        for (int ks = 0; ks < 2; ++ks) {
          const bf16x8_t pb = acc_half_bf16(p[sb], ks);
#pragma unroll
          for (int j = 0; j < JB; ++j)
            o[j] = mfma(lds_pair_read(Vt + (32 * j + c) * LDV, 32 * sb + 16 * ks, G), pb, o[j]);
        }
      }
    }
    __syncthreads();
  }
  if (tvalid) {
    const float inv = lsum > 0.f ? 1.f / lsum : 0.f;
    uint16_t* O = (uint16_t*)a.o + (long)(t - a.l) * H + h * D;
#pragma unroll
    for (int j = 0; j < JB; ++j)
#pragma unroll
      for (int v = 0; v < 16; v += 4) {
        const int col = 32 * j + 8 * (v >> 2) + 4 * G;
        *(uint2*)(O + col) = make_uint2(pack_bf16x2(o[j][v] * inv, o[j][v + 1] * inv),
                                        pack_bf16x2(o[j][v + 2] * inv, o[j][v + 3] * inv));
      }
    if (G == 0) a.lse[(long)h * a.Lmax + t] = (m + log2f(lsum)) * LN2;
  }
}

// ------------------------------------------------------ backward prologue

// D[h][t] = sum_j dO[t][h d + j] * O[t][h d + j]; one wave per (row, head).
template <int D>
__global__ __launch_bounds__(256) void attn_bwd_rowdot(AttnArgs a) {
  const int wave = (blockIdx.x * 256 + threadIdx.x) >> 6, lane = threadIdx.x & 63;
  const int n = a.r - a.l;
  if (wave >= n * a.heads) return;
  const int i = wave / a.heads, h = wave % a.heads;
  const uint16_t* dO = (const uint16_t*)a.dout + (long)i * a.H + h * D;
  const uint16_t* O = (const uint16_t*)a.o + (long)i * a.H + h * D;
  float s = 0.f;
  for (int j = lane; j < D; j += 64) s += to_f32(bf16{dO[j]}) * to_f32(bf16{O[j]});
  s = wave_sum(s);
  if (lane == 0) a.D[(long)h * a.Lmax + a.l + i] = s;
}

// ------------------------------------------------------------ dK / dV

template <int D, int NW>
__global__ __launch_bounds__(64 * NW) void attn_bwd_dkdv_mfma(AttnArgs a) {
  constexpr int NTH = 64 * NW, BQ = 32, LDQ = D + 8, LDT = BQ + 8, KS = D / 16, JB = D / 32;
  __shared__ __attribute__((aligned(16))) uint16_t Qs[BQ * LDQ];
  __shared__ __attribute__((aligned(16))) uint16_t Qt[D * LDT];
  __shared__ __attribute__((aligned(16))) uint16_t Os[BQ * LDQ];  // dO rows
  __shared__ __attribute__((aligned(16))) uint16_t Ot[D * LDT];   // dO transposed
  __shared__ float lse2_s[BQ], Dd_s[BQ];
  const int h = blockIdx.y, lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int G = lane >> 5, c = lane & 31, H = a.H;
  const int k_lo = blockIdx.x * 32 * NW;     // first key of the block
  const int s_w = k_lo + 32 * w;             // first key of this wave
  const int s_me = s_w + c;                  // this lane's key (column of S)
  const uint16_t* Kc = (const uint16_t*)a.kc + h * D;
  const uint16_t* Vc = (const uint16_t*)a.vc + h * D;
  const uint16_t* Q = (const uint16_t*)a.q + h * D;
  const uint16_t* dO = (const uint16_t*)a.dout + h * D;

  bf16x8_t kf[KS], vf[KS];
#pragma unroll
  for (int kk = 0; kk < KS; ++kk) {
    uint4 x = make_uint4(0, 0, 0, 0), y = make_uint4(0, 0, 0, 0);
    if (s_me < a.r) {
      x = *(const uint4*)(Kc + (long)s_me * H + 16 * kk + 8 * G);
      y = *(const uint4*)(Vc + (long)s_me * H + 16 * kk + 8 * G);
    }
    kf[kk] = __builtin_bit_cast(bf16x8_t, x);
    vf[kk] = __builtin_bit_cast(bf16x8_t, y);
  }
  f32x16_t dk[JB], dv[JB];
#pragma unroll
  for (int j = 0; j < JB; ++j) dk[j] = dv[j] = zero16();
  const float sl2 = a.scale * LOG2E;
  const int n = a.r - a.l;
  // query rows i = t - l that can see a key of this block: t >= k_lo
  const int i_begin = max(0, k_lo - a.l) & ~(BQ - 1);
  for (int i0 = i_begin; i0 < n; i0 += BQ) {
    const int qval = min(BQ, n - i0);
    lds_copy<BQ, D, LDQ, NTH>(Qs, Q + (long)i0 * H, H, qval);
    lds_copy_t<BQ, D, LDT, NTH>(Qt, Q + (long)i0 * H, H, qval);
    lds_copy<BQ, D, LDQ, NTH>(Os, dO + (long)i0 * H, H, qval);
    lds_copy_t<BQ, D, LDT, NTH>(Ot, dO + (long)i0 * H, H, qval);
    if (threadIdx.x < BQ) {
      const int tq = a.l + i0 + threadIdx.x;
      const bool ok = threadIdx.x < qval;
      lse2_s[threadIdx.x] = ok ? a.lse[(long)h * a.Lmax + tq] * LOG2E : 0.f;
      Dd_s[threadIdx.x] = ok ? a.D[(long)h * a.Lmax + tq] : 0.f;
    }
    __syncthreads();
    // the wave's keys [s_w, s_w + 32) meet queries up to l + i0 + qval - 1
    if (s_w <= a.l + i0 + qval - 1 && s_w < a.r) {
      f32x16_t s = zero16(), dp = zero16();
#pragma unroll
      for (int kk = 0; kk < KS; ++kk) {
        s = mfma(lds_read16(Qs + c * LDQ + 16 * kk + 8 * G), kf[kk], s);
        dp = mfma(lds_read16(Os + c * LDQ + 16 * kk + 8 * G), vf[kk], dp);
      }
      // s[v], dp[v]: query row qi = 8 (v / 4) + 4 G + v % 4 of the block, key s_me
      f32x16_t p, ds;
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int qi = 8 * (v >> 2) + 4 * G + (v & 3);
        const int tq = a.l + i0 + qi;
        const bool ok = qi < qval && s_me <= tq;
        const float pv = ok ? exp2f(s[v] * sl2 - lse2_s[qi]) : 0.f;
        p[v] = pv;
        ds[v] = pv * (dp[v] - Dd_s[qi]);
      }
#pragma unroll
      for (int ks = 0; ks < 2; ++ks) {
        const bf16x8_t pb = acc_half_bf16(p, ks), db = acc_half_bf16(ds, ks);
#pragma unroll
        for (int j = 0; j < JB; ++j) {
          dv[j] = mfma(pb, lds_pair_read(Ot + (32 * j + c) * LDT, 16 * ks, G), dv[j]);
          dk[j] = mfma(db, lds_pair_read(Qt + (32 * j + c) * LDT, 16 * ks, G), dk[j]);
        }
      }
    }
    __syncthreads();
  }
  // dk[j][v], dv[j][v]: key s_w + 8 (v / 4) + 4 G + v % 4, column 32 j + c
#pragma unroll
  for (int j = 0; j < JB; ++j)
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      const int key = s_w + 8 * (v >> 2) + 4 * G + (v & 3);
      if (key < a.r) {
        const long off = (long)key * H + h * D + 32 * j + c;
        a.dk[off] += dk[j][v] * a.scale;
        a.dv[off] += dv[j][v];
      }
    }
}

// ------------------------------------------------------------------- dQ

template <int D, int NW>
__global__ __launch_bounds__(64 * NW) void attn_bwd_dq_mfma(AttnArgs a) {
  constexpr int NTH = 64 * NW, BKV = 64, LDK = D + 8, LDT = BKV + 8, KS = D / 16, JB = D / 32;
  __shared__ __attribute__((aligned(16))) uint16_t Ks[BKV * LDK];
  __shared__ __attribute__((aligned(16))) uint16_t Kt[D * LDT];
  __shared__ __attribute__((aligned(16))) uint16_t Vs[BKV * LDK];
  const int h = blockIdx.y, lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int G = lane >> 5, c = lane & 31, H = a.H;
  const int q_lo = a.l + blockIdx.x * 32 * NW;
  const int t = q_lo + 32 * w + c;
  const bool tvalid = t < a.r;
  const int kend_blk = min(a.r, q_lo + 32 * NW);
  const int kend_w = min(a.r, q_lo + 32 * w + 32);
  const uint16_t* Kc = (const uint16_t*)a.kc + h * D;
  const uint16_t* Vc = (const uint16_t*)a.vc + h * D;

  bf16x8_t qf[KS], of[KS];
#pragma unroll
  for (int kk = 0; kk < KS; ++kk) {
    uint4 x = make_uint4(0, 0, 0, 0), y = make_uint4(0, 0, 0, 0);
    if (tvalid) {
      const long off = (long)(t - a.l) * H + h * D + 16 * kk + 8 * G;
      x = *(const uint4*)((const uint16_t*)a.q + off);
      y = *(const uint4*)((const uint16_t*)a.dout + off);
    }
    qf[kk] = __builtin_bit_cast(bf16x8_t, x);
    of[kk] = __builtin_bit_cast(bf16x8_t, y);
  }
  const float sl2 = a.scale * LOG2E;
  const float lse2 = tvalid ? a.lse[(long)h * a.Lmax + t] * LOG2E : 0.f;
  const float Dt = tvalid ? a.D[(long)h * a.Lmax + t] : 0.f;
  f32x16_t dq[JB];
#pragma unroll
  for (int j = 0; j < JB; ++j) dq[j] = zero16();

  for (int kb = 0; kb < kend_blk; kb += BKV) {
    const int kval = min(BKV, kend_blk - kb);
    lds_copy<BKV, D, LDK, NTH>(Ks, Kc + (long)kb * H, H, kval);
    lds_copy_t<BKV, D, LDT, NTH>(Kt, Kc + (long)kb * H, H, kval);
    lds_copy<BKV, D, LDK, NTH>(Vs, Vc + (long)kb * H, H, kval);
    __syncthreads();
#pragma unroll
    for (int sb = 0; sb < 2; ++sb) {
      if (kb + 32 * sb >= kend_w) break;
      f32x16_t s = zero16(), dp = zero16();
#pragma unroll
      for (int kk = 0; kk < KS; ++kk) {
        s = mfma(lds_read16(Ks + (32 * sb + c) * LDK + 16 * kk + 8 * G), qf[kk], s);
        dp = mfma(lds_read16(Vs + (32 * sb + c) * LDK + 16 * kk + 8 * G), of[kk], dp);
      }
      f32x16_t ds;
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int key = kb + 32 * sb + 8 * (v >> 2) + 4 * G + (v & 3);
        const bool ok = tvalid && key <= t;
        const float pv = ok ? exp2f(s[v] * sl2 - lse2) : 0.f;
        ds[v] = pv * (dp[v] - Dt);
      }
#pragma unroll
      for (int ks = 0; ks < 2; ++ks) {
        const bf16x8_t db = acc_half_bf16(ds, ks);
#pragma unroll
        for (int j = 0; j < JB; ++j)
          dq[j] = mfma(lds_pair_read(Kt + (32 * j + c) * LDT, 32 * sb + 16 * ks, G), db, dq[j]);
      }
    }
    __syncthreads();
  }
  if (tvalid) {
    uint16_t* dQ = (uint16_t*)a.dq + (long)(t - a.l) * a.ld_dq + h * D;
#pragma unroll
    for (int j = 0; j < JB; ++j)
#pragma unroll
      for (int v = 0; v < 16; v += 4) {
        const int col = 32 * j + 8 * (v >> 2) + 4 * G;
        *(uint2*)(dQ + col) =
            make_uint2(pack_bf16x2(dq[j][v] * a.scale, dq[j][v + 1] * a.scale),
                       pack_bf16x2(dq[j][v + 2] * a.scale, dq[j][v + 3] * a.scale));
      }
  }
}

constexpr int NWF = 4;  // waves per block

template <int D>
hipError_t fwd_d(const AttnArgs& a, hipStream_t s) {
  const int n = a.r - a.l;
  dim3 grid(cdiv(n, 32 * NWF), a.heads);
  attn_fwd_mfma<D, NWF><<<grid, 64 * NWF, 0, s>>>(a);
  return hipGetLastError();
}

template <int D>
hipError_t bwd_d(const AttnArgs& a, hipStream_t s) {
  const int n = a.r - a.l;
  attn_bwd_rowdot<D><<<cdiv((long)n * a.heads, 4), 256, 0, s>>>(a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  attn_bwd_dkdv_mfma<D, NWF><<<dim3(cdiv(a.r, 32 * NWF), a.heads), 64 * NWF, 0, s>>>(a);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  attn_bwd_dq_mfma<D, NWF><<<dim3(cdiv(n, 32 * NWF), a.heads), 64 * NWF, 0, s>>>(a);
  return hipGetLastError();
}

inline bool al16(const void* p) { return ((uintptr_t)p & 15) == 0; }

bool covered(const AttnArgs& a) {
  return (a.d == 64 || a.d == 128) && (a.H % 8) == 0 && al16(a.q) && al16(a.kc) && al16(a.vc);
}

}  // namespace

hipError_t attn_fwd_mfma_bf16(const AttnArgs& a, hipStream_t s) {
  if (!covered(a) || !al16(a.o)) return hipErrorNotSupported;
  return a.d == 128 ? fwd_d<128>(a, s) : fwd_d<64>(a, s);
}

hipError_t attn_bwd_mfma_bf16(const AttnArgs& a, hipStream_t s) {
  if (!covered(a) || !al16(a.dout) || !al16(a.dq) || (a.ld_dq % 8)) return hipErrorNotSupported;
  return a.d == 128 ? bwd_d<128>(a, s) : bwd_d<64>(a, s);
}

}  // namespace tp
