// Prefix-causal attention of a token slice on the CDNA4 matrix cores (bf16
// operands, fp32 accumulation, v_mfma_f32_32x32x16_bf16), head width 64 or 128.
//
// Queries t in [l, r) attend keys s <= t of the per-layer cache [0, r) (Eq. 2
// with every earlier slice's keys/values cached).
//
// MFMA fragment conventions (32 x 32 x 16): lane l = 32 G + c supplies row c of
// the left operand and column c of the right operand, 8 values each at its
// group's 8 reduction slots; accumulator element v of lane l is
// D[8 (v / 4) + 4 G + v % 4][c].  A score tile computed by one MFMA thus gives
// each lane one column and 16 rows; fed back as an operand, reduction slot e of
// group G stands for row 16 ks + (e < 4 ? 4 G + e : 8 + 4 G + e - 4)
// (ks = which half of the 32).  The other operand of such a product is read
// from an LDS tile with two transposing reads (ds_read_b64_tr_b16) whose row
// bases follow the same pairing, so tiles stay in their natural [token][d]
// orientation in LDS.
//
//  forward  : S^T = K Q^T (lane = one query: the online softmax is lane-local
//             plus one exchange with lane ^ 32), O^T += V^T P^T.
//  dK/dV    : one block of 32 keys per wave; S = Q K^T and dP = dO V^T (lane =
//             one key), dV += P^T dO, dK += dS^T Q; results are added to the
//             fp32 dK/dV buffer (each element owned by one lane: no atomics).
//  dQ       : one block of 32 queries per wave; S^T = K Q^T, dP^T = V dO^T,
//             dQ^T += K^T dS^T.
//  stored dS: the dK kernel also writes dS of every (key, query) block it
//             forms; dQ^T += K^T dS^T then streams it instead of forming the
//             scores and dP once more.
// K/V (or Q/dO) tiles move from HBM to a double-buffered LDS ring by the LDS
// DMA, so the next tile streams in while the current one is multiplied.
#include "tp_common.hpp"
#include "tp_kernels.hpp"
#include "tp_lds.hpp"

namespace tp {

namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

constexpr float LOG2E = 1.4426950408889634f;
constexpr float LN2 = 0.6931471805599453f;

typedef _Float16 f16x8_t __attribute__((ext_vector_type(8)));

__device__ inline f32x16_t mfma(u32x4 a, u32x4 b, f32x16_t c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, a),
                                                 __builtin_bit_cast(bf16x8_t, b), c, 0, 0, 0);
}
// fp16 operands (F16) or bf16
template <bool F16>
__device__ inline f32x16_t mfma_t(u32x4 a, u32x4 b, f32x16_t c) {
  if constexpr (F16)
    return __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(f16x8_t, a),
                                                  __builtin_bit_cast(f16x8_t, b), c, 0, 0, 0);
  else
    return mfma(a, b, c);
}

__device__ inline f32x16_t zero16() {
  f32x16_t z;
#pragma unroll
  for (int v = 0; v < 16; ++v) z[v] = 0.f;
  return z;
}

// Two fp32 values as round-to-nearest-even bf16 (lo in the low half), one
// v_cvt_pk_bf16_f32.
__device__ inline uint32_t pack_bf16x2(float lo, float hi) {
  typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
  typedef float f32x2_t __attribute__((ext_vector_type(2)));
  return __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2_t){lo, hi}, bf16x2_t));
}

// 2^x as the bare v_exp_f32 (results below the normal range flush to 0, which
// a softmax weight may do).
__device__ inline float exp2_fast(float x) { return __builtin_amdgcn_exp2f(x); }

// IEEE maximum (NaN-propagating; v_maximum3_f32 needs no operand
// canonicalisation, unlike fmaxf).
__device__ inline float fmax_ieee(float a, float b) { return __builtin_elementwise_maximum(a, b); }

// Lanes l and l ^ 32 combined: after v_permlane32_swap every lane holds the
// lower half's value in .x and the upper half's in .y, so both lanes of a pair
// compute op(lower, upper) and get the same result.
__device__ inline float2 halves(float v) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false,
                                                  false);
  return make_float2(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ inline float pair_max(float v) {
  const float2 h = halves(v);
  return fmax_ieee(h.x, h.y);
}
__device__ inline float pair_sum(float v) {
  const float2 h = halves(v);
  return h.x + h.y;
}

// 8 accumulator values (one reduction half) as a bf16 operand.
__device__ inline u32x4 acc_half_bf16(const f32x16_t& x, int ks) {
  u32x4 u;
  const int o = 8 * ks;
  u.x = pack_bf16x2(x[o + 0], x[o + 1]);
  u.y = pack_bf16x2(x[o + 2], x[o + 3]);
  u.z = pack_bf16x2(x[o + 4], x[o + 5]);
  u.w = pack_bf16x2(x[o + 6], x[o + 7]);
  return u;
}
// Two fp32 values as round-to-nearest-even fp16 (lo in the low half).
__device__ inline uint32_t pack_f16x2(float lo, float hi) {
  typedef _Float16 f16x2_t __attribute__((ext_vector_type(2)));
  typedef float f32x2_t __attribute__((ext_vector_type(2)));
  return __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2_t){lo, hi}, f16x2_t));
}
// 8 accumulator values as an fp16 (F16) or bf16 operand.
template <bool F16>
__device__ inline u32x4 acc_half(const f32x16_t& x, int ks) {
  if constexpr (F16) {
    u32x4 u;
    const int o = 8 * ks;
    u.x = pack_f16x2(x[o + 0], x[o + 1]);
    u.y = pack_f16x2(x[o + 2], x[o + 3]);
    u.z = pack_f16x2(x[o + 4], x[o + 5]);
    u.w = pack_f16x2(x[o + 6], x[o + 7]);
    return u;
  } else {
    return acc_half_bf16(x, ks);
  }
}

// Tile of rows x D bf16 in LDS, rows of 2D bytes whose 16-byte chunks are
// permuted by chunk ^ f(row).  f makes both the row-fragment reads (16
// consecutive rows at one chunk) and the transposing reads (8 rows x 4 chunks)
// use every bank group at most twice.
template <int D>
struct Tile {
  static constexpr int CPR = D / 8;
  __device__ static int f(int r) {
    if constexpr (D == 128) return ((r & 3) << 2) | ((r >> 2) & 3);
    else return (r >> 1) & 7;
  }
  // byte offset of chunk c of row r
  __device__ static uint32_t off(int r, int c) { return r * (2 * D) + ((c ^ f(r)) << 4); }
  // 8 consecutive d values [8c, 8c+8) of row r
  __device__ static u32x4 row8(uint32_t base, int r, int c) { return ds_read128(base + off(r, c)); }
  // transposed operand: this lane's column cb + (lane % 32) at rows
  // r0 + 4 G + (0..3) and r0 + 8 + 4 G + (0..3) (the pairing of the header)
  __device__ static u32x4 col8(uint32_t base, int r0, int cb, int lane) {
    const int g = lane >> 4, j = lane & 15;
    const int col = cb + 16 * (g & 1) + 4 * (j & 3);
    const int r = r0 + 4 * (g >> 1) + (j >> 2);
    const uint32_t inchunk = (col & 7) << 1;
    const u32x2 lo = ds_read_tr(base + off(r, col >> 3) + inchunk);
    const u32x2 hi = ds_read_tr(base + off(r + 8, col >> 3) + inchunk);
    return join(lo, hi);
  }
  // DMA of full ROWS-row tiles with this thread's chunk offsets (bytes from
  // the tile's first row, rows of ld elements) computed once, so a tile only
  // moves the wave-uniform origin; a tile with fewer valid rows takes `dma`.
  template <int ROWS, int NTH>
  struct Dma {
    static constexpr int CH = ROWS * CPR / NTH;
    uint32_t off[CH];
    int w;  // wave index, wave-uniform
    __device__ Dma(long ld, int wave) : w(wave) {
      const int lane = threadIdx.x & 63;
#pragma unroll
      for (int i = 0; i < CH; ++i) {
        const int s = i * NTH + w * 64 + lane;
        const int r = s / CPR, c = (s % CPR) ^ f(r);
        off[i] = (uint32_t)(((long)r * ld + c * 8) * 2);
      }
    }
    __device__ void issue(const uint16_t* G, long ld, int rvalid, uint16_t* lds) const {
      if (rvalid >= ROWS) {
#pragma unroll
        for (int i = 0; i < CH; ++i)
          dma16((const char*)G + off[i], lds + (i * NTH + w * 64) * 8);
      } else {
        dma<ROWS, NTH>(G, ld, rvalid, lds);
      }
    }
  };
  // DMA rows [0, ROWS) of a global [token][*] block (row stride ld elements);
  // rows >= rvalid repeat row rvalid - 1 (their products are masked).
  template <int ROWS, int NTH>
  __device__ static void dma(const uint16_t* G, long ld, int rvalid, uint16_t* lds) {
    constexpr int CH = ROWS * CPR / NTH;
    static_assert(CH * NTH == ROWS * CPR, "uneven tile DMA");
    const int lane = threadIdx.x & 63, w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
#pragma unroll
    for (int i = 0; i < CH; ++i) {
      const int s = i * NTH + w * 64 + lane;
      const int r = s / CPR, phys = s % CPR;
      const int c = phys ^ f(r);
      const int gr = min(r, rvalid - 1);
      dma16(G + (long)gr * ld + c * 8, lds + (i * NTH + w * 64) * 8);
    }
  }
};

// DMA of a 64-key x (128 NS)-query tile of the stored dS (32-query blocks of
// [key][32], qstride elements apart) into NS consecutive Tile<128> layouts
// (row = key); per-thread chunk offsets computed once; a tile with fewer valid
// rows repeats row rvalid - 1.
template <int NTH, int NS>
struct DsDma {
  static constexpr int ROWS = 64, CH = NS * ROWS * 16 / NTH;
  static_assert(CH * NTH == NS * ROWS * 16, "uneven tile DMA");
  uint32_t off[CH];
  int w;  // wave index, wave-uniform
  // slot sl of the tile: sub-tile sl / 1024, row and chunk within it
  __device__ static long src(int sl, long qstride, int rvalid) {
    const int t = sl >> 10, r = (sl >> 4) & 63, c = (sl & 15) ^ Tile<128>::f(r);
    return (4 * t + (c >> 2)) * qstride + min(r, rvalid - 1) * 32 + (c & 3) * 8;
  }
  __device__ DsDma(long qstride, int wave) : w(wave) {
    const int lane = threadIdx.x & 63;
#pragma unroll
    for (int i = 0; i < CH; ++i) off[i] = (uint32_t)(src(i * NTH + w * 64 + lane, qstride, ROWS) * 2);
  }
  // G: key 0 of the tile in the first query block
  __device__ void issue(const uint16_t* G, long qstride, int rvalid, uint16_t* lds) const {
    if (rvalid >= ROWS) {
#pragma unroll
      for (int i = 0; i < CH; ++i) dma16((const char*)G + off[i], lds + (i * NTH + w * 64) * 8);
    } else {
      const int lane = threadIdx.x & 63;
#pragma unroll
      for (int i = 0; i < CH; ++i)
        dma16(G + src(i * NTH + w * 64 + lane, qstride, rvalid), lds + (i * NTH + w * 64) * 8);
    }
  }
};

// Tile<128>::col8 for a tile whose columns are stored with bits 2 and 3 of the
// column index swapped (the stored dS): the 4-column blocks the transposing
// reads fetch move as a whole, so each lane still receives column cb + lane % 32.
__device__ inline u32x4 col8_swapped(uint32_t base, int r0, int cb, int lane) {
  using T = Tile<128>;
  const int g = lane >> 4, j = lane & 15;
  const int col = cb + 16 * (g & 1) + 4 * (j & 3);
  const int pc = (col & ~12) | ((col & 4) << 1) | ((col & 8) >> 1);
  const int r = r0 + 4 * (g >> 1) + (j >> 2);
  const uint32_t inchunk = (pc & 7) << 1;
  return join(ds_read_tr(base + T::off(r, pc >> 3) + inchunk),
              ds_read_tr(base + T::off(r + 8, pc >> 3) + inchunk));
}

// 16-bit operand values of keys >= r set to zero: slot e of group G stands for
// key r0 + 4 G + e (e < 4) or r0 + 8 + 4 G + e - 4, two slots per register,
// the lower one in the low half.
__device__ inline u32x4 mask_keys(u32x4 x, int r0, int G, int r) {
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int k = r0 + (q < 2 ? 4 * G + 2 * q : 8 + 4 * G + 2 * (q - 2));
    x[q] &= (k < r ? 0xffffu : 0u) | (k + 1 < r ? 0xffff0000u : 0u);
  }
  return x;
}

// ------------------------------------------------------------------ forward

// two waves per SIMD (registers capped at 256): one wave's softmax overlaps the
// other's matrix products
// SPLIT: this block takes only split blockIdx.z % nsplit of the keys and
// leaves the unnormalised output with its running maximum and sum.
// F16: q, k and v are fp16 (scores and P V on fp16 operands), else bf16.
template <int D, int NW, bool SPLIT, bool F16>
__global__ __launch_bounds__(64 * NW, 2) void attn_fwd_mfma(AttnArgs a0) {
  const AttnArgs a = attn_seq_view<uint16_t>(a0);
  const int zsp = SPLIT ? blockIdx.z % a.nsplit : 0;
  using T = Tile<D>;
  constexpr int NTH = 64 * NW, BKV = 64, KS = D / 16, JB = D / 32, ST = 2;
  constexpr int TILE = BKV * D, STAGE = 2 * TILE;       // elements: K then V
  extern __shared__ __attribute__((aligned(16))) uint16_t smem[];
  const int h = blockIdx.y, lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int G = lane >> 5, c = lane & 31, H = a.ld;  // H: row stride
  const int q_lo = a.l + blockIdx.x * 32 * NW;       // first query of the block
  const int t = q_lo + 32 * w + c;                    // this lane's query
  const bool tvalid = t < a.r;
  const int kend_blk = min(a.r, q_lo + 32 * NW);      // keys the block needs
  const int kend_w = min(a.r, q_lo + 32 * w + 32);    // keys this wave needs
  const uint16_t* Q = (const uint16_t*)a.q;
  const uint16_t* Kc = (const uint16_t*)a.kc + h * D;
  const uint16_t* Vc = (const uint16_t*)a.vc + h * D;
  const uint32_t sbase = lds_addr(smem);

  u32x4 qf[KS];
#pragma unroll
  for (int kk = 0; kk < KS; ++kk) {
    qf[kk] = u32x4{0, 0, 0, 0};
    if (tvalid) qf[kk] = *(const u32x4*)(Q + (long)(t - a.l) * H + h * D + 16 * kk + 8 * G);
  }
  // Online softmax in the log2 domain.  m is the reference maximum of the
  // lane's scaled scores (log2 units); it moves only when a block's maximum
  // exceeds it by more than RESCALE_LOG2 (and then for the whole wave), so the
  // O and lsum rescale is skipped for most blocks.  The unnormalised weights
  // stay below 2^RESCALE_LOG2, and O / lsum and lse are unchanged in exact
  // arithmetic.
  constexpr float RESCALE_LOG2 = 8.f;
  const float sl2 = a.scale * LOG2E;
  float m = -INFINITY, lsum = 0.f;
  f32x16_t o[JB];
#pragma unroll
  for (int j = 0; j < JB; ++j) o[j] = zero16();

  int nkb = (kend_blk + BKV - 1) / BKV, kb0 = 0;
  if constexpr (SPLIT) {
    kb0 = zsp * (a.kv_chunk / BKV);
    nkb = min(nkb, kb0 + a.kv_chunk / BKV);
  }
  const typename T::template Dma<BKV, NTH> kvd(H, __builtin_amdgcn_readfirstlane(w));
  auto issue = [&](int stage, int kb) {
    uint16_t* st = smem + stage * STAGE;
    const int rv = min(BKV, kend_blk - kb * BKV);
    kvd.issue(Kc + (long)kb * BKV * H, H, rv, st);
    kvd.issue(Vc + (long)kb * BKV * H, H, rv, st + TILE);
  };
  if (kb0 < nkb) issue(kb0 % ST, kb0);
  for (int kb = kb0; kb < nkb; ++kb) {
    wait_vm<0>();
    __builtin_amdgcn_s_barrier();
    if (kb + 1 < nkb) issue((kb + 1) % ST, kb + 1);
    const int kbase = kb * BKV;
    if (kbase < kend_w) {
      const uint32_t Kt = sbase + (kb % ST) * STAGE * 2, Vt = Kt + TILE * 2;
      f32x16_t p[2];  // raw scores, -inf where masked
#pragma unroll
      for (int sb = 0; sb < 2; ++sb) {
        // computed also for a sub-block past the wave's last query (its rows
        // exist in the tile; every such score is masked below)
        f32x16_t s;
        {
          u32x4 kf[KS];
#pragma unroll
          for (int kk = 0; kk < KS; ++kk) kf[kk] = T::row8(Kt, 32 * sb + c, 2 * kk + G);
          lgkm_wait(kf[0]);
#pragma unroll
          for (int kk = 1; kk < KS; ++kk) lgkm_tie(kf[kk]);
          s = mfma_t<F16>(kf[0], qf[0], zero16());
#pragma unroll
          for (int kk = 1; kk < KS; ++kk) s = mfma_t<F16>(kf[kk], qf[kk], s);
        }
        // keys of a sub-block that ends at or before the wave's first query
        // need no mask (all are <= every query of the wave and < r)
        if (kbase + 32 * sb + 31 <= q_lo + 32 * w && kbase + 32 * sb + 32 <= a.r) {
          p[sb] = s;
        } else {
#pragma unroll
          for (int v = 0; v < 16; ++v) {
            const int key = kbase + 32 * sb + 8 * (v >> 2) + 4 * G + (v & 3);
            p[sb][v] = (key <= t && key < a.r) ? s[v] : -INFINITY;
          }
        }
      }
      float mx = -INFINITY;
#pragma unroll
      for (int v = 0; v < 16; ++v) mx = fmax_ieee(mx, fmax_ieee(p[0][v], p[1][v]));
      mx = pair_max(mx) * sl2;
      if (__builtin_amdgcn_ballot_w64(mx > m + RESCALE_LOG2) != 0) {  // wave-uniform
        const float mnew = fmaxf(m, mx);
        // no visible key yet for this query (both stay -inf): nothing to scale
        const float alpha = mnew == -INFINITY ? 1.f : exp2_fast(m - mnew);
        lsum *= alpha;
#pragma unroll
        for (int j = 0; j < JB; ++j)
#pragma unroll
          for (int v = 0; v < 16; ++v) o[j][v] *= alpha;
        m = mnew;
      }
      // weights 2^(s sl2 - m); a lane with no visible key so far has only
      // masked scores (-inf) and gets zeros
      const float moff = m == -INFINITY ? 0.f : -m;
      float rs = 0.f;
#pragma unroll
      for (int sb = 0; sb < 2; ++sb)
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const float e = exp2_fast(__builtin_fmaf(p[sb][v], sl2, moff));
          p[sb][v] = e;
          rs += e;
        }
      lsum += pair_sum(rs);
#pragma unroll
      for (int sb = 0; sb < 2; ++sb) {
        if (kbase + 32 * sb >= kend_w) break;
#pragma unroll
        for (int ks = 0; ks < 2; ++ks) {
          const u32x4 pb = acc_half<F16>(p[sb], ks);
          u32x4 vf[JB];
#pragma unroll
          for (int j = 0; j < JB; ++j) vf[j] = T::col8(Vt, 32 * sb + 16 * ks, 32 * j, lane);
          lgkm_wait(vf[0]);
#pragma unroll
          for (int j = 1; j < JB; ++j) lgkm_tie(vf[j]);
#pragma unroll
          for (int j = 0; j < JB; ++j) o[j] = mfma_t<F16>(vf[j], pb, o[j]);
        }
      }
    }
  }
  if (SPLIT && tvalid) {
    // partial of split zsp: rows like o (stride H = ld), one [rows][a.H] plane per split
    const int n = a.r - a.l, s = blockIdx.z / a.nsplit;
    float* P = a.ws + (long)zsp * n * a.bs * a.H + (long)s * a.H + (long)(t - a.l) * H + h * D;
#pragma unroll
    for (int j = 0; j < JB; ++j)
#pragma unroll
      for (int v = 0; v < 16; v += 4)
        *(float4*)(P + 32 * j + 8 * (v >> 2) + 4 * G) =
            make_float4(o[j][v], o[j][v + 1], o[j][v + 2], o[j][v + 3]);
    if (G == 0) {
      float* ml = a.ws + (long)a.nsplit * n * a.bs * a.H +
                  ((((long)zsp * a.bs + s) * a.heads + h) * n + (t - a.l)) * 2;
      ml[0] = m;
      ml[1] = lsum;
    }
  } else if (tvalid) {
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
__global__ __launch_bounds__(256) void attn_bwd_rowdot(AttnArgs a0) {
  const AttnArgs a = attn_seq_view<uint16_t>(a0);
  const int wave = (blockIdx.x * 256 + threadIdx.x) >> 6, lane = threadIdx.x & 63;
  const int n = a.r - a.l;
  if (wave >= n * a.heads) return;
  const int i = wave / a.heads, h = wave % a.heads;
  const uint16_t* dO = (const uint16_t*)a.dout + (long)i * a.ld + h * D;
  const uint16_t* O = (const uint16_t*)a.o + (long)i * a.ld + h * D;
  float s = 0.f;
  for (int j = lane; j < D; j += 64) s += to_f32(bf16{dO[j]}) * to_f32(bf16{O[j]});
  s = wave_sum(s);
  if (lane == 0) a.D[(long)h * a.Lmax + a.l + i] = s;
}

// ------------------------------------------------------------ dK / dV

// Wait until at most BASE + k * PER vector memory instructions are in flight,
// k (wave-uniform, 0..KMAX) picking the immediate.
template <int BASE, int PER, int KMAX>
__device__ inline void wait_vm_stores(int k) {
  if constexpr (KMAX == 0) {
    wait_vm<BASE>();
  } else {
    if (k >= KMAX) wait_vm<BASE + KMAX * PER>();
    else wait_vm_stores<BASE, PER, KMAX - 1>(k);
  }
}

// Adds a wave's 32-key block of fp32 results, acc[j][v] * mul for key
// s0 + 8 (v / 4) + 4 G + v % 4 and column 32 j + c, into the fp32 buffer buf
// (this head's first column, rows of H); keys >= r are left out.  When all 32
// keys exist, the loads of column block j + 1 are issued before block j is
// added and stored, so the read latency is paid about once.
template <int JB>
__device__ inline void add_rows_f32(float* buf, const f32x16_t (&acc)[JB], float mul, int s0,
                                    int r, int H, int G, int c) {
  if (s0 + 32 <= r) {
    float* b = buf + (long)s0 * H + c;
    auto rowoff = [&](int v) { return (long)(8 * (v >> 2) + 4 * G + (v & 3)) * H; };
    float cur[16];
#pragma unroll
    for (int v = 0; v < 16; ++v) cur[v] = b[rowoff(v)];
#pragma unroll
    for (int j = 0; j < JB; ++j) {
      float nx[16];
      if (j + 1 < JB) {
#pragma unroll
        for (int v = 0; v < 16; ++v) nx[v] = b[rowoff(v) + 32 * (j + 1)];
      }
#pragma unroll
      for (int v = 0; v < 16; ++v) b[rowoff(v) + 32 * j] = cur[v] + acc[j][v] * mul;
      if (j + 1 < JB) {
#pragma unroll
        for (int v = 0; v < 16; ++v) cur[v] = nx[v];
      }
    }
  } else {
#pragma unroll
    for (int j = 0; j < JB; ++j)
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int key = s0 + 8 * (v >> 2) + 4 * G + (v & 3);
        if (key < r) buf[(long)key * H + 32 * j + c] += acc[j][v] * mul;
      }
  }
}

// MODE 1: dV (S, P, dV += P^T dO); MODE 2: dK (S, dP, dS, dK += dS^T Q);
// MODE 3: MODE 2 that also stores dS for the streaming dQ kernel.  Each holds
// one accumulator set and fits two waves per SIMD; the MODE 1 + 2 pair
// recomputes S once more than a kernel forming both would.
//
// Stored dS (MODE 3): one plane of pd_ld / 32 query blocks per sequence and
// head; query block qb (queries l + 32 qb ...) holds r rows of 32 values, row
// = key, at qb * r * 32 + key * 32, so a wave's stores of one block fill whole
// contiguous lines and a reader's tile of consecutive keys is one contiguous
// piece.  Values fp16 (F16) or bf16, as the dK product rounds them, in operand
// order: query 16 h + 4 G + e + 8 u (e < 4) at column 16 h + 8 G + 4 u + e,
// i.e. bits 2 and 3 of the query index swapped, so each lane stores the 8
// values of a reduction half with one 16-byte store.  A (32-key, 32-query) block is written when its first key is below r
// and not after the block's last query (masked entries as zeros), the same
// condition under which the dQ kernel reads it.
// ST query tiles form the LDS ring: tile qb + ST - 1 is requested while tile
// qb is multiplied.
// F16: q and k are fp16 (scores on fp16 operands; the dK kernel's dS product
// on fp16 dS); v and the gradients stay bf16.
template <int D, int NW, int MODE, int ST, bool F16>
__global__ __launch_bounds__(64 * NW, 2) void attn_bwd_dkdv_mfma(AttnArgs a0) {
  static_assert(MODE >= 1 && MODE <= 3, "dV (1), dK (2), dK storing dS (3)");
  const AttnArgs a = attn_seq_view<uint16_t>(a0);
  using T = Tile<D>;
  constexpr bool DO_K = MODE >= 2, DO_V = MODE == 1, STORE = MODE == 3;
  constexpr int NTH = 64 * NW, BQ = 32, KS = D / 16, JB = D / 32;
  constexpr int TILE = BQ * D;                           // elements
  constexpr int STAGE = 2 * TILE + NW * 128;             // Q, dO, then per-wave [lse | D]
  constexpr int PER_ISSUE = 2 * (BQ * D / 8) / NTH + 1;  // DMA instructions per tile
  extern __shared__ __attribute__((aligned(16))) uint16_t smem[];
  const int h = blockIdx.y, lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int G = lane >> 5, c = lane & 31, H = a.ld;  // H: row stride
  const int k_lo = blockIdx.x * 32 * NW;     // first key of the block
  const int s_w = k_lo + 32 * w;             // first key of this wave
  const int s_me = s_w + c;                  // this lane's key (column of S)
  const uint16_t* Kc = (const uint16_t*)a.kc + h * D;
  const uint16_t* Vc = (const uint16_t*)a.vc + h * D;
  const uint16_t* Q = (const uint16_t*)a.q + h * D;
  const uint16_t* dO = (const uint16_t*)a.dout + h * D;
  const uint32_t sbase = lds_addr(smem);

  // K fragments of the wave's keys stay in registers; the dK kernel keeps
  // the block's V rows (needed for dP) in LDS, loaded once after the
  // query-tile ring, and reads them per query block
  constexpr bool V_LDS = DO_K;
  // this lane's row in query block 0 of the stored dS plane (MODE 3)
  const long prow = STORE ? ((long)blockIdx.z * a.heads + h) * a.r * a.pd_ld + (long)s_me * 32 : 0;
  u32x4 kf[KS];
#pragma unroll
  for (int kk = 0; kk < KS; ++kk) {
    kf[kk] = u32x4{0, 0, 0, 0};
    if (s_me < a.r) kf[kk] = *(const u32x4*)(Kc + (long)s_me * H + 16 * kk + 8 * G);
  }
  f32x16_t dk[JB], dv[JB];
#pragma unroll
  for (int j = 0; j < JB; ++j) dk[j] = dv[j] = zero16();
  const float sl2 = a.scale * LOG2E;
  const int n = a.r - a.l;
  // query rows i = t - l that can see a key of this block: t >= k_lo
  const int i_begin = max(0, k_lo - a.l) & ~(BQ - 1);
  const int nqb = (n - i_begin + BQ - 1) / BQ;
  const float* lse_h = a.lse + (long)h * a.Lmax;
  const float* D_h = a.D + (long)h * a.Lmax;
  const typename T::template Dma<BQ, NTH> qd(H, __builtin_amdgcn_readfirstlane(w));
  auto issue = [&](int stage, int qb) {
    uint16_t* st = smem + stage * STAGE;
    const int i0 = i_begin + qb * BQ, qv = min(BQ, n - i0);
    qd.issue(Q + (long)i0 * H, H, qv, st);
    qd.issue(dO + (long)i0 * H, H, qv, st + TILE);
    // per-wave copy of lse (lanes 0..31) and D (lanes 32..63) of the block's queries
    const int tq = min(a.l + i0 + (lane & 31), a.Lmax - 1);
    dma4((lane < 32 ? lse_h : D_h) + tq, st + 2 * TILE + w * 128);
  };
  const uint32_t Vl = sbase + ST * STAGE * 2;  // V rows of the block's keys (V_LDS)
  if (nqb > 0) {
    if constexpr (V_LDS)
      T::template dma<32 * NW, NTH>(Vc + (long)k_lo * H, H, min(32 * NW, a.r - k_lo),
                                    smem + ST * STAGE);
    for (int i = 0; i < ST - 1 && i < nqb; ++i) issue(i, i);
  }
  // MODE 3: a query block that takes part issues STORES store instructions
  // (one 16-byte store per reduction half), counted by vmcnt like the DMA and
  // completing in issue order with it; `recent` has bit j set when block
  // qb - 1 - j did, so the stores of the ST - 1 blocks issued after tile qb's
  // DMA may stay in flight while waiting for that tile.  Were more store
  // instructions emitted, the wait would only be stricter.
  constexpr int STORES = 2;
  unsigned recent = 0;
  bool stored = false;
  for (int qb = 0; qb < nqb; ++qb) {
    // tile qb has landed once at most the ST - 2 later tiles (and the stores
    // issued after tile qb's DMA) are in flight
    if (qb + ST - 1 <= nqb) {
      if constexpr (STORE) {
        recent = ((recent << 1) | (stored ? 1u : 0u)) & ((1u << (ST - 1)) - 1);
        wait_vm_stores<(ST - 2) * PER_ISSUE, STORES, ST - 1>(__builtin_popcount(recent));
      } else {
        wait_vm<(ST - 2) * PER_ISSUE>();
      }
    } else {
      if constexpr (STORE) recent = ((recent << 1) | (stored ? 1u : 0u)) & ((1u << (ST - 1)) - 1);
      wait_vm<0>();
    }
    __builtin_amdgcn_s_barrier();
    if (qb + ST - 1 < nqb) issue((qb + ST - 1) % ST, qb + ST - 1);
    const int i0 = i_begin + qb * BQ, qval = min(BQ, n - i0);
    // the wave's keys [s_w, s_w + 32) meet queries up to l + i0 + qval - 1
    stored = s_w <= a.l + i0 + qval - 1 && s_w < a.r;
    if (stored) {
      const uint32_t Qt = sbase + (qb % ST) * STAGE * 2, Ot = Qt + TILE * 2;
      // lse and D of this lane's 16 query rows: 4 consecutive rows per v / 4
      const uint32_t LD = Qt + 2 * TILE * 2 + w * 256;
      u32x4 lq[4], dq4[4];
#pragma unroll
      for (int b = 0; b < 4; ++b) lq[b] = ds_read128(LD + (8 * b + 4 * G) * 4);
      f32x16_t s = zero16(), dp = zero16();
      {
        u32x4 qa[KS];
#pragma unroll
        for (int kk = 0; kk < KS; ++kk) qa[kk] = T::row8(Qt, c, 2 * kk + G);
        lgkm_wait(qa[0]);
#pragma unroll
        for (int kk = 1; kk < KS; ++kk) lgkm_tie(qa[kk]);
#pragma unroll
        for (int b = 0; b < 4; ++b) lgkm_tie(lq[b]);
#pragma unroll
        for (int kk = 0; kk < KS; ++kk) s = mfma_t<F16>(qa[kk], kf[kk], s);
      }
      // s[v]: query row qi = 8 (v / 4) + 4 G + v % 4 of the block, key s_me.
      // P first, so the lse values are dead before the dP product.
      // A full query block whose first query follows every key of the wave
      // needs no mask.
      f32x16_t p, ds;
      if (qval == BQ && s_w + 31 <= a.l + i0) {
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const float lse_q = __uint_as_float(lq[v >> 2][v & 3]);
          p[v] = exp2_fast(__builtin_fmaf(s[v], sl2, -lse_q * LOG2E));
        }
      } else {
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const int qi = 8 * (v >> 2) + 4 * G + (v & 3);
          const bool ok = qi < qval && s_me <= a.l + i0 + qi;
          const float lse_q = __uint_as_float(lq[v >> 2][v & 3]);
          p[v] = ok ? exp2_fast(__builtin_fmaf(s[v], sl2, -lse_q * LOG2E)) : 0.f;
        }
      }
      if constexpr (DO_K) {
#pragma unroll
        for (int b = 0; b < 4; ++b) dq4[b] = ds_read128(LD + 128 + (8 * b + 4 * G) * 4);
      }
      if constexpr (DO_K) {
        // dP = dO V^T in two halves of the head width, V rows from LDS (rows
        // of keys >= r repeat the last key; their scores are masked)
#pragma unroll
        for (int hf = 0; hf < 2; ++hf) {
          u32x4 oa[KS / 2], vr[KS / 2];
#pragma unroll
          for (int kk = 0; kk < KS / 2; ++kk) {
            const int k2 = hf * (KS / 2) + kk;
            vr[kk] = T::row8(Vl, 32 * w + c, 2 * k2 + G);
            oa[kk] = T::row8(Ot, c, 2 * k2 + G);
          }
          lgkm_wait(vr[0]);
#pragma unroll
          for (int kk = 1; kk < KS / 2; ++kk) lgkm_tie(vr[kk]);
#pragma unroll
          for (int kk = 0; kk < KS / 2; ++kk) lgkm_tie(oa[kk]);
          if (hf == 0) {
#pragma unroll
            for (int b = 0; b < 4; ++b) lgkm_tie(dq4[b]);
          }
#pragma unroll
          for (int kk = 0; kk < KS / 2; ++kk) dp = mfma(oa[kk], vr[kk], dp);
        }
      }
      if constexpr (DO_K) {
#pragma unroll
        for (int v = 0; v < 16; ++v) ds[v] = p[v] * (dp[v] - __uint_as_float(dq4[v >> 2][v & 3]));
      }
#pragma unroll
      for (int ks = 0; ks < 2; ++ks) {
        if constexpr (DO_V) {
          const u32x4 pb = acc_half_bf16(p, ks);
          u32x4 ob[JB];
#pragma unroll
          for (int j = 0; j < JB; ++j) ob[j] = T::col8(Ot, 16 * ks, 32 * j, lane);
          lgkm_wait(ob[0]);
#pragma unroll
          for (int j = 1; j < JB; ++j) lgkm_tie(ob[j]);
#pragma unroll
          for (int j = 0; j < JB; ++j) dv[j] = mfma(pb, ob[j], dv[j]);
        }
        if constexpr (DO_K) {
          const u32x4 db = acc_half<F16>(ds, ks);
          if constexpr (STORE) {
            if (s_me < a.r) *(u32x4*)(a.dst + prow + (long)(i0 >> 5) * a.r * 32 + 16 * ks + 8 * G) = db;
          }
          u32x4 qb2[JB];
#pragma unroll
          for (int j = 0; j < JB; ++j) qb2[j] = T::col8(Qt, 16 * ks, 32 * j, lane);
          lgkm_wait(qb2[0]);
#pragma unroll
          for (int j = 1; j < JB; ++j) lgkm_tie(qb2[j]);
#pragma unroll
          for (int j = 0; j < JB; ++j) dk[j] = mfma_t<F16>(db, qb2[j], dk[j]);
        }
      }
    }
  }
  // dk[j][v], dv[j][v]: key s_w + 8 (v / 4) + 4 G + v % 4, column 32 j + c
  if constexpr (DO_K) add_rows_f32<JB>(a.dk + h * D, dk, a.scale, s_w, a.r, H, G, c);
  if constexpr (DO_V) add_rows_f32<JB>(a.dv + h * D, dv, 1.f, s_w, a.r, H, G, c);
}

// ------------------------------------------------------------------- dQ

// SPLIT: this block takes only split blockIdx.z % nsplit of the keys and
// leaves its unscaled fp32 dQ partial.
// F16: q and k are fp16 (scores and the dS K product on fp16 operands).
template <int D, int NW, bool SPLIT, bool F16>
__global__ __launch_bounds__(64 * NW, 2) void attn_bwd_dq_mfma(AttnArgs a0) {
  const AttnArgs a = attn_seq_view<uint16_t>(a0);
  const int zsp = SPLIT ? blockIdx.z % a.nsplit : 0;
  using T = Tile<D>;
  constexpr int NTH = 64 * NW, BKV = 64, KS = D / 16, JB = D / 32, ST = 2;
  constexpr int TILE = BKV * D, STAGE = 2 * TILE;  // K then V
  extern __shared__ __attribute__((aligned(16))) uint16_t smem[];
  const int h = blockIdx.y, lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int G = lane >> 5, c = lane & 31, H = a.ld;  // H: row stride
  const int q_lo = a.l + blockIdx.x * 32 * NW;
  const int t = q_lo + 32 * w + c;
  const bool tvalid = t < a.r;
  const int kend_blk = min(a.r, q_lo + 32 * NW);
  const int kend_w = min(a.r, q_lo + 32 * w + 32);
  const uint16_t* Kc = (const uint16_t*)a.kc + h * D;
  const uint16_t* Vc = (const uint16_t*)a.vc + h * D;
  const uint32_t sbase = lds_addr(smem);

  u32x4 qf[KS], of[KS];
#pragma unroll
  for (int kk = 0; kk < KS; ++kk) {
    qf[kk] = of[kk] = u32x4{0, 0, 0, 0};
    if (tvalid) {
      const long off = (long)(t - a.l) * H + h * D + 16 * kk + 8 * G;
      qf[kk] = *(const u32x4*)((const uint16_t*)a.q + off);
      of[kk] = *(const u32x4*)((const uint16_t*)a.dout + off);
    }
  }
  const float sl2 = a.scale * LOG2E;
  const float lse2 = tvalid ? a.lse[(long)h * a.Lmax + t] * LOG2E : 0.f;
  const float Dt = tvalid ? a.D[(long)h * a.Lmax + t] : 0.f;
  f32x16_t dq[JB];
#pragma unroll
  for (int j = 0; j < JB; ++j) dq[j] = zero16();

  int nkb = (kend_blk + BKV - 1) / BKV, kb0 = 0;
  if constexpr (SPLIT) {
    kb0 = zsp * (a.kv_chunk / BKV);
    nkb = min(nkb, kb0 + a.kv_chunk / BKV);
  }
  const typename T::template Dma<BKV, NTH> kvd(H, __builtin_amdgcn_readfirstlane(w));
  auto issue = [&](int stage, int kb) {
    uint16_t* st = smem + stage * STAGE;
    const int rv = min(BKV, kend_blk - kb * BKV);
    kvd.issue(Kc + (long)kb * BKV * H, H, rv, st);
    kvd.issue(Vc + (long)kb * BKV * H, H, rv, st + TILE);
  };
  if (kb0 < nkb) issue(kb0 % ST, kb0);
  for (int kb = kb0; kb < nkb; ++kb) {
    wait_vm<0>();
    __builtin_amdgcn_s_barrier();
    if (kb + 1 < nkb) issue((kb + 1) % ST, kb + 1);
    const int kbase = kb * BKV;
    const uint32_t Kt = sbase + (kb % ST) * STAGE * 2, Vt = Kt + TILE * 2;
#pragma unroll
    for (int sb = 0; sb < 2; ++sb) {
      if (kbase + 32 * sb >= kend_w) break;
      f32x16_t s = zero16(), dp = zero16();
      // K fragments, then V fragments in the same registers: the V reads go out
      // once the S products have been issued
      {
        u32x4 ka[KS];
#pragma unroll
        for (int kk = 0; kk < KS; ++kk) ka[kk] = T::row8(Kt, 32 * sb + c, 2 * kk + G);
        lgkm_wait(ka[0]);
#pragma unroll
        for (int kk = 1; kk < KS; ++kk) lgkm_tie(ka[kk]);
#pragma unroll
        for (int kk = 0; kk < KS; ++kk) s = mfma_t<F16>(ka[kk], qf[kk], s);
      }
      {
        u32x4 va[KS];
#pragma unroll
        for (int kk = 0; kk < KS; ++kk) va[kk] = T::row8(Vt, 32 * sb + c, 2 * kk + G);
        lgkm_wait(va[0]);
#pragma unroll
        for (int kk = 1; kk < KS; ++kk) lgkm_tie(va[kk]);
#pragma unroll
        for (int kk = 0; kk < KS; ++kk) dp = mfma(va[kk], of[kk], dp);
      }
      // keys of a sub-block that ends at or before the wave's first query,
      // with all 32 queries of the wave valid, need no mask
      f32x16_t ds;
      if (kbase + 32 * sb + 31 <= q_lo + 32 * w && q_lo + 32 * w + 32 <= a.r) {
#pragma unroll
        for (int v = 0; v < 16; ++v)
          ds[v] = exp2_fast(__builtin_fmaf(s[v], sl2, -lse2)) * (dp[v] - Dt);
      } else {
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const int key = kbase + 32 * sb + 8 * (v >> 2) + 4 * G + (v & 3);
          const bool ok = tvalid && key <= t;
          const float pv = ok ? exp2_fast(__builtin_fmaf(s[v], sl2, -lse2)) : 0.f;
          ds[v] = pv * (dp[v] - Dt);
        }
      }
#pragma unroll
      for (int ks = 0; ks < 2; ++ks) {
        const u32x4 db = acc_half<F16>(ds, ks);
        u32x4 kt[JB];
#pragma unroll
        for (int j = 0; j < JB; ++j) kt[j] = T::col8(Kt, 32 * sb + 16 * ks, 32 * j, lane);
        lgkm_wait(kt[0]);
#pragma unroll
        for (int j = 1; j < JB; ++j) lgkm_tie(kt[j]);
#pragma unroll
        for (int j = 0; j < JB; ++j) dq[j] = mfma_t<F16>(kt[j], db, dq[j]);
      }
    }
  }
  if (SPLIT && tvalid) {
    const int n = a.r - a.l, s = blockIdx.z / a.nsplit;
    float* P = a.ws + (long)zsp * n * a.bs * a.H + (long)s * a.H + (long)(t - a.l) * H + h * D;
#pragma unroll
    for (int j = 0; j < JB; ++j)
#pragma unroll
      for (int v = 0; v < 16; v += 4)
        *(float4*)(P + 32 * j + 8 * (v >> 2) + 4 * G) =
            make_float4(dq[j][v], dq[j][v + 1], dq[j][v + 2], dq[j][v + 3]);
  } else if (tvalid) {
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

// ------------------------------------------------- dQ from the stored dS

// dQ^T += K^T dS^T over the dS the dK kernel stored: per 64-key tile, the K
// rows and the stored dS rows of the block's 32-query blocks (128 or 256
// queries) move through an LDS ring; each wave owns QH blocks of 32 queries.
// Rows of keys >= r (repeats in the last tile) are zeroed in the dS operand.
template <int D, int NW, int QH, int ST, bool F16>
__global__ __launch_bounds__(64 * NW, 2) void attn_bwd_dq_stream(AttnArgs a0) {
  const AttnArgs a = attn_seq_view<uint16_t>(a0);
  using TK = Tile<D>;
  constexpr int NTH = 64 * NW, BKV = 64, JB = D / 32, QB = 32 * QH * NW;
  static_assert(QB == 128 || QB == 256, "128 or 256 query columns per block");
  constexpr int TILE_K = BKV * D, STAGE = TILE_K + BKV * QB, NS = QB / 128;
  static_assert((BKV * D / 8) % NTH == 0 && (BKV * QB / 8) % NTH == 0, "uneven tile DMA");
  constexpr int PER_ISSUE = (BKV * D / 8) / NTH + (BKV * QB / 8) / NTH;
  extern __shared__ __attribute__((aligned(16))) uint16_t smem[];
  const int h = blockIdx.y, lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int G = lane >> 5, c = lane & 31, H = a.ld;  // H: row stride
  const int i_lo = blockIdx.x * QB, q_lo = a.l + i_lo;
  const long qstride = (long)a.r * 32;  // elements between query blocks
  const uint16_t* Sp =
      a.dst + ((long)blockIdx.z * a.heads + h) * a.r * a.pd_ld + (long)(i_lo >> 5) * qstride;
  const uint16_t* Kc = (const uint16_t*)a.kc + h * D;
  const int kend_blk = min(a.r, q_lo + QB);
  const uint32_t sbase = lds_addr(smem);
  f32x16_t dq[QH][JB];
#pragma unroll
  for (int qh = 0; qh < QH; ++qh)
#pragma unroll
    for (int j = 0; j < JB; ++j) dq[qh][j] = zero16();
  const int nkb = (kend_blk + BKV - 1) / BKV;
  const int wq = __builtin_amdgcn_readfirstlane(w);
  const typename TK::template Dma<BKV, NTH> kd(H, wq);
  const DsDma<NTH, NS> sd(qstride, wq);
  auto issue = [&](int stage, int kb) {
    uint16_t* st = smem + stage * STAGE;
    const int rv = min(BKV, a.r - kb * BKV);
    kd.issue(Kc + (long)kb * BKV * H, H, rv, st);
    sd.issue(Sp + (long)kb * BKV * 32, qstride, rv, st + TILE_K);
  };
  for (int i = 0; i < ST - 1 && i < nkb; ++i) issue(i, i);
  for (int kb = 0; kb < nkb; ++kb) {
    if (kb + ST - 1 <= nkb) wait_vm<(ST - 2) * PER_ISSUE>();
    else wait_vm<0>();
    __builtin_amdgcn_s_barrier();
    if (kb + ST - 1 < nkb) issue((kb + ST - 1) % ST, kb + ST - 1);
    const uint32_t Kt = sbase + (kb % ST) * STAGE * 2, St = Kt + TILE_K * 2;
#pragma unroll
    for (int sb = 0; sb < 2; ++sb) {
      const int k0 = kb * BKV + 32 * sb;
      // a 32-key block takes part when it starts before r and at or before the
      // query block's last query: the blocks whose dS the dK kernel stored
      bool act[QH], any = false;
#pragma unroll
      for (int qh = 0; qh < QH; ++qh) {
        act[qh] = k0 < min(a.r, q_lo + 32 * (QH * w + qh) + 32);
        any = any || act[qh];
      }
      if (!any) continue;
#pragma unroll
      for (int ks = 0; ks < 2; ++ks) {
        u32x4 kt[JB], db[QH];
#pragma unroll
        for (int j = 0; j < JB; ++j) kt[j] = TK::col8(Kt, 32 * sb + 16 * ks, 32 * j, lane);
#pragma unroll
        for (int qh = 0; qh < QH; ++qh) {
          const int cb = 32 * (QH * w + qh);  // the block's 128-column sub-tile, column
          db[qh] = col8_swapped(St + (cb >> 7) * BKV * 128 * 2, 32 * sb + 16 * ks, cb & 127, lane);
        }
        lgkm_wait(kt[0]);
#pragma unroll
        for (int j = 1; j < JB; ++j) lgkm_tie(kt[j]);
#pragma unroll
        for (int qh = 0; qh < QH; ++qh) lgkm_tie(db[qh]);
        if (k0 + 32 > a.r) {
#pragma unroll
          for (int qh = 0; qh < QH; ++qh) db[qh] = mask_keys(db[qh], k0 + 16 * ks, G, a.r);
        }
#pragma unroll
        for (int qh = 0; qh < QH; ++qh)
          if (act[qh]) {
#pragma unroll
            for (int j = 0; j < JB; ++j) dq[qh][j] = mfma_t<F16>(kt[j], db[qh], dq[qh][j]);
          }
      }
    }
  }
  // dq[qh][j][v]: column 32 j + 8 (v / 4) + 4 G + v % 4 of query
  // q_lo + 32 (QH w + qh) + c
#pragma unroll
  for (int qh = 0; qh < QH; ++qh) {
    const int t = q_lo + 32 * (QH * w + qh) + c;
    if (t < a.r) {
      uint16_t* dQ = (uint16_t*)a.dq + (long)(t - a.l) * a.ld_dq + h * D;
#pragma unroll
      for (int j = 0; j < JB; ++j)
#pragma unroll
        for (int v = 0; v < 16; v += 4) {
          const int col = 32 * j + 8 * (v >> 2) + 4 * G;
          *(uint2*)(dQ + col) =
              make_uint2(pack_bf16x2(dq[qh][j][v] * a.scale, dq[qh][j][v + 1] * a.scale),
                         pack_bf16x2(dq[qh][j][v + 2] * a.scale, dq[qh][j][v + 3] * a.scale));
        }
    }
  }
}

// ------------------------------------------------------ split combines

// At most MAX_SPLIT key-range splits per launch (plan_split).
constexpr int MAX_SPLIT = 8;

// Forward: one wave per (row, head) merges the splits' partials in split
// order: M = max_z m_z, L = sum_z l_z 2^(m_z - M), O = sum_z O_z 2^(m_z - M) / L.
// Every load (each split's (m, l) pair and its D / 64 partial values per
// lane) is issued before the first use, so the wave waits for memory once.
template <int D>
__global__ __launch_bounds__(256) void attn_fwd_combine(AttnArgs a) {
  constexpr int PER = D / 64;  // consecutive columns per lane
  static_assert(PER == 1 || PER == 2, "head width 64 or 128");
  const int n = a.r - a.l, lane = threadIdx.x & 63;
  const long rows = (long)n * a.bs, wave = ((long)blockIdx.x * 256 + threadIdx.x) >> 6;
  if (wave >= rows * a.heads) return;
  const int i = (int)(wave / a.heads), h = (int)(wave % a.heads);  // row i = (t - l) bs + s
  const int tl = i / a.bs, s = i % a.bs;
  const long plane = rows * a.H;
  const float* part = a.ws + (long)i * a.H + h * D + PER * lane;
  const float* ml = a.ws + a.nsplit * plane + (((long)s * a.heads + h) * n + tl) * 2;
  const long ml_split = (long)a.bs * a.heads * n * 2;
  float m[MAX_SPLIT], l[MAX_SPLIT], v[MAX_SPLIT][PER];
#pragma unroll
  for (int z = 0; z < MAX_SPLIT; ++z) {
    if (z < a.nsplit) {
      const float2 t = *(const float2*)(ml + z * ml_split);
      m[z] = t.x, l[z] = t.y;
      if constexpr (PER == 2) {
        const float2 u = *(const float2*)(part + z * plane);
        v[z][0] = u.x, v[z][1] = u.y;
      } else {
        v[z][0] = part[z * plane];
      }
    }
  }
  float M = -INFINITY;
#pragma unroll
  for (int z = 0; z < MAX_SPLIT; ++z)
    if (z < a.nsplit) M = fmaxf(M, m[z]);
  // weight of split z (0 for a split that saw no key of this query)
  float L = 0.f, acc[PER] = {};
#pragma unroll
  for (int z = 0; z < MAX_SPLIT; ++z) {
    if (z < a.nsplit) {
      const float f = m[z] == -INFINITY ? 0.f : exp2_fast(m[z] - M);
      L += l[z] * f;
#pragma unroll
      for (int e = 0; e < PER; ++e) acc[e] += v[z][e] * f;
    }
  }
  const float inv = L > 0.f ? 1.f / L : 0.f;
  uint16_t* O = (uint16_t*)a.o + (long)i * a.H + h * D + PER * lane;
  if constexpr (PER == 2)
    *(uint32_t*)O = pack_bf16x2(acc[0] * inv, acc[1] * inv);
  else
    O[0] = f32_to_bf16_bits(acc[0] * inv);
  if (lane == 0) a.lse[((long)s * a.heads + h) * a.Lmax + a.l + tl] = (M + log2f(L)) * LN2;
}

// dQ: the splits' partials added in split order, scaled, stored as bf16 rows.
__global__ __launch_bounds__(256) void attn_dq_combine(AttnArgs a) {
  const int n = a.r - a.l;
  const long rows = (long)n * a.bs, a8 = a.H / 8;
  const long e = (long)blockIdx.x * 256 + threadIdx.x;
  if (e >= rows * a8) return;
  const long i = e / a8, col = (e - i * a8) * 8;
  const long plane = rows * a.H;
  float acc[8] = {};
  // every split's values in flight before the first add (at most MAX_SPLIT)
  float4 u[MAX_SPLIT], w[MAX_SPLIT];
#pragma unroll
  for (int z = 0; z < MAX_SPLIT; ++z) {
    if (z < a.nsplit) {
      const float4* p = (const float4*)(a.ws + z * plane + i * a.H + col);
      u[z] = p[0], w[z] = p[1];
    }
  }
#pragma unroll
  for (int z = 0; z < MAX_SPLIT; ++z) {
    if (z < a.nsplit) {
      acc[0] += u[z].x, acc[1] += u[z].y, acc[2] += u[z].z, acc[3] += u[z].w;
      acc[4] += w[z].x, acc[5] += w[z].y, acc[6] += w[z].z, acc[7] += w[z].w;
    }
  }
  uint16_t* dst = (uint16_t*)a.dq + (i / a.bs) * a.ld_dq + (i % a.bs) * a.dq_seq + col;
  uint4 o;
  o.x = pack_bf16x2(acc[0] * a.scale, acc[1] * a.scale);
  o.y = pack_bf16x2(acc[2] * a.scale, acc[3] * a.scale);
  o.z = pack_bf16x2(acc[4] * a.scale, acc[5] * a.scale);
  o.w = pack_bf16x2(acc[6] * a.scale, acc[7] * a.scale);
  *(uint4*)dst = o;
}

constexpr int NWF = 4;  // waves per block

// Key-range splits for a query-parallel launch that fills under half of the
// 256 CUs: enough splits for about one block per CU, at most MAX_SPLIT, each
// of at least one 64-key block, within the scratch (measured: a launch of 192
// blocks is faster unsplit -- the partials' traffic outweighs the extra
// blocks).  Sets a.nsplit and a.kv_chunk; 1 = no split.
void plan_split(AttnArgs& a, bool with_ml) {
  a.nsplit = 1;
  const int n = a.r - a.l;
  const long wgs = (long)cdiv(n, 32 * NWF) * a.heads * a.bs;
  if (!a.ws || wgs >= 128) return;
  int ns = (int)std::min<long>(MAX_SPLIT, cdiv(256, wgs));
  ns = std::min(ns, cdiv(a.r, 64));
  const long per = (long)n * a.bs * a.H + (with_ml ? 2L * a.bs * a.heads * n : 0);
  while (ns > 1 && ns * per > a.ws_elems) --ns;
  if (ns < 2) return;
  a.kv_chunk = cdiv(cdiv(a.r, ns), 64) * 64;
  a.nsplit = cdiv(a.r, a.kv_chunk);
}
template <typename K>
hipError_t set_lds(K* fn, size_t bytes) {
  if (bytes <= 64 * 1024) return hipSuccess;
  return hipFuncSetAttribute((const void*)fn, hipFuncAttributeMaxDynamicSharedMemorySize,
                             (int)bytes);
}

template <int D, bool F16>
hipError_t fwd_d(const AttnArgs& a, hipStream_t s) {
  const int n = a.r - a.l;
  constexpr size_t lds = 2 * 2 * 64 * D * 2;
  AttnArgs b = a;
  plan_split(b, true);
  if (a.need) {
    *a.need = b.nsplit > 1 ? (long)b.nsplit * ((long)n * a.bs * a.H + 2L * a.bs * a.heads * n) : 0;
    return hipSuccess;
  }
  if (b.nsplit == 1) {
    hipError_t e = set_lds(attn_fwd_mfma<D, NWF, false, F16>, lds);
    if (e != hipSuccess) return e;
    attn_fwd_mfma<D, NWF, false, F16>
        <<<dim3(cdiv(n, 32 * NWF), a.heads, a.bs), 64 * NWF, lds, s>>>(a);
    return hipGetLastError();
  }
  hipError_t e = set_lds(attn_fwd_mfma<D, NWF, true, F16>, lds);
  if (e != hipSuccess) return e;
  attn_fwd_mfma<D, NWF, true, F16>
      <<<dim3(cdiv(n, 32 * NWF), a.heads, a.bs * b.nsplit), 64 * NWF, lds, s>>>(b);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  attn_fwd_combine<D><<<cdiv((long)n * a.bs * a.heads, 4), 256, 0, s>>>(b);
  return hipGetLastError();
}

template <int D, bool F16>
hipError_t dq_d(const AttnArgs& a, hipStream_t s) {
  const int n = a.r - a.l;
  hipError_t e;
  constexpr size_t lds_q = 2 * 2 * 64 * D * 2;
  AttnArgs b = a;
  plan_split(b, false);
  if (a.need) {
    *a.need = b.nsplit > 1 ? (long)b.nsplit * n * a.bs * a.H : 0;
    return hipSuccess;
  }
  if (b.nsplit == 1) {
    e = set_lds(attn_bwd_dq_mfma<D, NWF, false, F16>, lds_q);
    if (e != hipSuccess) return e;
    attn_bwd_dq_mfma<D, NWF, false, F16>
        <<<dim3(cdiv(n, 32 * NWF), a.heads, a.bs), 64 * NWF, lds_q, s>>>(a);
    return hipGetLastError();
  }
  e = set_lds(attn_bwd_dq_mfma<D, NWF, true, F16>, lds_q);
  if (e != hipSuccess) return e;
  attn_bwd_dq_mfma<D, NWF, true, F16>
      <<<dim3(cdiv(n, 32 * NWF), a.heads, a.bs * b.nsplit), 64 * NWF, lds_q, s>>>(b);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  attn_dq_combine<<<cdiv((long)n * a.bs * (a.H / 8), 256), 256, 0, s>>>(b);
  return hipGetLastError();
}

// Backward with stored dS, after the dV kernel: over query chunks of at most
// cq rows (a multiple of 256) whose dS planes fit the scratch, the dK kernel
// (MODE 3) writes the planes that the streaming dQ kernel then reads (the
// rows' D = rowsum(dO * O) is already computed for the whole slice).
template <int D, bool F16>
hipError_t bwd_stored(const AttnArgs& a, hipStream_t s, long cq) {
  constexpr int NWK = D == 128 ? 8 : 4, STK = D == 128 ? 4 : 2;
  constexpr size_t lds_k = STK * (2 * 32 * D + NWK * 128) * 2 + 32 * NWK * D * 2;
  // dQ: 256 queries per block (8 waves) when that fills the CUs, else 128
  constexpr int STQ = 2;
  constexpr size_t lds_q4 = STQ * (64 * D + 64 * 128) * 2, lds_q8 = STQ * (64 * D + 64 * 256) * 2;
  const bool q8 = (long)cdiv(std::min<long>(a.r - a.l, cq), 256) * a.heads * a.bs >= 128;
  hipError_t e = set_lds(attn_bwd_dkdv_mfma<D, NWK, 3, STK, F16>, lds_k);
  if (e == hipSuccess)
    e = q8 ? set_lds(attn_bwd_dq_stream<D, 8, 1, STQ, F16>, lds_q8)
           : set_lds(attn_bwd_dq_stream<D, 4, 1, STQ, F16>, lds_q4);
  if (e != hipSuccess) return e;
  const int n = a.r - a.l;
  for (int c0 = 0; c0 < n; c0 += (int)cq) {
    const int c1 = (int)std::min<long>(n, c0 + cq);
    AttnArgs b = a;
    b.l = a.l + c0, b.r = a.l + c1;
    b.q = (const uint16_t*)a.q + (long)c0 * a.ld;
    b.o = (uint16_t*)a.o + (long)c0 * a.ld;
    b.dout = (const uint16_t*)a.dout + (long)c0 * a.ld;
    b.dq = (uint16_t*)a.dq + (long)c0 * a.ld_dq;
    b.pd_ld = (long)cdiv(c1 - c0, 256) * 256;  // whole dQ blocks of either width
    b.dst = a.pd;
    attn_bwd_dkdv_mfma<D, NWK, 3, STK, F16>
        <<<dim3(cdiv(b.r, 32 * NWK), a.heads, a.bs), 64 * NWK, lds_k, s>>>(b);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    if (q8)
      attn_bwd_dq_stream<D, 8, 1, STQ, F16>
          <<<dim3(cdiv(c1 - c0, 256), a.heads, a.bs), 512, lds_q8, s>>>(b);
    else
      attn_bwd_dq_stream<D, 4, 1, STQ, F16>
          <<<dim3(cdiv(c1 - c0, 128), a.heads, a.bs), 256, lds_q4, s>>>(b);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

template <int D, bool F16>
hipError_t bwd_d(const AttnArgs& a, hipStream_t s) {
  const int n = a.r - a.l;
  if (a.need) return dq_d<D, F16>(a, s);  // only the dQ kernel takes split scratch
  attn_bwd_rowdot<D><<<dim3(cdiv((long)n * a.heads, 4), 1, a.bs), 256, 0, s>>>(a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  // dV kernel: 4 waves, a 4-tile ring (69 KB, two blocks per CU).  dK kernel:
  // the block's V rows stay in LDS; with head width 128 it runs 8 waves (256
  // keys) over a 4-tile ring (137 KB, one block per CU), with 64 4 waves over
  // a 2-tile ring.
  constexpr int STA = 4;
  constexpr int NWK = D == 128 ? 8 : 4, STK = D == 128 ? 4 : 2;
  constexpr size_t lds_a = STA * (2 * 32 * D + NWF * 128) * 2;
  constexpr size_t lds_k = STK * (2 * 32 * D + NWK * 128) * 2 + 32 * NWK * D * 2;
  if ((long)cdiv(a.r, 32 * NWF) * a.heads * a.bs < 128) {
    // few key blocks (few heads, short prefix): two-wave dV blocks and
    // four-wave dK blocks over two-tile rings, so more blocks share the CUs
    constexpr size_t lds_v2 = 2 * (2 * 32 * D + 2 * 128) * 2;
    constexpr size_t lds_k4 = 2 * (2 * 32 * D + 4 * 128) * 2 + 32 * 4 * D * 2;
    e = set_lds(attn_bwd_dkdv_mfma<D, 2, 1, 2, F16>, lds_v2);
    if (e != hipSuccess) return e;
    attn_bwd_dkdv_mfma<D, 2, 1, 2, F16>
        <<<dim3(cdiv(a.r, 64), a.heads, a.bs), 128, lds_v2, s>>>(a);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    e = set_lds(attn_bwd_dkdv_mfma<D, 4, 2, 2, F16>, lds_k4);
    if (e != hipSuccess) return e;
    attn_bwd_dkdv_mfma<D, 4, 2, 2, F16>
        <<<dim3(cdiv(a.r, 128), a.heads, a.bs), 256, lds_k4, s>>>(a);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    return dq_d<D, F16>(a, s);
  }
  e = set_lds(attn_bwd_dkdv_mfma<D, NWF, 1, STA, F16>, lds_a);
  if (e != hipSuccess) return e;
  attn_bwd_dkdv_mfma<D, NWF, 1, STA, F16>
      <<<dim3(cdiv(a.r, 32 * NWF), a.heads, a.bs), 64 * NWF, lds_a, s>>>(a);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (a.pd) {
    // query rows per chunk whose dS planes (whole 256-query blocks) fit
    const long cq = a.pd_elems / ((long)a.bs * a.heads * a.r) / 256 * 256;
    if (cq >= 256) return bwd_stored<D, F16>(a, s, cq);
  }
  e = set_lds(attn_bwd_dkdv_mfma<D, NWK, 2, STK, F16>, lds_k);
  if (e != hipSuccess) return e;
  attn_bwd_dkdv_mfma<D, NWK, 2, STK, F16>
      <<<dim3(cdiv(a.r, 32 * NWK), a.heads, a.bs), 64 * NWK, lds_k, s>>>(a);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  return dq_d<D, F16>(a, s);
}

inline bool al16(const void* p) { return ((uintptr_t)p & 15) == 0; }

bool covered(const AttnArgs& a) {
  return (a.d == 64 || a.d == 128) && (a.H % 8) == 0 && (a.ld % 8) == 0 && al16(a.q) &&
         al16(a.kc) && al16(a.vc);
}

}  // namespace

hipError_t attn_fwd_mfma_bf16(const AttnArgs& a, hipStream_t s) {
  if (!covered(a) || !al16(a.o)) return hipErrorNotSupported;
  if (a.f16) return a.d == 128 ? fwd_d<128, true>(a, s) : fwd_d<64, true>(a, s);
  return a.d == 128 ? fwd_d<128, false>(a, s) : fwd_d<64, false>(a, s);
}

hipError_t attn_bwd_mfma_bf16(const AttnArgs& a, hipStream_t s) {
  if (!covered(a) || !al16(a.dout) || !al16(a.dq) || (a.ld_dq % 8) || (a.dq_seq % 8))
    return hipErrorNotSupported;
  if (a.f16) return a.d == 128 ? bwd_d<128, true>(a, s) : bwd_d<64, true>(a, s);
  return a.d == 128 ? bwd_d<128, false>(a, s) : bwd_d<64, false>(a, s);
}

}  // namespace tp
