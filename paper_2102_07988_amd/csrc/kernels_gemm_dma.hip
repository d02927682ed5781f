// bf16 GEMM for k-aligned shapes: global -> LDS by the CDNA4 LDS DMA
// (global_load_lds_dwordx4, 16 bytes per lane straight into LDS), a ring of
// STAGES k-tiles in flight, and matrix-core reads straight from LDS:
//  - k-contiguous operand tiles ([row][64 k], 128-byte rows) are read with
//    ds_read_b128 (8 consecutive k for one row);
//  - operands contiguous along m/n stay in their global orientation in LDS
//    ([64 k][R], k-major) and are read with two ds_read_b64_tr_b16, the
//    transposing LDS read: within each 16-lane group, lane j addresses 4
//    consecutive columns of row k0 + j/4, and lane i receives column i of the
//    group's 16 columns at the 4 rows -- exactly 4 reduction values of one
//    MFMA row/column.
// Both layouts permute 16-byte chunks by an XOR of the row so that the DMA
// writes stay contiguous and the fragment reads avoid bank conflicts; the
// DMA lane order implements the permutation (each lane picks the global chunk
// that belongs at its LDS slot).
//
// LDS reads are issued as inline assembly with explicit lgkmcnt waits, and the
// DMA completion with explicit vmcnt waits before each barrier, so the
// compiler's conservative wait-for-all-DMA before LDS reads does not serialise
// the pipeline.
#include <algorithm>
#include <atomic>
#include <type_traits>

#include "tp_common.hpp"
#include "tp_epilogue.hpp"
#include "tp_kernels.hpp"

namespace tp {

hipError_t gemm_splitk_reduce(const GemmArgs& a, hipStream_t s);

namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef _Float16 f16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

__device__ inline uint32_t lds_addr(const void* p) {
  return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void*)p;
}

// k-contiguous tile of BK k per row: row r, 16-byte chunk c (k = 8c..8c+7) at
// r*2BK + 16*(c ^ swz_kc(r)).  Any 16 consecutive rows read at one chunk land
// on 16 distinct 16-byte bank groups.
template <int BK>
__device__ inline int swz_kc(int r) {
  if constexpr (BK == 64) return (r ^ (r >> 3)) & 7;
  else return (r >> 2) & 3;
}
// m/n-contiguous tile of R columns: k-row k, 16-byte chunk c at k*2R + 16*(c ^ swz_mc<R>(k)).
// A transposing read takes 32 bytes from each of 4 consecutive k-rows.  Rows of
// 256 or 512 bytes all start on bank 0, so the row's chunk index is XORed with
// 4 (k mod 4) (64-byte steps); rows of 384 bytes (R = 192) already alternate
// between bank 0 and bank 32, so XOR 4 on rows 2 and 3 of each 4 suffices and
// keeps the 24 chunks of a row within range.
template <int R>
__device__ inline int swz_mc(int k) {
  static_assert(R % 128 == 0 || R == 192, "transposing-read swizzle needs R = 128 j or 192");
  if constexpr (R == 192) return ((k >> 1) & 1) << 2;
  else return (k & 3) << 2;
}

typedef float f32x4v __attribute__((ext_vector_type(4)));

__device__ inline void dma16(const uint16_t* g, uint16_t* lds_wave_base) {
  __builtin_amdgcn_global_load_lds((const __attribute__((address_space(1))) void*)g,
                                   (__attribute__((address_space(3))) void*)lds_wave_base, 16, 0,
                                   0);
}

// DMA of one R x BK operand tile into LDS.  KC: X(r, k) = X[r * ld + k];
// MC: X(r, k) = X[k * ld + r].  Rows/columns past rmax are clamped to valid
// memory (their products are never stored); k is always in range (the caller
// guarantees whole k-tiles).  The per-lane part of every chunk address is a
// byte offset from the k-origin of the tile, computed once per output tile;
// each k-tile only moves the wave-uniform origin (X + k for KC, X + k * ld for
// MC), so the loads take the scalar-base + 32-bit vector-offset form.  The
// caller guarantees the offsets fit in 32 bits.
template <int R, int BK, int NTH, bool KC>
struct DmaPlan {
  static constexpr int CH = R * BK / 8 / NTH;  // 16-byte chunks per thread
  uint32_t off[CH];
  __device__ DmaPlan(long ld, int r0, int rmax, int w, int lane) {
#pragma unroll
    for (int i = 0; i < CH; ++i) {
      const int s = i * NTH + w * 64 + lane;  // LDS slot of this lane
      if constexpr (KC) {
        constexpr int CPR = BK / 8;  // chunks per row
        const int row = s / CPR, phys = s % CPR;
        const int logical = phys ^ swz_kc<BK>(row);
        const int gr = min(r0 + row, rmax - 1);
        off[i] = (uint32_t)(((long)gr * ld + logical * 8) * 2);
      } else {
        constexpr int CPR = R / 8;  // chunks per k-row
        const int krow = s / CPR, phys = s % CPR;
        const int logical = phys ^ swz_mc<R>(krow);
        const int gc = min(r0 + logical * 8, rmax - 8);
        off[i] = (uint32_t)(((long)krow * ld + gc) * 2);
      }
    }
  }
  // origin: X + k0 (KC) or X + k0 * ld (MC), wave-uniform; w: wave index (uniform)
  __device__ void issue(const uint16_t* origin, uint16_t* lds, int w) const {
#pragma unroll
    for (int i = 0; i < CH; ++i)
      dma16((const uint16_t*)((const char*)origin + off[i]), lds + (i * NTH + w * 64) * 8);
  }
};

__device__ inline u32x4 ds_read128(uint32_t addr) {
  u32x4 v;
  asm volatile("ds_read_b128 %0, %1" : "=v"(v) : "v"(addr));
  return v;
}
__device__ inline u32x2 ds_read_tr(uint32_t addr) {
  u32x2 v;
  asm volatile("ds_read_b64_tr_b16 %0, %1" : "=v"(v) : "v"(addr));
  return v;
}

// Fragment (8 reduction values at k0 + 8 G) of operand row/column `rc` for lane
// (G = lane / 32).  KC tiles: one 16-byte read; MC tiles: two transposing reads.
template <int R, int BK, bool KC>
__device__ inline u32x4 frag_read(uint32_t tile, int rc_base, int k0, int lane) {
  if constexpr (KC) {
    const int row = rc_base + (lane & 31), c = (k0 >> 3) + (lane >> 5);
    return ds_read128(tile + row * (2 * BK) + ((c ^ swz_kc<BK>(row)) << 4));
  } else {
    const int g = lane >> 4, j = lane & 15;
    const int col = rc_base + 16 * (g & 1) + 4 * (j & 3);
    const int kr0 = k0 + 8 * (g >> 1) + (j >> 2);
    u32x2 lo, hi;
    {
      const int kr = kr0;
      lo = ds_read_tr(tile + kr * (2 * R) + (((col >> 3) ^ swz_mc<R>(kr)) << 4) + ((col & 7) << 1));
    }
    {
      const int kr = kr0 + 4;
      hi = ds_read_tr(tile + kr * (2 * R) + (((col >> 3) ^ swz_mc<R>(kr)) << 4) + ((col & 7) << 1));
    }
    u32x4 r;
    r.x = lo.x;
    r.y = lo.y;
    r.z = hi.x;
    r.w = hi.y;
    return r;
  }
}

template <int N>
__device__ inline void wait_vm() {
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

// Wait until at most `pending` k-tiles (LPT DMA instructions each) are in flight.
template <int LPT, int MAXP>
__device__ inline void wait_tiles(int pending) {
  if constexpr (MAXP >= 1) {
    if (pending >= MAXP) {
      wait_vm<LPT * MAXP>();
      return;
    }
    wait_tiles<LPT, MAXP - 1>(pending);
  } else {
    wait_vm<0>();
  }
}

// XCD-aware output-tile order for launches of many tiles.  Workgroups are
// dispatched round-robin over the 8 XCDs (workgroup g runs on XCD g % 8) and
// each CU holds one workgroup, so the j-th workgroup of an XCD belongs to
// "round" j / 32 of that XCD's 32 CUs.  The 32 workgroups of one XCD and
// round cover a 4 x 8 super-tile of output tiles, so each k-slice of its 4
// A-panels and 8 B-panels is fetched into that XCD's L2 once while they run
// side by side.  Super-tile s of round r is r * 8 + xcd.
constexpr int WALK_PER_XCD = 32;

struct TileWalk {
  static constexpr int SM = 4, SN = 8;
  int tm, tn, stm, stn;
  __device__ TileWalk(int tiles_m, int tiles_n)
      : tm(tiles_m), tn(tiles_n), stm((tiles_m + SM - 1) / SM), stn((tiles_n + SN - 1) / SN) {}
  // output tile of workgroup (xcd, slot) in round r; -1 if that slot is idle
  __device__ int tile(int r, int xcd, int slot) const {
    const int s = r * 8 + xcd;
    if (s >= stm * stn) return -1;
    const int im = (s / stn) * SM + slot / SN, in = (s % stn) * SN + slot % SN;
    if (im >= tm || in >= tn) return -1;
    return im * tn + in;
  }
};

// STAGES k-tiles of A and SB of B are buffered.  SB == STAGES: one ring of
// (A, B) stages.  SB == STAGES + 1 == 3 ("B leads"): separate rings, the B
// operand (the weights of a slice-shaped product, streamed from HBM) one
// k-tile further ahead than A (activations, L2-resident).
// F16: both operands are fp16 (the mixed-precision query/key/value product),
// otherwise bf16.
template <int BM, int BN, int BK, int WGM, int WGN, bool A_KC, bool B_KC, int EPI, bool SPLIT,
          int STAGES, int SB, bool F16>
__global__ __launch_bounds__(64 * WGM * WGN) void gemm_dma_kernel(GemmArgs a) {
  constexpr int NTH = 64 * WGM * WGN;
  constexpr int WM = BM / WGM, WN = BN / WGN, FM = WM / 32, FN = WN / 32;
  constexpr int TILE_A = BM * BK, TILE_B = BN * BK, STAGE = TILE_A + TILE_B;  // elements
  constexpr int LPT = BK * (BM + BN) / 8 / NTH;  // DMA instructions per thread per k-tile
  static_assert(FM >= 1 && FN >= 1, "wave tile below 32 x 32");
  static_assert(WM % 32 == 0 && WN % 32 == 0, "wave tile not a multiple of 32 x 32");
  static_assert((BK * BM / 8) % NTH == 0 && (BK * BN / 8) % NTH == 0, "uneven DMA split");
  static_assert(LPT * (STAGES - 2) <= 63, "vmcnt range");
  constexpr bool BLEAD = SB > STAGES;
  static_assert(SB == STAGES || (STAGES == 2 && SB == 3), "unsupported ring shape");
  static_assert((BK / 16) % 2 == 0, "fragment buffers alternate per k-step across k-tiles");
  constexpr int LPT_B = BK * BN / 8 / NTH;
  extern __shared__ __attribute__((aligned(16))) uint16_t smem[];

  const uint16_t* A = (const uint16_t*)a.A;
  const uint16_t* B = (const uint16_t*)a.B;
  const long lda = A_KC ? a.sam : a.sak;
  const long ldb = B_KC ? a.sbn : a.sbk;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm0 = (wave / WGN) * WM, wn0 = (wave % WGN) * WN;
  const int kbeg = SPLIT ? blockIdx.z * a.k_split : 0;
  const int kend = SPLIT ? min(a.K, kbeg + a.k_split) : a.K;
  const int nk = (kend - kbeg) / BK;
  const uint32_t sbase = lds_addr(smem);

  int m0 = blockIdx.y * BM, n0 = blockIdx.x * BN;
  if (!SPLIT && a.walk) {
    const TileWalk walk(cdiv(a.M, BM), cdiv(a.N, BN));
    const int j = blockIdx.x / 8;
    const int tile = walk.tile(j / WALK_PER_XCD, blockIdx.x % 8, j % WALK_PER_XCD);
    if (tile < 0) return;  // uniform per workgroup
    m0 = (tile / walk.tn) * BM;
    n0 = (tile % walk.tn) * BN;
  }

  const int wu = __builtin_amdgcn_readfirstlane(wave);
  const DmaPlan<BM, BK, NTH, A_KC> plan_a(lda, m0, a.M, wu, lane);
  const DmaPlan<BN, BK, NTH, B_KC> plan_b(ldb, n0, a.N, wu, lane);
  auto issue_a = [&](int kt) {
    uint16_t* st = smem + (kt % STAGES) * (BLEAD ? TILE_A : STAGE);
    const long k = kbeg + kt * BK;
    plan_a.issue(A + (A_KC ? k : k * lda), st, wu);
  };
  auto issue_b = [&](int kt) {
    uint16_t* st = BLEAD ? smem + STAGES * TILE_A + (kt % SB) * TILE_B
                         : smem + (kt % STAGES) * STAGE + TILE_A;
    const long k = kbeg + kt * BK;
    plan_b.issue(B + (B_KC ? k : k * ldb), st, wu);
  };
  // DMA of the k-tiles that iteration kt brings in (their stages were last read
  // in iteration kt - 1, before its closing barrier)
  auto issue_next = [&](int kt) {
    if constexpr (BLEAD) {
      if (kt + 1 < nk) issue_a(kt + 1);
      if (kt + 2 < nk) issue_b(kt + 2);
    } else if (kt + STAGES - 1 < nk) {
      issue_a(kt + STAGES - 1);
      issue_b(kt + STAGES - 1);
    }
  };

  f32x16_t acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;

  if constexpr (BLEAD) {
    // issue order B0, A0, B1, then per iteration A(kt+1), B(kt+2): when
    // iteration kt starts, only B(kt+1) was issued after A(kt)
    issue_b(0);
    issue_a(0);
    if (nk > 1) issue_b(1);
  } else {
#pragma unroll
    for (int s = 0; s < STAGES - 1; ++s)
      if (s < nk) {
        issue_a(s);
        issue_b(s);
      }
  }

  // k-tile j has landed for every wave once at most the DMAs issued after it
  // are in flight (they complete in issue order) and the workgroup has met at
  // a barrier
  auto wait_tile = [&](int j) {
    if constexpr (BLEAD) {
      if (j + 1 < nk) wait_vm<LPT_B>();
      else wait_vm<0>();
    } else {
      wait_tiles<LPT, STAGES - 2>(min(STAGES - 2, nk - 1 - j));
    }
    __builtin_amdgcn_s_barrier();
  };
  auto tile_a = [&](int j) { return sbase + (j % STAGES) * (BLEAD ? TILE_A : STAGE) * 2; };
  auto tile_b = [&](int j) {
    return BLEAD ? sbase + (STAGES * TILE_A + (j % SB) * TILE_B) * 2 : tile_a(j) + TILE_A * 2;
  };
  u32x4 fa[2][FM], fb[2][FN];
  auto read_frags = [&](int buf, int j, int k0) {
    const uint32_t ta = tile_a(j), tb = tile_b(j);
#pragma unroll
    for (int i = 0; i < FM; ++i) fa[buf][i] = frag_read<BM, BK, A_KC>(ta, wm0 + 32 * i, k0, lane);
#pragma unroll
    for (int jj = 0; jj < FN; ++jj) fb[buf][jj] = frag_read<BN, BK, B_KC>(tb, wn0 + 32 * jj, k0, lane);
  };
  // wait for every LDS read issued so far, every fragment register of `buf` tied to the wait
  auto frags_ready = [&](int buf) {
    asm volatile("s_waitcnt lgkmcnt(0)" : "+v"(fa[buf][0]));
#pragma unroll
    for (int i = 1; i < FM; ++i) asm volatile("" : "+v"(fa[buf][i]));
#pragma unroll
    for (int jj = 0; jj < FN; ++jj) asm volatile("" : "+v"(fb[buf][jj]));
  };

  // One k-step runs the FM x FN matrix-core products of fragment buffer `cur`
  // and, one per product from the first product on, the fragment reads of the
  // next step into the other buffer, so the reads complete under the products
  // and the step ends with a single LDS wait.  Scheduling barriers pin that
  // order: the reads are inline assembly, which the scheduler would otherwise
  // let the products pass, leaving a wait in front of most of them.
  //
  // The k-tile boundary is software-pipelined: half of the last step's
  // products go out, then the wait and barrier for tile kt+1, then its first
  // fragment reads interleaved with the other half.  The DMA of the tile after
  // goes out right after the barrier for split (slice-shaped, weight-streaming)
  // products, after the last step's products for the others; either way into
  // the stage of tile kt, which every wave finished reading before the barrier.
  // The final k-tile is peeled (no next tile to wait for or read), so no
  // branch inside the loop holds products.
  constexpr int NR = FM + FN, NM = FM * FN;
  auto mfma_at = [&](int buf, int t) {
    const int i = t / FN, j = t % FN;
    if constexpr (F16)
      acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_f16(
          __builtin_bit_cast(f16x8_t, fa[buf][i]), __builtin_bit_cast(f16x8_t, fb[buf][j]),
          acc[i][j], 0, 0, 0);
    else
      acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
          __builtin_bit_cast(bf16x8_t, fa[buf][i]), __builtin_bit_cast(bf16x8_t, fb[buf][j]),
          acc[i][j], 0, 0, 0);
  };
  auto read_at = [&](int buf, uint32_t ta, uint32_t tb, int k0, int r) {
    if (r < FM) fa[buf][r] = frag_read<BM, BK, A_KC>(ta, wm0 + 32 * r, k0, lane);
    else fb[buf][r - FM] = frag_read<BN, BK, B_KC>(tb, wn0 + 32 * (r - FM), k0, lane);
  };
  // products [T0, NM) of `cur`; with RD, the reads of `nxt` (tile j, k-offset
  // k0) one per product from T0 on, any left over after the last product
  auto interleave = [&](auto t0c, auto rdc, int cur, int nxt, int j, int k0) {
    constexpr int T0 = decltype(t0c)::value;
    constexpr bool RD = decltype(rdc)::value;
    const uint32_t ta = tile_a(j), tb = tile_b(j);
#pragma unroll
    for (int t = T0; t < NM; ++t) {
      if constexpr (RD) {
        if (t - T0 < NR) read_at(nxt, ta, tb, k0, t - T0);
      }
      mfma_at(cur, t);
      __builtin_amdgcn_sched_barrier(0);
    }
    if constexpr (RD) {
#pragma unroll
      for (int r = NM - T0; r < NR; ++r) read_at(nxt, ta, tb, k0, r);
    }
  };
  using First = std::integral_constant<int, 0>;
  using Half = std::integral_constant<int, NM / 2>;
  using Yes = std::integral_constant<bool, true>;
  using No = std::integral_constant<bool, false>;
  auto ktile = [&](int kt, auto finalc) {
    constexpr bool FINAL = decltype(finalc)::value;
#pragma unroll
    for (int ks = 0; ks < BK / 16; ++ks) {
      const int cur = ks & 1, nxt = cur ^ 1;
      const bool last = ks + 1 == BK / 16;
      if (!last) {
        interleave(First{}, Yes{}, cur, nxt, kt, 16 * (ks + 1));
      } else if constexpr (!FINAL) {
#pragma unroll
        for (int t = 0; t < NM / 2; ++t) mfma_at(cur, t);
        __builtin_amdgcn_sched_barrier(0);
        wait_tile(kt + 1);
        if (SPLIT) issue_next(kt + 1);
        interleave(Half{}, Yes{}, cur, nxt, kt + 1, 0);
      } else {
        interleave(First{}, No{}, cur, nxt, 0, 0);
      }
      __builtin_amdgcn_sched_barrier(0);
      if (!FINAL && !SPLIT && last) issue_next(kt + 1);
      if (!(FINAL && last)) frags_ready(nxt);
    }
  };

  wait_tile(0);
  issue_next(0);
  read_frags(0, 0, 0);
  frags_ready(0);
  if (nk > 0) {
    for (int kt = 0; kt + 1 < nk; ++kt) ktile(kt, No{});
    ktile(nk - 1, Yes{});
  }
  // every outstanding DMA has been waited for: the last iteration waited for 0

  if constexpr (SPLIT || EPI == EPI_ACC_F32) {
    // fp32 outputs: each 32 x 32 sub-tile goes through a wave-private LDS patch
    // (in the ring stage no wave reads in the last iteration, or, with separate
    // rings, at the LDS base once every wave has left the loop)
    static_assert(WGM * WGN * 32 * 36 * 4 <= (BLEAD ? STAGES * TILE_A : STAGE) * 2,
                  "epilogue patch exceeds its region");
    if constexpr (BLEAD) __builtin_amdgcn_s_barrier();
    float* patch = (float*)(smem + (BLEAD ? 0 : (nk % STAGES) * STAGE)) + wave * (32 * 36);
    float* out = SPLIT ? a.ws + (long)blockIdx.z * a.M * a.N : (float*)a.C;
    const long ldo = SPLIT ? a.N : a.ldc;
    // sub-tile rows leave as whole 128-byte lines: in step q (0..3) lane l
    // takes row 8q + l/8, 16-byte chunk l%8
    const int er = lane >> 3, ec = (lane & 7) * 4;
    const bool full = m0 + wm0 + WM <= a.M && n0 + wn0 + WN <= a.N;
    auto dst_of = [&](int t, int q) {
      return out + (long)(m0 + wm0 + (t / FN) * 32 + 8 * q + er) * ldo + n0 + wn0 + (t % FN) * 32 +
             ec;
    };
    // fp32 +=: the destination values of the next P sub-tiles are in flight
    // while one is combined (a plain store with a.overwrite)
    constexpr int T = FM * FN, P = T < 4 ? T : 4;
    const bool add = !SPLIT && !a.overwrite;
    float4 pre[P][4];
    if (add && full) {
#pragma unroll
      for (int t = 0; t < P; ++t)
#pragma unroll
        for (int q = 0; q < 4; ++q) pre[t][q] = *(const float4*)dst_of(t, q);
    }
#pragma unroll
    for (int t = 0; t < T; ++t) {
      const int i = t / FN, j = t % FN;
#pragma unroll
      for (int v = 0; v < 16; ++v)
        patch[(8 * (v >> 2) + 4 * (lane >> 5) + (v & 3)) * 36 + (lane & 31)] = acc[i][j][v];
      float4 x[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) x[q] = *(const float4*)(patch + (8 * q + er) * 36 + ec);
      if (full) {
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          if (add) {
            const float4 o = pre[t % P][q];
            x[q].x += o.x, x[q].y += o.y, x[q].z += o.z, x[q].w += o.w;
          }
          if constexpr (SPLIT) {
            *(float4*)dst_of(t, q) = x[q];
          } else {
            // the fp32 weight gradient is not read again by this sequence's
            // kernels: a non-temporal store keeps it from displacing their
            // operands in the caches
            const f32x4v v = {x[q].x, x[q].y, x[q].z, x[q].w};
            __builtin_nontemporal_store(v, (f32x4v*)dst_of(t, q));
          }
        }
        if (add && t + P < T) {
#pragma unroll
          for (int q = 0; q < 4; ++q) pre[t % P][q] = *(const float4*)dst_of(t + P, q);
        }
      } else {
        const int n = n0 + wn0 + j * 32 + ec;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int m = m0 + wm0 + i * 32 + 8 * q + er;
          if (m < a.M) {
            float* dst = out + (long)m * ldo + n;
            const float xs[4] = {x[q].x, x[q].y, x[q].z, x[q].w};
#pragma unroll
            for (int e = 0; e < 4; ++e)
              if (n + e < a.N) dst[e] = add ? dst[e] + xs[e] : xs[e];
          }
        }
      }
    }
  } else {
    // bf16 outputs: each 32 x 32 sub-tile goes through the LDS patch and leaves
    // as 8-column row segments (in step q of 2, lane l takes row 16q + l/4,
    // columns 8 (l%4) .. +7), one 16-byte access per operand; N % 8 == 0, so a
    // segment is either inside the output or past its edge
    if constexpr (BLEAD) __builtin_amdgcn_s_barrier();
    float* patch = (float*)(smem + (BLEAD ? 0 : (nk % STAGES) * STAGE)) + wave * (32 * 36);
    const int er = lane >> 2, ec = (lane & 3) * 8;
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int j = 0; j < FN; ++j) {
#pragma unroll
        for (int v = 0; v < 16; ++v)
          patch[(8 * (v >> 2) + 4 * (lane >> 5) + (v & 3)) * 36 + (lane & 31)] = acc[i][j][v];
#pragma unroll
        for (int q = 0; q < 2; ++q) {
          const int r = 16 * q + er;
          const float4 u = *(const float4*)(patch + r * 36 + ec);
          const float4 w = *(const float4*)(patch + r * 36 + ec + 4);
          float x[8] = {u.x, u.y, u.z, u.w, w.x, w.y, w.z, w.w};
          const int m = m0 + wm0 + 32 * i + r, n = n0 + wn0 + 32 * j + ec;
          if (m < a.M && n < a.N) epi8<EPI>(a, m, n, x);
        }
      }
  }
}

template <int BM, int BN, int BK, int WGM, int WGN, bool A_KC, bool B_KC, int STAGES, int SB,
          bool SPLIT, bool F16>
hipError_t launch_dma(const GemmArgs& a, hipStream_t s) {
  constexpr int NTH = 64 * WGM * WGN;
  constexpr size_t lds = ((size_t)STAGES * BM + (size_t)SB * BN) * BK * 2;
  dim3 grid(cdiv(a.N, BN), cdiv(a.M, BM), SPLIT ? a.splits : 1);
  if (!SPLIT && a.walk) {
    // rounds of 8 super-tiles (one per XCD), 256 workgroups per round
    const int rounds =
        (cdiv(cdiv(a.M, BM), TileWalk::SM) * cdiv(cdiv(a.N, BN), TileWalk::SN) + 7) / 8;
    grid = dim3(rounds * 8 * WALK_PER_XCD, 1, 1);
  }
  // the dynamic-LDS limit is raised once per kernel and device (bit d of a
  // per-kernel mask; devices past 31 set it on every launch)
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) dev = 32;
#define TP_LAUNCH(E)                                                                         \
  do {                                                                                       \
    auto* fn = gemm_dma_kernel<BM, BN, BK, WGM, WGN, A_KC, B_KC, E, SPLIT, STAGES, SB, F16>;\
    static std::atomic<uint32_t> attr_set{0};                                                \
    const uint32_t bit = dev < 32 ? 1u << dev : 0u;                                          \
    if (!bit || !(attr_set.load(std::memory_order_acquire) & bit)) {                         \
      hipError_t e = hipFuncSetAttribute((const void*)fn,                                    \
                                         hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds); \
      if (e != hipSuccess) return e;                                                         \
      attr_set.fetch_or(bit, std::memory_order_release);                                     \
    }                                                                                        \
    fn<<<grid, NTH, lds, s>>>(a);                                                            \
  } while (0)
  if constexpr (SPLIT) {
    TP_LAUNCH(EPI_STORE);
  } else if constexpr (F16) {
    // fp16 operands: only the query/key/value product
    if (a.epi != EPI_QKV) return hipErrorNotSupported;
    TP_LAUNCH(EPI_QKV);
  } else if constexpr (!A_KC && !B_KC) {
    // m/n-contiguous operands on both sides: the weight-gradient products
    switch (a.epi) {
      case EPI_STORE: TP_LAUNCH(EPI_STORE); break;
      case EPI_ACC_F32: TP_LAUNCH(EPI_ACC_F32); break;
      default: return hipErrorNotSupported;
    }
  } else {
    switch (a.epi) {
      case EPI_STORE: TP_LAUNCH(EPI_STORE); break;
      case EPI_QKV: TP_LAUNCH(EPI_QKV); break;
      case EPI_RESID: TP_LAUNCH(EPI_RESID); break;
      case EPI_GELU: TP_LAUNCH(EPI_GELU); break;
      case EPI_DGELU: TP_LAUNCH(EPI_DGELU); break;
      case EPI_ACC_F32: TP_LAUNCH(EPI_ACC_F32); break;
      default: return hipErrorInvalidValue;
    }
  }
#undef TP_LAUNCH
  return hipGetLastError();
}


// One DMA GEMM launch.  Every configuration holds one workgroup per CU (its
// LDS ring takes most of the 160 KB), so when the tile count is low the
// reduction is split (whole k-tiles, the last split may be shorter).
// force_splits > 0 takes that many splits (at most; as k-tiles allow),
// otherwise the split count comes from the cost model below (<= 8 splits of
// >= 8 k-tiles).  With splits2 > 0 and 0 < cols1 < the column-tile count, the
// product runs as two split launches: column tiles [0, cols1) with
// force_splits splits, the rest with splits2 (when the partials fit), and one
// reduction over both.
template <int BM, int BN, int BK, int WGM, int WGN, bool A_KC, bool B_KC, int STAGES,
          int SB, bool F16>
hipError_t run_dma(GemmArgs a, hipStream_t s, int force_splits = 0, int splits2 = 0,
                   int cols1 = 0) {
  constexpr int CUS = 256;
  if (a.K % BK) return hipErrorNotSupported;
  const long tiles = (long)cdiv(a.M, BM) * cdiv(a.N, BN);
  const int nkt = a.K / BK;
  if (force_splits > 0 && splits2 > 0 && cols1 > 0 && (long)cols1 * BN < a.N && a.ws) {
    const int n1 = cols1 * BN, n2 = a.N - n1;
    const int ks1 = cdiv(nkt, std::min(force_splits, nkt)) * BK;
    const int ks2 = cdiv(nkt, std::min(splits2, nkt)) * BK;
    const int s1 = cdiv(a.K, ks1), s2 = cdiv(a.K, ks2);
    const long p1 = (long)s1 * a.M * n1, need = p1 + (long)s2 * a.M * n2;
    if (need <= a.ws_elems) {
      if (a.need) {
        *a.need = need;
        return hipSuccess;
      }
      GemmArgs g = a;
      g.N = n1, g.k_split = ks1, g.splits = s1;
      hipError_t e = launch_dma<BM, BN, BK, WGM, WGN, A_KC, B_KC, STAGES, SB, true, F16>(g, s);
      if (e != hipSuccess) return e;
      g = a;
      g.N = n2, g.k_split = ks2, g.splits = s2;
      g.B = (const uint16_t*)a.B + (long)n1 * a.sbn;
      g.ws = a.ws + p1, g.ws_elems = a.ws_elems - p1;
      e = launch_dma<BM, BN, BK, WGM, WGN, A_KC, B_KC, STAGES, SB, true, F16>(g, s);
      if (e != hipSuccess) return e;
      GemmArgs r = a;
      r.splits = s1, r.splits2 = s2, r.split_cols = n1;
      return gemm_splitk_reduce(r, s);
    }
  }
  int splits = 1;
  if (force_splits > 0) {
    splits = a.ws && (long)force_splits * a.M * a.N <= a.ws_elems ? std::min(force_splits, nkt) : 1;
  } else if (a.ws && tiles < 2 * CUS) {
    // time ~ rounds(s) / s of the unsplit main loop, plus the partial-sum
    // traffic (s fp32 products written and read back), which relative to the
    // weight stream of one round is about 2.2 M / K per split
    const double lam = 2.2 * (double)a.M / (double)a.K;
    double best = 1e30;
    for (int sp = 1; sp <= 8; ++sp) {
      if (sp > 1 && (nkt / sp < 8 || (long)sp * a.M * a.N > a.ws_elems)) break;
      const long wgs = tiles * sp;
      const double cost = (double)cdiv(wgs, CUS) / sp + (sp > 1 ? lam * sp : 0.0);
      if (cost < best - 1e-9) {
        best = cost;
        splits = sp;
      }
    }
  }
  if (a.need) {
    *a.need = splits > 1 ? (long)cdiv(a.K, cdiv(nkt, splits) * BK) * a.M * a.N : 0;
    return hipSuccess;
  }
  if (splits > 1) {
    a.k_split = cdiv(nkt, splits) * BK;
    a.splits = cdiv(a.K, a.k_split);
    hipError_t e = launch_dma<BM, BN, BK, WGM, WGN, A_KC, B_KC, STAGES, SB, true, F16>(a, s);
    if (e != hipSuccess) return e;
    return gemm_splitk_reduce(a, s);
  }
  // many tiles: XCD-aware super-tile order
  if (tiles >= 2 * CUS) a.walk = 1;
  return launch_dma<BM, BN, BK, WGM, WGN, A_KC, B_KC, STAGES, SB, false, F16>(a, s);
}

template <bool A_KC, bool B_KC, bool F16 = false>
hipError_t run_cfg_id(int cfg, const GemmArgs& a, hipStream_t s, int splits = 0, int splits2 = 0,
                      int cols1 = 0) {
  switch (cfg) {
    case 0: return run_dma<128, 128, 64, 2, 2, A_KC, B_KC, 4, 4, F16>(a, s, splits);
    case 1: return run_dma<256, 128, 64, 4, 2, A_KC, B_KC, 3, 3, F16>(a, s, splits);
    case 2: return run_dma<256, 256, 64, 2, 4, A_KC, B_KC, 2, 2, F16>(a, s, splits);
    case 3:
      return run_dma<256, 256, 64, 2, 4, A_KC, B_KC, 2, 3, F16>(a, s, splits, splits2, cols1);
    case 4:
      // 256 x 192: 256 tiles for a 256-row product of width 49152, 64 for 12288
      if constexpr (A_KC)
        return run_dma<256, 192, 64, 4, 2, A_KC, B_KC, 2, 3, F16>(a, s, splits, splits2, cols1);
      else return hipErrorNotSupported;
    default: return hipErrorNotSupported;
  }
}

// Tile shape and split count for a product whose A operand is k-contiguous
// (slice activations or output gradients times a weight matrix): the
// candidate (tiles, splits) with the smallest modelled time.  The model was
// fitted (log least squares, rms error 10 %) to a sweep of every candidate on
// the stage's products for hidden sizes 2048-12288, operation-partitioning
// shards and 128-512 rows:
//   t = max(rounds * (0.74 + kt * c_kt), rows_tiles * N * K * 2 B * 0.177 us/MB)
//       + (splits > 1 ? 5.7 + splits * M * N * 8 B / 5.8 MB/us : 0)
// with rounds = workgroups / 256 rounded up, kt = k-tiles per split and c_kt
// = 0.59 / 0.91 / 1.21 / 1.44 us for 128x128 / 256x128 / 256x192 / 256x256 tiles: a round of
// workgroups, not below the weight stream from HBM, plus the partial sums.
struct TileChoice {
  int cfg, splits;
  int splits2 = 0, cols1 = 0;  // two column groups (see run_dma), 0: one launch
};
TileChoice choose_tiles(const GemmArgs& a) {
  static const int kSplits[] = {1, 2, 3, 4, 5, 6, 8, 10, 12, 16};
  struct Cand {
    int cfg, bm, bn;
    double c_kt;
  };
  static const Cand kCands[] = {
      {0, 128, 128, 0.5931}, {1, 256, 128, 0.9088}, {4, 256, 192, 1.2088}, {3, 256, 256, 1.4367}};
  const int nkt = a.K / 64;
  double best = 1e300;
  TileChoice pick{3, 1};
  for (const Cand& c : kCands) {
    const long mt = cdiv(a.M, c.bm), tiles = mt * cdiv(a.N, c.bn);
    const double hbm = (double)mt * a.N * a.K * 2.0 / 1e6 * 0.1773;
    for (int sp : kSplits) {
      if (sp > nkt) break;
      if (sp > 1 && (!a.ws || (long)sp * a.M * a.N > a.ws_elems)) break;
      const int ks = cdiv(nkt, sp), s = cdiv(nkt, ks);
      const long rounds = cdiv(tiles * s, 256);
      double t = std::max(rounds * (0.7377 + ks * c.c_kt), hbm);
      if (s > 1) t += 5.6764 + (double)s * a.M * a.N * 8.0 / 1e6 / 5.7874;
      if (t < best) {
        best = t;
        pick = {c.cfg, s};
      }
    }
  }
  // Two launches over column groups: the first group's workgroups fill whole
  // rounds, the second group takes its own split count, so no round runs
  // part-empty the way a uniform split leaves the last one (the query/key/value
  // product of 144 tiles of 256 x 256: 2 x 128 + 16 x 16 workgroups against 3
  // x 144).  Taken when the model puts it 3 % under the best single launch.
  const double single = best;
  for (const Cand& c : kCands) {
    if (c.bm != 256 || c.bn < 192) continue;
    const long mt = cdiv(a.M, c.bm), tn = cdiv(a.N, c.bn);
    for (int sp1 : kSplits) {
      if (sp1 > nkt) break;
      const int ks1 = cdiv(nkt, sp1), e1 = cdiv(nkt, ks1);
      for (long r1 = 1;; ++r1) {
        const long cols1 = r1 * 256 / (mt * e1);
        if (cols1 >= tn) break;
        if (cols1 * mt * e1 != r1 * 256) continue;
        const long n1 = cols1 * c.bn, n2 = a.N - n1;
        const double hbm1 = (double)mt * n1 * a.K * 2.0 / 1e6 * 0.1773;
        const double hbm2 = (double)mt * n2 * a.K * 2.0 / 1e6 * 0.1773;
        for (int sp2 : kSplits) {
          if (sp2 > nkt) break;
          const int ks2 = cdiv(nkt, sp2), e2 = cdiv(nkt, ks2);
          const double part = (double)e1 * a.M * n1 + (double)e2 * a.M * n2;
          if (!a.ws || part > (double)a.ws_elems) break;
          const long r2 = cdiv(mt * (tn - cols1) * e2, 256);
          double t = std::max(r1 * (0.7377 + ks1 * c.c_kt), hbm1) +
                     std::max(r2 * (0.7377 + ks2 * c.c_kt), hbm2);
          t += 5.6764 + part * 8.0 / 1e6 / 5.7874;
          if (t < best && t < 0.97 * single) {
            best = t;
            pick = {c.cfg, e1, e2, (int)cols1};
          }
        }
      }
    }
  }
  return pick;
}

}  // namespace

// Explicit configuration (for measurement); -1 picks by shape.  Shapes the
// DMA path takes: K a multiple of BK; every operand dimension a multiple of 8;
// m/n-contiguous operands at least 128 wide.
hipError_t gemm_dma_bf16_cfg(int cfg, const GemmArgs& a, hipStream_t s) {
  if (a.M <= 0 || a.N <= 0) return hipSuccess;
  if (a.M % 8 || a.N % 8 || a.K % 32) return hipErrorNotSupported;
  const bool a_kc = a.sak == 1, b_kc = a.sbk == 1, a_mc = a.sam == 1, b_nc = a.sbn == 1;
  if (((uintptr_t)a.A & 15) || ((uintptr_t)a.B & 15)) return hipErrorNotSupported;
  const long lda = a_kc ? a.sam : a.sak, ldb = b_kc ? a.sbn : a.sbk;
  if ((lda & 7) || (ldb & 7)) return hipErrorNotSupported;
  // per-lane DMA offsets are 32-bit byte offsets from a k-origin
  auto fits = [](long rows, long ld) { return (rows + 1) * ld * 2 < (1l << 32); };
  if (!fits(a_kc ? a.M : 64, lda) || !fits(b_kc ? a.N : 64, ldb)) return hipErrorNotSupported;
  // fp32 outputs leave as 16-byte row segments, bf16 outputs (and their
  // operands) as 8-column segments
  if (a.epi == EPI_ACC_F32 && (((uintptr_t)a.C & 15) || (a.ldc & 3))) return hipErrorNotSupported;
  if (a.epi != EPI_ACC_F32 && !vec8_ok(a)) return hipErrorNotSupported;
  int splits = 0, splits2 = 0, cols1 = 0;
  if (cfg < 0) {
    // weight-gradient products (both operands m/n-contiguous): 256 x 256 tiles
    // over one (A, B) ring; products with a weight matrix as B: the modelled
    // best tile shape and split count (256 x 256 tiles keep the weight stream
    // a k-tile further ahead than the activations)
    if (a_mc && b_nc) {
      cfg = 2;
    } else {
      const TileChoice c = choose_tiles(a);
      cfg = c.cfg;
      splits = c.splits;
      splits2 = c.splits2;
      cols1 = c.cols1;
    }
  }
  if (a.in_f16) {
    // fp16 operands: the query/key/value product (activations times the fp16
    // weight copy, both k-contiguous)
    if (!(a_kc && b_kc) || a.epi != EPI_QKV) return hipErrorNotSupported;
    return run_cfg_id<true, true, true>(cfg, a, s, splits, splits2, cols1);
  }
  if (a_kc && b_kc) return run_cfg_id<true, true>(cfg, a, s, splits, splits2, cols1);
  if (a_kc && b_nc) return run_cfg_id<true, false>(cfg, a, s, splits, splits2, cols1);
  if (a_mc && b_nc) {
    if (a.M < 128 || a.N < 128) return hipErrorNotSupported;
    return run_cfg_id<false, false>(cfg, a, s);
  }
  return hipErrorNotSupported;
}

hipError_t gemm_dma_bf16(const GemmArgs& a, hipStream_t s) { return gemm_dma_bf16_cfg(-1, a, s); }

}  // namespace tp
