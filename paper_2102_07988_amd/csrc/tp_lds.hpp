// LDS DMA and explicit LDS reads for gfx950 kernels.
//
// global_load_lds (`dma16`, `dma4`): each active lane moves 16 (4) bytes from
// its own global address into LDS at the wave-uniform base + lane * 16 (4).
// The completion is tracked by vmcnt in issue order, so kernels wait with
// `wait_vm<N>()` (N = DMA instructions allowed to remain in flight) followed by
// a barrier.  LDS reads that feed the matrix cores are issued as inline
// assembly: the compiler does not see them, so it does not drain every
// outstanding DMA before each read; callers wait with lgkmcnt(0) tied to the
// registers the reads produced.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace tp {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

__device__ inline uint32_t lds_addr(const void* p) {
  return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void*)p;
}

__device__ inline void dma16(const void* g, void* lds_wave_base) {
  __builtin_amdgcn_global_load_lds((const __attribute__((address_space(1))) void*)g,
                                   (__attribute__((address_space(3))) void*)lds_wave_base, 16, 0,
                                   0);
}

__device__ inline void dma4(const void* g, void* lds_wave_base) {
  __builtin_amdgcn_global_load_lds((const __attribute__((address_space(1))) void*)g,
                                   (__attribute__((address_space(3))) void*)lds_wave_base, 4, 0,
                                   0);
}

__device__ inline u32x4 ds_read128(uint32_t addr) {
  u32x4 v;
  asm volatile("ds_read_b128 %0, %1" : "=v"(v) : "v"(addr));
  return v;
}

// Transposing read: within each group of 16 lanes, lane j supplies the address
// of 4 consecutive 16-bit elements of row j/4 at column block j%4; lane i then
// holds element i%4 of the rows supplied by lanes i/4, 4 + i/4, 8 + i/4 and
// 12 + i/4.  With lane j pointing at (row r0 + j/4, column c0 + 4 (j%4)), lane i
// receives column c0 + i at rows r0 .. r0 + 3.
__device__ inline u32x2 ds_read_tr(uint32_t addr) {
  u32x2 v;
  asm volatile("ds_read_b64_tr_b16 %0, %1" : "=v"(v) : "v"(addr));
  return v;
}

__device__ inline u32x4 join(u32x2 lo, u32x2 hi) {
  u32x4 r;
  r.x = lo.x;
  r.y = lo.y;
  r.z = hi.x;
  r.w = hi.y;
  return r;
}

// Wait for every LDS read issued so far; `x` is tied so its uses follow the wait.
__device__ inline void lgkm_wait(u32x4& x) { asm volatile("s_waitcnt lgkmcnt(0)" : "+v"(x)); }
// Orders a further register after a preceding lgkm_wait (no instruction).
__device__ inline void lgkm_tie(u32x4& x) { asm volatile("" : "+v"(x)); }

template <int N>
__device__ inline void wait_vm() {
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

// Wait until at most `pending` groups of LPT DMA instructions are in flight.
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

}  // namespace tp
