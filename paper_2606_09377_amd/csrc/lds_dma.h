// Operand tiles loaded straight from global memory into LDS on gfx950, and the bank
// swizzle of the tiles: shared by the GEMM and transposed-convolution kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <cstdint>

namespace vcr {

// LDS rows of BK floats, unpadded, as BK / 4 16-byte chunks; chunk c of tile row q sits at
// chunk c ^ swz(q).  A 16-byte LDS access serves 16 lanes per cycle over the 64 banks, so the
// swizzle spreads 16 consecutive rows at one chunk (the MFMA operand reads) over 16 distinct
// 4-bank groups; stores of whole rows are spread already.  (Rows whose offsets coincide
// modulo the 64 banks get different chunk positions.)  The pattern repeats every 16 rows.
template <int BK>
__device__ __forceinline__ int lds_swz(int row) {
  constexpr int CPR = BK / 4, RPG = 16 / CPR;
  return (row / RPG) & (CPR - 1);
}

// The LDS byte address of a __shared__ location (the value M0 takes for a load to LDS):
// computed once per kernel, outside the loops that issue the loads.
__device__ __forceinline__ uint32_t lds_addr(const float *p) {
  return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) float *)p;
}

// 16 bytes from global memory into LDS: lane i of the wave writes LDS byte address lds + 16 i
// (lds is wave-uniform).  Issued as inline assembly so that the compiler neither waits on the
// vector-memory counter before every LDS read of the loop nor counts these loads: the loop
// waits for them itself (wait_vmcnt) before the barrier that publishes a stage.  M0 carries
// the LDS address, with the one wait state a load to LDS needs after an M0 write.  M0 is
// clobbered without being restored: the kernels that call this have no other use of M0
// (checked in their ISA; saving and restoring it around every load cost 0.6% on the GEMM).
// Clobbering a register the compiler reserves draws a warning, silenced here.
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
__device__ __forceinline__ void dma16(const float *g, uint32_t lds) {
  asm volatile(
      "s_mov_b32 m0, %0\n\t"
      "s_nop 0\n\t"
      "global_load_lds_dwordx4 %1, off"
      :
      : "s"(__builtin_amdgcn_readfirstlane(lds)), "v"(g)
      : "memory", "m0");
}
// The same with the LDS location given as a pointer: the address conversion happens at every
// load.  (The GEMM kernels use this form: on the wide MLP it measured 1% faster than loads
// from precomputed addresses, which issue closer together; the convolutions gain 1% the other
// way round.)
__device__ __forceinline__ void dma16(const float *g, float *lds) {
  const uint32_t l = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) float *)lds;
  asm volatile(
      "s_mov_b32 m0, %0\n\t"
      "s_nop 0\n\t"
      "global_load_lds_dwordx4 %1, off"
      :
      : "s"(__builtin_amdgcn_readfirstlane(l)), "v"(g)
      : "memory", "m0");
}
#pragma clang diagnostic pop

// Workgroup barrier after this wave's LDS reads have completed, without the memory fences of
// __syncthreads (which wait for every outstanding vector-memory load, the prefetched stages
// included); the "memory" clobber keeps the compiler's LDS accesses on their side.
__device__ __forceinline__ void barrier_only() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

// s_waitcnt on the vector-memory counter alone (vmcnt <= N; gfx9 encoding: vmcnt in bits 3:0
// and 15:14, expcnt and lgkmcnt left at their maxima)
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (15 << 8) | ((N >> 4) << 14));
}

}  // namespace vcr
