// Device helpers shared by the kernels that stage operands through LDS:
// buffer resources (out-of-range offsets read zeros), LDS-DMA loads issued
// from inline assembly, explicit waits and barriers.
#pragma once

#include "foe_common.hpp"

namespace foe {

// Buffer resources end where the valid rows / K end: loads at offsets at or
// past the range return zeros, which handles ragged rows and K tails without
// branches.  kOob lies past every range used here.
constexpr uint32_t kOob = 0x80000000u;

// LDS-only workgroup barrier: waits for this wave's LDS operations and meets
// the other waves, but (unlike __syncthreads) does not drain outstanding
// global loads, so prefetches stay in flight across it.
__device__ __forceinline__ void lds_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

// LDS byte address of a __shared__ object: a generic address in the LDS
// aperture carries the aperture in its high 32 bits and the LDS offset in its
// low 32 bits (taking the low half avoids the null check of an address-space
// cast).
__device__ __forceinline__ uint32_t lds_addr(const void* p) { return (uint32_t)(uintptr_t)p; }
// Buffer resource built from wave-uniform (readfirstlane) fields, so that it
// is guaranteed to sit in SGPRs as the inline assembly below requires.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc_u(const void* base, uint32_t nbytes) {
  const uint64_t a = (uint64_t)(uintptr_t)base;
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)a);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(a >> 32));
  void* p = (void*)(uintptr_t)(((uint64_t)hi << 32) | lo);
  return __builtin_amdgcn_make_buffer_rsrc(p, (short)0, __builtin_amdgcn_readfirstlane(nbytes),
                                           0x00020000);
}
// LDS destination = lds + imm; imm is a constant once the call is inlined
// (the library is built with optimisation), so the per-instruction LDS
// addresses cost no registers.  An LDS-DMA load that reads M0 needs one wait
// state after the scalar write of M0 (the s_nop).
__device__ __forceinline__ void dma16(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t lds,
                                      int imm) {
  asm volatile("s_add_u32 m0, %2, %3\n\ts_nop 0\n\tbuffer_load_dwordx4 %0, %1, 0 offen lds" ::"v"(voff),
               "s"(r), "s"(lds), "i"(imm)
               : "memory");
}
// wait until at most N of this wave's vector memory operations are
// outstanding and its LDS operations are done, then meet the other waves
template <int N>
__device__ __forceinline__ void vm_barrier() {
  asm volatile("s_waitcnt vmcnt(%0)\n\ts_waitcnt lgkmcnt(0)\n\ts_barrier" ::"n"(N) : "memory");
}

// XOR swizzle of the 16-byte chunks of an LDS tile row of CPR chunks: chunk c
// of row r is stored in slot c ^ swz(r), so that 16 consecutive rows read at
// the same chunk touch every bank group once.
template <int CPR>
__device__ __forceinline__ int swz(int r) {
  static_assert(CPR == 4 || CPR == 8 || CPR == 16, "rows of 64, 128 or 256 bytes");
  if constexpr (CPR == 16) return r & 15;
  else if constexpr (CPR == 8) return (r & 7) ^ ((r >> 3) & 1);
  else return ((r >> 1) & 3) ^ ((r >> 3) & 1);
}

// wait until at most N of this wave's vector memory operations are outstanding
// (loads retire in issue order)
template <int N>
__device__ __forceinline__ void vm_wait() {
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

}  // namespace foe
