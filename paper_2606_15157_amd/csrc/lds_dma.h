// LDS DMA and vector-memory waits shared by the gfx950 kernels of librkv.
#pragma once

#include <hip/hip_runtime.h>

#include <stdint.h>

namespace rkv {
namespace {

// s_waitcnt vmcnt(N) (expcnt and lgkmcnt not waited for).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt is six bits");
  __builtin_amdgcn_s_waitcnt((N & 15) | (((N >> 4) & 3) << 14) | (7 << 4) | (15 << 8));
}

// 16 bytes per lane from global memory into LDS at lds_base + 16 lane (LDS DMA).  Issued as
// inline assembly so that the compiler does not conservatively wait for it before unrelated
// LDS reads; the issuing wave waits for it explicitly (vmcnt) before a barrier hands the data
// on.  lds_base must be wave-uniform.
// M0 is reserved by the compiler (it may hold a value across this statement), so the
// assembly saves it in a scratch SGPR and restores it after the DMA instruction has read it.
__device__ __forceinline__ void dma16(const void* src, uint32_t lds_base) {
  uint32_t saved;
  asm volatile(
      "s_mov_b32 %0, m0\n\ts_mov_b32 m0, %2\n\ts_nop 0\n\t"
      "global_load_lds_dwordx4 %1, off\n\ts_mov_b32 m0, %0"
      : "=&s"(saved)
      : "v"(src), "s"(lds_base)
      : "memory");
}
// Two of those 4 KiB apart: [base + off] -> lds_base and [base + 4096 + off] -> lds_base + 4096
// (+ 16 lane).  The instruction offset applies to the global and to the LDS address alike, so
// one base and one M0 value serve both.
__device__ __forceinline__ void dma16s_pair(const char* base, uint32_t off, uint32_t lds_base) {
  uint32_t saved;
  asm volatile(
      "s_mov_b32 %0, m0\n\ts_mov_b32 m0, %3\n\ts_nop 0\n\t"
      "global_load_lds_dwordx4 %1, %2 offset:-4096\n\t"
      "global_load_lds_dwordx4 %1, %2\n\ts_mov_b32 m0, %0"
      : "=&s"(saved)
      : "v"(off), "s"(base + 4096), "s"(lds_base + 4096u)
      : "memory");
}
__device__ __forceinline__ uint32_t lds_addr(const void* p) {
  return __builtin_amdgcn_readfirstlane(
      (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void*)p);
}

}  // namespace
}  // namespace rkv
