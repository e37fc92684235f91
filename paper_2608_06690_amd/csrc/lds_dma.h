// Global -> LDS copies (global_load_lds_dwordx4) and the waits and barriers around
// them, shared by the kernels that stage MFMA operands in LDS rings.
#pragma once
#include <type_traits>

#include "pmpe_internal.h"

namespace pmpe {

typedef __attribute__((address_space(3))) unsigned char lds_u8;

// 32-bit LDS address of a shared-memory pointer.
__device__ __forceinline__ uint32_t lds_addr(const void* p) {
  return (uint32_t)(uintptr_t)(const lds_u8*)p;
}

// Global -> LDS copy of 16 bytes per lane, addressed as a wave-uniform 64-bit base
// (SGPRs) plus a per-lane 32-bit byte offset: lane l's bytes land at lds_base + IMM +
// 16 * l (the LDS base is wave-uniform, held in M0). Written as inline assembly so that
// the compiler does not treat the copy as a pending LDS write that every later LDS read
// must wait for; a kernel waits for its own copies explicitly (wait_vmcnt) before a
// barrier and only then reads the stage they filled. The base and the LDS address are
// passed through readfirstlane so that they are held in SGPRs whatever the compiler can
// prove.
//
// The assembly must leave SCC alone: the compiler does not know that an asm statement
// changes it and may place one between its own SCC producer and consumer (the low and
// high halves of a 64-bit address add, a compare and its branch). So M0 is written with
// s_mov_b32 (which leaves SCC unchanged) from an LDS address the compiler has already
// summed, never with s_add_u32.
__device__ __forceinline__ const void* uniform_ptr(const void* p) {
  const uint64_t v = (uint64_t)(uintptr_t)p;
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)v);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(v >> 32));
  return (const void*)(uintptr_t)(((uint64_t)hi << 32) | lo);
}
// NT: non-temporal hint, for operands that are read once (streamed weights).
template <int IMM, bool NT>
__device__ __forceinline__ void dma16s(uint32_t byte_off, const void* base_, uint32_t lds_base_) {
  const void* base = uniform_ptr(base_);
  const uint32_t lds = __builtin_amdgcn_readfirstlane(lds_base_ + (uint32_t)IMM);
  if constexpr (NT)
    asm volatile(
        "s_mov_b32 m0, %2\n\t"
        "s_nop 0\n\t"
        "global_load_lds_dwordx4 %0, %1 offset:0 nt" ::"v"(byte_off),
        "s"(base), "s"(lds)
        : "memory", "m0");
  else
    asm volatile(
        "s_mov_b32 m0, %2\n\t"
        "s_nop 0\n\t"
        "global_load_lds_dwordx4 %0, %1 offset:0" ::"v"(byte_off),
        "s"(base), "s"(lds)
        : "memory", "m0");
}

// f(integral_constant<I>), ..., f(integral_constant<N-1>): copies whose LDS offset is an
// immediate (IMM of dma16s) are issued from a compile-time index.
template <int I, int N>
struct Unroll {
  template <class F>
  __device__ __forceinline__ static void run(F&& f) {
    f(std::integral_constant<int, I>{});
    Unroll<I + 1, N>::run(f);
  }
};
template <int N>
struct Unroll<N, N> {
  template <class F>
  __device__ __forceinline__ static void run(F&&) {}
};

template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

// Workgroup barrier without the full memory drain that __syncthreads() implies: the
// copies a stage depends on were already waited for (wait_vmcnt), and every LDS read
// of the previous stage was consumed by an MFMA before this point. Later stages'
// copies stay in flight across it.
__device__ __forceinline__ void barrier_raw() { asm volatile("s_barrier" ::: "memory"); }

}  // namespace pmpe
