// Direct global -> LDS copies (global_load_lds_dword{,x4}) and the waits that
// go with them, shared by the GEMM kernels that stage operands in LDS.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace moe {

// One 16-byte (or 4-byte) element per lane: lane l lands at LDS byte
// `lds + 16*l` (`lds + 4*l`); inactive lanes neither load nor write.  Issued
// as inline asm so the compiler does not treat every later LDS read as
// dependent on it; completion is awaited explicitly with vm_wait<N>().
// `lds` must be uniform across the wave.  An LDS-DMA that reads M0 needs one
// wait state after the SALU write of M0; the hazard recognizer cannot see
// inside inline asm, so the s_nop is written out here.
__device__ __forceinline__ void dma16(const void* gptr, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, off" ::"s"(__builtin_amdgcn_readfirstlane(lds)),
               "v"(gptr) : "memory", "m0");
}
// The same with the non-temporal hint: for data read exactly once (streamed
// weights), so it does not displace reused lines in L2.
__device__ __forceinline__ void dma16_nt(const void* gptr, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, off nt" ::"s"(__builtin_amdgcn_readfirstlane(lds)),
               "v"(gptr) : "memory", "m0");
}
__device__ __forceinline__ void dma4(const void* gptr, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dword %1, off" ::"s"(__builtin_amdgcn_readfirstlane(lds)),
               "v"(gptr) : "memory", "m0");
}
__device__ __forceinline__ uint32_t lds_addr(const void* p) {
  return __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(reinterpret_cast<uintptr_t>(p)));
}
// s_waitcnt with only the vector-memory count: at most N loads outstanding.
// The signal fences keep the compiler from moving LDS reads of the data the
// wait covers above it.
template <int N>
__device__ __forceinline__ void vm_wait() {
  static_assert(N >= 0 && N < 64, "vmcnt is 6 bits");
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
  __builtin_amdgcn_s_waitcnt(((N >> 4) & 3) << 14 | (0xF << 8) | (7 << 4) | (N & 0xF));
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
}
// s_waitcnt lgkmcnt(0): every LDS read issued so far has returned.
__device__ __forceinline__ void lds_wait() { __builtin_amdgcn_s_waitcnt(0xC07F); }
// Workgroup barrier without a memory fence (the fence of __syncthreads would
// also drain the loads still in flight for later stages).
__device__ __forceinline__ void bar() {
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
  __builtin_amdgcn_s_barrier();
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
}

}  // namespace moe
