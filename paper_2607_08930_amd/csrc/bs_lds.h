// Direct HBM -> LDS transfers (gfx950 global_load_lds) shared by the kernels
// that stage tiles through LDS rings.
//
// One wave instruction moves 64 lanes x 16 bytes: lane l fills bytes
// [16 l, 16 l + 16) of the 1 KiB LDS block at M0, from its own global address.
// The transfers are issued through inline assembly and waited for with
// explicit vmcnt counts: the compiler's waitcnt pass cannot see them and would
// otherwise drain every stage in flight before the first LDS read.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace bs {

typedef __attribute__((address_space(3))) void lds_void;

__device__ inline uint32_t lds_addr(const void* p) {
  return static_cast<uint32_t>(reinterpret_cast<uintptr_t>((lds_void*)p));
}

// One wave instruction: 64 lanes x 16 bytes, HBM -> LDS block at `lds` (wave-uniform).
__device__ inline void dma16(uint32_t lds, const void* gptr) {
  asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx4 %1, off" ::"s"(__builtin_amdgcn_readfirstlane(lds)),
               "v"(gptr)
               : "memory");
}
__device__ inline uint64_t uniform64(const void* p) {
  const uint64_t v = reinterpret_cast<uint64_t>(p);
  const uint32_t lo = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(v));
  const uint32_t hi = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(v >> 32));
  return (static_cast<uint64_t>(hi) << 32) | lo;
}
// Same, addressed as a wave-uniform base (SGPRs) plus a 32-bit per-lane byte offset.
__device__ inline void dma16_sv(uint32_t lds, uint64_t base, uint32_t off) {
  asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx4 %1, %2" ::"s"(__builtin_amdgcn_readfirstlane(lds)),
               "v"(off), "s"(uniform64(reinterpret_cast<const void*>(base)))
               : "memory");
}

// The same two transfers with the non-temporal hint: for tiles read exactly
// once (the step attention's K/V stream), so they do not displace lines that
// other work reuses. Kernels that share tiles through L2 (the output head,
// the refresh) use the plain forms.
__device__ inline void dma16_once(uint32_t lds, const void* gptr) {
  asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx4 %1, off nt" ::"s"(__builtin_amdgcn_readfirstlane(lds)),
               "v"(gptr)
               : "memory");
}
__device__ inline void dma16_sv_once(uint32_t lds, uint64_t base, uint32_t off) {
  asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx4 %1, %2 nt" ::"s"(__builtin_amdgcn_readfirstlane(lds)),
               "v"(off), "s"(uniform64(reinterpret_cast<const void*>(base)))
               : "memory");
}

// Wait until at most N (compile time) of this wave's vector-memory operations
// are outstanding. gfx9 encoding: vmcnt[3:0] | expcnt[6:4] | lgkmcnt[11:8] |
// vmcnt_hi[15:14]; counts above 63 wait for everything.
template <int N>
__device__ inline void wait_vm_c() {
  constexpr int n = N > 63 ? 0 : N;
  __builtin_amdgcn_s_waitcnt((n & 15) | ((n >> 4) << 14) | (7 << 4) | (15 << 8));
}

}  // namespace bs
