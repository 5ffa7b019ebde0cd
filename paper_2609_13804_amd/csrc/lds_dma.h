// Global -> LDS loads without register staging, shared by the matrix-core
// kernels (gemm.hip, encode.hip).
#pragma once

#include "sp_internal.h"

namespace sp {
namespace {

typedef __attribute__((address_space(3))) void* lptr_t;

// One 16-byte-per-lane global load straight into LDS (global_load_lds_dwordx4:
// lane i's bytes land at dst + 16 i, dst taken from M0, uniform in the wave).
// It is written as inline assembly so that the compiler does not track it:
// it models the builtin as an access that may touch both memory and LDS, and
// then waits for every outstanding LDS read (lgkmcnt(0)) wherever a fragment
// is consumed, including reads issued just before.  The caller awaits its
// completion explicitly (wait_vmcnt, then a barrier) before any wave reads
// what it filled.  The statement sets M0 itself, right before its load.  The
// compiler reserves M0 and does not preserve it across inline assembly, so the
// kernels that use this must not hold any other value in M0; in the generated
// code every write of M0 is this statement's (tests/test_codegen.py checks it).
__device__ __forceinline__ void lds_dma16(const void* src, char* dst) {
  const uint32_t l = __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)(lptr_t)dst);
  asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off"
               :: "v"(src), "s"(l) : "memory", "m0");
}

// s_waitcnt with only the vector-memory counter constrained (gfx9 encoding).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

}  // namespace
}  // namespace sp
