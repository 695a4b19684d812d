// Direct global -> LDS copies (gfx950 global_load_lds_dwordx4) and the LDS
// tile layouts of the GEMM kernels that are fed by them.
#pragma once
#include <hip/hip_runtime.h>

#include <cstdint>

namespace swsft {

// One direct global -> LDS copy of 16 bytes per lane: lane l writes
// LDS[lds_base + 16 l].  M0 holds the wave-uniform LDS base (with the NOP
// its write requires before the copy).  The copy counts in vmcnt like a
// load; it is waited for with wait_vmcnt, never by the compiler.
__device__ __forceinline__ void dma16(const void* g, unsigned lds_base) {
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, off"
               :
               : "s"(__builtin_amdgcn_readfirstlane(lds_base)), "v"(g)
               : "memory");
}

template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt immediate");
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

// Wait until at most `ahead` groups of P copies are outstanding (ahead <= A).
template <int A, int P>
__device__ __forceinline__ void wait_groups(int ahead) {
  if constexpr (A == 0) {
    wait_vmcnt<0>();
  } else {
    if (ahead >= A) wait_vmcnt<A * P>();
    else wait_groups<A - 1, P>(ahead);
  }
}

// LDS byte address of a shared-memory pointer (shared arrays start at LDS
// offset 0 of the aperture, so the low 32 bits of the generic address).
__device__ __forceinline__ unsigned lds_addr(const void* p) { return (unsigned)(uintptr_t)p; }

// Row-major K-contiguous tile, CPR 16-byte chunks per row: slot of chunk c of
// row r.  XOR-swizzled so that the 32 rows one MFMA operand read touches
// fall in distinct banks for 8- and for 16-lane groups of a 16-byte read.
template <int CPR>
__device__ __forceinline__ int swz(int r, int c) {
  static_assert(CPR == 4 || CPR == 8, "chunks per row");
  if constexpr (CPR == 4) return c ^ (((r >> 1) ^ (r >> 3)) & 3);
  else return c ^ ((r & 7) ^ ((r >> 3) & 1));
}

// K-major tile (row k holds consecutive M indices, at least 16 chunks):
// slot of chunk c of row k.  Rows k..k+3 of one transposed read land in
// four different 64-byte windows.
__device__ __forceinline__ int swz_t(int k, int c) { return c ^ ((k & 3) << 2); }

// K-major tile read by dword gathers (a lane takes 4 consecutive rows of one
// column, the two lane halves rows 4 apart; at least 16 chunks per row): the
// chunks of alternate groups of 4 rows are moved by 128 bytes so that the two
// halves of a wave hit different banks.  Self-inverse.
__device__ __forceinline__ int swz_k4(int k, int c) { return c ^ (((k >> 2) & 1) << 3); }

}  // namespace swsft
