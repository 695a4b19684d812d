// Building blocks of the register-staged MFMA GEMMs: the double-buffered
// main loop over K tiles, the LDS-staged epilogue, and the row loader of
// K-contiguous operand tiles.  Operands are staged in LDS K-contiguous and
// multiplied by MfmaTile (mfma_tile.h).
//
// Main loop: two LDS buffers and one barrier per K step; the global loads
// of step k+2 are in flight while step k is multiplied.  Epilogue: the
// accumulator tile goes through LDS so that results leave in 16-byte rows.
#pragma once

#include "mfma_tile.h"
#include "swsft_internal.h"

namespace swsft {
namespace {

constexpr int NT = 256;

struct SpinList {
  int s[kMaxSpins];
};

__device__ __forceinline__ int iabs(int v) { return v < 0 ? -v : v; }

template <typename T>
struct Vec16 {
  static constexpr int N = 16 / sizeof(T);
  union {
    uint4 u;
    T e[N];
  };
};

// LDS bytes of one operand stage and of the epilogue tile.
template <typename T, int BM, int BN, int BK>
struct GemmLds {
  static constexpr int LD = BK + LdsPad<T>::value;
  static constexpr int LDC = BN + (sizeof(T) == 4 ? 4 : 8);
  static constexpr size_t stage = (size_t)(BM + BN) * LD * sizeof(T);
  static constexpr size_t mainloop = 2 * stage;
  static constexpr size_t epilogue = (size_t)BM * LDC * sizeof(T);
  static constexpr size_t bytes = mainloop > epilogue ? mainloop : epilogue;
};

// Double-buffered main loop over nk K-tiles.  la / lb: load(kt) issues the
// global reads of K-tile kt into registers, store(lds) writes them to LDS.
template <typename T, int BM, int BN, int BK, int WM, int WN, class LA, class LB>
__device__ __forceinline__ void mainloop(MfmaTile<T, BM, BN, BK, WM, WN>& tile, LA& la, LB& lb,
                                         T* smem, int nk, int wm, int wn, int lane) {
  using G = GemmLds<T, BM, BN, BK>;
  constexpr int kStage = (BM + BN) * G::LD;  // elements per buffer (A then B)
  la.load(0);
  lb.load(0);
  la.store(smem);
  lb.store(smem + BM * G::LD);
  if (nk > 1) {
    la.load(1);
    lb.load(1);
  }
  __syncthreads();
  for (int kt = 0; kt < nk; ++kt) {
    T* cur = smem + (kt & 1) * kStage;
    T* nxt = smem + ((kt & 1) ^ 1) * kStage;
    if (kt + 1 < nk) {
      la.store(nxt);
      lb.store(nxt + BM * G::LD);
      if (kt + 2 < nk) {
        la.load(kt + 2);
        lb.load(kt + 2);
      }
    }
    tile.compute(cur, cur + BM * G::LD, wm, wn, lane);
    __syncthreads();
  }
}

// Epilogue: accumulators -> LDS tile [BM][LDC] of T -> `out(row, col, vec,
// n)` with up to VEC consecutive columns per call (n valid values).
template <typename T, int BM, int BN, int BK, int WM, int WN, class Out>
__device__ __forceinline__ void epilogue(const MfmaTile<T, BM, BN, BK, WM, WN>& tile, T* smem,
                                         int rows, int cols, int wm, int wn, int lane, int tid,
                                         Out&& out) {
  using G = GemmLds<T, BM, BN, BK>;
  constexpr int VEC = 16 / sizeof(T);
  tile.for_each(wm, wn, lane,
                [&](int row, int col, float v) { smem[row * G::LDC + col] = (T)v; });
  __syncthreads();
  constexpr int VPR = BN / VEC;
  for (int idx = tid; idx < BM * VPR; idx += NT) {
    const int row = idx / VPR;
    const int col = (idx % VPR) * VEC;
    if (row >= rows || col >= cols) continue;
    Vec16<T> v;
    v.u = *reinterpret_cast<const uint4*>(&smem[row * G::LDC + col]);
    out(row, col, v, cols - col < VEC ? cols - col : VEC);
  }
}

// K-contiguous operand tile of R rows from global rows given by row_ptr(r)
// (nullptr = zero row); columns >= K are zero.  Element k of a row is at
// row + k_base + (k - k_base) / BK * kstride + (k - k_base) % BK: kstride = BK
// for plain rows, the tile stride for K-tiled operands.  kVec: 16-byte loads (rows
// 16-byte aligned, K a multiple of the vector); else element loads.  The
// choice is a template flag: as a runtime branch the compiler merges both
// paths into element loads.
//
// Loads are never inside a per-lane branch: out-of-range lanes read a
// clamped valid address and the zero mask is applied when the registers are
// written to LDS, so the loads of a K step stay in flight together (a
// divergent if/else writing the same registers would force a wait on each).
template <typename T, int R, int BK, bool kVec>
struct RowLoader {
  static constexpr int VEC = 16 / sizeof(T);
  static constexpr int VPR = BK / VEC;
  static constexpr int NV = R * VPR;
  static constexpr int PER = (NV + NT - 1) / NT;
  static constexpr int LD = BK + LdsPad<T>::value;
  Vec16<T> reg[PER];
  const T* rows_[PER];
  bool rowok_[PER];
  unsigned ok_[PER];  // bit e: element e of reg[p] is in range
  int kv_[PER];
  int k_base, K;
  size_t kstride;  // elements between consecutive K tiles of a row

  template <class RowPtr>
  __device__ __forceinline__ void init(RowPtr&& row_ptr, const T* fallback, int k_base_, int K_,
                                       int tid, size_t kstride_ = BK) {
    k_base = k_base_;
    K = K_;
    kstride = kstride_;
#pragma unroll
    for (int p = 0; p < PER; ++p) {
      const int v = tid + p * NT;
      const T* r = (NV % NT == 0 || v < NV) ? row_ptr(v / VPR) : nullptr;
      rowok_[p] = r != nullptr;
      rows_[p] = r != nullptr ? r : fallback;
      kv_[p] = (v % VPR) * VEC;
    }
  }
  __device__ __forceinline__ void load(int kt) {
#pragma unroll
    for (int p = 0; p < PER; ++p) {
      const int k = k_base + kt * BK + kv_[p];
      const size_t off = k_base + kt * kstride + kv_[p];  // address of element k
      if constexpr (kVec) {
        const bool ok = rowok_[p] && k < K;
        reg[p].u = *reinterpret_cast<const uint4*>(rows_[p] + (ok ? off : 0));
        ok_[p] = ok ? 0xffu : 0u;
      } else {
        unsigned bits = 0;
#pragma unroll
        for (int e = 0; e < VEC; ++e) {
          const bool ok = rowok_[p] && k + e < K;
          reg[p].e[e] = rows_[p][ok ? off + e : 0];
          bits |= (ok ? 1u : 0u) << e;
        }
        ok_[p] = bits;
      }
    }
  }
  __device__ __forceinline__ void store(T* lds) {
    const int tid = threadIdx.x;
#pragma unroll
    for (int p = 0; p < PER; ++p) {
      const int v = tid + p * NT;
      if (NV % NT != 0 && v >= NV) break;
      const int r = v / VPR;
      if constexpr (kVec) {
        if (!ok_[p]) reg[p].u = make_uint4(0, 0, 0, 0);
      } else {
#pragma unroll
        for (int e = 0; e < VEC; ++e)
          if (!((ok_[p] >> e) & 1u)) reg[p].e[e] = (T)0.f;
      }
      if constexpr (sizeof(T) == 4) {
#pragma unroll
        for (int e = 0; e < VEC; ++e) lds[r * LD + kv_[p] + e] = reg[p].e[e];
      } else {
        *reinterpret_cast<uint4*>(&lds[r * LD + kv_[p]]) = reg[p].u;
      }
    }
  }
};

}  // namespace
}  // namespace swsft
