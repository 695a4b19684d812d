// Workgroup-level MFMA tile: C[BM x BN] += A[BM x BK] * B[BN x BK]^T with
// both operands staged in LDS K-contiguous (row pitch BK + pad).  Four
// waves in a WM x WN arrangement; each wave owns (BM/WM) x (BN/WN) as
// 32 x 32 MFMA blocks.
//   float : v_mfma_f32_32x32x2f32   (lane l: row l%32, k = l/32)
//   bf16  : v_mfma_f32_32x32x16_bf16 (lane l: row l%32, k = 8*(l/32) .. +7)
// Accumulator register r of lane l holds row 8*(r/4) + 4*(l/32) + r%4,
// column l%32 of its 32 x 32 block.
#pragma once

#include <hip/hip_runtime.h>

#include <type_traits>

namespace swsft {

typedef float v16f __attribute__((ext_vector_type(16)));
typedef __bf16 v8bf __attribute__((ext_vector_type(8)));

template <typename T>
struct LdsPad {
  // float: pitch BK+1 dwords makes the 32 rows read by one MFMA operand
  // fetch hit distinct banks; bf16: pitch BK+8 keeps 16-byte alignment for
  // the 128-bit operand reads and spreads rows over banks.
  static constexpr int value = std::is_same<T, float>::value ? 1 : 8;
};

template <typename T, int BM, int BN, int BK, int WM, int WN>
struct MfmaTile {
  static_assert(BM % (WM * 32) == 0 && BN % (WN * 32) == 0, "tile shape");
  static constexpr int TM = BM / (WM * 32);
  static constexpr int TN = BN / (WN * 32);
  static constexpr int LD = BK + LdsPad<T>::value;
  v16f acc[TM][TN];

  __device__ __forceinline__ void zero() {
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;
  }

  __device__ __forceinline__ void compute(const T* __restrict__ As, const T* __restrict__ Bs,
                                          int wm, int wn, int lane) {
    const int r = lane & 31;
    const int kh = lane >> 5;
    if constexpr (std::is_same<T, float>::value) {
#pragma unroll
      for (int kk = 0; kk < BK; kk += 2) {
        float a[TM], b[TN];
#pragma unroll
        for (int i = 0; i < TM; ++i) a[i] = As[((wm * TM + i) * 32 + r) * LD + kk + kh];
#pragma unroll
        for (int j = 0; j < TN; ++j) b[j] = Bs[((wn * TN + j) * 32 + r) * LD + kk + kh];
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
          for (int j = 0; j < TN; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(a[i], b[j], acc[i][j], 0, 0, 0);
      }
    } else {
#pragma unroll
      for (int kk = 0; kk < BK; kk += 16) {
        v8bf a[TM], b[TN];
#pragma unroll
        for (int i = 0; i < TM; ++i)
          a[i] = *reinterpret_cast<const v8bf*>(&As[((wm * TM + i) * 32 + r) * LD + kk + 8 * kh]);
#pragma unroll
        for (int j = 0; j < TN; ++j)
          b[j] = *reinterpret_cast<const v8bf*>(&Bs[((wn * TN + j) * 32 + r) * LD + kk + 8 * kh]);
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
          for (int j = 0; j < TN; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
      }
    }
  }

  // Visit every accumulator element as (row, col, value) in tile coordinates.
  template <class F>
  __device__ __forceinline__ void for_each(int wm, int wn, int lane, F&& f) const {
    const int col_l = lane & 31;
    const int row_l = 4 * (lane >> 5);
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int row = (wm * TM + i) * 32 + 8 * (r >> 2) + row_l + (r & 3);
          const int col = (wn * TN + j) * 32 + col_l;
          f(row, col, acc[i][j][r]);
        }
  }
};

}  // namespace swsft
