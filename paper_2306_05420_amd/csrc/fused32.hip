// Whole transforms of 32 x 32 float grids in one launch per direction.  At
// this size a map's spectrum (31 orders x 32 latitudes) is 8 KiB, so one
// workgroup keeps the spectra of 8 maps in LDS between the longitude DFT
// and the latitude GEMM, and the spectrum never goes through HBM (the
// five-stage path writes and reads it: 65 MB each way for the molecule-
// shaped batch).
//
//  fused32_fwd  8 maps (b, s, c0 .. c0 + 7), 64 KiB of contiguous x:
//               coalesced load into LDS -> one latitude row per thread,
//               32-point FFT in registers (the e^{-i m phi} sum of eq. (2))
//               -> X[m][j] in LDS -> per order m, the quadrature
//               coef[l^2+l+m][b][s][c] = sum_j T_s[m][l][j] X[m][j] on MFMA
//               16x16x4 f32 (T_s the plan's weighted table, read from L2).
//  fused32_inv  8 maps (b, t, c0 .. c0 + 7): per order m, the synthesis
//               Y[m][j] = sum_l T'_t[m][j][l] coef[l^2+l+m] on MFMA -> LDS
//               -> one latitude row per thread, 32-point inverse FFT in
//               registers (eq. (3)) -> one coalesced 64 KiB store of y.
//
// Operand layouts of v_mfma_f32_16x16x4f32 (one 16 x 16 block): lane l
// supplies A[l % 16][l / 16] and B[l / 16][l % 16] and receives
// D[4 (l / 16) + r][l % 16] in accumulator register r.  The contraction of
// a whole order is split over 8 (forward: 32 latitudes) or 4 (inverse: 16
// degrees) MFMAs, lane group q = l / 16 supplying latitudes 8 q + t
// (degrees 4 q + t) in MFMA t, so that each lane reads its operands as
// contiguous floats; A and B use the same assignment.
#include "fft_reg.h"
#include "swsft_internal.h"

namespace swsft {
namespace {

constexpr int kG = 32;      // grid size H = W
constexpr int kMaps = 8;    // maps per workgroup
constexpr int kRows = 256;  // (map, latitude row) pairs: one per thread in the FFTs
#ifndef SWSFT_FUSED32_NT
#define SWSFT_FUSED32_NT 512
#endif
// threads per workgroup: the FFTs use the first kRows; every wave takes
// orders in the per-order GEMMs, so more waves shorten each wave's chain of
// table (and coefficient) reads from L2 (molecule batch, 512 against 256
// threads: forward 12.9 -> 11.8 us, inverse 14.4 -> 13.3 us; 1024 threads
// would leave 64 registers per lane at two workgroups per CU and spill)
constexpr int kNT = SWSFT_FUSED32_NT;
constexpr int kWaves = kNT / 64;
constexpr int kRP = 68;     // floats per staged grid row (64 + 4: row starts 4 banks apart)
constexpr int kXP = 36;     // floats per (bin, column) row of the forward spectrum tile
constexpr int kMapStride = kG * kRP + 4;  // staged rows of one map (inverse)

typedef float v4f __attribute__((ext_vector_type(4)));

struct FSpins {
  int s[kMaxSpins];
};

__device__ __forceinline__ int fabs_i(int v) { return v < 0 ? -v : v; }

// x [B][S][C][32][32] complex -> coef [L^2][B][S][C] complex (C % 8 == 0)
__global__ void __launch_bounds__(kNT, 2 * kNT / 256)
    fused32_fwd_kernel(const float* __restrict__ x, const float* __restrict__ tab,
                       float* __restrict__ coef, int L, int B, int S, int C) {
  // staged x rows [256][kRP], then the spectrum [32 bins][16 columns][kXP]
  __shared__ __align__(16) float sm[kG * 16 * kXP];
  static_assert(kRows * kRP <= kG * 16 * kXP, "staged rows fit the spectrum tile");
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int M = 2 * L - 1;
  const int groups = C / kMaps;
  const int cg = blockIdx.x % groups, bs = blockIdx.x / groups;
  const int si = bs % S, b = bs / S;
  const size_t map0 = ((size_t)b * S + si) * C + (size_t)cg * kMaps;

  // the group's 8 maps (64 KiB, contiguous): 16-byte chunk c is row c / 16
  {
    constexpr int NU = kRows * 16 / kNT;  // 16-byte chunks per thread
    const v4f* src = reinterpret_cast<const v4f*>(x + map0 * kG * kG * 2);
    v4f buf[NU];
#pragma unroll
    for (int u = 0; u < NU; ++u) buf[u] = src[tid + kNT * u];
#pragma unroll
    for (int u = 0; u < NU; ++u) {
      const int c = tid + kNT * u;
      *reinterpret_cast<v4f*>(sm + (c >> 4) * kRP + (c & 15) * 4) = buf[u];
    }
  }
  __syncthreads();

  // thread tid < 256 = row (map = tid / 32, latitude j = tid % 32): X[k] = sum_q x[q] e^{-2 pi i q k / 32}
  float2 v[kG];
  if (tid < kRows) {
#pragma unroll
    for (int u = 0; u < 16; ++u) {
      const v4f q = *reinterpret_cast<const v4f*>(sm + tid * kRP + 4 * u);
      v[2 * u] = make_float2(q[0], q[1]);
      v[2 * u + 1] = make_float2(q[2], q[3]);
    }
    fft_reg<kG, -1>(v);
  }
  __syncthreads();  // every row is in registers before the spectrum overwrites it
  if (tid < kRows) {
    const int map = tid >> 5, j = tid & 31;
#pragma unroll
    for (int k = 0; k < kG; ++k) {
      sm[(k * 16 + 2 * map) * kXP + j] = v[k].x;
      sm[(k * 16 + 2 * map + 1) * kXP + j] = v[k].y;
    }
  }
  __syncthreads();

  // per order m (bin k = m mod 32): D[l][n] = sum_j T[m][l][j] X[k][j][n],
  // n = 2 map + re/im
  const int n = lane & 15, q = lane >> 4;
  const size_t row_stride = (size_t)S * C * 2;  // floats per coefficient row (l, m, b)
  for (int mi = wave; mi < M; mi += kWaves) {
    const int m = mi - (L - 1);
    const int k = m & (kG - 1);
    v4f a0 = {0.f, 0.f, 0.f, 0.f}, a1 = a0;
    if (n < L) {  // table row l = n; rows l >= L do not exist
      const v4f* ta = reinterpret_cast<const v4f*>(tab + (((size_t)si * M + mi) * L + n) * kG + 8 * q);
      a0 = ta[0];
      a1 = ta[1];
    }
    const v4f* xb = reinterpret_cast<const v4f*>(sm + (k * 16 + n) * kXP + 8 * q);
    const v4f b0 = xb[0], b1 = xb[1];
    v4f acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int t = 0; t < 4; ++t) acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a0[t], b0[t], acc, 0, 0, 0);
#pragma unroll
    for (int t = 0; t < 4; ++t) acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a1[t], b1[t], acc, 0, 0, 0);
    // the table is zero for l < max(|m|, |s|): those coefficients come out as 0
    const int lo = fabs_i(m);
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int l = 4 * q + r;
      if (l < L && l >= lo)
        coef[((size_t)(l * l + l + m) * B + b) * row_stride + (size_t)si * C * 2 +
             (size_t)(cg * kMaps + (n >> 1)) * 2 + (n & 1)] = acc[r];
    }
  }
}

// coef [L^2][Bc][S][C] complex (batch items 0 .. B-1 of Bc) -> y [B][S][C][32][32]
__global__ void __launch_bounds__(kNT, 2 * kNT / 256)
    fused32_inv_kernel(const float* __restrict__ coef, const float* __restrict__ tab,
                       float* __restrict__ y, int L, int Lp, int B, int Bc, int S, int C,
                       FSpins spins) {
  // spectrum rows [8 maps][32 latitudes][kRP]: (re, im) of bin k at 2 k
  __shared__ __align__(16) float sm[kMaps * kMapStride];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int M = 2 * L - 1;
  const int groups = C / kMaps;
  const int cg = blockIdx.x % groups, bs = blockIdx.x / groups;
  const int ti = bs % S, b = bs / S;
  const size_t map0 = ((size_t)b * S + ti) * C + (size_t)cg * kMaps;
  const int tabs = fabs_i(spins.s[ti]);

  // per order m: D[j][n] = sum_l T'[m][j][l] coef[l][m][n], two blocks of 16 latitudes
  const int n = lane & 15, q = lane >> 4;
  const size_t row_stride = (size_t)S * C * 2;
  for (int mi = wave; mi < M; mi += kWaves) {
    const int m = mi - (L - 1);
    const int k = m & (kG - 1);
    const int lo = fabs_i(m) > tabs ? fabs_i(m) : tabs;
    float bv[4];
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      const int l = 4 * q + t;  // rows l < max(|m|, |t|) do not exist: never read
      bv[t] = (l < L && l >= lo)
                  ? coef[((size_t)(l * l + l + m) * Bc + b) * row_stride + (size_t)ti * C * 2 +
                         (size_t)(cg * kMaps + (n >> 1)) * 2 + (n & 1)]
                  : 0.f;
    }
#pragma unroll
    for (int jb = 0; jb < 2; ++jb) {
      const v4f a = *reinterpret_cast<const v4f*>(
          tab + (((size_t)ti * M + mi) * kG + 16 * jb + n) * Lp + 4 * q);  // T'[m][j = 16 jb + n][4q ..]
      v4f acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int t = 0; t < 4; ++t) acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a[t], bv[t], acc, 0, 0, 0);
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int j = 16 * jb + 4 * q + r;
        sm[(n >> 1) * kMapStride + j * kRP + 2 * k + (n & 1)] = acc[r];
      }
    }
  }
  __syncthreads();

  // thread tid < 256 = row (map, j): bins with no order (L <= |m|) are zero;
  // y[q] = sum_k Y[k] e^{2 pi i q k / 32}
  if (tid < kRows) {
    float* row = sm + (tid >> 5) * kMapStride + (tid & 31) * kRP;
    float2 v[kG];
#pragma unroll
    for (int u = 0; u < 16; ++u) {
      const v4f w = *reinterpret_cast<const v4f*>(row + 4 * u);
      v[2 * u] = make_float2(w[0], w[1]);
      v[2 * u + 1] = make_float2(w[2], w[3]);
    }
#pragma unroll
    for (int kk = 0; kk < kG; ++kk)
      if (kk >= L && kk <= kG - L) v[kk] = make_float2(0.f, 0.f);
    fft_reg<kG, 1>(v);
#pragma unroll
    for (int u = 0; u < 16; ++u)
      *reinterpret_cast<v4f*>(row + 4 * u) = (v4f){v[2 * u].x, v[2 * u].y, v[2 * u + 1].x, v[2 * u + 1].y};
  }
  __syncthreads();

  // the group's 8 output maps (64 KiB, contiguous)
  v4f* dst = reinterpret_cast<v4f*>(y + map0 * kG * kG * 2);
#pragma unroll
  for (int u = 0; u < kRows * 16 / kNT; ++u) {
    const int c = tid + kNT * u, r = c >> 4;
    dst[c] = *reinterpret_cast<const v4f*>(sm + (r >> 5) * kMapStride + (r & 31) * kRP + (c & 15) * 4);
  }
}

}  // namespace

hipError_t launch_fused32_fwd(const Plan& p, int B, int C, const void* x, void* coef,
                              hipStream_t st) {
  const unsigned grid = (unsigned)((long long)B * p.n_in * (C / kMaps));
  hipLaunchKernelGGL(fused32_fwd_kernel, dim3(grid), dim3(kNT), 0, st, (const float*)x,
                     (const float*)p.tab_fwd, (float*)coef, p.L, B, p.n_in, C);
  return hipGetLastError();
}

hipError_t launch_fused32_inv(const Plan& p, int B, int C, const void* coef, void* y,
                              hipStream_t st) {
  FSpins so{};
  for (int i = 0; i < p.n_out; ++i) so.s[i] = p.spins_out[i];
  const unsigned grid = (unsigned)((long long)B * p.n_out * (C / kMaps));
  hipLaunchKernelGGL(fused32_inv_kernel, dim3(grid), dim3(kNT), 0, st, (const float*)coef,
                     (const float*)p.tab_inv, (float*)y, p.L, p.Lp, B,
                     p.coef_ldb > 0 ? p.coef_ldb : B, p.n_out, C, so);
  return hipGetLastError();
}

}  // namespace swsft
