// Longitude DFT as a dense matrix product on MFMA: the route the paper takes
// on TPUs (Method, "Efficient TPU implementation": DFT matrix multiplication
// instead of FFT; appendix "FFT vs DFT", Table 8), built here to compare with
// the register FFT of dft.hip on MI355X and to run grids whose width is not
// a power of two.
//
//   X[s][m][j/JT][(b,c)][re/im][j%JT] = sum_k x[b][s][c][j][k] exp(-2 pi i m k / W),  |m| < L
//
// as one real GEMM  out[r][2 mi + rho] = sum_K x[r][K] F[2 mi + rho][K]  over
// the rows r = (b, s, c, j) of x, whose interleaved (re, im) values are the K
// index as stored (K = 2k + re/im), against the expanded DFT matrix
//   F[2mi][2k] = cos t,   F[2mi][2k+1] = sin t,
//   F[2mi+1][2k] = -sin t, F[2mi+1][2k+1] = cos t,   t = 2 pi (m k mod W) / W,
// built once per plan in float64 and rounded to the storage type.  The
// quadrature weights stay folded into the latitude tables, as for the FFT.
#include "gemm_tile.h"
#include "mfma_tile.h"
#include "swsft_internal.h"
#include "xcd.h"

namespace swsft {
namespace {

template <typename T>
__global__ void dft_matrix_kernel(T* __restrict__ F, int W, int L) {
  const int K = blockIdx.x * blockDim.x + threadIdx.x;  // column: 2k + rho_in
  const int q = blockIdx.y;                              // row: 2 mi + rho_out
  if (K >= 2 * W) return;
  const int k = K >> 1, ri = K & 1, mi = q >> 1, ro = q & 1;
  const long long m = mi - (L - 1);
  const long long r = ((m * k) % W + W) % W;
  const double t = 2.0 * 3.14159265358979323846 * (double)r / (double)W;
  const double c = cos(t), s = sin(t);
  const double v = ro == 0 ? (ri == 0 ? c : s) : (ri == 0 ? -s : c);
  F[(size_t)q * 2 * W + K] = (T)(float)v;
}

template <typename T, int BM, int BN, int BK, int WM, int WN, bool kVec>
__global__ void __launch_bounds__(NT) dft_mm_kernel(const T* __restrict__ x, const T* __restrict__ F,
                                                    T* __restrict__ X, int rows, int W, int H,
                                                    int JT, int M, int S, int C, int BC,
                                                    int n_tiles_n) {
  using Tile = MfmaTile<T, BM, BN, BK, WM, WN>;
  using G = GemmLds<T, BM, BN, BK>;
  __shared__ __align__(16) T smem[G::bytes / sizeof(T)];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WN, wn = wave % WN;
  const int n_rows_t = (rows + BM - 1) / BM;
  // logical block = (row tile, column tile): the column tiles of one row tile
  // read the same rows of x and run next to each other on one XCD
  const int lbk = xcd_logical_block();
  if (lbk >= n_rows_t * n_tiles_n) return;
  const int nt = lbk % n_tiles_n, rt = lbk / n_tiles_n;
  const int r0 = rt * BM, q0 = nt * BN;
  const int K = 2 * W, N = 2 * M;
  RowLoader<T, BM, BK, kVec> la;
  RowLoader<T, BN, BK, kVec> lb;
  la.init([&](int r) -> const T* { return r0 + r < rows ? x + (size_t)(r0 + r) * K : nullptr; },
          x + (size_t)r0 * K, 0, K, tid);
  lb.init([&](int r) -> const T* { return q0 + r < N ? F + (size_t)(q0 + r) * K : nullptr; },
          F + (size_t)q0 * K, 0, K, tid);
  Tile tile;
  tile.zero();
  mainloop(tile, la, lb, smem, (K + BK - 1) / BK, wm, wn, lane);

  // epilogue: tile -> LDS [BM][LDC], then runs of VEC consecutive latitudes
  // of one column, written to the K-tiled spectrum
  tile.for_each(wm, wn, lane, [&](int row, int col, float v) { smem[row * G::LDC + col] = (T)v; });
  __syncthreads();
  constexpr int VEC = 16 / sizeof(T);
  constexpr int RUNS = BM / VEC;
  const int HT = H / JT;
  for (int idx = tid; idx < BN * RUNS; idx += NT) {
    const int col = idx / RUNS, row = (idx % RUNS) * VEC;
    const int q = q0 + col, r = r0 + row;
    if (q >= N || r >= rows) continue;
    const int mi = q >> 1, rho = q & 1;
    const int map = r / H, j = r - map * H;  // map = (b * S + s) * C + c
    const int c = map % C, bs = map / C, s = bs % S, b = bs / S;
    const size_t base = ((((size_t)s * M + mi) * HT + j / JT) * BC + (size_t)b * C + c) * 2 + rho;
    if (kVec && JT % VEC == 0 && r + VEC <= rows) {
      // the run stays in one latitude tile of one map (H and JT multiples of VEC)
      Vec16<T> v;
#pragma unroll
      for (int e = 0; e < VEC; ++e) v.e[e] = smem[(row + e) * G::LDC + col];
      *reinterpret_cast<uint4*>(&X[base * JT + j % JT]) = v.u;
    } else {
      for (int e = 0; e < VEC && r + e < rows; ++e) {
        const int re = r + e, me = re / H, je = re - me * H;
        const int ce = me % C, bse = me / C, se = bse % S, be = bse / S;
        const size_t o = ((((size_t)se * M + mi) * HT + je / JT) * BC + (size_t)be * C + ce) * 2 + rho;
        X[o * JT + je % JT] = smem[(row + e) * G::LDC + col];
      }
    }
  }
}

template <typename T>
hipError_t dft_mm_t(const Plan& p, int S, int B, int C, const void* x, void* X, hipStream_t st) {
  constexpr int BM = 128, BN = 128, BK = 32;
  const int rows = B * S * C * p.H;
  const int N = 2 * p.M;
  const int n_tiles_n = (N + BN - 1) / BN;
  const long long blocks = (long long)((rows + BM - 1) / BM) * n_tiles_n;
  constexpr int VEC = 16 / sizeof(T);
  const bool vec = (2 * p.W) % VEC == 0 && p.H % VEC == 0;
  auto kern = vec ? dft_mm_kernel<T, BM, BN, BK, 2, 2, true> : dft_mm_kernel<T, BM, BN, BK, 2, 2, false>;
  hipLaunchKernelGGL(kern, dim3(xcd_grid(blocks)), dim3(NT), 0, st, (const T*)x,
                     (const T*)p.dft_mat, (T*)X, rows, p.W, p.H, p.JT, p.M, S, C, B * C, n_tiles_n);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_dft_matrix(const Plan& p, hipStream_t st) {
  dim3 grid((2 * p.W + 255) / 256, 2 * p.M);
  if (p.dtype == SWSFT_BF16)
    hipLaunchKernelGGL(dft_matrix_kernel<__bf16>, grid, dim3(256), 0, st, (__bf16*)p.dft_mat, p.W, p.L);
  else
    hipLaunchKernelGGL(dft_matrix_kernel<float>, grid, dim3(256), 0, st, (float*)p.dft_mat, p.W, p.L);
  return hipGetLastError();
}

hipError_t launch_dft_fwd_matmul(const Plan& p, int S, int B, int C, const void* x, void* X,
                                 hipStream_t st) {
  if (p.dtype == SWSFT_BF16) return dft_mm_t<__bf16>(p, S, B, C, x, X, st);
  return dft_mm_t<float>(p, S, B, C, x, X, st);
}

}  // namespace swsft
