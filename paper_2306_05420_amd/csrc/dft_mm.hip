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

// The inverse longitude stage as a matrix product:
//   y[b][s][c][j][k] = sum_{|m| < L} Y[s][m][j/JT][(b,c)][re/im][j%JT] exp(+2 pi i m k / W)
// as one real GEMM  out[r][2k + rho] = sum_q Yrow[r][q] G[2k + rho][q]  over
// the rows r = (b, s, c, j) of y, with q = 2 mi + re/im the spectrum's value
// of order mi, and the expanded inverse DFT matrix
//   G[2k][2mi] = cos t,   G[2k][2mi+1] = -sin t,
//   G[2k+1][2mi] = sin t, G[2k+1][2mi+1] = cos t,   t = 2 pi (m k mod W) / W.
// In the K-tiled spectrum the rows of one order run along j (32 consecutive
// latitudes of one map are contiguous), so the A operand is staged in LDS
// K-major, [q][r], and its MFMA fragments are gathered along q.
// Rows of G are padded with zeros to dft_inv_pitch(M) values, so that every
// row starts 16-byte aligned and is read as whole vectors.
template <typename T>
__global__ void dft_matrix_inv_kernel(T* __restrict__ G, int W, int L) {
  const int q = blockIdx.x * blockDim.x + threadIdx.x;  // column: 2 mi + rho_in
  const int K = blockIdx.y;                              // row: 2k + rho_out
  const int M = 2 * L - 1;
  const int pitch = dft_inv_pitch(M);
  if (q >= pitch) return;
  double v = 0.0;
  if (q < 2 * M) {
    const int k = K >> 1, ro = K & 1, mi = q >> 1, ri = q & 1;
    const long long m = mi - (L - 1);
    const long long r = ((m * k) % W + W) % W;
    const double t = 2.0 * 3.14159265358979323846 * (double)r / (double)W;
    const double c = cos(t), s = sin(t);
    v = ro == 0 ? (ri == 0 ? c : -s) : (ri == 0 ? s : c);
  }
  G[(size_t)K * pitch + q] = (T)(float)v;
}

// A operand tile [BK][BM + PAD] (K-major) of the spectrum rows r0 .. r0+BM-1
// and values q = kt BK .. kt BK + BK - 1; VEC consecutive rows are one vector
// load when kVec (a run of VEC latitudes never leaves one latitude tile of
// one map).  Out-of-range rows and values are zero.
template <typename T, int BM, int BK, bool kVec>
struct SpecLoader {
  static constexpr int VEC = kVec ? 16 / sizeof(T) : 1;
  static constexpr int PAD = sizeof(T) == 4 ? 1 : 2;
  static constexpr int LDA = BM + PAD;
  static constexpr int VPK = BM / VEC;  // vectors per value q
  static constexpr int NV = BK * VPK;
  static constexpr int PER = (NV + NT - 1) / NT;
  T reg[PER][VEC];
  size_t rbase[PER];  // spectrum offset of the vector's first row at q = 0 (order 0, re)
  bool rok[PER];
  int kq[PER], rr[PER];
  int K;
  size_t mstride;     // elements between consecutive orders

  __device__ __forceinline__ void init(int r0, int rows, int H, int JT, int M, int S, int C,
                                       int BC, int K_, int tid) {
    K = K_;
    const int HT = H / JT;
    mstride = (size_t)HT * BC * 2 * JT;
#pragma unroll
    for (int p = 0; p < PER; ++p) {
      const int v = tid + p * NT;
      kq[p] = v / VPK;
      rr[p] = (v % VPK) * VEC;
      const int r = r0 + rr[p];
      rok[p] = (NV % NT == 0 || v < NV) && r < rows;
      const int rc = rok[p] ? r : 0;
      const int map = rc / H, j = rc - map * H;
      const int c = map % C, bs = map / C, s = bs % S, b = bs / S;
      rbase[p] = ((((size_t)s * M) * HT + j / JT) * BC + (size_t)b * C + c) * 2 * JT + j % JT;
    }
  }
  __device__ __forceinline__ void load(const T* __restrict__ Y, int kt, int rows, int r0, int H,
                                       int JT, int BC) {
#pragma unroll
    for (int p = 0; p < PER; ++p) {
      const int q = kt * BK + kq[p];
      const bool ok = rok[p] && q < K;
      const size_t off = ok ? rbase[p] + (size_t)(q >> 1) * mstride + (size_t)(q & 1) * JT : 0;
      if constexpr (kVec) {
        Vec16<T> v;
        v.u = *reinterpret_cast<const uint4*>(Y + off);
#pragma unroll
        for (int e = 0; e < VEC; ++e) reg[p][e] = ok ? v.e[e] : (T)0.f;
      } else {
        const T v = Y[off];
        reg[p][0] = ok ? v : (T)0.f;
      }
    }
  }
  __device__ __forceinline__ void store(T* lds) {
    const int tid = threadIdx.x;
#pragma unroll
    for (int p = 0; p < PER; ++p) {
      const int v = tid + p * NT;
      if (NV % NT != 0 && v >= NV) break;
#pragma unroll
      for (int e = 0; e < VEC; ++e) lds[kq[p] * LDA + rr[p] + e] = reg[p][e];
    }
  }
};

// MFMA tile whose A operand is K-major in LDS ([k][row], pitch LDA).
template <typename T, int BM, int BN, int BK, int WM, int WN, int LDA>
struct KMajorATile : MfmaTile<T, BM, BN, BK, WM, WN> {
  using Base = MfmaTile<T, BM, BN, BK, WM, WN>;
  using Base::acc;
  static constexpr int TM = Base::TM, TN = Base::TN, LD = Base::LD;
  __device__ __forceinline__ void compute(const T* __restrict__ As, const T* __restrict__ Bs,
                                          int wm, int wn, int lane) {
    const int r = lane & 31, kh = lane >> 5;
    if constexpr (std::is_same<T, float>::value) {
#pragma unroll
      for (int kk = 0; kk < BK; kk += 2) {
        float a[TM], b[TN];
#pragma unroll
        for (int i = 0; i < TM; ++i) a[i] = As[(kk + kh) * LDA + (wm * TM + i) * 32 + r];
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
#pragma unroll
          for (int e = 0; e < 8; ++e) a[i][e] = As[(kk + 8 * kh + e) * LDA + (wm * TM + i) * 32 + r];
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
};

// The double-buffered main loop of gemm_tile.h for a tile type with its own
// compute (the A region of a stage holds the K-major tile).
template <int BM, int BN, int BK, class Tile, class LA, class LB, typename T>
__device__ __forceinline__ void kmajor_mainloop(Tile& tile, LA& la, LB& lb, T* smem, int nk,
                                                int wm, int wn, int lane) {
  constexpr int LD = BK + LdsPad<T>::value;
  constexpr int kStage = (BM + BN) * LD;
  la.load(0);
  lb.load(0);
  la.store(smem);
  lb.store(smem + BM * LD);
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
      lb.store(nxt + BM * LD);
      if (kt + 2 < nk) {
        la.load(kt + 2);
        lb.load(kt + 2);
      }
    }
    tile.compute(cur, cur + BM * LD, wm, wn, lane);
    __syncthreads();
  }
}

template <typename T, int BM, int BN, int BK, int WM, int WN, bool kVec>
__global__ void __launch_bounds__(NT) dft_mm_inv_kernel(const T* __restrict__ Y,
                                                        const T* __restrict__ G,
                                                        T* __restrict__ y, int rows, int W, int H,
                                                        int JT, int M, int S, int C, int BC,
                                                        int n_tiles_n) {
  using LA = SpecLoader<T, BM, BK, kVec>;
  using Tile = KMajorATile<T, BM, BN, BK, WM, WN, LA::LDA>;
  using GL = GemmLds<T, BM, BN, BK>;
  static_assert(BK * LA::LDA <= BM * GL::LD, "K-major A tile fits the A region of a stage");
  __shared__ __align__(16) T smem[GL::bytes / sizeof(T)];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WN, wn = wave % WN;
  const int n_rows_t = (rows + BM - 1) / BM;
  // logical block = (row tile, column tile): the column tiles of one row tile
  // read the same spectrum values and run next to each other on one XCD
  const int lbk = xcd_logical_block();
  if (lbk >= n_rows_t * n_tiles_n) return;
  const int nt = lbk % n_tiles_n, rt = lbk / n_tiles_n;
  const int r0 = rt * BM, q0 = nt * BN;
  const int K = 2 * M, N = 2 * W;
  LA la;
  la.init(r0, rows, H, JT, M, S, C, BC, K, tid);
  // the A loader needs the spectrum pointer and geometry at each load
  struct ALoad {
    LA& la;
    const T* Y;
    int rows, r0, H, JT, BC;
    __device__ __forceinline__ void load(int kt) { la.load(Y, kt, rows, r0, H, JT, BC); }
    __device__ __forceinline__ void store(T* lds) { la.store(lds); }
  } al{la, Y, rows, r0, H, JT, BC};
  Tile tile;
  tile.zero();
  constexpr int VEC = 16 / sizeof(T);
  const int pitch = dft_inv_pitch(M);  // a multiple of VEC: whole 16-byte row reads
  RowLoader<T, BN, BK, true> lg;
  lg.init([&](int r) -> const T* { return q0 + r < N ? G + (size_t)(q0 + r) * pitch : nullptr; },
          G + (size_t)q0 * pitch, 0, K, tid);
  kmajor_mainloop<BM, BN, BK>(tile, al, lg, smem, (K + BK - 1) / BK, wm, wn, lane);
  // epilogue: rows r of y, columns 2k + rho contiguous
  epilogue(tile, smem, rows - r0, N - q0, wm, wn, lane, tid,
           [&](int row, int col, const Vec16<T>& v, int n) {
             T* dst = y + (size_t)(r0 + row) * N + q0 + col;
             if (n == VEC && (N % VEC) == 0) {
               *reinterpret_cast<uint4*>(dst) = v.u;
             } else {
               for (int e = 0; e < n; ++e) dst[e] = v.e[e];
             }
           });
}

template <typename T>
hipError_t dft_mm_inv_t(const Plan& p, int S, int B, int C, const void* Y, void* y,
                        hipStream_t st) {
  constexpr int BM = 128, BN = 128, BK = 32;
  const int rows = B * S * C * p.H;
  const int N = 2 * p.W;
  const int n_tiles_n = (N + BN - 1) / BN;
  const long long blocks = (long long)((rows + BM - 1) / BM) * n_tiles_n;
  constexpr int VEC = 16 / sizeof(T);
  const bool vec = p.JT % VEC == 0 && p.H % VEC == 0;
  auto kern = vec ? dft_mm_inv_kernel<T, BM, BN, BK, 2, 2, true>
                  : dft_mm_inv_kernel<T, BM, BN, BK, 2, 2, false>;
  hipLaunchKernelGGL(kern, dim3(xcd_grid(blocks)), dim3(NT), 0, st, (const T*)Y,
                     (const T*)p.dft_mat_inv, (T*)y, rows, p.W, p.H, p.JT, p.M, S, C, B * C,
                     n_tiles_n);
  return hipGetLastError();
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

hipError_t launch_dft_matrix_inv(const Plan& p, hipStream_t st) {
  dim3 grid((dft_inv_pitch(p.M) + 255) / 256, 2 * p.W);
  if (p.dtype == SWSFT_BF16)
    hipLaunchKernelGGL(dft_matrix_inv_kernel<__bf16>, grid, dim3(256), 0, st,
                       (__bf16*)p.dft_mat_inv, p.W, p.L);
  else
    hipLaunchKernelGGL(dft_matrix_inv_kernel<float>, grid, dim3(256), 0, st,
                       (float*)p.dft_mat_inv, p.W, p.L);
  return hipGetLastError();
}

hipError_t launch_dft_inv_matmul(const Plan& p, int S, int B, int C, const void* Y, void* y,
                                 hipStream_t st) {
  if (p.dtype == SWSFT_BF16) return dft_mm_inv_t<__bf16>(p, S, B, C, Y, y, st);
  return dft_mm_inv_t<float>(p, S, B, C, Y, y, st);
}

hipError_t launch_dft_fwd_matmul(const Plan& p, int S, int B, int C, const void* x, void* X,
                                 hipStream_t st) {
  if (p.dtype == SWSFT_BF16) return dft_mm_t<__bf16>(p, S, B, C, x, X, st);
  return dft_mm_t<float>(p, S, B, C, x, X, st);
}

}  // namespace swsft
