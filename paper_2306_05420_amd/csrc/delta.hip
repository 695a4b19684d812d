// The transforms by the paper's Wigner-Delta route (Background, eqs. (4)-(6)),
// with the J / G symmetries (eq. (5) and the G relation after eq. (6)) or
// without them, as chains of real MFMA GEMMs:
//
//  forward  X_m(theta_j) (longitude DFT)
//           -> theta GEMM: C_{m'} = sum_j q_j cos(m' theta_j) X_j,  S_{m'} = sum_j q_j sin(m' theta_j) X_j
//              (I_{m'} = C - iS, I_{-m'} = C + iS: the quadrature of the paper's I on the grid)
//           -> Delta GEMM: a_l = sum_{m'} P[l][m'] (C or S rows)       (the latitude kernels)
//  inverse  a_l -> Delta GEMM: G_{m'} = sum_l P[m'][l] a_l             (the latitude kernels)
//           -> theta GEMM: Y_j = sum_{m'} (cos, sin)(m' theta_j) G_{m'}  -> longitude DFT
//
// With the symmetries the product Delta^l_{m'm} Delta^l_{m'(-s)} is even or
// odd in m' by the parity of m + s, so only m' >= 0 enters and, per (s, m),
// only the cos or only the sin factor: one real table of L rows (forward) and
// every phase (-1)^s i^(m+s) is a real sign folded into the Delta tables.
// Without them all 2L - 1 values of m' are summed: the forward theta GEMM
// makes both C and S (2L rows) and multiplies one half by -i in its epilogue;
// the inverse theta GEMM makes cos and sin rows for every m' and combines
// them as Y = phase (Z_cos + i Z_sin).
//
// Intermediates (C/S, G) are K-tiled like the longitude spectra:
// [S][2L-1][R/32][n'][32], n' = (b, c, re/im), so the latitude kernels read
// them as their K operand.
#include "gemm_tile.h"
#include "mfma_tile.h"
#include "swsft_internal.h"
#include "wigner.h"
#include "xcd.h"

namespace swsft {
namespace {

constexpr double kPi = 3.14159265358979323846;

__device__ double dh_quadrature(int j, int H, int W) {
  // (2 pi / W) w_j, w_j the Driscoll--Healy weight of the offset grid
  const double theta = kPi * (2.0 * j + 1.0) / (2.0 * H);
  double acc = 0.0;
  for (int p = 0; p < H / 2; ++p) acc += sin((2.0 * p + 1.0) * theta) / (2.0 * p + 1.0);
  return (2.0 * kPi / W) * (4.0 / H) * sin(theta) * acc;
}

// theta tables (see the file comment); layouts:
//  fwd sym  [2 parities][L][H]: even w_{m'} q_j cos, odd 2 q_j sin    (w_0 = 1, else 2)
//  fwd full [2L][H]:            rows m' q_j cos, rows L + m' q_j sin
//  inv sym  [2][H][L]:          even w_{m'} cos, odd 2 sin
//  inv full [2H][2L]:           row 2j cos(m' theta_j), row 2j+1 sin, column m' + L - 1
template <typename T>
__global__ void theta_table_kernel(T* __restrict__ E, int variant, int H, int W, int L) {
  const int col = blockIdx.x * blockDim.x + threadIdx.x;
  const int row = blockIdx.y;
  const int z = blockIdx.z;  // parity for the symmetric tables
  double v = 0.0;
  if (variant == 0) {  // fwd sym: row m', col j
    if (col >= H) return;
    const double th = kPi * (2.0 * col + 1.0) / (2.0 * H), q = dh_quadrature(col, H, W);
    v = z == 0 ? (row == 0 ? 1.0 : 2.0) * q * cos(row * th) : 2.0 * q * sin(row * th);
    E[((size_t)z * L + row) * H + col] = (T)(float)v;
  } else if (variant == 1) {  // fwd full: row r in [0, 2L), col j
    if (col >= H) return;
    const double th = kPi * (2.0 * col + 1.0) / (2.0 * H), q = dh_quadrature(col, H, W);
    const int mp = row < L ? row : row - L;
    v = row < L ? q * cos(mp * th) : q * sin(mp * th);
    E[(size_t)row * H + col] = (T)(float)v;
  } else if (variant == 2) {  // inv sym: row j, col m'
    if (col >= L) return;
    const double th = kPi * (2.0 * row + 1.0) / (2.0 * H);
    v = z == 0 ? (col == 0 ? 1.0 : 2.0) * cos(col * th) : 2.0 * sin(col * th);
    E[((size_t)z * H + row) * L + col] = (T)(float)v;
  } else {  // inv full: row 2j + cos/sin, col m' + L - 1
    if (col >= 2 * L) return;
    const int j = row >> 1;
    const double th = kPi * (2.0 * j + 1.0) / (2.0 * H);
    const int mp = col - (L - 1);
    if (col < 2 * L - 1) v = (row & 1) ? sin(mp * th) : cos(mp * th);
    E[(size_t)row * 2 * L + col] = (T)(float)v;
  }
}

// (-1)^s i^(m+s) = sgn * i^odd
__device__ void phase_of(int m, int s, int& odd, double& sgn) {
  const int e = (((m + s) % 4) + 4) % 4;
  odd = e & 1;
  sgn = ((s & 1) ? -1.0 : 1.0) * ((e == 2 || e == 3) ? -1.0 : 1.0);
}

// Delta tables: one thread per (spin, m, m' >= 0) runs the recurrences of
// d^l_{+-m', m}(pi/2) and d^l_{+-m', -s}(pi/2) together over l and writes
// D+ = Delta_{m'm} Delta_{m'(-s)}, D- = Delta_{-m'm} Delta_{-m'(-s)} combinations:
//  variant 0 fwd sym  [S][M][L][L]    (row l, col m'):   sigma N_l D+
//  variant 1 fwd full [S][M][L][2L]   col m': sC N_l (D+ + D-), col L + m': sS N_l (D+ - D-)
//  variant 2 inv sym  [S][M][L][Lp]   (row m', col l):   sigma' N_l D-
//  variant 3 inv full [S][M][2L][Lp]  row m' + L - 1: N_l D-, row L - 1 - m': N_l D+
// (m' = 0 counted once; the signs as derived in the file comment)
template <typename T>
__global__ void delta_table_kernel(T* __restrict__ P, int variant, int s, int si, int L, int Lp) {
  const int mp = blockIdx.x * blockDim.x + threadIdx.x;
  const int mi = blockIdx.y;
  if (mp >= L) return;
  const int M = 2 * L - 1;
  const int m = mi - (L - 1);
  int odd;
  double sgn;
  phase_of(m, s, odd, sgn);
  WignerRec ap, bp, am, bm;
  ap.init(mp, m, 0.5 * kPi);
  bp.init(mp, -s, 0.5 * kPi);
  am.init(-mp, m, 0.5 * kPi);
  bm.init(-mp, -s, 0.5 * kPi);
  const size_t base = (size_t)si * M + mi;
  for (int l = 0; l < L; ++l) {
    const double Nl = sqrt((2.0 * l + 1.0) / (4.0 * kPi));
    const double Dp = ap.at(l) * bp.at(l), Dm = am.at(l) * bm.at(l);
    double v0 = 0.0, v1 = 0.0;
    switch (variant) {
      case 0:  // even: sigma = sgn; odd: J = -2i S folds to sgn (see above)
        P[(base * L + l) * L + mp] = (T)(float)(sgn * Nl * Dp);
        break;
      case 1:
        v0 = mp == 0 ? Dp : Dp + Dm;
        v1 = mp == 0 ? 0.0 : Dp - Dm;
        // even: C as is, S rotated by -i: (sgn, sgn); odd: C rotated: (-sgn, sgn)
        P[(base * L + l) * 2 * L + mp] = (T)(float)((odd ? -sgn : sgn) * Nl * v0);
        P[(base * L + l) * 2 * L + L + mp] = (T)(float)(sgn * Nl * v1);
        break;
      case 2:  // even: sgn; odd: -sgn (Y = sum 2 sin (i sgn i) ...)
        P[(base * L + mp) * Lp + l] = (T)(float)((odd ? -sgn : sgn) * Nl * Dm);
        break;
      default:
        P[(base * 2 * L + (L - 1 + mp)) * Lp + l] = (T)(float)(Nl * Dm);
        if (mp > 0) P[(base * 2 * L + (L - 1 - mp)) * Lp + l] = (T)(float)(Nl * Dp);
        break;
    }
    ap.advance_past(l);
    bp.advance_past(l);
    am.advance_past(l);
    bm.advance_past(l);
  }
}

// theta GEMM: per (spin, m): out[R_A][n'] = A[R_A][Kd] . In[Kd][n'] with the
// input and the output K-tiled ([K/32][N][32]); A is the table of the block's
// parity (tab_stride apart) or shared.  mode 0: plain; mode 1: rows
// [rot_lo, rot_lo + rot_n) of parity-0 blocks and [rot_lo1, ...) of parity-1
// blocks multiplied by -i; mode 2: output row r = phase (Z_{2r} + i Z_{2r+1}).
struct ThetaArgs {
  int L, Kd, RA, N, S, mode, rot0, rot1, rot_n;
  size_t tab_stride;
  int spins[kMaxSpins];
};

template <typename T, int BM, int BN, int BK, int WM, int WN, bool kVec>
__global__ void __launch_bounds__(NT) theta_gemm_kernel(const T* __restrict__ A0,
                                                        const T* __restrict__ in,
                                                        T* __restrict__ out, ThetaArgs a,
                                                        int n_row_t, int n_col_t) {
  using Tile = MfmaTile<T, BM, BN, BK, WM, WN>;
  using G = GemmLds<T, BM, BN, BK>;
  __shared__ __align__(16) T smem[G::bytes / sizeof(T)];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WN, wn = wave % WN;
  const int M = 2 * a.L - 1;
  int lbk = xcd_logical_block();
  if (lbk >= a.S * M * n_row_t * n_col_t) return;
  const int ct = lbk % n_col_t;
  lbk /= n_col_t;
  const int rt = lbk % n_row_t;
  lbk /= n_row_t;
  const int mi = mixed_order(lbk % M, a.L), si = lbk / M;
  const int m = mi - (a.L - 1), s = a.spins[si];
  int odd;
  double sgn;
  phase_of(m, s, odd, sgn);
  const T* A = A0 + (a.mode == 0 ? (size_t)odd * a.tab_stride : 0);
  const int RO = a.mode == 2 ? a.RA / 2 : a.RA;  // output rows
  const T* Bin = in + ((size_t)si * M + mi) * a.N * a.Kd;
  T* O = out + ((size_t)si * M + mi) * a.N * RO;
  const int r0 = rt * BM, n0 = ct * BN;
  RowLoader<T, BM, BK, kVec> la;
  RowLoader<T, BN, BK, kVec> lb;
  la.init([&](int r) -> const T* { return r0 + r < a.RA ? A + (size_t)(r0 + r) * a.Kd : nullptr; },
          A + (size_t)r0 * a.Kd, 0, a.Kd, tid);
  lb.init([&](int r) -> const T* { return n0 + r < a.N ? Bin + (size_t)(n0 + r) * 32 : nullptr; },
          Bin + (size_t)n0 * 32, 0, a.Kd, tid, (size_t)a.N * 32);
  Tile tile;
  tile.zero();
  mainloop(tile, la, lb, smem, (a.Kd + BK - 1) / BK, wm, wn, lane);
  tile.for_each(wm, wn, lane, [&](int row, int col, float v) { smem[row * G::LDC + col] = (T)v; });
  __syncthreads();
  // runs of 4 consecutive output rows of one column; rows and columns of the
  // tile are even-aligned, so a column's re/im partner and a row's cos/sin
  // partner are in the tile
  constexpr int RUN = 4;
  const int rows_here = a.mode == 2 ? BM / 2 : BM;
  const int ro0 = a.mode == 2 ? r0 / 2 : r0;
  const int rot_lo = odd ? a.rot1 : a.rot0;
  for (int idx = tid; idx < BN * (rows_here / RUN); idx += NT) {
    const int col = idx / (rows_here / RUN), rr = (idx % (rows_here / RUN)) * RUN;
    const int n = n0 + col;
    if (n >= a.N) continue;
    const int re = col & ~1, im = col | 1, is_im = col & 1;
    for (int e = 0; e < RUN; ++e) {
      const int ro = ro0 + rr + e;
      if (ro >= RO) break;
      float v;
      if (a.mode == 2) {
        const int t = rr + e;  // local output row: tile rows 2t (cos) and 2t+1 (sin)
        const float zr = (float)smem[(2 * t) * G::LDC + re] - (float)smem[(2 * t + 1) * G::LDC + im];
        const float zi = (float)smem[(2 * t) * G::LDC + im] + (float)smem[(2 * t + 1) * G::LDC + re];
        // times sgn * i^odd
        const float pr = odd ? -zi : zr, pi = odd ? zr : zi;
        v = (float)sgn * (is_im ? pi : pr);
      } else {
        const int t = rr + e;
        if (a.mode == 1 && ro >= rot_lo && ro < rot_lo + a.rot_n) {
          // times -i: (re, im) -> (im, -re)
          v = is_im ? -(float)smem[t * G::LDC + re] : (float)smem[t * G::LDC + im];
        } else {
          v = (float)smem[t * G::LDC + col];
        }
      }
      O[((size_t)(ro / 32) * a.N + n) * 32 + ro % 32] = (T)v;
    }
  }
}

template <typename T>
hipError_t theta_t(const T* A, const void* in, void* out, const ThetaArgs& a, hipStream_t st) {
  constexpr int BM = 128, BN = 128, BK = 32;
  const int n_row_t = (a.RA + BM - 1) / BM, n_col_t = (a.N + BN - 1) / BN;
  const long long blocks = (long long)a.S * (2 * a.L - 1) * n_row_t * n_col_t;
  constexpr int VEC = 16 / sizeof(T);
  auto kern = a.Kd % VEC == 0 ? theta_gemm_kernel<T, BM, BN, BK, 2, 2, true>
                              : theta_gemm_kernel<T, BM, BN, BK, 2, 2, false>;
  hipLaunchKernelGGL(kern, dim3(xcd_grid(blocks)), dim3(NT), 0, st, A, (const T*)in, (T*)out, a,
                     n_row_t, n_col_t);
  return hipGetLastError();
}

template <typename T>
hipError_t delta_tables_t(const Plan& p, hipStream_t st) {
  const int L = p.L, H = p.H, W = p.W, M = p.M;
  const bool sym = (p.flags & SWSFT_PLAN_DELTA_SYM) != 0;
  // theta tables
  if (sym) {
    hipLaunchKernelGGL(theta_table_kernel<T>, dim3((H + 63) / 64, L, 2), dim3(64), 0, st,
                       (T*)p.delta_theta_fwd, 0, H, W, L);
    hipLaunchKernelGGL(theta_table_kernel<T>, dim3((L + 63) / 64, H, 2), dim3(64), 0, st,
                       (T*)p.delta_theta_inv, 2, H, W, L);
  } else {
    hipLaunchKernelGGL(theta_table_kernel<T>, dim3((H + 63) / 64, 2 * L, 1), dim3(64), 0, st,
                       (T*)p.delta_theta_fwd, 1, H, W, L);
    hipLaunchKernelGGL(theta_table_kernel<T>, dim3((2 * L + 63) / 64, 2 * H, 1), dim3(64), 0, st,
                       (T*)p.delta_theta_inv, 3, H, W, L);
  }
  // Delta tables
  for (int si = 0; si < p.n_in; ++si)
    hipLaunchKernelGGL(delta_table_kernel<T>, dim3((L + 63) / 64, M), dim3(64), 0, st,
                       (T*)p.delta_fwd, sym ? 0 : 1, p.spins_in[si], si, L, p.Lp);
  for (int si = 0; si < p.n_out; ++si)
    hipLaunchKernelGGL(delta_table_kernel<T>, dim3((L + 63) / 64, M), dim3(64), 0, st,
                       (T*)p.delta_inv, sym ? 2 : 3, p.spins_out[si], si, L, p.Lp);
  return hipGetLastError();
}

}  // namespace

int delta_rows(const Plan& p) { return (p.flags & SWSFT_PLAN_DELTA_SYM) ? p.L : 2 * p.L; }

size_t delta_fwd_theta_elems(const Plan& p) { return (size_t)2 * p.L * p.H; }
size_t delta_inv_theta_elems(const Plan& p) {
  return (p.flags & SWSFT_PLAN_DELTA_SYM) ? (size_t)2 * p.H * p.L : (size_t)2 * p.H * 2 * p.L;
}
size_t delta_fwd_table_elems(const Plan& p) { return (size_t)p.M * p.L * delta_rows(p); }
size_t delta_inv_table_elems(const Plan& p) { return (size_t)p.M * delta_rows(p) * p.Lp; }

hipError_t launch_delta_tables(const Plan& p, hipStream_t st) {
  if (p.dtype == SWSFT_BF16) return delta_tables_t<__bf16>(p, st);
  return delta_tables_t<float>(p, st);
}

// forward theta GEMM: X (K-tiled over j) -> C/S (K-tiled over the R rows)
hipError_t launch_delta_theta_fwd(const Plan& p, int B, int C, const void* X, void* CS,
                                  hipStream_t st) {
  const bool sym = (p.flags & SWSFT_PLAN_DELTA_SYM) != 0;
  ThetaArgs a{};
  a.L = p.L;
  a.Kd = p.H;
  a.RA = delta_rows(p);
  a.N = 2 * B * C;
  a.S = p.n_in;
  a.mode = sym ? 0 : 1;
  a.rot0 = p.L;  // even parity: S rows times -i
  a.rot1 = 0;    // odd parity: C rows times -i
  a.rot_n = p.L;
  a.tab_stride = (size_t)p.L * p.H;
  for (int i = 0; i < p.n_in; ++i) a.spins[i] = p.spins_in[i];
  if (p.dtype == SWSFT_BF16) return theta_t<__bf16>((const __bf16*)p.delta_theta_fwd, X, CS, a, st);
  return theta_t<float>((const float*)p.delta_theta_fwd, X, CS, a, st);
}

// inverse theta GEMM: G (K-tiled over m') -> Y (K-tiled over j)
hipError_t launch_delta_theta_inv(const Plan& p, int B, int C, const void* G, void* Y,
                                  hipStream_t st) {
  const bool sym = (p.flags & SWSFT_PLAN_DELTA_SYM) != 0;
  ThetaArgs a{};
  a.L = p.L;
  a.Kd = delta_rows(p);
  a.RA = sym ? p.H : 2 * p.H;
  a.N = 2 * B * C;
  a.S = p.n_out;
  a.mode = sym ? 0 : 2;
  a.tab_stride = (size_t)p.H * p.L;
  for (int i = 0; i < p.n_out; ++i) a.spins[i] = p.spins_out[i];
  if (p.dtype == SWSFT_BF16) return theta_t<__bf16>((const __bf16*)p.delta_theta_inv, G, Y, a, st);
  return theta_t<float>((const float*)p.delta_theta_inv, G, Y, a, st);
}

}  // namespace swsft
