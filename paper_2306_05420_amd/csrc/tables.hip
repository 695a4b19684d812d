// Plan-time tables: Wigner-d / spin-weighted Legendre tables in float64,
// rounded once to the storage type.
//
// Forward table  Tf[s][m][l][j] = (2 pi / W) w_j (-1)^s N_l d^l_{m,-s}(theta_j)
// Inverse table  Ti[s][m][j][l] = (-1)^s N_l d^l_{m,-s}(theta_j)
// with N_l = sqrt((2l+1)/(4 pi)), theta_j = pi (2j+1)/(2H), w_j the
// Driscoll--Healy weights.  These are the latitude factors of the spin
// harmonics of eqs. (2)-(3); the paper factors the same d^l(theta) through
// Wigner Delta = d(pi/2) and a torus FFT (eqs. (4)-(6)), which we evaluate
// directly instead.  The backward pass uses the same values in the other
// layout: the unweighted factors l-major for the output spins (the adjoint of
// the synthesis is an unweighted analysis) and the weighted factors j-major
// for the input spins (the adjoint of the analysis is a weighted synthesis).
//
// One thread per (spin, m, j) runs the three-term recurrence in l from the
// single-term seed at l0 = max(|m|, |s|).
#include "swsft_internal.h"
#include "wigner.h"

namespace swsft {
namespace {

template <typename T>
__device__ __forceinline__ T to_storage(double v);
template <>
__device__ __forceinline__ float to_storage<float>(double v) { return (float)v; }
template <>
__device__ __forceinline__ __bf16 to_storage<__bf16>(double v) {
  // double -> float is exact enough here (|v| <= 1, relative 2^-24), then
  // round-to-nearest-even to bfloat16.
  return (__bf16)(float)v;
}

// weighted: include (2 pi / W) w_j; l_rows: layout [l][Hp] per (s, m), else [Hp][Lp]
template <typename T>
__global__ void tables_kernel(T* __restrict__ tab, int s, int si, bool weighted, bool l_rows,
                              int H, int W, int L, int Hp, int Lp) {
  const int j = blockIdx.x * blockDim.x + threadIdx.x;
  const int mi = blockIdx.y;
  if (j >= H) return;
  const int M = 2 * L - 1;
  const int m = mi - (L - 1);
  const int n = -s;
  const int am = m < 0 ? -m : m, an = n < 0 ? -n : n;
  const int l0 = am > an ? am : an;
  if (l0 >= L) return;
  const double pi = 3.14159265358979323846;
  const double theta = pi * (2.0 * j + 1.0) / (2.0 * H);
  const double c = cos(0.5 * theta), sn = sin(0.5 * theta), cb = cos(theta);
  double scale = (s & 1) ? -1.0 : 1.0;
  if (weighted) {
    // Driscoll--Healy weight on the offset grid, times the longitude step
    double acc = 0.0;
    for (int p = 0; p < H / 2; ++p) acc += sin((2.0 * p + 1.0) * theta) / (2.0 * p + 1.0);
    const double w = (4.0 / H) * sin(theta) * acc;
    scale *= (2.0 * pi / W) * w;
  }
  double dprev = 0.0, dcur = wigner_seed(m, n, c, sn);
  for (int l = l0; l < L; ++l) {
    const double Nl = sqrt((2.0 * l + 1.0) / (4.0 * pi));
    const double v = scale * Nl * dcur;
    if (l_rows) tab[(((size_t)si * M + mi) * L + l) * Hp + j] = to_storage<T>(v);
    else        tab[(((size_t)si * M + mi) * Hp + j) * Lp + l] = to_storage<T>(v);
    if (l + 1 < L) {
      const double lp = l + 1.0;
      const double a = lp * (2.0 * l + 1.0) / sqrt((lp * lp - (double)m * m) * (lp * lp - (double)n * n));
      const double t1 = (l == 0) ? cb * dcur : (cb - (double)m * n / (l * (l + 1.0))) * dcur;
      const double t2 = (l > l0) ? sqrt(((double)l * l - (double)m * m) * ((double)l * l - (double)n * n)) /
                                       (l * (2.0 * l + 1.0)) * dprev
                                 : 0.0;
      const double dn = a * (t1 - t2);
      dprev = dcur;
      dcur = dn;
    }
  }
}

__global__ void twiddle_kernel(float2* tw, int W) {
  const int r = blockIdx.x * blockDim.x + threadIdx.x;
  if (r >= W) return;
  // exp(-2 pi i r / W), phase reduced exactly: r < W
  const double a = -2.0 * 3.14159265358979323846 * (double)r / (double)W;
  tw[r] = make_float2((float)cos(a), (float)sin(a));
}

template <typename T>
hipError_t launch_tables_t(const Plan& p, hipStream_t st) {
  const int M = p.M;
  dim3 block(64);
  dim3 grid((p.H + 63) / 64, M);
  for (int si = 0; si < p.n_in; ++si) {
    hipLaunchKernelGGL(tables_kernel<T>, grid, block, 0, st, (T*)p.tab_fwd, p.spins_in[si], si,
                       true, true, p.H, p.W, p.L, p.Hp, p.Lp);
    hipLaunchKernelGGL(tables_kernel<T>, grid, block, 0, st, (T*)p.tab_bwd_syn, p.spins_in[si],
                       si, true, false, p.H, p.W, p.L, p.Hp, p.Lp);
  }
  for (int si = 0; si < p.n_out; ++si) {
    hipLaunchKernelGGL(tables_kernel<T>, grid, block, 0, st, (T*)p.tab_inv, p.spins_out[si], si,
                       false, false, p.H, p.W, p.L, p.Hp, p.Lp);
    hipLaunchKernelGGL(tables_kernel<T>, grid, block, 0, st, (T*)p.tab_bwd_ana, p.spins_out[si],
                       si, false, true, p.H, p.W, p.L, p.Hp, p.Lp);
  }
  hipLaunchKernelGGL(twiddle_kernel, dim3((p.W + 63) / 64), dim3(64), 0, st, p.twiddle, p.W);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_tables(const Plan& p, hipStream_t st) {
  if (p.dtype == SWSFT_BF16) return launch_tables_t<__bf16>(p, st);
  return launch_tables_t<float>(p, st);
}

}  // namespace swsft
