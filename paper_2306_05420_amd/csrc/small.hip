// Small grids (H = W <= 16): the transforms, and the layer, in two launches
// instead of five.  At these sizes every stage is a few microseconds of
// launch latency, not bandwidth, so one workgroup per map does a whole
// transform in LDS:
//
//  small_fwd  per input map (b, s, c): x -> longitude DFT (eq. (2)'s
//             e^{-i m phi} sum, plan twiddles) -> latitude quadrature with the
//             weighted table -> coef[l^2+l+m][b][s][c]
//  small_inv  per output map (b, t, c'): [the per-degree mixing of that output
//             channel over all input channels, filters shared across m] ->
//             latitude synthesis with the inverse table -> inverse longitude
//             DFT (eq. (3)) -> y[b][t][c'][j][k]
//
// Everything accumulates in float; the tables and twiddles are the plan's.
#include "swsft_internal.h"

namespace swsft {
namespace {

constexpr int kSmallNT = 256;

template <typename T>
__device__ __forceinline__ float2 ldc(const T* p, size_t i) {
  return make_float2((float)p[2 * i], (float)p[2 * i + 1]);
}
template <typename T>
__device__ __forceinline__ void stc(T* p, size_t i, float2 v) {
  p[2 * i] = (T)v.x;
  p[2 * i + 1] = (T)v.y;
}
__device__ __forceinline__ int iabs_s(int v) { return v < 0 ? -v : v; }

struct SmallSpins {
  int s[kMaxSpins];
};

// LDS of small_fwd: x [H][W], X [M][H], twiddles [W], the spin's weighted
// table [M][L][H] as float
template <typename T>
__global__ void __launch_bounds__(kSmallNT) small_fwd_kernel(const T* __restrict__ x,
                                                             const T* __restrict__ tab,
                                                             const float2* __restrict__ tw,
                                                             T* __restrict__ coef, int H, int W,
                                                             int L, int Hp, int B, int S, int C) {
  extern __shared__ float2 sm[];
  const int M = 2 * L - 1;
  float2* xs = sm;                // [H][W]
  float2* Xs = xs + H * W;        // [M][H]
  float2* tws = Xs + M * H;       // [W]
  float* ts = reinterpret_cast<float*>(tws + W);  // [M][L][H]
  const int map = blockIdx.x;     // (b * S + si) * C + c
  const int c = map % C, bs = map / C, si = bs % S, b = bs / S;
  const int tid = threadIdx.x;
  for (int i = tid; i < H * W; i += kSmallNT) xs[i] = ldc(x, (size_t)map * H * W + i);
  for (int i = tid; i < W; i += kSmallNT) tws[i] = tw[i];
  const T* tsrc = tab + (size_t)si * M * L * Hp;
  for (int i = tid; i < M * L * H; i += kSmallNT) {
    const int row = i / H, j = i - row * H;
    ts[i] = (float)tsrc[(size_t)row * Hp + j];
  }
  __syncthreads();
  for (int i = tid; i < M * H; i += kSmallNT) {
    const int mi = i / H, j = i - mi * H;
    const int m = mi - (L - 1);
    const int step = ((m % W) + W) % W;
    float2 acc = make_float2(0.f, 0.f);
    int r = 0;  // m k mod W
    for (int k = 0; k < W; ++k) {
      const float2 v = xs[j * W + k], w = tws[r];  // w = exp(-2 pi i m k / W)
      acc.x += v.x * w.x - v.y * w.y;
      acc.y += v.x * w.y + v.y * w.x;
      r += step;
      if (r >= W) r -= W;
    }
    Xs[i] = acc;
  }
  __syncthreads();
  for (int i = tid; i < L * L; i += kSmallNT) {
    int l = (int)sqrtf((float)i);
    while (l * l > i) --l;
    while ((l + 1) * (l + 1) <= i) ++l;
    const int m = i - l * l - l, mi = m + L - 1;
    const float* trow = ts + (mi * L + l) * H;  // zero below max(|m|, |s|)
    float2 acc = make_float2(0.f, 0.f);
    for (int j = 0; j < H; ++j) {
      const float t = trow[j];
      const float2 v = Xs[mi * H + j];
      acc.x += t * v.x;
      acc.y += t * v.y;
    }
    stc(coef, ((size_t)i * B + b) * S * C + (size_t)si * C + c, acc);
  }
}

// mix != 0: coef holds the input spins' coefficients [L^2][B][S_in][C_in] and
// K the filters; else coef holds the output spins' coefficients.  LDS: the
// map's coefficients [L^2], Y [M][H], twiddles [W], the spin's inverse table
// [M][H][L] as float, and with mixing the batch item's input coefficients
// [L^2][S_in C_in] and the output channel's filters [L][S_in C_in].
template <typename T>
__global__ void __launch_bounds__(kSmallNT) small_inv_kernel(
    const T* __restrict__ coef, const T* __restrict__ K, const T* __restrict__ tab,
    const float2* __restrict__ tw, T* __restrict__ y, int H, int W, int L, int Hp, int Lp, int B,
    int S_in, int C_in, int S_out, int C_out, SmallSpins sin_, SmallSpins sout_, int mix) {
  extern __shared__ float2 sm[];
  const int M = 2 * L - 1;
  const int KC = S_in * C_in;
  float2* cs = sm;               // [L^2]
  float2* Ys = cs + L * L;       // [M][H]
  float2* tws = Ys + M * H;      // [W]
  float2* as = tws + W;          // [L^2][KC] (mixing only)
  float2* ks = as + (mix ? L * L * KC : 0);       // [L][KC]
  float* ts = reinterpret_cast<float*>(ks + (mix ? L * KC : 0));  // [M][H][L]
  const int map = blockIdx.x;    // (b * S_out + t) * C_out + c'
  const int co = map % C_out, bt = map / C_out, ti = bt % S_out, b = bt / S_out;
  const int tspin = iabs_s(sout_.s[ti]);
  const int tid = threadIdx.x;
  for (int i = tid; i < W; i += kSmallNT) tws[i] = tw[i];
  const T* tsrc = tab + (size_t)ti * M * Hp * Lp;
  for (int i = tid; i < M * H * L; i += kSmallNT) {
    const int row = i / L, l = i - row * L;  // row = mi * H + j
    const int mi = row / H, j = row - mi * H;
    ts[i] = (float)tsrc[((size_t)mi * Hp + j) * Lp + l];
  }
  if (mix) {
    for (int i = tid; i < L * L * KC; i += kSmallNT) {
      const int r = i / KC, q = i - r * KC;
      as[i] = ldc(coef, ((size_t)r * B + b) * KC + q);
    }
    for (int i = tid; i < L * KC; i += kSmallNT) {
      const int l = i / KC, q = i - l * KC;
      ks[i] = ldc(K, (((size_t)l * S_out + ti) * C_out + co) * KC + q);
    }
  }
  __syncthreads();
  for (int i = tid; i < L * L; i += kSmallNT) {
    int l = (int)sqrtf((float)i);
    while (l * l > i) --l;
    while ((l + 1) * (l + 1) <= i) ++l;
    float2 acc = make_float2(0.f, 0.f);
    if (!mix) {
      acc = ldc(coef, ((size_t)i * B + b) * S_out * C_out + (size_t)ti * C_out + co);
    } else if (tspin <= l) {
      for (int q = 0; q < KC; ++q) {
        if (iabs_s(sin_.s[q / C_in]) > l) continue;
        const float2 k = ks[l * KC + q], a = as[i * KC + q];
        acc.x += k.x * a.x - k.y * a.y;
        acc.y += k.x * a.y + k.y * a.x;
      }
    }
    cs[i] = acc;
  }
  __syncthreads();
  for (int i = tid; i < M * H; i += kSmallNT) {
    const int mi = i / H;
    const int m = mi - (L - 1);
    const int am = m < 0 ? -m : m;
    const int lo = am > tspin ? am : tspin;
    const float* trow = ts + i * L;
    float2 acc = make_float2(0.f, 0.f);
    for (int l = lo; l < L; ++l) {
      const float t = trow[l];
      const float2 v = cs[l * l + l + m];
      acc.x += t * v.x;
      acc.y += t * v.y;
    }
    Ys[i] = acc;
  }
  __syncthreads();
  for (int i = tid; i < H * W; i += kSmallNT) {
    const int j = i / W, k = i - j * W;
    float2 acc = make_float2(0.f, 0.f);
    int r = ((-(L - 1) * k) % W + W) % W;  // m k mod W, m from -(L-1)
    for (int mi = 0; mi < M; ++mi) {
      const float2 v = Ys[mi * H + j], w = tws[r];  // conj(w) = exp(+2 pi i m k / W)
      acc.x += v.x * w.x + v.y * w.y;
      acc.y += v.y * w.x - v.x * w.y;
      r += k;
      if (r >= W) r -= W;
    }
    stc(y, (size_t)map * H * W + i, acc);
  }
}

SmallSpins small_spins(const int* s, int n) {
  SmallSpins r{};
  for (int i = 0; i < n && i < kMaxSpins; ++i) r.s[i] = s[i];
  return r;
}

}  // namespace

// Used up to H = 16: measured, the per-map kernels win over the five-stage
// path only while launch latency dominates (16^2: 22 -> 15 us per layer);
// at 32^2 staging each spin's table per workgroup costs more than it saves.
bool small_path(const Plan& p, int Cin) {
  return p.H <= 16 && p.fft_ok && !(p.flags & SWSFT_PLAN_DFT_MATMUL) && !is_delta(p) &&
         p.n_in * Cin <= 32;
}

hipError_t launch_small_fwd(const Plan& p, int B, int C, const void* x, void* coef,
                            hipStream_t st) {
  const size_t lds = (size_t)(p.H * p.W + p.M * p.H + p.W) * sizeof(float2) +
                     (size_t)p.M * p.L * p.H * sizeof(float);
  const unsigned grid = (unsigned)(B * p.n_in * C);
  auto kern = p.dtype == SWSFT_BF16 ? (const void*)small_fwd_kernel<__bf16>
                                    : (const void*)small_fwd_kernel<float>;
  const hipError_t e = ensure_dynamic_lds(kern, lds);
  if (e != hipSuccess) return e;
  if (p.dtype == SWSFT_BF16)
    hipLaunchKernelGGL(small_fwd_kernel<__bf16>, dim3(grid), dim3(kSmallNT), lds, st,
                       (const __bf16*)x, (const __bf16*)p.tab_fwd, p.twiddle, (__bf16*)coef, p.H,
                       p.W, p.L, p.Hp, B, p.n_in, C);
  else
    hipLaunchKernelGGL(small_fwd_kernel<float>, dim3(grid), dim3(kSmallNT), lds, st,
                       (const float*)x, (const float*)p.tab_fwd, p.twiddle, (float*)coef, p.H,
                       p.W, p.L, p.Hp, B, p.n_in, C);
  return hipGetLastError();
}

// K == nullptr: coef are the output spins' coefficients (no mixing)
hipError_t launch_small_inv(const Plan& p, int B, int C_in, int C_out, const void* coef,
                            const void* K, void* y, hipStream_t st) {
  const int mix = K != nullptr ? 1 : 0;
  const int KC = p.n_in * C_in;
  const size_t lds = (size_t)(p.L * p.L + p.M * p.H + p.W) * sizeof(float2) +
                     (mix ? (size_t)(p.L * p.L + p.L) * KC * sizeof(float2) : 0) +
                     (size_t)p.M * p.H * p.L * sizeof(float);
  const unsigned grid = (unsigned)(B * p.n_out * C_out);
  const SmallSpins si = small_spins(p.spins_in, p.n_in), so = small_spins(p.spins_out, p.n_out);
  auto kern = p.dtype == SWSFT_BF16 ? (const void*)small_inv_kernel<__bf16>
                                    : (const void*)small_inv_kernel<float>;
  const hipError_t e = ensure_dynamic_lds(kern, lds);
  if (e != hipSuccess) return e;
  if (p.dtype == SWSFT_BF16)
    hipLaunchKernelGGL(small_inv_kernel<__bf16>, dim3(grid), dim3(kSmallNT), lds, st,
                       (const __bf16*)coef, (const __bf16*)K, (const __bf16*)p.tab_inv, p.twiddle,
                       (__bf16*)y, p.H, p.W, p.L, p.Hp, p.Lp, B, p.n_in, C_in, p.n_out, C_out, si,
                       so, mix);
  else
    hipLaunchKernelGGL(small_inv_kernel<float>, dim3(grid), dim3(kSmallNT), lds, st,
                       (const float*)coef, (const float*)K, (const float*)p.tab_inv, p.twiddle,
                       (float*)y, p.H, p.W, p.L, p.Hp, p.Lp, B, p.n_in, C_in, p.n_out, C_out, si,
                       so, mix);
  return hipGetLastError();
}

}  // namespace swsft
