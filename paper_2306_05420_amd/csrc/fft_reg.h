// Small in-register FFTs with compile-time twiddles, and complex helpers.
#pragma once

#include <hip/hip_runtime.h>

namespace swsft {

constexpr double kPiD = 3.14159265358979323846264338327950288;

// Taylor series, |x| <= pi; evaluated by the compiler only.
constexpr double ct_sin(double x) {
  double term = x, sum = x;
  for (int n = 1; n < 40; ++n) {
    term *= -x * x / ((2.0 * n) * (2.0 * n + 1.0));
    sum += term;
  }
  return sum;
}
constexpr double ct_cos(double x) {
  double term = 1.0, sum = 1.0;
  for (int n = 1; n < 40; ++n) {
    term *= -x * x / ((2.0 * n - 1.0) * (2.0 * n));
    sum += term;
  }
  return sum;
}

// exp(-2 pi i k / N) for k < N, rounded from double.
template <int N>
struct RootTable {
  float re[N > 0 ? N : 1];
  float im[N > 0 ? N : 1];
  constexpr RootTable() : re(), im() {
    for (int k = 0; k < N; ++k) {
      double a = -2.0 * kPiD * k / N;
      if (a < -kPiD) a += 2.0 * kPiD;
      re[k] = (float)ct_cos(a);
      im[k] = (float)ct_sin(a);
    }
  }
};

template <int N>
struct Roots {
  static constexpr RootTable<N> t{};
};

__device__ __forceinline__ float2 cadd(float2 a, float2 b) { return make_float2(a.x + b.x, a.y + b.y); }
__device__ __forceinline__ float2 csub(float2 a, float2 b) { return make_float2(a.x - b.x, a.y - b.y); }
__device__ __forceinline__ float2 cmul(float2 a, float2 b) {
  return make_float2(a.x * b.x - a.y * b.y, a.x * b.y + a.y * b.x);
}
__device__ __forceinline__ float2 cmulc(float2 a, float2 b) {  // a * conj(b)
  return make_float2(a.x * b.x + a.y * b.y, a.y * b.x - a.x * b.y);
}

constexpr int ilog2(int n) { return n <= 1 ? 0 : 1 + ilog2(n / 2); }
constexpr int bitrev(int i, int bits) {
  int r = 0;
  for (int b = 0; b < bits; ++b) r |= ((i >> b) & 1) << (bits - 1 - b);
  return r;
}

// In-place length-N DFT of v: v[k] <- sum_q v[q] exp(SIGN 2 pi i q k / N).
// Radix-2 decimation in time, fully unrolled, twiddles folded to constants;
// the butterflies with twiddle 1 or -+i take no multiplies.
template <int N, int SIGN>
__device__ __forceinline__ void fft_reg(float2 (&v)[N]) {
  if constexpr (N > 1) {
    constexpr int bits = ilog2(N);
#pragma unroll
    for (int i = 0; i < N; ++i) {
      const int j = bitrev(i, bits);
      if (j > i) {
        float2 t = v[i];
        v[i] = v[j];
        v[j] = t;
      }
    }
#pragma unroll
    for (int half = 1; half < N; half *= 2) {
#pragma unroll
      for (int i = 0; i < N; i += 2 * half) {
#pragma unroll
        for (int k = 0; k < half; ++k) {
          const int idx = k * (N / (2 * half));
          const float wr = Roots<N>::t.re[idx];
          const float wi = (SIGN < 0 ? 1.0f : -1.0f) * Roots<N>::t.im[idx];
          const float2 a = v[i + k];
          const float2 b = v[i + k + half];
          float2 bw;
          if (idx == 0) {
            bw = b;
          } else if (4 * idx == N) {  // w = -i (forward) or +i (inverse): exact, no multiplies
            bw = SIGN < 0 ? make_float2(b.y, -b.x) : make_float2(-b.y, b.x);
          } else {
            bw = make_float2(b.x * wr - b.y * wi, b.x * wi + b.y * wr);
          }
          v[i + k] = cadd(a, bw);
          v[i + k + half] = csub(a, bw);
        }
      }
    }
  }
}

}  // namespace swsft
