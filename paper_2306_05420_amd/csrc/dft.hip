// Longitude DFT stages of the transform.
//
// Forward:  X[s][m][n][re/im][j] = sum_k x[b][s][c][j][k] exp(-2 pi i m k / W)
// Inverse:  y[b][s][c][j][k]     = sum_m Y[s][m][n][re/im][j] exp(+2 pi i m k / W)
// for orders |m| < L, n = b*C + c.  This is the e^{i m phi} factor of the
// harmonics in eqs. (2)-(3); the paper evaluates it as a dense DFT matrix
// product on TPU (Method, "Efficient TPU implementation"), here it is an
// in-register FFT because the stage is bound by HBM traffic, not flops.
//
// One workgroup handles JB consecutive rows j of one map.  Each row of W
// samples is split W = W1 * W2: W1 threads per row, each holding W2 samples
// strided by W1 (coalesced loads), a length-W2 register FFT, a twiddle, an
// LDS exchange, a length-W1 register FFT.  The spectrum is then staged in
// LDS as [m][re/im][j] and written with j fastest, so the output layout has
// the latitude index contiguous, which is the K dimension of the latitude
// GEMM that reads it.
#include "fft_reg.h"
#include "swsft_internal.h"

namespace swsft {
namespace {

template <typename T>
struct CplxIO;
template <>
struct CplxIO<float> {
  static __device__ __forceinline__ float2 load(const float* p, size_t i) {
    return reinterpret_cast<const float2*>(p)[i];
  }
  static __device__ __forceinline__ void store(float* p, size_t i, float2 v) {
    reinterpret_cast<float2*>(p)[i] = v;
  }
};
template <>
struct CplxIO<__bf16> {
  static __device__ __forceinline__ float2 load(const __bf16* p, size_t i) {
    const uint32_t u = reinterpret_cast<const uint32_t*>(p)[i];
    return make_float2(__uint_as_float(u << 16), __uint_as_float(u & 0xffff0000u));
  }
  static __device__ __forceinline__ void store(__bf16* p, size_t i, float2 v) {
    __bf16 r = (__bf16)v.x, q = (__bf16)v.y;
    const uint32_t u = (uint32_t)__builtin_bit_cast(uint16_t, r) |
                       ((uint32_t)__builtin_bit_cast(uint16_t, q) << 16);
    reinterpret_cast<uint32_t*>(p)[i] = u;
  }
};

template <typename T>
constexpr int stage_pitch(int JB) {
  return sizeof(T) == 4 ? 2 * JB + 1 : 2 * JB + 2;  // odd number of dwords
}

template <typename Tin, typename Tout, int W1, int W2>
__global__ void __launch_bounds__(256) dft_fwd_kernel(const Tin* __restrict__ x,
                                                      Tout* __restrict__ X,
                                                      const float2* __restrict__ tw, int S,
                                                      int C, int NBC, int H, int Hp, int L,
                                                      int JB) {
  constexpr int W = W1 * W2;
  extern __shared__ __align__(16) unsigned char smem[];
  const int RPP = blockDim.x / W1;
  const int tid = threadIdx.x;
  const int t = tid % W1;
  const int rr = tid / W1;
  const int nJB = H / JB;
  const int map = blockIdx.x / nJB;
  const int j0 = (blockIdx.x % nJB) * JB;
  const int c = map % C;
  const int si = (map / C) % S;
  const int b = map / (C * S);
  const int n = b * C + c;
  const int M = 2 * L - 1;
  const int SP = stage_pitch<Tout>(JB);
  float2* ex = reinterpret_cast<float2*>(smem);  // [RPP][W2][W1+1]
  Tout* stage = reinterpret_cast<Tout*>(ex + (size_t)RPP * W2 * (W1 + 1));  // [M][SP]

  const size_t row_base = ((size_t)map * H + j0) * W;  // complex index of row j0
  for (int r0 = 0; r0 < JB; r0 += RPP) {
    const int r = r0 + rr;
    float2 v[W2];
#pragma unroll
    for (int q = 0; q < W2; ++q) v[q] = CplxIO<Tin>::load(x, row_base + (size_t)r * W + t + W1 * q);
    fft_reg<W2, -1>(v);
#pragma unroll
    for (int k2 = 1; k2 < W2; ++k2) v[k2] = cmul(v[k2], tw[(t * k2) % W]);
    float2* exr = ex + (size_t)rr * W2 * (W1 + 1);
#pragma unroll
    for (int k2 = 0; k2 < W2; ++k2) exr[k2 * (W1 + 1) + t] = v[k2];
    __syncthreads();
#pragma unroll
    for (int i = 0; i < W2 / W1; ++i) {
      const int k2 = t + W1 * i;
      float2 u[W1];
#pragma unroll
      for (int tp = 0; tp < W1; ++tp) u[tp] = exr[k2 * (W1 + 1) + tp];
      fft_reg<W1, -1>(u);
#pragma unroll
      for (int k1 = 0; k1 < W1; ++k1) {
        const int f = k2 + W2 * k1;
        const int m = f < L ? f : f - W;
        if (m > -L && m < L) {
          Tout* sp = stage + (size_t)(m + L - 1) * SP;
          sp[r] = (Tout)u[k1].x;
          sp[JB + r] = (Tout)u[k1].y;
        }
      }
    }
    __syncthreads();
  }
  // X[si][mi][n][ri][j0 + r], r fastest
  const int total = M * 2 * JB;
  for (int idx = tid; idx < total; idx += blockDim.x) {
    const int r = idx % JB;
    const int ri = (idx / JB) & 1;
    const int mi = idx / (2 * JB);
    X[((((size_t)si * M + mi) * NBC + n) * 2 + ri) * Hp + j0 + r] = stage[(size_t)mi * SP + ri * JB + r];
  }
}

template <typename Tin, typename Tout, int W1, int W2>
__global__ void __launch_bounds__(256) dft_inv_kernel(const Tin* __restrict__ Y,
                                                      Tout* __restrict__ y,
                                                      const float2* __restrict__ tw, int S,
                                                      int C, int NBC, int H, int Hp, int L,
                                                      int JB) {
  constexpr int W = W1 * W2;
  extern __shared__ __align__(16) unsigned char smem[];
  const int RPP = blockDim.x / W1;
  const int tid = threadIdx.x;
  const int t = tid % W1;
  const int rr = tid / W1;
  const int nJB = H / JB;
  const int map = blockIdx.x / nJB;
  const int j0 = (blockIdx.x % nJB) * JB;
  const int c = map % C;
  const int si = (map / C) % S;
  const int b = map / (C * S);
  const int n = b * C + c;
  const int M = 2 * L - 1;
  const int SP = stage_pitch<Tin>(JB);
  float2* ex = reinterpret_cast<float2*>(smem);
  Tin* stage = reinterpret_cast<Tin*>(ex + (size_t)RPP * W2 * (W1 + 1));

  const int total = M * 2 * JB;
  for (int idx = tid; idx < total; idx += blockDim.x) {
    const int r = idx % JB;
    const int ri = (idx / JB) & 1;
    const int mi = idx / (2 * JB);
    stage[(size_t)mi * SP + ri * JB + r] = Y[((((size_t)si * M + mi) * NBC + n) * 2 + ri) * Hp + j0 + r];
  }
  __syncthreads();

  const size_t row_base = ((size_t)map * H + j0) * W;
  for (int r0 = 0; r0 < JB; r0 += RPP) {
    const int r = r0 + rr;
    float2 v[W2];
#pragma unroll
    for (int q = 0; q < W2; ++q) {
      const int f = t + W1 * q;
      const int m = f < L ? f : f - W;
      if (m > -L && m < L) {
        const Tin* sp = stage + (size_t)(m + L - 1) * SP;
        v[q] = make_float2((float)sp[r], (float)sp[JB + r]);
      } else {
        v[q] = make_float2(0.f, 0.f);
      }
    }
    fft_reg<W2, +1>(v);
#pragma unroll
    for (int k2 = 1; k2 < W2; ++k2) v[k2] = cmulc(v[k2], tw[(t * k2) % W]);
    float2* exr = ex + (size_t)rr * W2 * (W1 + 1);
    // the previous pass's readers of ex are done: the barrier below orders them
#pragma unroll
    for (int k2 = 0; k2 < W2; ++k2) exr[k2 * (W1 + 1) + t] = v[k2];
    __syncthreads();
#pragma unroll
    for (int i = 0; i < W2 / W1; ++i) {
      const int k2 = t + W1 * i;
      float2 u[W1];
#pragma unroll
      for (int tp = 0; tp < W1; ++tp) u[tp] = exr[k2 * (W1 + 1) + tp];
      fft_reg<W1, +1>(u);
#pragma unroll
      for (int k1 = 0; k1 < W1; ++k1)
        CplxIO<Tout>::store(y, row_base + (size_t)r * W + k2 + W2 * k1, u[k1]);
    }
    __syncthreads();
  }
}

// Rows per workgroup: 32 (64-byte bf16 / 128-byte f32 store runs) unless the
// exchange + staging LDS would exceed 80 KiB (two workgroups per CU), then 16.
template <typename Ts, int W1, int W2>
void dft_geometry(const Plan& p, int* JB, int* nthreads, size_t* lds) {
  for (int jb = p.H < 32 ? p.H : 32;; jb /= 2) {
    const int nt = jb * W1 < 256 ? jb * W1 : 256;
    const int rpp = nt / W1;
    const size_t l = (size_t)rpp * W2 * (W1 + 1) * sizeof(float2) +
                     (size_t)p.M * stage_pitch<Ts>(jb) * sizeof(Ts);
    if (l <= 80 * 1024 || jb <= 16 || jb <= rpp) {
      *JB = jb;
      *nthreads = nt;
      *lds = l;
      return;
    }
  }
}

template <typename Tin, typename Tout, int W1, int W2>
hipError_t launch_fwd_shape(const Plan& p, int S, int B, int C, const void* x, void* X,
                            hipStream_t st) {
  int JB, nthreads;
  size_t lds;
  dft_geometry<Tout, W1, W2>(p, &JB, &nthreads, &lds);
  auto kern = dft_fwd_kernel<Tin, Tout, W1, W2>;
  if (lds > 64 * 1024) {
    const hipError_t e = hipFuncSetAttribute((const void*)kern,
                                             hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
  }
  const long long blocks = (long long)B * S * C * (p.H / JB);
  hipLaunchKernelGGL(kern, dim3((unsigned)blocks), dim3(nthreads), lds, st, (const Tin*)x,
                     (Tout*)X, p.twiddle, S, C, B * C, p.H, p.Hp, p.L, JB);
  return hipGetLastError();
}

template <typename Tin, typename Tout, int W1, int W2>
hipError_t launch_inv_shape(const Plan& p, int S, int B, int C, const void* Y, void* y,
                            hipStream_t st) {
  int JB, nthreads;
  size_t lds;
  dft_geometry<Tin, W1, W2>(p, &JB, &nthreads, &lds);
  auto kern = dft_inv_kernel<Tin, Tout, W1, W2>;
  if (lds > 64 * 1024) {
    const hipError_t e = hipFuncSetAttribute((const void*)kern,
                                             hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
  }
  const long long blocks = (long long)B * S * C * (p.H / JB);
  hipLaunchKernelGGL(kern, dim3((unsigned)blocks), dim3(nthreads), lds, st, (const Tin*)Y,
                     (Tout*)y, p.twiddle, S, C, B * C, p.H, p.Hp, p.L, JB);
  return hipGetLastError();
}

#define SWSFT_W_CASES(X)                                                                 \
  X(2, 1, 2) X(4, 2, 2) X(8, 2, 4) X(16, 4, 4) X(32, 4, 8) X(64, 8, 8) X(128, 8, 16)     \
      X(256, 16, 16) X(512, 16, 32)

template <typename T>
hipError_t dispatch_fwd(const Plan& p, int S, int B, int C, const void* x, void* X,
                        hipStream_t st) {
  switch (p.W) {
#define CASE(Wv, a, b) \
  case Wv:             \
    return launch_fwd_shape<T, T, a, b>(p, S, B, C, x, X, st);
    SWSFT_W_CASES(CASE)
#undef CASE
    default:
      return hipErrorInvalidValue;
  }
}

template <typename T>
hipError_t dispatch_inv(const Plan& p, int S, int B, int C, const void* Y, void* y,
                        hipStream_t st) {
  switch (p.W) {
#define CASE(Wv, a, b) \
  case Wv:             \
    return launch_inv_shape<T, T, a, b>(p, S, B, C, Y, y, st);
    SWSFT_W_CASES(CASE)
#undef CASE
    default:
      return hipErrorInvalidValue;
  }
}

}  // namespace

hipError_t launch_dft_fwd(const Plan& p, int S, int B, int C, const void* x, void* X,
                          hipStream_t st) {
  if (p.dtype == SWSFT_BF16) return dispatch_fwd<__bf16>(p, S, B, C, x, X, st);
  return dispatch_fwd<float>(p, S, B, C, x, X, st);
}

hipError_t launch_dft_inv(const Plan& p, int S, int B, int C, const void* Y, void* y,
                          hipStream_t st) {
  if (p.dtype == SWSFT_BF16) return dispatch_inv<__bf16>(p, S, B, C, Y, y, st);
  return dispatch_inv<float>(p, S, B, C, Y, y, st);
}

}  // namespace swsft
