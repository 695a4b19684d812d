// Longitude DFT stages of the transform.
//
// Forward:  X[s][m][j][n][re/im] = sum_k x[b][s][c][j][k] exp(-2 pi i m k / W)
// Inverse:  y[b][s][c][j][k]     = sum_m Y[s][m][j][n][re/im] exp(+2 pi i m k / W)
// for orders |m| < L, n = b*C + c.  This is the e^{i m phi} factor of the
// harmonics in eqs. (2)-(3); the paper evaluates it as a dense DFT matrix
// product on TPU (Method, "Efficient TPU implementation"), here it is an
// in-register FFT because the stage is bound by HBM traffic, not flops.
//
// One workgroup handles JB consecutive rows j of one map.  Each row of W
// samples is split W = W1 * W2: W1 threads per row, each holding W2 samples
// strided by W1 (coalesced loads), a length-W2 register FFT, a twiddle, an
// LDS exchange, a length-W1 register FFT.  The spectrum is then staged in
// LDS as [m][re/im][j] and written with j fastest into the K-tiled layout
// X[s][m][j/JT][n][re/im][JT] (JT = 32): the latitude index, the K dimension
// of the latitude GEMM, is contiguous within a tile, and one tile of all
// maps is one contiguous block, so the GEMM reads whole 8 KiB blocks per K
// step and a block of rows of one map writes 128-byte runs.
#include "fft_reg.h"
#include "swsft_internal.h"
#include "xcd.h"

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

// Row pitch (elements) of the [m][re/im][j] staging buffer: a multiple of
// 16 bytes so whole 16-byte vectors move between LDS and HBM, and an odd
// multiple of 16 bytes so consecutive orders start in different banks.
template <typename T>
constexpr int stage_pitch(int JB) {
  return sizeof(T) == 4 ? 2 * JB + 4 : 2 * JB + 8;
}

// Raw register image of one complex input sample (loaded before any compute).
template <typename T>
struct Raw;
template <>
struct Raw<float> {
  using type = float2;
  static __device__ __forceinline__ type load(const float* p, size_t i) {
    return reinterpret_cast<const float2*>(p)[i];
  }
  static __device__ __forceinline__ float2 unpack(type v) { return v; }
};
template <>
struct Raw<__bf16> {
  using type = uint32_t;
  static __device__ __forceinline__ type load(const __bf16* p, size_t i) {
    return reinterpret_cast<const uint32_t*>(p)[i];
  }
  static __device__ __forceinline__ float2 unpack(type u) {
    return make_float2(__uint_as_float(u << 16), __uint_as_float(u & 0xffff0000u));
  }
};

constexpr int kMaxPasses = 2;

// Move the [M][2][JB] spectrum block between the LDS stage (pitch SP) and
// global memory at gbase[mi * mstride + (n * 2 + ri) * pitch + r] (gbase
// already offset to the spin, latitude tile and row), in 16-byte vectors
// when JB allows.
template <typename T, bool kToGlobal>
__device__ __forceinline__ void stage_copy(T* stage, T* gbase, int M, int JB, int SP,
                                           size_t mstride, size_t nbase, int pitch, int tid,
                                           int nthreads) {
  constexpr int VEC = 16 / sizeof(T);
  constexpr int BATCH = 8;  // global loads in flight per thread before their LDS stores
  if (JB % VEC == 0) {
    const int vpr = JB / VEC;
    const int total = M * 2 * vpr;
    for (int base = tid; base < total; base += BATCH * nthreads) {
      uint4 buf[BATCH];
#pragma unroll
      for (int u = 0; u < BATCH; ++u) {
        const int idx = base + u * nthreads;
        // no per-lane branch around a load: out-of-range lanes read vector 0
        const int id = idx < total ? idx : 0;
        const int vi = id % vpr;
        const int ri = (id / vpr) & 1;
        const int mi = id / (2 * vpr);
        uint4* s = reinterpret_cast<uint4*>(stage + (size_t)mi * SP + ri * JB + vi * VEC);
        uint4* g = reinterpret_cast<uint4*>(gbase + mi * mstride + (nbase * 2 + ri) * pitch + vi * VEC);
        if (kToGlobal) {
          if (idx < total) *g = *s;
        } else {
          buf[u] = *g;
        }
      }
      if (!kToGlobal) {
        // unconditional stores too (a lane past the end rewrites vector 0 with
        // the same data): a conditional store lets the compiler sink each
        // load next to it, which serializes the loads again
#pragma unroll
        for (int u = 0; u < BATCH; ++u) {
          const int idx = base + u * nthreads;
          const int id = idx < total ? idx : 0;
          const int vi = id % vpr;
          const int ri = (id / vpr) & 1;
          const int mi = id / (2 * vpr);
          *reinterpret_cast<uint4*>(stage + (size_t)mi * SP + ri * JB + vi * VEC) = buf[u];
        }
      }
    }
  } else {
    const int total = M * 2 * JB;
    for (int idx = tid; idx < total; idx += nthreads) {
      const int r = idx % JB;
      const int ri = (idx / JB) & 1;
      const int mi = idx / (2 * JB);
      T* s = stage + (size_t)mi * SP + ri * JB + r;
      T* g = gbase + mi * mstride + (nbase * 2 + ri) * pitch + r;
      if (kToGlobal) *g = *s;
      else *s = *g;
    }
  }
}

template <typename Tin, typename Tout, int W1, int W2>
__global__ void __launch_bounds__(256) dft_fwd_kernel(const Tin* __restrict__ x,
                                                      Tout* __restrict__ X,
                                                      const float2* __restrict__ tw, int S,
                                                      int C, int NB, int NBC, int H, int JT,
                                                      int L, int JB) {
  constexpr int W = W1 * W2;
  extern __shared__ __align__(16) unsigned char smem[];
  const int RPP = blockDim.x / W1;
  const int NP = JB / RPP;  // passes, <= kMaxPasses
  const int tid = threadIdx.x;
  const int t = tid % W1;
  const int rr = tid / W1;
  const int nJB = H / JB;
  // consecutive row blocks of a map (which share the 128-byte lines of the
  // transposed spectrum) are numbered together, so they run on one XCD
  const int lb = xcd_logical_block();
  if (lb >= S * C * NB * nJB) return;
  const int map = lb / nJB;
  const int j0 = (lb % nJB) * JB;
  const int c = map % C;
  const int si = (map / C) % S;
  const int b = map / (C * S);
  const int n = b * C + c;
  const int M = 2 * L - 1;
  const int SP = stage_pitch<Tout>(JB);
  // the exchange buffer [RPP][W2][W1+1] (during the FFTs) and the spectrum
  // stage [M][SP] (after them) share one allocation
  float2* ex = reinterpret_cast<float2*>(smem);
  Tout* stage = reinterpret_cast<Tout*>(smem);

  // every load of the block's JB rows is issued before any arithmetic
  const size_t row_base = ((size_t)map * H + j0) * W;  // complex index of row j0
  typename Raw<Tin>::type raw[kMaxPasses][W2];
#pragma unroll
  for (int p = 0; p < kMaxPasses; ++p)
    if (p < NP) {
#pragma unroll
      for (int q = 0; q < W2; ++q)
        raw[p][q] = Raw<Tin>::load(x, row_base + (size_t)(p * RPP + rr) * W + t + W1 * q);
    }
  float2* exr = ex + (size_t)rr * W2 * (W1 + 1);
  // spectra of all passes stay in registers until the exchange buffer is free:
  // spec[p][i * W1 + k1] is frequency t + W1 * i + W2 * k1 of row p * RPP + rr
  float2 spec[kMaxPasses][W2];
#pragma unroll
  for (int p = 0; p < kMaxPasses; ++p) {
    if (p >= NP) break;
    float2 v[W2];
#pragma unroll
    for (int q = 0; q < W2; ++q) v[q] = Raw<Tin>::unpack(raw[p][q]);
    fft_reg<W2, -1>(v);
#pragma unroll
    for (int k2 = 1; k2 < W2; ++k2) v[k2] = cmul(v[k2], tw[t * k2]);
    if (p > 0) __syncthreads();  // the previous pass has finished reading ex
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
      for (int k1 = 0; k1 < W1; ++k1) spec[p][i * W1 + k1] = u[k1];
    }
  }
  __syncthreads();  // every read of ex is done before the stage overwrites it
#pragma unroll
  for (int p = 0; p < kMaxPasses; ++p) {
    if (p >= NP) break;
    const int r = p * RPP + rr;
#pragma unroll
    for (int i = 0; i < W2 / W1; ++i)
#pragma unroll
      for (int k1 = 0; k1 < W1; ++k1) {
        const int f = t + W1 * i + W2 * k1;
        const int m = f < L ? f : f - W;
        if (m > -L && m < L) {
          Tout* sp = stage + (size_t)(m + L - 1) * SP;
          sp[r] = (Tout)spec[p][i * W1 + k1].x;
          sp[JB + r] = (Tout)spec[p][i * W1 + k1].y;
        }
      }
  }
  __syncthreads();
  // X[si][mi][n][ri][j0 + r]
  // X[si][mi][j0 / JT][n][ri][j0 % JT + r]
  const size_t tile = (size_t)NBC * 2 * JT;  // one latitude tile of one order
  stage_copy<Tout, true>(stage, X + ((size_t)si * M * (H / JT) + j0 / JT) * tile + j0 % JT, M, JB,
                         SP, (size_t)(H / JT) * tile, n, JT, tid, blockDim.x);
}

template <typename Tin, typename Tout, int W1, int W2>
__global__ void __launch_bounds__(256) dft_inv_kernel(const Tin* __restrict__ Y,
                                                      Tout* __restrict__ y,
                                                      const float2* __restrict__ tw, int S,
                                                      int C, int NB, int NBC, int H, int JT,
                                                      int L, int JB) {
  constexpr int W = W1 * W2;
  extern __shared__ __align__(16) unsigned char smem[];
  const int RPP = blockDim.x / W1;
  const int NP = JB / RPP;
  const int tid = threadIdx.x;
  const int t = tid % W1;
  const int rr = tid / W1;
  const int nJB = H / JB;
  // consecutive row blocks of a map (which share the 128-byte lines of the
  // transposed spectrum) are numbered together, so they run on one XCD
  const int lb = xcd_logical_block();
  if (lb >= S * C * NB * nJB) return;
  const int map = lb / nJB;
  const int j0 = (lb % nJB) * JB;
  const int c = map % C;
  const int si = (map / C) % S;
  const int b = map / (C * S);
  const int n = b * C + c;
  const int M = 2 * L - 1;
  const int SP = stage_pitch<Tin>(JB);
  // the spectrum stage [M][SP] (first) and the exchange buffer
  // [RPP][W2][W1+1] (during the FFTs) share one allocation
  Tin* stage = reinterpret_cast<Tin*>(smem);
  float2* ex = reinterpret_cast<float2*>(smem);

  const size_t tile = (size_t)NBC * 2 * JT;  // one latitude tile of one order
  stage_copy<Tin, false>(stage,
                         const_cast<Tin*>(Y) + ((size_t)si * M * (H / JT) + j0 / JT) * tile + j0 % JT,
                         M, JB, SP, (size_t)(H / JT) * tile, n, JT, tid, blockDim.x);
  __syncthreads();

  // the spectra of all passes are read into registers before the exchange
  // buffer overwrites the stage
  float2 v[kMaxPasses][W2];
#pragma unroll
  for (int p = 0; p < kMaxPasses; ++p) {
    if (p >= NP) break;
    const int r = p * RPP + rr;
#pragma unroll
    for (int q = 0; q < W2; ++q) {
      // branch-free: orders outside |m| < L read row 0 and are zeroed after
      const int f = t + W1 * q;
      const int m = f < L ? f : f - W;
      const bool ok = m > -L && m < L;
      const Tin* sp = stage + (size_t)(ok ? m + L - 1 : 0) * SP;
      const float re = (float)sp[r], im = (float)sp[JB + r];
      v[p][q] = make_float2(ok ? re : 0.f, ok ? im : 0.f);
    }
  }
  __syncthreads();

  const size_t row_base = ((size_t)map * H + j0) * W;
  float2* exr = ex + (size_t)rr * W2 * (W1 + 1);
#pragma unroll
  for (int p = 0; p < kMaxPasses; ++p) {
    if (p >= NP) break;
    const int r = p * RPP + rr;
    fft_reg<W2, +1>(v[p]);
#pragma unroll
    for (int k2 = 1; k2 < W2; ++k2) v[p][k2] = cmulc(v[p][k2], tw[t * k2]);
    if (p > 0) __syncthreads();  // the previous pass has finished reading ex
#pragma unroll
    for (int k2 = 0; k2 < W2; ++k2) exr[k2 * (W1 + 1) + t] = v[p][k2];
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
  }
}

// Rows per workgroup JB = NP * RPP: RPP rows are transformed at a time by
// 256 / W1 threads (fewer for small grids), NP <= 2 passes.  JB = 32 gives
// 64-byte (bf16) / 128-byte (f32) runs per order in the transposed layout.
#ifndef SWSFT_DFT_THREADS
#define SWSFT_DFT_THREADS 256
#endif
#ifndef SWSFT_DFT_JB
#define SWSFT_DFT_JB 32
#endif

template <typename Ts, int W1, int W2>
void dft_geometry(const Plan& p, int* JB, int* nthreads, size_t* lds) {
  int rpp = SWSFT_DFT_THREADS / W1;
  if (rpp < 1) rpp = 1;
  if (rpp > p.H) rpp = p.H;
  int jb = rpp;
  if (jb < SWSFT_DFT_JB && 2 * jb <= p.H) jb *= 2;  // a second pass when rows allow
  auto bytes = [&](int j) {  // exchange buffer and stage alias
    const size_t ex = (size_t)rpp * W2 * (W1 + 1) * sizeof(float2);
    const size_t stage = (size_t)p.M * stage_pitch<Ts>(j) * sizeof(Ts);
    return ex > stage ? ex : stage;
  };
  if (bytes(jb) > 160 * 1024) jb = rpp;  // one pass if two do not fit the CU's LDS
  *JB = jb;
  *nthreads = rpp * W1;
  *lds = bytes(jb);
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
  hipLaunchKernelGGL(kern, dim3(xcd_grid(blocks)), dim3(nthreads), lds, st, (const Tin*)x,
                     (Tout*)X, p.twiddle, S, C, B, B * C, p.H, p.JT, p.L, JB);
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
  hipLaunchKernelGGL(kern, dim3(xcd_grid(blocks)), dim3(nthreads), lds, st, (const Tin*)Y,
                     (Tout*)y, p.twiddle, S, C, B, B * C, p.H, p.JT, p.L, JB);
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
