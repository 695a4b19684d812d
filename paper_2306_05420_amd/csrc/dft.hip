// Longitude DFT stages of the transform.
//
// Forward:  X[s][m][j][n][re/im] = sum_k x[b][s][c][j][k] exp(-2 pi i m k / W)
// Inverse:  y[b][s][c][j][k]     = sum_m Y[s][m][j][n][re/im] exp(+2 pi i m k / W)
// for orders |m| < L, n = b*C + c.  This is the e^{i m phi} factor of the
// harmonics in eqs. (2)-(3); the paper evaluates it as a dense DFT matrix
// product on TPU (Method, "Efficient TPU implementation"), here it is an
// in-register FFT because the stage is bound by HBM traffic and VALU issue,
// not by flops.
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
//
// The grid is square (H == W), so the whole workgroup geometry is a
// compile-time function of W (index arithmetic folds to shifts), and a
// thread transforms NP adjacent rows: their values at one order are adjacent
// in the stage, so bfloat16 pairs move as one 32-bit LDS access.
#include "fft_reg.h"
#include "swsft_internal.h"
#include "xcd.h"

namespace swsft {
namespace {

#ifndef SWSFT_DFT_THREADS
#define SWSFT_DFT_THREADS 256
#endif

// Workgroup geometry for a length-W transform (W = W1 * W2, H = W rows).
template <int W1_, int W2_>
struct DftGeom {
  static constexpr int W1 = W1_, W2 = W2_, W = W1 * W2;
  static constexpr int RPP = SWSFT_DFT_THREADS / W1 < W ? SWSFT_DFT_THREADS / W1 : W;  // rows per pass
  static constexpr int NP = (RPP < 32 && 2 * RPP <= W) ? 2 : 1;  // passes (rows per thread)
  static constexpr int JB = RPP * NP;                            // rows per workgroup (== JT)
  static constexpr int NT = RPP * W1;
  static constexpr size_t ex_bytes = (size_t)RPP * W2 * (W1 + 1) * sizeof(float2);
  static_assert(W2 % W1 == 0 && W % JB == 0, "geometry");
};

// Row pitch (elements) of the [m][re/im][j] staging buffer: a multiple of
// 16 bytes so whole 16-byte vectors move between LDS and HBM, and an odd
// multiple of 16 bytes so consecutive orders start in different banks.
template <typename T, int JB>
constexpr int stage_pitch() {
  return sizeof(T) == 4 ? 2 * JB + 4 : 2 * JB + 8;
}

// Bytes of the shared allocation: the exchange buffer (during the FFTs) and
// the stage of M orders plus one spare row (after them) share it.
template <typename T, class G>
size_t dft_lds_bytes(int M) {
  const size_t stage = (size_t)(M + 1) * stage_pitch<T, G::JB>() * sizeof(T);
  return G::ex_bytes > stage ? G::ex_bytes : stage;
}

// Raw register image of one complex input sample (loaded before any compute).
template <typename T>
struct Raw;
// NT: the non-temporal hint (streams much larger than the caches).
template <>
struct Raw<float> {
  using type = float2;
  template <bool NT>
  static __device__ __forceinline__ type load(const float* p, size_t i) {
    typedef float f2v __attribute__((ext_vector_type(2)));
    if constexpr (NT) {
      const f2v v = __builtin_nontemporal_load(reinterpret_cast<const f2v*>(p) + i);
      return make_float2(v.x, v.y);
    }
    return reinterpret_cast<const float2*>(p)[i];
  }
  static __device__ __forceinline__ float2 unpack(type v) { return v; }
};
template <>
struct Raw<__bf16> {
  using type = uint32_t;
  template <bool NT>
  static __device__ __forceinline__ type load(const __bf16* p, size_t i) {
    if constexpr (NT) return __builtin_nontemporal_load(reinterpret_cast<const uint32_t*>(p) + i);
    return reinterpret_cast<const uint32_t*>(p)[i];
  }
  static __device__ __forceinline__ float2 unpack(type u) {
    return make_float2(__uint_as_float(u << 16), __uint_as_float(u & 0xffff0000u));
  }
};

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));

// Two floats -> packed bfloat16 pair (round to nearest even), one
// v_cvt_pk_bf16_f32.
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2_t){lo, hi}, bf16x2_t));
}

// One complex output sample; NT: the non-temporal hint.
template <bool NT>
__device__ __forceinline__ void store_cplx(float* p, size_t i, float2 v) {
  if constexpr (NT) {
    __builtin_nontemporal_store((f32x2_t){v.x, v.y}, reinterpret_cast<f32x2_t*>(p) + i);
    return;
  }
  reinterpret_cast<float2*>(p)[i] = v;
}
template <bool NT>
__device__ __forceinline__ void store_cplx(__bf16* p, size_t i, float2 v) {
  if constexpr (NT) {
    __builtin_nontemporal_store(pack_bf16x2(v.x, v.y), reinterpret_cast<uint32_t*>(p) + i);
    return;
  }
  reinterpret_cast<uint32_t*>(p)[i] = pack_bf16x2(v.x, v.y);
}

typedef unsigned v4u_t __attribute__((ext_vector_type(4)));

// LDS image of one pass's output rows of the inverse (W >= 64): WPC 32-bit
// words per complex sample, rows padded by 64 (bf16) or 128 (float) bytes so
// the rows one wave writes start in different banks.  The rows then leave as
// 16-byte vectors, whole 128-byte lines, where storing each thread's samples
// directly writes 64-byte pieces (W1 consecutive samples of a row).
template <typename T, int W>
struct OutStage {
  static constexpr bool ON = W >= 64;
  static constexpr int WPC = sizeof(T) == 2 ? 1 : 2;
  static constexpr int PITCH = W * WPC + 16 * WPC;  // words per row
  static constexpr int VPR = W * WPC / 4;           // 16-byte vectors per row
  static __device__ __forceinline__ void put(uint32_t* row, int col, float2 v) {
    if constexpr (WPC == 1) row[col] = pack_bf16x2(v.x, v.y);
    else *reinterpret_cast<float2*>(row + 2 * col) = v;
  }
};

// The NP values of rows NP*rr .. NP*rr+NP-1 at one stage position.
template <typename T, int NP>
struct StageVec;
template <>
struct StageVec<__bf16, 2> {
  static __device__ __forceinline__ void put(__bf16* p, const float (&v)[2]) {
    *reinterpret_cast<uint32_t*>(p) = pack_bf16x2(v[0], v[1]);
  }
  static __device__ __forceinline__ void get(const __bf16* p, float (&v)[2]) {
    const uint32_t u = *reinterpret_cast<const uint32_t*>(p);
    v[0] = __uint_as_float(u << 16);
    v[1] = __uint_as_float(u & 0xffff0000u);
  }
};
template <>
struct StageVec<__bf16, 1> {
  static __device__ __forceinline__ void put(__bf16* p, const float (&v)[1]) { *p = (__bf16)v[0]; }
  static __device__ __forceinline__ void get(const __bf16* p, float (&v)[1]) { v[0] = (float)*p; }
};
template <>
struct StageVec<float, 2> {
  static __device__ __forceinline__ void put(float* p, const float (&v)[2]) {
    *reinterpret_cast<float2*>(p) = make_float2(v[0], v[1]);
  }
  static __device__ __forceinline__ void get(const float* p, float (&v)[2]) {
    const float2 u = *reinterpret_cast<const float2*>(p);
    v[0] = u.x;
    v[1] = u.y;
  }
};
template <>
struct StageVec<float, 1> {
  static __device__ __forceinline__ void put(float* p, const float (&v)[1]) { *p = v[0]; }
  static __device__ __forceinline__ void get(const float* p, float (&v)[1]) { v[0] = *p; }
};

// Move the [M][2][JB] spectrum block between the LDS stage (pitch SP) and
// global memory at gbase[mi * mstride + (n * 2 + ri) * JB + r] (gbase
// already offset to the spin and latitude tile), in 16-byte vectors when JB
// allows.
template <typename T, bool kToGlobal, int JB, int SP, int NT>
__device__ __forceinline__ void stage_copy(T* stage, T* gbase, int M, size_t mstride, size_t n,
                                           int tid) {
  constexpr int VEC = 16 / sizeof(T);
  constexpr int BATCH = 8;  // global loads in flight per thread before their LDS stores
  if constexpr (JB % VEC == 0) {
    constexpr int VPR = JB / VEC;  // vectors per (order, re/im) run
    const int total = M * 2 * VPR;
    T* g0 = gbase + n * 2 * JB;
    for (int base = tid; base < total; base += BATCH * NT) {
      uint4 buf[BATCH];
#pragma unroll
      for (int u = 0; u < BATCH; ++u) {
        const int idx = base + u * NT;
        // no per-lane branch around a load: out-of-range lanes read vector 0
        const int id = idx < total ? idx : 0;
        const int vi = id % VPR, ri = (id / VPR) & 1, mi = id / (2 * VPR);
        uint4* s = reinterpret_cast<uint4*>(stage + mi * SP + ri * JB + vi * VEC);
        uint4* g = reinterpret_cast<uint4*>(g0 + mi * mstride + ri * JB + vi * VEC);
        if constexpr (kToGlobal) {
          if (idx < total) *g = *s;
        } else {
          buf[u] = *g;
        }
      }
      if constexpr (!kToGlobal) {
        // unconditional stores too (a lane past the end rewrites vector 0 with
        // the same data): a conditional store lets the compiler sink each
        // load next to it, which serializes the loads again
#pragma unroll
        for (int u = 0; u < BATCH; ++u) {
          const int idx = base + u * NT;
          const int id = idx < total ? idx : 0;
          const int vi = id % VPR, ri = (id / VPR) & 1, mi = id / (2 * VPR);
          *reinterpret_cast<uint4*>(stage + mi * SP + ri * JB + vi * VEC) = buf[u];
        }
      }
    }
  } else {
    const int total = M * 2 * JB;
    for (int idx = tid; idx < total; idx += NT) {
      const int r = idx % JB, ri = (idx / JB) & 1, mi = idx / (2 * JB);
      T* s = stage + mi * SP + ri * JB + r;
      T* g = gbase + mi * mstride + (n * 2 + ri) * JB + r;
      if constexpr (kToGlobal) *g = *s;
      else *s = *g;
    }
  }
}

// Map and row block of a logical block: consecutive row blocks of a map
// (which share the 128-byte lines of the transposed spectrum) are numbered
// together, so they run on one XCD.
struct MapBlock {
  int map, j0, si, n;
};
template <int JB, int H>
__device__ __forceinline__ bool map_block(int S, int C, int NB, MapBlock& mb) {
  constexpr int nJB = H / JB;
  const int lb = xcd_logical_block();
  if (lb >= S * C * NB * nJB) return false;
  mb.map = lb / nJB;
  mb.j0 = (lb % nJB) * JB;
  const int c = mb.map % C;
  mb.si = (mb.map / C) % S;
  mb.n = (mb.map / (C * S)) * C + c;
  return true;
}

// STREAM: the input rows are read with the non-temporal hint (see launch_dft_fwd).
template <typename Tin, typename Tout, int W1, int W2, bool STREAM>
__global__ void __launch_bounds__((DftGeom<W1, W2>::NT))
    dft_fwd_kernel(const Tin* __restrict__ x, Tout* __restrict__ X,
                   const float2* __restrict__ tw, int S, int C, int NB, int NBC, int L) {
  using G = DftGeom<W1, W2>;
  constexpr int W = G::W, H = W, NP = G::NP, JB = G::JB, NT = G::NT;
  constexpr int SP = stage_pitch<Tout, JB>();
  extern __shared__ __align__(16) unsigned char smem[];
  const int tid = threadIdx.x, t = tid % W1, rr = tid / W1;
  MapBlock mb;
  if (!map_block<JB, H>(S, C, NB, mb)) return;
  const int M = 2 * L - 1;
  // the exchange buffer [RPP][W2][W1+1] (during the FFTs) and the spectrum
  // stage [M + 1][SP] (after them) share one allocation
  float2* ex = reinterpret_cast<float2*>(smem);
  Tout* stage = reinterpret_cast<Tout*>(smem);

  // every load of the block's rows is issued before any arithmetic; this
  // thread's rows are NP * rr + p
  const size_t row_base = ((size_t)mb.map * H + mb.j0 + NP * rr) * W + t;
  typename Raw<Tin>::type raw[NP][W2];
#pragma unroll
  for (int p = 0; p < NP; ++p)
#pragma unroll
    for (int q = 0; q < W2; ++q) raw[p][q] = Raw<Tin>::template load<STREAM>(x, row_base + (size_t)p * W + W1 * q);
  float2 twr[W2];
#pragma unroll
  for (int k2 = 1; k2 < W2; ++k2) twr[k2] = tw[t * k2];

  float2* exr = ex + (size_t)rr * W2 * (W1 + 1);
  // spec[p][i * W1 + k1] is frequency t + W1 * i + W2 * k1 of row NP * rr + p
  float2 spec[NP][W2];
#pragma unroll
  for (int p = 0; p < NP; ++p) {
    float2 v[W2];
#pragma unroll
    for (int q = 0; q < W2; ++q) v[q] = Raw<Tin>::unpack(raw[p][q]);
    fft_reg<W2, -1>(v);
#pragma unroll
    for (int k2 = 1; k2 < W2; ++k2) v[k2] = cmul(v[k2], twr[k2]);
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
  for (int i = 0; i < W2 / W1; ++i)
#pragma unroll
    for (int k1 = 0; k1 < W1; ++k1) {
      const int f = t + W1 * i + W2 * k1;
      const int m = f < L ? f : f - W;
      // orders outside |m| < L go to the spare row M (never copied out)
      const int row = (m > -L && m < L) ? m + L - 1 : M;
      Tout* sp = stage + row * SP + NP * rr;
      float re[NP], im[NP];
#pragma unroll
      for (int p = 0; p < NP; ++p) {
        re[p] = spec[p][i * W1 + k1].x;
        im[p] = spec[p][i * W1 + k1].y;
      }
      StageVec<Tout, NP>::put(sp, re);
      StageVec<Tout, NP>::put(sp + JB, im);
    }
  __syncthreads();
  // X[si][mi][j0 / JT][n][ri][j0 % JT + r] with JT == JB
  const size_t tile = (size_t)NBC * 2 * JB;  // one latitude tile of one order
  stage_copy<Tout, true, JB, SP, NT>(stage, X + ((size_t)mb.si * M * (H / JB) + mb.j0 / JB) * tile,
                                     M, (size_t)(H / JB) * tile, mb.n, tid);
}

// STREAM: the output rows are written with the non-temporal hint.
template <typename Tin, typename Tout, int W1, int W2, bool STREAM>
__global__ void __launch_bounds__((DftGeom<W1, W2>::NT))
    dft_inv_kernel(const Tin* __restrict__ Y, Tout* __restrict__ y,
                   const float2* __restrict__ tw, int S, int C, int NB, int NBC, int L) {
  using G = DftGeom<W1, W2>;
  constexpr int W = G::W, H = W, NP = G::NP, JB = G::JB, NT = G::NT, RPP_ = G::RPP;
  constexpr int SP = stage_pitch<Tin, JB>();
  extern __shared__ __align__(16) unsigned char smem[];
  const int tid = threadIdx.x, t = tid % W1, rr = tid / W1;
  MapBlock mb;
  if (!map_block<JB, H>(S, C, NB, mb)) return;
  const int M = 2 * L - 1;
  // the spectrum stage [M][SP] (first) and the exchange buffer
  // [RPP][W2][W1+1] (during the FFTs) share one allocation
  Tin* stage = reinterpret_cast<Tin*>(smem);
  float2* ex = reinterpret_cast<float2*>(smem);
  // twiddles [k2][t] = tw[t k2], filled before any store of this workgroup:
  // a global load issued after the output stores would wait for them (vmcnt
  // counts stores too)
  __shared__ float2 twl[W];
  for (int i = tid; i < W; i += NT) twl[i] = tw[(i % W1) * (i / W1)];

  const size_t tile = (size_t)NBC * 2 * JB;  // one latitude tile of one order
  stage_copy<Tin, false, JB, SP, NT>(
      stage, const_cast<Tin*>(Y) + ((size_t)mb.si * M * (H / JB) + mb.j0 / JB) * tile, M,
      (size_t)(H / JB) * tile, mb.n, tid);
  __syncthreads();

  // the spectra of all passes are read into registers before the exchange
  // buffer overwrites the stage; orders outside |m| < L read row 0 and are
  // zeroed (branch-free)
  float2 v[NP][W2];
#pragma unroll
  for (int q = 0; q < W2; ++q) {
    const int f = t + W1 * q;
    const int m = f < L ? f : f - W;
    const bool ok = m > -L && m < L;
    const Tin* sp = stage + (ok ? m + L - 1 : 0) * SP + NP * rr;
    float re[NP], im[NP];
    StageVec<Tin, NP>::get(sp, re);
    StageVec<Tin, NP>::get(sp + JB, im);
#pragma unroll
    for (int p = 0; p < NP; ++p) v[p][q] = make_float2(ok ? re[p] : 0.f, ok ? im[p] : 0.f);
  }
  __syncthreads();

  const size_t row_base = ((size_t)mb.map * H + mb.j0 + NP * rr) * W;
  float2* exr = ex + (size_t)rr * W2 * (W1 + 1);
#pragma unroll
  for (int p = 0; p < NP; ++p) {
    fft_reg<W2, +1>(v[p]);
#pragma unroll
    for (int k2 = 1; k2 < W2; ++k2) v[p][k2] = cmulc(v[p][k2], twl[k2 * W1 + t]);
    if (p > 0) __syncthreads();  // the previous pass has finished reading ex
#pragma unroll
    for (int k2 = 0; k2 < W2; ++k2) exr[k2 * (W1 + 1) + t] = v[p][k2];
    __syncthreads();
    if constexpr (OutStage<Tout, W>::ON) {
      // the pass's RPP rows are staged in LDS (over the exchange buffer, once
      // every lane has read it) and leave as 16-byte vectors, whole rows
      using O = OutStage<Tout, W>;
      float2 uu[W2 / W1][W1];
#pragma unroll
      for (int i = 0; i < W2 / W1; ++i) {
        const int k2 = t + W1 * i;
#pragma unroll
        for (int tp = 0; tp < W1; ++tp) uu[i][tp] = exr[k2 * (W1 + 1) + tp];
        fft_reg<W1, +1>(uu[i]);
      }
      __syncthreads();  // every lane has read the exchange buffer
      uint32_t* os = reinterpret_cast<uint32_t*>(smem);
#pragma unroll
      for (int i = 0; i < W2 / W1; ++i)
#pragma unroll
        for (int k1 = 0; k1 < W1; ++k1)
          O::put(os + rr * O::PITCH, t + W1 * i + W2 * k1, uu[i][k1]);
      __syncthreads();
      uint32_t* yw = reinterpret_cast<uint32_t*>(y);
      for (int idx = tid; idx < RPP_ * O::VPR; idx += NT) {
        const int row = idx / O::VPR, vc = idx % O::VPR;
        const v4u_t val = *reinterpret_cast<const v4u_t*>(os + row * O::PITCH + 4 * vc);
        v4u_t* dst = reinterpret_cast<v4u_t*>(
            yw + ((size_t)mb.map * H + mb.j0 + NP * row + p) * W * O::WPC + 4 * vc);
        if constexpr (STREAM) __builtin_nontemporal_store(val, dst);
        else *dst = val;
      }
      continue;
    }
#pragma unroll
    for (int i = 0; i < W2 / W1; ++i) {
      const int k2 = t + W1 * i;
      float2 u[W1];
#pragma unroll
      for (int tp = 0; tp < W1; ++tp) u[tp] = exr[k2 * (W1 + 1) + tp];
      fft_reg<W1, +1>(u);
#pragma unroll
      for (int k1 = 0; k1 < W1; ++k1)
        store_cplx<STREAM>(y, row_base + (size_t)p * W + k2 + W2 * k1, u[k1]);
    }
  }
}

// Launches that move at least kStreamBytes (about half the 256 MB Infinity
// Cache) read their input (forward) or write their output (inverse) with the
// non-temporal hint: such a stream cannot stay cached anyway, and keeping it
// out leaves the cache to the spectrum the next stage reads (wx256: forward
// DFT 120 -> 106 us, layer 480 -> 462 us; at 33 MB (mol) the same hint costs
// 1.5-2.4x, since there everything fits).  Instantiated for W >= 128 only.
constexpr size_t kStreamBytes = size_t(128) << 20;
template <int W>
constexpr bool kHasStream = W >= 128;
template <int W>
bool streams_past_caches(size_t bytes) {
  return kHasStream<W> && bytes >= kStreamBytes;
}

template <class Kern>
hipError_t allow_lds(Kern kern, size_t lds) {
  return ensure_dynamic_lds((const void*)kern, lds);
}

template <typename Tin, typename Tout, int W1, int W2>
hipError_t launch_fwd_shape(const Plan& p, int S, int B, int C, const void* x, void* X,
                            hipStream_t st) {
  using G = DftGeom<W1, W2>;
  if (p.H != G::W || p.JT != G::JB) return hipErrorInvalidValue;
  const size_t lds = dft_lds_bytes<Tout, G>(p.M);
  const size_t bytes = (size_t)B * S * C * p.H * p.W * 2 * sizeof(Tin) + xy_elems(p, S, B, C) * sizeof(Tout);
  auto kern = streams_past_caches<W1 * W2>(bytes) ? dft_fwd_kernel<Tin, Tout, W1, W2, kHasStream<W1 * W2>>
                                                  : dft_fwd_kernel<Tin, Tout, W1, W2, false>;
  const hipError_t e = allow_lds(kern, lds);
  if (e != hipSuccess) return e;
  const long long blocks = (long long)B * S * C * (p.H / G::JB);
  hipLaunchKernelGGL(kern, dim3(xcd_grid(blocks)), dim3(G::NT), lds, st, (const Tin*)x, (Tout*)X,
                     p.twiddle, S, C, B, B * C, p.L);
  return hipGetLastError();
}

template <typename Tin, typename Tout, int W1, int W2>
hipError_t launch_inv_shape(const Plan& p, int S, int B, int C, const void* Y, void* y,
                            hipStream_t st) {
  using G = DftGeom<W1, W2>;
  if (p.H != G::W || p.JT != G::JB) return hipErrorInvalidValue;
  size_t lds = dft_lds_bytes<Tin, G>(p.M);
  using O = OutStage<Tout, G::W>;  // the output rows of a pass, staged over the same allocation
  if (O::ON && (size_t)G::RPP * O::PITCH * 4 > lds) lds = (size_t)G::RPP * O::PITCH * 4;
  const size_t bytes = xy_elems(p, S, B, C) * sizeof(Tin) + (size_t)B * S * C * p.H * p.W * 2 * sizeof(Tout);
  auto kern = streams_past_caches<W1 * W2>(bytes) ? dft_inv_kernel<Tin, Tout, W1, W2, kHasStream<W1 * W2>>
                                                  : dft_inv_kernel<Tin, Tout, W1, W2, false>;
  const hipError_t e = allow_lds(kern, lds);
  if (e != hipSuccess) return e;
  const long long blocks = (long long)B * S * C * (p.H / G::JB);
  hipLaunchKernelGGL(kern, dim3(xcd_grid(blocks)), dim3(G::NT), lds, st, (const Tin*)Y, (Tout*)y,
                     p.twiddle, S, C, B, B * C, p.L);
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
  if (p.flags & SWSFT_PLAN_DFT_MATMUL) return launch_dft_fwd_matmul(p, S, B, C, x, X, st);
  if (p.dtype == SWSFT_BF16) return dispatch_fwd<__bf16>(p, S, B, C, x, X, st);
  return dispatch_fwd<float>(p, S, B, C, x, X, st);
}

hipError_t launch_dft_inv(const Plan& p, int S, int B, int C, const void* Y, void* y,
                          hipStream_t st) {
  if (p.flags & SWSFT_PLAN_DFT_MATMUL) return launch_dft_inv_matmul(p, S, B, C, Y, y, st);
  if (p.dtype == SWSFT_BF16) return dispatch_inv<__bf16>(p, S, B, C, Y, y, st);
  return dispatch_inv<float>(p, S, B, C, Y, y, st);
}

}  // namespace swsft
