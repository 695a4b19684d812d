// Phase-collapse nonlinearity (Method, "Phase collapse nonlinearity"):
// at every grid point, x0 <- W1 x0 + W2 |x| + b over the C spin-0 channels;
// |x| stacks the moduli of all S*C channels in (spin, channel) order.  The
// other spins pass through unchanged.
//
// One workgroup owns 64 consecutive grid points of one batch item: it stages
// the spin-0 values and the moduli of every channel in LDS (each input
// element is read once), then produces the outputs of those points (below,
// as an MFMA GEMM when C is a multiple of 16).  x and y may be the same
// buffer: a workgroup reads all of its points before writing any.
#include "mfma_tile.h"
#include "swsft_internal.h"

namespace swsft {
namespace {

constexpr int PB = 64;   // grid points per workgroup
constexpr int NTP = 256;

template <typename T>
__device__ __forceinline__ float2 ld2(const T* p, size_t i) {
  return make_float2((float)p[2 * i], (float)p[2 * i + 1]);
}

template <typename T>
__global__ void __launch_bounds__(NTP) phase_collapse_kernel(
    const T* x, const float2* __restrict__ W1, const float2* __restrict__ W2,
    const float2* __restrict__ bias, T* y, int S, int C, int HW, int s0,
    int copy_others) {
  extern __shared__ __align__(16) unsigned char smem[];
  float2* z0 = reinterpret_cast<float2*>(smem);                // [C][PB]
  float* mag = reinterpret_cast<float*>(z0 + (size_t)C * PB);  // [S*C][PB]
  const int b = blockIdx.y;
  const int p0 = blockIdx.x * PB;
  const int np = HW - p0 < PB ? HW - p0 : PB;
  const int tid = threadIdx.x;
  const size_t map0 = (size_t)b * S * C;  // first map of this batch item
  for (int idx = tid; idx < S * C * PB; idx += NTP) {
    const int p = idx % PB;
    const int sc = idx / PB;
    if (p < np) {
      const size_t e = (map0 + sc) * HW + p0 + p;
      const float2 v = ld2(x, e);
      mag[sc * PB + p] = sqrtf(v.x * v.x + v.y * v.y);
      const int s = sc / C;
      if (s == s0) z0[(sc - s0 * C) * PB + p] = v;
      else if (copy_others) {
        y[2 * e] = x[2 * e];
        y[2 * e + 1] = x[2 * e + 1];
      }
    }
  }
  __syncthreads();
  const int SC = S * C;
  for (int idx = tid; idx < C * PB; idx += NTP) {
    const int p = idx % PB;
    const int co = idx / PB;
    if (p >= np) continue;
    float2 acc = bias[co];
    const float2* w1 = W1 + (size_t)co * C;
    for (int c = 0; c < C; ++c) {
      const float2 w = w1[c], z = z0[c * PB + p];
      acc.x += w.x * z.x - w.y * z.y;
      acc.y += w.x * z.y + w.y * z.x;
    }
    const float2* w2 = W2 + (size_t)co * SC;
    for (int sc = 0; sc < SC; ++sc) {
      const float a = mag[sc * PB + p];
      acc.x += w2[sc].x * a;
      acc.y += w2[sc].y * a;
    }
    const size_t e = (map0 + (size_t)s0 * C + co) * HW + p0 + p;
    y[2 * e] = (T)acc.x;
    y[2 * e + 1] = (T)acc.y;
  }
}

// MFMA form (C a multiple of 16): per workgroup of PM points, the real GEMM
//   out[2C][PM] = A[2C][K] . Z[K][PM],  K = 2C + S C,
// with Z = [Re z0; Im z0; |x|] staged in LDS (float) and the output rows
// (2 co + re/im) built from W1, W2 in the A operand:
//   row 2co:   [ Re W1[co][:], -Im W1[co][:], Re W2[co][:] ]
//   row 2co+1: [ Im W1[co][:],  Re W1[co][:], Im W2[co][:] ]
// v_mfma_f32_32x32x2f32: each wave owns 32 output rows and PM = 64 points
// (two 32-column tiles); the A values come from L2 one float per lane per
// step.  Z row k keeps its two 32-point halves rotated by 32 (k odd), so the
// two half-waves (rows k and k + 1) read different banks.
constexpr int PM = 64;

__device__ __forceinline__ int zcol(int k, int p) { return (p + ((k & 1) << 5)) & (PM - 1); }

template <typename T>
__global__ void __launch_bounds__(NTP) phase_collapse_mfma_kernel(
    const T* x, const float* __restrict__ W1, const float* __restrict__ W2,
    const float2* __restrict__ bias, T* y, int S, int C, int HW, int s0, int copy_others) {
  extern __shared__ __align__(16) float zs[];  // [K][PM]
  const int K = 2 * C + S * C, SC = S * C;
  const int b = blockIdx.y;
  const int p0 = blockIdx.x * PM;
  const int np = HW - p0 < PM ? HW - p0 : PM;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const size_t map0 = (size_t)b * S * C;
  // staging: SB loads in flight per thread before any of them is used
  constexpr int SB = 8;
  for (int base = 0; base < SC * PM; base += SB * NTP) {
    float2 v[SB];
#pragma unroll
    for (int u = 0; u < SB; ++u) {
      const int idx = base + u * NTP + tid;
      const int p = idx % PM, sc = idx / PM;
      v[u] = make_float2(0.f, 0.f);  // points past the end stage zeros
      if (idx < SC * PM && p < np) v[u] = ld2(x, (map0 + sc) * HW + p0 + p);
    }
#pragma unroll
    for (int u = 0; u < SB; ++u) {
      const int idx = base + u * NTP + tid;
      if (idx >= SC * PM) break;
      const int p = idx % PM, sc = idx / PM;
      zs[(2 * C + sc) * PM + zcol(2 * C + sc, p)] = sqrtf(v[u].x * v[u].x + v[u].y * v[u].y);
      const int s = sc / C;
      if (s == s0) {
        const int c = sc - s0 * C;
        zs[c * PM + zcol(c, p)] = v[u].x;
        zs[(C + c) * PM + zcol(C + c, p)] = v[u].y;
      } else if (copy_others && p < np) {
        const size_t e = (map0 + sc) * HW + p0 + p;
        y[2 * e] = (T)v[u].x;
        y[2 * e + 1] = (T)v[u].y;
      }
    }
  }
  __syncthreads();
  const int r32 = lane & 31, kh = lane >> 5;
  const int n_tiles = (2 * C) / 32;
  for (int rt = wave; rt < n_tiles; rt += NTP / 64) {
    const int m = rt * 32 + r32;  // this lane's A row
    const int co = m >> 1, ri = m & 1;
    v16f acc[2];
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[j][r] = 0.f;
    auto step = [&](int k, float a) {
      const float b0 = zs[k * PM + zcol(k, r32)];
      const float b1 = zs[k * PM + zcol(k, 32 + r32)];
      acc[0] = __builtin_amdgcn_mfma_f32_32x32x2f32(a, b0, acc[0], 0, 0, 0);
      acc[1] = __builtin_amdgcn_mfma_f32_32x32x2f32(a, b1, acc[1], 0, 0, 0);
    };
    // K runs over three regions (Re z0, Im z0, moduli), each a multiple of 16
    // long; a batch of U = 8 steps (16 k) lies inside one region, and the
    // next batch's A values are loaded before the current batch's MFMAs
    constexpr int U = 8;
    const int nb = K / (2 * U);
    auto load_batch = [&](int bi, float (&a)[U]) {
      const int k0 = bi * 2 * U;
      const float* w;
      float sgn = 1.f;
      int kk;
      if (k0 < C) {
        w = W1 + (size_t)co * C * 2 + ri;
        kk = k0;
      } else if (k0 < 2 * C) {  // row 2co takes -Im W1, row 2co+1 takes Re W1
        w = W1 + (size_t)co * C * 2 + (1 - ri);
        sgn = ri ? 1.f : -1.f;
        kk = k0 - C;
      } else {
        w = W2 + (size_t)co * SC * 2 + ri;
        kk = k0 - 2 * C;
      }
#pragma unroll
      for (int u = 0; u < U; ++u) a[u] = sgn * w[(size_t)(kk + 2 * u + kh) * 2];
    };
    float acur[U], anxt[U];
    load_batch(0, acur);
    for (int bi = 0; bi < nb; ++bi) {
      if (bi + 1 < nb) load_batch(bi + 1, anxt);
#pragma unroll
      for (int u = 0; u < U; ++u) step(bi * 2 * U + 2 * u + kh, acur[u]);
#pragma unroll
      for (int u = 0; u < U; ++u) acur[u] = anxt[u];
    }
    // rows (2co, 2co+1) of a column are registers (r, r+1), r even
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int p = j * 32 + r32;
      if (p >= np) continue;
#pragma unroll
      for (int r = 0; r < 16; r += 2) {
        const int row = rt * 32 + 8 * (r >> 2) + 4 * kh + (r & 3);
        const int c_out = row >> 1;
        const float2 bb = bias[c_out];
        const size_t e = (map0 + (size_t)s0 * C + c_out) * HW + p0 + p;
        y[2 * e] = (T)(acc[j][r] + bb.x);
        y[2 * e + 1] = (T)(acc[j][r + 1] + bb.y);
      }
    }
  }
}

template <typename T>
hipError_t launch_t(const Plan& p, int B, int C, const void* x, const float2* W1,
                    const float2* W2, const float2* bias, void* y, hipStream_t st, int s0) {
  const int HW = p.H * p.W;
  if (C % 16 == 0) {
    const size_t lds = (size_t)(2 * C + p.n_out * C) * PM * sizeof(float);
    auto kern = phase_collapse_mfma_kernel<T>;
    const hipError_t e = ensure_dynamic_lds((const void*)kern, lds);
    if (e != hipSuccess) return e;
    dim3 grid((HW + PM - 1) / PM, B);
    hipLaunchKernelGGL(kern, grid, dim3(NTP), lds, st, (const T*)x, (const float*)W1,
                       (const float*)W2, bias, (T*)y, p.n_out, C, HW, s0, x != y ? 1 : 0);
    return hipGetLastError();
  }
  const size_t lds = (size_t)C * PB * sizeof(float2) + (size_t)p.n_out * C * PB * sizeof(float);
  auto kern = phase_collapse_kernel<T>;
  const hipError_t e = ensure_dynamic_lds((const void*)kern, lds);
  if (e != hipSuccess) return e;
  dim3 grid((HW + PB - 1) / PB, B);
  hipLaunchKernelGGL(kern, grid, dim3(NTP), lds, st, (const T*)x, W1, W2, bias, (T*)y, p.n_out, C,
                     HW, s0, x != y ? 1 : 0);
  return hipGetLastError();
}

}  // namespace

// Largest channel count whose staging fits the 160 KiB LDS of a CU.
int phase_collapse_max_channels(int n_spins) {
  const int per_c = PB * (int)sizeof(float2) + n_spins * PB * (int)sizeof(float);
  return (160 * 1024) / per_c;
}

hipError_t launch_phase_collapse(const Plan& p, int B, int C, const void* x, const float2* W1,
                                 const float2* W2, const float2* bias, void* y,
                                 hipStream_t st) {
  int s0 = -1;
  for (int i = 0; i < p.n_out; ++i)
    if (p.spins_out[i] == 0) s0 = i;
  if (p.dtype == SWSFT_BF16) return launch_t<__bf16>(p, B, C, x, W1, W2, bias, y, st, s0);
  return launch_t<float>(p, B, C, x, W1, W2, bias, y, st, s0);
}

}  // namespace swsft
