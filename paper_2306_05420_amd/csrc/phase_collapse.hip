// Phase-collapse nonlinearity (Method, "Phase collapse nonlinearity"):
// at every grid point, x0 <- W1 x0 + W2 |x| + b over the C spin-0 channels;
// |x| stacks the moduli of all S*C channels in (spin, channel) order.  The
// other spins pass through unchanged.
//
// One workgroup owns PB consecutive grid points of one batch item: it stages
// the spin-0 values and the moduli of every channel in LDS (each input
// element is read once), then each thread produces outputs (c_out, point)
// with the point index fastest, so global reads and writes are coalesced and
// the weights are wave-uniform broadcasts.  x and y may be the same buffer:
// a workgroup reads all of its points before writing any.
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

template <typename T>
hipError_t launch_t(const Plan& p, int B, int C, const void* x, const float2* W1,
                    const float2* W2, const float2* bias, void* y, hipStream_t st, int s0) {
  const int HW = p.H * p.W;
  const size_t lds = (size_t)C * PB * sizeof(float2) + (size_t)p.n_out * C * PB * sizeof(float);
  auto kern = phase_collapse_kernel<T>;
  if (lds > 64 * 1024) {
    const hipError_t e = hipFuncSetAttribute((const void*)kern,
                                             hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
  }
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
