// Measurement helper, not part of the transform: the sustained rate of one
// MFMA instruction with both operands held in registers and no memory
// traffic, so that the contraction kernels can be stated against what the
// matrix units deliver on this chip besides the datasheet peak.
//
// Every wave keeps four independent accumulator chains (enough to cover the
// instruction latency with two or more waves per SIMD) and runs `iters`
// rounds of four MFMAs.  With random operands the registers hold bf16 / f32
// values with random signs and mantissas in [0.5, 2); with constant operands
// every value is 1.  The chip lowers its clock under the switching activity
// of random data, so the two rates differ.  Each lane writes one float (the
// sum of its accumulators) so that nothing is eliminated.
#include "mfma_tile.h"
#include "swsft_internal.h"

namespace swsft {
namespace {

__device__ __forceinline__ unsigned hash32(unsigned x) {
  x ^= x >> 16;
  x *= 0x7feb352du;
  x ^= x >> 15;
  x *= 0x846ca68bu;
  x ^= x >> 16;
  return x;
}

// two bf16 values with random signs and mantissas in [0.5, 2), or 1.0 twice
__device__ __forceinline__ unsigned bf16_pair(unsigned h, bool random) {
  if (!random) return 0x3f803f80u;
  const unsigned lo = (h & 0x807fu) | (((h >> 7) & 1u) ? 0x3f80u : 0x3f00u);
  const unsigned hi = ((h >> 16) & 0x807fu) | (((h >> 23) & 1u) ? 0x3f80u : 0x3f00u);
  return lo | (hi << 16);
}

__device__ __forceinline__ float f32_value(unsigned h, bool random) {
  if (!random) return 1.f;
  const unsigned bits = (h & 0x807fffffu) | (((h >> 23) & 1u) ? 0x3f800000u : 0x3f000000u);
  return __uint_as_float(bits);
}

typedef unsigned v4u __attribute__((ext_vector_type(4)));

template <bool BF16>
__global__ void __launch_bounds__(256) mfma_probe_kernel(float* __restrict__ out, long long iters,
                                                         int random) {
  const unsigned id = blockIdx.x * 256u + threadIdx.x;
  const bool rnd = random != 0;
  v16f acc[4];
#pragma unroll
  for (int c = 0; c < 4; ++c)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[c][r] = 0.f;
  if constexpr (BF16) {
    v8bf a[2], b[2];
#pragma unroll
    for (int o = 0; o < 2; ++o) {
      v4u va, vb;
#pragma unroll
      for (int d = 0; d < 4; ++d) {
        va[d] = bf16_pair(hash32(id * 16u + o * 8u + d), rnd);
        vb[d] = bf16_pair(hash32(id * 16u + o * 8u + 4u + d), rnd);
      }
      a[o] = __builtin_bit_cast(v8bf, va);
      b[o] = __builtin_bit_cast(v8bf, vb);
    }
    for (long long it = 0; it < iters; ++it) {
      acc[0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[0], b[0], acc[0], 0, 0, 0);
      acc[1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[1], b[0], acc[1], 0, 0, 0);
      acc[2] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[0], b[1], acc[2], 0, 0, 0);
      acc[3] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[1], b[1], acc[3], 0, 0, 0);
    }
  } else {
    const float a0 = f32_value(hash32(id * 4u), rnd), a1 = f32_value(hash32(id * 4u + 1u), rnd);
    const float b0 = f32_value(hash32(id * 4u + 2u), rnd), b1 = f32_value(hash32(id * 4u + 3u), rnd);
    for (long long it = 0; it < iters; ++it) {
      acc[0] = __builtin_amdgcn_mfma_f32_32x32x2f32(a0, b0, acc[0], 0, 0, 0);
      acc[1] = __builtin_amdgcn_mfma_f32_32x32x2f32(a1, b0, acc[1], 0, 0, 0);
      acc[2] = __builtin_amdgcn_mfma_f32_32x32x2f32(a0, b1, acc[2], 0, 0, 0);
      acc[3] = __builtin_amdgcn_mfma_f32_32x32x2f32(a1, b1, acc[3], 0, 0, 0);
    }
  }
  float s = 0.f;
#pragma unroll
  for (int c = 0; c < 4; ++c)
#pragma unroll
    for (int r = 0; r < 16; ++r) s += acc[c][r];
  out[id] = s;
}

}  // namespace

double mfma_probe_flops_per_wave_round(int dtype) {
  // four MFMAs per round: 32x32x16 bf16 (32768 flops) or 32x32x2 f32 (4096)
  return dtype == SWSFT_BF16 ? 4.0 * 2 * 32 * 32 * 16 : 4.0 * 2 * 32 * 32 * 2;
}

hipError_t launch_mfma_probe(int dtype, int random, long long iters, int n_waves, float* out,
                             hipStream_t st) {
  const unsigned blocks = (unsigned)(n_waves / 4);
  if (dtype == SWSFT_BF16)
    hipLaunchKernelGGL(mfma_probe_kernel<true>, dim3(blocks), dim3(256), 0, st, out, iters, random);
  else
    hipLaunchKernelGGL(mfma_probe_kernel<false>, dim3(blocks), dim3(256), 0, st, out, iters, random);
  return hipGetLastError();
}

}  // namespace swsft
