// Spectral batch normalization (Method, "Spectral batch normalization") on
// coefficients [L^2][B][S][C] (row l^2 + l + m, then batch, spin, channel).
//
// The l = 0 coefficient is the function's mean (times sqrt(4 pi)); by
// Parseval the other coefficients carry its variance.  Per (spin, channel):
//   var   = (1 / (4 pi B)) sum_{b, l >= 1, m} |a|^2    (batch statistics), or given,
//   out   = gamma a / sqrt(var + eps)                    for l >= 1,
//   out_0 = beta (spin 0; 0 for other spins)             for l = 0,
//   out  += skip                                         (optional).
//
// Three launches, all deterministic (no atomics):
//   bn_partial   each workgroup sums |a|^2 over a fixed range of rows for
//                every column (threads across a row: coalesced);
//   bn_finalize  per column: the partial sums in a fixed order -> var, scale;
//   bn_apply     elementwise, 4 complex values per thread.
#include "swsft_internal.h"

namespace swsft {
namespace {

constexpr int kNT = 256;
constexpr float kInv4Pi = 0.0795774715459476679f;  // 1 / (4 pi)

template <typename T>
__device__ __forceinline__ float2 ld_c(const T* p, size_t i) {
  return make_float2((float)p[2 * i], (float)p[2 * i + 1]);
}

// Threads are (row lane, column lane): TPR = min(ncol, 256) rounded down to a
// power of two threads share a row, 256 / TPR rows are read at once, and
// each thread keeps the sums of its columns (col, col + TPR, ...) in
// registers; the row lanes are combined through LDS at the end.
constexpr int kMaxColsPerThread = 8;

template <typename T>
__global__ void __launch_bounds__(kNT) bn_partial_kernel(const T* __restrict__ a,
                                                         float* __restrict__ partial, int rows,
                                                         int row_begin, int rows_per_blk, int ncol,
                                                         int tpr) {
  __shared__ float red[kNT * kMaxColsPerThread];
  const int rl = threadIdx.x / tpr, cl = threadIdx.x % tpr;
  const int rsub = kNT / tpr;
  const int ncpt = (ncol + tpr - 1) / tpr;  // columns per thread (<= kMaxColsPerThread)
  const int r0 = row_begin + blockIdx.x * rows_per_blk;
  const int r1 = min(r0 + rows_per_blk, rows);
  float acc[kMaxColsPerThread];
#pragma unroll
  for (int j = 0; j < kMaxColsPerThread; ++j) acc[j] = 0.f;
  int r = r0 + rl;
  // four rows in flight per thread
  for (; r + 3 * rsub < r1; r += 4 * rsub) {
#pragma unroll
    for (int j = 0; j < kMaxColsPerThread; ++j) {
      const int col = cl + j * tpr;
      if (j < ncpt && col < ncol) {
        const float2 v0 = ld_c(a, (size_t)r * ncol + col);
        const float2 v1 = ld_c(a, (size_t)(r + rsub) * ncol + col);
        const float2 v2 = ld_c(a, (size_t)(r + 2 * rsub) * ncol + col);
        const float2 v3 = ld_c(a, (size_t)(r + 3 * rsub) * ncol + col);
        acc[j] += (v0.x * v0.x + v0.y * v0.y) + (v1.x * v1.x + v1.y * v1.y) +
                  (v2.x * v2.x + v2.y * v2.y) + (v3.x * v3.x + v3.y * v3.y);
      }
    }
  }
  for (; r < r1; r += rsub) {
#pragma unroll
    for (int j = 0; j < kMaxColsPerThread; ++j) {
      const int col = cl + j * tpr;
      if (j < ncpt && col < ncol) {
        const float2 v = ld_c(a, (size_t)r * ncol + col);
        acc[j] += v.x * v.x + v.y * v.y;
      }
    }
  }
#pragma unroll
  for (int j = 0; j < kMaxColsPerThread; ++j) red[j * kNT + threadIdx.x] = acc[j];
  __syncthreads();
  // thread (rl = 0, cl) sums the row lanes of its columns in a fixed order
  if (rl == 0) {
    for (int j = 0; j < ncpt; ++j) {
      const int col = cl + j * tpr;
      if (col >= ncol) break;
      float sum = 0.f;
      for (int q = 0; q < rsub; ++q) sum += red[j * kNT + q * tpr + cl];
      partial[(size_t)blockIdx.x * ncol + col] = sum;
    }
  }
}

// One workgroup per 32 columns: 8 lanes per column sum the partial rows
// b = lane, lane + 8, ... (four loads in flight), then lane 0 adds the 8
// lane sums in order.
__global__ void __launch_bounds__(kNT) bn_finalize_kernel(const float* __restrict__ partial,
                                                          int nblk, int ncol, float inv_norm,
                                                          const float* __restrict__ var_in,
                                                          const float* __restrict__ gamma,
                                                          float eps, float* __restrict__ scale,
                                                          float* __restrict__ var_out) {
  __shared__ float red[kNT];
  const int lane = threadIdx.x / 32, cc = threadIdx.x % 32;
  const int col = blockIdx.x * 32 + cc;
  float acc = 0.f;
  if (var_in == nullptr && col < ncol) {
    float a0 = 0.f, a1 = 0.f, a2 = 0.f, a3 = 0.f;
    int b = lane;
    for (; b + 24 < nblk; b += 32) {
      a0 += partial[(size_t)b * ncol + col];
      a1 += partial[(size_t)(b + 8) * ncol + col];
      a2 += partial[(size_t)(b + 16) * ncol + col];
      a3 += partial[(size_t)(b + 24) * ncol + col];
    }
    for (; b < nblk; b += 8) a0 += partial[(size_t)b * ncol + col];
    acc = (a0 + a1) + (a2 + a3);
  }
  red[threadIdx.x] = acc;
  __syncthreads();
  if (lane != 0 || col >= ncol) return;
  float var;
  if (var_in != nullptr) {
    var = var_in[col];
  } else {
    float sum = 0.f;
    for (int q = 0; q < kNT / 32; ++q) sum += red[q * 32 + cc];
    var = sum * inv_norm;
  }
  scale[col] = gamma[col] / sqrtf(var + eps);
  if (var_out != nullptr) var_out[col] = var;
}

// 4 whole complex values as one 16-byte (bf16) or two 16-byte (float)
// accesses; n < 4 values fall back to element accesses
template <typename T>
__device__ __forceinline__ void ld4(const T* p, long long i0, int n, float2 (&v)[4]) {
  if (n == 4) {
    if constexpr (sizeof(T) == 4) {
      const float4 u = *reinterpret_cast<const float4*>(p + 2 * i0);
      const float4 w = *reinterpret_cast<const float4*>(p + 2 * i0 + 4);
      v[0] = make_float2(u.x, u.y); v[1] = make_float2(u.z, u.w);
      v[2] = make_float2(w.x, w.y); v[3] = make_float2(w.z, w.w);
    } else {
      typedef __bf16 v8b __attribute__((ext_vector_type(8)));
      const v8b u = *reinterpret_cast<const v8b*>(p + 2 * i0);
#pragma unroll
      for (int e = 0; e < 4; ++e) v[e] = make_float2((float)u[2 * e], (float)u[2 * e + 1]);
    }
  } else {
    // constant indices only (a runtime bound would put the array in memory)
#pragma unroll
    for (int e = 0; e < 4; ++e) v[e] = e < n ? ld_c(p, i0 + e) : make_float2(0.f, 0.f);
  }
}

template <typename T>
__device__ __forceinline__ void st4(T* p, long long i0, int n, const float2 (&v)[4]) {
  if (n == 4) {
    if constexpr (sizeof(T) == 4) {
      *reinterpret_cast<float4*>(p + 2 * i0) = make_float4(v[0].x, v[0].y, v[1].x, v[1].y);
      *reinterpret_cast<float4*>(p + 2 * i0 + 4) = make_float4(v[2].x, v[2].y, v[3].x, v[3].y);
    } else {
      typedef __bf16 v8b __attribute__((ext_vector_type(8)));
      v8b u;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        u[2 * e] = (__bf16)v[e].x;
        u[2 * e + 1] = (__bf16)v[e].y;
      }
      *reinterpret_cast<v8b*>(p + 2 * i0) = u;
    }
  } else {
#pragma unroll
    for (int e = 0; e < 4; ++e)
      if (e < n) {
        p[2 * (i0 + e)] = (T)v[e].x;
        p[2 * (i0 + e) + 1] = (T)v[e].y;
      }
  }
}

// rows [0, B) are degree 0; columns are (spin, channel), s0 the spin-0 slot or -1
template <typename T>
__global__ void __launch_bounds__(kNT) bn_apply_kernel(const T* a,  // may be out (in place)
                                                       const float* __restrict__ scale,
                                                       const float2* __restrict__ beta,
                                                       const T* skip, T* out,
                                                       long long n_cplx, int ncol, int C, int B,
                                                       int s0) {
  const long long i0 = ((long long)blockIdx.x * kNT + threadIdx.x) * 4;
  if (i0 >= n_cplx) return;
  const int n = n_cplx - i0 < 4 ? (int)(n_cplx - i0) : 4;
  float2 v[4], k[4];
  ld4(a, i0, n, v);
  if (skip != nullptr) ld4(skip, i0, n, k);
  float2 o[4];
  long long row = i0 / ncol;
  int col = (int)(i0 - row * ncol);
#pragma unroll
  for (int e = 0; e < 4; ++e, ++col) {
    if (col == ncol) {
      col = 0;
      ++row;
    }
    if (row < B) {  // degree 0: the bias for spin 0, else 0
      o[e] = (col / C == s0 && beta != nullptr) ? beta[col % C] : make_float2(0.f, 0.f);
    } else {
      const float sc = scale[col];
      o[e] = make_float2(v[e].x * sc, v[e].y * sc);
    }
    if (skip != nullptr) {
      o[e].x += k[e].x;
      o[e].y += k[e].y;
    }
  }
  st4(out, i0, n, o);
}

}  // namespace

int bn_partial_blocks(const Plan& p, int B) {
  const int rows = p.L * p.L * B - B;  // rows of degrees l >= 1
  int nblk = (rows + 63) / 64;         // at least 64 rows per workgroup
  return nblk < 1 ? 1 : (nblk > 256 ? 256 : nblk);
}

// threads per row: the largest power of two <= min(ncol, 256) that leaves
// at most kMaxColsPerThread columns per thread
int bn_threads_per_row(int ncol) {
  int t = 1;
  while (t * 2 <= ncol && t * 2 <= kNT) t *= 2;
  return t;
}

bool bn_supported(const Plan& p, int C) {
  const int ncol = p.n_out * C;
  return (ncol + bn_threads_per_row(ncol) - 1) / bn_threads_per_row(ncol) <= kMaxColsPerThread;
}

size_t bn_workspace_bytes(const Plan& p, int B, int C) {
  const int ncol = p.n_out * C;
  return ((size_t)bn_partial_blocks(p, B) * ncol + ncol) * sizeof(float);
}

template <typename T>
hipError_t bn_t(const Plan& p, int B, int C, const void* a, const float* gamma,
                const float2* beta, float eps, const float* var_in, float* var_out,
                const void* skip, void* out, float* ws, hipStream_t st) {
  const int ncol = p.n_out * C;
  const int rows = p.L * p.L * B;
  const int nblk = bn_partial_blocks(p, B);
  float* partial = ws;
  float* scale = ws + (size_t)nblk * ncol;
  if (var_in == nullptr) {
    const int body = rows - B;
    const int per = (body + nblk - 1) / nblk;
    hipLaunchKernelGGL(bn_partial_kernel<T>, dim3(nblk), dim3(kNT), 0, st, (const T*)a, partial,
                       rows, B, per, ncol, bn_threads_per_row(ncol));
  }
  hipLaunchKernelGGL(bn_finalize_kernel, dim3((ncol + 31) / 32), dim3(kNT), 0, st, partial,
                     nblk, ncol, kInv4Pi / (float)B, var_in, gamma, eps, scale, var_out);
  int s0 = -1;
  for (int i = 0; i < p.n_out; ++i)
    if (p.spins_out[i] == 0) s0 = i;
  const long long n = (long long)rows * ncol;
  const long long grid = (n + 4LL * kNT - 1) / (4LL * kNT);
  hipLaunchKernelGGL(bn_apply_kernel<T>, dim3((unsigned)grid), dim3(kNT), 0, st, (const T*)a, scale,
                     beta, (const T*)skip, (T*)out, n, ncol, C, B, s0);
  return hipGetLastError();
}

hipError_t launch_batch_norm(const Plan& p, int B, int C, const void* a, const float* gamma,
                             const float2* beta, float eps, const float* var_in, float* var_out,
                             const void* skip, void* out, void* ws, hipStream_t st) {
  if (p.dtype == SWSFT_BF16)
    return bn_t<__bf16>(p, B, C, a, gamma, beta, eps, var_in, var_out, skip, out, (float*)ws, st);
  return bn_t<float>(p, B, C, a, gamma, beta, eps, var_in, var_out, skip, out, (float*)ws, st);
}

}  // namespace swsft
