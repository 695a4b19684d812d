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
    // the biases of this lane's output rows, loaded before the stores start
    // (a load after them would wait for them: memory operations complete in
    // issue order)
    float2 bb[8];
#pragma unroll
    for (int r = 0; r < 16; r += 2) bb[r >> 1] = bias[(rt * 32 + 8 * (r >> 2) + 4 * kh + (r & 3)) >> 1];
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
        const size_t e = (map0 + (size_t)s0 * C + c_out) * HW + p0 + p;
        y[2 * e] = (T)(acc[j][r] + bb[r >> 1].x);
        y[2 * e + 1] = (T)(acc[j][r + 1] + bb[r >> 1].y);
      }
    }
  }
}

// Register form (C in {16, 32, 48, 64}, C + S C / 2 <= 128): one wave per 32
// grid points of one batch item, all 2C output rows.  Each lane loads the
// values of its point (lane % 32) for the channels of parity lane / 32
// straight into registers -- the B operand of v_mfma_f32_32x32x2f32 for
// Z = [Re z0; Im z0; |x|] -- so the input is read once, coalesced, and a wave
// holds all its inputs before it writes (x and y may be the same buffer).
// The moduli rows of Z take spin 0 first, then the other spins in order (a
// relabelling of the contraction index, applied to the W2 columns as well),
// so every register's channel is known at compile time.  The A operand (the
// rows 2co, 2co+1 above) is packed into LDS once per workgroup in the order
// the MFMA steps read it: float4 slot [row tile][step / 4][lane ^ (step / 4 %
// 16)] holds four consecutive steps.  Workgroups are persistent over the
// tiles of 32 points.
template <typename T>
__device__ __forceinline__ float2 ld_c2(const T* p) {
  if constexpr (sizeof(T) == 4) {
    return *reinterpret_cast<const float2*>(p);
  } else {
    typedef __bf16 b2 __attribute__((ext_vector_type(2)));
    const b2 v = *reinterpret_cast<const b2*>(p);
    return make_float2((float)v[0], (float)v[1]);
  }
}

template <typename T>
__device__ __forceinline__ void st_c2(T* p, float re, float im) {
  if constexpr (sizeof(T) == 4) {
    *reinterpret_cast<float2*>(p) = make_float2(re, im);
  } else {
    typedef __bf16 b2 __attribute__((ext_vector_type(2)));
    b2 v;
    v[0] = (__bf16)re;
    v[1] = (__bf16)im;
    *reinterpret_cast<b2*>(p) = v;
  }
}

// Registers per lane: Z (C + S C / 2), the next task's raw values (S C),
// the accumulators (C) and the A operands in flight.  Shapes above 200 run
// one wave per SIMD (workgroups of 4 waves) and so have the whole register
// file, accumulation registers included.
constexpr int reg_max_threads(int C, int S) { return 2 * C + 3 * S * C / 2 + C / 2 > 200 ? 256 : 512; }

template <typename T, int C, int S>
__global__ void __launch_bounds__(reg_max_threads(C, S)) phase_collapse_reg_kernel(
    const T* x, const float2* __restrict__ W1, const float2* __restrict__ W2,
    const float2* __restrict__ bias, T* y, int B, int HW, int s0, int copy_others) {
  constexpr int SC = S * C, K = 2 * C + SC, KS = K / 2, KQ = KS / 4, RT = 2 * C / 32;
  static_assert(C % 16 == 0 && KS % 4 == 0, "shape");
  extern __shared__ __align__(16) float4 apk[];  // [RT][KQ][64], then the bias
  float2* bsh = reinterpret_cast<float2*>(apk + RT * KQ * 64);  // [C]
  const int tid = threadIdx.x, lane = tid & 63;
  const int nt = blockDim.x, nw = nt >> 6;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int r32 = lane & 31, kh = lane >> 5;
  const int tiles_b = (HW + 31) >> 5;
  const int ntask = B * tiles_b;
  const size_t cs = 2 * (size_t)HW;  // elements from one channel to the next
  // spin slot of the i-th moduli block: spin 0 first, then the others in order
  auto slot_of = [&](int i) { return i == 0 ? s0 : (i - 1 < s0 ? i - 1 : i); };

  // raw values of this lane's point: channel 2 j + kh of spin slot i
  float2 v[S][C / 2];
  auto issue_loads = [&](int t) {
    const int b = t / tiles_b;  // wave-uniform: channel bases are scalar
    const int p = (t - b * tiles_b) * 32 + r32;
    const bool ok = p < HW;
    const unsigned lo = 2u * (unsigned)(kh * HW + (ok ? p : 0));  // lane offset
    const T* xb = x + (size_t)b * SC * cs + lo;
#pragma unroll
    for (int i = 0; i < S; ++i) {
      const int sp = slot_of(i);
#pragma unroll
      for (int j = 0; j < C / 2; ++j)
        v[i][j] = ok ? ld_c2(xb + (size_t)(sp * C + 2 * j) * cs) : make_float2(0.f, 0.f);
    }
  };
  // pack A.  Work item = (co, eight consecutive complex entries of row co of
  // W1 or of W2): a W1 chunk gives the Re z0 and the Im z0 columns, a W2
  // chunk the moduli columns.  All of a thread's items are loaded first, then
  // the first task's inputs are issued, then the items are written to LDS
  // (memory returns in issue order: this keeps the inputs in flight).
  constexpr int CH1 = C / 8, CH = C / 8 + SC / 8;  // chunks per co: W1, all
  constexpr int NITEM = C * CH;
  constexpr int U = (NITEM + 255) / 256;  // items per thread (>= 256 threads)
  float2 w[U][8];
#pragma unroll
  for (int u = 0; u < U; ++u) {
    const int it = u * nt + tid;
    const int co = it / CH, ch = it - co * CH;
    const float2* src;
    if (ch < CH1) {
      src = W1 + (size_t)co * C + 8 * ch;
    } else {
      const int r0 = 8 * (ch - CH1);  // relabelled moduli column
      src = W2 + (size_t)co * SC + slot_of(r0 / C) * C + (r0 % C);
    }
#pragma unroll
    for (int e = 0; e < 8; ++e) w[u][e] = it < NITEM ? src[e] : make_float2(0.f, 0.f);
  }
  // the bias goes to LDS: an epilogue read of global memory would wait for
  // the stores before it (memory operations complete in issue order)
  const float2 bias_t = tid < C ? bias[tid] : make_float2(0.f, 0.f);
  int task = blockIdx.x * nw + wave;
  if (task < ntask) issue_loads(task);
  __builtin_amdgcn_sched_barrier(0);
  if (tid < C) bsh[tid] = bias_t;
  {
    auto put = [&](int m, int k0, const float (&a)[8]) {  // A[m][k0 .. k0 + 8)
      const int q = k0 >> 3, rt = m >> 5, rr = m & 31;
      float4* row = apk + (size_t)(rt * KQ + q) * 64;
      row[rr ^ (q & 15)] = make_float4(a[0], a[2], a[4], a[6]);
      row[(rr + 32) ^ (q & 15)] = make_float4(a[1], a[3], a[5], a[7]);
    };
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int it = u * nt + tid;
      if (it >= NITEM) break;
      const int co = it / CH, ch = it - co * CH;
      float re[8], im[8], nim[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        re[e] = w[u][e].x;
        im[e] = w[u][e].y;
        nim[e] = -w[u][e].y;
      }
      if (ch < CH1) {
        put(2 * co, 8 * ch, re);  // row 2co:   Re W1 | -Im W1
        put(2 * co, C + 8 * ch, nim);
        put(2 * co + 1, 8 * ch, im);  // row 2co+1: Im W1 |  Re W1
        put(2 * co + 1, C + 8 * ch, re);
      } else {
        const int k0 = 2 * C + 8 * (ch - CH1);
        put(2 * co, k0, re);  // Re W2 | Im W2
        put(2 * co + 1, k0, im);
      }
    }
  }
  __syncthreads();

  float zr[C / 2], zi[C / 2], mg[SC / 2];
  auto lda = [&](int rt, int q) { return apk[(size_t)(rt * KQ + q) * 64 + (lane ^ (q & 15))]; };
  auto zval = [&](int st) -> float {
    return st < C / 2 ? zr[st] : (st < C ? zi[st - C / 2] : mg[st - C]);
  };
  // MFMA step groups [qa, qb) for every row tile; A of group q + 1 is read
  // while the MFMAs of group q run (the scheduling groups put the reads first)
  auto run = [&](v16f (&acc)[RT], float4 (&a)[RT], int qa, int qb) {
#pragma unroll
    for (int q = qa; q < qb; ++q) {
      float4 n[RT];
#pragma unroll
      for (int rt = 0; rt < RT; ++rt) n[rt] = q + 1 < KQ ? lda(rt, q + 1) : a[rt];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float z = zval(4 * q + e);
#pragma unroll
        for (int rt = 0; rt < RT; ++rt) {
          const float av = e == 0 ? a[rt].x : (e == 1 ? a[rt].y : (e == 2 ? a[rt].z : a[rt].w));
          acc[rt] = __builtin_amdgcn_mfma_f32_32x32x2f32(av, z, acc[rt], 0, 0, 0);
        }
      }
#pragma unroll
      for (int rt = 0; rt < RT; ++rt) a[rt] = n[rt];
      __builtin_amdgcn_sched_group_barrier(0x100, RT, 0);      // LDS reads
      __builtin_amdgcn_sched_group_barrier(0x008, 4 * RT, 0);  // MFMA
      __builtin_amdgcn_sched_barrier(0);
    }
  };

  for (; task < ntask; task += gridDim.x * nw) {
    const int b = task / tiles_b;
    const int p = (task - b * tiles_b) * 32 + r32;
    const bool ok = p < HW;
    v16f acc[RT];
#pragma unroll
    for (int rt = 0; rt < RT; ++rt)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[rt][r] = 0.f;
    float4 a[RT];
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) a[rt] = lda(rt, 0);
    // Z of this task: Re z0, Im z0 and the moduli (spin 0 first), and the
    // pass-through copy of the other spins
    {
      const unsigned lo = 2u * (unsigned)(kh * HW + (ok ? p : 0));
      T* yb = y + (size_t)b * SC * cs + lo;
#pragma unroll
      for (int i = 0; i < S; ++i) {
        const int sp = slot_of(i);
#pragma unroll
        for (int j = 0; j < C / 2; ++j) {
          if (i == 0) {
            zr[j] = v[0][j].x;
            zi[j] = v[0][j].y;
          } else if (copy_others && ok) {
            st_c2(yb + (size_t)(sp * C + 2 * j) * cs, v[i][j].x, v[i][j].y);
          }
          mg[i * (C / 2) + j] =
              __builtin_amdgcn_sqrtf(v[i][j].x * v[i][j].x + v[i][j].y * v[i][j].y);
        }
      }
    }
    __builtin_amdgcn_sched_barrier(0);
    // every raw value is consumed: the next task's loads overlap the MFMAs
    if (task + gridDim.x * nw < ntask) issue_loads(task + gridDim.x * nw);
    __builtin_amdgcn_sched_barrier(0);
    run(acc, a, 0, KQ);
    // rows (2co, 2co+1) of a column are registers (r, r+1), r even; the
    // output channel co = (row tile) 16 + 4 (r / 4) + (r % 4) / 2 + 2 kh is a
    // lane part (2 kh) plus a wave-uniform part
    if (ok) {
      T* yl = y + 2 * (((size_t)b * SC + (size_t)s0 * C + 2 * kh) * HW + p);
      const float2* bl = bsh + 2 * kh;
#pragma unroll
      for (int rt = 0; rt < RT; ++rt)
#pragma unroll
        for (int r = 0; r < 16; r += 2) {
          const int cu = rt * 16 + 4 * (r >> 2) + ((r & 3) >> 1);
          const float2 bb = bl[cu];
          st_c2(yl + (size_t)cu * cs, acc[rt][r] + bb.x, acc[rt][r + 1] + bb.y);
        }
    }
  }
}

template <typename T, int C, int S>
hipError_t launch_reg(const Plan& p, int B, const void* x, const float2* W1, const float2* W2,
                      const float2* bias, void* y, hipStream_t st, int s0) {
  constexpr int K = 2 * C + S * C;
  const size_t lds = (size_t)2 * C * K * sizeof(float) + C * sizeof(float2);
  auto kern = phase_collapse_reg_kernel<T, C, S>;
  const hipError_t e = ensure_dynamic_lds((const void*)kern, lds);
  if (e != hipSuccess) return e;
  const int HW = p.H * p.W;
  const long long ntask = (long long)B * ((HW + 31) / 32);
  const int nw = ntask >= 8LL * 256 && reg_max_threads(C, S) >= 512 ? 8 : 4;
  const int per_cu = (int)((160 * 1024) / lds) < 1 ? 1 : (int)((160 * 1024) / lds);
  long long blocks = (ntask + nw - 1) / nw;
  const long long cap = 256LL * (per_cu < 2 ? per_cu : 2);
  if (blocks > cap) blocks = cap;
  hipLaunchKernelGGL(kern, dim3((unsigned)blocks), dim3(64 * nw), lds, st, (const T*)x, W1, W2,
                     bias, (T*)y, B, HW, s0, x != y ? 1 : 0);
  return hipGetLastError();
}

// The register form for the shapes it is instantiated for, else nullptr.
template <typename T>
hipError_t (*reg_form(int C, int S))(const Plan&, int, const void*, const float2*, const float2*,
                                     const float2*, void*, hipStream_t, int) {
#define SWSFT_PC_REG(c, s) \
  if (C == c && S == s) return launch_reg<T, c, s>;
  SWSFT_PC_REG(16, 1) SWSFT_PC_REG(16, 2) SWSFT_PC_REG(16, 3)
  SWSFT_PC_REG(32, 1) SWSFT_PC_REG(32, 2) SWSFT_PC_REG(32, 3)
  SWSFT_PC_REG(48, 1) SWSFT_PC_REG(48, 2)
  SWSFT_PC_REG(64, 1) SWSFT_PC_REG(64, 2)
#undef SWSFT_PC_REG
  return nullptr;
}

template <typename T>
hipError_t launch_t(const Plan& p, int B, int C, const void* x, const float2* W1,
                    const float2* W2, const float2* bias, void* y, hipStream_t st, int s0) {
  const int HW = p.H * p.W;
  if (auto f = reg_form<T>(C, p.n_out)) return f(p, B, x, W1, W2, bias, y, st, s0);
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
