// Backward pass of the spectral convolution layer (Method, eqs. (2)-(3) and
// the per-degree mixing): the two kernels that have no forward counterpart.
//
//  filter_adjoint  KH[l][(s,c)][(t,c')] = conj(K[l][(t,c')][(s,c)]): the
//                  filters of the adjoint mixing K^H, in the row-major
//                  [out][in] layout that the mixing GEMM reads.
//  filter_grad     gK[l][(t,c')][(s,c)] = sum_{(m,b)} g[l][(m,b)][(t,c')] conj(a[l][(m,b)][(s,c)]),
//                  the derivative of a real loss with respect to the filters
//                  (one complex GEMM per degree l, contraction length (2l+1) B).
//
// filter_grad as a real MFMA GEMM: the complex product g conj(a) splits into
//   Re = sum gr ar + gi ai,  Im = sum gi ar - gr ai,
// so per 16-wide slice of output rows t' the tile takes 16 "real" rows and 16
// "imaginary" rows, and the contraction index is (k, rho), rho in {re, im}:
//   real rows: A = [gr | gi],   imaginary rows: A = [gi | -gr],   B = [ar ; ai].
// g and a are staged in LDS as separate real and imaginary planes [k][channel]
// (de-interleaved on the way in), so every MFMA operand is one plane read
// along k: ds_read_b64_tr_b16 for bf16 (lanes of a 16-lane group take 16
// consecutive channels, 4 consecutive k each), one dword per lane for fp32.
#include <type_traits>

#include "lds_dma.h"
#include "mfma_tile.h"
#include "swsft_internal.h"
#include "xcd.h"


namespace swsft {
namespace {

struct Spins {
  int s[kMaxSpins];
};

__device__ __forceinline__ int iabs_(int v) { return v < 0 ? -v : v; }

// ---------------------------------------------------------------- adjoint
constexpr int TA = 64;  // transpose tile (complex elements per side)

template <typename T>
struct Cplx;
template <>
struct Cplx<float> {
  typedef float2 type;
  __device__ static float2 conj(float2 v) { return make_float2(v.x, -v.y); }
};
template <>
struct Cplx<__bf16> {
  typedef unsigned type;  // (re, im) bf16 pair, im in the high half
  __device__ static unsigned conj(unsigned v) { return v ^ 0x80000000u; }
};

template <typename T>
__global__ void __launch_bounds__(256) filter_adjoint_kernel(const typename Cplx<T>::type* __restrict__ K,
                                                             typename Cplx<T>::type* __restrict__ KH,
                                                             int Nc, int Kc, int tiles_r, int tiles_c) {
  using V = typename Cplx<T>::type;
  __shared__ V tile[TA][TA + 1];
  const int per_l = tiles_r * tiles_c;
  const int l = blockIdx.x / per_l;
  const int t = blockIdx.x % per_l;
  const int r0 = (t / tiles_c) * TA, c0 = (t % tiles_c) * TA;
  const size_t base = (size_t)l * Nc * Kc;
  for (int idx = threadIdx.x; idx < TA * TA; idx += 256) {
    const int r = idx / TA, c = idx % TA;
    if (r0 + r < Nc && c0 + c < Kc) tile[r][c] = K[base + (size_t)(r0 + r) * Kc + c0 + c];
  }
  __syncthreads();
  for (int idx = threadIdx.x; idx < TA * TA; idx += 256) {
    const int c = idx / TA, r = idx % TA;  // output row (s,c), output column (t,c')
    if (r0 + r < Nc && c0 + c < Kc) KH[base + (size_t)(c0 + c) * Nc + r0 + r] = Cplx<T>::conj(tile[r][c]);
  }
}

// ---------------------------------------------------------------- filter gradient
constexpr int GBM = 64;   // output rows (t,c') per workgroup: 4 slices of 16
constexpr int GBN = 128;  // output columns (s,c) per workgroup: 4 MFMA columns of 32
constexpr int GBK = 32;   // contraction rows (m,b) per LDS stage
constexpr int GNT = 256;  // 4 waves, 2 x 2: each owns 2 row slices x 2 column tiles

template <typename T>
struct GradGeom {
  // Plane pitches and gaps in elements.  bf16: a row stride of 8 dwords past
  // a multiple of 32 puts the 4 rows of one transposed read on distinct
  // banks, and the real and imaginary g planes (read by neighbouring 16-lane
  // groups of one instruction) start 32 dwords apart modulo 64.  fp32: rows
  // k and k + 1 (the two half-waves) 32 dwords apart, the g planes 16 apart.
  static constexpr bool BF = std::is_same<T, __bf16>::value;
  static constexpr int PG = BF ? GBM + 16 : GBM + 32;
  static constexpr int PA = BF ? GBN + 16 : GBN + 32;
  static constexpr int PLANE_G = GBK * PG + (BF ? 64 : 16), PLANE_A = GBK * PA;
  static constexpr int G_CHUNKS = GBK * GBM / 4 / GNT;  // 4-complex chunks per thread
  static constexpr int A_CHUNKS = GBK * GBN / 4 / GNT;
  static constexpr int SMEM = (2 * PLANE_G + 2 * PLANE_A) * (int)sizeof(T);
};

typedef short v4s __attribute__((ext_vector_type(4)));

template <typename T>
struct Chunk {  // 4 consecutive complex values, de-interleaved
  float re[4], im[4];
};

template <typename T, bool VEC>
__device__ __forceinline__ void load_chunk(const T* __restrict__ src, size_t row_off, int col,
                                           int ncols, bool row_ok, Chunk<T>& ch) {
  // src row starts at row_off (reals); col is the first of 4 complex columns
#pragma unroll
  for (int e = 0; e < 4; ++e) ch.re[e] = ch.im[e] = 0.f;
  if (!row_ok) return;
  const T* p = src + row_off + 2 * (size_t)col;
  if constexpr (VEC) {
    if (col >= ncols) return;  // ncols % 4 == 0: a chunk is all in or all out
    if constexpr (std::is_same<T, float>::value) {
      const float4 u = *reinterpret_cast<const float4*>(p);
      const float4 v = *reinterpret_cast<const float4*>(p + 4);
      ch.re[0] = u.x; ch.im[0] = u.y; ch.re[1] = u.z; ch.im[1] = u.w;
      ch.re[2] = v.x; ch.im[2] = v.y; ch.re[3] = v.z; ch.im[3] = v.w;
    } else {
      typedef __bf16 v8b __attribute__((ext_vector_type(8)));
      const v8b u = *reinterpret_cast<const v8b*>(p);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        ch.re[e] = (float)u[2 * e];
        ch.im[e] = (float)u[2 * e + 1];
      }
    }
  } else {
#pragma unroll
    for (int e = 0; e < 4; ++e)
      if (col + e < ncols) {
        ch.re[e] = (float)p[2 * e];
        ch.im[e] = (float)p[2 * e + 1];
      }
  }
}

template <typename T>
__device__ __forceinline__ void store_chunk(T* re_plane, T* im_plane, int off, const Chunk<T>& ch) {
  if constexpr (std::is_same<T, float>::value) {
    *reinterpret_cast<float4*>(re_plane + off) = make_float4(ch.re[0], ch.re[1], ch.re[2], ch.re[3]);
    *reinterpret_cast<float4*>(im_plane + off) = make_float4(ch.im[0], ch.im[1], ch.im[2], ch.im[3]);
  } else {
    typedef __bf16 v4b __attribute__((ext_vector_type(4)));
    v4b r, i;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      r[e] = (__bf16)ch.re[e];
      i[e] = (__bf16)ch.im[e];
    }
    *reinterpret_cast<v4b*>(re_plane + off) = r;
    *reinterpret_cast<v4b*>(im_plane + off) = i;
  }
}

// lane i of a 16-lane group addresses row k + i/4, columns col + 4 (i%4) .. +3;
// lane L of the group receives plane[k + e][col + L] for e = 0..3
__device__ __forceinline__ v4s tr4(const __bf16* plane, int pitch, int k, int col, int gl) {
  const __bf16* p = plane + (k + (gl >> 2)) * pitch + col + 4 * (gl & 3);
  return __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      (__attribute__((address_space(3))) v4s*)((__attribute__((address_space(3))) __bf16*)p));
}

__device__ __forceinline__ v8bf cat8(v4s lo, v4s hi, unsigned flip) {
  typedef unsigned v4u __attribute__((ext_vector_type(4)));
  v4u u;
  u[0] = ((unsigned)(unsigned short)lo[0] | ((unsigned)(unsigned short)lo[1] << 16)) ^ flip;
  u[1] = ((unsigned)(unsigned short)lo[2] | ((unsigned)(unsigned short)lo[3] << 16)) ^ flip;
  u[2] = ((unsigned)(unsigned short)hi[0] | ((unsigned)(unsigned short)hi[1] << 16)) ^ flip;
  u[3] = ((unsigned)(unsigned short)hi[2] | ((unsigned)(unsigned short)hi[3] << 16)) ^ flip;
  return __builtin_bit_cast(v8bf, u);
}

// Degree numbering: q -> l alternates between the top and the bottom of the
// range (L-1, 0, L-2, 1, ...), so any run of consecutive q (one XCD's share
// of the grid) pairs long contractions with short ones.
__device__ __forceinline__ int paired_degree(int q, int L) { return (q & 1) ? (q >> 1) : L - 1 - (q >> 1); }

// Number of kc-row chunks of degree l's contraction (kc > 0).
__device__ __host__ __forceinline__ int grad_chunks(int l, int B, int kc) {
  return ((2 * l + 1) * B + kc - 1) / kc;
}

// Walks n = grad_chunks(l, B, kc) for l = 0, 1, ... with two divisions in
// all: the numerator (2l + 1) B + kc - 1 grows by 2B per degree, so its
// quotient and remainder by kc advance by those of 2B, plus a carry.
struct ChunkWalk {
  int n, rem, dn, dr, kc;
  __device__ ChunkWalk(int B, int kc_) : kc(kc_) {
    const int t = B + kc - 1;
    n = t / kc;
    rem = t - n * kc;
    dn = 2 * B / kc;
    dr = 2 * B - dn * kc;
  }
  __device__ void next() {
    n += dn;
    rem += dr;
    if (rem >= kc) {
      rem -= kc;
      ++n;
    }
  }
};

// kc == 0: one workgroup per (degree, tile), the whole contraction, gK
// written.  kc > 0: one workgroup per (degree, chunk of kc contraction rows,
// tile), chunks numbered by increasing degree; the raw float sums go to
// part[chunk][t'][s'] (complex) and filter_grad_reduce_kernel adds them up.
template <typename T, bool VEC>
__global__ void __launch_bounds__(GNT) filter_grad_kernel(const T* __restrict__ a,
                                                          const T* __restrict__ g, T* __restrict__ gK,
                                                          int L, int B, int Cin, int Cout, int n_in,
                                                          int n_out, Spins sin_, Spins sout_,
                                                          int tiles_r, int tiles_c, int kc,
                                                          float* __restrict__ part) {
  using G = GradGeom<T>;
  extern __shared__ __align__(16) unsigned char smem_raw[];
  T* Gr = reinterpret_cast<T*>(smem_raw);
  T* Gi = Gr + G::PLANE_G;
  T* Ar = Gi + G::PLANE_G;
  T* Ai = Ar + G::PLANE_A;

  const int per_l = tiles_r * tiles_c;
  const int lb = xcd_logical_block();
  int l, k_begin = 0, chunk = 0;
  if (kc == 0) {
    if (lb >= L * per_l) return;
    l = paired_degree(lb / per_l, L);
  } else {
    int q = lb / per_l;  // global chunk index
    ChunkWalk cw(B, kc);
    for (l = 0; l < L; ++l, cw.next()) {
      if (q < cw.n) break;
      q -= cw.n;
      chunk += cw.n;
    }
    if (l >= L) return;
    chunk += q;
    k_begin = q * kc;
  }
  const int tile = lb % per_l;
  const int r0 = (tile / tiles_c) * GBM, c0 = (tile % tiles_c) * GBN;
  const int Nc = n_out * Cout, Kc = n_in * Cin;
  const int Kdeg = (2 * l + 1) * B;                            // degree l's contraction length
  const int k_end = kc == 0 ? Kdeg : min(k_begin + kc, Kdeg);  // this workgroup's rows
  const int Kl = k_end - k_begin;
  const size_t row0 = (size_t)l * l * B + k_begin;             // first (m,b) row
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wr = wave >> 1, wc = wave & 1;

  // whole-tile spin test: every row or every column belongs to a spin that
  // does not exist at degree l
  bool rows_dead = true, cols_dead = true;
  for (int t = r0 / Cout; t <= (min(r0 + GBM, Nc) - 1) / Cout; ++t)
    if (iabs_(sout_.s[t]) <= l) rows_dead = false;
  for (int s = c0 / Cin; s <= (min(c0 + GBN, Kc) - 1) / Cin; ++s)
    if (iabs_(sin_.s[s]) <= l) cols_dead = false;

  v16f acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  if (!rows_dead && !cols_dead) {
    Chunk<T> cg[G::G_CHUNKS], ca[G::A_CHUNKS];
    auto load = [&](int k0) {
#pragma unroll
      for (int u = 0; u < G::G_CHUNKS; ++u) {
        const int idx = u * GNT + tid;
        const int kr = idx / (GBM / 4), cc = 4 * (idx % (GBM / 4));
        const bool ok = k0 + kr < Kl;
        load_chunk<T, VEC>(g, (row0 + k0 + kr) * Nc * 2, r0 + cc, Nc, ok, cg[u]);
      }
#pragma unroll
      for (int u = 0; u < G::A_CHUNKS; ++u) {
        const int idx = u * GNT + tid;
        const int kr = idx / (GBN / 4), cc = 4 * (idx % (GBN / 4));
        const bool ok = k0 + kr < Kl;
        load_chunk<T, VEC>(a, (row0 + k0 + kr) * Kc * 2, c0 + cc, Kc, ok, ca[u]);
      }
    };
    auto store = [&]() {
#pragma unroll
      for (int u = 0; u < G::G_CHUNKS; ++u) {
        const int idx = u * GNT + tid;
        const int kr = idx / (GBM / 4), cc = 4 * (idx % (GBM / 4));
        store_chunk<T>(Gr, Gi, kr * G::PG + cc, cg[u]);
      }
#pragma unroll
      for (int u = 0; u < G::A_CHUNKS; ++u) {
        const int idx = u * GNT + tid;
        const int kr = idx / (GBN / 4), cc = 4 * (idx % (GBN / 4));
        store_chunk<T>(Ar, Ai, kr * G::PA + cc, ca[u]);
      }
    };

    const int nkb = (Kl + GBK - 1) / GBK;
    load(0);
    store();
    __syncthreads();
    for (int kb = 0; kb < nkb; ++kb) {
      if (kb + 1 < nkb) load((kb + 1) * GBK);
      if constexpr (G::BF) {
        const int grp = lane >> 4, gl = lane & 15;
        const int half = grp & 1, kq = grp >> 1;
        const unsigned flip1 = half ? 0x80008000u : 0u;  // imaginary rows take -gr
#pragma unroll
        for (int ks = 0; ks < GBK; ks += 16) {
          const int kb8 = ks + 8 * kq;
#pragma unroll
          for (int rho = 0; rho < 2; ++rho) {
            const __bf16* pa = (rho == 0) == (half == 0) ? Gr : Gi;
            const __bf16* pb = rho == 0 ? Ar : Ai;
            v8bf av[2], bv[2];
#pragma unroll
            for (int i = 0; i < 2; ++i) {
              const int col = wr * 32 + i * 16;
              av[i] = cat8(tr4(pa, G::PG, kb8, col, gl), tr4(pa, G::PG, kb8 + 4, col, gl),
                           rho ? flip1 : 0u);
            }
#pragma unroll
            for (int j = 0; j < 2; ++j) {
              const int col = wc * 64 + j * 32 + 16 * half;
              bv[j] = cat8(tr4(pb, G::PA, kb8, col, gl), tr4(pb, G::PA, kb8 + 4, col, gl), 0u);
            }
#pragma unroll
            for (int i = 0; i < 2; ++i)
#pragma unroll
              for (int j = 0; j < 2; ++j)
                acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av[i], bv[j], acc[i][j], 0, 0, 0);
          }
        }
      } else {
        const int r32 = lane & 31, kh = lane >> 5, half = r32 >> 4;
        const float sgn1 = half ? -1.f : 1.f;
#pragma unroll 4
        for (int kk = 0; kk < GBK; kk += 2) {
          const int k = kk + kh;
#pragma unroll
          for (int rho = 0; rho < 2; ++rho) {
            const float* pa = (rho == 0) == (half == 0) ? Gr : Gi;
            const float* pb = rho == 0 ? Ar : Ai;
            float av[2], bv[2];
#pragma unroll
            for (int i = 0; i < 2; ++i)
              av[i] = (rho ? sgn1 : 1.f) * pa[k * G::PG + wr * 32 + i * 16 + (r32 & 15)];
#pragma unroll
            for (int j = 0; j < 2; ++j) bv[j] = pb[k * G::PA + wc * 64 + j * 32 + r32];
#pragma unroll
            for (int i = 0; i < 2; ++i)
#pragma unroll
              for (int j = 0; j < 2; ++j)
                acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(av[i], bv[j], acc[i][j], 0, 0, 0);
          }
        }
      }
      __syncthreads();
      if (kb + 1 < nkb) {
        store();
        __syncthreads();
      }
    }
  }

  // epilogue: registers (r, r + 8) of a lane are the real and imaginary parts
  // of one output; zeros where a spin does not exist at degree l (a split
  // contraction writes its raw float sums, the reduction applies them)
  if (kc != 0) {
    float* pout = part + (size_t)chunk * Nc * Kc * 2;
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        const int sc = c0 + wc * 64 + j * 32 + (lane & 31);
        if (sc >= Kc) continue;
#pragma unroll
        for (int r = 0; r < 8; ++r) {
          const int tc = r0 + wr * 32 + i * 16 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
          if (tc >= Nc) continue;
          *reinterpret_cast<float2*>(pout + ((size_t)tc * Kc + sc) * 2) =
              make_float2(acc[i][j][r], acc[i][j][r + 8]);
        }
      }
    return;
  }
  T* out = gK + (size_t)l * Nc * Kc * 2;
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int sc = c0 + wc * 64 + j * 32 + (lane & 31);
      if (sc >= Kc) continue;
      const bool col_live = iabs_(sin_.s[sc / Cin]) <= l;
#pragma unroll
      for (int r = 0; r < 8; ++r) {
        const int tc = r0 + wr * 32 + i * 16 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
        if (tc >= Nc) continue;
        const bool live = col_live && iabs_(sout_.s[tc / Cout]) <= l;
        const float re = live ? acc[i][j][r] : 0.f, im = live ? acc[i][j][r + 8] : 0.f;
        T* o = out + ((size_t)tc * Kc + sc) * 2;
        if constexpr (G::BF) {
          typedef float f32x2 __attribute__((ext_vector_type(2)));
          typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
          *reinterpret_cast<bf16x2*>(o) = __builtin_convertvector((f32x2){re, im}, bf16x2);
        } else {
          *reinterpret_cast<float2*>(o) = make_float2(re, im);
        }
      }
    }
}

Spins to_spins(const int* s, int n) {
  Spins r{};
  for (int i = 0; i < n && i < kMaxSpins; ++i) r.s[i] = s[i];
  return r;
}

// gK[l] = sum over the chunks of degree l of part[chunk], in chunk order
// (deterministic), zero where a spin does not exist at degree l.  Grid: L x
// ceil(Nc Kc / (256 V)) workgroups, V consecutive complex outputs per thread
// (V = 2 takes 16-byte loads and needs Nc Kc even).
template <typename T, int V>
__global__ void __launch_bounds__(256) filter_grad_reduce_kernel(const float* __restrict__ part,
                                                                 T* __restrict__ gK, int L, int B,
                                                                 int Cin, int Cout, int n_in,
                                                                 int n_out, Spins sin_, Spins sout_,
                                                                 int kc, int blocks_per_l) {
  using VF = typename std::conditional<V == 2, float4, float2>::type;
  const int l = blockIdx.x / blocks_per_l;
  const int Nc = n_out * Cout, Kc = n_in * Cin, NK = Nc * Kc;
  const int e = ((blockIdx.x % blocks_per_l) * 256 + threadIdx.x) * V;  // first output (t', s')
  if (l >= L || e >= NK) return;
  int base = 0;
  ChunkWalk cw(B, kc);
  for (int d = 0; d < l; ++d, cw.next()) base += cw.n;
  const int n = cw.n;
  const size_t stride = (size_t)NK / V;  // one chunk, in VF units
  const VF* p = reinterpret_cast<const VF*>(part) + ((size_t)base * NK + e) / V;
  float acc[2 * V] = {};
  auto add = [&](const VF& v) {
    const float* f = reinterpret_cast<const float*>(&v);
#pragma unroll
    for (int u = 0; u < 2 * V; ++u) acc[u] += f[u];
  };
  // four loads in flight; the sum order stays chunk order
  int c = 0;
  for (; c + 4 <= n; c += 4) {
    VF v[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) v[u] = p[(size_t)(c + u) * stride];
#pragma unroll
    for (int u = 0; u < 4; ++u) add(v[u]);
  }
  for (; c < n; ++c) add(p[(size_t)c * stride]);
  T* o = gK + ((size_t)l * NK + e) * 2;
#pragma unroll
  for (int u = 0; u < V; ++u) {
    const int tc = (e + u) / Kc, sc = e + u - tc * Kc;
    const bool live = iabs_(sout_.s[tc / Cout]) <= l && iabs_(sin_.s[sc / Cin]) <= l;
    o[2 * u] = (T)(live ? acc[2 * u] : 0.f);
    o[2 * u + 1] = (T)(live ? acc[2 * u + 1] : 0.f);
  }
}

// ---------------------------------------------------------------- bf16 filter gradient, split accumulators
// The same gradient as a complex GEMM per degree with separate real and
// imaginary accumulators, the contraction running over (k, rho):
//   Re gK[t'][s'] = sum_k gr ar + gi ai   (g and a as stored, (re, im) per k),
//   Im gK[t'][s'] = sum_k gi ar - gr ai   (each g pair turned into (gi, -gr) in registers).
// Both operands are K-major (row k = one coefficient row (m, b), channels
// contiguous); each tile is copied global -> LDS unchanged as [k][RA or RB
// complex columns] (swz_k4 chunk order) and a lane gathers the 4 consecutive
// contraction rows of its column as 4 dword reads, so one read of a g
// fragment feeds a real and an imaginary MFMA.  A wave owns TM x TN blocks of
// 32 x 32 complex outputs.  A real GEMM over the interleaved values, which
// keeps all four real products of every complex output until its epilogue,
// needs twice the accumulators per output; here the same registers hold
// twice the outputs, so a 128 x 128 complex tile copies each row of g and of
// a for 4 tiles (16 KB of copies per contraction row and degree at 512 x 512
// channels, against 24 KB for 256 x 128 real tiles) and reads half the LDS
// bytes per MFMA.  Contraction rows past (2l+1) B are copied from a clamped
// row and zeroed in LDS before use.
typedef unsigned v4u_t __attribute__((ext_vector_type(4)));

// Contraction rows per K step and (waves per workgroup as rows x columns of
// 64 x 64 complex wave tiles, stages); measured at 256^2, C = 256: 16 rows
// with 4 stages 131 us, 32 with 2 136 us, 8 with 8 143 us.
#ifndef SWSFT_GRAD_SPLIT_BK
#define SWSFT_GRAD_SPLIT_BK 16
#endif
#ifndef SWSFT_GRAD_SPLIT
#define SWSFT_GRAD_SPLIT 2, 2, 4
#endif

template <int WM, int WN, int ST>
struct GradSplitGeom {
  static constexpr int BK = SWSFT_GRAD_SPLIT_BK;  // contraction rows per K step
  static constexpr int TM = 2, TN = 2;     // 32 x 32 complex blocks per wave
  static constexpr int RA = 32 * TM * WM;  // complex rows t' per workgroup
  static constexpr int RB = 32 * TN * WN;  // complex columns s' per workgroup
  static constexpr int NW = WM * WN, NT = 64 * NW;
  static constexpr int PITCH_A = 4 * RA, PITCH_B = 4 * RB;  // bytes per k row
  static constexpr int RPI_A = 1024 / PITCH_A, LPR_A = 64 / RPI_A;
  static constexpr int RPI_B = 1024 / PITCH_B, LPR_B = 64 / RPI_B;
  static constexpr int A_BYTES = BK * PITCH_A, B_BYTES = BK * PITCH_B;
  static constexpr int NI_A = A_BYTES / 1024, NI = NI_A + B_BYTES / 1024;
  static constexpr int PER_WAVE = NI / NW;
  static constexpr int STAGE = A_BYTES + B_BYTES;
  static constexpr int SMEM = ST * STAGE;
  static_assert(PITCH_A <= 1024 && PITCH_B <= 1024 && 1024 % PITCH_A == 0 &&
                    1024 % PITCH_B == 0 && PITCH_A >= 256 && PITCH_B >= 256 && NI % NW == 0 &&
                    ST >= 2 && (ST - 2) * PER_WAVE < 64,
                "tile shape");
  static_assert(RA * RB * 4 <= SMEM, "staged output tile");
};

// (two workgroups per CU: at most 256 registers per lane)
template <int WM, int WN, int ST>
__global__ void __launch_bounds__((GradSplitGeom<WM, WN, ST>::NT), 2)
    filter_grad_split_kernel(const __bf16* __restrict__ a, const __bf16* __restrict__ g,
                             __bf16* __restrict__ gK, int L, int B, int Cin, int Cout, int n_in,
                             int n_out, Spins sin_, Spins sout_, int tiles_r, int tiles_c) {
  using G = GradSplitGeom<WM, WN, ST>;
  constexpr int BK = G::BK, TM = G::TM, TN = G::TN, RA = G::RA, RB = G::RB;
  extern __shared__ __align__(16) unsigned char smem[];  // the ring, then the output tile
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave / WN, wn = wave % WN;
  const int per_l = tiles_r * tiles_c;
  const int lb = xcd_logical_block();
  if (lb >= L * per_l) return;
  const int l = paired_degree(lb / per_l, L);
  const int tile = lb % per_l;
  const int Nc = n_out * Cout, Kc = n_in * Cin;
  const int r0 = (tile / tiles_c) * RA, c0 = (tile % tiles_c) * RB;  // first t', first s'
  const int Kl = (2 * l + 1) * B;
  const size_t row0 = (size_t)l * l * B;

  bool rows_dead = true, cols_dead = true;
  for (int t = r0 / Cout; t <= (min(r0 + RA, Nc) - 1) / Cout; ++t)
    if (iabs_(sout_.s[t]) <= l) rows_dead = false;
  for (int q = c0 / Cin; q <= (min(c0 + RB, Kc) - 1) / Cin; ++q)
    if (iabs_(sin_.s[q]) <= l) cols_dead = false;

  v16f acc_re[TM][TN], acc_im[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc_re[i][j][r] = acc_im[i][j][r] = 0.f;

  if (!rows_dead && !cols_dead) {
    // copy u of this wave: g rows (A tile) for copy index < NI_A, else a
    // rows; lane -> (k row of the step, 16-byte slot), the slot holding
    // chunk swz_k4(k, slot) of the row (4 complex columns, clamped to the
    // last whole chunk: those columns are never stored)
    const __bf16* src[G::PER_WAVE];
    int krow[G::PER_WAVE], pitch[G::PER_WAVE];
#pragma unroll
    for (int u = 0; u < G::PER_WAVE; ++u) {
      const int gi = wave * G::PER_WAVE + u;
      if (gi < G::NI_A) {
        const int k = gi * G::RPI_A + lane / G::LPR_A;
        const int col = min(r0 + 4 * swz_k4(k, lane % G::LPR_A), Nc - 4);
        src[u] = g + 2 * (size_t)col;
        krow[u] = k;
        pitch[u] = 2 * Nc;
      } else {
        const int k = (gi - G::NI_A) * G::RPI_B + lane / G::LPR_B;
        const int col = min(c0 + 4 * swz_k4(k, lane % G::LPR_B), Kc - 4);
        src[u] = a + 2 * (size_t)col;
        krow[u] = k;
        pitch[u] = 2 * Kc;
      }
    }
    const unsigned ring = lds_addr(smem);
    auto issue = [&](int i, int stage) {
      const unsigned base = ring + stage * G::STAGE + wave * G::PER_WAVE * 1024;
#pragma unroll
      for (int u = 0; u < G::PER_WAVE; ++u) {
        const int k = min(i * BK + krow[u], Kl - 1);  // past the degree: a row that exists
        dma16(src[u] + (row0 + k) * (size_t)pitch[u], base + u * 1024);
      }
    };
    const int nk = (Kl + BK - 1) / BK;
#pragma unroll
    for (int s = 0; s < ST - 1; ++s)
      if (s < nk) issue(s, s);
    const int r32 = lane & 31, kh = lane >> 5;
    // the 4 contraction rows 4c .. 4c + 3 of column col of a K-major tile
    auto gather = [](const unsigned char* tile, int pitch_b, int c, int col) {
      v4u_t y;
#pragma unroll
      for (int d = 0; d < 4; ++d) {
        const int kr = 4 * c + d;
        y[d] = *reinterpret_cast<const unsigned*>(tile + kr * pitch_b + swz_k4(kr, col >> 2) * 16 +
                                                  (col & 3) * 4);
      }
      return y;
    };
    for (int i = 0; i < nk; ++i) {
      const int issued = nk < i + ST - 1 ? nk : i + ST - 1;
      wait_groups<ST - 2, G::PER_WAVE>(issued - i - 1);
      __builtin_amdgcn_s_barrier();  // every wave's copies of step i landed; step i-1 is consumed
      if (i + ST - 1 < nk) issue(i + ST - 1, (i + ST - 1) % ST);
      unsigned char* As = smem + (i % ST) * G::STAGE;
      unsigned char* Bs = As + G::A_BYTES;
      const int kv = Kl - i * BK;  // valid rows of this step
      if (kv < BK) {
        // the clamped rows of the last step hold other data: zero them
        const int za = (BK - kv) * G::PITCH_A, zb = (BK - kv) * G::PITCH_B;
        for (int o = tid * 16; o < za; o += G::NT * 16)
          *reinterpret_cast<uint4*>(As + kv * G::PITCH_A + o) = make_uint4(0, 0, 0, 0);
        for (int o = tid * 16; o < zb; o += G::NT * 16)
          *reinterpret_cast<uint4*>(Bs + kv * G::PITCH_B + o) = make_uint4(0, 0, 0, 0);
        __syncthreads();
      }
#pragma unroll
      for (int kk = 0; kk < BK / 8; ++kk) {  // MFMA K steps of 8 rows (4 per lane half)
        const int c = 2 * kk + kh;
        v8bf xb[TN];
#pragma unroll
        for (int jj = 0; jj < TN; ++jj)
          xb[jj] = __builtin_bit_cast(v8bf, gather(Bs, G::PITCH_B, c, (wn * TN + jj) * 32 + r32));
#pragma unroll
        for (int ii = 0; ii < TM; ++ii) {
          const v4u_t x = gather(As, G::PITCH_A, c, (wm * TM + ii) * 32 + r32);
          v4u_t xi;
#pragma unroll
          for (int d = 0; d < 4; ++d)
            xi[d] = __builtin_amdgcn_alignbit(x[d], x[d], 16u) ^ 0x80000000u;  // (gi, -gr)
          const v8bf ar = __builtin_bit_cast(v8bf, x), ai = __builtin_bit_cast(v8bf, xi);
#pragma unroll
          for (int jj = 0; jj < TN; ++jj) {
            acc_re[ii][jj] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ar, xb[jj], acc_re[ii][jj], 0, 0, 0);
            acc_im[ii][jj] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ai, xb[jj], acc_im[ii][jj], 0, 0, 0);
          }
        }
      }
    }
    wait_vmcnt<0>();
  }

  // epilogue: register r of a lane holds row 8 (r / 4) + 4 (lane / 32) + r % 4
  // of its block, column lane % 32; the (re, im) bf16 pairs are staged in LDS
  // as the tile's [t'][s'] block (16-byte chunks of rows with bit 2 set moved
  // by 128 bytes), then written by all threads as 16-byte chunks along s'.
  // Outputs of spins that do not exist at this degree are zero.
  typedef float f32x2 __attribute__((ext_vector_type(2)));
  typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
  constexpr int RP = RB * 4;    // bytes per staged row
  constexpr int CPRO = RB / 4;  // 16-byte chunks per staged row
  __syncthreads();              // every wave is done with the ring
  const int col_l = lane & 31, row_l = 4 * (lane >> 5);
#pragma unroll
  for (int jj = 0; jj < TN; ++jj) {
    const int cl = (wn * TN + jj) * 32 + col_l;
    const int sc = c0 + cl;
    const bool col_live = sc < Kc && iabs_(sin_.s[(sc < Kc ? sc : 0) / Cin]) <= l;
#pragma unroll
    for (int ii = 0; ii < TM; ++ii)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int rl = (wm * TM + ii) * 32 + 8 * (r >> 2) + row_l + (r & 3);
        const int tc = r0 + rl;
        const bool live = col_live && tc < Nc && iabs_(sout_.s[(tc < Nc ? tc : 0) / Cout]) <= l;
        const f32x2 v = live ? (f32x2){acc_re[ii][jj][r], acc_im[ii][jj][r]} : (f32x2){0.f, 0.f};
        *reinterpret_cast<bf16x2*>(smem + rl * RP + swz_k4(rl, cl >> 2) * 16 + (cl & 3) * 4) =
            __builtin_convertvector(v, bf16x2);
      }
  }
  __syncthreads();
  __bf16* out = gK + (size_t)l * Nc * Kc * 2;
  for (int idx = tid; idx < RA * CPRO; idx += G::NT) {
    const int rl = idx / CPRO, ch = idx % CPRO;
    const int tc = r0 + rl, sc = c0 + 4 * ch;  // Kc % 4 == 0: whole chunks
    if (tc < Nc && sc < Kc)
      *reinterpret_cast<uint4*>(out + ((size_t)tc * Kc + sc) * 2) =
          *reinterpret_cast<const uint4*>(smem + rl * RP + swz_k4(rl, ch) * 16);
  }
}


template <int WM, int WN, int ST>
hipError_t filter_grad_split_t(const Plan& p, int B, int Cin, int Cout, const void* a,
                               const void* g, void* gK, hipStream_t st) {
  using G = GradSplitGeom<WM, WN, ST>;
  const int Nc = p.n_out * Cout, Kc = p.n_in * Cin;
  const int tiles_r = (Nc + G::RA - 1) / G::RA, tiles_c = (Kc + G::RB - 1) / G::RB;
  const long long blocks = (long long)p.L * tiles_r * tiles_c;
  const hipError_t e = ensure_dynamic_lds((const void*)filter_grad_split_kernel<WM, WN, ST>, G::SMEM);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((filter_grad_split_kernel<WM, WN, ST>), dim3(xcd_grid(blocks)), dim3(G::NT),
                     G::SMEM, st, (const __bf16*)a, (const __bf16*)g, (__bf16*)gK, p.L, B, Cin,
                     Cout, p.n_in, p.n_out, to_spins(p.spins_in, p.n_in),
                     to_spins(p.spins_out, p.n_out), tiles_r, tiles_c);
  return hipGetLastError();
}

bool grad_uses_dma(const Plan& p, int Cin, int Cout) {
  // bf16 rows as 16-byte chunks: channel counts with 2 S C % 8 == 0
  return p.dtype == SWSFT_BF16 && (2 * p.n_out * Cout) % 8 == 0 && (2 * p.n_in * Cin) % 8 == 0;
}

template <typename T>
hipError_t filter_grad_t(const Plan& p, int B, int Cin, int Cout, const void* a, const void* g,
                         void* gK, void* part, hipStream_t st) {
  if constexpr (std::is_same<T, __bf16>::value) {
    if (grad_uses_dma(p, Cin, Cout))
      return filter_grad_split_t<SWSFT_GRAD_SPLIT>(p, B, Cin, Cout, a, g, gK, st);
  }
  using G = GradGeom<T>;
  const int Nc = p.n_out * Cout, Kc = p.n_in * Cin;
  const int tiles_r = (Nc + GBM - 1) / GBM, tiles_c = (Kc + GBN - 1) / GBN;
  const int kc = filter_grad_split_rows(p, B, Cin, Cout);
  long long units = p.L;  // degrees, or chunks of split contractions
  if (kc > 0) {
    units = 0;
    for (int l = 0; l < p.L; ++l) units += grad_chunks(l, B, kc);
  }
  const long long blocks = units * tiles_r * tiles_c;
  const bool vec = Nc % 4 == 0 && Kc % 4 == 0;
  auto kern = vec ? filter_grad_kernel<T, true> : filter_grad_kernel<T, false>;
  const hipError_t e = ensure_dynamic_lds((const void*)kern, G::SMEM);
  if (e != hipSuccess) return e;
  const Spins si = to_spins(p.spins_in, p.n_in), so = to_spins(p.spins_out, p.n_out);
  hipLaunchKernelGGL(kern, dim3(xcd_grid(blocks)), dim3(GNT), G::SMEM, st, (const T*)a,
                     (const T*)g, (T*)gK, p.L, B, Cin, Cout, p.n_in, p.n_out, si, so, tiles_r,
                     tiles_c, kc, (float*)part);
  if (kc > 0) {
    const bool two = (Nc * Kc) % 2 == 0;
    const int per_l = (Nc * Kc + (two ? 511 : 255)) / (two ? 512 : 256);
    auto rk = two ? filter_grad_reduce_kernel<T, 2> : filter_grad_reduce_kernel<T, 1>;
    hipLaunchKernelGGL(rk, dim3((unsigned)((long long)p.L * per_l)), dim3(256), 0, st,
                       (const float*)part, (T*)gK, p.L, B, Cin, Cout, p.n_in, p.n_out, si, so, kc,
                       per_l);
  }
  return hipGetLastError();
}

template <typename T>
hipError_t filter_adjoint_t(const Plan& p, int Cin, int Cout, const void* K, void* KH,
                            hipStream_t st) {
  using V = typename Cplx<T>::type;
  const int Nc = p.n_out * Cout, Kc = p.n_in * Cin;
  const int tr = (Nc + TA - 1) / TA, tc = (Kc + TA - 1) / TA;
  hipLaunchKernelGGL(filter_adjoint_kernel<T>, dim3((unsigned)((long long)p.L * tr * tc)), dim3(256),
                     0, st, (const V*)K, (V*)KH, Nc, Kc, tr, tc);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_filter_adjoint(const Plan& p, int C_in, int C_out, const void* K, void* KH,
                                 hipStream_t st) {
  if (p.dtype == SWSFT_BF16) return filter_adjoint_t<__bf16>(p, C_in, C_out, K, KH, st);
  return filter_adjoint_t<float>(p, C_in, C_out, K, KH, st);
}

#ifndef SWSFT_GRAD_SPLIT_WG
#define SWSFT_GRAD_SPLIT_WG 384
#endif

// Contraction rows per chunk of the register-staged kernel: a multiple of
// the K stage, sized for about SWSFT_GRAD_SPLIT_WG workgroups, when one workgroup per
// (degree, tile) would leave CUs idle (few degrees, long contractions, as at
// small bandlimits with large batches); 0 when the contraction is not split.
int filter_grad_split_rows(const Plan& p, int B, int C_in, int C_out) {
  if (grad_uses_dma(p, C_in, C_out)) return 0;
  const int Nc = p.n_out * C_out, Kc = p.n_in * C_in;
  const long long tiles = (long long)((Nc + GBM - 1) / GBM) * ((Kc + GBN - 1) / GBN);
  if ((long long)p.L * tiles >= 256) return 0;
  const long long rows = (long long)p.L * p.L * B;  // all degrees' contraction rows
  long long kc = (rows * tiles + SWSFT_GRAD_SPLIT_WG - 1) / SWSFT_GRAD_SPLIT_WG;
  kc = (kc + GBK - 1) / GBK * GBK;
  if (kc >= (long long)(2 * p.L - 1) * B) return 0;  // no degree would be split
  return (int)kc;
}

size_t filter_grad_split_bytes(const Plan& p, int B, int C_in, int C_out) {
  const int kc = filter_grad_split_rows(p, B, C_in, C_out);
  if (kc == 0) return 0;
  size_t chunks = 0;
  for (int l = 0; l < p.L; ++l) chunks += grad_chunks(l, B, kc);
  return chunks * p.n_out * C_out * p.n_in * C_in * 2 * sizeof(float);
}

hipError_t launch_filter_grad(const Plan& p, int B, int C_in, int C_out, const void* a,
                              const void* g, void* gK, void* part, hipStream_t st) {
  if (p.dtype == SWSFT_BF16) return filter_grad_t<__bf16>(p, B, C_in, C_out, a, g, gK, part, st);
  return filter_grad_t<float>(p, B, C_in, C_out, a, g, gK, part, st);
}

}  // namespace swsft
