// The three contractions of the layer, as MFMA GEMMs.
//
//  lat_fwd  (eq. (2), latitude sum), per (spin s, order m):
//     coef[l*l+l+m][b][s][c] = sum_j Tf[s][m][l][j] X[s][m][n][re/im][j]
//     real GEMM: rows l in [|m|, L), columns n' = 2n + re/im, K = j.
//  mix      (per-degree products with filters shared across m), per l:
//     coef'[l][(m,b)][(t,c')] = sum_(s,c) coef[l][(m,b)][(s,c)] K[l][(t,c')][(s,c)]
//     complex GEMM written as a real GEMM with K doubled: the filter tile is
//     expanded in LDS into 2x2 real blocks [[re, -im], [im, re]].
//  lat_inv  (eq. (3), latitude sum), per (spin t, order m):
//     Y[t][m][n'][j] = sum_l coef'[l*l+l+m][b][t][c'][re/im] Ti[t][m][j][l]
//     real GEMM: rows n', columns j, K = l in [max(|m|,|t|), L).
//
// Every operand is staged in LDS K-contiguous; the tables and the X / Y
// intermediates are laid out so that their global rows already are, the
// mixing filters are stored output-major for the same reason, and only the
// coefficient operand of lat_inv is transposed on its way into LDS.
#include "mfma_tile.h"
#include "swsft_internal.h"

namespace swsft {
namespace {

constexpr int BK = 32;
constexpr int NT = 256;

struct SpinList {
  int s[kMaxSpins];
};

__device__ __forceinline__ int iabs(int v) { return v < 0 ? -v : v; }

// --------------------------------------------------------------------------
template <typename T, int BM, int BN, int WM, int WN>
__global__ void __launch_bounds__(NT) lat_fwd_kernel(const T* __restrict__ X,
                                                     const T* __restrict__ tab,
                                                     T* __restrict__ coef, int L, int H, int Hp,
                                                     int B, int C, int S, int n_row_tiles) {
  using Tile = MfmaTile<T, BM, BN, BK, WM, WN>;
  __shared__ __align__(16) T As[BM * Tile::LD];
  __shared__ __align__(16) T Bs[BN * Tile::LD];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WN, wn = wave % WN;
  const int M = 2 * L - 1;
  const int mi = blockIdx.y, si = blockIdx.z;
  const int m = mi - (L - 1);
  const int rt = blockIdx.x % n_row_tiles, nt = blockIdx.x / n_row_tiles;
  const int l_begin = iabs(m) + rt * BM;
  if (l_begin >= L) return;
  const int Np = 2 * B * C;
  const int n0 = nt * BN;
  const T* A0 = tab + (size_t)(si * M + mi) * L * Hp;
  const T* B0 = X + (size_t)(si * M + mi) * Np * Hp;
  auto arow = [&](int r) -> const T* {
    const int l = l_begin + r;
    return l < L ? A0 + (size_t)l * Hp : nullptr;
  };
  auto brow = [&](int r) -> const T* {
    const int np = n0 + r;
    return np < Np ? B0 + (size_t)np * Hp : nullptr;
  };
  Tile tile;
  tile.zero();
  KTileLoader<T, BM, BK, NT> la;
  KTileLoader<T, BN, BK, NT> lb;
  la.load(arow, 0, H, tid, true);
  lb.load(brow, 0, H, tid, true);
  for (int k0 = 0; k0 < H; k0 += BK) {
    __syncthreads();
    la.store(As, tid);
    lb.store(Bs, tid);
    __syncthreads();
    if (k0 + BK < H) {
      la.load(arow, k0 + BK, H, tid, true);
      lb.load(brow, k0 + BK, H, tid, true);
    }
    tile.compute(As, Bs, wm, wn, lane);
  }
  const int twoC = 2 * C;
  tile.for_each(wm, wn, lane, [&](int row, int col, float v) {
    const int l = l_begin + row;
    const int np = n0 + col;
    if (l < L && np < Np) {
      const int b = np / twoC;
      const int rem = np - b * twoC;
      coef[(((size_t)(l * l + l + m) * B + b) * S + si) * twoC + rem] = (T)v;
    }
  });
}

// --------------------------------------------------------------------------
template <typename T, int BM, int BN, int WM, int WN>
__global__ void __launch_bounds__(NT) mix_kernel(const T* __restrict__ coef,
                                                 const T* __restrict__ K, T* __restrict__ out,
                                                 int L, int B, int Cin, int Cout, int Sin,
                                                 int Sout, SpinList sin_, SpinList sout_) {
  using Tile = MfmaTile<T, BM, BN, BK, WM, WN>;
  __shared__ __align__(16) T As[BM * Tile::LD];
  __shared__ __align__(16) T Bs[BN * Tile::LD];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WN, wn = wave % WN;
  // work item -> (l, row tile); the largest degrees come first
  int t = blockIdx.x;
  int l = L - 1;
  for (; l >= 0; --l) {
    const int ntl = ((2 * l + 1) * B + BM - 1) / BM;
    if (t < ntl) break;
    t -= ntl;
  }
  if (l < 0) return;
  const int Mrows = (2 * l + 1) * B;
  const int row0 = t * BM;
  const int Kc = Sin * Cin, Nc = Sout * Cout;  // complex sizes
  const int Kp = 2 * Kc, Np = 2 * Nc;          // real sizes
  const int n0 = blockIdx.y * BN;
  const T* A0 = coef + (size_t)l * l * B * Kp;
  const T* K0 = K + (size_t)l * Nc * Kc * 2;
  const bool avec = (Kp % (16 / (int)sizeof(T))) == 0;
  auto arow = [&](int r) -> const T* {
    const int i = row0 + r;
    return i < Mrows ? A0 + (size_t)i * Kp : nullptr;
  };
  Tile tile;
  tile.zero();
  KTileLoader<T, BM, BK, NT> la;

  // filter operand: BN/2 complex rows x BK/2 complex columns per tile
  constexpr int VEC = 16 / sizeof(T);      // reals per 16-byte vector
  constexpr int VPR = BK / VEC;            // vectors per complex row of the tile
  constexpr int NVB = (BN / 2) * VPR;
  constexpr int PERB = (NVB + NT - 1) / NT;
  union Vec {
    uint4 u;
    T e[VEC];
  };
  Vec breg[PERB];
  const bool bvec = (Kp % VEC) == 0;
  auto load_b = [&](int k0) {
#pragma unroll
    for (int p = 0; p < PERB; ++p) {
      const int v = tid + p * NT;
      if (NVB % NT != 0 && v >= NVB) break;
      const int r = v / VPR;           // complex row within tile
      const int kv = (v % VPR) * VEC;  // real column within tile
      const int q = n0 / 2 + r;        // complex output index (t, c')
      const int k = k0 + kv;           // real input index (s, c, re/im)
      const bool qok = q < Nc && iabs(sout_.s[q < Nc ? q / Cout : 0]) <= l;
      const T* src = K0 + (size_t)q * Kp;
      if (qok && bvec && k + VEC <= Kp) {
        breg[p].u = *reinterpret_cast<const uint4*>(src + k);
      } else {
#pragma unroll
        for (int e = 0; e < VEC; ++e) breg[p].e[e] = (qok && k + e < Kp) ? src[k + e] : (T)0.f;
      }
      // input spins that do not exist at this degree take no part
#pragma unroll
      for (int e = 0; e < VEC; e += 2) {
        const int pc = (k + e) >> 1;
        if (pc < Kc && iabs(sin_.s[pc / Cin]) > l) {
          breg[p].e[e] = (T)0.f;
          breg[p].e[e + 1] = (T)0.f;
        }
      }
    }
  };
  auto store_b = [&]() {
#pragma unroll
    for (int p = 0; p < PERB; ++p) {
      const int v = tid + p * NT;
      if (NVB % NT != 0 && v >= NVB) break;
      const int r = v / VPR;
      const int kv = (v % VPR) * VEC;
      T* re_row = Bs + (2 * r) * Tile::LD + kv;      // output real part
      T* im_row = Bs + (2 * r + 1) * Tile::LD + kv;  // output imaginary part
#pragma unroll
      for (int e = 0; e < VEC; e += 2) {
        const T kr = breg[p].e[e], ki = breg[p].e[e + 1];
        re_row[e] = kr;
        re_row[e + 1] = -ki;
        im_row[e] = ki;
        im_row[e + 1] = kr;
      }
    }
  };

  la.load(arow, 0, Kp, tid, avec);
  load_b(0);
  for (int k0 = 0; k0 < Kp; k0 += BK) {
    __syncthreads();
    la.store(As, tid);
    store_b();
    __syncthreads();
    if (k0 + BK < Kp) {
      la.load(arow, k0 + BK, Kp, tid, avec);
      load_b(k0 + BK);
    }
    tile.compute(As, Bs, wm, wn, lane);
  }
  T* O0 = out + (size_t)l * l * B * Np;
  tile.for_each(wm, wn, lane, [&](int row, int col, float v) {
    const int i = row0 + row;
    const int np = n0 + col;
    if (i < Mrows && np < Np) O0[(size_t)i * Np + np] = (T)v;
  });
}

// --------------------------------------------------------------------------
template <typename T, int BM, int BN, int WM, int WN>
__global__ void __launch_bounds__(NT) lat_inv_kernel(const T* __restrict__ coef,
                                                     const T* __restrict__ tab,
                                                     T* __restrict__ Y, int L, int H, int Hp,
                                                     int Lp, int B, int C, int S,
                                                     SpinList sout_, int n_tiles_n) {
  using Tile = MfmaTile<T, BM, BN, BK, WM, WN>;
  __shared__ __align__(16) T As[BM * Tile::LD];
  __shared__ __align__(16) T Bs[BN * Tile::LD];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WN, wn = wave % WN;
  const int M = 2 * L - 1;
  const int mi = blockIdx.y, si = blockIdx.z;
  const int m = mi - (L - 1);
  const int spin = sout_.s[si];
  const int lo = iabs(m) > iabs(spin) ? iabs(m) : iabs(spin);
  const int nt = blockIdx.x % n_tiles_n, jt = blockIdx.x / n_tiles_n;
  const int Np = 2 * B * C;
  const int n0 = nt * BM, j0 = jt * BN;
  const int twoC = 2 * C;
  const int kb = (lo / 8) * 8;  // aligned start of the degree range
  const T* Tb = tab + (size_t)(si * M + mi) * Hp * Lp;
  auto brow = [&](int r) -> const T* {
    const int j = j0 + r;
    return j < H ? Tb + (size_t)j * Lp : nullptr;
  };
  Tile tile;
  tile.zero();
  KTileLoader<T, BN, BK, NT> lb;

  // coefficient operand, transposed into LDS: VEC consecutive n' per thread
  constexpr int VEC = 16 / sizeof(T);
  constexpr int VPC = BM / VEC;  // vectors per degree column of the tile
  constexpr int NVA = BK * VPC;
  constexpr int PERA = (NVA + NT - 1) / NT;
  union Vec {
    uint4 u;
    T e[VEC];
  };
  Vec areg[PERA];
  const bool avec = (twoC % VEC) == 0;
  auto load_a = [&](int k0) {
#pragma unroll
    for (int p = 0; p < PERA; ++p) {
      const int v = tid + p * NT;
      if (NVA % NT != 0 && v >= NVA) break;
      const int kl = v / VPC;
      const int nv = (v % VPC) * VEC;
      const int l = k0 + kl;
      const int np = n0 + nv;
      const bool lok = l >= lo && l < L;
      if (lok && avec && np + VEC <= Np) {
        const int b = np / twoC, rem = np - b * twoC;
        areg[p].u = *reinterpret_cast<const uint4*>(
            coef + (((size_t)(l * l + l + m) * B + b) * S + si) * twoC + rem);
      } else {
#pragma unroll
        for (int e = 0; e < VEC; ++e) {
          const int n2 = np + e;
          if (lok && n2 < Np) {
            const int b = n2 / twoC, rem = n2 - b * twoC;
            areg[p].e[e] = coef[(((size_t)(l * l + l + m) * B + b) * S + si) * twoC + rem];
          } else {
            areg[p].e[e] = (T)0.f;
          }
        }
      }
    }
  };
  auto store_a = [&]() {
#pragma unroll
    for (int p = 0; p < PERA; ++p) {
      const int v = tid + p * NT;
      if (NVA % NT != 0 && v >= NVA) break;
      const int kl = v / VPC;
      const int nv = (v % VPC) * VEC;
#pragma unroll
      for (int e = 0; e < VEC; ++e) As[(nv + e) * Tile::LD + kl] = areg[p].e[e];
    }
  };

  load_a(kb);
  lb.load(brow, kb, Lp, tid, true);
  for (int k0 = kb; k0 < L; k0 += BK) {
    __syncthreads();
    store_a();
    lb.store(Bs, tid);
    __syncthreads();
    if (k0 + BK < L) {
      load_a(k0 + BK);
      lb.load(brow, k0 + BK, Lp, tid, true);
    }
    tile.compute(As, Bs, wm, wn, lane);
  }
  T* Y0 = Y + (size_t)(si * M + mi) * Np * Hp;
  tile.for_each(wm, wn, lane, [&](int row, int col, float v) {
    const int np = n0 + row;
    const int j = j0 + col;
    if (np < Np && j < H) Y0[(size_t)np * Hp + j] = (T)v;
  });
}

SpinList make_spins(const int* s, int n) {
  SpinList r{};
  for (int i = 0; i < n && i < kMaxSpins; ++i) r.s[i] = s[i];
  return r;
}

template <typename T, int BM, int BN, int WM, int WN>
hipError_t lat_fwd_cfg(const Plan& p, int B, int C, const void* X, void* coef, hipStream_t st) {
  const int Np = 2 * B * C;
  const int nrt = (p.L + BM - 1) / BM;
  const int nnt = (Np + BN - 1) / BN;
  dim3 grid(nrt * nnt, p.M, p.n_in);
  hipLaunchKernelGGL((lat_fwd_kernel<T, BM, BN, WM, WN>), grid, dim3(NT), 0, st, (const T*)X,
                     (const T*)p.tab_fwd, (T*)coef, p.L, p.H, p.Hp, B, C, p.n_in, nrt);
  return hipGetLastError();
}

template <typename T>
hipError_t lat_fwd_t(const Plan& p, int B, int C, const void* X, void* coef, hipStream_t st) {
  if (p.L > 64) return lat_fwd_cfg<T, 128, 128, 2, 2>(p, B, C, X, coef, st);
  if (p.L > 32) return lat_fwd_cfg<T, 64, 128, 2, 2>(p, B, C, X, coef, st);
  return lat_fwd_cfg<T, 32, 128, 1, 4>(p, B, C, X, coef, st);
}

template <typename T, int BM, int BN, int WM, int WN>
hipError_t mix_cfg(const Plan& p, int B, int Cin, int Cout, const void* coef, const void* K,
                   void* out, hipStream_t st) {
  int tiles = 0;
  for (int l = 0; l < p.L; ++l) tiles += ((2 * l + 1) * B + BM - 1) / BM;
  const int Np = 2 * p.n_out * Cout;
  dim3 grid(tiles, (Np + BN - 1) / BN);
  hipLaunchKernelGGL((mix_kernel<T, BM, BN, WM, WN>), grid, dim3(NT), 0, st, (const T*)coef,
                     (const T*)K, (T*)out, p.L, B, Cin, Cout, p.n_in, p.n_out,
                     make_spins(p.spins_in, p.n_in), make_spins(p.spins_out, p.n_out));
  return hipGetLastError();
}

template <typename T>
hipError_t mix_t(const Plan& p, int B, int Cin, int Cout, const void* coef, const void* K,
                 void* out, hipStream_t st) {
  const int Np = 2 * p.n_out * Cout;
  if (Np >= 128) return mix_cfg<T, 128, 128, 2, 2>(p, B, Cin, Cout, coef, K, out, st);
  return mix_cfg<T, 128, 32, 4, 1>(p, B, Cin, Cout, coef, K, out, st);
}

template <typename T, int BM, int BN, int WM, int WN>
hipError_t lat_inv_cfg(const Plan& p, int B, int C, const void* coef, void* Y, hipStream_t st) {
  const int Np = 2 * B * C;
  const int nnt = (Np + BM - 1) / BM;
  const int njt = (p.H + BN - 1) / BN;
  dim3 grid(nnt * njt, p.M, p.n_out);
  hipLaunchKernelGGL((lat_inv_kernel<T, BM, BN, WM, WN>), grid, dim3(NT), 0, st,
                     (const T*)coef, (const T*)p.tab_inv, (T*)Y, p.L, p.H, p.Hp, p.Lp, B, C,
                     p.n_out, make_spins(p.spins_out, p.n_out), nnt);
  return hipGetLastError();
}

template <typename T>
hipError_t lat_inv_t(const Plan& p, int B, int C, const void* coef, void* Y, hipStream_t st) {
  if (p.H >= 128) return lat_inv_cfg<T, 128, 128, 2, 2>(p, B, C, coef, Y, st);
  if (p.H >= 64) return lat_inv_cfg<T, 128, 64, 2, 2>(p, B, C, coef, Y, st);
  return lat_inv_cfg<T, 128, 32, 4, 1>(p, B, C, coef, Y, st);
}

}  // namespace

hipError_t launch_lat_fwd(const Plan& p, int B, int C, const void* X, void* coef,
                          hipStream_t st) {
  if (p.dtype == SWSFT_BF16) return lat_fwd_t<__bf16>(p, B, C, X, coef, st);
  return lat_fwd_t<float>(p, B, C, X, coef, st);
}

hipError_t launch_mix(const Plan& p, int B, int Cin, int Cout, const void* coef, const void* K,
                      void* out, hipStream_t st) {
  if (p.dtype == SWSFT_BF16) return mix_t<__bf16>(p, B, Cin, Cout, coef, K, out, st);
  return mix_t<float>(p, B, Cin, Cout, coef, K, out, st);
}

hipError_t launch_lat_inv(const Plan& p, int B, int C, const void* coef, void* Y,
                          hipStream_t st) {
  if (p.dtype == SWSFT_BF16) return lat_inv_t<__bf16>(p, B, C, coef, Y, st);
  return lat_inv_t<float>(p, B, C, coef, Y, st);
}

}  // namespace swsft
