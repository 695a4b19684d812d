// The three contractions of the layer, as MFMA GEMMs.
//
//  lat_fwd  (eq. (2), latitude sum), per (spin s, order m):
//     coef[l*l+l+m][b][s][c] = sum_j Tf[s][m][l][j] X[s][m][j][n][re/im]
//     real GEMM: rows l in [|m|, L), columns n' = 2n + re/im, K = j.
//  mix      (per-degree products with filters shared across m), per l:
//     coef'[l][(m,b)][(t,c')] = sum_(s,c) coef[l][(m,b)][(s,c)] K[l][(t,c')][(s,c)]
//     complex GEMM written as a real GEMM with K doubled: each filter row is
//     expanded in LDS into the two real rows (re, -im, ...) and (im, re, ...).
//  lat_inv  (eq. (3), latitude sum), per (spin t, order m):
//     Y[t][m][j][n'] = sum_l coef'[l*l+l+m][b][t][c'][re/im] Ti[t][m][j][l]
//     real GEMM: rows n', columns j, K = l in [max(|m|,|t|), L).
//
// Every operand is staged in LDS K-contiguous; the tables and the K-tiled X /
// Y spectra ([j/32][n'][32]) are laid out so that their global rows already
// are, the
// mixing filters are stored output-major for the same reason, and only the
// coefficient operand of lat_inv is transposed on its way into LDS.
//
// Main loop, epilogue and row loader: gemm_tile.h.
#include "gemm_tile.h"
#include "mfma_tile.h"
#include "swsft_internal.h"
#include "xcd.h"

namespace swsft {
namespace {

// --------------------------------------------------------------------------
// lat_fwd
// --------------------------------------------------------------------------
template <typename T, int BM, int BN, int BK, int WM, int WN, bool kVec>
__global__ void __launch_bounds__(NT) lat_fwd_kernel(const T* __restrict__ X,
                                                     const T* __restrict__ tab,
                                                     T* __restrict__ coef, int L, int H, int Hp,
                                                     int JT, int B, int C, int S, int n_row_tiles,
                                                     int n_tiles_n) {
  using Tile = MfmaTile<T, BM, BN, BK, WM, WN>;
  using G = GemmLds<T, BM, BN, BK>;
  __shared__ __align__(16) T smem[G::bytes / sizeof(T)];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WN, wn = wave % WN;
  const int M = 2 * L - 1;
  // logical block = ((s, order, row tile), column tile): the column tiles of
  // one (s, m, row tile) share its table tile and run on one XCD
  int lbk = xcd_logical_block();
  if (lbk >= S * M * n_row_tiles * n_tiles_n) return;
  const int nt = lbk % n_tiles_n;
  lbk /= n_tiles_n;
  const int rt = lbk % n_row_tiles;
  lbk /= n_row_tiles;
  const int mi = mixed_order(lbk % M, L), si = lbk / M;
  const int m = mi - (L - 1);
  const int l_begin = iabs(m) + rt * BM;
  if (l_begin >= L) return;
  const int Np = 2 * B * C;
  const int n0 = nt * BN;
  const T* A0 = tab + (size_t)(si * M + mi) * L * Hp;
  const T* B0 = X + (size_t)(si * M + mi) * Np * H;  // K-tiled: [H/JT][Np][JT]
  RowLoader<T, BM, BK, kVec> la;
  RowLoader<T, BN, BK, kVec> lb;
  la.init([&](int r) -> const T* { const int l = l_begin + r; return l < L ? A0 + (size_t)l * Hp : nullptr; },
          A0 + (size_t)l_begin * Hp, 0, H, tid);
  lb.init([&](int r) -> const T* { const int np = n0 + r; return np < Np ? B0 + (size_t)np * JT : nullptr; },
          B0 + (size_t)n0 * JT, 0, H, tid, (size_t)Np * JT);
  Tile tile;
  tile.zero();
  mainloop(tile, la, lb, smem, (H + BK - 1) / BK, wm, wn, lane);
  const int twoC = 2 * C;
  epilogue(tile, smem, L - l_begin, Np - n0, wm, wn, lane, tid,
           [&](int row, int col, const Vec16<T>& v, int n) {
             const int l = l_begin + row;
             const size_t rowbase = ((size_t)(l * l + l + m) * B) * S * twoC;
             const int np = n0 + col;
             if (kVec && n == Vec16<T>::N) {
               const int b = np / twoC, rem = np - b * twoC;
               *reinterpret_cast<uint4*>(&coef[rowbase + ((size_t)b * S + si) * twoC + rem]) = v.u;
             } else {
#pragma unroll
               for (int e = 0; e < Vec16<T>::N; ++e) {
                 if (e >= n) break;
                 const int b = (np + e) / twoC, rem = np + e - b * twoC;
                 coef[rowbase + ((size_t)b * S + si) * twoC + rem] = v.e[e];
               }
             }
           });
}

// --------------------------------------------------------------------------
// mix
// --------------------------------------------------------------------------
// Filter operand: BN/2 complex filter rows q (output (t, c')) become the BN
// real rows (2q: re, -im pairs; 2q+1: im, re pairs) of the real GEMM.
// Input spins that do not exist at degree l are zeroed: per K tile when a
// tile lies inside one spin's channel block, else per element.
template <typename T, int BN, int BK, bool kVec>
struct FilterLoader {
  static constexpr int VEC = 16 / sizeof(T);   // reals per vector
  static constexpr int VPR = BK / VEC;
  static constexpr int NV = (BN / 2) * VPR;
  static constexpr int PER = (NV + NT - 1) / NT;
  static constexpr int LD = BK + LdsPad<T>::value;
  Vec16<T> reg[PER];
  const T* rows_[PER];
  bool rowok_[PER];
  unsigned ok_[PER];
  int kv_[PER];
  int Kp, Cin, l;
  bool tile_spin;
  unsigned dead_;  // bit si: input spin si does not exist at degree l

  __device__ __forceinline__ void init(const T* K0, int n0, int Nc, int Kp_, int Cin_, int Cout,
                                       int l_, const SpinList& sin, const SpinList& sout,
                                       int tid) {
    Kp = Kp_;
    Cin = Cin_;
    l = l_;
    tile_spin = ((2 * Cin) % BK) == 0;
    dead_ = 0;
    for (int i = 0; i < kMaxSpins; ++i)
      if (i * Cin < Kp / 2 && iabs(sin.s[i]) > l) dead_ |= 1u << i;
#pragma unroll
    for (int p = 0; p < PER; ++p) {
      const int v = tid + p * NT;
      const int q = n0 / 2 + v / VPR;
      const bool ok = (NV % NT == 0 || v < NV) && q < Nc && iabs(sout.s[q < Nc ? q / Cout : 0]) <= l;
      rowok_[p] = ok;
      rows_[p] = ok ? K0 + (size_t)q * Kp : K0;
      kv_[p] = (v % VPR) * VEC;
    }
  }
  __device__ __forceinline__ void load(int kt) {
    // tile-uniform spin test (scalar)
    const bool tile_dead = tile_spin && ((dead_ >> ((kt * BK) / (2 * Cin))) & 1u);
#pragma unroll
    for (int p = 0; p < PER; ++p) {
      const int k = kt * BK + kv_[p];
      unsigned bits;
      if constexpr (kVec) {
        const bool ok = rowok_[p] && k < Kp;
        reg[p].u = *reinterpret_cast<const uint4*>(rows_[p] + (ok ? k : 0));
        bits = ok ? 0xffu : 0u;
      } else {
        bits = 0;
#pragma unroll
        for (int e = 0; e < VEC; ++e) {
          const bool ok = rowok_[p] && k + e < Kp;
          reg[p].e[e] = rows_[p][ok ? k + e : 0];
          bits |= (ok ? 1u : 0u) << e;
        }
      }
      if (tile_spin) {
        if (tile_dead) bits = 0;
      } else {
#pragma unroll
        for (int e = 0; e < VEC; e += 2) {
          const int pc = (k + e) >> 1;
          if (pc < Kp / 2 && ((dead_ >> (pc / Cin)) & 1u)) bits &= ~(3u << e);
        }
      }
      ok_[p] = bits;
    }
  }
  __device__ __forceinline__ void store(T* lds) {
    const int tid = threadIdx.x;
#pragma unroll
    for (int p = 0; p < PER; ++p) {
      const int v = tid + p * NT;
      if (NV % NT != 0 && v >= NV) break;
      const int r = v / VPR;
      if (ok_[p] == 0) {
        reg[p].u = make_uint4(0, 0, 0, 0);
      } else if (ok_[p] != 0xffu) {
#pragma unroll
        for (int e = 0; e < VEC; ++e)
          if (!((ok_[p] >> e) & 1u)) reg[p].e[e] = (T)0.f;
      }
      T* re_row = lds + (2 * r) * LD + kv_[p];
      T* im_row = lds + (2 * r + 1) * LD + kv_[p];
      if constexpr (sizeof(T) == 2) {
        // packed (re, im) bf16 pairs: (re, -im) flips the sign bit of the high
        // half, (im, re) swaps the halves
        const uint4 a = reg[p].u;
        const uint4 neg = make_uint4(a.x ^ 0x80000000u, a.y ^ 0x80000000u, a.z ^ 0x80000000u,
                                     a.w ^ 0x80000000u);
        const uint4 bsw = make_uint4((a.x >> 16) | (a.x << 16), (a.y >> 16) | (a.y << 16),
                                     (a.z >> 16) | (a.z << 16), (a.w >> 16) | (a.w << 16));
        *reinterpret_cast<uint4*>(re_row) = neg;
        *reinterpret_cast<uint4*>(im_row) = bsw;
      } else {
#pragma unroll
        for (int e = 0; e < VEC; e += 2) {
          const T kr = reg[p].e[e], ki = reg[p].e[e + 1];
          re_row[e] = kr;
          re_row[e + 1] = -ki;
          im_row[e] = ki;
          im_row[e + 1] = kr;
        }
      }
    }
  }
};

template <typename T, int BM, int BN, int BK, int WM, int WN, bool kVec>
__global__ void __launch_bounds__(NT) mix_kernel(const T* __restrict__ coef,
                                                 const T* __restrict__ K, T* __restrict__ out,
                                                 int L, int B, int Cin, int Cout, int Sin,
                                                 int Sout, SpinList sin_, SpinList sout_) {
  using Tile = MfmaTile<T, BM, BN, BK, WM, WN>;
  extern __shared__ __align__(16) unsigned char mix_smem[];  // GemmLds<T, BM, BN, BK>::bytes
  T* smem = reinterpret_cast<T*>(mix_smem);
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WN, wn = wave % WN;
  // logical block = ((l, row tile), column tile), largest degrees first: all
  // tiles of one degree (its filter block and coefficient rows) are numbered
  // together and run on one XCD
  const int Np_ = 2 * Sout * Cout;
  const int n_tiles_n = (Np_ + BN - 1) / BN;
  int lbk = xcd_logical_block();
  const int ntile = lbk % n_tiles_n;
  int t = lbk / n_tiles_n;
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
  const int n0 = ntile * BN;
  const T* A0 = coef + (size_t)l * l * B * Kp;
  const T* K0 = K + (size_t)l * Nc * Kc * 2;
  RowLoader<T, BM, BK, kVec> la;
  la.init([&](int r) -> const T* { const int i = row0 + r; return i < Mrows ? A0 + (size_t)i * Kp : nullptr; },
          A0 + (size_t)row0 * Kp, 0, Kp, tid);
  FilterLoader<T, BN, BK, kVec> lb;
  lb.init(K0, n0, Nc, Kp, Cin, Cout, l, sin_, sout_, tid);
  Tile tile;
  tile.zero();
  mainloop(tile, la, lb, smem, (Kp + BK - 1) / BK, wm, wn, lane);
  T* O0 = out + ((size_t)l * l * B + row0) * Np + n0;
  epilogue(tile, smem, Mrows - row0, Np - n0, wm, wn, lane, tid,
           [&](int row, int col, const Vec16<T>& v, int n) {
             T* dst = O0 + (size_t)row * Np + col;
             if (kVec && n == Vec16<T>::N) {
               *reinterpret_cast<uint4*>(dst) = v.u;
             } else {
#pragma unroll
               for (int e = 0; e < Vec16<T>::N; ++e)
                 if (e < n) dst[e] = v.e[e];
             }
           });
}

// --------------------------------------------------------------------------
// lat_inv
// --------------------------------------------------------------------------
// Coefficient operand transposed into LDS: each thread reads 16-byte runs
// of consecutive n' for two consecutive degrees and writes degree pairs;
// consecutive lanes take consecutive degree pairs of the same n' run, so the
// pair writes of a wave fall in distinct banks.  Loads use clamped
// addresses; the zero mask is applied at the LDS store.
template <typename T, int BM, int BK, bool kVec>
struct CoefTLoader {
  static constexpr int VEC = 16 / sizeof(T);
  static constexpr int NV = (BK / 2) * (BM / VEC);
  static constexpr int PER = (NV + NT - 1) / NT;
  static constexpr int LD = BK + LdsPad<T>::value;
  Vec16<T> reg[PER][2];
  unsigned ok_[PER][2];
  const T* coef;
  int m, B, S, si, twoC, Np, n0, lo, L, k_base;

  __device__ __forceinline__ size_t offset(int l, int n2) const {
    const int b = n2 / twoC, rem = n2 - b * twoC;
    return ((size_t)(l * l + l + m) * B + b) * S * twoC + (size_t)si * twoC + rem;
  }
  __device__ __forceinline__ void load(int kt) {
    const int tid = threadIdx.x;
#pragma unroll
    for (int p = 0; p < PER; ++p) {
      const int v = tid + p * NT;
      const int kl = 2 * (v % (BK / 2));
      const int np = n0 + (v / (BK / 2)) * VEC;
      const bool vok = NV % NT == 0 || v < NV;
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const int l = k_base + kt * BK + kl + h;
        const bool lok = vok && l >= lo && l < L;
        if constexpr (kVec) {
          const bool ok = lok && np < Np;
          reg[p][h].u = *reinterpret_cast<const uint4*>(coef + (ok ? offset(l, np) : 0));
          ok_[p][h] = ok ? 0xffu : 0u;
        } else {
          unsigned bits = 0;
#pragma unroll
          for (int e = 0; e < VEC; ++e) {
            const bool ok = lok && np + e < Np;
            reg[p][h].e[e] = coef[ok ? offset(l, np + e) : 0];
            bits |= (ok ? 1u : 0u) << e;
          }
          ok_[p][h] = bits;
        }
      }
    }
  }
  __device__ __forceinline__ void store(T* lds) {
    const int tid = threadIdx.x;
#pragma unroll
    for (int p = 0; p < PER; ++p) {
      const int v = tid + p * NT;
      if (NV % NT != 0 && v >= NV) break;
      const int kl = 2 * (v % (BK / 2));
      const int nv = (v / (BK / 2)) * VEC;
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        if (ok_[p][h] == 0) {
          reg[p][h].u = make_uint4(0, 0, 0, 0);
        } else if (ok_[p][h] != 0xffu) {
#pragma unroll
          for (int e = 0; e < VEC; ++e)
            if (!((ok_[p][h] >> e) & 1u)) reg[p][h].e[e] = (T)0.f;
        }
      }
      if constexpr (sizeof(T) == 2) {
#pragma unroll
        for (int e = 0; e < VEC; ++e) {
          const uint32_t lo16 = __builtin_bit_cast(uint16_t, reg[p][0].e[e]);
          const uint32_t hi16 = __builtin_bit_cast(uint16_t, reg[p][1].e[e]);
          *reinterpret_cast<uint32_t*>(&lds[(nv + e) * LD + kl]) = lo16 | (hi16 << 16);
        }
      } else {
#pragma unroll
        for (int e = 0; e < VEC; ++e) {
          lds[(nv + e) * LD + kl] = reg[p][0].e[e];
          lds[(nv + e) * LD + kl + 1] = reg[p][1].e[e];
        }
      }
    }
  }
};

template <typename T, int BM, int BN, int BK, int WM, int WN, bool kVec>
__global__ void __launch_bounds__(NT) lat_inv_kernel(const T* __restrict__ coef,
                                                     const T* __restrict__ tab,
                                                     T* __restrict__ Y, int L, int H, int Hp,
                                                     int JT, int Lp, int B, int Bc, int C, int S,
                                                     SpinList sout_, int n_tiles_n) {
  using Tile = MfmaTile<T, BM, BN, BK, WM, WN>;
  using G = GemmLds<T, BM, BN, BK>;
  __shared__ __align__(16) T smem[G::bytes / sizeof(T)];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WN, wn = wave % WN;
  const int M = 2 * L - 1;
  // logical block = ((s, order, j tile), n' tile): the n' tiles of one
  // (s, m, j tile) share its table tile and run on one XCD
  const int n_tiles_j = (H + BN - 1) / BN;
  int lbk = xcd_logical_block();
  if (lbk >= S * M * n_tiles_j * n_tiles_n) return;
  const int nt = lbk % n_tiles_n;
  lbk /= n_tiles_n;
  const int jt = lbk % n_tiles_j;
  lbk /= n_tiles_j;
  const int mi = mixed_order(lbk % M, L), si = lbk / M;
  const int m = mi - (L - 1);
  const int spin = sout_.s[si];
  const int lo = iabs(m) > iabs(spin) ? iabs(m) : iabs(spin);
  const int Np = 2 * B * C;
  const int n0 = nt * BM, j0 = jt * BN;
  const int kb = (lo / 8) * 8;  // aligned start of the degree range
  const T* Tb = tab + (size_t)(si * M + mi) * Hp * Lp;
  CoefTLoader<T, BM, BK, kVec> la;
  la.coef = coef;
  la.m = m;
  la.B = Bc;  // rows of the coefficient array hold Bc batch items
  la.S = S;
  la.si = si;
  la.twoC = 2 * C;
  la.Np = Np;
  la.n0 = n0;
  la.lo = lo;
  la.L = L;
  la.k_base = kb;
  RowLoader<T, BN, BK, true> lb;  // table rows: Lp is a multiple of 32
  lb.init([&](int r) -> const T* { const int j = j0 + r; return j < H ? Tb + (size_t)j * Lp : nullptr; },
          Tb + (size_t)j0 * Lp, kb, Lp, tid);
  Tile tile;
  tile.zero();
  mainloop(tile, la, lb, smem, (L - kb + BK - 1) / BK, wm, wn, lane);
  // Y K-tiled: [H/JT][Np][JT]; element (n', j) at (j / JT) Np JT + n' JT + j % JT
  T* Y0 = Y + (size_t)(si * M + mi) * Np * H;
  const size_t tstride = (size_t)Np * JT;
  epilogue(tile, smem, Np - n0, H - j0, wm, wn, lane, tid,
           [&](int row, int col, const Vec16<T>& v, int n) {
             const int np = n0 + row, j = j0 + col;
             if (n == Vec16<T>::N) {  // 8 consecutive j inside one tile (JT is a multiple of 8)
               *reinterpret_cast<uint4*>(Y0 + (j / JT) * tstride + (size_t)np * JT + j % JT) = v.u;
             } else {
#pragma unroll
               for (int e = 0; e < Vec16<T>::N; ++e)
                 if (e < n) Y0[((j + e) / JT) * tstride + (size_t)np * JT + (j + e) % JT] = v.e[e];
             }
           });
}

SpinList make_spins(const int* s, int n) {
  SpinList r{};
  for (int i = 0; i < n && i < kMaxSpins; ++i) r.s[i] = s[i];
  return r;
}

// K step of each contraction for bf16 storage (float uses 32).
#ifndef SWSFT_BK_LAT_FWD
#define SWSFT_BK_LAT_FWD 32
#endif
#ifndef SWSFT_BK_MIX
#define SWSFT_BK_MIX 32
#endif
#ifndef SWSFT_BK_LAT_INV
#define SWSFT_BK_LAT_INV 32
#endif
template <typename T, int kBf16>
constexpr int kBK = sizeof(T) == 2 ? kBf16 : 32;

template <typename T, int BM, int BN, int WM, int WN>
hipError_t lat_fwd_cfg(const Plan& p, int B, int C, const void* X, void* coef, hipStream_t st) {
  const int Np = 2 * B * C;
  const int nrt = (p.L + BM - 1) / BM;
  const int nnt = (Np + BN - 1) / BN;
  const long long blocks = (long long)nrt * nnt * p.M * p.n_in;
  constexpr int VEC = 16 / sizeof(T);
  auto kern = (p.H % VEC == 0 && (2 * C) % VEC == 0) ? lat_fwd_kernel<T, BM, BN, kBK<T, SWSFT_BK_LAT_FWD>, WM, WN, true>
                                                      : lat_fwd_kernel<T, BM, BN, kBK<T, SWSFT_BK_LAT_FWD>, WM, WN, false>;
  hipLaunchKernelGGL(kern, dim3(xcd_grid(blocks)), dim3(NT), 0, st, (const T*)X, (const T*)p.tab_fwd,
                     (T*)coef, p.L, p.H, p.Hp, p.JT, B, C, p.n_in, nrt, nnt);
  return hipGetLastError();
}

#ifndef SWSFT_LAT_FWD_TILE
#define SWSFT_LAT_FWD_TILE 128, 128, 2, 2
#endif

template <typename T>
hipError_t lat_fwd_t(const Plan& p, int B, int C, const void* X, void* coef, hipStream_t st) {
  if (p.L > 64) return lat_fwd_cfg<T, SWSFT_LAT_FWD_TILE>(p, B, C, X, coef, st);
  if (p.L > 32) return lat_fwd_cfg<T, 64, 128, 2, 2>(p, B, C, X, coef, st);
  return lat_fwd_cfg<T, 32, 128, 1, 4>(p, B, C, X, coef, st);
}

// Workgroups of the mixing GEMM with BM x BN tiles.
long long mix_blocks(const Plan& p, int B, int Cout, int BM, int BN) {
  long long tiles = 0;
  for (int l = 0; l < p.L; ++l) tiles += ((2 * l + 1) * B + BM - 1) / BM;
  return tiles * ((2 * p.n_out * Cout + BN - 1) / BN);
}

// K step of the float mixing GEMM (bf16 uses SWSFT_BK_MIX).
#ifndef SWSFT_BK_MIX_F32
#define SWSFT_BK_MIX_F32 32
#endif

template <typename T, int BM, int BN, int WM, int WN>
hipError_t mix_cfg(const Plan& p, int B, int Cin, int Cout, const void* coef, const void* K,
                   void* out, hipStream_t st) {
  const int Np = 2 * p.n_out * Cout, Kp = 2 * p.n_in * Cin;
  const long long blocks = mix_blocks(p, B, Cout, BM, BN);
  constexpr int VEC = 16 / sizeof(T);
  constexpr int BK = sizeof(T) == 2 ? SWSFT_BK_MIX : SWSFT_BK_MIX_F32;
  auto kern = (Kp % VEC == 0 && Np % VEC == 0) ? mix_kernel<T, BM, BN, BK, WM, WN, true>
                                               : mix_kernel<T, BM, BN, BK, WM, WN, false>;
  const size_t lds = GemmLds<T, BM, BN, BK>::bytes;
  const hipError_t e = ensure_dynamic_lds((const void*)kern, lds);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(kern, dim3(xcd_grid(blocks)), dim3(NT), lds, st, (const T*)coef, (const T*)K,
                     (T*)out, p.L, B, Cin, Cout, p.n_in, p.n_out, make_spins(p.spins_in, p.n_in),
                     make_spins(p.spins_out, p.n_out));
  return hipGetLastError();
}

// Tile of the large-channel mixing GEMM (rows x columns, waves per dim): the
// largest of 128 x 128, 64 x 128 and 64 x 64 that still gives two
// workgroups per CU (the degrees are few and short at small bandlimits, and
// a 128 x 128 tiling then leaves CUs idle).
template <typename T>
hipError_t mix_t(const Plan& p, int B, int Cin, int Cout, const void* coef, const void* K,
                 void* out, hipStream_t st) {
  const int Np = 2 * p.n_out * Cout;
  constexpr long long kWant = 2LL * 256;
  if (Np >= 128) {
    if (mix_blocks(p, B, Cout, 128, 128) >= kWant)
      return mix_cfg<T, 128, 128, 2, 2>(p, B, Cin, Cout, coef, K, out, st);
    if (mix_blocks(p, B, Cout, 64, 128) >= kWant)
      return mix_cfg<T, 64, 128, 2, 2>(p, B, Cin, Cout, coef, K, out, st);
    return mix_cfg<T, 64, 64, 2, 2>(p, B, Cin, Cout, coef, K, out, st);
  }
  return mix_cfg<T, 128, 32, 4, 1>(p, B, Cin, Cout, coef, K, out, st);
}

template <typename T, int BM, int BN, int WM, int WN>
hipError_t lat_inv_cfg(const Plan& p, int B, int C, const void* coef, void* Y, hipStream_t st) {
  const int Np = 2 * B * C;
  const int nnt = (Np + BM - 1) / BM;
  const int njt = (p.H + BN - 1) / BN;
  const long long blocks = (long long)nnt * njt * p.M * p.n_out;
  constexpr int VEC = 16 / sizeof(T);
  auto kern = ((2 * C) % VEC == 0) ? lat_inv_kernel<T, BM, BN, kBK<T, SWSFT_BK_LAT_INV>, WM, WN, true>
                                   : lat_inv_kernel<T, BM, BN, kBK<T, SWSFT_BK_LAT_INV>, WM, WN, false>;
  hipLaunchKernelGGL(kern, dim3(xcd_grid(blocks)), dim3(NT), 0, st, (const T*)coef,
                     (const T*)p.tab_inv, (T*)Y, p.L, p.H, p.Hp, p.JT, p.Lp, B,
                     p.coef_ldb > 0 ? p.coef_ldb : B, C, p.n_out,
                     make_spins(p.spins_out, p.n_out), nnt);
  return hipGetLastError();
}

#ifndef SWSFT_LAT_INV_TILE
#define SWSFT_LAT_INV_TILE 128, 128, 2, 2
#endif

template <typename T>
hipError_t lat_inv_t(const Plan& p, int B, int C, const void* coef, void* Y, hipStream_t st) {
  if (p.H >= 128) return lat_inv_cfg<T, SWSFT_LAT_INV_TILE>(p, B, C, coef, Y, st);
  if (p.H >= 64) return lat_inv_cfg<T, 128, 64, 2, 2>(p, B, C, coef, Y, st);
  return lat_inv_cfg<T, 128, 32, 4, 1>(p, B, C, coef, Y, st);
}

}  // namespace

#ifndef SWSFT_DMA
#define SWSFT_DMA 1
#endif

hipError_t launch_lat_fwd(const Plan& p, int B, int C, const void* X, void* coef,
                          hipStream_t st) {
  if (SWSFT_DMA && lat_fwd_dma_supported(p, B, C)) return launch_lat_fwd_dma(p, B, C, X, coef, st);
  if (p.dtype == SWSFT_BF16) return lat_fwd_t<__bf16>(p, B, C, X, coef, st);
  return lat_fwd_t<float>(p, B, C, X, coef, st);
}

hipError_t launch_mix(const Plan& p, int B, int Cin, int Cout, const void* coef, const void* K,
                      void* out, hipStream_t st) {
  if (SWSFT_DMA && mix_dma_supported(p, Cin, Cout))
    return launch_mix_dma(p, B, Cin, Cout, coef, K, out, st);
  if (p.dtype == SWSFT_BF16) return mix_t<__bf16>(p, B, Cin, Cout, coef, K, out, st);
  return mix_t<float>(p, B, Cin, Cout, coef, K, out, st);
}

hipError_t launch_lat_inv(const Plan& p, int B, int C, const void* coef, void* Y,
                          hipStream_t st) {
  if (SWSFT_DMA && lat_inv_dma_supported(p, B, C)) return launch_lat_inv_dma(p, B, C, coef, Y, st);
  if (p.dtype == SWSFT_BF16) return lat_inv_t<__bf16>(p, B, C, coef, Y, st);
  return lat_inv_t<float>(p, B, C, coef, Y, st);
}

}  // namespace swsft
