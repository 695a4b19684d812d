// Latitude stages of the transform (bfloat16 and float storage), as GEMMs
// whose operands are copied global -> LDS directly
// (global_load_lds_dwordx4; see lds_dma.h) into a ring of K steps.
//
//   forward  coef[l][m][b][s][c] = sum_j Tf[s][m][l][j] X[s][m][j][b c]      (eq. (4))
//   inverse  Y[s][m][j][b c]     = sum_l Ti[s][m][j][l] coef'[l][m][b][s][c]  (eq. (3))
//
// X, Y and the coefficients are complex, stored as (re, im) pairs, so each
// (s, m) is one real GEMM with N = 2 B C.  The tables already hold the
// quadrature weights (forward) and are zero below max(|m|, |s|), so the
// triangular degree ranges need no masking inside the K loop.
//
// Forward: A = table rows l (K = j contiguous), B = spectrum rows n' from the
// K-tiled layout [H/32][2BC][32] (16 rows x 32 latitudes = one contiguous
// KiB).  Inverse: the coefficient operand is stored l-major, so its tile
// enters LDS K-major ([l][n']) and MFMA fragments are read from it with the
// transposed LDS read (ds_read_b64_tr_b16), two per fragment; B = table rows
// j (K = l contiguous).  Each wave owns 64 x 64 outputs (2 x 2 MFMA
// 32x32x16 tiles).
#include <type_traits>

#include "lds_dma.h"
#include "mfma_tile.h"
#include "swsft_internal.h"
#include "xcd.h"

namespace swsft {
namespace {

constexpr int kJT = 32;  // latitude tile of the K-tiled spectra

struct SpinList {
  int s[kMaxSpins];
};

__device__ __forceinline__ int iabs_(int v) { return v < 0 ? -v : v; }
__device__ __forceinline__ int imin_(int a, int b) { return a < b ? a : b; }

typedef unsigned v4u __attribute__((ext_vector_type(4)));
typedef short v4s __attribute__((ext_vector_type(4)));
typedef short v8s __attribute__((ext_vector_type(8)));

// Accumulators of a wave's 64 x 64 block -> LDS tile [rows][LDC] of bf16.
__device__ __forceinline__ void acc_to_lds(const v16f (&acc)[2][2], __bf16* cs, int LDC, int wm,
                                           int wn, int lane) {
  const int col_l = lane & 31, row_l = 4 * (lane >> 5);
#pragma unroll
  for (int ii = 0; ii < 2; ++ii)
#pragma unroll
    for (int jj = 0; jj < 2; ++jj)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = wm * 64 + ii * 32 + 8 * (r >> 2) + row_l + (r & 3);
        const int col = wn * 64 + jj * 32 + col_l;
        cs[row * LDC + col] = (__bf16)acc[ii][jj][r];
      }
}

__device__ __forceinline__ void zero_acc(v16f (&acc)[2][2]) {
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;
}

// ---------------------------------------------------------------------------
// forward
// ---------------------------------------------------------------------------
template <int BK, int RA, int RB, int ST>
struct FwdGeom {
  static constexpr int WM = RA / 64, WN = RB / 64;
  static constexpr int NW = WM * WN, NT = 64 * NW;
  static constexpr int PITCH = 2 * BK;  // bytes per tile row
  static constexpr int CPR = PITCH / 16;
  static constexpr int RPI = 1024 / PITCH;  // rows per 1 KiB copy
  static constexpr int LPR = 64 / RPI;      // lanes per row
  static constexpr int NI = (RA + RB) / RPI;
  static constexpr int PER_WAVE = NI / NW;
  static constexpr int STAGE = (RA + RB) * PITCH;
  static constexpr int LDC = RB + 8;
  static constexpr int RING = ST * STAGE, CTILE = RA * LDC * 2;
  static constexpr int SMEM = RING > CTILE ? RING : CTILE;
  static_assert(BK % kJT == 0 && RA % RPI == 0 && NI % NW == 0 && RA % 64 == 0 &&
                    RB % 64 == 0 && ST >= 2 && (ST - 2) * PER_WAVE < 64,
                "tile shape");
};

template <int BK, int RA, int RB, int ST>
__global__ void __launch_bounds__((FwdGeom<BK, RA, RB, ST>::NT))
    lat_fwd_dma_kernel(const __bf16* __restrict__ X, const __bf16* __restrict__ tab,
                       __bf16* __restrict__ coef, int L, int H, int B, int C, int S,
                       int n_row_tiles, int n_tiles_n) {
  using G = FwdGeom<BK, RA, RB, ST>;
  __shared__ __align__(16) unsigned char smem[G::SMEM];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / G::WN, wn = wave % G::WN;
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
  const int l_begin = iabs_(m) + rt * RA;
  if (l_begin >= L) return;
  const int Np = 2 * B * C;
  const int n0 = nt * RB;
  const __bf16* A0 = tab + (size_t)(si * M + mi) * L * H;  // rows l of H latitudes
  const __bf16* B0 = X + (size_t)(si * M + mi) * Np * H;   // [H/32][Np][32]

  // copy g = wave * PER_WAVE + u moves stage rows [g RPI, (g + 1) RPI) of
  // [A rows; B rows]; rows past the end are clamped (their outputs are
  // discarded)
  const __bf16* src[G::PER_WAVE];
  int step[G::PER_WAVE];  // elements between consecutive K steps
#pragma unroll
  for (int u = 0; u < G::PER_WAVE; ++u) {
    const int g = wave * G::PER_WAVE + u;
    const int tr = g * G::RPI + lane / G::LPR, slot = lane % G::LPR;
    if (tr < RA) {
      const int l = imin_(l_begin + tr, L - 1);
      src[u] = A0 + (size_t)l * H + swz<G::CPR>(tr, slot) * 8;
      step[u] = BK;
    } else {
      const int rb = tr - RA;
      const int np = imin_(n0 + rb, Np - 1);
      const int k = swz<G::CPR>(rb, slot) * 8;  // latitude offset inside the K step
      src[u] = B0 + (size_t)(k / kJT) * Np * kJT + (size_t)np * kJT + k % kJT;
      step[u] = (BK / kJT) * Np * kJT;
    }
  }
  const unsigned ring = lds_addr(smem);
  auto issue = [&](int i, int stage) {
    const unsigned base = ring + stage * G::STAGE + wave * G::PER_WAVE * 1024;
#pragma unroll
    for (int u = 0; u < G::PER_WAVE; ++u) dma16(src[u] + (size_t)i * step[u], base + u * 1024);
  };

  v16f acc[2][2];
  zero_acc(acc);
  const int nk = H / BK;
#pragma unroll
  for (int s = 0; s < ST - 1; ++s)
    if (s < nk) issue(s, s);
  const int r32 = lane & 31, kh = lane >> 5;
  // The K loop for NL row blocks of 32 degrees that exist (l < L); blocks of
  // the tile past the last degree (orders |m| near L leave most of a tile
  // empty) issue neither operand reads nor MFMAs.  NL is wave-uniform.
  auto k_loop = [&](auto nl) {
    constexpr int NL = decltype(nl)::value;
    for (int i = 0; i < nk; ++i) {
      const int issued = nk < i + ST - 1 ? nk : i + ST - 1;
      wait_groups<ST - 2, G::PER_WAVE>(issued - i - 1);
      __builtin_amdgcn_s_barrier();  // step i landed for every wave; step i-1 is consumed
      if (i + ST - 1 < nk) issue(i + ST - 1, (i + ST - 1) % ST);
      if constexpr (NL > 0) {
        const unsigned char* As = smem + (i % ST) * G::STAGE;
        const unsigned char* Bs = As + RA * G::PITCH;
#pragma unroll
        for (int kk = 0; kk < BK / 16; ++kk) {
          const int c = 2 * kk + kh;
          v8bf a[2], b[2];
#pragma unroll
          for (int ii = 0; ii < NL; ++ii) {
            const int r = wm * 64 + ii * 32 + r32;
            a[ii] = *reinterpret_cast<const v8bf*>(As + r * G::PITCH + swz<G::CPR>(r, c) * 16);
          }
#pragma unroll
          for (int jj = 0; jj < 2; ++jj) {
            const int r = wn * 64 + jj * 32 + r32;
            b[jj] = *reinterpret_cast<const v8bf*>(Bs + r * G::PITCH + swz<G::CPR>(r, c) * 16);
          }
#pragma unroll
          for (int ii = 0; ii < NL; ++ii)
#pragma unroll
            for (int jj = 0; jj < 2; ++jj)
              acc[ii][jj] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[ii], b[jj], acc[ii][jj], 0, 0, 0);
        }
      }
    }
  };
  const int wrow = __builtin_amdgcn_readfirstlane(l_begin + wm * 64);
  if (wrow + 32 < L) k_loop(std::integral_constant<int, 2>{});
  else if (wrow < L) k_loop(std::integral_constant<int, 1>{});
  else k_loop(std::integral_constant<int, 0>{});
  wait_vmcnt<0>();
  __syncthreads();

  // epilogue: rows l, columns n' = (b, c, re/im); 8 columns stay inside one
  // b because 2C is a multiple of 8 (rows past L are not stored)
  __bf16* cs = reinterpret_cast<__bf16*>(smem);
  acc_to_lds(acc, cs, G::LDC, wm, wn, lane);
  __syncthreads();
  const int twoC = 2 * C;
  constexpr int VPR = RB / 8;
  for (int idx = tid; idx < RA * VPR; idx += G::NT) {
    const int row = idx / VPR, col = (idx % VPR) * 8;
    const int l = l_begin + row, np = n0 + col;
    if (l >= L || np >= Np) continue;
    const int b = np / twoC, rem = np - b * twoC;
    const uint4 v = *reinterpret_cast<const uint4*>(&cs[row * G::LDC + col]);
    *reinterpret_cast<uint4*>(&coef[((size_t)(l * l + l + m) * B + b) * S * twoC +
                                    (size_t)si * twoC + rem]) = v;
  }
}

// Float forward: K steps of 32 latitudes (128 bytes per row and copy); each
// of the 4 waves owns 32 rows l x 64 columns n' (two MFMA 32x32x2 chains;
// a 16-byte chunk's four latitudes feed two steps, lane half kh taking
// latitudes 2 kh and 2 kh + 1 from one 8-byte read of each operand); the
// workgroup covers 32 WM rows x 64 WN columns.
template <int WM, int WN, int ST>
struct FwdGeomF {
  static constexpr int BK = 32, PITCH = 4 * BK, CPR = PITCH / 16;
  static constexpr int RPI = 1024 / PITCH, LPR = 64 / RPI;
  static constexpr int NW = WM * WN, NT = 64 * NW;
  static constexpr int RA = 32 * WM, RB = 64 * WN;
  static constexpr int NI = (RA + RB) / RPI, PER_WAVE = NI / NW;
  static constexpr int STAGE = (RA + RB) * PITCH;
  static constexpr int LDC = RB + 4;  // floats per row of the output tile
  static constexpr int RING = ST * STAGE, CTILE = RA * LDC * 4;
  static constexpr int SMEM = RING > CTILE ? RING : CTILE;
  static_assert(BK == kJT && (RA + RB) % RPI == 0 && NI % NW == 0 && ST >= 1 &&
                    (ST - 2) * PER_WAVE < 64,
                "tile shape");
};

template <int WM, int WN, int ST>
__global__ void __launch_bounds__((FwdGeomF<WM, WN, ST>::NT))
    lat_fwd_dma_f32_kernel(const float* __restrict__ X, const float* __restrict__ tab,
                           float* __restrict__ coef, int L, int H, int B, int C, int S,
                           int n_row_tiles, int n_tiles_n) {
  using G = FwdGeomF<WM, WN, ST>;
  constexpr int RA = G::RA, RB = G::RB, BK = G::BK;
  extern __shared__ __align__(16) unsigned char smem[];  // G::SMEM bytes
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WN, wn = wave % WN;
  const int M = 2 * L - 1;
  // logical block = ((s, order, row tile), column tile), as for bf16
  int lbk = xcd_logical_block();
  if (lbk >= S * M * n_row_tiles * n_tiles_n) return;
  const int nt = lbk % n_tiles_n;
  lbk /= n_tiles_n;
  const int rt = lbk % n_row_tiles;
  lbk /= n_row_tiles;
  const int mi = mixed_order(lbk % M, L), si = lbk / M;
  const int m = mi - (L - 1);
  const int l_begin = iabs_(m) + rt * RA;
  if (l_begin >= L) return;
  const int Np = 2 * B * C;
  const int n0 = nt * RB;
  const float* A0 = tab + (size_t)(si * M + mi) * L * H;  // rows l of H latitudes
  const float* B0 = X + (size_t)(si * M + mi) * Np * H;   // [H/32][Np][32]

  const float* src[G::PER_WAVE];
  int step[G::PER_WAVE];  // elements between consecutive K steps
#pragma unroll
  for (int u = 0; u < G::PER_WAVE; ++u) {
    const int g = wave * G::PER_WAVE + u;
    const int tr = g * G::RPI + lane / G::LPR, slot = lane % G::LPR;
    if (tr < RA) {
      const int l = imin_(l_begin + tr, L - 1);
      src[u] = A0 + (size_t)l * H + swz<G::CPR>(tr, slot) * 4;
      step[u] = BK;
    } else {
      const int rb = tr - RA;
      const int np = imin_(n0 + rb, Np - 1);
      src[u] = B0 + (size_t)np * kJT + swz<G::CPR>(rb, slot) * 4;
      step[u] = Np * kJT;
    }
  }
  const unsigned ring = lds_addr(smem);
  auto issue = [&](int i, int stage) {
    const unsigned base = ring + stage * G::STAGE + wave * G::PER_WAVE * 1024;
#pragma unroll
    for (int u = 0; u < G::PER_WAVE; ++u) dma16(src[u] + (size_t)i * step[u], base + u * 1024);
  };

  v16f acc[2];
#pragma unroll
  for (int j = 0; j < 2; ++j)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[j][r] = 0.f;
  const int nk = H / BK;
#pragma unroll
  for (int s = 0; s < ST - 1; ++s)
    if (s < nk) issue(s, s);
  const int r32 = lane & 31, kh = lane >> 5;
  const int ra = wm * 32 + r32;
  if constexpr (ST == 1) issue(0, 0);  // one stage: a single K step (checked by the launcher)
  for (int i = 0; i < nk; ++i) {
    if constexpr (ST == 1) {
      wait_vmcnt<0>();
      __builtin_amdgcn_s_barrier();
    } else {
      const int issued = nk < i + ST - 1 ? nk : i + ST - 1;
      wait_groups<ST - 2, G::PER_WAVE>(issued - i - 1);
      __builtin_amdgcn_s_barrier();  // step i landed for every wave; step i-1 is consumed
      if (i + ST - 1 < nk) issue(i + ST - 1, (i + ST - 1) % ST);
    }
    const unsigned char* As = smem + (i % ST) * G::STAGE;
    const unsigned char* Bs = As + RA * G::PITCH;
    // a chunk's four latitudes feed two MFMA steps; lane half kh takes
    // latitudes 2 kh and 2 kh + 1 of it (steps 0 and 1) from one 8-byte read
    auto lda = [&](int cc) {
      return *reinterpret_cast<const float2*>(As + ra * G::PITCH + swz<G::CPR>(ra, cc) * 16 +
                                              kh * 8);
    };
    auto ldb = [&](int jj, int cc) {
      const int r = wn * 64 + jj * 32 + r32;
      return *reinterpret_cast<const float2*>(Bs + r * G::PITCH + swz<G::CPR>(r, cc) * 16 + kh * 8);
    };
    // chunk cc + 1 is read while the MFMAs of chunk cc run
    float2 av = lda(0), bv0 = ldb(0, 0), bv1 = ldb(1, 0);
#pragma unroll
    for (int cc = 0; cc < G::CPR; ++cc) {  // four latitudes = two MFMA steps
      float2 nav = av, nb0 = bv0, nb1 = bv1;
      if (cc + 1 < G::CPR) {
        nav = lda(cc + 1);
        nb0 = ldb(0, cc + 1);
        nb1 = ldb(1, cc + 1);
      }
#pragma unroll
      for (int e = 0; e < 2; ++e) {
        const float a = e ? av.y : av.x;
        const float b0 = e ? bv0.y : bv0.x;
        const float b1 = e ? bv1.y : bv1.x;
        acc[0] = __builtin_amdgcn_mfma_f32_32x32x2f32(a, b0, acc[0], 0, 0, 0);
        acc[1] = __builtin_amdgcn_mfma_f32_32x32x2f32(a, b1, acc[1], 0, 0, 0);
      }
      av = nav;
      bv0 = nb0;
      bv1 = nb1;
      if (cc + 1 < G::CPR) __builtin_amdgcn_sched_group_barrier(0x100, 3, 0);  // LDS reads
      __builtin_amdgcn_sched_group_barrier(0x008, 4, 0);                       // MFMA
      __builtin_amdgcn_sched_barrier(0);
    }
  }
  wait_vmcnt<0>();
  __syncthreads();

  // epilogue: rows l, columns n' = (b, c, re/im) through LDS; 4 columns stay
  // inside one b because 2C is a multiple of 4
  float* cs = reinterpret_cast<float*>(smem);
  {
    const int col_l = lane & 31, row_l = 4 * (lane >> 5);
#pragma unroll
    for (int jj = 0; jj < 2; ++jj)
#pragma unroll
      for (int r = 0; r < 16; ++r)
        cs[(wm * 32 + 8 * (r >> 2) + row_l + (r & 3)) * G::LDC + wn * 64 + jj * 32 + col_l] =
            acc[jj][r];
  }
  __syncthreads();
  const int twoC = 2 * C;
  constexpr int VPR = RB / 4;
  for (int idx = tid; idx < RA * VPR; idx += G::NT) {
    const int row = idx / VPR, col = (idx % VPR) * 4;
    const int l = l_begin + row, np = n0 + col;
    if (l >= L || np >= Np) continue;
    const int b = np / twoC, rem = np - b * twoC;
    *reinterpret_cast<float4*>(&coef[((size_t)(l * l + l + m) * B + b) * S * twoC +
                                     (size_t)si * twoC + rem]) =
        *reinterpret_cast<const float4*>(&cs[row * G::LDC + col]);
  }
}

// ---------------------------------------------------------------------------
// inverse
// ---------------------------------------------------------------------------
template <int RA, int RB, int ST>
struct InvGeom {
  static constexpr int BK = 32;  // degrees per K step
  static constexpr int WM = RA / 64, WN = RB / 64;
  static constexpr int NW = WM * WN, NT = 64 * NW;
  static constexpr int PITCH_A = 2 * RA;  // bytes per degree row of the coefficient tile
  static constexpr int RPI_A = 1024 / PITCH_A, LPR_A = 64 / RPI_A;
  static constexpr int PITCH_B = 2 * BK, CPR_B = PITCH_B / 16;
  static constexpr int RPI_B = 1024 / PITCH_B, LPR_B = 64 / RPI_B;
  static constexpr int A_BYTES = BK * PITCH_A, B_BYTES = RB * PITCH_B;
  static constexpr int NI_A = A_BYTES / 1024, NI = NI_A + B_BYTES / 1024;
  static constexpr int PER_WAVE = NI / NW;
  static constexpr int STAGE = A_BYTES + B_BYTES;
  static constexpr int LDC = RB + 8;
  static constexpr int RING = ST * STAGE, CTILE = RA * LDC * 2;
  static constexpr int SMEM = RING > CTILE ? RING : CTILE;
  static_assert(PITCH_A >= 256 && PITCH_A <= 1024 && NI % NW == 0 && RA % 64 == 0 &&
                    RB % 64 == 0 && ST >= 2 && (ST - 2) * PER_WAVE < 64,
                "tile shape");
};

// Transposed read of 4 consecutive degrees for one n' from the K-major tile.
__device__ __forceinline__ v4s tr_read(const unsigned char* tile, int pitch, int k, int col) {
  const unsigned char* p = tile + k * pitch + swz_t(k, col >> 3) * 16 + (col & 7) * 2;
  return __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      (__attribute__((address_space(3))) v4s*)((__attribute__((address_space(3))) unsigned char*)p));
}

template <int RA, int RB, int ST>
__global__ void __launch_bounds__((InvGeom<RA, RB, ST>::NT))
    lat_inv_dma_kernel(const __bf16* __restrict__ coef, const __bf16* __restrict__ tab,
                       __bf16* __restrict__ Y, int L, int H, int Lp, int B, int Bc, int C, int S,
                       SpinList sout_, int n_tiles_n) {
  using G = InvGeom<RA, RB, ST>;
  constexpr int BK = G::BK;
  __shared__ __align__(16) unsigned char smem[G::SMEM];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / G::WN, wn = wave % G::WN;
  const int M = 2 * L - 1;
  // logical block = ((s, order, j tile), n' tile): the n' tiles of one
  // (s, m, j tile) share its table tile and run on one XCD
  const int n_tiles_j = (H + RB - 1) / RB;
  int lbk = xcd_logical_block();
  if (lbk >= S * M * n_tiles_j * n_tiles_n) return;
  const int nt = lbk % n_tiles_n;
  lbk /= n_tiles_n;
  const int jt = lbk % n_tiles_j;
  lbk /= n_tiles_j;
  const int mi = mixed_order(lbk % M, L), si = lbk / M;
  const int m = mi - (L - 1);
  const int spin = sout_.s[si];
  const int lo = iabs_(m) > iabs_(spin) ? iabs_(m) : iabs_(spin);
  const int Np = 2 * B * C, twoC = 2 * C;
  const int n0 = nt * RA, j0 = jt * RB;
  const int b0 = n0 / twoC;  // the n' tile lies inside one b (2C % RA == 0)
  const int kb = (lo / BK) * BK;
  const int nk = (Lp - kb) / BK;  // Lp is a multiple of BK; table columns >= L are zero
  const __bf16* Tb = tab + (size_t)(si * M + mi) * H * Lp;

  // copies g < NI_A: coefficient degree rows k = g RPI_A + lane / LPR_A of
  // the step; degrees below lo or past L are clamped to a row that exists
  // (the table is zero there); copies g >= NI_A: table rows j
  const __bf16* csrc = coef + (size_t)b0 * S * twoC + (size_t)si * twoC + (n0 - b0 * twoC);
  const size_t row_elems = (size_t)Bc * S * twoC;  // elements per coefficient row (l, m)
  int ka[G::PER_WAVE], ca[G::PER_WAVE];
  const __bf16* bsrc[G::PER_WAVE];
#pragma unroll
  for (int u = 0; u < G::PER_WAVE; ++u) {
    const int g = wave * G::PER_WAVE + u;
    if (g < G::NI_A) {
      const int k = g * G::RPI_A + lane / G::LPR_A;
      ka[u] = k;
      ca[u] = swz_t(k, lane % G::LPR_A) * 8;
      bsrc[u] = nullptr;
    } else {
      const int gb = g - G::NI_A;
      const int tr = gb * G::RPI_B + lane / G::LPR_B, slot = lane % G::LPR_B;
      const int j = imin_(j0 + tr, H - 1);
      ka[u] = 0;
      ca[u] = 0;
      bsrc[u] = Tb + (size_t)j * Lp + kb + swz<G::CPR_B>(tr, slot) * 8;
    }
  }
  const unsigned ring = lds_addr(smem);
  auto issue = [&](int i, int stage) {
    const unsigned base = ring + stage * G::STAGE + wave * G::PER_WAVE * 1024;
#pragma unroll
    for (int u = 0; u < G::PER_WAVE; ++u) {
      const __bf16* p;
      if (wave * G::PER_WAVE + u < G::NI_A) {
        int l = kb + i * BK + ka[u];
        l = l < lo ? lo : l;
        l = l > L - 1 ? L - 1 : l;  // last, so that a row of the array is read even if lo >= L
        p = csrc + (size_t)(l * l + l + m) * row_elems + ca[u];
      } else {
        p = bsrc[u] + i * BK;
      }
      dma16(p, base + u * 1024);
    }
  };

  v16f acc[2][2];
  zero_acc(acc);
#pragma unroll
  for (int s = 0; s < ST - 1; ++s)
    if (s < nk) issue(s, s);
  const int r32 = lane & 31, kh = lane >> 5;
  const int q4 = (lane & 15) >> 2, c4 = 4 * (lane & 3);
  const int r0 = 16 * ((lane >> 4) & 1);
  for (int i = 0; i < nk; ++i) {
    const int issued = nk < i + ST - 1 ? nk : i + ST - 1;
    wait_groups<ST - 2, G::PER_WAVE>(issued - i - 1);
    __builtin_amdgcn_s_barrier();
    if (i + ST - 1 < nk) issue(i + ST - 1, (i + ST - 1) % ST);
    const unsigned char* As = smem + (i % ST) * G::STAGE;
    const unsigned char* Bs = As + G::A_BYTES;
#pragma unroll
    for (int kk = 0; kk < BK / 16; ++kk) {
      v8bf a[2], b[2];
      const int kbase = kk * 16 + 8 * kh + q4;
#pragma unroll
      for (int ii = 0; ii < 2; ++ii) {
        const int col = wm * 64 + ii * 32 + r0 + c4;
        const v4s lo4 = tr_read(As, G::PITCH_A, kbase, col);
        const v4s hi4 = tr_read(As, G::PITCH_A, kbase + 4, col);
        a[ii] = __builtin_bit_cast(v8bf, __builtin_shufflevector(lo4, hi4, 0, 1, 2, 3, 4, 5, 6, 7));
      }
#pragma unroll
      for (int jj = 0; jj < 2; ++jj) {
        const int r = wn * 64 + jj * 32 + r32;
        b[jj] = *reinterpret_cast<const v8bf*>(Bs + r * G::PITCH_B +
                                               swz<G::CPR_B>(r, 2 * kk + kh) * 16);
      }
#pragma unroll
      for (int ii = 0; ii < 2; ++ii)
#pragma unroll
        for (int jj = 0; jj < 2; ++jj)
          acc[ii][jj] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[ii], b[jj], acc[ii][jj], 0, 0, 0);
    }
  }
  wait_vmcnt<0>();
  __syncthreads();

  // epilogue: rows n', columns j; Y K-tiled [H/32][Np][32]: 8 consecutive j
  // of one n' are one 16-byte vector inside a latitude tile
  __bf16* cs = reinterpret_cast<__bf16*>(smem);
  acc_to_lds(acc, cs, G::LDC, wm, wn, lane);
  __syncthreads();
  __bf16* Y0 = Y + (size_t)(si * M + mi) * Np * H;
  const size_t tstride = (size_t)Np * kJT;
  constexpr int VPR = RB / 8;
  for (int idx = tid; idx < RA * VPR; idx += G::NT) {
    const int row = idx / VPR, col = (idx % VPR) * 8;
    const int np = n0 + row, j = j0 + col;
    if (np >= Np || j >= H) continue;
    const uint4 v = *reinterpret_cast<const uint4*>(&cs[row * G::LDC + col]);
    *reinterpret_cast<uint4*>(Y0 + (j / kJT) * tstride + (size_t)np * kJT + j % kJT) = v;
  }
}

// Float inverse: K steps of 32 degrees.  The coefficient tile enters LDS
// K-major ([l][n'], 4 RA bytes per degree row, 16-byte chunks of rows with
// degree bit 1 set moved by 128 bytes so that the two lane halves of a read
// hit different banks); of a chunk's four degrees 4c .. 4c + 3, lane half kh
// takes 4c + 2 kh and 4c + 2 kh + 1 (steps 0 and 1): one float of the
// coefficient tile per step and one 8-byte read of its table row j (K = l
// contiguous) per chunk.  Each wave owns TM x TN (TM TN = 2) MFMA 32x32x2 blocks of
// (n', j); the n' tile may span several batch items (a lane keeps its own
// column offset, only the degree row moves per K step).
template <int TM, int WM, int WN, int ST>
struct InvGeomF {
  static constexpr int BK = 32;  // degrees per K step
  static constexpr int TN = 2 / TM;
  static constexpr int NW = WM * WN, NT = 64 * NW;
  static constexpr int RA = 32 * TM * WM, RB = 32 * TN * WN;  // n' rows, j columns
  static constexpr int PITCH_A = 4 * RA, CPR_A = PITCH_A / 16;
  static constexpr int RPI_A = 1024 / PITCH_A, LPR_A = 64 / RPI_A;
  static constexpr int PITCH_B = 4 * BK, CPR_B = PITCH_B / 16;
  static constexpr int RPI_B = 1024 / PITCH_B, LPR_B = 64 / RPI_B;
  static constexpr int A_BYTES = BK * PITCH_A, B_BYTES = RB * PITCH_B;
  static constexpr int NI_A = A_BYTES / 1024, NI = NI_A + B_BYTES / 1024;
  static constexpr int PER_WAVE = NI / NW;
  static constexpr int STAGE = A_BYTES + B_BYTES;
  static constexpr int LDC = RB + 4;  // floats per row of the output tile
  static constexpr int RING = ST * STAGE, CTILE = RA * LDC * 4;
  static constexpr int SMEM = RING > CTILE ? RING : CTILE;
  static_assert(TM * TN == 2 && PITCH_A >= 256 && PITCH_A <= 1024 && B_BYTES % 1024 == 0 &&
                    NI % NW == 0 && ST >= 1 && (ST - 2) * PER_WAVE < 64,
                "tile shape");
};

// chunk slot of a degree row of the float coefficient tile: the 16-byte
// chunks of degree rows with bit 1 set move by 128 bytes, so the two lane
// halves of a read (degrees 4c + e and 4c + 2 + e) hit different banks
__device__ __forceinline__ int swa(int k, int c) { return c ^ (((k >> 1) & 1) << 3); }

template <int TM, int WM, int WN, int ST>
__global__ void __launch_bounds__((InvGeomF<TM, WM, WN, ST>::NT))
    lat_inv_dma_f32_kernel(const float* __restrict__ coef, const float* __restrict__ tab,
                           float* __restrict__ Y, int L, int H, int Lp, int B, int Bc, int C,
                           int S, SpinList sout_, int n_tiles_n) {
  using G = InvGeomF<TM, WM, WN, ST>;
  constexpr int BK = G::BK, TN = G::TN, RA = G::RA, RB = G::RB;
  extern __shared__ __align__(16) unsigned char smem[];  // G::SMEM bytes
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WN, wn = wave % WN;
  const int M = 2 * L - 1;
  // logical block = ((s, order, j tile), n' tile), as for bf16
  const int n_tiles_j = (H + RB - 1) / RB;
  int lbk = xcd_logical_block();
  if (lbk >= S * M * n_tiles_j * n_tiles_n) return;
  const int nt = lbk % n_tiles_n;
  lbk /= n_tiles_n;
  const int jt = lbk % n_tiles_j;
  lbk /= n_tiles_j;
  const int mi = mixed_order(lbk % M, L), si = lbk / M;
  const int m = mi - (L - 1);
  const int spin = sout_.s[si];
  const int lo = iabs_(m) > iabs_(spin) ? iabs_(m) : iabs_(spin);
  const int Np = 2 * B * C, twoC = 2 * C;
  const int n0 = nt * RA, j0 = jt * RB;
  const int kb = (lo / BK) * BK;
  const int nk = (Lp - kb) / BK;  // Lp is a multiple of BK; table columns >= L are zero
  const float* Tb = tab + (size_t)(si * M + mi) * H * Lp;
  const size_t row_elems = (size_t)Bc * S * twoC;  // elements per coefficient row (l, m)

  // copies g < NI_A: coefficient degree rows k of the step, this lane's chunk
  // of n' (its batch item and offset fixed); copies g >= NI_A: table rows j
  int ka[G::PER_WAVE];
  size_t coff[G::PER_WAVE];
  const float* bsrc[G::PER_WAVE];
#pragma unroll
  for (int u = 0; u < G::PER_WAVE; ++u) {
    const int g = wave * G::PER_WAVE + u;
    if (g < G::NI_A) {
      const int k = g * G::RPI_A + lane / G::LPR_A;
      const int np = imin_(n0 + 4 * swa(k, lane % G::LPR_A), Np - 4);
      const int b = np / twoC, rem = np - b * twoC;
      ka[u] = k;
      coff[u] = (size_t)b * S * twoC + (size_t)si * twoC + rem;
      bsrc[u] = nullptr;
    } else {
      const int gb = g - G::NI_A;
      const int tr = gb * G::RPI_B + lane / G::LPR_B, slot = lane % G::LPR_B;
      const int j = imin_(j0 + tr, H - 1);
      ka[u] = 0;
      coff[u] = 0;
      bsrc[u] = Tb + (size_t)j * Lp + kb + swz<G::CPR_B>(tr, slot) * 4;
    }
  }
  const unsigned ring = lds_addr(smem);
  auto issue = [&](int i, int stage) {
    const unsigned base = ring + stage * G::STAGE + wave * G::PER_WAVE * 1024;
#pragma unroll
    for (int u = 0; u < G::PER_WAVE; ++u) {
      const float* p;
      if (wave * G::PER_WAVE + u < G::NI_A) {
        int l = kb + i * BK + ka[u];
        l = l < lo ? lo : l;
        l = l > L - 1 ? L - 1 : l;  // last, so that a row of the array is read even if lo >= L
        p = coef + (size_t)(l * l + l + m) * row_elems + coff[u];
      } else {
        p = bsrc[u] + i * BK;
      }
      dma16(p, base + u * 1024);
    }
  };

  v16f acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;
#pragma unroll
  for (int s = 0; s < ST - 1; ++s)
    if (s < nk) issue(s, s);
  if constexpr (ST == 1) issue(0, 0);  // one stage: a single K step (checked by the launcher)
  const int r32 = lane & 31, kh = lane >> 5;
  for (int i = 0; i < nk; ++i) {
    if constexpr (ST == 1) {
      wait_vmcnt<0>();
      __builtin_amdgcn_s_barrier();
    } else {
      const int issued = nk < i + ST - 1 ? nk : i + ST - 1;
      wait_groups<ST - 2, G::PER_WAVE>(issued - i - 1);
      __builtin_amdgcn_s_barrier();
      if (i + ST - 1 < nk) issue(i + ST - 1, (i + ST - 1) % ST);
    }
    const unsigned char* As = smem + (i % ST) * G::STAGE;
    const unsigned char* Bs = As + G::A_BYTES;
    auto lda = [&](int ii, int k) {  // A[n'][degree k] of this lane's row block ii
      const int n = wm * 32 * TM + ii * 32 + r32;
      return *reinterpret_cast<const float*>(As + k * G::PITCH_A + swa(k, n >> 2) * 16 + (n & 3) * 4);
    };
    // a chunk's four degrees feed two MFMA steps; lane half kh takes degrees
    // 2 kh and 2 kh + 1 of it (steps 0 and 1), one 8-byte table read
    auto ldb = [&](int jj, int cc) {
      const int r = wn * 32 * TN + jj * 32 + r32;
      return *reinterpret_cast<const float2*>(Bs + r * G::PITCH_B + swz<G::CPR_B>(r, cc) * 16 +
                                              kh * 8);
    };
#pragma unroll
    for (int cc = 0; cc < G::CPR_B; ++cc) {  // four degrees = two MFMA steps
      float2 bv[TN];
#pragma unroll
      for (int jj = 0; jj < TN; ++jj) bv[jj] = ldb(jj, cc);
#pragma unroll
      for (int e = 0; e < 2; ++e) {
        float a[TM];
#pragma unroll
        for (int ii = 0; ii < TM; ++ii) a[ii] = lda(ii, 4 * cc + 2 * kh + e);
#pragma unroll
        for (int jj = 0; jj < TN; ++jj) {
          const float b = e ? bv[jj].y : bv[jj].x;
#pragma unroll
          for (int ii = 0; ii < TM; ++ii)
            acc[ii][jj] = __builtin_amdgcn_mfma_f32_32x32x2f32(a[ii], b, acc[ii][jj], 0, 0, 0);
        }
      }
    }
  }
  wait_vmcnt<0>();
  __syncthreads();

  // epilogue: rows n', columns j through LDS; Y K-tiled [H/32][Np][32]: 4
  // consecutive j of one n' are one 16-byte vector inside a latitude tile
  float* cs = reinterpret_cast<float*>(smem);
  {
    const int col_l = lane & 31, row_l = 4 * (lane >> 5);
#pragma unroll
    for (int ii = 0; ii < TM; ++ii)
#pragma unroll
      for (int jj = 0; jj < TN; ++jj)
#pragma unroll
        for (int r = 0; r < 16; ++r)
          cs[(wm * 32 * TM + ii * 32 + 8 * (r >> 2) + row_l + (r & 3)) * G::LDC + wn * 32 * TN +
             jj * 32 + col_l] = acc[ii][jj][r];
  }
  __syncthreads();
  float* Y0 = Y + (size_t)(si * M + mi) * Np * H;
  const size_t tstride = (size_t)Np * kJT;
  constexpr int VPR = RB / 4;
  for (int idx = tid; idx < RA * VPR; idx += G::NT) {
    const int row = idx / VPR, col = (idx % VPR) * 4;
    const int np = n0 + row, j = j0 + col;
    if (np >= Np || j >= H) continue;
    *reinterpret_cast<float4*>(Y0 + (j / kJT) * tstride + (size_t)np * kJT + j % kJT) =
        *reinterpret_cast<const float4*>(&cs[row * G::LDC + col]);
  }
}

// forward: BK, rows l, columns n', stages; the wide tile when 2BC allows it
#ifndef SWSFT_LAT_FWD_DMA_WIDE
#define SWSFT_LAT_FWD_DMA_WIDE 32, 128, 256, 3
#endif
#ifndef SWSFT_LAT_FWD_DMA
#define SWSFT_LAT_FWD_DMA 32, 128, 128, 3
#endif
// inverse: rows n', columns j, stages; the wide tile when 2C allows it
#ifndef SWSFT_LAT_INV_DMA_WIDE
#define SWSFT_LAT_INV_DMA_WIDE 256, 128, 3
#endif
#ifndef SWSFT_LAT_INV_DMA
#define SWSFT_LAT_INV_DMA 128, 128, 3
#endif

template <int BK, int RA, int RB, int ST>
hipError_t fwd_geom(const Plan& p, int B, int C, const void* X, void* coef, hipStream_t st) {
  const int Np = 2 * B * C;
  const int nrt = (p.L + RA - 1) / RA, nnt = (Np + RB - 1) / RB;
  const long long blocks = (long long)p.n_in * p.M * nrt * nnt;
  hipLaunchKernelGGL((lat_fwd_dma_kernel<BK, RA, RB, ST>), dim3(xcd_grid(blocks)),
                     dim3(FwdGeom<BK, RA, RB, ST>::NT), 0, st, (const __bf16*)X,
                     (const __bf16*)p.tab_fwd, (__bf16*)coef, p.L, p.H, B, C, p.n_in, nrt, nnt);
  return hipGetLastError();
}

template <int WM, int WN, int ST>
hipError_t fwd_geom_f32(const Plan& p, int B, int C, const void* X, void* coef, hipStream_t st) {
  using G = FwdGeomF<WM, WN, ST>;
  const int Np = 2 * B * C;
  const int nrt = (p.L + G::RA - 1) / G::RA, nnt = (Np + G::RB - 1) / G::RB;
  const long long blocks = (long long)p.n_in * p.M * nrt * nnt;
  auto kern = lat_fwd_dma_f32_kernel<WM, WN, ST>;
  const hipError_t e = ensure_dynamic_lds((const void*)kern, G::SMEM);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(kern, dim3(xcd_grid(blocks)), dim3(G::NT), G::SMEM, st, (const float*)X,
                     (const float*)p.tab_fwd, (float*)coef, p.L, p.H, B, C, p.n_in, nrt, nnt);
  return hipGetLastError();
}

template <int RA, int RB, int ST>
hipError_t inv_geom(const Plan& p, int B, int C, const void* coef, void* Y, hipStream_t st) {
  const int Np = 2 * B * C;
  const int nnt = (Np + RA - 1) / RA, njt = (p.H + RB - 1) / RB;
  const long long blocks = (long long)p.n_out * p.M * njt * nnt;
  SpinList so{};
  for (int i = 0; i < p.n_out; ++i) so.s[i] = p.spins_out[i];
  hipLaunchKernelGGL((lat_inv_dma_kernel<RA, RB, ST>), dim3(xcd_grid(blocks)),
                     dim3(InvGeom<RA, RB, ST>::NT), 0, st, (const __bf16*)coef,
                     (const __bf16*)p.tab_inv, (__bf16*)Y, p.L, p.H, p.Lp, B,
                     p.coef_ldb > 0 ? p.coef_ldb : B, C, p.n_out, so, nnt);
  return hipGetLastError();
}

template <int TM, int WM, int WN, int ST>
hipError_t inv_geom_f32(const Plan& p, int B, int C, const void* coef, void* Y, hipStream_t st) {
  using G = InvGeomF<TM, WM, WN, ST>;
  const int Np = 2 * B * C;
  const int nnt = (Np + G::RA - 1) / G::RA, njt = (p.H + G::RB - 1) / G::RB;
  const long long blocks = (long long)p.n_out * p.M * njt * nnt;
  SpinList so{};
  for (int i = 0; i < p.n_out; ++i) so.s[i] = p.spins_out[i];
  auto kern = lat_inv_dma_f32_kernel<TM, WM, WN, ST>;
  const hipError_t e = ensure_dynamic_lds((const void*)kern, G::SMEM);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(kern, dim3(xcd_grid(blocks)), dim3(G::NT), G::SMEM, st, (const float*)coef,
                     (const float*)p.tab_inv, (float*)Y, p.L, p.H, p.Lp, B,
                     p.coef_ldb > 0 ? p.coef_ldb : B, C, p.n_out, so, nnt);
  return hipGetLastError();
}

template <int BK, int RA, int RB, int ST>
constexpr int fwd_bk(int) { return BK; }
template <int BK, int RA, int RB, int ST>
constexpr int fwd_rb(int) { return RB; }
template <int RA, int RB, int ST>
constexpr int inv_ra(int) { return RA; }

}  // namespace

bool lat_fwd_dma_supported(const Plan& p, int B, int C) {
  constexpr int BK = fwd_bk<SWSFT_LAT_FWD_DMA>(0);
  static_assert(fwd_bk<SWSFT_LAT_FWD_DMA_WIDE>(0) == BK, "wide tile");
  // float: columns 2BC >= 1024 (narrower ones leave too few workgroups; the
  // register-staged kernel takes them)
  if (p.dtype == SWSFT_F32)
    return p.H % kJT == 0 && p.Hp == p.H && p.JT == kJT && C % 2 == 0 && 2 * B * C >= 1024;
  return p.dtype == SWSFT_BF16 && p.H >= BK && p.H % BK == 0 && p.Hp == p.H && p.JT == kJT &&
         (2 * C) % 8 == 0;
}

bool lat_inv_dma_supported(const Plan& p, int B, int C) {
  constexpr int RA = inv_ra<SWSFT_LAT_INV_DMA>(0);
  static_assert(inv_ra<SWSFT_LAT_INV_DMA_WIDE>(0) % RA == 0, "wide tile");
  // float: columns 2BC >= 1024, as for the forward
  if (p.dtype == SWSFT_F32)
    return p.H % kJT == 0 && p.JT == kJT && p.Hp == p.H && p.Lp % 32 == 0 && C % 2 == 0 &&
           2 * B * C >= 1024;
  return p.dtype == SWSFT_BF16 && p.H % kJT == 0 && p.JT == kJT && (2 * C) % RA == 0 &&
         p.Lp % InvGeom<SWSFT_LAT_INV_DMA>::BK == 0 && p.Hp == p.H;
}

// float geometries at H = 32 (WM, WN, ST of FwdGeomF; TM, WM, WN, ST of InvGeomF)
#ifndef SWSFT_LAT_FWD_F32_H32
#define SWSFT_LAT_FWD_F32_H32 1, 4, 1
#endif
#ifndef SWSFT_LAT_INV_F32_H32
#define SWSFT_LAT_INV_F32_H32 2, 4, 1, 1
#endif
// and for H > 32 (forward: 32 rows l x 256 columns with 2 stages, measured
// against 64 x 128 with 2 or 3 stages, 32 x 128 and 64 x 64: wx128 31.5 -> 30.1 us)
#ifndef SWSFT_LAT_FWD_F32
#define SWSFT_LAT_FWD_F32 1, 4, 2
#endif
#ifndef SWSFT_LAT_INV_F32
#define SWSFT_LAT_INV_F32 1, 2, 2, 2
#endif

hipError_t launch_lat_fwd_dma(const Plan& p, int B, int C, const void* X, void* coef,
                              hipStream_t st) {
  // float: 32 rows l x 256 columns; a single K step (H = 32) needs a single
  // stage, which leaves room for 4 workgroups per CU
  if (p.dtype == SWSFT_F32) {
    if (p.H == kJT) return fwd_geom_f32<SWSFT_LAT_FWD_F32_H32>(p, B, C, X, coef, st);
    return fwd_geom_f32<SWSFT_LAT_FWD_F32>(p, B, C, X, coef, st);
  }
  if ((2 * B * C) % fwd_rb<SWSFT_LAT_FWD_DMA_WIDE>(0) == 0)
    return fwd_geom<SWSFT_LAT_FWD_DMA_WIDE>(p, B, C, X, coef, st);
  return fwd_geom<SWSFT_LAT_FWD_DMA>(p, B, C, X, coef, st);
}

hipError_t launch_lat_inv_dma(const Plan& p, int B, int C, const void* coef, void* Y,
                              hipStream_t st) {
  // float: 256 n' x 32 j in one stage when H = 32 (then L <= 16 < 32: one K
  // step); else 64 n' x 128 j with two stages
  if (p.dtype == SWSFT_F32) {
    if (p.H == kJT) return inv_geom_f32<SWSFT_LAT_INV_F32_H32>(p, B, C, coef, Y, st);
    return inv_geom_f32<SWSFT_LAT_INV_F32>(p, B, C, coef, Y, st);
  }
  if ((2 * C) % inv_ra<SWSFT_LAT_INV_DMA_WIDE>(0) == 0)
    return inv_geom<SWSFT_LAT_INV_DMA_WIDE>(p, B, C, coef, Y, st);
  return inv_geom<SWSFT_LAT_INV_DMA>(p, B, C, coef, Y, st);
}

}  // namespace swsft
