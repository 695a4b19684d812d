// Per-degree mixing GEMM fed by direct global -> LDS loads
// (global_load_lds_dwordx4) into a ring of LDS stages: bfloat16 storage
// first, the float form below.
//
//   coef'[l][(m,b)][(t,c')] = sum_(s,c) coef[l][(m,b)][(s,c)] K[l][(t,c')][(s,c)]
//
// (Background, "Spherical CNNs": convolution as products of coefficients
// with filters shared across m; Fig. 2 "*K".)  The complex product is a real
// GEMM whose rows are the coefficient rows expanded in registers: row 2i is
// coef row i with the imaginary parts negated, row 2i+1 is coef row i with
// real and imaginary parts swapped; both operands then enter LDS unchanged,
// so the hardware copies them from HBM/L2 without passing through registers
// and several K steps are in flight per workgroup.
//
// Tile geometry (template parameters): BK reals of every row per K step (64
// = one whole 128-byte line per row and copy), RA coefficient rows (2 RA
// expanded GEMM rows) x RB filter rows (complex outputs) per workgroup, ST
// K steps resident in LDS.  Each wave owns 64 expanded rows x 64 outputs.
//
// Preconditions (checked by the launcher): K' = 2 S_in C_in with each input
// spin's channel block a whole number of K steps; bf16 also C_out % 4 == 0.
//
// The adjoint mixing of the backward pass is computed straight from the
// filters as stored (ADJ mode of the split kernel below and of the float
// kernel):
//   coef'[l][(m,b)][(s,c)] = sum_(t,c') g[l][(m,b)][(t,c')] conj(K[l][(t,c')][(s,c)]),
// the contraction now running over the filter rows, so the filter tile is
// copied k-major ([contraction rows][RB outputs]) and a lane gathers its
// contraction rows of one output.  No conjugate-transposed copy of the
// filters is made.
#include <type_traits>

#include "lds_dma.h"
#include "mfma_tile.h"
#include "swsft_internal.h"
#include "xcd.h"

namespace swsft {
namespace {

constexpr int kMaxKp = 8192;  // 2 S_in C_in

struct Spins {
  int s[kMaxSpins];
};

__device__ __forceinline__ int iabs_(int v) { return v < 0 ? -v : v; }

template <int BK, int RA, int RB, int ST>
struct MixGeom {
  static constexpr int WM = 2 * RA / 64, WN = RB / 64;
  static constexpr int NW = WM * WN, NT = 64 * NW;  // waves, threads
  static constexpr int PITCH = 2 * BK;               // bytes per tile row
  static constexpr int CPR = PITCH / 16;             // 16-byte chunks per row
  static constexpr int RPI = 1024 / PITCH;           // rows per 1 KiB copy
  static constexpr int LPR = 64 / RPI;               // lanes per row
  static constexpr int NI = (RA + RB) / RPI;         // copies per stage
  static constexpr int NI_A = RA / RPI;              // of which coefficient rows
  static constexpr int PER_WAVE = NI / NW;
  static constexpr int STAGE = (RA + RB) * PITCH;
  static constexpr int SMEM = ST * STAGE;  // the ring (the epilogue needs no LDS)
  static constexpr int MAX_KT = kMaxKp / BK;
  static_assert(RA % RPI == 0 && NI % NW == 0 && RA % 32 == 0 && RB % 64 == 0, "tile shape");
  static_assert(ST >= 2 && (ST - 2) * PER_WAVE < 64, "stages");
};

template <int BK, int RA, int RB, int ST>
__global__ void __launch_bounds__((MixGeom<BK, RA, RB, ST>::NT))
    mix_dma_kernel(const __bf16* __restrict__ coef, const __bf16* __restrict__ K,
                   __bf16* __restrict__ out, int L, int B, int Cin, int Cout, int Sin, int Sout,
                   Spins sin_, Spins sout_) {
  using G = MixGeom<BK, RA, RB, ST>;
  __shared__ __align__(16) unsigned char smem[G::SMEM];
  __shared__ int live[G::MAX_KT];
  __shared__ int n_live_s;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / G::WN, wn = wave % G::WN;
  const int Kc = Sin * Cin, Nc = Sout * Cout;
  const int Kp = 2 * Kc;
  const int n_tiles_n = (Nc + RB - 1) / RB;

  // logical block = ((l, row tile), column tile), largest degrees first
  int lbk = xcd_logical_block();
  const int ntile = lbk % n_tiles_n;
  int t = lbk / n_tiles_n;
  int l = L - 1;
  for (; l >= 0; --l) {
    const int ntl = ((2 * l + 1) * B + RA - 1) / RA;
    if (t < ntl) break;
    t -= ntl;
  }
  if (l < 0) return;
  const int Mrows = (2 * l + 1) * B;
  const int row0 = t * RA;
  const int q0 = ntile * RB;

  // K steps of input spins that exist at this degree (whole channel blocks)
  if (tid == 0) {
    const int per_spin = 2 * Cin / BK;
    int n = 0;
    for (int si = 0; si < Sin; ++si)
      if (iabs_(sin_.s[si]) <= l)
        for (int k = 0; k < per_spin; ++k) live[n++] = si * per_spin + k;
    n_live_s = n;
  }
  __syncthreads();
  const int nk = n_live_s;

  const __bf16* A0 = coef + (size_t)l * l * B * Kp;  // rows (m, b) of degree l
  const __bf16* K0 = K + (size_t)l * Nc * Kp;        // filter rows q of degree l
  const unsigned ring_base = lds_addr(smem);

  // copy g = wave * PER_WAVE + u moves tile rows [g RPI, (g + 1) RPI) of the
  // stage [A rows; B rows]; rows past the end of the matrix are clamped to
  // its last row (their products are discarded)
  const __bf16* gsrc[G::PER_WAVE];
  bool is_a[G::PER_WAVE];  // wave-uniform
#pragma unroll
  for (int u = 0; u < G::PER_WAVE; ++u) {
    const int g = wave * G::PER_WAVE + u;
    is_a[u] = g < G::NI_A;
    if (is_a[u]) {
      const int tr = g * G::RPI + lane / G::LPR;  // row of the stage
      const int row = row0 + tr < Mrows ? row0 + tr : Mrows - 1;
      gsrc[u] = A0 + (size_t)row * Kp + swz<G::CPR>(tr, lane % G::LPR) * 8;
    } else {
      const int rb = (g - G::NI_A) * G::RPI + lane / G::LPR;
      const int q = q0 + rb < Nc ? q0 + rb : Nc - 1;
      gsrc[u] = K0 + (size_t)q * Kp + swz<G::CPR>(rb, lane % G::LPR) * 8;
    }
  }
  auto issue = [&](int i, int stage) {
    const int koff = live[i] * BK;  // along the rows of both operands
    const unsigned base = ring_base + stage * G::STAGE + wave * G::PER_WAVE * 1024;
#pragma unroll
    for (int u = 0; u < G::PER_WAVE; ++u) dma16(gsrc[u] + koff, base + u * 1024);
  };

  typedef unsigned v4u __attribute__((ext_vector_type(4)));
  v16f acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  // prologue: K steps 0 .. ST-2 in flight
#pragma unroll
  for (int s = 0; s < ST - 1; ++s)
    if (s < nk) issue(s, s);

  const int r32 = lane & 31, kh = lane >> 5;
  // odd expanded rows (im, re): rotate by 16 bits; even rows (re, -im): flip
  // the high half's sign (the row parity is the lane parity)
  const unsigned rot = (lane & 1) ? 16u : 0u;
  const unsigned sgn = (lane & 1) ? 0u : 0x80000000u;
  for (int i = 0; i < nk; ++i) {
    // K step i has landed once at most (issued - i - 1) steps are outstanding
    const int issued = nk < i + ST - 1 ? nk : i + ST - 1;
    wait_groups<ST - 2, G::PER_WAVE>(issued - i - 1);
    __builtin_amdgcn_s_barrier();  // every wave's copies of step i landed; step i-1 is consumed
    if (i + ST - 1 < nk) issue(i + ST - 1, (i + ST - 1) % ST);
    const unsigned char* As = smem + (i % ST) * G::STAGE;
    const unsigned char* Bs = As + RA * G::PITCH;
#pragma unroll
    for (int kk = 0; kk < BK / 16; ++kk) {  // 16-wide MFMA K steps
      const int c = 2 * kk + kh;
      v8bf a[2], b[2];
#pragma unroll
      for (int ii = 0; ii < 2; ++ii) {
        const int cr = (wm * 64 + ii * 32 + r32) >> 1;  // coefficient row of the expanded row
        const v4u x = *reinterpret_cast<const v4u*>(As + cr * G::PITCH + swz<G::CPR>(cr, c) * 16);
        v4u y;
#pragma unroll
        for (int d = 0; d < 4; ++d) y[d] = __builtin_amdgcn_alignbit(x[d], x[d], rot) ^ sgn;
        a[ii] = __builtin_bit_cast(v8bf, y);
      }
#pragma unroll
      for (int jj = 0; jj < 2; ++jj) {
        const int rb = wn * 64 + jj * 32 + r32;
        b[jj] = *reinterpret_cast<const v8bf*>(Bs + rb * G::PITCH + swz<G::CPR>(rb, c) * 16);
      }
#pragma unroll
      for (int ii = 0; ii < 2; ++ii)
#pragma unroll
        for (int jj = 0; jj < 2; ++jj)
          acc[ii][jj] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[ii], b[jj], acc[ii][jj], 0, 0, 0);
    }
  }
  wait_vmcnt<0>();

  // epilogue straight from the accumulators: registers r and r + 1 (r even)
  // of a lane hold expanded rows 2i and 2i + 1 of its column q, i.e. the real
  // and imaginary part of output (row0 + i, q0 + q); packed as one bf16 pair,
  // the 32 lanes of a row write 128 contiguous bytes.  Output spins that do
  // not exist at this degree are written as zero.
  typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
  typedef float f32x2_t __attribute__((ext_vector_type(2)));
  const int Np = 2 * Nc;
  const int col_l = lane & 31, row_l = 4 * (lane >> 5);
#pragma unroll
  for (int jj = 0; jj < 2; ++jj) {
    const int q = q0 + wn * 64 + jj * 32 + col_l;
    const bool qok = q < Nc;
    const bool tok = qok && iabs_(sout_.s[(qok ? q : 0) / Cout]) <= l;
#pragma unroll
    for (int ii = 0; ii < 2; ++ii)
#pragma unroll
      for (int r = 0; r < 16; r += 2) {
        const int er = wm * 64 + ii * 32 + 8 * (r >> 2) + row_l + (r & 3);  // even
        const int row = row0 + (er >> 1);
        if (!qok || row >= Mrows) continue;
        const f32x2_t v = tok ? (f32x2_t){acc[ii][jj][r], acc[ii][jj][r + 1]} : (f32x2_t){0.f, 0.f};
        *reinterpret_cast<bf16x2_t*>(out + ((size_t)l * l * B + row) * Np + 2 * q) =
            __builtin_convertvector(v, bf16x2_t);
      }
  }
}

template <int BK, int RA, int RB, int ST>
hipError_t launch_geom(const Plan& p, int B, int Cin, int Cout, const void* coef, const void* K,
                       void* out, hipStream_t st) {
  using G = MixGeom<BK, RA, RB, ST>;
  Spins si{}, so{};
  for (int i = 0; i < p.n_in; ++i) si.s[i] = p.spins_in[i];
  for (int i = 0; i < p.n_out; ++i) so.s[i] = p.spins_out[i];
  int tiles = 0;
  for (int l = 0; l < p.L; ++l) tiles += ((2 * l + 1) * B + RA - 1) / RA;
  const int Nc = p.n_out * Cout;
  const long long blocks = (long long)tiles * ((Nc + RB - 1) / RB);
  hipLaunchKernelGGL((mix_dma_kernel<BK, RA, RB, ST>), dim3(xcd_grid(blocks)), dim3(G::NT), 0,
                     st, (const __bf16*)coef, (const __bf16*)K, (__bf16*)out, p.L, B, Cin, Cout,
                     p.n_in, p.n_out, si, so);
  return hipGetLastError();
}

// Forward mixing, bfloat16, with separate real and imaginary accumulators.
//
// A lane reads 16 bytes of its coefficient row (four complex values) once per
// 16-wide K step and forms both operands in registers: (re, -im) for the
// real part of the product and (im, re) for the imaginary part, against the
// filter values as stored (re, im).  So the 32 rows of an MFMA operand are
// 32 distinct coefficient rows and each LDS read feeds two MFMAs; the
// expanded-row kernel above reads every coefficient row twice (once per
// expanded row) and feeds one.  Each wave owns TM x TN blocks of 32
// coefficient rows x 32 outputs (2 TM TN accumulators); the workgroup covers
// WM x WN waves.  Row blocks past the last row of the degree issue no MFMA
// and no operand read (wave-uniform branch), so short degrees cost about
// their own rows rather than a whole tile.  Both operands enter a ring of ST
// LDS stages by direct copies of whole 128-byte lines per row (64-wide K
// steps), swizzled as in the kernel above.
typedef unsigned v4u_t __attribute__((ext_vector_type(4)));

template <int WM, int WN, int ST>
struct MixGeomS {
  static constexpr int BK = 64;                  // reals per row per K step
  static constexpr int TM = 2, TN = 2;           // 32 x 32 blocks per wave
  static constexpr int RA = 32 * TM * WM;        // coefficient rows per workgroup
  static constexpr int RB = 32 * TN * WN;        // outputs per workgroup
  static constexpr int NW = WM * WN, NT = 64 * NW;
  static constexpr int PITCH = 2 * BK, CPR = PITCH / 16;
  static constexpr int RPI = 1024 / PITCH, LPR = 64 / RPI;
  static constexpr int NI = (RA + RB) / RPI, NI_A = RA / RPI;
  static constexpr int PER_WAVE = NI / NW;
  static constexpr int STAGE = (RA + RB) * PITCH;
  static constexpr int SMEM = ST * STAGE;
  static constexpr int MAX_KT = kMaxKp / BK;
  // k-major filter tile of the adjoint: BK / 2 contraction rows of RB outputs
  static constexpr int PITCH_T = 4 * RB;
  static constexpr int RPI_T = PITCH_T <= 1024 ? 1024 / PITCH_T : 1;
  static constexpr int LPR_T = 64 / RPI_T;
  static_assert(RA % RPI == 0 && NI % NW == 0, "tile shape");
  static_assert(ST >= 2 && (ST - 2) * PER_WAVE < 64, "stages");
};

// ADJ: the adjoint mixing of the backward pass from the filters as stored
// (Cin, Sin, sin_ describe the contraction side, i.e. the forward's outputs;
// Cout, Sout, sout_ the results, the forward's inputs): the filter tile is
// copied k-major ([32 contraction rows][RB outputs], swz_k4 chunk order) and
// a lane gathers its 4 consecutive contraction rows of one output as 4 dword
// reads; with g = (gr, gi) and K = (Kr, Ki), Re = gr Kr + gi Ki takes the
// coefficient values as stored and Im = gi Kr - gr Ki takes them as
// (gi, -gr).  (256^2, C = 256: 94 us against 101 us for the expanded-row
// form with the same gathers, which issued 1.25x the MFMAs.)
template <int WM, int WN, int ST, bool REG, bool ADJ = false>
__global__ void __launch_bounds__((MixGeomS<WM, WN, ST>::NT))
    mix_split_kernel(const __bf16* __restrict__ coef, const __bf16* __restrict__ K,
                     __bf16* __restrict__ out, int L, int B, int Cin, int Cout, int Sin, int Sout,
                     Spins sin_, Spins sout_) {
  using G = MixGeomS<WM, WN, ST>;
  constexpr int TM = G::TM, TN = G::TN, RA = G::RA, RB = G::RB, BK = G::BK;
  static_assert(!ADJ || (!REG && G::PITCH_T <= 1024 && 1024 % G::PITCH_T == 0 &&
                         (BK / 2) % G::RPI_T == 0 && (BK / 2) * G::PITCH_T == RB * G::PITCH),
                "adjoint filter tile");
  extern __shared__ __align__(16) unsigned char smem[];  // G::SMEM bytes: the ring, then the output tile
  __shared__ int live[G::MAX_KT];
  __shared__ int n_live_s;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave / WN, wn = wave % WN;
  const int Kc = Sin * Cin, Nc = Sout * Cout;
  const int Kp = 2 * Kc;
  const int n_tiles_n = (Nc + RB - 1) / RB;

  // logical block = ((l, row tile), column tile), largest degrees first
  const int lbk = xcd_logical_block();
  const int ntile = lbk % n_tiles_n;
  int t = lbk / n_tiles_n;
  int l = L - 1;
  for (; l >= 0; --l) {
    const int ntl = ((2 * l + 1) * B + RA - 1) / RA;
    if (t < ntl) break;
    t -= ntl;
  }
  if (l < 0) return;
  const int Mrows = (2 * l + 1) * B;
  const int row0 = t * RA;
  const int q0 = ntile * RB;

  if (tid == 0) {
    const int per_spin = 2 * Cin / BK;
    int n = 0;
    for (int si = 0; si < Sin; ++si)
      if (iabs_(sin_.s[si]) <= l)
        for (int k = 0; k < per_spin; ++k) live[n++] = si * per_spin + k;
    n_live_s = n;
  }
  __syncthreads();
  const int nk = n_live_s;

  const __bf16* A0 = coef + (size_t)l * l * B * Kp;
  const __bf16* K0 = K + (size_t)l * Nc * Kp;
  const unsigned ring_base = lds_addr(smem);

  const __bf16* gsrc[G::PER_WAVE];
  bool is_a[G::PER_WAVE];
#pragma unroll
  for (int u = 0; u < G::PER_WAVE; ++u) {
    const int g = wave * G::PER_WAVE + u;
    is_a[u] = g < G::NI_A;
    if (is_a[u]) {
      const int tr = g * G::RPI + lane / G::LPR;
      const int row = row0 + tr < Mrows ? row0 + tr : Mrows - 1;
      gsrc[u] = A0 + (size_t)row * Kp + swz<G::CPR>(tr, lane % G::LPR) * 8;
    } else if (!ADJ) {
      const int rb = (g - G::NI_A) * G::RPI + lane / G::LPR;
      const int q = q0 + rb < Nc ? q0 + rb : Nc - 1;
      gsrc[u] = K0 + (size_t)q * Kp + swz<G::CPR>(rb, lane % G::LPR) * 8;
    } else {
      // contraction row kb of the step, 4 outputs per chunk; chunks past the
      // last output are clamped to it (their products are discarded)
      const int kb = (g - G::NI_A) * G::RPI_T + lane / G::LPR_T;
      const int q = min(q0 + 4 * swz_k4(kb, lane % G::LPR_T), Nc - 4);
      gsrc[u] = K0 + (size_t)kb * (2 * Nc) + 2 * q;
    }
  }
  auto issue = [&](int i, int stage) {
    const int koff = live[i] * BK;  // along coefficient rows
    const size_t koff_b = ADJ ? (size_t)live[i] * (BK / 2) * (2 * Nc) : (size_t)koff;
    const unsigned base = ring_base + stage * G::STAGE + wave * G::PER_WAVE * 1024;
#pragma unroll
    for (int u = 0; u < G::PER_WAVE; ++u) dma16(gsrc[u] + (is_a[u] ? koff : koff_b), base + u * 1024);
  };
  // Register-staged copies (REG): thread t moves the 16-byte chunks
  // t + NT u of the stage [A rows; B rows] (8 consecutive threads one
  // 128-byte row segment) through registers; global reads of step i + 2 are
  // in flight while step i is multiplied and step i + 1 is written to LDS.
  constexpr int NLD = REG ? (RA + RB) * G::CPR / G::NT : 1;
  static_assert(!REG || ((RA + RB) * G::CPR) % G::NT == 0, "register staging");
  const __bf16* rsrc[NLD];
  int rdst[NLD];
  v4u_t stg[NLD];
  if constexpr (REG) {
#pragma unroll
    for (int u = 0; u < NLD; ++u) {
      const int id = tid + G::NT * u, tr = id / G::CPR, c = id % G::CPR;
      if (tr < RA) {
        const int row = row0 + tr < Mrows ? row0 + tr : Mrows - 1;
        rsrc[u] = A0 + (size_t)row * Kp + c * 8;
      } else {
        const int q = q0 + tr - RA < Nc ? q0 + tr - RA : Nc - 1;
        rsrc[u] = K0 + (size_t)q * Kp + c * 8;
      }
      rdst[u] = tr * G::PITCH + swz<G::CPR>(tr, c) * 16;
    }
  }
  auto rload = [&](int i) {
    const int koff = live[i] * BK;
#pragma unroll
    for (int u = 0; u < NLD; ++u) stg[u] = *reinterpret_cast<const v4u_t*>(rsrc[u] + koff);
  };
  auto rstore = [&](int stage) {
#pragma unroll
    for (int u = 0; u < NLD; ++u)
      *reinterpret_cast<v4u_t*>(smem + stage * G::STAGE + rdst[u]) = stg[u];
  };

  v16f acc_re[TM][TN], acc_im[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc_re[i][j][r] = acc_im[i][j][r] = 0.f;

  // row blocks of this wave that hold rows of the degree (wave-uniform)
  bool blk_live[TM];
#pragma unroll
  for (int i = 0; i < TM; ++i) blk_live[i] = row0 + (wm * TM + i) * 32 < Mrows;

  if constexpr (!REG) {
#pragma unroll
    for (int s = 0; s < ST - 1; ++s)
      if (s < nk) issue(s, s);
  } else {
    static_assert(!REG || ST == 2, "register staging double-buffers");
    if (nk > 0) {
      rload(0);
      rstore(0);
    }
    if (nk > 1) rload(1);
    __syncthreads();
  }

  const int r32 = lane & 31, kh = lane >> 5;
  // The K loop for NL live row blocks (0: the wave only copies and waits at
  // the barriers); the operands of the next 16-wide step are read from LDS
  // while the MFMAs of the current one run.
  auto k_loop = [&](auto nl) {
    constexpr int NL = decltype(nl)::value;
    for (int i = 0; i < nk; ++i) {
      if constexpr (!REG) {
        const int issued = nk < i + ST - 1 ? nk : i + ST - 1;
        wait_groups<ST - 2, G::PER_WAVE>(issued - i - 1);
        __builtin_amdgcn_s_barrier();  // every wave's copies of step i landed; step i-1 is consumed
        if (i + ST - 1 < nk) issue(i + ST - 1, (i + ST - 1) % ST);
      }
      if constexpr (NL > 0) {
        const unsigned char* As = smem + (i % ST) * G::STAGE;
        const unsigned char* Bs = As + RA * G::PITCH;
        auto read = [&](int kk, v4u_t (&xa)[TM], v8bf (&xb)[TN]) {
          const int c = 2 * kk + kh;
#pragma unroll
          for (int jj = 0; jj < TN; ++jj) {
            const int rb = (wn * TN + jj) * 32 + r32;
            if constexpr (!ADJ) {
              xb[jj] = *reinterpret_cast<const v8bf*>(Bs + rb * G::PITCH + swz<G::CPR>(rb, c) * 16);
            } else {
              // contraction rows 4c .. 4c + 3 of output rb: (re, im) each
              v4u_t y;
#pragma unroll
              for (int d = 0; d < 4; ++d) {
                const int kr = 4 * c + d;
                y[d] = *reinterpret_cast<const unsigned*>(Bs + kr * G::PITCH_T +
                                                          swz_k4(kr, rb >> 2) * 16 + (rb & 3) * 4);
              }
              xb[jj] = __builtin_bit_cast(v8bf, y);
            }
          }
#pragma unroll
          for (int ii = 0; ii < NL; ++ii) {
            const int cr = (wm * TM + ii) * 32 + r32;
            xa[ii] = *reinterpret_cast<const v4u_t*>(As + cr * G::PITCH + swz<G::CPR>(cr, c) * 16);
          }
        };
        v4u_t xa[TM], na[TM];
        v8bf xb[TN], nb[TN];
        read(0, xa, xb);
#pragma unroll
        for (int kk = 0; kk < BK / 16; ++kk) {
          if (kk + 1 < BK / 16) read(kk + 1, na, nb);
#pragma unroll
          for (int ii = 0; ii < NL; ++ii) {
            v4u_t xr, xi;
#pragma unroll
            for (int d = 0; d < 4; ++d) {
              const unsigned sw = __builtin_amdgcn_alignbit(xa[ii][d], xa[ii][d], 16u);
              xr[d] = ADJ ? xa[ii][d] : xa[ii][d] ^ 0x80000000u;  // (re, im) / (re, -im)
              xi[d] = ADJ ? sw ^ 0x80000000u : sw;                // (im, -re) / (im, re)
            }
            const v8bf ar = __builtin_bit_cast(v8bf, xr), ai = __builtin_bit_cast(v8bf, xi);
#pragma unroll
            for (int jj = 0; jj < TN; ++jj) {
              acc_re[ii][jj] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ar, xb[jj], acc_re[ii][jj], 0, 0, 0);
              acc_im[ii][jj] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ai, xb[jj], acc_im[ii][jj], 0, 0, 0);
            }
          }
          if (kk + 1 < BK / 16) {
#pragma unroll
            for (int ii = 0; ii < NL; ++ii) xa[ii] = na[ii];
#pragma unroll
            for (int jj = 0; jj < TN; ++jj) xb[jj] = nb[jj];
          }
        }
      }
      if constexpr (REG) {
        if (i + 1 < nk) rstore((i + 1) % 2);  // step i + 1 (its stage was consumed in step i - 1)
        __syncthreads();                       // step i + 1 visible; step i consumed
        if (i + 2 < nk) rload(i + 2);
      }
    }
  };
  static_assert(TM == 2, "live-block dispatch");
  if (blk_live[1]) k_loop(std::integral_constant<int, 2>{});
  else if (blk_live[0]) k_loop(std::integral_constant<int, 1>{});
  else k_loop(std::integral_constant<int, 0>{});
  wait_vmcnt<0>();

  if constexpr (RA * RB * 4 <= G::SMEM) {
    // the tile's outputs as bf16 pairs in LDS ([RA rows][RB outputs], the
    // 16-byte chunks of rows with bit 2 set moved by 128 bytes so the two
    // row groups of a write hit different banks), then 16-byte stores (256 x
    // 256 layer: mixing 96.2 -> 92.6 us against the pair stores below)
    typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
    typedef float f32x2_t __attribute__((ext_vector_type(2)));
    constexpr int RP = RB * 4;  // bytes per staged row
    auto slot = [](int row, int chunk) { return chunk ^ (((row >> 2) & 1) << 3); };
    __syncthreads();  // every wave is done with the ring
    const int col_l = lane & 31, row_l = 4 * (lane >> 5);
#pragma unroll
    for (int jj = 0; jj < TN; ++jj) {
      const int cl = (wn * TN + jj) * 32 + col_l;
      const int q = q0 + cl;
      const bool tok = q < Nc && iabs_(sout_.s[(q < Nc ? q : 0) / Cout]) <= l;
#pragma unroll
      for (int ii = 0; ii < TM; ++ii) {
        if (!blk_live[ii]) continue;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int rl = (wm * TM + ii) * 32 + 8 * (r >> 2) + row_l + (r & 3);
          const f32x2_t v = tok ? (f32x2_t){acc_re[ii][jj][r], acc_im[ii][jj][r]} : (f32x2_t){0.f, 0.f};
          *reinterpret_cast<bf16x2_t*>(smem + rl * RP + slot(rl, cl >> 2) * 16 + (cl & 3) * 4) =
              __builtin_convertvector(v, bf16x2_t);
        }
      }
    }
    __syncthreads();
    const int Np = 2 * Nc;
    constexpr int CPRO = RB / 4;  // 16-byte chunks per staged row
    for (int idx = tid; idx < RA * CPRO; idx += G::NT) {
      const int rl = idx / CPRO, c = idx % CPRO;
      const int row = row0 + rl, q = q0 + 4 * c;
      if (row >= Mrows || q >= Nc) continue;
      *reinterpret_cast<uint4*>(out + ((size_t)l * l * B + row) * Np + 2 * q) =
          *reinterpret_cast<const uint4*>(smem + rl * RP + slot(rl, c) * 16);
    }
    return;
  }

  // register r of a lane holds row 8 (r / 4) + 4 kh + r % 4 of its block,
  // column lane % 32: one complex output, stored as one bf16 pair (the 32
  // lanes of a row write 128 contiguous bytes).  Output spins that do not
  // exist at this degree are written as zero.
  typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
  typedef float f32x2_t __attribute__((ext_vector_type(2)));
  const int Np = 2 * Nc;
  const int col_l = lane & 31, row_l = 4 * (lane >> 5);
#pragma unroll
  for (int jj = 0; jj < TN; ++jj) {
    const int q = q0 + (wn * TN + jj) * 32 + col_l;
    const bool qok = q < Nc;
    const bool tok = qok && iabs_(sout_.s[(qok ? q : 0) / Cout]) <= l;
#pragma unroll
    for (int ii = 0; ii < TM; ++ii) {
      if (!blk_live[ii]) continue;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = row0 + (wm * TM + ii) * 32 + 8 * (r >> 2) + row_l + (r & 3);
        if (!qok || row >= Mrows) continue;
        const f32x2_t v = tok ? (f32x2_t){acc_re[ii][jj][r], acc_im[ii][jj][r]} : (f32x2_t){0.f, 0.f};
        *reinterpret_cast<bf16x2_t*>(out + ((size_t)l * l * B + row) * Np + 2 * q) =
            __builtin_convertvector(v, bf16x2_t);
      }
    }
  }
}

template <int WM, int WN, int ST, bool REG, bool ADJ = false>
hipError_t launch_split(const Plan& p, int B, int Cin, int Cout, const void* coef, const void* K,
                        void* out, hipStream_t st) {
  using G = MixGeomS<WM, WN, ST>;
  Spins si{}, so{};
  for (int i = 0; i < p.n_in; ++i) si.s[i] = p.spins_in[i];
  for (int i = 0; i < p.n_out; ++i) so.s[i] = p.spins_out[i];
  long long tiles = 0;
  for (int l = 0; l < p.L; ++l) tiles += ((2 * l + 1) * B + G::RA - 1) / G::RA;
  const int Nc = p.n_out * Cout;
  const long long blocks = tiles * ((Nc + G::RB - 1) / G::RB);
  const hipError_t e = ensure_dynamic_lds((const void*)mix_split_kernel<WM, WN, ST, REG, ADJ>, G::SMEM);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((mix_split_kernel<WM, WN, ST, REG, ADJ>), dim3(xcd_grid(blocks)), dim3(G::NT), G::SMEM,
                     st, (const __bf16*)coef, (const __bf16*)K, (__bf16*)out, p.L, B, Cin, Cout,
                     p.n_in, p.n_out, si, so);
  return hipGetLastError();
}

// Float form.  K steps of 32 floats (16 complex entries: one 128-byte line
// per row and copy).  Each wave owns one block of 32 expanded rows (16
// coefficient rows) x TN blocks of 32 outputs, MFMA 32x32x2 f32; the
// workgroup covers WM x WN such wave tiles, i.e. 16 WM coefficient rows x
// 32 TN WN outputs.  The contraction order inside a 16-byte chunk (complex
// entries 2c, 2c + 1) is chosen so that each lane needs only one entry: the
// chunk's first MFMA step pairs the real parts of the filter values, the
// second the imaginary parts, and lane half kh holds entry 2c + kh; so a lane
// reads 8 bytes of its coefficient row and 8 of its filter row, and its A
// values are (re, -im) for even expanded rows, (im, re) for odd ones (mol
// mixing 18.5 -> 17.5 us, wx128 36.8 -> 34.7 us against picking two of the
// four floats of a whole 16-byte read).
template <int WM, int WN, int ST, int TN>
struct MixGeomF {
  static constexpr int BK = 32;                 // floats per row per K step
  static constexpr int PITCH = 4 * BK;          // bytes per tile row
  static constexpr int CPR = PITCH / 16;        // 16-byte chunks per row
  static constexpr int RPI = 1024 / PITCH;      // rows per 1 KiB copy
  static constexpr int LPR = 64 / RPI;          // lanes per row
  static constexpr int NW = WM * WN, NT = 64 * NW;
  static constexpr int RA = 16 * WM, RB = 32 * TN * WN;
  static constexpr int NI = (RA + RB) / RPI;    // copies per stage
  static constexpr int PER_WAVE = NI / NW;
  static constexpr int STAGE = (RA + RB) * PITCH;
  static constexpr int SMEM = ST * STAGE;
  static constexpr int MAX_KT = kMaxKp / BK;
  static constexpr int NI_A = RA / RPI;  // copies of coefficient rows
  // k-major filter tile of the adjoint: BK / 2 contraction rows of RB outputs
  static constexpr int PITCH_T = 8 * RB;
  static constexpr int RPI_T = PITCH_T <= 1024 ? 1024 / PITCH_T : 1;
  static constexpr int LPR_T = 64 / RPI_T;
  static_assert((RA + RB) % RPI == 0 && NI % NW == 0 && RA % RPI == 0, "tile shape");
  static_assert(ST >= 2 && (ST - 2) * PER_WAVE < 64, "stages");
};

// ADJ: the adjoint from the filters as stored, as for bfloat16 above; the
// A values are (re, im) for even rows, (im, -re) for odd ones, and a lane
// reads its filter entry (contraction row 2c + kh, its output column) as 8
// bytes of the k-major tile (32 lanes: 256 contiguous bytes).
template <int WM, int WN, int ST, int TN, bool ADJ>
__global__ void __launch_bounds__((MixGeomF<WM, WN, ST, TN>::NT))
    mix_dma_f32_kernel(const float* __restrict__ coef, const float* __restrict__ K,
                       float* __restrict__ out, int L, int B, int Cin, int Cout, int Sin,
                       int Sout, Spins sin_, Spins sout_) {
  using G = MixGeomF<WM, WN, ST, TN>;
  static_assert(!ADJ || (G::PITCH_T <= 1024 && 1024 % G::PITCH_T == 0 &&
                         (G::BK / 2) % G::RPI_T == 0 && (G::BK / 2) * G::PITCH_T == G::RB * G::PITCH),
                "adjoint filter tile");
  constexpr int RA = G::RA, RB = G::RB, BK = G::BK;
  extern __shared__ __align__(16) unsigned char smem[];  // G::SMEM bytes: the ring
  __shared__ int live[G::MAX_KT];
  __shared__ int n_live_s;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WN, wn = wave % WN;
  const int Kc = Sin * Cin, Nc = Sout * Cout;
  const int Kp = 2 * Kc;
  const int n_tiles_n = (Nc + RB - 1) / RB;

  // logical block = ((l, row tile), column tile), largest degrees first
  const int lbk = xcd_logical_block();
  const int ntile = lbk % n_tiles_n;
  int t = lbk / n_tiles_n;
  int l = L - 1;
  for (; l >= 0; --l) {
    const int ntl = ((2 * l + 1) * B + RA - 1) / RA;
    if (t < ntl) break;
    t -= ntl;
  }
  if (l < 0) return;
  const int Mrows = (2 * l + 1) * B;
  const int row0 = t * RA;
  const int q0 = ntile * RB;

  // K steps of input spins that exist at this degree (whole channel blocks)
  if (tid == 0) {
    const int per_spin = 2 * Cin / BK;
    int n = 0;
    for (int si = 0; si < Sin; ++si)
      if (iabs_(sin_.s[si]) <= l)
        for (int k = 0; k < per_spin; ++k) live[n++] = si * per_spin + k;
    n_live_s = n;
  }
  __syncthreads();
  const int nk = n_live_s;

  const float* A0 = coef + (size_t)l * l * B * Kp;  // rows (m, b) of degree l
  const float* K0 = K + (size_t)l * Nc * Kp;        // filter rows q of degree l
  const unsigned ring_base = lds_addr(smem);

  // copy g = wave * PER_WAVE + u moves tile rows [g RPI, (g + 1) RPI) of the
  // stage [A rows; B rows]; rows past the end of a matrix are clamped to its
  // last row (their products are discarded)
  const float* gsrc[G::PER_WAVE];
  bool is_a[G::PER_WAVE];  // wave-uniform
#pragma unroll
  for (int u = 0; u < G::PER_WAVE; ++u) {
    const int g = wave * G::PER_WAVE + u;
    is_a[u] = g < G::NI_A;
    if (is_a[u]) {
      const int tr = g * G::RPI + lane / G::LPR;
      const int row = row0 + tr < Mrows ? row0 + tr : Mrows - 1;
      gsrc[u] = A0 + (size_t)row * Kp + swz<G::CPR>(tr, lane % G::LPR) * 4;
    } else if (!ADJ) {
      const int rb = (g - G::NI_A) * G::RPI + lane / G::LPR;
      const int q = q0 + rb < Nc ? q0 + rb : Nc - 1;
      gsrc[u] = K0 + (size_t)q * Kp + swz<G::CPR>(rb, lane % G::LPR) * 4;
    } else {
      // contraction row kb of the step, 2 outputs per chunk; chunks past the
      // last output are clamped to it (their products are discarded)
      const int kb = (g - G::NI_A) * G::RPI_T + lane / G::LPR_T;
      const int q = min(q0 + 2 * (lane % G::LPR_T), Nc - 2);
      gsrc[u] = K0 + (size_t)kb * (2 * Nc) + 2 * q;
    }
  }
  auto issue = [&](int i, int stage) {
    const int koff = live[i] * BK;  // along coefficient rows
    const size_t koff_b = ADJ ? (size_t)live[i] * (BK / 2) * (2 * Nc) : (size_t)koff;
    const unsigned base = ring_base + stage * G::STAGE + wave * G::PER_WAVE * 1024;
#pragma unroll
    for (int u = 0; u < G::PER_WAVE; ++u) dma16(gsrc[u] + (is_a[u] ? koff : koff_b), base + u * 1024);
  };

  v16f acc[TN];
#pragma unroll
  for (int j = 0; j < TN; ++j)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[j][r] = 0.f;

#pragma unroll
  for (int s = 0; s < ST - 1; ++s)
    if (s < nk) issue(s, s);

  const int r32 = lane & 31, kh = lane >> 5;
  const int cr = wm * 16 + (r32 >> 1);  // coefficient row of this lane's A row
  for (int i = 0; i < nk; ++i) {
    const int issued = nk < i + ST - 1 ? nk : i + ST - 1;
    wait_groups<ST - 2, G::PER_WAVE>(issued - i - 1);
    __builtin_amdgcn_s_barrier();  // every wave's copies of step i landed; step i-1 is consumed
    if (i + ST - 1 < nk) issue(i + ST - 1, (i + ST - 1) % ST);
    const unsigned char* As = smem + (i % ST) * G::STAGE;
    const unsigned char* Bs = As + RA * G::PITCH;
    // the two MFMA steps of a 16-byte chunk (complex entries 2cc, 2cc + 1)
    // take the real parts (step 0) and then the imaginary parts (step 1),
    // lane half kh holding entry 2cc + kh: each lane reads only its 8-byte
    // half of both operands.  Row parity picks the expansion: forward
    // (re | -im) / (im | re), adjoint (re | im) / (im | -re).
    const bool odd = (r32 & 1) != 0;
    auto lda2 = [&](int cc) {
      return *reinterpret_cast<const float2*>(As + cr * G::PITCH + swz<G::CPR>(cr, cc) * 16 +
                                              kh * 8);
    };
    auto ldb2 = [&](int jj, int cc) {
      const int q = wn * 32 * TN + jj * 32 + r32;
      if constexpr (!ADJ)
        return *reinterpret_cast<const float2*>(Bs + q * G::PITCH + swz<G::CPR>(q, cc) * 16 +
                                                kh * 8);
      else
        return *reinterpret_cast<const float2*>(Bs + (2 * cc + kh) * G::PITCH_T + q * 8);
    };
    float2 a2 = lda2(0), b2[TN];
#pragma unroll
    for (int jj = 0; jj < TN; ++jj) b2[jj] = ldb2(jj, 0);
#pragma unroll
    for (int cc = 0; cc < G::CPR; ++cc) {
      float2 na = a2, nb[TN];
#pragma unroll
      for (int jj = 0; jj < TN; ++jj) nb[jj] = b2[jj];
      if (cc + 1 < G::CPR) {
        na = lda2(cc + 1);
#pragma unroll
        for (int jj = 0; jj < TN; ++jj) nb[jj] = ldb2(jj, cc + 1);
      }
      const float a0 = odd ? a2.y : a2.x;
      const float a1 = ADJ ? (odd ? -a2.x : a2.y) : (odd ? a2.x : -a2.y);
#pragma unroll
      for (int jj = 0; jj < TN; ++jj)
        acc[jj] = __builtin_amdgcn_mfma_f32_32x32x2f32(a0, b2[jj].x, acc[jj], 0, 0, 0);
#pragma unroll
      for (int jj = 0; jj < TN; ++jj)
        acc[jj] = __builtin_amdgcn_mfma_f32_32x32x2f32(a1, b2[jj].y, acc[jj], 0, 0, 0);
      a2 = na;
#pragma unroll
      for (int jj = 0; jj < TN; ++jj) b2[jj] = nb[jj];
      if (cc + 1 < G::CPR) __builtin_amdgcn_sched_group_barrier(0x100, 1 + TN, 0);  // LDS reads
      __builtin_amdgcn_sched_group_barrier(0x008, 2 * TN, 0);                      // MFMA
      __builtin_amdgcn_sched_barrier(0);
    }
  }
  wait_vmcnt<0>();

  // registers r and r + 1 (r even) of a lane hold expanded rows 2i and 2i + 1
  // of its column q: the real and imaginary part of output (row0 + i, q0 + q)
  const int col_l = lane & 31, row_l = 4 * (lane >> 5);
#pragma unroll
  for (int jj = 0; jj < TN; ++jj) {
    const int q = q0 + wn * 32 * TN + jj * 32 + col_l;
    const bool qok = q < Nc;
    const bool tok = qok && iabs_(sout_.s[(qok ? q : 0) / Cout]) <= l;
#pragma unroll
    for (int r = 0; r < 16; r += 2) {
      const int er = wm * 32 + 8 * (r >> 2) + row_l + (r & 3);  // even
      const int row = row0 + (er >> 1);
      if (!qok || row >= Mrows) continue;
      const float2 v = tok ? make_float2(acc[jj][r], acc[jj][r + 1]) : make_float2(0.f, 0.f);
      *reinterpret_cast<float2*>(out + ((size_t)l * l * B + row) * (2 * Nc) + 2 * q) = v;
    }
  }
}

template <int WM, int WN, int ST, int TN, bool ADJ = false>
hipError_t launch_geom_f32(const Plan& p, int B, int Cin, int Cout, const void* coef,
                           const void* K, void* out, hipStream_t st) {
  using G = MixGeomF<WM, WN, ST, TN>;
  Spins si{}, so{};
  for (int i = 0; i < p.n_in; ++i) si.s[i] = p.spins_in[i];
  for (int i = 0; i < p.n_out; ++i) so.s[i] = p.spins_out[i];
  long long tiles = 0;
  for (int l = 0; l < p.L; ++l) tiles += ((2 * l + 1) * B + G::RA - 1) / G::RA;
  const int Nc = p.n_out * Cout;
  const long long blocks = tiles * ((Nc + G::RB - 1) / G::RB);
  const hipError_t e =
      ensure_dynamic_lds((const void*)mix_dma_f32_kernel<WM, WN, ST, TN, ADJ>, G::SMEM);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((mix_dma_f32_kernel<WM, WN, ST, TN, ADJ>), dim3(xcd_grid(blocks)), dim3(G::NT), G::SMEM, st,
                     (const float*)coef, (const float*)K, (float*)out, p.L, B, Cin, Cout, p.n_in,
                     p.n_out, si, so);
  return hipGetLastError();
}

// Tile shape: 128 coefficient rows x 128 outputs, two 64-wide K steps
// resident (two workgroups of 8 waves per CU); channel counts that are a
// multiple of 16 but not of 32 take 32-wide K steps.
#ifndef SWSFT_MIX_DMA_BK
#define SWSFT_MIX_DMA_BK 64
#endif
#ifndef SWSFT_MIX_DMA_RA
#define SWSFT_MIX_DMA_RA 128
#endif
#ifndef SWSFT_MIX_DMA_RB
#define SWSFT_MIX_DMA_RB 128
#endif
#ifndef SWSFT_MIX_DMA_STAGES
#define SWSFT_MIX_DMA_STAGES 2
#endif
// bf16 forward with split real / imaginary accumulators: WM, WN, ST of MixGeomS
#ifndef SWSFT_MIX_SPLIT
#define SWSFT_MIX_SPLIT 1
#endif
#ifndef SWSFT_MIX_SPLIT_GEOM
#define SWSFT_MIX_SPLIT_GEOM 2, 2, 2
#endif
// 1: the split kernel stages its operands through registers instead of
// direct global -> LDS copies
#ifndef SWSFT_MIX_SPLIT_REG
#define SWSFT_MIX_SPLIT_REG 0
#endif
// float: WM, WN, ST, TN of MixGeomF
#ifndef SWSFT_MIX_DMA_F32
#define SWSFT_MIX_DMA_F32 2, 2, 4, 1
#endif
#ifndef SWSFT_MIX_F32_MIN_OUT
#define SWSFT_MIX_F32_MIN_OUT 64
#endif

}  // namespace

bool mix_dma_supported(const Plan& p, int Cin, int Cout) {
  // float: outputs of at least 64 (narrower ones run as fast register-staged)
  if (p.dtype == SWSFT_F32)
    return (2 * Cin) % 32 == 0 && 2 * p.n_in * Cin <= kMaxKp && p.n_out * Cout >= SWSFT_MIX_F32_MIN_OUT;
  return p.dtype == SWSFT_BF16 && (2 * Cin) % 32 == 0 && 2 * p.n_in * Cin <= kMaxKp &&
         Cout % 4 == 0;
}

bool mix_adj_dma_supported(const Plan& p, int Cin, int Cout) {
  if (p.dtype == SWSFT_F32)  // as the forward float kernel; outputs in 16-byte pairs
    return (2 * Cin) % 32 == 0 && 2 * p.n_in * Cin <= kMaxKp &&
           p.n_out * Cout >= SWSFT_MIX_F32_MIN_OUT && (p.n_out * Cout) % 2 == 0;
  return p.dtype == SWSFT_BF16 && (2 * Cin) % 64 == 0 && 2 * p.n_in * Cin <= kMaxKp &&
         Cout % 4 == 0;
}

hipError_t launch_mix_adj_dma(const Plan& p, int B, int Cin, int Cout, const void* coef,
                              const void* K, void* out, hipStream_t st) {
  if (p.dtype == SWSFT_F32)
    return launch_geom_f32<SWSFT_MIX_DMA_F32, true>(p, B, Cin, Cout, coef, K, out, st);
  return launch_split<SWSFT_MIX_SPLIT_GEOM, false, true>(p, B, Cin, Cout, coef, K, out, st);
}

hipError_t launch_mix_dma(const Plan& p, int B, int Cin, int Cout, const void* coef,
                          const void* K, void* out, hipStream_t st) {
  // float: 32 coefficient rows x 64 outputs, one 32 x 32 block per wave, 4 K
  // steps resident (measured against 32 x 128 with 3 steps, 16 x 128, 32 x 64
  // with 2 waves and 64 x 64 with 8 waves: mol 19.4 -> 18.3 us, wx128 42.3 -> 36.4 us)
  if (p.dtype == SWSFT_F32) return launch_geom_f32<SWSFT_MIX_DMA_F32>(p, B, Cin, Cout, coef, K, out, st);
#if SWSFT_MIX_SPLIT
  if ((2 * Cin) % 64 == 0)
    return launch_split<SWSFT_MIX_SPLIT_GEOM, SWSFT_MIX_SPLIT_REG != 0>(p, B, Cin, Cout, coef, K, out,
                                                                        st);
#endif
  if ((2 * Cin) % SWSFT_MIX_DMA_BK == 0)
    return launch_geom<SWSFT_MIX_DMA_BK, SWSFT_MIX_DMA_RA, SWSFT_MIX_DMA_RB, SWSFT_MIX_DMA_STAGES>(
        p, B, Cin, Cout, coef, K, out, st);
  return launch_geom<32, 128, 128, 4>(p, B, Cin, Cout, coef, K, out, st);
}

}  // namespace swsft
