// Per-degree mixing GEMM for bfloat16 storage, fed by direct global -> LDS
// loads (global_load_lds_dwordx4) into a ring of LDS stages.
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
// Preconditions (checked by the launcher): bf16, K' = 2 S_in C_in a multiple
// of 32, each input spin's channel block a whole number of 32-wide K steps.
#include "mfma_tile.h"
#include "swsft_internal.h"
#include "xcd.h"

namespace swsft {
namespace {

constexpr int kNT = 256;     // 4 waves
constexpr int kBK = 32;      // bf16 per row per K step (64 bytes)
constexpr int kRowsA = 64;   // coefficient rows per tile (128 expanded GEMM rows)
constexpr int kRowsB = 128;  // filter rows (complex outputs) per tile
constexpr int kStages = 4;
constexpr int kStageBytes = (kRowsA + kRowsB) * kBK * 2;
constexpr int kMaxKTiles = 256;  // K' <= 8192

struct Spins {
  int s[kMaxSpins];
};

__device__ __forceinline__ int iabs_(int v) { return v < 0 ? -v : v; }

// LDS slot of 16-byte chunk c of tile row r: chunks are XOR-swizzled so that
// the 32 rows one MFMA operand read touches fall in distinct banks.
__device__ __forceinline__ int swz(int r, int c) { return c ^ (((r >> 1) ^ (r >> 3)) & 3); }

// One direct global -> LDS copy of 16 bytes per lane: lane l writes
// LDS[lds_base + 16 l].  M0 holds the wave-uniform LDS base (with the NOP
// its write requires before the copy).
__device__ __forceinline__ void dma16(const void* g, unsigned lds_base) {
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, off"
               :
               : "s"(__builtin_amdgcn_readfirstlane(lds_base)), "v"(g)
               : "memory");
}

template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 16, "vmcnt immediate");
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

__global__ void __launch_bounds__(kNT) mix_dma_kernel(const __bf16* __restrict__ coef,
                                                      const __bf16* __restrict__ K,
                                                      __bf16* __restrict__ out, int L, int B,
                                                      int Cin, int Cout, int Sin, int Sout,
                                                      Spins sin_, Spins sout_) {
  __shared__ __align__(16) unsigned char ring[kStages * kStageBytes];
  __shared__ int live[kMaxKTiles];
  __shared__ int n_live_s;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;  // 2 x 2 waves, 64 expanded rows x 64 cols each
  const int Kc = Sin * Cin, Nc = Sout * Cout;
  const int Kp = 2 * Kc;
  const int n_tiles_n = (Nc + kRowsB - 1) / kRowsB;

  // logical block = ((l, row tile), column tile), largest degrees first
  int lbk = xcd_logical_block();
  const int ntile = lbk % n_tiles_n;
  int t = lbk / n_tiles_n;
  int l = L - 1;
  for (; l >= 0; --l) {
    const int ntl = ((2 * l + 1) * B + kRowsA - 1) / kRowsA;
    if (t < ntl) break;
    t -= ntl;
  }
  if (l < 0) return;
  const int Mrows = (2 * l + 1) * B;
  const int row0 = t * kRowsA;
  const int q0 = ntile * kRowsB;

  // K steps of input spins that exist at this degree (whole channel blocks)
  if (tid == 0) {
    const int per_spin = 2 * Cin / kBK;
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
  const unsigned ring_base = (unsigned)(uintptr_t)ring;

  // each wave copies 16 rows (one 1 KiB instruction) of A and 32 rows of B
  const int ra = wave * 16 + (lane >> 2);
  const int slot = lane & 3;
  const int rowA = row0 + ra < Mrows ? row0 + ra : Mrows - 1;  // clamp: rows past the end are discarded
  const __bf16* gA = A0 + (size_t)rowA * Kp + swz(ra, slot) * 8;
  const __bf16* gB[2];
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const int rb = wave * 32 + h * 16 + (lane >> 2);
    const int q = q0 + rb < Nc ? q0 + rb : Nc - 1;
    gB[h] = K0 + (size_t)q * Kp + swz(rb, slot) * 8;
  }
  auto issue = [&](int i, int stage) {
    const int koff = live[i] * kBK;
    const unsigned base = ring_base + stage * kStageBytes;
    dma16(gA + koff, base + wave * 16 * 64);
    dma16(gB[0] + koff, base + kRowsA * 64 + (wave * 32) * 64);
    dma16(gB[1] + koff, base + kRowsA * 64 + (wave * 32 + 16) * 64);
  };
  constexpr int kPerTile = 3;  // DMA instructions per wave per K step

  typedef unsigned v4u __attribute__((ext_vector_type(4)));
  v16f acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  // prologue: K steps 0 .. kStages-2 in flight
#pragma unroll
  for (int s = 0; s < kStages - 1; ++s)
    if (s < nk) issue(s, s);

  const int r32 = lane & 31, kh = lane >> 5;
  const unsigned rot = (lane & 1) ? 16u : 0u;
  const unsigned sgn = (lane & 1) ? 0u : 0x80000000u;
  for (int i = 0; i < nk; ++i) {
    // K step i has landed once at most (issued - i - 1) steps are outstanding
    const int issued = nk < i + kStages - 1 ? nk : i + kStages - 1;
    const int ahead = issued - i - 1;
    if (ahead >= 2) wait_vmcnt<2 * kPerTile>();
    else if (ahead == 1) wait_vmcnt<kPerTile>();
    else wait_vmcnt<0>();
    __builtin_amdgcn_s_barrier();  // every wave's copies of step i landed; step i-1 is consumed
    if (i + kStages - 1 < nk) issue(i + kStages - 1, (i + kStages - 1) % kStages);
    const unsigned char* st = ring + (i % kStages) * kStageBytes;
    const unsigned char* As = st;
    const unsigned char* Bs = st + kRowsA * 64;
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) {  // two 16-wide MFMA K steps per 32-wide tile
      const int c = 2 * kk + kh;
      v8bf a[2], b[2];
#pragma unroll
      for (int ii = 0; ii < 2; ++ii) {
        const int er = wm * 64 + ii * 32 + r32;  // expanded GEMM row
        const int cr = er >> 1;                  // coefficient row in the tile
        v4u x = *reinterpret_cast<const v4u*>(As + cr * 64 + swz(cr, c) * 16);
        // odd rows (im, re): rotate by 16 bits; even rows (re, -im): flip the
        // high half's sign (er & 1 == lane & 1, selected without branches)
        v4u y;
#pragma unroll
        for (int d = 0; d < 4; ++d) y[d] = __builtin_amdgcn_alignbit(x[d], x[d], rot) ^ sgn;
        a[ii] = __builtin_bit_cast(v8bf, y);
      }
#pragma unroll
      for (int jj = 0; jj < 2; ++jj) {
        const int rb = wn * 64 + jj * 32 + r32;
        b[jj] = *reinterpret_cast<const v8bf*>(Bs + rb * 64 + swz(rb, c) * 16);
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

  // epilogue: C[er][q] -> out row (row0 + er/2), real column 2q + er%2, via LDS
  constexpr int LDC = 2 * kRowsB + 8;  // bf16 per LDS row
  __bf16* cs = reinterpret_cast<__bf16*>(ring);
  const int col_l = lane & 31, row_l = 4 * (lane >> 5);
#pragma unroll
  for (int ii = 0; ii < 2; ++ii)
#pragma unroll
    for (int jj = 0; jj < 2; ++jj)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int er = wm * 64 + ii * 32 + 8 * (r >> 2) + row_l + (r & 3);
        const int q = wn * 64 + jj * 32 + col_l;
        cs[(er >> 1) * LDC + 2 * q + (er & 1)] = (__bf16)acc[ii][jj][r];
      }
  __syncthreads();
  const int Np = 2 * Nc;
  __bf16* O0 = out + ((size_t)l * l * B + row0) * Np + 2 * q0;
  const int rows = Mrows - row0 < kRowsA ? Mrows - row0 : kRowsA;
  const int cols = 2 * (Nc - q0 < kRowsB ? Nc - q0 : kRowsB);
  constexpr int VPR = 2 * kRowsB / 8;
  for (int idx = tid; idx < kRowsA * VPR; idx += kNT) {
    const int row = idx / VPR;
    const int col = (idx % VPR) * 8;
    if (row >= rows || col >= cols) continue;
    uint4 v = *reinterpret_cast<const uint4*>(&cs[row * LDC + col]);
    // output spins that do not exist at this degree are zero
    const int tq = (q0 + col / 2) / Cout;  // 8 reals = 4 complex outputs, one spin (Cout % 4 == 0)
    if (iabs_(sout_.s[tq]) > l) v = make_uint4(0, 0, 0, 0);
    *reinterpret_cast<uint4*>(O0 + (size_t)row * Np + col) = v;
  }
}

}  // namespace

bool mix_dma_supported(const Plan& p, int Cin, int Cout) {
  const int Kp = 2 * p.n_in * Cin;
  return p.dtype == SWSFT_BF16 && (2 * Cin) % kBK == 0 && Kp / kBK <= kMaxKTiles &&
         Cout % 4 == 0;
}

hipError_t launch_mix_dma(const Plan& p, int B, int Cin, int Cout, const void* coef,
                          const void* K, void* out, hipStream_t st) {
  Spins si{}, so{};
  for (int i = 0; i < p.n_in; ++i) si.s[i] = p.spins_in[i];
  for (int i = 0; i < p.n_out; ++i) so.s[i] = p.spins_out[i];
  int tiles = 0;
  for (int l = 0; l < p.L; ++l) tiles += ((2 * l + 1) * B + kRowsA - 1) / kRowsA;
  const int Nc = p.n_out * Cout;
  const long long blocks = (long long)tiles * ((Nc + kRowsB - 1) / kRowsB);
  hipLaunchKernelGGL(mix_dma_kernel, dim3(xcd_grid(blocks)), dim3(kNT), 0, st,
                     (const __bf16*)coef, (const __bf16*)K, (__bf16*)out, p.L, B, Cin, Cout,
                     p.n_in, p.n_out, si, so);
  return hipGetLastError();
}

}  // namespace swsft
