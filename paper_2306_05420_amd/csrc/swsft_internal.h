// Internal declarations shared by the host API and the kernel launchers.
#pragma once

#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>
#include <string>

#include "../../include/swsft.h"

namespace swsft {

constexpr int kMaxSpins = 8;
constexpr int kMaxTimedLaunches = 4096;

enum Stage : int {
  kStageDftFwd = 0,
  kStageLatFwd = 1,
  kStageMix = 2,
  kStageLatInv = 3,
  kStageDftInv = 4,
  kStagePhaseCollapse = 5,
  kStageTables = 6,
  kStageFilterGrad = 7,
  kStageFilterAdjoint = 8,
  kStageBatchNorm = 9,
  kStageDeltaTheta = 10,
  kStageSmallFwd = 11,
  kStageSmallInv = 12,
  kNumStages = 13
};

inline int round_up(int x, int m) { return (x + m - 1) / m * m; }

struct Plan {
  int device = 0;
  int H = 0, W = 0, L = 0;
  int Hp = 0;  // H rounded up to a multiple of 8 (row pitch of the forward tables)
  int JT = 0;  // latitude tile of the X / Y spectra: min(H, 32), the latitude GEMMs' K step
  int Lp = 0;  // L rounded up to a multiple of 32 (row pitch of inverse tables: whole K steps)
  int M = 0;   // number of orders, 2L - 1
  int n_in = 0, n_out = 0;
  int spins_in[kMaxSpins] = {0};
  int spins_out[kMaxSpins] = {0};
  int dtype = SWSFT_F32;
  size_t elem = 4;  // bytes of one real of the storage type
  // device tables
  void* tab_fwd = nullptr;  // [n_in][M][L][Hp]
  void* tab_inv = nullptr;  // [n_out][M][Hp][Lp]   (rows j < H used)
  // backward pass: weighted factors j-major for spins_in (adjoint of the
  // analysis), unweighted factors l-major for spins_out (adjoint of the synthesis)
  void* tab_bwd_syn = nullptr;  // [n_in][M][Hp][Lp]
  void* tab_bwd_ana = nullptr;  // [n_out][M][L][Hp]
  float2* twiddle = nullptr;  // [W]: exp(-2 pi i r / W)
  // creation flags (SWSFT_PLAN_*); with SWSFT_PLAN_DFT_MATMUL the forward
  // longitude stage is a dense DFT GEMM against dft_mat [2M][2W]
  // batch count of the coefficient array the latitude synthesis reads (0: the
  // call's B): lets lat_inv run on a batch range of a larger array
  int coef_ldb = 0;
  unsigned flags = 0;
  void* dft_mat = nullptr;
  void* dft_mat_inv = nullptr;  // [2W][2M]: the inverse longitude stage of SWSFT_PLAN_DFT_MATMUL
  // Wigner-Delta route (SWSFT_PLAN_DELTA / SWSFT_PLAN_DELTA_SYM): theta tables
  // and Delta tables, layouts in delta.hip
  void* delta_theta_fwd = nullptr;
  void* delta_theta_inv = nullptr;
  void* delta_fwd = nullptr;  // [n_in][M][L][R]
  void* delta_inv = nullptr;  // [n_out][M][R][Lp]
  bool fft_ok = true;  // W is a size of the register FFT (a power of two <= 512)
  // stage timing
  bool timing = false;
  int n_timed = 0;
  hipEvent_t* ev = nullptr;  // 2 * kMaxTimedLaunches
  int* ev_stage = nullptr;   // kMaxTimedLaunches

  size_t fwd_table_elems() const { return (size_t)M * L * Hp; }
  size_t inv_table_elems() const { return (size_t)M * Hp * Lp; }
};

// Sizes (in reals of the storage type) of the intermediate buffers.
// X / Y spectra, K-tiled: [S][2L-1][H/JT][B*C][re/im][JT], so that one
// latitude tile of all maps is one contiguous block.
inline size_t xy_elems(const Plan& p, int S, int B, int C) {
  return (size_t)S * p.M * (size_t)B * C * 2 * p.H;
}
inline size_t coef_elems(const Plan& p, int S, int B, int C) {
  return (size_t)p.L * p.L * (size_t)B * S * C * 2;
}

// The library-owned workspace of spin_sph_conv_forward_noalloc (noalloc.hip):
// a file-scope device array of this many bytes on every device.
constexpr size_t kNoAllocScratchBytes = size_t(128) << 20;
// Look up (once per device, with that device current) and remember the
// device address of the array; scratch_of returns it (NULL if never looked up).
hipError_t register_scratch(int device);
void* scratch_of(int device);

// Raise a kernel's dynamic LDS limit to `bytes` (no-op up to 64 KiB).  The
// attribute is set once per (device, kernel) and size: later launches make no
// runtime call, so a launch sequence can be captured in a graph once it has
// run eagerly.
hipError_t ensure_dynamic_lds(const void* kern, size_t bytes);

// ---- kernel launchers (return hipGetLastError() of the launch) ----
hipError_t launch_tables(const Plan& p, hipStream_t st);

// x [B][S][C][H][W] -> X [S][M][H/JT][B*C][2][JT]
hipError_t launch_dft_fwd(const Plan& p, int S, int B, int C, const void* x, void* X,
                          hipStream_t st);
// the dense-DFT forward longitude stage (dft_mm.hip) and its plan-time matrix
hipError_t launch_dft_fwd_matmul(const Plan& p, int S, int B, int C, const void* x, void* X,
                                 hipStream_t st);
hipError_t launch_dft_matrix(const Plan& p, hipStream_t st);
// the dense-DFT inverse longitude stage (dft_mm.hip) and its plan-time matrix
// [2W][dft_inv_pitch(M)] (rows padded with zeros to a multiple of 8 values)
__host__ __device__ inline int dft_inv_pitch(int M) { return (2 * M + 7) / 8 * 8; }
hipError_t launch_dft_inv_matmul(const Plan& p, int S, int B, int C, const void* Y, void* y,
                                 hipStream_t st);
hipError_t launch_dft_matrix_inv(const Plan& p, hipStream_t st);
// the Wigner-Delta route (delta.hip): R = L rows (with the symmetries) or 2L
int delta_rows(const Plan& p);
size_t delta_fwd_theta_elems(const Plan& p);
size_t delta_inv_theta_elems(const Plan& p);
size_t delta_fwd_table_elems(const Plan& p);
size_t delta_inv_table_elems(const Plan& p);
hipError_t launch_delta_tables(const Plan& p, hipStream_t st);
hipError_t launch_delta_theta_fwd(const Plan& p, int B, int C, const void* X, void* CS,
                                  hipStream_t st);
hipError_t launch_delta_theta_inv(const Plan& p, int B, int C, const void* G, void* Y,
                                  hipStream_t st);
inline bool is_delta(const Plan& p) {
  return (p.flags & (SWSFT_PLAN_DELTA | SWSFT_PLAN_DELTA_SYM)) != 0;
}
// [S][M][R/32][2 B C][32] intermediate of the Delta route (0 without it)
inline size_t delta_elems(const Plan& p, int S, int B, int C) {
  return is_delta(p) ? (size_t)S * p.M * delta_rows(p) * 2 * (size_t)B * C : 0;
}
// small grids (small.hip): whole transforms per map in one launch each
bool small_path(const Plan& p, int Cin);
hipError_t launch_small_fwd(const Plan& p, int B, int C, const void* x, void* coef,
                            hipStream_t st);
hipError_t launch_small_inv(const Plan& p, int B, int C_in, int C_out, const void* coef,
                            const void* K, void* y, hipStream_t st);
// Y [S][M][H/JT][B*C][2][JT] -> y [B][S][C][H][W]
hipError_t launch_dft_inv(const Plan& p, int S, int B, int C, const void* Y, void* y,
                          hipStream_t st);
// X (spins_in) -> coef [L^2][B][S_in][C]
hipError_t launch_lat_fwd(const Plan& p, int B, int C, const void* X, void* coef,
                          hipStream_t st);
// coef' [L^2][B][S_out][C] -> Y (spins_out)
hipError_t launch_lat_inv(const Plan& p, int B, int C, const void* coef, void* Y,
                          hipStream_t st);
// coef [L^2][B][S_in][C_in] x K -> coef' [L^2][B][S_out][C_out]
hipError_t launch_mix(const Plan& p, int B, int C_in, int C_out, const void* coef,
                      const void* K, void* coef_out, hipStream_t st);
// Backward pass (backward.hip, gemm.hip).
// KH[l][(s,c)][(t,c')] = conj(K[l][(t,c')][(s,c)]): the filters of the adjoint mixing
hipError_t launch_filter_adjoint(const Plan& p, int C_in, int C_out, const void* K, void* KH,
                                 hipStream_t st);
// gK[l][(t,c')][(s,c)] = sum_{(m,b)} g[l][(m,b)][(t,c')] conj(a[l][(m,b)][(s,c)]), zero
// where |s| > l or |t| > l; a [L^2][B][S_in][C_in], g [L^2][B][S_out][C_out].
// part: filter_grad_split_bytes(p, B, C_in, C_out) bytes of workspace (the
// partial sums of a split contraction; unused when that is 0).
size_t filter_grad_split_bytes(const Plan& p, int B, int C_in, int C_out);
int filter_grad_split_rows(const Plan& p, int B, int C_in, int C_out);
hipError_t launch_filter_grad(const Plan& p, int B, int C_in, int C_out, const void* a,
                              const void* g, void* gK, void* part, hipStream_t st);
// Spectral batch norm on coefficients [L^2][B][S_out][C] of plan p's output
// spins (batch_norm.hip); ws holds bn_workspace_bytes(p, B, C) bytes.
size_t bn_workspace_bytes(const Plan& p, int B, int C);
bool bn_supported(const Plan& p, int C);  // S_out * C <= 2048
hipError_t launch_batch_norm(const Plan& p, int B, int C, const void* a, const float* gamma,
                             const float2* beta, float eps, const float* var_in, float* var_out,
                             const void* skip, void* out, void* ws, hipStream_t st);
// bf16 latitude GEMMs fed by direct global -> LDS copies (see lat_dma.hip).
bool lat_fwd_dma_supported(const Plan& p, int B, int C);
bool lat_inv_dma_supported(const Plan& p, int B, int C);
hipError_t launch_lat_fwd_dma(const Plan& p, int B, int C, const void* X, void* coef,
                              hipStream_t st);
hipError_t launch_lat_inv_dma(const Plan& p, int B, int C, const void* coef, void* Y,
                              hipStream_t st);
// Mixing fed by direct global -> LDS copies (bf16 and float; see mix_dma.hip).
bool mix_dma_supported(const Plan& p, int C_in, int C_out);
hipError_t launch_mix_dma(const Plan& p, int B, int C_in, int C_out, const void* coef,
                          const void* K, void* coef_out, hipStream_t st);
// The adjoint mixing from the filters as stored (DMA kernels): with plan p whose
// input spins are the layer's output spins, coef_out[l][(m,b)][(s,c)] =
// sum_(t,c') coef[l][(m,b)][(t,c')] conj(K[l][(t,c')][(s,c)]), K the layer's
// filters [L][S_p_in][C_in][S_p_out][C_out] (C_in, C_out of this call).
bool mix_adj_dma_supported(const Plan& p, int C_in, int C_out);
hipError_t launch_mix_adj_dma(const Plan& p, int B, int C_in, int C_out, const void* coef,
                              const void* K, void* coef_out, hipStream_t st);
// Largest channel count the phase-collapse kernel stages in LDS for n_spins.
int phase_collapse_max_channels(int n_spins);
hipError_t launch_phase_collapse(const Plan& p, int B, int C, const void* x,
                                 const float2* W1, const float2* W2, const float2* bias,
                                 void* y, hipStream_t st);
// Whole transforms of 32 x 32 float grids in one launch per direction
// (fused32.hip): the longitude spectrum stays in LDS.  C (maps per batch
// item and spin) a multiple of 8.
inline bool fused32_ok(const Plan& p, int C) {
  return p.H == 32 && p.W == 32 && p.dtype == SWSFT_F32 && p.fft_ok &&
         !(p.flags & SWSFT_PLAN_DFT_MATMUL) && !is_delta(p) && C % 8 == 0 && p.Hp == 32 &&
         p.L <= 16 && p.Lp % 4 == 0;
}
// x [B][S_in][C][32][32] -> coef [L^2][B][S_in][C] with p.tab_fwd
hipError_t launch_fused32_fwd(const Plan& p, int B, int C, const void* x, void* coef,
                              hipStream_t st);
// coef [L^2][Bc][S_out][C] (Bc = p.coef_ldb or B) -> y [B][S_out][C][32][32] with p.tab_inv
hipError_t launch_fused32_inv(const Plan& p, int B, int C, const void* coef, void* y,
                              hipStream_t st);
// Measurement helper (probe.hip): n_waves waves (a multiple of 4) each run
// `iters` rounds of four register-only MFMAs of the dtype's shape; out holds
// 64 n_waves floats.
double mfma_probe_flops_per_wave_round(int dtype);
hipError_t launch_mfma_probe(int dtype, int random, long long iters, int n_waves, float* out,
                             hipStream_t st);

}  // namespace swsft
