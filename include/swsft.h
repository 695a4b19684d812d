/*
 * swsft.h — C ABI of the MI355X (gfx950) spectral spin-weighted spherical
 * convolution library.
 *
 * The layer (Esteves, Slotine, Makadia, "Scaling Spherical CNNs", ICML 2023)
 * is: forward spin-weighted spherical Fourier transform (Background, eq. (2)),
 * per-degree mixing of spins and channels by filters shared across the order
 * m (Background, "Spherical CNNs": convolution as products of spin-weighted
 * harmonic coefficients; Fig. 2, "*K"), inverse transform (eq. (3)).  The
 * phase-collapse nonlinearity of the Method section ("Phase collapse
 * nonlinearity") is provided for stacking layers.
 *
 * Conventions shared by every call
 * --------------------------------
 *  Grid       H x W equiangular, H == W, H even: colatitude
 *             theta_j = pi (2j+1) / (2H), longitude phi_k = 2 pi k / W.
 *             Quadrature: Driscoll--Healy weights on that grid.
 *  Bandlimit  degrees 0 <= l < L, 1 <= L <= H/2; orders |m| <= l.
 *  Harmonics  sY_lm(theta, phi) = (-1)^s sqrt((2l+1)/(4 pi)) d^l_{m,-s}(theta)
 *             e^{i m phi}, with d^1_{10}(b) = -sin(b)/sqrt(2).  This is the
 *             convention in which the paper's eqs. (4) and (6) hold.
 *  Complex    every complex array is interleaved (re, im) pairs of the plan's
 *             storage type: float for SWSFT_F32, bfloat16 for SWSFT_BF16.
 *  Layouts    (all C-contiguous, device memory)
 *    spatial       x, y     [B][S][C][H][W]       complex
 *    coefficients  coef     [L*L][B][S][C]        complex, row l*l + l + m;
 *                  rows with l < |s| are written as 0 and ignored on input
 *    filters       K        [L][S_out][C_out][S_in][C_in]   complex;
 *                  output spin/channel first, like a dense-layer weight;
 *                  entries with l < max(|s_in|, |s_out|) are ignored;
 *                  S_out C_out S_in C_in <= 2^30 (one degree's block),
 *                  else SWSFT_E_UNSUPPORTED
 *  Sizes      1 <= B <= 65535, 1 <= C <= 2^20 and B C <= 2^26 for every
 *             channel count C (SWSFT_E_INVALID otherwise)
 *  S is the number of spins of the side concerned; spins are the plan's
 *  spins_in (forward transform, conv input) or spins_out (inverse transform,
 *  conv output, phase collapse), in the order given to swsft_plan_create.
 *
 * Ownership and streams
 *  The plan owns its device tables (allocated by swsft_plan_create on the
 *  current device, freed by swsft_plan_destroy).  The caller owns every
 *  per-call buffer, including a workspace of at least swsft_workspace_bytes.
 *  Calls never allocate, never synchronize and enqueue all work on `stream`
 *  (a hipStream_t; NULL is the null stream) of the plan's device; results are
 *  ready when the stream reaches them.  A plan is immutable after creation
 *  (apart from the stage-timing record, see swsft_stage_timing); calls on
 *  different streams may run concurrently if their workspaces and outputs
 *  are distinct.
 *
 * Errors
 *  Every call validates its arguments on the host before enqueuing
 *  anything; on SWSFT_E_INVALID / SWSFT_E_WORKSPACE / SWSFT_E_UNSUPPORTED
 *  nothing was enqueued.  SWSFT_E_HIP reports a failed HIP call (text in
 *  swsft_last_error()).  Nothing aborts and no C++ exception crosses the ABI.
 */
#ifndef SWSFT_H
#define SWSFT_H

#include <stddef.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct swsft_plan_s* swsft_plan;

typedef enum {
  SWSFT_OK = 0,
  SWSFT_E_INVALID = 1,     /* bad argument; nothing enqueued                  */
  SWSFT_E_UNSUPPORTED = 2, /* valid in the paper's terms, not implemented here */
  SWSFT_E_ALLOC = 3,       /* device allocation failed in swsft_plan_create   */
  SWSFT_E_HIP = 4,         /* a HIP call failed                               */
  SWSFT_E_WORKSPACE = 5    /* workspace NULL or smaller than required         */
} swsft_status;

typedef enum {
  SWSFT_F32 = 0,  /* float storage, float accumulation                   */
  SWSFT_BF16 = 1  /* bfloat16 storage, float accumulation (MFMA bf16)    */
} swsft_dtype;

/* Plan creation flags (swsft_plan_create_ex). */
typedef enum {
  /* Forward and inverse longitude stages as dense DFT matrix products on
   * MFMA (the route the paper takes on TPUs: Method, "Efficient TPU
   * implementation"; appendix "FFT vs DFT", Table 8) instead of the register
   * FFT.  Also admits widths the FFT does not take: any even W (H <= 32 or a
   * multiple of 32), e.g. 96 or 768.  The plan then also holds the two
   * expanded DFT matrices. */
  SWSFT_PLAN_DFT_MATMUL = 1,
  /* Latitude stages by the paper's Wigner-Delta route (Background, eqs.
   * (4)-(6)): a Fourier sum in theta on the grid (quadrature weights folded
   * in) followed by the Delta^l_{m'm} Delta^l_{m'(-s)} contraction, both as
   * MFMA GEMMs, for swsft_forward, swsft_inverse and spin_sph_conv_forward.
   * DELTA sums all m' in [-l, l] (eq. (4), eq. (6) for every G_{m'm});
   * DELTA_SYM uses the J / G symmetries (eq. (5): m' >= 0 only).  Needs L a
   * multiple of 32; not with the backward pass or the residual block. */
  SWSFT_PLAN_DELTA = 2,
  SWSFT_PLAN_DELTA_SYM = 4
} swsft_plan_flags;

typedef enum {
  SWSFT_OP_FORWARD = 0, /* swsft_forward          */
  SWSFT_OP_INVERSE = 1, /* swsft_inverse          */
  SWSFT_OP_CONV = 2,    /* spin_sph_conv_forward  */
  SWSFT_OP_CONV_BACKWARD = 3, /* spin_sph_conv_backward */
  SWSFT_OP_BATCH_NORM = 4     /* spin_sph_spectral_batch_norm (C_out = C, C_in ignored) */
} swsft_op;

/*
 * Create a plan for H x W grids with bandlimit L (Background, eqs. (2)-(3)).
 *  H, W        grid size; H == W (the transform needs equal sample counts on
 *              both axes, appendix "WeatherBench"), H even.  Implemented:
 *              W a power of two in [2, 512] (with SWSFT_PLAN_DFT_MATMUL
 *              any even W up to 32 or multiple of 32); other sizes return
 *              SWSFT_E_UNSUPPORTED.
 *  L           bandlimit, 1 <= L <= H/2 (L < H/2 is spectral pooling:
 *              Method, "Spectral pooling").
 *  spins_in    host array of n_spins_in distinct spins, |s| < L, 1..8 of them.
 *  spins_out   host array of n_spins_out distinct spins, |s| < L, 1..8.
 *  dtype       a swsft_dtype.
 *  out         receives the plan (unchanged on error).
 * Builds, on the current device, the Wigner-d tables of every spin in float64
 * (recursion in l) rounded once to the storage type, and the DFT twiddles.
 * Synchronizes the device before returning.
 */
swsft_status swsft_plan_create(int H, int W, int L, const int* spins_in, int n_spins_in,
                               const int* spins_out, int n_spins_out, int dtype,
                               swsft_plan* out);

/* swsft_plan_create with creation flags (swsft_plan_flags; 0 is
 * swsft_plan_create).  With SWSFT_PLAN_DFT_MATMUL the plan also holds the
 * expanded forward and inverse DFT matrices, [2(2L-1)][2W] and
 * [2W][2(2L-1)] reals of the storage type. */
swsft_status swsft_plan_create_ex(int H, int W, int L, const int* spins_in, int n_spins_in,
                                  const int* spins_out, int n_spins_out, int dtype,
                                  unsigned flags, swsft_plan* out);

/* Free the plan's device tables.  NULL-safe.  The caller must make sure no
 * enqueued call still uses the plan. */
void swsft_plan_destroy(swsft_plan p);

/* Workspace bytes needed by one call of `op` (a swsft_op) with batch B and
 * channel counts C_in, C_out (C_out is ignored for SWSFT_OP_FORWARD, C_in
 * for SWSFT_OP_INVERSE).  Returns 0 for invalid arguments. */
size_t swsft_workspace_bytes(swsft_plan p, int op, int B, int C_in, int C_out);

/*
 * Forward transform, eq. (2), of every (b, s, c) map on spins_in:
 *  coef[l*l+l+m][b][s][c] = int f conj(sY_lm) dx, by Driscoll--Healy
 *  quadrature (exact for fields band-limited to l < L).
 *  x     [B][S_in][C][H][W] complex, read only.
 *  coef  [L*L][B][S_in][C] complex, written (rows l < |s| set to 0).
 *  ws    workspace of ws_bytes >= swsft_workspace_bytes(p, SWSFT_OP_FORWARD, B, C, 0).
 *  coef and ws must not overlap each other or x (SWSFT_E_INVALID).
 */
swsft_status swsft_forward(swsft_plan p, int B, int C, const void* x, void* coef, void* ws,
                           size_t ws_bytes, void* stream);

/*
 * Inverse transform, eq. (3), on spins_out:
 *  y[b][s][c](theta_j, phi_k) = sum_{l>=|s|} sum_{|m|<=l} coef[l*l+l+m][b][s][c] sY_lm.
 *  coef  [L*L][B][S_out][C] complex, read only (rows l < |s| ignored).
 *  y     [B][S_out][C][H][W] complex, written.
 *  ws    workspace of ws_bytes >= swsft_workspace_bytes(p, SWSFT_OP_INVERSE, B, 0, C).
 *  y and ws must not overlap each other or coef (SWSFT_E_INVALID).
 */
swsft_status swsft_inverse(swsft_plan p, int B, int C, const void* coef, void* y, void* ws,
                           size_t ws_bytes, void* stream);

/*
 * The spectral spin-weighted spherical convolution layer (Background,
 * "Spherical CNNs"; Fig. 2's FT -> *K -> IFT):
 *  a  = forward(x)                                   on spins_in
 *  a'[l*l+l+m][b][t][c'] = sum_{s: |s|<=l} sum_c K[l][t][c'][s][c] a[l*l+l+m][b][s][c]
 *                          for |t| <= l (else 0)
 *  y  = inverse(a')                                  on spins_out
 *  x        [B][S_in][C_in][H][W] complex, read only.
 *  filters  [L][S_out][C_out][S_in][C_in] complex, read only.
 *  y        [B][S_out][C_out][H][W] complex, written.
 *  ws       workspace of ws_bytes >= swsft_workspace_bytes(p, SWSFT_OP_CONV, B, C_in, C_out).
 *  y and ws must not overlap each other, x or filters (SWSFT_E_INVALID).
 */
swsft_status spin_sph_conv_forward(swsft_plan p, int B, int C_in, int C_out, const void* x,
                                   const void* filters, void* y, void* ws, size_t ws_bytes,
                                   void* stream);

/*
 * Backward pass of spin_sph_conv_forward: the gradients that training needs.
 * For a real loss L with output gradient grad_y = dL/dy in the convention
 * dL = Re sum conj(grad_y) dy (the convention of torch's complex autograd),
 * the layer y = G(K F x) -- F the quadrature analysis of eq. (2), K the
 * per-degree mixing, G the synthesis of eq. (3), all linear -- has
 *   grad_x       = F^H (K^H (G^H grad_y)),
 *   grad_filters[l][t][c'][s][c] = sum_{|m|<=l, b} g[l*l+l+m][b][t][c'] conj(a[l*l+l+m][b][s][c]),
 * with g = G^H grad_y (the analysis sum of eq. (2) without quadrature
 * weights), a = F x, and zeros where |s| > l or |t| > l.  F^H is the
 * synthesis of eq. (3) weighted by (2 pi / W) w_j; K^H applies conj(K).
 *  x             [B][S_in][C_in][H][W] complex; read when grad_filters != NULL
 *                and coef_x is NULL.
 *  coef_x        [L*L][B][S_in][C_in] complex, the input's coefficients F x as
 *                saved by spin_sph_conv_forward_train (or swsft_forward), or
 *                NULL to compute them from x (one more forward transform).
 *  filters       [L][S_out][C_out][S_in][C_in] complex; read when grad_x != NULL.
 *  grad_y        [B][S_out][C_out][H][W] complex, read only.
 *  grad_x        [B][S_in][C_in][H][W] complex, written; NULL: not computed.
 *  grad_filters  [L][S_out][C_out][S_in][C_in] complex, written; NULL: not computed.
 *  At least one output must be requested.  Outputs and the workspace must not
 *  overlap each other or an input that is read; an input that no requested output needs
 *  (x for grad_x alone, filters for grad_filters alone) may be NULL.
 *  Returns SWSFT_E_INVALID / SWSFT_E_WORKSPACE on bad arguments before any
 *  launch, SWSFT_E_HIP if a launch fails.  Results are deterministic: no
 *  atomics; where the filter-gradient contraction over (m, b) is split across
 *  workgroups, the partial sums (kept in the workspace) are added in a fixed
 *  order, so repeated calls are bit-identical.
 *  ws  workspace of ws_bytes >= swsft_workspace_bytes(p, SWSFT_OP_CONV_BACKWARD, B, C_in, C_out).
 */
swsft_status spin_sph_conv_backward(swsft_plan p, int B, int C_in, int C_out, const void* x,
                                    const void* coef_x, const void* filters, const void* grad_y,
                                    void* grad_x, void* grad_filters, void* ws, size_t ws_bytes,
                                    void* stream);

/*
 * spin_sph_conv_forward without a caller workspace, for callers that cannot
 * allocate device memory (code under graph capture, tight serving loops,
 * harnesses that forbid hipMalloc).  The workspace is a static array of
 * 128 MiB that the library holds on every device it runs on until the
 * process ends; its device address is looked up when a plan is created on
 * that device, and this call allocates, frees and synchronizes nothing.
 *  x, filters, y   as for spin_sph_conv_forward (y must not overlap x).
 * Returns SWSFT_E_UNSUPPORTED, with nothing enqueued, when the layer needs
 * more than 128 MiB of workspace (swsft_workspace_bytes(p, SWSFT_OP_CONV, B,
 * C_in, C_out) > 134217728; e.g. the 256 x 256, C = 256, B = 2 layer).
 * Every call on a device shares that device's array: calls that may overlap
 * in time on one device (other streams, other threads) race and must be
 * serialized by the caller.  The array keeps the last call's contents; the
 * layer reads nothing of it that the same call has not written.
 */
swsft_status spin_sph_conv_forward_noalloc(swsft_plan p, int B, int C_in, int C_out,
                                           const void* x, const void* filters, void* y,
                                           void* stream);

/*
 * spin_sph_conv_forward that also writes the input's coefficients F x
 * (eq. (2); [L*L][B][S_in][C_in] complex, the layout of swsft_forward) to
 * coef_x, for the backward pass to reuse: training saves them instead of
 * transforming x again.  Same workspace as spin_sph_conv_forward; coef_x must
 * not overlap any other argument.
 */
swsft_status spin_sph_conv_forward_train(swsft_plan p, int B, int C_in, int C_out, const void* x,
                                         const void* filters, void* y, void* coef_x, void* ws,
                                         size_t ws_bytes, void* stream);

/*
 * Phase-collapse nonlinearity (Method, "Phase collapse nonlinearity") on a
 * spatial feature map with the plan's spins_out, which must contain spin 0:
 * at every grid point, x0 <- W1 x0 + W2 |x| + b, where x0 are the C spin-0
 * channels and |x| the moduli of all S_out*C channels stacked in (spin,
 * channel) order; channels of other spins are passed through unchanged.
 *  x     [B][S_out][C][H][W] complex (storage type), read only.
 *  W1    [C][C] complex float (interleaved), row = output channel.
 *  W2    [C][S_out*C] complex float, row = output channel.
 *  bias  [C] complex float.
 *  y     [B][S_out][C][H][W] complex, written; y == x (in place) is allowed,
 *        any other overlap is not.
 *  W1, W2 and bias must be 8-byte aligned, x and y 16-byte aligned.
 * Returns SWSFT_E_INVALID if spin 0 is not in spins_out, SWSFT_E_UNSUPPORTED
 * if C exceeds the channel count whose staging fits one CU's LDS for S_out
 * spins (160 for two spins).
 */
swsft_status spin_sph_phase_collapse(swsft_plan p, int B, int C, const void* x,
                                     const void* W1, const void* W2, const void* bias,
                                     void* y, void* stream);

/*
 * The per-degree mixing alone (Background, "Spherical CNNs": convolution as
 * products of coefficients, filters shared across m; Fig. 2 "*K"):
 *   coef_out[l*l+l+m][b][t][c'] = sum_{s, |s| <= l} sum_c K[l][t][c'][s][c] coef[l*l+l+m][b][s][c]
 * for |t| <= l, else 0.
 *  coef      [L*L][B][S_in][C_in] complex, read only.
 *  filters   [L][S_out][C_out][S_in][C_in] complex, read only.
 *  coef_out  [L*L][B][S_out][C_out] complex, written; must not overlap the inputs.
 * Needs no workspace.
 */
swsft_status spin_sph_mix(swsft_plan p, int B, int C_in, int C_out, const void* coef,
                          const void* filters, void* coef_out, void* stream);

/*
 * Spectral batch normalization (Method, "Spectral batch normalization") of
 * coefficients of the plan's output spins.  The l = 0 coefficient is the
 * function's mean times sqrt(4 pi), and by Parseval the remaining ones carry
 * its variance over the sphere, so per (spin s, channel c):
 *   var[s][c] = (1 / (4 pi B)) sum_b sum_{l >= 1} sum_m |coef|^2    (batch statistics)
 *   out = gamma[s][c] coef / sqrt(var[s][c] + eps)                   for l >= 1
 *   out[0][b][s0][c] = beta[c] (spin 0), 0 for the other spins       for l = 0
 *   out += skip                                                      (if skip != NULL)
 *  coef     [L*L][B][S_out][C] complex (storage type).
 *  gamma    [S_out][C] float, device.  beta: [C] complex float, device, or NULL (0).
 *  eps      >= 0, added under the square root.
 *  var_in   [S_out][C] float (device) to normalise with given statistics (e.g.
 *           running averages at inference), or NULL for batch statistics.
 *  var_out  [S_out][C] float (device) receiving the variance used, or NULL.
 *  skip     [L*L][B][S_out][C] complex added after normalising (the Fourier-
 *           space residual connection of Fig. 2), or NULL.
 *  out      [L*L][B][S_out][C] complex; out == coef and out == skip are allowed.
 *  ws       >= swsft_workspace_bytes(p, SWSFT_OP_BATCH_NORM, B, 1, C) bytes.
 * The statistics are summed in float32 in a fixed order (deterministic).
 * S_out * C above 2048 returns SWSFT_E_UNSUPPORTED.
 */
swsft_status spin_sph_spectral_batch_norm(swsft_plan p, int B, int C, const void* coef,
                                          const float* gamma, const void* beta, float eps,
                                          const float* var_in, float* var_out, const void* skip,
                                          void* out, void* ws, size_t ws_bytes, void* stream);

/*
 * Parameters of the residual block; every pointer is device memory.
 *  K1, K2          [L][S][C][S][C] complex filters in the plans' storage type.
 *  gamma1, gamma2  [S][C] float; beta1, beta2 [C] complex float or NULL.
 *  pc*_W1 [C][C], pc*_W2 [C][S*C], pc*_b [C]: complex float phase-collapse parameters.
 *  eps             batch-norm epsilon (>= 0).
 *  var1_out, var2_out  [S][C] float receiving the batch variances, or NULL.
 */
typedef struct swsft_block_params {
  const void* K1;
  const void* K2;
  const float* gamma1;
  const void* beta1;
  const float* gamma2;
  const void* beta2;
  const void* pc1_W1;
  const void* pc1_W2;
  const void* pc1_b;
  const void* pc2_W1;
  const void* pc2_W2;
  const void* pc2_b;
  float eps;
  float* var1_out;
  float* var2_out;
} swsft_block_params;

/* Workspace bytes of spin_sph_residual_block_forward (0 for invalid arguments). */
size_t swsft_block_workspace_bytes(swsft_plan p_in, swsft_plan p_out, int B, int C);

/*
 * The residual block of Fig. 2 (Method, "Spectral pooling and efficient
 * residual block"), with the skip connection between Fourier coefficients:
 *   a = FT(x)                                   with p_in (grid H_in, bandlimit L)
 *   z = PC1(IFT(BN1(K1 * a)))                   with p_out (grid H_out)
 *   y = PC2(IFT(BN2(K2 * FT(z)) + a))
 * FT / IFT are swsft_forward / swsft_inverse, K * the per-degree mixing, BN
 * the spectral batch norm with batch statistics, PC the phase collapse.
 * Spectral pooling: L < H_in / 2 skips the coefficients of degree >= L in
 * the first transform, and H_out = 2 L puts the output on the coarser grid;
 * H_out = H_in is the block without pooling.
 *  p_in, p_out  plans with the same device, dtype, bandlimit L, and the same
 *               spin list S (containing 0) as both spins_in and spins_out.
 *  x   [B][S][C][H_in][W_in] complex, read only.
 *  y   [B][S][C][H_out][W_out] complex, written; must not overlap x.
 *  ws  >= swsft_block_workspace_bytes(p_in, p_out, B, C) bytes.
 * Stage timing, if enabled, is recorded on p_out.  Channel limits: those of
 * the phase collapse and of the batch norm (S * C <= 2048).
 */
swsft_status spin_sph_residual_block_forward(swsft_plan p_in, swsft_plan p_out, int B, int C,
                                             const void* x, const swsft_block_params* params,
                                             void* y, void* ws, size_t ws_bytes, void* stream);

/* Static text for a status code. */
const char* swsft_status_string(int status);

/* Detail of the last non-OK status returned on this thread ("" if none). */
const char* swsft_last_error(void);

/*
 * Stage timing for measurement.  When enabled on a plan, each kernel launch
 * of the calls above is bracketed by HIP events recorded on the call's
 * stream.  swsft_stage_times synchronizes those events, adds each stage's
 * elapsed milliseconds and launch count into ms[i] and launches[i] for
 * i < n (stage i is named by swsft_stage_name(i)), clears the record and
 * returns the number of stages.  Disabled by default; enabling costs two
 * event records per launch.  At most 4096 launches are recorded between
 * reads; later ones are not timed.  The record is shared by every call on
 * the plan: while timing is enabled, each launch and each read-out takes one
 * library-wide lock, so calls from several threads stay correct (and are
 * serialised launch by launch); a plan without timing takes no lock.
 */
swsft_status swsft_stage_timing(swsft_plan p, int enable);
int swsft_stage_times(swsft_plan p, double* ms, long long* launches, int n);
const char* swsft_stage_name(int stage);

/*
 * Copy a plan table to host memory (synchronous; for tests).
 *  which 0: forward table, [2L-1][L][Hp] per spins_in entry `spin_index`:
 *           (2 pi / W) w_j (-1)^s sqrt((2l+1)/(4 pi)) d^l_{m,-s}(theta_j),
 *           row (m + L - 1, l), zero for l < max(|m|, |s|), Hp = H rounded
 *           up to a multiple of 8 (padding columns are 0).
 *  which 1: inverse table, [2L-1][H][Lp] per spins_out entry:
 *           (-1)^s sqrt((2l+1)/(4 pi)) d^l_{m,-s}(theta_j), Lp = L rounded
 *           up to a multiple of 32 (padding columns are 0).
 *  which 2: backward synthesis table, [2L-1][H][Lp] per spins_in entry: the
 *           values of table 0 in the layout of table 1.
 *  which 3: backward analysis table, [2L-1][L][Hp] per spins_out entry: the
 *           values of table 1 in the layout of table 0.
 *  Elements are of the plan's storage type.  `bytes` must equal the table
 *  size; returns SWSFT_E_INVALID otherwise.
 */
swsft_status swsft_plan_table(swsft_plan p, int which, int spin_index, void* host_dst,
                              size_t bytes);

/*
 * Measurement helper, not part of the transform: enqueue on `stream` one
 * kernel in which n_waves waves (a multiple of 4, 4 <= n_waves <= 2^20) each
 * run `iters` (1 <= iters <= 2^24) rounds of four independent MFMAs with
 * both operands held in registers and no memory traffic:
 * v_mfma_f32_32x32x16_bf16 for dtype SWSFT_BF16, v_mfma_f32_32x32x2f32 for
 * SWSFT_F32.  random_operands != 0 fills the operand registers with values
 * of random sign and mantissa in [0.5, 2), 0 with ones (the chip's clock
 * depends on the switching activity, so the two rates differ).  `out`
 * (device, 64 n_waves floats, caller-owned) receives one checksum per lane.
 * *flops_out (host, may be NULL) receives the MFMA flops the kernel issues:
 * n_waves iters (4 x 2 x 32 x 32 x 16) for bf16, (4 x 2 x 32 x 32 x 2) for
 * f32.  The caller times the kernel on its stream (e.g. with events) to get
 * the sustained rate against which the contraction kernels are quoted.
 */
swsft_status swsft_probe_mfma(int dtype, int random_operands, long long iters, int n_waves,
                              float* out, double* flops_out, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* SWSFT_H */
