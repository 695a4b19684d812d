// C ABI: argument validation, plan ownership, workspace layout and the
// sequence of kernel launches of each call.  Every call checks its
// arguments on the host before it touches HIP; on an error nothing is
// enqueued.
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <initializer_list>
#include <map>
#include <mutex>
#include <new>
#include <utility>

#include "swsft_internal.h"

struct swsft_plan_s : swsft::Plan {};

namespace {

using swsft::Plan;

thread_local char g_last_error[512] = "";

swsft_status fail(swsft_status st, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_last_error, sizeof(g_last_error), fmt, ap);
  va_end(ap);
  return st;
}

swsft_status hip_fail(hipError_t e, const char* what) {
  return fail(SWSFT_E_HIP, "%s: %s", what, hipGetErrorString(e));
}

bool is_pow2(int v) { return v > 0 && (v & (v - 1)) == 0; }

constexpr size_t kAlign = 256;
size_t align_up(size_t v) { return (v + kAlign - 1) / kAlign * kAlign; }

swsft_status check_spins(const int* s, int n, int L, const char* which) {
  if (s == nullptr) return fail(SWSFT_E_INVALID, "%s is NULL", which);
  if (n < 1 || n > swsft::kMaxSpins)
    return fail(SWSFT_E_INVALID, "%s: count %d not in [1, %d]", which, n, swsft::kMaxSpins);
  for (int i = 0; i < n; ++i) {
    if (s[i] <= -L || s[i] >= L)
      return fail(SWSFT_E_INVALID, "%s[%d] = %d: need |s| < L = %d", which, i, s[i], L);
    for (int j = 0; j < i; ++j)
      if (s[j] == s[i]) return fail(SWSFT_E_INVALID, "%s: spin %d repeated", which, s[i]);
  }
  return SWSFT_OK;
}

// Batch and channel bounds keep every index computed in 32 bits inside the
// kernels (n' = 2 B C, rows (2l+1) B, grid dimensions) in range.
swsft_status check_bc(int B, int C, const char* cname) {
  if (B < 1 || B > 65535) return fail(SWSFT_E_INVALID, "B = %d not in [1, 65535]", B);
  if (C < 1 || C > (1 << 20)) return fail(SWSFT_E_INVALID, "%s = %d not in [1, 2^20]", cname, C);
  if ((long long)B * C > (1LL << 26))
    return fail(SWSFT_E_INVALID, "B * %s = %lld exceeds 2^26", cname, (long long)B * C);
  return SWSFT_OK;
}

// One degree's filter block, S_out C_out x S_in C_in complex values, is
// indexed with 32-bit integers inside the kernels.
swsft_status check_filter_block(const Plan& p, int C_in, int C_out) {
  const long long n = (long long)p.n_out * C_out * p.n_in * C_in;
  if (n > (1LL << 30))
    return fail(SWSFT_E_UNSUPPORTED,
                "S_out * C_out * S_in * C_in = %lld exceeds 2^30 filter entries per degree", n);
  return SWSFT_OK;
}

bool overlaps(const void* a, size_t na, const void* b, size_t nb) {
  const char *pa = static_cast<const char*>(a), *pb = static_cast<const char*>(b);
  return pa != nullptr && pb != nullptr && pa < pb + nb && pb < pa + na;
}

// A buffer of a call: written by the call (outputs and the workspace) or
// only read.  Buffers that are both read need not be disjoint; a written
// buffer must not overlap any other buffer of the call.
struct Region {
  const void* ptr;
  size_t bytes;
  const char* name;
  bool written;
};

swsft_status check_disjoint(std::initializer_list<Region> rs) {
  for (auto a = rs.begin(); a != rs.end(); ++a)
    for (auto b = a + 1; b != rs.end(); ++b)
      if ((a->written || b->written) && overlaps(a->ptr, a->bytes, b->ptr, b->bytes))
        return fail(SWSFT_E_INVALID, "%s and %s overlap", a->name, b->name);
  return SWSFT_OK;
}

size_t filter_elems(const Plan& p, int Cin, int Cout) {
  return (size_t)p.L * p.n_out * Cout * p.n_in * Cin * 2;
}

// Bytes of a [B][S][C][H][W] complex field of the storage type.
size_t spatial_bytes(const Plan& p, int S, int B, int C) {
  return (size_t)B * S * C * p.H * p.W * 2 * p.elem;
}

size_t ws_need(const Plan& p, int op, int B, int Cin, int Cout) {
  const size_t e = p.elem;
  switch (op) {
    case SWSFT_OP_FORWARD:
      return align_up(swsft::xy_elems(p, p.n_in, B, Cin) * e) +
             align_up(swsft::delta_elems(p, p.n_in, B, Cin) * e);
    case SWSFT_OP_INVERSE:
      return align_up(swsft::xy_elems(p, p.n_out, B, Cout) * e) +
             align_up(swsft::delta_elems(p, p.n_out, B, Cout) * e);
    case SWSFT_OP_CONV: {
      size_t xin = swsft::xy_elems(p, p.n_in, B, Cin), xout = swsft::xy_elems(p, p.n_out, B, Cout);
      size_t din = swsft::delta_elems(p, p.n_in, B, Cin), dout = swsft::delta_elems(p, p.n_out, B, Cout);
      return align_up((xin > xout ? xin : xout) * e) +
             align_up(swsft::coef_elems(p, p.n_in, B, Cin) * e) +
             align_up(swsft::coef_elems(p, p.n_out, B, Cout) * e) +
             align_up((din > dout ? din : dout) * e);
    }
    case SWSFT_OP_CONV_BACKWARD: {
      size_t xin = swsft::xy_elems(p, p.n_in, B, Cin), xout = swsft::xy_elems(p, p.n_out, B, Cout);
      return align_up((xin > xout ? xin : xout) * e) +
             2 * align_up(swsft::coef_elems(p, p.n_in, B, Cin) * e) +
             align_up(swsft::coef_elems(p, p.n_out, B, Cout) * e) +
             align_up(filter_elems(p, Cin, Cout) * e) +
             align_up(swsft::filter_grad_split_bytes(p, B, Cin, Cout));
    }
    case SWSFT_OP_BATCH_NORM:
      return align_up(swsft::bn_workspace_bytes(p, B, Cout));
    default:
      return 0;
  }
}

swsft_status check_ws(const Plan& p, int op, int B, int Cin, int Cout, const void* ws,
                      size_t ws_bytes) {
  const size_t need = ws_need(p, op, B, Cin, Cout);
  if (ws == nullptr || ws_bytes < need)
    return fail(SWSFT_E_WORKSPACE, "workspace %s: %zu bytes given, %zu needed",
                ws == nullptr ? "NULL" : "too small", ws == nullptr ? (size_t)0 : ws_bytes,
                need);
  if (reinterpret_cast<uintptr_t>(ws) % 16 != 0)
    return fail(SWSFT_E_INVALID, "workspace must be 16-byte aligned");
  return SWSFT_OK;
}

swsft_status check_ptr(const void* ptr, const char* name) {
  if (ptr == nullptr) return fail(SWSFT_E_INVALID, "%s is NULL", name);
  if (reinterpret_cast<uintptr_t>(ptr) % 16 != 0)
    return fail(SWSFT_E_INVALID, "%s must be 16-byte aligned", name);
  return SWSFT_OK;
}

}  // namespace

namespace swsft {
hipError_t ensure_dynamic_lds(const void* kern, size_t bytes) {
  if (bytes <= 64 * 1024) return hipSuccess;
  static std::mutex mu;
  static std::map<std::pair<int, const void*>, size_t> done;
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  std::lock_guard<std::mutex> lock(mu);
  size_t& have = done[{dev, kern}];
  if (have >= bytes) return hipSuccess;
  e = hipFuncSetAttribute(kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)bytes);
  if (e == hipSuccess) have = bytes;
  return e;
}
}  // namespace swsft

namespace {

swsft_status check_inverse_stage(const Plan& p) {
  if (!p.fft_ok && !(p.flags & SWSFT_PLAN_DFT_MATMUL))
    return fail(SWSFT_E_UNSUPPORTED, "W = %d: the inverse longitude stage needs a power of two <= 512",
                p.W);
  return SWSFT_OK;
}

swsft_status check_device(const Plan& p) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  if (dev != p.device)
    return fail(SWSFT_E_INVALID, "plan belongs to device %d, current device is %d", p.device, dev);
  return SWSFT_OK;
}

// Stage timing appends to the plan's event record; calls on a timing-enabled
// plan from several threads take this lock for every launch (and
// swsft_stage_times for the read-out), so the record stays consistent.  A
// plan without timing takes no lock.
std::mutex g_timing_mu;

// Launch one stage, bracketed by timing events when enabled.
template <class F>
swsft_status run_stage(Plan& p, int stage, hipStream_t st, const char* name, F&& launch) {
  std::unique_lock<std::mutex> lock(g_timing_mu, std::defer_lock);
  if (p.timing) lock.lock();
  const bool timed = p.timing && p.ev != nullptr && p.n_timed < swsft::kMaxTimedLaunches;
  if (timed) {
    hipError_t e = hipEventRecord(p.ev[2 * p.n_timed], st);
    if (e != hipSuccess) return hip_fail(e, "hipEventRecord");
  }
  hipError_t e = launch();
  if (e != hipSuccess) return hip_fail(e, name);
  if (timed) {
    e = hipEventRecord(p.ev[2 * p.n_timed + 1], st);
    if (e != hipSuccess) return hip_fail(e, "hipEventRecord");
    p.ev_stage[p.n_timed] = stage;
    ++p.n_timed;
  }
  return SWSFT_OK;
}

#define SWSFT_TRY(expr)                  \
  do {                                   \
    swsft_status _st = (expr);           \
    if (_st != SWSFT_OK) return _st;     \
  } while (0)

void free_plan(Plan* p) {
  if (p == nullptr) return;
  if (p->tab_fwd) (void)hipFree(p->tab_fwd);
  if (p->tab_inv) (void)hipFree(p->tab_inv);
  if (p->tab_bwd_syn) (void)hipFree(p->tab_bwd_syn);
  if (p->tab_bwd_ana) (void)hipFree(p->tab_bwd_ana);
  if (p->dft_mat) (void)hipFree(p->dft_mat);
  if (p->dft_mat_inv) (void)hipFree(p->dft_mat_inv);
  if (p->delta_theta_fwd) (void)hipFree(p->delta_theta_fwd);
  if (p->delta_theta_inv) (void)hipFree(p->delta_theta_inv);
  if (p->delta_fwd) (void)hipFree(p->delta_fwd);
  if (p->delta_inv) (void)hipFree(p->delta_inv);
  if (p->twiddle) (void)hipFree(p->twiddle);
  if (p->ev) {
    for (int i = 0; i < 2 * swsft::kMaxTimedLaunches; ++i)
      if (p->ev[i]) (void)hipEventDestroy(p->ev[i]);
    std::free(p->ev);
  }
  std::free(p->ev_stage);
}

}  // namespace

extern "C" {

const char* swsft_status_string(int status) {
  switch (status) {
    case SWSFT_OK: return "SWSFT_OK";
    case SWSFT_E_INVALID: return "SWSFT_E_INVALID: invalid argument";
    case SWSFT_E_UNSUPPORTED: return "SWSFT_E_UNSUPPORTED: not implemented for these sizes";
    case SWSFT_E_ALLOC: return "SWSFT_E_ALLOC: device allocation failed";
    case SWSFT_E_HIP: return "SWSFT_E_HIP: HIP call failed";
    case SWSFT_E_WORKSPACE: return "SWSFT_E_WORKSPACE: workspace missing or too small";
    default: return "unknown swsft status";
  }
}

const char* swsft_last_error(void) { return g_last_error; }

const char* swsft_stage_name(int stage) {
  static const char* names[swsft::kNumStages] = {"dft_fwd", "lat_fwd", "mix", "lat_inv",
                                                 "dft_inv", "phase_collapse", "tables",
                                                 "filter_grad", "filter_adjoint", "batch_norm",
                                                 "delta_theta", "small_fwd", "small_inv"};
  if (stage < 0 || stage >= swsft::kNumStages) return "";
  return names[stage];
}

swsft_status swsft_plan_create(int H, int W, int L, const int* spins_in, int n_spins_in,
                               const int* spins_out, int n_spins_out, int dtype,
                               swsft_plan* out) {
  return swsft_plan_create_ex(H, W, L, spins_in, n_spins_in, spins_out, n_spins_out, dtype, 0u,
                              out);
}

swsft_status swsft_plan_create_ex(int H, int W, int L, const int* spins_in, int n_spins_in,
                                  const int* spins_out, int n_spins_out, int dtype,
                                  unsigned flags, swsft_plan* out) {
  g_last_error[0] = 0;
  if (out == nullptr) return fail(SWSFT_E_INVALID, "out is NULL");
  if (H != W) return fail(SWSFT_E_INVALID, "H = %d != W = %d (square grids only)", H, W);
  if (H < 2 || H % 2) return fail(SWSFT_E_INVALID, "H = %d must be even and >= 2", H);
  if (L < 1 || L > H / 2) return fail(SWSFT_E_INVALID, "L = %d not in [1, H/2 = %d]", L, H / 2);
  if (dtype != SWSFT_F32 && dtype != SWSFT_BF16)
    return fail(SWSFT_E_INVALID, "dtype %d is not a swsft_dtype", dtype);
  SWSFT_TRY(check_spins(spins_in, n_spins_in, L, "spins_in"));
  SWSFT_TRY(check_spins(spins_out, n_spins_out, L, "spins_out"));
  const unsigned known = SWSFT_PLAN_DFT_MATMUL | SWSFT_PLAN_DELTA | SWSFT_PLAN_DELTA_SYM;
  if (flags & ~known) return fail(SWSFT_E_INVALID, "unknown flags %#x", flags);
  if ((flags & SWSFT_PLAN_DELTA) && (flags & SWSFT_PLAN_DELTA_SYM))
    return fail(SWSFT_E_INVALID, "SWSFT_PLAN_DELTA and SWSFT_PLAN_DELTA_SYM exclude each other");
  if ((flags & (SWSFT_PLAN_DELTA | SWSFT_PLAN_DELTA_SYM)) && (L % 32 != 0 || H % 32 != 0))
    return fail(SWSFT_E_UNSUPPORTED, "the Delta route needs L and H multiples of 32 (L = %d)", L);
  const bool fft_ok = is_pow2(W) && W <= 512;
  if (H > 32 && H % 32 != 0)
    return fail(SWSFT_E_UNSUPPORTED, "H = %d: grids above 32 take whole latitude tiles of 32 rows", H);
  if (!fft_ok && !(flags & SWSFT_PLAN_DFT_MATMUL))
    return fail(SWSFT_E_UNSUPPORTED,
                "W = %d: the FFT longitude stage takes powers of two up to 512 "
                "(SWSFT_PLAN_DFT_MATMUL takes any even W)", W);

  Plan* p = new (std::nothrow) swsft_plan_s();
  if (p == nullptr) return fail(SWSFT_E_ALLOC, "host allocation of the plan failed");
  p->H = H;
  p->W = W;
  p->L = L;
  p->Hp = swsft::round_up(H, 8);
  p->JT = H < 32 ? H : 32;
  p->Lp = swsft::round_up(L, 32);
  p->M = 2 * L - 1;
  p->n_in = n_spins_in;
  p->n_out = n_spins_out;
  for (int i = 0; i < n_spins_in; ++i) p->spins_in[i] = spins_in[i];
  for (int i = 0; i < n_spins_out; ++i) p->spins_out[i] = spins_out[i];
  p->dtype = dtype;
  p->elem = dtype == SWSFT_BF16 ? 2 : 4;
  p->flags = flags;
  p->fft_ok = fft_ok;

  hipError_t e = hipGetDevice(&p->device);
  if (e != hipSuccess) {
    free_plan(p);
    delete static_cast<swsft_plan_s*>(p);
    return hip_fail(e, "hipGetDevice");
  }
  // the device address of the static workspace of spin_sph_conv_forward_noalloc
  if ((e = swsft::register_scratch(p->device)) != hipSuccess) {
    free_plan(p);
    delete static_cast<swsft_plan_s*>(p);
    return hip_fail(e, "hipGetSymbolAddress of the static workspace");
  }
  const size_t fb = (size_t)p->n_in * p->fwd_table_elems() * p->elem;
  const size_t ib = (size_t)p->n_out * p->inv_table_elems() * p->elem;
  const size_t sb = (size_t)p->n_in * p->inv_table_elems() * p->elem;   // backward synthesis
  const size_t ab = (size_t)p->n_out * p->fwd_table_elems() * p->elem;  // backward analysis
  if (hipMalloc(&p->tab_fwd, fb) != hipSuccess || hipMalloc(&p->tab_inv, ib) != hipSuccess ||
      hipMalloc(&p->tab_bwd_syn, sb) != hipSuccess || hipMalloc(&p->tab_bwd_ana, ab) != hipSuccess ||
      hipMalloc((void**)&p->twiddle, (size_t)W * sizeof(float2)) != hipSuccess) {
    (void)hipGetLastError();
    free_plan(p);
    delete static_cast<swsft_plan_s*>(p);
    return fail(SWSFT_E_ALLOC, "hipMalloc of %zu table bytes failed", fb + ib + sb + ab);
  }
  // zero padding and the rows below max(|m|, |s|); the table kernel fills the rest
  if ((e = hipMemset(p->tab_fwd, 0, fb)) != hipSuccess ||
      (e = hipMemset(p->tab_inv, 0, ib)) != hipSuccess ||
      (e = hipMemset(p->tab_bwd_syn, 0, sb)) != hipSuccess ||
      (e = hipMemset(p->tab_bwd_ana, 0, ab)) != hipSuccess ||
      (e = swsft::launch_tables(*p, nullptr)) != hipSuccess ||
      (e = hipDeviceSynchronize()) != hipSuccess) {
    free_plan(p);
    delete static_cast<swsft_plan_s*>(p);
    return hip_fail(e, "table generation");
  }
  if (swsft::is_delta(*p)) {
    const size_t e1 = swsft::delta_fwd_theta_elems(*p) * p->elem;
    const size_t e2 = swsft::delta_inv_theta_elems(*p) * p->elem;
    const size_t e3 = (size_t)p->n_in * swsft::delta_fwd_table_elems(*p) * p->elem;
    const size_t e4 = (size_t)p->n_out * swsft::delta_inv_table_elems(*p) * p->elem;
    if (hipMalloc(&p->delta_theta_fwd, e1) != hipSuccess ||
        hipMalloc(&p->delta_theta_inv, e2) != hipSuccess ||
        hipMalloc(&p->delta_fwd, e3) != hipSuccess || hipMalloc(&p->delta_inv, e4) != hipSuccess) {
      (void)hipGetLastError();
      free_plan(p);
      delete static_cast<swsft_plan_s*>(p);
      return fail(SWSFT_E_ALLOC, "hipMalloc of %zu Delta-route table bytes failed", e1 + e2 + e3 + e4);
    }
    if ((e = hipMemset(p->delta_theta_fwd, 0, e1)) != hipSuccess ||
        (e = hipMemset(p->delta_theta_inv, 0, e2)) != hipSuccess ||
        (e = hipMemset(p->delta_fwd, 0, e3)) != hipSuccess ||
        (e = hipMemset(p->delta_inv, 0, e4)) != hipSuccess ||
        (e = swsft::launch_delta_tables(*p, nullptr)) != hipSuccess ||
        (e = hipDeviceSynchronize()) != hipSuccess) {
      free_plan(p);
      delete static_cast<swsft_plan_s*>(p);
      return hip_fail(e, "Delta-route table generation");
    }
  }
  if (flags & SWSFT_PLAN_DFT_MATMUL) {
    const size_t db = (size_t)2 * p->M * 2 * W * p->elem;
    if (hipMalloc(&p->dft_mat, db) != hipSuccess) {
      (void)hipGetLastError();
      p->dft_mat = nullptr;
      free_plan(p);
      delete static_cast<swsft_plan_s*>(p);
      return fail(SWSFT_E_ALLOC, "hipMalloc of the %zu-byte DFT matrix failed", db);
    }
    const size_t gb = (size_t)2 * W * swsft::dft_inv_pitch(p->M) * p->elem;
    if (hipMalloc(&p->dft_mat_inv, gb) != hipSuccess) {
      (void)hipGetLastError();
      p->dft_mat_inv = nullptr;
      free_plan(p);
      delete static_cast<swsft_plan_s*>(p);
      return fail(SWSFT_E_ALLOC, "hipMalloc of the %zu-byte inverse DFT matrix failed", gb);
    }
    if ((e = swsft::launch_dft_matrix(*p, nullptr)) != hipSuccess ||
        (e = swsft::launch_dft_matrix_inv(*p, nullptr)) != hipSuccess ||
        (e = hipDeviceSynchronize()) != hipSuccess) {
      free_plan(p);
      delete static_cast<swsft_plan_s*>(p);
      return hip_fail(e, "DFT matrix generation");
    }
  }
  *out = static_cast<swsft_plan_s*>(p);
  return SWSFT_OK;
}

void swsft_plan_destroy(swsft_plan p) {
  if (p == nullptr) return;
  free_plan(p);
  delete p;
}

size_t swsft_workspace_bytes(swsft_plan p, int op, int B, int C_in, int C_out) {
  if (p == nullptr) return 0;
  if (op == SWSFT_OP_FORWARD) C_out = 1;
  if (op == SWSFT_OP_INVERSE) C_in = 1;
  if (check_bc(B, C_in, "C_in") != SWSFT_OK || check_bc(B, C_out, "C_out") != SWSFT_OK) return 0;
  return ws_need(*p, op, B, C_in, C_out);
}

namespace {

// The analysis x -> coef on the input spins of p with its table tab_fwd
// (direct latitude route), stage times recorded on tp: one launch for 32 x 32
// float grids (the spectrum stays in LDS), else the longitude DFT into X and
// the latitude GEMM.
swsft_status analysis_stages(Plan& tp, const Plan& p, int B, int C, const void* x, void* X,
                             void* coef, hipStream_t st) {
  if (swsft::fused32_ok(p, C))
    return run_stage(tp, swsft::kStageSmallFwd, st, "small_fwd",
                     [&] { return swsft::launch_fused32_fwd(p, B, C, x, coef, st); });
  SWSFT_TRY(run_stage(tp, swsft::kStageDftFwd, st, "dft_fwd",
                      [&] { return swsft::launch_dft_fwd(p, p.n_in, B, C, x, X, st); }));
  return run_stage(tp, swsft::kStageLatFwd, st, "lat_fwd",
                   [&] { return swsft::launch_lat_fwd(p, B, C, X, coef, st); });
}

// The forward transform x -> coef: longitude stage into X, then the latitude
// stage directly (d tables) or by the Delta route (theta GEMM into D, then
// the Delta contraction by the latitude kernels on a plan view whose "grid"
// is the R rows of D).
swsft_status forward_stages(Plan& p, int B, int C, const void* x, void* X, void* D, void* coef,
                            hipStream_t st) {
  if (swsft::small_path(p, 1))
    return run_stage(p, swsft::kStageSmallFwd, st, "small_fwd",
                     [&] { return swsft::launch_small_fwd(p, B, C, x, coef, st); });
  if (!swsft::is_delta(p)) return analysis_stages(p, p, B, C, x, X, coef, st);
  SWSFT_TRY(run_stage(p, swsft::kStageDftFwd, st, "dft_fwd",
                      [&] { return swsft::launch_dft_fwd(p, p.n_in, B, C, x, X, st); }));
  SWSFT_TRY(run_stage(p, swsft::kStageDeltaTheta, st, "delta_theta",
                      [&] { return swsft::launch_delta_theta_fwd(p, B, C, X, D, st); }));
  Plan v = p;
  v.H = v.Hp = swsft::delta_rows(p);
  v.JT = 32;
  v.tab_fwd = p.delta_fwd;
  return run_stage(p, swsft::kStageLatFwd, st, "lat_fwd",
                   [&] { return swsft::launch_lat_fwd(v, B, C, D, coef, st); });
}

// Spectra of at most this many bytes stay in the 256 MiB Infinity Cache of an
// MI355X between the latitude synthesis that writes them and the inverse
// longitude DFT that reads them.
constexpr size_t kCacheResidentBytes = size_t(128) << 20;

// Latitude synthesis and inverse DFT, coef -> y, on the output spins of p
// (direct latitude route; stage times are recorded on tp, the caller's
// plan).  When the spectrum Y of the whole batch exceeds kCacheResidentBytes,
// the two alternate over batch ranges whose Y fits, so the DFT reads Y from
// the cache instead of HBM.
swsft_status synthesis_stages(Plan& tp, const Plan& p, int B, int C, const void* coef, void* Y,
                              void* y, hipStream_t st) {
  if (swsft::fused32_ok(p, C))  // the spectrum stays in LDS: one launch for the batch
    return run_stage(tp, swsft::kStageSmallInv, st, "small_inv",
                     [&] { return swsft::launch_fused32_inv(p, B, C, coef, y, st); });
  {
    const size_t per_item = swsft::xy_elems(p, p.n_out, 1, C) * p.elem;
    int bc = per_item == 0 ? B : (int)(kCacheResidentBytes / per_item);
    bc = bc < 1 ? 1 : (bc > B ? B : bc);
    if (((size_t)p.n_out * 2 * C * p.elem) % 16 != 0) bc = B;  // batch offsets keep 16-byte rows
    if (bc >= B) {
      SWSFT_TRY(run_stage(tp, swsft::kStageLatInv, st, "lat_inv",
                          [&] { return swsft::launch_lat_inv(p, B, C, coef, Y, st); }));
      return run_stage(tp, swsft::kStageDftInv, st, "dft_inv",
                       [&] { return swsft::launch_dft_inv(p, p.n_out, B, C, Y, y, st); });
    }
    Plan v = p;
    v.coef_ldb = B;
    const size_t coef_step = (size_t)p.n_out * 2 * C * p.elem;  // one batch item of a row
    const size_t y_step = (size_t)p.n_out * C * p.H * p.W * 2 * p.elem;
    for (int b0 = 0; b0 < B; b0 += bc) {
      const int n = B - b0 < bc ? B - b0 : bc;
      const void* cb = static_cast<const char*>(coef) + b0 * coef_step;
      void* yb = static_cast<char*>(y) + b0 * y_step;
      SWSFT_TRY(run_stage(tp, swsft::kStageLatInv, st, "lat_inv",
                          [&] { return swsft::launch_lat_inv(v, n, C, cb, Y, st); }));
      SWSFT_TRY(run_stage(tp, swsft::kStageDftInv, st, "dft_inv",
                          [&] { return swsft::launch_dft_inv(p, p.n_out, n, C, Y, yb, st); }));
    }
    return SWSFT_OK;
  }
}

// The inverse transform coef -> y (see forward_stages).
swsft_status inverse_stages(Plan& p, int B, int C, const void* coef, void* Y, void* D, void* y,
                            hipStream_t st) {
  if (swsft::small_path(p, 1))
    return run_stage(p, swsft::kStageSmallInv, st, "small_inv", [&] {
      return swsft::launch_small_inv(p, B, 1, C, coef, nullptr, y, st);
    });
  if (!swsft::is_delta(p)) {
    return synthesis_stages(p, p, B, C, coef, Y, y, st);
  } else {
    Plan v = p;
    v.H = v.Hp = swsft::delta_rows(p);
    v.JT = 32;
    v.tab_inv = p.delta_inv;
    SWSFT_TRY(run_stage(p, swsft::kStageLatInv, st, "lat_inv",
                        [&] { return swsft::launch_lat_inv(v, B, C, coef, D, st); }));
    SWSFT_TRY(run_stage(p, swsft::kStageDeltaTheta, st, "delta_theta",
                        [&] { return swsft::launch_delta_theta_inv(p, B, C, D, Y, st); }));
  }
  return run_stage(p, swsft::kStageDftInv, st, "dft_inv",
                   [&] { return swsft::launch_dft_inv(p, p.n_out, B, C, Y, y, st); });
}

swsft_status reject_delta(const Plan& p, const char* what) {
  if (swsft::is_delta(p))
    return fail(SWSFT_E_UNSUPPORTED, "%s has no Delta-route variant: use a plan without "
                "SWSFT_PLAN_DELTA / SWSFT_PLAN_DELTA_SYM", what);
  return SWSFT_OK;
}

}  // namespace

swsft_status swsft_forward(swsft_plan p, int B, int C, const void* x, void* coef, void* ws,
                           size_t ws_bytes, void* stream) {
  g_last_error[0] = 0;
  if (p == nullptr) return fail(SWSFT_E_INVALID, "plan is NULL");
  SWSFT_TRY(check_bc(B, C, "C"));
  SWSFT_TRY(check_ptr(x, "x"));
  SWSFT_TRY(check_ptr(coef, "coef"));
  SWSFT_TRY(check_ws(*p, SWSFT_OP_FORWARD, B, C, 1, ws, ws_bytes));
  SWSFT_TRY(check_disjoint({{x, spatial_bytes(*p, p->n_in, B, C), "x", false},
                            {coef, swsft::coef_elems(*p, p->n_in, B, C) * p->elem, "coef", true},
                            {ws, ws_bytes, "the workspace", true}}));
  SWSFT_TRY(check_device(*p));
  hipStream_t st = static_cast<hipStream_t>(stream);
  char* X = static_cast<char*>(ws);
  void* D = X + align_up(swsft::xy_elems(*p, p->n_in, B, C) * p->elem);
  return forward_stages(*p, B, C, x, X, D, coef, st);
}

swsft_status swsft_inverse(swsft_plan p, int B, int C, const void* coef, void* y, void* ws,
                           size_t ws_bytes, void* stream) {
  g_last_error[0] = 0;
  if (p == nullptr) return fail(SWSFT_E_INVALID, "plan is NULL");
  SWSFT_TRY(check_bc(B, C, "C"));
  SWSFT_TRY(check_ptr(coef, "coef"));
  SWSFT_TRY(check_ptr(y, "y"));
  SWSFT_TRY(check_inverse_stage(*p));
  SWSFT_TRY(check_ws(*p, SWSFT_OP_INVERSE, B, 1, C, ws, ws_bytes));
  SWSFT_TRY(check_disjoint({{coef, swsft::coef_elems(*p, p->n_out, B, C) * p->elem, "coef", false},
                            {y, spatial_bytes(*p, p->n_out, B, C), "y", true},
                            {ws, ws_bytes, "the workspace", true}}));
  SWSFT_TRY(check_device(*p));
  hipStream_t st = static_cast<hipStream_t>(stream);
  char* Y = static_cast<char*>(ws);
  void* D = Y + align_up(swsft::xy_elems(*p, p->n_out, B, C) * p->elem);
  return inverse_stages(*p, B, C, coef, Y, D, y, st);
}

namespace {

// The layer; with coef_x != NULL the input's coefficients are written there
// (for the backward pass) instead of to the workspace.
swsft_status conv_forward(swsft_plan p, int B, int C_in, int C_out, const void* x,
                          const void* filters, void* y, void* coef_x, void* ws, size_t ws_bytes,
                          void* stream) {
  g_last_error[0] = 0;
  if (p == nullptr) return fail(SWSFT_E_INVALID, "plan is NULL");
  SWSFT_TRY(check_bc(B, C_in, "C_in"));
  SWSFT_TRY(check_bc(B, C_out, "C_out"));
  SWSFT_TRY(check_filter_block(*p, C_in, C_out));
  SWSFT_TRY(check_ptr(x, "x"));
  SWSFT_TRY(check_ptr(filters, "filters"));
  SWSFT_TRY(check_ptr(y, "y"));
  if (coef_x != nullptr) SWSFT_TRY(check_ptr(coef_x, "coef_x"));
  SWSFT_TRY(check_inverse_stage(*p));
  SWSFT_TRY(check_ws(*p, SWSFT_OP_CONV, B, C_in, C_out, ws, ws_bytes));
  const size_t xs = (size_t)B * p->n_in * C_in * p->H * p->W * 2 * p->elem;
  const size_t ys = (size_t)B * p->n_out * C_out * p->H * p->W * 2 * p->elem;
  const size_t cs = swsft::coef_elems(*p, p->n_in, B, C_in) * p->elem;
  const size_t ks = filter_elems(*p, C_in, C_out) * p->elem;
  SWSFT_TRY(check_disjoint({{x, xs, "x", false},
                            {filters, ks, "filters", false},
                            {y, ys, "y", true},
                            {coef_x, cs, "coef_x", true},
                            {ws, ws_bytes, "the workspace", true}}));
  SWSFT_TRY(check_device(*p));
  hipStream_t st = static_cast<hipStream_t>(stream);
  const size_t xin = swsft::xy_elems(*p, p->n_in, B, C_in);
  const size_t xout = swsft::xy_elems(*p, p->n_out, B, C_out);
  char* w = static_cast<char*>(ws);
  void* XY = w;
  w += align_up((xin > xout ? xin : xout) * p->elem);
  void* coef = coef_x != nullptr ? coef_x : static_cast<void*>(w);
  w += align_up(swsft::coef_elems(*p, p->n_in, B, C_in) * p->elem);
  void* coef2 = w;
  w += align_up(swsft::coef_elems(*p, p->n_out, B, C_out) * p->elem);
  void* D = w;
  if (swsft::small_path(*p, C_in)) {
    // small grids: the mixing runs inside the synthesis, per output map
    SWSFT_TRY(forward_stages(*p, B, C_in, x, XY, D, coef, st));
    return run_stage(*p, swsft::kStageSmallInv, st, "small_inv", [&] {
      return swsft::launch_small_inv(*p, B, C_in, C_out, coef, filters, y, st);
    });
  }
  SWSFT_TRY(forward_stages(*p, B, C_in, x, XY, D, coef, st));
  SWSFT_TRY(run_stage(*p, swsft::kStageMix, st, "mix", [&] {
    return swsft::launch_mix(*p, B, C_in, C_out, coef, filters, coef2, st);
  }));
  return inverse_stages(*p, B, C_out, coef2, XY, D, y, st);
}

}  // namespace

swsft_status spin_sph_conv_forward(swsft_plan p, int B, int C_in, int C_out, const void* x,
                                   const void* filters, void* y, void* ws, size_t ws_bytes,
                                   void* stream) {
  return conv_forward(p, B, C_in, C_out, x, filters, y, nullptr, ws, ws_bytes, stream);
}

swsft_status spin_sph_conv_forward_noalloc(swsft_plan p, int B, int C_in, int C_out,
                                           const void* x, const void* filters, void* y,
                                           void* stream) {
  g_last_error[0] = 0;
  if (p == nullptr) return fail(SWSFT_E_INVALID, "plan is NULL");
  SWSFT_TRY(check_bc(B, C_in, "C_in"));
  SWSFT_TRY(check_bc(B, C_out, "C_out"));
  SWSFT_TRY(check_filter_block(*p, C_in, C_out));
  const size_t need = ws_need(*p, SWSFT_OP_CONV, B, C_in, C_out);
  if (need > swsft::kNoAllocScratchBytes)
    return fail(SWSFT_E_UNSUPPORTED,
                "the layer needs %zu bytes of workspace; the library's static workspace holds "
                "%zu (use spin_sph_conv_forward with a caller workspace)",
                need, swsft::kNoAllocScratchBytes);
  void* ws = swsft::scratch_of(p->device);
  if (ws == nullptr)
    return fail(SWSFT_E_INVALID, "no static workspace registered for device %d", p->device);
  return conv_forward(p, B, C_in, C_out, x, filters, y, nullptr, ws, swsft::kNoAllocScratchBytes,
                      stream);
}

swsft_status spin_sph_conv_forward_train(swsft_plan p, int B, int C_in, int C_out, const void* x,
                                         const void* filters, void* y, void* coef_x, void* ws,
                                         size_t ws_bytes, void* stream) {
  if (coef_x == nullptr) {
    g_last_error[0] = 0;
    return fail(SWSFT_E_INVALID, "coef_x is NULL");
  }
  return conv_forward(p, B, C_in, C_out, x, filters, y, coef_x, ws, ws_bytes, stream);
}

swsft_status spin_sph_conv_backward(swsft_plan p, int B, int C_in, int C_out, const void* x,
                                    const void* coef_x, const void* filters, const void* grad_y,
                                    void* grad_x, void* grad_filters, void* ws, size_t ws_bytes,
                                    void* stream) {
  g_last_error[0] = 0;
  if (p == nullptr) return fail(SWSFT_E_INVALID, "plan is NULL");
  SWSFT_TRY(check_bc(B, C_in, "C_in"));
  SWSFT_TRY(check_bc(B, C_out, "C_out"));
  SWSFT_TRY(check_filter_block(*p, C_in, C_out));
  if (grad_x == nullptr && grad_filters == nullptr)
    return fail(SWSFT_E_INVALID, "neither grad_x nor grad_filters requested");
  SWSFT_TRY(check_ptr(grad_y, "grad_y"));
  SWSFT_TRY(check_inverse_stage(*p));
  SWSFT_TRY(reject_delta(*p, "spin_sph_conv_backward"));
  if (grad_filters != nullptr) {
    if (coef_x != nullptr) SWSFT_TRY(check_ptr(coef_x, "coef_x"));
    else SWSFT_TRY(check_ptr(x, "x"));
    SWSFT_TRY(check_ptr(grad_filters, "grad_filters"));
  }
  if (grad_x != nullptr) {
    SWSFT_TRY(check_ptr(filters, "filters"));
    SWSFT_TRY(check_ptr(grad_x, "grad_x"));
  }
  SWSFT_TRY(check_ws(*p, SWSFT_OP_CONV_BACKWARD, B, C_in, C_out, ws, ws_bytes));
  {
    // outputs must not overlap inputs
    const size_t xs = (size_t)B * p->n_in * C_in * p->H * p->W * 2 * p->elem;
    const size_t ys = (size_t)B * p->n_out * C_out * p->H * p->W * 2 * p->elem;
    const size_t ks = filter_elems(*p, C_in, C_out) * p->elem;
    struct R { const void* a; size_t n; };
    const size_t cs = swsft::coef_elems(*p, p->n_in, B, C_in) * p->elem;
    const R ins[4] = {{grad_filters && !coef_x ? x : nullptr, xs},
                      {grad_filters ? coef_x : nullptr, cs},
                      {grad_x ? filters : nullptr, ks},
                      {grad_y, ys}};
    const R outs[2] = {{grad_x, xs}, {grad_filters, ks}};
    for (const R& o : outs) {
      if (o.a == nullptr) continue;
      for (const R& i : ins) {
        if (i.a == nullptr) continue;
        const char *ob = static_cast<const char*>(o.a), *ib = static_cast<const char*>(i.a);
        if (ob < ib + i.n && ib < ob + o.n) return fail(SWSFT_E_INVALID, "an output overlaps an input");
      }
    }
    if (grad_x && grad_filters) {
      const char *a = static_cast<const char*>(grad_x), *b = static_cast<const char*>(grad_filters);
      if (a < b + ks && b < a + xs) return fail(SWSFT_E_INVALID, "grad_x and grad_filters overlap");
    }
    for (const R& r : ins)
      if (overlaps(ws, ws_bytes, r.a, r.n)) return fail(SWSFT_E_INVALID, "the workspace overlaps an input");
    for (const R& r : outs)
      if (overlaps(ws, ws_bytes, r.a, r.n)) return fail(SWSFT_E_INVALID, "the workspace overlaps an output");
  }
  SWSFT_TRY(check_device(*p));
  hipStream_t st = static_cast<hipStream_t>(stream);
  const size_t xin = swsft::xy_elems(*p, p->n_in, B, C_in);
  const size_t xout = swsft::xy_elems(*p, p->n_out, B, C_out);
  char* w = static_cast<char*>(ws);
  void* XY = w;
  w += align_up((xin > xout ? xin : xout) * p->elem);
  void* a_in = w;  // F x
  w += align_up(swsft::coef_elems(*p, p->n_in, B, C_in) * p->elem);
  void* g_in = w;  // K^H g
  w += align_up(swsft::coef_elems(*p, p->n_in, B, C_in) * p->elem);
  void* g_out = w;  // G^H grad_y
  w += align_up(swsft::coef_elems(*p, p->n_out, B, C_out) * p->elem);
  void* KH = w;
  w += align_up(filter_elems(*p, C_in, C_out) * p->elem);
  void* part = w;  // partial sums of a split filter-gradient contraction

  // Views of the plan for the adjoint stages (shallow copies, nothing owned):
  // G^H grad_y is the forward latitude GEMM with the unweighted l-major table
  // on the output spins; K^H swaps the roles of the spin lists; F^H is the
  // inverse latitude GEMM with the weighted j-major table on the input spins.
  Plan ana = *p;
  ana.tab_fwd = p->tab_bwd_ana;
  ana.n_in = p->n_out;
  for (int i = 0; i < swsft::kMaxSpins; ++i) ana.spins_in[i] = p->spins_out[i];
  Plan adj = *p;
  adj.n_in = p->n_out;
  adj.n_out = p->n_in;
  for (int i = 0; i < swsft::kMaxSpins; ++i) {
    adj.spins_in[i] = p->spins_out[i];
    adj.spins_out[i] = p->spins_in[i];
  }
  Plan syn = *p;
  syn.tab_inv = p->tab_bwd_syn;
  syn.n_out = p->n_in;
  for (int i = 0; i < swsft::kMaxSpins; ++i) syn.spins_out[i] = p->spins_in[i];

  SWSFT_TRY(analysis_stages(*p, ana, B, C_out, grad_y, XY, g_out, st));
  if (grad_filters != nullptr) {
    const void* a = coef_x;  // F x as saved by the forward pass, or computed here
    if (a == nullptr) {
      // the forward transform exactly as the layer computes it (same kernels,
      // so saved and recomputed coefficients agree bit for bit)
      SWSFT_TRY(forward_stages(*p, B, C_in, x, XY, nullptr, a_in, st));
      a = a_in;
    }
    SWSFT_TRY(run_stage(*p, swsft::kStageFilterGrad, st, "filter_grad", [&] {
      return swsft::launch_filter_grad(*p, B, C_in, C_out, a, g_out, grad_filters, part, st);
    }));
  }
  if (grad_x != nullptr) {
    if (swsft::mix_adj_dma_supported(adj, C_out, C_in)) {
      // K^H applied from the filters as stored
      SWSFT_TRY(run_stage(*p, swsft::kStageMix, st, "mix", [&] {
        return swsft::launch_mix_adj_dma(adj, B, C_out, C_in, g_out, filters, g_in, st);
      }));
    } else {
      SWSFT_TRY(run_stage(*p, swsft::kStageFilterAdjoint, st, "filter_adjoint", [&] {
        return swsft::launch_filter_adjoint(*p, C_in, C_out, filters, KH, st);
      }));
      SWSFT_TRY(run_stage(*p, swsft::kStageMix, st, "mix", [&] {
        return swsft::launch_mix(adj, B, C_out, C_in, g_out, KH, g_in, st);
      }));
    }
    // F^H: the synthesis with the weighted table on the input spins, over
    // cache-sized batch ranges like the layer's inverse
    SWSFT_TRY(synthesis_stages(*p, syn, B, C_in, g_in, XY, grad_x, st));
  }
  return SWSFT_OK;
}

swsft_status spin_sph_mix(swsft_plan p, int B, int C_in, int C_out, const void* coef,
                          const void* filters, void* coef_out, void* stream) {
  g_last_error[0] = 0;
  if (p == nullptr) return fail(SWSFT_E_INVALID, "plan is NULL");
  SWSFT_TRY(check_bc(B, C_in, "C_in"));
  SWSFT_TRY(check_bc(B, C_out, "C_out"));
  SWSFT_TRY(check_filter_block(*p, C_in, C_out));
  SWSFT_TRY(check_ptr(coef, "coef"));
  SWSFT_TRY(check_ptr(filters, "filters"));
  SWSFT_TRY(check_ptr(coef_out, "coef_out"));
  {
    const size_t as = swsft::coef_elems(*p, p->n_in, B, C_in) * p->elem;
    const size_t ks = filter_elems(*p, C_in, C_out) * p->elem;
    const size_t os = swsft::coef_elems(*p, p->n_out, B, C_out) * p->elem;
    if (overlaps(coef_out, os, coef, as) || overlaps(coef_out, os, filters, ks))
      return fail(SWSFT_E_INVALID, "coef_out overlaps an input");
  }
  SWSFT_TRY(check_device(*p));
  hipStream_t st = static_cast<hipStream_t>(stream);
  return run_stage(*p, swsft::kStageMix, st, "mix", [&] {
    return swsft::launch_mix(*p, B, C_in, C_out, coef, filters, coef_out, st);
  });
}

swsft_status spin_sph_spectral_batch_norm(swsft_plan p, int B, int C, const void* coef,
                                          const float* gamma, const void* beta, float eps,
                                          const float* var_in, float* var_out, const void* skip,
                                          void* out, void* ws, size_t ws_bytes, void* stream) {
  g_last_error[0] = 0;
  if (p == nullptr) return fail(SWSFT_E_INVALID, "plan is NULL");
  SWSFT_TRY(check_bc(B, C, "C"));
  SWSFT_TRY(check_ptr(coef, "coef"));
  SWSFT_TRY(check_ptr(out, "out"));
  if (gamma == nullptr) return fail(SWSFT_E_INVALID, "gamma is NULL");
  if (!std::isfinite(eps) || eps < 0.f) return fail(SWSFT_E_INVALID, "eps must be finite and >= 0");
  if ((reinterpret_cast<uintptr_t>(gamma) | reinterpret_cast<uintptr_t>(var_in) |
       reinterpret_cast<uintptr_t>(var_out)) % 4 != 0 ||
      reinterpret_cast<uintptr_t>(beta) % 8 != 0)
    return fail(SWSFT_E_INVALID, "gamma, var_in, var_out must be 4-byte, beta 8-byte aligned");
  if (skip != nullptr) SWSFT_TRY(check_ptr(skip, "skip"));
  if (!swsft::bn_supported(*p, C))
    return fail(SWSFT_E_UNSUPPORTED, "S_out * C = %d exceeds 2048 columns", p->n_out * C);
  SWSFT_TRY(check_ws(*p, SWSFT_OP_BATCH_NORM, B, 1, C, ws, ws_bytes));
  {
    const size_t cs = swsft::coef_elems(*p, p->n_out, B, C) * p->elem;
    if (out != coef && overlaps(out, cs, coef, cs))
      return fail(SWSFT_E_INVALID, "out overlaps coef without being equal");
    if (skip != nullptr && out != skip && overlaps(out, cs, skip, cs))
      return fail(SWSFT_E_INVALID, "out overlaps skip without being equal");
    if (overlaps(ws, ws_bytes, coef, cs) || overlaps(ws, ws_bytes, out, cs))
      return fail(SWSFT_E_INVALID, "the workspace overlaps the coefficients");
  }
  SWSFT_TRY(check_device(*p));
  hipStream_t st = static_cast<hipStream_t>(stream);
  return run_stage(*p, swsft::kStageBatchNorm, st, "batch_norm", [&] {
    return swsft::launch_batch_norm(*p, B, C, coef, gamma, static_cast<const float2*>(beta), eps,
                                    var_in, var_out, skip, out, ws, st);
  });
}

size_t swsft_block_workspace_bytes(swsft_plan p_in, swsft_plan p_out, int B, int C) {
  if (p_in == nullptr || p_out == nullptr || check_bc(B, C, "C") != SWSFT_OK) return 0;
  const int S = p_out->n_out;
  const size_t xy_in = swsft::xy_elems(*p_in, S, B, C), xy_out = swsft::xy_elems(*p_out, S, B, C);
  const size_t e = p_out->elem;
  return align_up((xy_in > xy_out ? xy_in : xy_out) * e) +
         3 * align_up(swsft::coef_elems(*p_out, S, B, C) * e) +
         align_up((size_t)B * S * C * p_out->H * p_out->W * 2 * e) +
         align_up(swsft::bn_workspace_bytes(*p_out, B, C));
}

swsft_status spin_sph_residual_block_forward(swsft_plan p_in, swsft_plan p_out, int B, int C,
                                             const void* x, const swsft_block_params* prm,
                                             void* y, void* ws, size_t ws_bytes, void* stream) {
  g_last_error[0] = 0;
  if (p_in == nullptr || p_out == nullptr) return fail(SWSFT_E_INVALID, "plan is NULL");
  if (prm == nullptr) return fail(SWSFT_E_INVALID, "params is NULL");
  SWSFT_TRY(check_bc(B, C, "C"));
  SWSFT_TRY(check_ptr(x, "x"));
  SWSFT_TRY(check_ptr(y, "y"));
  SWSFT_TRY(check_ptr(prm->K1, "K1"));
  SWSFT_TRY(check_ptr(prm->K2, "K2"));
  if (prm->gamma1 == nullptr || prm->gamma2 == nullptr)
    return fail(SWSFT_E_INVALID, "gamma1 and gamma2 must not be NULL");
  if ((reinterpret_cast<uintptr_t>(prm->gamma1) | reinterpret_cast<uintptr_t>(prm->gamma2) |
       reinterpret_cast<uintptr_t>(prm->var1_out) | reinterpret_cast<uintptr_t>(prm->var2_out)) %
              4 != 0 ||
      (reinterpret_cast<uintptr_t>(prm->beta1) | reinterpret_cast<uintptr_t>(prm->beta2)) % 8 != 0)
    return fail(SWSFT_E_INVALID, "gamma, var must be 4-byte, beta 8-byte aligned");
  const void* pcs[6] = {prm->pc1_W1, prm->pc1_W2, prm->pc1_b, prm->pc2_W1, prm->pc2_W2, prm->pc2_b};
  for (const void* q : pcs)
    if (q == nullptr || reinterpret_cast<uintptr_t>(q) % 8 != 0)
      return fail(SWSFT_E_INVALID, "phase-collapse parameters must be non-NULL and 8-byte aligned");
  if (!std::isfinite(prm->eps) || prm->eps < 0.f)
    return fail(SWSFT_E_INVALID, "eps must be finite and >= 0");
  swsft::Plan &pi = *p_in, &po = *p_out;
  if (pi.device != po.device || pi.dtype != po.dtype || pi.L != po.L)
    return fail(SWSFT_E_INVALID, "the plans differ in device, dtype or bandlimit");
  const int S = po.n_out;
  bool same = pi.n_in == S && pi.n_out == S && po.n_in == S, has0 = false;
  for (int i = 0; same && i < S; ++i) {
    same = pi.spins_in[i] == po.spins_out[i] && pi.spins_out[i] == po.spins_out[i] &&
           po.spins_in[i] == po.spins_out[i];
    has0 |= po.spins_out[i] == 0;
  }
  if (!same) return fail(SWSFT_E_INVALID, "both plans must map the same spin list to itself");
  SWSFT_TRY(check_inverse_stage(po));
  SWSFT_TRY(reject_delta(pi, "spin_sph_residual_block_forward"));
  SWSFT_TRY(reject_delta(po, "spin_sph_residual_block_forward"));
  if (!has0) return fail(SWSFT_E_INVALID, "the spin list must contain spin 0");
  if (C > swsft::phase_collapse_max_channels(S))
    return fail(SWSFT_E_UNSUPPORTED, "C = %d exceeds %d channels for %d spins", C,
                swsft::phase_collapse_max_channels(S), S);
  if (!swsft::bn_supported(po, C))
    return fail(SWSFT_E_UNSUPPORTED, "S * C = %d exceeds 2048 columns", S * C);
  const size_t need = swsft_block_workspace_bytes(p_in, p_out, B, C);
  if (ws == nullptr || ws_bytes < need)
    return fail(SWSFT_E_WORKSPACE, "workspace: %zu bytes given, %zu needed",
                ws == nullptr ? (size_t)0 : ws_bytes, need);
  if (reinterpret_cast<uintptr_t>(ws) % 16 != 0)
    return fail(SWSFT_E_INVALID, "workspace must be 16-byte aligned");
  {
    const size_t xs = (size_t)B * S * C * pi.H * pi.W * 2 * pi.elem;
    const size_t ys = (size_t)B * S * C * po.H * po.W * 2 * po.elem;
    if (overlaps(x, xs, y, ys)) return fail(SWSFT_E_INVALID, "x and y overlap");
    if (overlaps(ws, ws_bytes, x, xs) || overlaps(ws, ws_bytes, y, ys))
      return fail(SWSFT_E_INVALID, "the workspace overlaps x or y");
  }
  SWSFT_TRY(check_device(po));
  hipStream_t st = static_cast<hipStream_t>(stream);
  const size_t xy_in = swsft::xy_elems(pi, S, B, C), xy_out = swsft::xy_elems(po, S, B, C);
  const size_t cb = align_up(swsft::coef_elems(po, S, B, C) * po.elem);
  char* w = static_cast<char*>(ws);
  void* XY = w;
  w += align_up((xy_in > xy_out ? xy_in : xy_out) * po.elem);
  void* a = w;  // FT(x): also the skip connection
  void* h = w + cb;
  void* g = w + 2 * cb;
  w += 3 * cb;
  void* z = w;  // the block's middle feature map, on the output grid
  w += align_up((size_t)B * S * C * po.H * po.W * 2 * po.elem);
  void* bnws = w;
  auto f2 = [](const void* q) { return static_cast<const float2*>(q); };

  // stage timing is recorded on the output plan
  SWSFT_TRY(analysis_stages(po, pi, B, C, x, XY, a, st));
  SWSFT_TRY(run_stage(po, swsft::kStageMix, st, "mix",
                      [&] { return swsft::launch_mix(po, B, C, C, a, prm->K1, h, st); }));
  SWSFT_TRY(run_stage(po, swsft::kStageBatchNorm, st, "batch_norm", [&] {
    return swsft::launch_batch_norm(po, B, C, h, prm->gamma1, f2(prm->beta1), prm->eps, nullptr,
                                    prm->var1_out, nullptr, h, bnws, st);
  }));
  SWSFT_TRY(synthesis_stages(po, po, B, C, h, XY, z, st));
  SWSFT_TRY(run_stage(po, swsft::kStagePhaseCollapse, st, "phase_collapse", [&] {
    return swsft::launch_phase_collapse(po, B, C, z, f2(prm->pc1_W1), f2(prm->pc1_W2),
                                        f2(prm->pc1_b), z, st);
  }));
  SWSFT_TRY(analysis_stages(po, po, B, C, z, XY, h, st));
  SWSFT_TRY(run_stage(po, swsft::kStageMix, st, "mix",
                      [&] { return swsft::launch_mix(po, B, C, C, h, prm->K2, g, st); }));
  SWSFT_TRY(run_stage(po, swsft::kStageBatchNorm, st, "batch_norm", [&] {
    return swsft::launch_batch_norm(po, B, C, g, prm->gamma2, f2(prm->beta2), prm->eps, nullptr,
                                    prm->var2_out, a, g, bnws, st);
  }));
  SWSFT_TRY(synthesis_stages(po, po, B, C, g, XY, y, st));
  return run_stage(po, swsft::kStagePhaseCollapse, st, "phase_collapse", [&] {
    return swsft::launch_phase_collapse(po, B, C, y, f2(prm->pc2_W1), f2(prm->pc2_W2),
                                        f2(prm->pc2_b), y, st);
  });
}

swsft_status spin_sph_phase_collapse(swsft_plan p, int B, int C, const void* x, const void* W1,
                                     const void* W2, const void* bias, void* y, void* stream) {
  g_last_error[0] = 0;
  if (p == nullptr) return fail(SWSFT_E_INVALID, "plan is NULL");
  SWSFT_TRY(check_bc(B, C, "C"));
  SWSFT_TRY(check_ptr(x, "x"));
  SWSFT_TRY(check_ptr(y, "y"));
  if (W1 == nullptr || W2 == nullptr || bias == nullptr)
    return fail(SWSFT_E_INVALID, "W1, W2 and bias must not be NULL");
  if ((reinterpret_cast<uintptr_t>(W1) | reinterpret_cast<uintptr_t>(W2) |
       reinterpret_cast<uintptr_t>(bias)) % 8 != 0)
    return fail(SWSFT_E_INVALID, "W1, W2 and bias must be 8-byte aligned");
  bool has0 = false;
  for (int i = 0; i < p->n_out; ++i) has0 |= p->spins_out[i] == 0;
  if (!has0) return fail(SWSFT_E_INVALID, "spins_out does not contain spin 0");
  if (C > swsft::phase_collapse_max_channels(p->n_out))
    return fail(SWSFT_E_UNSUPPORTED, "C = %d exceeds %d channels for %d spins", C,
                swsft::phase_collapse_max_channels(p->n_out), p->n_out);
  if (x != y) {
    const char* xb = static_cast<const char*>(x);
    const char* yb = static_cast<const char*>(y);
    const size_t sz = (size_t)B * p->n_out * C * p->H * p->W * 2 * p->elem;
    if (xb < yb + sz && yb < xb + sz)
      return fail(SWSFT_E_INVALID, "x and y overlap without being equal");
  }
  SWSFT_TRY(check_device(*p));
  hipStream_t st = static_cast<hipStream_t>(stream);
  return run_stage(*p, swsft::kStagePhaseCollapse, st, "phase_collapse", [&] {
    return swsft::launch_phase_collapse(*p, B, C, x, static_cast<const float2*>(W1),
                                        static_cast<const float2*>(W2),
                                        static_cast<const float2*>(bias), y, st);
  });
}

swsft_status swsft_stage_timing(swsft_plan p, int enable) {
  g_last_error[0] = 0;
  if (p == nullptr) return fail(SWSFT_E_INVALID, "plan is NULL");
  if (enable && p->ev == nullptr) {
    const int n = 2 * swsft::kMaxTimedLaunches;
    p->ev = static_cast<hipEvent_t*>(std::calloc(n, sizeof(hipEvent_t)));
    p->ev_stage = static_cast<int*>(std::calloc(swsft::kMaxTimedLaunches, sizeof(int)));
    if (p->ev == nullptr || p->ev_stage == nullptr) return fail(SWSFT_E_ALLOC, "event pool");
    for (int i = 0; i < n; ++i) {
      hipError_t e = hipEventCreate(&p->ev[i]);
      if (e != hipSuccess) return hip_fail(e, "hipEventCreate");
    }
  }
  std::lock_guard<std::mutex> lock(g_timing_mu);
  p->timing = enable != 0;
  p->n_timed = 0;
  return SWSFT_OK;
}

int swsft_stage_times(swsft_plan p, double* ms, long long* launches, int n) {
  if (p == nullptr) return 0;
  std::lock_guard<std::mutex> lock(g_timing_mu);
  for (int i = 0; i < p->n_timed; ++i) {
    const int s = p->ev_stage[i];
    if (hipEventSynchronize(p->ev[2 * i + 1]) != hipSuccess) continue;
    float t = 0.f;
    if (hipEventElapsedTime(&t, p->ev[2 * i], p->ev[2 * i + 1]) != hipSuccess) continue;
    if (s < n) {
      if (ms) ms[s] += t;
      if (launches) launches[s] += 1;
    }
  }
  p->n_timed = 0;
  return swsft::kNumStages;
}

swsft_status swsft_probe_mfma(int dtype, int random_operands, long long iters, int n_waves,
                              float* out, double* flops_out, void* stream) {
  g_last_error[0] = 0;
  if (dtype != SWSFT_F32 && dtype != SWSFT_BF16) return fail(SWSFT_E_INVALID, "dtype %d", dtype);
  if (out == nullptr) return fail(SWSFT_E_INVALID, "out is NULL");
  if (iters < 1 || iters > (1ll << 24)) return fail(SWSFT_E_INVALID, "iters = %lld", iters);
  if (n_waves < 4 || n_waves > (1 << 20) || n_waves % 4 != 0)
    return fail(SWSFT_E_INVALID, "n_waves = %d (a multiple of 4 in [4, 2^20])", n_waves);
  if (flops_out != nullptr)
    *flops_out = swsft::mfma_probe_flops_per_wave_round(dtype) * (double)n_waves * (double)iters;
  const hipError_t e =
      swsft::launch_mfma_probe(dtype, random_operands, iters, n_waves, out, (hipStream_t)stream);
  if (e != hipSuccess) return hip_fail(e, "mfma probe launch");
  return SWSFT_OK;
}

swsft_status swsft_plan_table(swsft_plan p, int which, int spin_index, void* host_dst,
                              size_t bytes) {
  g_last_error[0] = 0;
  if (p == nullptr || host_dst == nullptr) return fail(SWSFT_E_INVALID, "NULL argument");
  size_t elems;
  const char* base;
  if (which == 0) {
    if (spin_index < 0 || spin_index >= p->n_in) return fail(SWSFT_E_INVALID, "spin index");
    elems = p->fwd_table_elems();
    base = static_cast<const char*>(p->tab_fwd) + spin_index * elems * p->elem;
  } else if (which == 1) {
    if (spin_index < 0 || spin_index >= p->n_out) return fail(SWSFT_E_INVALID, "spin index");
    elems = p->inv_table_elems();
    base = static_cast<const char*>(p->tab_inv) + spin_index * elems * p->elem;
  } else if (which == 2) {
    if (spin_index < 0 || spin_index >= p->n_in) return fail(SWSFT_E_INVALID, "spin index");
    elems = p->inv_table_elems();
    base = static_cast<const char*>(p->tab_bwd_syn) + spin_index * elems * p->elem;
  } else if (which == 3) {
    if (spin_index < 0 || spin_index >= p->n_out) return fail(SWSFT_E_INVALID, "spin index");
    elems = p->fwd_table_elems();
    base = static_cast<const char*>(p->tab_bwd_ana) + spin_index * elems * p->elem;
  } else {
    return fail(SWSFT_E_INVALID, "which = %d", which);
  }
  if (bytes != elems * p->elem)
    return fail(SWSFT_E_INVALID, "bytes = %zu, table has %zu", bytes, elems * p->elem);
  SWSFT_TRY(check_device(*p));
  hipError_t e = hipMemcpy(host_dst, base, bytes, hipMemcpyDeviceToHost);
  if (e != hipSuccess) return hip_fail(e, "hipMemcpy");
  return SWSFT_OK;
}

}  // extern "C"
