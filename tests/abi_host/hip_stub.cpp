// Host-only stand-ins for the HIP runtime and for the library's kernel
// launchers, so that the C-ABI layer (csrc/swsft_api.cpp) can be built with
// -fsanitize=address,undefined and exercised on a machine without a GPU.
//
// "Device memory" is host memory from posix_memalign, registered per
// allocation.  Every launcher checks that each buffer it would read or write
// lies inside one registered allocation, with the extent the kernel's
// documented layout gives, then reads every byte it would read and writes
// every byte it would write, so AddressSanitizer sees any pointer
// arithmetic of the API layer that leaves a buffer.  No kernel runs.
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <mutex>
#include <vector>

#include "../../paper_2306_05420_amd/csrc/swsft_internal.h"

struct ihipEvent_t {
  int id;
};

namespace stub {

struct Alloc {
  char* p;
  size_t n;
};
std::vector<Alloc>& allocs() {
  static std::vector<Alloc> v;
  return v;
}
std::mutex mu;
long long launches = 0;

void die(const char* what, const void* p, size_t n) {
  std::fprintf(stderr, "STUB FAILURE: %s: [%p, +%zu) is not inside one allocation\n", what, p, n);
  std::abort();
}

const Alloc* find(const void* p, size_t n) {
  const char* c = static_cast<const char*>(p);
  for (const Alloc& a : allocs())
    if (c >= a.p && c + n <= a.p + a.n) return &a;
  return nullptr;
}

volatile unsigned sink = 0;

void rd(const char* what, const void* p, size_t n) {
  if (n == 0) return;
  if (p == nullptr || find(p, n) == nullptr) die(what, p, n);
  const unsigned char* c = static_cast<const unsigned char*>(p);
  unsigned s = 0;
  for (size_t i = 0; i < n; ++i) s += c[i];
  sink = sink + s;
}

void wr(const char* what, void* p, size_t n) {
  if (n == 0) return;
  if (p == nullptr || find(p, n) == nullptr) die(what, p, n);
  std::memset(p, 0x3c, n);
}

void count() {
  std::lock_guard<std::mutex> l(mu);
  ++launches;
}

}  // namespace stub

extern "C" long long stub_launch_count() { return stub::launches; }

// ---- HIP runtime -----------------------------------------------------------

hipError_t hipGetDevice(int* d) {
  *d = 0;
  return hipSuccess;
}
hipError_t hipMalloc(void** ptr, size_t n) {
  void* p = nullptr;
  if (posix_memalign(&p, 256, n == 0 ? 1 : n) != 0) return hipErrorOutOfMemory;
  std::lock_guard<std::mutex> l(stub::mu);
  stub::allocs().push_back({static_cast<char*>(p), n});
  *ptr = p;
  return hipSuccess;
}
hipError_t hipFree(void* p) {
  if (p == nullptr) return hipSuccess;
  std::lock_guard<std::mutex> l(stub::mu);
  auto& v = stub::allocs();
  for (size_t i = 0; i < v.size(); ++i)
    if (v[i].p == p) {
      std::free(p);
      v.erase(v.begin() + i);
      return hipSuccess;
    }
  std::fprintf(stderr, "STUB FAILURE: hipFree of %p, not an allocation\n", p);
  std::abort();
}
hipError_t hipMemset(void* p, int v, size_t n) {
  if (stub::find(p, n) == nullptr) stub::die("hipMemset", p, n);
  std::memset(p, v, n);
  return hipSuccess;
}
hipError_t hipMemcpy(void* dst, const void* src, size_t n, hipMemcpyKind) {
  stub::rd("hipMemcpy source", src, n);
  std::memcpy(dst, src, n);
  return hipSuccess;
}
hipError_t hipDeviceSynchronize(void) { return hipSuccess; }
hipError_t hipGetLastError(void) { return hipSuccess; }
const char* hipGetErrorString(hipError_t) { return "stub"; }
hipError_t hipFuncSetAttribute(const void*, hipFuncAttribute, int) { return hipSuccess; }
hipError_t hipEventCreate(hipEvent_t* e) {
  *e = new ihipEvent_t{0};
  return hipSuccess;
}
hipError_t hipEventDestroy(hipEvent_t e) {
  delete e;
  return hipSuccess;
}
hipError_t hipEventRecord(hipEvent_t e, hipStream_t) {
  e->id++;
  return hipSuccess;
}
hipError_t hipEventSynchronize(hipEvent_t) { return hipSuccess; }
hipError_t hipEventElapsedTime(float* ms, hipEvent_t, hipEvent_t) {
  *ms = 0.001f;
  return hipSuccess;
}

// ---- sizes and launchers -------------------------------------------------

namespace swsft {

namespace {
size_t spatial(const Plan& p, int S, int B, int C) {
  return (size_t)B * S * C * p.H * p.W * 2 * p.elem;
}
size_t coefb(const Plan& p, int S, int B, int C) { return coef_elems(p, S, B, C) * p.elem; }
size_t filt(const Plan& p, int Cin, int Cout) {
  return (size_t)p.L * p.n_out * Cout * p.n_in * Cin * 2 * p.elem;
}
unsigned char g_scratch_store[1];  // replaced by a registered allocation below
void* g_scratch = nullptr;
}  // namespace

int delta_rows(const Plan& p) { return (p.flags & SWSFT_PLAN_DELTA_SYM) ? p.L : 2 * p.L; }
size_t delta_fwd_theta_elems(const Plan& p) { return (size_t)2 * p.L * p.H; }
size_t delta_inv_theta_elems(const Plan& p) {
  return (p.flags & SWSFT_PLAN_DELTA_SYM) ? (size_t)2 * p.H * p.L : (size_t)2 * p.H * 2 * p.L;
}
size_t delta_fwd_table_elems(const Plan& p) { return (size_t)p.M * p.L * delta_rows(p); }
size_t delta_inv_table_elems(const Plan& p) { return (size_t)p.M * delta_rows(p) * p.Lp; }
bool small_path(const Plan& p, int Cin) {
  return p.H <= 16 && p.fft_ok && !(p.flags & SWSFT_PLAN_DFT_MATMUL) && !is_delta(p) &&
         p.n_in * Cin <= 32;
}
bool bn_supported(const Plan& p, int C) { return p.n_out * C <= 2048; }
size_t bn_workspace_bytes(const Plan& p, int B, int C) {
  const int rows = p.L * p.L * B - B;
  int nblk = (rows + 63) / 64;
  nblk = nblk < 1 ? 1 : (nblk > 256 ? 256 : nblk);
  return ((size_t)nblk * p.n_out * C + p.n_out * C) * sizeof(float);
}
size_t filter_grad_split_bytes(const Plan& p, int B, int C_in, int C_out) {
  // float plans: one chunk of partial sums per degree (exercises the buffer)
  return p.dtype == SWSFT_F32 ? (size_t)p.L * p.n_out * C_out * p.n_in * C_in * 2 * sizeof(float)
                              : 0;
}
int phase_collapse_max_channels(int n_spins) { return 320 / n_spins; }
bool mix_adj_dma_supported(const Plan& p, int Cin, int Cout) {
  return p.dtype == SWSFT_BF16 && (2 * Cin) % 64 == 0 && Cout % 4 == 0;
}

hipError_t register_scratch(int device) {
  if (device != 0) return hipErrorInvalidDevice;
  if (g_scratch == nullptr && hipMalloc(&g_scratch, kNoAllocScratchBytes) != hipSuccess)
    return hipErrorOutOfMemory;
  (void)g_scratch_store;
  return hipSuccess;
}
void* scratch_of(int device) { return device == 0 ? g_scratch : nullptr; }

hipError_t launch_tables(const Plan& p, hipStream_t) {
  stub::count();
  stub::wr("tab_fwd", p.tab_fwd, p.n_in * p.fwd_table_elems() * p.elem);
  stub::wr("tab_inv", p.tab_inv, p.n_out * p.inv_table_elems() * p.elem);
  stub::wr("tab_bwd_syn", p.tab_bwd_syn, p.n_in * p.inv_table_elems() * p.elem);
  stub::wr("tab_bwd_ana", p.tab_bwd_ana, p.n_out * p.fwd_table_elems() * p.elem);
  stub::wr("twiddle", p.twiddle, (size_t)p.W * sizeof(float2));
  return hipSuccess;
}
hipError_t launch_dft_matrix(const Plan& p, hipStream_t) {
  stub::count();
  stub::wr("dft_mat", p.dft_mat, (size_t)2 * p.M * 2 * p.W * p.elem);
  return hipSuccess;
}
hipError_t launch_dft_matrix_inv(const Plan& p, hipStream_t) {
  stub::count();
  stub::wr("dft_mat_inv", p.dft_mat_inv, (size_t)2 * p.W * dft_inv_pitch(p.M) * p.elem);
  return hipSuccess;
}
hipError_t launch_delta_tables(const Plan& p, hipStream_t) {
  stub::count();
  stub::wr("delta_theta_fwd", p.delta_theta_fwd, delta_fwd_theta_elems(p) * p.elem);
  stub::wr("delta_theta_inv", p.delta_theta_inv, delta_inv_theta_elems(p) * p.elem);
  stub::wr("delta_fwd", p.delta_fwd, p.n_in * delta_fwd_table_elems(p) * p.elem);
  stub::wr("delta_inv", p.delta_inv, p.n_out * delta_inv_table_elems(p) * p.elem);
  return hipSuccess;
}
hipError_t launch_dft_fwd(const Plan& p, int S, int B, int C, const void* x, void* X,
                          hipStream_t) {
  stub::count();
  stub::rd("dft_fwd x", x, spatial(p, S, B, C));
  stub::wr("dft_fwd X", X, xy_elems(p, S, B, C) * p.elem);
  return hipSuccess;
}
hipError_t launch_dft_inv(const Plan& p, int S, int B, int C, const void* Y, void* y,
                          hipStream_t) {
  stub::count();
  stub::rd("dft_inv Y", Y, xy_elems(p, S, B, C) * p.elem);
  stub::wr("dft_inv y", y, spatial(p, S, B, C));
  return hipSuccess;
}
hipError_t launch_lat_fwd(const Plan& p, int B, int C, const void* X, void* coef, hipStream_t) {
  stub::count();
  stub::rd("lat_fwd X", X, xy_elems(p, p.n_in, B, C) * p.elem);
  stub::rd("lat_fwd table", p.tab_fwd, p.n_in * p.fwd_table_elems() * p.elem);
  stub::wr("lat_fwd coef", coef, coefb(p, p.n_in, B, C));
  return hipSuccess;
}
hipError_t launch_lat_inv(const Plan& p, int B, int C, const void* coef, void* Y, hipStream_t) {
  stub::count();
  const int ldb = p.coef_ldb > 0 ? p.coef_ldb : B;
  const size_t row = (size_t)ldb * p.n_out * 2 * C * p.elem;  // one coefficient row (l, m)
  stub::rd("lat_inv coef", coef, ((size_t)p.L * p.L - 1) * row + (size_t)B * p.n_out * 2 * C * p.elem);
  stub::rd("lat_inv table", p.tab_inv, p.n_out * p.inv_table_elems() * p.elem);
  stub::wr("lat_inv Y", Y, xy_elems(p, p.n_out, B, C) * p.elem);
  return hipSuccess;
}
hipError_t launch_mix(const Plan& p, int B, int Cin, int Cout, const void* coef, const void* K,
                      void* out, hipStream_t) {
  stub::count();
  stub::rd("mix coef", coef, coefb(p, p.n_in, B, Cin));
  stub::rd("mix filters", K, filt(p, Cin, Cout));
  stub::wr("mix out", out, coefb(p, p.n_out, B, Cout));
  return hipSuccess;
}
hipError_t launch_mix_adj_dma(const Plan& p, int B, int Cin, int Cout, const void* coef,
                              const void* K, void* out, hipStream_t) {
  stub::count();
  stub::rd("mix_adj coef", coef, coefb(p, p.n_in, B, Cin));
  stub::rd("mix_adj filters", K, (size_t)p.L * p.n_in * Cin * p.n_out * Cout * 2 * p.elem);
  stub::wr("mix_adj out", out, coefb(p, p.n_out, B, Cout));
  return hipSuccess;
}
hipError_t launch_filter_adjoint(const Plan& p, int Cin, int Cout, const void* K, void* KH,
                                 hipStream_t) {
  stub::count();
  stub::rd("filter_adjoint K", K, filt(p, Cin, Cout));
  stub::wr("filter_adjoint KH", KH, filt(p, Cin, Cout));
  return hipSuccess;
}
hipError_t launch_filter_grad(const Plan& p, int B, int Cin, int Cout, const void* a,
                              const void* g, void* gK, void* part, hipStream_t) {
  stub::count();
  stub::rd("filter_grad a", a, coefb(p, p.n_in, B, Cin));
  stub::rd("filter_grad g", g, coefb(p, p.n_out, B, Cout));
  stub::wr("filter_grad gK", gK, filt(p, Cin, Cout));
  stub::wr("filter_grad partial sums", part, filter_grad_split_bytes(p, B, Cin, Cout));
  return hipSuccess;
}
hipError_t launch_small_fwd(const Plan& p, int B, int C, const void* x, void* coef, hipStream_t) {
  stub::count();
  stub::rd("small_fwd x", x, spatial(p, p.n_in, B, C));
  stub::wr("small_fwd coef", coef, coefb(p, p.n_in, B, C));
  return hipSuccess;
}
hipError_t launch_small_inv(const Plan& p, int B, int Cin, int Cout, const void* coef,
                            const void* K, void* y, hipStream_t) {
  stub::count();
  if (K != nullptr) {
    stub::rd("small_inv coef", coef, coefb(p, p.n_in, B, Cin));
    stub::rd("small_inv filters", K, filt(p, Cin, Cout));
  } else {
    stub::rd("small_inv coef", coef, coefb(p, p.n_out, B, Cout));
  }
  stub::wr("small_inv y", y, spatial(p, p.n_out, B, Cout));
  return hipSuccess;
}
hipError_t launch_batch_norm(const Plan& p, int B, int C, const void* a, const float* gamma,
                             const float2* beta, float, const float* var_in, float* var_out,
                             const void* skip, void* out, void* ws, hipStream_t) {
  stub::count();
  const size_t cs = coefb(p, p.n_out, B, C);
  stub::rd("batch_norm coef", a, cs);
  stub::rd("batch_norm gamma", gamma, (size_t)p.n_out * C * sizeof(float));
  if (beta) stub::rd("batch_norm beta", beta, (size_t)C * sizeof(float2));
  if (var_in) stub::rd("batch_norm var_in", var_in, (size_t)p.n_out * C * sizeof(float));
  if (skip) stub::rd("batch_norm skip", skip, cs);
  if (var_in == nullptr) stub::wr("batch_norm workspace", ws, bn_workspace_bytes(p, B, C));
  if (var_out) stub::wr("batch_norm var_out", var_out, (size_t)p.n_out * C * sizeof(float));
  stub::wr("batch_norm out", out, cs);
  return hipSuccess;
}
hipError_t launch_phase_collapse(const Plan& p, int B, int C, const void* x, const float2* W1,
                                 const float2* W2, const float2* bias, void* y, hipStream_t) {
  stub::count();
  stub::rd("phase_collapse x", x, spatial(p, p.n_out, B, C));
  stub::rd("phase_collapse W1", W1, (size_t)C * C * sizeof(float2));
  stub::rd("phase_collapse W2", W2, (size_t)C * p.n_out * C * sizeof(float2));
  stub::rd("phase_collapse bias", bias, (size_t)C * sizeof(float2));
  stub::wr("phase_collapse y", y, spatial(p, p.n_out, B, C));
  return hipSuccess;
}
hipError_t launch_delta_theta_fwd(const Plan& p, int B, int C, const void* X, void* CS,
                                  hipStream_t) {
  stub::count();
  stub::rd("delta_theta_fwd X", X, xy_elems(p, p.n_in, B, C) * p.elem);
  stub::wr("delta_theta_fwd CS", CS, delta_elems(p, p.n_in, B, C) * p.elem);
  return hipSuccess;
}
hipError_t launch_fused32_fwd(const Plan& p, int B, int C, const void* x, void* coef,
                              hipStream_t) {
  stub::count();
  stub::rd("fused32_fwd x", x, spatial(p, p.n_in, B, C));
  stub::rd("fused32_fwd table", p.tab_fwd, p.n_in * p.fwd_table_elems() * p.elem);
  stub::wr("fused32_fwd coef", coef, coefb(p, p.n_in, B, C));
  return hipSuccess;
}
hipError_t launch_fused32_inv(const Plan& p, int B, int C, const void* coef, void* y,
                              hipStream_t) {
  stub::count();
  const int ldb = p.coef_ldb > 0 ? p.coef_ldb : B;
  const size_t row = (size_t)ldb * p.n_out * 2 * C * p.elem;  // one coefficient row (l, m)
  stub::rd("fused32_inv coef", coef, ((size_t)p.L * p.L - 1) * row + (size_t)B * p.n_out * 2 * C * p.elem);
  stub::rd("fused32_inv table", p.tab_inv, p.n_out * p.inv_table_elems() * p.elem);
  stub::wr("fused32_inv y", y, spatial(p, p.n_out, B, C));
  return hipSuccess;
}
double mfma_probe_flops_per_wave_round(int dtype) {
  return dtype == SWSFT_BF16 ? 4.0 * 2 * 32 * 32 * 16 : 4.0 * 2 * 32 * 32 * 2;
}
hipError_t launch_mfma_probe(int, int, long long, int n_waves, float* out, hipStream_t) {
  stub::count();
  stub::wr("mfma_probe out", out, (size_t)n_waves * 64 * sizeof(float));
  return hipSuccess;
}
hipError_t launch_delta_theta_inv(const Plan& p, int B, int C, const void* G, void* Y,
                                  hipStream_t) {
  stub::count();
  stub::rd("delta_theta_inv G", G, delta_elems(p, p.n_out, B, C) * p.elem);
  stub::wr("delta_theta_inv Y", Y, xy_elems(p, p.n_out, B, C) * p.elem);
  return hipSuccess;
}

}  // namespace swsft
