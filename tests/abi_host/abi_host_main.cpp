// Drives every entry point of include/swsft.h against the host stubs of
// hip_stub.cpp: valid calls on buffers of exactly the documented sizes
// (AddressSanitizer reports any access past them), and invalid calls that
// must be refused before anything is launched.  Prints "ALL OK" and exits 0
// when every expectation holds.
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <thread>
#include <vector>

#include <hip/hip_runtime_api.h>

#include "../../include/swsft.h"

extern "C" long long stub_launch_count();

namespace {

int g_fail = 0;

#define EXPECT(cond)                                                           \
  do {                                                                         \
    if (!(cond)) {                                                             \
      std::fprintf(stderr, "FAILED %s:%d: %s (%s)\n", __FILE__, __LINE__, #cond, \
                   swsft_last_error());                                        \
      ++g_fail;                                                                \
    }                                                                          \
  } while (0)

struct Buf {
  void* p = nullptr;
  size_t n = 0;
  explicit Buf(size_t bytes) : n(bytes) {
    if (hipMalloc(&p, bytes) != hipSuccess) std::abort();
    std::memset(p, 0, bytes);
  }
  ~Buf() { (void)hipFree(p); }
  Buf(const Buf&) = delete;
  Buf& operator=(const Buf&) = delete;
};

struct Shape {
  int H, L;
  std::vector<int> si, so;
  int dtype;
  unsigned flags;
  int B, Ci, Co;
};

size_t elem(int dtype) { return dtype == SWSFT_BF16 ? 2 : 4; }

void exercise(const Shape& s) {
  std::printf("shape H=%d L=%d S_in=%zu S_out=%zu dtype=%d flags=%u B=%d C=%d->%d\n", s.H, s.L,
              s.si.size(), s.so.size(), s.dtype, s.flags, s.B, s.Ci, s.Co);
  swsft_plan p = nullptr;
  EXPECT(swsft_plan_create_ex(s.H, s.H, s.L, s.si.data(), (int)s.si.size(), s.so.data(),
                              (int)s.so.size(), s.dtype, s.flags, &p) == SWSFT_OK);
  if (p == nullptr) return;
  const size_t e = elem(s.dtype);
  const int Si = (int)s.si.size(), So = (int)s.so.size(), B = s.B, L = s.L, H = s.H;
  const size_t xs = (size_t)B * Si * s.Ci * H * H * 2 * e;
  const size_t ys = (size_t)B * So * s.Co * H * H * 2 * e;
  const size_t ai = (size_t)L * L * B * Si * s.Ci * 2 * e;
  const size_t ao = (size_t)L * L * B * So * s.Co * 2 * e;
  const size_t ks = (size_t)L * So * s.Co * Si * s.Ci * 2 * e;
  Buf x(xs), y(ys), a_in(ai), a_out(ao), K(ks), gx(xs), gK(ks), gy(ys), cx(ai);
  const bool delta = (s.flags & (SWSFT_PLAN_DELTA | SWSFT_PLAN_DELTA_SYM)) != 0;

  {  // forward
    const size_t n = swsft_workspace_bytes(p, SWSFT_OP_FORWARD, B, s.Ci, 0);
    EXPECT(n > 0);
    Buf ws(n);
    EXPECT(swsft_forward(p, B, s.Ci, x.p, a_in.p, ws.p, n, nullptr) == SWSFT_OK);
    EXPECT(swsft_forward(p, B, s.Ci, x.p, a_in.p, ws.p, n - 1, nullptr) == SWSFT_E_WORKSPACE);
    EXPECT(swsft_forward(p, B, s.Ci, x.p, x.p, ws.p, n, nullptr) == SWSFT_E_INVALID);
    EXPECT(swsft_forward(p, B, s.Ci, x.p, ws.p, ws.p, n, nullptr) == SWSFT_E_INVALID);
    EXPECT(swsft_forward(p, 0, s.Ci, x.p, a_in.p, ws.p, n, nullptr) == SWSFT_E_INVALID);
  }
  {  // inverse
    const size_t n = swsft_workspace_bytes(p, SWSFT_OP_INVERSE, B, 0, s.Co);
    Buf ws(n);
    EXPECT(swsft_inverse(p, B, s.Co, a_out.p, y.p, ws.p, n, nullptr) == SWSFT_OK);
    EXPECT(swsft_inverse(p, B, s.Co, a_out.p, ws.p, ws.p, n, nullptr) == SWSFT_E_INVALID);
  }
  {  // the layer, with timing on, and the layer saving F x
    const size_t n = swsft_workspace_bytes(p, SWSFT_OP_CONV, B, s.Ci, s.Co);
    Buf ws(n);
    EXPECT(swsft_stage_timing(p, 1) == SWSFT_OK);
    EXPECT(spin_sph_conv_forward(p, B, s.Ci, s.Co, x.p, K.p, y.p, ws.p, n, nullptr) == SWSFT_OK);
    double ms[16] = {0};
    long long cnt[16] = {0};
    EXPECT(swsft_stage_times(p, ms, cnt, 16) > 0);
    long long total = 0;
    for (long long c : cnt) total += c;
    EXPECT(total > 0);
    EXPECT(swsft_stage_timing(p, 0) == SWSFT_OK);
    EXPECT(spin_sph_conv_forward(p, B, s.Ci, s.Co, x.p, K.p, x.p, ws.p, n, nullptr) ==
           SWSFT_E_INVALID);  // y overlaps x
    EXPECT(spin_sph_conv_forward(p, B, s.Ci, s.Co, x.p, y.p, y.p, ws.p, n, nullptr) ==
           SWSFT_E_INVALID);  // y overlaps the filters
    if (!delta) {
      EXPECT(spin_sph_conv_forward_train(p, B, s.Ci, s.Co, x.p, K.p, y.p, cx.p, ws.p, n,
                                         nullptr) == SWSFT_OK);
      EXPECT(spin_sph_conv_forward_train(p, B, s.Ci, s.Co, x.p, K.p, y.p, ws.p, ws.p, n,
                                         nullptr) == SWSFT_E_INVALID);
    }
    const swsft_status na = spin_sph_conv_forward_noalloc(p, B, s.Ci, s.Co, x.p, K.p, y.p, nullptr);
    EXPECT(na == SWSFT_OK || (na == SWSFT_E_UNSUPPORTED && n > (size_t(128) << 20)));
  }
  if (!delta) {  // backward: both gradients, from x and from saved coefficients, each alone
    const size_t n = swsft_workspace_bytes(p, SWSFT_OP_CONV_BACKWARD, B, s.Ci, s.Co);
    Buf ws(n);
    EXPECT(spin_sph_conv_backward(p, B, s.Ci, s.Co, x.p, nullptr, K.p, gy.p, gx.p, gK.p, ws.p, n,
                                  nullptr) == SWSFT_OK);
    EXPECT(spin_sph_conv_backward(p, B, s.Ci, s.Co, nullptr, cx.p, K.p, gy.p, gx.p, gK.p, ws.p,
                                  n, nullptr) == SWSFT_OK);
    EXPECT(spin_sph_conv_backward(p, B, s.Ci, s.Co, nullptr, nullptr, K.p, gy.p, gx.p, nullptr,
                                  ws.p, n, nullptr) == SWSFT_OK);
    EXPECT(spin_sph_conv_backward(p, B, s.Ci, s.Co, x.p, nullptr, nullptr, gy.p, nullptr, gK.p,
                                  ws.p, n, nullptr) == SWSFT_OK);
    EXPECT(spin_sph_conv_backward(p, B, s.Ci, s.Co, x.p, nullptr, K.p, gy.p, gx.p, gK.p, gx.p, n,
                                  nullptr) == SWSFT_E_INVALID);  // workspace overlaps grad_x
  }
  // the mixing alone
  EXPECT(spin_sph_mix(p, B, s.Ci, s.Co, a_in.p, K.p, a_out.p, nullptr) == SWSFT_OK);
  EXPECT(spin_sph_mix(p, B, s.Ci, s.Co, a_in.p, K.p, K.p, nullptr) == SWSFT_E_INVALID);
  bool has0 = false;
  for (int v : s.so) has0 |= v == 0;
  if (has0 && s.Co <= 160) {  // phase collapse, out of place and in place
    Buf W1((size_t)s.Co * s.Co * 8), W2((size_t)s.Co * So * s.Co * 8), b((size_t)s.Co * 8);
    Buf y2(ys);
    EXPECT(spin_sph_phase_collapse(p, B, s.Co, y.p, W1.p, W2.p, b.p, y2.p, nullptr) == SWSFT_OK);
    EXPECT(spin_sph_phase_collapse(p, B, s.Co, y.p, W1.p, W2.p, b.p, y.p, nullptr) == SWSFT_OK);
  }
  if (So * s.Co <= 2048) {  // batch norm: batch statistics with skip, given statistics in place
    const size_t n = swsft_workspace_bytes(p, SWSFT_OP_BATCH_NORM, B, 1, s.Co);
    Buf ws(n), gamma((size_t)So * s.Co * 4), beta((size_t)s.Co * 8), var((size_t)So * s.Co * 4);
    Buf skip(ao), out(ao);
    EXPECT(spin_sph_spectral_batch_norm(p, B, s.Co, a_out.p, (const float*)gamma.p, beta.p, 1e-5f,
                                        nullptr, (float*)var.p, skip.p, out.p, ws.p, n,
                                        nullptr) == SWSFT_OK);
    EXPECT(spin_sph_spectral_batch_norm(p, B, s.Co, a_out.p, (const float*)gamma.p, nullptr,
                                        1e-5f, (const float*)var.p, nullptr, nullptr, a_out.p,
                                        ws.p, n, nullptr) == SWSFT_OK);
    EXPECT(spin_sph_spectral_batch_norm(p, B, s.Co, a_out.p, (const float*)gamma.p, nullptr,
                                        1e-5f, nullptr, nullptr, nullptr, out.p, a_out.p, n,
                                        nullptr) == SWSFT_E_INVALID);  // workspace overlaps coef
  }
  {  // table read-back into exactly sized host memory
    const size_t Hp = (size_t)(H + 7) / 8 * 8, Lp = (size_t)(L + 31) / 32 * 32;
    const size_t fb = (size_t)(2 * L - 1) * L * Hp * e, ib = (size_t)(2 * L - 1) * H * Lp * e;
    std::vector<unsigned char> hf(fb), hi(ib);
    EXPECT(swsft_plan_table(p, 0, 0, hf.data(), fb) == SWSFT_OK);
    EXPECT(swsft_plan_table(p, 1, So - 1, hi.data(), ib) == SWSFT_OK);
    EXPECT(swsft_plan_table(p, 0, 0, hf.data(), fb - 1) == SWSFT_E_INVALID);
    EXPECT(swsft_plan_table(p, 0, Si, hf.data(), fb) == SWSFT_E_INVALID);
  }
  swsft_plan_destroy(p);
}

void block(int dtype) {
  const int S[2] = {0, 1};
  const int C = 8, B = 3, Hi = 32, Ho = 16, L = 8;
  swsft_plan pi = nullptr, po = nullptr;
  EXPECT(swsft_plan_create(Hi, Hi, L, S, 2, S, 2, dtype, &pi) == SWSFT_OK);
  EXPECT(swsft_plan_create(Ho, Ho, L, S, 2, S, 2, dtype, &po) == SWSFT_OK);
  const size_t e = elem(dtype);
  Buf x((size_t)B * 2 * C * Hi * Hi * 2 * e), y((size_t)B * 2 * C * Ho * Ho * 2 * e);
  Buf K1((size_t)L * 2 * C * 2 * C * 2 * e), K2((size_t)L * 2 * C * 2 * C * 2 * e);
  Buf g1(2 * C * 4), g2(2 * C * 4), b1(C * 8), b2(C * 8), v1(2 * C * 4), v2(2 * C * 4);
  Buf w11(C * C * 8), w12(C * 2 * C * 8), bb1(C * 8), w21(C * C * 8), w22(C * 2 * C * 8), bb2(C * 8);
  swsft_block_params prm{K1.p, K2.p, (const float*)g1.p, b1.p, (const float*)g2.p, b2.p,
                         w11.p, w12.p, bb1.p, w21.p, w22.p, bb2.p, 1e-5f,
                         (float*)v1.p, (float*)v2.p};
  const size_t n = swsft_block_workspace_bytes(pi, po, B, C);
  EXPECT(n > 0);
  Buf ws(n);
  EXPECT(spin_sph_residual_block_forward(pi, po, B, C, x.p, &prm, y.p, ws.p, n, nullptr) ==
         SWSFT_OK);
  EXPECT(spin_sph_residual_block_forward(pi, po, B, C, x.p, &prm, y.p, ws.p, n - 1, nullptr) ==
         SWSFT_E_WORKSPACE);
  swsft_plan_destroy(pi);
  swsft_plan_destroy(po);
}

void timing_from_threads() {
  // calls on a timing-enabled plan from several threads: the record stays
  // consistent (every launch counted once)
  const int S[1] = {0};
  swsft_plan p = nullptr;
  EXPECT(swsft_plan_create(32, 32, 16, S, 1, S, 1, SWSFT_F32, &p) == SWSFT_OK);
  const int B = 2, C = 4;
  const size_t xs = (size_t)B * C * 32 * 32 * 8, as = (size_t)16 * 16 * B * C * 8;
  const size_t n = swsft_workspace_bytes(p, SWSFT_OP_FORWARD, B, C, 0);
  EXPECT(swsft_stage_timing(p, 1) == SWSFT_OK);
  const int kThreads = 4, kCalls = 50;
  std::vector<std::thread> th;
  for (int t = 0; t < kThreads; ++t)
    th.emplace_back([&] {
      Buf x(xs), a(as), ws(n);
      for (int i = 0; i < kCalls; ++i)
        EXPECT(swsft_forward(p, B, C, x.p, a.p, ws.p, n, nullptr) == SWSFT_OK);
    });
  for (auto& t : th) t.join();
  double ms[16] = {0};
  long long cnt[16] = {0};
  swsft_stage_times(p, ms, cnt, 16);
  EXPECT(cnt[0] == kThreads * kCalls && cnt[1] == kThreads * kCalls);  // dft_fwd, lat_fwd
  swsft_plan_destroy(p);
}

}  // namespace

int main() {
  const std::vector<Shape> shapes = {
      {16, 8, {0}, {0, 1}, SWSFT_F32, 0, 1, 4, 4},                     // small-grid path
      {32, 16, {0, 1}, {0, 1}, SWSFT_F32, 0, 4, 16, 8},                // float, split filter gradient
      {64, 32, {1, -2}, {2, 0}, SWSFT_BF16, 0, 2, 64, 64},             // bf16, |s| = 2
      {64, 32, {0, 1}, {0, 1, -1}, SWSFT_BF16, 0, 3, 32, 44},          // ragged bf16 mixing
      {64, 32, {0}, {0, 1}, SWSFT_F32, SWSFT_PLAN_DELTA_SYM, 2, 8, 8},  // Delta route
      {64, 32, {0}, {0}, SWSFT_BF16, SWSFT_PLAN_DELTA, 1, 8, 8},
      {96, 48, {0, 1}, {1}, SWSFT_F32, SWSFT_PLAN_DFT_MATMUL, 2, 3, 5},  // DFT-matrix route
      {256, 128, {0, 1}, {0, 1}, SWSFT_BF16, 0, 2, 16, 16},            // the 256 x 256 grid
  };
  for (const Shape& s : shapes) exercise(s);
  block(SWSFT_F32);
  block(SWSFT_BF16);
  timing_from_threads();
  {
    // the MFMA probe writes exactly 64 floats per wave; bad arguments are refused
    Buf out((size_t)8 * 64 * sizeof(float));
    double flops = 0.0;
    EXPECT(swsft_probe_mfma(SWSFT_BF16, 1, 10, 8, (float*)out.p, &flops, nullptr) == SWSFT_OK);
    EXPECT(flops == 8.0 * 10 * 4 * 2 * 32 * 32 * 16);
    EXPECT(swsft_probe_mfma(SWSFT_F32, 0, 10, 8, (float*)out.p, nullptr, nullptr) == SWSFT_OK);
    EXPECT(swsft_probe_mfma(SWSFT_BF16, 1, 10, 6, (float*)out.p, nullptr, nullptr) == SWSFT_E_INVALID);
    EXPECT(swsft_probe_mfma(SWSFT_BF16, 1, 0, 8, (float*)out.p, nullptr, nullptr) == SWSFT_E_INVALID);
    EXPECT(swsft_probe_mfma(7, 1, 10, 8, (float*)out.p, nullptr, nullptr) == SWSFT_E_INVALID);
    EXPECT(swsft_probe_mfma(SWSFT_BF16, 1, 10, 8, nullptr, nullptr, nullptr) == SWSFT_E_INVALID);
  }
  std::printf("%lld stub launches\n", stub_launch_count());
  if (g_fail) {
    std::printf("%d expectation(s) failed\n", g_fail);
    return 1;
  }
  std::printf("ALL OK\n");
  return 0;
}
