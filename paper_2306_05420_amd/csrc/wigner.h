// Wigner (small) d by the three-term recurrence in l, in float64: shared by
// the plan-time table kernels.
#pragma once

#include <hip/hip_runtime.h>

namespace swsft {

// d^{l0}_{m n}(theta) at l0 = max(|m|, |n|): sqrt(C(2 l0, a)) c^a s^b times a
// sign, c = cos(theta/2), s = sin(theta/2), a + b = 2 l0.  Evaluated as a
// running product so no factorial or power is formed on its own.
__device__ inline double wigner_seed(int m, int n, double c, double s) {
  const int am = m < 0 ? -m : m, an = n < 0 ? -n : n;
  const int l0 = am > an ? am : an;
  int a, b;
  bool neg;
  if (am >= an) {
    if (m == l0) { a = l0 + n; b = l0 - n; neg = (b & 1); }   // d_{l,n}
    else         { a = l0 - n; b = l0 + n; neg = false; }     // d_{-l,n}
  } else {
    if (n == l0) { a = l0 + m; b = l0 - m; neg = false; }     // d_{m,l}
    else         { a = l0 - m; b = l0 + m; neg = (b & 1); }   // d_{m,-l}
  }
  double v = 1.0;
  for (int i = 1; i <= a; ++i) v *= c * sqrt((double)(b + i) / (double)i);
  for (int i = 0; i < b; ++i) v *= s;
  return neg ? -v : v;
}

// d^l_{mn}(beta) for l = 0, 1, ... visited in order: at(l) is the value at
// degree l (0 below l0 = max(|m|, |n|)), advance_past(l) then moves the
// recurrence from degree l to l + 1,
//   d^{l+1} = (l+1)(2l+1) / sqrt(((l+1)^2-m^2)((l+1)^2-n^2))
//             * [ (cos b - m n/(l(l+1))) d^l - sqrt((l^2-m^2)(l^2-n^2)) / (l(2l+1)) d^{l-1} ].
struct WignerRec {
  int m, n, l0, l;
  double cb, prev, cur;
  __device__ void init(int m_, int n_, double beta) {
    m = m_;
    n = n_;
    const int am = m < 0 ? -m : m, an = n < 0 ? -n : n;
    l0 = am > an ? am : an;
    l = l0;
    cb = cos(beta);
    prev = 0.0;
    cur = wigner_seed(m, n, cos(0.5 * beta), sin(0.5 * beta));
  }
  __device__ double at(int deg) const { return deg < l0 ? 0.0 : cur; }
  __device__ void advance_past(int deg) {
    if (deg < l0) return;
    const double lp = l + 1.0;
    const double a = lp * (2.0 * l + 1.0) / sqrt((lp * lp - (double)m * m) * (lp * lp - (double)n * n));
    const double t1 = (l == 0) ? cb * cur : (cb - (double)m * n / (l * (l + 1.0))) * cur;
    const double t2 = (l > l0) ? sqrt(((double)l * l - (double)m * m) * ((double)l * l - (double)n * n)) /
                                     (l * (2.0 * l + 1.0)) * prev
                               : 0.0;
    prev = cur;
    cur = a * (t1 - t2);
    ++l;
  }
};

}  // namespace swsft
