// twiddles.cpp -- host generation of the twiddle table (float64 math, rounded once).
#include "twiddles.hpp"

#include <cmath>

#include "plan.hpp"

namespace rdfft {

HostC32 unit_root(long long j, long long M) {
  long long a = j % M;
  if (a < 0) a += M;
  // quadrant q and position r within it: angle = (pi/2) * (q + r/M), 0 <= r < M
  const long long q = (4 * a) / M;
  const long long r = 4 * a - q * M;
  const double half_pi = 1.57079632679489661923132169163975;
  double c, s;
  if (2 * r <= M) {
    const double phi = half_pi * (double)r / (double)M;
    c = std::cos(phi);
    s = std::sin(phi);
  } else {  // reflect about pi/4 so the argument stays in [0, pi/4]
    const double phi = half_pi * (double)(M - r) / (double)M;
    c = std::sin(phi);
    s = std::cos(phi);
  }
  double cc, ss;  // cos and sin of the full angle
  switch (q) {
    case 0: cc = c; ss = s; break;
    case 1: cc = -s; ss = c; break;
    case 2: cc = -c; ss = -s; break;
    default: cc = s; ss = -c; break;
  }
  return HostC32{(float)cc, (float)(-ss)};
}

std::vector<HostC32> build_twiddle_table() {
  std::vector<HostC32> t((size_t)kTableEntries);
  for (int logn = 0; logn <= kMaxLogN; ++logn) {
    for (int q = 1; q < num_passes(logn); ++q) {
      const int R = radix(logn, q), Ns = stride_before(logn, q);
      const int off = pass_table_offset(logn, q);
      const int L = tw_loaded(R);
      for (int k = 0; k < Ns; ++k)
        for (int r = 1; r <= L; ++r) t[(size_t)off + (size_t)k * L + r - 1] = unit_root((long long)r * k, (long long)Ns * R);
    }
    const int N = 1 << logn, off = post_table_offset(logn);
    const float inv_n = 1.0f / (2.0f * (float)N);
    for (int k = 0; k < N / 2; ++k) {
      const HostC32 w = unit_root(k, 2LL * N);                      // (cos, -sin)
      t[(size_t)off + k] = HostC32{0.5f * w.y, -0.5f * w.x};         // (1/2) (-i) W
      t[(size_t)off + N / 2 + k] = HostC32{inv_n * w.y, inv_n * w.x};  // (1/n) i conj(W)
    }
  }
  return t;
}

}  // namespace rdfft
