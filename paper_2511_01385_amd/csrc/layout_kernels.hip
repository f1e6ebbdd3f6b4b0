// layout_kernels.hip -- in-place conversion between the two packed spectrum layouts.
//
// pairs       (this library):  P[0] = (Y_0, Y_{n/2}),  P[k] = (Re Y_k, Im Y_k), 1 <= k < N
// halfcomplex (Sec. 4.1, the paper's layout): slot k = Re Y_k for 0 <= k <= n/2 and
//             slot n-k = Im Y_k for 1 <= k < n/2
// with n = 2N.  Pair slot k thus maps to the real slots (k, n-k), and pair slot 0 to
// (0, N).  The conversion only moves values, bit for bit.  Each row is read completely
// into registers before any of its slots is written, so the rows need no scratch.
#include <hip/hip_runtime.h>

#include "fft_device.hpp"
#include "launch.hpp"

namespace rdfft {

template <int LOGN>
struct LayoutPlan {
  static constexpr int N = 1 << LOGN;  // pair slots per row
  static constexpr int TPR = N < 1024 ? N : 1024;
  static constexpr int KPT = N / TPR;  // pair slots per thread
  static constexpr int RW = TPR >= 256 ? 1 : 256 / TPR;
  static constexpr int WG = TPR * RW;
};

// Pair is the storage of one pair slot (two scalars), Scalar that of one real slot.
template <int LOGN, class Pair, class Scalar, bool TO_HC>
__global__ void __launch_bounds__(LayoutPlan<LOGN>::WG) layout_kernel(Scalar* buf, int64_t rows) {
  using L = LayoutPlan<LOGN>;
  constexpr int N = L::N, TPR = L::TPR, KPT = L::KPT;
  const int tid = threadIdx.x;
  const int rho = tid / TPR;
  const int t = tid - rho * TPR;
  const int64_t row = (int64_t)blockIdx.x * L::RW + rho;
  const bool active = row < rows;
  Scalar* const s = buf + (active ? row : 0) * (int64_t)(2 * N);  // real slots of the row
  Pair* const p = reinterpret_cast<Pair*>(s);                     // its pair slots

  // slot k = t + j*TPR; its two real slots in the halfcomplex layout are (k, 2N-k), or
  // (0, N) for k == 0
  Scalar a[KPT], b[KPT];
  static_for<KPT>([&](auto jc) {
    constexpr int j = decltype(jc)::value;
    const int k = t + j * TPR;
    if constexpr (TO_HC) {
      const Pair v = p[k];
      a[j] = v.x;
      b[j] = v.y;
    } else {
      a[j] = s[k];
      b[j] = s[k == 0 ? N : 2 * N - k];
    }
  });
  // Every load of the row must have returned before any thread of the row stores: no
  // store depends on another thread's loads, and the workgroup barrier orders LDS, not
  // global memory, so the compiler may otherwise sink the loads below it.  The empty asm
  // statements consume the loaded values ahead of the barrier.
#pragma unroll
  for (int j = 0; j < KPT; ++j) asm volatile("" ::"v"(a[j]), "v"(b[j]));
  row_sync<TPR>();
  if (!active) return;
  static_for<KPT>([&](auto jc) {
    constexpr int j = decltype(jc)::value;
    const int k = t + j * TPR;
    if constexpr (TO_HC) {
      s[k] = a[j];
      s[k == 0 ? N : 2 * N - k] = b[j];
    } else {
      Pair v;
      v.x = a[j];
      v.y = b[j];
      p[k] = v;
    }
  });
}

struct alignas(4) U16x2 {
  uint16_t x, y;
};

template <int LOGN, class Pair, class Scalar, bool TO_HC>
static hipError_t launch_layout(void* buf, int64_t rows, hipStream_t stream) {
  using L = LayoutPlan<LOGN>;
  const int64_t max_blocks = kMaxGridThreads / L::WG;
  Scalar* base = static_cast<Scalar*>(buf);
  for (int64_t r0 = 0; r0 < rows;) {
    const int64_t blocks = std::min<int64_t>((rows - r0 + L::RW - 1) / L::RW, max_blocks);
    const int64_t nrows = std::min<int64_t>(blocks * L::RW, rows - r0);
    hipLaunchKernelGGL((layout_kernel<LOGN, Pair, Scalar, TO_HC>), dim3((unsigned)blocks), dim3(L::WG), 0, stream,
                       base + r0 * (int64_t)(2 * L::N), nrows);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    r0 += nrows;
  }
  return hipSuccess;
}

using LayoutLauncher = hipError_t (*)(void*, int64_t, hipStream_t);

template <int... L>
static std::array<LayoutLauncher, sizeof...(L)> make_layout_table(bool bf16, bool to_hc,
                                                                 std::integer_sequence<int, L...>) {
  return {(bf16 ? (to_hc ? &launch_layout<L, U16x2, uint16_t, true> : &launch_layout<L, U16x2, uint16_t, false>)
                : (to_hc ? &launch_layout<L, float2, float, true> : &launch_layout<L, float2, float, false>))...};
}

hipError_t launch_layout_convert(void* buf, int64_t rows, int logn, bool half16, bool to_halfcomplex,
                                 hipStream_t stream) {
  static const auto seq = std::make_integer_sequence<int, kMaxLogN + 1>{};
  static const std::array<LayoutLauncher, kMaxLogN + 1> tables[4] = {
      make_layout_table(false, false, seq), make_layout_table(false, true, seq), make_layout_table(true, false, seq),
      make_layout_table(true, true, seq)};
  return tables[(half16 ? 2 : 0) + (to_halfcomplex ? 1 : 0)][logn](buf, rows, stream);
}

}  // namespace rdfft
