// rows_kernel.hpp -- the batched in-place row transform kernel and its launcher, shared by
// rdfft_kernels.hip (spectra in the pairs layout) and rdfft_hc_kernels.hip (spectra in the
// halfcomplex layout of Sec. 4.1, Memory Layout).
//
// A workgroup owns RW whole rows (RowPlan::RW); every row is read once from HBM into
// registers, transformed through LDS, and written back to the same addresses, so the
// call needs no memory beyond the caller's buffer (Sec. 4.1, rdFFT algorithm).  Every
// thread's loads of a row feed the LDS writes of the first exchange, which a row
// barrier separates from any thread's stores, so the row is read completely before any
// of its slots is written, whatever the layout.
#pragma once

#include <hip/hip_runtime.h>

#include "fft_device.hpp"
#include "launch.hpp"

namespace rdfft {

// exchange rounds per pass of the row kernels
template <int LOGN, class Acc>
constexpr int row_chunks() {  // 16-bit storage: the bf16 table
  return std::is_same<Acc, GlobalF32>::value ? kChunks[LOGN] : kChunksBf16[LOGN];
}

// HC: the spectrum side of the row (the forward's output, the inverse's input) is in the
// halfcomplex layout; the signal side is always the pairs (x_{2m}, x_{2m+1}).
template <int LOGN, class Acc, class Elem, bool INV, bool HC>
__global__ void __launch_bounds__(RowPlan<LOGN>::WG) rdfft_rows_kernel(Elem* buf, int64_t rows,
                                                                        const float2* __restrict__ tw) {
  constexpr int CH = row_chunks<LOGN, Acc>();
  using P = RowPlan<LOGN, CH>;
  constexpr int LDS_ROW = P::LDS_F2 > 0 ? P::LDS_F2 : 1;
  __shared__ float2 lds[P::RW * LDS_ROW];
  const int tid = threadIdx.x;
  const int rho = tid / P::TPR;
  const int t = tid - rho * P::TPR;
  const int64_t row = (int64_t)blockIdx.x * P::RW + rho;
  const bool active = row < rows;
  Elem* const rp = buf + (active ? row : 0) * (int64_t)P::N;
  const Acc acc{rp};
  float2* my = lds + rho * LDS_ROW;
  if constexpr (HC) {
    using H = Halfcomplex<Acc>;
    const H hc{reinterpret_cast<typename H::scalar_t*>(rp), P::N};
    if constexpr (!INV) row_forward<LOGN, false, Acc, H, CH, mirror_ok<LOGN>()>(t, active, acc, hc, my, tw);
    else row_inverse<LOGN, false, H, Acc, CH>(t, active, hc, acc, my, tw);
  } else {
    if constexpr (!INV) row_forward<LOGN, false, Acc, Acc, CH, mirror_ok<LOGN>()>(t, active, acc, acc, my, tw);
    else row_inverse<LOGN, false, Acc, Acc, CH>(t, active, acc, acc, my, tw);
  }
}

template <int LOGN, class Acc, class Elem, bool INV, bool HC>
static hipError_t launch_rows(void* buf, int64_t rows, const float2* tw, hipStream_t stream) {
  using P = RowPlan<LOGN>;
  // keep every launch within the grid limit
  const int64_t max_blocks = kMaxGridThreads / P::WG;
  Elem* base = static_cast<Elem*>(buf);
  for (int64_t r0 = 0; r0 < rows;) {
    const int64_t blocks = std::min<int64_t>((rows - r0 + P::RW - 1) / P::RW, max_blocks);
    const int64_t nrows = std::min<int64_t>(blocks * P::RW, rows - r0);
    hipLaunchKernelGGL((rdfft_rows_kernel<LOGN, Acc, Elem, INV, HC>), dim3((unsigned)blocks), dim3(P::WG), 0, stream,
                       base + r0 * (int64_t)P::N, nrows, tw);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    r0 += nrows;
  }
  return hipSuccess;
}

using RowLauncher = hipError_t (*)(void*, int64_t, const float2*, hipStream_t);

template <class Acc, class Elem, bool HC, int... L>
static std::array<RowLauncher, sizeof...(L)> make_row_table(bool inv, std::integer_sequence<int, L...>) {
  return {(inv ? &launch_rows<L, Acc, Elem, true, HC> : &launch_rows<L, Acc, Elem, false, HC>)...};
}

// [storage][inverse][logn] launchers of one layout
template <bool HC>
static hipError_t launch_rows_of_layout(void* buf, int64_t rows, int logn, int storage, bool inv, const float2* tw,
                                        hipStream_t stream) {
  static const auto seq = std::make_integer_sequence<int, kMaxLogN + 1>{};
  static const std::array<RowLauncher, kMaxLogN + 1> tables[3][2] = {
      {make_row_table<GlobalF32, float2, HC>(false, seq), make_row_table<GlobalF32, float2, HC>(true, seq)},
      {make_row_table<GlobalBF16, uint32_t, HC>(false, seq), make_row_table<GlobalBF16, uint32_t, HC>(true, seq)},
      {make_row_table<GlobalF16, uint32_t, HC>(false, seq), make_row_table<GlobalF16, uint32_t, HC>(true, seq)}};
  return tables[storage][inv ? 1 : 0][logn](buf, rows, tw, stream);
}

}  // namespace rdfft
