// rdfft_kernels.hip -- batched in-place rdFFT / irdFFT row kernels (spectra in the pairs
// layout) and the twiddle table.
#include <hip/hip_runtime.h>

#include "rows_kernel.hpp"

namespace rdfft {

// The library's only device-resident data: the twiddle factors of every plan.
__device__ __attribute__((aligned(16))) float2 g_twiddles[kTableEntries];

hipError_t launch_rdfft_rows(void* buf, int64_t rows, int logn, int storage, bool inv, const float2* tw,
                             hipStream_t stream, int) {
  return launch_rows_of_layout<false>(buf, rows, logn, storage, inv, tw, stream);
}

hipError_t upload_twiddles(const void* host, size_t bytes, const float2** dev_ptr) {
  hipError_t e = hipMemcpyToSymbol(HIP_SYMBOL(g_twiddles), host, bytes, 0, hipMemcpyHostToDevice);
  if (e != hipSuccess) return e;
  void* p = nullptr;
  e = hipGetSymbolAddress(&p, HIP_SYMBOL(g_twiddles));
  if (e != hipSuccess) return e;
  *dev_ptr = static_cast<const float2*>(p);
  return hipSuccess;
}

}  // namespace rdfft
