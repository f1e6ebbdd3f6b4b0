// rdfft_hc_kernels.hip -- the in-place row transforms with the spectrum in the paper's
// halfcomplex layout (Sec. 4.1, Memory Layout): the forward writes, and the inverse reads,
// Re Y_k at real slot k and Im Y_k at real slot n - k.  The arithmetic is that of the
// pairs-layout kernels (rdfft_kernels.hip), so the results equal theirs followed by the
// layout conversion bit for bit, in one pass over HBM instead of two.
#include <hip/hip_runtime.h>

#include "rows_kernel.hpp"

namespace rdfft {

hipError_t launch_rdfft_rows_hc(void* buf, int64_t rows, int logn, int storage, bool inv, const float2* tw,
                                hipStream_t stream) {
  return launch_rows_of_layout<true>(buf, rows, logn, storage, inv, tw, stream);
}

}  // namespace rdfft
