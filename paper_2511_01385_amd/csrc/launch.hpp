// launch.hpp -- host-side launchers exported by the kernel translation units.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <algorithm>
#include <array>
#include <utility>

namespace rdfft {

// Storage types of the row kernels (the values of rdfft_dtype_t)
constexpr int kStorageF32 = 0, kStorageBF16 = 1, kStorageF16 = 2;

// Work-items per launch: each grid dimension holds fewer than 2^32 of them, so launches
// are split to stay at or below this.
constexpr int64_t kMaxGridThreads = (int64_t)1 << 31;

// In-place forward (inv = false) or inverse rdFFT of `rows` rows of 2^(logn+1) elements
// (rows >= 1) stored as `storage`.
hipError_t launch_rdfft_rows(void* buf, int64_t rows, int logn, int storage, bool inv, const float2* tw,
                             hipStream_t stream, int num_cu);
// The same transforms with the spectrum in the halfcomplex layout (the forward's output,
// the inverse's input).
hipError_t launch_rdfft_rows_hc(void* buf, int64_t rows, int logn, int storage, bool inv, const float2* tw,
                                hipStream_t stream);

// In-place conversion of `rows` packed spectra of 2^(logn+1) elements between the pairs
// layout and the halfcomplex layout (rows >= 1); half16 = 16-bit storage (bf16 or f16).
hipError_t launch_layout_convert(void* buf, int64_t rows, int logn, bool half16, bool to_halfcomplex,
                                 hipStream_t stream);

// Rows whose half-length N = n/2 is 2^a 3^b 5^c but not a power of two, N <= 16384
// (mixed_kernels.hip): the transforms and the layout converters, rows >= 1.
constexpr int64_t kMixedMaxHalf = 16384;
bool mixed_length_supported(int64_t n);
hipError_t launch_mixed_rows(void* buf, int64_t rows, int64_t n, int storage, bool inv, bool halfcomplex,
                             hipStream_t stream);
hipError_t launch_mixed_layout(void* buf, int64_t rows, int64_t n, bool half16, bool to_halfcomplex,
                               hipStream_t stream);

// Copies the host twiddle table to the current device; returns its device address.
hipError_t upload_twiddles(const void* host, size_t bytes, const float2** dev_ptr);

struct BcaArgs {
  const void* x;
  const void* c;      // packed spectra [q][kb][p]
  void* y;            // forward output, or backward upstream gradient gy
  void* dx;           // backward only
  float* dc;          // backward only
  int64_t tokens;
  int q, kb, logp;    // p = 2^logp
  int storage;        // kStorageF32, kStorageBF16 or kStorageF16
};

hipError_t launch_bca_forward(const BcaArgs& a, const float2* tw, hipStream_t stream, int num_cu);

// Independent layers of one shape (bca_forward_batched / bca_backward_batched): up to
// kMaxBatch of them per launch, layer b of a launch in grid row blockIdx.y.
constexpr int kMaxBatch = 32;
struct BcaBatch {
  int count;
  const void* x[kMaxBatch];
  const void* c[kMaxBatch];
  void* y[kMaxBatch];  // forward output, or backward upstream gradient gy
  void* dx[kMaxBatch];
  float* dc[kMaxBatch];
};
// whether layers of this shape run in one grid per launch (the wave kernels' square layers;
// the backward only with dx apart from gy); other batches run layer by layer
bool bca_batch_fused(int logp, int q, int kb, int storage, bool backward);
// shape: BcaArgs whose pointers are unused; the backward zeroes and fills every dc
hipError_t launch_bca_forward_batched(const BcaArgs& shape, const BcaBatch& b, const float2* tw, hipStream_t stream,
                                      int num_cu);
hipError_t launch_bca_backward_batched(const BcaArgs& shape, const BcaBatch& b, const float2* tw, hipStream_t stream,
                                       int num_cu);
// also zeroes dc first and transforms it to the time domain afterwards
hipError_t launch_bca_backward(const BcaArgs& a, const float2* tw, hipStream_t stream, int num_cu);

// whether the fused forward (or backward) kernel handles p = 2^logp with q x kb blocks
bool bca_shape_supported(int logp, int q, int kb, bool backward);

// The multi-pass layer for 8192 < p <= 65536 (bca_multipass.hip), q * kb <= 65535.  In
// place (y == x in the forward, dx == gy in the backward, so q == kb) it takes at most
// kMpMaxInPlaceBlocks blocks: a per-bin product holds that many values.  The backward
// launcher expects dc zeroed and leaves it as packed spectra.
constexpr int kMpMaxInPlaceBlocks = 8;
bool bca_multipass_supported(int logp, int q, int kb, bool backward);
// The forward of a single circulant (q == kb == 1) of p = 2^(kCirculantLogN+1) = 8192 as
// one row kernel per token (bca_multipass.hip), the spectrum handed from the forward to
// the inverse transform in registers.
constexpr int kCirculantLogN = 12;
hipError_t launch_bca_circulant(const BcaArgs& a, const float2* tw, hipStream_t stream);
hipError_t launch_bca_multipass(const BcaArgs& a, bool backward, const float2* tw, hipStream_t stream, int num_cu);

}  // namespace rdfft
