// bca_kernels.hip -- dispatch of the fused block-circulant layer (Sec. 3.3, Eqs. (4)-(5))
// to the kernels of bca_kernels.hpp (instantiated per storage type in
// bca_store_{f32,bf16,f16}.hip) and the multi-pass layer of bca_multipass.hip, plus the
// two small kernels every storage type shares: the fill of dc and the second stage of
// the two-stage dC sum.
#include <hip/hip_runtime.h>

#include "bca_kernels.hpp"

namespace rdfft {

// Second stage of the two-stage dC sum: dc[e] += the partials of workgroups
// b in [blockIdx.y*kReduceGroup, +kReduceGroup) (zeroed dc, one float32 atomic pair per
// thread and group of workgroups).  Workgroup b's slot e lies at
// stage[(b + c*groups)*tile_f2 + e - c*chunk], c = e / chunk.
__global__ void __launch_bounds__(256) bca_dc_reduce_kernel(const float2* __restrict__ stage, float* __restrict__ dc,
                                                            int qkn, int chunk, int groups, int64_t tile_f2) {
  const int e = blockIdx.x * 256 + threadIdx.x;
  if (e >= qkn) return;
  const int ch = e / chunk;
  const int b0 = blockIdx.y * kReduceGroup;
  const int b1 = b0 + kReduceGroup < groups ? b0 + kReduceGroup : groups;
  const float2* p = stage + ((int64_t)ch * groups + b0) * tile_f2 + (e - ch * chunk);
  float2 v = make_float2(0.f, 0.f);
#pragma unroll 8
  for (int b = b0; b < b1; ++b, p += tile_f2) v = c_add(v, *p);
  unsafeAtomicAdd(dc + 2 * (int64_t)e, v.x);
  unsafeAtomicAdd(dc + 2 * (int64_t)e + 1, v.y);
}

__global__ void fill_zero_kernel(float* __restrict__ p, int64_t count) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < count; i += (int64_t)gridDim.x * blockDim.x)
    p[i] = 0.f;
}

hipError_t launch_fill_zero(float* p, int64_t count, hipStream_t stream) {
  const int blocks = (int)std::min<int64_t>((count + 255) / 256, 1024);
  hipLaunchKernelGGL(fill_zero_kernel, dim3(blocks), dim3(256), 0, stream, p, count);
  return hipGetLastError();
}

hipError_t launch_dc_reduce(const float2* stage, float* dc, int qkn, int chunk, int groups, int64_t tile_f2,
                            hipStream_t stream) {
  const dim3 rgrid((unsigned)((qkn + 255) / 256), (unsigned)((groups + kReduceGroup - 1) / kReduceGroup));
  hipLaunchKernelGGL(bca_dc_reduce_kernel, rgrid, dim3(256), 0, stream, stage, dc, qkn, chunk, groups, tile_f2);
  return hipGetLastError();
}

static const BcaStoreTables& store_tables(int storage) {
  static const BcaStoreTables t[kStorages] = {bca_tables_f32(), bca_tables_bf16(), bca_tables_f16()};
  return t[storage];
}

bool bca_shape_supported(int logp, int q, int kb, bool backward) {
  const int logn = logp - 1;
  if (logn > kBcaMaxLogN) return bca_multipass_supported(logp, q, kb, backward);
  if (logn < 0) return false;
  // one token's spectra must fit in LDS; the backward also needs room for the dC slots
  // of at least one block next to two spectra (block ranges cover the rest)
  if (tokens_per_tile(logn, kb, q, 1, 256, kLdsLimit) == 0) return false;
  if (!backward) return true;
  int ia = 0, jb = 0;
  dc_chunk(logn, q, kb, &ia, &jb);
  return ia > 0;
}

hipError_t launch_bca_forward(const BcaArgs& a, const float2* tw, hipStream_t stream, int num_cu) {
  if (a.storage < 0 || a.storage >= kStorages) return hipErrorInvalidValue;
  const BcaStoreTables& t = store_tables(a.storage);
  if (a.logp - 1 > kBcaMaxLogN) return launch_bca_multipass(a, false, tw, stream, num_cu);
  if (a.logp - 1 == kCirculantLogN && a.q == 1 && a.kb == 1) return launch_bca_circulant(a, tw, stream);
  if (a.q == a.kb && a.q <= kSqMaxBlocks) {
    const BcaBwdFn fn = t.sq_fwd[a.q - 1][a.logp - 1];
    if (fn != nullptr) return fn(a, tw, stream, num_cu);
  }
  return t.fwd[a.logp - 1](a, tw, stream);
}

hipError_t launch_bca_backward(const BcaArgs& a, const float2* tw, hipStream_t stream, int num_cu) {
  if (a.storage < 0 || a.storage >= kStorages) return hipErrorInvalidValue;
  const BcaStoreTables& t = store_tables(a.storage);
  const int64_t slots = (int64_t)a.q * a.kb * ((int64_t)1 << (a.logp - 1)) * 2;
  // the square-layer kernels zero dc themselves (in the kernel when the dC sum is staged);
  // every other path finds it zeroed
  BcaBwdFn sq_fn = nullptr;
  if (a.tokens > 0 && a.logp - 1 <= kBcaMaxLogN && a.q == a.kb && a.q <= kSqMaxBlocks)
    sq_fn = t.sq_bwd[a.q - 1][a.logp - 1];
  hipError_t e = hipSuccess;
  if (sq_fn == nullptr) {
    e = launch_fill_zero(a.dc, slots, stream);
    if (e != hipSuccess || a.tokens == 0) return e;
  }
  if (sq_fn != nullptr) {
    e = sq_fn(a, tw, stream, num_cu);
  } else if (a.logp - 1 > kBcaMaxLogN) {
    e = launch_bca_multipass(a, true, tw, stream, num_cu);
  } else {
    e = t.bwd[a.logp - 1](a, tw, stream, num_cu);
  }
  if (e != hipSuccess) return e;
  // dc holds sum_t conj(X) . G as packed spectra; transform them in place to time domain
  return launch_rdfft_rows(a.dc, (int64_t)a.q * a.kb, a.logp - 1, kStorageF32, true, tw, stream, num_cu);
}

}  // namespace rdfft
