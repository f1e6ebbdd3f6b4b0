// bca_kernels.hip -- dispatch of the fused block-circulant layer (Sec. 3.3, Eqs. (4)-(5))
// to the kernels of bca_kernels.hpp (instantiated per storage type in
// bca_store_{f32,bf16,f16}.hip) and the multi-pass layer of bca_multipass.hip, plus the
// two small kernels every storage type shares: the fill of dc and the second stage of
// the two-stage dC sum (fused with dc's inverse transform).
#include <hip/hip_runtime.h>

#include "bca_kernels.hpp"

namespace rdfft {

// Second stage of the two-stage dC sum, fused with the inverse transform of dc.  A
// workgroup takes one (i, j) row of dC and one group of kReduceGroup workgroups' partial
// sums: its threads add those partials slot by slot into an LDS region, the row's
// threads transform the sum to the time domain in place and add the result into dc
// (zeroed beforehand) with float32 atomics.  The inverse transform is linear, so the sum over the groups of the
// transformed group sums is the transform of the full sum.  Workgroup b's partial of
// slot e = ij*N + k lies at stage[(b + c*groups)*tile_f2 + e - c*chunk], c = e / chunk.
struct AtomicAddF32 {  // a time-domain row of dc, added into
  float* base;
  __device__ __forceinline__ void store(int m, float2 v) const {
    unsafeAtomicAdd(base + 2 * m, v.x);
    unsafeAtomicAdd(base + 2 * m + 1, v.y);
  }
};

// threads of the finish kernel: a row of more than 64 threads synchronises with workgroup
// barriers, so the workgroup is that one row; shorter rows synchronise at wave level only,
// and the workgroup has one thread per slot (at least 64, at most 1024) for the sums
template <int LOGN>
constexpr int finish_wg() {
  constexpr int N = RowPlan<LOGN>::N;
  return RowPlan<LOGN>::TPR > 64 ? RowPlan<LOGN>::TPR : (N < 64 ? 64 : (N > 1024 ? 1024 : N));
}

// Layer b of a batch (grid row blockIdx.y when MAXB > 1) reads p.stage[b] and adds into p.dc[b].
template <int LOGN, int MAXB>
__global__ void __launch_bounds__(finish_wg<LOGN>()) bca_dc_finish_kernel(FinishPtrs<MAXB> fp, int rows_ij, int chunk,
                                                                          int groups, int64_t tile_f2,
                                                                          const float2* __restrict__ tw) {
  const int bi = MAXB == 1 ? 0 : (int)blockIdx.y;
  const float2* __restrict__ stage = fp.stage[bi];
  float* __restrict__ dc = fp.dc[bi];
  using P = RowPlan<LOGN>;
  constexpr int N = P::N, TPR = P::TPR, WG = finish_wg<LOGN>();
  constexpr int REG = P::LDS_F2 > lds_padded_size(N) ? P::LDS_F2 : lds_padded_size(N);
  __shared__ float2 reg[REG];
  // one unit per workgroup: every thread sums slots, then the first row group transforms
  const int ij = blockIdx.x % rows_ij, gg = blockIdx.x / rows_ij;
  const int b0 = gg * kReduceGroup;
  const int b1 = b0 + kReduceGroup < groups ? b0 + kReduceGroup : groups;
  for (int k = threadIdx.x; k < N; k += WG) {
    const int e = ij * N + k;
    const int ch = e / chunk;
    const float2* p = stage + ((int64_t)ch * groups + b0) * tile_f2 + (e - ch * chunk);
    // all of a full group's loads in flight at once
    float2 part[kReduceGroup];
    if (b1 - b0 == kReduceGroup) {
      static_for<kReduceGroup>([&](auto bc) { part[decltype(bc)::value] = p[decltype(bc)::value * tile_f2]; });
    } else {
      for (int b = 0; b < kReduceGroup; ++b) {
        part[b] = make_float2(0.f, 0.f);
        if (b < b1 - b0) part[b] = p[b * tile_f2];
      }
    }
    float2 v = part[0];
    static_for<kReduceGroup - 1>([&](auto bc) { v = c_add(v, part[decltype(bc)::value + 1]); });
    reg[lds_pad(k)] = v;
  }
  __syncthreads();
  if (threadIdx.x < TPR)  // the whole workgroup when TPR > 64
    row_inverse<LOGN, true>((int)threadIdx.x, true, LdsSpectrum{reg}, AtomicAddF32{dc + (int64_t)ij * 2 * N}, reg, tw);
}

template <int LOGN, int MAXB>
static hipError_t dc_finish_launch(const FinishPtrs<MAXB>& fp, int count, int rows_ij, int chunk, int groups,
                                   int64_t tile_f2, const float2* tw, hipStream_t stream) {
  const int units = rows_ij * ((groups + kReduceGroup - 1) / kReduceGroup);
  hipLaunchKernelGGL((bca_dc_finish_kernel<LOGN, MAXB>), dim3((unsigned)units, (unsigned)count),
                     dim3(finish_wg<LOGN>()), 0, stream, fp, rows_ij, chunk, groups, tile_f2, tw);
  return hipGetLastError();
}

template <int MAXB, int... L>
static std::array<hipError_t (*)(const FinishPtrs<MAXB>&, int, int, int, int, int64_t, const float2*, hipStream_t),
                  sizeof...(L)>
dc_finish_table(std::integer_sequence<int, L...>) {
  return {&dc_finish_launch<L, MAXB>...};
}

hipError_t launch_dc_finish(const float2* stage, float* dc, int rows_ij, int logn, int chunk, int groups,
                            int64_t tile_f2, const float2* tw, hipStream_t stream) {
  static const auto tab = dc_finish_table<1>(std::make_integer_sequence<int, kBcaMaxLogN + 1>{});
  if (logn < 0 || logn > kBcaMaxLogN) return hipErrorInvalidValue;
  const FinishPtrs<1> fp{{stage}, {dc}};
  return tab[logn](fp, 1, rows_ij, chunk, groups, tile_f2, tw, stream);
}

hipError_t launch_dc_finish_batched(const FinishPtrs<kMaxBatch>& fp, int count, int rows_ij, int logn, int chunk,
                                    int groups, int64_t tile_f2, const float2* tw, hipStream_t stream) {
  static const auto tab = dc_finish_table<kMaxBatch>(std::make_integer_sequence<int, kBcaMaxLogN + 1>{});
  if (logn < 0 || logn > kBcaMaxLogN || count < 1 || count > kMaxBatch) return hipErrorInvalidValue;
  return tab[logn](fp, count, rows_ij, chunk, groups, tile_f2, tw, stream);
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
    BcaBwdFn fn = t.wave_fwd[a.q - 1][a.logp - 1];
    if (fn == nullptr) fn = t.sq_fwd[a.q - 1][a.logp - 1];
    if (fn != nullptr) return fn(a, tw, stream, num_cu);
  }
  return t.fwd[a.logp - 1](a, tw, stream);
}

bool bca_batch_fused(int logp, int q, int kb, int storage, bool backward) {
  if (storage < 0 || storage >= kStorages || q != kb || q < 1 || q > kSqMaxBlocks) return false;
  const int logn = logp - 1;
  if (logn < 0 || logn > kBcaMaxLogN) return false;
  const BcaStoreTables& t = store_tables(storage);
  return (backward ? t.wave_bwd_batched : t.wave_fwd_batched)[q - 1][logn] != nullptr;
}

hipError_t launch_bca_forward_batched(const BcaArgs& a, const BcaBatch& b, const float2* tw, hipStream_t stream,
                                      int num_cu) {
  if (!bca_batch_fused(a.logp, a.q, a.kb, a.storage, false) || b.count < 1 || b.count > kMaxBatch)
    return hipErrorInvalidValue;
  return store_tables(a.storage).wave_fwd_batched[a.q - 1][a.logp - 1](a, b, tw, stream, num_cu);
}

// Every layer's dx apart from its gy (the caller checks): the staged two-stage dC sum, which
// also zeroes dc and leaves it in the time domain.
hipError_t launch_bca_backward_batched(const BcaArgs& a, const BcaBatch& b, const float2* tw, hipStream_t stream,
                                       int num_cu) {
  if (!bca_batch_fused(a.logp, a.q, a.kb, a.storage, true) || b.count < 1 || b.count > kMaxBatch || a.tokens < 1)
    return hipErrorInvalidValue;
  for (int i = 0; i < b.count; ++i)
    if (b.dx[i] == b.y[i]) return hipErrorInvalidValue;
  return store_tables(a.storage).wave_bwd_batched[a.q - 1][a.logp - 1](a, b, tw, stream, num_cu);
}

hipError_t launch_bca_backward(const BcaArgs& a, const float2* tw, hipStream_t stream, int num_cu) {
  if (a.storage < 0 || a.storage >= kStorages) return hipErrorInvalidValue;
  const BcaStoreTables& t = store_tables(a.storage);
  const int64_t slots = (int64_t)a.q * a.kb * ((int64_t)1 << (a.logp - 1)) * 2;
  // the square-layer kernels zero dc themselves (in the kernel when the dC sum is staged);
  // every other path finds it zeroed
  BcaBwdFn sq_fn = nullptr;
  if (a.tokens > 0 && a.logp - 1 <= kBcaMaxLogN && a.q == a.kb && a.q <= kSqMaxBlocks) {
    sq_fn = t.wave_bwd[a.q - 1][a.logp - 1];
    if (sq_fn == nullptr) sq_fn = t.sq_bwd[a.q - 1][a.logp - 1];
  }
  hipError_t e = hipSuccess;
  if (sq_fn == nullptr) {
    e = launch_fill_zero(a.dc, slots, stream);
    if (e != hipSuccess || a.tokens == 0) return e;
  }
  // the square-layer kernels also leave dc in the time domain
  if (sq_fn != nullptr) return sq_fn(a, tw, stream, num_cu);
  if (a.logp - 1 > kBcaMaxLogN) {
    e = launch_bca_multipass(a, true, tw, stream, num_cu);
  } else {
    e = t.bwd[a.logp - 1](a, tw, stream, num_cu);
  }
  if (e != hipSuccess) return e;
  // dc holds sum_t conj(X) . G as packed spectra; transform them in place to time domain
  return launch_rdfft_rows(a.dc, (int64_t)a.q * a.kb, a.logp - 1, kStorageF32, true, tw, stream, num_cu);
}

}  // namespace rdfft
