// bca_kernels.hip -- fused block-circulant layer kernels (Sec. 3.3, Eqs. (4)-(5)).
//
// A workgroup takes a tile of TT tokens at a time and keeps every spectrum of the
// tile in LDS, in the packed pair layout of the row transforms:
//   forward : X_j = rdFFT(x_j)  ->  Y_i = sum_j C_ij . X_j  ->  y_i = irdFFT(Y_i)
//   backward: X_j = rdFFT(x_j), G_i = rdFFT(g_i)
//             dC_ij += conj(X_j) . G_i          (float32 accumulators in registers)
//             dX_j   = sum_i conj(C_ij) . G_i  ->  dx_j = irdFFT(dX_j)
// so no intermediate tensor ever reaches HBM.  Slot 0 of a packed spectrum holds
// the two real bins Y_0 and Y_{p/2}; every product acts on them as two real
// products (conjugation is the identity there).  The per-workgroup dC partial sums
// are added into the caller's dc buffer with float32 atomics; a final in-place
// irdFFT of dc (stream-ordered after this kernel) yields the time-domain gradient.
#include <hip/hip_runtime.h>

#include "fft_device.hpp"
#include "launch.hpp"

namespace rdfft {

constexpr int kBcaThreads = 256;
constexpr int kBcaMaxAcc = 32;  // dC pair slots accumulated per thread

template <int LOGN>
struct BcaPlan {
  using P = RowPlan<LOGN>;
  static constexpr int N = P::N;
  static constexpr int TPR = P::TPR;
  static_assert(TPR <= kBcaThreads, "row too long for the fused layer kernel");
  static constexpr int NG = kBcaThreads / TPR;  // row groups per workgroup
  static constexpr int REGION = P::LDS_F2 > lds_padded_size(N) ? P::LDS_F2 : lds_padded_size(N);
};

// a . b on packed pair slots (slot 0 = two real bins)
__device__ __forceinline__ float2 slot_mul(float2 a, float2 b, bool slot0) {
  const float re = slot0 ? a.x * b.x : fmaf(a.x, b.x, -a.y * b.y);
  const float im = slot0 ? a.y * b.y : fmaf(a.x, b.y, a.y * b.x);
  return make_float2(re, im);
}
// conj(a) . b on packed pair slots
__device__ __forceinline__ float2 slot_cmul(float2 a, float2 b, bool slot0) {
  const float re = slot0 ? a.x * b.x : fmaf(a.x, b.x, a.y * b.y);
  const float im = slot0 ? a.y * b.y : fmaf(a.x, b.y, -a.y * b.x);
  return make_float2(re, im);
}

template <class Elem>
struct Acc;
template <>
struct Acc<float2> {
  using In = ConstF32;
  using Out = GlobalF32;
};
template <>
struct Acc<uint32_t> {
  using In = ConstBF16;
  using Out = GlobalBF16;
};

extern __shared__ float2 bca_lds[];

// x: [T][kb*N] pairs, c: [q][kb][N] pairs, y: [T][q*N] pairs (all in storage type Elem)
template <int LOGN, class Elem>
__global__ void __launch_bounds__(kBcaThreads) bca_forward_kernel(const Elem* __restrict__ x, const Elem* __restrict__ c,
                                                                  Elem* y, int64_t tokens, int q, int kb, int tt_per_tile,
                                                                  const float2* __restrict__ tw) {
  using B = BcaPlan<LOGN>;
  using In = typename Acc<Elem>::In;
  using Out = typename Acc<Elem>::Out;
  constexpr int N = B::N, TPR = B::TPR, NG = B::NG, REG = B::REGION;
  const int tid = threadIdx.x;
  const int grp = tid / TPR, t = tid - grp * TPR;
  const int TT = tt_per_tile;
  float2* const xs = bca_lds;                        // TT*kb regions
  float2* const ys = bca_lds + (size_t)TT * kb * REG;  // TT*q regions
  float2* const dummy = bca_lds + (size_t)TT * (kb + q) * REG;
  const int64_t tok0 = (int64_t)blockIdx.x * TT;

  // Phase A: X_j = rdFFT(x_j) for every (token, j) of the tile, into LDS
  const int nx = TT * kb;
  for (int s0 = 0; s0 < nx; s0 += NG) {
    const int s = s0 + grp;
    const bool valid = s < nx;
    const int tt = valid ? s / kb : 0, j = valid ? s - tt * kb : 0;
    const bool act = valid && tok0 + tt < tokens;
    float2* reg = valid ? xs + (size_t)s * REG : dummy;
    const In src{x + ((act ? tok0 + tt : 0) * kb + j) * (int64_t)N};
    row_forward<LOGN, true>(t, act, src, LdsSpectrum{reg}, reg, tw);
  }
  __syncthreads();

  // Phase B: Y_i[k] = sum_j C_ij[k] . X_j[k]
  const In cin{c};
  for (int e = tid; e < q * N; e += kBcaThreads) {
    const int i = e / N, k = e - i * N;
    const bool s0 = k == 0;
    for (int tt = 0; tt < TT; ++tt) {
      float2 acc = make_float2(0.f, 0.f);
      for (int j = 0; j < kb; ++j) {
        const float2 cv = cin.load((i * kb + j) * N + k);
        const float2 xv = xs[(size_t)(tt * kb + j) * REG + lds_pad(k)];
        const float2 pr = slot_mul(cv, xv, s0);
        acc.x += pr.x;
        acc.y += pr.y;
      }
      ys[(size_t)(tt * q + i) * REG + lds_pad(k)] = acc;
    }
  }
  __syncthreads();

  // Phase C: y_i = irdFFT(Y_i)
  const int ny = TT * q;
  for (int s0 = 0; s0 < ny; s0 += NG) {
    const int s = s0 + grp;
    const bool valid = s < ny;
    const int tt = valid ? s / q : 0, i = valid ? s - tt * q : 0;
    const bool act = valid && tok0 + tt < tokens;
    float2* reg = valid ? ys + (size_t)s * REG : dummy;
    const Out dst{y + ((act ? tok0 + tt : 0) * q + i) * (int64_t)N};
    row_inverse<LOGN, true>(t, act, LdsSpectrum{reg}, dst, reg, tw);
  }
}

// gy: [T][q*N] pairs (read), dx: [T][kb*N] pairs (written; may alias gy when kb == q),
// dc: [q][kb][N] float2 slots, receives the spectral partial sums (atomically)
template <int LOGN, class Elem>
__global__ void __launch_bounds__(kBcaThreads) bca_backward_kernel(const Elem* __restrict__ x, const Elem* __restrict__ c,
                                                                   const Elem* gy, Elem* dx, float* __restrict__ dc,
                                                                   int64_t tokens, int q, int kb, int tt_per_tile,
                                                                   int64_t ntiles, const float2* __restrict__ tw) {
  using B = BcaPlan<LOGN>;
  using In = typename Acc<Elem>::In;
  using Out = typename Acc<Elem>::Out;
  constexpr int N = B::N, TPR = B::TPR, NG = B::NG, REG = B::REGION;
  const int tid = threadIdx.x;
  const int grp = tid / TPR, t = tid - grp * TPR;
  const int TT = tt_per_tile;
  float2* const xs = bca_lds;                        // TT*kb regions: X, then dX
  float2* const gs = bca_lds + (size_t)TT * kb * REG;  // TT*q regions: G
  float2* const dummy = bca_lds + (size_t)TT * (kb + q) * REG;
  const int qkn = q * kb * N;
  const In cin{c};

  float2 acc[kBcaMaxAcc];
  static_for<kBcaMaxAcc>([&](auto uc) { acc[decltype(uc)::value] = make_float2(0.f, 0.f); });

  for (int64_t tile = blockIdx.x; tile < ntiles; tile += gridDim.x) {
    const int64_t tok0 = tile * TT;
    const int nvalid = (int)(tokens - tok0 < TT ? tokens - tok0 : TT);

    // Phase A: X_j = rdFFT(x_j), G_i = rdFFT(g_i)
    const int nx = TT * kb, ns = TT * (kb + q);
    for (int s0 = 0; s0 < ns; s0 += NG) {
      const int s = s0 + grp;
      const bool valid = s < ns;
      float2* reg = valid ? bca_lds + (size_t)s * REG : dummy;
      // choose the source without branching around the transform: its barriers
      // must be reached by every lane of every wave
      const Elem* srcp = x;
      bool act = false;
      if (valid && s < nx) {
        const int tt = s / kb, j = s - tt * kb;
        act = tt < nvalid;
        srcp = x + ((act ? tok0 + tt : 0) * kb + j) * (int64_t)N;
      } else if (valid) {
        const int sg = s - nx;
        const int tt = sg / q, i = sg - tt * q;
        act = tt < nvalid;
        srcp = gy + ((act ? tok0 + tt : 0) * q + i) * (int64_t)N;
      }
      row_forward<LOGN, true>(t, act, In{srcp}, LdsSpectrum{reg}, reg, tw);
    }
    __syncthreads();

    // Phase B1: dC_ij[k] += sum_t conj(X_tj[k]) . G_ti[k]
    static_for<kBcaMaxAcc>([&](auto uc) {
      constexpr int u = decltype(uc)::value;
      const int e = tid + u * kBcaThreads;
      if (e < qkn) {
        const int k = e & (N - 1);
        const int ij = e / N;
        const int i = ij / kb, j = ij - i * kb;
        const bool s0 = k == 0;
        for (int tt = 0; tt < nvalid; ++tt) {
          const float2 xv = xs[(size_t)(tt * kb + j) * REG + lds_pad(k)];
          const float2 gv = gs[(size_t)(tt * q + i) * REG + lds_pad(k)];
          const float2 pr = slot_cmul(xv, gv, s0);
          acc[u].x += pr.x;
          acc[u].y += pr.y;
        }
      }
    });
    __syncthreads();

    // Phase B2: dX_j[k] = sum_i conj(C_ij[k]) . G_i[k], written over X_j
    for (int e = tid; e < kb * N; e += kBcaThreads) {
      const int j = e / N, k = e - j * N;
      const bool s0 = k == 0;
      for (int tt = 0; tt < TT; ++tt) {
        float2 sum = make_float2(0.f, 0.f);
        for (int i = 0; i < q; ++i) {
          const float2 cv = cin.load((i * kb + j) * N + k);
          const float2 gv = gs[(size_t)(tt * q + i) * REG + lds_pad(k)];
          const float2 pr = slot_cmul(cv, gv, s0);
          sum.x += pr.x;
          sum.y += pr.y;
        }
        xs[(size_t)(tt * kb + j) * REG + lds_pad(k)] = sum;
      }
    }
    __syncthreads();

    // Phase C: dx_j = irdFFT(dX_j)
    for (int s0 = 0; s0 < nx; s0 += NG) {
      const int s = s0 + grp;
      const bool valid = s < nx;
      const int tt = valid ? s / kb : 0, j = valid ? s - tt * kb : 0;
      const bool act = valid && tt < nvalid;
      float2* reg = valid ? xs + (size_t)s * REG : dummy;
      const Out dst{dx + ((act ? tok0 + tt : 0) * kb + j) * (int64_t)N};
      row_inverse<LOGN, true>(t, act, LdsSpectrum{reg}, dst, reg, tw);
    }
    __syncthreads();
  }

  static_for<kBcaMaxAcc>([&](auto uc) {
    constexpr int u = decltype(uc)::value;
    const int e = tid + u * kBcaThreads;
    if (e < qkn) {
      unsafeAtomicAdd(dc + 2 * (int64_t)e, acc[u].x);
      unsafeAtomicAdd(dc + 2 * (int64_t)e + 1, acc[u].y);
    }
  });
}

__global__ void fill_zero_kernel(float* __restrict__ p, int64_t count) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < count; i += (int64_t)gridDim.x * blockDim.x)
    p[i] = 0.f;
}

// ----------------------------------------------------------------------------------
// host side

static int region_bytes(int logn) {
  static const int sizes[kMaxLogN + 1] = {
      BcaPlan<0>::REGION,  BcaPlan<1>::REGION,  BcaPlan<2>::REGION,  BcaPlan<3>::REGION,
      BcaPlan<4>::REGION,  BcaPlan<5>::REGION,  BcaPlan<6>::REGION,  BcaPlan<7>::REGION,
      BcaPlan<8>::REGION,  BcaPlan<9>::REGION,  BcaPlan<10>::REGION, BcaPlan<11>::REGION,
      BcaPlan<12>::REGION, 0, 0, 0};
  return sizes[logn] * (int)sizeof(float2);
}

constexpr int kBcaMaxLogN = 12;      // p <= 8192
constexpr int kLdsLimit = 160 * 1024;  // gfx950 LDS per workgroup
constexpr int kLdsTarget = 64 * 1024;  // aim for two workgroups per CU

// tokens per tile so that a tile's spectra fit the LDS target; 0 if one token does not fit
static int tokens_per_tile(int logn, int segs_per_token, int64_t tokens) {
  const int rb = region_bytes(logn);
  const int64_t per_tok = (int64_t)segs_per_token * rb;
  if (per_tok + rb > kLdsLimit) return 0;
  int64_t tt = (kLdsTarget - rb) / per_tok;
  if (tt < 1) tt = 1;
  if (tt > tokens) tt = tokens;
  if (tt < 1) tt = 1;
  return (int)tt;
}

template <class K>
static hipError_t set_lds_limit(K kernel) {
  return hipFuncSetAttribute(reinterpret_cast<const void*>(kernel), hipFuncAttributeMaxDynamicSharedMemorySize,
                             kLdsLimit);
}

template <int LOGN, class Elem>
static hipError_t fwd_impl(const BcaArgs& a, const float2* tw, hipStream_t stream) {
  const int TT = tokens_per_tile(LOGN, a.kb + a.q, a.tokens);
  if (TT == 0) return hipErrorInvalidValue;
  const size_t lds = (size_t)(TT * (a.kb + a.q) + 1) * region_bytes(LOGN);
  static const hipError_t attr = set_lds_limit(bca_forward_kernel<LOGN, Elem>);
  if (attr != hipSuccess) return attr;
  const int64_t tiles = (a.tokens + TT - 1) / TT;
  hipLaunchKernelGGL((bca_forward_kernel<LOGN, Elem>), dim3((unsigned)tiles), dim3(kBcaThreads), lds, stream,
                     static_cast<const Elem*>(a.x), static_cast<const Elem*>(a.c), static_cast<Elem*>(a.y), a.tokens,
                     a.q, a.kb, TT, tw);
  return hipGetLastError();
}

template <int LOGN, class Elem>
static hipError_t bwd_impl(const BcaArgs& a, const float2* tw, hipStream_t stream, int num_cu) {
  const int TT = tokens_per_tile(LOGN, a.kb + a.q, a.tokens);
  if (TT == 0) return hipErrorInvalidValue;
  const size_t lds = (size_t)(TT * (a.kb + a.q) + 1) * region_bytes(LOGN);
  static const hipError_t attr = set_lds_limit(bca_backward_kernel<LOGN, Elem>);
  if (attr != hipSuccess) return attr;
  const int64_t tiles = (a.tokens + TT - 1) / TT;
  const int per_cu = lds <= (size_t)kLdsTarget ? 2 : 1;
  const int64_t grid = std::min<int64_t>(tiles, (int64_t)num_cu * per_cu);
  hipLaunchKernelGGL((bca_backward_kernel<LOGN, Elem>), dim3((unsigned)grid), dim3(kBcaThreads), lds, stream,
                     static_cast<const Elem*>(a.x), static_cast<const Elem*>(a.c), static_cast<const Elem*>(a.y),
                     static_cast<Elem*>(a.dx), a.dc, a.tokens, a.q, a.kb, TT, tiles, tw);
  return hipGetLastError();
}

using BcaFn = hipError_t (*)(const BcaArgs&, const float2*, hipStream_t);
using BcaBwdFn = hipError_t (*)(const BcaArgs&, const float2*, hipStream_t, int);

template <int... L>
static std::array<BcaFn, sizeof...(L)> fwd_table(bool bf16, std::integer_sequence<int, L...>) {
  return {(bf16 ? &fwd_impl<L, uint32_t> : &fwd_impl<L, float2>)...};
}
template <int... L>
static std::array<BcaBwdFn, sizeof...(L)> bwd_table(bool bf16, std::integer_sequence<int, L...>) {
  return {(bf16 ? &bwd_impl<L, uint32_t> : &bwd_impl<L, float2>)...};
}

bool bca_shape_supported(int logp, int q, int kb) {
  const int logn = logp - 1;
  if (logn < 0 || logn > kBcaMaxLogN) return false;
  if ((int64_t)q * kb * (1 << logn) > (int64_t)kBcaThreads * kBcaMaxAcc) return false;
  return tokens_per_tile(logn, kb + q, 1) > 0;
}

hipError_t launch_bca_forward(const BcaArgs& a, const float2* tw, hipStream_t stream) {
  static const auto seq = std::make_integer_sequence<int, kBcaMaxLogN + 1>{};
  static const std::array<BcaFn, kBcaMaxLogN + 1> tab[2] = {fwd_table(false, seq), fwd_table(true, seq)};
  return tab[a.bf16 ? 1 : 0][a.logp - 1](a, tw, stream);
}

hipError_t launch_bca_backward(const BcaArgs& a, const float2* tw, hipStream_t stream, int num_cu) {
  static const auto seq = std::make_integer_sequence<int, kBcaMaxLogN + 1>{};
  static const std::array<BcaBwdFn, kBcaMaxLogN + 1> tab[2] = {bwd_table(false, seq), bwd_table(true, seq)};
  const int64_t slots = (int64_t)a.q * a.kb * ((int64_t)1 << (a.logp - 1)) * 2;
  const int blocks = (int)std::min<int64_t>((slots + 255) / 256, 1024);
  hipLaunchKernelGGL(fill_zero_kernel, dim3(blocks), dim3(256), 0, stream, a.dc, slots);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || a.tokens == 0) return e;
  e = tab[a.bf16 ? 1 : 0][a.logp - 1](a, tw, stream, num_cu);
  if (e != hipSuccess) return e;
  // dc holds sum_t conj(X) . G as packed spectra; transform them in place to time domain
  return launch_rdfft_rows(a.dc, (int64_t)a.q * a.kb, a.logp - 1, false, true, tw, stream);
}

}  // namespace rdfft
