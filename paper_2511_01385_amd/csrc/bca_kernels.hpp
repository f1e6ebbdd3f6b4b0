// bca_kernels.hpp -- fused block-circulant layer kernels (Sec. 3.3, Eqs. (4)-(5)), as
// templates over the storage type.  bca_store_{f32,bf16,f16}.hip instantiate them, one
// storage type per translation unit; bca_kernels.hip holds the dispatch.
//
// A workgroup takes a tile of TT tokens at a time and keeps every spectrum of the
// tile in LDS, in the packed pair layout of the row transforms:
//   forward : X_j = rdFFT(x_j)  ->  Y_i = sum_j C_ij . X_j  ->  y_i = irdFFT(Y_i)
//   backward: X_j = rdFFT(x_j), G_i = rdFFT(g_i)
//             dC_ij += conj(X_j) . G_i          (float32 partial sums in LDS)
//             dX_j   = sum_i conj(C_ij) . G_i  ->  dx_j = irdFFT(dX_j)
// so no intermediate tensor ever reaches HBM.  Slot 0 of a packed spectrum holds
// the two real bins Y_0 and Y_{p/2}; every product acts on them as two real
// products (conjugation is the identity there).  The backward runs one wide persistent
// workgroup per CU; its dC partial sums stay in LDS (or registers) for all of its tiles
// and are then added into the caller's dc buffer with float32 atomics (each workgroup
// starting at a different offset), or, for the square-layer kernel when dx is not gy,
// staged in the gy rows the workgroup has consumed and summed by a second kernel; a final
// in-place irdFFT of dc (stream-ordered after the kernels) yields the time-domain
// gradient.  A single circulant of p = 8192 and blocks beyond 8192 are routed to the row
// kernels of bca_multipass.hip.
#pragma once

#include <hip/hip_runtime.h>

#include "fft_device.hpp"
#include "launch.hpp"

namespace rdfft {

template <int LOGN>
struct BcaPlan {
  using P = RowPlan<LOGN>;
  static constexpr int N = P::N;
  static constexpr int TPR = P::TPR;
  static_assert(TPR <= 256, "row too long for the fused layer kernels");
  // forward: 256 threads, or two row groups for the longest rows
  static constexpr int FWD_WG = 2 * TPR > 256 ? 2 * TPR : 256;
  // backward: one wide workgroup per CU keeps the number of dC partial sums (and so
  // of atomics) small; 1024 threads when the plan is light on registers
  static constexpr int BWD_WG = (P::E <= 8 && TPR <= 128) ? 1024 : 512;
  static constexpr int REGION = P::LDS_F2 > lds_padded_size(N) ? P::LDS_F2 : lds_padded_size(N);
};

// acc + a.b (or acc + conj(a).b) on packed pair slots.  Slot 0 (S0) holds the two real
// bins Y_0 and Y_{p/2}: there the product is two real products and conj is the identity.
template <bool S0, bool CONJ>
__device__ __forceinline__ float2 slot_mac(float2 acc, float2 a, float2 b) {
  if constexpr (S0) return make_float2(fmaf(a.x, b.x, acc.x), fmaf(a.y, b.y, acc.y));
  if constexpr (!CONJ) return make_float2(fmaf(a.x, b.x, fmaf(-a.y, b.y, acc.x)), fmaf(a.x, b.y, fmaf(a.y, b.x, acc.y)));
  return make_float2(fmaf(a.x, b.x, fmaf(a.y, b.y, acc.x)), fmaf(a.x, b.y, fmaf(-a.y, b.x, acc.y)));
}

// the pair type a storage struct keeps in memory
template <class St>
using ElemOf = typename St::Elem;

extern __shared__ float2 bca_lds[];

// x: [T][kb*N] pairs, c: [q][kb][N] pairs, y: [T][q*N] pairs (all in the storage type St).
// y may be x itself (kb == q): a workgroup reads a tile's x rows before it writes the
// tile's y rows, and no other workgroup touches them, so x is not declared restrict.
template <int LOGN, class St, int WG = BcaPlan<LOGN>::FWD_WG>
__global__ void __launch_bounds__(WG) bca_forward_kernel(const ElemOf<St>* x, const ElemOf<St>* __restrict__ c,
                                                                  ElemOf<St>* y, int64_t tokens, int q, int kb, int tt_per_tile,
                                                                  const float2* __restrict__ tw) {
  using B = BcaPlan<LOGN>;
  using In = typename St::In;
  using Out = typename St::Out;
  constexpr int N = B::N, TPR = B::TPR, NG = WG / TPR, REG = B::REGION;
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

  // Phase B: Y_i[k] = sum_j C_ij[k] . X_j[k]; a thread takes one (token, bin) and all i, j.
  // Bin 0 is slot 0 and takes the branch with real products (one lane of one wave).
  const In cin{c};
  for (int it = tid; it < TT * N; it += WG) {
    const int tt = it / N, k = it - tt * N;
    const float2* xk = xs + (size_t)tt * kb * REG + lds_pad(k);
    float2* yk = ys + (size_t)tt * q * REG + lds_pad(k);
    auto block_sum = [&](auto s0c) {
      constexpr bool S0 = decltype(s0c)::value;
      int ci = k;  // pair index of C_ij[k] = (i*kb + j)*N + k
      for (int i = 0; i < q; ++i) {
        float2 a = make_float2(0.f, 0.f);
        // unrolled so that several L2 loads of C are in flight at once
#pragma unroll 4
        for (int j = 0; j < kb; ++j) a = slot_mac<S0, false>(a, cin.load(ci + j * N), xk[j * REG]);
        ci += kb * N;
        yk[i * REG] = a;
      }
    };
    if (k == 0) block_sum(std::true_type{});
    else block_sum(std::false_type{});
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

// General backward.  gy: [T][q*N] pairs (read), dx: [T][kb*N] pairs (written; may alias
// gy when kb == q), dc: [q][kb][N] float2 slots, receives spectral partial sums (atomically).
// A launch covers the output blocks i0 <= i < i0+ia and input blocks j0 <= j < j0+jb and
// does the dx path (mode & kBwdDx; needs every block: i0 = j0 = 0, ia = q, jb = kb), the dC
// accumulation (mode & kBwdDc), or both.  Layers whose q*kb*(p/2) dC slots do not fit
// in LDS run dC launches over block ranges that do, then one dx launch (last, since dx
// may be gy).
constexpr int kBwdDx = 1, kBwdDc = 2;

template <int LOGN, class St, int WG = BcaPlan<LOGN>::BWD_WG>
__global__ void __launch_bounds__(WG) bca_backward_kernel(const ElemOf<St>* __restrict__ x, const ElemOf<St>* __restrict__ c,
                                                                   const ElemOf<St>* gy, ElemOf<St>* dx, float* __restrict__ dc,
                                                                   int64_t tokens, int q, int kb, int i0, int ia,
                                                                   int j0, int jb, int mode, int tt_per_tile,
                                                                   int64_t ntiles, const float2* __restrict__ tw) {
  using B = BcaPlan<LOGN>;
  using In = typename St::In;
  using Out = typename St::Out;
  constexpr int N = B::N, TPR = B::TPR, NG = WG / TPR, REG = B::REGION;
  const int tid = threadIdx.x;
  const int grp = tid / TPR, t = tid - grp * TPR;
  const int TT = tt_per_tile;
  const bool do_dx = (mode & kBwdDx) != 0, do_dc = (mode & kBwdDc) != 0;
  float2* const xs = bca_lds;                        // TT*jb regions: X, then dX
  float2* const gs = bca_lds + (size_t)TT * jb * REG;  // TT*ia regions: G
  float2* const dummy = bca_lds + (size_t)TT * (jb + ia) * REG;
  float2* const acc = dummy + REG;                   // ia*jb*N dC partial sums (pair slots)
  const int qkn = do_dc ? ia * jb * N : 0;
  const In cin{c};

  for (int e = tid; e < qkn; e += WG) acc[e] = make_float2(0.f, 0.f);

  for (int64_t tile = blockIdx.x; tile < ntiles; tile += gridDim.x) {
    const int64_t tok0 = tile * TT;
    const int nvalid = (int)(tokens - tok0 < TT ? tokens - tok0 : TT);

    // Phase A: X_j = rdFFT(x_j), G_i = rdFFT(g_i) for the launch's blocks
    const int nx = TT * jb, ns = TT * (jb + ia);
    for (int s0 = 0; s0 < ns; s0 += NG) {
      const int s = s0 + grp;
      const bool valid = s < ns;
      float2* reg = valid ? bca_lds + (size_t)s * REG : dummy;
      // choose the source without branching around the transform: its barriers
      // must be reached by every lane of every wave
      const ElemOf<St>* srcp = x;
      bool act = false;
      if (valid && s < nx) {
        const int tt = s / jb, j = j0 + s - tt * jb;
        act = tt < nvalid;
        srcp = x + ((act ? tok0 + tt : 0) * kb + j) * (int64_t)N;
      } else if (valid) {
        const int sg = s - nx;
        const int tt = sg / ia, i = i0 + sg - tt * ia;
        act = tt < nvalid;
        srcp = gy + ((act ? tok0 + tt : 0) * q + i) * (int64_t)N;
      }
      row_forward<LOGN, true>(t, act, In{srcp}, LdsSpectrum{reg}, reg, tw);
    }
    __syncthreads();

    // Phase B1: dC_ij[k] += sum_t conj(X_tj[k]) . G_ti[k]; each slot has one owner thread
    for (int e = tid; e < qkn; e += WG) {
      const int k = e & (N - 1);
      const int ij = e / N;
      const int ii = ij / jb, jj = ij - ii * jb;
      const float2* xp = xs + (size_t)jj * REG + lds_pad(k);
      const float2* gp = gs + (size_t)ii * REG + lds_pad(k);
      auto contract = [&](auto s0c) {
        constexpr bool S0 = decltype(s0c)::value;
        float2 sum = acc[e];
#pragma unroll 4
        for (int tt = 0; tt < nvalid; ++tt) sum = slot_mac<S0, true>(sum, xp[(size_t)tt * jb * REG], gp[(size_t)tt * ia * REG]);
        acc[e] = sum;
      };
      if (k == 0) contract(std::true_type{});
      else contract(std::false_type{});
    }
    if (!do_dx) {
      __syncthreads();
      continue;
    }
    __syncthreads();

    // Phase B2: dX_j[k] = sum_i conj(C_ij[k]) . G_i[k], written over X_j
    for (int it = tid; it < TT * N; it += WG) {
      const int tt = it / N, k = it - tt * N;
      const float2* gk = gs + (size_t)tt * q * REG + lds_pad(k);
      float2* xk = xs + (size_t)tt * kb * REG + lds_pad(k);
      auto grad_x = [&](auto s0c) {
        constexpr bool S0 = decltype(s0c)::value;
        for (int j = 0; j < kb; ++j) {
          float2 a = make_float2(0.f, 0.f);
          const int ci = j * N + k;  // pair index of C_0j[k]; C_ij[k] is i*kb*N further
#pragma unroll 4
          for (int i = 0; i < q; ++i) a = slot_mac<S0, true>(a, cin.load(ci + i * kb * N), gk[i * REG]);
          xk[j * REG] = a;
        }
      };
      if (k == 0) grad_x(std::true_type{});
      else grad_x(std::false_type{});
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

  if (!do_dc) return;
  __syncthreads();
  // fold this workgroup's partial sums into dc; workgroup b starts 64*b slots in, so
  // that the workgroups, which all finish together, do not queue on the same addresses
  const int shift = (int)(((unsigned)blockIdx.x * 64u) % (unsigned)qkn);
  for (int e0 = tid; e0 < qkn; e0 += WG) {
    int e = e0 + shift;
    if (e >= qkn) e -= qkn;
    const float2 v = acc[e];
    const int k = e & (N - 1);
    const int ij = e / N;
    const int ii = ij / jb, jj = ij - ii * jb;
    const int64_t d = ((int64_t)(i0 + ii) * kb + (j0 + jj)) * N + k;
    unsafeAtomicAdd(dc + 2 * d, v.x);
    unsafeAtomicAdd(dc + 2 * d + 1, v.y);
  }
}

// Forward for square layers (q == kb == QB) with few blocks: a persistent workgroup
// whose threads own fixed bins for the whole kernel and keep C_ij[k] for them in
// registers (read from HBM once per workgroup rather than once per token).  With TB > 1
// threads per bin the TB threads split the output blocks i into TJ groups and the
// tokens of a tile into TS phases; with BT > 1 bins per thread a thread takes bins kt,
// kt+WG, ...
template <int LOGN, int QB, int WG>
struct BcaSqFwd {
  static constexpr int N = BcaPlan<LOGN>::N;
  static constexpr int TB = WG >= N ? WG / N : 1;
  static constexpr int BT = WG >= N ? 1 : N / WG;
  static constexpr int TJ = TB % QB == 0 ? QB : (QB % TB == 0 ? TB : 1);  // output-block groups
  static constexpr int TS = TB / TJ;                                        // token phases
  static constexpr int IPT = QB / TJ;                                       // output blocks per thread
  static constexpr int NSL = IPT * QB;
  // the 512-bin layers (p = 1024) run two 512-thread workgroups per CU, four waves per SIMD,
  // which leaves a wave 128 VGPRs: ask the compiler to stay within them
  static constexpr int MIN_WAVES = (WG == 512 && N == 512) ? 4 : 1;
};
constexpr int kFwdSqWG = 512;

template <int LOGN, class St, int QB, int WG = kFwdSqWG>
__global__ void __launch_bounds__(WG) __attribute__((amdgpu_waves_per_eu(BcaSqFwd<LOGN, QB, WG>::MIN_WAVES)))
bca_forward_sq_kernel(const ElemOf<St>* x, const ElemOf<St>* __restrict__ c,
                                                                     ElemOf<St>* y, int64_t tokens, int tt_per_tile,
                                                                     int64_t ntiles, const float2* __restrict__ tw) {
  using B = BcaPlan<LOGN>;
  using S = BcaSqFwd<LOGN, QB, WG>;
  using In = typename St::In;
  using Out = typename St::Out;
  constexpr int N = B::N, TPR = B::TPR, NG = WG / TPR, REG = B::REGION;
  constexpr int TB = S::TB, BT = S::BT, TJ = S::TJ, TS = S::TS, IPT = S::IPT, NSL = S::NSL;
  static_assert(TJ * IPT == QB && TS * TJ == TB, "inconsistent split");
  const int tid = threadIdx.x;
  const int grp = tid / TPR, t = tid - grp * TPR;
  const int u = TB > 1 ? tid / N : 0;
  const int kt = TB > 1 ? tid - u * N : tid;
  const int i0 = (u % TJ) * IPT;  // first output block of this thread
  const int tu = u / TJ;          // token phase
  const int TT = tt_per_tile;
  // With one thread per bin, Y_i[k] overwrites X_i[k]: the thread has read every X_j[k]
  // before it writes, and no other thread touches bin k, so a token needs QB regions.
  constexpr bool INPLACE = TB == 1;
  float2* const xs = bca_lds;                                         // TT*QB regions: X
  float2* const ys = INPLACE ? xs : bca_lds + (size_t)TT * QB * REG;  // TT*QB regions: Y
  // spare region for row groups without a transform (allocated only when some exist)
  float2* const dummy = bca_lds + (size_t)TT * (INPLACE ? 1 : 2) * QB * REG;

  // slot (ii, j) is sl = ii*QB + j for output block i = i0 + ii
  typename In::raw_t cr[BT][NSL];
  {
    const In cin{c};
    static_for<BT>([&](auto wc) {
      constexpr int w = decltype(wc)::value;
      static_for<NSL>([&](auto sc) {
        constexpr int sl = decltype(sc)::value, ii = sl / QB, j = sl % QB;
        cr[w][sl] = cin.load_raw(((i0 + ii) * QB + j) * N + kt + w * WG);  // C_ij[k]
      });
    });
  }

  for (int64_t tile = blockIdx.x; tile < ntiles; tile += gridDim.x) {
    const int64_t tok0 = tile * TT;
    const int nvalid = (int)(tokens - tok0 < TT ? tokens - tok0 : TT);

    // Phase A: X_j = rdFFT(x_j)
    const int nx = TT * QB;
    for (int s0 = 0; s0 < nx; s0 += NG) {
      const int s = s0 + grp;
      const bool valid = s < nx;
      const int tt = valid ? s / QB : 0, j = valid ? s - tt * QB : 0;
      const bool act = valid && tt < nvalid;
      float2* reg = valid ? xs + (size_t)s * REG : dummy;
      const In src{x + ((act ? tok0 + tt : 0) * QB + j) * (int64_t)N};
      row_forward<LOGN, true>(t, act, src, LdsSpectrum{reg}, reg, tw);
    }
    __syncthreads();

    // Phase B: Y_i[k] = sum_j C_ij[k] . X_j[k]
    static_for<BT>([&](auto wc) {
      constexpr int w = decltype(wc)::value;
      const int k = kt + w * WG;
      const int pk = lds_pad(k);
      auto block_sum = [&](auto s0c) {
        constexpr bool S0 = decltype(s0c)::value;
        for (int tt = tu; tt < nvalid; tt += TS) {
          const float2* xk = xs + (size_t)tt * QB * REG + pk;
          float2* yk = ys + ((size_t)tt * QB + i0) * REG + pk;
          float2 X[QB];
          static_for<QB>([&](auto jc) { X[decltype(jc)::value] = xk[decltype(jc)::value * REG]; });
          static_for<IPT>([&](auto ic) {
            constexpr int ii = decltype(ic)::value;
            float2 a = make_float2(0.f, 0.f);
            static_for<QB>([&](auto jc) {
              constexpr int j = decltype(jc)::value;
              a = slot_mac<S0, false>(a, In::widen(cr[w][ii * QB + j]), X[j]);
            });
            yk[ii * REG] = a;
          });
        }
      };
      if (k == 0) block_sum(std::true_type{});
      else block_sum(std::false_type{});
    });
    __syncthreads();

    // Phase C: y_i = irdFFT(Y_i)
    for (int s0 = 0; s0 < nx; s0 += NG) {
      const int s = s0 + grp;
      const bool valid = s < nx;
      const int tt = valid ? s / QB : 0, i = valid ? s - tt * QB : 0;
      const bool act = valid && tt < nvalid;
      float2* reg = valid ? ys + (size_t)s * REG : dummy;
      const Out dst{y + ((act ? tok0 + tt : 0) * QB + i) * (int64_t)N};
      row_inverse<LOGN, true>(t, act, LdsSpectrum{reg}, dst, reg, tw);
    }
    __syncthreads();
  }
}

// Backward for square layers (q == kb == QB) with few blocks: every thread owns a fixed
// set of (bin, input block) slots for the whole kernel, keeps C_ij[k] and its dC_ij[k]
// partial sums for them in registers, and so touches LDS only to read X_j[k], G_i[k]
// and to write dX_j[k].  With TB > 1 threads per bin (WG > N), the TB threads of a bin
// split the input blocks j into TJ groups and the tokens of a tile into TS phases; with
// BT > 1 bins per thread (N > WG) a thread takes bins kt, kt+WG, ...
constexpr int gcd_int(int a, int b) { return b == 0 ? a : gcd_int(b, a % b); }

template <int LOGN, int QB, int WG>
struct BcaSq {
  static constexpr int N = BcaPlan<LOGN>::N;
  static constexpr int TB = WG >= N ? WG / N : 1;
  static constexpr int BT = WG >= N ? 1 : N / WG;
  static constexpr int TJ = gcd_int(TB, QB);  // input-block groups per bin
  static constexpr int TS = TB / TJ;          // token phases per bin
  static constexpr int JPT = QB / TJ;         // input blocks per thread
  static constexpr int NSL = QB * JPT;        // (i, j) slots per bin per thread
};

template <int LOGN, class St, int QB, int WG = BcaPlan<LOGN>::BWD_WG>
__global__ void __launch_bounds__(WG) bca_backward_sq_kernel(const ElemOf<St>* __restrict__ x, const ElemOf<St>* __restrict__ c,
                                                                      const ElemOf<St>* gy, ElemOf<St>* dx, float* __restrict__ dc,
                                                                      int64_t tokens, int tt_per_tile, int64_t ntiles,
                                                                      float2* stage, int64_t tile_f2, int chunk,
                                                                      const float2* __restrict__ tw) {
  using B = BcaPlan<LOGN>;
  using S = BcaSq<LOGN, QB, WG>;
  using In = typename St::In;
  using Out = typename St::Out;
  constexpr int N = B::N, TPR = B::TPR, NG = WG / TPR, REG = B::REGION;
  constexpr int TB = S::TB, BT = S::BT, TJ = S::TJ, TS = S::TS, JPT = S::JPT, NSL = S::NSL;
  const int tid = threadIdx.x;
  const int grp = tid / TPR, t = tid - grp * TPR;
  const int u = TB > 1 ? tid / N : 0;         // which of the bin's TB threads
  const int kt = TB > 1 ? tid - u * N : tid;  // first bin of this thread
  const int j0 = (u % TJ) * JPT;              // first input block of this thread
  const int tu = u / TJ;                      // token phase
  const int TT = tt_per_tile;
  float2* const xs = bca_lds;                         // TT*QB regions: X, then dX
  float2* const gs = bca_lds + (size_t)TT * QB * REG;  // TT*QB regions: G
  // spare region for row groups without a transform (allocated only when some exist)
  float2* const dummy = bca_lds + (size_t)TT * 2 * QB * REG;
  if (stage != nullptr) {
    // two-stage sum: this kernel never touches dc, and the reduce kernel that adds into it
    // runs after it on the stream, so dc is zeroed here instead of by a launch of its own
    for (int64_t e = (int64_t)blockIdx.x * WG + tid; e < 2 * (int64_t)QB * QB * N; e += (int64_t)gridDim.x * WG)
      dc[e] = 0.f;
  }

  // slot (i, jj) is sl = i*JPT + jj, for input block j = j0 + jj.  C is kept in its
  // storage form (half the registers for 16-bit storage) and widened where it is used.
  typename In::raw_t cr[BT][NSL];
  float2 dcr[BT][NSL];
  {
    const In cin{c};
    static_for<BT>([&](auto wc) {
      constexpr int w = decltype(wc)::value;
      static_for<NSL>([&](auto sc) {
        constexpr int sl = decltype(sc)::value, i = sl / JPT, jj = sl % JPT;
        cr[w][sl] = cin.load_raw((i * QB + j0 + jj) * N + kt + w * WG);  // C_ij[k]
        dcr[w][sl] = make_float2(0.f, 0.f);
      });
    });
  }

  for (int64_t tile = blockIdx.x; tile < ntiles; tile += gridDim.x) {
    const int64_t tok0 = tile * TT;
    const int nvalid = (int)(tokens - tok0 < TT ? tokens - tok0 : TT);

    // Phase A: X_j = rdFFT(x_j), G_i = rdFFT(g_i)
    const int nx = TT * QB, ns = 2 * TT * QB;
    for (int s0 = 0; s0 < ns; s0 += NG) {
      const int s = s0 + grp;
      const bool valid = s < ns;
      float2* reg = valid ? bca_lds + (size_t)s * REG : dummy;
      const int sx = s < nx ? s : s - nx;
      const int tt = sx / QB, j = sx - tt * QB;
      const bool act = valid && tt < nvalid;
      const ElemOf<St>* base = s < nx ? x : gy;
      const ElemOf<St>* srcp = base + ((act ? tok0 + tt : 0) * QB + j) * (int64_t)N;
      row_forward<LOGN, true>(t, act, In{srcp}, LdsSpectrum{reg}, reg, tw);
    }
    __syncthreads();

    // Phase B: per (token, bin): dC_ij += conj(X_j) . G_i and dX_j = sum_i conj(C_ij) . G_i
    static_for<BT>([&](auto wc) {
      constexpr int w = decltype(wc)::value;
      const int k = kt + w * WG;
      const int pk = lds_pad(k);
      auto contract = [&](auto s0c) {
        constexpr bool S0 = decltype(s0c)::value;
        for (int tt = tu; tt < nvalid; tt += TS) {
          float2* xk = xs + ((size_t)tt * QB + j0) * REG + pk;
          const float2* gk = gs + (size_t)tt * QB * REG + pk;
          float2 X[JPT], G[QB];
          static_for<JPT>([&](auto jc) { X[decltype(jc)::value] = xk[decltype(jc)::value * REG]; });
          static_for<QB>([&](auto ic) { G[decltype(ic)::value] = gk[decltype(ic)::value * REG]; });
          static_for<JPT>([&](auto jc) {
            constexpr int jj = decltype(jc)::value;
            float2 d = make_float2(0.f, 0.f);
            static_for<QB>([&](auto ic) {
              constexpr int i = decltype(ic)::value;
              dcr[w][i * JPT + jj] = slot_mac<S0, true>(dcr[w][i * JPT + jj], X[jj], G[i]);
              d = slot_mac<S0, true>(d, In::widen(cr[w][i * JPT + jj]), G[i]);
            });
            xk[jj * REG] = d;
          });
        }
      };
      if (k == 0) contract(std::true_type{});
      else contract(std::false_type{});
    });
    __syncthreads();

    // Phase C: dx_j = irdFFT(dX_j)
    for (int s0 = 0; s0 < nx; s0 += NG) {
      const int s = s0 + grp;
      const bool valid = s < nx;
      const int tt = valid ? s / QB : 0, j = valid ? s - tt * QB : 0;
      const bool act = valid && tt < nvalid;
      float2* reg = valid ? xs + (size_t)s * REG : dummy;
      const Out dst{dx + ((act ? tok0 + tt : 0) * QB + j) * (int64_t)N};
      row_inverse<LOGN, true>(t, act, LdsSpectrum{reg}, dst, reg, tw);
    }
    __syncthreads();
  }

  // Fold the partial sums into dc (slot e = (i*QB + j)*N + k, float2).  They are staged
  // in LDS as [TS][QB*QB*N], the TS token phases summed, and the atomics issued from a
  // rotated start: workgroup b begins 64*b slots in, so that the workgroups, which all
  // finish together, do not queue on the same addresses.
  constexpr int QKN = QB * QB * N;
  float2* const part = bca_lds;
  static_for<BT>([&](auto wc) {
    constexpr int w = decltype(wc)::value;
    static_for<NSL>([&](auto sc) {
      constexpr int sl = decltype(sc)::value, i = sl / JPT, jj = sl % JPT;
      part[(size_t)tu * QKN + (i * QB + j0 + jj) * N + kt + w * WG] = dcr[w][sl];
    });
  });
  __syncthreads();
  if (stage != nullptr) {
    // Two-stage sum (dx is not gy): the partial sums go to the gy rows of this workgroup's
    // first tiles, which it alone has read and nobody reads again, chunk c of them (chunk
    // float2 each) to tile blockIdx.x + c*gridDim.x; bca_dc_finish_kernel then adds the
    // workgroups' partials into dc.
    for (int e = tid; e < QKN; e += WG) {
      float2 v = part[e];
      static_for<TS - 1>([&](auto pc) { v = c_add(v, part[(size_t)(decltype(pc)::value + 1) * QKN + e]); });
      const int ch = e / chunk;
      stage[((int64_t)blockIdx.x + (int64_t)ch * gridDim.x) * tile_f2 + (e - ch * chunk)] = v;
    }
    return;
  }
  const int shift = (int)(((unsigned)blockIdx.x * 64u) % (unsigned)QKN);
  for (int e0 = tid; e0 < QKN; e0 += WG) {
    int e = e0 + shift;
    if (e >= QKN) e -= QKN;
    float2 v = part[e];
    static_for<TS - 1>([&](auto pc) { v = c_add(v, part[(size_t)(decltype(pc)::value + 1) * QKN + e]); });
    unsafeAtomicAdd(dc + 2 * (int64_t)e, v.x);
    unsafeAtomicAdd(dc + 2 * (int64_t)e + 1, v.y);
  }
}

// The fill of dc, and the second stage of the two-stage dC sum (bca_kernels.hip): the
// staged partials of `groups` workgroups for rows_ij rows of n = 2^(logn+1), summed in
// groups of kReduceGroup workgroups, transformed to the time domain and added into the
// zeroed dc.
constexpr int kReduceGroup = 16;
constexpr int64_t kStageMinAtomics = (int64_t)1 << 21;
hipError_t launch_dc_finish(const float2* stage, float* dc, int rows_ij, int logn, int chunk, int groups,
                            int64_t tile_f2, const float2* tw, hipStream_t stream);
hipError_t launch_fill_zero(float* p, int64_t count, hipStream_t stream);

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

constexpr int kBcaMaxLogN = 12;        // p <= 8192
constexpr int kLdsLimit = 160 * 1024;  // gfx950 LDS per workgroup
constexpr int kFwdLdsTarget = 64 * 1024;  // forward: aim for two workgroups per CU

template <int LOGN>
static int fwd_wg() { return BcaPlan<LOGN>::FWD_WG; }
static int bwd_wg(int logn) {
  static const int wg[kBcaMaxLogN + 1] = {
      BcaPlan<0>::BWD_WG, BcaPlan<1>::BWD_WG, BcaPlan<2>::BWD_WG,  BcaPlan<3>::BWD_WG,  BcaPlan<4>::BWD_WG,
      BcaPlan<5>::BWD_WG, BcaPlan<6>::BWD_WG, BcaPlan<7>::BWD_WG,  BcaPlan<8>::BWD_WG,  BcaPlan<9>::BWD_WG,
      BcaPlan<10>::BWD_WG, BcaPlan<11>::BWD_WG, BcaPlan<12>::BWD_WG};
  return wg[logn];
}
static int tpr_of(int logn) {
  static const int tpr[kBcaMaxLogN + 1] = {
      BcaPlan<0>::TPR, BcaPlan<1>::TPR, BcaPlan<2>::TPR, BcaPlan<3>::TPR,  BcaPlan<4>::TPR,  BcaPlan<5>::TPR,
      BcaPlan<6>::TPR, BcaPlan<7>::TPR, BcaPlan<8>::TPR, BcaPlan<9>::TPR, BcaPlan<10>::TPR, BcaPlan<11>::TPR,
      BcaPlan<12>::TPR};
  return tpr[logn];
}

// Tokens per tile: a tile's spectra plus one spare region must fit the LDS budget; the
// tile is grown until every row group has a transform in the output phase.  0 when a
// single token does not fit.
static int tokens_per_tile(int logn, int kb, int q, int64_t tokens, int wg, int budget) {
  const int rb = region_bytes(logn);
  const int64_t per_tok = (int64_t)(kb + q) * rb;
  if (per_tok + rb > budget) return 0;
  const int ng = wg / tpr_of(logn);
  int64_t tt = 1;
  while ((tt + 1) * per_tok + rb <= budget && tt * kb < ng && tt < tokens && tt < 64) ++tt;
  return (int)tt;
}

template <class K>
static hipError_t set_lds_limit(K kernel) {
  return hipFuncSetAttribute(reinterpret_cast<const void*>(kernel), hipFuncAttributeMaxDynamicSharedMemorySize,
                             kLdsLimit);
}

template <int LOGN, class St>
static hipError_t fwd_impl(const BcaArgs& a, const float2* tw, hipStream_t stream) {
  constexpr int WG = BcaPlan<LOGN>::FWD_WG;
  // aim for two workgroups per CU; a token whose spectra exceed that budget gets the whole LDS
  int TT = tokens_per_tile(LOGN, a.kb, a.q, a.tokens, WG, std::max(kFwdLdsTarget, 3 * region_bytes(LOGN)));
  if (TT == 0) TT = tokens_per_tile(LOGN, a.kb, a.q, a.tokens, WG, kLdsLimit);
  if (TT == 0) return hipErrorInvalidValue;
  const size_t lds = (size_t)(TT * (a.kb + a.q) + 1) * region_bytes(LOGN);
  static const hipError_t attr = set_lds_limit(bca_forward_kernel<LOGN, St>);
  if (attr != hipSuccess) return attr;
  // one workgroup per tile, in launches within the grid limit
  const int64_t per_launch = (kMaxGridThreads / WG) * TT;
  constexpr int64_t N = (int64_t)1 << LOGN;
  for (int64_t t0 = 0; t0 < a.tokens; t0 += per_launch) {
    const int64_t nt = std::min<int64_t>(per_launch, a.tokens - t0);
    const int64_t tiles = (nt + TT - 1) / TT;
    hipLaunchKernelGGL((bca_forward_kernel<LOGN, St>), dim3((unsigned)tiles), dim3(WG), lds, stream,
                       static_cast<const ElemOf<St>*>(a.x) + t0 * a.kb * N, static_cast<const ElemOf<St>*>(a.c),
                       static_cast<ElemOf<St>*>(a.y) + t0 * a.q * N, nt, a.q, a.kb, TT, tw);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

// LDS of the backward's dC partial sums: q*kb*p/2 pair slots of float2
static int64_t dc_lds_bytes(int logn, int q, int kb) { return (int64_t)q * kb * ((int64_t)1 << logn) * 8; }

template <int LOGN, class St>
static hipError_t bwd_launch(const BcaArgs& a, const float2* tw, hipStream_t stream, int num_cu, int i0, int ia,
                             int j0, int jb, int mode) {
  constexpr int WG = BcaPlan<LOGN>::BWD_WG;
  const int64_t acc_bytes = (mode & kBwdDc) ? dc_lds_bytes(LOGN, ia, jb) : 0;
  const int TT = tokens_per_tile(LOGN, jb, ia, a.tokens, WG, kLdsLimit - (int)acc_bytes);
  if (TT == 0) return hipErrorInvalidValue;
  const size_t lds = (size_t)(TT * (jb + ia) + 1) * region_bytes(LOGN) + (size_t)acc_bytes;
  static const hipError_t attr = set_lds_limit(bca_backward_kernel<LOGN, St>);
  if (attr != hipSuccess) return attr;
  const int64_t tiles = (a.tokens + TT - 1) / TT;
  // persistent workgroups, as many as fit at once: fewer workgroups, fewer dC partials
  const int per_cu = std::max(1, std::min<int>(kLdsLimit / (int)lds, 2048 / WG));
  const int64_t grid = std::min<int64_t>(tiles, (int64_t)num_cu * per_cu);
  hipLaunchKernelGGL((bca_backward_kernel<LOGN, St>), dim3((unsigned)grid), dim3(WG), lds, stream,
                     static_cast<const ElemOf<St>*>(a.x), static_cast<const ElemOf<St>*>(a.c), static_cast<const ElemOf<St>*>(a.y),
                     static_cast<ElemOf<St>*>(a.dx), a.dc, a.tokens, a.q, a.kb, i0, ia, j0, jb, mode, TT, tiles, tw);
  return hipGetLastError();
}

// Largest block ranges (ia output x jb input blocks) whose dC slots and spectra fit in LDS
// together with one token (0 when even one block does not fit).
static void dc_chunk(int logn, int q, int kb, int* ia, int* jb) {
  const int64_t rb = region_bytes(logn), blk = dc_lds_bytes(logn, 1, 1);
  int best_a = 0, best_b = 0;
  for (int A = 1; A <= q; ++A) {
    for (int Bj = kb; Bj >= 1; --Bj) {
      if (A * Bj * blk + (int64_t)(A + Bj + 1) * rb <= kLdsLimit) {
        const int64_t chunks = (int64_t)((q + A - 1) / A) * ((kb + Bj - 1) / Bj);
        const int64_t best = best_a ? (int64_t)((q + best_a - 1) / best_a) * ((kb + best_b - 1) / best_b) : INT64_MAX;
        if (chunks < best) best_a = A, best_b = Bj;
        break;
      }
    }
  }
  *ia = best_a;
  *jb = best_b;
}

template <int LOGN, class St>
static hipError_t bwd_impl(const BcaArgs& a, const float2* tw, hipStream_t stream, int num_cu) {
  constexpr int WG = BcaPlan<LOGN>::BWD_WG;
  const int64_t acc_bytes = dc_lds_bytes(LOGN, a.q, a.kb);
  if (acc_bytes < kLdsLimit && tokens_per_tile(LOGN, a.kb, a.q, a.tokens, WG, kLdsLimit - (int)acc_bytes) > 0)
    return bwd_launch<LOGN, St>(a, tw, stream, num_cu, 0, a.q, 0, a.kb, kBwdDx | kBwdDc);
  // too many blocks for one LDS-resident dC: dC over block ranges, then the dx path.  The
  // dC launches read gy, and dx may be gy itself, so the dx launch (which reads a tile's gy
  // rows before it writes that tile's dx rows) comes last on the stream.
  int ia = 0, jb = 0;
  dc_chunk(LOGN, a.q, a.kb, &ia, &jb);
  if (ia == 0) return hipErrorInvalidValue;
  hipError_t e = hipSuccess;
  for (int i0 = 0; i0 < a.q && e == hipSuccess; i0 += ia)
    for (int j0 = 0; j0 < a.kb && e == hipSuccess; j0 += jb)
      e = bwd_launch<LOGN, St>(a, tw, stream, num_cu, i0, std::min(ia, a.q - i0), j0, std::min(jb, a.kb - j0),
                                 kBwdDc);
  if (e != hipSuccess) return e;
  return bwd_launch<LOGN, St>(a, tw, stream, num_cu, 0, a.q, 0, a.kb, kBwdDx);
}

// Square layers with few blocks: register-resident C and dC (bca_backward_sq_kernel)
constexpr int kSqMaxBlocks = 4;  // q == kb <= 4
constexpr int kSqMaxSlots = 16;  // C and dC values per thread: bins per thread * q * kb

// Tokens per tile of the square-layer kernels: the largest TT (at most 64 and the token
// count) whose TT*rpt spectra, plus a spare region when TT*QB transforms leave some of
// the ng row groups idle, fit in `budget` bytes.  0 when one token does not fit.
// Tokens per tile of the square-layer kernels: the most whose regions fit `budget`, at most
// 64, and (spread > 0) at most tokens / spread, so that a short batch still reaches `spread`
// workgroups.  The forward spreads over the CUs (the 256-wide layer's 128 tokens: 2 tiles of 64,
// 7.5 us; 128 tiles of 1, 4.0 us); the backward does not, since every workgroup adds a dC
// partial sum (1024-wide, 512 tokens: 31 us as is, 40 us spread).
static int sq_tokens_per_tile(int logn, int rpt, int qb, int ng, int64_t tokens, int64_t budget, bool* spare,
                              int spread = 0) {
  const int64_t rb = region_bytes(logn);
  int64_t top = std::min<int64_t>(64, std::max<int64_t>(tokens, 1));
  if (spread > 0) top = std::min<int64_t>(top, std::max<int64_t>(1, (tokens + spread - 1) / spread));
  for (int tt = (int)top; tt >= 1; --tt) {
    const bool sp = (tt * qb) % ng != 0;
    if ((tt * rpt + (sp ? 1 : 0)) * rb <= budget) {
      *spare = sp;
      return tt;
    }
  }
  return 0;
}

template <int LOGN, int QB>
constexpr bool sq_fwd_fits() {
  using S = BcaSqFwd<LOGN, QB, kFwdSqWG>;
  return BcaPlan<LOGN>::TPR <= kFwdSqWG / 2 && S::BT * S::NSL <= kSqMaxSlots && S::TS <= 8;
}

template <int LOGN, class St, int QB>
static hipError_t fwd_sq_impl(const BcaArgs& a, const float2* tw, hipStream_t stream, int num_cu) {
  constexpr int WG = kFwdSqWG;
  using S = BcaSqFwd<LOGN, QB, WG>;
  constexpr int rpt = (S::TB == 1 ? 1 : 2) * QB;  // regions per token (Y over X when TB == 1)
  constexpr int ng = WG / BcaPlan<LOGN>::TPR;
  // two workgroups per CU, or one when a token's spectra need more than half the LDS
  bool spare = false;
  int TT = sq_tokens_per_tile(LOGN, rpt, QB, ng, a.tokens, kLdsLimit / 2, &spare, num_cu);
  if (TT == 0) TT = sq_tokens_per_tile(LOGN, rpt, QB, ng, a.tokens, kLdsLimit, &spare, num_cu);
  if (TT == 0) return hipErrorInvalidValue;
  const size_t lds = (size_t)(TT * rpt + (spare ? 1 : 0)) * region_bytes(LOGN);
  static const hipError_t attr = set_lds_limit(bca_forward_sq_kernel<LOGN, St, QB>);
  if (attr != hipSuccess) return attr;
  const int64_t tiles = (a.tokens + TT - 1) / TT;
  const int per_cu = std::max(1, std::min<int>(kLdsLimit / (int)lds, 2048 / WG));
  const int64_t grid = std::min<int64_t>(tiles, (int64_t)num_cu * per_cu);
  hipLaunchKernelGGL((bca_forward_sq_kernel<LOGN, St, QB>), dim3((unsigned)grid), dim3(WG), lds, stream,
                     static_cast<const ElemOf<St>*>(a.x), static_cast<const ElemOf<St>*>(a.c), static_cast<ElemOf<St>*>(a.y), a.tokens,
                     TT, tiles, tw);
  return hipGetLastError();
}

template <int LOGN, int QB>
constexpr bool sq_fits() {
  using S = BcaSq<LOGN, QB, BcaPlan<LOGN>::BWD_WG>;
  return S::BT * S::NSL <= kSqMaxSlots && S::TS <= 8;  // short rows: many threads per bin
}

template <int LOGN, class St, int QB>
static hipError_t bwd_sq_impl(const BcaArgs& a, const float2* tw, hipStream_t stream, int num_cu) {
  constexpr int WG = BcaPlan<LOGN>::BWD_WG;
  using S = BcaSq<LOGN, QB, WG>;
  bool spare = false;
  const int TT = sq_tokens_per_tile(LOGN, 2 * QB, QB, WG / BcaPlan<LOGN>::TPR, a.tokens, kLdsLimit, &spare);
  if (TT == 0) return hipErrorInvalidValue;
  const size_t spectra = (size_t)(TT * 2 * QB + (spare ? 1 : 0)) * region_bytes(LOGN);
  const size_t part = (size_t)S::TS * QB * QB * S::N * sizeof(float2);  // [TS][QB*QB*N]
  const size_t lds = std::max(spectra, part);
  if (lds > (size_t)kLdsLimit) return hipErrorInvalidValue;
  static const hipError_t attr = set_lds_limit(bca_backward_sq_kernel<LOGN, St, QB>);
  if (attr != hipSuccess) return attr;
  const int64_t tiles = (a.tokens + TT - 1) / TT;
  const int per_cu = std::max(1, std::min<int>(kLdsLimit / (int)lds, 2048 / WG));
  const int64_t grid = std::min<int64_t>(tiles, (int64_t)num_cu * per_cu);
  // Two-stage dC sum when dx has its own buffer: each workgroup's partial sums (QKN float2)
  // fit in the gy rows of its first `chunks` tiles, all of them full tiles
  constexpr int QKN = QB * QB * S::N;
  const int64_t tile_bytes = (int64_t)TT * QB * S::N * (int64_t)sizeof(ElemOf<St>);
  const int64_t tile_f2 = tile_bytes / (int64_t)sizeof(float2);
  const int chunk = (int)std::max<int64_t>(1, std::min<int64_t>(QKN, tile_f2));
  const int64_t chunks = (QKN + chunk - 1) / chunk;
  // (worth a second launch only when the atomics it replaces are many: 4.2M float32 atomics
  // for the 4096-wide layer took ~24 us, 0.6M for the 768-wide one less than the launch)
  const bool staged = a.dx != a.y && tile_bytes % (int64_t)sizeof(float2) == 0 && chunks * grid <= a.tokens / TT &&
                      2 * (int64_t)QKN * grid >= kStageMinAtomics;
  float2* const stage = staged ? static_cast<float2*>(a.y) : nullptr;
  if (!staged) {  // the kernel's atomics add into dc
    const hipError_t ez = launch_fill_zero(a.dc, 2 * (int64_t)QKN, stream);
    if (ez != hipSuccess) return ez;
  }
  hipLaunchKernelGGL((bca_backward_sq_kernel<LOGN, St, QB>), dim3((unsigned)grid), dim3(WG), lds, stream,
                     static_cast<const ElemOf<St>*>(a.x), static_cast<const ElemOf<St>*>(a.c), static_cast<const ElemOf<St>*>(a.y),
                     static_cast<ElemOf<St>*>(a.dx), a.dc, a.tokens, TT, tiles, stage, tile_f2, chunk, tw);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (staged) return launch_dc_finish(stage, a.dc, QB * QB, LOGN, chunk, (int)grid, tile_f2, tw, stream);
  // dc holds sum_t conj(X) . G as packed spectra; transform them in place to the time domain
  return launch_rdfft_rows(a.dc, (int64_t)QB * QB, LOGN, kStorageF32, true, tw, stream, num_cu);
}

// ----------------------------------------------------------------------------------
// Square layers (q == kb == QB) with short blocks, whose rows fit inside one wavefront
// (TPR <= 64, at least 64 bins).  Every wave works on its own groups of TW tokens: its
// transforms, per-bin products and inverse transforms synchronise at wave level only, so
// no wave waits for another; a workgroup's waves share nothing but the backward's final
// dC reduction.  Lane l owns bins l, l + 64, ... (BL of them): it reads C_ij[k] for a bin
// once per group (from L1/L2: C is small) and, in the backward, keeps its dC_ij[k] sums in
// registers for the whole kernel.
//
// Each group first takes a copy of the twiddle pointer that the compiler cannot see
// through: otherwise it hoists the loop-invariant twiddle reads of every transform out of
// the group loop and keeps them all in registers, which spilled.
template <int LOGN, int QB>
struct BcaWave {
  using P = RowPlan<LOGN>;
  static constexpr int N = P::N, TPR = P::TPR;
  static constexpr int G = TPR <= 64 ? 64 / TPR : 1;  // rows one wave transforms at a time
  static constexpr int BL = N >= 64 ? N / 64 : 1;      // bins per lane
  static constexpr int REG = BcaPlan<LOGN>::REGION;
  static constexpr int CS = BL * QB * QB;                // dC slots per lane
};
// waves per workgroup: the forward's workgroups are independent sets of waves; the
// backward runs one wider workgroup per CU, whose waves add their dC before it leaves
constexpr int kWaveFwdNW = 4, kWaveBwdNW = 8;
// asked of the compiler: at least this many waves per SIMD (at most 128 VGPRs), so that a
// CU keeps enough waves in flight to cover their memory and LDS latency.  The backward
// runs one workgroup of kWaveBwdNW waves per CU, two per SIMD, so more registers cost it
// nothing (and its dC sums live in them).
constexpr int kWaveMinWaves = 4, kWaveBwdMinWaves = 2;

template <int LOGN, int QB>
constexpr bool wave_fits(bool backward) {
  using W = BcaWave<LOGN, QB>;
  return W::TPR <= 64 && W::N >= 64 && W::N <= 256 && (backward ? W::CS <= 18 : W::CS <= 32);
}

// Tokens per wave group: the rows of a group (QB per token and direction) fill whole
// rounds of G row slots where that keeps a wave's LDS small; otherwise short groups.
template <int LOGN, int QB>
constexpr int wave_tokens() {
  constexpr int G = BcaWave<LOGN, QB>::G;
  return G % QB == 0 ? G / QB : (G >= 2 * QB ? G / QB : 1);
}

// The tensors of the layers a wave-kernel launch serves: layer b (grid row blockIdx.y when
// MAXB > 1) reads x[b], c[b] and writes y[b] (forward), or reads x[b], c[b], y[b] = gy and
// writes dx[b], dc[b] (backward).
template <class St, int MAXB>
struct WavePtrs {
  const ElemOf<St>* x[MAXB];
  const ElemOf<St>* c[MAXB];
  ElemOf<St>* y[MAXB];
  ElemOf<St>* dx[MAXB];
  float* dc[MAXB];
};

// Forward: per group, X_j = rdFFT(x_j) into the wave's LDS regions, Y_i = sum_j C_ij X_j
// per bin written over X_i (a lane reads every X_j[k] of its bin before it writes), then
// y_i = irdFFT(Y_i).  y may be x: a wave reads its group's x rows before it writes the
// group's y rows, and no other wave touches them.
template <int LOGN, class St, int QB, int TW, int MAXB, int NW = kWaveFwdNW>
__global__ void __launch_bounds__(64 * NW) __attribute__((amdgpu_waves_per_eu(kWaveMinWaves)))
bca_forward_wave_kernel(WavePtrs<St, MAXB> ptrs, int64_t tokens, int64_t ngroups, const float2* __restrict__ tw) {
  const int bi = MAXB == 1 ? 0 : (int)blockIdx.y;
  const ElemOf<St>* x = ptrs.x[bi];
  const ElemOf<St>* __restrict__ c = ptrs.c[bi];
  ElemOf<St>* y = ptrs.y[bi];
  using W = BcaWave<LOGN, QB>;
  using In = typename St::In;
  using Out = typename St::Out;
  constexpr int N = W::N, TPR = W::TPR, G = W::G, BL = W::BL, REG = W::REG;
  constexpr int NR = TW * QB, ROUNDS = (NR + G - 1) / G;
  constexpr int WREGS = NR + (NR % G != 0 ? 1 : 0);  // + a spare region for idle row slots
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int grp = lane / TPR, t = lane - grp * TPR;
  float2* const xs = bca_lds + (size_t)wave * WREGS * REG;
  float2* const spare = xs + (size_t)NR * REG;
  const int64_t wstride = (int64_t)gridDim.x * NW;
  for (int64_t gi = (int64_t)blockIdx.x * NW + wave; gi < ngroups; gi += wstride) {
    const int64_t tok0 = gi * TW;
    const int nvalid = (int)(tokens - tok0 < TW ? tokens - tok0 : TW);
    const float2* twg = tw;
    asm volatile("" : "+s"(twg));
    // (runtime loops over the rounds: unrolled, the compiler hoists every round's loads)
#pragma unroll 1
    for (int r = 0; r < ROUNDS; ++r) {
      const int s = r * G + grp;
      const bool valid = s < NR;
      const int tt = valid ? s / QB : 0, j = valid ? s - tt * QB : 0;
      const bool act = valid && tt < nvalid;
      float2* reg = valid ? xs + (size_t)s * REG : spare;
      const In src{x + ((act ? tok0 + tt : 0) * QB + j) * (int64_t)N};
      row_forward<LOGN, true>(t, act, src, LdsSpectrum{reg}, reg, twg);
    }
    row_sync<64>();
    static_for<BL>([&](auto bc) {
      constexpr int b = decltype(bc)::value;
      const int k = lane + 64 * b;
      typename In::raw_t cb[QB * QB];
      {
        const In cin{c};
        static_for<QB * QB>([&](auto sc) { cb[decltype(sc)::value] = cin.load_raw(decltype(sc)::value * N + k); });
      }
      for (int tt = 0; tt < nvalid; ++tt) {
        float2* xk = xs + (size_t)tt * QB * REG + lds_pad(k);
        auto block_sum = [&](auto s0c) {
          constexpr bool S0 = decltype(s0c)::value;
          float2 X[QB];
          static_for<QB>([&](auto jc) { X[decltype(jc)::value] = xk[decltype(jc)::value * REG]; });
          static_for<QB>([&](auto ic) {
            constexpr int i = decltype(ic)::value;
            float2 a = make_float2(0.f, 0.f);
            static_for<QB>([&](auto jc) {
              constexpr int j = decltype(jc)::value;
              a = slot_mac<S0, false>(a, In::widen(cb[i * QB + j]), X[j]);
            });
            xk[i * REG] = a;
          });
        };
        if (b == 0 && lane == 0) block_sum(std::true_type{});
        else block_sum(std::false_type{});
      }
    });
    row_sync<64>();
#pragma unroll 1
    for (int r = 0; r < ROUNDS; ++r) {
      const int s = r * G + grp;
      const bool valid = s < NR;
      const int tt = valid ? s / QB : 0, i = valid ? s - tt * QB : 0;
      const bool act = valid && tt < nvalid;
      float2* reg = valid ? xs + (size_t)s * REG : spare;
      const Out dst{y + ((act ? tok0 + tt : 0) * QB + i) * (int64_t)N};
      row_inverse<LOGN, true>(t, act, LdsSpectrum{reg}, dst, reg, twg);
    }
    row_sync<64>();  // the next group's transforms reuse the regions
  }
}

// Backward: per group, X_j = rdFFT(x_j) and G_i = rdFFT(g_i) into LDS; per bin
// dC_ij += conj(X_j) G_i (registers, summed over all of the wave's groups) and
// dX_j = sum_i conj(C_ij) G_i written over X_j; dx_j = irdFFT(dX_j).  At the end the
// workgroup's four waves add their dC in LDS, and the sum goes to dc by float32 atomics
// (stage == nullptr; dc zeroed beforehand) or is written to `stage` at
// blockIdx.x * stage_f2 for bca_dc_finish_kernel (then this kernel zeroes dc).
template <int LOGN, class St, int QB, int TW, int MAXB, int NW = kWaveBwdNW>
__global__ void __launch_bounds__(64 * NW) __attribute__((amdgpu_waves_per_eu(kWaveBwdMinWaves)))
bca_backward_wave_kernel(WavePtrs<St, MAXB> ptrs, int64_t tokens, int64_t ngroups, int staged, int64_t stage_f2,
                         const float2* __restrict__ tw) {
  const int bi = MAXB == 1 ? 0 : (int)blockIdx.y;
  const ElemOf<St>* __restrict__ x = ptrs.x[bi];
  const ElemOf<St>* __restrict__ c = ptrs.c[bi];
  const ElemOf<St>* gy = ptrs.y[bi];
  ElemOf<St>* dx = ptrs.dx[bi];
  float* __restrict__ dc = ptrs.dc[bi];
  float2* const stage = staged ? reinterpret_cast<float2*>(ptrs.y[bi]) : nullptr;
  using W = BcaWave<LOGN, QB>;
  using In = typename St::In;
  using Out = typename St::Out;
  constexpr int N = W::N, TPR = W::TPR, G = W::G, BL = W::BL, REG = W::REG, CS = W::CS;
  constexpr int NR = TW * QB, NA = 2 * NR;
  constexpr int ROUNDS_A = (NA + G - 1) / G, ROUNDS_C = (NR + G - 1) / G;
  constexpr int WREGS = NA + (NA % G != 0 || NR % G != 0 ? 1 : 0);
  constexpr int QKN = QB * QB * N;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int grp = lane / TPR, t = lane - grp * TPR;
  float2* const xs = bca_lds + (size_t)wave * WREGS * REG;  // NR regions: X, then dX
  float2* const gs = xs + (size_t)NR * REG;                   // NR regions: G
  float2* const spare = xs + (size_t)NA * REG;
  if (stage != nullptr) {
    // the reduce kernel that adds into dc runs after this one on the stream
    for (int64_t e = (int64_t)blockIdx.x * (64 * NW) + threadIdx.x; e < 2 * (int64_t)QKN;
         e += (int64_t)gridDim.x * (64 * NW))
      dc[e] = 0.f;
  }
  float2 dcr[CS];
  static_for<CS>([&](auto sc) { dcr[decltype(sc)::value] = make_float2(0.f, 0.f); });

  const int64_t wstride = (int64_t)gridDim.x * NW;
  for (int64_t gi = (int64_t)blockIdx.x * NW + wave; gi < ngroups; gi += wstride) {
    const int64_t tok0 = gi * TW;
    const int nvalid = (int)(tokens - tok0 < TW ? tokens - tok0 : TW);
    const float2* twg = tw;
    asm volatile("" : "+s"(twg));
#pragma unroll 1
    for (int r = 0; r < ROUNDS_A; ++r) {
      const int s = r * G + grp;
      const bool valid = s < NA;
      const int sx = s < NR ? s : s - NR;
      const int tt = valid ? sx / QB : 0, j = valid ? sx - tt * QB : 0;
      const bool act = valid && tt < nvalid;
      float2* reg = valid ? xs + (size_t)s * REG : spare;
      const ElemOf<St>* base = s < NR ? x : gy;
      const In src{base + ((act ? tok0 + tt : 0) * QB + j) * (int64_t)N};
      row_forward<LOGN, true>(t, act, src, LdsSpectrum{reg}, reg, twg);
    }
    row_sync<64>();
    static_for<BL>([&](auto bc) {
      constexpr int b = decltype(bc)::value;
      const int k = lane + 64 * b;
      typename In::raw_t cb[QB * QB];
      {
        const In cin{c};
        static_for<QB * QB>([&](auto sc) { cb[decltype(sc)::value] = cin.load_raw(decltype(sc)::value * N + k); });
      }
      for (int tt = 0; tt < nvalid; ++tt) {
        float2* xk = xs + (size_t)tt * QB * REG + lds_pad(k);
        const float2* gk = gs + (size_t)tt * QB * REG + lds_pad(k);
        auto contract = [&](auto s0c) {
          constexpr bool S0 = decltype(s0c)::value;
          float2 X[QB], Gv[QB];
          static_for<QB>([&](auto jc) { X[decltype(jc)::value] = xk[decltype(jc)::value * REG]; });
          static_for<QB>([&](auto ic) { Gv[decltype(ic)::value] = gk[decltype(ic)::value * REG]; });
          static_for<QB>([&](auto jc) {
            constexpr int j = decltype(jc)::value;
            float2 d = make_float2(0.f, 0.f);
            static_for<QB>([&](auto ic) {
              constexpr int i = decltype(ic)::value, sl = b * QB * QB + i * QB + j;
              dcr[sl] = slot_mac<S0, true>(dcr[sl], X[j], Gv[i]);
              d = slot_mac<S0, true>(d, In::widen(cb[i * QB + j]), Gv[i]);
            });
            xk[j * REG] = d;
          });
        };
        if (b == 0 && lane == 0) contract(std::true_type{});
        else contract(std::false_type{});
      }
    });
    row_sync<64>();
#pragma unroll 1
    for (int r = 0; r < ROUNDS_C; ++r) {
      const int s = r * G + grp;
      const bool valid = s < NR;
      const int tt = valid ? s / QB : 0, j = valid ? s - tt * QB : 0;
      const bool act = valid && tt < nvalid;
      float2* reg = valid ? xs + (size_t)s * REG : spare;
      const Out dst{dx + ((act ? tok0 + tt : 0) * QB + j) * (int64_t)N};
      row_inverse<LOGN, true>(t, act, LdsSpectrum{reg}, dst, reg, twg);
    }
    row_sync<64>();
  }

  // the workgroup's dC: wave w's slot (i*QB + j)*N + k at part[w*QKN + ...]
  __syncthreads();
  float2* const part = bca_lds;
  static_for<BL>([&](auto bc) {
    constexpr int b = decltype(bc)::value;
    static_for<QB * QB>([&](auto sc) {
      constexpr int sl = decltype(sc)::value;
      part[(size_t)wave * QKN + sl * N + lane + 64 * b] = dcr[b * QB * QB + sl];
    });
  });
  __syncthreads();
  if (stage != nullptr) {
    for (int e = threadIdx.x; e < QKN; e += (64 * NW)) {
      float2 v = part[e];
      static_for<NW - 1>([&](auto wc) { v = c_add(v, part[(size_t)(decltype(wc)::value + 1) * QKN + e]); });
      stage[(int64_t)blockIdx.x * stage_f2 + e] = v;
    }
    return;
  }
  const int shift = (int)(((unsigned)blockIdx.x * 64u) % (unsigned)QKN);
  for (int e0 = threadIdx.x; e0 < QKN; e0 += (64 * NW)) {
    int e = e0 + shift;
    if (e >= QKN) e -= QKN;
    float2 v = part[e];
    static_for<NW - 1>([&](auto wc) { v = c_add(v, part[(size_t)(decltype(wc)::value + 1) * QKN + e]); });
    unsafeAtomicAdd(dc + 2 * (int64_t)e, v.x);
    unsafeAtomicAdd(dc + 2 * (int64_t)e + 1, v.y);
  }
}

// LDS of one workgroup of the wave kernels
template <int LOGN, int QB>
constexpr size_t wave_lds_bytes(bool backward) {
  using W = BcaWave<LOGN, QB>;
  constexpr int TW = wave_tokens<LOGN, QB>(), NR = TW * QB;
  const int nw = backward ? kWaveBwdNW : kWaveFwdNW;
  const int na = backward ? 2 * NR : NR;
  const bool spare = na % W::G != 0 || NR % W::G != 0;
  const size_t spectra = (size_t)nw * (na + (spare ? 1 : 0)) * W::REG * sizeof(float2);
  const size_t part = backward ? (size_t)nw * QB * QB * W::N * sizeof(float2) : 0;
  return spectra > part ? spectra : part;
}

// Wave-kernel launches for `count` layers of one shape (count <= MAXB).  Layers share the
// chip: each gets about 1/count of the workgroups one layer alone would get.
template <int LOGN, class St, int QB, int MAXB>
static hipError_t fwd_wave_launch(const WavePtrs<St, MAXB>& ptrs, int count, int64_t tokens, const float2* tw,
                                  hipStream_t stream, int num_cu) {
  constexpr int TW = wave_tokens<LOGN, QB>(), NW = kWaveFwdNW;
  constexpr size_t lds = wave_lds_bytes<LOGN, QB>(false);
  static_assert(lds <= (size_t)kLdsLimit, "wave groups too large for LDS");
  static const hipError_t attr = set_lds_limit(bca_forward_wave_kernel<LOGN, St, QB, TW, MAXB>);
  if (attr != hipSuccess) return attr;
  const int64_t groups = (tokens + TW - 1) / TW;
  // every wave takes groups until none are left; enough workgroups for a full chip
  const int per_cu = std::max(1, std::min<int>(kLdsLimit / (int)lds, 2048 / (64 * NW)));
  const int64_t slots = ((int64_t)num_cu * per_cu + count - 1) / count;
  const int64_t grid = std::max<int64_t>(1, std::min<int64_t>((groups + NW - 1) / NW, slots));
  hipLaunchKernelGGL((bca_forward_wave_kernel<LOGN, St, QB, TW, MAXB>), dim3((unsigned)grid, (unsigned)count),
                     dim3(64 * NW), lds, stream, ptrs, tokens, groups, tw);
  return hipGetLastError();
}

template <int LOGN, class St, int QB>
static hipError_t fwd_wave_impl(const BcaArgs& a, const float2* tw, hipStream_t stream, int num_cu) {
  const WavePtrs<St, 1> p{{static_cast<const ElemOf<St>*>(a.x)}, {static_cast<const ElemOf<St>*>(a.c)},
                          {static_cast<ElemOf<St>*>(a.y)}, {nullptr}, {nullptr}};
  return fwd_wave_launch<LOGN, St, QB, 1>(p, 1, a.tokens, tw, stream, num_cu);
}

// The two-stage dC sum of `count` layers: layer b's partials in its own gy rows, its sum in
// its own dc (bca_kernels.hip)
template <int MAXB>
struct FinishPtrs {
  const float2* stage[MAXB];
  float* dc[MAXB];
};
hipError_t launch_dc_finish_batched(const FinishPtrs<kMaxBatch>& p, int count, int rows_ij, int logn, int chunk,
                                    int groups, int64_t tile_f2, const float2* tw, hipStream_t stream);

template <int LOGN, class St, int QB, int MAXB>
static hipError_t bwd_wave_launch(const WavePtrs<St, MAXB>& ptrs, int count, bool apart, int64_t tokens,
                                  const float2* tw, hipStream_t stream, int num_cu) {
  using W = BcaWave<LOGN, QB>;
  constexpr int TW = wave_tokens<LOGN, QB>(), NW = kWaveBwdNW;
  constexpr size_t lds = wave_lds_bytes<LOGN, QB>(true);
  static_assert(lds <= (size_t)kLdsLimit, "wave groups too large for LDS");
  constexpr int QKN = QB * QB * W::N;
  static const hipError_t attr = set_lds_limit(bca_backward_wave_kernel<LOGN, St, QB, TW, MAXB>);
  if (attr != hipSuccess) return attr;
  const int64_t groups = (tokens + TW - 1) / TW;
  // one workgroup per CU in all: fewer workgroups, fewer dC partial sums to add
  const int64_t grid = std::max<int64_t>(1, std::min<int64_t>((groups + NW - 1) / NW, num_cu / count));
  // Two-stage dC sum when dx has its own buffer (apart): workgroup b's first groups are the
  // tokens [b*NW*TW, (b+1)*NW*TW), whose gy rows only it reads; once all its waves are
  // done it writes its partial sums there (QKN float2 must fit those rows, all of them
  // valid tokens)
  const int64_t region_f2 = (int64_t)NW * TW * QB * W::N * (int64_t)sizeof(ElemOf<St>) / (int64_t)sizeof(float2);
  const bool staged = apart && region_f2 >= QKN && grid * NW * TW <= tokens;
  if (!staged && count > 1) {
    // too few tokens to stage a batch's partial sums: the layers one by one
    for (int b = 0; b < count; ++b) {
      const WavePtrs<St, 1> p1{{ptrs.x[b]}, {ptrs.c[b]}, {ptrs.y[b]}, {ptrs.dx[b]}, {ptrs.dc[b]}};
      const hipError_t e1 = bwd_wave_launch<LOGN, St, QB, 1>(p1, 1, apart, tokens, tw, stream, num_cu);
      if (e1 != hipSuccess) return e1;
    }
    return hipSuccess;
  }
  if (!staged) {
    const hipError_t ez = launch_fill_zero(ptrs.dc[0], 2 * (int64_t)QKN, stream);
    if (ez != hipSuccess) return ez;
  }
  hipLaunchKernelGGL((bca_backward_wave_kernel<LOGN, St, QB, TW, MAXB>), dim3((unsigned)grid, (unsigned)count),
                     dim3(64 * NW), lds, stream, ptrs, tokens, groups, staged ? 1 : 0, region_f2, tw);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (staged) {
    if (count == 1)
      return launch_dc_finish(reinterpret_cast<const float2*>(ptrs.y[0]), ptrs.dc[0], QB * QB, LOGN, QKN, (int)grid,
                              region_f2, tw, stream);
    FinishPtrs<kMaxBatch> f{};
    for (int b = 0; b < count; ++b) {
      f.stage[b] = reinterpret_cast<const float2*>(ptrs.y[b]);
      f.dc[b] = ptrs.dc[b];
    }
    return launch_dc_finish_batched(f, count, QB * QB, LOGN, QKN, (int)grid, region_f2, tw, stream);
  }
  return launch_rdfft_rows(ptrs.dc[0], (int64_t)QB * QB, LOGN, kStorageF32, true, tw, stream, num_cu);
}

template <int LOGN, class St, int QB>
static hipError_t bwd_wave_impl(const BcaArgs& a, const float2* tw, hipStream_t stream, int num_cu) {
  const WavePtrs<St, 1> p{{static_cast<const ElemOf<St>*>(a.x)}, {static_cast<const ElemOf<St>*>(a.c)},
                          {static_cast<ElemOf<St>*>(a.y)}, {static_cast<ElemOf<St>*>(a.dx)}, {a.dc}};
  return bwd_wave_launch<LOGN, St, QB, 1>(p, 1, a.dx != a.y, a.tokens, tw, stream, num_cu);
}

// Batches: kMaxBatch-wide pointer lists, count layers in grid rows
template <int LOGN, class St>
static WavePtrs<St, kMaxBatch> batch_ptrs(const BcaBatch& b) {
  WavePtrs<St, kMaxBatch> p{};
  for (int i = 0; i < b.count; ++i) {
    p.x[i] = static_cast<const ElemOf<St>*>(b.x[i]);
    p.c[i] = static_cast<const ElemOf<St>*>(b.c[i]);
    p.y[i] = static_cast<ElemOf<St>*>(b.y[i]);
    p.dx[i] = static_cast<ElemOf<St>*>(b.dx[i]);
    p.dc[i] = b.dc[i];
  }
  return p;
}
template <int LOGN, class St, int QB>
static hipError_t fwd_wave_batched(const BcaArgs& a, const BcaBatch& b, const float2* tw, hipStream_t stream,
                                   int num_cu) {
  return fwd_wave_launch<LOGN, St, QB, kMaxBatch>(batch_ptrs<LOGN, St>(b), b.count, a.tokens, tw, stream, num_cu);
}
template <int LOGN, class St, int QB>
static hipError_t bwd_wave_batched(const BcaArgs& a, const BcaBatch& b, const float2* tw, hipStream_t stream,
                                   int num_cu) {
  return bwd_wave_launch<LOGN, St, QB, kMaxBatch>(batch_ptrs<LOGN, St>(b), b.count, true, a.tokens, tw, stream,
                                                  num_cu);
}

using BcaFn = hipError_t (*)(const BcaArgs&, const float2*, hipStream_t);
using BcaBwdFn = hipError_t (*)(const BcaArgs&, const float2*, hipStream_t, int);

template <int LOGN, class St, int QB>
static constexpr BcaBwdFn sq_fwd_entry() {
  if constexpr (sq_fwd_fits<LOGN, QB>()) return &fwd_sq_impl<LOGN, St, QB>;
  else return nullptr;
}
template <class St, int QB, int... L>
static std::array<BcaBwdFn, sizeof...(L)> sq_fwd_row(std::integer_sequence<int, L...>) {
  return {sq_fwd_entry<L, St, QB>()...};
}

template <int LOGN, class St, int QB>
static constexpr BcaBwdFn sq_entry() {
  if constexpr (sq_fits<LOGN, QB>()) return &bwd_sq_impl<LOGN, St, QB>;
  else return nullptr;
}
template <class St, int QB, int... L>
static std::array<BcaBwdFn, sizeof...(L)> sq_row(std::integer_sequence<int, L...>) {
  return {sq_entry<L, St, QB>()...};
}

template <class St, int... L>
static std::array<BcaFn, sizeof...(L)> fwd_row(std::integer_sequence<int, L...>) {
  return {&fwd_impl<L, St>...};
}
template <class St, int... L>
static std::array<BcaBwdFn, sizeof...(L)> bwd_row(std::integer_sequence<int, L...>) {
  return {&bwd_impl<L, St>...};
}

constexpr int kStorages = 3;  // indexed by BcaArgs::storage: float32, bf16, f16
using SeqP = std::make_integer_sequence<int, kBcaMaxLogN + 1>;
using SqTable = std::array<std::array<BcaBwdFn, kBcaMaxLogN + 1>, kSqMaxBlocks>;

template <class St>
static SqTable sq_fwd_tables() {
  return {sq_fwd_row<St, 1>(SeqP{}), sq_fwd_row<St, 2>(SeqP{}), sq_fwd_row<St, 3>(SeqP{}), sq_fwd_row<St, 4>(SeqP{})};
}
template <class St>
static SqTable sq_bwd_tables() {
  return {sq_row<St, 1>(SeqP{}), sq_row<St, 2>(SeqP{}), sq_row<St, 3>(SeqP{}), sq_row<St, 4>(SeqP{})};
}

// The launchers of one storage type, indexed by log2(p/2) (and q - 1 for the square-layer
// kernels; nullptr where those kernels do not fit).
using BcaBatchFn = hipError_t (*)(const BcaArgs&, const BcaBatch&, const float2*, hipStream_t, int);
using BatchTable = std::array<std::array<BcaBatchFn, kBcaMaxLogN + 1>, kSqMaxBlocks>;

struct BcaStoreTables {
  std::array<BcaFn, kBcaMaxLogN + 1> fwd;
  std::array<BcaBwdFn, kBcaMaxLogN + 1> bwd;
  SqTable sq_fwd;
  SqTable sq_bwd;
  SqTable wave_fwd;
  SqTable wave_bwd;
  BatchTable wave_fwd_batched;
  BatchTable wave_bwd_batched;
};

template <int LOGN, class St, int QB>
static constexpr BcaBwdFn wave_entry(bool backward) {
  if constexpr (wave_fits<LOGN, QB>(true)) {
    return backward ? &bwd_wave_impl<LOGN, St, QB> : &fwd_wave_impl<LOGN, St, QB>;
  } else if constexpr (wave_fits<LOGN, QB>(false)) {
    return backward ? nullptr : &fwd_wave_impl<LOGN, St, QB>;
  } else {
    return nullptr;
  }
}
template <class St, int QB, int... L>
static std::array<BcaBwdFn, sizeof...(L)> wave_row(bool backward, std::integer_sequence<int, L...>) {
  return {wave_entry<L, St, QB>(backward)...};
}
template <class St>
static SqTable wave_tables(bool backward) {
  return {wave_row<St, 1>(backward, SeqP{}), wave_row<St, 2>(backward, SeqP{}), wave_row<St, 3>(backward, SeqP{}),
          wave_row<St, 4>(backward, SeqP{})};
}

template <int LOGN, class St, int QB>
static constexpr BcaBatchFn batch_entry(bool backward) {
  if constexpr (wave_fits<LOGN, QB>(true)) {
    return backward ? &bwd_wave_batched<LOGN, St, QB> : &fwd_wave_batched<LOGN, St, QB>;
  } else if constexpr (wave_fits<LOGN, QB>(false)) {
    return backward ? nullptr : &fwd_wave_batched<LOGN, St, QB>;
  } else {
    return nullptr;
  }
}
template <class St, int QB, int... L>
static std::array<BcaBatchFn, sizeof...(L)> batch_row(bool backward, std::integer_sequence<int, L...>) {
  return {batch_entry<L, St, QB>(backward)...};
}
template <class St>
static BatchTable batch_tables(bool backward) {
  return {batch_row<St, 1>(backward, SeqP{}), batch_row<St, 2>(backward, SeqP{}), batch_row<St, 3>(backward, SeqP{}),
          batch_row<St, 4>(backward, SeqP{})};
}

template <class St>
BcaStoreTables make_store_tables() {
  return {fwd_row<St>(SeqP{}),     bwd_row<St>(SeqP{}),     sq_fwd_tables<St>(),    sq_bwd_tables<St>(),
          wave_tables<St>(false), wave_tables<St>(true),  batch_tables<St>(false), batch_tables<St>(true)};
}

BcaStoreTables bca_tables_f32();
BcaStoreTables bca_tables_bf16();
BcaStoreTables bca_tables_f16();

}  // namespace rdfft
