// bca_multipass.hip -- the block-circulant layer for blocks too long for one workgroup's
// LDS budget next to a second spectrum: 8192 < p <= 65536.
//
// The steps of Eqs. (4)-(5) run as separate passes over HBM.  The intermediate spectra
// live in the caller's own output buffers, so the layer still needs no memory beyond
// them:
//   forward   X_tj = FFT(x_tj) into y's segment j (when kb <= q and kb <= 8), then per
//             bin Y_ti = sum_j C_ij X_tj in place, then y_ti = IFFT(Y_ti) in place.
//             Other shapes (y distinct from x) take one pass per input block j instead:
//             the transform of x_tj hands each bin of X_tj to the store, which adds
//             C_ij X_tj into every Y_ti in y (the first pass writes), so no input
//             spectrum is staged; then y_ti = IFFT(Y_ti).  A single circulant
//             (q == kb == 1) runs both transforms and the product in one row kernel, the
//             spectrum staying in registers (p <= 32768), or takes the product as the
//             inverse loads (p = 65536).
//   backward  G_ti = FFT(g_ti) in place in gy; X_tj = FFT(x_tj) into dx; per bin
//             dC_ij = sum_t conj(X_tj) G_ti (float32 atomics into dc); per bin
//             dX_tj = sum_i conj(C_ij) G_ti into dx; dx_tj = IFFT(dX_tj) in place; the
//             caller's dc rows are then inverted like the fused path's.  With
//             q == kb == 1 the dx product is applied as the inverse loads.
//             When dx is gy (Sec. 5.1.1, overwriting the grad_output; q == kb <= 8)
//             there is nowhere to stage X: its transform hands each bin to the store,
//             which adds conj(X_tj) G_ti into dc_ij for every i (float32 atomics), and
//             dX_tj then replaces G_tj per bin in place in gy.
// The intermediate spectra are stored in the layer's storage type (the in-place
// transform keeps a spectrum in the storage of its input, Sec. 4.1); the arithmetic is
// float32 throughout.
#include <hip/hip_runtime.h>

#include "fft_device.hpp"
#include "launch.hpp"

namespace rdfft {

namespace {

constexpr int kMpMinLogN = 13;  // p = 16384
constexpr int kMpMaxLogN = 15;  // p = 65536
constexpr int kMpMaxKb = kMpMaxInPlaceBlocks;  // blocks a per-bin product thread holds

// elementwise product of pair slot m with the matching slot of a spectrum w (times
// conj(w) when CONJ); slot 0 holds the two real bins Y_0 and Y_{n/2}
template <bool CONJ>
__device__ __forceinline__ float2 slot_mul(int m, float2 a, float2 w) {
  const float2 re = make_float2(a.x * w.x, a.y * w.y);
  return m == 0 ? re : c_mul<CONJ>(a, w);
}

// the pair type a storage struct keeps in memory
template <class St>
using ElemOf = typename St::Elem;

template <int LOGN, class St>
constexpr int mp_chunks() {
  return St::kHalf ? kChunksBf16[LOGN] : kChunks[LOGN];
}

// Load accessor that returns the product of a stored spectrum slot with the matching
// slot of one block spectrum (times its conjugate when CONJ)
template <class GAcc, class CAcc, bool CONJ>
struct MulLoad {
  using raw_t = float2;
  GAcc g;
  CAcc c;
  __device__ __forceinline__ static float2 widen(raw_t r) { return r; }
  __device__ __forceinline__ raw_t load_raw(int m) const { return slot_mul<CONJ>(m, g.load(m), c.load(m)); }
  __device__ __forceinline__ float2 load(int m) const { return load_raw(m); }
};

// Forward transform of rows r < rows of src into dst row (r / gin) * gout + r % gin
// (src == dst with gin == gout is the in-place transform).
template <int LOGN, class St>
__global__ void __launch_bounds__((RowPlan<LOGN, mp_chunks<LOGN, St>()>::WG))
    mp_forward_kernel(const ElemOf<St>* src, ElemOf<St>* dst, int64_t rows, int gin, int gout, const float2* __restrict__ tw) {
  constexpr int CH = mp_chunks<LOGN, St>();
  using P = RowPlan<LOGN, CH>;
  static_assert(P::RW == 1, "one row per workgroup");
  using S = St;
  __shared__ float2 lds[P::LDS_F2];
  const int t = threadIdx.x;
  const int64_t row = blockIdx.x;
  if (row >= rows) return;  // whole workgroup: no barrier is skipped by part of it
  const int64_t out_row = (row / gin) * gout + row % gin;
  const typename S::In in{src + row * (int64_t)P::N};
  const typename S::Out out{dst + out_row * (int64_t)P::N};
  row_forward<LOGN, false, typename S::In, typename S::Out, CH>(t, true, in, out, lds, tw);
}

// Post-pass destinations that consume a spectrum bin by bin instead of storing it.
// YAccumulate: the bins of X_tj (token t, input block j) add C_ij X_tj into Y_ti for
// every output block i, in y's segments (stored in the layer's storage type; `first`
// writes instead of adding).
template <class St>
struct YAccumulate {
  ElemOf<St>* y;             // Y_t0
  const ElemOf<St>* c;       // C_0j
  int q;
  int64_t n_slots, cstride;  // pair slots per row; between C_ij and C_(i+1)j
  bool first;
  __device__ __forceinline__ void store(int m, float2 xv) const {
    for (int i = 0; i < q; ++i) {
      float2 v = slot_mul<false>(m, xv, St::In::widen(c[i * cstride + m]));
      ElemOf<St>* yp = y + i * n_slots + m;
      if (!first) v = c_add(v, St::Out::widen(*yp));
      *yp = St::Out::narrow(v);
    }
  }
};

// DcAccumulate: the bins of X_tj add conj(X_tj) G_ti into dc_ij (float32 atomics) for
// every output block i, G_ti being the upstream spectra in gy.
template <class St>
struct DcAccumulate {
  const ElemOf<St>* g;        // G_t0
  float* dc;                  // dc_0j, float32 pairs
  int q;
  int64_t n_slots, dcstride;  // pair slots per row; between dc_ij and dc_(i+1)j
  __device__ __forceinline__ void store(int m, float2 xv) const {
    for (int i = 0; i < q; ++i) {
      const float2 v = slot_mul<true>(m, St::In::widen(g[i * n_slots + m]), xv);  // G . conj(X)
      float* d = dc + 2 * (i * dcstride + m);
      unsafeAtomicAdd(d, v.x);
      unsafeAtomicAdd(d + 1, v.y);
    }
  }
};

// Forward pass for input block j of every token: row t of the grid transforms x_tj and
// adds C_ij X_tj into y_t's output segments.  One launch per j, in order.
template <int LOGN, class St>
__global__ void __launch_bounds__((RowPlan<LOGN, mp_chunks<LOGN, St>()>::WG))
    mp_fwd_accumulate_kernel(const ElemOf<St>* x, ElemOf<St>* y, const ElemOf<St>* c, int64_t tokens, int q, int kb,
                             int j, const float2* __restrict__ tw) {
  constexpr int CH = mp_chunks<LOGN, St>();
  using P = RowPlan<LOGN, CH>;
  static_assert(P::RW == 1, "one row per workgroup");
  __shared__ float2 lds[P::LDS_F2];
  const int64_t tok = blockIdx.x;
  if (tok >= tokens) return;  // whole workgroup
  constexpr int64_t N = P::N;
  const typename St::In in{x + (tok * kb + j) * N};
  const YAccumulate<St> acc{y + tok * q * N, c + (int64_t)j * N, q, N, (int64_t)kb * N, j == 0};
  row_forward<LOGN, false, typename St::In, YAccumulate<St>, CH>(threadIdx.x, true, in, acc, lds, tw);
}

// dC for the in-place backward: row r = t*kb + j of the grid transforms x_tj and adds
// conj(X_tj) G_ti into dc_ij for every i.
template <int LOGN, class St>
__global__ void __launch_bounds__((RowPlan<LOGN, mp_chunks<LOGN, St>()>::WG))
    mp_dc_accumulate_kernel(const ElemOf<St>* x, const ElemOf<St>* g, float* dc, int64_t rows, int q, int kb,
                            const float2* __restrict__ tw) {
  constexpr int CH = mp_chunks<LOGN, St>();
  using P = RowPlan<LOGN, CH>;
  static_assert(P::RW == 1, "one row per workgroup");
  __shared__ float2 lds[P::LDS_F2];
  const int64_t row = blockIdx.x;
  if (row >= rows) return;  // whole workgroup
  constexpr int64_t N = P::N;
  const int64_t tok = row / kb;
  const int j = (int)(row - tok * kb);
  const typename St::In in{x + row * N};
  const DcAccumulate<St> acc{g + tok * q * N, dc + 2 * (int64_t)j * N, q, N, (int64_t)kb * N};
  row_forward<LOGN, false, typename St::In, DcAccumulate<St>, CH>(threadIdx.x, true, in, acc, lds, tw);
}

// dst row r = IFFT(spec . src row r), or IFFT(conj(spec) . src row r) when CONJ: the
// last step of a single-block layer's forward (in place) and of its dx.  Every load of
// a row precedes its first store, so src may be dst.
template <int LOGN, class St, bool CONJ>
__global__ void __launch_bounds__((RowPlan<LOGN, mp_chunks<LOGN, St>()>::WG))
    mp_inverse_mul_kernel(const ElemOf<St>* src, ElemOf<St>* dst, const ElemOf<St>* spec, int64_t rows, const float2* __restrict__ tw) {
  constexpr int CH = mp_chunks<LOGN, St>();
  using P = RowPlan<LOGN, CH>;
  static_assert(P::RW == 1, "one row per workgroup");
  using S = St;
  __shared__ float2 lds[P::LDS_F2];
  const int t = threadIdx.x;
  const int64_t row = blockIdx.x;
  if (row >= rows) return;
  const MulLoad<typename S::In, typename S::In, CONJ> in{typename S::In{src + row * (int64_t)P::N},
                                                              typename S::In{spec}};
  const typename S::Out out{dst + row * (int64_t)P::N};
  row_inverse<LOGN, false, decltype(in), typename S::Out, CH>(t, true, in, out, lds, tw);
}

// y row r = IFFT(spec . FFT(x row r)) for one block spectrum spec (a single circulant,
// q == kb == 1): the forward post-pass leaves thread t the slots the inverse pre-pass of
// the same thread reads (RegSpectrum), so the row goes from x to y in one pass over HBM.
// Every load of a row precedes its first store, so x may be y.
template <int LOGN, class St>
__global__ void __launch_bounds__((RowPlan<LOGN, mp_chunks<LOGN, St>()>::WG))
    mp_circulant_kernel(const ElemOf<St>* x, ElemOf<St>* y, const ElemOf<St>* spec, int64_t rows, const float2* __restrict__ tw) {
  constexpr int CH = mp_chunks<LOGN, St>();
  using P = RowPlan<LOGN, CH>;
  static_assert(P::RW == 1, "one row per workgroup");
  constexpr int N = P::N, E = P::E, TPR = P::TPR;
  constexpr int R0 = radix(LOGN, 0), BPT0 = E / R0;
  using S = St;
  __shared__ float2 lds[P::LDS_F2];
  const int t = threadIdx.x;
  const int64_t row = blockIdx.x;
  if (row >= rows) return;
  typename S::In::raw_t raw[E];
  load_forward<LOGN>(t, typename S::In{x + row * (int64_t)N}, raw);
  float2 lo[E / 2], hi[E / 2];
  // DST_IN_LDS: a barrier after the post-pass's last LDS read, before the inverse's writes
  row_forward_loaded<LOGN, true, typename S::In, RegSpectrum, CH>(t, true, raw, RegSpectrum{lo, hi}, lds, tw);
  // Y . C on slot k_j = t + j*TPR and its partner; slot 0 (thread 0, j = 0) holds the two
  // real bins Y_0, Y_{n/2}, and its partner is the complex bin N/2
  const typename S::In cin{spec};
  static_for<E / 2>([&](auto jc) {
    constexpr int j = decltype(jc)::value;
    const int k = t + j * TPR;
    if constexpr (j == 0) {
      const bool z = t == 0;
      const float2 c0 = cin.load(k), ch = cin.load(z ? N / 2 : N - k);
      lo[0] = z ? make_float2(lo[0].x * c0.x, lo[0].y * c0.y) : c_mul<false>(lo[0], c0);
      hi[0] = c_mul<false>(hi[0], ch);
    } else {
      lo[j] = c_mul<false>(lo[j], cin.load(k));
      hi[j] = c_mul<false>(hi[j], cin.load(N - k));
    }
  });
  // the inverse reads slot m = t + TPR*(b + BPT0*r) at raw[b*R0 + r], its partner at
  // raw[b*R0 + R0/2 + r]
  float2 inv[E];
  static_for<BPT0>([&](auto bc) {
    constexpr int b = decltype(bc)::value;
    static_for<R0 / 2>([&](auto rc) {
      constexpr int r = decltype(rc)::value;
      inv[b * R0 + r] = lo[b + BPT0 * r];
      inv[b * R0 + R0 / 2 + r] = hi[b + BPT0 * r];
    });
  });
  row_inverse_loaded<LOGN, false, RegSource, typename S::Out, CH>(t, true, inv, typename S::Out{y + row * (int64_t)N},
                                                                  lds, tw);
}

// Per bin, in place in y: Y_ti = sum_j C_ij X_tj, with X_tj in y's segment j (kb <= q).
// One thread owns slot m of one token across all segments, so it reads every X_tj[m]
// before it writes any Y_ti[m].
template <class St>
__global__ void __launch_bounds__(256) mp_fwd_product_kernel(ElemOf<St>* y, const ElemOf<St>* c, int64_t tokens, int q, int kb,
                                                             int nslots, int xblocks) {
  const int64_t b = blockIdx.x;
  const int64_t tok = b / xblocks;
  const int m = (int)(b - tok * xblocks) * 256 + threadIdx.x;
  if (tok >= tokens || m >= nslots) return;
  ElemOf<St>* yt = y + tok * (int64_t)q * nslots;
  float2 xv[kMpMaxKb];
#pragma unroll
  for (int j = 0; j < kMpMaxKb; ++j)
    if (j < kb) xv[j] = St::Out::widen(yt[(int64_t)j * nslots + m]);
  for (int i = 0; i < q; ++i) {
    const ElemOf<St>* ci = c + (int64_t)i * kb * nslots + m;
    float2 acc = make_float2(0.f, 0.f);
#pragma unroll
    for (int j = 0; j < kMpMaxKb; ++j)
      if (j < kb) acc = c_add(acc, slot_mul<false>(m, xv[j], St::Out::widen(ci[(int64_t)j * nslots])));
    yt[(int64_t)i * nslots + m] = St::Out::narrow(acc);
  }
}

// Per bin: dX_tj = sum_i conj(C_ij) G_ti into dx (G in gy).  Thread: slot m of (t, j).
template <class St>
__global__ void __launch_bounds__(256) mp_dx_product_kernel(const ElemOf<St>* g, const ElemOf<St>* c, ElemOf<St>* dx, int64_t tokens,
                                                            int q, int kb, int nslots, int xblocks) {
  const int64_t b = blockIdx.x;
  const int64_t row = b / xblocks;  // t * kb + j
  const int m = (int)(b - row * xblocks) * 256 + threadIdx.x;
  if (row >= tokens * kb || m >= nslots) return;
  const int64_t tok = row / kb;
  const int j = (int)(row - tok * kb);
  const ElemOf<St>* gt = g + tok * (int64_t)q * nslots + m;
  const ElemOf<St>* cj = c + (int64_t)j * nslots + m;
  float2 acc = make_float2(0.f, 0.f);
  for (int i = 0; i < q; ++i)
    acc = c_add(acc, slot_mul<true>(m, St::Out::widen(gt[(int64_t)i * nslots]), St::Out::widen(cj[(int64_t)i * kb * nslots])));
  dx[row * nslots + m] = St::Out::narrow(acc);
}

// In place in gy (dx == gy, q == kb): per bin, dX_tj = sum_i conj(C_ij) G_ti replaces G_tj.
// One thread owns slot m of one token across all segments, so it reads every G_ti[m]
// before it writes any dX_tj[m].
template <class St>
__global__ void __launch_bounds__(256) mp_dx_inplace_kernel(ElemOf<St>* g, const ElemOf<St>* c, int64_t tokens, int q,
                                                            int nslots, int xblocks) {
  const int64_t b = blockIdx.x;
  const int64_t tok = b / xblocks;
  const int m = (int)(b - tok * xblocks) * 256 + threadIdx.x;
  if (tok >= tokens || m >= nslots) return;
  ElemOf<St>* gt = g + tok * (int64_t)q * nslots;
  float2 gv[kMpMaxKb];
#pragma unroll
  for (int i = 0; i < kMpMaxKb; ++i)
    if (i < q) gv[i] = St::Out::widen(gt[(int64_t)i * nslots + m]);
  for (int j = 0; j < q; ++j) {
    float2 acc = make_float2(0.f, 0.f);
#pragma unroll
    for (int i = 0; i < kMpMaxKb; ++i)
      if (i < q) acc = c_add(acc, slot_mul<true>(m, gv[i], St::Out::widen(c[((int64_t)i * q + j) * nslots + m])));
    gt[(int64_t)j * nslots + m] = St::Out::narrow(acc);
  }
}

// dC_ij[m] += sum_{t in chunk} conj(X_tj[m]) G_ti[m]; grid (slot blocks, q*kb, chunks).
template <class St>
__global__ void __launch_bounds__(256) mp_dc_kernel(const ElemOf<St>* xs, const ElemOf<St>* g, float* dc, int64_t tokens, int q,
                                                    int kb, int nslots, int64_t tch) {
  const int m = blockIdx.x * 256 + threadIdx.x;
  if (m >= nslots) return;
  const int pair = blockIdx.y;  // i * kb + j
  const int i = pair / kb, j = pair - (pair / kb) * kb;
  const int64_t t0 = (int64_t)blockIdx.z * tch;
  const int64_t t1 = t0 + tch < tokens ? t0 + tch : tokens;
  const ElemOf<St>* xp = xs + (t0 * kb + j) * (int64_t)nslots + m;
  const ElemOf<St>* gp = g + (t0 * q + i) * (int64_t)nslots + m;
  const int64_t xstep = (int64_t)kb * nslots, gstep = (int64_t)q * nslots;
  float2 acc = make_float2(0.f, 0.f);
#pragma unroll 8
  for (int64_t tok = t0; tok < t1; ++tok, xp += xstep, gp += gstep)
    acc = c_add(acc, slot_mul<true>(m, St::Out::widen(*gp), St::Out::widen(*xp)));
  float* d = dc + 2 * ((int64_t)pair * nslots + m);
  unsafeAtomicAdd(d, acc.x);
  unsafeAtomicAdd(d + 1, acc.y);
}

// workgroups per launch: a dimension of the grid holds fewer than 2^32 work-items
constexpr int64_t kMaxGrid256 = kMaxGridThreads / 256;

template <int LOGN, class St>
hipError_t forward_rows(const void* src, void* dst, int64_t rows, int gin, int gout, const float2* tw,
                        hipStream_t stream) {
  constexpr int N = 1 << LOGN;
  using P = RowPlan<LOGN, mp_chunks<LOGN, St>()>;
  const ElemOf<St>* s = static_cast<const ElemOf<St>*>(src);
  ElemOf<St>* d = static_cast<ElemOf<St>*>(dst);
  for (int64_t r0 = 0; r0 < rows;) {
    const int64_t nr = std::min<int64_t>(rows - r0, kMaxGridThreads / P::WG);
    // chunks start at a multiple of gin so the destination mapping restarts cleanly
    const int64_t step = nr == rows - r0 ? nr : (nr / gin) * gin;
    hipLaunchKernelGGL((mp_forward_kernel<LOGN, St>), dim3((unsigned)step), dim3(P::WG), 0, stream,
                       s + r0 * (int64_t)N, d + (r0 / gin) * gout * (int64_t)N, step, gin, gout, tw);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    r0 += step;
  }
  return hipSuccess;
}

template <int LOGN, class St, bool CONJ>
hipError_t inverse_mul_rows(const void* src, void* dst, const void* spec, int64_t rows, const float2* tw,
                            hipStream_t stream) {
  constexpr int N = 1 << LOGN;
  using P = RowPlan<LOGN, mp_chunks<LOGN, St>()>;
  for (int64_t r0 = 0; r0 < rows;) {
    const int64_t nr = std::min<int64_t>(rows - r0, kMaxGridThreads / P::WG);
    hipLaunchKernelGGL((mp_inverse_mul_kernel<LOGN, St, CONJ>), dim3((unsigned)nr), dim3(P::WG), 0, stream,
                       static_cast<const ElemOf<St>*>(src) + r0 * (int64_t)N, static_cast<ElemOf<St>*>(dst) + r0 * (int64_t)N,
                       static_cast<const ElemOf<St>*>(spec), nr, tw);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    r0 += nr;
  }
  return hipSuccess;
}

// 1-D grid of (unit, block) pairs, `per` blocks per unit, in launches of at most
// kMaxGrid256 blocks
template <class F>
hipError_t per_row_slots(int64_t nrows, int per, F launch) {
  const int64_t rows_per = std::max<int64_t>(1, kMaxGrid256 / per);
  for (int64_t r0 = 0; r0 < nrows; r0 += rows_per) {
    const int64_t nr = std::min<int64_t>(rows_per, nrows - r0);
    launch(r0, nr, (unsigned)(nr * per));
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

template <int LOGN, class St>
hipError_t circulant_rows(const void* x, void* y, const void* spec, int64_t rows, const float2* tw,
                          hipStream_t stream) {
  constexpr int N = 1 << LOGN;
  using P = RowPlan<LOGN, mp_chunks<LOGN, St>()>;
  for (int64_t r0 = 0; r0 < rows;) {
    const int64_t nr = std::min<int64_t>(rows - r0, kMaxGridThreads / P::WG);
    hipLaunchKernelGGL((mp_circulant_kernel<LOGN, St>), dim3((unsigned)nr), dim3(P::WG), 0, stream,
                       static_cast<const ElemOf<St>*>(x) + r0 * (int64_t)N, static_cast<ElemOf<St>*>(y) + r0 * (int64_t)N,
                       static_cast<const ElemOf<St>*>(spec), nr, tw);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    r0 += nr;
  }
  return hipSuccess;
}

template <int LOGN, class St>
hipError_t mp_forward(const BcaArgs& a, const float2* tw, hipStream_t stream, int num_cu) {
  constexpr int N = 1 << LOGN;
  constexpr int storage = St::kId;
  const int64_t xrows = a.tokens * a.kb;
  // single circulant: one fused row pass where the registers hold both spectra (p <= 32768);
  // for p = 65536 the row already fills the registers, so forward, then inverse with the
  // product taken as it loads
  if constexpr (LOGN < kMpMaxLogN) {
    if (a.q == 1 && a.kb == 1) return circulant_rows<LOGN, St>(a.x, a.y, a.c, xrows, tw, stream);
  }
  if (a.kb > a.q || a.kb > kMpMaxKb) {
    // no room to stage the input spectra in y: one accumulating pass per input block
    if (a.x == a.y) return hipErrorInvalidValue;  // in place needs q == kb <= kMpMaxKb
    using P = RowPlan<LOGN, mp_chunks<LOGN, St>()>;
    const int64_t per_launch = kMaxGridThreads / P::WG;
    for (int j = 0; j < a.kb; ++j) {
      for (int64_t t0 = 0; t0 < a.tokens; t0 += per_launch) {
        const int64_t nt = std::min<int64_t>(per_launch, a.tokens - t0);
        hipLaunchKernelGGL((mp_fwd_accumulate_kernel<LOGN, St>), dim3((unsigned)nt), dim3(P::WG), 0, stream,
                           static_cast<const ElemOf<St>*>(a.x) + t0 * a.kb * (int64_t)N,
                           static_cast<ElemOf<St>*>(a.y) + t0 * a.q * (int64_t)N, static_cast<const ElemOf<St>*>(a.c), nt,
                           a.q, a.kb, j, tw);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
      }
    }
    return launch_rdfft_rows(a.y, a.tokens * a.q, LOGN, storage, true, tw, stream, num_cu);
  }
  hipError_t e = forward_rows<LOGN, St>(a.x, a.y, xrows, a.kb, a.q, tw, stream);
  if (e != hipSuccess) return e;
  if (a.q == 1 && a.kb == 1) return inverse_mul_rows<LOGN, St, false>(a.y, a.y, a.c, xrows, tw, stream);
  const int xblocks = (N + 255) / 256;
  ElemOf<St>* y = static_cast<ElemOf<St>*>(a.y);
  e = per_row_slots(a.tokens, xblocks, [&](int64_t r0, int64_t nr, unsigned blocks) {
    hipLaunchKernelGGL(mp_fwd_product_kernel<St>, dim3(blocks), dim3(256), 0, stream, y + r0 * (int64_t)a.q * N,
                       static_cast<const ElemOf<St>*>(a.c), nr, a.q, a.kb, N, xblocks);
  });
  if (e != hipSuccess) return e;
  return launch_rdfft_rows(a.y, a.tokens * a.q, LOGN, storage, true, tw, stream, num_cu);
}

template <int LOGN, class St>
hipError_t mp_backward(const BcaArgs& a, const float2* tw, hipStream_t stream, int num_cu) {
  constexpr int N = 1 << LOGN;
  constexpr int storage = St::kId;
  const int64_t grows = a.tokens * a.q, xrows = a.tokens * a.kb;
  // G = FFT(g) in place
  hipError_t e = launch_rdfft_rows(a.y, grows, LOGN, storage, false, tw, stream, num_cu);
  if (e != hipSuccess) return e;
  const int xblocks = (N + 255) / 256;
  if (a.dx == a.y) {
    // in place (q == kb <= kMpMaxKb): dC from the transforms of x as they complete, then
    // dX per bin over G, then its inverse
    if (a.q != a.kb || a.q > kMpMaxKb) return hipErrorInvalidValue;
    using P = RowPlan<LOGN, mp_chunks<LOGN, St>()>;
    const int64_t per_launch = kMaxGridThreads / P::WG;
    for (int64_t r0 = 0; r0 < xrows;) {
      // launches start at whole tokens
      const int64_t nr = std::min<int64_t>((per_launch / a.kb) * a.kb, xrows - r0);
      const int64_t t0 = r0 / a.kb;
      hipLaunchKernelGGL((mp_dc_accumulate_kernel<LOGN, St>), dim3((unsigned)nr), dim3(P::WG), 0, stream,
                         static_cast<const ElemOf<St>*>(a.x) + r0 * (int64_t)N,
                         static_cast<const ElemOf<St>*>(a.y) + t0 * a.q * (int64_t)N, a.dc, nr, a.q, a.kb, tw);
      e = hipGetLastError();
      if (e != hipSuccess) return e;
      r0 += nr;
    }
    if (a.q == 1) return inverse_mul_rows<LOGN, St, true>(a.y, a.y, a.c, xrows, tw, stream);
    ElemOf<St>* g = static_cast<ElemOf<St>*>(a.y);
    e = per_row_slots(a.tokens, xblocks, [&](int64_t t0, int64_t nt, unsigned blocks) {
      hipLaunchKernelGGL(mp_dx_inplace_kernel<St>, dim3(blocks), dim3(256), 0, stream, g + t0 * a.q * (int64_t)N,
                         static_cast<const ElemOf<St>*>(a.c), nt, a.q, N, xblocks);
    });
    if (e != hipSuccess) return e;
    return launch_rdfft_rows(a.y, xrows, LOGN, storage, true, tw, stream, num_cu);
  }
  // X = FFT(x) into dx
  e = forward_rows<LOGN, St>(a.x, a.dx, xrows, 1, 1, tw, stream);
  if (e != hipSuccess) return e;
  // dC: slot blocks x pairs x token chunks, about 2048 workgroups in all (q * kb <= 65535)
  const int pairs = a.q * a.kb;
  int64_t chunks = std::max<int64_t>(1, 2048 / ((int64_t)xblocks * pairs));
  chunks = std::min<int64_t>(chunks, std::max<int64_t>(1, a.tokens / 16));
  int64_t tch = std::max<int64_t>((a.tokens + chunks - 1) / chunks, (a.tokens + 65534) / 65535);
  chunks = (a.tokens + tch - 1) / tch;
  hipLaunchKernelGGL(mp_dc_kernel<St>, dim3(xblocks, pairs, (unsigned)chunks), dim3(256), 0, stream,
                     static_cast<const ElemOf<St>*>(a.dx), static_cast<const ElemOf<St>*>(a.y), a.dc, a.tokens, a.q, a.kb, N,
                     tch);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (a.q == 1 && a.kb == 1) return inverse_mul_rows<LOGN, St, true>(a.y, a.dx, a.c, xrows, tw, stream);
  // dX into dx, then its inverse in place; launches cover whole tokens
  ElemOf<St>* dx = static_cast<ElemOf<St>*>(a.dx);
  e = per_row_slots(a.tokens, xblocks * a.kb, [&](int64_t t0, int64_t nt, unsigned blocks) {
    hipLaunchKernelGGL(mp_dx_product_kernel<St>, dim3(blocks), dim3(256), 0, stream,
                       static_cast<const ElemOf<St>*>(a.y) + t0 * a.q * (int64_t)N, static_cast<const ElemOf<St>*>(a.c),
                       dx + t0 * a.kb * (int64_t)N, nt, a.q, a.kb, N, xblocks);
  });
  if (e != hipSuccess) return e;
  return launch_rdfft_rows(a.dx, xrows, LOGN, storage, true, tw, stream, num_cu);
}

using MpFn = hipError_t (*)(const BcaArgs&, const float2*, hipStream_t, int);
using SeqMp = std::make_integer_sequence<int, kMpMaxLogN - kMpMinLogN + 1>;
using MpRow = std::array<MpFn, kMpMaxLogN - kMpMinLogN + 1>;

template <class St, int... L>
MpRow mp_row(bool backward, std::integer_sequence<int, L...>) {
  return {(backward ? &mp_backward<L + kMpMinLogN, St> : &mp_forward<L + kMpMinLogN, St>)...};
}

}  // namespace

bool bca_multipass_supported(int logp, int q, int kb, bool) {
  const int logn = logp - 1;
  if (logn < kMpMinLogN || logn > kMpMaxLogN) return false;
  return (int64_t)q * kb <= 65535;  // the dC grid's second dimension
}

hipError_t launch_bca_circulant(const BcaArgs& a, const float2* tw, hipStream_t stream) {
  if (a.logp - 1 != kCirculantLogN || a.q != 1 || a.kb != 1) return hipErrorInvalidValue;
  switch (a.storage) {
    case kStorageF32: return circulant_rows<kCirculantLogN, StoreF32>(a.x, a.y, a.c, a.tokens, tw, stream);
    case kStorageBF16: return circulant_rows<kCirculantLogN, StoreBF16>(a.x, a.y, a.c, a.tokens, tw, stream);
    case kStorageF16: return circulant_rows<kCirculantLogN, StoreF16>(a.x, a.y, a.c, a.tokens, tw, stream);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_bca_multipass(const BcaArgs& a, bool backward, const float2* tw, hipStream_t stream, int num_cu) {
  // [direction][storage]
  static const MpRow tab[2][3] = {
      {mp_row<StoreF32>(false, SeqMp{}), mp_row<StoreBF16>(false, SeqMp{}), mp_row<StoreF16>(false, SeqMp{})},
      {mp_row<StoreF32>(true, SeqMp{}), mp_row<StoreBF16>(true, SeqMp{}), mp_row<StoreF16>(true, SeqMp{})}};
  if (a.storage < 0 || a.storage > 2) return hipErrorInvalidValue;
  return tab[backward ? 1 : 0][a.storage][a.logp - 1 - kMpMinLogN](a, tw, stream, num_cu);
}

}  // namespace rdfft
