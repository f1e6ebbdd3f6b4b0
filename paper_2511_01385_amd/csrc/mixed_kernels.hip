// mixed_kernels.hip -- rdFFT rows whose half-length has factors 3 and 5.
//
// Even n = 2N with N = 2^a 3^b 5^c that is not a power of two, N <= 16384.  The
// transform is the one of the power-of-two kernels (Sec. 4.1): the N-point complex DFT of
// z_m = x_{2m} + i x_{2m+1} followed by the post-pass that pairs bins k and N-k, and the
// inverse pre-pass (1/n folded in) followed by the conjugate passes.  Here one workgroup
// owns one row, keeps all N complex points in LDS, and runs a Stockham pass per radix
// (5, 3, then 8/4/2) with the radix picked at run time; the twiddles come from the
// hardware sine and cosine of the fraction k/M in revolutions, and a butterfly's higher
// powers from products of its first one, so these plans need no table.
#include <hip/hip_runtime.h>

#include "fft_device.hpp"
#include "launch.hpp"

namespace rdfft {

namespace {

constexpr int kMixedMaxPasses = 16;
constexpr int kMixedMaxPerThread = 16;  // complex points per thread (N / blockDim <= 16)

struct MixedPlan {
  int n_half;  // N
  int passes;
  int radix[kMixedMaxPasses];
};

// -i * a (forward) or +i * a (inverse)
template <bool INV>
__device__ __forceinline__ float2 mul_mi(float2 a) {
  return INV ? make_float2(-a.y, a.x) : make_float2(a.y, -a.x);
}

template <int R, bool INV>
struct DftOdd;

// 3 points: y1, y2 = (v0 - (v1+v2)/2) -+ i (sqrt(3)/2) (v1 - v2)
template <bool INV>
struct DftOdd<3, INV> {
  __device__ __forceinline__ static void run(float2* v) {
    constexpr float s3 = 0.866025403784438646763723f;  // sin(2 pi / 3)
    const float2 a = c_add(v[1], v[2]), b = c_scale(c_sub(v[1], v[2]), s3);
    const float2 t = make_float2(fmaf(-0.5f, a.x, v[0].x), fmaf(-0.5f, a.y, v[0].y));
    v[0] = c_add(v[0], a);
    const float2 ib = mul_mi<INV>(b);
    v[1] = c_add(t, ib);
    v[2] = c_sub(t, ib);
  }
};

// 5 points with c1 = cos(2 pi/5), c2 = cos(4 pi/5), s1 = sin(2 pi/5), s2 = sin(4 pi/5):
//   y1, y4 = v0 + c1 (v1+v4) + c2 (v2+v3) -+ i (s1 (v1-v4) + s2 (v2-v3))
//   y2, y3 = v0 + c2 (v1+v4) + c1 (v2+v3) -+ i (s2 (v1-v4) - s1 (v2-v3))
template <bool INV>
struct DftOdd<5, INV> {
  __device__ __forceinline__ static void run(float2* v) {
    constexpr float c1 = 0.309016994374947424102293f, c2 = -0.809016994374947424102293f;
    constexpr float s1 = 0.951056516295153572116439f, s2 = 0.587785252292473129168706f;
    const float2 a1 = c_add(v[1], v[4]), a2 = c_add(v[2], v[3]);
    const float2 b1 = c_sub(v[1], v[4]), b2 = c_sub(v[2], v[3]);
    const float2 v0 = v[0];
    const float2 t1 = make_float2(fmaf(c2, a2.x, fmaf(c1, a1.x, v0.x)), fmaf(c2, a2.y, fmaf(c1, a1.y, v0.y)));
    const float2 t2 = make_float2(fmaf(c1, a2.x, fmaf(c2, a1.x, v0.x)), fmaf(c1, a2.y, fmaf(c2, a1.y, v0.y)));
    const float2 u1 = make_float2(fmaf(s2, b2.x, s1 * b1.x), fmaf(s2, b2.y, s1 * b1.y));
    const float2 u2 = make_float2(fmaf(-s1, b2.x, s2 * b1.x), fmaf(-s1, b2.y, s2 * b1.y));
    v[0] = c_add(v0, c_add(a1, a2));
    const float2 iu1 = mul_mi<INV>(u1), iu2 = mul_mi<INV>(u2);
    v[1] = c_add(t1, iu1);
    v[4] = c_sub(t1, iu1);
    v[2] = c_add(t2, iu2);
    v[3] = c_sub(t2, iu2);
  }
};

template <int R, bool INV>
__device__ __forceinline__ void dft_any(float2* v) {
  if constexpr (R == 3 || R == 5) DftOdd<R, INV>::run(v);
  else Dft<R, INV>::run(v);
}

// exp(-+ 2 pi i num / den) for 0 <= num < den, from the hardware sine and cosine of the
// angle in revolutions, num / den (V_SIN_F32 / V_COS_F32 take their argument in turns, so
// no reduction by pi is needed); the caller passes inv_den = 1/den (one division per pass,
// not per twiddle).  Transform errors stay at 1e-7 .. 6e-7 relative (fp64 reference),
// against 1e-7 .. 3e-7 with sincospif, whose argument reduction costs more instructions.
template <bool INV>
__device__ __forceinline__ float2 unit_root_dev(int num, float inv_den) {
  const float x = (float)num * inv_den;  // revolutions
  const float s = __builtin_amdgcn_sinf(x), c = __builtin_amdgcn_cosf(x);
  return make_float2(c, INV ? s : -s);
}

// One Stockham pass of radix R over the row in LDS: butterfly j < B = N/R reads
// in[j + r*B], multiplies input r by W_{Ns*R}^{r*k} (k = j mod Ns), runs the R-point DFT
// and writes out[(j/Ns)*Ns*R + k + r*Ns].  All reads of the pass precede its writes.  A
// thread's butterflies are T apart, so their k follow from the first one by adding T mod Ns
// (no division per butterfly).  (Padding the row as the power-of-two kernels do made these
// passes slower: their strides are multiples of 3 and 5.)
template <int R, bool INV>
__device__ __forceinline__ void mixed_pass(float2* lds, int N, int Ns) {
  constexpr int MB = (kMixedMaxPerThread + R - 1) / R;  // butterflies per thread, at most
  const int B = N / R, T = blockDim.x, t = threadIdx.x;
  float2 v[MB][R];
#pragma unroll
  for (int s = 0; s < MB; ++s) {
    const int j = t + s * T;
    if (j < B) {
#pragma unroll
      for (int r = 0; r < R; ++r) v[s][r] = lds[j + r * B];
    }
  }
  __syncthreads();
  const float inv_den = 1.0f / (float)(Ns * R);
  const int step = T % Ns;
  int k = t % Ns;  // k of butterfly t + s*T, advanced by step per s
#pragma unroll
  for (int s = 0; s < MB; ++s) {
    const int j = t + s * T;
    if (s > 0) {
      k += step;
      if (k >= Ns) k -= Ns;
    }
    if (j < B) {
      if (Ns > 1) {
        const float2 w1 = unit_root_dev<INV>(k, inv_den);
        float2 w = w1;
#pragma unroll
        for (int r = 1; r < R; ++r) {
          v[s][r] = c_mul<false>(v[s][r], w);
          if (r + 1 < R) w = c_mul<false>(w, w1);
        }
      }
      dft_any<R, INV>(v[s]);
      const int o = (j - k) * R + k;
#pragma unroll
      for (int r = 0; r < R; ++r) lds[o + r * Ns] = v[s][r];
    }
  }
  __syncthreads();
}

template <bool INV>
__device__ __forceinline__ void mixed_passes(float2* lds, const MixedPlan& plan) {
  int Ns = 1;
  for (int q = 0; q < plan.passes; ++q) {
    const int R = plan.radix[q];
    switch (R) {
      case 2: mixed_pass<2, INV>(lds, plan.n_half, Ns); break;
      case 3: mixed_pass<3, INV>(lds, plan.n_half, Ns); break;
      case 4: mixed_pass<4, INV>(lds, plan.n_half, Ns); break;
      case 5: mixed_pass<5, INV>(lds, plan.n_half, Ns); break;
      default: mixed_pass<8, INV>(lds, plan.n_half, Ns); break;
    }
    Ns *= R;
  }
}

// HC: the spectrum (the forward's output, the inverse's input) in the halfcomplex layout.
template <class Acc, class Elem, bool INV, bool HC>
__global__ void __launch_bounds__(1024) mixed_rows_kernel(Elem* buf, MixedPlan plan) {
  extern __shared__ float2 mixed_lds[];
  const int N = plan.n_half, T = blockDim.x, t = threadIdx.x;
  Elem* const rp = buf + (int64_t)blockIdx.x * N;
  const Acc sig{rp};                                   // the signal pairs (x_{2m}, x_{2m+1})
  const auto spec = spectrum_view<HC, Acc>(rp, N);  // the packed spectrum
  if constexpr (!INV) {
    for (int m = t; m < N; m += T) mixed_lds[m] = sig.load(m);
  } else {
    // pre-pass: Z~_m = (s + i conj(W_n^m) d) / n, Z~_{N-m} = conj(s - i conj(W_n^m) d) / n with
    // s = Y_m + conj(Y_{N-m}), d = Y_m - conj(Y_{N-m}); slot 0 holds (Y_0, Y_{n/2})
    const float sc = 1.0f / (2.0f * N), inv_n = 1.0f / (float)(2 * N);
    for (int m = t; 2 * m <= N; m += T) {
      const float2 ya = spec.load(m);
      if (m == 0) {
        mixed_lds[0] = make_float2(sc * (ya.x + ya.y), sc * (ya.x - ya.y));
        continue;
      }
      const float2 yb = c_conj(spec.load(N - m));
      const float2 s = c_add(ya, yb), d = c_sub(ya, yb);
      const float2 w = unit_root_dev<true>(m, inv_n);         // conj(W_n^m)
      const float2 q = c_mul<false>(d, make_float2(-sc * w.y, sc * w.x));  // i conj(W_n^m) d / n
      mixed_lds[m] = make_float2(fmaf(s.x, sc, q.x), fmaf(s.y, sc, q.y));
      if (2 * m != N) mixed_lds[N - m] = make_float2(fmaf(s.x, sc, -q.x), -fmaf(s.y, sc, -q.y));
    }
  }
  __syncthreads();
  mixed_passes<INV>(mixed_lds, plan);
  if constexpr (!INV) {
    // post-pass: Y_k = s/2 + (-i W_n^k / 2) d, Y_{N-k} = conj(s/2 - (-i W_n^k / 2) d) with
    // s = Z_k + conj(Z_{N-k}), d = Z_k - conj(Z_{N-k}); slot 0 = (Y_0, Y_{n/2})
    const float inv_n = 1.0f / (float)(2 * N);
    for (int k = t; 2 * k <= N; k += T) {
      const float2 a = mixed_lds[k];
      if (k == 0) {
        spec.store(0, make_float2(a.x + a.y, a.x - a.y));
        continue;
      }
      const float2 b = c_conj(mixed_lds[N - k]);
      const float2 s = c_add(a, b), d = c_sub(a, b);
      const float2 w = unit_root_dev<false>(k, inv_n);  // W_n^k
      const float2 q = c_mul<false>(d, make_float2(0.5f * w.y, -0.5f * w.x));  // -i W_n^k d / 2
      spec.store(k, make_float2(fmaf(s.x, 0.5f, q.x), fmaf(s.y, 0.5f, q.y)));
      if (2 * k != N) spec.store(N - k, make_float2(fmaf(s.x, 0.5f, -q.x), -fmaf(s.y, 0.5f, -q.y)));
    }
  } else {
    for (int m = t; m < N; m += T) sig.store(m, mixed_lds[m]);
  }
}

template <class K>
hipError_t allow_lds(K kernel) {
  return hipFuncSetAttribute(reinterpret_cast<const void*>(kernel), hipFuncAttributeMaxDynamicSharedMemorySize,
                             160 * 1024);
}

template <class Acc, class Elem, bool INV, bool HC>
hipError_t launch_mixed(void* buf, int64_t rows, const MixedPlan& plan, int threads, hipStream_t stream) {
  static const hipError_t attr = allow_lds(mixed_rows_kernel<Acc, Elem, INV, HC>);
  if (attr != hipSuccess) return attr;
  const size_t lds = (size_t)plan.n_half * sizeof(float2);
  Elem* base = static_cast<Elem*>(buf);
  const int64_t max_rows = kMaxGridThreads / threads;
  for (int64_t r0 = 0; r0 < rows; r0 += max_rows) {
    const int64_t nr = std::min<int64_t>(max_rows, rows - r0);
    hipLaunchKernelGGL((mixed_rows_kernel<Acc, Elem, INV, HC>), dim3((unsigned)nr), dim3(threads), lds, stream,
                       base + r0 * plan.n_half, plan);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

// Radices of N = 2^a 3^b 5^c: fives, threes, then eights and one four or two
bool make_plan(int64_t n_half, MixedPlan* plan) {
  if (n_half < 1 || n_half > kMixedMaxHalf || (n_half & (n_half - 1)) == 0) return false;
  int64_t m = n_half;
  int q = 0;
  auto push = [&](int r) {
    if (q >= kMixedMaxPasses) return false;
    plan->radix[q++] = r;
    m /= r;
    return true;
  };
  while (m % 5 == 0)
    if (!push(5)) return false;
  while (m % 3 == 0)
    if (!push(3)) return false;
  while (m % 8 == 0)
    if (!push(8)) return false;
  if (m == 4 && !push(4)) return false;
  if (m == 2 && !push(2)) return false;
  if (m != 1) return false;
  plan->n_half = (int)n_half;
  plan->passes = q;
  return true;
}

// In-place pairs <-> halfcomplex conversion of one row per workgroup (the permutation of
// the power-of-two converters), staged through LDS so that every slot is read before any
// is written.  Pair slot k maps to the real slots (k, n-k), and slot 0 to (0, N).
template <class Pair, class Scalar, bool TO_HC>
__global__ void __launch_bounds__(1024) mixed_layout_kernel(Scalar* buf, int n_half) {
  extern __shared__ float2 mixed_lds[];
  Pair* lds = reinterpret_cast<Pair*>(mixed_lds);
  const int N = n_half, T = blockDim.x, t = threadIdx.x;
  Scalar* const s = buf + (int64_t)blockIdx.x * (2 * N);
  Pair* const p = reinterpret_cast<Pair*>(s);
  for (int k = t; k < N; k += T) {
    if constexpr (TO_HC) {
      lds[k] = p[k];
    } else {
      Pair v;
      v.x = s[k];
      v.y = s[k == 0 ? N : 2 * N - k];
      lds[k] = v;
    }
  }
  __syncthreads();
  for (int k = t; k < N; k += T) {
    const Pair v = lds[k];
    if constexpr (TO_HC) {
      s[k] = v.x;
      s[k == 0 ? N : 2 * N - k] = v.y;
    } else {
      p[k] = v;
    }
  }
}

struct alignas(4) Half2 {
  uint16_t x, y;
};

template <class Pair, class Scalar, bool TO_HC>
hipError_t launch_mixed_layout_t(void* buf, int64_t rows, int n_half, int threads, hipStream_t stream) {
  static const hipError_t attr = allow_lds(mixed_layout_kernel<Pair, Scalar, TO_HC>);
  if (attr != hipSuccess) return attr;
  const size_t lds = (size_t)n_half * sizeof(Pair);
  Scalar* base = static_cast<Scalar*>(buf);
  const int64_t max_rows = kMaxGridThreads / threads;
  for (int64_t r0 = 0; r0 < rows; r0 += max_rows) {
    const int64_t nr = std::min<int64_t>(max_rows, rows - r0);
    hipLaunchKernelGGL((mixed_layout_kernel<Pair, Scalar, TO_HC>), dim3((unsigned)nr), dim3(threads), lds, stream,
                       base + r0 * 2 * n_half, n_half);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

int threads_for(int64_t n_half) {
  // n_half / threads <= kMixedMaxPerThread bounds every pass's butterflies per thread
  return (int)std::min<int64_t>(1024, std::max<int64_t>(64, ((n_half + 16 * 64 - 1) / (16 * 64)) * 64));
}

}  // namespace

bool mixed_length_supported(int64_t n) {
  MixedPlan p;
  return n % 2 == 0 && make_plan(n / 2, &p);
}

hipError_t launch_mixed_rows(void* buf, int64_t rows, int64_t n, int storage, bool inv, bool halfcomplex,
                             hipStream_t stream) {
  MixedPlan plan;
  if (!make_plan(n / 2, &plan)) return hipErrorInvalidValue;
  const int threads = threads_for(n / 2);
  using Fn = hipError_t (*)(void*, int64_t, const MixedPlan&, int, hipStream_t);
  static const Fn table[2][3][2] = {
      {{&launch_mixed<GlobalF32, float2, false, false>, &launch_mixed<GlobalF32, float2, true, false>},
       {&launch_mixed<GlobalBF16, uint32_t, false, false>, &launch_mixed<GlobalBF16, uint32_t, true, false>},
       {&launch_mixed<GlobalF16, uint32_t, false, false>, &launch_mixed<GlobalF16, uint32_t, true, false>}},
      {{&launch_mixed<GlobalF32, float2, false, true>, &launch_mixed<GlobalF32, float2, true, true>},
       {&launch_mixed<GlobalBF16, uint32_t, false, true>, &launch_mixed<GlobalBF16, uint32_t, true, true>},
       {&launch_mixed<GlobalF16, uint32_t, false, true>, &launch_mixed<GlobalF16, uint32_t, true, true>}}};
  return table[halfcomplex ? 1 : 0][storage][inv ? 1 : 0](buf, rows, plan, threads, stream);
}

}  // namespace rdfft

namespace rdfft {

hipError_t launch_mixed_layout(void* buf, int64_t rows, int64_t n, bool half16, bool to_halfcomplex,
                               hipStream_t stream) {
  MixedPlan plan;
  if (!make_plan(n / 2, &plan)) return hipErrorInvalidValue;
  using Fn = hipError_t (*)(void*, int64_t, int, int, hipStream_t);
  static const Fn table[2][2] = {
      {&launch_mixed_layout_t<float2, float, false>, &launch_mixed_layout_t<float2, float, true>},
      {&launch_mixed_layout_t<Half2, uint16_t, false>, &launch_mixed_layout_t<Half2, uint16_t, true>}};
  return table[half16 ? 1 : 0][to_halfcomplex ? 1 : 0](buf, rows, (int)(n / 2), threads_for(n / 2), stream);
}

}  // namespace rdfft
