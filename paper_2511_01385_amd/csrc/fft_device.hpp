// fft_device.hpp -- device building blocks of the row transforms (gfx950, wave64).
//
// One row of n = 2N reals is transformed by TPR cooperating threads that each hold
// E complex values in registers.  The N-point complex DFT of z_m = x_{2m} + i x_{2m+1}
// runs as a Stockham sequence of radix-R passes (plan.hpp): every pass is a set of
// register-resident radix-R DFTs preceded by twiddle multiplies; consecutive passes
// exchange data through the row's LDS region.  The real-signal spectrum then follows
// from a post-pass that pairs bins k and N-k (Sec. 4.1: the output of a real FFT is
// conjugate-symmetric, so the n/2+1 bins Y_0..Y_{n/2} are squeezed into n reals).
//
// Packed ("pairs") layout of the result, as complex pair slots P[0..N-1]:
//   P[0] = (Y_0, Y_{n/2}),  P[k] = Y_k for 1 <= k < N.
//
// The inverse runs the pre-pass (the algebraic inverse of the post-pass, with the
// 1/n scale folded in) and the same passes with conjugated twiddles.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>
#include <utility>

#include "plan.hpp"

namespace rdfft {

// ----------------------------------------------------------------------------------
// compile-time loops
template <class F, int... Is>
__device__ __forceinline__ void static_for_impl(F&& f, std::integer_sequence<int, Is...>) {
  (f(std::integral_constant<int, Is>{}), ...);
}
template <int N, class F>
__device__ __forceinline__ void static_for(F&& f) {
  static_for_impl(f, std::make_integer_sequence<int, N>{});
}

// ----------------------------------------------------------------------------------
// complex arithmetic on float2
__device__ __forceinline__ float2 c_add(float2 a, float2 b) { return make_float2(a.x + b.x, a.y + b.y); }
__device__ __forceinline__ float2 c_sub(float2 a, float2 b) { return make_float2(a.x - b.x, a.y - b.y); }
__device__ __forceinline__ float2 c_conj(float2 a) { return make_float2(a.x, -a.y); }
__device__ __forceinline__ float2 c_scale(float2 a, float s) { return make_float2(a.x * s, a.y * s); }

// a * w, or a * conj(w) when CONJ
template <bool CONJ>
__device__ __forceinline__ float2 c_mul(float2 a, float2 w) {
  if constexpr (!CONJ) return make_float2(fmaf(a.x, w.x, -a.y * w.y), fmaf(a.x, w.y, a.y * w.x));
  else return make_float2(fmaf(a.x, w.x, a.y * w.y), fmaf(a.y, w.x, -a.x * w.y));
}

// cos(2 pi m / 64), m in [0, 16]; the rest follows by symmetry
constexpr double kCos64[17] = {1.0,
                               0.99518472667219688624483695310948,
                               0.98078528040323044912618223613424,
                               0.95694033573220886493579788698027,
                               0.92387953251128675612818318939679,
                               0.88192126434835502971275686366039,
                               0.83146961230254523707878837761791,
                               0.77301045336273696081090660975847,
                               0.70710678118654752440084436210485,
                               0.63439328416364549821517161322549,
                               0.55557023301960222474283081394853,
                               0.47139673682599764855638762590867,
                               0.38268343236508977172845998403040,
                               0.29028467725446236763619237581740,
                               0.19509032201612826784828486847702,
                               0.09801714032956060199419556388864,
                               0.0};
constexpr double cos64(int m) {
  m &= 63;
  return m <= 16 ? kCos64[m] : m <= 32 ? -kCos64[32 - m] : m <= 48 ? -kCos64[m - 32] : kCos64[64 - m];
}
constexpr double sin64(int m) { return cos64(m - 16); }

// a * exp(-+ 2 pi i J / R): forward sign unless INV.  R divides 64.
template <int R, int J, bool INV>
__device__ __forceinline__ float2 rot(float2 a) {
  constexpr int j = ((J % R) + R) % R;
  if constexpr (j == 0) {
    return a;
  } else if constexpr (2 * j == R) {
    return make_float2(-a.x, -a.y);
  } else if constexpr (4 * j == R) {
    return INV ? make_float2(-a.y, a.x) : make_float2(a.y, -a.x);
  } else if constexpr (4 * j == 3 * R) {
    return INV ? make_float2(a.y, -a.x) : make_float2(-a.y, a.x);
  } else {
    static_assert(64 % R == 0, "constant rotations need R | 64");
    constexpr float c = (float)cos64(j * (64 / R));
    constexpr float s = (float)sin64(j * (64 / R));
    if constexpr (!INV) return make_float2(fmaf(a.x, c, a.y * s), fmaf(a.y, c, -a.x * s));
    else return make_float2(fmaf(a.x, c, -a.y * s), fmaf(a.y, c, a.x * s));
  }
}

// ----------------------------------------------------------------------------------
// In-register DFT of R points, natural order in and out:
//   v[k] <- sum_j v[j] exp(-+ 2 pi i j k / R)
template <int R, bool INV>
struct Dft;

template <bool INV>
struct Dft<1, INV> {
  __device__ __forceinline__ static void run(float2*) {}
};

template <bool INV>
struct Dft<2, INV> {
  __device__ __forceinline__ static void run(float2* v) {
    const float2 a = v[0], b = v[1];
    v[0] = c_add(a, b);
    v[1] = c_sub(a, b);
  }
};

template <bool INV>
struct Dft<4, INV> {
  __device__ __forceinline__ static void run(float2* v) {
    const float2 a0 = c_add(v[0], v[2]), a1 = c_sub(v[0], v[2]);
    const float2 a2 = c_add(v[1], v[3]), a3 = rot<4, 1, INV>(c_sub(v[1], v[3]));
    v[0] = c_add(a0, a2);
    v[2] = c_sub(a0, a2);
    v[1] = c_add(a1, a3);
    v[3] = c_sub(a1, a3);
  }
};

// a <- a + W b and b <- a - W b for the constant W = W_M^J (exp(-2 pi i J / M), its
// conjugate when INV).  W is written as (-i)^q cos(phi) (1 - i tan(phi)) with |phi| <= pi/4:
// the factor (1 - i tan(phi)) costs two FMAs, (-i)^q only swaps and negates, and cos(phi)
// rides in the FMAs of the sum and difference, so a butterfly costs six instructions
// (four when phi = 0) instead of a complex multiply plus an add and a subtract.
template <int M, int J, bool INV>
__device__ __forceinline__ void bfly2(float2& a, float2& b) {
  static_assert(64 % M == 0, "constant rotations need M | 64");
  constexpr int j = ((J % M) + M) % M * (64 / M);  // the angle in units of 2 pi / 64
  constexpr int q = ((j + 8) / 16) % 4;              // nearest quarter turn
  constexpr int phi = j - 16 * ((j + 8) / 16);       // the rest, in [-8, 8)
  float2 e = b;
  if constexpr (phi != 0) {
    constexpr float t = (float)(sin64(phi) / cos64(phi));
    // (1 -+ i t) b
    e = INV ? make_float2(fmaf(-t, b.y, b.x), fmaf(t, b.x, b.y)) : make_float2(fmaf(t, b.y, b.x), fmaf(-t, b.x, b.y));
  }
  // (-i)^q e, or i^q e for the inverse
  constexpr int qq = INV ? (4 - q) % 4 : q;
  if constexpr (qq == 1) e = make_float2(e.y, -e.x);
  else if constexpr (qq == 2) e = make_float2(-e.x, -e.y);
  else if constexpr (qq == 3) e = make_float2(-e.y, e.x);
  if constexpr (phi == 0) {
    const float2 s = c_add(a, e), d = c_sub(a, e);
    a = s;
    b = d;
  } else {
    constexpr float c = (float)cos64(phi);
    const float2 s = make_float2(fmaf(c, e.x, a.x), fmaf(c, e.y, a.y));
    const float2 d = make_float2(fmaf(-c, e.x, a.x), fmaf(-c, e.y, a.y));
    a = s;
    b = d;
  }
}

// DFT of R points of the inputs W_M^{nJ} x[n] (conjugate rotations when INV), natural order
// in and out, by radix-2 decimation in time: the even and odd halves are DFTs of the same
// form with 2J, and output k pairs with k + R/2 through the constant W_R^k W_M^J = W_M^{J + kM/R}.
template <int R, int M, int J, bool INV>
struct TwDft {
  __device__ __forceinline__ static void run(float2* x) {
    float2 e[R / 2], o[R / 2];
    static_for<R / 2>([&](auto mc) {
      constexpr int m = decltype(mc)::value;
      e[m] = x[2 * m];
      o[m] = x[2 * m + 1];
    });
    TwDft<R / 2, M, 2 * J, INV>::run(e);
    TwDft<R / 2, M, 2 * J, INV>::run(o);
    static_for<R / 2>([&](auto kc) {
      constexpr int k = decltype(kc)::value;
      bfly2<M, J + k * (M / R), INV>(e[k], o[k]);
      x[k] = e[k];
      x[k + R / 2] = o[k];
    });
  }
};
template <int M, int J, bool INV>
struct TwDft<1, M, J, INV> {
  __device__ __forceinline__ static void run(float2*) {}
};

template <bool INV>
struct Dft<8, INV> : TwDft<8, 8, 0, INV> {};
template <bool INV>
struct Dft<16, INV> : TwDft<16, 16, 0, INV> {};
// R = 32 as 8 DFTs of 4 points over stride-8 inputs, then 4 rotated DFTs of 8 points
// (n = 8 n1 + n2, k = k1 + 4 k2): the same instruction count as the radix-2 recursion,
// with shorter live ranges at a thread's 128-register limit.
template <bool INV>
struct Dft<32, INV> {
  __device__ __forceinline__ static void run(float2* v) {
    float2 u[8][4];
    static_for<8>([&](auto n2c) {
      constexpr int n2 = decltype(n2c)::value;
      static_for<4>([&](auto n1c) { u[n2][decltype(n1c)::value] = v[8 * decltype(n1c)::value + n2]; });
      Dft<4, INV>::run(u[n2]);
    });
    static_for<4>([&](auto k1c) {
      constexpr int k1 = decltype(k1c)::value;
      float2 w[8];
      static_for<8>([&](auto n2c) { w[decltype(n2c)::value] = u[decltype(n2c)::value][k1]; });
      TwDft<8, 32, k1, INV>::run(w);
      static_for<8>([&](auto k2c) { v[k1 + 4 * decltype(k2c)::value] = w[decltype(k2c)::value]; });
    });
  }
};

// ----------------------------------------------------------------------------------
// Row storage accessors (complex-pair indexed).  load_raw fetches a slot in its storage
// form and widen turns that into float2, so a caller can issue a row's loads early and
// widen them when it computes; load(m) == widen(load_raw(m)).
struct GlobalF32 {
  using raw_t = float2;
  float2* base;
  __device__ __forceinline__ static float2 widen(raw_t r) { return r; }
  __device__ __forceinline__ static raw_t narrow(float2 v) { return v; }
  __device__ __forceinline__ raw_t load_raw(int m) const { return base[m]; }
  __device__ __forceinline__ float2 load(int m) const { return base[m]; }
  __device__ __forceinline__ void store(int m, float2 v) const { base[m] = v; }
};

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));

__device__ __forceinline__ float2 bf16x2_to_f32(uint32_t u) {
  return make_float2(__uint_as_float(u << 16), __uint_as_float(u & 0xffff0000u));
}
__device__ __forceinline__ uint32_t f32_to_bf16x2(float2 v) {  // round to nearest even
  const f32x2_t f = {v.x, v.y};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f, bf16x2_t));
}

struct GlobalBF16 {
  using raw_t = uint32_t;
  uint32_t* base;
  __device__ __forceinline__ static float2 widen(raw_t r) { return bf16x2_to_f32(r); }
  __device__ __forceinline__ static raw_t narrow(float2 v) { return f32_to_bf16x2(v); }
  __device__ __forceinline__ raw_t load_raw(int m) const { return base[m]; }
  __device__ __forceinline__ float2 load(int m) const { return bf16x2_to_f32(base[m]); }
  __device__ __forceinline__ void store(int m, float2 v) const { base[m] = f32_to_bf16x2(v); }
};

typedef _Float16 f16x2_t __attribute__((ext_vector_type(2)));

__device__ __forceinline__ float2 f16x2_to_f32(uint32_t u) {
  const f32x2_t f = __builtin_convertvector(__builtin_bit_cast(f16x2_t, u), f32x2_t);
  return make_float2(f.x, f.y);
}
__device__ __forceinline__ uint32_t f32_to_f16x2(float2 v) {  // round to nearest even
  const f32x2_t f = {v.x, v.y};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f, f16x2_t));
}

struct GlobalF16 {
  using raw_t = uint32_t;
  uint32_t* base;
  __device__ __forceinline__ static float2 widen(raw_t r) { return f16x2_to_f32(r); }
  __device__ __forceinline__ static raw_t narrow(float2 v) { return f32_to_f16x2(v); }
  __device__ __forceinline__ raw_t load_raw(int m) const { return base[m]; }
  __device__ __forceinline__ float2 load(int m) const { return f16x2_to_f32(base[m]); }
  __device__ __forceinline__ void store(int m, float2 v) const { base[m] = f32_to_f16x2(v); }
};

// Read-only views (inputs that must never be written)
struct ConstF32 {
  using raw_t = float2;
  const float2* base;
  __device__ __forceinline__ static float2 widen(raw_t r) { return r; }
  __device__ __forceinline__ raw_t load_raw(int m) const { return base[m]; }
  __device__ __forceinline__ float2 load(int m) const { return base[m]; }
};
struct ConstBF16 {
  using raw_t = uint32_t;
  const uint32_t* base;
  __device__ __forceinline__ static float2 widen(raw_t r) { return bf16x2_to_f32(r); }
  __device__ __forceinline__ raw_t load_raw(int m) const { return base[m]; }
  __device__ __forceinline__ float2 load(int m) const { return bf16x2_to_f32(base[m]); }
};
struct ConstF16 {
  using raw_t = uint32_t;
  const uint32_t* base;
  __device__ __forceinline__ static float2 widen(raw_t r) { return f16x2_to_f32(r); }
  __device__ __forceinline__ raw_t load_raw(int m) const { return base[m]; }
  __device__ __forceinline__ float2 load(int m) const { return f16x2_to_f32(base[m]); }
};

// The accessor moved by g slots, for the accessors that are plain pointers: a butterfly's
// loads and stores then take one address each and compile-time offsets that the memory
// instructions carry as immediates.  Other accessors (LDS, halfcomplex) index as before.
template <class A>
struct PlainPointer : std::false_type {};
template <> struct PlainPointer<GlobalF32> : std::true_type {};
template <> struct PlainPointer<GlobalBF16> : std::true_type {};
template <> struct PlainPointer<GlobalF16> : std::true_type {};
template <> struct PlainPointer<ConstF32> : std::true_type {};
template <> struct PlainPointer<ConstBF16> : std::true_type {};
template <> struct PlainPointer<ConstF16> : std::true_type {};
// ... used by plans with at most 16 values per thread: the 32-value plan (n = 65536) is at its
// register limit and spills with the extra live addresses
template <class A, int LOGN>
constexpr bool shifted_access() { return PlainPointer<A>::value && kElems[LOGN] <= 16; }

// A row's packed spectrum in the halfcomplex layout (Sec. 4.1, Memory Layout): Re Y_k at
// real slot k (0 <= k <= N) and Im Y_k at real slot 2N - k (1 <= k < N).  Pair slot m of the
// pairs layout is thus the two real slots (m, 2N - m), and pair slot 0 = (Y_0, Y_{n/2}) the
// slots (0, N).  G is the row's pairs accessor (GlobalF32, GlobalBF16 or GlobalF16), which
// gives a pair's storage form; every pair is read and written as two scalars.
template <class G>
struct Halfcomplex {
  using raw_t = typename G::raw_t;
  static constexpr bool kF32 = std::is_same<raw_t, float2>::value;
  using scalar_t = typename std::conditional<kF32, float, uint16_t>::type;
  scalar_t* base;  // real slot 0 of the row
  int N;           // pair slots per row (n / 2)
  __device__ __forceinline__ int partner(int m) const { return m == 0 ? N : 2 * N - m; }
  __device__ __forceinline__ static float2 widen(raw_t r) { return G::widen(r); }
  __device__ __forceinline__ raw_t load_raw(int m) const {
    const scalar_t a = base[m], b = base[partner(m)];
    if constexpr (kF32) {
      return make_float2(a, b);
    } else {
      return (uint32_t)a | ((uint32_t)b << 16);
    }
  }
  __device__ __forceinline__ float2 load(int m) const { return widen(load_raw(m)); }
  __device__ __forceinline__ void store(int m, float2 v) const {
    const raw_t r = G::narrow(v);
    if constexpr (kF32) {
      base[m] = r.x;
      base[partner(m)] = r.y;
    } else {
      base[m] = (uint16_t)(r & 0xffffu);
      base[partner(m)] = (uint16_t)(r >> 16);
    }
  }
};

// The spectrum side of a row at p (n = 2N reals): halfcomplex (HC) or pairs.
template <bool HC, class G, class Elem>
__device__ __forceinline__ auto spectrum_view(Elem* p, int N) {
  if constexpr (HC) {
    return Halfcomplex<G>{reinterpret_cast<typename Halfcomplex<G>::scalar_t*>(p), N};
  } else {
    return G{p};
  }
}

// Storage types of the layer kernels: the pair type in memory (Elem), its read-only and
// read-write row accessors, and the value of rdfft_dtype_t it stands for.  bf16 and f16
// share the 32-bit pair type, so the layer kernels are instantiated per storage struct.
struct StoreF32 {
  using Elem = float2;
  using In = ConstF32;
  using Out = GlobalF32;
  static constexpr int kId = 0;
  static constexpr bool kHalf = false;
};
struct StoreBF16 {
  using Elem = uint32_t;
  using In = ConstBF16;
  using Out = GlobalBF16;
  static constexpr int kId = 1;
  static constexpr bool kHalf = true;
};
struct StoreF16 {
  using Elem = uint32_t;
  using In = ConstF16;
  using Out = GlobalF16;
  static constexpr int kId = 2;
  static constexpr bool kHalf = true;
};


// A packed spectrum kept in a row's (padded) LDS region
struct LdsSpectrum {
  using raw_t = float2;
  float2* base;
  __device__ __forceinline__ static float2 widen(raw_t r) { return r; }
  __device__ __forceinline__ raw_t load_raw(int m) const { return base[lds_pad(m)]; }
  __device__ __forceinline__ float2 load(int m) const { return base[lds_pad(m)]; }
  __device__ __forceinline__ void store(int m, float2 v) const { base[lds_pad(m)] = v; }
};

// A packed spectrum kept in the caller's registers.  The forward post-pass of thread t
// produces the pair slots k_j = t + j*TPR, j < E/2, and their partners N - k_j (N/2 for
// k_j == 0); these are exactly the slots the inverse pre-pass of the same thread reads
// (load_inverse), so a row can pass from one transform to the other without an exchange.
struct RegSpectrum {
  float2* lo;  // [E/2]: slot k_j
  float2* hi;  // [E/2]: slot N - k_j, or N/2 for k_j == 0
};
// Its counterpart as a source: raw values already in float32
struct RegSource {
  using raw_t = float2;
  __device__ __forceinline__ static float2 widen(raw_t r) { return r; }
};

// lds_pad(base + j*stride) == lds_pad(base) + pad_step(j*stride) whenever the low four
// bits of base plus those of j*stride stay below 16.  Every Stockham exchange address has
// that form (base's low bits are below the sub-transform stride, or the stride is a
// multiple of 16), so one padded base per butterfly plus compile-time offsets suffices.
constexpr int pad_step(int d) { return d + (d >> 4); }

// Synchronises the TPR threads that share one row's LDS region.  When the row lives
// inside one wavefront (TPR divides 64) no workgroup barrier is needed: all LDS
// operations of a CU are performed wavefront-wide in one global order, so a wave's
// later LDS reads observe its earlier LDS writes, and only compiler code motion has to
// be stopped.  Rows spanning several waves use the workgroup barrier.
template <int TPR>
__device__ __forceinline__ void row_sync() {
  if constexpr (TPR <= 64) {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  } else {
    __syncthreads();
  }
}

// ----------------------------------------------------------------------------------
template <int LOGN, int CH = kChunks[LOGN]>
struct RowPlan {
  static constexpr int N = 1 << LOGN;
  static constexpr int NP = num_passes(LOGN);
  static constexpr int E = kElems[LOGN];
  static constexpr int C = CH;
  static constexpr int TPR = N / E;                       // threads per row
  static constexpr int RW = TPR >= 256 ? 1 : 256 / TPR;   // rows per 256-thread workgroup
  static constexpr int WG = TPR * RW;
  // LDS float2 per row: one exchange chunk, or the half-spectrum partner exchange, at a
  // stride that keeps the rows of one wavefront on different banks
  static constexpr int LDS_F2_STD = TPR == 1 ? 0 : lds_row_stride(N / C > N / 2 ? N / C : N / 2, TPR);
  static constexpr int LDS_F2_WIDE = plan_has_wide_exchange(LOGN, CH) ? lds_pad_wide(N - 1) + 1 : 0;
  static constexpr int LDS_F2 = LDS_F2_STD > LDS_F2_WIDE ? LDS_F2_STD : LDS_F2_WIDE;
  static_assert(plan_is_consistent(LOGN), "inconsistent plan");
  static_assert(exchange_split_ok(LOGN, CH), "an exchange's split LDS addresses differ from the padded index");

};

// Mirrored last pass.  When the last pass gives each thread two butterflies and the row
// has exactly half as many threads as that pass has butterflies (TPR = N/(2 RL)), thread t
// can take butterflies t and N/RL - t (thread 0: 0 and N/(2 RL)).  Bin k = g + r N/RL of
// butterfly g and its post-pass partner N - k then sit in the same thread, and the forward
// post-pass needs no LDS exchange.  Only the standalone row kernels use it: the layer
// kernels read the spectrum in the plain order.  It costs ~2% more VALU instructions (the
// selects for thread 0) for one LDS round trip and one barrier fewer: timed, that pays for
// n >= 2048 and not for n = 64 or 256, so shorter rows keep the exchange.
template <int LOGN>
constexpr bool mirror_ok() {
  using P = RowPlan<LOGN>;
  if constexpr (LOGN < 10 || P::NP < 2) {
    return false;
  } else {
    constexpr int RL = radix(LOGN, P::NP - 1);
    return P::E / RL == 2 && 2 * P::TPR == P::N / RL && P::TPR > 1;
  }
}

// Butterfly of slot b of thread t in pass Q (b a compile-time constant at every call).
template <int LOGN, int Q, bool MIR>
__device__ __forceinline__ int bfly(int t, int b) {
  using P = RowPlan<LOGN>;
  if constexpr (MIR && Q == P::NP - 1) {
    constexpr int NsL = P::N / radix(LOGN, Q);
    return b == 0 ? t : (t == 0 ? NsL / 2 : NsL - t);
  } else {
    return t + b * P::TPR;
  }
}

// One Stockham pass q: twiddles (q > 0) then radix-R DFTs on the thread's butterflies.
template <int LOGN, int Q, bool INV, bool MIR = false>
__device__ __forceinline__ void stockham_compute(float2* v, int t, const float2* __restrict__ tw) {
  using P = RowPlan<LOGN>;
  constexpr int R = radix(LOGN, Q);
  constexpr int Ns = stride_before(LOGN, Q);
  constexpr int BPT = P::E / R;
  if constexpr (Q > 0) {
    constexpr int kOff = pass_table_offset(LOGN, Q);  // forced to a compile-time constant
    constexpr int L = tw_loaded(R);
    static_assert(kOff % 2 == 0 && L % 2 == 0, "twiddle pairs must be 16-byte aligned");
    const float4* __restrict__ twq = reinterpret_cast<const float4*>(tw + kOff);
    static_for<BPT>([&](auto bc) {
      constexpr int b = decltype(bc)::value;
      const int g = bfly<LOGN, Q, MIR>(t, b);
      const int k = g & (Ns - 1);
      // w[r] = W_{Ns*R}^{r*k}: the stored powers r <= L, then w[r] = w[r - L] * w[L]
      float2 w[R > L ? R : L + 1];
      static_for<L / 2>([&](auto ic) {
        constexpr int i = decltype(ic)::value;
        const float4 pr = twq[k * (L / 2) + i];
        w[2 * i + 1] = make_float2(pr.x, pr.y);
        w[2 * i + 2] = make_float2(pr.z, pr.w);
      });
      static_for<R - 1>([&](auto rc) {
        constexpr int r = decltype(rc)::value + 1;
        if constexpr (r > L) w[r] = c_mul<false>(w[r - L], w[L]);
        v[b * R + r] = c_mul<INV>(v[b * R + r], w[r]);
      });
    });
  }
  static_for<BPT>([&](auto bc) { Dft<R, INV>::run(&v[decltype(bc)::value * R]); });
}

// Exchange the outputs of pass Q into the inputs of pass Q+1 through LDS.
// Pass Q writes out[(g/Ns)*Ns*R + (g mod Ns) + r*Ns]; pass Q+1 reads in[g + r*(N/R')].
// With C chunks, round c moves the outputs whose destination lies in chunk c: butterfly
// g writes into chunk g / (N/(R*C)), which is decided by the butterfly slot b when a
// thread holds at least C butterflies and by the thread index when it holds one; the
// reads of round c are those with r in chunk c.
template <int LOGN, int Q, int CH, bool MIR = false>
__device__ __forceinline__ void stockham_exchange(float2* v, int t, float2* lds) {
  using P = RowPlan<LOGN, CH>;
  constexpr int N = P::N, E = P::E, C = P::C, TPR = P::TPR;
  constexpr int R = radix(LOGN, Q), Ns = stride_before(LOGN, Q), BPT = E / R;
  constexpr int R2 = radix(LOGN, Q + 1), BPT2 = E / R2;
  constexpr int CS = N / C;  // slots per chunk
  static_assert(C == 1 || ((BPT % C == 0 || BPT == 1) && R2 % C == 0), "chunking needs C | BPT (or BPT = 1) and C | R'");
  // every address of this exchange goes through one padding rule, the wide one where it applies
  constexpr bool WIDE = wide_exchange(LOGN, Q, C);
  const auto xp = [](int i) { return WIDE ? lds_pad_wide(i) : lds_pad(i); };
  float2 nv[E];
  static_for<C>([&](auto cc) {
    constexpr int c = decltype(cc)::value;
    static_for<BPT>([&](auto bc) {
      constexpr int b = decltype(bc)::value;
      auto write = [&]() {
        const int g = t + b * TPR;
        const int k = g & (Ns - 1);
        const int pb = xp((g - k) * R + k - c * CS);
        static_for<R>([&](auto rc) {
          constexpr int r = decltype(rc)::value;
          lds[pb + xp(r * Ns)] = v[b * R + r];
        });
      };
      if constexpr (BPT % C == 0) {
        if constexpr (b / (BPT / C) == c) write();
      } else if (t / (TPR / C) == c) {  // one butterfly per thread: no barrier inside
        write();
      }
    });
    row_sync<TPR>();
    static_for<BPT2>([&](auto bc) {
      constexpr int b = decltype(bc)::value;
      const int pg = xp(bfly<LOGN, Q + 1, MIR>(t, b));
      static_for<R2>([&](auto rc) {
        constexpr int r = decltype(rc)::value;
        // chunk c starts at r = c*R2/C, i.e. at index c*CS: the address is g + (r - c*R2/C)*(N/R2)
        if constexpr (r / (R2 / C) == c) nv[b * R2 + r] = lds[pg + xp((r - c * (R2 / C)) * (N / R2))];
      });
    });
    row_sync<TPR>();
  });
  static_for<E>([&](auto ic) { v[decltype(ic)::value] = nv[decltype(ic)::value]; });
}

template <int LOGN, int Q, bool INV, int CH = kChunks[LOGN], bool MIR = false>
__device__ __forceinline__ void stockham_from(float2* v, int t, float2* lds, const float2* __restrict__ tw) {
  stockham_compute<LOGN, Q, INV, MIR>(v, t, tw);
  if constexpr (Q + 1 < RowPlan<LOGN>::NP) {
    stockham_exchange<LOGN, Q, CH, MIR>(v, t, lds);
    stockham_from<LOGN, Q + 1, INV, CH, MIR>(v, t, lds, tw);
  }
}

// ----------------------------------------------------------------------------------
// Forward rdFFT of one row, in two steps so that a caller can issue the loads of one
// row before it computes another:
//   load_forward        thread t's first-pass inputs in storage form: slot
//                       g + r*(N/R0) at raw[b*R0 + r], g = t + b*TPR
//   row_forward_loaded  the transform of those inputs
//   t      thread index within the row's TPR threads
//   active false for padding rows past the end of the batch: their loads read a valid
//          row and their results are not stored
//   dst    output packed pairs P[k]
//   lds    the row's LDS region (RowPlan::LDS_F2 float2); may be the storage of dst
//          when DST_IN_LDS (then a barrier separates the last LDS read from the stores)
template <int LOGN, class Src>
__device__ __forceinline__ void load_forward(int t, const Src& src, typename Src::raw_t* raw) {
  using P = RowPlan<LOGN>;
  if constexpr (LOGN == 0) {
    raw[0] = src.load_raw(0);
  } else {
    constexpr int N = P::N, E = P::E, TPR = P::TPR, R0 = radix(LOGN, 0), BPT0 = E / R0;
    static_for<BPT0>([&](auto bc) {
      constexpr int b = decltype(bc)::value;
      const int g = t + b * TPR;
      if constexpr (shifted_access<Src, LOGN>()) {
        const auto* p = src.base + g;
        static_for<R0>([&](auto rc) {
          constexpr int r = decltype(rc)::value;
          raw[b * R0 + r] = p[r * (N / R0)];
        });
      } else {
        static_for<R0>([&](auto rc) {
          constexpr int r = decltype(rc)::value;
          raw[b * R0 + r] = src.load_raw(g + r * (N / R0));
        });
      }
    });
  }
}

template <int LOGN, bool DST_IN_LDS, class Src, class Dst, int CH = kChunks[LOGN], bool MIR = false>
__device__ __forceinline__ void row_forward_loaded(int t, bool active, const typename Src::raw_t* raw,
                                                   const Dst& dst, float2* lds, const float2* __restrict__ tw) {
  static_assert(!MIR || (mirror_ok<LOGN>() && !DST_IN_LDS), "mirrored last pass: standalone rows only");
  using P = RowPlan<LOGN>;
  constexpr int N = P::N, E = P::E, TPR = P::TPR;
  if constexpr (LOGN == 0) {
    // n = 2: Y_0 = x0 + x1, Y_1 = x0 - x1.  The barrier stays outside any branch.
    const float2 z = Src::widen(raw[0]);
    if constexpr (DST_IN_LDS) row_sync<TPR>();
    if (active) dst.store(0, make_float2(z.x + z.y, z.x - z.y));
    return;
  } else {
    float2 v[E];
    static_for<E>([&](auto ic) { v[decltype(ic)::value] = Src::widen(raw[decltype(ic)::value]); });
    stockham_from<LOGN, 0, false, CH, MIR>(v, t, lds, tw);

    // Post-pass.  After the last pass thread t holds Z_m at m = g_b + r*(N/RL).
    constexpr int RL = radix(LOGN, P::NP - 1), BPL = E / RL, NsL = N / RL;
    constexpr int kPostOff = post_table_offset(LOGN);
    const float2* __restrict__ twp = tw + kPostOff;
    if constexpr (MIR) {
      // thread t holds butterfly g0 = t in v[0, RL) and g1 = N/RL - t in v[RL, 2 RL); thread
      // 0 holds g0 = 0 and g1 = N/(2 RL), each of which pairs with itself
      if (!active) return;
      const bool z = t == 0;
      const float2 tw0 = twp[t];  // -i W_n^t / 2
      // slots j >= RL/2: other threads pair v[j] (bin t + j N/RL) with v[2RL-1-j]; thread 0
      // pairs v[RL + j] (bin N/(2RL) + j N/RL of its second butterfly) with the same v[2RL-1-j],
      // so only the first operand, the twiddle (-i W_n^{N/(2RL)} / 2 = -i W_{4RL} / 2) and
      // the bins' base differ
      const float2 tw1 = z ? rot<4 * RL, 1, false>(make_float2(0.f, -0.5f)) : tw0;
      const int kb1 = z ? NsL / 2 : t;
      static_for<RL>([&](auto jc) {
        constexpr int j = decltype(jc)::value;
        float2 a, pt, twj;
        int k;
        if constexpr (j < RL / 2) {
          a = v[j];
          pt = (j == 0 || !z) ? v[2 * RL - 1 - j] : v[RL - j];
          k = t + j * NsL;
          twj = tw0;
        } else {
          a = z ? v[RL + j] : v[j];
          pt = v[2 * RL - 1 - j];
          k = kb1 + j * NsL;
          twj = tw1;
        }
        const float2 bc2 = c_conj(pt);
        const float2 s = c_add(a, bc2), d = c_sub(a, bc2);
        const float2 q = c_mul<false>(d, rot<2 * RL, j, false>(twj));
        float2 lo = make_float2(fmaf(s.x, 0.5f, q.x), fmaf(s.y, 0.5f, q.y));
        float2 hi = make_float2(fmaf(s.x, 0.5f, -q.x), -fmaf(s.y, 0.5f, -q.y));
        int hi_idx = N - k;
        if constexpr (j == 0) {
          // thread 0: slot 0 = (Y_0, Y_{n/2}) and Y_{N/2} = conj(Z_{N/2}) (v[RL/2])
          const float2 zh = c_conj(v[RL / 2]);
          lo = z ? make_float2(a.x + a.y, a.x - a.y) : lo;
          hi = z ? zh : hi;
          hi_idx = z ? N / 2 : hi_idx;
        }
        if constexpr (shifted_access<Dst, LOGN>()) {
          // bins k = kb + j N/RL from kb's address, partners N - k from N - kb's (thread
          // 0's first partner is slot N/2)
          constexpr int jj = j < RL / 2 ? j : j - RL / 2;
          auto* lo_p = dst.base + (j < RL / 2 ? t : kb1 + (RL / 2) * NsL);
          auto* hi_p = dst.base + (N - (j < RL / 2 ? t : kb1 + (RL / 2) * NsL));
          lo_p[jj * NsL] = Dst::narrow(lo);
          if constexpr (j == 0) (z ? dst.base + N / 2 : hi_p)[0] = Dst::narrow(hi);
          else hi_p[-jj * NsL] = Dst::narrow(hi);
        } else {
          dst.store(k, lo);
          dst.store(hi_idx, hi);
        }
      });
      return;
    }
    float2 partner[E / 2];
    if constexpr (TPR == 1) {
      // the whole row is in this thread's registers: Z_{N-k} is v at N-k
      static_for<BPL>([&](auto bc) {
        constexpr int b = decltype(bc)::value;
        static_for<RL / 2>([&](auto rc) {
          constexpr int r = decltype(rc)::value;
          constexpr int k = b + r * NsL;
          if constexpr (k != 0) {
            constexpr int mk = N - k;
            partner[b * (RL / 2) + r] = v[(mk % NsL) * RL + mk / NsL];
          } else {
            partner[b * (RL / 2) + r] = make_float2(0.f, 0.f);  // unused: slot 0 is special
          }
        });
      });
      if constexpr (DST_IN_LDS) row_sync<TPR>();
    } else {
      static_for<BPL>([&](auto bc) {
        constexpr int b = decltype(bc)::value;
        const int pg = lds_pad(t + b * TPR);
        static_for<RL / 2>([&](auto rc) {
          constexpr int r = decltype(rc)::value;  // element r + RL/2 sits at g + r*NsL past N/2
          lds[pg + pad_step(r * NsL)] = v[b * RL + r + RL / 2];
        });
      });
      row_sync<TPR>();
      static_for<BPL>([&](auto bc) {
        constexpr int b = decltype(bc)::value;
        const int g = t + b * TPR;
        // Z_{N-k} for k = g + r*NsL sits at N/2 - k = (NsL - g) + (RL/2 - 1 - r)*NsL;
        // k == 0 reads index N/2 (never written); its value is unused
        const int pq = lds_pad(NsL - g);
        static_for<RL / 2>([&](auto rc) {
          constexpr int r = decltype(rc)::value;
          if constexpr (NsL % 16 == 0) {
            partner[b * (RL / 2) + r] = lds[pq + pad_step((RL / 2 - 1 - r) * NsL)];
          } else {
            partner[b * (RL / 2) + r] = lds[lds_pad(N / 2 - g - r * NsL)];
          }
        });
      });
      if constexpr (DST_IN_LDS) row_sync<TPR>();
    }
    if (!active) return;
    static_for<BPL>([&](auto bc) {
      constexpr int b = decltype(bc)::value;
      const int g = t + b * TPR;
      const float2 twg = twp[g];  // -i W_n^g / 2
      static_for<RL / 2>([&](auto rc) {
        constexpr int r = decltype(rc)::value;
        const int k = g + r * NsL;
        const float2 a = v[b * RL + r];
        const float2 bc2 = c_conj(partner[b * (RL / 2) + r]);
        const float2 s = c_add(a, bc2), d = c_sub(a, bc2);
        // Y_k = s/2 + (-i W_n^k / 2) d,  Y_{N-k} = conj(s/2 - (-i W_n^k / 2) d), with
        // W_n^k = W_n^g W_{2RL}^r (k = 0: the slot-0 select replaces the result)
        const float2 q = c_mul<false>(d, rot<2 * RL, r, false>(twg));
        float2 lo = make_float2(fmaf(s.x, 0.5f, q.x), fmaf(s.y, 0.5f, q.y));
        float2 hi = make_float2(fmaf(s.x, 0.5f, -q.x), -fmaf(s.y, 0.5f, -q.y));
        int hi_idx = N - k;
        if constexpr (b == 0 && r == 0) {
          // k == 0 (thread 0): slot 0 = (Y_0, Y_{n/2}) = (Re Z_0 + Im Z_0, Re Z_0 - Im Z_0)
          // and Y_{N/2} = conj(Z_{N/2}); chosen by selects so the stores stay uniform
          const bool z = t == 0;
          const float2 zh = c_conj(v[RL / 2]);
          lo = z ? make_float2(a.x + a.y, a.x - a.y) : lo;
          hi = z ? zh : hi;
          hi_idx = z ? N / 2 : hi_idx;
        }
        if constexpr (std::is_same<Dst, RegSpectrum>::value) {
          // k = t + TPR*(b + BPL*r): register index j = b + BPL*r
          dst.lo[b + BPL * r] = lo;
          dst.hi[b + BPL * r] = hi;
        } else if constexpr (shifted_access<Dst, LOGN>()) {
          // bins g + r N/RL from g's address, partners N - g - r N/RL from N - g's (thread
          // 0's first partner is slot N/2)
          auto* lo_p = dst.base + g;
          auto* hi_p = dst.base + (N - g);
          lo_p[r * NsL] = Dst::narrow(lo);
          if constexpr (b == 0 && r == 0) (t == 0 ? dst.base + N / 2 : hi_p)[0] = Dst::narrow(hi);
          else hi_p[-r * NsL] = Dst::narrow(hi);
        } else {
          dst.store(k, lo);
          dst.store(hi_idx, hi);
        }
      });
    });
  }
}

template <int LOGN, bool DST_IN_LDS, class Src, class Dst, int CH = kChunks[LOGN], bool MIR = false>
__device__ __forceinline__ void row_forward(int t, bool active, const Src& src, const Dst& dst, float2* lds,
                                            const float2* __restrict__ tw) {
  typename Src::raw_t raw[RowPlan<LOGN>::E];
  load_forward<LOGN>(t, src, raw);
  row_forward_loaded<LOGN, DST_IN_LDS, Src, Dst, CH, MIR>(t, active, raw, dst, lds, tw);
}

// ----------------------------------------------------------------------------------
// Inverse rdFFT of one row: packed pairs P[k] -> pairs (x_{2m}, x_{2m+1}) (dst), split
// like the forward:
//   load_inverse        thread t's pre-pass inputs in storage form: for m = g + r*(N/R0),
//                       r < R0/2, slot m at raw[b*R0 + r] and its partner N - m (N/2 for
//                       m == 0) at raw[b*R0 + R0/2 + r]
//   row_inverse_loaded  the transform of those inputs
// SRC_IN_LDS: the loads read this row's LDS region (a barrier then separates them from
// the first LDS write).
template <int LOGN, class Src>
__device__ __forceinline__ void load_inverse(int t, const Src& src, typename Src::raw_t* raw) {
  using P = RowPlan<LOGN>;
  if constexpr (LOGN == 0) {
    raw[0] = src.load_raw(0);
  } else {
    constexpr int N = P::N, E = P::E, TPR = P::TPR, R0 = radix(LOGN, 0), BPT0 = E / R0;
    static_for<BPT0>([&](auto bc) {
      constexpr int b = decltype(bc)::value;
      const int g = t + b * TPR;
      if constexpr (shifted_access<Src, LOGN>()) {
        // slots g + r S0 from one address, partners N - g - r S0 from another (thread 0's
        // first partner is slot N/2)
        const auto* lo = src.base + g;
        const auto* hi = src.base + (N - g);
        static_for<R0 / 2>([&](auto rc) {
          constexpr int r = decltype(rc)::value;
          raw[b * R0 + r] = lo[r * (N / R0)];
          if constexpr (b == 0 && r == 0) raw[b * R0 + R0 / 2 + r] = (t == 0 ? src.base + N / 2 : hi)[0];
          else raw[b * R0 + R0 / 2 + r] = hi[-r * (N / R0)];
        });
      } else {
        static_for<R0 / 2>([&](auto rc) {
          constexpr int r = decltype(rc)::value;
          const int m = g + r * (N / R0);
          // m == 0 only for thread 0 at (b, r) = (0, 0); it pairs with slot N/2 instead of N
          const bool z = (b == 0 && r == 0) ? (t == 0) : false;
          raw[b * R0 + r] = src.load_raw(m);
          raw[b * R0 + R0 / 2 + r] = src.load_raw(z ? N / 2 : N - m);
        });
      }
    });
  }
}

template <int LOGN, bool SRC_IN_LDS, class Src, class Dst, int CH = kChunks[LOGN]>
__device__ __forceinline__ void row_inverse_loaded(int t, bool active, const typename Src::raw_t* raw,
                                                   const Dst& dst, float2* lds, const float2* __restrict__ tw) {
  using P = RowPlan<LOGN>;
  constexpr int N = P::N, E = P::E, TPR = P::TPR;
  constexpr float sc = 1.0f / (2.0f * N);  // 1/n
  if constexpr (LOGN == 0) {
    const float2 y = Src::widen(raw[0]);
    if (active) dst.store(0, make_float2(0.5f * (y.x + y.y), 0.5f * (y.x - y.y)));
    return;
  } else {
    constexpr int R0 = radix(LOGN, 0), BPT0 = E / R0;
    constexpr int kPostOff = post_table_offset(LOGN);
    const float2* __restrict__ twp = tw + kPostOff;
    float2 v[E];
    float2 mirror[E / 2];  // Z~_{N-m} for this thread's jobs m < N/2
    float2 zhalf;          // Z~_{N/2} = conj(Y_{N/2}) * 2/n (meaningful in thread 0 only)
    static_for<BPT0>([&](auto bc) {
      constexpr int b = decltype(bc)::value;
      const int g = t + b * TPR;
      const float2 twg = twp[N / 2 + g];  // i conj(W_n^g) / n
      static_for<R0 / 2>([&](auto rc) {
        constexpr int r = decltype(rc)::value;
        const bool z = (b == 0 && r == 0) ? (t == 0) : false;
        const float2 ya = Src::widen(raw[b * R0 + r]);
        const float2 yb = c_conj(Src::widen(raw[b * R0 + R0 / 2 + r]));
        const float2 s = c_add(ya, yb), d = c_sub(ya, yb);
        // Z~_m = (s + i conj(W_n^m) d) / n,  Z~_{N-m} = conj(s - i conj(W_n^m) d) / n for
        // m = g + r*N/R0, with conj(W_n^m) = conj(W_n^g) conj(W_{2R0}^r)
        const float2 q = c_mul<false>(d, rot<2 * R0, r, true>(twg));
        float2 lo = make_float2(fmaf(s.x, sc, q.x), fmaf(s.y, sc, q.y));
        float2 hi = make_float2(fmaf(s.x, sc, -q.x), -fmaf(s.y, sc, -q.y));
        if constexpr (b == 0 && r == 0) {
          // Z~_0 = ((Y_0 + Y_{n/2}) + i (Y_0 - Y_{n/2})) / n ;  Z~_{N/2} = conj(Y_{N/2}) * 2/n
          lo = z ? make_float2(sc * (ya.x + ya.y), sc * (ya.x - ya.y)) : lo;
          zhalf = c_scale(yb, 2.0f * sc);
        }
        v[b * R0 + r] = lo;
        mirror[b * (R0 / 2) + r] = hi;
      });
    });
    if constexpr (TPR == 1) {
      // the partner values are this thread's own upper-half inputs
      v[R0 / 2] = zhalf;
      static_for<BPT0>([&](auto bc) {
        constexpr int b = decltype(bc)::value;
        static_for<R0 / 2>([&](auto rc) {
          constexpr int r = decltype(rc)::value;
          constexpr int m = b + r * (N / R0);
          if constexpr (m != 0) {
            constexpr int mm = N - m;
            v[(mm % (N / R0)) * R0 + mm / (N / R0)] = mirror[b * (R0 / 2) + r];
          }
        });
      });
    } else {
      if constexpr (SRC_IN_LDS) row_sync<TPR>();
      constexpr int S0 = N / R0;
      static_for<BPT0>([&](auto bc) {
        constexpr int b = decltype(bc)::value;
        const int g = t + b * TPR;
        // Z~_{N-m} for m = g + r*S0 goes to N/2 - m = (S0 - g) + (R0/2 - 1 - r)*S0; the
        // m == 0 element (thread 0) lands on index N/2, which nobody reads
        const int pq = lds_pad(S0 - g);
        static_for<R0 / 2>([&](auto rc) {
          constexpr int r = decltype(rc)::value;
          if constexpr (S0 % 16 == 0) {
            lds[pq + pad_step((R0 / 2 - 1 - r) * S0)] = mirror[b * (R0 / 2) + r];
          } else {
            lds[lds_pad(N / 2 - g - r * S0)] = mirror[b * (R0 / 2) + r];
          }
        });
      });
      // element m = N/2 (thread 0) reads index 0, which no mirror write touches
      if (t == 0) lds[0] = zhalf;
      row_sync<TPR>();
      static_for<BPT0>([&](auto bc) {
        constexpr int b = decltype(bc)::value;
        const int g = t + b * TPR;
        const int pg = lds_pad(g);
        static_for<R0 / 2>([&](auto rc) {
          constexpr int r = decltype(rc)::value;  // element r + R0/2 is at m - N/2 = g + r*S0
          v[b * R0 + r + R0 / 2] = lds[pg + pad_step(r * S0)];
        });
      });
      row_sync<TPR>();
    }
    stockham_from<LOGN, 0, true, CH>(v, t, lds, tw);
    if (!active) return;
    constexpr int RL = radix(LOGN, P::NP - 1), BPL = E / RL, NsL = N / RL;
    static_for<BPL>([&](auto bc) {
      constexpr int b = decltype(bc)::value;
      const int g = t + b * TPR;
      if constexpr (shifted_access<Dst, LOGN>()) {
        auto* p = dst.base + g;
        static_for<RL>([&](auto rc) {
          constexpr int r = decltype(rc)::value;
          p[r * NsL] = Dst::narrow(v[b * RL + r]);
        });
      } else {
        static_for<RL>([&](auto rc) {
          constexpr int r = decltype(rc)::value;
          dst.store(g + r * NsL, v[b * RL + r]);
        });
      }
    });
  }
}

template <int LOGN, bool SRC_IN_LDS, class Src, class Dst, int CH = kChunks[LOGN]>
__device__ __forceinline__ void row_inverse(int t, bool active, const Src& src, const Dst& dst, float2* lds,
                                            const float2* __restrict__ tw) {
  typename Src::raw_t raw[RowPlan<LOGN>::E];
  load_inverse<LOGN>(t, src, raw);
  row_inverse_loaded<LOGN, SRC_IN_LDS, Src, Dst, CH>(t, active, raw, dst, lds, tw);
}

}  // namespace rdfft
