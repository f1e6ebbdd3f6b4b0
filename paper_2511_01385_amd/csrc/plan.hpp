// plan.hpp -- compile-time transform plans and twiddle-table layout.
//
// A real row of n = 2N samples is viewed as N complex points z_m = x_{2m} + i x_{2m+1}
// (the interleaved pairs already are that view).  The row transform computes the
// N-point complex DFT of z with a Stockham (self-sorting) sequence of radix passes
// held in registers and exchanged through LDS, then the real-to-packed post-pass
// that turns Z into the n/2+1 real-signal bins Y_k (Sec. 4.1, "Squeeze N+2 into N").
//
// Shared by the host table generator and the device kernels of this library.
#pragma once

#include <stdint.h>

namespace rdfft {

constexpr int kMaxLogN = 15;  // N = 32768 complex points, n = 65536 reals

// Radix sequence per log2(N).  Pass q multiplies the sub-transform size by kPlan[q].
constexpr int kPlan[kMaxLogN + 1][5] = {
    {0},              // N = 1: handled by the post-pass alone
    {2},              // 2
    {4},              // 4
    {8},              // 8
    {16},             // 16
    {8, 4},           // 32
    {8, 8},           // 64
    {16, 8},          // 128
    {16, 16},         // 256
    {8, 8, 8},        // 512
    {16, 8, 8},       // 1024
    {16, 16, 8},      // 2048
    {16, 16, 16},     // 4096
    {16, 16, 8, 4},   // 8192
    {16, 16, 16, 4},  // 16384
    {32, 32, 32},     // 32768
};

// Complex values each thread holds (E) and LDS exchange chunks (C).  With C > 1 a
// pass-to-pass exchange is split into C rounds so that one round fits in LDS.
constexpr int kElems[kMaxLogN + 1] = {1, 2, 4, 8, 16, 8, 8, 16, 16, 8, 16, 16, 16, 16, 16, 32};
constexpr int kChunks[kMaxLogN + 1] = {1, 1, 1, 1, 1, 1, 1, 1, 1, 1, 1, 1, 1, 1, 1, 2};
// The bf16 row kernels of rows n >= 2048 also exchange in two rounds: the halved LDS region
// admits more resident waves, which pays where the arithmetic, not HBM, bounds the time.
constexpr int kChunksBf16[kMaxLogN + 1] = {1, 1, 1, 1, 1, 1, 1, 1, 1, 1, 2, 2, 2, 2, 2, 2};

constexpr int num_passes(int logn) {
  int k = 0;
  while (k < 5 && kPlan[logn][k] != 0) ++k;
  return k;
}

constexpr int radix(int logn, int q) { return kPlan[logn][q]; }

// product of the radices of passes before q
constexpr int stride_before(int logn, int q) {
  int s = 1;
  for (int i = 0; i < q; ++i) s *= kPlan[logn][i];
  return s;
}

constexpr bool plan_is_consistent(int logn) {
  int prod = 1;
  for (int q = 0; q < num_passes(logn); ++q) {
    prod *= radix(logn, q);
    if (kElems[logn] % radix(logn, q) != 0) return false;
  }
  return prod == (1 << logn);
}

// Twiddles of pass q >= 1 with radix R: butterfly k < Ns multiplies its input r by
// W_{Ns*R}^{r*k}, 1 <= r < R.  Only the first tw_loaded(R) powers are stored, at
// [k*L + r - 1] for 1 <= r <= L (L = tw_loaded(R), even, so a butterfly reads them as
// 16-byte pairs); the kernels form the others as products, W^{rk} = W^{(r-L)k} W^{Lk}.
// Every table read costs a vector-memory instruction, and those, not the arithmetic,
// bound the row kernels when each power is read on its own.
constexpr int tw_loaded(int R) { return R >= 8 ? 4 : 2; }
constexpr int pass_table_size(int logn, int q) {
  return q == 0 ? 0 : tw_loaded(radix(logn, q)) * stride_before(logn, q);
}

// Post-pass twiddles, 0 <= k < N/2, with the post-pass scale folded in (exact: powers of two):
//   forward  [k]       = (1/2) * (-i) * W_n^k
//   inverse  [N/2 + k] = (1/n) * i * conj(W_n^k),   W_n^k = exp(-2 pi i k / (2N)).
// A thread reads the entry of its first bin only: its other bins lie N/R apart (R the
// radix of the last pass, or of the first for the inverse), and W_n^{N/R} = W_{2R} is a
// compile-time constant.
constexpr int post_table_size(int logn) { return 2 * ((1 << logn) / 2); }

constexpr int plan_table_size(int logn) {
  int s = 0;
  for (int q = 0; q < num_passes(logn); ++q) s += pass_table_size(logn, q);
  return s + post_table_size(logn);
}

constexpr int plan_table_offset(int logn) {
  int s = 0;
  for (int l = 0; l < logn; ++l) s += plan_table_size(l);
  return s;
}

constexpr int pass_table_offset(int logn, int q) {
  int s = plan_table_offset(logn);
  for (int i = 0; i < q; ++i) s += pass_table_size(logn, i);
  return s;
}

constexpr int post_table_offset(int logn) {
  return plan_table_offset(logn) + plan_table_size(logn) - post_table_size(logn);
}

constexpr int kTableEntries = plan_table_offset(kMaxLogN + 1);  // float2 entries

// LDS padding: one float2 of padding after every 16, so that the strided
// Stockham writes of the early passes spread over all banks.
constexpr int lds_pad(int i) { return i + (i >> 4); }
constexpr int lds_padded_size(int count) { return count + (count >> 4) + 1; }

// The exchange after a radix-8 pass of stride 8 (the n = 1024 plan 8.8.8) writes groups of 8
// consecutive slots 64 apart, and lds_pad puts neighbouring groups on overlapping banks (one
// extra cycle per 16 lanes).  Four more slots of padding every 64 move every other group by
// half the banks.  That padding stays additive over the exchange's base-plus-offset addresses
// (write bases 64m + j with j < 8 and offsets below 64; read offsets multiples of 64) whenever
// the next pass's sub-transform stride N/R' is a multiple of 64, which the test requires.
constexpr int lds_pad_wide(int i) { return i + (i >> 4) + 4 * (i >> 6); }
constexpr bool wide_exchange(int logn, int q, int chunks) {
  return chunks == 1 && q + 1 < num_passes(logn) && stride_before(logn, q) == 8 && radix(logn, q) == 8 &&
         ((1 << logn) / radix(logn, q + 1)) % 64 == 0;
}
constexpr bool plan_has_wide_exchange(int logn, int chunks) {
  bool any = false;
  for (int q = 0; q + 1 < num_passes(logn); ++q) any = any || wide_exchange(logn, q, chunks);
  return any;
}

// The exchanges address LDS as pad(base) + pad(offset): a per-butterfly base and compile-time
// offsets.  pad(base + offset) - pad(base) - pad(offset) is the carry out of the low four
// bits (plus four times the carry out of the low six for lds_pad_wide), so the split is exact
// when (base & 15) + (offset & 15) < 16 (and (base & 63) + (offset & 63) < 64) for every pair.
// exchange_split_ok checks that for every exchange of a plan, over all residues of the bases
// mod 64 and the largest low bits of the offsets, so a plan or padding that breaks it does not
// compile.  (The post-pass and pre-pass partner exchanges take the split form only when their
// offsets are multiples of 16, which carry nothing.)
constexpr bool split_carry_free(int base, int off_low4, int off_low6, bool wide) {
  return (base & 15) + off_low4 < 16 && (!wide || (base & 63) + off_low6 < 64);
}
constexpr bool exchange_split_ok(int logn, int chunks) {
  if (logn == 0) return true;
  const int N = 1 << logn, NP = num_passes(logn), CS = N / chunks;
  if (chunks > 1 && CS % 64 != 0) return false;  // a chunk's origin must leave the low bits alone
  for (int q = 0; q + 1 < NP; ++q) {
    const int R = radix(logn, q), Ns = stride_before(logn, q), R2 = radix(logn, q + 1);
    const bool wide = wide_exchange(logn, q, chunks);
    // writes: base (g - k) R + k - c CS, offsets r Ns (r < R)
    int l4 = 0, l6 = 0;
    for (int r = 0; r < R; ++r) {
      l4 = (r * Ns) % 16 > l4 ? (r * Ns) % 16 : l4;
      l6 = (r * Ns) % 64 > l6 ? (r * Ns) % 64 : l6;
    }
    const int nm = N / (R * Ns) < 64 ? N / (R * Ns) : 64, nk = Ns < 64 ? Ns : 64;
    for (int m = 0; m < nm; ++m)
      for (int k = 0; k < nk; ++k)
        if (!split_carry_free((Ns * R * m + k) % 64, l4, l6, wide)) return false;
    // reads: base g < N/R', offsets j N/R' (j < R'/chunks)
    l4 = 0, l6 = 0;
    for (int j = 0; j < R2 / chunks; ++j) {
      l4 = (j * (N / R2)) % 16 > l4 ? (j * (N / R2)) % 16 : l4;
      l6 = (j * (N / R2)) % 64 > l6 ? (j * (N / R2)) % 64 : l6;
    }
    const int ng = N / R2 < 64 ? N / R2 : 64;
    for (int g = 0; g < ng; ++g)
      if (!split_carry_free(g, l4, l6, wide)) return false;
  }
  return true;
}

// Stride between the LDS regions of rows that share a wavefront.  ds_write_b64 and the
// paired ds_read2_b64 serve 16 lanes per cycle from 32 four-byte banks, so the 16/TPR rows
// in such a group should fall on disjoint banks: one row's lanes cover 2*TPR words, which
// asks for a stride of TPR float2 modulo 16.  Rows of 16 or more threads need nothing.
constexpr int lds_row_stride(int count, int tpr) {
  return tpr >= 16 ? lds_padded_size(count) : lds_padded_size(count) + ((tpr - lds_padded_size(count) % 16) % 16 + 16) % 16;
}

}  // namespace rdfft
