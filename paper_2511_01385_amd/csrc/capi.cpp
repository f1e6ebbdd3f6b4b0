// capi.cpp -- the library's extern "C" entry points (declared in include/rdfft.h).
//
// Every entry point validates its arguments on the host before making any HIP call,
// then enqueues its kernels on the caller's stream.  Nothing here allocates device
// memory; the per-device twiddle table is a static __device__ array filled on first
// use.
#include <hip/hip_runtime.h>
#include <stdint.h>
#include <string.h>

#include <atomic>
#include <mutex>
#include <vector>

#include "launch.hpp"
#include "plan.hpp"
#include "rdfft.h"
#include "twiddles.hpp"

namespace {

constexpr int kMaxDevices = 64;

struct DeviceState {
  std::atomic<const float2*> tw{nullptr};
  int num_cu = 0;
};

DeviceState g_dev[kMaxDevices];
std::mutex g_init_mu;

bool is_pow2(int64_t v) { return v > 0 && (v & (v - 1)) == 0; }

int ilog2(int64_t v) {
  int l = 0;
  while ((int64_t(1) << l) < v) ++l;
  return l;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// [a, a+na) and [b, b+nb) share a byte
bool overlaps(const void* a, int64_t na, const void* b, int64_t nb) {
  const uintptr_t x = reinterpret_cast<uintptr_t>(a), y = reinterpret_cast<uintptr_t>(b);
  return na > 0 && nb > 0 && x < y + (uintptr_t)nb && y < x + (uintptr_t)na;
}

int elem_bytes(int dtype) { return dtype == RDFFT_F32 ? 4 : 2; }

// products of sizes that must not overflow int64
bool mul_ok(int64_t a, int64_t b, int64_t* out) {
  if (a < 0 || b < 0) return false;
  if (a != 0 && b > INT64_MAX / a) return false;
  *out = a * b;
  return true;
}

int ensure_device(const float2** tw, int* num_cu) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return RDFFT_EDEVICE;
  DeviceState& st = g_dev[dev];
  const float2* p = st.tw.load(std::memory_order_acquire);
  if (p == nullptr) {
    std::lock_guard<std::mutex> lock(g_init_mu);
    p = st.tw.load(std::memory_order_relaxed);
    if (p == nullptr) {
      hipDeviceProp_t prop;
      if (hipGetDeviceProperties(&prop, dev) != hipSuccess) return RDFFT_EDEVICE;
      if (strncmp(prop.gcnArchName, "gfx950", 6) != 0) return RDFFT_EDEVICE;
      static const std::vector<rdfft::HostC32> host = rdfft::build_twiddle_table();
      if (rdfft::upload_twiddles(host.data(), host.size() * sizeof(rdfft::HostC32), &p) != hipSuccess)
        return RDFFT_EDEVICE;
      st.num_cu = prop.multiProcessorCount;
      st.tw.store(p, std::memory_order_release);
    }
  }
  *tw = p;
  if (num_cu) *num_cu = st.num_cu;
  return RDFFT_OK;
}

int check_transform(const void* buf, int64_t rows, int64_t n, int dtype) {
  if (dtype != RDFFT_F32 && dtype != RDFFT_BF16 && dtype != RDFFT_F16) return RDFFT_EINVAL;
  if (rows < 0) return RDFFT_EINVAL;
  if (n < 2 || (n & 1)) return RDFFT_EINVAL;
  if (is_pow2(n) ? n > (int64_t(2) << rdfft::kMaxLogN) : !rdfft::mixed_length_supported(n))
    return RDFFT_EUNSUPPORTED;
  if (rows == 0) return RDFFT_OK;
  int64_t count = 0, bytes = 0;
  if (!mul_ok(rows, n, &count) || !mul_ok(count, elem_bytes(dtype), &bytes)) return RDFFT_EINVAL;
  if (buf == nullptr || !aligned16(buf)) return RDFFT_EINVAL;
  return RDFFT_OK;
}

// hc: the spectrum side of the transform in the halfcomplex layout instead of pairs
int transform(void* buf, int64_t rows, int64_t n, int dtype, rdfft_stream_t stream, bool inv, bool hc) {
  int st = check_transform(buf, rows, n, dtype);
  if (st != RDFFT_OK || rows == 0) return st;
  const float2* tw = nullptr;
  int num_cu = 0;
  st = ensure_device(&tw, &num_cu);
  if (st != RDFFT_OK) return st;
  const hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  hipError_t e;
  if (!is_pow2(n)) e = rdfft::launch_mixed_rows(buf, rows, n, dtype, inv, hc, s);
  else if (hc) e = rdfft::launch_rdfft_rows_hc(buf, rows, ilog2(n) - 1, dtype, inv, tw, s);
  else e = rdfft::launch_rdfft_rows(buf, rows, ilog2(n) - 1, dtype, inv, tw, s, num_cu);
  return e == hipSuccess ? RDFFT_OK : RDFFT_ELAUNCH;
}

int convert(void* buf, int64_t rows, int64_t n, int dtype, rdfft_stream_t stream, bool to_hc) {
  int st = check_transform(buf, rows, n, dtype);
  if (st != RDFFT_OK || rows == 0) return st;
  // the kernels need no twiddles, but the device check is the same
  const float2* tw = nullptr;
  st = ensure_device(&tw, nullptr);
  if (st != RDFFT_OK) return st;
  const hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  const hipError_t e = is_pow2(n) ? rdfft::launch_layout_convert(buf, rows, ilog2(n) - 1, dtype != RDFFT_F32, to_hc, s)
                                  : rdfft::launch_mixed_layout(buf, rows, n, dtype != RDFFT_F32, to_hc, s);
  return e == hipSuccess ? RDFFT_OK : RDFFT_ELAUNCH;
}

struct BcaShape {
  int q = 0, kb = 0, logp = 0;
  int64_t x_bytes = 0, y_bytes = 0, c_bytes = 0, dc_bytes = 0;
};

int check_bca(const void* x, const void* c, const void* y, int64_t d_in, int64_t d_out, int64_t p, int64_t tokens,
              int dtype, bool backward, BcaShape* sh) {
  if (dtype != RDFFT_F32 && dtype != RDFFT_BF16 && dtype != RDFFT_F16) return RDFFT_EINVAL;
  if (tokens < 0 || d_in <= 0 || d_out <= 0 || p <= 0) return RDFFT_EINVAL;
  if (p < 2 || (p & 1)) return RDFFT_EINVAL;
  if (d_in % p != 0 || d_out % p != 0) return RDFFT_EINVAL;
  if (!is_pow2(p)) return RDFFT_EUNSUPPORTED;
  const int64_t q = d_out / p, kb = d_in / p;
  if (q > (1 << 20) || kb > (1 << 20)) return RDFFT_EUNSUPPORTED;
  sh->q = (int)q;
  sh->kb = (int)kb;
  sh->logp = ilog2(p);
  if (!rdfft::bca_shape_supported(sh->logp, sh->q, sh->kb, backward)) return RDFFT_EUNSUPPORTED;
  const int s = elem_bytes(dtype);
  int64_t t = 0;
  if (!mul_ok(tokens, d_in, &t) || !mul_ok(t, s, &sh->x_bytes)) return RDFFT_EINVAL;
  if (!mul_ok(tokens, d_out, &t) || !mul_ok(t, s, &sh->y_bytes)) return RDFFT_EINVAL;
  if (!mul_ok(q * kb, p, &t) || !mul_ok(t, s, &sh->c_bytes)) return RDFFT_EINVAL;
  sh->dc_bytes = t * 4;
  if (c == nullptr || !aligned16(c)) return RDFFT_EINVAL;
  if (tokens > 0) {
    if (x == nullptr || y == nullptr || !aligned16(x) || !aligned16(y)) return RDFFT_EINVAL;
    if (overlaps(c, sh->c_bytes, x, sh->x_bytes) || overlaps(c, sh->c_bytes, y, sh->y_bytes)) return RDFFT_EINVAL;
  }
  return RDFFT_OK;
}

// bca_forward's checks beyond check_bca (tokens > 0): y may be x itself (an in-place layer)
// only when the shapes agree
int check_forward_alias(const void* x, const void* y, int64_t d_in, int64_t d_out, int64_t p, const BcaShape& sh) {
  if (y == x) {
    if (d_in != d_out) return RDFFT_EINVAL;
    if (p > 8192 && sh.q > rdfft::kMpMaxInPlaceBlocks) return RDFFT_EUNSUPPORTED;
  } else if (overlaps(x, sh.x_bytes, y, sh.y_bytes)) {
    return RDFFT_EINVAL;
  }
  return RDFFT_OK;
}

// bca_backward's checks beyond check_bca
int check_backward_grads(const void* x, const void* c_spectra, const void* gy, const void* dx, const float* dc,
                         int64_t d_in, int64_t d_out, int64_t p, int64_t tokens, const BcaShape& sh) {
  if (dc == nullptr || !aligned16(dc)) return RDFFT_EINVAL;
  if (overlaps(dc, sh.dc_bytes, c_spectra, sh.c_bytes)) return RDFFT_EINVAL;
  if (tokens > 0) {
    if (dx == nullptr || !aligned16(dx)) return RDFFT_EINVAL;
    if (overlaps(x, sh.x_bytes, gy, sh.y_bytes)) return RDFFT_EINVAL;
    if (overlaps(dx, sh.x_bytes, x, sh.x_bytes) || overlaps(dx, sh.x_bytes, c_spectra, sh.c_bytes)) return RDFFT_EINVAL;
    if (dx == gy) {
      if (d_in != d_out) return RDFFT_EINVAL;
      if (p > 8192 && sh.q > rdfft::kMpMaxInPlaceBlocks) return RDFFT_EUNSUPPORTED;
    } else if (overlaps(dx, sh.x_bytes, gy, sh.y_bytes)) {
      return RDFFT_EINVAL;
    }
    if (overlaps(dc, sh.dc_bytes, x, sh.x_bytes) || overlaps(dc, sh.dc_bytes, gy, sh.y_bytes) ||
        overlaps(dc, sh.dc_bytes, dx, sh.x_bytes))
      return RDFFT_EINVAL;
  }
  return RDFFT_OK;
}

// Layers of a batch: nothing one layer writes may overlap anything of another layer (reads
// may share buffers, e.g. one x for several layers).
struct Span {
  const void* p;
  int64_t bytes;
  bool written;
};
bool batch_disjoint(const std::vector<std::vector<Span>>& layers) {
  for (size_t a = 0; a < layers.size(); ++a)
    for (size_t b = a + 1; b < layers.size(); ++b)
      for (const Span& u : layers[a])
        for (const Span& v : layers[b])
          if ((u.written || v.written) && overlaps(u.p, u.bytes, v.p, v.bytes)) return false;
  return true;
}

constexpr int kMaxBatchCount = 1024;

}  // namespace

extern "C" {

int rdfft_forward(void* buf, int64_t rows, int64_t n, rdfft_dtype_t dtype, rdfft_stream_t stream) {
  return transform(buf, rows, n, dtype, stream, false, false);
}

int rdfft_inverse(void* buf, int64_t rows, int64_t n, rdfft_dtype_t dtype, rdfft_stream_t stream) {
  return transform(buf, rows, n, dtype, stream, true, false);
}

int rdfft_forward_halfcomplex(void* buf, int64_t rows, int64_t n, rdfft_dtype_t dtype, rdfft_stream_t stream) {
  return transform(buf, rows, n, dtype, stream, false, true);
}

int rdfft_inverse_halfcomplex(void* buf, int64_t rows, int64_t n, rdfft_dtype_t dtype, rdfft_stream_t stream) {
  return transform(buf, rows, n, dtype, stream, true, true);
}

int rdfft_pairs_to_halfcomplex(void* buf, int64_t rows, int64_t n, rdfft_dtype_t dtype, rdfft_stream_t stream) {
  return convert(buf, rows, n, dtype, stream, true);
}

int rdfft_halfcomplex_to_pairs(void* buf, int64_t rows, int64_t n, rdfft_dtype_t dtype, rdfft_stream_t stream) {
  return convert(buf, rows, n, dtype, stream, false);
}

int bca_forward(const void* x, const void* c_spectra, void* y, bca_grads_t* grads, int64_t d_in, int64_t d_out,
                int64_t p, int64_t tokens, rdfft_dtype_t dtype, rdfft_stream_t stream) {
  if (grads != nullptr) return RDFFT_EINVAL;
  BcaShape sh;
  int st = check_bca(x, c_spectra, y, d_in, d_out, p, tokens, dtype, false, &sh);
  if (st != RDFFT_OK) return st;
  if (tokens == 0) return RDFFT_OK;
  st = check_forward_alias(x, y, d_in, d_out, p, sh);
  if (st != RDFFT_OK) return st;
  const float2* tw = nullptr;
  int num_cu = 0;
  st = ensure_device(&tw, &num_cu);
  if (st != RDFFT_OK) return st;
  rdfft::BcaArgs a{x, c_spectra, y, nullptr, nullptr, tokens, sh.q, sh.kb, sh.logp, dtype};
  return rdfft::launch_bca_forward(a, tw, reinterpret_cast<hipStream_t>(stream), num_cu) == hipSuccess
             ? RDFFT_OK
             : RDFFT_ELAUNCH;
}

int bca_backward(const void* x, const void* c_spectra, void* gy, bca_grads_t* grads, int64_t d_in, int64_t d_out,
                 int64_t p, int64_t tokens, rdfft_dtype_t dtype, rdfft_stream_t stream) {
  if (grads == nullptr) return RDFFT_EINVAL;
  BcaShape sh;
  int st = check_bca(x, c_spectra, gy, d_in, d_out, p, tokens, dtype, true, &sh);
  if (st != RDFFT_OK) return st;
  float* dc = grads->dc;
  void* dx = grads->dx;
  st = check_backward_grads(x, c_spectra, gy, dx, dc, d_in, d_out, p, tokens, sh);
  if (st != RDFFT_OK) return st;
  const float2* tw = nullptr;
  int num_cu = 0;
  st = ensure_device(&tw, &num_cu);
  if (st != RDFFT_OK) return st;
  rdfft::BcaArgs a{x, c_spectra, gy, dx, dc, tokens, sh.q, sh.kb, sh.logp, dtype};
  return rdfft::launch_bca_backward(a, tw, reinterpret_cast<hipStream_t>(stream), num_cu) == hipSuccess
             ? RDFFT_OK
             : RDFFT_ELAUNCH;
}

int bca_forward_batched(int count, const void* const* x, const void* const* c_spectra, void* const* y, int64_t d_in,
                        int64_t d_out, int64_t p, int64_t tokens, rdfft_dtype_t dtype, rdfft_stream_t stream) {
  if (count < 0 || count > kMaxBatchCount) return RDFFT_EINVAL;
  if (count == 0) return RDFFT_OK;
  if (x == nullptr || c_spectra == nullptr || y == nullptr) return RDFFT_EINVAL;
  BcaShape sh;
  std::vector<std::vector<Span>> spans((size_t)count);
  for (int b = 0; b < count; ++b) {
    int st = check_bca(x[b], c_spectra[b], y[b], d_in, d_out, p, tokens, dtype, false, &sh);
    if (st != RDFFT_OK) return st;
    if (tokens > 0) {
      st = check_forward_alias(x[b], y[b], d_in, d_out, p, sh);
      if (st != RDFFT_OK) return st;
    }
    spans[b] = {{x[b], sh.x_bytes, false}, {c_spectra[b], sh.c_bytes, false}, {y[b], sh.y_bytes, true}};
  }
  if (tokens == 0) return RDFFT_OK;
  if (!batch_disjoint(spans)) return RDFFT_EINVAL;
  const float2* tw = nullptr;
  int num_cu = 0;
  int st = ensure_device(&tw, &num_cu);
  if (st != RDFFT_OK) return st;
  const hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  if (rdfft::bca_batch_fused(sh.logp, sh.q, sh.kb, dtype, false)) {
    const rdfft::BcaArgs shape{nullptr, nullptr, nullptr, nullptr, nullptr, tokens, sh.q, sh.kb, sh.logp, dtype};
    for (int b0 = 0; b0 < count; b0 += rdfft::kMaxBatch) {
      rdfft::BcaBatch bt{};
      bt.count = count - b0 < rdfft::kMaxBatch ? count - b0 : rdfft::kMaxBatch;
      for (int i = 0; i < bt.count; ++i) {
        bt.x[i] = x[b0 + i];
        bt.c[i] = c_spectra[b0 + i];
        bt.y[i] = y[b0 + i];
      }
      if (rdfft::launch_bca_forward_batched(shape, bt, tw, s, num_cu) != hipSuccess) return RDFFT_ELAUNCH;
    }
    return RDFFT_OK;
  }
  for (int b = 0; b < count; ++b) {
    const rdfft::BcaArgs a{x[b], c_spectra[b], y[b], nullptr, nullptr, tokens, sh.q, sh.kb, sh.logp, dtype};
    if (rdfft::launch_bca_forward(a, tw, s, num_cu) != hipSuccess) return RDFFT_ELAUNCH;
  }
  return RDFFT_OK;
}

int bca_backward_batched(int count, const void* const* x, const void* const* c_spectra, void* const* gy,
                         const bca_grads_t* grads, int64_t d_in, int64_t d_out, int64_t p, int64_t tokens,
                         rdfft_dtype_t dtype, rdfft_stream_t stream) {
  if (count < 0 || count > kMaxBatchCount) return RDFFT_EINVAL;
  if (count == 0) return RDFFT_OK;
  if (x == nullptr || c_spectra == nullptr || gy == nullptr || grads == nullptr) return RDFFT_EINVAL;
  BcaShape sh;
  bool apart = true;  // every layer's dx apart from its gy
  std::vector<std::vector<Span>> spans((size_t)count);
  for (int b = 0; b < count; ++b) {
    int st = check_bca(x[b], c_spectra[b], gy[b], d_in, d_out, p, tokens, dtype, true, &sh);
    if (st != RDFFT_OK) return st;
    st = check_backward_grads(x[b], c_spectra[b], gy[b], grads[b].dx, grads[b].dc, d_in, d_out, p, tokens, sh);
    if (st != RDFFT_OK) return st;
    apart = apart && grads[b].dx != gy[b];
    spans[b] = {{x[b], sh.x_bytes, false},
                {c_spectra[b], sh.c_bytes, false},
                {gy[b], sh.y_bytes, true},
                {grads[b].dx, tokens > 0 ? sh.x_bytes : 0, true},
                {grads[b].dc, sh.dc_bytes, true}};
  }
  if (!batch_disjoint(spans)) return RDFFT_EINVAL;
  const float2* tw = nullptr;
  int num_cu = 0;
  int st = ensure_device(&tw, &num_cu);
  if (st != RDFFT_OK) return st;
  const hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  if (tokens > 0 && apart && rdfft::bca_batch_fused(sh.logp, sh.q, sh.kb, dtype, true)) {
    const rdfft::BcaArgs shape{nullptr, nullptr, nullptr, nullptr, nullptr, tokens, sh.q, sh.kb, sh.logp, dtype};
    for (int b0 = 0; b0 < count; b0 += rdfft::kMaxBatch) {
      rdfft::BcaBatch bt{};
      bt.count = count - b0 < rdfft::kMaxBatch ? count - b0 : rdfft::kMaxBatch;
      for (int i = 0; i < bt.count; ++i) {
        bt.x[i] = x[b0 + i];
        bt.c[i] = c_spectra[b0 + i];
        bt.y[i] = gy[b0 + i];
        bt.dx[i] = grads[b0 + i].dx;
        bt.dc[i] = grads[b0 + i].dc;
      }
      if (rdfft::launch_bca_backward_batched(shape, bt, tw, s, num_cu) != hipSuccess) return RDFFT_ELAUNCH;
    }
    return RDFFT_OK;
  }
  for (int b = 0; b < count; ++b) {
    const rdfft::BcaArgs a{x[b], c_spectra[b], gy[b], grads[b].dx, grads[b].dc, tokens, sh.q, sh.kb, sh.logp, dtype};
    if (rdfft::launch_bca_backward(a, tw, s, num_cu) != hipSuccess) return RDFFT_ELAUNCH;
  }
  return RDFFT_OK;
}

int rdfft_init(void) {
  const float2* tw = nullptr;
  return ensure_device(&tw, nullptr);
}

int64_t rdfft_table_bytes(void) { return (int64_t)rdfft::kTableEntries * 8; }

const char* rdfft_status_string(int status) {
  switch (status) {
    case RDFFT_OK: return "RDFFT_OK";
    case RDFFT_EINVAL: return "RDFFT_EINVAL: invalid argument";
    case RDFFT_EUNSUPPORTED: return "RDFFT_EUNSUPPORTED: valid but unsupported size";
    case RDFFT_ELAUNCH: return "RDFFT_ELAUNCH: HIP kernel launch failed";
    case RDFFT_EDEVICE: return "RDFFT_EDEVICE: no usable gfx950 device or table upload failed";
    default: return "unknown rdfft status";
  }
}

}  // extern "C"
