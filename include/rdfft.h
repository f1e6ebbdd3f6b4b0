/*
 * rdfft.h -- C ABI of the MI355X (gfx950) in-place real-domain FFT library.
 *
 * Implements the method of "Memory-Efficient Training with In-Place FFT
 * Implementation" (arXiv 2511.01385): a real FFT whose spectrum is written back
 * into the input's own n real slots (rdFFT), its inverse, and the
 * block-circulant linear layer (forward and backward) computed with them.
 *
 * Conventions shared by every entry point
 * --------------------------------------
 * - All pointers are DEVICE pointers on the current HIP device, 16-byte
 *   aligned.  The caller owns every buffer; the library keeps no pointer after
 *   the enqueued work completes.
 * - Every call validates its arguments on the host before any HIP call; on
 *   failure it returns a negative rdfft_status_t and enqueues nothing.
 * - Work is enqueued on `stream` (NULL = the default stream) and the call
 *   returns without synchronising.  Faults during execution surface at the
 *   caller's next synchronisation.
 * - No call allocates device memory.  The only device memory the library owns
 *   is a static table of twiddle factors (rdfft_table_bytes()), copied to each
 *   device the first time that device is used (or by rdfft_init()); that first
 *   use performs a synchronous copy and must not happen under stream capture.
 * - dtype selects the storage type of the transformed data; arithmetic is
 *   float32 throughout, bf16 and f16 values are widened exactly and rounded to
 *   nearest even on store (an f16 result beyond 65504 becomes an infinity).
 *
 * Packed spectrum layout ("pairs"), for a row of even length n:
 *   slot 0 = Y_0 (DC, real), slot 1 = Y_{n/2} (Nyquist, real),
 *   slots 2k, 2k+1 = Re Y_k, Im Y_k for 1 <= k < n/2,
 * where Y_k = sum_m x_m exp(-2 pi i k m / n)  (Sec. 3.1, Eq. (1), forward,
 * unnormalised).  The other half of the spectrum is conj-symmetric
 * (Sec. 3.1, Theorem 1) and DC/Nyquist are real (Sec. 4.1, "Squeeze N+2 into
 * N"), so these n reals hold the whole spectrum.
 */
#ifndef RDFFT_H
#define RDFFT_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#if defined(__GNUC__)
#define RDFFT_API __attribute__((visibility("default")))
#else
#define RDFFT_API
#endif

/* Same type as hipStream_t. */
struct ihipStream_t;
typedef struct ihipStream_t *rdfft_stream_t;

typedef enum {
  RDFFT_F32 = 0,  /* IEEE float32 storage */
  RDFFT_BF16 = 1, /* bfloat16 storage */
  RDFFT_F16 = 2   /* IEEE float16 storage */
} rdfft_dtype_t;

typedef enum {
  RDFFT_OK = 0,
  RDFFT_EINVAL = -1,       /* invalid argument (null/misaligned pointer, bad size, overlap) */
  RDFFT_EUNSUPPORTED = -2, /* valid but not implemented (n > 65536, n/2 with a prime factor
                              above 5 or beyond 16384 when not a power of two, p > 65536,
                              and the long-block limits of bca_forward / bca_backward) */
  RDFFT_ELAUNCH = -3,      /* HIP reported an error when enqueuing */
  RDFFT_EDEVICE = -4       /* no usable gfx950 device, or the twiddle table upload failed */
} rdfft_status_t;

/*
 * rdfft_forward -- in-place real FFT of `rows` rows (Sec. 4.1, rdFFT algorithm;
 * Sec. 3.1 Eq. (1), forward).
 *   buf   rows x n elements of `dtype`, row-major, row stride n.  On entry the
 *         real samples x_0..x_{n-1} of each row; on return the packed spectrum
 *         of that row in the layout above.
 *   rows  >= 0; rows == 0 is a no-op (buf may then be NULL).
 *   n     even, 2 <= n: a power of two up to 65536, or n = 2N with N = 2^a 3^b 5^c
 *         up to 16384 (mixed-radix rows: one workgroup per row, the row in LDS,
 *         twiddles from the hardware sine and cosine).  Odd n -> RDFFT_EINVAL (no Nyquist bin,
 *         Theorem 1); any other even n -> RDFFT_EUNSUPPORTED.
 * No memory beyond buf is read or written (apart from the twiddle table).
 */
RDFFT_API int rdfft_forward(void *buf, int64_t rows, int64_t n, rdfft_dtype_t dtype, rdfft_stream_t stream);

/*
 * rdfft_inverse -- in-place inverse of rdfft_forward (Sec. 4.2; Sec. 3.1
 * Eq. (1), inverse, with the 1/n normalisation of Sec. 3.2):
 *   x_m = (1/n) sum_{k=0}^{n-1} Y_k exp(+2 pi i k m / n),  Y_{n-k} = conj(Y_k),
 * with the imaginary parts of Y_0 and Y_{n/2} taken as zero.  Any n reals are
 * a valid packed spectrum.  Arguments and errors as rdfft_forward.
 */
RDFFT_API int rdfft_inverse(void *buf, int64_t rows, int64_t n, rdfft_dtype_t dtype, rdfft_stream_t stream);

/*
 * rdfft_pairs_to_halfcomplex / rdfft_halfcomplex_to_pairs -- in-place change of
 * the packed layout of `rows` spectra between the pairs layout above and the
 * paper's halfcomplex layout (Sec. 4.1, "Memory Layout"):
 *   halfcomplex: slot k = Re Y_k for 0 <= k <= n/2, slot n-k = Im Y_k for
 *                1 <= k < n/2
 * (so pair slot k, i.e. elements 2k and 2k+1, maps to elements k and n-k, and
 * pair slot 0 to elements 0 and n/2).  Values are moved bit for bit; NaN
 * payloads included.  rdfft_inverse expects the pairs layout, so a spectrum
 * converted to halfcomplex must be converted back before it is inverted (or
 * inverted with rdfft_inverse_halfcomplex).
 * Arguments and errors as rdfft_forward.
 */
RDFFT_API int rdfft_pairs_to_halfcomplex(void *buf, int64_t rows, int64_t n, rdfft_dtype_t dtype, rdfft_stream_t stream);
RDFFT_API int rdfft_halfcomplex_to_pairs(void *buf, int64_t rows, int64_t n, rdfft_dtype_t dtype, rdfft_stream_t stream);

/*
 * rdfft_forward_halfcomplex / rdfft_inverse_halfcomplex -- the in-place transforms
 * with the spectrum in the halfcomplex layout above (Sec. 4.1, Memory Layout) instead
 * of pairs: the forward leaves Re Y_k at element k and Im Y_k at element n-k, the
 * inverse reads them from there.  The results equal rdfft_forward followed by
 * rdfft_pairs_to_halfcomplex (and rdfft_halfcomplex_to_pairs followed by
 * rdfft_inverse) bit for bit, in one pass over the data instead of two.  Arguments
 * and errors as rdfft_forward.
 */
RDFFT_API int rdfft_forward_halfcomplex(void *buf, int64_t rows, int64_t n, rdfft_dtype_t dtype, rdfft_stream_t stream);
RDFFT_API int rdfft_inverse_halfcomplex(void *buf, int64_t rows, int64_t n, rdfft_dtype_t dtype, rdfft_stream_t stream);

/* Gradient outputs of bca_backward. */
typedef struct {
  void *dx;  /* [tokens][d_in] in dtype: dL/dx */
  float *dc; /* [q][kb][p] float32: dL/dc, time-domain first columns, OVERWRITTEN (not accumulated) */
} bca_grads_t;

/*
 * bca_forward -- block-circulant layer y = W x per token (Sec. 3.3; Eq. (4)
 * per block: y_i = IFFT( sum_j FFT(c_ij) . FFT(x_j) )).
 *   W is d_out x d_in, tiled into q x kb circulant blocks of size p
 *   (q = d_out/p, kb = d_in/p); block (i, j) is the circulant matrix whose
 *   first column is c_ij, C[m][r] = c_ij[(m - r) mod p], and maps input segment
 *   j of a token to output segment i.
 *   x          [tokens][d_in] in dtype, read only.
 *   c_spectra  [q][kb][p] in dtype, read only: row (i, j) is the packed
 *              spectrum (rdfft_forward of c_ij).
 *   y          [tokens][d_out] in dtype, written.  y == x is allowed when
 *              d_in == d_out (a truly in-place layer, Sec. 5.1.1); any other
 *              overlap with x or c_spectra -> RDFFT_EINVAL.
 *   grads      reserved, must be NULL.
 *   dtype      RDFFT_F32, RDFFT_BF16 or RDFFT_F16: the storage of x, c_spectra and y
 *              (float32 arithmetic; 16-bit stores round to nearest even).
 *   p          power of two, 2 <= p <= 65536 (larger -> RDFFT_EUNSUPPORTED);
 *              must divide d_in and d_out (Table 1 marks such shapes N/A) -> else RDFFT_EINVAL.
 *   tokens     >= 0; 0 is a no-op (x and y may then be NULL).
 * Blocks beyond 8192 (p = 16384, 32768, 65536) run as passes over HBM with q * kb <= 65535
 * (else RDFFT_EUNSUPPORTED).  With kb <= q and kb <= 8 they stage the input spectra in y;
 * other shapes add each input block's contribution into y's spectra, one pass per block.
 * Either way the intermediate spectra are stored in dtype (for 16-bit storage, one more
 * rounding of each staged spectrum, or of each of the kb partial sums).  In place
 * (y == x) they need q = kb <= 8 (else RDFFT_EUNSUPPORTED).
 */
RDFFT_API int bca_forward(const void *x, const void *c_spectra, void *y, bca_grads_t *grads, int64_t d_in,
                int64_t d_out, int64_t p, int64_t tokens, rdfft_dtype_t dtype, rdfft_stream_t stream);

/*
 * bca_backward -- gradients of the block-circulant layer (Sec. 3.3, Eq. (5)):
 *   dx_j  = IFFT( sum_i conj(FFT(c_ij)) . FFT(g_i) )          per token,
 *   dc_ij = IFFT( sum_t conj(FFT(x_{t,j})) . FFT(g_{t,i}) )   summed over tokens,
 * with g = dL/dy.
 *   x          [tokens][d_in] in dtype, read only.
 *   c_spectra  [q][kb][p] in dtype, read only (as bca_forward).
 *   gy         [tokens][d_out] in dtype: the upstream gradient.  Its contents
 *              are unspecified on return (the layer may use it as work space,
 *              Sec. 5.1.1 "overwriting the grad_output").
 *   grads->dx  [tokens][d_in] in dtype, written; may equal gy when d_in == d_out.
 *              Blocks beyond 8192 stage the input spectra in dx while gy holds the
 *              upstream ones; with dx == gy (q = kb <= 8 there, else RDFFT_EUNSUPPORTED)
 *              each token's input spectra go straight into float32 atomic sums of dc.
 *   grads->dc  [q][kb][p] float32, written (overwritten, not accumulated).
 *              Summed with float32 atomics, so the last bits may vary run to run.
 *   Other arguments as bca_forward.  tokens == 0 writes dc = 0.
 * Any other overlap between the buffers -> RDFFT_EINVAL.
 */
RDFFT_API int bca_backward(const void *x, const void *c_spectra, void *gy, bca_grads_t *grads, int64_t d_in,
                 int64_t d_out, int64_t p, int64_t tokens, rdfft_dtype_t dtype, rdfft_stream_t stream);

/*
 * bca_forward_batched / bca_backward_batched -- `count` independent layers of one shape
 * (the same d_in, d_out, p, tokens and dtype, each with its own tensors), such as the query
 * and value adapters of every layer of an encoder (Sec. 5.1.2), in one call.  Square layers
 * of 128 <= p <= 512 with q = kb <= 4 (the ones whose transforms fit a wavefront) run the
 * layers side by side in the same launches, which fills the chip where one layer alone
 * cannot; the backward does so when every dx is apart from its gy.  Other batches run
 * their layers one after another.  Results equal those of bca_forward / bca_backward on
 * each layer (dc up to the order of its float32 sums).
 *   count      0 <= count <= 1024 (0: no-op); else RDFFT_EINVAL.
 *   x, c_spectra, y / gy
 *              host arrays of `count` device pointers, entry b as the argument of the
 *              single-layer call for layer b.
 *   grads      host array of `count` bca_grads_t (backward only).
 * Within a layer the aliasing rules of the single-layer calls hold.  Across layers, buffers
 * that are only read may be shared (one x for several layers), but nothing a layer writes
 * (y; gy, dx, dc) may overlap any buffer of another layer -> RDFFT_EINVAL.  All layers are
 * checked before anything is enqueued.
 */
RDFFT_API int bca_forward_batched(int count, const void *const *x, const void *const *c_spectra, void *const *y,
                                  int64_t d_in, int64_t d_out, int64_t p, int64_t tokens, rdfft_dtype_t dtype,
                                  rdfft_stream_t stream);
RDFFT_API int bca_backward_batched(int count, const void *const *x, const void *const *c_spectra, void *const *gy,
                                   const bca_grads_t *grads, int64_t d_in, int64_t d_out, int64_t p, int64_t tokens,
                                   rdfft_dtype_t dtype, rdfft_stream_t stream);

/* Uploads the twiddle table to the current device (synchronously) if not done yet.
 * Optional: every entry point does it on first use.  Returns RDFFT_OK or RDFFT_EDEVICE. */
RDFFT_API int rdfft_init(void);

/* Bytes of the static twiddle table held on each device the library has used. */
RDFFT_API int64_t rdfft_table_bytes(void);

/* Human-readable name of a status code (static string). */
RDFFT_API const char *rdfft_status_string(int status);

#ifdef __cplusplus
}
#endif

#endif /* RDFFT_H */
