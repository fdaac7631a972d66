/*
 * hadacore.h -- C ABI of libhadacore: batched, normalized Walsh-Hadamard
 * transform of fp16/bf16 rows on AMD Instinct MI355X (gfx950).
 *
 * Operation (HadaCore, arXiv 2412.08832, Sec. 2.1-2.2 and Sec. 2.4):
 * for every row i < m of an m x n matrix x of 16-bit floats,
 *
 *     out[i][j] = scale * sum_{k<n} (-1)^popcount(j & k) * in[i][k],  j < n,
 *
 * i.e. each row is multiplied on the right by the Sylvester-ordered
 * Walsh-Hadamard matrix H_n (natural order, +-1 entries), and by `scale`.
 * The normalized transform of the paper is scale = 1/sqrt(n); H_n is never
 * stored.  n is a power of two from 1 to 2^16: the paper's sizes are 2^7 to
 * 2^15 (Sec. 2.3-2.4 and Sec. 3.2 bound them at 2^15); the smaller ones and
 * 2^16 are supported as well (n = 1 is the identity times `scale`), and
 * hadamard_transform_ws goes on to 2^20.  In-place operation
 * (Appendix B) is supported.
 *
 * Numerics: inputs are scaled before any addition -- by `scale`, or by its
 * power-of-two part with the remaining factor (in [1, 2)) applied at the end --
 * so that large bf16 rows cannot overflow fp32 partial sums; all intermediates
 * are fp32 and the result is rounded once to the output dtype with
 * round-to-nearest-even.  Subnormals are preserved.
 * NaN/Inf propagate as IEEE arithmetic dictates.  Results are deterministic:
 * repeated calls, and in-place vs out-of-place calls, give identical bits.
 *
 * Memory: all pointers are DEVICE pointers owned by the caller; the library
 * never allocates, frees or retains them.  Rows are contiguous (element
 * stride 1) and start every `row_stride` elements; elements between n and the
 * row stride are neither read nor written.  Row strides are at most 2^26
 * elements (bytes for quantized codes), which keeps every offset inside a
 * group of rows handled by one wave below 2^32 bytes, and multiples of
 * min(n, 8) elements (codes: min(n, 16) bytes), so that every row starts on a
 * boundary of its access width.
 *
 * Streams: work is enqueued asynchronously on `stream` (a hipStream_t; NULL
 * means the default stream), which must belong to the current device (the
 * architecture check and launch shape use it), and the call returns without
 * synchronizing.
 * Buffers must stay alive until that work completes.  Faults in the enqueued
 * kernel surface at the caller's next synchronization, not here.  A call
 * enqueues kernel launches only (no allocation, memset or synchronization),
 * so it can be captured into a HIP graph once the first call on a device has
 * run outside capture (that call caches the device check); calls on
 * different streams may run concurrently.
 *
 * Kernels: per transform size the library picks one of two front ends for the
 * first stages, both giving results within fp32 rounding of each other: fp32
 * VALU butterflies, or one radix-32 step on the matrix cores (MFMA) applied
 * directly to the 16-bit inputs (n >= 128 only).  The environment variable
 * HADACORE_VARIANT set to "valu" or "mfma" forces one of them for n >= 128
 * (testing and tuning; read on every call); unset keeps the measured per-size
 * choice.
 *
 * Launches: a call is one kernel launch, or two for the two-pass sizes; m so
 * large that a launch would exceed 2^31 work-items (2^33 elements) is split
 * into several launches of consecutive rows on the same stream, with the
 * same result.
 *
 * Output alignment (performance only): an output (or code array) that starts
 * on a 128-byte boundary, with contiguous rows or a row pitch and row size
 * that are multiples of 128 bytes, takes a store path that is 1-3% faster at
 * most sizes.  Any other valid layout gives the same bytes.
 *
 * Errors: arguments are validated synchronously before anything is enqueued;
 * on error nothing is enqueued and a nonzero status is returned.  No call
 * aborts or throws.  The library keeps no state beyond a per-device cache of
 * the architecture check, the compute-unit count and the address of the
 * scratch array of hadamard_transform_ws_noalloc, and is safe to call from
 * several host threads.
 */
#ifndef HADACORE_H
#define HADACORE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define HADACORE_VERSION 10200 /* 1.2.0: hadamard_transform_ws_noalloc */

typedef int32_t hadacore_dtype;
#define HADACORE_FP16 0 /* IEEE binary16 */
#define HADACORE_BF16 1 /* bfloat16 */

typedef int32_t hadacore_status;
#define HADACORE_SUCCESS 0
#define HADACORE_ERROR_INVALID_VALUE 1      /* m < 0, null pointer with m > 0, non-finite scale */
#define HADACORE_ERROR_INVALID_SIZE 2       /* n not a power of two in [1, 65536] (2^20 for _ws) */
#define HADACORE_ERROR_INVALID_DTYPE 3      /* dtype not HADACORE_FP16 / HADACORE_BF16 */
#define HADACORE_ERROR_INVALID_STRIDE 4     /* row stride < n, > 2^26, or not a multiple of min(n, 8) */
#define HADACORE_ERROR_MISALIGNED 5         /* in or out not 16-byte aligned */
#define HADACORE_ERROR_OVERLAP 6            /* in/out overlap without being the same layout */
#define HADACORE_ERROR_LAUNCH 7             /* the HIP runtime rejected the kernel launch */
#define HADACORE_ERROR_UNSUPPORTED_DEVICE 8 /* current device is not gfx950 */
#define HADACORE_ERROR_TOO_LARGE 9          /* m >= 2^31, or m * row stride > 2^40 */
#define HADACORE_ERROR_WORKSPACE 10         /* workspace NULL or below the required size */
#define HADACORE_ERROR_SCRATCH 11           /* hadamard_transform_ws_noalloc: needs more than
                                               HADACORE_NOALLOC_SCRATCH_BYTES of workspace */

/*
 * hadamard_transform -- out = scale * in * H_n for m dense rows of n elements.
 *   in     device pointer to m*n 16-bit values, 16-byte aligned (read only
 *          unless in == out)
 *   out    device pointer to m*n 16-bit values, 16-byte aligned; out == in
 *          selects in-place operation, any other overlap is rejected
 *   m      number of rows, >= 0; m == 0 returns HADACORE_SUCCESS and enqueues
 *          nothing (pointers may then be NULL)
 *   n      transform length, a power of two in [1, 65536]
 *   dtype  HADACORE_FP16 or HADACORE_BF16 (input and output share it)
 *   scale  finite fp32 multiplier; 1/sqrt(n) gives the orthonormal transform
 *   stream hipStream_t to enqueue on (NULL = default stream)
 * Same as hadamard_transform_strided with both row strides equal to n.
 */
hadacore_status hadamard_transform(const void *in, void *out, int64_t m, int64_t n,
                                   hadacore_dtype dtype, float scale, void *stream);

/*
 * hadamard_transform_strided -- as hadamard_transform, with row i of the input
 * at in + i*in_row_stride and row i of the output at out + i*out_row_stride
 * (strides in elements, each >= n, <= 2^26 and a multiple of min(n, 8)).  In-place operation
 * requires in == out and in_row_stride == out_row_stride.
 */
hadacore_status hadamard_transform_strided(const void *in, int64_t in_row_stride, void *out,
                                           int64_t out_row_stride, int64_t m, int64_t n,
                                           hadacore_dtype dtype, float scale, void *stream);

/*
 * hadamard_transform_workspace_size -- bytes of device workspace that
 * hadamard_transform_ws needs for m rows of n elements: 4*m*n (one fp32 value
 * per element) for 2^16 < n <= 2^20, 0 for n <= 2^16.  Returns 0 as well for
 * arguments hadamard_transform_ws rejects; the call reports why.
 */
int64_t hadamard_transform_workspace_size(int64_t m, int64_t n);

/*
 * hadamard_transform_ws -- as hadamard_transform_strided, for n up to 2^20.
 * Sizes above 2^16 (the paper's range ends at 2^15, Sec. 3.2) do not fit one
 * workgroup's registers in fp32, so they run in two passes
 * through a caller-provided fp32 workspace: pass 1 applies `scale` and the
 * stages on index bits 15..log2(n)-1 (between the 2^15-element blocks of a
 * row), pass 2 the stages on bits 0..14 within each block, and rounds once.
 * Every intermediate stays fp32, so the numerics are those of the one-pass
 * sizes; the HBM traffic is 12 bytes per element instead of 4.  For n <= 2^16
 * the call is hadamard_transform_strided and the workspace is not touched.
 *   workspace        device pointer, 16-byte aligned, at least
 *                    hadamard_transform_workspace_size(m, n) bytes, not
 *                    overlapping in or out (NULL allowed for n <= 2^16)
 *   workspace_bytes  its size in bytes
 * The workspace is scratch: its contents on return are unspecified, and two
 * calls in flight at once need two workspaces.  Other arguments, strides,
 * streams and errors as for hadamard_transform_strided, plus
 * HADACORE_ERROR_WORKSPACE.  The quantizing entry points stop at n = 2^16.
 */
hadacore_status hadamard_transform_ws(const void *in, int64_t in_row_stride, void *out,
                                      int64_t out_row_stride, int64_t m, int64_t n,
                                      hadacore_dtype dtype, float scale, void *workspace,
                                      int64_t workspace_bytes, void *stream);

/*
 * hadamard_transform_ws_noalloc -- hadamard_transform_ws for callers that
 * cannot allocate device memory (code under HIP graph capture, tight serving
 * loops, harnesses that forbid hipMalloc): the same kernels and results, with
 * the fp32 workspace taken from a fixed array inside the library instead of
 * an argument.  The call itself allocates nothing (no hipMalloc, hipFree or
 * allocating library routine).
 *   The array is HADACORE_NOALLOC_SCRATCH_BYTES (32 MiB) of device memory per
 *   GPU, held from the library's first use on that GPU until the process
 *   ends; for n > 2^16 the call needs hadamard_transform_workspace_size(m, n)
 *   <= HADACORE_NOALLOC_SCRATCH_BYTES (m * n <= 2^23 elements: e.g. 64 rows of
 *   2^17, 8 rows of 2^20) and returns HADACORE_ERROR_SCRATCH beyond that,
 *   enqueuing nothing.  For n <= 2^16 it is hadamard_transform_strided.
 *   Every call on one GPU uses that GPU's one array: calls that can overlap
 *   in time on the same GPU (different streams, host threads) race and give
 *   undefined results; calls in one stream's order are safe.  Nothing in the
 *   array needs to start at zero (pass 1 writes all of it before pass 2
 *   reads).  The first call on a device looks up that device's address of the
 *   array (HADACORE_ERROR_LAUNCH if the runtime cannot give it); run that call
 *   outside graph capture.
 * Other arguments, strides, streams and errors as for hadamard_transform_ws.
 */
#define HADACORE_NOALLOC_SCRATCH_BYTES (32LL << 20)
hadacore_status hadamard_transform_ws_noalloc(const void *in, int64_t in_row_stride, void *out,
                                              int64_t out_row_stride, int64_t m, int64_t n,
                                              hadacore_dtype dtype, float scale, void *stream);

/*
 * hadamard_transform_fp8 -- the transform fused with per-row quantization to
 * OCP FP8 e4m3 (the fused Hadamard transform + quantization that the paper
 * names as future work, Sec. 5; rotations precede FP8 attention, Sec. 4.2).
 * For every row i, with y = scale * in[i] * H_n computed as above:
 *     amax_i          = max_j |y_j|   (NaN ignored unless the row is all NaN)
 *     out_scales[i]   = amax_i / 448  (fp32, correctly rounded)
 *     out_codes[i][j] = e4m3 round-to-nearest-even of y_j * (448 / amax_i)
 *                       (448/amax_i taken as 0 where it is not finite: a zero
 *                       or NaN row, or amax_i < 448 * 2^-128, whose codes are
 *                       then +-0)
 * so that y_j ~ decode_e4m3(out_codes[i][j]) * out_scales[i].  e4m3: 1 sign,
 * 4 exponent (bias 7) and 3 fraction bits, largest finite 448, 0x7f NaN.
 *   in              device pointer, m rows of n 16-bit values at in_row_stride
 *                   elements (>= n, <= 2^26, multiple of min(n, 8)), 16-byte
 *                   aligned
 *   out_codes       device pointer, m rows of n bytes at out_row_stride bytes
 *                   (>= n, <= 2^26, multiple of min(n, 16)), 16-byte aligned
 *   out_scales      device pointer to m floats, 4-byte aligned
 * The three ranges must not overlap (OVERLAP otherwise).  Other arguments,
 * streams, ownership and errors as for hadamard_transform.
 */
hadacore_status hadamard_transform_fp8(const void *in, int64_t in_row_stride, void *out_codes,
                                       int64_t out_row_stride, float *out_scales, int64_t m,
                                       int64_t n, hadacore_dtype dtype, float scale, void *stream);

/*
 * hadamard_transform_int8 -- the transform fused with symmetric per-row INT8
 * quantization, the integer counterpart of hadamard_transform_fp8 (rotations
 * spread outliers so that one scale per row loses less, Sec. 1).  For every
 * row i, with y = scale * in[i] * H_n computed as above and amax_i as for FP8:
 *     out_scales[i]   = amax_i / 127  (fp32, correctly rounded)
 *     out_codes[i][j] = round-half-to-even of y_j * (127 / amax_i), an int8 in
 *                       [-127, 127] (the product rounded to fp32 first)
 * so that y_j ~ out_codes[i][j] * out_scales[i].  A row whose amax is 0, Inf or
 * NaN, or so small that 127 / amax_i overflows fp32 (amax_i < 127 * 2^-128),
 * gets all-zero codes; its scale is still amax_i / 127.  Arguments, layout,
 * alignment, overlap rules, streams and errors as for hadamard_transform_fp8.
 */
hadacore_status hadamard_transform_int8(const void *in, int64_t in_row_stride, void *out_codes,
                                        int64_t out_row_stride, float *out_scales, int64_t m,
                                        int64_t n, hadacore_dtype dtype, float scale, void *stream);

/*
 * hadacore_stream_copy -- copies `bytes` bytes from device pointer `src` to
 * device pointer `dst` with 16-byte vector loads and stores on `stream`.  Both
 * pointers 16-byte aligned, bytes a multiple of 16, ranges disjoint.  It moves
 * the same HBM bytes per element as the transform and serves as its measured
 * bandwidth ceiling (the paper's Appendix B compares against a device copy).
 */
hadacore_status hadacore_stream_copy(const void *src, void *dst, int64_t bytes, void *stream);

/* Static, human-readable name of a status code (never NULL). */
const char *hadacore_status_string(hadacore_status status);

/* HADACORE_VERSION of the loaded library. */
int32_t hadacore_version(void);

#ifdef __cplusplus
}
#endif

#endif /* HADACORE_H */
