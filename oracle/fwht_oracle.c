/*
 * fwht_oracle.c -- plain, slow, obviously-correct fp64 CPU reference for the
 * batched normalized Walsh-Hadamard transform (HadaCore, arXiv 2412.08832).
 *
 * TEST INFRASTRUCTURE ONLY.  This file is the oracle that GPU results are
 * judged against.  Only the test suite, the smoke check and the benchmark's
 * CPU-baseline leg may load it.  It shares no code, header, table or helper
 * with the HIP library: it has its own 16-bit decoders and its own loops.
 *
 * What it computes (per row i of an m x n matrix x, n a power of two):
 *     y[i][j] = s * sum_k (-1)^popcount(j & k) * x[i][k]
 * i.e. every row multiplied by the Sylvester-ordered Walsh-Hadamard matrix
 * H_n (paper Sec. 2.1: +-1 entries, orthogonal, power-of-two sizes built by
 * Sylvester's recursion H_2k = [[H_k, H_k], [H_k, -H_k]]), scaled by s.
 * The caller passes s; the paper's normalization (Sec. 2.2, the per-stage
 * division by sqrt 2 in its FWHT listing) is the special case s = 1/sqrt(n).
 *
 * Also: oracle_fwht_fp8 and oracle_fwht_int8, the transform followed by
 * per-row FP8 (e4m3) or INT8 quantization (see their comments), with their own
 * encoders and decoder.
 *
 * Two independent routes are provided for the transform itself:
 *   oracle_fwht_f64        -- the iterative radix-2 FWHT of Sec. 2.2: stage
 *                             sizes h = 1, 2, 4, ..., n/2; within a stage,
 *                             blocks of 2h, pairs (j, j+h) replaced by
 *                             (a+b, a-b); natural (Sylvester) order, in place
 *                             on a double copy of the row; s applied once at
 *                             the end.
 *   oracle_fwht_direct_f64 -- the plain definition above, O(n) per requested
 *                             output, for sampled checks at any size.
 *
 * Readings of the paper taken here (all listed in the design notes):
 *   - order: natural/Sylvester, H[j][k] = (-1)^popcount(j&k) (Sec. 2.1-2.2);
 *   - direction: the transform acts along each row, x * H (Sec. 2.4);
 *   - normalization: one multiplication by the caller's scale at the end,
 *     equal in exact arithmetic to the per-stage 1/sqrt 2 of Sec. 2.2;
 *   - arithmetic: fp64 throughout; inputs decoded exactly.
 *
 * Exactness: every fp16 value is an integer multiple of 2^-24 and every
 * partial sum of a row with sum|x| < 2^29 stays an integer multiple of 2^-24
 * below 2^53, so the unscaled fp16 transform is exact in fp64; only the final
 * multiplication by s rounds.
 *
 * Build: plain C11, -O2, no SIMD intrinsics, no fast-math.
 */
#include <math.h>
#include <pthread.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define ORACLE_FP16 0
#define ORACLE_BF16 1

/* IEEE binary16: 1 sign bit, 5 exponent bits (bias 15), 10 fraction bits. */
double oracle_decode_fp16(uint16_t h)
{
    int sign = (h >> 15) & 1;
    int expo = (h >> 10) & 0x1f;
    int frac = h & 0x3ff;
    double v;
    if (expo == 0) {
        v = ldexp((double)frac, -24);              /* zero or subnormal */
    } else if (expo == 31) {
        v = frac ? NAN : INFINITY;
    } else {
        v = ldexp((double)(1024 + frac), expo - 25); /* (1.f) * 2^(e-15) */
    }
    return sign ? -v : v;
}

/* bfloat16: 1 sign bit, 8 exponent bits (bias 127), 7 fraction bits. */
double oracle_decode_bf16(uint16_t b)
{
    int sign = (b >> 15) & 1;
    int expo = (b >> 7) & 0xff;
    int frac = b & 0x7f;
    double v;
    if (expo == 0) {
        v = ldexp((double)frac, -133);             /* zero or subnormal */
    } else if (expo == 255) {
        v = frac ? NAN : INFINITY;
    } else {
        v = ldexp((double)(128 + frac), expo - 134); /* (1.f) * 2^(e-127) */
    }
    return sign ? -v : v;
}

static double decode(uint16_t bits, int dtype)
{
    return dtype == ORACLE_BF16 ? oracle_decode_bf16(bits) : oracle_decode_fp16(bits);
}

static int is_pow2(int64_t n) { return n > 0 && (n & (n - 1)) == 0; }

/*
 * Unscaled in-place FWHT of a double vector of length n (power of two),
 * following the iterative algorithm of Sec. 2.2: the outer loop doubles the
 * transform size, the middle loop walks the blocks of 2h elements, the inner
 * loop forms the sum and difference of each pair (j, j+h).
 */
void oracle_fwht_vec_f64(double *v, int64_t n)
{
    for (int64_t h = 1; h < n; h *= 2) {
        for (int64_t i = 0; i < n; i += 2 * h) {
            for (int64_t j = i; j < i + h; ++j) {
                double a = v[j];
                double b = v[j + h];
                v[j] = a + b;
                v[j + h] = a - b;
            }
        }
    }
}

/* Decode rows of a row-strided 16-bit matrix into a dense m x n double array. */
int oracle_decode_rows(const uint16_t *in, int64_t in_stride, int64_t m, int64_t n,
                       int dtype, double *out)
{
    if (m < 0 || n < 0 || in_stride < n) return 1;
    for (int64_t i = 0; i < m; ++i)
        for (int64_t k = 0; k < n; ++k)
            out[i * n + k] = decode(in[i * in_stride + k], dtype);
    return 0;
}

typedef struct {
    const uint16_t *in;
    int64_t in_stride, n, row0, row1;
    int dtype;
    double scale;
    double *out;
} fwht_job;

static void *fwht_rows_worker(void *arg)
{
    const fwht_job *jb = (const fwht_job *)arg;
    for (int64_t i = jb->row0; i < jb->row1; ++i) {
        double *row = jb->out + i * jb->n;
        const uint16_t *src = jb->in + i * jb->in_stride;
        for (int64_t k = 0; k < jb->n; ++k) row[k] = decode(src[k], jb->dtype);
        oracle_fwht_vec_f64(row, jb->n);
        for (int64_t k = 0; k < jb->n; ++k) row[k] *= jb->scale;
    }
    return NULL;
}

/*
 * y = s * x * H_n for every row, via the iterative FWHT.  `in` is row-strided
 * (in_stride >= n elements); `out` is a dense m x n double array.  Rows are
 * split into contiguous blocks over `nthreads` POSIX threads (<= 1: serial).
 * Returns 0 on success, 1 on bad arguments.
 */
int oracle_fwht_f64(const uint16_t *in, int64_t in_stride, int64_t m, int64_t n,
                    int dtype, double scale, double *out, int nthreads)
{
    if (m < 0 || !is_pow2(n) || in_stride < n) return 1;
    if (dtype != ORACLE_FP16 && dtype != ORACLE_BF16) return 1;
    if (m == 0) return 0;
    if (nthreads < 1) nthreads = 1;
    if (nthreads > m) nthreads = (int)m;
    fwht_job *jobs = (fwht_job *)calloc((size_t)nthreads, sizeof(fwht_job));
    pthread_t *tids = (pthread_t *)calloc((size_t)nthreads, sizeof(pthread_t));
    if (!jobs || !tids) { free(jobs); free(tids); return 1; }
    for (int t = 0; t < nthreads; ++t) {
        jobs[t].in = in;
        jobs[t].in_stride = in_stride;
        jobs[t].n = n;
        jobs[t].row0 = m * t / nthreads;
        jobs[t].row1 = m * (t + 1) / nthreads;
        jobs[t].dtype = dtype;
        jobs[t].scale = scale;
        jobs[t].out = out;
    }
    int spawned = 0;
    for (int t = 1; t < nthreads; ++t) {
        if (pthread_create(&tids[t], NULL, fwht_rows_worker, &jobs[t]) != 0) break;
        spawned = t;
    }
    fwht_rows_worker(&jobs[0]);
    for (int t = 1; t <= spawned; ++t) pthread_join(tids[t], NULL);
    for (int t = spawned + 1; t < nthreads; ++t) fwht_rows_worker(&jobs[t]);
    free(jobs);
    free(tids);
    return 0;
}

static int popcount64(uint64_t v)
{
    int c = 0;
    while (v) { v &= v - 1; ++c; }
    return c;
}

/*
 * The plain definition, one output at a time: for each requested (row, col)
 * pair, out[t] = s * sum_k (-1)^popcount(col & k) * x[row][k], summed in
 * index order k = 0..n-1.  Used for sampled checks where a full transform of
 * the whole matrix is not wanted.  Returns 0 on success, 1 on bad arguments.
 */
int oracle_fwht_direct_f64(const uint16_t *in, int64_t in_stride, int64_t n, int dtype,
                           double scale, const int64_t *rows, const int64_t *cols,
                           int64_t count, double *out)
{
    if (!is_pow2(n) || in_stride < n || count < 0) return 1;
    if (dtype != ORACLE_FP16 && dtype != ORACLE_BF16) return 1;
    for (int64_t t = 0; t < count; ++t) {
        if (cols[t] < 0 || cols[t] >= n || rows[t] < 0) return 1;
        const uint16_t *src = in + rows[t] * in_stride;
        double acc = 0.0;
        for (int64_t k = 0; k < n; ++k) {
            double x = decode(src[k], dtype);
            if (popcount64((uint64_t)(cols[t] & k)) & 1)
                acc -= x;
            else
                acc += x;
        }
        out[t] = acc * scale;
    }
    return 0;
}

/* ---- fused transform + FP8 quantization -------------------------------------
 *
 * The paper names a fused Hadamard transform and quantization as future work
 * (Sec. 5; the rotation exists to spread outliers before low-precision
 * attention, Sec. 1 and Sec. 4.2).  Reading taken here: each transformed row
 * y_i is quantized to OCP FP8 e4m3 (finite max 448, no infinities) with one
 * fp32 scale per row,
 *     amax_i = max_j |y_ij|   (NaN entries ignored unless all are NaN)
 *     s_i    = amax_i / 448
 *     q_ij   = e4m3_rne(y_ij * inv_i),  inv_i = 448 / amax_i if that is finite, else 0
 * so that y_ij ~ decode(q_ij) * s_i.  inv_i = 0 covers a zero row, a NaN row
 * and a row so small (amax_i < 448 * 2^-128) that the multiplier overflows
 * fp32: its codes are all zero, which is within amax_i of every element.  The quantization decision is taken in
 * fp32, as the GPU kernel takes it: y is the fp64 transform rounded once to
 * fp32, and s, inv and the product are fp32 operations.
 */

/* e4m3 (OCP "fn" variant): 1 sign, 4 exponent bits (bias 7), 3 fraction bits;
 * exponent field 15 with fraction 7 is NaN; there is no infinity. */
double oracle_decode_e4m3(uint8_t q)
{
    int sign = (q >> 7) & 1;
    int expo = (q >> 3) & 0xf;
    int frac = q & 0x7;
    double v;
    if (expo == 15 && frac == 7) return NAN;
    if (expo == 0)
        v = ldexp((double)frac, -9);               /* subnormal: frac * 2^-9 */
    else
        v = ldexp((double)(8 + frac), expo - 10);  /* (1.f) * 2^(e-7) */
    return sign ? -v : v;
}

/* Round-to-nearest-even of a float to e4m3.  464 is the tie between 448 and
 * the missing 480 and rounds to the even 448; larger magnitudes and NaN give
 * NaN (0x7f with the sign). */
uint8_t oracle_encode_e4m3(float x)
{
    uint8_t sign = signbit(x) ? 0x80 : 0x00;
    double a = fabs((double)x);
    if (isnan(x) || a > 464.0) return (uint8_t)(sign | 0x7f);
    /* candidates are k * 2^(e-3) in the binade [2^e, 2^(e+1)), e >= -6;
     * below 2^-6 the spacing is 2^-9 (subnormals) */
    int e;
    double spacing;
    if (a < ldexp(1.0, -6)) {
        spacing = ldexp(1.0, -9);
    } else {
        frexp(a, &e);          /* a = f * 2^e, f in [0.5, 1) */
        spacing = ldexp(1.0, e - 1 - 3);
    }
    double k = a / spacing;            /* exact: spacing is a power of two */
    double kf = floor(k);
    double r = k - kf;
    if (r > 0.5 || (r == 0.5 && fmod(kf, 2.0) != 0.0)) kf += 1.0;
    double v = kf * spacing;           /* rounded magnitude, <= 448 */
    /* encode v */
    if (v == 0.0) return sign;
    if (v < ldexp(1.0, -6)) return (uint8_t)(sign | (uint8_t)(v / ldexp(1.0, -9)));
    frexp(v, &e);                      /* v = f * 2^e, 2^(e-1) <= v < 2^e */
    int biased = (e - 1) + 7;
    int frac = (int)(v / ldexp(1.0, e - 1 - 3)) - 8;
    return (uint8_t)(sign | (biased << 3) | frac);
}

/* fp32 maximum that ignores NaN unless both operands are NaN. */
static float max_ignoring_nan(float a, float b)
{
    if (isnan(a)) return b;
    if (isnan(b)) return a;
    return a > b ? a : b;
}

/* The largest |y_k| of a row of n fp32 values (NaN ignored unless all are NaN). */
static float row_amax(const float *y, int64_t n)
{
    float amax = NAN;
    for (int64_t k = 0; k < n; ++k) amax = max_ignoring_nan(amax, fabsf(y[k]));
    return amax;
}

/* FP8 quantization of one row of n fp32 values: n codes and one scale. */
static void quantize_row_fp8(const float *y, int64_t n, uint8_t *codes, float *scale)
{
    const float amax = row_amax(y, n);
    const float s = amax / 448.0f;
    const float q = 448.0f / amax;
    const float inv = isfinite(q) ? q : 0.0f;
    *scale = s;
    for (int64_t k = 0; k < n; ++k) codes[k] = oracle_encode_e4m3(y[k] * inv);
}

/* Decodes row i, transforms it in fp64 and rounds y = row * scale once to fp32. */
static void transform_row_fp32(const uint16_t *src, int64_t n, int dtype, double scale,
                               double *row, float *y)
{
    for (int64_t k = 0; k < n; ++k) row[k] = decode(src[k], dtype);
    oracle_fwht_vec_f64(row, n);
    for (int64_t k = 0; k < n; ++k) y[k] = (float)(row[k] * scale);
}

/*
 * Fused transform + quantization of m rows: codes (m x n bytes, row stride
 * out_stride) and scales (m floats).  Returns 0 on success, 1 on bad
 * arguments.
 */
int oracle_fwht_fp8(const uint16_t *in, int64_t in_stride, int64_t m, int64_t n, int dtype,
                    double scale, uint8_t *codes, int64_t out_stride, float *scales)
{
    if (m < 0 || !is_pow2(n) || in_stride < n || out_stride < n) return 1;
    if (dtype != ORACLE_FP16 && dtype != ORACLE_BF16) return 1;
    double *row = (double *)malloc((size_t)n * sizeof(double));
    float *y = (float *)malloc((size_t)n * sizeof(float));
    if (!row || !y) { free(row); free(y); return 1; }
    for (int64_t i = 0; i < m; ++i) {
        transform_row_fp32(in + i * in_stride, n, dtype, scale, row, y);
        quantize_row_fp8(y, n, codes + i * out_stride, &scales[i]);
    }
    free(row);
    free(y);
    return 0;
}

/*
 * The same quantization without the transform: m rows of n fp32 values
 * (dense) to codes (m x n) and scales (m).  The baseline of the
 * rotation-versus-quantization comparison.  Returns 0, or 1 on bad arguments.
 */
int oracle_quantize_fp8(const float *y, int64_t m, int64_t n, uint8_t *codes, float *scales)
{
    if (m < 0 || n < 1) return 1;
    for (int64_t i = 0; i < m; ++i) quantize_row_fp8(y + i * n, n, codes + i * n, &scales[i]);
    return 0;
}

/* ---- fused transform + INT8 quantization ------------------------------------
 *
 * The symmetric per-row INT8 counterpart of the FP8 path: the integer format
 * that rotation-based quantization schemes target (the rotation spreads
 * outliers so that one scale per row loses less, Sec. 1).  With amax_i as for
 * FP8,
 *     s_i  = amax_i / 127
 *     q_ij = round_half_even(y_ij * inv_i),  inv_i = 127 / amax_i,
 * an integer in [-127, 127] (|y_ij * inv_i| <= 127 up to one fp32 rounding),
 * so that y_ij ~ q_ij * s_i.  A row whose amax is 0, +Inf or NaN gets all-zero
 * codes (INT8 has no NaN, and 127/Inf would turn every y * inv into 0 or NaN),
 * and so does a row so small (amax_i < 127 * 2^-128) that 127 / amax_i
 * overflows fp32: zero is within amax_i of every element.
 * As for FP8 the decision is taken in fp32: y is the fp64 transform rounded
 * once to fp32, and s, inv and the product are fp32 operations.
 */

/* Round-half-to-even of v to an integer, saturated to [-127, 127]; NaN -> 0. */
int8_t oracle_encode_int8(float v)
{
    if (isnan(v)) return 0;
    double f = floor((double)v);
    const double r = (double)v - f;
    if (r > 0.5 || (r == 0.5 && fmod(f, 2.0) != 0.0)) f += 1.0;
    if (f > 127.0) f = 127.0;
    if (f < -127.0) f = -127.0;
    return (int8_t)f;
}

/* INT8 quantization of one row of n fp32 values: n codes and one scale. */
static void quantize_row_int8(const float *y, int64_t n, int8_t *codes, float *scale)
{
    const float amax = row_amax(y, n);
    *scale = amax / 127.0f;
    const float q = 127.0f / amax;
    const int usable = isfinite(amax) && isfinite(q);
    const float inv = usable ? q : 0.0f;
    for (int64_t k = 0; k < n; ++k) codes[k] = usable ? oracle_encode_int8(y[k] * inv) : 0;
}

/*
 * Fused transform + INT8 quantization of m rows: codes (m x n int8, row stride
 * out_stride) and scales (m floats).  Returns 0 on success, 1 on bad
 * arguments.
 */
int oracle_fwht_int8(const uint16_t *in, int64_t in_stride, int64_t m, int64_t n, int dtype,
                     double scale, int8_t *codes, int64_t out_stride, float *scales)
{
    if (m < 0 || !is_pow2(n) || in_stride < n || out_stride < n) return 1;
    if (dtype != ORACLE_FP16 && dtype != ORACLE_BF16) return 1;
    double *row = (double *)malloc((size_t)n * sizeof(double));
    float *y = (float *)malloc((size_t)n * sizeof(float));
    if (!row || !y) { free(row); free(y); return 1; }
    for (int64_t i = 0; i < m; ++i) {
        transform_row_fp32(in + i * in_stride, n, dtype, scale, row, y);
        quantize_row_int8(y, n, codes + i * out_stride, &scales[i]);
    }
    free(row);
    free(y);
    return 0;
}

/* INT8 quantization without the transform (see oracle_quantize_fp8). */
int oracle_quantize_int8(const float *y, int64_t m, int64_t n, int8_t *codes, float *scales)
{
    if (m < 0 || n < 1) return 1;
    for (int64_t i = 0; i < m; ++i) quantize_row_int8(y + i * n, n, codes + i * n, &scales[i]);
    return 0;
}
