/*
 * dps_oracle.c -- reference oracle for the nested-precision linear layer of
 * Dual-Mode Precision Serving (DPS, "Dual-Mode Precision LLM Serving with
 * Semi-Unified Memory").
 *
 * TEST INFRASTRUCTURE.  Only the test suite, the smoke check and the
 * benchmark's CPU-baseline leg load this library.  The product (the HIP
 * library under paper_2609_34380_amd/csrc) never calls it, links it or shares
 * a line of code with it, and this file includes nothing from there.
 *
 * Everything here is the plain definition, written to be checked by eye:
 *   - numbers are decoded from their bit fields by closed form (never by a
 *     hardware conversion or a bit shift into another format);
 *   - products are accumulated in fp64 in the natural k order;
 *   - the only parallelism is OpenMP over independent output rows.
 * All arrays are host memory.  Functions return 0 on success and a negative
 * value if an argument would make them read or write out of bounds.
 *
 * Readings of the paper this oracle takes (where the text leaves a choice):
 *   - the FP8 part of a nested FP16 weight is the upper byte (sign, five
 *     exponent bits, the two most significant mantissa bits), taken by
 *     truncation, and the residual is the lower byte (Sec. IV-A "Dynamic
 *     Networks and a Nested Model"; Sec. IV-B "Persistent Region"; Sec. IV-C,
 *     restoration paragraph);
 *   - the residual plane is a logical byte stream in the weight's row-major
 *     order, stored in fixed-size chunks placed by a slot table (Sec. IV-B
 *     "Shared Region": physical units mapped behind one virtual tensor);
 *   - fast-mode prefill quantizes each activation row to OCP E4M3 with a
 *     dynamic power-of-two scale (per-token dynamic activations as in
 *     Sec. V-A "Baselines"; the power of two is chosen so that scaling is
 *     exact and only one rounding happens);
 *   - the E4M3 nesting (Sec. IV-B "Persistent Region") keeps the sign, the
 *     four low exponent bits and the three leading mantissa bits; the dropped
 *     exponent MSB is zero for every weight it is used on, so the FP8 part
 *     read as OCP E4M3 (bias 7) is the FP16 value times 2^8, truncated, and
 *     the fast-mode weight is E4M3(upper) * 2^-8.  The residual is the seven
 *     low mantissa bits, kept in the low bits of a byte;
 *   - the per-layer encoding choice (Sec. IV-C, "Dual-mode serving"
 *     paragraph: E5M2 for layers whose range E4M3 cannot express) takes E4M3
 *     exactly when every weight of the layer nests losslessly (exponent MSB
 *     zero) and its E4M3 part is a number, i.e. |w| < 1.875; the largest
 *     fast-mode magnitude is then 448 * 2^-8 = 1.75.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#ifdef _OPENMP
#include <omp.h>
#endif

/* ------------------------------------------------------------------------ */
/* Number formats (Sec. II-B: ExMy = x exponent bits, y mantissa bits).      */
/* ------------------------------------------------------------------------ */

/* FP16 = E5M10, exponent bias 15.
 *   e in 1..30 : (-1)^s * 2^(e-15) * (1 + m/1024)
 *   e == 0     : (-1)^s * 2^(-14)  * (m/1024)          (subnormal, and +-0)
 *   e == 31    : +-inf if m == 0, NaN otherwise                               */
double oracle_fp16_value(uint16_t b)
{
    int s = (b >> 15) & 1;
    int e = (b >> 10) & 31;
    int m = b & 1023;
    double sign = s ? -1.0 : 1.0;
    if (e == 31)
        return m == 0 ? sign * INFINITY : NAN;
    if (e == 0)
        return sign * ldexp((double)m / 1024.0, -14);
    return sign * ldexp(1.0 + (double)m / 1024.0, e - 15);
}

/* FP8 E5M2 (same five-bit exponent and bias as FP16, Sec. II-B), bias 15.
 *   e in 1..30 : (-1)^s * 2^(e-15) * (1 + m/4)
 *   e == 0     : (-1)^s * 2^(-14)  * (m/4)
 *   e == 31    : +-inf if m == 0, NaN otherwise                               */
double oracle_e5m2_value(uint8_t b)
{
    int s = (b >> 7) & 1;
    int e = (b >> 2) & 31;
    int m = b & 3;
    double sign = s ? -1.0 : 1.0;
    if (e == 31)
        return m == 0 ? sign * INFINITY : NAN;
    if (e == 0)
        return sign * ldexp((double)m / 4.0, -14);
    return sign * ldexp(1.0 + (double)m / 4.0, e - 15);
}

/* FP8 E4M3 in the OCP "FN" flavour: bias 7, no infinities, the single NaN
 * pattern per sign is e == 15 && m == 7, largest finite value 448.
 *   e in 1..15 : (-1)^s * 2^(e-7) * (1 + m/8)
 *   e == 0     : (-1)^s * 2^(-6)  * (m/8)                                     */
double oracle_e4m3_value(uint8_t b)
{
    int s = (b >> 7) & 1;
    int e = (b >> 3) & 15;
    int m = b & 7;
    double sign = s ? -1.0 : 1.0;
    if (e == 15 && m == 7)
        return NAN;
    if (e == 0)
        return sign * ldexp((double)m / 8.0, -6);
    return sign * ldexp(1.0 + (double)m / 8.0, e - 7);
}

/* Nearest E4M3 value to v with ties going to the code whose mantissa is
 * even, found by scanning every non-negative finite code.  |v| must not
 * exceed 448 (returns -1 otherwise).  The sign bit is v's sign bit, so a
 * negative value that rounds to zero gives negative zero (0x80).            */
int oracle_e4m3_rne(double v, uint8_t *out)
{
    double a = fabs(v);
    if (!(a <= 448.0))
        return -1;
    int best = 0;
    double best_err = INFINITY;
    for (int c = 0; c <= 0x7E; ++c) {
        double err = fabs(oracle_e4m3_value((uint8_t)c) - a);
        if (err < best_err || (err == best_err && (c & 1) == 0 && (best & 1) == 1)) {
            best = c;
            best_err = err;
        }
    }
    *out = (uint8_t)(best | (signbit(v) ? 0x80 : 0));
    return 0;
}

/* ------------------------------------------------------------------------ */
/* Residual addressing (Sec. IV-B "Shared Region").                          */
/* ------------------------------------------------------------------------ */

/* Byte i of a residual's logical stream lives in chunk i / C at offset
 * i mod C; chunk c is stored in pool slot slots[c].  Returns the physical
 * byte offset into the pool, or -1 if the chunk or its slot is out of range. */
int64_t oracle_residual_addr(int64_t i, const int32_t *slots, int64_t n_chunks,
                             int32_t log2_chunk, int64_t pool_bytes)
{
    int64_t chunk_bytes = (int64_t)1 << log2_chunk;
    int64_t c = i / chunk_bytes;
    if (i < 0 || c >= n_chunks)
        return -1;
    int64_t slot = slots[c];
    int64_t phys = slot * chunk_bytes + (i % chunk_bytes);
    if (slot < 0 || phys >= pool_bytes)
        return -1;
    return phys;
}

static int check_residual(int64_t numel, const int32_t *slots, int64_t n_chunks,
                          int32_t log2_chunk, int64_t pool_bytes)
{
    if (log2_chunk < 0 || log2_chunk > 40)
        return -1;
    int64_t chunk_bytes = (int64_t)1 << log2_chunk;
    if (numel == 0)
        return 0;
    int64_t used = (numel - 1) / chunk_bytes + 1;
    if (used > n_chunks)
        return -1;
    for (int64_t c = 0; c < used; ++c)
        if (slots[c] < 0 || ((int64_t)slots[c] + 1) * chunk_bytes > pool_bytes)
            return -1;
    return 0;
}

/* ------------------------------------------------------------------------ */
/* Split and merge (Sec. IV-A, Sec. IV-B "Persistent Region").               */
/* ------------------------------------------------------------------------ */

enum { ORACLE_ENC_E5M2 = 0, ORACLE_ENC_E4M3 = 1 };

/* The two nested parts of the FP16 word b with fields sign s, exponent e
 * (5 bits), mantissa m (10 bits):
 *   E5M2: upper = s | e | m's 2 leading bits,         residual = m's 8 low bits
 *   E4M3: upper = s | e's 4 low bits | m's 3 leading, residual = m's 7 low bits
 * Field arithmetic only, so each line can be checked against the layouts.  */
static void nest_word(int enc, uint16_t b, uint8_t *hi, uint8_t *lo)
{
    int s = b / 32768, e = (b / 1024) % 32, m = b % 1024;
    if (enc == ORACLE_ENC_E5M2) {
        *hi = (uint8_t)(s * 128 + e * 4 + m / 256);
        *lo = (uint8_t)(m % 256);
    } else {
        *hi = (uint8_t)(s * 128 + (e % 16) * 8 + m / 128);
        *lo = (uint8_t)(m % 128);
    }
}

/* Inverse of nest_word: the FP16 word the two parts describe.  For E4M3 the
 * exponent MSB is zero and only the residual byte's seven low bits count.  */
static uint16_t unnest_word(int enc, uint8_t hi, uint8_t lo)
{
    int s = hi / 128;
    if (enc == ORACLE_ENC_E5M2) {
        int e = (hi / 4) % 32, mh = hi % 4;
        return (uint16_t)(s * 32768 + e * 1024 + mh * 256 + lo);
    }
    int e = (hi / 8) % 16, mh = hi % 8;
    return (uint16_t)(s * 32768 + e * 1024 + mh * 128 + lo % 128);
}

/* Fast-mode weight value of an upper byte: E5M2 as stored, or E4M3 scaled
 * back by 2^-8 (the E4M3 bias 7 against FP16's 15).                        */
double oracle_fast_value(int enc, uint8_t hi)
{
    if (enc == ORACLE_ENC_E5M2)
        return oracle_e5m2_value(hi);
    return ldexp(oracle_e4m3_value(hi), -8);
}

/* Per-layer encoding: E4M3 when every word nests losslessly into it and its
 * E4M3 part is a number, else E5M2.  An empty layer gets E4M3.             */
int oracle_select_enc(const uint16_t *w, int64_t numel)
{
    for (int64_t i = 0; i < numel; ++i) {
        int e = (w[i] / 1024) % 32;
        uint8_t hi, lo;
        nest_word(ORACLE_ENC_E4M3, w[i], &hi, &lo);
        if (e >= 16 || isnan(oracle_e4m3_value(hi)))
            return ORACLE_ENC_E5M2;
    }
    return ORACLE_ENC_E4M3;
}

/* FP16 words -> upper bytes (the FP8 part kept in the persistent region)
 * and residual bytes (written through the chunk table).  E4M3 on a word
 * whose exponent MSB is set keeps the fields above all the same (the MSB is
 * lost); oracle_select_enc tells whether a layer has such words.          */
int oracle_split(int enc, const uint16_t *w, int64_t numel, uint8_t *hi, uint8_t *pool,
                 int64_t pool_bytes, const int32_t *slots, int64_t n_chunks,
                 int32_t log2_chunk)
{
    if (enc != ORACLE_ENC_E5M2 && enc != ORACLE_ENC_E4M3)
        return -1;
    if (check_residual(numel, slots, n_chunks, log2_chunk, pool_bytes))
        return -1;
    for (int64_t i = 0; i < numel; ++i) {
        int64_t p = oracle_residual_addr(i, slots, n_chunks, log2_chunk, pool_bytes);
        if (p < 0)
            return -1;
        nest_word(enc, w[i], &hi[i], &pool[p]);
    }
    return 0;
}

/* Upper byte and residual byte -> the FP16 word.                          */
int oracle_merge(int enc, const uint8_t *hi, const uint8_t *pool, int64_t pool_bytes,
                 const int32_t *slots, int64_t n_chunks, int32_t log2_chunk,
                 int64_t numel, uint16_t *w_out)
{
    if (enc != ORACLE_ENC_E5M2 && enc != ORACLE_ENC_E4M3)
        return -1;
    if (check_residual(numel, slots, n_chunks, log2_chunk, pool_bytes))
        return -1;
    for (int64_t i = 0; i < numel; ++i) {
        int64_t p = oracle_residual_addr(i, slots, n_chunks, log2_chunk, pool_bytes);
        if (p < 0)
            return -1;
        w_out[i] = unnest_word(enc, hi[i], pool[p]);
    }
    return 0;
}

/* ------------------------------------------------------------------------ */
/* Residual backup and restore (Sec. IV-B "Residual Backup"; Sec. IV-C,     */
/* restoration paragraph).  The backup is the residual's logical byte       */
/* stream, contiguous in host memory.                                       */
/* ------------------------------------------------------------------------ */

/* Restore logical chunks [c0, c1) of a residual from its backup: byte i of
 * those chunks (i < numel) is written to the pool where the chunk table puts
 * it.  Every other pool byte is left as it was.                            */
int oracle_restore(const uint8_t *backup, int64_t numel, int64_t c0, int64_t c1,
                   uint8_t *pool, int64_t pool_bytes, const int32_t *slots,
                   int64_t n_chunks, int32_t log2_chunk)
{
    if (check_residual(numel, slots, n_chunks, log2_chunk, pool_bytes))
        return -1;
    int64_t chunk_bytes = (int64_t)1 << log2_chunk;
    int64_t used = numel == 0 ? 0 : (numel - 1) / chunk_bytes + 1;  /* chunks holding bytes */
    if (c0 < 0 || c1 < c0 || c1 > used)
        return -1;
    for (int64_t i = c0 * chunk_bytes; i < c1 * chunk_bytes && i < numel; ++i) {
        int64_t p = oracle_residual_addr(i, slots, n_chunks, log2_chunk, pool_bytes);
        if (p < 0)
            return -1;
        pool[p] = backup[i];
    }
    return 0;
}

/* The backup itself: the logical stream read back through the table.      */
int oracle_backup(const uint8_t *pool, int64_t pool_bytes, const int32_t *slots,
                  int64_t n_chunks, int32_t log2_chunk, int64_t numel, uint8_t *backup)
{
    if (check_residual(numel, slots, n_chunks, log2_chunk, pool_bytes))
        return -1;
    for (int64_t i = 0; i < numel; ++i) {
        int64_t p = oracle_residual_addr(i, slots, n_chunks, log2_chunk, pool_bytes);
        if (p < 0)
            return -1;
        backup[i] = pool[p];
    }
    return 0;
}

/* ------------------------------------------------------------------------ */
/* Nested linear layer (Sec. IV-C "Overall concept" and the GroupedGEMM     */
/* paragraph): Y[r][c] = sum_k X[r][k] * W[c][k].                           */
/*   full mode : W = the FP16 value of (upper byte, residual byte)          */
/*   fast mode : W = oracle_fast_value(upper byte); the residual is not     */
/*               read at all (pool and slots may be NULL).                  */
/* ------------------------------------------------------------------------ */

enum { ORACLE_FULL = 0, ORACLE_FAST = 1 };

/* sum_{kk < k} a[kk] * b[kk] in fp64, in the natural k order.              */
static double dot(const double *a, const double *b, int64_t k)
{
    double acc = 0.0;
    for (int64_t kk = 0; kk < k; ++kk)
        acc += a[kk] * b[kk];
    return acc;
}

/* Rows [r0, r1) of the FP16 matrix x [.][k], decoded once into a new fp64
 * array [r1 - r0][k] (NULL if it cannot be allocated).                    */
static double *decode_fp16_rows(const uint16_t *x, int64_t r0, int64_t r1, int64_t k)
{
    int64_t cnt = (r1 - r0) * k;
    double *v = (double *)malloc(sizeof(double) * (size_t)(cnt > 0 ? cnt : 1));
    if (!v)
        return NULL;
    for (int64_t i = 0; i < cnt; ++i)
        v[i] = oracle_fp16_value(x[r0 * k + i]);
    return v;
}

/* Weight element (c, k) of the expert whose elements start at logical
 * offset w_base (e * n * k for expert e).  Fills row c of the decoded
 * weight into wrow[0..k).                                                  */
static void decode_weight_row(int mode, int enc, const uint8_t *hi, const uint8_t *pool,
                              int64_t pool_bytes, const int32_t *slots,
                              int64_t n_chunks, int32_t log2_chunk,
                              int64_t w_base, int64_t c, int64_t k, double *wrow)
{
    for (int64_t kk = 0; kk < k; ++kk) {
        int64_t i = w_base + c * k + kk;
        if (mode == ORACLE_FAST) {
            wrow[kk] = oracle_fast_value(enc, hi[i]);
        } else {
            int64_t p = oracle_residual_addr(i, slots, n_chunks, log2_chunk, pool_bytes);
            wrow[kk] = oracle_fp16_value(unnest_word(enc, hi[i], p < 0 ? 0 : pool[p]));
        }
    }
}

/* Dense or grouped linear.  Rows [offsets[e], offsets[e+1]) of x use expert
 * e's weights (elements e*n*k ... (e+1)*n*k - 1 of hi and of the residual
 * stream).  Dense is experts == 1 with offsets {0, rows}.  y is fp64
 * [rows][n].  hi holds experts*n*k bytes.                                   */
int oracle_linear_grouped(int mode, int enc, const uint16_t *x, const int64_t *offsets,
                          int64_t experts, int64_t n, int64_t k,
                          const uint8_t *hi, const uint8_t *pool, int64_t pool_bytes,
                          const int32_t *slots, int64_t n_chunks, int32_t log2_chunk,
                          double *y)
{
    if (mode != ORACLE_FULL && mode != ORACLE_FAST)
        return -1;
    if (enc != ORACLE_ENC_E5M2 && enc != ORACLE_ENC_E4M3)
        return -1;
    if (experts < 1 || n < 0 || k < 0 || offsets[0] != 0)
        return -1;
    for (int64_t e = 0; e < experts; ++e)
        if (offsets[e + 1] < offsets[e])
            return -1;
    if (mode == ORACLE_FULL &&
        check_residual(experts * n * k, slots, n_chunks, log2_chunk, pool_bytes))
        return -1;

    int bad = 0;
    for (int64_t e = 0; e < experts; ++e) {
        int64_t r0 = offsets[e], r1 = offsets[e + 1];
        if (r1 == r0)
            continue;
        int64_t w_base = e * n * k;
        double *xv = decode_fp16_rows(x, r0, r1, k);
        if (!xv)
            return -1;
#pragma omp parallel
        {
            double *wrow = (double *)malloc(sizeof(double) * (size_t)(k > 0 ? k : 1));
            if (!wrow) {
#pragma omp atomic write
                bad = 1;
            } else {
#pragma omp for schedule(static)
                for (int64_t c = 0; c < n; ++c) {
                    decode_weight_row(mode, enc, hi, pool, pool_bytes, slots, n_chunks,
                                      log2_chunk, w_base, c, k, wrow);
                    for (int64_t r = r0; r < r1; ++r)
                        y[r * n + c] = dot(xv + (r - r0) * k, wrow, k);
                }
                free(wrow);
            }
        }
        free(xv);
    }
    return bad ? -1 : 0;
}

int oracle_linear(int mode, int enc, const uint16_t *x, int64_t m, int64_t n, int64_t k,
                  const uint8_t *hi, const uint8_t *pool, int64_t pool_bytes,
                  const int32_t *slots, int64_t n_chunks, int32_t log2_chunk,
                  double *y)
{
    int64_t offsets[2] = {0, m};
    return oracle_linear_grouped(mode, enc, x, offsets, 1, n, k, hi, pool, pool_bytes,
                                 slots, n_chunks, log2_chunk, y);
}

/* Dense linear restricted to the listed output rows (for sampled checks of
 * large problems): y[j][c] = sum_k X[rows[j]][k] * W[c][k].               */
int oracle_linear_rows(int mode, int enc, const uint16_t *x, const int64_t *rows,
                       int64_t n_rows, int64_t n, int64_t k, const uint8_t *hi,
                       const uint8_t *pool, int64_t pool_bytes, const int32_t *slots,
                       int64_t n_chunks, int32_t log2_chunk, double *y)
{
    if (mode != ORACLE_FULL && mode != ORACLE_FAST)
        return -1;
    if (enc != ORACLE_ENC_E5M2 && enc != ORACLE_ENC_E4M3)
        return -1;
    if (mode == ORACLE_FULL &&
        check_residual(n * k, slots, n_chunks, log2_chunk, pool_bytes))
        return -1;
    /* the listed rows of x, decoded once */
    double *xv = (double *)malloc(sizeof(double) * (size_t)(n_rows * k > 0 ? n_rows * k : 1));
    if (!xv)
        return -1;
    for (int64_t j = 0; j < n_rows; ++j)
        for (int64_t kk = 0; kk < k; ++kk)
            xv[j * k + kk] = oracle_fp16_value(x[rows[j] * k + kk]);
    int bad = 0;
#pragma omp parallel
    {
        double *wrow = (double *)malloc(sizeof(double) * (size_t)(k > 0 ? k : 1));
        if (!wrow) {
#pragma omp atomic write
            bad = 1;
        } else {
#pragma omp for schedule(static)
            for (int64_t c = 0; c < n; ++c) {
                decode_weight_row(mode, enc, hi, pool, pool_bytes, slots, n_chunks,
                                  log2_chunk, 0, c, k, wrow);
                for (int64_t j = 0; j < n_rows; ++j)
                    y[j * n + c] = dot(xv + j * k, wrow, k);
            }
            free(wrow);
        }
    }
    free(xv);
    return bad ? -1 : 0;
}

/* ------------------------------------------------------------------------ */
/* Fast-mode prefill with FP8 activations.                                  */
/* ------------------------------------------------------------------------ */

/* Row r: a = max_k |X[r][k]|; the scale s is the smallest power of two with
 * a <= 448 * s (s = 1 when a == 0); Xq[r][k] = nearest E4M3 to X[r][k] / s
 * (ties to even).  Division by a power of two is exact, so there is a single
 * rounding per element.  Returns -1 on a non-finite input.                */
int oracle_act_quant(const uint16_t *x, int64_t m, int64_t k, uint8_t *xq, double *scale)
{
    for (int64_t r = 0; r < m; ++r) {
        double a = 0.0;
        for (int64_t kk = 0; kk < k; ++kk) {
            double v = oracle_fp16_value(x[r * k + kk]);
            if (!isfinite(v))
                return -1;
            if (fabs(v) > a)
                a = fabs(v);
        }
        double s = 1.0;
        if (a > 0.0) {
            while (a > 448.0 * s)
                s *= 2.0;
            while (a <= 448.0 * (s / 2.0))
                s /= 2.0;
        }
        scale[r] = s;
        for (int64_t kk = 0; kk < k; ++kk)
            if (oracle_e4m3_rne(oracle_fp16_value(x[r * k + kk]) / s, &xq[r * k + kk]))
                return -1;
    }
    return 0;
}

/* Y[r][c] = s_r * sum_k E4M3(Xq[r][k]) * oracle_fast_value(hi[c][k]).    */
int oracle_linear_fp8(int enc, const uint8_t *xq, const double *scale, int64_t m, int64_t n,
                      int64_t k, const uint8_t *hi, double *y)
{
    if (enc != ORACLE_ENC_E5M2 && enc != ORACLE_ENC_E4M3)
        return -1;
    /* the E4M3 activation codes, decoded once */
    double *xv = (double *)malloc(sizeof(double) * (size_t)(m * k > 0 ? m * k : 1));
    if (!xv)
        return -1;
    for (int64_t i = 0; i < m * k; ++i)
        xv[i] = oracle_e4m3_value(xq[i]);
    int bad = 0;
#pragma omp parallel
    {
        double *wrow = (double *)malloc(sizeof(double) * (size_t)(k > 0 ? k : 1));
        if (!wrow) {
#pragma omp atomic write
            bad = 1;
        } else {
#pragma omp for schedule(static)
            for (int64_t c = 0; c < n; ++c) {
                for (int64_t kk = 0; kk < k; ++kk)
                    wrow[kk] = oracle_fast_value(enc, hi[c * k + kk]);
                for (int64_t r = 0; r < m; ++r)
                    y[r * n + c] = scale[r] * dot(xv + r * k, wrow, k);
            }
            free(wrow);
        }
    }
    free(xv);
    return bad ? -1 : 0;
}

/* Number of OpenMP threads the linear routines run on.                    */
int oracle_num_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/* Threads the linear routines run on from now on (n >= 1); returns the
 * previous count.  Only the benchmark's CPU baseline changes it, to time the
 * oracle on one core as well as on all of them.                          */
int oracle_set_num_threads(int n)
{
    int prev = oracle_num_threads();
#ifdef _OPENMP
    if (n >= 1)
        omp_set_num_threads(n);
#endif
    return prev;
}
