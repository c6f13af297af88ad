/*
 * rfq_oracle.c -- plain, slow, obviously-correct CPU oracle for Residual
 * Fallback Quantization (RFQ) with MXFP4 codes.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product path may link, load or
 * call this file; only the test suite, the smoke check and the CPU-baseline
 * leg of the benchmark use it.  It shares no source, header, table or helper
 * with the GPU library.
 *
 * Every value is carried in double precision.  All inputs handled here
 * (fp32 and bf16 activations, E2M1 grid points times powers of two) are exact
 * in double, so quantization decisions are taken on exact values.
 *
 * What is computed, with the passage of the paper it follows:
 *   - MX block scale, Sec. 3.2 Eq. (3), read with the OCP MX rule that the
 *     shared exponent is floor(log2(amax)) minus the largest exponent of the
 *     element format (2 for E2M1).
 *   - MX element quantization, Sec. 3.2 Eq. (4); element format E2M1
 *     (Sec. 3.2.2: 1 sign, 2 exponent, 1 mantissa bit), round to nearest with
 *     ties to even, saturating at +-6.
 *   - Primary quantization of activations and weights, Sec. 4.3 Eq. (8).
 *   - Residual DeltaX = X - Xtilde, Sec. 4.3 Eq. (9), and its quantization
 *     with the same quantizer, Eq. (10), with its own block scale.
 *   - The RFQ product, Sec. 4.3 Eq. (11) / Algorithm 1, with the fallback
 *     indicator phi fixed to 1 (every block carries a residual), 0 (plain
 *     MXFP4), or given per activation tile of ORACLE_PHI_ROWS rows by
 *     ORACLE_PHI_K reduction columns (Algorithm 1 takes phi(p, r) as an input
 *     over blocks of P_s x R_s; these are the library's tile sizes).
 *   - Two rules that produce such a phi map (the paper states none): phi = 1
 *     where a tile's residual codes are not all zero (the residual term of
 *     the other tiles is exactly zero), or where a tile holds a primary scale
 *     byte at least a threshold (a large block maximum marks an outlier).
 *   - Dequantization X ~ Xtilde + phi * Xhat, Sec. 4.3 Eq. (12).
 *   - SwiGLU intermediate h = bf16(silu(g) * u) for the MLP workload (not
 *     from the paper; used to chain two RFQ products).
 *
 * Planted mistakes: building with -DORACLE_PLANT=<n> (n >= 1) swaps in one
 * plausible error at a marked site, so that the test suite can show that its
 * pins catch it.  The default build (ORACLE_PLANT undefined, i.e. 0) has none.
 *
 * Storage conventions shared with the GPU library only through the written
 * interface (not through code): a 4-bit code is sign<<3 | magnitude index,
 * two codes per byte with the lower-indexed element in the low nibble,
 * codes[row][K/2] and scales[row][K/32] row-major, one E8M0 byte per block
 * (value 2^(byte-127)).
 */
#include <math.h>
#ifdef _OPENMP
#include <omp.h>
#endif
#include <stdint.h>
#include <stddef.h>
#include <string.h>

#define ORACLE_BLOCK 32
#define ORACLE_PHI_ROWS 64
#if ORACLE_PLANT == 12
#define ORACLE_PHI_K 128        /* planted: phi tile width halved */
#else
#define ORACLE_PHI_K 256
#endif

#ifndef ORACLE_PLANT
#define ORACLE_PLANT 0
#endif

/* E2M1 magnitudes indexed by the 3-bit magnitude field (Sec. 3.2.2):
 * exponent bias 1, one mantissa bit, exponent field 0 is subnormal. */
static double e2m1_magnitude(int mag3)
{
    int ebits = (mag3 >> 1) & 3;
    int mbit = mag3 & 1;
    if (ebits == 0)
        return 0.5 * mbit;                      /* subnormal: 0 or 0.5 */
    return ldexp(1.0 + 0.5 * mbit, ebits - 1);  /* 1, 1.5, 2, 3, 4, 6 */
}

/* Value of one 4-bit code (Sec. 3.2.2). */
double oracle_e2m1_value(int code)
{
    double m = e2m1_magnitude(code & 7);
    return (code & 8) ? -m : m;
}

/* floor(log2(a)) for finite a > 0, exactly, through frexp: a = f * 2^p with
 * f in [0.5, 1) gives floor(log2 a) = p - 1. */
static int floor_log2(double a)
{
    int p;
    (void)frexp(a, &p);
    return p - 1;
}

/* Shared block exponent, Eq. (3) with the OCP MX offset: e = floor(log2 amax)
 * - 2, clamped to the E8M0 range [-127, 127]; an all-zero block takes the
 * lower clamp. */
int oracle_block_exponent(double amax)
{
    int e;
    if (amax == 0.0)
        return -127;
    e = floor_log2(amax) - 2;
#if ORACLE_PLANT == 1
    e = floor_log2(amax);                  /* planted: Eq. (3) without -emax */
#endif
#if ORACLE_PLANT == 2
    e = floor_log2(amax) - 1;              /* planted: off-by-one offset */
#endif
    if (e < -127)
        e = -127;
    if (e > 127)
        e = 127;
    return e;
}

/* Element quantization, Eq. (4): y = x / 2^e is exact; round |y| to the
 * nearest E2M1 magnitude, ties to the even magnitude index (the one whose
 * mantissa bit is 0), values above 6 saturate to 6.  The sign is kept, also
 * for a value that rounds to zero. */
int oracle_e2m1_encode(double y)
{
    double a = fabs(y);
    int best = 0;
    if (a > 6.0)
        a = 6.0;        /* saturate to the largest E2M1 magnitude */
    double best_d = a;  /* distance to magnitude 0 */
    int m;
    for (m = 1; m < 8; ++m) {
        double d = fabs(a - e2m1_magnitude(m));
#if ORACLE_PLANT == 3
        if (d < best_d || d == best_d) {   /* planted: ties away from zero */
#else
        if (d < best_d || (d == best_d && (m & 1) == 0)) {
#endif
            best = m;
            best_d = d;
        }
    }
#if ORACLE_PLANT == 4
    if (best == 0)
        return 0;                          /* planted: sign of zero dropped */
#endif
    return (signbit(y) ? 8 : 0) | best;
}

static void put_nibble(uint8_t *row_codes, int64_t k, int code)
{
    uint8_t *b = row_codes + k / 2;
#if ORACLE_PLANT == 5
    k ^= 1;                                /* planted: nibble order swapped */
#endif
    if (k & 1)
        *b = (uint8_t)((*b & 0x0F) | (code << 4));
    else
        *b = (uint8_t)((*b & 0xF0) | code);
}

static int get_nibble(const uint8_t *row_codes, int64_t k)
{
    uint8_t b = row_codes[k / 2];
#if ORACLE_PLANT == 5
    k ^= 1;
#endif
    return (k & 1) ? (b >> 4) : (b & 0x0F);
}

/* Quantize one block of 32 values (Eq. 3 + Eq. 4).  Writes 32 codes into
 * the packed row at element offset k0 and returns the E8M0 byte.  If deq is
 * not NULL it receives the dequantized values (Eq. 12, first term). */
static uint8_t quantize_block(const double *x, uint8_t *row_codes, int64_t k0,
                              double *deq)
{
    double amax = 0.0;
    int i, e;
    for (i = 0; i < ORACLE_BLOCK; ++i)
        if (fabs(x[i]) > amax)
            amax = fabs(x[i]);
    e = oracle_block_exponent(amax);
    for (i = 0; i < ORACLE_BLOCK; ++i) {
        double y = ldexp(x[i], -e);
        int c = oracle_e2m1_encode(y);
        put_nibble(row_codes, k0 + i, c);
        if (deq)
            deq[i] = ldexp(oracle_e2m1_value(c), e);
    }
    return (uint8_t)(e + 127);
}

/*
 * Primary quantization Q(X), Eq. (8), and -- when r_codes is not NULL -- the
 * residual DeltaX = X - deq(Q(X)), Eq. (9), quantized with its own block
 * scale, Eq. (10).  x is rows x K row-major (K a multiple of 32).
 * Outputs: codes rows x K/2 bytes, scales rows x K/32 bytes.
 */
void oracle_rfq_quantize(const double *x, int64_t rows, int64_t K,
                         uint8_t *q_codes, uint8_t *q_scales,
                         uint8_t *r_codes, uint8_t *r_scales)
{
    int64_t nb = K / ORACLE_BLOCK;
    int64_t m;
#pragma omp parallel for schedule(static)
    for (m = 0; m < rows; ++m) {
        int64_t b;
        for (b = 0; b < nb; ++b) {
            const double *xb = x + m * K + b * ORACLE_BLOCK;
            double deq[ORACLE_BLOCK], res[ORACLE_BLOCK];
            int i;
            q_scales[m * nb + b] =
                quantize_block(xb, q_codes + m * (K / 2), b * ORACLE_BLOCK, deq);
            if (r_codes) {
                for (i = 0; i < ORACLE_BLOCK; ++i)
                    res[i] = xb[i] - deq[i];
#if ORACLE_PLANT == 6
                for (i = 0; i < ORACLE_BLOCK; ++i)
                    res[i] = xb[i];        /* planted: residual of x, not of x - q */
#endif
                r_scales[m * nb + b] =
                    quantize_block(res, r_codes + m * (K / 2), b * ORACLE_BLOCK, NULL);
            }
        }
    }
}

/* Dequantization of one code tensor, Eq. (12) term by term:
 * out[row][k] = value(code) * 2^(scale - 127). */
void oracle_dequant(const uint8_t *codes, const uint8_t *scales, int64_t rows,
                    int64_t K, double *out)
{
    int64_t nb = K / ORACLE_BLOCK;
    int64_t m;
#pragma omp parallel for schedule(static)
    for (m = 0; m < rows; ++m) {
        int64_t k;
        for (k = 0; k < K; ++k) {
            int c = get_nibble(codes + m * (K / 2), k);
            int e = (int)scales[m * nb + k / ORACLE_BLOCK] - 127;
            out[m * K + k] = ldexp(oracle_e2m1_value(c), e);
        }
    }
}

/* One output of the RFQ product, Eq. (11): the primary and the residual
 * contraction are summed separately over k in increasing order, then added.
 * bound receives sum_k |q w| + |r w| (the scale of the rounding error any
 * fp32 evaluation may make). */
static void gemm_one(const uint8_t *qc, const uint8_t *qs,
                     const uint8_t *rc, const uint8_t *rs,
                     const uint8_t *wc, const uint8_t *ws, const uint8_t *phi,
                     int64_t K, int64_t m, int64_t n, double *z, double *bound)
{
    int64_t phi_cols = (K + ORACLE_PHI_K - 1) / ORACLE_PHI_K;
    int64_t nb = K / ORACLE_BLOCK;
    double zq = 0.0, zr = 0.0, bsum = 0.0;
    int64_t k;
    for (k = 0; k < K; ++k) {
        int64_t b = k / ORACLE_BLOCK;
#if ORACLE_PLANT == 11
        int64_t kw = (k + 1) % K;          /* planted: misaligned weight index */
#else
        int64_t kw = k;
#endif
        double w = ldexp(oracle_e2m1_value(get_nibble(wc + n * (K / 2), kw)),
                         (int)ws[n * nb + b] - 127);
#if ORACLE_PLANT == 7
        w = ldexp(oracle_e2m1_value(get_nibble(wc + n * (K / 2), k)),
                  (int)qs[m * nb + b] - 127);  /* planted: wrong scale operand */
#endif
        double q = ldexp(oracle_e2m1_value(get_nibble(qc + m * (K / 2), k)),
                         (int)qs[m * nb + b] - 127);
        zq += q * w;
        bsum += fabs(q * w);
        if (rc && (!phi || phi[(m / ORACLE_PHI_ROWS) * phi_cols + k / ORACLE_PHI_K])) {
            double r = ldexp(oracle_e2m1_value(get_nibble(rc + m * (K / 2), k)),
                             (int)rs[m * nb + b] - 127);
            zr += r * w;
            bsum += fabs(r * w);
        }
    }
    *z = zq + zr;
#if ORACLE_PLANT == 8
    *z = zq;                               /* planted: residual term dropped */
#endif
    *bound = bsum;
}

/* Full RFQ product Z[M][N] with a phi map phi[ceil(M/64)][ceil(K/256)]
 * (nonzero: the tile's residual term is included; NULL: phi = 1; rc NULL:
 * phi = 0), weights stored [N][K] with blocks along K.  The bound covers the
 * terms included. */
void oracle_gemm_phi(const uint8_t *qc, const uint8_t *qs,
                     const uint8_t *rc, const uint8_t *rs,
                     const uint8_t *wc, const uint8_t *ws, const uint8_t *phi,
                     int64_t M, int64_t N, int64_t K, double *z, double *bound)
{
    int64_t m;
#pragma omp parallel for schedule(dynamic, 1)
    for (m = 0; m < M; ++m) {
        int64_t n;
        for (n = 0; n < N; ++n)
            gemm_one(qc, qs, rc, rs, wc, ws, phi, K, m, n, z + m * N + n,
                     bound + m * N + n);
    }
}

/* Full RFQ product with phi = 1 (phi = 0 when rc is NULL). */
void oracle_gemm(const uint8_t *qc, const uint8_t *qs,
                 const uint8_t *rc, const uint8_t *rs,
                 const uint8_t *wc, const uint8_t *ws,
                 int64_t M, int64_t N, int64_t K, double *z, double *bound)
{
    oracle_gemm_phi(qc, qs, rc, rs, wc, ws, NULL, M, N, K, z, bound);
}

/* phi map [ceil(M/64)][ceil(K/256)] by one of two rules (the paper gives
 * none): rule 0 sets phi where some residual code of the tile has a nonzero
 * magnitude, rule 1 where some primary scale byte of the tile is at least
 * threshold. */
void oracle_fallback_map(const uint8_t *rc, const uint8_t *qs, int64_t M, int64_t K,
                         int rule, int threshold, uint8_t *phi)
{
    int64_t nb = K / ORACLE_BLOCK;
    int64_t pr = (M + ORACLE_PHI_ROWS - 1) / ORACLE_PHI_ROWS;
    int64_t pc = (K + ORACLE_PHI_K - 1) / ORACLE_PHI_K;
    int64_t t;
#pragma omp parallel for schedule(static)
    for (t = 0; t < pr * pc; ++t) {
        int64_t p = t / pc, c = t % pc, m, k;
        int on = 0;
        for (m = p * ORACLE_PHI_ROWS; m < M && m < (p + 1) * ORACLE_PHI_ROWS; ++m) {
            for (k = c * ORACLE_PHI_K; k < K && k < (c + 1) * ORACLE_PHI_K; ++k) {
                if (rule == 0) {
                    if ((get_nibble(rc + m * (K / 2), k) & 7) != 0)
                        on = 1;
                } else {
#if ORACLE_PLANT == 13
                    if ((int)qs[m * nb + k / ORACLE_BLOCK] > threshold)   /* planted: > */
#else
                    if ((int)qs[m * nb + k / ORACLE_BLOCK] >= threshold)
#endif
                        on = 1;
                }
            }
        }
        phi[t] = (uint8_t)on;
    }
}

/* The same product at count sampled (row, col) positions. */
void oracle_gemm_sampled(const uint8_t *qc, const uint8_t *qs,
                         const uint8_t *rc, const uint8_t *rs,
                         const uint8_t *wc, const uint8_t *ws,
                         int64_t K, const int64_t *rows, const int64_t *cols,
                         int64_t count, double *z, double *bound)
{
    int64_t i;
#pragma omp parallel for schedule(static)
    for (i = 0; i < count; ++i)
        gemm_one(qc, qs, rc, rs, wc, ws, NULL, K, rows[i], cols[i], z + i, bound + i);
}

/* Round a double to the nearest bfloat16 value (8 significant bits, the
 * exponent range of binary32), ties to even, overflow to infinity. */
double oracle_round_bf16(double v)
{
    int p;
    double f;
    if (v == 0.0 || isnan(v) || isinf(v))
        return v;
    if (fabs(v) < ldexp(1.0, -126))                     /* subnormal range */
        return ldexp(nearbyint(ldexp(v, 133)), -133);
    f = frexp(v, &p);                                    /* |f| in [0.5, 1) */
#if ORACLE_PLANT == 9
    f = ldexp(trunc(ldexp(f, 8)), -8);     /* planted: truncation */
#else
    f = ldexp(nearbyint(ldexp(f, 8)), -8);
#endif
    v = ldexp(f, p);
    if (fabs(v) >= ldexp(1.0, 128))
        return v > 0 ? INFINITY : -INFINITY;
    return v;
}

/* SwiGLU intermediate for the MLP workload: h = bf16(silu(g) * u) with
 * silu(g) = g / (1 + exp(-g)). */
void oracle_swiglu(const double *g, const double *u, int64_t n, double *h)
{
    int64_t i;
#pragma omp parallel for schedule(static)
    for (i = 0; i < n; ++i)
#if ORACLE_PLANT == 10
        h[i] = oracle_round_bf16(g[i] / (1.0 + exp(g[i])) * u[i]);  /* planted: sign */
#else
        h[i] = oracle_round_bf16(g[i] / (1.0 + exp(-g[i])) * u[i]);
#endif
}

/* Exact residual values DeltaX (Eq. 9) for inspection by tests. */
void oracle_residual(const double *x, int64_t rows, int64_t K, double *res)
{
    int64_t nb = K / ORACLE_BLOCK;
    int64_t m;
    for (m = 0; m < rows; ++m) {
        int64_t b;
        uint8_t scratch[ORACLE_BLOCK / 2];
        for (b = 0; b < nb; ++b) {
            double deq[ORACLE_BLOCK];
            int i;
            const double *xb = x + m * K + b * ORACLE_BLOCK;
            memset(scratch, 0, sizeof scratch);
            (void)quantize_block(xb, scratch, 0, deq);
            for (i = 0; i < ORACLE_BLOCK; ++i)
                res[m * K + b * ORACLE_BLOCK + i] = xb[i] - deq[i];
        }
    }
}

/* Number of threads the parallel loops above use (1 without OpenMP). */
int oracle_num_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/* Sets the number of threads of later parallel loops (for timing the oracle
 * single-threaded); no effect without OpenMP. */
void oracle_set_num_threads(int n)
{
#ifdef _OPENMP
    if (n > 0) omp_set_num_threads(n);
#else
    (void)n;
#endif
}
