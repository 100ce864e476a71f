/*
 * CPU oracle for the signaled + reordered GEMM path -- TEST INFRASTRUCTURE.
 *
 * Only the test suite, the smoke check and the benchmark's CPU-baseline leg
 * may load this library. The GPU path never calls it and shares no code with
 * it. Everything here is deliberately plain: fp64 arithmetic, loops in the
 * order the definitions are written, one rounding to the storage dtype at
 * the end.
 *
 * Contents (each cites the passage it follows):
 *   - binary16 / bfloat16 decode and round-to-nearest-even encode, written
 *     from the IEEE 754 format definitions;
 *   - the GEMM C = A x B of Section 2.1.1 (A^{MxK} x B^{KxN}), with B handed
 *     over as W = B^T [N, K]; exact products, fp64 sums, one RNE rounding;
 *   - the AllReduce / ReduceScatter stand-in of the consumer: the
 *     correctly rounded sum of a local and a peer partial (Section 2.3.1:
 *     AllReduce reduces the GEMM partial results of all GPUs);
 *   - RMSNorm after the post-communication reorder (Section 6.6 evaluates an
 *     RMSNorm kernel fused with the post-communication reordering):
 *     y = h / sqrt(mean(h^2) + eps) * gamma with h = x + bias.
 *
 * Build: gcc -O2 -ffp-contract=off -fopenmp -shared -fPIC (see build.py).
 */
#include <math.h>
#include <stdint.h>
#include <string.h>

#define DT_FP16 0
#define DT_BF16 1

/* ---- storage formats --------------------------------------------------- */

/* binary16: 1 sign bit, 5 exponent bits (bias 15), 10 fraction bits. */
double fo_orc_half_to_f64(uint16_t h) {
    int sign = (h >> 15) & 1;
    int e = (h >> 10) & 0x1F;
    int f = h & 0x3FF;
    double v;
    if (e == 0)
        v = ldexp((double)f, -24);                 /* subnormal: f * 2^-24 */
    else if (e == 31)
        v = f ? NAN : INFINITY;
    else
        v = ldexp((double)(1024 + f), e - 25);     /* 1.f * 2^(e-15) */
    return sign ? -v : v;
}

/* bfloat16: 1 sign bit, 8 exponent bits (bias 127), 7 fraction bits. */
double fo_orc_bf16_to_f64(uint16_t b) {
    int sign = (b >> 15) & 1;
    int e = (b >> 7) & 0xFF;
    int f = b & 0x7F;
    double v;
    if (e == 0)
        v = ldexp((double)f, -133);                /* subnormal: f * 2^-133 */
    else if (e == 255)
        v = f ? NAN : INFINITY;
    else
        v = ldexp((double)(128 + f), e - 134);     /* 1.f * 2^(e-127) */
    return sign ? -v : v;
}

/*
 * Round a double to a binary format with `p` significand bits (including the
 * hidden bit), minimum normal exponent `emin` and maximum exponent `emax`,
 * ties to even. Returns the encoded magnitude bits; `ebits`/`fbits` give the
 * field widths. Scaling by powers of two is exact in double, and nearbyint()
 * in the default rounding mode rounds half to even.
 */
static uint16_t encode_rne(double x, int p, int emin, int emax, int fbits, int ebits) {
    uint16_t sign = signbit(x) ? (uint16_t)(1u << (fbits + ebits)) : 0;
    uint16_t exp_all_ones = (uint16_t)(((1u << ebits) - 1) << fbits);
    if (isnan(x))
        return (uint16_t)(sign | exp_all_ones | (1u << (fbits - 1)));
    double a = fabs(x);
    if (isinf(a))
        return (uint16_t)(sign | exp_all_ones);
    if (a < ldexp(1.0, emin)) {
        /* subnormal range: quantum 2^(emin - p + 1) */
        double q = nearbyint(ldexp(a, -(emin - p + 1)));
        /* q may reach 2^(p-1): the encoding then reads as the smallest normal */
        return (uint16_t)(sign | (uint16_t)q);
    }
    int e2;
    frexp(a, &e2);              /* a = m * 2^e2, m in [0.5, 1) */
    int E = e2 - 1;             /* a in [2^E, 2^(E+1)) */
    double s = nearbyint(ldexp(a, -(E - p + 1)));   /* significand in [2^(p-1), 2^p] */
    if (s == ldexp(1.0, p)) {   /* rounded up to the next binade */
        s = ldexp(1.0, p - 1);
        E += 1;
    }
    if (E > emax)
        return (uint16_t)(sign | exp_all_ones);     /* overflow to infinity */
    int bias = (1 << (ebits - 1)) - 1;
    uint16_t field_e = (uint16_t)(E + bias);
    uint16_t field_f = (uint16_t)((uint32_t)s - (1u << (p - 1)));
    return (uint16_t)(sign | (uint16_t)(field_e << fbits) | field_f);
}

uint16_t fo_orc_f64_to_half(double x) { return encode_rne(x, 11, -14, 15, 10, 5); }
uint16_t fo_orc_f64_to_bf16(double x) { return encode_rne(x, 8, -126, 127, 7, 8); }

static double dec(uint16_t v, int dtype) {
    return dtype == DT_FP16 ? fo_orc_half_to_f64(v) : fo_orc_bf16_to_f64(v);
}
static uint16_t enc(double v, int dtype) {
    return dtype == DT_FP16 ? fo_orc_f64_to_half(v) : fo_orc_f64_to_bf16(v);
}

void fo_orc_decode(const uint16_t* in, int64_t n, int dtype, double* out) {
    #pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; ++i) out[i] = dec(in[i], dtype);
}

void fo_orc_encode(const double* in, int64_t n, int dtype, uint16_t* out) {
    #pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; ++i) out[i] = enc(in[i], dtype);
}

/* ---- GEMM ------------------------------------------------------------- */

/*
 * C[i, n] = sum_k A[i, k] * B[k, n] with B[k, n] = W[n, k].
 * A is [M, K] row-major, W is [N, K] row-major, C is [M, N] row-major fp64.
 * Products of two fp16 (or bf16) values are exact in fp64; the sum runs in
 * plain k order. Only rows rows[0..nrows) and columns [n0, n1) are computed
 * (pass all rows and [0, N) for the full product); results go to
 * C[r * ldc + (n - n0)] for the r-th listed row.
 */
void fo_orc_gemm_rows(const uint16_t* A, const uint16_t* W, int dtype,
                      int64_t K, const int64_t* rows, int64_t nrows,
                      int64_t n0, int64_t n1, double* C, int64_t ldc) {
    #pragma omp parallel for schedule(dynamic, 1)
    for (int64_t r = 0; r < nrows; ++r) {
        const uint16_t* a = A + rows[r] * K;
        for (int64_t n = n0; n < n1; ++n) {
            const uint16_t* w = W + n * K;
            double acc = 0.0;
            for (int64_t k = 0; k < K; ++k)
                acc += dec(a[k], dtype) * dec(w[k], dtype);
            C[r * ldc + (n - n0)] = acc;
        }
    }
}

/* Same product on operands already widened to fp64 (faster for large runs). */
void fo_orc_gemm_f64(const double* A, const double* W, int64_t M, int64_t N,
                     int64_t K, const int64_t* rows, int64_t nrows,
                     int64_t n0, int64_t n1, double* C, int64_t ldc) {
    (void)M; (void)N;
    #pragma omp parallel for schedule(dynamic, 1)
    for (int64_t r = 0; r < nrows; ++r) {
        const double* a = A + rows[r] * K;
        for (int64_t n = n0; n < n1; ++n) {
            const double* w = W + n * K;
            double acc = 0.0;
            for (int64_t k = 0; k < K; ++k)
                acc += a[k] * w[k];
            C[r * ldc + (n - n0)] = acc;
        }
    }
}

/* ---- consumer stand-in ------------------------------------------------- */

/*
 * out = RNE(a + b). Two fp16 (or bf16) values add exactly in fp64, so this
 * is the correctly rounded sum, the value any correct reduction of two
 * partials must produce.
 */
void fo_orc_add(const uint16_t* a, const uint16_t* b, int64_t n, int dtype, uint16_t* out) {
    #pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; ++i)
        out[i] = enc(dec(a[i], dtype) + dec(b[i], dtype), dtype);
}

/* ---- RMSNorm ----------------------------------------------------------- */

/*
 * For each of `rows` rows of length n: h = x + bias (bias optional),
 * y = h / sqrt(mean(h^2) + eps) * gamma (gamma optional, else 1), rounded
 * once to the storage dtype. With do_norm == 0 only y = RNE(h) is produced.
 */
void fo_orc_rmsnorm(const uint16_t* x, int64_t rows, int64_t n,
                    const uint16_t* bias, const uint16_t* gamma, double eps,
                    int do_norm, int dtype, uint16_t* out) {
    #pragma omp parallel for schedule(static)
    for (int64_t r = 0; r < rows; ++r) {
        const uint16_t* xr = x + r * n;
        double ss = 0.0;
        for (int64_t c = 0; c < n; ++c) {
            double h = dec(xr[c], dtype) + (bias ? dec(bias[c], dtype) : 0.0);
            ss += h * h;
        }
        double inv = do_norm ? 1.0 / sqrt(ss / (double)n + eps) : 1.0;
        for (int64_t c = 0; c < n; ++c) {
            double h = dec(xr[c], dtype) + (bias ? dec(bias[c], dtype) : 0.0);
            double g = (do_norm && gamma) ? dec(gamma[c], dtype) : 1.0;
            out[r * n + c] = enc(do_norm ? h * inv * g : h, dtype);
        }
    }
}

/* Number of OpenMP threads the oracle runs with. */
int fo_orc_num_threads(void) {
#ifdef _OPENMP
    extern int omp_get_max_threads(void);
    return omp_get_max_threads();
#else
    return 1;
#endif
}
