/*
 * oracle.c - CPU oracle for the weight-streaming read path.
 *
 * TEST INFRASTRUCTURE ONLY.  Only the tests, the smoke check and the benchmark's CPU-baseline leg
 * may load this library; the product path (the GPU library and its binding) never does, and the two
 * share no code, header, table or helper.
 *
 * Plain and slow on purpose, so that it can be checked against the paper by eye:
 *   - every stored value is decoded to double by the rules of its format (written out below);
 *   - every sum runs in double, in ascending index order, one term at a time;
 *   - rows are independent, so the optional OpenMP split over rows never changes a result.
 *
 * What it computes (the operations the paper measures, Sec. 3.1 "matched protocol" and Sec. 6.2):
 *   probe      s = sum_i buf[i]                       (the pure-read reference streams every byte)
 *   gemv16     y_i = sum_k W[i,k] * x[k]              (single-token GEMV over a row-major (M, K)
 *                                                      matrix with strides (K, 1), Alg. 1)
 *   q4 dequant w[i,k] = q[i,k] * s[i, floor(k / 32)]  (32 signed int4 codes share one fp16 scale)
 *   gemv_q4    y_i = sum_k w[i,k] * x[k]
 *   i8 dequant w[i,k] = q[i,k] * s[i]                 (the paper's packed int8 weights with fp16 row
 *                                                      scales, Sec. 3.1)
 *   gemv_i8    y_i = sum_k w[i,k] * x[k]
 * Build: gcc -O2 -ffp-contract=off -fPIC -shared -fopenmp (no fast-math, no contraction).
 */
#include <math.h>
#include <stdint.h>

/* ---- decoding of the storage formats ------------------------------------------------------ */

/* IEEE binary16: sign 1, exponent 5 (bias 15), fraction 10. */
double ora_f16_to_f64(uint16_t h) {
    int sign = h >> 15;
    int e = (h >> 10) & 0x1F;
    int f = h & 0x3FF;
    double v;
    if (e == 0)
        v = ldexp((double)f, -24);                /* subnormal: f * 2^-14 * 2^-10 */
    else if (e == 31)
        v = f ? NAN : INFINITY;
    else
        v = ldexp((double)(1024 + f), e - 25);    /* (1 + f/2^10) * 2^(e-15) */
    return sign ? -v : v;
}

/* bfloat16: sign 1, exponent 8 (bias 127), fraction 7. */
double ora_bf16_to_f64(uint16_t b) {
    int sign = b >> 15;
    int e = (b >> 7) & 0xFF;
    int f = b & 0x7F;
    double v;
    if (e == 0)
        v = ldexp((double)f, -133);               /* subnormal: f * 2^-126 * 2^-7 */
    else if (e == 255)
        v = f ? NAN : INFINITY;
    else
        v = ldexp((double)(128 + f), e - 134);    /* (1 + f/2^7) * 2^(e-127) */
    return sign ? -v : v;
}

/* Signed int4 in two's complement: codes 0..7 are 0..7, codes 8..15 are -8..-1. */
/* Two's-complement int8 from its byte. */
int ora_int8(unsigned byte) {
    byte &= 0xFF;
    return byte >= 128 ? (int)byte - 256 : (int)byte;
}

int ora_int4(unsigned code) {
    code &= 0xF;
    return code >= 8 ? (int)code - 16 : (int)code;
}

enum { ORA_F16 = 1, ORA_BF16 = 2 };

static double dec16(uint16_t v, int fmt) {
    return fmt == ORA_BF16 ? ora_bf16_to_f64(v) : ora_f16_to_f64(v);
}

/* ---- streaming-read probe ------------------------------------------------------------------ */

/* s = ((buf[0] + buf[1]) + buf[2]) + ... in double. */
double ora_probe_sum(const float* buf, int64_t n) {
    double s = 0.0;
    for (int64_t i = 0; i < n; ++i) s += (double)buf[i];
    return s;
}

/* ---- 16-bit GEMV ----------------------------------------------------------------------------- */

/* y[i] = sum_k W[i*K + k] * x[k], W and x both fp16 (fmt 1) or both bf16 (fmt 2). */
void ora_gemv16(const uint16_t* W, const uint16_t* x, int64_t M, int64_t K, int fmt, double* y,
                int threads) {
#pragma omp parallel for schedule(static) num_threads(threads > 0 ? threads : 1)
    for (int64_t i = 0; i < M; ++i) {
        double acc = 0.0;
        for (int64_t k = 0; k < K; ++k) acc += dec16(W[i * K + k], fmt) * dec16(x[k], fmt);
        y[i] = acc;
    }
}

/* ---- 4-bit block quantisation ------------------------------------------------------------------ */

/* Weight (i, k) of a q4 matrix: codes uint8 (M, K/2), element k of row i in byte k/2, low nibble for
 * even k and high nibble for odd k; scales fp16 (M, K/32). */
double ora_q4_weight(const uint8_t* Wq, const uint16_t* S, int64_t K, int64_t i, int64_t k) {
    uint8_t byte = Wq[i * (K / 2) + k / 2];
    unsigned code = (k % 2 == 0) ? (byte & 0xF) : (byte >> 4);
    int q = ora_int4(code);
    double s = ora_f16_to_f64(S[i * (K / 32) + k / 32]);
    return (double)q * s;
}

/* w (M, K) in double: every dequantised weight. */
void ora_dequant_q4(const uint8_t* Wq, const uint16_t* S, int64_t M, int64_t K, double* w) {
    for (int64_t i = 0; i < M; ++i)
        for (int64_t k = 0; k < K; ++k) w[i * K + k] = ora_q4_weight(Wq, S, K, i, k);
}

/* y[i] = sum_k w[i,k] * x[k], x fp16. */
void ora_gemv_q4(const uint8_t* Wq, const uint16_t* S, const uint16_t* x, int64_t M, int64_t K,
                 double* y, int threads) {
#pragma omp parallel for schedule(static) num_threads(threads > 0 ? threads : 1)
    for (int64_t i = 0; i < M; ++i) {
        double acc = 0.0;
        for (int64_t k = 0; k < K; ++k) acc += ora_q4_weight(Wq, S, K, i, k) * ora_f16_to_f64(x[k]);
        y[i] = acc;
    }
}

/* int8 weights with one fp16 scale per row (Sec. 3.1): Wq (M, K) bytes row-major, S[M]. */
double ora_i8_weight(const uint8_t* Wq, const uint16_t* S, int64_t K, int64_t i, int64_t k) {
    int q = ora_int8(Wq[i * K + k]);
    double row_scale = ora_f16_to_f64(S[i]);
    return (double)q * row_scale;
}

void ora_gemv_i8(const uint8_t* Wq, const uint16_t* S, const uint16_t* x, int64_t M, int64_t K,
                 double* y, int threads) {
#pragma omp parallel for schedule(static) num_threads(threads > 0 ? threads : 1)
    for (int64_t i = 0; i < M; ++i) {
        double acc = 0.0;
        for (int64_t k = 0; k < K; ++k) acc += ora_i8_weight(Wq, S, K, i, k) * ora_f16_to_f64(x[k]);
        y[i] = acc;
    }
}
