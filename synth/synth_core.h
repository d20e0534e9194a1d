/*
 * synth_core.h - the generator's draws and encoders, compiled for the host (synth.c) and for the
 * GPU (synth_dev.hip) from this one definition, so both produce the same bits: everything below is
 * integer arithmetic, or IEEE double addition and multiplication built without contraction.
 * Part of the input generator only: neither the oracle nor the GPU library includes it.
 */
#ifndef SYNTH_CORE_H
#define SYNTH_CORE_H

#include <math.h>
#include <stdint.h>
#include <string.h>

#ifdef __HIPCC__
#define SYNTH_FN __host__ __device__ static inline
#else
#define SYNTH_FN static inline
#endif

#define SYNTH_GAMMA 0x9E3779B97F4A7C15ULL
#define SYNTH_SLOTS 65536
#define SYNTH_CAP (1ULL << 48)                         /* 2^64 / SYNTH_SLOTS */

SYNTH_FN uint64_t synth_mix64(uint64_t z) {
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
    return z ^ (z >> 31);
}

/* SplitMix64 output number c + 1 for counter c = (stream << 40) | e under `seed`. */
SYNTH_FN uint64_t synth_draw(uint64_t seed, uint64_t stream, uint64_t e) {
    const uint64_t c = (stream << 40) | (e & ((1ULL << 40) - 1));
    return synth_mix64(seed + (c + 1) * SYNTH_GAMMA);
}

SYNTH_FN double synth_top53(uint64_t u) { return (double)(u >> 11) * 0x1p-53; }

/* Round a double to a binary format with `mbits` stored significand bits and exponent bias `bias`
 * (fp16: 10, 15; bf16: 7, 127), nearest-even, with subnormals and overflow to infinity. */
SYNTH_FN uint16_t synth_enc_rne_slow(double v, int mbits, int bias) {
    uint64_t bits;
    memcpy(&bits, &v, 8);
    const uint16_t sign = (uint16_t)((bits >> 63) << 15);
    const int emax_field = 2 * bias + 1;               /* all-ones exponent field */
    const uint16_t inf = (uint16_t)(emax_field << mbits);
    if (isnan(v)) return sign | inf | (uint16_t)(1u << (mbits - 1));
    const double a = fabs(v);
    if (a == 0.0) return sign;
    if (isinf(a)) return sign | inf;
    int e;
    frexp(a, &e);                                       /* a in [2^(e-1), 2^e) */
    int ulp_exp = e - 1 - mbits;                        /* spacing of the format in that binade */
    const int ulp_min = 1 - bias - mbits;               /* spacing of the subnormals */
    if (ulp_exp < ulp_min) ulp_exp = ulp_min;
    const double r = rint(ldexp(a, -ulp_exp));          /* exact scaling, then nearest-even */
    uint32_t ri = (uint32_t)r;
    const uint32_t one = 1u << mbits;                   /* the implicit leading bit */
    if (ulp_exp == ulp_min && ri < one) return sign | (uint16_t)ri;  /* subnormal (or zero) */
    if (ri == 2 * one) { ri = one; ulp_exp += 1; }      /* rounding carried into the next binade */
    const int efield = ulp_exp + bias + mbits;          /* value = ri * 2^(efield - bias - mbits) */
    if (efield >= emax_field) return sign | inf;
    return sign | (uint16_t)((efield << mbits) | (ri - one));
}

/* Same rounding on the bit pattern when the result is a normal number of the target format:
 * keep the top mbits + 1 significand bits, adding just under half an ulp plus the kept lsb, so
 * that exact halves round to even. */
SYNTH_FN uint16_t synth_enc_rne(double v, int mbits, int bias) {
    uint64_t bits;
    memcpy(&bits, &v, 8);
    const int e = (int)((bits >> 52) & 0x7FF) - 1023;
    if (e < 1 - bias || e > bias) return synth_enc_rne_slow(v, mbits, bias);
    const int shift = 52 - mbits;
    const uint64_t mant = (bits & ((1ULL << 52) - 1)) | (1ULL << 52);
    uint64_t r = (mant + ((1ULL << (shift - 1)) - 1) + ((mant >> shift) & 1)) >> shift;
    int ef = e + bias;
    if (r >> (mbits + 1)) { r >>= 1; ef += 1; }         /* carry into the next binade */
    if (ef >= 2 * bias + 1) return synth_enc_rne_slow(v, mbits, bias);
    const uint16_t sign = (uint16_t)((bits >> 63) << 15);
    return sign | (uint16_t)((ef << mbits) | (uint16_t)(r & ((1u << mbits) - 1)));
}

SYNTH_FN uint16_t synth_enc16(double v, int fmt) {
    return fmt == 2 ? synth_enc_rne(v, 7, 127) : synth_enc_rne(v, 10, 15);
}

/* Walker alias draw: the top 16 bits pick a slot, the low 48 bits accept its code or take the
   alias. */
SYNTH_FN uint16_t synth_table_draw(const uint64_t* q, const uint16_t* alias, uint64_t u) {
    const unsigned i = (unsigned)(u >> 48);
    return (u & (SYNTH_CAP - 1)) < q[i] ? (uint16_t)i : alias[i];
}

/* Uniform on [-1, 1) on the 2^-23 grid. */
SYNTH_FN float synth_grid_value(uint64_t u) {
    const int64_t k = (int64_t)(u >> 40);
    return (float)(k - (1 << 23)) * 0x1p-23f;
}

/* Signed int4 uniform on {-8..7}. */
SYNTH_FN int synth_int4_value(uint64_t u) { return (int)(u >> 60) - 8; }

/* Byte j of a packed int4 stream starting at element e0 (even): elements e0 + 2j (low nibble) and
   e0 + 2j + 1 (high nibble). */
SYNTH_FN uint8_t synth_q4_byte(uint64_t seed, uint64_t stream, uint64_t e0, int64_t j) {
    const int lo = synth_int4_value(synth_draw(seed, stream, e0 + 2 * (uint64_t)j));
    const int hi = synth_int4_value(synth_draw(seed, stream, e0 + 2 * (uint64_t)j + 1));
    return (uint8_t)((lo & 0xF) | ((hi & 0xF) << 4));
}

/* Signed int8 uniform on {-128..127}: top 8 bits of the draw minus 128. */
SYNTH_FN int8_t synth_int8_value(uint64_t u) { return (int8_t)((int)(u >> 56) - 128); }

/* Uniform on [lo, hi), rounded to fp16 / bf16. */
SYNTH_FN uint16_t synth_uniform16_value(uint64_t u, double lo, double hi, int fmt) {
    return synth_enc16(lo + (hi - lo) * synth_top53(u), fmt);
}

#endif
