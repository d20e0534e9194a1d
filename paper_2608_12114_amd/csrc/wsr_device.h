/*
 * wsr_device.h - device building blocks of the weight-streaming kernels (gfx950, wave64).
 *
 * Design (CDNA4): a batch-1 GEMV reads each weight byte once and does one multiply-add per weight,
 * far below any matrix-core ridge, so it runs on the vector ALUs and is bound by HBM bandwidth.
 *  - A wavefront owns whole rows: its 64 lanes cover a row in 16-byte chunks, so every load
 *    instruction of the wave reads 1 KiB of one row, contiguous and aligned.
 *  - Row indices are wave-uniform values held in scalar registers (the wave id goes through
 *    readfirstlane), so row bases, table reads and loop control run on the scalar unit and the
 *    vector ALUs only decode and multiply.  Pointers are global-address-space, giving plain global
 *    loads with a scalar base and a 32-bit lane offset.
 *  - Weights are loaded non-temporally (each byte is used once); activations use the normal cache
 *    path, since every row of the matrix rereads them.
 *  - Each lane accumulates in fp32 with packed two-element dot products (v_dot2c_f32_f16 /
 *    v_dot2c_f32_bf16); a row's 64 lane sums are combined with DPP lane moves inside each 16-lane
 *    row and two cross-row swaps, so LDS is needed only where several waves share a result.
 *  - Every accumulation order is fixed, so results do not depend on where the operands live, on the
 *    grid size or on which wave handled which row.
 */
#ifndef WSR_DEVICE_H
#define WSR_DEVICE_H

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "wsr_internal.h"

namespace wsr {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef _Float16 h2_t __attribute__((ext_vector_type(2)));
typedef __bf16 b2_t __attribute__((ext_vector_type(2)));

/* global-address-space views of caller pointers */
typedef __attribute__((address_space(1))) const u32x4 g_u32x4;
typedef __attribute__((address_space(1))) const uint16_t g_u16;
typedef __attribute__((address_space(1))) float g_f32;

constexpr int WAVE = 64;

template <typename T>
__device__ __forceinline__ T as_global(const void* p) { return (T)p; }

__device__ __forceinline__ u32x4 load_once(g_u32x4* p) { return __builtin_nontemporal_load(p); }
__device__ __forceinline__ u32x4 load_reused(g_u32x4* p) { return *p; }
__device__ __forceinline__ u32x4 zero4() { return u32x4{0u, 0u, 0u, 0u}; }

/* The wave's index inside its block, as a uniform (scalar) value. */
/* Raw buffer access: a wave-uniform base in a scalar resource, a 32-bit lane offset, a scalar
   offset and an immediate, with no per-lane address arithmetic.  Every access here is in bounds
   by construction, so the resource's range check is left open (num_records = 2^32 - 1); the word
   0x00020000 is the gfx9 family's format for untyped buffer access.  aux 2 marks a load
   non-temporal (read once). */
typedef __amdgpu_buffer_rsrc_t rsrc_t;
__device__ __forceinline__ rsrc_t buffer_of(const void* base) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, -1, 0x00020000);
}
__device__ __forceinline__ u32x4 buf_once(rsrc_t r, uint32_t v, uint32_t s) {
    return __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(r, v, s, 2));
}
__device__ __forceinline__ u32x4 buf_reused(rsrc_t r, uint32_t v, uint32_t s) {
    return __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(r, v, s, 0));
}
__device__ __forceinline__ uint32_t buf_u16(rsrc_t r, uint32_t v, uint32_t s) {
    return __builtin_amdgcn_raw_buffer_load_b16(r, v, s, 0);
}
/* 16 bytes per lane from memory straight into LDS: lane i's bytes land at lds + 16 i (lds
   wave-uniform).  The load counts in vmcnt like any other; nothing orders a later LDS read of the
   same bytes after it except an explicit wait (wait_vm). */
__device__ __forceinline__ void buf_to_lds(rsrc_t r, u32x4* lds, uint32_t v, uint32_t s) {
    __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (__attribute__((address_space(3))) void*)lds, 16, v, s, 0, 0);
}

/* A wave-uniform pointer held in scalar registers, so that a load from it plus a 32-bit lane
   offset and a constant takes the scalar-base form (no per-lane address arithmetic). */
__device__ __forceinline__ const char* uniform_ptr(const char* p) {
    const uint64_t v = reinterpret_cast<uint64_t>(p);
    const uint64_t lo = (uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)v);
    const uint64_t hi = (uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)(v >> 32));
    return reinterpret_cast<const char*>(hi << 32 | lo);
}

__device__ __forceinline__ int wave_in_block() {
    return __builtin_amdgcn_readfirstlane((int)(threadIdx.x / WAVE));
}

/* acc + a.lo*b.lo + a.hi*b.hi for two packed 16-bit pairs, fp32 accumulate. */
template <int FMT>
__device__ __forceinline__ float dot2(uint32_t a, uint32_t b, float acc) {
    if constexpr (FMT == FMT_BF16)
        return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(b2_t, a), __builtin_bit_cast(b2_t, b),
                                               acc, false);
    else
        return __builtin_amdgcn_fdot2(__builtin_bit_cast(h2_t, a), __builtin_bit_cast(h2_t, b), acc,
                                      false);
}

/* Eight products of one 16-byte chunk, in element order. */
template <int FMT>
__device__ __forceinline__ float dot8(u32x4 w, u32x4 x, float acc) {
    acc = dot2<FMT>(w.x, x.x, acc);
    acc = dot2<FMT>(w.y, x.y, acc);
    acc = dot2<FMT>(w.z, x.z, acc);
    acc = dot2<FMT>(w.w, x.w, acc);
    return acc;
}

/* ---- wavefront reductions ------------------------------------------------------------------ */

/* DPP controls: quad permutes, then mirrors inside 8- and 16-lane groups. */
constexpr int DPP_XOR1 = 0xB1;          /* quad_perm [1,0,3,2] */
constexpr int DPP_XOR2 = 0x4E;          /* quad_perm [2,3,0,1] */
constexpr int DPP_HALF_MIRROR = 0x141;  /* lane i <-> 7-i inside each 8 */
constexpr int DPP_MIRROR = 0x140;       /* lane i <-> 15-i inside each 16 */

template <int CTRL>
__device__ __forceinline__ float dpp_f32(float v) {
    return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), CTRL,
                                                                 0xF, 0xF, false));
}

template <int CTRL>
__device__ __forceinline__ double dpp_f64(double v) {
    uint64_t u = __builtin_bit_cast(uint64_t, v);
    int lo = __builtin_amdgcn_update_dpp(0, (int)(uint32_t)u, CTRL, 0xF, 0xF, false);
    int hi = __builtin_amdgcn_update_dpp(0, (int)(uint32_t)(u >> 32), CTRL, 0xF, 0xF, false);
    return __builtin_bit_cast(double, ((uint64_t)(uint32_t)hi << 32) | (uint32_t)lo);
}

/* Lane exchanges of the row reductions, in the order they are applied: lanes 32 apart, 16 apart,
   mirrored inside each 16-lane row (i <-> 15 - i), then the two quad swaps and the mirror inside
   each 8-lane half.  Each step pairs every lane with one partner, and together they join all 64. */
/* The six exchanges of a wave reduction, in the order every reduction here uses.  Level k pairs
   lane l with a partner that differs from l in lane bit 5 - k, and before level k every lane
   differing from l only in lower bits holds the same set of partial sums, so the extra low bits
   flipped by the mirrors do not matter: level 0 l ^ 32, level 1 l ^ 16, level 2 the row mirror
   (l ^ 15), level 3 the half-row mirror (l ^ 7), level 4 l ^ 2, level 5 l ^ 1. */
template <int LEVEL>
__device__ __forceinline__ float xchg(float v) {
    if constexpr (LEVEL == 0) return __shfl_xor(v, 32);
    else if constexpr (LEVEL == 1) return __shfl_xor(v, 16);
    else if constexpr (LEVEL == 2) return dpp_f32<DPP_MIRROR>(v);
    else if constexpr (LEVEL == 3) return dpp_f32<DPP_HALF_MIRROR>(v);
    else if constexpr (LEVEL == 4) return dpp_f32<DPP_XOR2>(v);
    else return dpp_f32<DPP_XOR1>(v);
}

/* One transposed step: lanes whose `bit` is set keep the upper half of the row list and send the
   lower half to their partner, which keeps the lower half. */
template <int LEVEL, int N>
__device__ __forceinline__ void halve_rows(float (&a)[N], int n, bool upper) {
    const int h = n / 2;
#pragma unroll
    for (int j = 0; j < N / 2; ++j) {
        if (j < h) {
            const float send = upper ? a[j] : a[j + h];
            const float keep = upper ? a[j + h] : a[j];
            a[j] = keep + xchg<LEVEL>(send);
        }
    }
}

/* Totals over the 64 lanes of N per-lane partial sums (N = 1, 2, 4, ..., 256: rows, or rows times
   activation columns).  The first min(log2 N, 6) exchanges split the list between partner lanes
   instead of duplicating it, so N sums cost about as much as one.  Afterwards, for N <= 64, lane l
   holds the total of entry l / (64 / N) in a[0]; for N > 64, lane l holds the totals of entries
   l * (N / 64) + j in a[j], j < N / 64.  Every entry is summed by the same tree of pairwise additions
   whatever N is (each level adds a lane's partial to its partner's, and a + b == b + a), so a
   result does not depend on how rows or columns were grouped. */
template <int LEVEL, int N>
__device__ __forceinline__ void halve_level(float (&a)[N], int lane) {
    constexpr int n = N >> LEVEL;                 /* entries still held before this level */
    if constexpr (n >= 2) halve_rows<LEVEL, N>(a, n, lane & (32 >> LEVEL));
}

template <int N>
__device__ __forceinline__ void wave_sum_entries(float (&a)[N], int lane) {
    static_assert(N >= 1 && N <= 256 && (N & (N - 1)) == 0, "N must be a power of two up to 256");
    halve_level<0, N>(a, lane);
    halve_level<1, N>(a, lane);
    halve_level<2, N>(a, lane);
    halve_level<3, N>(a, lane);
    halve_level<4, N>(a, lane);
    halve_level<5, N>(a, lane);
    if constexpr (N < 2) a[0] += xchg<0>(a[0]);
    if constexpr (N < 4) a[0] += xchg<1>(a[0]);
    if constexpr (N < 8) a[0] += xchg<2>(a[0]);
    if constexpr (N < 16) a[0] += xchg<3>(a[0]);
    if constexpr (N < 32) a[0] += xchg<4>(a[0]);
    if constexpr (N < 64) a[0] += xchg<5>(a[0]);
}

template <int N>
__device__ __forceinline__ float wave_sum_rows(float (&a)[N], int lane) {
    static_assert(N <= 64, "one total per lane needs N <= 64");
    wave_sum_entries<N>(a, lane);
    return a[0];
}

/* Single-row form: every lane ends with the same total. */
__device__ __forceinline__ float wave_sum(float v) {
    float a[1] = {v};
    return wave_sum_rows<1>(a, 0);
}

__device__ __forceinline__ double wave_sum(double v) {
    v += dpp_f64<DPP_XOR1>(v);
    v += dpp_f64<DPP_XOR2>(v);
    v += dpp_f64<DPP_HALF_MIRROR>(v);
    v += dpp_f64<DPP_MIRROR>(v);
    v += __shfl_xor(v, 16);
    v += __shfl_xor(v, 32);
    return v;
}

/* ---- 16-bit rows -------------------------------------------------------------------------------

   Rows [i, i + R) of matrix d (i wave-uniform, all R rows valid).  A pass over K moves in steps of
   U chunks per lane (U * 64 chunks = U KiB per row per step); only a ragged last step masks its
   lanes.  Lane l accumulates chunks l, l + 64, l + 128, ... of each row in that order, whatever R
   and U are, so every row's result is independent of how rows were grouped. */
template <int FMT, int R, int U>
__device__ __forceinline__ void group16(const char* W, g_u32x4* x, g_f32* y, int64_t nc, int64_t i,
                                        int lane) {
    constexpr int STEP = WAVE * U;
    float acc[R];
    g_u32x4* wr[R];
#pragma unroll
    for (int r = 0; r < R; ++r) {
        acc[r] = 0.f;
        wr[r] = as_global<g_u32x4*>(W + (i + r) * nc * 16);
    }
    int64_t c0 = 0;
    for (; c0 + STEP <= nc; c0 += STEP) {
        u32x4 xv[U], wv[R][U];
#pragma unroll
        for (int u = 0; u < U; ++u) xv[u] = load_reused(x + c0 + u * WAVE + lane);
#pragma unroll
        for (int r = 0; r < R; ++r)
#pragma unroll
            for (int u = 0; u < U; ++u) wv[r][u] = load_once(wr[r] + c0 + u * WAVE + lane);
#pragma unroll
        for (int r = 0; r < R; ++r)
#pragma unroll
            for (int u = 0; u < U; ++u) acc[r] = dot8<FMT>(wv[r][u], xv[u], acc[r]);
    }
    if (c0 < nc) {  /* ragged last step */
        u32x4 xv[U], wv[R][U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int64_t c = c0 + u * WAVE + lane;
            xv[u] = c < nc ? load_reused(x + c) : zero4();
#pragma unroll
            for (int r = 0; r < R; ++r) wv[r][u] = c < nc ? load_once(wr[r] + c) : zero4();
        }
#pragma unroll
        for (int r = 0; r < R; ++r)
#pragma unroll
            for (int u = 0; u < U; ++u) acc[r] = dot8<FMT>(wv[r][u], xv[u], acc[r]);
    }
    const float s = wave_sum_rows<R>(acc, lane);
    if ((lane & (WAVE / R - 1)) == 0) y[i + lane / (WAVE / R)] = s;
}

/* Rows [i, i + R) against T activation columns read with one pass over the weights.  Column t of
   the activations starts xcs 16-byte chunks after column 0 and its outputs ycs floats after
   column 0's.  Each lane accumulates every (row, column) pair over the same chunk sequence as
   group16, and the R * T sums go through the same reduction tree, so every column's result equals
   the single-column result bit for bit. */
template <int FMT, int R, int U, int T>
__device__ __forceinline__ void group16_cols(const char* W, g_u32x4* x, int64_t xcs, g_f32* y, int64_t ycs,
                                             int64_t nc, int64_t i, int lane) {
    constexpr int STEP = WAVE * U;
    constexpr int N = R * T;
    float acc[N];                                   /* entry t * R + r */
    g_u32x4* wr[R];
#pragma unroll
    for (int r = 0; r < R; ++r) wr[r] = as_global<g_u32x4*>(W + (i + r) * nc * 16);
#pragma unroll
    for (int e = 0; e < N; ++e) acc[e] = 0.f;
    int64_t c0 = 0;
    for (; c0 + STEP <= nc; c0 += STEP) {
        u32x4 xv[T][U], wv[R][U];
#pragma unroll
        for (int t = 0; t < T; ++t)
#pragma unroll
            for (int u = 0; u < U; ++u) xv[t][u] = load_reused(x + t * xcs + c0 + u * WAVE + lane);
#pragma unroll
        for (int r = 0; r < R; ++r)
#pragma unroll
            for (int u = 0; u < U; ++u) wv[r][u] = load_once(wr[r] + c0 + u * WAVE + lane);
#pragma unroll
        for (int t = 0; t < T; ++t)
#pragma unroll
            for (int r = 0; r < R; ++r)
#pragma unroll
                for (int u = 0; u < U; ++u) acc[t * R + r] = dot8<FMT>(wv[r][u], xv[t][u], acc[t * R + r]);
    }
    if (c0 < nc) {  /* ragged last step */
        u32x4 xv[T][U], wv[R][U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int64_t c = c0 + u * WAVE + lane;
#pragma unroll
            for (int t = 0; t < T; ++t) xv[t][u] = c < nc ? load_reused(x + t * xcs + c) : zero4();
#pragma unroll
            for (int r = 0; r < R; ++r) wv[r][u] = c < nc ? load_once(wr[r] + c) : zero4();
        }
#pragma unroll
        for (int t = 0; t < T; ++t)
#pragma unroll
            for (int r = 0; r < R; ++r)
#pragma unroll
                for (int u = 0; u < U; ++u) acc[t * R + r] = dot8<FMT>(wv[r][u], xv[t][u], acc[t * R + r]);
    }
    wave_sum_entries<N>(acc, lane);
    if constexpr (N <= WAVE) {
        if ((lane & (WAVE / N - 1)) == 0) {
            const int e = lane / (WAVE / N);
            y[(e / R) * ycs + i + e % R] = acc[0];
        }
    } else {
#pragma unroll
        for (int j = 0; j < N / WAVE; ++j) {
            const int e = lane * (N / WAVE) + j;
            y[(e / R) * ycs + i + e % R] = acc[j];
        }
    }
}

/* Launch shape of the multi-column 16-bit row loops: rows per wave R and chunks per lane per step U
   for T columns.  A step loads R U weight chunks and T U activation chunks per lane, so tall row
   groups keep the activation reloads (from L2) below the weight stream; measured on the 70B
   sweep, these shapes hold the weight stream at 7.1, 6.9, 6.5 and 4.6 TB/s for T = 2, 4, 8, 16. */
template <int T> struct Cols16 { static constexpr int R = 1, U = 8; };
template <> struct Cols16<2> { static constexpr int R = 4, U = 4; };
template <> struct Cols16<4> { static constexpr int R = 8, U = 1; };
template <> struct Cols16<8> { static constexpr int R = 16, U = 1; };
template <> struct Cols16<16> { static constexpr int R = 8, U = 1; };

/* Rows [r0, r1) of matrix d for tokens token0 .. token0 + T - 1 in one pass over the weights. */
template <int FMT, int T, int R = Cols16<T>::R, int U = Cols16<T>::U>
__device__ __forceinline__ void rows16_cols(const DevMat& d, int64_t r0, int64_t r1, int32_t token0,
                                            int lane) {
    const char* W = static_cast<const char*>(d.w);
    g_u32x4* x = as_global<g_u32x4*>(static_cast<const char*>(d.x) + token0 * d.x_stride);
    g_f32* y = as_global<g_f32*>(reinterpret_cast<char*>(d.y) + token0 * d.y_stride);
    const int64_t xcs = d.x_stride / 16, ycs = d.y_stride / 4;
    int64_t i = r0;
    for (; i + R <= r1; i += R) group16_cols<FMT, R, U, T>(W, x, xcs, y, ycs, d.nc, i, lane);
    for (; i < r1; ++i) group16_cols<FMT, 1, U, T>(W, x, xcs, y, ycs, d.nc, i, lane);
}

/* Rows [r0, r1) of matrix d at token `token` (r0, r1 wave-uniform): groups of R rows, then the
   remaining rows one at a time. */
template <int FMT, int R, int U>
__device__ __forceinline__ void rows16(const DevMat& d, int64_t r0, int64_t r1, int32_t token,
                                       int lane) {
    const char* W = static_cast<const char*>(d.w);
    g_u32x4* x = as_global<g_u32x4*>(static_cast<const char*>(d.x) + token * d.x_stride);
    g_f32* y = as_global<g_f32*>(reinterpret_cast<char*>(d.y) + token * d.y_stride);
    int64_t i = r0;
    for (; i + R <= r1; i += R) group16<FMT, R, U>(W, x, y, d.nc, i, lane);
    for (; i < r1; ++i) group16<FMT, 1, U>(W, x, y, d.nc, i, lane);
}

/* ---- q4 rows -----------------------------------------------------------------------------------

   A 16-byte chunk of codes is exactly one block of 32 weights; lane l takes blocks l, l + 64, ...
   of each row, so a wave load reads 1 KiB of codes and each lane needs one scale per block.

   In-register decode: with v = q + 8 (the code XOR 8), masking a code word with 0x000F000F gives
   two fp16 subnormals v * 2^-24 (elements k and k + 4), and 0x00F000F0 gives 16 v * 2^-24; the
   same masks after a shift by 8 give the other two pairs.  XOR and AND fuse into one three-input
   bit operation, so a code word of 8 weights costs four bit operations, one shift and four packed
   dot products, and the decoded values are exact.  Per block the dot products sum to
   Se = 2^-24 (sum_even q x + 8 Xe) and So = 2^-20 (sum_odd q x + 8 Xo), Xe and Xo being the block's
   activation sums over even and odd k; Se + So / 16 - 2^-24 (8 Xe + 8 Xo) is sum q x in units of
   2^-24, where the offset term depends on the activations only and is formed once per block and
   shared by the R rows.  The row total is scaled by 2^24 at the end (exact).  The offset is small
   (8 times an activation sum), so the fp32 sums keep nearly full precision, and a unit activation
   vector gives y = q * s exactly. */
constexpr uint32_t Q4_SIGN = 0x88888888u;
constexpr uint32_t Q4_LO = 0x000F000Fu, Q4_HI = 0x00F000F0u;
constexpr uint32_t F16_OFS_EVEN = 0x00080008u;   /* 8 * 2^-24 in both halves (fp16 subnormal)   */
constexpr uint32_t F16_OFS_ODD = 0x00800080u;    /* 16 * 8 * 2^-24                              */

/* Activation pairs of one block, in the order the decode produces weights: for code dword d,
   p[4d] = (x[8d], x[8d+4]), p[4d+1] = (x[8d+1], x[8d+5]), p[4d+2] = (x[8d+2], x[8d+6]),
   p[4d+3] = (x[8d+3], x[8d+7]); plus the block's offset term. */
struct Q4X {
    uint32_t p[16];
    float off;
};

__device__ __forceinline__ void q4_prep(const u32x4 (&xv)[4], Q4X& q) {
#pragma unroll
    for (int d = 0; d < 4; ++d) {
        const uint32_t X0 = xv[d].x, X1 = xv[d].y, X2 = xv[d].z, X3 = xv[d].w;
        q.p[4 * d + 0] = __builtin_amdgcn_perm(X2, X0, 0x05040100u);
        q.p[4 * d + 1] = __builtin_amdgcn_perm(X2, X0, 0x07060302u);
        q.p[4 * d + 2] = __builtin_amdgcn_perm(X3, X1, 0x05040100u);
        q.p[4 * d + 3] = __builtin_amdgcn_perm(X3, X1, 0x07060302u);
    }
    float ce = 0.f, co = 0.f;
#pragma unroll
    for (int d = 0; d < 4; ++d) {
        ce = dot2<FMT_F16>(F16_OFS_EVEN, q.p[4 * d + 0], ce);
        co = dot2<FMT_F16>(F16_OFS_ODD, q.p[4 * d + 1], co);
        ce = dot2<FMT_F16>(F16_OFS_EVEN, q.p[4 * d + 2], ce);
        co = dot2<FMT_F16>(F16_OFS_ODD, q.p[4 * d + 3], co);
    }
    q.off = __builtin_fmaf(co, 0.0625f, ce);
}

/* sum_k q x over one block, in units of 2^-24. */
__device__ __forceinline__ float q4_block_dot(u32x4 w, const Q4X& q) {
    float se = 0.f, so = 0.f;
    const uint32_t wd[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
    for (int d = 0; d < 4; ++d) {
        const uint32_t w0 = wd[d], w8 = wd[d] >> 8;
        se = dot2<FMT_F16>((w0 ^ Q4_SIGN) & Q4_LO, q.p[4 * d + 0], se);
        so = dot2<FMT_F16>((w0 ^ Q4_SIGN) & Q4_HI, q.p[4 * d + 1], so);
        se = dot2<FMT_F16>((w8 ^ Q4_SIGN) & Q4_LO, q.p[4 * d + 2], se);
        so = dot2<FMT_F16>((w8 ^ Q4_SIGN) & Q4_HI, q.p[4 * d + 3], so);
    }
    return __builtin_fmaf(so, 0.0625f, se) - q.off;
}

__device__ __forceinline__ float f16_bits_to_f32(uint16_t b) {
    return (float)__builtin_bit_cast(_Float16, b);
}

/* Registers of one step of R rows: U blocks per lane, their scales and the activations. */
template <int R, int U>
struct Q4Step {
    u32x4 w[R][U];
    uint16_t s[R][U];
    u32x4 x[U][4];
};

/* Loads of the step at block b0 for rows wr[r] / sr[r] (all U * 64 blocks inside the row). */
template <int R, int U>
__device__ __forceinline__ void q4_load(Q4Step<R, U>& st, g_u32x4* const (&wr)[R], g_u16* const (&sr)[R],
                                        g_u32x4* x, int64_t b0, int lane) {
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
        for (int j = 0; j < 4; ++j) st.x[u][j] = load_reused(x + 4 * (b0 + u * WAVE + lane) + j);
#pragma unroll
    for (int r = 0; r < R; ++r)
#pragma unroll
        for (int u = 0; u < U; ++u) {
            st.w[r][u] = load_once(wr[r] + b0 + u * WAVE + lane);
            st.s[r][u] = sr[r][b0 + u * WAVE + lane];
        }
}

/* Same, for a ragged last step: lanes past the row end load nothing and contribute zero. */
template <int R, int U>
__device__ __forceinline__ void q4_load_masked(Q4Step<R, U>& st, g_u32x4* const (&wr)[R],
                                               g_u16* const (&sr)[R], g_u32x4* x, int64_t b0,
                                               int64_t nb, int lane) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
        const int64_t b = b0 + u * WAVE + lane;
        const bool ok = b < nb;
#pragma unroll
        for (int j = 0; j < 4; ++j) st.x[u][j] = ok ? load_reused(x + 4 * b + j) : zero4();
#pragma unroll
        for (int r = 0; r < R; ++r) {
            st.w[r][u] = ok ? load_once(wr[r] + b) : zero4();
            st.s[r][u] = ok ? sr[r][b] : (uint16_t)0;
        }
    }
}

template <int R, int U>
__device__ __forceinline__ void q4_compute(const Q4Step<R, U>& st, float (&acc)[R]) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
        Q4X q;
        q4_prep(st.x[u], q);
#pragma unroll
        for (int r = 0; r < R; ++r)
            acc[r] = __builtin_fmaf(f16_bits_to_f32(st.s[r][u]), q4_block_dot(st.w[r][u], q), acc[r]);
    }
}

template <int R>
__device__ __forceinline__ void q4_store(g_f32* y, int64_t i, float (&acc)[R], int lane) {
    const float s = wave_sum_rows<R>(acc, lane) * 16777216.0f;   /* undo the 2^-24 unit (exact) */
    if ((lane & (WAVE / R - 1)) == 0) y[i + lane / (WAVE / R)] = s;
#pragma unroll
    for (int r = 0; r < R; ++r) acc[r] = 0.f;
}

/* Rows [i, i + R), any block count: one step at a time. */
template <int R, int U>
__device__ __forceinline__ void q4_group(g_u32x4* Wq, g_u16* S, g_u32x4* x, g_f32* y, int64_t nb,
                                         int64_t i, int lane) {
    constexpr int STEP = WAVE * U;
    float acc[R];
    g_u32x4* wr[R];
    g_u16* sr[R];
#pragma unroll
    for (int r = 0; r < R; ++r) {
        acc[r] = 0.f;
        wr[r] = Wq + (i + r) * nb;
        sr[r] = S + (i + r) * nb;
    }
    for (int64_t b0 = 0; b0 < nb; b0 += STEP) {
        Q4Step<R, U> st;
        if (b0 + STEP <= nb) q4_load<R, U>(st, wr, sr, x, b0, lane);
        else q4_load_masked<R, U>(st, wr, sr, x, b0, nb, lane);
        q4_compute<R, U>(st, acc);
    }
    q4_store<R>(y, i, acc, lane);
}

/* Rows [i, i + R) of a q4 matrix against T activation columns in one pass over the codes: each
   row's block is decoded once per step and dotted with every column's activation pairs.  Per
   (row, column) the arithmetic and its order are those of q4_block_dot and q4_store, and the
   R * T totals share the reduction tree, so each column equals the single-column result bit for
   bit.  Column t of x starts xcs 16-byte chunks after column 0, its outputs ycs floats after. */
template <int R, int T>
__device__ __forceinline__ void q4_group_cols(g_u32x4* Wq, g_u16* S, g_u32x4* x, int64_t xcs, g_f32* y,
                                              int64_t ycs, int64_t nb, int64_t i, int lane) {
    constexpr int N = R * T;
    float acc[N];                                   /* entry t * R + r */
#pragma unroll
    for (int e = 0; e < N; ++e) acc[e] = 0.f;
    g_u32x4* wr[R];
    g_u16* sr[R];
#pragma unroll
    for (int r = 0; r < R; ++r) {
        wr[r] = Wq + (i + r) * nb;
        sr[r] = S + (i + r) * nb;
    }
    for (int64_t b0 = 0; b0 < nb; b0 += WAVE) {
        const int64_t b = b0 + lane;
        const bool ok = b < nb;
        u32x4 xv[T][4], wv[R];
        uint16_t sv[R];
#pragma unroll
        for (int t = 0; t < T; ++t)
#pragma unroll
            for (int j = 0; j < 4; ++j) xv[t][j] = ok ? load_reused(x + t * xcs + 4 * b + j) : zero4();
#pragma unroll
        for (int r = 0; r < R; ++r) {
            wv[r] = ok ? load_once(wr[r] + b) : zero4();
            sv[r] = ok ? sr[r][b] : (uint16_t)0;
        }
        uint32_t dec[R][16];                        /* decoded subnormal pairs, q4_block_dot's order */
#pragma unroll
        for (int r = 0; r < R; ++r) {
            const uint32_t wd[4] = {wv[r].x, wv[r].y, wv[r].z, wv[r].w};
#pragma unroll
            for (int d = 0; d < 4; ++d) {
                const uint32_t w0 = wd[d], w8 = wd[d] >> 8;
                dec[r][4 * d + 0] = (w0 ^ Q4_SIGN) & Q4_LO;
                dec[r][4 * d + 1] = (w0 ^ Q4_SIGN) & Q4_HI;
                dec[r][4 * d + 2] = (w8 ^ Q4_SIGN) & Q4_LO;
                dec[r][4 * d + 3] = (w8 ^ Q4_SIGN) & Q4_HI;
            }
        }
#pragma unroll
        for (int t = 0; t < T; ++t) {
            Q4X q;
            q4_prep(xv[t], q);
#pragma unroll
            for (int r = 0; r < R; ++r) {
                float se = 0.f, so = 0.f;
#pragma unroll
                for (int d = 0; d < 4; ++d) {
                    se = dot2<FMT_F16>(dec[r][4 * d + 0], q.p[4 * d + 0], se);
                    so = dot2<FMT_F16>(dec[r][4 * d + 1], q.p[4 * d + 1], so);
                    se = dot2<FMT_F16>(dec[r][4 * d + 2], q.p[4 * d + 2], se);
                    so = dot2<FMT_F16>(dec[r][4 * d + 3], q.p[4 * d + 3], so);
                }
                const float blk = __builtin_fmaf(so, 0.0625f, se) - q.off;
                acc[t * R + r] = __builtin_fmaf(f16_bits_to_f32(sv[r]), blk, acc[t * R + r]);
            }
        }
    }
    wave_sum_entries<N>(acc, lane);
    if constexpr (N <= WAVE) {
        if ((lane & (WAVE / N - 1)) == 0) {
            const int e = lane / (WAVE / N);
            y[(e / R) * ycs + i + e % R] = acc[0] * 16777216.0f;   /* undo the 2^-24 unit (exact) */
        }
    } else {
#pragma unroll
        for (int j = 0; j < N / WAVE; ++j) {
            const int e = lane * (N / WAVE) + j;
            y[(e / R) * ycs + i + e % R] = acc[j] * 16777216.0f;
        }
    }
}

/* Rows per wave of the multi-column q4 loop for T = 1, 2, 4, 8 columns (the T raw activation
   blocks and R decoded rows stay in registers, so T stops at 8).  A 16-byte code block needs 64
   bytes of activations per column, so a step reloads 4 T / R activation bytes (from L2) per code
   byte; with registers for only R T sums, that traffic, not HBM, sets the rate of these passes. */
template <int T> struct Cols4 { static constexpr int R = 8; };
template <> struct Cols4<2> { static constexpr int R = 4; };
template <> struct Cols4<4> { static constexpr int R = 4; };
template <> struct Cols4<8> { static constexpr int R = 2; };

/* Rows [r0, r1) of a q4 matrix for tokens token0 .. token0 + T - 1 in one pass over the codes. */
template <int T, int R = Cols4<T>::R>
__device__ __forceinline__ void rows_q4_cols(const DevMat& d, int64_t r0, int64_t r1, int32_t token0,
                                             int lane) {
    static_assert(T <= 8, "q4 takes at most 8 columns per pass");
    g_u32x4* Wq = as_global<g_u32x4*>(d.w);
    g_u16* S = as_global<g_u16*>(d.s);
    g_u32x4* x = as_global<g_u32x4*>(static_cast<const char*>(d.x) + token0 * d.x_stride);
    g_f32* y = as_global<g_f32*>(reinterpret_cast<char*>(d.y) + token0 * d.y_stride);
    const int64_t xcs = d.x_stride / 16, ycs = d.y_stride / 4;
    int64_t i = r0;
    for (; i + R <= r1; i += R) q4_group_cols<R, T>(Wq, S, x, xcs, y, ycs, d.nc, i, lane);
    for (; i < r1; ++i) q4_group_cols<1, T>(Wq, S, x, xcs, y, ycs, d.nc, i, lane);
}

/* ---- int8 rows with fp16 row scales -------------------------------------------------------------

   The paper's protocol format (Sec. 3.1): w[i,k] = q[i,k] * s[i], q two's-complement int8, one fp16
   scale per row.  A 16-byte chunk holds 16 codes; lane l takes chunks l, l + 64, ... of each row.
   Decode: with u = q + 128 (the code XOR 0x80), masking a code word with 0x00FF00FF gives two exact
   fp16 subnormals u * 2^-24 (codes 0 and 2 of the word) and the same after a shift by 8 gives codes
   1 and 3; XOR and AND fuse into one three-input bit operation, so a word of 4 codes costs two bit
   operations, one shift and two packed dot products.  Per chunk the products sum to
   2^-24 (sum q x + 128 X), X the chunk's activation sum; the offset 2^-24 * 128 X depends on the
   activations only and is formed once per chunk and shared by the rows.  The row total is scaled by
   2^24 (exact) and then by the row scale, so a unit activation vector gives y = q * s exactly. */
constexpr uint32_t I8_SIGN = 0x80808080u, I8_LOHALF = 0x00FF00FFu;
constexpr uint32_t F16_I8_OFS = 0x00800080u;       /* 128 * 2^-24 in both halves (fp16 subnormal) */

/* Activation pairs of one chunk in the order the decode produces codes: for code word d,
   p[2d] = (x[4d], x[4d+2]), p[2d+1] = (x[4d+1], x[4d+3]); plus the chunk's offset term. */
struct I8X {
    uint32_t p[8];
    float off;
};

__device__ __forceinline__ void i8_prep(u32x4 x0, u32x4 x1, I8X& q) {
    const uint32_t X[8] = {x0.x, x0.y, x0.z, x0.w, x1.x, x1.y, x1.z, x1.w};
    float off = 0.f;
#pragma unroll
    for (int d = 0; d < 4; ++d) {
        q.p[2 * d + 0] = __builtin_amdgcn_perm(X[2 * d + 1], X[2 * d], 0x05040100u);
        q.p[2 * d + 1] = __builtin_amdgcn_perm(X[2 * d + 1], X[2 * d], 0x07060302u);
        off = dot2<FMT_F16>(F16_I8_OFS, q.p[2 * d + 0], off);
        off = dot2<FMT_F16>(F16_I8_OFS, q.p[2 * d + 1], off);
    }
    q.off = off;
}

/* sum_k q x over one chunk, in units of 2^-24. */
__device__ __forceinline__ float i8_chunk_dot(u32x4 w, const I8X& q) {
    const uint32_t wd[4] = {w.x, w.y, w.z, w.w};
    float t = 0.f;
#pragma unroll
    for (int d = 0; d < 4; ++d) {
        t = dot2<FMT_F16>((wd[d] ^ I8_SIGN) & I8_LOHALF, q.p[2 * d + 0], t);
        t = dot2<FMT_F16>((wd[d] >> 8 ^ 0x00800080u) & I8_LOHALF, q.p[2 * d + 1], t);
    }
    return t - q.off;
}

/* Rows [i, i + R) of an int8 matrix against T activation columns (T = 1: a single GEMV) in one
   pass over the codes.  Column t of x starts xcs 16-byte chunks after column 0 (two chunks of x
   per chunk of codes), its outputs ycs floats after.  Every (row, column) sum follows the same
   chunk sequence and reduction tree whatever R, U and T are, so results do not depend on them. */
template <int R, int U, int T>
__device__ __forceinline__ void group_i8(g_u32x4* Wq, const uint16_t* S, g_u32x4* x, int64_t xcs, g_f32* y,
                                         int64_t ycs, int64_t nc, int64_t i, int lane) {
    constexpr int STEP = WAVE * U;
    constexpr int N = R * T;
    float acc[N];                                   /* entry t * R + r */
#pragma unroll
    for (int e = 0; e < N; ++e) acc[e] = 0.f;
    g_u32x4* wr[R];
#pragma unroll
    for (int r = 0; r < R; ++r) wr[r] = Wq + (i + r) * nc;
    for (int64_t c0 = 0; c0 < nc; c0 += STEP) {
        u32x4 xv[T][U][2], wv[R][U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int64_t c = c0 + u * WAVE + lane;
            const bool ok = c < nc;
#pragma unroll
            for (int t = 0; t < T; ++t) {
                xv[t][u][0] = ok ? load_reused(x + t * xcs + 2 * c) : zero4();
                xv[t][u][1] = ok ? load_reused(x + t * xcs + 2 * c + 1) : zero4();
            }
#pragma unroll
            for (int r = 0; r < R; ++r) wv[r][u] = ok ? load_once(wr[r] + c) : zero4();
        }
#pragma unroll
        for (int u = 0; u < U; ++u)
#pragma unroll
            for (int t = 0; t < T; ++t) {
                I8X q;
                i8_prep(xv[t][u][0], xv[t][u][1], q);
#pragma unroll
                for (int r = 0; r < R; ++r) acc[t * R + r] += i8_chunk_dot(wv[r][u], q);
            }
    }
    wave_sum_entries<N>(acc, lane);
    auto out = [&](int e, float v) {
        const float rs = f16_bits_to_f32(S[i + e % R]);
        y[(e / R) * ycs + i + e % R] = v * 16777216.0f * rs;   /* 2^24 exact, then the row scale */
    };
    if constexpr (N <= WAVE) {
        if ((lane & (WAVE / N - 1)) == 0) out(lane / (WAVE / N), acc[0]);
    } else {
#pragma unroll
        for (int j = 0; j < N / WAVE; ++j) out(lane * (N / WAVE) + j, acc[j]);
    }
}

/* Rows per wave and chunks per lane per step of the int8 sweep loops for T columns (T <= 8): eight
   rows share each activation chunk's preparation, one chunk per lane per step keeps the register
   count low enough for several waves per SIMD. */
template <int T> struct ColsI8 { static constexpr int R = 8, U = 1; };
/* The same for the standalone int8 GEMV kernels (one group of R rows per wave). */
template <int T> struct GemvI8 { static constexpr int R = 4, U = 1; };
template <> struct GemvI8<2> { static constexpr int R = 4, U = 2; };
template <> struct GemvI8<4> { static constexpr int R = 8, U = 1; };
template <> struct GemvI8<8> { static constexpr int R = 8, U = 1; };
/* Register sets in flight in the single-column int8 row loop. */
constexpr int I8_NB = 3;

/* Rows [r0, r1) of an int8 matrix for tokens token0 .. token0 + T - 1 in one pass over the codes. */
template <int T, int R = ColsI8<T>::R, int U = ColsI8<T>::U>
__device__ __forceinline__ void rows_i8(const DevMat& d, int64_t r0, int64_t r1, int32_t token0, int lane) {
    static_assert(T <= 8, "int8 takes at most 8 columns per pass");
    g_u32x4* Wq = as_global<g_u32x4*>(d.w);
    const uint16_t* S = static_cast<const uint16_t*>(d.s);
    g_u32x4* x = as_global<g_u32x4*>(static_cast<const char*>(d.x) + token0 * d.x_stride);
    g_f32* y = as_global<g_f32*>(reinterpret_cast<char*>(d.y) + token0 * d.y_stride);
    const int64_t xcs = d.x_stride / 16, ycs = d.y_stride / 4;
    int64_t i = r0;
    for (; i + R <= r1; i += R) group_i8<R, U, T>(Wq, S, x, xcs, y, ycs, d.nc, i, lane);
    for (; i < r1; ++i) group_i8<1, U, T>(Wq, S, x, xcs, y, ycs, d.nc, i, lane);
}

/* One step of the int8 row loop: R rows x U chunks of codes and the U activation chunk pairs. */
template <int R, int U>
struct I8Step {
    u32x4 w[R][U];
    u32x4 x[U][2];
};

/* Rows [r0, r1) of an int8 matrix, one column, with NB register sets in flight: while one unit
   (group of R rows, step) is decoded the loads of the next NB - 1 units are outstanding, across
   row-group boundaries, as in the q4 loop below.  Needs rows made of whole steps (nc a multiple of
   64 U); otherwise, and for the rows left over, group_i8 runs.  Every sum takes the chunks and
   the reduction tree of group_i8, so the results are those of rows_i8<1>. */
template <int R, int U, int NB>
__device__ __forceinline__ void rows_i8_pipe(const DevMat& d, int64_t r0, int64_t r1, int32_t token, int lane) {
    g_u32x4* Wq = as_global<g_u32x4*>(d.w);
    const uint16_t* S = static_cast<const uint16_t*>(d.s);
    g_u32x4* x = as_global<g_u32x4*>(static_cast<const char*>(d.x) + token * d.x_stride);
    g_f32* y = as_global<g_f32*>(reinterpret_cast<char*>(d.y) + token * d.y_stride);
    const int64_t nc = d.nc;
    constexpr int STEP = WAVE * U;
    const int64_t ngroups = (r1 - r0) / R;
    int64_t i = r0;
    if (ngroups > 0 && nc > 0 && nc % STEP == 0) {
        const int64_t steps = nc / STEP;                 /* steps per row group */
        const int64_t n = ngroups * steps;               /* units */
        float acc[R];
#pragma unroll
        for (int r = 0; r < R; ++r) acc[r] = 0.f;
        int64_t gl = 0, kl = 0;                          /* next unit to load   */
        int64_t gc = 0, kc = 0;                          /* next unit to decode */
        auto load = [&](I8Step<R, U>& st) {
            const int64_t i0 = r0 + gl * R;
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int64_t c = kl * STEP + u * WAVE + lane;
                st.x[u][0] = load_reused(x + 2 * c);
                st.x[u][1] = load_reused(x + 2 * c + 1);
#pragma unroll
                for (int r = 0; r < R; ++r) st.w[r][u] = load_once(Wq + (i0 + r) * nc + c);
            }
            if (++kl == steps) { kl = 0; ++gl; }
        };
        auto decode = [&](const I8Step<R, U>& st) {
#pragma unroll
            for (int u = 0; u < U; ++u) {
                I8X q;
                i8_prep(st.x[u][0], st.x[u][1], q);
#pragma unroll
                for (int r = 0; r < R; ++r) acc[r] += i8_chunk_dot(st.w[r][u], q);
            }
            if (kc + 1 == steps) {
                const int64_t i0 = r0 + gc * R;
                wave_sum_entries<R>(acc, lane);
                if ((lane & (WAVE / R - 1)) == 0) {
                    const int e = lane / (WAVE / R);
                    y[i0 + e] = acc[0] * 16777216.0f * f16_bits_to_f32(S[i0 + e]);
                }
#pragma unroll
                for (int r = 0; r < R; ++r) acc[r] = 0.f;
            }
            if (++kc == steps) { kc = 0; ++gc; }
        };
        I8Step<R, U> buf[NB];
#pragma unroll
        for (int j = 0; j < NB - 1; ++j)
            if (j < n) load(buf[j]);
        int64_t u = 0;                                   /* buf[j] holds unit u + j, j < NB - 1 */
        for (; u + 2 * NB - 1 <= n; u += NB) {
#pragma unroll
            for (int j = 0; j < NB; ++j) {
                load(buf[(j + NB - 1) % NB]);            /* unit u + j + NB - 1 */
                __builtin_amdgcn_sched_barrier(0);       /* keep those loads ahead of the decode */
                decode(buf[j]);                          /* unit u + j */
            }
        }
#pragma unroll
        for (int j = 0; j < 2 * NB - 1; ++j) {
            if (u + j < n) {
                if (u + j + NB - 1 < n) load(buf[(j + NB - 1) % NB]);
                decode(buf[j % NB]);
            }
        }
        i = r0 + ngroups * R;
    }
    for (; i + R <= r1; i += R) group_i8<R, U, 1>(Wq, S, x, 0, y, 0, nc, i, lane);
    for (; i < r1; ++i) group_i8<1, U, 1>(Wq, S, x, 0, y, 0, nc, i, lane);
}

/* Rows [r0, r1) of a q4 matrix.  With NB >= 2, when rows hold whole steps (nb a multiple of 64 U),
   the units (group of R rows, step) run as one software pipeline over NB register sets: the loads
   of the NB - 1 units after the current one are in flight while it is decoded.  The main loop is
   unrolled by NB so every set is named statically and its loads are unconditional, which keeps
   the waits exact; the last units are decoded after it.  Remaining rows go one at a time. */
template <int R, int U, int NB = 2>
__device__ __forceinline__ void rows_q4(const DevMat& d, int64_t r0, int64_t r1, int32_t token,
                                        int lane) {
    g_u32x4* Wq = as_global<g_u32x4*>(d.w);
    g_u16* S = as_global<g_u16*>(d.s);
    g_u32x4* x = as_global<g_u32x4*>(static_cast<const char*>(d.x) + token * d.x_stride);
    g_f32* y = as_global<g_f32*>(reinterpret_cast<char*>(d.y) + token * d.y_stride);
    const int64_t nb = d.nc;
    constexpr int STEP = WAVE * U;
    const int64_t ngroups = (r1 - r0) / R;
    int64_t i_end = r0 + ngroups * R;
    if (NB < 2) {
        for (int64_t i = r0; i < i_end; i += R) q4_group<R, U>(Wq, S, x, y, nb, i, lane);
    } else if (ngroups > 0 && nb % STEP == 0 && nb > 0) {
        const int64_t steps = nb / STEP;                 /* steps per row group */
        const int64_t n = ngroups * steps;               /* units */
        float acc[R];
#pragma unroll
        for (int r = 0; r < R; ++r) acc[r] = 0.f;
        int64_t gl = 0, kl = 0;                          /* next unit to load    */
        int64_t gc = 0, kc = 0;                          /* next unit to decode  */
        /* Raw buffer loads: a resource per row group and a scalar offset per row and step (rows of a
           group lie within 2^28 bytes) over one lane offset, where 64-bit row pointers cost several
           scalar instructions per row and step (8B q4: 95 -> 25 scalar instructions per unit in the
           main loop, the same 164 registers; the rate moved by under 0.3 %, the outputs not at all). */
        const rsrc_t rx = buffer_of(uniform_ptr(static_cast<const char*>(d.x) + (int64_t)token * d.x_stride));
        rsrc_t rw = rx, rsc = rx;                        /* this group's codes and scales */
        const uint32_t vl = 16u * (uint32_t)lane, vx = 64u * (uint32_t)lane;
        const uint32_t rcb = (uint32_t)(nb * 16), rsb = (uint32_t)(nb * 2);   /* row bytes of codes, scales */
        auto load = [&](Q4Step<R, U>& st) {
            if (kl == 0) {
                const int64_t i = r0 + gl * R;
                rw = buffer_of(uniform_ptr(static_cast<const char*>(d.w) + i * nb * 16));
                rsc = buffer_of(uniform_ptr(static_cast<const char*>(d.s) + i * nb * 2));
            }
            const uint32_t kb = (uint32_t)(kl * STEP);   /* the step's first block */
#pragma unroll
            for (int u = 0; u < U; ++u)
#pragma unroll
                for (int j = 0; j < 4; ++j)
                    st.x[u][j] = buf_reused(rx, vx + (uint32_t)(4096 * u + 16 * j), 64u * kb);
#pragma unroll
            for (int r = 0; r < R; ++r)
#pragma unroll
                for (int u = 0; u < U; ++u) {
                    st.w[r][u] = buf_once(rw, vl + (uint32_t)(1024 * u), r * rcb + 16u * kb);
                    st.s[r][u] = (uint16_t)buf_u16(rsc, (vl >> 3) + (uint32_t)(128 * u), r * rsb + 2u * kb);
                }
            if (++kl == steps) { kl = 0; ++gl; }
        };
        auto decode = [&](const Q4Step<R, U>& st) {
            q4_compute<R, U>(st, acc);
            if (kc + 1 == steps) q4_store<R>(y, r0 + gc * R, acc, lane);
            if (++kc == steps) { kc = 0; ++gc; }
        };
        Q4Step<R, U> buf[NB];
#pragma unroll
        for (int j = 0; j < NB - 1; ++j)
            if (j < n) load(buf[j]);
        int64_t u = 0;                                   /* buf[j] holds unit u + j, j < NB - 1 */
        for (; u + 2 * NB - 1 <= n; u += NB) {
#pragma unroll
            for (int j = 0; j < NB; ++j) {
                load(buf[(j + NB - 1) % NB]);            /* unit u + j + NB - 1 */
                __builtin_amdgcn_sched_barrier(0);       /* keep those loads ahead of the decode */
                decode(buf[j]);                          /* unit u + j */
            }
        }
#pragma unroll
        for (int j = 0; j < 2 * NB - 1; ++j) {
            if (u + j < n) {
                if (u + j + NB - 1 < n) load(buf[(j + NB - 1) % NB]);
                decode(buf[j % NB]);
            }
        }
    } else {
        i_end = r0;
    }
    for (int64_t i = i_end; i < r1; ++i) q4_group<1, U>(Wq, S, x, y, nb, i, lane);
}

/* ceil(a / b) for a >= 0, b > 0.  A 64-bit division expands to a long dependent sequence on this
   target, so values that fit 32 bits (every range of a matrix below 4 GiB) take the 32-bit form. */
__device__ __forceinline__ int64_t ceil_div(int64_t a, int64_t b) {
    const uint64_t n = (uint64_t)(a + b - 1);
    if (((n | (uint64_t)b) >> 32) == 0) return (int64_t)((uint32_t)n / (uint32_t)b);
    return (int64_t)(n / (uint64_t)b);
}

/* Last matrix whose stream starts at or before byte lo: from the hint when it still holds, else by
   bisection over the dense offset array (8 bytes per matrix, so it stays in the scalar cache). */
__device__ __forceinline__ int first_matrix(const int64_t* __restrict__ cost, int nmat, int64_t lo, int hint) {
    int a = hint;
    if (cost[a] > lo) a = 0;
    if (a + 1 < nmat && cost[a + 1] <= lo) {
        int b = nmat - 1;
        while (a < b) {
            const int mid = (a + b + 1) >> 1;
            if (cost[mid] <= lo) a = mid; else b = mid - 1;
        }
    }
    return a;
}


template <int FMT, int R16, int U16, int RQ, int UQ, int QNB = 2, int T = 1, int RC = Cols16<T>::R,
          int UC = Cols16<T>::U, int RQC = Cols4<(T <= 8 ? T : 8)>::R>
__device__ __forceinline__ void stream_range(const DevMat* __restrict__ tab, const int64_t* __restrict__ cost,
                                             int nmat, int64_t lo, int64_t hi, int32_t token, int lane,
                                             int& hint) {
    for (int m = first_matrix(cost, nmat, lo, hint); m < nmat; ++m) {
        const DevMat d = tab[m];
        if (d.cost0 >= hi) break;
        hint = m;
        const int fmt = FMT ? FMT : d.fmt;
        const int64_t g = fmt == FMT_Q4 ? (T == 1 ? RQ : RQC)
                        : fmt == FMT_I8 ? ColsI8<(T <= 8 ? T : 8)>::R
                                        : (T == 1 ? R16 : RC);
        /* a byte range maps to rows by rounding both ends up to the next group of g rows */
        const int64_t r0 = lo > d.cost0 ? ceil_div(lo - d.cost0, d.row_bytes * g) * g : 0;
        const int64_t e1 = ceil_div(hi - d.cost0, d.row_bytes * g) * g;
        const int64_t r1 = d.M < e1 ? d.M : e1;
        if (r0 >= r1) continue;
        if constexpr (T == 1) {
            if ((FMT == 0 || FMT == FMT_F16) && fmt == FMT_F16)
                rows16<FMT_F16, R16, U16>(d, r0, r1, token, lane);
            else if ((FMT == 0 || FMT == FMT_BF16) && fmt == FMT_BF16)
                rows16<FMT_BF16, R16, U16>(d, r0, r1, token, lane);
            else if ((FMT == 0 || FMT == FMT_Q4) && fmt == FMT_Q4)
                rows_q4<RQ, UQ, QNB>(d, r0, r1, token, lane);
            else if ((FMT == 0 || FMT == FMT_I8) && fmt == FMT_I8)
                rows_i8_pipe<ColsI8<1>::R, ColsI8<1>::U, I8_NB>(d, r0, r1, token, lane);
        } else {                                        /* tokens token .. token + T - 1 together */
            if ((FMT == 0 || FMT == FMT_F16) && fmt == FMT_F16)
                rows16_cols<FMT_F16, T, RC, UC>(d, r0, r1, token, lane);
            else if ((FMT == 0 || FMT == FMT_BF16) && fmt == FMT_BF16)
                rows16_cols<FMT_BF16, T, RC, UC>(d, r0, r1, token, lane);
            else if constexpr (T <= 8) {
                if ((FMT == 0 || FMT == FMT_Q4) && fmt == FMT_Q4) rows_q4_cols<T, RQC>(d, r0, r1, token, lane);
                else if ((FMT == 0 || FMT == FMT_I8) && fmt == FMT_I8) rows_i8<T>(d, r0, r1, token, lane);
            }
        }
    }
}

}  // namespace wsr

#endif
