/*
 * wsr_device.h - device building blocks of the weight-streaming kernels (gfx950, wave64).
 *
 * Design (CDNA4): a batch-1 GEMV reads each weight byte once and does one multiply-add per weight,
 * far below any matrix-core ridge, so it runs on the vector ALUs and is bound by HBM bandwidth.
 *  - A wavefront owns whole rows: its 64 lanes cover a row in 16-byte chunks, so every load
 *    instruction of the wave reads 1 KiB of one row, contiguous and aligned.
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

constexpr int WAVE = 64;

__device__ __forceinline__ u32x4 load_once(const u32x4* p) { return __builtin_nontemporal_load(p); }
__device__ __forceinline__ u32x4 load_reused(const u32x4* p) { return *p; }
__device__ __forceinline__ u32x4 zero4() { return u32x4{0u, 0u, 0u, 0u}; }

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

/* Butterfly sum over the 64 lanes.  Each step adds a value to its partner's, and a + b == b + a,
   so all lanes end with the same bits and the association order is fixed. */
__device__ __forceinline__ float wave_sum(float v) {
    v += dpp_f32<DPP_XOR1>(v);
    v += dpp_f32<DPP_XOR2>(v);
    v += dpp_f32<DPP_HALF_MIRROR>(v);
    v += dpp_f32<DPP_MIRROR>(v);
    v += __shfl_xor(v, 16);
    v += __shfl_xor(v, 32);
    return v;
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

   Rows [r0, r1) of matrix d at token `token`, R rows per pass over K.  A pass over K moves in steps
   of U chunks per lane (U * 64 chunks = U KiB per row per step); only a ragged last step masks its
   lanes.  Lane l accumulates chunks l, l + 64, l + 128, ... of each row in that order. */
template <int FMT, int R, int U>
__device__ __forceinline__ void rows16(const DevMat& d, int64_t r0, int64_t r1, int32_t token,
                                       int lane) {
    const u32x4* __restrict__ W = static_cast<const u32x4*>(d.w);
    const u32x4* __restrict__ x =
        reinterpret_cast<const u32x4*>(static_cast<const char*>(d.x) + token * d.x_stride);
    float* __restrict__ y = reinterpret_cast<float*>(reinterpret_cast<char*>(d.y) + token * d.y_stride);
    const int64_t nc = d.nc;
    constexpr int STEP = WAVE * U;
    for (int64_t i = r0; i < r1; i += R) {
        float acc[R];
#pragma unroll
        for (int r = 0; r < R; ++r) acc[r] = 0.f;
        for (int64_t c0 = 0; c0 < nc; c0 += STEP) {
            u32x4 xv[U], wv[R][U];
            if (c0 + STEP <= nc) {
#pragma unroll
                for (int u = 0; u < U; ++u) xv[u] = load_reused(x + c0 + u * WAVE + lane);
#pragma unroll
                for (int r = 0; r < R; ++r) {
                    if (i + r < r1) {
                        const u32x4* wr = W + (i + r) * nc + c0 + lane;
#pragma unroll
                        for (int u = 0; u < U; ++u) wv[r][u] = load_once(wr + u * WAVE);
                    } else {
#pragma unroll
                        for (int u = 0; u < U; ++u) wv[r][u] = zero4();
                    }
                }
            } else {
#pragma unroll
                for (int u = 0; u < U; ++u) {
                    const int64_t c = c0 + u * WAVE + lane;
                    xv[u] = c < nc ? load_reused(x + c) : zero4();
                }
#pragma unroll
                for (int r = 0; r < R; ++r) {
#pragma unroll
                    for (int u = 0; u < U; ++u) {
                        const int64_t c = c0 + u * WAVE + lane;
                        wv[r][u] = (i + r < r1 && c < nc) ? load_once(W + (i + r) * nc + c) : zero4();
                    }
                }
            }
#pragma unroll
            for (int r = 0; r < R; ++r)
#pragma unroll
                for (int u = 0; u < U; ++u) acc[r] = dot8<FMT>(wv[r][u], xv[u], acc[r]);
        }
#pragma unroll
        for (int r = 0; r < R; ++r) {
            const float s = wave_sum(acc[r]);
            if (lane == 0 && i + r < r1) y[i + r] = s;
        }
    }
}

/* ---- q4 rows -----------------------------------------------------------------------------------

   A 16-byte chunk of codes is exactly one block of 32 weights; lane l takes blocks l, l + 64, ...
   of each row, so a wave load reads 1 KiB of codes and each lane needs one scale per block.

   In-register decode: with v = q + 8 (the code XOR 8), masking a code word with 0x000F000F gives
   two fp16 subnormals v * 2^-24 (elements k and k + 4), and 0x00F000F0 gives 16 v * 2^-24; the
   same masks after a shift by 8 give the other two pairs, so one AND per pair decodes the word and
   the values are exact.  Packed dot products with activation pairs then sum, per block,
   Se = 2^-24 (sum_even q x + 8 Xe) and So = 2^-20 (sum_odd q x + 8 Xo), with Xe and Xo the
   block's activation sums over even and odd k; the offset terms are computed once per block from
   the activations alone and subtracted, and the block scale times 2^24 (exact) multiplies the
   result.  The offset is small (8 Xe, not the value magnitude 1024 + v of a normal fp16), so the
   fp32 sums keep nearly full precision, and a unit activation vector gives y = q * s exactly.
*/
constexpr uint32_t Q4_LO = 0x000F000Fu, Q4_HI = 0x00F000F0u;
constexpr uint32_t F16_OFS_EVEN = 0x00080008u;   /* 8 * 2^-24 in both halves (fp16 subnormal)   */
constexpr uint32_t F16_OFS_ODD = 0x00800080u;    /* 16 * 8 * 2^-24                              */

/* Activation pairs of one block, in the order the decode produces weights: for code dword d,
   p[4d] = (x[8d], x[8d+4]), p[4d+1] = (x[8d+1], x[8d+5]), p[4d+2] = (x[8d+2], x[8d+6]),
   p[4d+3] = (x[8d+3], x[8d+7]); plus the even/odd offset terms. */
struct Q4X {
    uint32_t p[16];
    float ce, co;
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
    q.ce = ce;
    q.co = co;
}

__device__ __forceinline__ float q4_block_dot(u32x4 w, const Q4X& q) {
    float se = 0.f, so = 0.f;
    const uint32_t wd[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
    for (int d = 0; d < 4; ++d) {
        const uint32_t t = wd[d] ^ 0x88888888u;
        const uint32_t t8 = t >> 8;
        se = dot2<FMT_F16>(t & Q4_LO, q.p[4 * d + 0], se);
        so = dot2<FMT_F16>(t & Q4_HI, q.p[4 * d + 1], so);
        se = dot2<FMT_F16>(t8 & Q4_LO, q.p[4 * d + 2], se);
        so = dot2<FMT_F16>(t8 & Q4_HI, q.p[4 * d + 3], so);
    }
    return (se - q.ce) + (so - q.co) * 0.0625f;   /* sum_k q x, in units of 2^-24 */
}

/* fp16 block scale times 2^24 (exact), undoing the 2^-24 unit of the decoded values. */
__device__ __forceinline__ float q4_scale(uint16_t b) {
    return (float)__builtin_bit_cast(_Float16, b) * 16777216.0f;
}

template <int R, int U>
__device__ __forceinline__ void rows_q4(const DevMat& d, int64_t r0, int64_t r1, int32_t token,
                                        int lane) {
    const u32x4* __restrict__ Wq = static_cast<const u32x4*>(d.w);
    const uint16_t* __restrict__ S = static_cast<const uint16_t*>(d.s);
    const u32x4* __restrict__ x =
        reinterpret_cast<const u32x4*>(static_cast<const char*>(d.x) + token * d.x_stride);
    float* __restrict__ y = reinterpret_cast<float*>(reinterpret_cast<char*>(d.y) + token * d.y_stride);
    const int64_t nb = d.nc;
    constexpr int STEP = WAVE * U;
    for (int64_t i = r0; i < r1; i += R) {
        float acc[R];
#pragma unroll
        for (int r = 0; r < R; ++r) acc[r] = 0.f;
        for (int64_t b0 = 0; b0 < nb; b0 += STEP) {
            u32x4 xv[U][4], wv[R][U];
            uint16_t sv[R][U];
            bool ok[U];
#pragma unroll
            for (int u = 0; u < U; ++u) ok[u] = b0 + u * WAVE + lane < nb;
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int64_t b = b0 + u * WAVE + lane;
#pragma unroll
                for (int j = 0; j < 4; ++j) xv[u][j] = ok[u] ? load_reused(x + 4 * b + j) : zero4();
            }
#pragma unroll
            for (int r = 0; r < R; ++r) {
#pragma unroll
                for (int u = 0; u < U; ++u) {
                    const int64_t b = b0 + u * WAVE + lane;
                    const bool live = i + r < r1 && ok[u];
                    wv[r][u] = live ? load_once(Wq + (i + r) * nb + b) : zero4();
                    sv[r][u] = live ? S[(i + r) * nb + b] : (uint16_t)0;
                }
            }
#pragma unroll
            for (int u = 0; u < U; ++u) {
                Q4X q;
                q4_prep(xv[u], q);
#pragma unroll
                for (int r = 0; r < R; ++r)
                    acc[r] = __builtin_fmaf(q4_scale(sv[r][u]), q4_block_dot(wv[r][u], q), acc[r]);
            }
        }
#pragma unroll
        for (int r = 0; r < R; ++r) {
            const float s = wave_sum(acc[r]);
            if (lane == 0 && i + r < r1) y[i + r] = s;
        }
    }
}

}  // namespace wsr

#endif
