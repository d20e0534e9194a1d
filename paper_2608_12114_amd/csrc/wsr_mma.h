/*
 * wsr_mma.h - row loops of the batched decode sweep on the matrix cores (gfx950).
 *
 * Several tokens per pass over the weights turn the decode GEMV into a small matrix product
 * (Sec. 3.4, 5.2: several activation columns per weight read); from about four tokens on, the
 * vector-ALU loops of wsr_device.h are bound by their per-token dot products, so these loops hand
 * the products to v_mfma_f32_16x16x32.
 */
#ifndef WSR_MMA_H
#define WSR_MMA_H

#include <type_traits>

#include "wsr_device.h"
#include "wsr_mma_launch.h"

namespace wsr {

/* Rows [r0, r1) of matrix d that the byte range [lo, hi) of the weight stream covers.  A byte
   boundary maps to the first group of g rows starting at or after it, the same way for the ranges
   on both sides, so the ranges still cover each row once and break only between whole groups. */
struct RowRange {
    int64_t r0, r1;
};
__device__ __forceinline__ RowRange range_rows(const DevMat& d, int64_t lo, int64_t hi, int64_t g) {
    const int64_t r0 = lo > d.cost0 ? ceil_div(lo - d.cost0, d.row_bytes * g) * g : 0;
    const int64_t e1 = ceil_div(hi - d.cost0, d.row_bytes * g) * g;
    return RowRange{r0, d.M < e1 ? d.M : e1};
}

/* ---- matrix-core rows: up to 16 tokens per pass over the weights ----------------------------------

   With several tokens per pass the packed dot products of the loops above cost one instruction per
   weight pair per token, and from about four tokens on the vector ALUs, not HBM, set the rate.
   These loops hand the products to the matrix cores instead.  A wave owns tiles of 16 rows; per
   32-element slab of K it forms D = X^T W^T for the tile with one v_mfma_f32_16x16x32: the A
   operand holds 16 token slots of activations (slots past the pass's tokens repeat its first token
   and their results are never stored), the B operand 16 weight rows decoded to fp16.  Decoded
   weights are exact.  An int8 code becomes q as 1024 + (q + 128), formed by one bit operation,
   minus 1024 + 128 by one packed fp16 subtraction.  A q4 code becomes (q + 8) 2^-24, the fp16
   subnormal whose mantissa is the biased code, formed by one bit operation alone; the bias term
   8 2^-24 times the slab's activation sum is the same for every row, so one more matrix instruction
   per slab, with -8 2^-24 in every weight position, gives it for all tiles at once, and it enters
   each tile's instruction as the accumulator input.  A row group's q4 sums are scaled back by 2^24
   when stored, which is exact.  16-bit weights are used as stored.  Every product is exact in
   fp32, and the scales multiply the fp32 slab sums, but the matrix core adds a slab's products in
   an order of its own, so these results agree with the other loops within rounding, not bit for
   bit.
   Operand layout (checked on the device): lane i holds A[i%16][8(i/16)+j], B[8(i/16)+j][i%16] and
   D[4(i/16)+j][i%16].  K may be permuted inside a slab as long as A and B follow the same order;
   the decoders give (k0,k4,k1,k5,k2,k6,k3,k7) for a q4 word and (k0,k2,k1,k3,k4,k6,k5,k7) for two
   int8 words, and the activation loaders permute x to match.  A q4 scale covers one block of 32, so
   a slab is one block: the four words a lane loaded in chunk jj (block b0 + 4 jj + i/16 of row i%16) are
   transposed between the four 16-lane groups with two rounds of lane swaps, and each block's product is formed
   alone and added with its row's scale.  int8 scales are per row and multiply the finished sum. */
typedef _Float16 h8_t __attribute__((ext_vector_type(8)));
typedef __bf16 b8_t __attribute__((ext_vector_type(8)));
typedef float f4_t __attribute__((ext_vector_type(4)));

constexpr int MMA_TOKENS = 16;              /* token columns per tile                               */

template <int FMT>
__device__ __forceinline__ f4_t mma16(u32x4 a, u32x4 b, f4_t c) {
    if constexpr (FMT == FMT_BF16)
        return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(b8_t, a), __builtin_bit_cast(b8_t, b), c,
                                                       0, 0, 0);
    else
        return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(h8_t, a), __builtin_bit_cast(h8_t, b), c,
                                                      0, 0, 0);
}

/* v - bias in both fp16 halves of a word holding 1024 + v (exact for the small integers here). */
__device__ __forceinline__ uint32_t f16_sub_bias(uint32_t v, uint32_t neg_bias) {
    return __builtin_bit_cast(uint32_t, __builtin_bit_cast(h2_t, v) + __builtin_bit_cast(h2_t, neg_bias));
}

/* One q4 code word (code k in nibble k) as 8 fp16 subnormals (q + 8) 2^-24, order
   (k0,k4,k1,k5,k2,k6,k3,k7): code ^ 8 = q + 8 is the whole mantissa.  Taking the bias out here
   would cost a packed subtraction per pair; the slab's bias instruction takes it out instead
   (8B q4 at 16 tokens: 512 -> 386 vector instructions per unit of 64 rows x 256 weights). */
__device__ __forceinline__ u32x4 q4_word_sub(uint32_t w) {
    constexpr uint32_t M = 0x000F000Fu, E = 0x00080008u;
    return u32x4{(w & M) ^ E, ((w >> 4) & M) ^ E, ((w >> 8) & M) ^ E, ((w >> 12) & M) ^ E};
}
constexpr uint32_t Q4_NEG_BIAS = 0x80088008u;   /* -8 2^-24 in both fp16 halves  */
constexpr float Q4_UNSCALE = 0x1p24f;           /* what q4 sums are multiplied by */

/* Two int8 code words (codes k0..k3, k4..k7) as 8 fp16 integers, order (k0,k2,k1,k3,k4,k6,k5,k7). */
__device__ __forceinline__ u32x4 i8_words_f16(uint32_t w0, uint32_t w1) {
    constexpr uint32_t M = 0x00FF00FFu, E = 0x64806480u, NEG = 0xE480E480u;   /* 1024 + (code ^ 128); -1152 */
    return u32x4{f16_sub_bias((w0 & M) ^ E, NEG), f16_sub_bias(((w0 >> 8) & M) ^ E, NEG),
                 f16_sub_bias((w1 & M) ^ E, NEG), f16_sub_bias(((w1 >> 8) & M) ^ E, NEG)};
}

/* Eight activations x0..x7 (16 bytes) in the q4 decoder's order and in the int8 decoder's order. */
__device__ __forceinline__ u32x4 x8_q4_order(u32x4 u) {
    return u32x4{__builtin_amdgcn_perm(u.z, u.x, 0x05040100u), __builtin_amdgcn_perm(u.z, u.x, 0x07060302u),
                 __builtin_amdgcn_perm(u.w, u.y, 0x05040100u), __builtin_amdgcn_perm(u.w, u.y, 0x07060302u)};
}
__device__ __forceinline__ u32x4 x8_i8_order(u32x4 u) {
    return u32x4{__builtin_amdgcn_perm(u.y, u.x, 0x05040100u), __builtin_amdgcn_perm(u.y, u.x, 0x07060302u),
                 __builtin_amdgcn_perm(u.w, u.z, 0x05040100u), __builtin_amdgcn_perm(u.w, u.z, 0x07060302u)};
}

/* Lane group g (lanes 16g .. 16g + 15) holds the four words of block g in w; afterwards it holds
   word g of blocks 0, 1, 2, 3 in w.x, w.y, w.z, w.w (a 4 x 4 transpose between the groups). */
__device__ __forceinline__ u32x4 transpose_groups(u32x4 w) {
    const auto s02 = __builtin_amdgcn_permlane32_swap(w.x, w.z, false, false);
    const auto s13 = __builtin_amdgcn_permlane32_swap(w.y, w.w, false, false);
    const auto s01 = __builtin_amdgcn_permlane16_swap(s02[0], s13[0], false, false);
    const auto s23 = __builtin_amdgcn_permlane16_swap(s02[1], s13[1], false, false);
    return u32x4{s01[0], s01[1], s23[0], s23[1]};
}

/* Weights arrive as whole 128-byte lines.  The load of a tile's half b (rows 8 b .. 8 b + 7) gives
   lane (g, c) row 8 b + c % 8 of the tile at byte 16 (g + 4 (c / 8)) of the step's line, so eight
   lanes cover each line.  Moving the upper eight lanes of every 16-lane row of half 0 into the
   lower eight of half 1 and back (row shifts by 8; a lane whose source falls outside its row keeps
   its own value) leaves lane (g, c) with row c at byte 16 g of the line in the first register and
   at byte 64 + 16 g in the second: chunks 0 and 1 of the matrix instructions' layout. */
__device__ __forceinline__ void lines_to_slabs(u32x4& a, u32x4& b) {
    constexpr int ROW_SHL8 = 0x108, ROW_SHR8 = 0x118;
    u32x4 lo, hi;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        lo[k] = (uint32_t)__builtin_amdgcn_update_dpp((int)a[k], (int)b[k], ROW_SHR8, 0xF, 0xF, false);
        hi[k] = (uint32_t)__builtin_amdgcn_update_dpp((int)b[k], (int)a[k], ROW_SHL8, 0xF, 0xF, false);
    }
    a = lo;
    b = hi;
}

/* One step of the matrix-core loops: 128 bytes of every row.  The matrix instructions want chunk jj
   (jj = 0, 1) of lane group g at byte 64 jj + 16 g of the step, 64 bytes of each of 16 rows per
   register; the loads read the step as whole 128-byte lines, two per tile, and lines_to_slabs puts
   them in that layout (HBM delivers about half its rate to loads of 64 bytes of each of 16 rows).
   SLABS is the number of matrix instructions per tile and step, K the weights per row and step. */
template <int FMT> struct MmaStep { static constexpr int J = 2, SLABS = 2, K = 64; };     /* 8 per chunk   */
template <> struct MmaStep<FMT_Q4> { static constexpr int J = 2, SLABS = 8, K = 256; };   /* 32 per chunk  */
template <> struct MmaStep<FMT_I8> { static constexpr int J = 2, SLABS = 4, K = 128; };   /* 16 per chunk  */

/* Registers of one unit (a group of NT tiles, one step): the chunks of each tile and the scales
   (q4: the step's eight block scales of each tile's row, as fp16 pairs; int8: each tile's row
   scale).  The activations go through LDS. */
template <int FMT, int NT>
struct MmaUnit {
    static constexpr int J = MmaStep<FMT>::J, SL = MmaStep<FMT>::SLABS;
    static constexpr int NS = FMT == FMT_Q4 ? 4 : 1;
    u32x4 w[NT][J];
    uint32_t s[NT][NS];
};

/* Byte offset of slab s's eight activations within a step, past the lane group's own offset
   (16 g, or 32 g for int8): 16-bit and q4 slab s covers weights 32 s .. 32 s + 31 of the step
   (q4: one block), int8 slab s half s % 2 of chunk s / 2. */
template <int FMT>
constexpr int mma_x_byte(int s) { return FMT == FMT_I8 ? 128 * (s / 2) + 16 * (s % 2) : 64 * s; }

__device__ __forceinline__ u32x4 keep_if(bool ok, u32x4 v) { return ok ? v : zero4(); }

/* The activations stay out of the register ring: each unit's activation slabs go straight from
   memory into a two-unit ring in the wave's LDS and are read back slab by slab as they are
   multiplied (8B q4 at 16 tokens 13.7k -> 14.1k tok/s, int8 protocol 74.7k -> 80.8k, 70B bf16
   +0.5 to +0.9 %).  Where a step's eight q4 block scales of a row are one aligned 16-byte run
   (WHOLE), the scales of MMA_SCALE_STEPS steps of the group's rows come into LDS at once, one
   load of 64 lanes per 16 rows (64 contiguous bytes of each row), where loading a step's scales
   into registers took one instruction per tile, each returning the same 16 bytes of a row to all
   four lane groups, and touched a cache line per row per step (8B q4 at 16 tokens: 15.7k ->
   17.8k tok/s; at 4 tokens 4.4k -> 4.9k).  mma_ring_slots counts the ring's slots of 64 chunks of 16 bytes: the two units'
   activations, then (q4) one block of scales for row groups of NT tiles. */
constexpr int MMA_SCALE_STEPS = 4;
template <int FMT, int NT>
constexpr int mma_ring_slots() { return 2 * MmaStep<FMT>::SLABS + (FMT == FMT_Q4 ? NT : 0); }

/* Wait until no LDS operation of the wave is outstanding. */
__device__ __forceinline__ void wait_lds_idle() { __builtin_amdgcn_s_waitcnt(0xF | 0x70 | (3 << 14)); }

/* Wait until at most n vector memory operations are outstanding (an LDS-DMA load's data is in LDS
   once it has left the count; operations leave it in the order they were issued). */
template <int N>
__device__ __forceinline__ void wait_vm() {
    static_assert(N >= 0 && N < 64, "vmcnt holds 0..63");
    __builtin_amdgcn_s_waitcnt((N & 15) | 0x70 | 0xF00 | ((N >> 4) << 14));
}

/* Rows [r0, r1) of matrix d for tokens token0 .. token0 + ntok - 1 (ntok <= 16), NT tiles of 16
   rows per group.  The units (group, step) run as a two-set register pipeline, as in rows_q4: the
   loads of the next unit are in flight while the current one is multiplied.  Each load adds a
   32-bit lane offset and a constant to a wave-uniform base, so it costs no vector arithmetic; the
   lane offsets are set once per group, with rows past r1 clamped to row r1 - 1 (read, never
   stored), and token slots past ntok read the first token (never stored).  Where a row's length
   is not a whole number of steps, its last step is moved back to end at the row's end and the
   values the previous step already covered are zeroed when it is multiplied (masking them as they
   arrive would make each load wait at once).  Rows shorter than one step (SHORT) clamp each
   lane's offset instead.  Where rows hold a whole number of steps (WHOLE), no step is ever moved
   back and the loop carries no mask (16-bit and int8: the mask's selects cost 40 % of a 16-bit
   unit's vector instructions).  For q4, WHOLE also asks for 16-byte aligned scales: a step's
   eight block scales of a row are then one 16-byte run and come through LDS in blocks of four
   steps (below); otherwise each is loaded into registers alone.
   The caller keeps 16 NT rows of codes and 16 tokens of activations within 2^31 bytes.  The
   activations (and, with WHOLE, the q4 scales) come from the LDS ring, which leaves the register
   ring to the weights. */
template <int FMT, int NT, bool WHOLE, bool SHORT>
__device__ __forceinline__ void rows_mma(const DevMat& d, int64_t r0, int64_t r1, int32_t token0, int ntok, int lane,
                                         u32x4* __restrict__ xlds) {
    using Unit = MmaUnit<FMT, NT>;
    constexpr int J = Unit::J, SL = Unit::SL, SK = MmaStep<FMT>::K, SB = 64 * J;   /* SB: row bytes per step */
    constexpr int XG = FMT == FMT_I8 ? 32 : 16;                  /* x bytes per lane group within a step */
    const int c = lane & 15, g = lane >> 4;                      /* token slot and tile row; group       */
    const int64_t nc = d.nc;                                     /* blocks (q4) or 16-byte chunks        */
    const int64_t crb = nc * 16;                                 /* code (or weight) bytes per row       */
    const int64_t kelem = FMT == FMT_Q4 ? nc * 32 : FMT == FMT_I8 ? nc * 16 : nc * 8;
    const int32_t steps = (int32_t)((crb + SB - 1) / SB);       /* at most 2^19 (rows up to 32 MiB) */
    const int64_t ngroups = (r1 - r0 + 16 * NT - 1) / (16 * NT);
    const int64_t n = ngroups * steps;                           /* units */
    if (n == 0) return;
    const rsrc_t rx = buffer_of(uniform_ptr(static_cast<const char*>(d.x) + (int64_t)token0 * d.x_stride));
    const int64_t srow = FMT == FMT_Q4 ? nc * 2 : 2;             /* scale bytes per row */
    f4_t acc[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) acc[t] = f4_t{0.f, 0.f, 0.f, 0.f};
    int64_t gl = 0, gc = 0;                                      /* group of the next unit to load, multiply */
    int32_t kl = 0, kc = 0;                                      /* and its step                             */
    int lbuf = 0, mbuf = 0;                                      /* LDS ring half of the next load, multiply */
    rsrc_t rw = buffer_of(d.w), rs = buffer_of(d.w);             /* this group's row r0 of codes, scales */
    uint32_t vr[NT], vs[NT];                                     /* lane offsets: row of each tile */
    /* q4 WHOLE: the block of scales of steps 4 m .. 4 m + 3 of the group's 16 NT rows comes into
       LDS with the first of those steps, NT loads of 16 rows each: lane i of load j brings row
       r = 16 j + i / 4 at step 4 m + ((i % 4) ^ (r / 2 % 4)), into block slot 4 r + i % 4 (the
       rotation spreads a tile's 16 rows of one step over the LDS banks).  The block is overwritten
       when the next one comes, one unit before the old block's last unit is multiplied, so that
       unit's scales are read into its registers at the end of the unit before it (scar). */
    constexpr bool S_LDS = FMT == FMT_Q4 && WHOLE;
    constexpr int NBD = S_LDS ? NT : 0;                          /* loads of a scale block */
    constexpr int SBLK = 2 * SL * WAVE;                          /* the block's first slot */
    uint32_t vsb[NBD > 0 ? NBD : 1] = {};                        /* row 16 j + i / 4 of lane i, load j */
    const uint32_t skk = (uint32_t)((lane & 3) ^ ((lane >> 3) & 3));   /* its step within the block */
    bool scar = false;                                           /* the next unit's scales are in its registers */
    /* Ring activations reach LDS as whole 128-byte lines: load q of a unit (line p = q / 2 of the
       step, token half h = q % 2) gives lane i token 8 h + i / 8 at chunk (i % 8) ^ (i / 8) of line
       p, which holds slabs 2 p and 2 p + 1 (q4: chunk 4 (s % 2) + g of slab s for lane group g;
       int8: chunk s % 2 + 2 g).  The chunks are stored rotated by token so that the slab reads, 16
       tokens of one chunk per lane group, spread over the LDS banks.  Lane (c, g) reads slab s at
       slot 128 (s / 2) + rd[s % 2] of the ring.  Whole lines halve the cache lines each load
       touches (8B q4 at 16 tokens: 13.9k -> 15.3k tok/s). */
    const int xi = lane >> 3, xc = (lane & 7) ^ xi;
    uint32_t xt[2];                                              /* the token row of each half */
#pragma unroll
    for (int h = 0; h < 2; ++h) xt[h] = (uint32_t)((8 * h + xi < ntok ? 8 * h + xi : 0) * d.x_stride);
    int rd[2];
#pragma unroll
    for (int e = 0; e < 2; ++e)
        rd[e] = (c >> 3) * WAVE + (c & 7) * 8 + ((FMT == FMT_I8 ? e + 2 * g : 4 * e + g) ^ (c & 7));
    static_assert(2 * SL + NBD <= mma_ring_slots<FMT, NT>(), "LDS ring slots");
    uint32_t vh[NT];                                             /* the row of the tile's second half */
    const uint32_t lc = 16 * (g + 4 * (c >> 3));                 /* the lane's byte within a 128-byte line */
    static_assert(J == 2, "a step is one line of each row");
    /* the scales of step k of tile t's row c (lane (c, g)) from the block */
    auto read_scales = [&](Unit& v, int32_t k) {
        if constexpr (S_LDS) {
#pragma unroll
            for (int t = 0; t < NT; ++t) {
                const u32x4 x = xlds[SBLK + 4 * (16 * t + c) + ((k % MMA_SCALE_STEPS) ^ ((c >> 1) & 3))];
                v.s[t][0] = x.x, v.s[t][1] = x.y, v.s[t][2] = x.z, v.s[t][3] = x.w;
            }
        }
    };
    auto load = [&](Unit& u) {
        if (kl == 0) {
            const int64_t i0 = r0 + gl * 16 * NT;
            rw = buffer_of(uniform_ptr(static_cast<const char*>(d.w) + i0 * crb));
            if constexpr (FMT == FMT_Q4 || FMT == FMT_I8)
                rs = buffer_of(uniform_ptr(static_cast<const char*>(d.s) + i0 * srow));
#pragma unroll
            for (int t = 0; t < NT; ++t) {
                const int64_t rr = std::min<int64_t>(i0 + 16 * t + c, r1 - 1) - i0;   /* the row lane c multiplies */
                vs[t] = (uint32_t)(rr * srow);
                vr[t] = (uint32_t)((std::min<int64_t>(i0 + 16 * t + (c & 7), r1 - 1) - i0) * crb);
                vh[t] = (uint32_t)((std::min<int64_t>(i0 + 16 * t + 8 + (c & 7), r1 - 1) - i0) * crb);
            }
#pragma unroll
            for (int j = 0; j < NBD; ++j)
                vsb[j] = (uint32_t)((std::min<int64_t>(i0 + 16 * j + (lane >> 2), r1 - 1) - i0) * srow);
        }
        /* the last step ends at the row's end; offsets stay below 2^31 (the caller's limits) */
        const uint32_t kb = SHORT ? 0 : (uint32_t)std::min<int64_t>((int64_t)kl * SB, crb - SB);
        const uint32_t xo = SHORT ? 0 : (uint32_t)(std::min<int64_t>((int64_t)kl * SK, kelem - SK) * 2);
        const uint32_t b0 = SHORT ? 0 : (uint32_t)std::min<int64_t>((int64_t)kl * 8, nc - 8);   /* q4: first block */
        if (S_LDS && kl % MMA_SCALE_STEPS == 0) {              /* a new block of scales, first of all */
            wait_lds_idle();                                     /* the old block's reads are done */
            const uint32_t so = (uint32_t)std::min<int64_t>(kl + skk, steps - 1) * 16;   /* the last block may be short */
#pragma unroll
            for (int j = 0; j < NBD; ++j) buf_to_lds(rs, xlds + SBLK + j * WAVE, vsb[j] + so, 0);
        }
        {
            /* the slabs next, so that every load issued after them is counted by wait_vm; a row
               shorter than one step clamps each lane's activation offset */
            u32x4* ring = xlds + (lbuf ? SL * WAVE : 0);
#pragma unroll
            for (int q = 0; q < SL; ++q) {
                const int p = q >> 1, h = q & 1;
                const uint32_t v = SHORT ? xt[h] + 2 * (uint32_t)std::min<int64_t>(64 * p + 8 * xc, kelem - 8)
                                         : xt[h] + 16 * xc + 128 * p;
                buf_to_lds(rx, ring + q * WAVE, v, xo);
            }
            lbuf ^= 1;
            __builtin_amdgcn_sched_barrier(0);
        }
        /* a row shorter than one step clamps each lane's weight offset */
        const uint32_t lw = SHORT ? (uint32_t)std::min<int64_t>(lc, crb - 16) : lc;
#pragma unroll
        for (int t = 0; t < NT; ++t)
#pragma unroll
            for (int jj = 0; jj < J; ++jj) u.w[t][jj] = buf_once(rw, (jj ? vh[t] : vr[t]) + lw, kb);
#pragma unroll
        for (int t = 0; t < NT; ++t) {
            if constexpr (FMT == FMT_Q4) {
                if constexpr (!WHOLE) {                          /* (WHOLE: in the LDS ring) */
                    uint32_t h[8];
#pragma unroll
                    for (int j = 0; j < 8; ++j) h[j] = buf_u16(rs, vs[t], (uint32_t)std::min<int64_t>(b0 + j, nc - 1) * 2);
#pragma unroll
                    for (int j = 0; j < 4; ++j) u.s[t][j] = h[2 * j] | h[2 * j + 1] << 16;
                }
            } else if constexpr (FMT == FMT_I8) {
                if (kl + 1 == steps) u.s[t][0] = buf_u16(rs, vs[t], 0);   /* read only by the group's last step */
            }
        }
        if (++kl == steps) { kl = 0; ++gl; }
    };
    /* Vector memory operations each load() issues after its loads into LDS (weights, scales; the
       int8 row scales, loaded on a group's last step only, are left out: a wait that counts fewer
       later loads than were issued still covers the ring). */
    constexpr int AFTER_X = NT * J + (FMT == FMT_Q4 ? (WHOLE ? 0 : 8 * NT) : 0);
    constexpr int PER_UNIT = SL + AFTER_X;                       /* plus NBD where a scale block starts */
    auto multiply = [&](Unit& u, Unit& un, auto next_loaded) {   /* un: the next unit's registers */
        const int64_t i0 = r0 + gc * 16 * NT;
        const int32_t k1 = kc + 1 == steps ? 0 : kc + 1;         /* the next unit's step, and the one after */
        const int32_t k2 = k1 + 1 == steps ? 0 : k1 + 1;
        /* the step's first weight, and the first one it has not already covered */
        const int64_t e0 = SHORT ? 0 : std::min<int64_t>((int64_t)kc * SK, kelem - SK), e1 = SHORT ? 0 : (int64_t)kc * SK;
#pragma unroll
        for (int t = 0; t < NT; ++t) lines_to_slabs(u.w[t][0], u.w[t][1]);
        {
            if constexpr (FMT == FMT_Q4) {
#pragma unroll
                for (int t = 0; t < NT; ++t)
#pragma unroll
                    for (int jj = 0; jj < J; ++jj) u.w[t][jj] = transpose_groups(u.w[t][jj]);
            }
            /* the unit's slabs are in LDS once no more than the loads issued after them remain (the
               next unit's scale block, if it starts one, was issued after them too) */
            constexpr int AFTER = AFTER_X + (decltype(next_loaded)::value ? PER_UNIT : 0);
            if (S_LDS && decltype(next_loaded)::value && k1 % MMA_SCALE_STEPS == 0)
                wait_vm<(AFTER + NBD < 63 ? AFTER + NBD : 63)>();
            else
                wait_vm<(AFTER < 63 ? AFTER : 63)>();
            __builtin_amdgcn_sched_barrier(0);
            const u32x4* ring = xlds + (mbuf ? SL * WAVE : 0);
            mbuf ^= 1;
            if constexpr (S_LDS) {
                if (!scar) read_scales(u, kc);
            }
            /* a short row or a moved-back last step (never with WHOLE: known at compile time) */
            const bool masked = SHORT || (!WHOLE && e0 < e1);
            auto slab = [&](int sl) -> u32x4 {
                u32x4 xs = ring[(sl >> 1) * 2 * WAVE + rd[sl & 1]];
                if (__builtin_expect(masked, 0)) {
                    const int64_t e = e0 + (XG * g + mma_x_byte<FMT>(sl)) / 2;
                    xs = keep_if(e >= e1 && e < kelem, xs);
                }
                return xs;
            };
            if constexpr (FMT != FMT_Q4 && FMT != FMT_I8) {       /* 16-bit */
                if (__builtin_expect(masked, 0)) {               /* 16-bit weights there may not be finite */
#pragma unroll
                    for (int t = 0; t < NT; ++t)
#pragma unroll
                        for (int jj = 0; jj < J; ++jj) {
                            const int64_t e = e0 + 32 * jj + 8 * g;
                            u.w[t][jj] = keep_if(e >= e1 && e < kelem, u.w[t][jj]);
                        }
                }
                u32x4 xs[SL];
#pragma unroll
                for (int sl = 0; sl < SL; ++sl) xs[sl] = slab(sl);
#pragma unroll
                for (int t = 0; t < NT; ++t)
#pragma unroll
                    for (int jj = 0; jj < J; ++jj) acc[t] = mma16<FMT>(xs[jj], u.w[t][jj], acc[t]);
            } else if constexpr (FMT == FMT_I8) {
                u32x4 xs[SL];
#pragma unroll
                for (int sl = 0; sl < SL; ++sl) xs[sl] = x8_i8_order(slab(sl));
#pragma unroll
                for (int t = 0; t < NT; ++t)
#pragma unroll
                    for (int jj = 0; jj < J; ++jj) {
                        acc[t] = mma16<FMT_F16>(xs[2 * jj], i8_words_f16(u.w[t][jj].x, u.w[t][jj].y), acc[t]);
                        acc[t] = mma16<FMT_F16>(xs[2 * jj + 1], i8_words_f16(u.w[t][jj].z, u.w[t][jj].w), acc[t]);
                    }
            } else {
                /* Each slab's products are scaled and summed while the next slab's matrix instructions
                   run, and the sum is pinned there: left alone, the compiler sinks every scaled sum to
                   the end of the unit and keeps all 32 products live (128 registers, one wave per SIMD
                   instead of two). */
                f4_t pend[NT];
                float psc[NT];
#pragma unroll
                for (int sl = 0; sl < SL; ++sl) {                   /* slab sl: block e0 / 32 + sl of each row */
                    const u32x4 xs = x8_q4_order(slab(sl));
                    const f4_t bias = mma16<FMT_F16>(xs, u32x4{Q4_NEG_BIAS, Q4_NEG_BIAS, Q4_NEG_BIAS, Q4_NEG_BIAS},
                                                     f4_t{0.f, 0.f, 0.f, 0.f});
                    f4_t p[NT];                                  /* 2^-24 q x per row and token */
#pragma unroll
                    for (int t = 0; t < NT; ++t) p[t] = mma16<FMT_F16>(xs, q4_word_sub(u.w[t][sl / 4][sl % 4]), bias);
#pragma unroll
                    for (int t = 0; t < NT; ++t) {
                        if (sl > 0) {
                            acc[t] += psc[t] * pend[t];
                            __asm__ volatile("" : "+v"(acc[t]));
                        }
                        float sc = f16_bits_to_f32((uint16_t)(u.s[t][sl / 2] >> (16 * (sl % 2))));
                        if constexpr (!WHOLE) {
                            const int64_t b = e0 / 32 + sl;
                            sc = b >= e1 / 32 && b < nc ? sc : 0.f;
                        }
                        pend[t] = p[t];
                        psc[t] = sc;
                    }
                    __builtin_amdgcn_sched_barrier(0);               /* two slabs' values live at a time */
                }
#pragma unroll
                for (int t = 0; t < NT; ++t) {
                    acc[t] += psc[t] * pend[t];
                    __asm__ volatile("" : "+v"(acc[t]));
                }
            }
            /* The next unit's scales, where the unit after it brings a new block before the next
               unit is multiplied; a block of one step (the group's last) is waited for first. */
            if constexpr (S_LDS && decltype(next_loaded)::value) {
                scar = k2 % MMA_SCALE_STEPS == 0;
                if (scar) {
                    if (k1 % MMA_SCALE_STEPS == 0) wait_vm<(SL + NT * J < 63 ? SL + NT * J : 63)>();
                    read_scales(un, k1);
                }
            }
        }
        if (kc + 1 == steps) {                                   /* end of a group: store, reset */
            /* lane (c, g) holds tokens 4 g .. 4 g + 3 of row c of each tile */
#pragma unroll
            for (int t = 0; t < NT; ++t) {
                const int64_t r = i0 + 16 * t + c;
                float rs = 1.f;
                if constexpr (FMT == FMT_I8) rs = f16_bits_to_f32((uint16_t)u.s[t][0]);
                if constexpr (FMT == FMT_Q4) rs = Q4_UNSCALE;
                if (r < r1) {
#pragma unroll
                    for (int jj = 0; jj < 4; ++jj) {
                        const int tok = 4 * g + jj;
                        if (tok < ntok)                          /* a global (not flat) store keeps the load waits exact */
                            as_global<g_f32*>(reinterpret_cast<char*>(d.y) + (int64_t)(token0 + tok) * d.y_stride)[r] =
                                acc[t][jj] * rs;
                    }
                }
                acc[t] = f4_t{0.f, 0.f, 0.f, 0.f};
            }
        }
        if (++kc == steps) { kc = 0; ++gc; }
    };
    Unit buf[2];
    const std::true_type next_loaded;
    const std::false_type last;
    load(buf[0]);
    if constexpr (S_LDS) {                                       /* one-step groups: unit 1 brings a new block */
        if (steps == 1 && n > 1) {
            wait_vm<(SL + NT * J < 63 ? SL + NT * J : 63)>();
            read_scales(buf[0], 0);
            scar = true;
        }
    }
    int64_t u = 0;                                               /* buf[0] holds unit u */
    for (; u + 3 <= n; u += 2) {
        load(buf[1]);                                            /* unit u + 1 */
        __builtin_amdgcn_sched_barrier(0);
        multiply(buf[0], buf[1], next_loaded);                   /* unit u     */
        load(buf[0]);                                            /* unit u + 2 */
        __builtin_amdgcn_sched_barrier(0);
        multiply(buf[1], buf[0], next_loaded);                   /* unit u + 1 */
    }
    /* one or two units left, unit u in buf[0] */
    if (u + 1 < n) {
        load(buf[1]);
        __builtin_amdgcn_sched_barrier(0);
        multiply(buf[0], buf[1], next_loaded);
        multiply(buf[1], buf[0], last);
    } else {
        multiply(buf[0], buf[1], last);
    }
}

constexpr int mma_base_fmt(int fmt) { return fmt == FMT_Q4_WHOLE ? FMT_Q4 : fmt; }

/* The matrix-core sweep over the byte range [lo, hi) of the weight stream (groups of 16 NT rows). */
template <int FMT, int NT>
__device__ __forceinline__ void stream_range_mma(const DevMat* __restrict__ tab, const int64_t* __restrict__ cost,
                                                 int nmat, int64_t lo, int64_t hi, int64_t tail, int64_t main_rows,
                                                 int32_t token0, int ntok, int lane, int& hint, u32x4* xlds) {
    for (int m = first_matrix(cost, nmat, lo, hint); m < nmat; ++m) {
        const DevMat d = tab[m];
        if (d.cost0 >= hi) break;
        hint = m;
        constexpr int F = mma_base_fmt(FMT);
        const int fmt = F ? F : d.fmt;
        RowRange rr = range_rows(d, lo, hi, 16 * NT);
        if (tail > 0) {              /* rows below the main region's last boundary are not the tail's */
            const int64_t fl = tail > d.cost0 ? ceil_div(tail - d.cost0, d.row_bytes * main_rows) * main_rows : 0;
            const int64_t f = fl < d.M ? fl : d.M;
            rr.r0 = rr.r0 > f ? rr.r0 : f;
            rr.r1 = rr.r1 > f ? rr.r1 : f;
        }
        if (rr.r0 >= rr.r1) continue;
        const bool short_rows = d.nc * 16 < 128;                 /* under one step */
#define WSR_ROWS(F, W, SH) rows_mma<F, NT, W, SH>(d, rr.r0, rr.r1, token0, ntok, lane, xlds)
        const bool whole = d.nc % 8 == 0;                        /* 128-byte steps: 8 chunks or blocks */
        if constexpr (FMT == FMT_Q4_WHOLE) {                     /* the launcher checked every matrix */
            WSR_ROWS(FMT_Q4, true, false);
        } else if ((F == 0 || F == FMT_F16) && fmt == FMT_F16) {
            if (short_rows) WSR_ROWS(FMT_F16, false, true);
            else if (whole) WSR_ROWS(FMT_F16, true, false);
            else WSR_ROWS(FMT_F16, false, false);
        } else if ((F == 0 || F == FMT_BF16) && fmt == FMT_BF16) {
            if (short_rows) WSR_ROWS(FMT_BF16, false, true);
            else if (whole) WSR_ROWS(FMT_BF16, true, false);
            else WSR_ROWS(FMT_BF16, false, false);
        } else if ((F == 0 || F == FMT_Q4) && fmt == FMT_Q4) {
            if (short_rows) WSR_ROWS(FMT_Q4, false, true);
            else if (whole && (reinterpret_cast<uintptr_t>(d.s) & 15) == 0) WSR_ROWS(FMT_Q4, true, false);
            else WSR_ROWS(FMT_Q4, false, false);
        } else if ((F == 0 || F == FMT_I8) && fmt == FMT_I8) {
            if (short_rows) WSR_ROWS(FMT_I8, false, true);
            else if (whole) WSR_ROWS(FMT_I8, true, false);
            else WSR_ROWS(FMT_I8, false, false);
        }
#undef WSR_ROWS
    }
}

}  // namespace wsr

#endif
