// Implicit-GEMM quantized convolution for small images: a workgroup keeps
// whole padded images (or row bands of larger ones) in LDS and its filters in
// registers.  Same computation as the other convolution kernels (Sec. III-A
// Eq. (2), Sec. III-B Eq. (6), scale-and-clamp compression or the staircase
// of Eq. (4), Sec. IV-A fused max-pooling), laid out for layers whose
// per-tile bookkeeping would dominate the general kernels: a network's first
// layer (K = kh*kw*3 for 3 image channels), the later layers of a small
// network (16x16 and 8x8 images of 32 channels) and layers with about one
// general tile per compute unit (32x32x64 images at batch 64, in row bands).
//   * A workgroup owns one 32-channel group (grid.y) and walks groups of
//     whole images (several small images per step so that every wave has
//     work): each padded image is staged once in LDS, unpacked to int8 (8-bit
//     codes offset by -128, pads included); the next group's bytes are
//     loaded into registers while the current one is computed.  Images too
//     large for one tile (BAND) are walked in bands of output rows instead:
//     a step stages the band's input rows plus the kh - 1 rows of its halo,
//     rows above or below the image as pads.
//   * The filters of the group live in registers for the whole kernel (one
//     16-byte fragment per lane and K step); wide-pixel filters arrive
//     through LDS once (coalesced loads of the group's rows, expanded to
//     int8 there), and the group's compression plans (or staircase
//     thresholds) are computed once, by wave 0, while the first step is
//     staged.
//   * A wave computes two MFMA row tiles of 32 output pixels at a time with
//     v_mfma_i32_32x32x32_i8 (rows = pixels, columns = channels).  A row tile
//     is 1, 2 or 4 output rows of an image WOP = 32, 16 or 8 pixels wide
//     (narrower images leave lanes idle), so the lane's pixel is fixed per
//     tile and every im2col tap is an LDS read at a compile-time offset from
//     one per-lane base.
//   * K order.  Pixels of 32 unpacked bytes or more: K steps walk the taps
//     and the 32-byte chunks of each tap; the two halves of a wave (lanes
//     0-31, 32-63) take the two 16-byte halves of a chunk.  One-word pixels
//     (4-16 unpacked bytes): the halves take the filter's upper and lower
//     band of ceil(kh/2) rows in the same slot order (bands past the filter's
//     last row and slots past the band carry zero weights); 8-bit tiles then
//     store a pixel pair per slot, so a run of four taps along a filter row
//     is two aligned 8-byte reads.
//   * The 2x2 max-pooling is taken on the accumulators (the compression is
//     non-decreasing in the accumulator whenever the multiplier is positive,
//     and the staircase level always is, so the maximum commutes with it)
//     and only the pooled values are compressed; with a non-positive
//     multiplier each code is compressed first and the codes are pooled.
//     The four outputs of a window always sit in one lane.
//   * Outputs in whole rows of pixels of one or two 32-channel groups are
//     assembled per wave in LDS and leave as one group-wide store per pixel
//     (unpooled: unpacked code bytes, packed on the read-back with byte
//     permutes; pooled: codes of neighbouring channels packed across lanes
//     with DPP moves first); other shapes store bytes straight from the
//     lanes.
#pragma once

#include "conv_m32_impl.h"

namespace qnn {

// Slot order of the K dimension within one half band (DY filter rows x KW
// columns) for one-word pixels, TPF taps per 16-byte fragment (U = unpacked
// bytes per pixel: 4, 8 or 16).  U = 8, 16: the taps in raster order.
// U = 4 (8-bit codes): first every run of four horizontally adjacent taps of
// a filter row (one fragment each, read as two aligned 8-byte pixel pairs),
// then the leftover columns of all rows, four to a fragment.  tap(i) =
// ky * 256 + kx, or -1 for an empty slot (zero weight, nothing read).
template <int U, int KW, int DY>
struct BandTaps {
    static constexpr int TPF = 16 / U;
    static constexpr int NT = DY * KW;
    static constexpr int RUNS = U == 4 ? KW / 4 : 0;
    static constexpr int LEFT = KW % 4;
    static constexpr int NR = DY * RUNS;
    static constexpr int NF = U == 4 ? NR + (DY * LEFT + 3) / 4 : (NT + TPF - 1) / TPF;
    static constexpr int tap(int i)
    {
        if (U != 4)
            return i < NT ? (i / KW) * 256 + i % KW : -1;
        const int f = i / 4, t = i % 4;
        if (f < NR)
            return (f / (RUNS > 0 ? RUNS : 1)) * 256 + (f % (RUNS > 0 ? RUNS : 1)) * 4 + t;
        const int j = (f - NR) * 4 + t;
        return (LEFT > 0 && j < DY * LEFT) ? (j / (LEFT > 0 ? LEFT : 1)) * 256 + RUNS * 4 + j % (LEFT > 0 ? LEFT : 1)
                                          : -1;
    }
};

// Half-word pixels (4 channels at 4 bits, codes n0..n3): activations as the
// bytes n0, n2, n1, n3 and weights as 16 times the same order, the K order
// of the 4-bit packed words (stage_word<4>, w4_word) within one 16-bit pixel.
__device__ __forceinline__ uint32_t stage_half4(uint32_t v)
{
    return (v & 0x0F0Fu) | (((v >> 4) & 0x0F0Fu) << 16);
}
__device__ __forceinline__ uint32_t w4_half(uint32_t v)
{
    return ((v << 4) & 0xF0F0u) | ((v & 0xF0F0u) << 16);
}

// Geometry of one instance: BITS-bit codes, pixels of P packed bytes.
template <int BITS, int P, int KH, int KW, int WOP>
struct ImgGeom {
    static constexpr int U = P * 8 / BITS;             // unpacked bytes per pixel
    static constexpr bool CHUNK = U >= 32;             // K split by 16-byte halves of 32-byte chunks
    // tile slot bytes: 8-bit one-word pixels a pair; pixels of 32 unpacked
    // bytes or more one pixel and 16 bytes of padding (an odd number of
    // 16-byte units apart, the 16-byte im2col reads of 8 neighbouring lanes
    // fall in 8 different bank quads; with slots a power of two apart they
    // hit 2 or 4 times the same banks)
    static constexpr int SB = U == 4 ? 8 : (U >= 32 ? U + 16 : U);
    static constexpr int PP = WOP + KW - 1;            // tile pitch, slots
    static constexpr int RB = PP * SB;                 // tile row, bytes
    static constexpr int RT = 32 / WOP;                // image rows per MFMA row tile
    static constexpr int DY = (KH + 1) / 2;            // band rows (one-word pixels)
    static constexpr int CPT = CHUNK ? U / 32 : 1;     // 32-byte chunks per tap
    typedef BandTaps<CHUNK ? 16 : U, KW, DY> BT;
    static constexpr int TPF = CHUNK ? 1 : BT::TPF;    // taps per fragment
    static constexpr int KS = CHUNK ? KH * KW * CPT : BT::NF;  // 32-deep K steps
    static constexpr int WB = CHUNK ? 16 * BITS / 8 : 4;  // packed filter bytes behind one fragment slot
    // CHUNK filters pass through LDS unpacked: fragment unit u = 2 * (K
    // step) + lane half of channel c at u * FP + 16 c (FP: one unit of all 32
    // channels, padded); FLDS bytes in all.  XLDS: the LDS beyond the image
    // tiles (filters, then 32 channel plans of 64 bytes and a vote word,
    // then each wave's output staging: 64 pixels of one 32-channel group, one
    // code byte per channel, OPS bytes apart)
    static constexpr int FP = 33 * 16;
    static constexpr int FLDS = CHUNK ? 2 * KS * FP : 0;
    static constexpr int OPS = 48;
    static constexpr int XLDS = FLDS + 32 * 64 + 16 + 4 * 64 * OPS;
};

// One 16-byte im2col fragment for K step S of the pixel whose tile slot is
// at p (lane half already folded into p): compile-time offsets.
template <int BITS, int P, int KH, int KW, int WOP, int S>
__device__ __forceinline__ v4i img_frag(const uint8_t *p)
{
    typedef ImgGeom<BITS, P, KH, KW, WOP> G;
    constexpr int SB = G::SB, PP = G::PP;
    if constexpr (G::CHUNK) {
        constexpr int t = S / G::CPT, j = S % G::CPT;
        return *(const v4i *)(p + ((t / KW) * PP + t % KW) * SB + 32 * j);
    } else if constexpr (G::U == 4) {
        typedef typename G::BT TP;
        uint32_t d[4];
#pragma unroll
        for (int t = 0; t < 4; t += 2) {
            const int t0 = TP::tap(S * 4 + t), t1 = TP::tap(S * 4 + t + 1);
            if (t0 >= 0 && t1 == t0 + 1) {
                const uint2 v = *(const uint2 *)(p + ((t0 >> 8) * PP + (t0 & 255)) * SB);
                d[t] = v.x;
                d[t + 1] = v.y;
            } else {
                d[t] = t0 >= 0 ? *(const uint32_t *)(p + ((t0 >> 8) * PP + (t0 & 255)) * SB) : 0u;
                d[t + 1] = t1 >= 0 ? *(const uint32_t *)(p + ((t1 >> 8) * PP + (t1 & 255)) * SB) : 0u;
            }
        }
        return (v4i){(int32_t)d[0], (int32_t)d[1], (int32_t)d[2], (int32_t)d[3]};
    } else if constexpr (G::U == 8) {
        typedef typename G::BT TP;
        uint2 d[2];
#pragma unroll
        for (int t = 0; t < 2; ++t) {
            const int tp = TP::tap(S * 2 + t);
            d[t] = tp >= 0 ? *(const uint2 *)(p + ((tp >> 8) * PP + (tp & 255)) * SB) : make_uint2(0, 0);
        }
        return (v4i){(int32_t)d[0].x, (int32_t)d[0].y, (int32_t)d[1].x, (int32_t)d[1].y};
    } else {
        typedef typename G::BT TP;
        constexpr int tp = TP::tap(S);
        if constexpr (tp >= 0)
            return *(const v4i *)(p + ((tp >> 8) * PP + (tp & 255)) * SB);
        else
            return (v4i){0, 0, 0, 0};
    }
}

// Both row tiles' fragments and MFMAs of K steps S .. KS-1 (unrolled through
// the template recursion, so every offset is an immediate).
template <int BITS, int P, int KH, int KW, int WOP, int S>
__device__ __forceinline__ void img_steps(const uint8_t *p0, const uint8_t *p1, const v4i *A, v16i &acc0,
                                          v16i &acc1)
{
    if constexpr (S < ImgGeom<BITS, P, KH, KW, WOP>::KS) {
        const v4i b0 = img_frag<BITS, P, KH, KW, WOP, S>(p0);
        const v4i b1 = img_frag<BITS, P, KH, KW, WOP, S>(p1);
        if constexpr (S == 0) {
            acc0 = __builtin_amdgcn_mfma_i32_32x32x32_i8(b0, A[S], (v16i){}, 0, 0, 0);
            acc1 = __builtin_amdgcn_mfma_i32_32x32x32_i8(b1, A[S], (v16i){}, 0, 0, 0);
        } else {
            acc0 = __builtin_amdgcn_mfma_i32_32x32x32_i8(b0, A[S], acc0, 0, 0, 0);
            acc1 = __builtin_amdgcn_mfma_i32_32x32x32_i8(b1, A[S], acc1, 0, 0, 0);
        }
        img_steps<BITS, P, KH, KW, WOP, S + 1>(p0, p1, A, acc0, acc1);
    }
}

// The same K steps with the im2col fragments read D steps ahead of their
// MFMAs: a ring of D + 1 fragment pairs, the order held by scheduling
// barriers (left to itself the compiler reads each pair right before its
// MFMAs and waits out the local-memory latency at every step).  Used for
// row bands, whose 18 K steps per tile pair make that latency a chain
// (INT-4 batch-64 layer 6.93 -> 6.65 us, measured side by side); the
// shorter K loops of whole small images gain nothing from it.
template <int BITS, int P, int KH, int KW, int WOP, int S, int D>
__device__ __forceinline__ void img_pipe(const uint8_t *p0, const uint8_t *p1, const v4i *A, v16i &acc0,
                                         v16i &acc1, v4i *b0, v4i *b1)
{
    constexpr int KS = ImgGeom<BITS, P, KH, KW, WOP>::KS;
    if constexpr (S < KS) {
        if constexpr (S + D < KS) {
            b0[(S + D) % (D + 1)] = img_frag<BITS, P, KH, KW, WOP, S + D>(p0);
            b1[(S + D) % (D + 1)] = img_frag<BITS, P, KH, KW, WOP, S + D>(p1);
        }
        __builtin_amdgcn_sched_barrier(0);
        constexpr int k = S % (D + 1);
        if constexpr (S == 0) {
            acc0 = __builtin_amdgcn_mfma_i32_32x32x32_i8(b0[k], A[S], (v16i){}, 0, 0, 0);
            acc1 = __builtin_amdgcn_mfma_i32_32x32x32_i8(b1[k], A[S], (v16i){}, 0, 0, 0);
        } else {
            acc0 = __builtin_amdgcn_mfma_i32_32x32x32_i8(b0[k], A[S], acc0, 0, 0, 0);
            acc1 = __builtin_amdgcn_mfma_i32_32x32x32_i8(b1[k], A[S], acc1, 0, 0, 0);
        }
        __builtin_amdgcn_sched_barrier(0);
        img_pipe<BITS, P, KH, KW, WOP, S + 1, D>(p0, p1, A, acc0, acc1, b0, b1);
    }
}

template <int BITS, int P, int KH, int KW, int WOP, int S, int D>
__device__ __forceinline__ void img_pipe_fill(const uint8_t *p0, const uint8_t *p1, v4i *b0, v4i *b1)
{
    if constexpr (S < D && S < ImgGeom<BITS, P, KH, KW, WOP>::KS) {
        b0[S] = img_frag<BITS, P, KH, KW, WOP, S>(p0);
        b1[S] = img_frag<BITS, P, KH, KW, WOP, S>(p1);
        img_pipe_fill<BITS, P, KH, KW, WOP, S + 1, D>(p0, p1, b0, b1);
    }
}

template <int BITS, int P, int KH, int KW, int WOP, int D>
__device__ __forceinline__ void img_steps_ahead(const uint8_t *p0, const uint8_t *p1, const v4i *A, v16i &acc0,
                                                v16i &acc1)
{
    v4i b0[D + 1], b1[D + 1];
    img_pipe_fill<BITS, P, KH, KW, WOP, 0, D>(p0, p1, b0, b1);
    img_pipe<BITS, P, KH, KW, WOP, 0, D>(p0, p1, A, acc0, acc1, b0, b1);
}

// Scale-and-clamp code of one (scaled) accumulator from the channel's plan
// (requant_plan): any mode.
template <int SL>
__device__ __forceinline__ uint32_t img_code(int32_t accd, const int4 &e0, const int4 &e1, int32_t lo, int32_t hi)
{
    if (e1.z >= 3) {
        const int32_t d = __builtin_elementwise_sub_sat(accd, e0.x);
        const uint32_t dc = (uint32_t)min(max(d, 0), e0.y);
        const uint64_t rs = ((uint64_t)(uint32_t)e1.y << 32) | (uint32_t)e0.w;
        return (uint32_t)(((uint64_t)dc * (uint32_t)e0.z + rs) >> e1.x);
    }
    const int32_t acc32 = accd >> SL;
    int64_t r;
    if (e1.z) {
        const int32_t d = __builtin_elementwise_sub_sat(acc32, e0.x);
        const uint32_t dc = (uint32_t)min(max(d, 0), e0.y);
        uint32_t q;
        if (e1.z == 1)
            q = (__umul24(dc, (uint32_t)e0.z) + (uint32_t)e0.w) >> e1.y;
        else
            q = (uint32_t)(((uint64_t)dc * (uint32_t)e0.z + (uint32_t)e0.w) >> e1.y);
        r = (int64_t)e1.x + (int64_t)q;
    } else {
        const int64_t vv = (int64_t)acc32 + (int64_t)(((uint64_t)(uint32_t)e0.y << 32) | (uint32_t)e0.x);
        r = round_shift(vv * (int64_t)e0.z, e0.w);
    }
    r = r < lo ? lo : (r > hi ? hi : r);
    return (uint32_t)r;
}

// Mode-3 plans whose clamp interval lies in the signed 24-bit range (every
// channel's code fits the 32-bit form): with p = (L, H, mult, C) from
// img_plan3, the code is ((med3(acc, L, H) * mult + C) mod 2^32) >> shift,
// three instructions.  med3(acc, L, H) - L is the strict form's clamped
// difference and C = n0 - L * mult (mod 2^32), so the 32-bit multiply-add
// wraps to the exact strict-form value, which is below 2^32.  acc must come
// from an instruction the compiler sees (here: the maximum of a pooling
// window), not straight from a matrix instruction: the compiler inserts no
// wait states before an asm reader.
__device__ __forceinline__ uint32_t img_code3(int32_t accd, const int4 &p, int32_t sh)
{
    int32_t x, y;
    __asm__("v_med3_i32 %0, %1, %2, %3" : "=v"(x) : "v"(accd), "v"(p.x), "v"(p.y));
    __asm__("v_mad_i32_i24 %0, %1, %2, %3" : "=v"(y) : "v"(x), "v"(p.z), "v"(p.w));
    return (uint32_t)y >> sh;
}

// The three-instruction form of a mode-3 plan (e0 = (A, DS, mult, RS), the
// strict form's clamp base, width, multiplier and rounding term): clamp
// interval [L, H] = [A, A + DS], C = RS - A * mult mod 2^32; false when L, H
// or mult leave the signed 24-bit range of v_mad_i32_i24.
__device__ __forceinline__ bool img_plan3(const int4 &e0, const int4 &e1, int4 &p)
{
    const int64_t L = e0.x, H = (int64_t)e0.x + e0.y;
    p = make_int4(e0.x, (int32_t)H, e0.z, (int32_t)((uint32_t)e0.w - (uint32_t)e0.x * (uint32_t)e0.z));
    return e1.z == 3 && L >= -(1 << 23) && H < (1 << 23) && e0.z < (1 << 23);
}

// Mode-3 plans only (every channel's code fits the 32-bit form): a
// saturating subtract, a median-of-three clamp to [0, e0.y] (e0.y >= 0), a
// 24-bit multiply-add and a shift.
__device__ __forceinline__ uint32_t img_code3s(int32_t accd, const int4 &e0, const int4 &e1)
{
    const int32_t d = __builtin_elementwise_sub_sat(accd, e0.x);
    int32_t dc;
    __asm__("v_med3_i32 %0, %1, 0, %2" : "=v"(dc) : "v"(d), "v"(e0.y));
    return (__umul24((uint32_t)dc, (uint32_t)e0.z) + (uint32_t)e0.w) >> e1.x;
}

// Mode-3 and mode-4 plans (the strict form; products up to 64 bits): a
// saturating subtract, the clamp, one 32x32->64 multiply-add and a shift.
__device__ __forceinline__ uint32_t img_code4(int32_t accd, const int4 &e0, const int4 &e1)
{
    const int32_t d = __builtin_elementwise_sub_sat(accd, e0.x);
    int32_t dc;
    __asm__("v_med3_i32 %0, %1, 0, %2" : "=v"(dc) : "v"(d), "v"(e0.y));
    const uint64_t rs = ((uint64_t)(uint32_t)e1.y << 32) | (uint32_t)e0.w;
    return (uint32_t)(((uint64_t)(uint32_t)dc * (uint32_t)e0.z + rs) >> e1.x);
}

// Packs the codes of neighbouring channels into one output byte across
// lanes (lane = channel): 4 bits, lanes 2k and 2k+1; 2 bits, lanes 4k..4k+3,
// the lower channel in the lower bits.  Every lane of the wave takes part;
// the byte is complete on the lanes whose channel is a multiple of 8/BITS.
template <int BITS>
__device__ __forceinline__ uint32_t img_pack_lanes(uint32_t code)
{
    if (BITS == 8)
        return code;
    // quad_perm [1,0,3,2]: the neighbour's code
    uint32_t v = code | ((uint32_t)__builtin_amdgcn_update_dpp(0, (int)code, 0xB1, 0xF, 0xF, false) << BITS);
    if (BITS == 2)  // quad_perm [2,3,0,1]: the other pair
        v |= (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x4E, 0xF, 0xF, false) << 4;
    return v;
}

// Packs the 32 codes of one pixel's 32-channel group (one byte each in LDS,
// 16-byte aligned, channel order) into 4 * BITS bytes, the lower channel in
// the lower bits, and stores them (dst aligned to 4 * BITS).
template <int BITS>
__device__ __forceinline__ void img_pack_store(uint8_t *dst, const uint8_t *src)
{
    const uint4 lo = *(const uint4 *)src, hi = *(const uint4 *)(src + 16);
    if constexpr (BITS == 8) {
        *(uint4 *)dst = lo;
        *(uint4 *)(dst + 16) = hi;
    } else if constexpr (BITS == 4) {
        // bytes 2i and 2i + 1 -> one byte (even channel in the low nibble)
        const uint32_t d[8] = {lo.x, lo.y, lo.z, lo.w, hi.x, hi.y, hi.z, hi.w};
        uint32_t o[4];
#pragma unroll
        for (int m = 0; m < 4; ++m) {
            const uint32_t e = __builtin_amdgcn_perm(d[2 * m + 1], d[2 * m], 0x06040200u);
            const uint32_t od = __builtin_amdgcn_perm(d[2 * m + 1], d[2 * m], 0x07050301u);
            o[m] = e | (od << 4);
        }
        *(uint4 *)dst = make_uint4(o[0], o[1], o[2], o[3]);
    } else {
        // the four bytes of each word -> one byte, 2 bits each
        const uint32_t d[8] = {lo.x, lo.y, lo.z, lo.w, hi.x, hi.y, hi.z, hi.w};
        uint32_t y[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const uint32_t x = d[i] | (d[i] >> 6);  // byte 0: b0 | b1 << 2, byte 2: b2 | b3 << 2
            y[i] = x | (x >> 12);                   // byte 0: the packed byte
        }
        const uint32_t w0 = __builtin_amdgcn_perm(
            __builtin_amdgcn_perm(y[3], y[2], 0x0c0c0400u), __builtin_amdgcn_perm(y[1], y[0], 0x0c0c0400u),
            0x05040100u);
        const uint32_t w1 = __builtin_amdgcn_perm(
            __builtin_amdgcn_perm(y[7], y[6], 0x0c0c0400u), __builtin_amdgcn_perm(y[5], y[4], 0x0c0c0400u),
            0x05040100u);
        *(uint2 *)dst = make_uint2(w0, w1);
    }
}

// Staircase level of a (scaled) accumulator for non-decreasing thresholds:
// the balanced comparison tree of Sec. III-A (Eq. (4)), ceil(log2(NT + 1))
// comparisons, each choosing the next threshold with selects (no indexing).
// Equals the number of thresholds at or below acc (stair_level) whenever the
// thresholds are sorted.
template <int NT>
__device__ __forceinline__ uint32_t stair_tree(int32_t acc, const int32_t *T)
{
    if constexpr (NT == 15) {
        const bool c3 = acc >= T[7];
        const bool c2 = acc >= (c3 ? T[11] : T[3]);
        const int32_t u = c3 ? T[9] : T[1], v = c3 ? T[13] : T[5];
        const bool c1 = acc >= (c2 ? v : u);
        const int32_t a0 = c3 ? T[8] : T[0], a1 = c3 ? T[10] : T[2], a2 = c3 ? T[12] : T[4],
                      a3 = c3 ? T[14] : T[6];
        const int32_t b0 = c2 ? a2 : a0, b1 = c2 ? a3 : a1;
        const bool c0 = acc >= (c1 ? b1 : b0);
        return (c3 ? 8u : 0u) | (c2 ? 4u : 0u) | (c1 ? 2u : 0u) | (c0 ? 1u : 0u);
    } else if constexpr (NT == 3) {
        const bool c1 = acc >= T[1];
        const bool c0 = acc >= (c1 ? T[2] : T[0]);
        return (c1 ? 2u : 0u) | (c0 ? 1u : 0u);
    } else {
        return stair_level<NT>(acc, T);
    }
}

// The same tree with its last two levels' thresholds read from the lane's
// threshold column in LDS (T[i] at col[32 i]: the 32 lanes of a half-wave
// read 32 consecutive words, one per bank), at the index the bits decided so
// far give: for 15 thresholds the code is built one bit per comparison and
// only T[3], T[7] and T[11] are held in registers.
// 2 x + (acc >= t): the comparison's result is the carry into the add (two
// instructions; written out because the compiler builds the bit with a select
// and an or).  Only vcc, a vector-written lane mask, is clobbered.
__device__ __forceinline__ uint32_t stair_bit(uint32_t x, int32_t acc, int32_t t)
{
    uint32_t r;
    __asm__("v_cmp_ge_i32_e32 vcc, %1, %2\n\tv_addc_co_u32_e32 %0, vcc, %3, %3, vcc"
            : "=v"(r)
            : "v"(acc), "v"(t), "v"(x)
            : "vcc");
    return r;
}

template <int NT>
__device__ __forceinline__ uint32_t stair_tree_col(int32_t acc, const int32_t *T, const int32_t *col)
{
    if constexpr (NT == 15) {
        uint32_t x = acc >= T[7] ? 1u : 0u;                      // count >= 8
        x = stair_bit(x, acc, x ? T[11] : T[3]);                 // q: count >= 4 q
        x = stair_bit(x, acc, col[32 * (4 * x + 1)]);            // count >= 4 q + 2
        return stair_bit(x, acc, col[32 * (2 * x)]);             // count >= 4 q + 2 c1 + 1
    } else {
        return stair_tree<NT>(acc, T);
    }
}

// A compile-time int (the byte stride of an output pixel in the store fast
// paths).
template <int V>
struct ImgConst {
    static constexpr int value = V;
};

// 2x2 pooling windows of a pair of row tiles: window k (0..7) holds the
// registers (tile, v) of its four outputs and its pooled row (relative to
// the pair's first pooled row) and pooled column (without the lane half's
// share 2*h, which every window adds).  WOP = 32: a tile is one row, the
// window spans both tiles; WOP = 16: a tile is two rows, v and v + 8 are one
// column of both; WOP = 8: a tile is four rows, v and v + 4.
template <int WOP>
struct PoolWin {
    static constexpr int v0(int k)  // first register of window k
    {
        return WOP == 32 ? 2 * k : (WOP == 16 ? 2 * (k & 3) : ((k & 2) << 2) + 2 * (k & 1));
    }
    static constexpr int t0(int k) { return WOP == 32 ? 0 : k >> 2; }   // tile of the first row
    static constexpr int t1(int k) { return WOP == 32 ? 1 : k >> 2; }   // tile of the second row
    static constexpr int dv(int)  // register step from the first row to the second
    {
        return WOP == 32 ? 0 : (WOP == 16 ? 8 : 4);
    }
    static constexpr int prow(int k) { return WOP == 32 ? 0 : (WOP == 16 ? k >> 2 : 2 * (k >> 2) + ((k >> 1) & 1)); }
    static constexpr int pcol(int k)
    {
        // column of the window's first output (without 4h), halved
        return WOP == 32 ? 4 * (k >> 1) + (k & 1) : (WOP == 16 ? 4 * ((k & 3) >> 1) + (k & 1) : (k & 1));
    }
};

// The leading scalar arguments repeat the fields of a that the first input
// loads depend on (and the grid width): built with kernel-argument preloading,
// they are in scalar registers when the waves start, so the first loads issue
// without waiting for a scalar-load round trip (INT-4 batch-64 layer cold 6.76
// -> 6.16 us, INT-8 batch-1 layer 4.87 -> 4.49 us, measured side by side).
template <int BITS, int P, int KH, int KW, int WOP, bool POOL, bool BAND, bool STAIR>
__global__ void __launch_bounds__(256) conv_img_kernel(const uint8_t *px, int32_t pngroups,
                                                       int32_t pbands, int32_t pbrows, int32_t ptrows, int32_t pph,
                                                       int32_t ph_, int32_t pw_, uint32_t pdbm, uint32_t pdbs,
                                                       int32_t pgx, int32_t pm, ImgArgs a)
{
    a.x = px;
    a.m = pm;
    a.ngroups = pngroups;
    a.bands = pbands;
    a.brows = pbrows;
    a.trows = ptrows;
    a.ph = pph;
    a.h = ph_;
    a.w_ = pw_;
    a.div_bands.mul = pdbm;
    a.div_bands.shr = pdbs;
    const int gxn = pgx;
    static_assert(!STAIR || BITS != 8, "the staircase epilogue is built at 4 and 2 bits");
    typedef ImgGeom<BITS, P, KH, KW, WOP> G;
    static_assert(!BAND || P >= 16, "row bands are built for pixels of whole 16-byte quads");
    static_assert(P != 2 || BITS == 4, "half-word pixels are built at 4 bits (4 channels)");
    constexpr int NW = 4, NT = 256;
    constexpr int SB = G::SB, PP = G::PP, RB = G::RB, RT = G::RT, DY = G::DY, KS = G::KS;
    constexpr int SL = BITS == 4 ? 4 : (BITS == 2 ? 6 : 0);  // log2 of the weight scale
    constexpr int UPF = BAND ? 3 : 2;                         // prefetched 16-byte quads per thread
    constexpr int WROW = KH * KW * P;                         // packed bytes per filter bank
    extern __shared__ __align__(16) uint8_t smem[];
    const int tid = threadIdx.x;
    const int lane = tid & 63, r32 = lane & 31, h = lane >> 5;
    const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform
    const int gy = blockIdx.y;
    const int ch = gy * 32 + r32;
    const bool live = ch < a.m;
    const int npix = a.h * a.w_;
    const int imgq = npix * P / 16;  // 16-byte quads per image (P = 4: with a.quads)

    // ---- the first image group's bytes ----
    uint4 pf[UPF];
    auto issue = [&](int grp) {
        if constexpr (BAND) {
            // band of image img: tile row r is input row r0 + r; quads of
            // rows outside the image stay zero (staged as the pad code)
            const int img = (int)fdiv((uint32_t)grp, a.div_bands);
            const int r0 = (grp - img * a.bands) * a.brows - a.ph;
            const int rowq = a.w_ * (P / 16);
            const int qlo = max(0, -r0) * rowq, qhi = min(a.trows, a.h - r0) * rowq;
            const uint8_t *src = a.x + ((int64_t)img * a.h + r0) * a.w_ * P;
#pragma unroll
            for (int u = 0; u < UPF; ++u) {
                const int q = tid + u * NT;
                pf[u] = make_uint4(0, 0, 0, 0);
                if (q >= qlo && q < qhi)
                    pf[u] = *(const uint4 *)(src + (int64_t)q * 16);
            }
            return;
        }
        const int i0 = grp * a.ipw;
        const int ni = min(a.ipw, a.n - i0);
        const uint8_t *src = a.x + (size_t)i0 * npix * P;
#pragma unroll
        for (int u = 0; u < UPF; ++u) {
            const int q = tid + u * NT;
            pf[u] = make_uint4(0, 0, 0, 0);
            if (a.quads) {
                if (q < ni * imgq)
                    pf[u] = *(const uint4 *)(src + (size_t)q * 16);
            } else if constexpr (P == 4) {
                // one-word pixels, npix not a multiple of 4 (a single image per step)
                const uint32_t *s4 = (const uint32_t *)src;
                if (4 * q < npix)
                    pf[u].x = s4[4 * q];
                if (4 * q + 1 < npix)
                    pf[u].y = s4[4 * q + 1];
                if (4 * q + 2 < npix)
                    pf[u].z = s4[4 * q + 2];
                if (4 * q + 3 < npix)
                    pf[u].w = s4[4 * q + 3];
            } else {
                // half-word pixels, npix not a multiple of 8 (a single image per step)
                const uint16_t *s2 = (const uint16_t *)src;
                uint32_t d[4] = {0, 0, 0, 0};
#pragma unroll
                for (int j = 0; j < 8; ++j)
                    if (8 * q + j < npix)
                        d[j >> 1] |= (uint32_t)s2[8 * q + j] << (16 * (j & 1));
                pf[u] = make_uint4(d[0], d[1], d[2], d[3]);
            }
        }
    };
    // row bands: the workgroups of one XCD (dispatched round-robin over the
    // eight, workgroup i on XCD i mod 8; with the grid width a multiple of 8 both
    // channel groups of a band land on the same XCD) take consecutive bands,
    // so the halo rows two bands of an image share are fetched into one L2
    int grp = blockIdx.x;
    if (BAND && gxn % 8 == 0)
        grp = (int)(blockIdx.x % 8) * (gxn / 8) + (int)(blockIdx.x / 8);
    if (grp < a.ngroups)
        issue(grp);
    // the channel parameters of the plans (wave 0: bias, multiplier and
    // shift, or the staircase thresholds), requested right after the first
    // input bytes: the plans are on the way to the first barrier
    int32_t p_bias = 0, p_mult = 0, p_shift = 0;
    constexpr int NTH = (1 << BITS) - 1;  // staircase thresholds per channel (4 and 2 bits)
    int32_t p_tau[STAIR ? NTH : 1];
    if (wv == 0 && live) {
        if (a.bias)
            p_bias = a.bias[ch];
        if (a.epi == EPI_REQUANT) {
            p_mult = a.mult[ch];
            p_shift = a.shift[ch];
        }
        if constexpr (STAIR) {
#pragma unroll
            for (int k = 0; k < NTH; ++k)
                p_tau[k] = a.thresh[(size_t)ch * NTH + k];
        }
    }
    // ---- wide-pixel filters: the group's 32 filter rows are contiguous;
    // the threads that stage them (waves 1-3 when wave 0 computes the plans)
    // load them as 16-byte quads right after the image bytes, before any
    // other work ----
    constexpr bool early_plans = BITS != 8 || G::CHUNK;
    constexpr int QPR = WROW / 16;                                   // quads per filter row
    constexpr int FT = early_plans ? NT - 64 : NT;                   // staging threads
    constexpr int FQ = G::CHUNK ? (32 * QPR + FT - 1) / FT : 1;      // quads per staging thread
    const int ft = early_plans ? tid - 64 : tid;
    uint4 fq[FQ];
    if constexpr (G::CHUNK) {
        const int nq = min(32, a.m - gy * 32) * QPR;
        const uint8_t *wg = a.w + (size_t)gy * 32 * WROW;
#pragma unroll
        for (int i = 0; i < FQ; ++i) {
            const int q = ft + i * FT;
            fq[i] = make_uint4(0, 0, 0, 0);
            if (ft >= 0 && q < nq)
                fq[i] = *(const uint4 *)(wg + (size_t)q * 16);
        }
    }

    // ---- filters: the lane's fragment of every K step as int8 (4-/2-bit
    // weights as 16*w / 64*w) ----
    // LDS behind the image tiles: the unpacked filter units (CHUNK), then the
    // group's compression plans and fast-path votes
    uint8_t *sF = smem + (size_t)a.ipw * a.tile_bytes;
    // the requantization plans (e0 of the 32 channels, then their e1, then
    // their three-instruction forms: lanes read consecutive 16-byte
    // entries), or [16][32 channels] staircase thresholds on the kernel's
    // accumulator scale
    int4 *sPlan = (int4 *)(sF + G::FLDS);
    int *sVote = (int *)(sPlan + 128);
    uint8_t *sOut = (uint8_t *)(sPlan + 129) + wv * 64 * G::OPS;  // this wave's output staging
    // first layers (one-word and half-word pixels, pooled, one 32-channel
    // group per output pixel): every pooled code of a step goes into an LDS
    // copy of the step's output images, which leaves with full-wave 16-byte
    // stores after the step's last barrier (the launch adds its LDS: ipw
    // images of hp x wp pixels of ypb bytes)
    uint8_t *sStep = (uint8_t *)(sPlan + 129) + 4 * 64 * G::OPS;
    const bool bulk = P <= 4 && POOL && a.ypb == 4 * BITS && a.wp == WOP / 2 && a.pairs * G::RT <= a.hp;
    // STAIR instances compute only the staircase (Eq. (4)); the others every
    // other epilogue (a separate instance keeps each one's code small)
    constexpr bool stair = STAIR;
    // pads: every image tile holds the zero code once (staged: -128 at 8
    // bits); each step then overwrites only its interior (bands: also their
    // pad rows).  The barrier after the filter units also orders this fill
    // before the first staging
    {
        const uint32_t f = BITS == 8 ? 0x80808080u : 0u;
        const uint4 f4 = make_uint4(f, f, f, f);
        for (int i = tid; i < a.ipw * a.tile_bytes / 16; i += NT)
            ((uint4 *)smem)[i] = f4;
    }
    // ---- the group's compression plans (requant_plan) and the wave-uniform
    // fast paths: every channel in the 32-bit strict form with its clamp
    // interval in the signed 24-bit range (three instructions per code,
    // img_plan3); in the 32-bit strict form; in the 32- or 64-bit strict
    // form; every channel's code non-decreasing in the accumulator (positive
    // multiplier).  Computed by wave 0 (whose lanes hold
    // the same 32 channels as every wave's) and shared through LDS (read
    // after the first staging barrier).  Sub-byte plans need no filter sums
    // and 8-bit ones of 16-byte filter units read theirs from the filter
    // rows: wave 0 computes them before the filter staging, which the other
    // waves do; the remaining 8-bit plans (one-word pixels) follow the
    // filter fragments, while the other waves stage the first step ----
    v4i A[KS];
    auto compute_plans = [&]() {
        int32_t wsum = 0;
        if (BITS == 8 && G::CHUNK) {
            // the channel's filter sum straight from its row: lane half h
            // adds the 16-byte units h, h + 2, ... (four bytes per dot
            // product with ones)
            if (live) {
                const uint4 *wr = (const uint4 *)(a.w + (size_t)ch * WROW);
#pragma unroll
                for (int u = 0; u < KS; ++u) {
                    const uint4 v = wr[2 * u + h];
                    wsum = __builtin_amdgcn_sdot4((int)v.x, 0x01010101, wsum, false);
                    wsum = __builtin_amdgcn_sdot4((int)v.y, 0x01010101, wsum, false);
                    wsum = __builtin_amdgcn_sdot4((int)v.z, 0x01010101, wsum, false);
                    wsum = __builtin_amdgcn_sdot4((int)v.w, 0x01010101, wsum, false);
                }
            }
            wsum += __shfl_xor(wsum, 32, 64);  // the other lane half's share of the channel
        } else if (BITS == 8) {
#pragma unroll
            for (int s = 0; s < KS; ++s)
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const uint32_t d = (uint32_t)A[s][i];
                    wsum += (int)(int8_t)d + (int)(int8_t)(d >> 8) + (int)(int8_t)(d >> 16) + (int)(int8_t)(d >> 24);
                }
            wsum += __shfl_xor(wsum, 32, 64);  // the other lane half's share of the channel
        }
        if constexpr (stair) {
            // staircase (Eq. (4)): the thresholds moved onto the scaled
            // accumulator, S (tau - bias) clamped to int32 (stair_thresholds)
            __align__(16) int32_t T16[16];
            stair_thresholds(live ? p_tau : nullptr, NTH, p_bias, SL, T16);
            if (h == 0) {
#pragma unroll
                for (int k = 0; k < 16; ++k)
                    ((int32_t *)sPlan)[32 * k + r32] = T16[k];
            }
            // every channel's thresholds non-decreasing (the scaling and the
            // clamp keep their order): the comparison tree applies
            bool sorted = true;
#pragma unroll
            for (int k = 0; k + 1 < NTH; ++k)
                sorted = sorted && T16[k] <= T16[k + 1];
            const bool vs = __all(sorted);
            if (lane == 0)
                *sVote = vs ? 8 : 0;
        } else {
            int4 q0, q1;
            int64_t b = p_bias;
            if (BITS == 8)
                b += 128 * (int64_t)wsum;
            const int sh = p_shift < 0 ? 0 : (p_shift > 62 ? 62 : p_shift);
            requant_plan(b, p_mult, sh, a.clip_lo, a.clip_hi, a.epi == EPI_REQUANT, SL, q0, q1);
            int4 p3;
            const bool ok3 = img_plan3(q0, q1, p3);
            const bool v3 = __all(!live || ok3);
            const bool v3s = __all(!live || q1.z == 3);
            const bool v34 = __all(!live || q1.z == 3 || q1.z == 4);
            const bool vm = __all(!live || q1.z != 0 || q0.z > 0);
            if (h == 0) {
                sPlan[r32] = q0;
                sPlan[32 + r32] = q1;
                sPlan[64 + r32] = p3;
            }
            if (lane == 0)
                *sVote = (v3 ? 1 : 0) | (v34 ? 2 : 0) | (vm ? 4 : 0) | (v3s ? 16 : 0);
        }
    };
    if (early_plans && wv == 0)
        compute_plans();
    if constexpr (G::CHUNK) {
        // the fragment of K step s (tap s / CPT, chunk s % CPT) for lane half
        // h is packed bytes [(2 s + h) * WB, + WB) of the channel's row: unit
        // 2 s + h.  Every unit of the loaded quads is expanded to 16 int8
        // values and unit u of channel c stored at u * FP + 16 c (units of
        // missing channels are zero)
        constexpr int WB = G::WB, FP = G::FP, UPQ = 16 / WB;
#pragma unroll
        for (int i = 0; i < FQ; ++i) {
            const int q = ft + i * FT;
            if (ft < 0 || (32 * QPR % FT != 0 && q >= 32 * QPR))
                break;
            const uint4 v = fq[i];
            const int c = q / QPR;
            uint8_t *dst = sF + (q - c * QPR) * UPQ * FP + c * 16;
            if (BITS == 8) {
                *(uint4 *)dst = v;
            } else if (BITS == 4) {
                const uint2 w0 = w4_word(v.x), w1 = w4_word(v.y), w2 = w4_word(v.z), w3 = w4_word(v.w);
                *(uint4 *)dst = make_uint4(w0.x, w0.y, w1.x, w1.y);
                *(uint4 *)(dst + FP) = make_uint4(w2.x, w2.y, w3.x, w3.y);
            } else {
                *(uint4 *)dst = w2_word(v.x);
                *(uint4 *)(dst + FP) = w2_word(v.y);
                *(uint4 *)(dst + 2 * FP) = w2_word(v.z);
                *(uint4 *)(dst + 3 * FP) = w2_word(v.w);
            }
        }
    }
    if constexpr (!G::CHUNK) {
        const uint8_t *wb = a.w + (size_t)(live ? ch : 0) * WROW;
        typedef typename G::BT TP;
#pragma unroll
        for (int s = 0; s < KS; ++s) {
            uint32_t d[4];
#pragma unroll
            for (int t = 0; t < G::TPF; ++t) {
                const int tp = TP::tap(s * G::TPF + t);
                const int ky = (tp >> 8) + h * DY, kx = tp & 255;
                uint32_t v = 0;
                if (tp >= 0 && live && ky < KH)
                    v = P == 2 ? (uint32_t)*(const uint16_t *)(wb + (ky * KW + kx) * 2)
                               : *(const uint32_t *)(wb + (ky * KW + kx) * 4);
                if (BITS == 8) {
                    d[t] = v;
                } else if (P == 2) {
                    d[t] = w4_half(v);
                } else if (BITS == 4) {
                    const uint2 e = w4_word(v);
                    d[2 * t] = e.x;
                    d[2 * t + 1] = e.y;
                } else {
                    const uint4 e = w2_word(v);
                    d[0] = e.x;
                    d[1] = e.y;
                    d[2] = e.z;
                    d[3] = e.w;
                }
            }
            A[s] = (v4i){(int32_t)d[0], (int32_t)d[1], (int32_t)d[2], (int32_t)d[3]};
        }
    }

    __syncthreads();
    if constexpr (G::CHUNK) {
#pragma unroll
        for (int s = 0; s < KS; ++s)
            A[s] = *(const v4i *)(sF + (2 * s + h) * G::FP + r32 * 16);
    }

    if (!early_plans && wv == 0)
        compute_plans();

    const bool st_ok = live && (r32 % (8 / BITS)) == 0;
    const int ch_byte = gy * 4 * BITS + ((r32 * BITS) >> 3);
    // the lane's pixel in a row tile: image row T*RT + r32/WOP, column r32%WOP
    const int lrow = r32 / WOP, lcol = r32 % WOP;
    const int lane_slot = (lrow * PP + lcol) * SB + (G::CHUNK ? 16 * h : h * DY * RB);
    for (; grp < a.ngroups; grp += gxn) {
        // the step's first image, its image count and the first output row
        // of its tiles (non-zero for the later bands of an image)
        int i0, ni, orow0;
        if constexpr (BAND) {
            i0 = (int)fdiv((uint32_t)grp, a.div_bands);
            ni = 1;
            orow0 = (grp - i0 * a.bands) * a.brows;
        } else {
            i0 = grp * a.ipw;
            ni = min(a.ipw, a.n - i0);
            orow0 = 0;
        }
        // stage the prefetched bytes into the tile interiors
#pragma unroll
        for (int u = 0; u < UPF; ++u) {
            const int q = tid + u * NT;
            if (P <= 4) {
                // 16 / P one-word (or half-word) pixels per quad (one image
                // per step when the image is not a whole number of quads)
                constexpr int PPQ = 16 / P;
                const int ii = a.quads ? (int)fdiv((uint32_t)q, a.div_imgq) : 0;
                const int p0 = PPQ * (q - ii * imgq);
                if (ii < ni && p0 < npix) {
                    uint8_t *tile = smem + ii * a.tile_bytes;
                    int iy = (int)fdiv((uint32_t)p0, a.div_w);
                    int ix = p0 - iy * a.w_;
                    const uint32_t wd[4] = {pf[u].x, pf[u].y, pf[u].z, pf[u].w};
#pragma unroll
                    for (int j = 0; j < PPQ; ++j) {
                        if (p0 + j < npix) {
                            uint8_t *dst = tile + ((iy + a.ph) * PP + ix + a.pw) * SB;
                            if constexpr (P == 2) {
                                // one unpacked word per pixel, pixel pairs per slot as at 8 bits
                                const uint32_t e = stage_half4(wd[j >> 1] >> (16 * (j & 1)));
                                *(uint32_t *)dst = e;
                                if (ix + a.pw > 0)
                                    *(uint32_t *)(dst - 4) = e;
                            } else {
                                stage_word<BITS>(dst, wd[j]);
                                if (BITS == 8 && ix + a.pw > 0)
                                    stage_word<BITS>(dst - 4, wd[j]);  // second pixel of the slot on its left
                            }
                        }
                        if (++ix == a.w_) {
                            ix = 0;
                            ++iy;
                        }
                    }
                }
            } else {
                // one quad is part of one pixel (P / 16 quads per pixel); a
                // band step holds one tile of a.trows rows
                int ii, qi;
                if constexpr (BAND) {
                    ii = q < a.trows * a.w_ * (P / 16) ? 0 : 1;
                    qi = q;
                } else {
                    ii = (int)fdiv((uint32_t)q, a.div_imgq);
                    qi = q - ii * imgq;
                }
                const int pix = qi / (P / 16);
                const int part = qi - pix * (P / 16);
                if (ii < ni) {
                    const int iy = (int)fdiv((uint32_t)pix, a.div_w);
                    const int ix = pix - iy * a.w_;
                    // whole images: interior rows below ph pad rows; bands:
                    // every tile row staged (pads as zero quads)
                    const int ty = BAND ? iy : iy + a.ph;
                    uint8_t *dst = smem + ii * a.tile_bytes + (ty * PP + ix + a.pw) * SB + part * (16 * 8 / BITS);
                    stage_word<BITS>(dst, pf[u].x);
                    stage_word<BITS>(dst + 32 / BITS, pf[u].y);
                    stage_word<BITS>(dst + 64 / BITS, pf[u].z);
                    stage_word<BITS>(dst + 96 / BITS, pf[u].w);
                }
            }
        }
        __syncthreads();
        const int4 e0 = sPlan[r32], e1 = sPlan[32 + r32];
        const int votes = *sVote;
        const bool all3 = (votes & 1) != 0, all34 = (votes & 2) != 0, mono = (votes & 4) != 0,
                   all3s = (votes & 16) != 0;
        // (the rare compression forms store straight from the lanes)
        const bool bulk_step = bulk && (stair || all3 || all3s || all34);
        const int64_t bt = (int64_t)(((uint64_t)(uint32_t)e0.y << 32) | (uint32_t)e0.x);  // raw: bias (+ 128 wsum)
        if (grp + gxn < a.ngroups)
            issue(grp + gxn);

        // work items: (image of the step, pair of row tiles), item = image *
        // pairs + pair; wave wv takes items wv, wv + NW, ...  The epilogue
        // gets the pair's first output row (even).
        const int items = ni * a.pairs;
        auto run = [&](auto epi) {
            for (int it = wv; it < items; it += NW) {
                const int ii = (int)fdiv((uint32_t)it, a.div_pairs);
                const int tp = it - ii * a.pairs;
                const uint8_t *p0 = smem + ii * a.tile_bytes + 2 * tp * RT * RB + lane_slot;
                v16i c0, c1;
                if constexpr (BAND)
                    img_steps_ahead<BITS, P, KH, KW, WOP, 4>(p0, p0 + RT * RB, A, c0, c1);
                else
                    img_steps<BITS, P, KH, KW, WOP, 0>(p0, p0 + RT * RB, A, c0, c1);
                // an opaque copy of the lane half keeps the general paths'
                // per-register pixel indexes and bounds checks in this body
                // (hoisted out of the loop they would hold a register or a
                // lane mask per output register throughout)
                int hx = h;
                __asm__ volatile("" : "+v"(hx));
                epi(i0 + ii, orow0 + 2 * tp * RT, hx, c0, c1);
            }
        };
        // the lane's staircase thresholds (read per step: registers only in
        // the staircase epilogue) from its column of the threshold-major
        // table (T[k] of the 32 channels at words 32 k ..)
        const int32_t *stair_col = (const int32_t *)sPlan + r32;
        auto stair_T = [&](int32_t *T) {
#pragma unroll
            for (int k = 0; k < NTH; ++k)
                T[k] = stair_col[32 * k];
        };
        // ---- epilogues: lane (r32, h) holds channel ch for tile pixels
        // p = 8*(v/4) + 4h + v%4 (register v): image row T*RT + p/WOP,
        // column p%WOP.  The form (every channel in the 32-bit or the 64-bit
        // strict plan, or any plan) is chosen once per step, outside the
        // tile loop.  Codes go straight to memory as bytes ----
        if constexpr (POOL) {
            typedef PoolWin<WOP> PW;
            // pooled rows of the pair start at orow / 2
            auto store_pool = [&](int img, int orow, int hx, const uint32_t *code) {
                uint32_t byte[8];
#pragma unroll
                for (int k = 0; k < 8; ++k)
                    byte[k] = img_pack_lanes<BITS>(code[k]);
                // whole pooled rows of pixels of one or two 32-channel
                // groups: the pair's 16 pooled pixels are assembled (packed
                // across lanes) in the wave's LDS staging (no barrier: the
                // wave reads only what it wrote) and leave as one group-wide
                // store per pixel.  (Packing them on the read-back instead,
                // as the unpooled path does, costs the one-word-pixel
                // instances 20-30 registers and a wave per SIMD)
                if (bulk_step) {
                    constexpr int WP = WOP / 2, YG = 4 * BITS;
                    if (st_ok) {
                        uint8_t *ob = sStep + (size_t)(img - i0) * a.hp * a.wp * YG + ((r32 * BITS) >> 3);
#pragma unroll
                        for (int k = 0; k < 8; ++k)
                            ob[(((orow >> 1) + PW::prow(k)) * WP + PW::pcol(k) + 2 * h) * YG] = (uint8_t)byte[k];
                    }
                    return;
                }
                auto fast = [&](auto yp) {
                    constexpr int YP = decltype(yp)::value, WP = WOP / 2, YG = 4 * BITS;
                    if (st_ok) {
#pragma unroll
                        for (int k = 0; k < 8; ++k)
                            sOut[(PW::prow(k) * WP + PW::pcol(k) + 2 * h) * YG + ((r32 * BITS) >> 3)] = (uint8_t)byte[k];
                    }
                    __asm__ volatile("" ::: "memory");
                    if (lane < 16) {
                        uint8_t *yt = a.y + (size_t)img * a.hp * a.wp * a.ypb + gy * YG +
                                      ((size_t)((orow >> 1) + lane / WP) * WP + lane % WP) * YP;
                        if constexpr (YG >= 16) {
#pragma unroll
                            for (int i = 0; i < YG; i += 16) {
                                // a first layer's output (its largest
                                // stream, twice its input at 8 bits) is
                                // written past the caches (INT-8 / INT-4
                                // CIFAR first layer 30.8 -> 29.4 / 28.3 ->
                                // 27.2 us, measured side by side; no gain
                                // on the later layers)
                                if constexpr (P <= 4)
                                    __builtin_nontemporal_store(*(const v4i *)(sOut + lane * YG + i), (v4i *)(yt + i));
                                else
                                    *(uint4 *)(yt + i) = *(const uint4 *)(sOut + lane * YG + i);
                            }
                        } else {
                            *(uint2 *)yt = *(const uint2 *)(sOut + lane * YG);
                        }
                    }
                    __asm__ volatile("" ::: "memory");
                };
                const bool rows = a.wp == WOP / 2 && (orow >> 1) + RT <= a.hp;
                if (rows && a.ypb == 4 * BITS) {
                    fast(ImgConst<4 * BITS>());
                } else if (rows && a.ypb == 8 * BITS) {
                    fast(ImgConst<8 * BITS>());
                } else {
                    if (!st_ok)
                        return;
                    uint8_t *yb = a.y + (size_t)img * a.hp * a.wp * a.ypb + ch_byte;
#pragma unroll
                    for (int k = 0; k < 8; ++k) {
                        const int pr = (orow >> 1) + PW::prow(k), pc = PW::pcol(k) + 2 * hx;
                        if (pr < a.hp && pc < a.wp)
                            yb[((size_t)pr * a.wp + pc) * a.ypb] = (uint8_t)byte[k];
                    }
                }
            };
            auto win = [&](int k, const v16i &c0, const v16i &c1, int32_t &x0, int32_t &x1, int32_t &y0,
                           int32_t &y1) {
                const int v = PW::v0(k), d = PW::dv(k);
                const v16i &ta = PW::t0(k) ? c1 : c0;
                const v16i &tb = PW::t1(k) ? c1 : c0;
                x0 = ta[v];
                x1 = ta[v + 1];
                y0 = tb[v + d];
                y1 = tb[v + d + 1];
            };
            if constexpr (stair) {
                // the level is non-decreasing in the accumulator for any
                // thresholds: the window's maximum is counted
                auto stair_pool = [&](auto tree) {
                    run([&](int img, int orow, int hx, const v16i &c0, const v16i &c1) {
                        int32_t T[NTH];
                        stair_T(T);
                        uint32_t code[8];
#pragma unroll
                        for (int k = 0; k < 8; ++k) {
                            int32_t x0, x1, y0, y1;
                            win(k, c0, c1, x0, x1, y0, y1);
                            const int32_t mx = max(max(x0, x1), max(y0, y1));
                            code[k] = decltype(tree)::value ? stair_tree_col<NTH>(mx, T, stair_col) : stair_level<NTH>(mx, T);
                        }
                        store_pool(img, orow, hx, code);
                    });
                };
                if (votes & 8)
                    stair_pool(ImgConst<1>());
                else
                    stair_pool(ImgConst<0>());
            } else if (all3) {
                const int4 p3 = sPlan[64 + r32];
                run([&](int img, int orow, int hx, const v16i &c0, const v16i &c1) {
                    uint32_t code[8];
#pragma unroll
                    for (int k = 0; k < 8; ++k) {
                        int32_t x0, x1, y0, y1;
                        win(k, c0, c1, x0, x1, y0, y1);
                        code[k] = img_code3(max(max(x0, x1), max(y0, y1)), p3, e1.x);
                    }
                    store_pool(img, orow, hx, code);
                });
            } else if (all3s) {
                run([&](int img, int orow, int hx, const v16i &c0, const v16i &c1) {
                    uint32_t code[8];
#pragma unroll
                    for (int k = 0; k < 8; ++k) {
                        int32_t x0, x1, y0, y1;
                        win(k, c0, c1, x0, x1, y0, y1);
                        code[k] = img_code3s(max(max(x0, x1), max(y0, y1)), e0, e1);
                    }
                    store_pool(img, orow, hx, code);
                });
            } else if (all34) {
                run([&](int img, int orow, int hx, const v16i &c0, const v16i &c1) {
                    uint32_t code[8];
#pragma unroll
                    for (int k = 0; k < 8; ++k) {
                        int32_t x0, x1, y0, y1;
                        win(k, c0, c1, x0, x1, y0, y1);
                        code[k] = img_code4(max(max(x0, x1), max(y0, y1)), e0, e1);
                    }
                    store_pool(img, orow, hx, code);
                });
            } else {
                // rare forms (plans outside the strict form, or multipliers
                // that are not positive): one pooled value at a time, kept
                // rolled so their 64-bit temporaries do not crowd the
                // registers of the fast forms
                run([&](int img, int orow, int hx, const v16i &c0, const v16i &c1) {
                    uint8_t *yb = a.y + (size_t)img * a.hp * a.wp * a.ypb + ch_byte;
#pragma unroll 1
                    for (int k = 0; k < 8; ++k) {
                        int32_t x0, x1, y0, y1;
                        // the window's registers, selected at run time
                        const int v = WOP == 32 ? 2 * k : (WOP == 16 ? 2 * (k & 3) : ((k & 2) << 2) + 2 * (k & 1));
                        const int d = WOP == 32 ? 0 : (WOP == 16 ? 8 : 4);
                        const bool sa = WOP == 32 ? false : (k >> 2) != 0;
                        const bool sb = WOP == 32 ? true : (k >> 2) != 0;
                        x0 = sa ? c1[v] : c0[v];
                        x1 = sa ? c1[v + 1] : c0[v + 1];
                        y0 = sb ? c1[v + d] : c0[v + d];
                        y1 = sb ? c1[v + d + 1] : c0[v + d + 1];
                        uint32_t code;
                        if (mono)
                            code = img_code<SL>(max(max(x0, x1), max(y0, y1)), e0, e1, a.clip_lo, a.clip_hi);
                        else
                            code = max(max(img_code<SL>(x0, e0, e1, a.clip_lo, a.clip_hi),
                                           img_code<SL>(x1, e0, e1, a.clip_lo, a.clip_hi)),
                                       max(img_code<SL>(y0, e0, e1, a.clip_lo, a.clip_hi),
                                           img_code<SL>(y1, e0, e1, a.clip_lo, a.clip_hi)));
                        const uint32_t byte = img_pack_lanes<BITS>(code);
                        const int pr = (orow >> 1) + (WOP == 32 ? 0 : (WOP == 16 ? k >> 2 : 2 * (k >> 2) + ((k >> 1) & 1)));
                        const int pc = (WOP == 32 ? 4 * (k >> 1) + (k & 1)
                                                  : (WOP == 16 ? 4 * ((k & 3) >> 1) + (k & 1) : (k & 1))) + 2 * hx;
                        if (st_ok && pr < a.hp && pc < a.wp)
                            yb[((size_t)pr * a.wp + pc) * a.ypb] = (uint8_t)byte;
                    }
                });
            }
        } else if (!stair && a.epi == EPI_RAW32) {
            run([&](int img, int orow, int hx, const v16i &c0, const v16i &c1) {
                if (!live)
                    return;
#pragma unroll
                for (int t = 0; t < 2; ++t) {
#pragma unroll
                    for (int v = 0; v < 16; ++v) {
                        const int p = 8 * (v >> 2) + 4 * hx + (v & 3);
                        const int oy = orow + t * RT + p / WOP, ox = p % WOP;
                        const int32_t av = t ? c1[v] : c0[v];
                        if (oy < a.ho && ox < a.wo)
                            ((int32_t *)a.y)[(((size_t)img * a.ho + oy) * a.wo + ox) * a.m + ch] =
                                (int32_t)(uint32_t)(uint64_t)((int64_t)(av >> SL) + bt);
                    }
                }
            });
        } else {
            auto store_tiles = [&](int img, int orow, int hx, const uint32_t *code) {
                // whole rows of pixels of one or two 32-channel groups: every
                // lane writes its channel's code bytes into the wave's LDS
                // staging (no barrier: the wave reads only what it wrote);
                // each lane then packs one of the pair's 64 pixels and stores
                // it with one group-wide store (packing across lanes and byte
                // stores straight from them cost 2-4 vector instructions per
                // code and 32 store instructions per wave)
                auto fast = [&](auto yp) {
                    constexpr int YP = decltype(yp)::value, YG = 4 * BITS;
#pragma unroll
                    for (int v = 0; v < 32; ++v)
                        sOut[((v >> 4) * 32 + 8 * ((v & 15) >> 2) + 4 * h + (v & 3)) * G::OPS + r32] = (uint8_t)code[v];
                    __asm__ volatile("" ::: "memory");
                    uint8_t *yt = a.y + (size_t)img * a.ho * a.wo * a.ypb + gy * YG + ((size_t)orow * WOP + lane) * YP;
                    img_pack_store<BITS>(yt, sOut + lane * G::OPS);
                    __asm__ volatile("" ::: "memory");
                };
                const bool rows = a.wo == WOP && orow + 2 * RT <= a.ho;
                if (rows && a.ypb == 4 * BITS) {
                    fast(ImgConst<4 * BITS>());
                } else if (rows && a.ypb == 8 * BITS) {
                    fast(ImgConst<8 * BITS>());
                } else {
                    uint32_t byte[32];
#pragma unroll
                    for (int v = 0; v < 32; ++v)
                        byte[v] = img_pack_lanes<BITS>(code[v]);
                    if (!st_ok)
                        return;
                    uint8_t *yb = a.y + (size_t)img * a.ho * a.wo * a.ypb + ch_byte;
#pragma unroll
                    for (int v = 0; v < 32; ++v) {
                        const int p = 8 * ((v & 15) >> 2) + 4 * hx + (v & 3);
                        const int oy = orow + (v >> 4) * RT + p / WOP, ox = p % WOP;
                        if (oy < a.ho && ox < a.wo)
                            yb[((size_t)oy * a.wo + ox) * a.ypb] = (uint8_t)byte[v];
                    }
                }
            };
            if constexpr (stair) {
                // sorted thresholds (every channel): the comparison tree;
                // otherwise the count
                auto stair_tiles = [&](auto tree) {
                    run([&](int img, int orow, int hx, const v16i &c0, const v16i &c1) {
                        int32_t T[NTH];
                        stair_T(T);
                        uint32_t code[32];
#pragma unroll
                        for (int v = 0; v < 16; ++v) {
                            if (decltype(tree)::value) {
                                code[v] = stair_tree_col<NTH>(c0[v], T, stair_col);
                                code[16 + v] = stair_tree_col<NTH>(c1[v], T, stair_col);
                            } else {
                                code[v] = stair_level<NTH>(c0[v], T);
                                code[16 + v] = stair_level<NTH>(c1[v], T);
                            }
                        }
                        store_tiles(img, orow, hx, code);
                    });
                };
                if (votes & 8)
                    stair_tiles(ImgConst<1>());
                else
                    stair_tiles(ImgConst<0>());
            } else if (all3s) {
                // (not the three-instruction form: its inline-asm clamp would
                // be the first reader of the matrix results)
                run([&](int img, int orow, int hx, const v16i &c0, const v16i &c1) {
                    uint32_t code[32];
#pragma unroll
                    for (int v = 0; v < 16; ++v) {
                        code[v] = img_code3s(c0[v], e0, e1);
                        code[16 + v] = img_code3s(c1[v], e0, e1);
                    }
                    store_tiles(img, orow, hx, code);
                });
            } else if (all34) {
                run([&](int img, int orow, int hx, const v16i &c0, const v16i &c1) {
                    uint32_t code[32];
#pragma unroll
                    for (int v = 0; v < 16; ++v) {
                        code[v] = img_code4(c0[v], e0, e1);
                        code[16 + v] = img_code4(c1[v], e0, e1);
                    }
                    store_tiles(img, orow, hx, code);
                });
            } else {
                run([&](int img, int orow, int hx, const v16i &c0, const v16i &c1) {
                    uint8_t *yb = a.y + (size_t)img * a.ho * a.wo * a.ypb + ch_byte;
#pragma unroll
                    for (int t = 0; t < 2; ++t) {
#pragma unroll 1
                        for (int v = 0; v < 16; ++v) {
                            const uint32_t byte = img_pack_lanes<BITS>(
                                img_code<SL>(t ? c1[v] : c0[v], e0, e1, a.clip_lo, a.clip_hi));
                            const int p = 8 * (v >> 2) + 4 * hx + (v & 3);
                            const int oy = orow + t * RT + p / WOP, ox = p % WOP;
                            if (st_ok && oy < a.ho && ox < a.wo)
                                yb[((size_t)oy * a.wo + ox) * a.ypb] = (uint8_t)byte;
                        }
                    }
                });
            }
        }
        __syncthreads();  // every wave is done with this step's tiles
        if (bulk_step) {
            // the step's images are consecutive in the output: one flat copy,
            // past the caches (the output is the layer's largest stream;
            // CIFAR first layer INT-8 / INT-4 29.5 -> 27.3 / 26.9 -> 25.7 us
            // against each row pair's 16-lane stores, measured side by side)
            const int nb16 = ni * a.hp * a.wp * (4 * BITS) / 16;
            uint8_t *yo = a.y + (size_t)i0 * a.hp * a.wp * a.ypb;
            for (int i = tid; i < nb16; i += NT)
                __builtin_nontemporal_store(*(const v4i *)(sStep + 16 * i), (v4i *)(yo + 16 * (size_t)i));
        }
    }
}

// Grid: as many workgroups as the device holds at once (image groups each),
// so no workgroup starts only after others have finished.
template <typename K>
hipError_t launch_img_grid(K kernel, const ImgArgs &a, int flds, int cus, hipStream_t s, size_t extra = 0)
{
    const size_t lds = (size_t)a.ipw * a.tile_bytes + flds + extra;
    if (lds > 64 * 1024) {
        // past the default dynamic LDS limit: raise it to the CU's 160 KB
        // (once per instance)
        static bool attr_set = false;
        if (!attr_set) {
            if (hipFuncSetAttribute((const void *)kernel, hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024) !=
                hipSuccess)
                (void)hipGetLastError();
            attr_set = true;
        }
    }
    int per_cu = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kernel, 256, lds) != hipSuccess || per_cu < 1)
        per_cu = 1;
    const int gy = (a.m + 31) / 32;
    int64_t gx = ((int64_t)cus * per_cu + gy - 1) / gy;
    if (gx > a.ngroups)
        gx = a.ngroups;
    if (gx < 1)
        gx = 1;
    hipLaunchKernelGGL(kernel, dim3((unsigned)gx, (unsigned)gy), dim3(256), lds, s, a.x, a.ngroups, a.bands,
                       a.brows, a.trows, a.ph, a.h, a.w_, a.div_bands.mul, a.div_bands.shr, (int32_t)gx, a.m, a);
    return hipGetLastError();
}

template <int BITS, int P, int K, int WOP, bool BAND = false>
hipError_t launch_img(const ImgArgs &a, int cus, hipStream_t s)
{
    constexpr int FLDS = ImgGeom<BITS, P, K, K, WOP>::XLDS;
    // pooled first layers: the step's output images in LDS
    const size_t step_out = P <= 4 && a.pool ? (size_t)a.ipw * a.hp * a.wp * a.ypb : 0;
    if constexpr (BITS != 8) {
        if (a.epi == EPI_STAIR) {
            if (a.pool)
                return launch_img_grid(conv_img_kernel<BITS, P, K, K, WOP, true, BAND, true>, a, FLDS, cus, s,
                                       step_out);
            return launch_img_grid(conv_img_kernel<BITS, P, K, K, WOP, false, BAND, true>, a, FLDS, cus, s);
        }
    }
    if (a.pool)
        return launch_img_grid(conv_img_kernel<BITS, P, K, K, WOP, true, BAND, false>, a, FLDS, cus, s,
                               step_out);
    return launch_img_grid(conv_img_kernel<BITS, P, K, K, WOP, false, BAND, false>, a, FLDS, cus, s);
}

}  // namespace qnn
