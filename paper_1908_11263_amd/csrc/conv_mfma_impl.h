// Implicit-GEMM quantized convolution on the gfx950 int8 matrix cores.
//
// Computes Sec. III-A Eq. (2) / Sec. III-B Eq. (6) for 8-, 4- and 2-bit
// layers: every output O(m, x, y) is the dot product of filter bank W(m) with
// the im2col column of pixel (x, y), accumulated in 32 bits, followed by the
// per-channel scale-and-clamp compression (Sec. III-A) or a raw int32 store.
//
// GEMM view.  Rows = output channels (A operand = weights), columns = output
// pixels (B operand = im2col), K = kh*kw*C.  One workgroup (4 waves) owns a
// tile of 16*MR output channels and 64*NC output pixels (a block of output
// rows/columns of one image, or several whole small images); each wave
// computes all 16*MR channels for 16*NC of the pixels with
// v_mfma_i32_16x16x64_i8.  As in the paper's multi-core split (Sec. IV-B),
// workgroups are spread over output pixels and the filter banks are shared:
// each workgroup stages its filter tile once and then walks a grid-stride
// sequence of pixel tiles.
//
// Local memory (LDS) holds
//   * the filter tile as int8 in the order the MFMA consumes it;
//   * the input tile plus its halo, unpacked to int8 once per tile, so each
//     input byte is expanded once and then read by all kh*kw taps that use it
//     (im2col exists only as addresses into this tile, never materialised);
//   * the packed output tile, copied out with coalesced stores.
//
// Exact integer tricks (each leaves the accumulator exact):
//   * 8-bit activations are unsigned, the matrix cores multiply signed bytes:
//     x - 128 is staged (x ^ 0x80) and 128 * sum_k w[m, k] is added back;
//     padding taps (x = 0) are staged as -128, so the identity holds there too.
//   * 4-/2-bit weights are staged as 16*w / 64*w (the code shifted into the
//     top of the byte, so no sign extension is needed) and the accumulator
//     is shifted right by 4 / 6 afterwards, which is exact.
#pragma once

#include "qnn_internal.h"

namespace qnn {

typedef int32_t v4i __attribute__((ext_vector_type(4)));

// Sub-byte K order.  Within each packed 32-bit word (8 INT-4 or 16 INT-2
// codes, lowest channel in the lowest bits) the unpacked bytes are stored
// field-major: INT-4 word -> [c0 c2 c4 c6 | c1 c3 c5 c7], INT-2 word ->
// [c0 c4 c8 c12 | c1 c5 c9 c13 | c2 ... | c3 ... c15].  Weights and
// activations use the same order at the same K positions (packed words of a
// filter row and of a pixel both start at multiples of 8 / 16 channels), so
// every dot product is unchanged, and each unpack is a mask and a shift.

// Activations, one packed word -> 4 (INT-8, offset by -128), 8 or 16 bytes.
template <int BITS>
__device__ __forceinline__ void stage_word(uint8_t *dst, uint32_t v)
{
    if (BITS == 8) {
        *(uint32_t *)dst = v ^ 0x80808080u;
    } else if (BITS == 4) {
        *(uint2 *)dst = make_uint2(v & 0x0F0F0F0Fu, (v >> 4) & 0x0F0F0F0Fu);
    } else {
        *(uint4 *)dst = make_uint4(v & 0x03030303u, (v >> 2) & 0x03030303u, (v >> 4) & 0x03030303u,
                                   (v >> 6) & 0x03030303u);
    }
}

// INT-2 codes as FP4 (OCP e2m1: sign, 2-bit exponent with bias 1, 1-bit
// mantissa) for the 32x32x64 f8f6f4 matrix instruction.  The nibbles 0000,
// 0001, 0010, 0011 encode 0, 0.5, 1, 1.5, so an activation code x placed in
// a nibble IS the e2m1 value x/2; a weight code (two's complement b1 b0)
// becomes w/2: 01 -> 0001 (0.5), 10 -> 1010 (-1), 11 -> 1001 (-0.5).  Every
// product is then x*w/4, restored by an exponent-2 block scale.  One packed
// word (16 codes) -> 8 bytes: the even-position codes c0 c2 .. c14 in the low
// word's nibbles 0..7 and the odd ones in the high word's (the same order for
// weights and activations, so the dot products are unchanged).
__device__ __forceinline__ uint2 x2_word_f4(uint32_t v)
{
    return make_uint2(v & 0x33333333u, (v >> 2) & 0x33333333u);
}

__device__ __forceinline__ uint32_t w2_nibbles_f4(uint32_t t)
{
    const uint32_t o = t & 0x11111111u;  // b0 of every nibble
    const uint32_t s = t & 0x22222222u;  // b1 (the sign) of every nibble
    return (s << 2) | (s & ~(o << 1)) | o;
}

__device__ __forceinline__ uint2 w2_word_f4(uint32_t v)
{
    const uint2 t = x2_word_f4(v);
    return make_uint2(w2_nibbles_f4(t.x), w2_nibbles_f4(t.y));
}

// INT-1 codes (value 2*bit - 1 for weights and activations alike) as e2m1
// +1.0 (0010) and -1.0 (1010): one packed word (32 codes) -> 16 bytes, word
// j of the result holding codes j, j+4, .., j+28 in its nibbles 0..7.
__device__ __forceinline__ uint4 b1_word_f4(uint32_t v)
{
    const uint32_t m = 0x11111111u, neg = 0xAAAAAAAAu;
    return make_uint4(neg ^ ((v & m) << 3), neg ^ (((v >> 1) & m) << 3), neg ^ (((v >> 2) & m) << 3),
                      neg ^ (((v >> 3) & m) << 3));
}

// Weights, one packed word -> 8 (INT-4) or 16 (INT-2) bytes holding 16*w /
// 64*w: the code moved to the top of its byte is exactly that signed byte.
__device__ __forceinline__ uint2 w4_word(uint32_t v)
{
    return make_uint2((v << 4) & 0xF0F0F0F0u, v & 0xF0F0F0F0u);
}

__device__ __forceinline__ uint4 w2_word(uint32_t v)
{
    return make_uint4((v << 6) & 0xC0C0C0C0u, (v << 4) & 0xC0C0C0C0u, (v << 2) & 0xC0C0C0C0u,
                      v & 0xC0C0C0C0u);
}

__device__ __forceinline__ int wave_sum(int s)
{
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1)
        s += __shfl_xor(s, off, 64);
    return s;
}

// Rounding right shift floor(t / 2^s + 1/2) without forming t + 2^(s-1):
// with t = q*2^s + r (0 <= r < 2^s) the result is q + [r >= 2^(s-1)], and
// r >= 2^(s-1) is bit s-1 of t.
__device__ __forceinline__ int64_t round_shift(int64_t t, int s)
{
    return s == 0 ? t : (t >> s) + ((t >> (s - 1)) & 1);
}

// Stage 16 packed weight bytes as int8 at dst: 16, 32 or 64 bytes for 8, 4,
// 2 bits, in the sub-byte K order above.
template <int BITS>
__device__ __forceinline__ void stage_w16(int8_t *dst, uint4 v)
{
    if (BITS == 8) {
        *(uint4 *)dst = v;
    } else if (BITS == 4) {
        const uint2 a = w4_word(v.x), b = w4_word(v.y), c = w4_word(v.z), d = w4_word(v.w);
        *(uint4 *)dst = make_uint4(a.x, a.y, b.x, b.y);
        *(uint4 *)(dst + 16) = make_uint4(c.x, c.y, d.x, d.y);
    } else {
        *(uint4 *)dst = w2_word(v.x);
        *(uint4 *)(dst + 16) = w2_word(v.y);
        *(uint4 *)(dst + 32) = w2_word(v.z);
        *(uint4 *)(dst + 48) = w2_word(v.w);
    }
}

// Per-channel requantization plan.  For mult > 0 the compressed code is a
// non-decreasing step function of the accumulator: it is lo up to a_base and
// hi from a_base + D on, and in between
//   y = Q + ((d * mult + R) >> shift),  d = acc - a_base in [0, D],
// with (a_base + bias) * mult + 2^(shift-1) = Q * 2^shift + R.  When D and
// mult fit 24 bits this is exact with one 24-bit multiply-add per output if
// R + D * mult < 2^32 (mode 1), else with a 32x32->64 multiply-add (mode 2);
// other channels use the direct 64-bit form.  Two 16-byte words per channel:
//   modes 3, 4: e0 = {S t_lo, S D, mult, S n0 lo}, e1 = {shift + log2 S, S n0 hi, mode, 0}
//               (mode 3 when the expression fits 32 bits, mode 4 with a 64-bit product)
//   modes 1, 2: e0 = {a_base, D, mult, R}, e1 = {Q, shift, mode, 0}
//   direct:     e0 = {bias lo, bias hi, mult, shift}, e1 = {0, 0, 0, 0}
// (RAW32 uses the slow word's bias only.)
// floor(a / b) for 0 < b < 2^31 and |a| < 2^40: the hardware reciprocal of b
// refined by two Newton steps times a is within one of the true quotient
// (within 2^-10 of it: relative error below 2^-50), and the estimate is
// corrected exactly in integers.  No division sequence: its steps share the
// VCC register, which keeps two divisions from overlapping.
__device__ __forceinline__ int64_t floor_div_pos(int64_t a, int64_t b)
{
    const double bd = (double)b;
    double r = __builtin_amdgcn_rcp(bd);
    r = __builtin_fma(__builtin_fma(-bd, r, 1.0), r, r);
    r = __builtin_fma(__builtin_fma(-bd, r, 1.0), r, r);
    const int64_t q = (int64_t)__builtin_floor((double)a * r);
    const int64_t rem = a - q * b;
    return q + (int64_t)(rem >= b) - (int64_t)(rem < 0);
}

__device__ __forceinline__ void requant_plan(int64_t bias, int32_t mult, int32_t shift, int32_t lo,
                                             int32_t hi, bool requant, int scale_log2, int4 &e0,
                                             int4 &e1)
{
    e0 = make_int4((int32_t)(uint32_t)(uint64_t)bias, (int32_t)(bias >> 32), mult, shift);
    e1 = make_int4(0, 0, 0, 0);
    if (!requant || mult <= 0 || shift > 30 || bias > ((int64_t)1 << 40) || bias < -((int64_t)1 << 40))
        return;
    const int64_t half = shift > 0 ? ((int64_t)1 << (shift - 1)) : 0;
    const int64_t two_s = (int64_t)1 << shift;
    // smallest accumulator whose code reaches p: ceil((p 2^s - half) / mult) - bias
    const int64_t t_lo = -floor_div_pos(half - (int64_t)lo * two_s, mult) - bias;
    const int64_t t_hi = -floor_div_pos(half - (int64_t)hi * two_s, mult) - bias;
    // Strict form (modes 3, 4): with mult <= 2^shift the code rises by at most one
    // per accumulator unit, so it is exactly lo at t_lo and hi at t_hi and
    //   code = (clamp(acc' - S t_lo, 0, S D) * mult + S n0) >> (shift + log2 S)
    // on the scaled accumulator acc' = S acc (S = 16 / 64 for 4 / 2 bits), where
    // n0 = (t_lo + bias) mult + 2^(shift-1) = lo 2^shift + R, 0 <= R < 2^shift.
    if (mult <= two_s && lo >= 0 && shift + scale_log2 <= 31) {
        const int64_t S = (int64_t)1 << scale_log2;
        const int64_t Dn = t_hi - t_lo;
        const int64_t n0s = (t_lo + bias) * (int64_t)mult + half;
        const int64_t A = S * t_lo;
        if (A >= INT32_MIN && A <= INT32_MAX && Dn >= 0 && S * Dn < (1 << 24) && mult < (1 << 24) &&
            n0s >= 0 && S * (n0s + Dn * (int64_t)mult) < ((int64_t)1 << 62)) {
            const int64_t rs = S * n0s;
            // mode 3: the whole expression fits 32 bits; mode 4: 64-bit multiply-add
            const int md = S * (n0s + Dn * (int64_t)mult) < ((int64_t)1 << 32) ? 3 : 4;
            e0 = make_int4((int32_t)A, (int32_t)(S * Dn), mult, (int32_t)(uint32_t)rs);
            e1 = make_int4(shift + scale_log2, (int32_t)(rs >> 32), md, 0);
            return;
        }
    }
    const int64_t a_base = t_lo - 1;
    const int64_t D = t_hi - a_base;
    if (a_base < INT32_MIN || t_hi > INT32_MAX || D < 0 || D >= (1 << 24) || mult >= (1 << 24))
        return;
    const int64_t n0 = (a_base + bias) * (int64_t)mult + half;
    const int64_t Q = n0 >> shift;
    const int64_t R = n0 - Q * two_s;
    if (Q < INT32_MIN || Q > INT32_MAX)
        return;
    e0 = make_int4((int32_t)a_base, (int32_t)D, mult, (int32_t)(uint32_t)R);
    // mode 1: R + D * mult fits 32 bits; mode 2: it needs the 64-bit product
    e1 = make_int4((int32_t)Q, shift, R + D * (int64_t)mult < ((int64_t)1 << 32) ? 1 : 2, 0);
}

// Staircase thresholds of one channel (Sec. III-A, Eq. (4)) moved onto the
// kernel's accumulator: acc + bias >= tau  <=>  S acc >= S (tau - bias), with
// S = 2^scale_log2 the weight scale of the sub-byte staging.  Values are
// clamped to int32: S acc never equals INT32_MAX (an odd number, S acc is a
// multiple of S), so the clamped comparisons keep their results.  Unused
// slots (and missing channels) hold INT32_MAX, which no accumulator reaches.
__device__ __forceinline__ void stair_thresholds(const int32_t *tau, int nt, int64_t bias,
                                                 int scale_log2, int32_t *dst16)
{
#pragma unroll
    for (int p = 0; p < 16; ++p) {
        int32_t v = INT32_MAX;
        if (tau && p < nt) {
            int64_t t = ((int64_t)tau[p] - bias) * ((int64_t)1 << scale_log2);
            t = t < INT32_MIN ? INT32_MIN : (t > INT32_MAX ? INT32_MAX : t);
            v = (int32_t)t;
        }
        dst16[p] = v;
    }
}

// Staircase level of a (scaled) accumulator: the number of thresholds at or
// below it.
template <int NT>
__device__ __forceinline__ uint32_t stair_level(int32_t acc, const int32_t *T)
{
    uint32_t code = 0;
#pragma unroll
    for (int p = 0; p < NT; ++p)
        code += acc >= T[p] ? 1u : 0u;
    return code;
}

// One batch of U packed-input quads of a tile: issue the loads ...
// (F4: INT-2 codes staged as e2m1 nibbles, 4 bits per code, instead of bytes)
template <int BITS, bool Q16, int U, int NT = 256, bool F4 = false>
__device__ __forceinline__ void halo_issue(const ConvArgs &a, int b0, int totq, int n0, int iy0,
                                           int ix0, uint4 *v, int *dst)
{
    constexpr int QB = Q16 ? 16 : 4;
    constexpr int QU = QB * (F4 ? 4 : 8) / BITS;
    const uint8_t *x = a.x;
#pragma unroll
    for (int u = 0; u < U; ++u) {
        const int idx = b0 + u * NT;
        const int pix = (int)fdiv((uint32_t)idx, a.div_pbq);
        const int q = idx - pix * a.pbq;
        const int hrow = (int)fdiv((uint32_t)pix, a.div_hwd);
        const int hx = pix - hrow * a.hwd;
        const int tI = (int)fdiv((uint32_t)hrow, a.div_hh);
        const int hy = hrow - tI * a.hh;
        const int nn = n0 + tI, iy = iy0 + hy, ix = ix0 + hx;
        const bool live = idx < totq;
        dst[u] = live ? pix * a.ps + q * QU : -1;
        // one predicate (unsigned compares also reject negative rows and
        // columns); the input pixel index fits 31 bits (n*h*w < 2^31)
        const bool ok = live && nn < a.n && (uint32_t)iy < (uint32_t)a.h && (uint32_t)ix < (uint32_t)a.w_;
        const uint32_t gpix = ((uint32_t)nn * (uint32_t)a.h + (uint32_t)iy) * (uint32_t)a.w_ + (uint32_t)ix;
        const uint8_t *src = x + (size_t)gpix * (uint32_t)a.pb + q * QB;
        v[u] = make_uint4(0, 0, 0, 0);
        if (ok) {
            if (Q16)
                v[u] = *(const uint4 *)src;
            else
                v[u].x = *(const uint32_t *)src;
        }
    }
}

// ... and unpack them into the LDS tile.
template <int BITS, bool Q16, int U, bool F4 = false>
__device__ __forceinline__ void halo_store(uint8_t *sX, const uint4 *v, const int *dst)
{
    constexpr int W = (F4 ? 16 : 32) / BITS;  // staged bytes per packed word
#pragma unroll
    for (int u = 0; u < U; ++u) {
        if (dst[u] >= 0) {
            uint8_t *d = sX + dst[u];
            if (F4 && BITS == 1) {
                *(uint4 *)d = b1_word_f4(v[u].x);
                if (Q16) {
                    *(uint4 *)(d + 16) = b1_word_f4(v[u].y);
                    *(uint4 *)(d + 32) = b1_word_f4(v[u].z);
                    *(uint4 *)(d + 48) = b1_word_f4(v[u].w);
                }
                continue;
            }
            if (F4) {
                const uint2 p = x2_word_f4(v[u].x);
                if (Q16) {
                    const uint2 q = x2_word_f4(v[u].y), r = x2_word_f4(v[u].z), t = x2_word_f4(v[u].w);
                    *(uint4 *)d = make_uint4(p.x, p.y, q.x, q.y);
                    *(uint4 *)(d + 16) = make_uint4(r.x, r.y, t.x, t.y);
                } else {
                    *(uint2 *)d = p;
                }
                continue;
            }
            stage_word<BITS>(d, v[u].x);
            if (Q16) {
                stage_word<BITS>(d + W, v[u].y);
                stage_word<BITS>(d + 2 * W, v[u].z);
                stage_word<BITS>(d + 3 * W, v[u].w);
            }
        }
    }
}

// Whole tile (or the part after the first batch) in batches of U.
template <int BITS, bool Q16, int U, int NT = 256, bool F4 = false>
__device__ __forceinline__ void halo_stage_from(const ConvArgs &a, uint8_t *sX, int b_first, int n0,
                                                int iy0, int ix0)
{
    const int totq = a.ti * a.hh * a.hwd * a.pbq;
    for (int b0 = b_first; b0 < totq; b0 += NT * U) {
        uint4 v[U];
        int dst[U];
        halo_issue<BITS, Q16, U, NT, F4>(a, b0, totq, n0, iy0, ix0, v, dst);
        halo_store<BITS, Q16, U, F4>(sX, v, dst);
    }
}

// Tile index -> first image / output row / output column.
struct TileXY {
    int n0, oy0, ox0, iy0, ix0;
};

__device__ __forceinline__ TileXY tile_xy(const ConvArgs &a, int tile)
{
    TileXY r;
    const int tq = (int)fdiv((uint32_t)tile, a.div_tx);
    const int tx = tile - tq * a.tiles_x;
    const int tn = (int)fdiv((uint32_t)tq, a.div_ty);
    const int ty = tq - tn * a.tiles_y;
    r.n0 = tn * a.ti;
    r.oy0 = ty * a.th;
    r.ox0 = tx * a.tw;
    r.iy0 = r.oy0 * a.sh - a.ph;
    r.ix0 = r.ox0 * a.sw - a.pw;
    return r;
}

template <int BITS, int MR, int NC, bool AL16>
__global__ void __launch_bounds__(256, 2) conv_mfma_kernel(ConvArgs a)
{
    extern __shared__ __align__(16) uint8_t smem[];
    constexpr int MT = 16 * MR;
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wv = tid >> 6;
    const int m0 = blockIdx.y * MT;
    const int kch = 4 * a.ksteps;

    int8_t *sW = (int8_t *)smem;
    int32_t *sTab = (int32_t *)(smem + a.off_tab);
    int32_t *sNat = sTab + kch;
    int32_t *sVld = sNat + kch;
    int32_t *sWsum = (int32_t *)(smem + a.off_wsum);           // [MT] filter sums (8 bits), [4] votes
    int4 *sEpi = (int4 *)(smem + a.off_wsum + 4 * MT + 16);      // [MT][4]: plan (2) or 16 thresholds
    uint8_t *sX = smem + a.off_x;
    uint8_t *sOut = smem + a.off_out;

    // ---- prologue: every independent load is issued before any is used ----
    // per-channel epilogue parameters (one thread per channel)
    // (channel ch = wave + 4 * lane, so every wave computes a quarter of the plans)
    const int pch = wv + 4 * lane;
    const bool has_ch = lane < MT / 4;
    int32_t p_bias = 0, p_mult = 0, p_shift = 0;
    if (has_ch && m0 + pch < a.m) {
        if (a.bias)
            p_bias = a.bias[m0 + pch];
        if (a.epi == EPI_REQUANT) {
            p_mult = a.mult[m0 + pch];
            p_shift = a.shift[m0 + pch];
        }
    }
    // filter tile, first batch (contiguous rows, natural order = chunk order)
    const bool wfast = !a.row_mode && (a.wrow & 15) == 0;
    const int qrow = a.wrow >> 4;
    const int nq = MT * qrow;
    constexpr int UW = 8;
    uint4 wq[UW];
    if (wfast) {
#pragma unroll
        for (int u = 0; u < UW; ++u) {
            const int idx = tid + u * 256;
            const int row = (int)fdiv((uint32_t)idx, a.div_qrow);
            wq[u] = make_uint4(0, 0, 0, 0);
            if (idx < nq && m0 + row < a.m)
                wq[u] = *(const uint4 *)(a.w + (size_t)(m0 + row) * a.wrow + (idx - row * qrow) * 16);
        }
    }
    // input tile of the first pixel tile, first batch
    int tile = blockIdx.x;
    TileXY T = tile_xy(a, tile < a.ntiles ? tile : 0);
    constexpr int UH = 4;
    uint4 hq[UH];
    int hd[UH];
    const int totq = a.ti * a.hh * a.hwd * a.pbq;
    if (a.quad16)
        halo_issue<BITS, true, UH>(a, tid, tile < a.ntiles ? totq : 0, T.n0, T.iy0, T.ix0, hq, hd);
    else
        halo_issue<BITS, false, UH>(a, tid, tile < a.ntiles ? totq : 0, T.n0, T.iy0, T.ix0, hq, hd);

    // K-chunk tables: chunk j = 16 consecutive K bytes.  sTab: offset of the
    // chunk in the input tile relative to a pixel's top-left tap; sNat: offset
    // in the natural (ky, kx, c) order of a filter bank; sVld: bytes of the
    // chunk that belong to the filter (the rest meets zero weights).
    for (int j = tid; j < kch; j += 256) {
        int hoff = 0, nat = 0, vld = 0;
        if (j < a.kchunks) {
            if (a.row_mode) {
                int ky = (int)fdiv((uint32_t)j, a.div_tab_a), r = (j - ky * a.cpr) * 16;
                hoff = ky * a.hwd * a.ps + r;
                nat = ky * a.row_len + r;
                vld = min(16, a.row_len - r);
            } else {
                int cpt = a.c8 >> 4;
                int tap = (int)fdiv((uint32_t)j, a.div_tab_a), c16 = j - tap * cpt;
                int ky = (int)fdiv((uint32_t)tap, a.div_tab_kw), kx = tap - ky * a.kw;
                hoff = (ky * a.hwd + kx) * a.ps + c16 * 16;
                nat = j * 16;
                vld = 16;
            }
        }
        sTab[j] = hoff;
        sNat[j] = nat;
        sVld[j] = vld;
    }
    __syncthreads();

    // filter tile -> int8 (4-/2-bit codes scaled by 16 / 64), chunk order
    const int ncol = kch * 4;
    if (wfast) {
#pragma unroll
        for (int u = 0; u < UW; ++u) {
            const int idx = tid + u * 256;
            if (idx < nq) {
                const int row = (int)fdiv((uint32_t)idx, a.div_qrow);
                stage_w16<BITS>(sW + row * a.kp + (idx - row * qrow) * (128 / BITS), wq[u]);
            }
        }
        for (int b0 = tid + 256 * UW; b0 < nq; b0 += 256 * UW) {
#pragma unroll
            for (int u = 0; u < UW; ++u) {
                const int idx = b0 + u * 256;
                const int row = (int)fdiv((uint32_t)idx, a.div_qrow);
                wq[u] = make_uint4(0, 0, 0, 0);
                if (idx < nq && m0 + row < a.m)
                    wq[u] = *(const uint4 *)(a.w + (size_t)(m0 + row) * a.wrow + (idx - row * qrow) * 16);
            }
#pragma unroll
            for (int u = 0; u < UW; ++u) {
                const int idx = b0 + u * 256;
                if (idx < nq) {
                    const int row = (int)fdiv((uint32_t)idx, a.div_qrow);
                    stage_w16<BITS>(sW + row * a.kp + (idx - row * qrow) * (128 / BITS), wq[u]);
                }
            }
        }
        // zero the chunks that round K up to whole MFMA steps
        const int padc = kch - a.kchunks;
        for (int i = tid; i < MT * padc; i += 256) {
            const int row = i / padc;
            *(uint4 *)(sW + row * a.kp + (a.kchunks + i - row * padc) * 16) = make_uint4(0, 0, 0, 0);
        }
    } else {
        // general order (row walk for small C): one 4-byte LDS word per item
        const int nit = MT * ncol;
        constexpr int U = 4;
        for (int b0 = tid; b0 < nit; b0 += 256 * U) {
            uint32_t v[U];
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int idx = b0 + u * 256;
                const int row = (int)fdiv((uint32_t)idx, a.div_ncol);
                const int col = idx - row * ncol;
                const int j = col >> 2, d = col & 3;
                const int mg = m0 + row;
                v[u] = 0;
                if (idx < nit && mg < a.m && 4 * d < sVld[j]) {
                    const uint8_t *wr = a.w + (size_t)mg * a.wrow;
                    const int e = sNat[j] + 4 * d;
                    if (BITS == 8) {
                        v[u] = *(const uint32_t *)(wr + e);
                    } else if (BITS == 4) {
                        // bytes e..e+3 of the K order are one half of packed word e / 8
                        const uint2 h = w4_word(*(const uint32_t *)(wr + ((e >> 3) << 2)));
                        v[u] = (e & 4) ? h.y : h.x;
                    } else {
                        // bytes e..e+3 are field (e / 4) % 4 of packed word e / 16
                        const uint4 f = w2_word(*(const uint32_t *)(wr + ((e >> 4) << 2)));
                        const int k = (e >> 2) & 3;
                        v[u] = k == 0 ? f.x : (k == 1 ? f.y : (k == 2 ? f.z : f.w));
                    }
                }
            }
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int idx = b0 + u * 256;
                if (idx < nit) {
                    const int row = (int)fdiv((uint32_t)idx, a.div_ncol);
                    const int col = idx - row * ncol;
                    *(uint32_t *)(sW + row * a.kp + col * 4) = v[u];
                }
            }
        }
    }
    // input tile of the first pixel tile: first batch, then the rest
    if (tile < a.ntiles) {
        if (a.quad16) {
            halo_store<BITS, true, UH>(sX, hq, hd);
            halo_stage_from<BITS, true, UH>(a, sX, tid + 256 * UH, T.n0, T.iy0, T.ix0);
        } else {
            halo_store<BITS, false, UH>(sX, hq, hd);
            halo_stage_from<BITS, false, UH>(a, sX, tid + 256 * UH, T.n0, T.iy0, T.ix0);
        }
    }
    __syncthreads();

    // filter sums for the unsigned 8-bit fold, then the requantization plans
    if (BITS == 8) {
        for (int row = wv; row < MT; row += 4) {
            int s = 0;
            for (int col = lane; col < ncol; col += 64) {
                uint32_t v = *(const uint32_t *)(sW + row * a.kp + col * 4);
                s += (int)(int8_t)v + (int)(int8_t)(v >> 8) + (int)(int8_t)(v >> 16) +
                     (int)(int8_t)(v >> 24);
            }
            s = wave_sum(s);
            if (lane == 0)
                sWsum[row] = s;
        }
        __syncthreads();
    }
    constexpr int SL = BITS == 4 ? 4 : (BITS == 2 ? 6 : 0);  // log2 of the weight scale
    constexpr int NT = BITS == 8 ? 1 : (1 << BITS) - 1;       // staircase thresholds per channel
    int mode = 0;
    if (has_ch && a.epi == EPI_STAIR) {
        const bool live = m0 + pch < a.m;
        stair_thresholds(live ? a.thresh + (size_t)(m0 + pch) * NT : nullptr, NT, p_bias, SL,
                         (int32_t *)(sEpi + 4 * pch));
        mode = 5;
    } else if (has_ch) {
        int4 e0, e1;
        if (m0 + pch < a.m) {
            int64_t b = p_bias;
            if (BITS == 8)
                b += 128 * (int64_t)sWsum[pch];
            p_shift = p_shift < 0 ? 0 : (p_shift > 62 ? 62 : p_shift);
            requant_plan(b, p_mult, p_shift, a.clip_lo, a.clip_hi, a.epi == EPI_REQUANT, SL, e0, e1);
        } else {
            // missing channel: a strict plan that yields code 0 (and RAW32 skips it)
            e0 = make_int4(0, 0, 0, 0);
            e1 = make_int4(0, 0, 3, 0);
        }
        sEpi[4 * pch] = e0;
        sEpi[4 * pch + 1] = e1;
        mode = e1.z;
    }
    // workgroup-uniform epilogue selection: per-wave votes in LDS, then the
    // barrier that also publishes sEpi
    {
        const bool v3 = __all(!has_ch || mode == 3);
        const bool v4 = __all(!has_ch || mode == 3 || mode == 4);
        const bool v32 = __all(!has_ch || mode == 1);
        const bool v64 = __all(!has_ch || mode == 1 || mode == 2);
        if (lane == 0)
            sWsum[MT + wv] = (v32 ? 1 : 0) | (v64 ? 2 : 0) | (v3 ? 4 : 0) | (v4 ? 8 : 0);
    }
    __syncthreads();
    const int votes = sWsum[MT] & sWsum[MT + 1] & sWsum[MT + 2] & sWsum[MT + 3];
    const bool all3 = (votes & 4) != 0;
    const bool all4 = (votes & 8) != 0 && !all3;
    const bool all32 = (votes & 1) != 0 && !all3;
    const bool all64 = (votes & 2) != 0 && !all3;
    const bool full = m0 + MT <= a.m;

    const int tile_px = a.ti * a.th * a.tw;
    const int g = lane >> 4, r16 = lane & 15;

    for (bool first = true; tile < a.ntiles; tile += gridDim.x, first = false) {
        if (!first) {
            T = tile_xy(a, tile);
            if (a.quad16)
                halo_stage_from<BITS, true, UH>(a, sX, tid, T.n0, T.iy0, T.ix0);
            else
                halo_stage_from<BITS, false, UH>(a, sX, tid, T.n0, T.iy0, T.ix0);
            __syncthreads();
        }

        // ---- main loop: MR x NC MFMA tiles per 64-deep K step ----
        int base[NC];
#pragma unroll
        for (int c = 0; c < NC; ++c) {
            const int p = wv * 16 * NC + c * 16 + r16;
            base[c] = 0;
            if (p < tile_px) {
                const int tI = (int)fdiv((uint32_t)p, a.div_tile_px);
                const int rem = p - tI * a.th * a.tw;
                const int py = (int)fdiv((uint32_t)rem, a.div_tw);
                const int px = rem - py * a.tw;
                base[c] = ((tI * a.hh + py * a.sh) * a.hwd + px * a.sw) * a.ps;
            }
        }
        v4i acc[MR][NC];
#pragma unroll
        for (int t = 0; t < MR; ++t)
#pragma unroll
            for (int c = 0; c < NC; ++c)
                acc[t][c] = (v4i){0, 0, 0, 0};
        const int8_t *aRow = sW + r16 * a.kp + g * 16;
        // software pipeline: fragments of K step ks + 1 are read while the
        // MFMAs of step ks run
        v4i av[MR], bv[NC];
        auto load_frags = [&](int ks, v4i *A, v4i *B) {
            const int off = sTab[ks * 4 + g];
#pragma unroll
            for (int t = 0; t < MR; ++t)
                A[t] = *(const v4i *)(aRow + t * 16 * a.kp + ks * 64);
#pragma unroll
            for (int c = 0; c < NC; ++c) {
                const uint8_t *bp = sX + base[c] + off;
                if (AL16) {
                    B[c] = *(const v4i *)bp;
                } else {
                    const int32_t *b4 = (const int32_t *)bp;
                    B[c] = (v4i){b4[0], b4[1], b4[2], b4[3]};
                }
            }
        };
        load_frags(0, av, bv);
        for (int ks = 0; ks < a.ksteps; ++ks) {
            v4i an[MR], bn[NC];
            if (ks + 1 < a.ksteps)
                load_frags(ks + 1, an, bn);
#pragma unroll
            for (int t = 0; t < MR; ++t)
#pragma unroll
                for (int c = 0; c < NC; ++c)
                    acc[t][c] = __builtin_amdgcn_mfma_i32_16x16x64_i8(av[t], bv[c], acc[t][c], 0, 0, 0);
#pragma unroll
            for (int t = 0; t < MR; ++t)
                av[t] = an[t];
#pragma unroll
            for (int c = 0; c < NC; ++c)
                bv[c] = bn[c];
        }

        // the plan reads below do not depend on the tile; an opaque zero keeps
        // the compiler from hoisting all of them out of the tile loop (which
        // would hold every channel's plan in registers)
        int ez = 0;
        __asm__ volatile("" : "+v"(ez));
        const int4 *ep = sEpi + ez;
        // ---- epilogue: lane (r16, g) of tile (t, c) holds channels
        // t*16 + 4g + {0..3} of pixel c*16 + r16 of its wave ----
        int gpix[NC];
#pragma unroll
        for (int c = 0; c < NC; ++c) {
            const int p = wv * 16 * NC + c * 16 + r16;
            gpix[c] = -1;
            if (p < tile_px) {
                const int tI = (int)fdiv((uint32_t)p, a.div_tile_px);
                const int rem = p - tI * a.th * a.tw;
                const int py = (int)fdiv((uint32_t)rem, a.div_tw);
                const int px = rem - py * a.tw;
                const int nn = T.n0 + tI, oy = T.oy0 + py, ox = T.ox0 + px;
                if (nn < a.n && oy < a.ho && ox < a.wo)
                    gpix[c] = (nn * a.ho + oy) * a.wo + ox;
            }
        }
        if (a.epi == EPI_RAW32) {
#pragma unroll
            for (int t = 0; t < MR; ++t)
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const int mrow = t * 16 + 4 * g + i + ez;
                    if (m0 + mrow >= a.m)
                        continue;
                    const int4 e0 = ep[4 * mrow];
                    const int64_t bt = (int64_t)(((uint64_t)(uint32_t)e0.y << 32) | (uint32_t)e0.x);
#pragma unroll
                    for (int c = 0; c < NC; ++c) {
                        int32_t acc32 = acc[t][c][i];
                        if (BITS == 4)
                            acc32 >>= 4;
                        else if (BITS == 2)
                            acc32 >>= 6;
                        if (gpix[c] >= 0)
                            ((int32_t *)a.y)[(size_t)gpix[c] * a.m + m0 + mrow] =
                                (int32_t)(uint32_t)(uint64_t)(acc32 + bt);
                    }
                }
        } else {
            uint32_t packed[MR][NC];
#pragma unroll
            for (int t = 0; t < MR; ++t)
#pragma unroll
                for (int c = 0; c < NC; ++c)
                    packed[t][c] = 0;
            if (BITS != 8 && a.epi == EPI_STAIR) {
                // staircase (Eq. (4)): count the channel's thresholds at or below acc'
#pragma unroll
                for (int t = 0; t < MR; ++t)
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        const int4 *tp = ep + 4 * (t * 16 + 4 * g + i + ez);
                        int32_t T[16];
#pragma unroll
                        for (int k = 0; k < 4; ++k) {
                            const int4 q4 = tp[k];
                            T[4 * k] = q4.x;
                            T[4 * k + 1] = q4.y;
                            T[4 * k + 2] = q4.z;
                            T[4 * k + 3] = q4.w;
                        }
#pragma unroll
                        for (int c = 0; c < NC; ++c)
                            packed[t][c] |= stair_level<NT>((int32_t)acc[t][c][i], T) << (i * BITS);
                    }
            } else if (all3 || all4) {
                // strict plan: code = (clamp(acc' - A, 0, DS) * mult + RS) >> shift'
#pragma unroll
                for (int t = 0; t < MR; ++t) {
                    int4 e0[4], e1[4];
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        e0[i] = ep[4 * (t * 16 + 4 * g + i + ez)];
                        e1[i] = ep[4 * (t * 16 + 4 * g + i + ez) + 1];
                    }
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
#pragma unroll
                        for (int c = 0; c < NC; ++c) {
                            const int32_t d = __builtin_elementwise_sub_sat((int32_t)acc[t][c][i], e0[i].x);
                            const uint32_t dc = (uint32_t)min(max(d, 0), e0[i].y);
                            uint32_t code;
                            if (all3) {
                                code = (__umul24(dc, (uint32_t)e0[i].z) + (uint32_t)e0[i].w) >> e1[i].x;
                            } else {
                                const uint64_t rs = ((uint64_t)(uint32_t)e1[i].y << 32) | (uint32_t)e0[i].w;
                                code = (uint32_t)(((uint64_t)dc * (uint32_t)e0[i].z + rs) >> e1[i].x);
                            }
                            packed[t][c] |= code << (i * BITS);
                        }
                    }
                    __builtin_amdgcn_sched_barrier(0);
                }
            } else if (all32 || all64) {
                // plan form: code = clip(Q + ((clamp(acc - a_base, 0, D) * mult + R) >> shift))
#pragma unroll
                for (int t = 0; t < MR; ++t) {
                    int4 e0[4], e1[4];
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        e0[i] = ep[4 * (t * 16 + 4 * g + i + ez)];
                        e1[i] = ep[4 * (t * 16 + 4 * g + i + ez) + 1];
                    }
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        const bool live = full || (m0 + t * 16 + 4 * g + i + ez < a.m);
#pragma unroll
                        for (int c = 0; c < NC; ++c) {
                            int32_t acc32 = acc[t][c][i];
                            if (BITS == 4)
                                acc32 >>= 4;
                            else if (BITS == 2)
                                acc32 >>= 6;
                            const int32_t d = __builtin_elementwise_sub_sat(acc32, e0[i].x);
                            const uint32_t dc = (uint32_t)min(max(d, 0), e0[i].y);
                            uint32_t q;
                            if (all32) {
                                q = (__umul24(dc, (uint32_t)e0[i].z) + (uint32_t)e0[i].w) >> e1[i].y;
                            } else {
                                const uint64_t tt = (uint64_t)dc * (uint32_t)e0[i].z + (uint32_t)e0[i].w;
                                q = (uint32_t)(tt >> e1[i].y);
                            }
                            int32_t code = min(max(e1[i].x + (int32_t)q, a.clip_lo), a.clip_hi);
                            if (!live)
                                code = 0;
                            packed[t][c] |= (uint32_t)code << (i * BITS);
                        }
                    }
                    __builtin_amdgcn_sched_barrier(0);
                }
            } else {
                // general form, channel by channel
#pragma unroll
                for (int t = 0; t < MR; ++t)
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        const int mrow = t * 16 + 4 * g + i + ez;
                        if (m0 + mrow >= a.m)
                            continue;
                        const int4 e0 = ep[4 * mrow];
                        const int4 e1 = ep[4 * mrow + 1];
#pragma unroll
                        for (int c = 0; c < NC; ++c) {
                            if (e1.z >= 3) {
                                const int32_t d = __builtin_elementwise_sub_sat((int32_t)acc[t][c][i], e0.x);
                                const uint32_t dc = (uint32_t)min(max(d, 0), e0.y);
                                const uint64_t rs = ((uint64_t)(uint32_t)e1.y << 32) | (uint32_t)e0.w;
                                packed[t][c] |= (uint32_t)(((uint64_t)dc * (uint32_t)e0.z + rs) >> e1.x) << (i * BITS);
                                continue;
                            }
                            int32_t acc32 = acc[t][c][i];
                            if (BITS == 4)
                                acc32 >>= 4;
                            else if (BITS == 2)
                                acc32 >>= 6;
                            int64_t r;
                            if (e1.z) {
                                const int32_t d = __builtin_elementwise_sub_sat(acc32, e0.x);
                                const uint32_t dc = (uint32_t)min(max(d, 0), e0.y);
                                const uint64_t tt = (uint64_t)dc * (uint32_t)e0.z + (uint32_t)e0.w;
                                r = (int64_t)e1.x + (int64_t)(tt >> e1.y);
                            } else {
                                const int64_t v = (int64_t)acc32 +
                                    (int64_t)(((uint64_t)(uint32_t)e0.y << 32) | (uint32_t)e0.x);
                                r = round_shift(v * (int64_t)e0.z, e0.w);
                            }
                            r = r < a.clip_lo ? a.clip_lo : (r > a.clip_hi ? a.clip_hi : r);
                            packed[t][c] |= (uint32_t)r << (i * BITS);
                        }
                    }
            }
#pragma unroll
            for (int t = 0; t < MR; ++t)
#pragma unroll
                for (int c = 0; c < NC; ++c) {
                    const int p = wv * 16 * NC + c * 16 + r16;
                    if (p < tile_px) {
                        uint8_t *o = sOut + p * a.ot_b + (t * 16 + 4 * g) * BITS / 8;
                        if (BITS == 8)
                            *(uint32_t *)o = packed[t][c];
                        else if (BITS == 4)
                            *(uint16_t *)o = (uint16_t)packed[t][c];
                        else
                            *o = (uint8_t)packed[t][c];
                    }
                }
        }
        __syncthreads();

        // ---- coalesced copy of the packed output tile ----
        if (a.epi != EPI_RAW32 && a.contig) {
            // the tile's valid pixels are consecutive output pixels and the tile
            // holds every channel: one flat copy
            const int valid = a.ti == 1 ? min(a.th, a.ho - T.oy0) * a.wo
                                        : min(a.ti, a.n - T.n0) * a.ho * a.wo;
            const size_t first = a.ti == 1 ? ((size_t)T.n0 * a.ho + T.oy0) * a.wo : (size_t)T.n0 * a.ho * a.wo;
            uint8_t *dst = a.y + first * a.ypb;
            const int nbytes = valid * a.ypb;
            if ((a.ypb & 15) == 0) {
                for (int o = tid * 16; o < nbytes; o += 256 * 16)
                    *(uint4 *)(dst + o) = *(const uint4 *)(sOut + o);
            } else {
                for (int o = tid * 4; o < nbytes; o += 256 * 4)
                    *(uint32_t *)(dst + o) = *(const uint32_t *)(sOut + o);
            }
        } else if (a.epi != EPI_RAW32) {
            const int ob0 = m0 * BITS / 8;
            const int obn = min(a.ot_b, a.ypb - ob0);
            const int tq4 = tile_px * a.obq;
            for (int idx = tid; idx < tq4; idx += 256) {
                const int p = (int)fdiv((uint32_t)idx, a.div_obq);
                const int q = idx - p * a.obq;
                const int tI = (int)fdiv((uint32_t)p, a.div_tile_px);
                const int rem = p - tI * a.th * a.tw;
                const int py = (int)fdiv((uint32_t)rem, a.div_tw);
                const int px = rem - py * a.tw;
                const int nn = T.n0 + tI, oy = T.oy0 + py, ox = T.ox0 + px;
                if (nn >= a.n || oy >= a.ho || ox >= a.wo)
                    continue;
                const size_t gp = (size_t)(nn * a.ho + oy) * a.wo + ox;
                if (a.oquad16) {
                    if (4 * q < obn)
                        *(uint32_t *)(a.y + gp * a.ypb + ob0 + 4 * q) =
                            *(const uint32_t *)(sOut + p * a.ot_b + 4 * q);
                } else {
                    if (q < obn)
                        a.y[gp * a.ypb + ob0 + q] = sOut[p * a.ot_b + q];
                }
            }
        }
        // the next tile's input staging overwrites sX / sOut only after every
        // wave passed the barrier above; its own barrier follows the staging
    }
}

template <int BITS>
hipError_t launch_conv_mfma_bits(const ConvArgs &a, int mr, int nc, int al16, dim3 grid,
                                 hipStream_t s)
{
#define QNN_CASE(MR_, NC_, AL_)                                                                 \
    if (mr == MR_ && nc == NC_ && al16 == AL_) {                                                \
        static bool attr_set = false;                                                           \
        auto *k = conv_mfma_kernel<BITS, MR_, NC_, (AL_ != 0)>;                                 \
        if (!attr_set) {                                                                        \
            if (hipFuncSetAttribute((const void *)k, hipFuncAttributeMaxDynamicSharedMemorySize,  \
                                    a.lds_bytes > 64 * 1024 ? 160 * 1024 : 64 * 1024) != hipSuccess) \
                (void)hipGetLastError();                                                        \
            attr_set = true;                                                                    \
        }                                                                                       \
        hipLaunchKernelGGL(k, grid, dim3(256), a.lds_bytes, s, a);                              \
        return hipGetLastError();                                                               \
    }
    QNN_CASE(1, 1, 0) QNN_CASE(1, 2, 0) QNN_CASE(1, 4, 0)
    QNN_CASE(2, 1, 0) QNN_CASE(2, 2, 0) QNN_CASE(2, 4, 0)
    QNN_CASE(4, 1, 0) QNN_CASE(4, 2, 0) QNN_CASE(4, 4, 0)
    QNN_CASE(1, 1, 1) QNN_CASE(1, 2, 1) QNN_CASE(1, 4, 1)
    QNN_CASE(2, 1, 1) QNN_CASE(2, 2, 1) QNN_CASE(2, 4, 1)
    QNN_CASE(4, 1, 1) QNN_CASE(4, 2, 1) QNN_CASE(4, 4, 1)
#undef QNN_CASE
    return hipErrorInvalidValue;
}

}  // namespace qnn
