// Implicit-GEMM quantized convolution on v_mfma_i32_32x32x32_i8.
//
// Same computation as conv_mfma_kernel (Sec. III-A Eq. (2), Sec. III-B
// Eq. (6), scale-and-clamp compression of Sec. III-A), for layers wide enough
// to fill 32-row matrix tiles.  Differences:
//   * each wave computes 32*WM output channels x 32*WN output pixels with
//     32x32x32 MFMAs (the larger instruction sustains a higher fraction of
//     the matrix-core peak);
//   * the filter tile stays PACKED in LDS (4 / 2 bits per weight), copied from
//     memory without any unpacking, and each A fragment is expanded to int8 in
//     registers just before use (3 / 7 mask-and-shift ops per fragment), which
//     halves / quarters both the LDS footprint and the LDS traffic of the
//     A operand; the input tile is still unpacked once per tile.
// The sub-byte K order (field-major within each packed word) is the one of
// conv_mfma_impl.h, for weights and activations alike.
#pragma once

#include "conv_mfma_impl.h"

namespace qnn {

typedef int32_t v16i __attribute__((ext_vector_type(16)));
typedef int32_t v8i __attribute__((ext_vector_type(8)));
typedef float v16f __attribute__((ext_vector_type(16)));

// Packed form of one A fragment (16 K bytes of one output channel) and its
// expansion to int8 (4-/2-bit codes scaled by 16 / 64).
template <int BITS> struct PackedA { typedef v4i type; };
template <> struct PackedA<4> { typedef uint2 type; };
template <> struct PackedA<2> { typedef uint32_t type; };

template <int BITS>
__device__ __forceinline__ v4i expand_a(v4i p) { return p; }

// FP4 mode (INT-2 layers on the e2m1 matrix instruction): filter fragments
// are staged as 16 bytes of e2m1 nibbles per lane (no expansion), and the
// accumulators are fp32 (exact: every partial sum is an integer below 2^24).
template <bool F4, int BITS> struct FragA { typedef typename PackedA<BITS>::type type; };
template <int BITS> struct FragA<true, BITS> { typedef v4i type; };
template <bool F4> struct AccTile { typedef v16i type; };
template <> struct AccTile<true> { typedef v16f type; };

// One 32x32x64 e2m1 MFMA: rows = A (16 bytes per lane, 32 codes), columns =
// B.  At 2 bits the exponent-2 scale on A restores the factor 1/4 of the
// x/2, w/2 encoding; 1-bit values (+1, -1) are encoded as they are (E8M0
// scale bytes: 127 + 2 or 127, and 127 on B).
template <int BITS>
__device__ __forceinline__ v16f mfma_f4(v4i a, v4i b, v16f c)
{
    const v8i a8 = {a.x, a.y, a.z, a.w, 0, 0, 0, 0};
    const v8i b8 = {b.x, b.y, b.z, b.w, 0, 0, 0, 0};
    return __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a8, b8, c, 4, 4, 0, BITS == 1 ? 127 : 129,
                                                           0, 127);
}

// 16 packed INT-2 / INT-1 weight bytes (64 / 128 codes) -> 32 / 64 bytes of
// e2m1 nibbles.
template <int BITS>
__device__ __forceinline__ void store_w16_f4(uint8_t *dst, uint4 v)
{
    if (BITS == 1) {
        *(uint4 *)dst = b1_word_f4(v.x);
        *(uint4 *)(dst + 16) = b1_word_f4(v.y);
        *(uint4 *)(dst + 32) = b1_word_f4(v.z);
        *(uint4 *)(dst + 48) = b1_word_f4(v.w);
    } else {
        const uint2 a = w2_word_f4(v.x), b = w2_word_f4(v.y), c = w2_word_f4(v.z), d = w2_word_f4(v.w);
        *(uint4 *)dst = make_uint4(a.x, a.y, b.x, b.y);
        *(uint4 *)(dst + 16) = make_uint4(c.x, c.y, d.x, d.y);
    }
}

// One packed 4-byte weight word in FP4 mode: 8 (INT-2) or 16 (INT-1) bytes.
template <int BITS>
__device__ __forceinline__ void store_w4_f4(uint8_t *dst, uint32_t v)
{
    if (BITS == 1)
        *(uint4 *)dst = b1_word_f4(v);
    else
        *(uint2 *)dst = w2_word_f4(v);
}

template <int BITS>
__device__ __forceinline__ v4i expand_a(uint2 d)
{
    const uint2 x = w4_word(d.x), y = w4_word(d.y);
    return (v4i){(int32_t)x.x, (int32_t)x.y, (int32_t)y.x, (int32_t)y.y};
}

template <int BITS>
__device__ __forceinline__ v4i expand_a(uint32_t d)
{
    const uint4 f = w2_word(d);
    return (v4i){(int32_t)f.x, (int32_t)f.y, (int32_t)f.z, (int32_t)f.w};
}

// Store 16 packed bytes at an LDS address aligned to 16 (8 bits), 8 (4 bits) or
// 4 (2 bits) bytes: the packed row stride is an odd multiple of one A
// fragment's packed size, which keeps fragment reads free of bank conflicts.
template <int BITS>
__device__ __forceinline__ void store_packed16(uint8_t *dst, uint4 v)
{
    if (BITS == 8) {
        *(uint4 *)dst = v;
    } else if (BITS == 4) {
        *(uint2 *)dst = make_uint2(v.x, v.y);
        *(uint2 *)(dst + 8) = make_uint2(v.z, v.w);
    } else {
        *(uint32_t *)dst = v.x;
        *(uint32_t *)(dst + 4) = v.y;
        *(uint32_t *)(dst + 8) = v.z;
        *(uint32_t *)(dst + 12) = v.w;
    }
}

// Packs 32/BITS one-byte codes (LDS address aligned to 4 / 8 / 16 bytes) into
// one 32-bit word of the packed layout: lowest channel in the lowest bits.
template <int BITS>
__device__ __forceinline__ uint32_t pack_codes_word(const uint8_t *src)
{
    if (BITS == 8) {
        return *(const uint32_t *)src;
    } else if (BITS == 4) {
        // bytes 0 and 2 of v | v >> 4 hold channel pairs (2j, 2j+1)
        const uint2 v = *(const uint2 *)src;
        const uint32_t x = v.x | (v.x >> 4), y = v.y | (v.y >> 4);
        return __builtin_amdgcn_perm(y, x, 0x06040200u);
    } else if (BITS == 1) {
        // 32 bytes of 0 / 1: per word, bits 0..3 of t | t >> 14 (t = v | v >> 7)
        // are its 4 codes
        const uint4 a = *(const uint4 *)src, b = *(const uint4 *)(src + 16);
        const uint32_t w[8] = {a.x, a.y, a.z, a.w, b.x, b.y, b.z, b.w};
        uint32_t r = 0;
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const uint32_t t = w[i] | (w[i] >> 7);
            r |= ((t | (t >> 14)) & 15u) << (4 * i);
        }
        return r;
    } else {
        // byte 0 of u = v | v >> 6, then u | u >> 12, holds channels 0..3
        const uint4 v = *(const uint4 *)src;
        uint32_t u0 = v.x | (v.x >> 6), u1 = v.y | (v.y >> 6);
        uint32_t u2 = v.z | (v.z >> 6), u3 = v.w | (v.w >> 6);
        u0 |= u0 >> 12;
        u1 |= u1 >> 12;
        u2 |= u2 >> 12;
        u3 |= u3 >> 12;
        const uint32_t lo = __builtin_amdgcn_perm(u1, u0, 0x0c0c0400u);
        const uint32_t hi = __builtin_amdgcn_perm(u3, u2, 0x0c0c0400u);
        return __builtin_amdgcn_perm(hi, lo, 0x05040100u);
    }
}

// Byte-wise maximum of two words of one-byte codes (two 16-bit maxima on
// the even and the odd bytes).
__device__ __forceinline__ uint32_t max_bytes(uint32_t a, uint32_t b)
{
    typedef unsigned short u16x2 __attribute__((ext_vector_type(2)));
    const u16x2 lo = __builtin_elementwise_max(__builtin_bit_cast(u16x2, a & 0x00FF00FFu),
                                               __builtin_bit_cast(u16x2, b & 0x00FF00FFu));
    const u16x2 hi = __builtin_elementwise_max(__builtin_bit_cast(u16x2, (a >> 8) & 0x00FF00FFu),
                                               __builtin_bit_cast(u16x2, (b >> 8) & 0x00FF00FFu));
    return __builtin_bit_cast(uint32_t, lo) | (__builtin_bit_cast(uint32_t, hi) << 8);
}

// Code bytes of a 2x2 window: the byte-wise maximum of the four pixels'
// runs of 32/BITS codes (4 / 8 / 16 bytes), written to out.
template <int BITS>
__device__ __forceinline__ void max4_codes(const uint8_t *p00, const uint8_t *p01, const uint8_t *p10,
                                           const uint8_t *p11, uint8_t *out)
{
    constexpr int NW = 8 / BITS;  // 32-bit words of codes
#pragma unroll
    for (int i = 0; i < NW; ++i) {
        const uint32_t a = *(const uint32_t *)(p00 + 4 * i), b = *(const uint32_t *)(p01 + 4 * i);
        const uint32_t c = *(const uint32_t *)(p10 + 4 * i), d = *(const uint32_t *)(p11 + 4 * i);
        *(uint32_t *)(out + 4 * i) = max_bytes(max_bytes(a, b), max_bytes(c, d));
    }
}

// One output byte from 8/BITS one-byte codes.
template <int BITS>
__device__ __forceinline__ uint8_t pack_codes_byte(const uint8_t *src)
{
    uint32_t b = 0;
#pragma unroll
    for (int i = 0; i < 8 / BITS; ++i)
        b |= (uint32_t)src[i] << (i * BITS);
    return (uint8_t)b;
}

// EXT: the staircase epilogue, the fused pooling and the next-tile input
// prefetch are compiled in; the plain instances (scale-and-clamp and raw
// layers with one tile per workgroup) carry none of them.
// UA: 4- / 2-bit filters staged in LDS already unpacked to int8 (16*w /
// 64*w), so the main loop reads 16-byte filter fragments and spends no
// vector instructions expanding them (instantiated for 4-bit layers walked
// tap by tap).
template <int BITS, int WM, int WN, bool AL16, bool EXT, int NW, bool F4 = false, bool UA = false>
__global__ void __launch_bounds__(64 * NW, 8 / NW) conv_m32_kernel(ConvArgs a)
{
    extern __shared__ __align__(16) uint8_t smem[];
    constexpr int NT = 64 * NW;   // threads: NW waves of 32*WN pixels each
    constexpr int MT = 32 * WM;
    // LDS bytes of one K chunk of a filter row: packed codes (16 K values),
    // or 16 bytes of e2m1 nibbles (32 K values) in FP4 mode
    constexpr int CB = (F4 || UA) ? 16 : 2 * BITS;
    // staged bytes per packed byte: 2 / 4 at 2 / 1 bits in FP4 mode, 8/BITS
    // for unpacked filters
    constexpr int XR = F4 ? 4 / BITS : (UA ? 8 / BITS : 1);
    // threshold epilogues (the staircase, and the binary threshold as a
    // one-step staircase) are compiled into the extended instances and into
    // every 1-bit one
    constexpr bool THR = EXT || BITS == 1;
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wv = tid >> 6;
    const int m0 = blockIdx.y * MT;
    const int kch = a.kch;

    uint8_t *sW = smem;                                          // [MT][kp] packed, chunk order
    int32_t *sTab = (int32_t *)(smem + a.off_tab);
    int32_t *sNat = sTab + kch;
    int32_t *sVld = sNat + kch;
    int32_t *sWsum = (int32_t *)(smem + a.off_wsum);            // [MT] filter sums, [8] votes
    int4 *sEpi = (int4 *)(smem + a.off_wsum + 4 * MT + 32);      // [MT][4]: plan (2) or 16 thresholds
    uint8_t *sX = smem + a.off_x;
    uint8_t *sC = smem + a.off_out;                              // [pixel][cs] one byte per code

    // ---- prologue: every independent load is issued before any is used ----
    // the input tile first: its loads are the longest chain of the prologue
    int tile = blockIdx.x;
    TileXY T = tile_xy(a, tile < a.ntiles ? tile : 0);
    constexpr int UH = 4;
    uint4 hq[UH];
    int hd[UH];
    const int totq = a.ti * a.hh * a.hwd * a.pbq;
    if (a.quad16)
        halo_issue<BITS, true, UH, NT, F4>(a, tid, tile < a.ntiles ? totq : 0, T.n0, T.iy0, T.ix0, hq, hd);
    else
        halo_issue<BITS, false, UH, NT, F4>(a, tid, tile < a.ntiles ? totq : 0, T.n0, T.iy0, T.ix0, hq, hd);
    // filter tile: packed rows m0 .. m0+MT-1 are one contiguous run and, when
    // the K walk is tap by tap, already in chunk order: a plain copy
    const bool wfast = !a.row_mode && (a.wrow & 15) == 0;
    const int qrow = a.wrow >> 4;
    const int nq = MT * qrow;
    // quads of the rows that exist (rows past the last channel stay zero)
    const int nqv = min(MT, a.m - m0) * qrow;
    const uint4 *wsrc = (const uint4 *)(a.w + (size_t)m0 * a.wrow);
    constexpr int UW = NW == 8 ? 3 : 6;
    uint4 wq[UW];
    if (wfast) {
#pragma unroll
        for (int u = 0; u < UW; ++u) {
            const int idx = tid + u * NT;
            wq[u] = make_uint4(0, 0, 0, 0);
            if (idx < nqv)
                wq[u] = wsrc[idx];
        }
    }
    // per-channel parameters and plans: computed by (at most) four waves,
    // one per SIMD, so an eight-wave workgroup pays for them once per SIMD
    constexpr int PW = NW < 4 ? NW : 4;
    const int pch = wv + PW * lane;
    const bool has_ch = wv < PW && lane < MT / PW;
    int32_t p_bias = 0, p_mult = 0, p_shift = 0;
    if (has_ch && m0 + pch < a.m) {
        if (a.bias)
            p_bias = a.bias[m0 + pch];
        if (a.epi == EPI_REQUANT) {
            p_mult = a.mult[m0 + pch];
            p_shift = a.shift[m0 + pch];
        }
    }

    // requantization plans (sub-byte layers: they need no filter sums, so they
    // are computed while the loads above are in flight) and the votes that
    // select a workgroup-uniform epilogue
    // log2 of the weight scale the accumulator carries (16 / 64 for packed
    // 4- / 2-bit fragments; none in FP4 mode, whose block scale removes it)
    constexpr int SL = F4 ? 0 : (BITS == 4 ? 4 : (BITS == 2 ? 6 : 0));
    constexpr int NTH = BITS == 8 ? 1 : (1 << BITS) - 1;  // staircase thresholds per channel
    auto make_plans = [&](const int32_t *wsum) {
        int mode = 0;
        if (THR && has_ch && (a.epi == EPI_STAIR || a.epi == EPI_THRESH1)) {
            const bool live = m0 + pch < a.m;
            stair_thresholds(live ? a.thresh + (size_t)(m0 + pch) * NTH : nullptr, NTH, p_bias, SL,
                             (int32_t *)(sEpi + 4 * pch));
            mode = 5;
        } else if (has_ch) {
            int4 e0, e1;
            if (m0 + pch < a.m) {
                int64_t b = p_bias;
                if (BITS == 8)
                    b += 128 * (int64_t)wsum[pch];
                const int sh = p_shift < 0 ? 0 : (p_shift > 62 ? 62 : p_shift);
                requant_plan(b, p_mult, sh, a.clip_lo, a.clip_hi, a.epi == EPI_REQUANT, SL, e0, e1);
            } else {
                e0 = make_int4(0, 0, 0, 0);
                e1 = make_int4(0, 0, 3, 0);
            }
            sEpi[4 * pch] = e0;
            sEpi[4 * pch + 1] = e1;
            mode = e1.z;
        }
        const bool v3 = __all(!has_ch || mode == 3);
        const bool v4 = __all(!has_ch || mode == 3 || mode == 4);
        if (lane == 0)
            sWsum[MT + wv] = (v3 ? 4 : 0) | (v4 ? 8 : 0);
    };
    if (BITS != 8)
        make_plans(nullptr);

    // K-chunk tables: chunk j of the reduction starts at byte hoff of a
    // pixel's window in the input tile (sTab, in main-loop order) and at
    // unpacked byte sNat[j] of a filter row; sVld[j] bytes of it are real
    // (the rest pads K)
    for (int j = tid; j < kch; j += NT) {
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
        // pair-major order for the main loop: step pair, lane half, step
        sTab[((j >> 2) * 2 + (j & 1)) * 2 + ((j >> 1) & 1)] = hoff;
        sNat[j] = nat;
        sVld[j] = vld;
    }
    __syncthreads();

    if (wfast) {
#pragma unroll
        for (int u = 0; u < UW; ++u) {
            const int idx = tid + u * NT;
            if (idx < nq) {
                const int row = (int)fdiv((uint32_t)idx, a.div_qrow);
                if (F4)
                    store_w16_f4<BITS>(sW + row * a.kp + (idx - row * qrow) * 16 * XR, wq[u]);
                else
                    if (UA)
                        stage_w16<BITS>((int8_t *)(sW + row * a.kp + (idx - row * qrow) * 16 * XR), wq[u]);
                    else
                        store_packed16<BITS>(sW + row * a.kp + (idx - row * qrow) * 16, wq[u]);
            }
        }
        for (int b0 = tid + NT * UW; b0 < nq; b0 += NT * UW) {
#pragma unroll
            for (int u = 0; u < UW; ++u) {
                const int idx = b0 + u * NT;
                wq[u] = make_uint4(0, 0, 0, 0);
                if (idx < nqv)
                    wq[u] = wsrc[idx];
            }
#pragma unroll
            for (int u = 0; u < UW; ++u) {
                const int idx = b0 + u * NT;
                if (idx < nq) {
                    const int row = (int)fdiv((uint32_t)idx, a.div_qrow);
                    if (F4)
                        store_w16_f4<BITS>(sW + row * a.kp + (idx - row * qrow) * 16 * XR, wq[u]);
                    else
                        if (UA)
                            stage_w16<BITS>((int8_t *)(sW + row * a.kp + (idx - row * qrow) * 16 * XR), wq[u]);
                        else
                            store_packed16<BITS>(sW + row * a.kp + (idx - row * qrow) * 16, wq[u]);
                }
            }
        }
        // zero the packed bytes of the chunks that round K up to whole steps
        const int padw = (kch - a.kchunks) * CB / 4;
        for (int i = tid; i < MT * padw; i += NT) {
            const int row = i / padw;
            *(uint32_t *)(sW + row * a.kp + a.kchunks * CB + 4 * (i - row * padw)) = 0u;
        }
    } else {
        // general order (row walk for small C): one packed 4-byte word per
        // item, staged as IB bytes (itself, or 8 / 16 bytes of e2m1 nibbles)
        constexpr int IB = 4 * XR;
        const int wpr = kch * CB / IB;  // items per staged row
        const int nit = MT * wpr;
        constexpr int U = 4;
        for (int b0 = tid; b0 < nit; b0 += NT * U) {
            uint32_t v[U];
            bool ok[U];
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int idx = b0 + u * NT;
                const int row = (int)fdiv((uint32_t)idx, a.div_ncol);
                const int col = idx - row * wpr;
                const int j = col / (CB / IB), d = col - j * (CB / IB);
                const int mg = m0 + row;
                // the chunk's packed offset in the filter row and its real bytes
                const int pnat = F4 ? sNat[j] / XR : sNat[j] * BITS / 8;
                const int pvld = F4 ? sVld[j] / XR : sVld[j] * BITS / 8;
                v[u] = 0;
                ok[u] = idx < nit && mg < a.m && 4 * d < pvld;
                if (ok[u])
                    v[u] = *(const uint32_t *)(a.w + (size_t)mg * a.wrow + pnat + 4 * d);
            }
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int idx = b0 + u * NT;
                if (idx < nit) {
                    const int row = (int)fdiv((uint32_t)idx, a.div_ncol);
                    uint8_t *dst = sW + row * a.kp + IB * (idx - row * wpr);
                    if (UA && BITS == 4)
                        *(uint2 *)dst = w4_word(v[u]);
                    else if (UA && BITS == 2)
                        *(uint4 *)dst = w2_word(v[u]);
                    else if (!F4)
                        *(uint32_t *)dst = v[u];
                    else if (ok[u])
                        store_w4_f4<BITS>(dst, v[u]);
                    else if (BITS == 1)
                        *(uint4 *)dst = make_uint4(0, 0, 0, 0);  // K padding: e2m1 zeros
                    else
                        *(uint2 *)dst = make_uint2(0, 0);
                }
            }
        }
    }
    if (tile < a.ntiles) {
        if (a.quad16) {
            halo_store<BITS, true, UH, F4>(sX, hq, hd);
            halo_stage_from<BITS, true, UH, NT, F4>(a, sX, tid + NT * UH, T.n0, T.iy0, T.ix0);
        } else {
            halo_store<BITS, false, UH, F4>(sX, hq, hd);
            halo_stage_from<BITS, false, UH, NT, F4>(a, sX, tid + NT * UH, T.n0, T.iy0, T.ix0);
        }
    }
    __syncthreads();

    // filter sums for the unsigned 8-bit fold, then the 8-bit plans
    if (BITS == 8) {
        const int wpr = kch * 4;
        for (int row = wv; row < MT; row += NW) {
            int s = 0;
            for (int col = lane; col < wpr; col += 64) {
                uint32_t v = *(const uint32_t *)(sW + row * a.kp + col * 4);
                s += (int)(int8_t)v + (int)(int8_t)(v >> 8) + (int)(int8_t)(v >> 16) +
                     (int)(int8_t)(v >> 24);
            }
            s = wave_sum(s);
            if (lane == 0)
                sWsum[row] = s;
        }
        __syncthreads();
        make_plans(sWsum);
        __syncthreads();
    }
    int votes = sWsum[MT];
#pragma unroll
    for (int w = 1; w < NW; ++w)
        votes &= sWsum[MT + w];
    const bool all3 = (votes & 4) != 0;

    const int tile_px = a.ti * a.th * a.tw;
    const int h = lane >> 5, r32 = lane & 31;
    // next-tile input prefetch (extended instances, which the host picks for
    // workgroups with more than one tile): for wave tiles of up to two 32x32
    // MFMA tiles (wider ones would spill the extra registers)
    constexpr bool PREF = EXT && WM * WN <= 2;
    // code-staging pixel stride (the planner sizes sC with the same value):
    // a compile-time stride turns every staging address into an immediate
    // offset
    constexpr int cs = MT + 16;

    for (bool first = true; tile < a.ntiles; tile += gridDim.x, first = false) {
        if (!first) {
            if (a.alias_out)
                __syncthreads();  // the previous tile's copy-out still reads sC = sX
            // with PREF the first batch of this tile's input arrived in
            // registers during the previous tile's epilogue; the rest is
            // staged now
            if (PREF) {
                if (a.quad16) {
                    halo_store<BITS, true, UH, F4>(sX, hq, hd);
                    halo_stage_from<BITS, true, UH, NT, F4>(a, sX, tid + NT * UH, T.n0, T.iy0, T.ix0);
                } else {
                    halo_store<BITS, false, UH, F4>(sX, hq, hd);
                    halo_stage_from<BITS, false, UH, NT, F4>(a, sX, tid + NT * UH, T.n0, T.iy0, T.ix0);
                }
            } else {
                T = tile_xy(a, tile);
                if (a.quad16)
                    halo_stage_from<BITS, true, UH, NT, F4>(a, sX, tid, T.n0, T.iy0, T.ix0);
                else
                    halo_stage_from<BITS, false, UH, NT, F4>(a, sX, tid, T.n0, T.iy0, T.ix0);
            }
            __syncthreads();
        }

        // ---- main loop: WN x WM 32x32 tiles per 32-deep K step.  The MFMA's
        // row operand is the im2col fragment (pixels) and its column operand
        // the filter fragment (channels), so each lane ends up holding one
        // output channel of 16 pixels per tile ----
        int base[WN];
#pragma unroll
        for (int c = 0; c < WN; ++c) {
            const int p = wv * 32 * WN + c * 32 + r32;
            base[c] = 0;
            if (p < tile_px) {
                const int tI = (int)fdiv((uint32_t)p, a.div_tile_px);
                const int rem = p - tI * a.th * a.tw;
                const int py = (int)fdiv((uint32_t)rem, a.div_tw);
                const int px = rem - py * a.tw;
                base[c] = ((tI * a.hh + py * a.sh) * a.hwd + px * a.sw) * a.ps;
            }
        }
        // accumulators: the first K step's MFMAs start from zero
        typedef typename AccTile<F4>::type ACC;
        ACC acc[WM][WN];
        const uint8_t *aRow = sW + r32 * a.kp + h * CB;
        // filter fragments are read in packed form (2 / 1 registers for 4 / 2
        // bits) and expanded right before their MFMAs; two register sets
        // alternate, so the reads of step k+1 are in flight during step k
        typedef typename FragA<F4 || UA, BITS>::type PA;
        auto load_frags = [&](int ks, int off, PA *A, v4i *B) {
#pragma unroll
            for (int t = 0; t < WM; ++t)
                A[t] = *(const PA *)(aRow + t * 32 * a.kp + ks * 2 * CB);
#pragma unroll
            for (int c = 0; c < WN; ++c) {
                const uint8_t *bp = sX + base[c] + off;
                if (AL16) {
                    B[c] = *(const v4i *)bp;
                } else {
                    const int32_t *b4 = (const int32_t *)bp;
                    B[c] = (v4i){b4[0], b4[1], b4[2], b4[3]};
                }
            }
        };
        auto mfma_step = [&](const PA *A, const v4i *B, bool zero) {
#pragma unroll
            for (int t = 0; t < WM; ++t) {
                const v4i av = expand_a<BITS>(A[t]);
#pragma unroll
                for (int c = 0; c < WN; ++c) {
                    const ACC cin = zero ? (ACC){} : acc[t][c];
                    if constexpr (F4)
                        acc[t][c] = mfma_f4<BITS>(B[c], av, cin);
                    else
                        acc[t][c] = __builtin_amdgcn_mfma_i32_32x32x32_i8(B[c], av, cin, 0, 0, 0);
                }
            }
        };
        // K steps come in pairs (the planner rounds them up to an even count);
        // the two register sets alternate, and the reads of a pair's steps are
        // issued one step before their MFMAs.  One 8-byte table read gives a
        // lane both offsets of a pair.  The scheduling barriers keep this
        // order (the counter that tracks local-memory reads completes them in
        // issue order, so a read issued early is never waited for late).
        PA a0[WM], a1[WM];
        v4i b0[WN], b1[WN];
        const int npairs = a.ksteps >> 1;
        const int2 *tab2 = (const int2 *)sTab + h;
        {
            const int2 o = tab2[0];
            __builtin_amdgcn_sched_barrier(0);
            load_frags(0, o.x, a0, b0);
            __builtin_amdgcn_sched_barrier(0);
            load_frags(1, o.y, a1, b1);
            __builtin_amdgcn_sched_barrier(0);
        }
        {
            // the first pair (there is always one), peeled: its first MFMAs
            // take a zero accumulator instead of zeroed registers
            const int pn = min(1, npairs - 1);
            const int2 o = tab2[2 * pn];
            __builtin_amdgcn_sched_barrier(0);
            mfma_step(a0, b0, true);
            __builtin_amdgcn_sched_barrier(0);
            load_frags(2 * pn, o.x, a0, b0);
            __builtin_amdgcn_sched_barrier(0);
            mfma_step(a1, b1, false);
            __builtin_amdgcn_sched_barrier(0);
            load_frags(2 * pn + 1, o.y, a1, b1);
            __builtin_amdgcn_sched_barrier(0);
        }
        for (int pr = 1; pr < npairs; ++pr) {
            const int pn = min(pr + 1, npairs - 1);
            const int2 o = tab2[2 * pn];
            __builtin_amdgcn_sched_barrier(0);
            mfma_step(a0, b0, false);
            __builtin_amdgcn_sched_barrier(0);
            load_frags(2 * pn, o.x, a0, b0);
            __builtin_amdgcn_sched_barrier(0);
            mfma_step(a1, b1, false);
            __builtin_amdgcn_sched_barrier(0);
            load_frags(2 * pn + 1, o.y, a1, b1);
            __builtin_amdgcn_sched_barrier(0);
        }

        // the next tile's first input batch is loaded into registers now, so
        // its latency hides behind this tile's epilogue and copy-out
        const int next = tile + gridDim.x;
        TileXY Tn = T;
        if (PREF && next < a.ntiles) {
            Tn = tile_xy(a, next);
            if (a.quad16)
                halo_issue<BITS, true, UH, NT, F4>(a, tid, totq, Tn.n0, Tn.iy0, Tn.ix0, hq, hd);
            else
                halo_issue<BITS, false, UH, NT, F4>(a, tid, totq, Tn.n0, Tn.iy0, Tn.ix0, hq, hd);
        }

        if (a.alias_out)
            __syncthreads();  // every wave is done reading sX before sC = sX is written

        // ---- epilogue: lane (r32, h) of tile (t, c) holds output channel
        // t*32 + r32 for pixels c*32 + 8*(v/4) + 4*h + v%4 (register v) ----
        if (a.epi == EPI_RAW32) {
            // an opaque zero keeps the per-register pixel arithmetic below
            // inside the tile loop (hoisted, it would occupy registers
            // throughout)
            int ez = 0;
            __asm__ volatile("" : "+v"(ez));
#pragma unroll
            for (int t = 0; t < WM; ++t) {
                const int mg = m0 + t * 32 + r32;
                const int4 e0 = sEpi[4 * (t * 32 + r32)];
                const int64_t bt = (int64_t)(((uint64_t)(uint32_t)e0.y << 32) | (uint32_t)e0.x);
#pragma unroll
                for (int c = 0; c < WN; ++c)
#pragma unroll
                    for (int v = 0; v < 16; ++v) {
                        const int p = wv * 32 * WN + c * 32 + 8 * (v >> 2) + 4 * h + (v & 3) + ez;
                        if (mg >= a.m || p >= tile_px)
                            continue;
                        const int tI = (int)fdiv((uint32_t)p, a.div_tile_px);
                        const int rem = p - tI * a.th * a.tw;
                        const int py = (int)fdiv((uint32_t)rem, a.div_tw);
                        const int px = rem - py * a.tw;
                        const int nn = T.n0 + tI, oy = T.oy0 + py, ox = T.ox0 + px;
                        if (nn >= a.n || oy >= a.ho || ox >= a.wo)
                            continue;
                        const int32_t acc32 = (int32_t)acc[t][c][v] >> SL;
                        const size_t gp = (size_t)(nn * a.ho + oy) * a.wo + ox;
                        ((int32_t *)a.y)[gp * a.m + mg] = (int32_t)(uint32_t)(uint64_t)(acc32 + bt);
                    }
            }
        } else {
            // each lane applies the plan of its own channel: one plan per tile
            // row in registers, one code byte per output into local memory
#pragma unroll
            for (int t = 0; t < WM; ++t) {
                const int ch = t * 32 + r32;
                if (THR && BITS != 8 && (a.epi == EPI_STAIR || a.epi == EPI_THRESH1)) {
                    // staircase (Eq. (4)): count the channel's thresholds at or below
                    // acc' (one threshold: the binary output of Eq. (5))
                    int32_t T[16];
                    if (NTH == 1) {
                        T[0] = ((const int32_t *)(sEpi + 4 * ch))[0];
                    } else {
#pragma unroll
                        for (int k = 0; k < 4; ++k) {
                            const int4 q4 = sEpi[4 * ch + k];
                            T[4 * k] = q4.x;
                            T[4 * k + 1] = q4.y;
                            T[4 * k + 2] = q4.z;
                            T[4 * k + 3] = q4.w;
                        }
                    }
#pragma unroll
                    for (int c = 0; c < WN; ++c) {
                        uint8_t *dst = sC + (wv * 32 * WN + c * 32 + 4 * h) * cs + ch;
#pragma unroll
                        for (int v = 0; v < 16; ++v)
                            dst[(8 * (v >> 2) + (v & 3)) * cs] = (uint8_t)stair_level<NTH>((int32_t)acc[t][c][v], T);
                    }
                    continue;
                }
                const int4 e0 = sEpi[4 * ch];
                const int4 e1 = sEpi[4 * ch + 1];
#pragma unroll
                for (int c = 0; c < WN; ++c) {
                    uint8_t *dst = sC + (wv * 32 * WN + c * 32 + 4 * h) * cs + ch;
                    if (all3) {
                        // code = (clamp(acc' - A, 0, DS) * mult + RS) >> shift', all in 32 bits
#pragma unroll
                        for (int v = 0; v < 16; ++v) {
                            const int32_t d = __builtin_elementwise_sub_sat((int32_t)acc[t][c][v], e0.x);
                            const uint32_t dc = (uint32_t)min(max(d, 0), e0.y);
                            const uint32_t code = (__umul24(dc, (uint32_t)e0.z) + (uint32_t)e0.w) >> e1.x;
                            dst[(8 * (v >> 2) + (v & 3)) * cs] = (uint8_t)code;
                        }
                    } else {
#pragma unroll
                        for (int v = 0; v < 16; ++v) {
                            const int32_t accd = (int32_t)acc[t][c][v];
                            uint32_t code;
                            if (e1.z >= 3) {
                                const int32_t d = __builtin_elementwise_sub_sat(accd, e0.x);
                                const uint32_t dc = (uint32_t)min(max(d, 0), e0.y);
                                const uint64_t rs = ((uint64_t)(uint32_t)e1.y << 32) | (uint32_t)e0.w;
                                code = (uint32_t)(((uint64_t)dc * (uint32_t)e0.z + rs) >> e1.x);
                            } else {
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
                                    const int64_t vv = (int64_t)acc32 +
                                        (int64_t)(((uint64_t)(uint32_t)e0.y << 32) | (uint32_t)e0.x);
                                    r = round_shift(vv * (int64_t)e0.z, e0.w);
                                }
                                r = r < a.clip_lo ? a.clip_lo : (r > a.clip_hi ? a.clip_hi : r);
                                code = (uint32_t)r;
                            }
                            dst[(8 * (v >> 2) + (v & 3)) * cs] = (uint8_t)code;
                        }
                    }
                }
            }
        }
        __syncthreads();

        // ---- pack the staged codes and copy them out with coalesced stores ----
        if (EXT && a.epi != EPI_RAW32 && a.pool) {
            // fused 2x2 / stride-2 max-pooling: each pooled pixel takes the
            // byte-wise maximum of its window's codes (windows lie inside the
            // tile: even tile height and width, or whole images)
            const int ob0 = m0 * BITS / 8;
            const int obn = min(a.ot_b, a.ypb - ob0);
            constexpr int CPW = 32 / BITS;
            const int thp = a.th >> 1, twp = a.tw >> 1;
            const int npq = a.ti * thp * twp * a.obq;
            for (int idx = tid; idx < npq; idx += NT) {
                const int pp = (int)fdiv((uint32_t)idx, a.div_obq);
                const int q = idx - pp * a.obq;
                const int tI = (int)fdiv((uint32_t)pp, a.div_ptile);
                const int rem = pp - tI * thp * twp;
                const int pr = (int)fdiv((uint32_t)rem, a.div_ptw);
                const int pc = rem - pr * twp;
                const int nn = T.n0 + tI, oy = (T.oy0 >> 1) + pr, ox = (T.ox0 >> 1) + pc;
                if (nn >= a.n || oy >= a.hp || ox >= a.wp)
                    continue;
                const int p00 = tI * a.th * a.tw + 2 * pr * a.tw + 2 * pc;
                const size_t gp = (size_t)(nn * a.hp + oy) * a.wp + ox;
                if (a.oquad16) {
                    if (4 * q < obn) {
                        __align__(16) uint8_t mx[CPW];
                        const uint8_t *s0 = sC + p00 * cs + q * CPW;
                        max4_codes<BITS>(s0, s0 + cs, s0 + a.tw * cs, s0 + (a.tw + 1) * cs, mx);
                        *(uint32_t *)(a.y + gp * a.ypb + ob0 + 4 * q) = pack_codes_word<BITS>(mx);
                    }
                } else if (q < obn) {
                    // byte-granular tail: 8/BITS codes per output byte
                    uint32_t b = 0;
                    const uint8_t *s0 = sC + p00 * cs + q * (8 / BITS);
#pragma unroll
                    for (int i = 0; i < 8 / BITS; ++i) {
                        const uint8_t c0 = max(s0[i], s0[cs + i]);
                        const uint8_t c1 = max(s0[a.tw * cs + i], s0[(a.tw + 1) * cs + i]);
                        b |= (uint32_t)max(c0, c1) << (i * BITS);
                    }
                    a.y[gp * a.ypb + ob0 + q] = (uint8_t)b;
                }
            }
        } else if (a.epi != EPI_RAW32) {
            const int ob0 = m0 * BITS / 8;
            const int obn = min(a.ot_b, a.ypb - ob0);
            constexpr int CPW = 32 / BITS;  // codes per output word
            if (a.contig) {
                // the tile's valid pixels are consecutive output pixels and the
                // tile holds every channel: consecutive words of the output
                const int valid = a.ti == 1 ? min(a.th, a.ho - T.oy0) * a.wo
                                            : min(a.ti, a.n - T.n0) * a.ho * a.wo;
                const size_t first_px = a.ti == 1 ? ((size_t)T.n0 * a.ho + T.oy0) * a.wo
                                                  : (size_t)T.n0 * a.ho * a.wo;
                uint32_t *dst = (uint32_t *)(a.y + first_px * a.ypb);
                const int nw = valid * a.obq;
                if ((a.obq & 3) == 0) {
                    // four words (16 bytes) per store
                    for (int i4 = tid * 4; i4 < nw; i4 += NT * 4) {
                        const int p = (int)fdiv((uint32_t)i4, a.div_obq);
                        const uint8_t *src = sC + p * cs + (i4 - p * a.obq) * CPW;
                        *(uint4 *)(dst + i4) = make_uint4(pack_codes_word<BITS>(src), pack_codes_word<BITS>(src + CPW),
                                                          pack_codes_word<BITS>(src + 2 * CPW),
                                                          pack_codes_word<BITS>(src + 3 * CPW));
                    }
                } else {
                    for (int idx = tid; idx < nw; idx += NT) {
                        const int p = (int)fdiv((uint32_t)idx, a.div_obq);
                        const int q = idx - p * a.obq;
                        dst[idx] = pack_codes_word<BITS>(sC + p * cs + q * CPW);
                    }
                }
            } else if (a.oquad16 && (a.obq & 3) == 0 && obn == 4 * a.obq && (a.ypb & 15) == 0 &&
                       (ob0 & 15) == 0) {
                // whole 16-byte quads of a pixel's channel range (aligned):
                // one thread per pixel of the tile, its tile coordinates
                // computed once, 16-byte stores (INT-2 batch-256 layer
                // 15.1 -> 14.1 us against one thread per 4-byte word)
                const int nq = a.obq >> 2;
                for (int p = tid; p < tile_px; p += NT) {
                    const int tI = (int)fdiv((uint32_t)p, a.div_tile_px);
                    const int rem = p - tI * a.th * a.tw;
                    const int py = (int)fdiv((uint32_t)rem, a.div_tw);
                    const int px = rem - py * a.tw;
                    const int nn = T.n0 + tI, oy = T.oy0 + py, ox = T.ox0 + px;
                    if (nn >= a.n || oy >= a.ho || ox >= a.wo)
                        continue;
                    const size_t gp = (size_t)(nn * a.ho + oy) * a.wo + ox;
                    uint4 *dst = (uint4 *)(a.y + gp * a.ypb + ob0);
                    for (int j = 0; j < nq; ++j) {
                        const uint8_t *src = sC + p * cs + 4 * j * CPW;
                        dst[j] = make_uint4(pack_codes_word<BITS>(src), pack_codes_word<BITS>(src + CPW),
                                            pack_codes_word<BITS>(src + 2 * CPW),
                                            pack_codes_word<BITS>(src + 3 * CPW));
                    }
                }
            } else {
                const int tq4 = tile_px * a.obq;
                for (int idx = tid; idx < tq4; idx += NT) {
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
                                pack_codes_word<BITS>(sC + p * cs + q * CPW);
                    } else {
                        if (q < obn)
                            a.y[gp * a.ypb + ob0 + q] = pack_codes_byte<BITS>(sC + p * cs + q * (8 / BITS));
                    }
                }
            }
        }
        // the next tile's input staging overwrites sX / sC only after every
        // wave passed the barrier above; its own barrier follows the staging
        if (PREF)
            T = Tn;
    }
}

template <int BITS, bool F4 = false>
hipError_t launch_conv_m32_bits(const ConvArgs &a, int wm, int wn, int al16, int nw, dim3 grid, hipStream_t s)
{
#define QNN_CASE32_XU(WM_, WN_, AL_, EXT_, NW_, UA_)                                            \
    if (wm == WM_ && wn == WN_ && al16 == AL_ && ext == EXT_ && nw == NW_ && ua == UA_) {       \
        static bool attr_set = false;                                                           \
        auto *k = conv_m32_kernel<BITS, WM_, WN_, (AL_ != 0), EXT_, NW_, F4, UA_>;              \
        if (!attr_set) {                                                                        \
            if (hipFuncSetAttribute((const void *)k, hipFuncAttributeMaxDynamicSharedMemorySize,  \
                                    a.lds_bytes > 64 * 1024 ? 160 * 1024 : 64 * 1024) != hipSuccess) \
                (void)hipGetLastError();                                                        \
            attr_set = true;                                                                    \
        }                                                                                       \
        hipLaunchKernelGGL(k, grid, dim3(64 * NW_), a.lds_bytes, s, a);                         \
        return hipGetLastError();                                                               \
    }
#define QNN_CASE32_X(WM_, WN_, AL_, EXT_, NW_) QNN_CASE32_XU(WM_, WN_, AL_, EXT_, NW_, false)
#define QNN_CASE32(WM_, WN_, AL_) QNN_CASE32_X(WM_, WN_, AL_, false, 4) QNN_CASE32_X(WM_, WN_, AL_, true, 4)
    const bool ext = a.pool != 0 || a.epi == EPI_STAIR || (int64_t)grid.x < a.ntiles;
    const bool ua = a.wunpack != 0;
    if constexpr (!F4 && BITS == 4) {
        // filters staged unpacked (4-bit layers walked tap by tap)
#define QNN_CASE32_U(WM_, WN_)                                                                  \
        QNN_CASE32_XU(WM_, WN_, 1, false, 4, true) QNN_CASE32_XU(WM_, WN_, 1, true, 4, true)    \
        QNN_CASE32_XU(WM_, WN_, 1, false, 8, true)
        QNN_CASE32_U(1, 1) QNN_CASE32_U(2, 1) QNN_CASE32_U(1, 2) QNN_CASE32_U(2, 2)
#undef QNN_CASE32_U
    }
    QNN_CASE32(1, 1, 0) QNN_CASE32(1, 2, 0) QNN_CASE32(2, 1, 0) QNN_CASE32(2, 2, 0)
    QNN_CASE32(1, 1, 1) QNN_CASE32(1, 2, 1) QNN_CASE32(2, 1, 1) QNN_CASE32(2, 2, 1)
    // eight-wave workgroups: plain instances for layers with one tile per workgroup
    QNN_CASE32_X(1, 1, 1, false, 8) QNN_CASE32_X(2, 1, 1, false, 8)
    QNN_CASE32_X(1, 2, 1, false, 8) QNN_CASE32_X(2, 2, 1, false, 8)
    if constexpr (F4) {
        // the e2m1 path also walks several tiles per eight-wave workgroup
        // (one workgroup per compute unit keeps its staged filter rows)
        QNN_CASE32_X(1, 1, 1, true, 8) QNN_CASE32_X(2, 1, 1, true, 8)
        QNN_CASE32_X(1, 2, 1, true, 8) QNN_CASE32_X(2, 2, 1, true, 8)
    }
    if constexpr (BITS == 8 && !F4) {
        // 128-channel wave tiles: 8-bit only (the sub-byte expansion does not fit
        // two workgroups' register budget at this width)
        QNN_CASE32(4, 1, 0) QNN_CASE32(4, 1, 1)
    }
#undef QNN_CASE32
#undef QNN_CASE32_X
#undef QNN_CASE32_XU
    return hipErrorInvalidValue;
}

}  // namespace qnn
