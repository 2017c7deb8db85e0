// Implicit-GEMM quantized convolution for layers whose input pixel is ONE
// packed 32-bit word: a network's first layer (3-4 image channels at 8 bits,
// up to 8 at 4 bits, up to 16 at 2 bits), stride 1, 3x3 or 5x5 filters,
// output rows of at most 32 pixels.  Same computation as the other
// convolution kernels (Sec. III-A Eq. (2), Sec. III-B Eq. (6), scale-and-
// clamp compression, Sec. IV-A fused max-pooling), laid out for a K of only
// kh*kw taps of one word each, where the general kernels spend most of their
// instructions on per-tile bookkeeping:
//   * a workgroup owns one 32-channel group and walks whole images: the
//     padded image is staged once in LDS (unpacked to int8, pads included),
//     the next image's words are loaded into registers while the current one
//     is computed;
//   * the filters of the group live in registers for the whole kernel (one
//     16-byte fragment per lane and K step), never in LDS;
//   * a wave computes two output rows (32 pixels each) at a time with
//     v_mfma_i32_32x32x32_i8, rows = pixels, columns = channels;
//   * K order: the two halves of a wave (lanes 0-31, 32-63) cover the
//     filter's upper and lower band of ceil(kh/2) rows in the same slot
//     order, so every im2col tap is an LDS read at a compile-time offset
//     from one per-lane base (bands past the filter's last row and slots
//     past the band carry zero weights); 8-bit tiles store a pixel pair per
//     slot, so a run of four taps along a filter row is two aligned 8-byte
//     reads;
//   * the 2x2 max-pooling is taken on the accumulators (the compression is
//     non-decreasing in the accumulator whenever the multiplier is positive,
//     so the maximum commutes with it) and only the pooled values are
//     compressed; with a non-positive multiplier each code is compressed
//     first and the codes are pooled;
//   * codes leave as bytes straight from the lanes (4-/2-bit codes of
//     neighbouring channels packed across lanes with DPP moves), with no
//     staging through LDS.
#include "conv_m32_impl.h"

namespace qnn {

// Slot order of the K dimension within one half band (DY filter rows x KW
// columns), TPF taps per 16-byte fragment.  4- and 2-bit layers: the taps in
// raster order.  8-bit layers (4-byte taps): first every run of four
// horizontally adjacent taps of a filter row (one fragment each, read as two
// aligned 8-byte pixel pairs), then the leftover columns of all rows, four
// to a fragment.  tap(i) = ky * 256 + kx, or -1 for an empty slot (zero
// weight, nothing read).
template <int BITS, int KW, int DY>
struct Px4Taps {
    static constexpr int TPF = BITS == 8 ? 4 : (BITS == 4 ? 2 : 1);
    static constexpr int NT = DY * KW;
    static constexpr int RUNS = BITS == 8 ? KW / 4 : 0;
    static constexpr int LEFT = KW % 4;
    static constexpr int NR = DY * RUNS;
    static constexpr int NF = BITS == 8 ? NR + (DY * LEFT + 3) / 4 : (NT + TPF - 1) / TPF;
    static constexpr int tap(int i)
    {
        if (BITS != 8)
            return i < NT ? (i / KW) * 256 + i % KW : -1;
        const int f = i / 4, t = i % 4;
        if (f < NR)
            return (f / (RUNS > 0 ? RUNS : 1)) * 256 + (f % (RUNS > 0 ? RUNS : 1)) * 4 + t;
        const int j = (f - NR) * 4 + t;
        return (LEFT > 0 && j < DY * LEFT) ? (j / (LEFT > 0 ? LEFT : 1)) * 256 + RUNS * 4 + j % (LEFT > 0 ? LEFT : 1)
                                          : -1;
    }
};

// One 16-byte im2col fragment of the pixel whose tile slot is at p, for K
// step S: compile-time offsets into the tile (pitch PP slots of SB bytes).
// 8-bit tiles hold a pixel pair per slot (the pixel and its right
// neighbour), so two adjacent taps are one aligned 8-byte read.
template <int BITS, int KW, int DY, int PP, int S>
__device__ __forceinline__ v4i px4_frag(const uint8_t *p)
{
    typedef Px4Taps<BITS, KW, DY> TP;
    constexpr int SB = BITS == 8 ? 8 : 32 / BITS;
    constexpr int TPF = TP::TPF;
    if constexpr (BITS == 8) {
        uint32_t d[4];
#pragma unroll
        for (int t = 0; t < 4; t += 2) {
            const int t0 = TP::tap(S * TPF + t), t1 = TP::tap(S * TPF + t + 1);
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
    } else if constexpr (BITS == 4) {
        uint2 d[2];
#pragma unroll
        for (int t = 0; t < 2; ++t) {
            const int tp = TP::tap(S * TPF + t);
            d[t] = tp >= 0 ? *(const uint2 *)(p + ((tp >> 8) * PP + (tp & 255)) * SB) : make_uint2(0, 0);
        }
        return (v4i){(int32_t)d[0].x, (int32_t)d[0].y, (int32_t)d[1].x, (int32_t)d[1].y};
    } else {
        constexpr int tp = TP::tap(S);
        if constexpr (tp >= 0)
            return *(const v4i *)(p + ((tp >> 8) * PP + (tp & 255)) * SB);
        else
            return (v4i){0, 0, 0, 0};
    }
}

// Both rows' fragments and MFMAs of K steps S .. KS-1 (unrolled through the
// template recursion, so every offset is an immediate).
template <int BITS, int KW, int DY, int PP, int KS, int S>
__device__ __forceinline__ void px4_steps(const uint8_t *p0, const uint8_t *p1, const v4i *A, v16i &acc0,
                                          v16i &acc1)
{
    if constexpr (S < KS) {
        const v4i b0 = px4_frag<BITS, KW, DY, PP, S>(p0);
        const v4i b1 = px4_frag<BITS, KW, DY, PP, S>(p1);
        if constexpr (S == 0) {
            acc0 = __builtin_amdgcn_mfma_i32_32x32x32_i8(b0, A[S], (v16i){}, 0, 0, 0);
            acc1 = __builtin_amdgcn_mfma_i32_32x32x32_i8(b1, A[S], (v16i){}, 0, 0, 0);
        } else {
            acc0 = __builtin_amdgcn_mfma_i32_32x32x32_i8(b0, A[S], acc0, 0, 0, 0);
            acc1 = __builtin_amdgcn_mfma_i32_32x32x32_i8(b1, A[S], acc1, 0, 0, 0);
        }
        px4_steps<BITS, KW, DY, PP, KS, S + 1>(p0, p1, A, acc0, acc1);
    }
}

// Scale-and-clamp code of one (scaled) accumulator from the channel's plan
// (requant_plan): any mode.
template <int SL>
__device__ __forceinline__ uint32_t px4_code(int32_t accd, const int4 &e0, const int4 &e1, int32_t lo,
                                             int32_t hi)
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

// Mode-3 plans only (every channel's code fits the 32-bit form): a
// saturating subtract, a median-of-three clamp to [0, e0.y] (e0.y >= 0), a
// 24-bit multiply-add and a shift.
__device__ __forceinline__ uint32_t px4_code3(int32_t accd, const int4 &e0, const int4 &e1)
{
    const int32_t d = __builtin_elementwise_sub_sat(accd, e0.x);
    int32_t dc;
    __asm__("v_med3_i32 %0, %1, 0, %2" : "=v"(dc) : "v"(d), "v"(e0.y));
    return (__umul24((uint32_t)dc, (uint32_t)e0.z) + (uint32_t)e0.w) >> e1.x;
}

// Mode-3 and mode-4 plans (the strict form; products up to 64 bits): a
// saturating subtract, the clamp, one 32x32->64 multiply-add and a shift.
__device__ __forceinline__ uint32_t px4_code4(int32_t accd, const int4 &e0, const int4 &e1)
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
__device__ __forceinline__ uint32_t px4_pack_lanes(uint32_t code)
{
    if (BITS == 8)
        return code;
    // quad_perm [1,0,3,2]: the neighbour's code
    uint32_t v = code | ((uint32_t)__builtin_amdgcn_update_dpp(0, (int)code, 0xB1, 0xF, 0xF, false) << BITS);
    if (BITS == 2)  // quad_perm [2,3,0,1]: the other pair
        v |= (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x4E, 0xF, 0xF, false) << 4;
    return v;
}

template <int BITS, int KH, int KW, bool POOL>
__global__ void __launch_bounds__(256) conv_px4_kernel(Px4Args a)
{
    constexpr int NW = 4, NT = 256;
    constexpr int UB = 32 / BITS;              // staged (int8) bytes per pixel
    constexpr int SB = BITS == 8 ? 8 : UB;     // tile slot bytes (8 bits: a pixel pair)
    constexpr int PP = 32 + KW - 1;            // tile pitch, slots
    constexpr int RB = PP * SB;                // tile row, bytes
    constexpr int DY = (KH + 1) / 2;           // filter rows per half band
    typedef Px4Taps<BITS, KW, DY> TP;
    constexpr int TPF = TP::TPF;               // taps per 16-byte fragment
    constexpr int KS = TP::NF;                 // 32-deep K steps
    constexpr int SL = BITS == 4 ? 4 : (BITS == 2 ? 6 : 0);  // log2 of the weight scale
    constexpr int UPF = 2;                     // prefetched 4-pixel groups per thread
    constexpr int WROW = KH * KW * 4;          // packed bytes per filter bank
    extern __shared__ __align__(16) uint8_t smem[];
    uint8_t *sX = smem;
    const int tid = threadIdx.x;
    const int lane = tid & 63, r32 = lane & 31, h = lane >> 5;
    const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform
    const int gy = blockIdx.y;
    const int ch = gy * 32 + r32;
    const bool live = ch < a.m;
    const int npix = a.h * a.w_;

    // ---- the first image's words: issued before anything else ----
    uint4 pf[UPF];
    auto issue = [&](int img) {
        const uint32_t *src = a.x + (size_t)img * (uint32_t)npix;
#pragma unroll
        for (int u = 0; u < UPF; ++u) {
            const int p0 = 4 * (tid + u * NT);
            pf[u] = make_uint4(0, 0, 0, 0);
            if (a.quads) {
                if (p0 < npix)
                    pf[u] = *(const uint4 *)(src + p0);
            } else {
                if (p0 < npix)
                    pf[u].x = src[p0];
                if (p0 + 1 < npix)
                    pf[u].y = src[p0 + 1];
                if (p0 + 2 < npix)
                    pf[u].z = src[p0 + 2];
                if (p0 + 3 < npix)
                    pf[u].w = src[p0 + 3];
            }
        }
    };
    int img = blockIdx.x;
    if (img < a.n)
        issue(img);

    // ---- filters: the lane's fragment of every K step, expanded to int8
    // (4-/2-bit weights as 16*w / 64*w) ----
    v4i A[KS];
    int wsum = 0;
    {
        const uint8_t *wb = a.w + (size_t)(live ? ch : 0) * WROW;
#pragma unroll
        for (int s = 0; s < KS; ++s) {
            uint32_t d[4];
#pragma unroll
            for (int t = 0; t < TPF; ++t) {
                const int tp = TP::tap(s * TPF + t);
                const int ky = (tp >> 8) + h * DY, kx = tp & 255;
                uint32_t v = 0;
                if (tp >= 0 && live && ky < KH)
                    v = *(const uint32_t *)(wb + (ky * KW + kx) * 4);
                if (BITS == 8) {
                    d[t] = v;
                    wsum += (int)(int8_t)v + (int)(int8_t)(v >> 8) + (int)(int8_t)(v >> 16) + (int)(int8_t)(v >> 24);
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
    if (BITS == 8)
        wsum += __shfl_xor(wsum, 32, 64);  // the other band's half of the channel

    // ---- the channel's compression plan (requant_plan) ----
    int32_t p_bias = 0, p_mult = 0, p_shift = 0;
    if (live) {
        if (a.bias)
            p_bias = a.bias[ch];
        if (a.epi == EPI_REQUANT) {
            p_mult = a.mult[ch];
            p_shift = a.shift[ch];
        }
    }
    int4 e0, e1;
    {
        int64_t b = p_bias;
        if (BITS == 8)
            b += 128 * (int64_t)wsum;
        const int sh = p_shift < 0 ? 0 : (p_shift > 62 ? 62 : p_shift);
        requant_plan(b, p_mult, sh, a.clip_lo, a.clip_hi, a.epi == EPI_REQUANT, SL, e0, e1);
    }
    // wave-uniform fast paths: every channel in the 32-bit strict form; every
    // channel's code non-decreasing in the accumulator (positive multiplier)
    const bool all3 = __all(!live || e1.z == 3);
    const bool all34 = __all(!live || e1.z == 3 || e1.z == 4);
    const bool mono = __all(!live || e1.z != 0 || e0.z > 0);
    const int64_t bt = (int64_t)(((uint64_t)(uint32_t)e0.y << 32) | (uint32_t)e0.x);  // raw: bias (+ 128 wsum)

    // ---- pads: the whole tile holds the zero code once (staged: -128 at 8
    // bits); each image then overwrites only its interior ----
    {
        const uint32_t f = BITS == 8 ? 0x80808080u : 0u;
        const uint4 f4 = make_uint4(f, f, f, f);
        for (int i = tid; i < a.tile_bytes / 16; i += NT)
            ((uint4 *)sX)[i] = f4;
    }
    __syncthreads();

    const int nrp = (a.ho + 1) >> 1;  // output row pairs
    for (; img < a.n; img += gridDim.x) {
        // stage the prefetched words into the tile interior
#pragma unroll
        for (int u = 0; u < UPF; ++u) {
            const int p0 = 4 * (tid + u * NT);
            if (p0 < npix) {
                int iy = (int)fdiv((uint32_t)p0, a.div_w);
                int ix = p0 - iy * a.w_;
                const uint32_t wd[4] = {pf[u].x, pf[u].y, pf[u].z, pf[u].w};
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    if (p0 + j < npix) {
                        uint8_t *dst = sX + ((iy + a.ph) * PP + ix + a.pw) * SB;
                        stage_word<BITS>(dst, wd[j]);
                        if (BITS == 8 && ix + a.pw > 0)
                            stage_word<BITS>(dst - 4, wd[j]);  // second pixel of the slot on its left
                    }
                    if (++ix == a.w_) {
                        ix = 0;
                        ++iy;
                    }
                }
            }
        }
        __syncthreads();
        if (img + (int)gridDim.x < a.n)
            issue(img + gridDim.x);

        // row pairs rp = wv, wv + NW, ... of this image go to this wave
        // (pooled layers stop at the last complete pair of rows)
        const int nl = POOL ? a.hp : nrp;
        auto mfma_rows = [&](int rp, v16i &c0, v16i &c1) {
            const uint8_t *p0 = sX + (2 * rp * PP + r32) * SB + h * DY * RB;
            px4_steps<BITS, KW, DY, PP, KS, 0>(p0, p0 + RB, A, c0, c1);
        };
        auto run_rows = [&](auto epi) {
            for (int rp = wv; rp < nl; rp += NW) {
                v16i x0, x1;
                mfma_rows(rp, x0, x1);
                epi(rp, x0, x1);
            }
        };
        // ---- epilogues: lane (r32, h) holds channel ch for pixels
        // ox = 8*(v/4) + 4h + v%4 (register v) of rows 2rp, 2rp+1; the form
        // (every channel in the 32-bit or the 64-bit strict plan, or any
        // plan) is chosen once per image, outside the row loop ----
        // codes go straight to memory as bytes: a lane stores the byte of its
        // channel (and of its neighbours', packed across lanes at 4 / 2 bits)
        // for each of its pixels; a row of M = 32 channels is a run of whole
        // bytes, so the stores of a wave cover contiguous spans
        const bool st_ok = live && (r32 % (8 / BITS)) == 0;
        const int ch_byte = gy * 4 * BITS + ((r32 * BITS) >> 3);
        if constexpr (POOL) {
            // pooled pixel of value k (0..7): 4*(k/2) + 2h + k%2
            auto store_pool = [&](int rp, const uint32_t *code) {
                uint32_t byte[8];
#pragma unroll
                for (int k = 0; k < 8; ++k)
                    byte[k] = px4_pack_lanes<BITS>(code[k]);
                if (!st_ok)
                    return;
                uint8_t *yb = a.y + ((size_t)img * a.hp + rp) * a.wp * a.ypb + ch_byte;
                if (a.ypb == 4 * BITS && a.wp >= 16) {
                    // one 32-channel group, whole rows: compile-time strides
                    yb += 2 * h * (4 * BITS);
#pragma unroll
                    for (int k = 0; k < 8; ++k)
                        yb[(4 * (k >> 1) + (k & 1)) * (4 * BITS)] = (uint8_t)byte[k];
                } else {
#pragma unroll
                    for (int k = 0; k < 8; ++k) {
                        const int px = 4 * (k >> 1) + 2 * h + (k & 1);
                        if (px < a.wp)
                            yb[(size_t)px * a.ypb] = (uint8_t)byte[k];
                    }
                }
            };
            if (all3) {
                run_rows([&](int rp, const v16i &c0, const v16i &c1) {
                    uint32_t code[8];
#pragma unroll
                    for (int k = 0; k < 8; ++k)
                        code[k] = px4_code3(max(max(c0[2 * k], c0[2 * k + 1]), max(c1[2 * k], c1[2 * k + 1])), e0, e1);
                    store_pool(rp, code);
                });
            } else if (all34) {
                run_rows([&](int rp, const v16i &c0, const v16i &c1) {
                    uint32_t code[8];
#pragma unroll
                    for (int k = 0; k < 8; ++k)
                        code[k] = px4_code4(max(max(c0[2 * k], c0[2 * k + 1]), max(c1[2 * k], c1[2 * k + 1])), e0, e1);
                    store_pool(rp, code);
                });
            } else {
                // rare forms (plans outside the strict form, or multipliers
                // that are not positive): one pooled value at a time, kept
                // rolled so their 64-bit temporaries do not crowd the
                // registers of the fast forms
                run_rows([&](int rp, const v16i &c0, const v16i &c1) {
                    uint8_t *yb = a.y + ((size_t)img * a.hp + rp) * a.wp * a.ypb + ch_byte;
#pragma unroll 1
                    for (int k = 0; k < 8; ++k) {
                        const int32_t a0 = c0[2 * k], a1 = c0[2 * k + 1], b0 = c1[2 * k], b1 = c1[2 * k + 1];
                        uint32_t code;
                        if (mono)
                            code = px4_code<SL>(max(max(a0, a1), max(b0, b1)), e0, e1, a.clip_lo, a.clip_hi);
                        else
                            code = max(max(px4_code<SL>(a0, e0, e1, a.clip_lo, a.clip_hi),
                                           px4_code<SL>(a1, e0, e1, a.clip_lo, a.clip_hi)),
                                       max(px4_code<SL>(b0, e0, e1, a.clip_lo, a.clip_hi),
                                           px4_code<SL>(b1, e0, e1, a.clip_lo, a.clip_hi)));
                        const uint32_t byte = px4_pack_lanes<BITS>(code);
                        const int px = 4 * (k >> 1) + 2 * h + (k & 1);
                        if (st_ok && px < a.wp)
                            yb[(size_t)px * a.ypb] = (uint8_t)byte;
                    }
                });
            }
        } else if (a.epi == EPI_RAW32) {
            run_rows([&](int rp, const v16i &c0, const v16i &c1) {
#pragma unroll
                for (int r = 0; r < 2; ++r) {
                    const int oy = 2 * rp + r;
                    if (oy >= a.ho || !live)
                        continue;
                    int32_t *yr = (int32_t *)a.y + ((size_t)img * a.ho + oy) * a.wo * a.m + ch;
#pragma unroll
                    for (int v = 0; v < 16; ++v) {
                        const int ox = 8 * (v >> 2) + 4 * h + (v & 3);
                        const int32_t av = r ? c1[v] : c0[v];
                        if (ox < a.wo)
                            yr[(size_t)ox * a.m] = (int32_t)(uint32_t)(uint64_t)((int64_t)(av >> SL) + bt);
                    }
                }
            });
        } else {
            // output pixel of value v (0..15): 8*(v/4) + 4h + v%4
            auto store_row = [&](int oy, const uint32_t *code) {
                uint32_t byte[16];
#pragma unroll
                for (int v = 0; v < 16; ++v)
                    byte[v] = px4_pack_lanes<BITS>(code[v]);
                if (!st_ok || oy >= a.ho)
                    return;
                uint8_t *yb = a.y + ((size_t)img * a.ho + oy) * a.wo * a.ypb + ch_byte;
                if (a.ypb == 4 * BITS && a.wo >= 32) {
                    yb += 4 * h * (4 * BITS);
#pragma unroll
                    for (int v = 0; v < 16; ++v)
                        yb[(8 * (v >> 2) + (v & 3)) * (4 * BITS)] = (uint8_t)byte[v];
                } else {
#pragma unroll
                    for (int v = 0; v < 16; ++v) {
                        const int ox = 8 * (v >> 2) + 4 * h + (v & 3);
                        if (ox < a.wo)
                            yb[(size_t)ox * a.ypb] = (uint8_t)byte[v];
                    }
                }
            };
            if (all3) {
                run_rows([&](int rp, const v16i &c0, const v16i &c1) {
                    uint32_t code[16];
#pragma unroll
                    for (int v = 0; v < 16; ++v)
                        code[v] = px4_code3(c0[v], e0, e1);
                    store_row(2 * rp, code);
#pragma unroll
                    for (int v = 0; v < 16; ++v)
                        code[v] = px4_code3(c1[v], e0, e1);
                    store_row(2 * rp + 1, code);
                });
            } else if (all34) {
                run_rows([&](int rp, const v16i &c0, const v16i &c1) {
                    uint32_t code[16];
#pragma unroll
                    for (int v = 0; v < 16; ++v)
                        code[v] = px4_code4(c0[v], e0, e1);
                    store_row(2 * rp, code);
#pragma unroll
                    for (int v = 0; v < 16; ++v)
                        code[v] = px4_code4(c1[v], e0, e1);
                    store_row(2 * rp + 1, code);
                });
            } else {
                run_rows([&](int rp, const v16i &c0, const v16i &c1) {
#pragma unroll
                    for (int r = 0; r < 2; ++r) {
                        const int oy = 2 * rp + r;
                        if (oy >= a.ho)
                            break;
                        uint8_t *yb = a.y + ((size_t)img * a.ho + oy) * a.wo * a.ypb + ch_byte;
#pragma unroll 1
                        for (int v = 0; v < 16; ++v) {
                            const uint32_t byte = px4_pack_lanes<BITS>(
                                px4_code<SL>(r ? c1[v] : c0[v], e0, e1, a.clip_lo, a.clip_hi));
                            const int ox = 8 * (v >> 2) + 4 * h + (v & 3);
                            if (st_ok && ox < a.wo)
                                yb[(size_t)ox * a.ypb] = (uint8_t)byte;
                        }
                    }
                });
            }
        }
        __syncthreads();  // every wave is done with this image's tile
    }
}

// Grid: as many workgroups as the device holds at once (whole images each),
// so no workgroup starts only after others have finished.
template <typename K>
hipError_t launch_px4_grid(K kernel, const Px4Args &a, int cus, hipStream_t s)
{
    const size_t lds = (size_t)a.tile_bytes;
    int per_cu = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kernel, 256, lds) != hipSuccess || per_cu < 1)
        per_cu = 1;
    const int gy = (a.m + 31) / 32;
    int64_t gx = ((int64_t)cus * per_cu + gy - 1) / gy;
    if (gx > a.n)
        gx = a.n;
    if (gx < 1)
        gx = 1;
    hipLaunchKernelGGL(kernel, dim3((unsigned)gx, (unsigned)gy), dim3(256), lds, s, a);
    return hipGetLastError();
}

template <int BITS, int KH, int KW>
hipError_t launch_px4(const Px4Args &a, int cus, hipStream_t s)
{
    if (a.pool)
        return launch_px4_grid(conv_px4_kernel<BITS, KH, KW, true>, a, cus, s);
    return launch_px4_grid(conv_px4_kernel<BITS, KH, KW, false>, a, cus, s);
}

hipError_t launch_conv_px4(const Px4Args &a, int bits, int kh, int kw, int cus, hipStream_t s)
{
    const int k = kh == kw ? kh : 0;
#define QNN_PX4(B_, K_)                             \
    if (bits == B_ && k == K_)                      \
        return launch_px4<B_, K_, K_>(a, cus, s);
    QNN_PX4(8, 3) QNN_PX4(8, 5) QNN_PX4(4, 3) QNN_PX4(4, 5) QNN_PX4(2, 3) QNN_PX4(2, 5)
#undef QNN_PX4
    return hipErrorInvalidValue;
}

}  // namespace qnn
