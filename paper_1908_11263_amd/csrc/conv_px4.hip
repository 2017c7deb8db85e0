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
//     filter's upper and lower band of ceil(kh/2) rows, tap by tap in the
//     same order, so every im2col tap is an LDS read at a compile-time
//     offset from one per-lane base (bands past the filter's last row and
//     slots past the band carry zero weights);
//   * the 2x2 max-pooling is taken on the accumulators (the compression is
//     non-decreasing in the accumulator whenever the multiplier is positive,
//     so the maximum commutes with it) and only the pooled values are
//     compressed; with a non-positive multiplier each code is compressed
//     first and the codes are pooled.
#include "conv_m32_impl.h"

namespace qnn {

// One 16-byte im2col fragment (TPF taps of UB staged bytes) of the pixel at
// p, for K step S: compile-time offsets into the tile (pitch PP pixels).
template <int BITS, int KW, int PP, int NTH, int S>
__device__ __forceinline__ v4i px4_frag(const uint8_t *p)
{
    constexpr int UB = 32 / BITS;
    constexpr int TPF = 16 / UB;
    if constexpr (BITS == 8) {
        int32_t d[4];
#pragma unroll
        for (int t = 0; t < 4; ++t) {
            const int i = S * TPF + t;
            d[t] = i < NTH ? *(const int32_t *)(p + ((i / KW) * PP + i % KW) * UB) : 0;
        }
        return (v4i){d[0], d[1], d[2], d[3]};
    } else if constexpr (BITS == 4) {
        uint2 d[2];
#pragma unroll
        for (int t = 0; t < 2; ++t) {
            const int i = S * TPF + t;
            d[t] = i < NTH ? *(const uint2 *)(p + ((i / KW) * PP + i % KW) * UB) : make_uint2(0, 0);
        }
        return (v4i){(int32_t)d[0].x, (int32_t)d[0].y, (int32_t)d[1].x, (int32_t)d[1].y};
    } else {
        constexpr int i = S;
        if constexpr (i < NTH)
            return *(const v4i *)(p + ((i / KW) * PP + i % KW) * UB);
        else
            return (v4i){0, 0, 0, 0};
    }
}

// Both rows' fragments and MFMAs of K steps S .. KS-1 (unrolled through the
// template recursion, so every offset is an immediate).
template <int BITS, int KW, int PP, int NTH, int KS, int S>
__device__ __forceinline__ void px4_steps(const uint8_t *p0, const uint8_t *p1, const v4i *A, v16i &acc0,
                                          v16i &acc1)
{
    if constexpr (S < KS) {
        const v4i b0 = px4_frag<BITS, KW, PP, NTH, S>(p0);
        const v4i b1 = px4_frag<BITS, KW, PP, NTH, S>(p1);
        if constexpr (S == 0) {
            acc0 = __builtin_amdgcn_mfma_i32_32x32x32_i8(b0, A[S], (v16i){}, 0, 0, 0);
            acc1 = __builtin_amdgcn_mfma_i32_32x32x32_i8(b1, A[S], (v16i){}, 0, 0, 0);
        } else {
            acc0 = __builtin_amdgcn_mfma_i32_32x32x32_i8(b0, A[S], acc0, 0, 0, 0);
            acc1 = __builtin_amdgcn_mfma_i32_32x32x32_i8(b1, A[S], acc1, 0, 0, 0);
        }
        px4_steps<BITS, KW, PP, NTH, KS, S + 1>(p0, p1, A, acc0, acc1);
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

// Mode-3 plans only (every channel's code fits the 32-bit form).
__device__ __forceinline__ uint32_t px4_code3(int32_t accd, const int4 &e0, const int4 &e1)
{
    const int32_t d = __builtin_elementwise_sub_sat(accd, e0.x);
    const uint32_t dc = (uint32_t)min(max(d, 0), e0.y);
    return (__umul24(dc, (uint32_t)e0.z) + (uint32_t)e0.w) >> e1.x;
}

// Makes this wave's LDS writes visible to its own later LDS reads (and keeps
// the compiler from moving LDS accesses across the point).
__device__ __forceinline__ void wave_lds_sync()
{
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

template <int BITS, int KH, int KW, bool POOL>
__global__ void __launch_bounds__(256) conv_px4_kernel(Px4Args a)
{
    constexpr int NW = 4, NT = 256;
    constexpr int UB = 32 / BITS;              // staged (int8) bytes per pixel
    constexpr int PP = 32 + KW - 1;            // tile pitch, pixels
    constexpr int RB = PP * UB;                // tile row, bytes
    constexpr int DY = (KH + 1) / 2;           // filter rows per half band
    constexpr int NTH = DY * KW;               // taps per half band
    constexpr int TPF = 16 / UB;               // taps per 16-byte fragment
    constexpr int KS = (NTH + TPF - 1) / TPF;  // 32-deep K steps
    constexpr int SL = BITS == 4 ? 4 : (BITS == 2 ? 6 : 0);  // log2 of the weight scale
    constexpr int NPX = POOL ? 16 : 32;        // staged output pixels per wave
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
    uint8_t *sC = smem + a.tile_bytes + wv * NPX * 32;
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
                const int i = s * TPF + t;
                const int ky = i / KW + h * DY, kx = i % KW;
                uint32_t v = 0;
                if (i < NTH && live && ky < KH)
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
    // output words of this channel group per pixel (the group's channels
    // fill whole words: M * bits is a multiple of 32)
    const int mv = min(32, a.m - gy * 32);
    const int wpp = mv * BITS / 32;
    const int wi = lane & 7;
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
                    if (p0 + j < npix)
                        stage_word<BITS>(sX + ((iy + a.ph) * PP + ix + a.pw) * UB, wd[j]);
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

        for (int rp = wv; rp < nrp; rp += NW) {
            const uint8_t *p0 = sX + (2 * rp * PP + r32) * UB + h * DY * RB;
            v16i acc0, acc1;
            px4_steps<BITS, KW, PP, NTH, KS, 0>(p0, p0 + RB, A, acc0, acc1);

            // ---- epilogue: lane (r32, h) holds channel ch for pixels
            // ox = 8*(v/4) + 4h + v%4 (register v) of rows 2rp, 2rp+1 ----
            if (POOL) {
                if (rp >= a.hp)
                    continue;
#pragma unroll
                for (int k = 0; k < 8; ++k) {
                    const int32_t a0 = acc0[2 * k], a1 = acc0[2 * k + 1];
                    const int32_t c0 = acc1[2 * k], c1 = acc1[2 * k + 1];
                    uint32_t code;
                    if (mono) {
                        const int32_t mx = max(max(a0, a1), max(c0, c1));
                        code = all3 ? px4_code3(mx, e0, e1) : px4_code<SL>(mx, e0, e1, a.clip_lo, a.clip_hi);
                    } else {
                        code = max(max(px4_code<SL>(a0, e0, e1, a.clip_lo, a.clip_hi),
                                       px4_code<SL>(a1, e0, e1, a.clip_lo, a.clip_hi)),
                                   max(px4_code<SL>(c0, e0, e1, a.clip_lo, a.clip_hi),
                                       px4_code<SL>(c1, e0, e1, a.clip_lo, a.clip_hi)));
                    }
                    const int px = 4 * (k >> 1) + 2 * h + (k & 1);
                    sC[px * 32 + r32] = (uint8_t)code;
                }
                wave_lds_sync();
                uint8_t *yrow = a.y + ((size_t)img * a.hp + rp) * a.wp * a.ypb + gy * 4 * BITS + wi * 4;
#pragma unroll
                for (int j = 0; j < 2; ++j) {
                    const int px = (lane >> 3) + 8 * j;
                    if (px < a.wp && wi < wpp)
                        *(uint32_t *)(yrow + (size_t)px * a.ypb) = pack_codes_word<BITS>(sC + px * 32 + wi * (32 / BITS));
                }
                wave_lds_sync();
            } else {
                // one output row at a time (rows 2rp and 2rp+1)
                auto row_out = [&](const v16i &acc, int oy) {
                    if (oy >= a.ho)
                        return;
                    if (a.epi == EPI_RAW32) {
                        if (!live)
                            return;
                        int32_t *yr = (int32_t *)a.y + ((size_t)img * a.ho + oy) * a.wo * a.m + ch;
#pragma unroll
                        for (int v = 0; v < 16; ++v) {
                            const int ox = 8 * (v >> 2) + 4 * h + (v & 3);
                            if (ox < a.wo)
                                yr[(size_t)ox * a.m] = (int32_t)(uint32_t)(uint64_t)((int64_t)(acc[v] >> SL) + bt);
                        }
                        return;
                    }
#pragma unroll
                    for (int v = 0; v < 16; ++v) {
                        const uint32_t code = all3 ? px4_code3(acc[v], e0, e1)
                                                   : px4_code<SL>(acc[v], e0, e1, a.clip_lo, a.clip_hi);
                        const int ox = 8 * (v >> 2) + 4 * h + (v & 3);
                        sC[ox * 32 + r32] = (uint8_t)code;
                    }
                    wave_lds_sync();
                    uint8_t *yrow = a.y + ((size_t)img * a.ho + oy) * a.wo * a.ypb + gy * 4 * BITS + wi * 4;
#pragma unroll
                    for (int j = 0; j < 4; ++j) {
                        const int px = (lane >> 3) + 8 * j;
                        if (px < a.wo && wi < wpp)
                            *(uint32_t *)(yrow + (size_t)px * a.ypb) =
                                pack_codes_word<BITS>(sC + px * 32 + wi * (32 / BITS));
                    }
                    wave_lds_sync();
                };
                row_out(acc0, 2 * rp);
                row_out(acc1, 2 * rp + 1);
            }
        }
        __syncthreads();  // every wave is done with this image's tile
    }
}

template <int BITS, int KH, int KW>
hipError_t launch_px4(const Px4Args &a, dim3 grid, hipStream_t s)
{
    const size_t lds = (size_t)a.tile_bytes + 4 * (a.pool ? 16 : 32) * 32;
    if (a.pool)
        hipLaunchKernelGGL((conv_px4_kernel<BITS, KH, KW, true>), grid, dim3(256), lds, s, a);
    else
        hipLaunchKernelGGL((conv_px4_kernel<BITS, KH, KW, false>), grid, dim3(256), lds, s, a);
    return hipGetLastError();
}

hipError_t launch_conv_px4(const Px4Args &a, int bits, int kh, int kw, dim3 grid, hipStream_t s)
{
    const int k = kh == kw ? kh : 0;
#define QNN_PX4(B_, K_)                             \
    if (bits == B_ && k == K_)                      \
        return launch_px4<B_, K_, K_>(a, grid, s);
    QNN_PX4(8, 3) QNN_PX4(8, 5) QNN_PX4(4, 3) QNN_PX4(4, 5) QNN_PX4(2, 3) QNN_PX4(2, 5)
#undef QNN_PX4
    return hipErrorInvalidValue;
}

}  // namespace qnn
