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

// Four 4-bit two's complement weights (16 bits, lowest element in the low
// nibble) -> four bytes holding 16*w each.
__device__ __forceinline__ uint32_t w4_to_s8x16(uint32_t u)
{
    return ((u & 0xFu) << 4) | ((u & 0xF0u) << 8) | ((u & 0xF00u) << 12) | ((u & 0xF000u) << 16);
}

// Four 2-bit two's complement weights (one byte) -> four bytes holding 64*w.
__device__ __forceinline__ uint32_t w2_to_s8x64(uint32_t u)
{
    return ((u & 0x3u) << 6) | ((u & 0xCu) << 12) | ((u & 0x30u) << 18) | ((u & 0xC0u) << 24);
}

// Eight unsigned 4-bit activations -> eight bytes (natural order).
__device__ __forceinline__ uint2 a4_to_u8(uint32_t v)
{
    uint2 r;
    r.x = (v & 0xFu) | ((v & 0xF0u) << 4) | ((v & 0xF00u) << 8) | ((v & 0xF000u) << 12);
    v >>= 16;
    r.y = (v & 0xFu) | ((v & 0xF0u) << 4) | ((v & 0xF00u) << 8) | ((v & 0xF000u) << 12);
    return r;
}

// Four unsigned 2-bit activations (one byte) -> four bytes.
__device__ __forceinline__ uint32_t a2_byte_to_u8(uint32_t u)
{
    return (u & 0x3u) | ((u & 0xCu) << 6) | ((u & 0x30u) << 12) | ((u & 0xC0u) << 18);
}

// Stage one packed 4-byte word of activations at `dst` (unpacked bytes).
template <int BITS>
__device__ __forceinline__ void stage_word(uint8_t *dst, uint32_t v)
{
    if (BITS == 8) {
        *(uint32_t *)dst = v ^ 0x80808080u;
    } else if (BITS == 4) {
        *(uint2 *)dst = a4_to_u8(v);
    } else {
        uint4 o;
        o.x = a2_byte_to_u8(v & 0xFFu);
        o.y = a2_byte_to_u8((v >> 8) & 0xFFu);
        o.z = a2_byte_to_u8((v >> 16) & 0xFFu);
        o.w = a2_byte_to_u8(v >> 24);
        *(uint4 *)dst = o;
    }
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

template <int BITS, int MR, int NC, bool AL16>
__global__ void __launch_bounds__(256) conv_mfma_kernel(ConvArgs a)
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
    int32_t *sWsum = (int32_t *)(smem + a.off_wsum);
    uint8_t *sX = smem + a.off_x;
    uint8_t *sOut = smem + a.off_out;

    // (1) K-chunk tables: chunk j = 16 consecutive K bytes.  sTab: offset of
    // the chunk in the input tile relative to a pixel's top-left tap; sNat:
    // offset in the natural (ky, kx, c) order of a filter bank; sVld: bytes of
    // the chunk that belong to the filter (the rest meets zero weights).
    for (int j = tid; j < kch; j += 256) {
        int hoff = 0, nat = 0, vld = 0;
        if (j < a.kchunks) {
            if (a.row_mode) {
                int ky = j / a.cpr, r = (j - ky * a.cpr) * 16;
                hoff = ky * a.hwd * a.ps + r;
                nat = ky * a.row_len + r;
                vld = min(16, a.row_len - r);
            } else {
                int cpt = a.c8 >> 4;
                int tap = j / cpt, c16 = j - tap * cpt;
                int ky = tap / a.kw, kx = tap - ky * a.kw;
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

    // (2) Filter tile -> int8 in chunk order (rows = output channels).
    const int ncol = kch * 4;
    for (int row = wv; row < MT; row += 4) {
        const int mg = m0 + row;
        const uint8_t *wr = a.w + (size_t)min(mg, a.m - 1) * a.wrow;
        for (int col = lane; col < ncol; col += 64) {
            const int j = col >> 2, d = col & 3;
            uint32_t val = 0;
            if (mg < a.m && 4 * d < sVld[j]) {
                const int e = sNat[j] + 4 * d;
                if (BITS == 8)
                    val = *(const uint32_t *)(wr + e);
                else if (BITS == 4)
                    val = w4_to_s8x16(*(const uint16_t *)(wr + (e >> 1)));
                else
                    val = w2_to_s8x64(wr[e >> 2]);
            }
            *(uint32_t *)(sW + row * a.kp + col * 4) = val;
        }
    }
    __syncthreads();
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
    }

    const int tile_px = a.ti * a.th * a.tw;
    const int g = lane >> 4, r16 = lane & 15;
    const int quad_b = a.quad16 ? 16 : 4;
    const int quad_u = quad_b * 8 / BITS;  // unpacked bytes per quad

    for (int tile = blockIdx.x; tile < a.ntiles; tile += gridDim.x) {
        const int tq = (int)fdiv((uint32_t)tile, a.div_tx);
        const int tx = tile - tq * a.tiles_x;
        const int tn = (int)fdiv((uint32_t)tq, a.div_ty);
        const int ty = tq - tn * a.tiles_y;
        const int n0 = tn * a.ti, oy0 = ty * a.th, ox0 = tx * a.tw;
        const int iy0 = oy0 * a.sh - a.ph, ix0 = ox0 * a.sw - a.pw;

        // (3) Input tile + halo -> LDS, unpacked to int8, one quad per thread step.
        const int totq = a.ti * a.hh * a.hwd * a.pbq;
        for (int idx = tid; idx < totq; idx += 256) {
            const int pix = (int)fdiv((uint32_t)idx, a.div_pbq);
            const int q = idx - pix * a.pbq;
            const int hrow = (int)fdiv((uint32_t)pix, a.div_hwd);
            const int hx = pix - hrow * a.hwd;
            const int tI = (int)fdiv((uint32_t)hrow, a.div_hh);
            const int hy = hrow - tI * a.hh;
            const int nn = n0 + tI, iy = iy0 + hy, ix = ix0 + hx;
            const bool in = nn < a.n && iy >= 0 && iy < a.h && ix >= 0 && ix < a.w_;
            const uint8_t *src = a.x + (((size_t)(in ? nn : 0) * a.h + (in ? iy : 0)) * a.w_ +
                                        (in ? ix : 0)) * a.pb + q * quad_b;
            uint8_t *dst = sX + pix * a.ps + q * quad_u;
            if (a.quad16) {
                uint4 v = in ? *(const uint4 *)src : make_uint4(0, 0, 0, 0);
                constexpr int U = 32 / BITS;  // unpacked bytes per packed word
                stage_word<BITS>(dst, v.x);
                stage_word<BITS>(dst + U, v.y);
                stage_word<BITS>(dst + 2 * U, v.z);
                stage_word<BITS>(dst + 3 * U, v.w);
            } else {
                uint32_t v = in ? *(const uint32_t *)src : 0u;
                stage_word<BITS>(dst, v);
            }
        }
        __syncthreads();

        // (4) Main loop: MR x NC MFMA tiles per 64-deep K step.
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
#pragma unroll 2
        for (int ks = 0; ks < a.ksteps; ++ks) {
            const int off = sTab[ks * 4 + g];
            v4i av[MR], bv[NC];
#pragma unroll
            for (int t = 0; t < MR; ++t)
                av[t] = *(const v4i *)(aRow + t * 16 * a.kp + ks * 64);
#pragma unroll
            for (int c = 0; c < NC; ++c) {
                const uint8_t *bp = sX + base[c] + off;
                if (AL16) {
                    bv[c] = *(const v4i *)bp;
                } else {
                    const int32_t *b4 = (const int32_t *)bp;
                    bv[c] = (v4i){b4[0], b4[1], b4[2], b4[3]};
                }
            }
#pragma unroll
            for (int t = 0; t < MR; ++t)
#pragma unroll
                for (int c = 0; c < NC; ++c)
                    acc[t][c] = __builtin_amdgcn_mfma_i32_16x16x64_i8(av[t], bv[c], acc[t][c], 0, 0, 0);
        }

        // (5) Epilogue.  Lane (r16, g) of tile (t, c) holds channels
        // t*16 + 4g + {0..3} of pixel c*16 + r16 of its wave.
#pragma unroll
        for (int c = 0; c < NC; ++c) {
            const int p = wv * 16 * NC + c * 16 + r16;
            int gpix = -1;
            if (p < tile_px) {
                const int tI = (int)fdiv((uint32_t)p, a.div_tile_px);
                const int rem = p - tI * a.th * a.tw;
                const int py = (int)fdiv((uint32_t)rem, a.div_tw);
                const int px = rem - py * a.tw;
                const int nn = n0 + tI, oy = oy0 + py, ox = ox0 + px;
                if (nn < a.n && oy < a.ho && ox < a.wo)
                    gpix = (nn * a.ho + oy) * a.wo + ox;
            }
#pragma unroll
            for (int t = 0; t < MR; ++t) {
                const int mb = t * 16 + 4 * g;
                uint32_t packed = 0;
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const int m = m0 + mb + i;
                    if (m >= a.m)
                        continue;
                    int64_t accv = acc[t][c][i];
                    if (BITS == 8)
                        accv += 128 * (int64_t)sWsum[mb + i];
                    else if (BITS == 4)
                        accv >>= 4;
                    else
                        accv >>= 6;
                    const int64_t v = accv + (a.bias ? (int64_t)a.bias[m] : 0);
                    if (a.epi == EPI_RAW32) {
                        if (gpix >= 0)
                            ((int32_t *)a.y)[(size_t)gpix * a.m + m] = (int32_t)(uint32_t)(uint64_t)v;
                    } else {
                        int s = a.shift[m];
                        s = s < 0 ? 0 : (s > 62 ? 62 : s);
                        int64_t r = round_shift(v * (int64_t)a.mult[m], s);
                        r = r < a.clip_lo ? a.clip_lo : (r > a.clip_hi ? a.clip_hi : r);
                        packed |= (uint32_t)r << (i * BITS);
                    }
                }
                if (a.epi != EPI_RAW32 && p < tile_px) {
                    uint8_t *o = sOut + p * a.ot_b + mb * BITS / 8;
                    if (BITS == 8)
                        *(uint32_t *)o = packed;
                    else if (BITS == 4)
                        *(uint16_t *)o = (uint16_t)packed;
                    else
                        *o = (uint8_t)packed;
                }
            }
        }
        __syncthreads();

        // (6) Coalesced copy of the packed output tile.
        if (a.epi != EPI_RAW32) {
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
                const int nn = n0 + tI, oy = oy0 + py, ox = ox0 + px;
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
            hipFuncSetAttribute((const void *)k, hipFuncAttributeMaxDynamicSharedMemorySize,    \
                                160 * 1024);                                                    \
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
