// INT-1 (binary) convolution by XNOR and population count (Sec. III-A,
// Eq. (5); Sec. IV-A "Binary Convolution Kernel").
//
// Each lane owns one output pixel.  General form (any filter volume): the
// lane walks its receptive field one packed 32-channel word at a time and,
// for 32 output channels at once, adds popcount(~(x ^ w)) to 32 counters.  The filter words are the
// same for every lane of a wave, so they are fetched by scalar loads and fed
// to v_xnor_b32 / v_bcnt_u32_b32 as scalar operands: two vector instructions
// per 32 binary MACs.  Padding taps hold bit 0 (value -1).  The +-1 dot
// product is 2 * popcount - K; the output bit of channel m is
// (dot + bias[m] >= thresh[m]), 32 channels packed per output word.
#include "qnn_internal.h"

namespace qnn {

template <int KB>
__global__ void __launch_bounds__(256) conv_xnor_kernel(const uint32_t *__restrict__ xg,
                                                        const uint32_t *__restrict__ wgl, XnorArgs a)
{
    const int p = blockIdx.x * 256 + threadIdx.x;
    const bool live = p < a.npix;
    const int pc = live ? p : a.npix - 1;
    const int q = (int)fdiv((uint32_t)pc, a.div_wo);
    const int ox = pc - q * a.wo;
    const int n = (int)fdiv((uint32_t)q, a.div_ho);
    const int oy = q - n * a.ho;
    const int ngroups = (a.m + 31) >> 5;

    for (int grp = 0; grp < ngroups; ++grp) {
        uint32_t pop[32];
#pragma unroll
        for (int i = 0; i < 32; ++i)
            pop[i] = 0;
        const uint32_t *wg = wgl + (size_t)grp * 32 * a.kd;
        const int nvalid = min(32, a.m - grp * 32);
        for (int ky = 0; ky < a.kh; ++ky) {
            const int iy = oy * a.sh - a.ph + ky;
            for (int kx = 0; kx < a.kw; ++kx) {
                const int ix = ox * a.sw - a.pw + kx;
                const bool in = iy >= 0 && iy < a.h && ix >= 0 && ix < a.w_;
                const uint32_t *xp = xg + ((size_t)(n * a.h + (in ? iy : 0)) * a.w_ + (in ? ix : 0)) * a.cd;
                const uint32_t *wt = wg + (size_t)(ky * a.kw + kx) * a.cd;
                for (int d0 = 0; d0 < a.cd; d0 += KB) {
                    uint32_t xv[KB];
#pragma unroll
                    for (int d = 0; d < KB; ++d)
                        xv[d] = in ? xp[d0 + d] : 0u;
                    if (nvalid == 32) {
#pragma unroll
                        for (int mm = 0; mm < 32; ++mm)
#pragma unroll
                            for (int d = 0; d < KB; ++d)
                                pop[mm] += __popc(~(xv[d] ^ wt[(size_t)mm * a.kd + d0 + d]));
                    } else {
#pragma unroll
                        for (int mm = 0; mm < 32; ++mm) {
                            if (mm < nvalid) {
#pragma unroll
                                for (int d = 0; d < KB; ++d)
                                    pop[mm] += __popc(~(xv[d] ^ wt[(size_t)mm * a.kd + d0 + d]));
                            }
                        }
                    }
                }
            }
        }
        if (!live)
            continue;
        if (a.epi == EPI_RAW32) {
            int32_t *yr = (int32_t *)a.y + (size_t)p * a.m + grp * 32;
            for (int mm = 0; mm < nvalid; ++mm) {
                int64_t dot = 2 * (int64_t)pop[mm] - a.kbits;
                int64_t v = dot + (a.bias ? a.bias[grp * 32 + mm] : 0);
                yr[mm] = (int32_t)(uint32_t)(uint64_t)v;
            }
        } else {
            uint32_t word = 0;
#pragma unroll
            for (int mm = 0; mm < 32; ++mm) {
                if (mm < nvalid) {
                    const int m = grp * 32 + mm;
                    int64_t dot = 2 * (int64_t)pop[mm] - a.kbits;
                    int64_t v = dot + (a.bias ? a.bias[m] : 0);
                    word |= (v >= a.thresh[m] ? 1u : 0u) << mm;
                }
            }
            uint8_t *yb = a.y + (size_t)p * a.ypb + grp * 4;
            const int nb = min(4, a.ypb - grp * 4);
            if (nb == 4 && (a.ypb & 3) == 0) {
                *(uint32_t *)yb = word;
            } else {
                for (int b = 0; b < nb; ++b)
                    yb[b] = (uint8_t)(word >> (8 * b));
            }
        }
    }
}

// Register-resident variant (filter volume KD words, a multiple of 8, known
// at compile time): a lane gathers its whole im2col column (zero bits for
// padding taps) once, then walks the output channels of its workgroup's
// channel group (the split over workgroups keeps several waves per SIMD to
// hide the scalar-load latency).  Channel m's KD filter words arrive by
// scalar loads in 8-word blocks that alternate between two register sets,
// one block ahead of their use.  The lane counts mismatching bits,
// popcount(x ^ w): with K taps of +-1 values, the dot product is
// K - 2 * mismatches, so no complement is needed (two vector instructions
// per 32 binary MACs, and with KD fixed no scalar bookkeeping per block).
template <int KD>
__global__ void __launch_bounds__(256) conv_xnor_res_kernel(const uint32_t *__restrict__ xg,
                                                            const uint32_t *__restrict__ wgl,
                                                            const int32_t *__restrict__ bias,
                                                            const int32_t *__restrict__ thresh,
                                                            XnorArgs a)
{
    // workgroup -> (channel group, pixel block), the group varying fastest:
    // consecutive workgroups go to different XCDs, so each XCD (and the
    // scalar caches of its compute units) sees the filters of few groups
    const int grp = (int)(blockIdx.x % (unsigned)a.ngroups);
    const int p = (int)(blockIdx.x / (unsigned)a.ngroups) * 256 + threadIdx.x;
    const bool live = p < a.npix;
    const int pc = live ? p : a.npix - 1;
    const int q = (int)fdiv((uint32_t)pc, a.div_wo);
    const int ox = pc - q * a.wo;
    const int n = (int)fdiv((uint32_t)q, a.div_ho);
    const int oy = q - n * a.ho;

    // the lane's im2col column: taps in (ky, kx) order, cd words each
    uint32_t xv[KD];
    if ((a.cd & 3) == 0) {
        // whole 16-byte quads: the tap position advances in wave-uniform steps
        int tap = 0, d = 0, ky = 0, kx = 0;
#pragma unroll
        for (int k = 0; k < KD; k += 4) {
            const int iy = oy * a.sh - a.ph + ky, ix = ox * a.sw - a.pw + kx;
            uint4 v = make_uint4(0, 0, 0, 0);
            if ((uint32_t)iy < (uint32_t)a.h && (uint32_t)ix < (uint32_t)a.w_)
                v = *(const uint4 *)(xg + ((size_t)(n * a.h + iy) * a.w_ + ix) * a.cd + d);
            xv[k] = v.x;
            xv[k + 1] = v.y;
            xv[k + 2] = v.z;
            xv[k + 3] = v.w;
            d += 4;
            if (d == a.cd) {
                d = 0;
                ++tap;
                if (++kx == a.kw) {
                    kx = 0;
                    ++ky;
                }
            }
        }
        (void)tap;
    } else {
#pragma unroll
        for (int k = 0; k < KD; ++k) {
            const int tap = (int)fdiv((uint32_t)k, a.div_cd);
            const int d = k - tap * a.cd;
            const int ky = (int)fdiv((uint32_t)tap, a.div_kw);
            const int kx = tap - ky * a.kw;
            const int iy = oy * a.sh - a.ph + ky, ix = ox * a.sw - a.pw + kx;
            xv[k] = 0u;
            if (iy >= 0 && iy < a.h && ix >= 0 && ix < a.w_)
                xv[k] = xg[((size_t)(n * a.h + iy) * a.w_ + ix) * a.cd + d];
        }
    }

    const int mb = grp * a.mgrp;
    const int me = min(a.m, mb + a.mgrp);
    int32_t b_cur = bias ? bias[mb] : 0;
    int32_t t_cur = a.epi == EPI_RAW32 ? 0 : thresh[mb];
    uint32_t word = 0;
    for (int m = mb; m < me; ++m) {
        // the next channel's bias and threshold are fetched now, used next
        const int mn = m + 1 < me ? m + 1 : m;
        const int32_t b_next = bias ? bias[mn] : 0;
        const int32_t t_next = a.epi == EPI_RAW32 ? 0 : thresh[mn];
        // Block b + 1 is requested after the first word of block b is used:
        // a wait for scalar loads covers every load in flight, so requesting
        // it earlier would make the wait for block b also wait for b + 1.
        // The scheduling barriers keep this order; the empty asm keeps the
        // accumulating popcounts from being regrouped into three-input adds.
        const uint4 *wr = (const uint4 *)(wgl + (size_t)m * KD);
        uint4 s0 = wr[0], s1 = wr[1], t0, t1;
        uint32_t mis = 0;
#pragma unroll
        for (int kb = 0; kb < KD; kb += 8) {
            const bool odd = (kb >> 3) & 1;
            const uint4 c0 = odd ? t0 : s0, c1 = odd ? t1 : s1;
            const uint32_t w8[8] = {c0.x, c0.y, c0.z, c0.w, c1.x, c1.y, c1.z, c1.w};
            mis = __popc(xv[kb] ^ w8[0]) + mis;
            __asm__("" : "+v"(mis));
            __builtin_amdgcn_sched_barrier(0);
            if (kb + 8 < KD) {
                if (odd) {
                    s0 = wr[(kb + 8) / 4];
                    s1 = wr[(kb + 8) / 4 + 1];
                } else {
                    t0 = wr[(kb + 8) / 4];
                    t1 = wr[(kb + 8) / 4 + 1];
                }
            }
            __builtin_amdgcn_sched_barrier(0);
#pragma unroll
            for (int i = 1; i < 8; ++i) {
                mis = __popc(xv[kb + i] ^ w8[i]) + mis;
                __asm__("" : "+v"(mis));
            }
            __builtin_amdgcn_sched_barrier(0);
        }
        const int64_t v = (int64_t)a.kbits - 2 * (int64_t)mis + b_cur;
        if (a.epi == EPI_RAW32) {
            if (live)
                ((int32_t *)a.y)[(size_t)p * a.m + m] = (int32_t)(uint32_t)(uint64_t)v;
        } else {
            word |= (v >= t_cur ? 1u : 0u) << (m & 31);
            if ((m & 31) == 31 || m == me - 1) {
                if (live) {
                    uint8_t *yb = a.y + (size_t)p * a.ypb + (m >> 5) * 4;
                    const int nb = min(4, a.ypb - (m >> 5) * 4);
                    if (nb == 4 && (a.ypb & 3) == 0) {
                        *(uint32_t *)yb = word;
                    } else {
                        for (int b = 0; b < nb; ++b)
                            yb[b] = (uint8_t)(word >> (8 * b));
                    }
                }
                word = 0;
            }
        }
        b_cur = b_next;
        t_cur = t_next;
    }
}

hipError_t launch_conv_xnor(const XnorArgs &a, hipStream_t s)
{
    dim3 grid((a.npix + 255) / 256);
    // channel groups of mgrp (a multiple of 32) along grid.y
    dim3 grid_res(grid.x * a.ngroups);
    if (a.kd % 8 == 0 && a.kd <= 128) {
        switch (a.kd / 8) {
#define QNN_XR(J_)                                                                                          \
        case J_:                                                                                            \
            hipLaunchKernelGGL(conv_xnor_res_kernel<8 * J_>, grid_res, dim3(256), 0, s, a.x, a.w, a.bias,  \
                               a.thresh, a);                                                                \
            break;
            QNN_XR(1) QNN_XR(2) QNN_XR(3) QNN_XR(4) QNN_XR(5) QNN_XR(6) QNN_XR(7) QNN_XR(8)
            QNN_XR(9) QNN_XR(10) QNN_XR(11) QNN_XR(12) QNN_XR(13) QNN_XR(14) QNN_XR(15) QNN_XR(16)
#undef QNN_XR
        }
    }
    if (a.kd % 8 == 0 && a.kd <= 128)
        return hipGetLastError();
    if (a.cd % 8 == 0)
        hipLaunchKernelGGL(conv_xnor_kernel<8>, grid, dim3(256), 0, s, a.x, a.w, a);
    else if (a.cd % 4 == 0)
        hipLaunchKernelGGL(conv_xnor_kernel<4>, grid, dim3(256), 0, s, a.x, a.w, a);
    else if (a.cd % 2 == 0)
        hipLaunchKernelGGL(conv_xnor_kernel<2>, grid, dim3(256), 0, s, a.x, a.w, a);
    else
        hipLaunchKernelGGL(conv_xnor_kernel<1>, grid, dim3(256), 0, s, a.x, a.w, a);
    return hipGetLastError();
}

}  // namespace qnn
