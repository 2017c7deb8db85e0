// Fully connected layer with raw int32 outputs (Sec. IV-A: a convolution
// whose filter covers the whole input; the network's classifier, Sec. V-E):
// y[n][j] = sum_k X[n][k] * W[j][k] + bias[j] over the K = h*w*c codes of
// image n in NHWC order.  The layer is a thin GEMM (few output channels, a
// long K) bound by reading X once, so it gets its own kernel instead of the
// convolution tiles, whose 64-pixel tiles leave most compute units idle:
//   * a workgroup owns 16 images and 16 output channels (grid.y over
//     channel groups); its four waves split K four ways and each issues
//     v_mfma_i32_16x16x64_i8 (rows = images, columns = channels) on
//     fragments loaded straight from memory into registers (no LDS
//     staging: every byte of X is used once);
//   * 8-bit codes are offset by -128 (x ^ 0x80) and 128 * sum_k W[j][k] is
//     added back; 4-/2-bit codes are unpacked in registers, weights as
//     16*w / 64*w and the accumulator shifted back (both exact);
//   * the four partial accumulators (and filter sums) are added through LDS.
#include "conv_mfma_impl.h"

namespace qnn {

// 16 K values of one row from its packed bytes at p, as int8 (activations:
// unsigned codes, 8-bit ones offset by -128; weights: two's complement,
// sub-byte ones scaled by 16 / 64), in the sub-byte K order of the
// convolution kernels (field-major within each packed word).
template <int BITS, bool WEIGHT>
__device__ __forceinline__ v4i lin_frag(const uint8_t *p, bool live)
{
    uint32_t d[4] = {0, 0, 0, 0};
    if (BITS == 8) {
        if (live) {
            const uint4 v = *(const uint4 *)p;
            d[0] = v.x;
            d[1] = v.y;
            d[2] = v.z;
            d[3] = v.w;
        }
        if (!WEIGHT) {
#pragma unroll
            for (int i = 0; i < 4; ++i)
                d[i] ^= 0x80808080u;
        }
    } else if (BITS == 4) {
        uint2 v = make_uint2(0, 0);
        if (live)
            v = *(const uint2 *)p;
        const uint2 a = WEIGHT ? w4_word(v.x) : make_uint2(v.x & 0x0F0F0F0Fu, (v.x >> 4) & 0x0F0F0F0Fu);
        const uint2 b = WEIGHT ? w4_word(v.y) : make_uint2(v.y & 0x0F0F0F0Fu, (v.y >> 4) & 0x0F0F0F0Fu);
        d[0] = a.x;
        d[1] = a.y;
        d[2] = b.x;
        d[3] = b.y;
    } else {
        const uint32_t v = live ? *(const uint32_t *)p : 0u;
        const uint4 a = WEIGHT ? w2_word(v)
                               : make_uint4(v & 0x03030303u, (v >> 2) & 0x03030303u, (v >> 4) & 0x03030303u,
                                            (v >> 6) & 0x03030303u);
        d[0] = a.x;
        d[1] = a.y;
        d[2] = a.z;
        d[3] = a.w;
    }
    return (v4i){(int32_t)d[0], (int32_t)d[1], (int32_t)d[2], (int32_t)d[3]};
}

template <int BITS>
__global__ void __launch_bounds__(256) linear_raw_kernel(const uint8_t *__restrict__ x,
                                                         const uint8_t *__restrict__ w,
                                                         const int32_t *__restrict__ bias, int32_t *__restrict__ y,
                                                         int32_t n, int32_t m, int32_t kb, int32_t ksteps)
{
    __shared__ int32_t sAcc[4][64][4];
    __shared__ int32_t sSum[4][64];
    constexpr int SL = BITS == 4 ? 4 : (BITS == 2 ? 6 : 0);  // log2 of the weight scale
    constexpr int FB = 16 * BITS / 8;                          // packed bytes of a 16-value fragment
    const int tid = threadIdx.x, lane = tid & 63;
    const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int r16 = lane & 15, kq = lane >> 4;
    const int img = blockIdx.x * 16 + r16;   // A row of this lane
    const int ch = blockIdx.y * 16 + r16;    // B column of this lane
    const bool xin = img < n, win = ch < m;
    const uint8_t *xr = x + (size_t)(xin ? img : 0) * kb + kq * FB;
    const uint8_t *wr = w + (size_t)(win ? ch : 0) * kb + kq * FB;
    v4i acc = {0, 0, 0, 0};
    int wsum = 0;
    // wave wv takes K steps wv, wv + 4, ...: 64 values each, 16 per lane
    // group; four of its steps at a time have all their loads issued before
    // their products (one memory round trip per four steps)
    auto step = [&](const v4i &a, const v4i &b) {
        if (BITS == 8) {
#pragma unroll
            for (int i = 0; i < 4; ++i)
                wsum = __builtin_amdgcn_sdot4((int)b[i], 0x01010101, wsum, false);
        }
        acc = __builtin_amdgcn_mfma_i32_16x16x64_i8(a, b, acc, 0, 0, 0);
    };
    int s = wv;
    for (; s + 12 < ksteps; s += 16) {
        v4i fa[4], fb[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            fa[u] = lin_frag<BITS, false>(xr + (size_t)(s + 4 * u) * 4 * FB, xin);
            fb[u] = lin_frag<BITS, true>(wr + (size_t)(s + 4 * u) * 4 * FB, win);
        }
#pragma unroll
        for (int u = 0; u < 4; ++u)
            step(fa[u], fb[u]);
    }
    for (; s < ksteps; s += 4)
        step(lin_frag<BITS, false>(xr + (size_t)s * 4 * FB, xin), lin_frag<BITS, true>(wr + (size_t)s * 4 * FB, win));
    // lane l holds channel l%16 for images 4*(l/16) + i
#pragma unroll
    for (int i = 0; i < 4; ++i)
        sAcc[wv][lane][i] = acc[i];
    sSum[wv][lane] = wsum;
    __syncthreads();
    if (wv != 0)
        return;
    int64_t bt = 0;
    if (BITS == 8) {
        // the channel's filter sum: its four lane groups in each of the four waves
        int s = 0;
#pragma unroll
        for (int q = 0; q < 4; ++q)
#pragma unroll
            for (int g = 0; g < 4; ++g)
                s += sSum[q][g * 16 + r16];
        bt = 128 * (int64_t)s;
    }
    if (bias && win)
        bt += bias[ch];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int32_t v = sAcc[0][lane][i] + sAcc[1][lane][i] + sAcc[2][lane][i] + sAcc[3][lane][i];
        const int im = blockIdx.x * 16 + 4 * kq + i;
        if (win && im < n)
            y[(size_t)im * m + ch] = (int32_t)(uint32_t)(uint64_t)((int64_t)(v >> SL) + bt);
    }
}

hipError_t launch_linear_raw(const uint8_t *x, const uint8_t *w, const int32_t *bias, int32_t *y, int32_t n,
                             int32_t m, int32_t k, int bits, hipStream_t s)
{
    const int32_t kb = (int32_t)((int64_t)k * bits / 8);
    const int32_t ksteps = k / 64;
    dim3 grid((unsigned)((n + 15) / 16), (unsigned)((m + 15) / 16));
    if (bits == 8)
        hipLaunchKernelGGL(linear_raw_kernel<8>, grid, dim3(256), 0, s, x, w, bias, y, n, m, kb, ksteps);
    else if (bits == 4)
        hipLaunchKernelGGL(linear_raw_kernel<4>, grid, dim3(256), 0, s, x, w, bias, y, n, m, kb, ksteps);
    else if (bits == 2)
        hipLaunchKernelGGL(linear_raw_kernel<2>, grid, dim3(256), 0, s, x, w, bias, y, n, m, kb, ksteps);
    else
        return hipErrorInvalidValue;
    return hipGetLastError();
}

}  // namespace qnn
