// Max-pooling over packed unsigned codes and signed 8-bit ReLU (Sec. IV-A:
// ReLU is a max with zero, max-pooling the maximum over a window; both split
// over pixels across the parallel units, Sec. IV-B).
//
// Pooling works on one packed 32-bit word (32/b channels) per lane.  The word
// is split into 16/b pairs of b-bit fields that sit in the two 16-bit halves
// of a register, and the maximum over the window is taken with packed 16-bit
// unsigned max, so no field ever needs sign handling or per-byte extraction.
#include "qnn_internal.h"

namespace qnn {

typedef unsigned short u16x2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ u16x2 as_u16x2(uint32_t v)
{
    return __builtin_bit_cast(u16x2, v);
}

template <int BITS>
__global__ void __launch_bounds__(256) maxpool_kernel(PoolArgs a)
{
    constexpr int S = 16 / BITS;                   // field pairs per word
    constexpr uint32_t FM = (1u << BITS) - 1u;
    constexpr uint32_t MASK = FM | (FM << 16);     // one field in each half
    const int idx = blockIdx.x * 256 + threadIdx.x;
    if (idx >= a.total)
        return;
    const int pix = (int)fdiv((uint32_t)idx, a.div_pbd);
    const int d = idx - pix * a.pbd;
    const int q = (int)fdiv((uint32_t)pix, a.div_wo);
    const int ox = pix - q * a.wo;
    const int n = (int)fdiv((uint32_t)q, a.div_ho);
    const int oy = q - n * a.ho;
    const uint32_t *x = (const uint32_t *)a.x;
    u16x2 best[S];
#pragma unroll
    for (int s = 0; s < S; ++s)
        best[s] = (u16x2){0, 0};
    for (int ky = 0; ky < a.kh; ++ky) {
        const int iy = oy * a.sh + ky;
        for (int kx = 0; kx < a.kw; ++kx) {
            const int ix = ox * a.sw + kx;
            const uint32_t v = x[(((size_t)n * a.h + iy) * a.w_ + ix) * a.pbd + d];
#pragma unroll
            for (int s = 0; s < S; ++s)
                best[s] = __builtin_elementwise_max(best[s], as_u16x2((v >> (s * BITS)) & MASK));
        }
    }
    uint32_t out = 0;
#pragma unroll
    for (int s = 0; s < S; ++s)
        out |= __builtin_bit_cast(uint32_t, best[s]) << (s * BITS);
    ((uint32_t *)a.y)[idx] = out;
}

hipError_t launch_maxpool(const PoolArgs &a, int bits, hipStream_t s)
{
    dim3 grid((a.total + 255) / 256);
    if (bits == 8)
        hipLaunchKernelGGL(maxpool_kernel<8>, grid, dim3(256), 0, s, a);
    else if (bits == 4)
        hipLaunchKernelGGL(maxpool_kernel<4>, grid, dim3(256), 0, s, a);
    else if (bits == 2)
        hipLaunchKernelGGL(maxpool_kernel<2>, grid, dim3(256), 0, s, a);
    else
        return hipErrorInvalidValue;
    return hipGetLastError();
}

// y = max(x, 0) on signed bytes, four per word: a byte is negative when its
// top bit is set; (neg << 8) - neg turns each such top bit into a 0xFF byte
// mask without carries between bytes.
__global__ void __launch_bounds__(256) relu_s8_kernel(const uint8_t *x, uint8_t *y, size_t count)
{
    const size_t words = count / 4;
    const size_t i = (size_t)blockIdx.x * 256 + threadIdx.x;
    if (i < words) {
        const uint32_t v = ((const uint32_t *)x)[i];
        const uint32_t neg = (v >> 7) & 0x01010101u;
        const uint32_t mask = (neg << 8) - neg;
        ((uint32_t *)y)[i] = v & ~mask;
    } else if (i < words + (count & 3)) {
        const size_t b = words * 4 + (i - words);
        const int8_t v = (int8_t)x[b];
        y[b] = (uint8_t)(v > 0 ? v : 0);
    }
}

hipError_t launch_relu_s8(const uint8_t *x, uint8_t *y, size_t count, hipStream_t s)
{
    const size_t items = count / 4 + (count & 3);
    dim3 grid((unsigned)((items + 255) / 256));
    hipLaunchKernelGGL(relu_s8_kernel, grid, dim3(256), 0, s, x, y, count);
    return hipGetLastError();
}

}  // namespace qnn
