// Measurement kernels (include/qnn_calib.h): the matrix-core, vector
// XNOR/popcount and copy rates of the device, the shader clock and the empty
// launch, measured beside the layer so that its throughput is reported
// against what this device sustains as well as against the published peaks.
#include "qnn.h"
#include "qnn_calib.h"
#include "qnn_internal.h"

namespace {

typedef int32_t c4i __attribute__((ext_vector_type(4)));
typedef int32_t c16i __attribute__((ext_vector_type(16)));

constexpr int32_t kMaxBlocks = 1 << 20;
constexpr int32_t kMaxIters = 1 << 24;

// Wave 0's shader-clock cycles and reference ticks over the timed loop.
__device__ __forceinline__ void store_clock(int64_t *clk, uint64_t t0, uint64_t r0)
{
    const uint64_t t1 = __builtin_amdgcn_s_memtime();
    const uint64_t r1 = __builtin_amdgcn_s_memrealtime();
    if (clk && threadIdx.x == 0) {
        clk[2 * blockIdx.x] = (int64_t)(t1 - t0);
        clk[2 * blockIdx.x + 1] = (int64_t)(r1 - r0);
    }
}

// Four independent accumulator chains per wave (the 32x32x32 instruction's
// latency is covered by the other chains and the other waves of the SIMD).
__global__ void __launch_bounds__(256) calib_mfma_kernel(int iters, int32_t *out, int64_t *clk)
{
    const int tid = threadIdx.x;
    const c4i a = {tid, tid * 3 + 1, tid ^ 0x55, tid + 7};
    const c4i b = {tid * 5, tid + 1, tid ^ 0x33, 0x01010101};
    c16i c0 = {}, c1 = {}, c2 = {}, c3 = {};
    const uint64_t t0 = __builtin_amdgcn_s_memtime();
    const uint64_t r0 = __builtin_amdgcn_s_memrealtime();
    for (int i = 0; i < iters; ++i) {
        c0 = __builtin_amdgcn_mfma_i32_32x32x32_i8(a, b, c0, 0, 0, 0);
        c1 = __builtin_amdgcn_mfma_i32_32x32x32_i8(b, a, c1, 0, 0, 0);
        c2 = __builtin_amdgcn_mfma_i32_32x32x32_i8(a, a, c2, 0, 0, 0);
        c3 = __builtin_amdgcn_mfma_i32_32x32x32_i8(b, b, c3, 0, 0, 0);
    }
    int32_t s = 0;
#pragma unroll
    for (int v = 0; v < 16; ++v)
        s += c0[v] ^ c1[v] ^ c2[v] ^ c3[v];
    store_clock(clk, t0, r0);
    out[(size_t)blockIdx.x * 256 + tid] = s;
}

struct Words8 {
    uint32_t w[8];
};

// The binary kernel's inner step: one xor with a wave-uniform word (a kernel
// argument, hence a scalar operand) and one accumulating popcount per word.
// The empty asm statements make every word look rewritten each iteration,
// so neither instruction is hoisted out of the loop, and keep the counts
// from being regrouped into three-input adds.
__global__ void __launch_bounds__(256) calib_xnor_kernel(int iters, Words8 w, int32_t *out, int64_t *clk)
{
    const uint32_t tid = threadIdx.x + blockIdx.x * 256u;
    uint32_t x[8];
#pragma unroll
    for (int j = 0; j < 8; ++j)
        x[j] = tid * (2654435761u + 2u * j) ^ (0x9E3779B9u >> j);
    // two running counts, so consecutive popcounts do not depend on each other
    uint32_t acc[2] = {0, 0};
    const uint64_t t0 = __builtin_amdgcn_s_memtime();
    const uint64_t r0 = __builtin_amdgcn_s_memrealtime();
    for (int i = 0; i < iters; ++i) {
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            __asm__ volatile("" : "+v"(x[j]));
            acc[j & 1] = __popc(x[j] ^ w.w[j]) + acc[j & 1];
            __asm__ volatile("" : "+v"(acc[j & 1]));
        }
    }
    store_clock(clk, t0, r0);
    out[tid] = (int32_t)(acc[0] + acc[1]);
}

// Grid-stride copy, four 16-byte quads in flight per thread.
__global__ void __launch_bounds__(256) calib_copy_kernel(const uint4 *__restrict__ src, uint4 *__restrict__ dst,
                                                         size_t quads)
{
    const size_t stride = (size_t)gridDim.x * 256;
    size_t i = (size_t)blockIdx.x * 256 + threadIdx.x;
    for (; i + 3 * stride < quads; i += 4 * stride) {
        const uint4 v0 = src[i], v1 = src[i + stride], v2 = src[i + 2 * stride], v3 = src[i + 3 * stride];
        dst[i] = v0;
        dst[i + stride] = v1;
        dst[i + 2 * stride] = v2;
        dst[i + 3 * stride] = v3;
    }
    for (; i < quads; i += stride)
        dst[i] = src[i];
}

__global__ void __launch_bounds__(256) calib_empty_kernel() {}

bool aligned16(const void *p) { return ((uintptr_t)p & 15u) == 0; }

qnn_status launched() { return hipGetLastError() == hipSuccess ? QNN_OK : QNN_ERR_LAUNCH; }

qnn_status check_loop(int32_t blocks, int32_t iters, const int32_t *out, const int64_t *clk)
{
    if (!out)
        return QNN_ERR_NULL;
    if (blocks < 1 || blocks > kMaxBlocks || iters < 1 || iters > kMaxIters)
        return QNN_ERR_PARAM;
    if (!aligned16(out) || (clk && !aligned16(clk)))
        return QNN_ERR_ALIGN;
    return QNN_OK;
}

}  // namespace

extern "C" {

qnn_status qnn_calib_mfma_i8(int32_t blocks, int32_t iters, int32_t *out_dev, int64_t *clk_dev, void *stream)
{
    qnn_status st = check_loop(blocks, iters, out_dev, clk_dev);
    if (st != QNN_OK)
        return st;
    if ((st = qnn_device_check()) != QNN_OK)
        return st;
    hipLaunchKernelGGL(calib_mfma_kernel, dim3(blocks), dim3(256), 0, (hipStream_t)stream, iters, out_dev,
                       clk_dev);
    return launched();
}

qnn_status qnn_calib_xnor(int32_t blocks, int32_t iters, int32_t *out_dev, int64_t *clk_dev, void *stream)
{
    qnn_status st = check_loop(blocks, iters, out_dev, clk_dev);
    if (st != QNN_OK)
        return st;
    if ((st = qnn_device_check()) != QNN_OK)
        return st;
    Words8 w;
    for (int j = 0; j < 8; ++j)
        w.w[j] = 0x6A09E667u * (uint32_t)(j + 1);
    hipLaunchKernelGGL(calib_xnor_kernel, dim3(blocks), dim3(256), 0, (hipStream_t)stream, iters, w, out_dev,
                       clk_dev);
    return launched();
}

qnn_status qnn_calib_copy(const void *src_dev, void *dst_dev, size_t bytes, void *stream)
{
    if (!src_dev || !dst_dev)
        return QNN_ERR_NULL;
    if (bytes % 16 != 0 || !aligned16(src_dev) || !aligned16(dst_dev))
        return QNN_ERR_ALIGN;
    if (bytes > ((size_t)1 << 40))
        return QNN_ERR_SHAPE;
    const uintptr_t s = (uintptr_t)src_dev, d = (uintptr_t)dst_dev;
    if (bytes && s < d + bytes && d < s + bytes)
        return QNN_ERR_PARAM;
    qnn_status st = qnn_device_check();
    if (st != QNN_OK)
        return st;
    if (bytes == 0)
        return QNN_OK;
    int dev = 0, cus = 256;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus < 1)
        cus = 256;
    const size_t quads = bytes / 16;
    size_t grid = (size_t)cus * 8;
    if (grid > (quads + 255) / 256)
        grid = (quads + 255) / 256;
    hipLaunchKernelGGL(calib_copy_kernel, dim3((unsigned)grid), dim3(256), 0, (hipStream_t)stream,
                       (const uint4 *)src_dev, (uint4 *)dst_dev, quads);
    return launched();
}

qnn_status qnn_calib_empty(int32_t blocks, void *stream)
{
    if (blocks < 1 || blocks > kMaxBlocks)
        return QNN_ERR_PARAM;
    qnn_status st = qnn_device_check();
    if (st != QNN_OK)
        return st;
    hipLaunchKernelGGL(calib_empty_kernel, dim3(blocks), dim3(256), 0, (hipStream_t)stream);
    return launched();
}

}  // extern "C"
