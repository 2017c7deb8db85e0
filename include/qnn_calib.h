/*
 * qnn_calib.h - measurement kernels of the quantized-convolution library.
 *
 * These entry points do none of the layer's arithmetic.  They measure, on the
 * device the library runs on, the denominators against which the layer's
 * throughput is reported: the int8 matrix-core rate (the dense contraction of
 * Sec. III-A Eq. (2) runs on v_mfma_i32_32x32x32_i8), the vector XNOR /
 * population-count rate of the binary kernel (Sec. III-A Eq. (5), Sec. IV-A),
 * the HBM copy bandwidth the memory-bound layers stream at, the shader clock
 * the kernels run at, and the cost of an empty launch.
 *
 * Conventions as in qnn.h: caller-owned device memory, 16-byte aligned device
 * pointers (QNN_ERR_ALIGN), asynchronous on `stream` (a hipStream_t; NULL =
 * the null stream), every argument check on the host before any device call,
 * a qnn_status for every error (QNN_ERR_DEVICE without a gfx950 device,
 * QNN_ERR_LAUNCH when the launch fails).
 */
#ifndef QNN_CALIB_H
#define QNN_CALIB_H

#include <stddef.h>
#include <stdint.h>

#include "qnn.h"

#ifdef __cplusplus
extern "C" {
#endif

/*
 * Matrix-core rate: `blocks` workgroups of 4 waves, each wave issuing
 * `iters` x 4 independent v_mfma_i32_32x32x32_i8 (32768 multiply-adds each;
 * MACs in all = blocks * 4 * iters * 4 * 32768).
 *   out_dev: int32 [blocks * 256], one reduction of the accumulators per lane
 *            (keeps the products live; contents unspecified).
 *   clk_dev: int64 [blocks * 2] or NULL: per workgroup, the shader-clock
 *            cycles (s_memtime) and the 100 MHz reference ticks
 *            (s_memrealtime) that wave 0 spent in the loop.
 * blocks in [1, 2^20], iters in [1, 2^24] (QNN_ERR_PARAM).
 */
qnn_status qnn_calib_mfma_i8(int32_t blocks, int32_t iters, int32_t *out_dev, int64_t *clk_dev,
                             void *stream);

/*
 * Vector XNOR/popcount rate in the binary kernel's form: per lane and
 * iteration, 8 words each through one v_xor_b32 with a wave-uniform operand
 * and one accumulating v_bcnt_u32_b32 (binary MACs in all = blocks * 256 *
 * iters * 8 * 32).  out_dev, clk_dev, limits as qnn_calib_mfma_i8.
 */
qnn_status qnn_calib_xnor(int32_t blocks, int32_t iters, int32_t *out_dev, int64_t *clk_dev,
                          void *stream);

/*
 * Device copy of `bytes` bytes (a multiple of 16, at most 2^40) from src_dev
 * to dst_dev with 16-byte loads and stores (the buffers must not overlap):
 * the HBM bandwidth a streaming kernel reaches (bytes read + bytes written
 * per second), and the known traffic that scales the memory counters.
 */
qnn_status qnn_calib_copy(const void *src_dev, void *dst_dev, size_t bytes, void *stream);

/* An empty kernel of `blocks` workgroups of 256 threads (blocks in
 * [1, 2^20]): the launch floor under which no kernel's duration falls. */
qnn_status qnn_calib_empty(int32_t blocks, void *stream);

#ifdef __cplusplus
}
#endif

#endif /* QNN_CALIB_H */
