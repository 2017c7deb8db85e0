/*
 * qnn.h - C ABI of the MI355X (gfx950) quantized-convolution library.
 *
 * The library implements the hot path of PULP-NN (Garofalo et al., "PULP-NN:
 * Accelerating Quantized Neural Networks on Parallel Ultra-Low-Power RISC-V
 * Processors"): the convolution layer over INT-8, INT-4, INT-2 and INT-1 data
 * with a wide integer accumulator and a per-output-channel compression back to
 * the layer's bit-width, plus the fully connected, max-pooling and ReLU
 * helpers of the same library.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * Layout.  Activations are NHWC ("Height-Width-Channel", Sec. III-B): channel
 *   stride 1, then width, then height, then image.  Weights of a convolution
 *   are M x kh x kw x C (one filter bank per output channel, Sec. III-B,
 *   Eq. (6)), each bank's codes contiguous in (ky, kx, c) order.
 * Packing (Sec. IV-A, "Sub-byte Extensions").  A b-bit tensor stores 8/b
 *   codes per byte; the lower channel sits in the less significant bits.  One
 *   pixel occupies ceil(C*b/8) bytes ("pixel bytes"); convolution, pooling
 *   and linear inputs require pixel bytes to be a multiple of 4 (pad C with
 *   zero channels and zero weights, which leaves every result unchanged).
 *   One exception: a convolution also takes 2-byte pixels of 4 channels at
 *   4 bits (a network's first layer: 3 image channels and a zero channel)
 *   when the whole-image kernel covers it (see QNN_TILE_IMAGE: stride 1,
 *   3x3 or 5x5 filters, output rows of at most 32 pixels), else
 *   QNN_ERR_ALIGN.
 * Values.  Activations are unsigned codes (0 .. 2^b - 1) for b = 8, 4, 2;
 *   weights are two's complement codes (-2^(b-1) .. 2^(b-1) - 1).  At b = 1
 *   both operands hold +1 (bit 1) or -1 (bit 0) (Sec. III-A, Eq. (5)).
 *   Padding taps of a convolution hold code 0 (value 0, or -1 at one bit).
 * Accumulation (Sec. III-A, Eq. (2); Sec. III-B, Eq. (6)).  acc[n,oy,ox,m] =
 *   sum over ky < kh, kx < kw, c < C of X[n, oy*sh - ph + ky, ox*sw - pw + kx, c]
 *   * W[m, ky, kx, c] (cross-correlation), exact.  Output size per axis is
 *   floor((in + 2*pad - k) / stride) + 1.
 * Epilogues (Sec. III-A compression; Sec. IV-A binary kernel):
 *   QNN_EPI_REQUANT (b = 8, 4, 2; output b bits):
 *     y = clip(floor(((acc + bias[m]) * mult[m]) / 2^shift[m] + 1/2), lo, hi),
 *     computed without overflow; needs 0 <= lo <= hi <= 2^b - 1 and
 *     shift[m] in [0, 62] (out-of-range shifts give unspecified codes; they
 *     never fault).
 *   QNN_EPI_THRESH1 (b = 1; output 1 bit): y = (acc + bias[m] >= thresh[m]).
 *   QNN_EPI_STAIR (b = 4, 2; output b bits; Sec. III-A, Eq. (4)): thresh
 *     holds T = 2^b - 1 thresholds per channel, channel-major
 *     (thresh[m*T + p - 1] = tau_p); y is the level p of the interval
 *     [tau_p, tau_{p+1}) that holds acc + bias[m] (tau_0 = -inf,
 *     tau_{2^b} = +inf), compared exactly in 64 bits.  For thresholds that
 *     are not non-decreasing, y is the number of thresholds at or below
 *     acc + bias[m] (the same level whenever they are sorted).
 *   QNN_EPI_RAW32 (any b; output int32 per channel): y = acc + bias[m],
 *     reduced modulo 2^32.
 *   bias may be NULL (zero).
 * Limits.  The filter volume K = kh*kw*C must satisfy K*max|x|*max|w| < 2^31
 *   for the kernels' 32-bit accumulators: K <= 65793 at 8 bits, 1118481 at
 *   4 bits, 5592405 at 2 bits, 2^31 - 1 at 1 bit (QNN_ERR_OVERFLOW).  The
 *   8/4/2-bit convolution stages one filter tile (16 output channels x K) and
 *   one input tile in the 160 KB local memory of a compute unit; shapes that
 *   cannot fit return QNN_ERR_UNSUPPORTED.
 * Memory and streams.  Every device pointer is caller-owned device memory and
 *   must be 16-byte aligned (QNN_ERR_ALIGN).  The library allocates no device
 *   memory and keeps no state besides a per-device capability check.  Work is
 *   enqueued asynchronously on `stream` (a hipStream_t; NULL = the null
 *   stream); outputs are valid once the stream has reached that point.
 * Errors.  Every function returns a qnn_status and never aborts.  All argument
 *   checks run on the host before any device call; a failed check launches
 *   nothing.  N = 0 is valid and launches nothing.
 */
#ifndef QNN_H
#define QNN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define QNN_ABI_VERSION 8

typedef enum {
    QNN_OK = 0,
    QNN_ERR_NULL = 1,        /* a required pointer is NULL */
    QNN_ERR_BITS = 2,        /* unsupported or mismatched bit-width */
    QNN_ERR_SHAPE = 3,       /* negative/zero size, empty output, output descriptor mismatch */
    QNN_ERR_PARAM = 4,       /* stride/pad/window/epilogue parameter out of range */
    QNN_ERR_ALIGN = 5,       /* pixel bytes not a multiple of 4, or device pointer not 16-B aligned */
    QNN_ERR_OVERFLOW = 6,    /* the 32-bit accumulator could overflow (K too large) */
    QNN_ERR_UNSUPPORTED = 7, /* shape beyond the kernels' local-memory limits */
    QNN_ERR_DEVICE = 8,      /* no usable gfx950 device is current */
    QNN_ERR_LAUNCH = 9       /* the kernel launch failed */
} qnn_status;

typedef enum {
    QNN_EPI_REQUANT = 0,
    QNN_EPI_THRESH1 = 1,
    QNN_EPI_RAW32 = 2,
    QNN_EPI_STAIR = 3
} qnn_epilogue;

/* An NHWC tensor: n images of h x w pixels with c channels of `bits` bits
 * (bits = 32 means int32 elements, used by QNN_EPI_RAW32 outputs). */
typedef struct {
    int32_t n, h, w, c, bits;
} qnn_tensor;

/* Convolution geometry: kernel size, strides (>= 1) and zero-code padding (>= 0). */
typedef struct {
    int32_t kh, kw, stride_h, stride_w, pad_h, pad_w;
} qnn_conv_geom;

/* Epilogue parameters.  Arrays are device pointers of M entries. */
typedef struct {
    int32_t kind;            /* a qnn_epilogue value */
    const int32_t *bias;     /* [M] or NULL */
    const int32_t *mult;     /* [M], QNN_EPI_REQUANT */
    const int8_t *shift;     /* [M], QNN_EPI_REQUANT, each in [0, 62] */
    const int32_t *thresh;   /* [M] (QNN_EPI_THRESH1) or [M][2^b - 1] (QNN_EPI_STAIR) */
    int32_t clip_lo, clip_hi;/* QNN_EPI_REQUANT output range */
} qnn_epi;

/* qnn_tile.kernel values. */
#define QNN_TILE_MFMA16 16 /* v_mfma_i32_16x16x64_i8 */
#define QNN_TILE_MFMA32 32 /* v_mfma_i32_32x32x32_i8 */
/* INT-2 and INT-1 layers: v_mfma_scale_f32_32x32x64_f8f6f4 on FP4 (e2m1)
 * operands.  Every INT-2 code is an exact e2m1 value (activations x as x/2,
 * weights w as w/2, products rescaled by a block exponent of 2), so is every
 * INT-1 value (+1, -1), and every partial sum is an integer below 2^24, so
 * the fp32 accumulator and hence the output equal the integer paths' bit for
 * bit, at twice the int8 matrix-core rate per instruction.  INT-1 layers take
 * QNN_EPI_THRESH1 or QNN_EPI_RAW32 as on the XNOR path.  The library never
 * picks this path by itself. */
#define QNN_TILE_FP4 4
/* Small images, a workgroup keeping whole padded images in local memory and
 * its filters in registers: stride 1, 3x3 or 5x5 filters, output rows of at
 * most 32 pixels, images of at most 8 KB, QNN_EPI_REQUANT (also fused with
 * max-pooling) or QNN_EPI_RAW32, M*bits a multiple of 32, and input pixels
 * of 4 packed bytes (a network's first layer: e.g. 3 image channels padded
 * to 4 at 8 bits), of 2 packed bytes (4 channels at 4 bits), or of 16 / 32
 * packed bytes (32 channels at 4 / 8 bits, 64
 * at 2 / 4 bits) with at most 28 K steps of 32 (5x5 filters: 32 channels at
 * 8 or 4 bits).  The library picks it by itself for every layer that
 * qualifies; tile_m = tile_n = waves = 0.  A layer that does not qualify
 * gives QNN_ERR_UNSUPPORTED. */
#define QNN_TILE_IMAGE 1

/* Tile shape of the matrix-core convolution kernels, for exploration and
 * tuning (the library otherwise picks it per layer). */
typedef struct {
    int32_t kernel;  /* a QNN_TILE_* value */
    int32_t tile_m;  /* MFMA tiles per wave along output channels: 1, 2, 4 (4 at MFMA32: 8 bits only;
                        FP4: 1, 2, or 0 with tile_n = waves = 0 to let the library pick) */
    int32_t tile_n;  /* MFMA tiles per wave along output pixels: 1, 2, 4 (MFMA32, FP4: 1, 2) */
    int32_t waves;   /* waves per workgroup: 4; or 8 at MFMA32 / FP4 for scale-and-clamp and raw
                        layers whose filter taps are whole 16-byte chunks of the staged pixel
                        (channels a multiple of 16; 32 at FP4), tile_m and tile_n <= 2, when each
                        workgroup gets a single tile */
} qnn_tile;

/* Library ABI version (QNN_ABI_VERSION). */
int32_t qnn_abi_version(void);

/* Static description of a status code (a qnn_status value; any other value
 * gives "unknown status"); never NULL. */
const char *qnn_status_string(int32_t status);

/* Checks that the current HIP device is a gfx950 GPU.  Called implicitly by
 * every device entry point; QNN_ERR_DEVICE when no such device is current. */
qnn_status qnn_device_check(void);

/* Bytes of one pixel of `t` (ceil(c*bits/8), or 4*c at bits = 32). */
size_t qnn_pixel_bytes(const qnn_tensor *t);

/* Bytes of the whole tensor `t` (n*h*w pixel bytes); 0 if t is NULL. */
size_t qnn_tensor_bytes(const qnn_tensor *t);

/* Output descriptor of a convolution of `x` with M filters of geometry `g`
 * and epilogue `kind` (Sec. III-B, Eq. (6)).  Host only. */
qnn_status qnn_conv2d_out_shape(const qnn_tensor *x, int32_t m, const qnn_conv_geom *g,
                                int32_t kind, qnn_tensor *y);

/*
 * Quantized convolution layer (Sec. III-A Eq. (2); Sec. III-B Eq. (6);
 * Sec. IV-A INT-8 / sub-byte / binary kernels).
 *   x, x_dev: input descriptor and packed NHWC device data (bits 8, 4, 2, 1).
 *   m, w_dev: number of filters and packed M x kh x kw x C weights at the
 *             same bit-width as the input.
 *   g:        geometry; e: epilogue (REQUANT at 8/4/2 bits, STAIR at 4/2 bits,
 *             THRESH1 at 1 bit, RAW32 at any).
 *   y, y_dev: output descriptor (must equal qnn_conv2d_out_shape) and device
 *             buffer of qnn_tensor_bytes(y) bytes; must not overlap the inputs.
 */
qnn_status qnn_conv2d(const qnn_tensor *x, const void *x_dev, int32_t m, const void *w_dev,
                      const qnn_conv_geom *g, const qnn_epi *e, const qnn_tensor *y, void *y_dev,
                      void *stream);

/*
 * Fully connected layer (Sec. IV-A: a convolution whose filter covers the
 * whole input, so no im2col is needed): y[n, j] = sum_i X[n, i] * W[j, i]
 * over the K = h*w*c elements of image n in NHWC order, then the epilogue.
 *   x: input descriptor (pixel bytes a multiple of 4); w_dev: M x K packed
 *   weights; y: descriptor {n, 1, 1, m, out_bits}.
 */
qnn_status qnn_linear(const qnn_tensor *x, const void *x_dev, int32_t m, const void *w_dev,
                      const qnn_epi *e, const qnn_tensor *y, void *y_dev, void *stream);

/*
 * qnn_conv2d with a caller-chosen tile shape (the MI355X counterpart of the
 * paper's study of register-blocked kernel sizes, Sec. IV-C / Fig. 9) or
 * matrix instruction (QNN_TILE_FP4: the sub-byte SIMD the paper's outlook in
 * Sec. VI asks for, on MI355X's FP4 matrix cores): identical results,
 * different speed.  8-, 4- and 2-bit inputs (QNN_TILE_FP4: 2- and 1-bit only,
 * else QNN_ERR_BITS; filter volume kh*kw*C above 2796202 at 2 bits or 2^24
 * at 1 bit QNN_ERR_OVERFLOW; other tiles at 1 bit: QNN_ERR_PARAM);
 * shapes that are not built return QNN_ERR_PARAM, tiles that do not fit the
 * local memory (or a single-tile eight-wave plan that the device cannot
 * hold) QNN_ERR_UNSUPPORTED.
 */
qnn_status qnn_conv2d_tiled(const qnn_tensor *x, const void *x_dev, int32_t m, const void *w_dev,
                            const qnn_conv_geom *g, const qnn_epi *e, const qnn_tile *tile,
                            const qnn_tensor *y, void *y_dev, void *stream);

/*
 * Convolution fused with the 2x2 / stride-2 max-pooling that follows it in
 * the paper's network (Sec. IV-A pooling kernel): y = maxpool_2x2/2 of the
 * codes qnn_conv2d would produce, floor output size, in one pass (the
 * convolution's output never reaches memory).
 *   e:      QNN_EPI_REQUANT (8/4/2 bits) or QNN_EPI_STAIR (4/2 bits); other
 *           epilogues give QNN_ERR_PARAM.
 *   pool_k, pool_s: pooling window and stride; only 2 and 2 are defined
 *           (QNN_ERR_PARAM otherwise).
 *   y:      {n, floor(Ho/2), floor(Wo/2), m, bits}, Ho x Wo being the
 *           convolution output size (each at least 2, else QNN_ERR_SHAPE).
 * Everything else (layouts, limits, errors, streams) as qnn_conv2d.
 */
qnn_status qnn_conv2d_maxpool(const qnn_tensor *x, const void *x_dev, int32_t m, const void *w_dev,
                              const qnn_conv_geom *g, const qnn_epi *e, int32_t pool_k,
                              int32_t pool_s, const qnn_tensor *y, void *y_dev, void *stream);

/*
 * Max-pooling on unsigned codes (Sec. IV-A): window kh x kw, strides sh, sw,
 * no padding, floor output size.  bits 8, 4 or 2; y = {n, ho, wo, c, bits}.
 */
qnn_status qnn_maxpool2d(const qnn_tensor *x, const void *x_dev, int32_t kh, int32_t kw,
                         int32_t sh, int32_t sw, const qnn_tensor *y, void *y_dev, void *stream);

/* ReLU on `count` signed 8-bit values (Sec. IV-A): y = max(x, 0); y_dev may
 * equal x_dev (in place). */
qnn_status qnn_relu_s8(const void *x_dev, void *y_dev, size_t count, void *stream);

/* Host helpers: pack `count` unsigned codes (one per byte, each < 2^bits)
 * into the packed format (ceil(count*bits/8) bytes, zero tail bits), and the
 * inverse, producing values (two's complement if is_signed; +-1 at bits = 1). */
qnn_status qnn_pack_host(const uint8_t *codes, size_t count, int32_t bits, uint8_t *out);
qnn_status qnn_unpack_host(const uint8_t *packed, size_t count, int32_t bits, int32_t is_signed,
                           int32_t *out);

#ifdef __cplusplus
}
#endif

#endif /* QNN_H */
