// Internal declarations shared by the host dispatcher and the gfx950 kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace qnn {

// Division by a run-time constant: q = (umulhi(n, mul) + n) >> shr, exact for
// 0 <= n < 2^31 (round-up magic number; d = 1 gives mul = 1, shr = 0).
struct FastDiv {
    uint32_t d, mul, shr;
};

inline FastDiv make_fastdiv(uint32_t d)
{
    FastDiv f;
    f.d = d;
    uint32_t l = 0;
    while ((1ull << l) < d)
        ++l;
    f.shr = l;
    f.mul = (uint32_t)((((1ull << l) - d) << 32) / d + 1);
    return f;
}

__device__ __forceinline__ uint32_t fdiv(uint32_t n, const FastDiv &f)
{
    return (__umulhi(n, f.mul) + n) >> f.shr;
}

enum { EPI_REQUANT = 0, EPI_THRESH1 = 1, EPI_RAW32 = 2, EPI_STAIR = 3 };

// Arguments of the int8-MFMA implicit-GEMM convolution (8/4/2-bit inputs).
// GEMM view: rows = output channels (A = weights), columns = output pixels
// (B = im2col of the input tile held in local memory), K = kh*kw*C.
struct ConvArgs {
    const uint8_t *x;      // packed NHWC input
    const uint8_t *w;      // packed OHWI weights
    uint8_t *y;            // packed NHWC output (codes) or int32 [pix][M]
    const int32_t *bias, *mult;
    const int8_t *shift;
    const int32_t *thresh; // staircase thresholds [M][2^bits - 1]
    int32_t n, h, w_, pb;  // input size, packed bytes per pixel
    int32_t c8;            // bytes of a staged pixel: channels (int8), or channels / 2 (e2m1)
    int32_t m, kh, kw, sh, sw, ph, pw, ho, wo;
    int32_t wrow;          // packed bytes per filter bank
    int32_t epi, clip_lo, clip_hi, ypb;  // ypb: output bytes per pixel
    // tiling of the output: tile = ti images x th rows x tw columns
    int32_t ti, th, tw, tiles_x, tiles_y, ntiles;
    int32_t hh, hwd, ps;   // halo rows / columns, local-memory pixel stride
    int32_t kchunks, ksteps, kp;  // 16-byte K chunks, MFMA K steps, weight row stride in LDS
    int32_t kch;           // chunks including the padding to whole K steps
    int32_t ot_b;          // packed output bytes per pixel of a channel tile
    int32_t cs;            // 32x32 kernel: bytes per pixel of the one-byte-per-code output staging
    int32_t alias_out;     // 32x32 kernel: the output staging reuses the input tile's local memory
    int32_t off_tab, off_wsum, off_x, off_out, lds_bytes;
    int32_t row_mode, row_len, cpr;  // K walk per filter row when C*1B is not a multiple of 16
    FastDiv div_pbq;       // packed 16-byte (or 4-byte) quads per pixel
    FastDiv div_hwd;       // halo columns
    FastDiv div_hh;        // halo rows
    FastDiv div_tile_px;   // th*tw
    FastDiv div_tw;
    FastDiv div_tx, div_ty;   // tiles_x, tiles_y
    FastDiv div_obq;       // output quads per pixel in the copy-out
    FastDiv div_qrow;      // packed 16-byte quads per filter bank
    FastDiv div_ncol;      // 4-byte words per staged filter row
    FastDiv div_tab_a;     // K-chunk table: chunks per filter row (row walk) or per tap
    FastDiv div_tab_kw;    // K-chunk table: filter columns
    int32_t pbq, quad16;   // quads per pixel, 1 if the quad is 16 bytes else 4 bytes
    int32_t ob0, obn, obq, oquad16;  // copy-out byte offset, byte count, quads, quad size flag
    int32_t contig;        // tile = consecutive output pixels with every channel: flat copy-out
    // fused 2x2 / stride-2 max-pooling of the codes (32x32 kernel): pooled
    // output size, and divisors of a tile's pooled pixel grid
    int32_t pool, hp, wp;
    FastDiv div_ptile;     // (th/2)*(tw/2) pooled pixels per image of a tile
    FastDiv div_ptw;       // tw/2
    int32_t wunpack;       // 32x32 kernel: 4-/2-bit filters staged unpacked to int8
};

// Arguments of the whole-image convolution (conv_img_kernel): small images
// (input pixels of 4, 16 or 32 packed bytes, output rows of at most 32
// pixels), stride 1; a workgroup walks groups of whole images, one
// 32-channel group per grid row.
struct ImgArgs {
    const uint8_t *x;      // packed NHWC input
    const uint8_t *w;      // packed OHWI weights
    uint8_t *y;            // packed NHWC codes (pooled or not) or int32 [pix][M]
    const int32_t *bias, *mult;
    const int8_t *shift;
    int32_t n, h, w_, m, ph, pw, ho, wo;
    int32_t epi, clip_lo, clip_hi, ypb;
    int32_t pool, hp, wp;
    int32_t tile_bytes;    // LDS bytes of one padded, unpacked image tile
    int32_t ipw;           // images per workgroup step
    int32_t ngroups;       // ceil(n / ipw)
    int32_t pairs;         // pairs of 32-pixel MFMA row tiles per image
    int32_t quads;         // 1: an image step is loaded as 16-byte quads
    FastDiv div_w;         // input width
    FastDiv div_pairs;     // pairs
    FastDiv div_imgq;      // 16-byte quads per image
    // row bands (images too large for one tile): a step is one band of brows
    // output rows of one image; its tile holds trows = brows + kh - 1 input
    // rows (rows outside the image as pads) and div_imgq counts the tile's
    // quads.  bands = 0 in whole-image mode.
    int32_t bands, brows, trows;
    FastDiv div_bands;
    const int32_t *thresh; // staircase thresholds [M][2^bits - 1] (EPI_STAIR)
};

// Arguments of the INT-1 XNOR/popcount convolution.
struct XnorArgs {
    const uint32_t *x;     // packed NHWC bits, cd dwords per pixel
    const uint32_t *w;     // packed M x kh x kw x C bits, kd dwords per bank
    uint8_t *y;
    const int32_t *bias, *thresh;
    int32_t n, h, w_, cd;
    int32_t m, kh, kw, sh, sw, ph, pw, ho, wo;
    int32_t kd, kbits, epi, ypb;
    int32_t npix;
    int32_t mgrp;          // output channels per workgroup (multiple of 32), register-resident kernel
    int32_t ngroups;       // channel groups (ceil(m / mgrp))
    FastDiv div_wo, div_ho, div_cd, div_kw;
};

struct PoolArgs {
    const uint8_t *x;
    uint8_t *y;
    int32_t n, h, w_, pbd;     // pbd: dwords per pixel
    int32_t kh, kw, sh, sw, ho, wo;
    int32_t total;             // output dwords
    FastDiv div_pbd, div_wo, div_ho;
};

hipError_t launch_conv_mfma_b8(const ConvArgs &a, int mr, int nc, int al16, dim3 grid, hipStream_t s);
hipError_t launch_conv_mfma_b4(const ConvArgs &a, int mr, int nc, int al16, dim3 grid, hipStream_t s);
hipError_t launch_conv_mfma_b2(const ConvArgs &a, int mr, int nc, int al16, dim3 grid, hipStream_t s);
hipError_t launch_conv_m32_b8(const ConvArgs &a, int wm, int wn, int al16, int nw, dim3 grid, hipStream_t s);
hipError_t launch_conv_m32_b4(const ConvArgs &a, int wm, int wn, int al16, int nw, dim3 grid, hipStream_t s);
hipError_t launch_conv_m32_b2(const ConvArgs &a, int wm, int wn, int al16, int nw, dim3 grid, hipStream_t s);
// INT-2 and INT-1 through the e2m1 (FP4) matrix instruction
hipError_t launch_conv_m32_f4(const ConvArgs &a, int wm, int wn, int al16, int nw, dim3 grid, hipStream_t s);
hipError_t launch_conv_m32_f4b1(const ConvArgs &a, int wm, int wn, int al16, int nw, dim3 grid, hipStream_t s);
hipError_t launch_conv_xnor(const XnorArgs &a, hipStream_t s);
// whole-image kernel; hipErrorInvalidValue for a shape with no built
// instance; the grid fills the cus compute units with resident workgroups
hipError_t launch_conv_img_p4(const ImgArgs &a, int bits, int k, int cus, hipStream_t s);
hipError_t launch_conv_img_p2(const ImgArgs &a, int bits, int k, int cus, hipStream_t s);
hipError_t launch_conv_img_p16(const ImgArgs &a, int bits, int k, int wop, int cus, hipStream_t s);
hipError_t launch_conv_img_p32(const ImgArgs &a, int bits, int k, int wop, int cus, hipStream_t s);
// fully connected layer with raw outputs: K a multiple of 64 (linear.hip)
hipError_t launch_linear_raw(const uint8_t *x, const uint8_t *w, const int32_t *bias, int32_t *y, int32_t n,
                             int32_t m, int32_t k, int bits, hipStream_t s);
hipError_t launch_maxpool(const PoolArgs &a, int bits, hipStream_t s);
hipError_t launch_relu_s8(const uint8_t *x, uint8_t *y, size_t count, hipStream_t s);

}  // namespace qnn
