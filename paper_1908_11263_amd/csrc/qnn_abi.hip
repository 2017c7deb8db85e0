// C ABI of the quantized-convolution library: argument validation (entirely
// on the host, before any device call), tile planning and kernel dispatch.
#include <mutex>
#include <string.h>

#include "qnn.h"
#include "qnn_internal.h"

using namespace qnn;

namespace {

constexpr int kMaxDevices = 64;
constexpr int kLdsBytes = 160 * 1024;
constexpr int kPlanCus = 256;  // compute units of an MI355X; the grid uses the queried count

struct DeviceInfo {
    int checked = 0;  // 0 unknown, 1 ok, -1 not usable
    int cus = 0;
};

std::mutex g_mu;
DeviceInfo g_dev[kMaxDevices];

qnn_status device_info(int *cus)
{
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices)
        return QNN_ERR_DEVICE;
    std::lock_guard<std::mutex> lock(g_mu);
    DeviceInfo &d = g_dev[dev];
    if (d.checked == 0) {
        hipDeviceProp_t prop;
        if (hipGetDeviceProperties(&prop, dev) != hipSuccess) {
            d.checked = -1;
        } else {
            d.checked = strncmp(prop.gcnArchName, "gfx950", 6) == 0 ? 1 : -1;
            d.cus = prop.multiProcessorCount;
        }
    }
    if (d.checked != 1)
        return QNN_ERR_DEVICE;
    if (cus)
        *cus = d.cus;
    return QNN_OK;
}

bool valid_bits(int b) { return b == 1 || b == 2 || b == 4 || b == 8; }

int64_t pixel_bytes64(const qnn_tensor *t)
{
    if (t->bits == 32)
        return 4 * (int64_t)t->c;
    return ((int64_t)t->c * t->bits + 7) / 8;
}

bool aligned16(const void *p) { return ((uintptr_t)p & 15u) == 0; }

int32_t out_dim(int32_t in, int32_t k, int32_t s, int32_t p)
{
    int64_t span = (int64_t)in + 2 * (int64_t)p - k;
    if (span < 0)
        return 0;
    return (int32_t)(span / s + 1);
}

int out_bits_for(int32_t kind, int32_t in_bits)
{
    if (kind == QNN_EPI_REQUANT || kind == QNN_EPI_STAIR)
        return in_bits;
    if (kind == QNN_EPI_THRESH1)
        return 1;
    return 32;
}

int64_t max_k_for(int bits)
{
    // K * max|x'| * max|w'| < 2^31 on the accumulator the kernels keep, and
    // K * max|x| * max|w| < 2^31 for the true accumulator.
    switch (bits) {
    case 8: return 65793;     // 255 * 128 * K < 2^31 (true); 128 * 128 * K < 2^31 (offset form)
    case 4: return 1118481;   // 15 * 128 * K < 2^31 (weights staged as 16 * w)
    case 2: return 5592405;   // 3 * 128 * K < 2^31 (weights staged as 64 * w)
    default: return 2147483647;
    }
}

qnn_status check_tensor(const qnn_tensor *t)
{
    if (t->n < 0 || t->h < 1 || t->w < 1 || t->c < 1)
        return QNN_ERR_SHAPE;
    if ((int64_t)t->n * t->h * t->w * pixel_bytes64(t) > ((int64_t)1 << 40))
        return QNN_ERR_SHAPE;
    return QNN_OK;
}

qnn_status check_epi(const qnn_epi *e, int bits, int32_t m)
{
    (void)m;
    switch (e->kind) {
    case QNN_EPI_REQUANT:
        if (bits == 1)
            return QNN_ERR_BITS;
        if (!e->mult || !e->shift)
            return QNN_ERR_NULL;
        if (e->clip_lo < 0 || e->clip_lo > e->clip_hi || e->clip_hi > (1 << bits) - 1)
            return QNN_ERR_PARAM;
        break;
    case QNN_EPI_THRESH1:
        if (bits != 1)
            return QNN_ERR_BITS;
        if (!e->thresh)
            return QNN_ERR_NULL;
        break;
    case QNN_EPI_STAIR:
        if (bits != 4 && bits != 2)
            return QNN_ERR_BITS;
        if (!e->thresh)
            return QNN_ERR_NULL;
        break;
    case QNN_EPI_RAW32:
        break;
    default:
        return QNN_ERR_PARAM;
    }
    return QNN_OK;
}

// Fits an output tile of PT pixels and MT channels: fills the tile geometry,
// LDS offsets and tile counts of `c`; returns the LDS bytes, or -1.
int64_t fit_tile(ConvArgs &c, int MT, int PT, int bits, int obits, int64_t w_bytes, int64_t tab_bytes,
                 bool code_staging, bool alias = false)
{
    int ti, th, tw;
    if (c.pool && (int64_t)c.ho * c.wo >= PT) {
        // pooled tiles hold whole 2x2 windows: an even width (or the whole
        // row) and an even height (or the rest of the image), at least two rows
        ti = 1;
        tw = c.wo <= PT / 2 ? c.wo : PT / 2;
        th = PT / tw;
        if (th > c.ho)
            th = c.ho;
        if (th < c.ho && (th & 1))
            th -= 1;
    } else if ((int64_t)c.ho * c.wo >= PT) {
        ti = 1;
        tw = c.wo < PT ? c.wo : PT;
        th = PT / tw;
        if (th > c.ho)
            th = c.ho;
    } else {
        ti = PT / (c.ho * c.wo);
        if (ti > c.n)
            ti = c.n > 0 ? c.n : 1;
        th = c.ho;
        tw = c.wo;
    }
    const int hh = (th - 1) * c.sh + c.kh;
    const int hwd = (tw - 1) * c.sw + c.kw;
    const int64_t x_bytes = (int64_t)ti * hh * hwd * c.ps + 64;
    const int ot_b = obits == 32 ? 0 : MT * bits / 8;
    // output staging: the packed tile, or one byte per code with a pixel
    // stride of MT + 16 (the two pixel groups a wave writes at once, 4 pixels
    // apart, then fall in different LDS banks)
    const int cs = obits == 32 ? 0 : (code_staging ? MT + 16 : ot_b);
    const int64_t o_bytes = (int64_t)PT * cs;
    int64_t off = w_bytes;
    off = (off + 15) & ~(int64_t)15;
    const int64_t off_tab = off;
    off += tab_bytes;
    off = (off + 15) & ~(int64_t)15;
    const int64_t off_wsum = off;
    off += 4 * MT + 32 + 64 * MT;   // filter sums, votes, per-channel plans or staircase thresholds
    off = (off + 15) & ~(int64_t)15;
    const int64_t off_x = off;
    off += (x_bytes + 15) & ~(int64_t)15;
    // the output staging either follows the input tile or, when asked for
    // and small enough, reuses it (the kernel then separates the two uses
    // with barriers)
    const bool share = alias && o_bytes <= x_bytes;
    if (alias && !share)
        return -1;
    const int64_t off_out = share ? off_x : off;
    if (!share)
        off += o_bytes;
    if (off > kLdsBytes)
        return -1;
    c.ti = ti;
    c.th = th;
    c.tw = tw;
    c.hh = hh;
    c.hwd = hwd;
    c.ot_b = ot_b;
    c.cs = cs;
    c.alias_out = share ? 1 : 0;
    c.off_tab = (int32_t)off_tab;
    c.off_wsum = (int32_t)off_wsum;
    c.off_x = (int32_t)off_x;
    c.off_out = (int32_t)off_out;
    c.lds_bytes = (int32_t)off;
    c.tiles_x = (c.wo + tw - 1) / tw;
    c.tiles_y = (c.ho + th - 1) / th;
    const int64_t tiles_n = (c.n + ti - 1) / ti;
    const int64_t nt = tiles_n * c.tiles_y * c.tiles_x;
    if (nt > (int64_t)1 << 30)
        return -1;
    c.ntiles = (int32_t)nt;
    return off;
}

// K walk common to both kernels: 16-byte K chunks, tap by tap when a pixel
// is a whole number of chunks, else along each filter row.
void plan_k_walk(ConvArgs &a, int &al16)
{
    const int c8 = a.c8;
    a.row_mode = (c8 % 16) != 0;
    if (a.row_mode) {
        a.row_len = a.kw * c8;
        a.cpr = (a.row_len + 15) / 16;
        a.kchunks = a.kh * a.cpr;
        a.ps = c8;
    } else {
        a.row_len = 0;
        a.cpr = 0;
        a.kchunks = a.kh * a.kw * (c8 / 16);
        // keep the pixel stride an odd multiple of 16 bytes, so 16 lanes
        // reading 16 neighbouring pixels hit 16 different bank groups
        a.ps = ((c8 / 16) % 2 == 0) ? c8 + 16 : c8;
    }
    al16 = a.row_mode ? 0 : 1;
}

// 16x16x64 kernel: candidates in order of preference (widest channel tile,
// then widest pixel tile); the first that fits the local memory and gives at
// least two tiles per compute unit, else the one with the most tiles (small
// layers are latency-bound and want parallelism).
qnn_status plan_conv_mfma(ConvArgs &a, int bits, int &mr, int &nc, int &al16,
                          const qnn_tile *force = nullptr)
{
    plan_k_walk(a, al16);
    a.ksteps = (a.kchunks + 3) / 4;
    a.kch = 4 * a.ksteps;
    a.kp = a.ksteps * 64 + 16;
    const int obits = a.epi == EPI_RAW32 ? 32 : bits;
    const int64_t tab_bytes = 3 * 4 * (int64_t)a.kch;
    if (force) {
        ConvArgs c = a;
        if (fit_tile(c, 16 * force->tile_m, 64 * force->tile_n, bits, obits,
                     (int64_t)16 * force->tile_m * a.kp, tab_bytes, false) < 0)
            return QNN_ERR_UNSUPPORTED;
        a = c;
        mr = force->tile_m;
        nc = force->tile_n;
        return QNN_OK;
    }
    const int mr_first = a.m <= 16 ? 1 : (a.m <= 32 ? 2 : 4);
    ConvArgs best = a;
    int best_mr = 0, best_nc = 0;
    int64_t best_units = -1;
    for (int cmr = mr_first; cmr >= 1; cmr >>= 1) {
        for (int cnc = 4; cnc >= 1; cnc >>= 1) {
            if (cmr * cnc > 8)
                continue;  // 64 x 256 tiles exceed the register budget of two workgroups per CU
            ConvArgs c = a;
            if (fit_tile(c, 16 * cmr, 64 * cnc, bits, obits, (int64_t)16 * cmr * a.kp, tab_bytes, false) < 0)
                continue;
            const int64_t units = (int64_t)c.ntiles * ((c.m + 16 * cmr - 1) / (16 * cmr));
            if (units >= 2 * kPlanCus) {
                a = c;
                mr = cmr;
                nc = cnc;
                return QNN_OK;
            }
            if (units > best_units) {
                best = c;
                best_units = units;
                best_mr = cmr;
                best_nc = cnc;
            }
        }
    }
    if (best_units < 0)
        return QNN_ERR_UNSUPPORTED;
    a = best;
    mr = best_mr;
    nc = best_nc;
    return QNN_OK;
}

// 32x32x32 kernel with packed filters in LDS: used when the layer has at
// least 32 output channels and enough tiles for two per compute unit; the
// preferred tile keeps two workgroups per compute unit in the local memory.
// f4: INT-2 layer on the e2m1 instruction (filter rows staged as 16 bytes of
// nibbles per 32-deep K chunk, like an 8-bit layer of half the channels).
qnn_status plan_conv_m32(ConvArgs &a, int bits, int &wm, int &wn, int &al16, int &nw,
                         bool allow_nw8 = true, const qnn_tile *force = nullptr, bool f4 = false, int cus = 0)
{
    nw = 4;
    // fused pooling runs on this kernel whatever the layer's width, and so
    // does the e2m1 path (chosen by the caller)
    if (a.m < 32 && !a.pool && !force && !f4)
        return QNN_ERR_UNSUPPORTED;
    ConvArgs b = a;
    plan_k_walk(b, al16);
    // measured per layer: the 32x32 kernel wins every layer except 8-bit ones
    // with a K walk along filter rows (pixels of less than 16 bytes)
    if (bits == 8 && b.row_mode && !a.pool && !force)
        return QNN_ERR_UNSUPPORTED;
    b.ksteps = 2 * ((b.kchunks + 3) / 4);  // an even number of 32-deep steps
    b.kch = 2 * b.ksteps;
    // 4-bit filters walked tap by tap are staged unpacked to int8: the main
    // loop then spends no vector instructions expanding them, for twice the
    // filter bytes in LDS (measured faster at 4 bits; at 2 bits the fourfold
    // filter bytes cost more than the expansion)
    const bool unpack = !f4 && bits == 4 && al16;
    b.wunpack = unpack ? 1 : 0;
    const int cb = (f4 || unpack) ? 16 : 2 * bits;  // LDS bytes of a filter row per 16-byte K chunk
    b.kp = (b.kch + 1) * cb;         // odd multiple of cb: conflict-free fragment reads
    const int obits = b.epi == EPI_RAW32 ? 32 : bits;
    const int64_t tab_bytes = 3 * 4 * (int64_t)b.kch;
    if (force) {
        const int MT = 32 * force->tile_m;
        if (force->waves == 8 && (!al16 || a.pool || a.epi == EPI_STAIR))
            return QNN_ERR_PARAM;
        ConvArgs c = b;
        const int PT = 32 * force->tile_n * force->waves;
        int64_t lds = fit_tile(c, MT, PT, bits, obits, (int64_t)MT * b.kp, tab_bytes, true);
        if (lds < 0 || lds > kLdsBytes) {
            c = b;
            lds = fit_tile(c, MT, PT, bits, obits, (int64_t)MT * b.kp, tab_bytes, true, true);
        }
        if (lds < 0 || lds > kLdsBytes)
            return QNN_ERR_UNSUPPORTED;
        a = c;
        wm = force->tile_m;
        wn = force->tile_n;
        nw = force->waves;
        return QNN_OK;
    }
    static const int cand[5][2] = {{4, 1}, {2, 2}, {2, 1}, {1, 2}, {1, 1}};
    // the e2m1 path: eight-wave tiles first, whenever one fits the local
    // memory, one workgroup per compute unit walking its channel group's
    // tiles.  Its staged filter rows are 2x / 4x the packed ones (INT-2 /
    // INT-1), so sharing them between more pixels pays most here (INT-1
    // batch-1024 layer: 2x1 eight-wave tiles 33.6 us with one tile per
    // workgroup, 25.5 us walking four, against 51.0 us for the 1x1 four-wave
    // tile the general rule below picks), as long as the tiles give every
    // compute unit a workgroup (INT-2 batch-64 32x32x64 layer: 2x2 tiles
    // leave half the device idle, 9.07 us against 7.2 us for 2x1)
    if (f4 && allow_nw8 && !a.pool && a.epi != EPI_STAIR && al16) {
        for (int i = 1; i < 5; ++i) {
            const int cwm = cand[i][0], cwn = cand[i][1];
            const int MT = 32 * cwm;
            if ((MT > 32 && MT - 32 >= b.m) || MT > ((b.m + 31) / 32) * 32)
                continue;
            ConvArgs c8 = b;
            const int64_t lds8 = fit_tile(c8, MT, 256 * cwn, bits, obits, (int64_t)MT * b.kp, tab_bytes, true);
            if (lds8 < 0 || lds8 > kLdsBytes)
                continue;
            if (i < 4 && (int64_t)c8.ntiles * ((b.m + MT - 1) / MT) < cus)
                continue;
            a = c8;
            wm = cwm;
            wn = cwn;
            nw = 8;
            return QNN_OK;
        }
    }
    // pass 2 (pooled layers and the e2m1 path, which have no other kernel to
    // fall back on): any tile that fits, even with few tiles
    const bool last_resort = a.pool || f4;
    for (int pass = 0; pass < (last_resort ? 3 : 2); ++pass) {
        const int64_t lds_cap = pass == 0 ? kLdsBytes / 2 : kLdsBytes;
        for (int i = 0; i < 5; ++i) {
            const int cwm = cand[i][0], cwn = cand[i][1];
            if (cwm == 4 && bits != 8)
                continue;  // not instantiated: exceeds the register budget
            const int MT = 32 * cwm;
            if (MT > 32 && MT - 32 >= b.m)
                continue;  // at least one full 32-channel row tile per extra tile row
            if (MT > ((b.m + 31) / 32) * 32)
                continue;
            ConvArgs c = b;
            int64_t lds = fit_tile(c, MT, 128 * cwn, bits, obits, (int64_t)MT * b.kp, tab_bytes, true);
            if (lds < 0 || lds > lds_cap) {
                c = b;
                lds = fit_tile(c, MT, 128 * cwn, bits, obits, (int64_t)MT * b.kp, tab_bytes, true, true);
            }
            if (lds < 0 || lds > lds_cap)
                continue;
            const int64_t units = (int64_t)c.ntiles * ((c.m + MT - 1) / MT);
            if (units < 2 * kPlanCus && !(last_resort && pass == 2))
                continue;
            a = c;
            wm = cwm;
            wn = cwn;
            // eight waves per workgroup, twice the pixels: for plain layers
            // whose four-wave plan gives every workgroup a single tile (the
            // prologue -- filter tile, plans, tables -- is then shared by
            // twice the work); instantiated for wave tiles of up to 2x2
            // MFMA tiles with 16-byte aligned fragments
            if (allow_nw8 && !a.pool && a.epi != EPI_STAIR && wm <= 2 && al16 &&
                units <= 2 * kPlanCus) {
                ConvArgs c8 = b;
                const int64_t lds8 = fit_tile(c8, MT, 256 * cwn, bits, obits, (int64_t)MT * b.kp, tab_bytes, true);
                if (lds8 >= 0 && lds8 <= kLdsBytes) {
                    a = c8;
                    nw = 8;
                }
            }
            return QNN_OK;
        }
    }
    return QNN_ERR_UNSUPPORTED;
}

// Whole-image kernel (conv_img_kernel): stride 1, 3x3 or 5x5 filters, output
// rows of at most 32 pixels, scale-and-clamp or (4 and 2 bits) staircase
// outputs (pooled or not) or raw outputs,
// channel groups that fill whole output words, and pixels of
//   * 4 packed bytes (8, 4 or 2 bits: a network's first layer), or
//   * 16 / 32 packed bytes whose unpacked pixel is a whole number of 32-byte
//     chunks, with at most 28 K steps (filters held in registers);
// a group of whole images per workgroup step (prefetched in at most 8 KB,
// the tiles in at most 64 KB of LDS), or, for larger images of 32-byte
// pixels and rows of 17 to 32 outputs, one band of 8 output rows per step
// (its kh + 7 input rows prefetched in at most 12 KB).  Fills everything but
// the pointers and ypb; false when the layer does not qualify.
bool plan_img(ImgArgs &p, const qnn_tensor *x, int32_t m, const qnn_conv_geom *g, const qnn_epi *e,
              int32_t ho, int32_t wo, bool pool, int &pbytes, int &wop)
{
    const int bits = x->bits;
    if (bits != 8 && bits != 4 && bits != 2)
        return false;
    const int64_t pb = pixel_bytes64(x);
    if (g->stride_h != 1 || g->stride_w != 1)
        return false;
    if (!(g->kh == g->kw && (g->kh == 3 || g->kh == 5)))
        return false;
    if (!(e->kind == QNN_EPI_REQUANT || (e->kind == QNN_EPI_RAW32 && !pool) ||
          (e->kind == QNN_EPI_STAIR && bits != 8)))
        return false;
    if (((int64_t)m * bits) % 32 != 0 || wo > 32)
        return false;
    const int64_t u = pb * 8 / bits;  // unpacked bytes per pixel
    const int taps = g->kh * g->kw;
    if (pb == 4 || (pb == 2 && bits == 4)) {
        wop = 32;
    } else if (pb == 16 || pb == 32) {
        if (u < 32 || taps * (u / 32) > 28)
            return false;
        // built: 16-byte pixels at 4 and 2 bits, 32-byte pixels at 8 and 4
        // bits, 5x5 filters only with a single chunk per tap
        if ((pb == 16 && bits == 8) || (pb == 32 && bits == 2))
            return false;
        wop = wo <= 8 ? 8 : (wo <= 16 ? 16 : 32);
    } else {
        return false;
    }
    pbytes = (int)pb;
    const int64_t npix = (int64_t)x->h * x->w;
    const int64_t img_bytes = npix * pb;
    // tile slot bytes (8-bit one-word pixels: a pair; wide pixels: padded by
    // 16 bytes, an odd number of 16-byte units, against bank conflicts)
    const int sb = u == 4 ? 8 : (u >= 32 ? (int)u + 16 : (int)u);
    const int pp = wop + g->kw - 1;           // tile pitch, slots
    const int rt = 32 / wop;                  // image rows per MFMA row tile
    if (img_bytes > 8192) {
        // row bands: built for 32-byte pixels with 32-pixel row tiles
        if (!(pb == 32 && wop == 32))
            return false;
        const int brows = 2 * rt * 4;         // a pair of row tiles per wave
        const int trows = brows + g->kh - 1;
        const int64_t bands = (ho + brows - 1) / brows;
        if ((int64_t)trows * x->w * pb > 3 * 256 * 16 || (int64_t)x->n * bands > INT32_MAX)
            return false;
        memset(&p, 0, sizeof(p));
        p.bias = e->bias;
        p.mult = e->mult;
        p.shift = e->shift;
        p.thresh = e->thresh;
        p.n = x->n; p.h = x->h; p.w_ = x->w; p.m = m;
        p.ph = g->pad_h; p.pw = g->pad_w; p.ho = ho; p.wo = wo;
        p.epi = e->kind;
        p.clip_lo = e->clip_lo;
        p.clip_hi = e->clip_hi;
        p.pool = pool ? 1 : 0;
        p.hp = ho / 2;
        p.wp = wo / 2;
        p.tile_bytes = (int32_t)(((int64_t)trows * pp * sb + 15) & ~(int64_t)15);
        p.ipw = 1;
        p.ngroups = (int32_t)(x->n * bands);
        p.pairs = brows / (2 * rt);
        p.quads = 1;
        p.div_w = make_fastdiv((uint32_t)x->w);
        p.div_pairs = make_fastdiv((uint32_t)p.pairs);
        p.div_imgq = make_fastdiv((uint32_t)(trows * x->w * pb / 16));
        p.bands = (int32_t)bands;
        p.brows = brows;
        p.trows = trows;
        p.div_bands = make_fastdiv((uint32_t)bands);
        return true;
    }
    const int64_t tiles = (ho + rt - 1) / rt;
    const int64_t pairs = (tiles + 1) / 2;
    const int extra = u >= 32 ? g->kh - 1 : 2 * ((g->kh + 1) / 2) - 1;
    const int64_t rows = 2 * pairs * rt + extra;
    const int64_t tile = (rows * pp * sb + 15) & ~(int64_t)15;
    // images per step: enough row-tile pairs for the four waves, within the
    // prefetch registers and 64 KB of LDS; several only when the step is a
    // whole number of 16-byte quads
    int64_t ipw = (4 + pairs - 1) / pairs;
    // one-word and half-word pixels: at least two images per step (half as
    // many steps, staging phases and barriers; measured 5% faster on the
    // 32x32 first layers)
    if (pb <= 4 && ipw < 2)
        ipw = 2;
    if (ipw > 8192 / img_bytes)
        ipw = 8192 / img_bytes;
    if (ipw > (64 * 1024) / tile)
        ipw = (64 * 1024) / tile;
    if (img_bytes % 16 != 0)
        ipw = 1;
    if (ipw < 1)
        return false;
    memset(&p, 0, sizeof(p));
    p.bias = e->bias;
    p.mult = e->mult;
    p.shift = e->shift;
    p.thresh = e->thresh;
    p.n = x->n; p.h = x->h; p.w_ = x->w; p.m = m;
    p.ph = g->pad_h; p.pw = g->pad_w; p.ho = ho; p.wo = wo;
    p.epi = e->kind;
    p.clip_lo = e->clip_lo;
    p.clip_hi = e->clip_hi;
    p.pool = pool ? 1 : 0;
    p.hp = ho / 2;
    p.wp = wo / 2;
    p.tile_bytes = (int32_t)tile;
    p.ipw = (int32_t)ipw;
    p.ngroups = (int32_t)((x->n + ipw - 1) / ipw);
    p.pairs = (int32_t)pairs;
    p.quads = img_bytes % 16 == 0 ? 1 : 0;
    p.div_w = make_fastdiv((uint32_t)x->w);
    p.div_pairs = make_fastdiv((uint32_t)pairs);
    p.div_imgq = make_fastdiv((uint32_t)(img_bytes / 16 > 0 ? img_bytes / 16 : 1));
    return true;
}

qnn_status run_conv(const qnn_tensor *x, const void *x_dev, int32_t m, const void *w_dev,
                    const qnn_conv_geom *g, const qnn_epi *e, const qnn_tensor *y, void *y_dev,
                    void *stream, bool pool = false, const qnn_tile *force = nullptr)
{
    if (!x || !g || !e || !y)
        return QNN_ERR_NULL;
    if (!valid_bits(x->bits))
        return QNN_ERR_BITS;
    qnn_status st = check_tensor(x);
    if (st != QNN_OK)
        return st;
    if (m < 1)
        return QNN_ERR_SHAPE;
    if (g->kh < 1 || g->kw < 1 || g->stride_h < 1 || g->stride_w < 1 || g->pad_h < 0 ||
        g->pad_w < 0 || g->pad_h > 1024 || g->pad_w > 1024 || g->kh > 4096 || g->kw > 4096)
        return QNN_ERR_PARAM;
    st = check_epi(e, x->bits, m);
    if (st != QNN_OK)
        return st;
    const int obits = out_bits_for(e->kind, x->bits);
    const int32_t ho = out_dim(x->h, g->kh, g->stride_h, g->pad_h);
    const int32_t wo = out_dim(x->w, g->kw, g->stride_w, g->pad_w);
    if (ho < 1 || wo < 1)
        return QNN_ERR_SHAPE;
    if (pool) {
        if (e->kind != QNN_EPI_REQUANT && e->kind != QNN_EPI_STAIR)
            return QNN_ERR_PARAM;
        if (ho < 2 || wo < 2 || y->n != x->n || y->h != ho / 2 || y->w != wo / 2 || y->c != m)
            return QNN_ERR_SHAPE;
    } else if (y->n != x->n || y->h != ho || y->w != wo || y->c != m) {
        return QNN_ERR_SHAPE;
    }
    if (y->bits != obits)
        return QNN_ERR_BITS;
    const int64_t pb = pixel_bytes64(x);
    // whole 4-byte pixels; or half-word pixels (4 channels at 4 bits), which
    // only the whole-image kernel reads (checked where it is chosen)
    const bool half_word = (int64_t)x->c * x->bits == 16 && x->bits == 4;
    if ((int64_t)x->c * x->bits % 32 != 0 && !half_word)
        return QNN_ERR_ALIGN;
    const int64_t K = (int64_t)g->kh * g->kw * x->c;
    if (K > max_k_for(x->bits))
        return QNN_ERR_OVERFLOW;
    // the e2m1 path: INT-2 / INT-1 codes staged as nibbles, half a byte per
    // channel; its fp32 accumulation is exact while every partial sum stays
    // below 2^24 in magnitude (|x * w| <= 3 * 2, or 1, per term)
    const bool f4 = force && force->kernel == QNN_TILE_FP4;
    if (f4 && K * (x->bits == 1 ? 1 : 6) > ((int64_t)1 << 24))
        return QNN_ERR_OVERFLOW;
    if ((int64_t)x->n * ho * wo >= ((int64_t)1 << 31) || (int64_t)x->n * x->h * x->w >= ((int64_t)1 << 31))
        return QNN_ERR_SHAPE;
    if (x->n == 0)
        return QNN_OK;
    if (!x_dev || !w_dev || !y_dev)
        return QNN_ERR_NULL;
    if (!aligned16(x_dev) || !aligned16(w_dev) || !aligned16(y_dev))
        return QNN_ERR_ALIGN;
    hipStream_t s = (hipStream_t)stream;
    const int ypb = (int)pixel_bytes64(y);
    int cus = 0;

    if (x->bits == 1 && !f4) {
        st = device_info(&cus);
        if (st != QNN_OK)
            return st;
        XnorArgs a;
        memset(&a, 0, sizeof(a));
        a.x = (const uint32_t *)x_dev;
        a.w = (const uint32_t *)w_dev;
        a.y = (uint8_t *)y_dev;
        a.bias = e->bias;
        a.thresh = e->thresh;
        a.n = x->n; a.h = x->h; a.w_ = x->w; a.cd = (int32_t)(pb / 4);
        a.m = m; a.kh = g->kh; a.kw = g->kw; a.sh = g->stride_h; a.sw = g->stride_w;
        a.ph = g->pad_h; a.pw = g->pad_w; a.ho = ho; a.wo = wo;
        a.kd = g->kh * g->kw * a.cd;
        a.kbits = (int32_t)K;
        a.epi = e->kind;
        a.ypb = ypb;
        a.npix = x->n * ho * wo;
        {
            // channel groups: enough waves per SIMD (about 4) to hide the
            // latency of the scalar filter loads, groups of at least 32
            const int64_t waves = ((int64_t)a.npix + 63) / 64;
            int64_t groups = (4 * 4 * (int64_t)cus + waves - 1) / waves;
            const int64_t maxg = (m + 31) / 32;
            groups = groups < 1 ? 1 : (groups > maxg ? maxg : groups);
            a.mgrp = (int32_t)((((m + groups - 1) / groups) + 31) / 32 * 32);
            a.ngroups = (m + a.mgrp - 1) / a.mgrp;
        }
        a.div_wo = make_fastdiv((uint32_t)wo);
        a.div_ho = make_fastdiv((uint32_t)ho);
        a.div_cd = make_fastdiv((uint32_t)a.cd);
        a.div_kw = make_fastdiv((uint32_t)a.kw);
        return launch_conv_xnor(a, s) == hipSuccess ? QNN_OK : QNN_ERR_LAUNCH;
    }

    // small images (a network's first layer, or later layers of 8- to
    // 32-pixel-wide images): the whole-image kernel, unless the caller
    // forces another tile
    const bool force_img = force && force->kernel == QNN_TILE_IMAGE;
    if (!f4 && (!force || force_img)) {
        ImgArgs p;
        int pbytes = 0, wop = 0;
        if (plan_img(p, x, m, g, e, ho, wo, pool, pbytes, wop)) {
            st = device_info(&cus);
            if (st != QNN_OK)
                return st;
            p.x = (const uint8_t *)x_dev;
            p.w = (const uint8_t *)w_dev;
            p.y = (uint8_t *)y_dev;
            p.ypb = ypb;
            hipError_t err;
            if (pbytes == 2)
                err = launch_conv_img_p2(p, x->bits, g->kh, cus, s);
            else if (pbytes == 4)
                err = launch_conv_img_p4(p, x->bits, g->kh, cus, s);
            else if (pbytes == 16)
                err = launch_conv_img_p16(p, x->bits, g->kh, wop, cus, s);
            else
                err = launch_conv_img_p32(p, x->bits, g->kh, wop, cus, s);
            return err == hipSuccess ? QNN_OK : QNN_ERR_LAUNCH;
        }
        if (force_img)
            return half_word ? QNN_ERR_ALIGN : QNN_ERR_UNSUPPORTED;
    }
    if (half_word)
        return QNN_ERR_ALIGN;

    // a filter covering the whole image with raw outputs (the network's
    // classifier): the fully connected kernel, unless the caller forces a tile
    if (!force && e->kind == QNN_EPI_RAW32 && x->bits != 1 && g->kh == x->h && g->kw == x->w &&
        g->pad_h == 0 && g->pad_w == 0 && K % 64 == 0) {
        st = device_info(&cus);
        if (st != QNN_OK)
            return st;
        return launch_linear_raw((const uint8_t *)x_dev, (const uint8_t *)w_dev, e->bias, (int32_t *)y_dev,
                                 x->n, m, (int32_t)K, x->bits, s) == hipSuccess ? QNN_OK : QNN_ERR_LAUNCH;
    }

    ConvArgs a;
    memset(&a, 0, sizeof(a));
    a.x = (const uint8_t *)x_dev;
    a.w = (const uint8_t *)w_dev;
    a.y = (uint8_t *)y_dev;
    a.bias = e->bias;
    a.mult = e->mult;
    a.shift = e->shift;
    a.thresh = e->thresh;
    a.n = x->n; a.h = x->h; a.w_ = x->w; a.pb = (int32_t)pb; a.c8 = x->c;
    a.m = m; a.kh = g->kh; a.kw = g->kw; a.sh = g->stride_h; a.sw = g->stride_w;
    a.ph = g->pad_h; a.pw = g->pad_w; a.ho = ho; a.wo = wo;
    a.wrow = (int32_t)(K * x->bits / 8);
    a.epi = e->kind;
    a.clip_lo = e->clip_lo;
    a.clip_hi = e->clip_hi;
    a.ypb = ypb;
    a.pool = pool ? 1 : 0;
    a.hp = ho / 2;
    a.wp = wo / 2;
    int mr = 0, nc = 0, al16 = 0, wm = 0, wn = 0;
    int nw = 4;
    if (f4)
        a.c8 = x->c / 2;
    const ConvArgs a0 = a;
    bool use32;
    if (f4) {
        // tile_m = 0: the library picks the tile, as for qnn_conv2d
        // (the device's compute units steer the pick; a missing device is
        // reported after the shape checks, below)
        if (force->tile_m != 0 || device_info(&cus) != QNN_OK)
            cus = 0;
        st = plan_conv_m32(a, x->bits, wm, wn, al16, nw, force->tile_m == 0,
                           force->tile_m == 0 ? nullptr : force, true, cus);
        if (st != QNN_OK)
            return st;
        use32 = true;
    } else if (force) {
        st = force->kernel == 32 ? plan_conv_m32(a, x->bits, wm, wn, al16, nw, false, force)
                                 : plan_conv_mfma(a, x->bits, mr, nc, al16, force);
        if (st != QNN_OK)
            return st;
        use32 = force->kernel == 32;
    } else {
        use32 = plan_conv_m32(a, x->bits, wm, wn, al16, nw) == QNN_OK;
        if (!use32 && pool)
            return QNN_ERR_UNSUPPORTED;
        if (!use32) {
            st = plan_conv_mfma(a, x->bits, mr, nc, al16);
            if (st != QNN_OK)
                return st;
        }
    }
    st = device_info(&cus);
    if (st != QNN_OK)
        return st;
    if (use32 && nw == 8 && a.ntiles > cus && !f4) {
        // an eight-wave plan needs one tile per workgroup and one workgroup
        // per compute unit (the e2m1 path also has eight-wave instances that
        // walk several tiles): on a device with fewer compute units the
        // layer takes four waves
        if (force && !(f4 && force->tile_m == 0))
            return QNN_ERR_UNSUPPORTED;
        a = a0;
        if (plan_conv_m32(a, x->bits, wm, wn, al16, nw, false, nullptr, f4) != QNN_OK)
            return QNN_ERR_UNSUPPORTED;
    }
    a.quad16 = (pb % 16) == 0;
    a.pbq = (int32_t)(a.quad16 ? pb / 16 : pb / 4);
    a.div_pbq = make_fastdiv((uint32_t)a.pbq);
    a.div_hwd = make_fastdiv((uint32_t)a.hwd);
    a.div_hh = make_fastdiv((uint32_t)a.hh);
    a.div_tile_px = make_fastdiv((uint32_t)(a.th * a.tw));
    a.div_tw = make_fastdiv((uint32_t)a.tw);
    a.div_tx = make_fastdiv((uint32_t)a.tiles_x);
    a.div_ty = make_fastdiv((uint32_t)a.tiles_y);
    if (a.epi != EPI_RAW32) {
        a.oquad16 = (ypb % 4) == 0;   // copy whole 4-byte words when every tile's range is word-sized
        a.obq = a.oquad16 ? a.ot_b / 4 : a.ot_b;
    } else {
        a.oquad16 = 0;
        a.obq = 1;
    }
    a.div_obq = make_fastdiv((uint32_t)a.obq);
    const int MT = use32 ? 32 * wm : 16 * mr;
    a.contig = a.epi != EPI_RAW32 && !a.pool && a.tw == a.wo && (a.ti == 1 || a.th == a.ho) &&
               a.ot_b == ypb && (ypb % 4) == 0 && m <= MT;
    a.div_qrow = make_fastdiv((uint32_t)(a.wrow / 16 > 0 ? a.wrow / 16 : 1));
    a.div_tab_a = make_fastdiv((uint32_t)(a.row_mode ? a.cpr : (a.c8 >> 4 > 0 ? a.c8 >> 4 : 1)));
    a.div_tab_kw = make_fastdiv((uint32_t)a.kw);
    a.div_ptile = make_fastdiv((uint32_t)((a.th / 2) * (a.tw / 2) > 0 ? (a.th / 2) * (a.tw / 2) : 1));
    a.div_ptw = make_fastdiv((uint32_t)(a.tw / 2 > 0 ? a.tw / 2 : 1));
    // staging items per filter row: int8 words (16x16 kernel), packed words,
    // or 8-byte e2m1 groups (one packed word each)
    a.div_ncol = make_fastdiv((uint32_t)(f4 ? a.kch * x->bits : (use32 ? a.kch * x->bits / 2 : 4 * a.kch)));
    const int mtiles = (m + MT - 1) / MT;
    const int per_cu = (a.lds_bytes * 2 <= kLdsBytes && nw == 4) ? 2 : 1;
    int64_t gx = (int64_t)cus * per_cu;
    if (f4 && nw == 8)
        gx = cus / mtiles > 1 ? cus / mtiles : 1;  // one workgroup per compute unit in all
    if (gx > a.ntiles)
        gx = a.ntiles;
    if (gx < 1)
        gx = 1;
    dim3 grid((unsigned)gx, (unsigned)mtiles);
    hipError_t err;
    if (f4) {
        err = x->bits == 1 ? launch_conv_m32_f4b1(a, wm, wn, al16, nw, grid, s)
                           : launch_conv_m32_f4(a, wm, wn, al16, nw, grid, s);
    } else if (use32) {
        if (x->bits == 8)
            err = launch_conv_m32_b8(a, wm, wn, al16, nw, grid, s);
        else if (x->bits == 4)
            err = launch_conv_m32_b4(a, wm, wn, al16, nw, grid, s);
        else
            err = launch_conv_m32_b2(a, wm, wn, al16, nw, grid, s);
    } else if (x->bits == 8) {
        err = launch_conv_mfma_b8(a, mr, nc, al16, grid, s);
    } else if (x->bits == 4) {
        err = launch_conv_mfma_b4(a, mr, nc, al16, grid, s);
    } else {
        err = launch_conv_mfma_b2(a, mr, nc, al16, grid, s);
    }
    return err == hipSuccess ? QNN_OK : QNN_ERR_LAUNCH;
}

}  // namespace

extern "C" {

int32_t qnn_abi_version(void) { return QNN_ABI_VERSION; }

const char *qnn_status_string(int32_t status)
{
    // compared as an integer: a value outside the enumeration is no
    // qnn_status, and loading it as one would be undefined
    switch (status) {
    case QNN_OK: return "ok";
    case QNN_ERR_NULL: return "a required pointer is NULL";
    case QNN_ERR_BITS: return "unsupported or mismatched bit-width";
    case QNN_ERR_SHAPE: return "invalid or inconsistent tensor shape";
    case QNN_ERR_PARAM: return "parameter out of range";
    case QNN_ERR_ALIGN: return "pixel bytes not a multiple of 4 or device pointer not 16-byte aligned";
    case QNN_ERR_OVERFLOW: return "filter volume too large for the 32-bit accumulator";
    case QNN_ERR_UNSUPPORTED: return "shape exceeds the kernels' local-memory limits";
    case QNN_ERR_DEVICE: return "no usable gfx950 device is current";
    case QNN_ERR_LAUNCH: return "kernel launch failed";
    }
    return "unknown status";
}

qnn_status qnn_device_check(void) { return device_info(nullptr); }

size_t qnn_pixel_bytes(const qnn_tensor *t)
{
    if (!t || t->c < 0)
        return 0;
    return (size_t)pixel_bytes64(t);
}

size_t qnn_tensor_bytes(const qnn_tensor *t)
{
    if (!t || t->n < 0 || t->h < 0 || t->w < 0 || t->c < 0)
        return 0;
    return (size_t)t->n * t->h * t->w * (size_t)pixel_bytes64(t);
}

qnn_status qnn_conv2d_out_shape(const qnn_tensor *x, int32_t m, const qnn_conv_geom *g,
                                int32_t kind, qnn_tensor *y)
{
    if (!x || !g || !y)
        return QNN_ERR_NULL;
    if (!valid_bits(x->bits))
        return QNN_ERR_BITS;
    if (check_tensor(x) != QNN_OK || m < 1)
        return QNN_ERR_SHAPE;
    if (g->kh < 1 || g->kw < 1 || g->stride_h < 1 || g->stride_w < 1 || g->pad_h < 0 || g->pad_w < 0)
        return QNN_ERR_PARAM;
    if (kind != QNN_EPI_REQUANT && kind != QNN_EPI_THRESH1 && kind != QNN_EPI_RAW32 &&
        kind != QNN_EPI_STAIR)
        return QNN_ERR_PARAM;
    if ((kind == QNN_EPI_REQUANT && x->bits == 1) || (kind == QNN_EPI_THRESH1 && x->bits != 1) ||
        (kind == QNN_EPI_STAIR && x->bits != 4 && x->bits != 2))
        return QNN_ERR_BITS;
    const int32_t ho = out_dim(x->h, g->kh, g->stride_h, g->pad_h);
    const int32_t wo = out_dim(x->w, g->kw, g->stride_w, g->pad_w);
    if (ho < 1 || wo < 1)
        return QNN_ERR_SHAPE;
    y->n = x->n;
    y->h = ho;
    y->w = wo;
    y->c = m;
    y->bits = out_bits_for(kind, x->bits);
    return QNN_OK;
}

qnn_status qnn_conv2d(const qnn_tensor *x, const void *x_dev, int32_t m, const void *w_dev,
                      const qnn_conv_geom *g, const qnn_epi *e, const qnn_tensor *y, void *y_dev,
                      void *stream)
{
    return run_conv(x, x_dev, m, w_dev, g, e, y, y_dev, stream);
}

qnn_status qnn_conv2d_tiled(const qnn_tensor *x, const void *x_dev, int32_t m, const void *w_dev,
                            const qnn_conv_geom *g, const qnn_epi *e, const qnn_tile *tile,
                            const qnn_tensor *y, void *y_dev, void *stream)
{
    if (!tile)
        return QNN_ERR_NULL;
    if (x && x->bits == 1 && tile->kernel != QNN_TILE_FP4)
        return QNN_ERR_PARAM;  // the XNOR kernel has no matrix tiles
    const int tm = tile->tile_m, tn = tile->tile_n;
    bool built = false;
    if (tile->kernel == QNN_TILE_FP4) {
        if (x && x->bits != 2 && x->bits != 1)
            return QNN_ERR_BITS;
        built = (tm == 0 && tn == 0 && tile->waves == 0) ||
                ((tile->waves == 4 || tile->waves == 8) && (tn == 1 || tn == 2) && (tm == 1 || tm == 2));
    } else if (tile->kernel == QNN_TILE_IMAGE) {
        built = tm == 0 && tn == 0 && tile->waves == 0;
    } else if (tile->kernel == 16)
        built = tile->waves == 4 && (tm == 1 || tm == 2 || tm == 4) && (tn == 1 || tn == 2 || tn == 4);
    else if (tile->kernel == 32)
        built = (tile->waves == 4 || tile->waves == 8) && (tn == 1 || tn == 2) &&
                (tm == 1 || tm == 2 || (tm == 4 && tn == 1 && tile->waves == 4 && x && x->bits == 8));
    if (!built)
        return QNN_ERR_PARAM;
    return run_conv(x, x_dev, m, w_dev, g, e, y, y_dev, stream, false, tile);
}

qnn_status qnn_conv2d_maxpool(const qnn_tensor *x, const void *x_dev, int32_t m, const void *w_dev,
                              const qnn_conv_geom *g, const qnn_epi *e, int32_t pool_k,
                              int32_t pool_s, const qnn_tensor *y, void *y_dev, void *stream)
{
    if (pool_k != 2 || pool_s != 2)
        return QNN_ERR_PARAM;
    if (x && x->bits == 1)
        return QNN_ERR_BITS;
    return run_conv(x, x_dev, m, w_dev, g, e, y, y_dev, stream, true);
}

qnn_status qnn_linear(const qnn_tensor *x, const void *x_dev, int32_t m, const void *w_dev,
                      const qnn_epi *e, const qnn_tensor *y, void *y_dev, void *stream)
{
    if (!x || !e || !y)
        return QNN_ERR_NULL;
    if (y->h != 1 || y->w != 1)
        return QNN_ERR_SHAPE;
    qnn_conv_geom g = {x->h, x->w, 1, 1, 0, 0};
    return run_conv(x, x_dev, m, w_dev, &g, e, y, y_dev, stream);
}

qnn_status qnn_maxpool2d(const qnn_tensor *x, const void *x_dev, int32_t kh, int32_t kw,
                         int32_t sh, int32_t sw, const qnn_tensor *y, void *y_dev, void *stream)
{
    if (!x || !y)
        return QNN_ERR_NULL;
    if (x->bits != 8 && x->bits != 4 && x->bits != 2)
        return QNN_ERR_BITS;
    qnn_status st = check_tensor(x);
    if (st != QNN_OK)
        return st;
    if (kh < 1 || kw < 1 || sh < 1 || sw < 1)
        return QNN_ERR_PARAM;
    const int32_t ho = out_dim(x->h, kh, sh, 0), wo = out_dim(x->w, kw, sw, 0);
    if (ho < 1 || wo < 1)
        return QNN_ERR_SHAPE;
    if (y->n != x->n || y->h != ho || y->w != wo || y->c != x->c)
        return QNN_ERR_SHAPE;
    if (y->bits != x->bits)
        return QNN_ERR_BITS;
    const int64_t pb = pixel_bytes64(x);
    if ((int64_t)x->c * x->bits % 32 != 0)
        return QNN_ERR_ALIGN;
    const int64_t total = (int64_t)x->n * ho * wo * (pb / 4);
    if (total >= ((int64_t)1 << 31) || (int64_t)x->n * x->h * x->w >= ((int64_t)1 << 31))
        return QNN_ERR_SHAPE;
    if (x->n == 0)
        return QNN_OK;
    if (!x_dev || !y_dev)
        return QNN_ERR_NULL;
    if (!aligned16(x_dev) || !aligned16(y_dev))
        return QNN_ERR_ALIGN;
    st = device_info(nullptr);
    if (st != QNN_OK)
        return st;
    PoolArgs a;
    memset(&a, 0, sizeof(a));
    a.x = (const uint8_t *)x_dev;
    a.y = (uint8_t *)y_dev;
    a.n = x->n; a.h = x->h; a.w_ = x->w; a.pbd = (int32_t)(pb / 4);
    a.kh = kh; a.kw = kw; a.sh = sh; a.sw = sw; a.ho = ho; a.wo = wo;
    a.total = (int32_t)total;
    a.div_pbd = make_fastdiv((uint32_t)a.pbd);
    a.div_wo = make_fastdiv((uint32_t)wo);
    a.div_ho = make_fastdiv((uint32_t)ho);
    return launch_maxpool(a, x->bits, (hipStream_t)stream) == hipSuccess ? QNN_OK : QNN_ERR_LAUNCH;
}

qnn_status qnn_relu_s8(const void *x_dev, void *y_dev, size_t count, void *stream)
{
    if (count == 0)
        return QNN_OK;
    if (!x_dev || !y_dev)
        return QNN_ERR_NULL;
    if (!aligned16(x_dev) || !aligned16(y_dev))
        return QNN_ERR_ALIGN;
    if (count >= ((size_t)1 << 40))
        return QNN_ERR_SHAPE;
    qnn_status st = device_info(nullptr);
    if (st != QNN_OK)
        return st;
    return launch_relu_s8((const uint8_t *)x_dev, (uint8_t *)y_dev, count, (hipStream_t)stream) ==
                   hipSuccess
               ? QNN_OK
               : QNN_ERR_LAUNCH;
}

qnn_status qnn_pack_host(const uint8_t *codes, size_t count, int32_t bits, uint8_t *out)
{
    if (!valid_bits(bits))
        return QNN_ERR_BITS;
    if (count == 0)
        return QNN_OK;
    if (!codes || !out)
        return QNN_ERR_NULL;
    const unsigned mask = (1u << bits) - 1u;
    for (size_t i = 0; i < count; ++i)
        if (codes[i] > mask)
            return QNN_ERR_PARAM;
    const size_t nbytes = (count * (size_t)bits + 7) / 8;
    memset(out, 0, nbytes);
    const int per = 8 / bits;
    for (size_t i = 0; i < count; ++i)
        out[i / per] |= (uint8_t)(codes[i] << ((i % per) * bits));
    return QNN_OK;
}

qnn_status qnn_unpack_host(const uint8_t *packed, size_t count, int32_t bits, int32_t is_signed,
                           int32_t *out)
{
    if (!valid_bits(bits))
        return QNN_ERR_BITS;
    if (count == 0)
        return QNN_OK;
    if (!packed || !out)
        return QNN_ERR_NULL;
    const int per = 8 / bits;
    const unsigned mask = (1u << bits) - 1u;
    for (size_t i = 0; i < count; ++i) {
        const unsigned code = (packed[i / per] >> ((i % per) * bits)) & mask;
        int32_t v;
        if (bits == 1)
            v = code ? 1 : -1;
        else if (is_signed && (code >> (bits - 1)))
            v = (int32_t)code - (1 << bits);
        else
            v = (int32_t)code;
        out[i] = v;
    }
    return QNN_OK;
}

}  // extern "C"
