/*
 * Reference (oracle) implementation of the quantized convolution layer of
 * PULP-NN (Garofalo et al., "PULP-NN: Accelerating Quantized Neural Networks
 * on Parallel Ultra-Low-Power RISC-V Processors").
 *
 * TEST INFRASTRUCTURE ONLY.  This file is the plain, slow, obviously correct
 * CPU definition that the GPU library is checked against.  Only the test
 * suite, the smoke check and the benchmark's CPU-baseline leg may load it.
 * It shares no code, header, table or helper with the GPU library.
 *
 * What is computed (all integer, no floating point):
 *   - Sec. III-A, Eq. (2): the layer accumulates Phi = sum_i W_i * X_i over
 *     the receptive field, in a wide integer accumulator.
 *   - Sec. III-B, Eq. (6): the output O(m, x, y) is the dot product of the
 *     m-th filter bank with the im2col column of the output pixel, i.e. the
 *     C x kw x kh input values under the filter (cross-correlation, no flip).
 *   - Sec. III-B: tensors are stored Height-Width-Channel, channel stride 1.
 *   - Sec. III-A: INT-8 outputs are compressed back by scaling and clamping;
 *     this library uses a per-channel integer multiplier, a rounding right
 *     shift and a clip (reading of the "scaling and clamp" step).
 *   - Sec. III-A, Eq. (5) and Sec. IV-A "Binary Convolution Kernel": INT-1
 *     values are +1/-1 and the output bit comes from one threshold per
 *     channel.  This oracle uses the +1/-1 product form; the XNOR/popcount
 *     form is checked against it by the tests.
 *   - Sec. IV-A "Sub-byte Extensions": INT-4 / INT-2 / INT-1 values are
 *     stored compactly, several per byte.
 *   - Sec. IV-A "INT-8 Kernels": ReLU is a max with zero, max-pooling takes
 *     the maximum over a window; the fully connected layer is a dot product
 *     of the whole input with each weight row.
 *
 * Readings where the paper is silent (each one is listed with its reason in
 * the design notes of the repository):
 *   - sub-byte packing: the lower channel occupies the less significant bits;
 *     the unused high bits of a pixel's last byte are zero;
 *   - activations are unsigned codes for 8/4/2 bits; weights are two's
 *     complement codes; for 1 bit both operands take the value 2*bit - 1;
 *   - padding taps hold code 0 (value 0, or -1 for 1 bit);
 *   - requantization: y = clip(floor((acc + bias) * mult / 2^shift + 1/2));
 *     the product is taken without any overflow;
 *   - binary threshold: bit = (acc + bias >= thresh), acc the +1/-1 dot;
 *   - staircase compression (Sec. III-A, Eq. (4)), 4 and 2 bits: each
 *     channel has 2^Q - 1 thresholds tau_1 .. tau_{2^Q-1} and the output is
 *     the level p of the interval [tau_p, tau_{p+1}) that holds acc + bias
 *     (tau_0 = -inf, tau_{2^Q} = +inf).  For thresholds that are not
 *     non-decreasing the intervals overlap or leave gaps; the library then
 *     defines the output as the number of thresholds at or below acc + bias,
 *     which is the same level whenever the thresholds are sorted;
 *   - RAW32 returns acc + bias reduced modulo 2^32 (two's complement).
 */
#include <stdint.h>
#include <stddef.h>
#include <string.h>
#include <stdlib.h>
#include <pthread.h>

enum { ORC_REQUANT = 0, ORC_THRESH1 = 1, ORC_RAW32 = 2, ORC_STAIR = 3 };

/* Number of bytes that hold `count` codes of `bits` bits (whole bytes). */
size_t oracle_packed_bytes(size_t count, int bits)
{
    return (count * (size_t)bits + 7) / 8;
}

/* Unsigned code of element `i` in a packed run of `bits`-bit codes
 * (Sec. IV-A, sub-byte storage; lower element in the lower bits). */
static unsigned get_code(const uint8_t *run, size_t i, int bits)
{
    size_t bit = i * (size_t)bits;
    unsigned byte = run[bit / 8];
    unsigned mask = (1u << bits) - 1u;
    if (bits == 8)
        return byte;
    return (byte >> (bit % 8)) & mask;
}

static void put_code(uint8_t *run, size_t i, int bits, unsigned code)
{
    size_t bit = i * (size_t)bits;
    unsigned mask = (1u << bits) - 1u;
    if (bits == 8) {
        run[bit / 8] = (uint8_t)code;
        return;
    }
    run[bit / 8] = (uint8_t)((run[bit / 8] & ~(mask << (bit % 8))) | ((code & mask) << (bit % 8)));
}

/* Activation value of a code: unsigned for 8/4/2 bits, +1/-1 for 1 bit. */
static int64_t act_value(unsigned code, int bits)
{
    if (bits == 1)
        return code ? 1 : -1;
    return (int64_t)code;
}

/* Weight value of a code: two's complement of `bits` bits, +1/-1 for 1 bit
 * (Sec. III-A, Eq. (1): W = q(w) * 2^(Q-1) is a signed integer). */
static int64_t wgt_value(unsigned code, int bits)
{
    if (bits == 1)
        return code ? 1 : -1;
    if (code >= (1u << (bits - 1)))
        return (int64_t)code - ((int64_t)1 << bits);
    return (int64_t)code;
}

/* Exported decode/encode of whole runs, used by the packing pins. */
void oracle_unpack(const uint8_t *packed, size_t count, int bits, int is_signed, int32_t *out)
{
    for (size_t i = 0; i < count; ++i) {
        unsigned code = get_code(packed, i, bits);
        out[i] = (int32_t)(is_signed ? wgt_value(code, bits) : act_value(code, bits));
    }
}

void oracle_pack(const uint32_t *codes, size_t count, int bits, uint8_t *out)
{
    memset(out, 0, oracle_packed_bytes(count, bits));
    for (size_t i = 0; i < count; ++i)
        put_code(out, i, bits, codes[i]);
}

/* floor(a / 2^s) for s >= 0, written as a floor division (no reliance on the
 * behaviour of >> on negative numbers). */
static __int128 floor_div_pow2(__int128 a, int s)
{
    __int128 d = (__int128)1 << s;
    __int128 q = a / d;
    if ((a % d) != 0 && a < 0)
        q -= 1;
    return q;
}

/* Staircase compression of Sec. III-A, Eq. (4): Y = sum_p p * chi_[tau_p,
 * tau_{p+1})(phi) over p = 0 .. 2^Q - 1 with tau_0 = -inf, tau_{2^Q} = +inf.
 * `tau` holds tau_1 .. tau_{2^Q-1}.  With non-decreasing thresholds exactly
 * one interval holds phi; otherwise the count of thresholds at or below phi
 * is returned (the library's definition for unsorted thresholds). */
static unsigned staircase(int64_t phi, const int32_t *tau, int q)
{
    const int levels = 1 << q;
    int sorted = 1;
    for (int p = 1; p + 1 < levels; ++p)
        if (tau[p] < tau[p - 1])
            sorted = 0;
    if (sorted) {
        for (int p = 0; p < levels; ++p) {
            /* interval [tau_p, tau_{p+1}): lower end tau_p (p >= 1) */
            int above_lower = p == 0 || phi >= (int64_t)tau[p - 1];
            int below_upper = p == levels - 1 || phi < (int64_t)tau[p];
            if (above_lower && below_upper)
                return (unsigned)p;
        }
    }
    unsigned count = 0;
    for (int p = 1; p < levels; ++p)
        if (phi >= (int64_t)tau[p - 1])
            ++count;
    return count;
}

/* INT-8 / sub-byte compression by scale and clamp (Sec. III-A). */
static int64_t requant(int64_t v, int32_t mult, int shift, int32_t lo, int32_t hi)
{
    __int128 t = (__int128)v * (__int128)mult;
    __int128 r;
    if (shift == 0)
        r = t;
    else
        r = floor_div_pow2(t + ((__int128)1 << (shift - 1)), shift);
    if (r < lo)
        r = lo;
    if (r > hi)
        r = hi;
    return (int64_t)r;
}

typedef struct {
    /* input */
    const uint8_t *x;
    int32_t n, h, w, c, bits;
    /* weights, M x kh x kw x C (OHWI), same bit-width */
    const uint8_t *wt;
    int32_t m, kh, kw, sh, sw, ph, pw;
    /* epilogue */
    int32_t epi;
    const int32_t *bias, *mult, *thresh;
    const int8_t *shift;
    int32_t clip_lo, clip_hi;
    /* outputs */
    int64_t *acc;  /* optional raw accumulators [N][Ho][Wo][M] */
    uint8_t *y;    /* optional epilogue output */
    int32_t ho, wo;
    /* image range for one thread */
    int32_t n0, n1;
} conv_job;

/* Eq. (2) / Eq. (6): plain nested loops over every output element. */
static void *conv_worker(void *arg)
{
    const conv_job *j = (const conv_job *)arg;
    const size_t xpix = oracle_packed_bytes((size_t)j->c, j->bits);
    const size_t wrow = oracle_packed_bytes((size_t)j->kh * j->kw * j->c, j->bits);
    const int obits = (j->epi == ORC_REQUANT || j->epi == ORC_STAIR) ? j->bits : (j->epi == ORC_THRESH1 ? 1 : 32);
    const size_t ypix = obits == 32 ? (size_t)j->m * 4 : oracle_packed_bytes((size_t)j->m, obits);
    for (int32_t n = j->n0; n < j->n1; ++n)
        for (int32_t oy = 0; oy < j->ho; ++oy)
            for (int32_t ox = 0; ox < j->wo; ++ox) {
                size_t opix = ((size_t)n * j->ho + oy) * j->wo + ox;
                uint8_t *yp = j->y ? j->y + opix * ypix : NULL;
                if (yp && obits != 32)
                    memset(yp, 0, ypix);
                for (int32_t mm = 0; mm < j->m; ++mm) {
                    const uint8_t *wrun = j->wt + (size_t)mm * wrow;
                    int64_t acc = 0;
                    for (int32_t ky = 0; ky < j->kh; ++ky)
                        for (int32_t kx = 0; kx < j->kw; ++kx) {
                            int32_t iy = oy * j->sh - j->ph + ky;
                            int32_t ix = ox * j->sw - j->pw + kx;
                            int inside = iy >= 0 && iy < j->h && ix >= 0 && ix < j->w;
                            const uint8_t *xrun = inside
                                ? j->x + (((size_t)n * j->h + iy) * j->w + ix) * xpix
                                : NULL;
                            for (int32_t cc = 0; cc < j->c; ++cc) {
                                /* padding taps hold code 0 */
                                unsigned xc = inside ? get_code(xrun, (size_t)cc, j->bits) : 0u;
                                size_t wi = ((size_t)ky * j->kw + kx) * j->c + cc;
                                unsigned wc = get_code(wrun, wi, j->bits);
                                acc += act_value(xc, j->bits) * wgt_value(wc, j->bits);
                            }
                        }
                    if (j->acc)
                        j->acc[opix * j->m + mm] = acc;
                    if (!yp)
                        continue;
                    int64_t b = j->bias ? j->bias[mm] : 0;
                    if (j->epi == ORC_REQUANT) {
                        int64_t q = requant(acc + b, j->mult[mm], j->shift[mm], j->clip_lo, j->clip_hi);
                        put_code(yp, (size_t)mm, obits, (unsigned)q);
                    } else if (j->epi == ORC_THRESH1) {
                        put_code(yp, (size_t)mm, 1, (acc + b >= (int64_t)j->thresh[mm]) ? 1u : 0u);
                    } else if (j->epi == ORC_STAIR) {
                        const int nt = (1 << j->bits) - 1;
                        put_code(yp, (size_t)mm, obits, staircase(acc + b, j->thresh + (size_t)mm * nt, j->bits));
                    } else {
                        uint32_t r = (uint32_t)(uint64_t)(acc + b); /* modulo 2^32 */
                        memcpy(yp + (size_t)mm * 4, &r, 4);
                    }
                }
            }
    return NULL;
}

/* Output size along one axis: floor((in + 2*pad - k) / stride) + 1. */
int32_t oracle_out_dim(int32_t in, int32_t k, int32_t stride, int32_t pad)
{
    int32_t span = in + 2 * pad - k;
    if (span < 0 || stride < 1)
        return 0;
    return span / stride + 1;
}

/*
 * Quantized convolution.  Returns 0 on success, -1 on an argument the oracle
 * does not define.  `acc` (int64 [N][Ho][Wo][M]) and `y` are each optional.
 * y holds packed codes (REQUANT and STAIR at the input bit-width, THRESH1
 * at 1 bit; STAIR reads 2^bits - 1 thresholds per channel, channel-major) or
 * little-endian int32 values (RAW32), one output pixel after the other.
 */
int oracle_conv2d(const uint8_t *x, int32_t n, int32_t h, int32_t w, int32_t c, int32_t bits,
                  const uint8_t *wt, int32_t m, int32_t kh, int32_t kw,
                  int32_t sh, int32_t sw, int32_t ph, int32_t pw,
                  int32_t epi, const int32_t *bias, const int32_t *mult, const int8_t *shift,
                  const int32_t *thresh, int32_t clip_lo, int32_t clip_hi,
                  int64_t *acc, uint8_t *y, int32_t nthreads)
{
    if (!(bits == 1 || bits == 2 || bits == 4 || bits == 8))
        return -1;
    if (n < 0 || h < 1 || w < 1 || c < 1 || m < 1 || kh < 1 || kw < 1 || sh < 1 || sw < 1 ||
        ph < 0 || pw < 0)
        return -1;
    if (epi == ORC_REQUANT && (bits == 1 || !mult || !shift))
        return -1;
    if (epi == ORC_THRESH1 && (bits != 1 || !thresh))
        return -1;
    if (epi == ORC_STAIR && ((bits != 4 && bits != 2) || !thresh))
        return -1;
    if (epi < ORC_REQUANT || epi > ORC_STAIR)
        return -1;
    int32_t ho = oracle_out_dim(h, kh, sh, ph), wo = oracle_out_dim(w, kw, sw, pw);
    if (ho < 1 || wo < 1)
        return -1;
    if (nthreads < 1)
        nthreads = 1;
    if (nthreads > n)
        nthreads = n > 0 ? n : 1;
    conv_job base = {x, n, h, w, c, bits, wt, m, kh, kw, sh, sw, ph, pw, epi, bias, mult, thresh,
                     shift, clip_lo, clip_hi, acc, y, ho, wo, 0, n};
    if (nthreads == 1) {
        conv_worker(&base);
        return 0;
    }
    pthread_t *tid = (pthread_t *)calloc((size_t)nthreads, sizeof(pthread_t));
    conv_job *jobs = (conv_job *)calloc((size_t)nthreads, sizeof(conv_job));
    for (int32_t t = 0; t < nthreads; ++t) {
        jobs[t] = base;
        jobs[t].n0 = (int32_t)((int64_t)n * t / nthreads);
        jobs[t].n1 = (int32_t)((int64_t)n * (t + 1) / nthreads);
        pthread_create(&tid[t], NULL, conv_worker, &jobs[t]);
    }
    for (int32_t t = 0; t < nthreads; ++t)
        pthread_join(tid[t], NULL);
    free(tid);
    free(jobs);
    return 0;
}

/*
 * Fully connected layer (Sec. IV-A): out[n][j] = sum_i X[n][i] * W[j][i],
 * i running over the whole input of image n in its stored (HWC) order,
 * followed by the same epilogue as the convolution.
 */
int oracle_linear(const uint8_t *x, int32_t n, int32_t k, int32_t bits,
                  const uint8_t *wt, int32_t m,
                  int32_t epi, const int32_t *bias, const int32_t *mult, const int8_t *shift,
                  const int32_t *thresh, int32_t clip_lo, int32_t clip_hi,
                  int64_t *acc, uint8_t *y)
{
    if (!(bits == 1 || bits == 2 || bits == 4 || bits == 8) || n < 0 || k < 1 || m < 1)
        return -1;
    if (epi == ORC_STAIR && ((bits != 4 && bits != 2) || !thresh))
        return -1;
    const size_t xrow = oracle_packed_bytes((size_t)k, bits);
    const int obits = (epi == ORC_REQUANT || epi == ORC_STAIR) ? bits : (epi == ORC_THRESH1 ? 1 : 32);
    const size_t yrow = obits == 32 ? (size_t)m * 4 : oracle_packed_bytes((size_t)m, obits);
    for (int32_t nn = 0; nn < n; ++nn) {
        uint8_t *yp = y ? y + (size_t)nn * yrow : NULL;
        if (yp && obits != 32)
            memset(yp, 0, yrow);
        for (int32_t j = 0; j < m; ++j) {
            int64_t s = 0;
            for (int32_t i = 0; i < k; ++i)
                s += act_value(get_code(x + (size_t)nn * xrow, (size_t)i, bits), bits) *
                     wgt_value(get_code(wt + (size_t)j * xrow, (size_t)i, bits), bits);
            if (acc)
                acc[(size_t)nn * m + j] = s;
            if (!yp)
                continue;
            int64_t b = bias ? bias[j] : 0;
            if (epi == ORC_REQUANT)
                put_code(yp, (size_t)j, obits, (unsigned)requant(s + b, mult[j], shift[j], clip_lo, clip_hi));
            else if (epi == ORC_THRESH1)
                put_code(yp, (size_t)j, 1, (s + b >= (int64_t)thresh[j]) ? 1u : 0u);
            else if (epi == ORC_STAIR)
                put_code(yp, (size_t)j, obits, staircase(s + b, thresh + (size_t)j * ((1 << bits) - 1), bits));
            else {
                uint32_t r = (uint32_t)(uint64_t)(s + b);
                memcpy(yp + (size_t)j * 4, &r, 4);
            }
        }
    }
    return 0;
}

/* Max-pooling over unsigned codes (Sec. IV-A), no padding, floor size. */
int oracle_maxpool2d(const uint8_t *x, int32_t n, int32_t h, int32_t w, int32_t c, int32_t bits,
                     int32_t kh, int32_t kw, int32_t sh, int32_t sw, uint8_t *y)
{
    if (!(bits == 2 || bits == 4 || bits == 8) || kh < 1 || kw < 1 || sh < 1 || sw < 1)
        return -1;
    int32_t ho = oracle_out_dim(h, kh, sh, 0), wo = oracle_out_dim(w, kw, sw, 0);
    if (ho < 1 || wo < 1)
        return -1;
    const size_t pix = oracle_packed_bytes((size_t)c, bits);
    for (int32_t nn = 0; nn < n; ++nn)
        for (int32_t oy = 0; oy < ho; ++oy)
            for (int32_t ox = 0; ox < wo; ++ox) {
                uint8_t *yp = y + (((size_t)nn * ho + oy) * wo + ox) * pix;
                memset(yp, 0, pix);
                for (int32_t cc = 0; cc < c; ++cc) {
                    unsigned best = 0;
                    for (int32_t ky = 0; ky < kh; ++ky)
                        for (int32_t kx = 0; kx < kw; ++kx) {
                            const uint8_t *xp =
                                x + (((size_t)nn * h + oy * sh + ky) * w + ox * sw + kx) * pix;
                            unsigned v = get_code(xp, (size_t)cc, bits);
                            if (v > best)
                                best = v;
                        }
                    put_code(yp, (size_t)cc, bits, best);
                }
            }
    return 0;
}

/* ReLU on signed 8-bit values: max(v, 0) (Sec. IV-A). */
void oracle_relu_s8(const int8_t *x, size_t count, int8_t *y)
{
    for (size_t i = 0; i < count; ++i)
        y[i] = x[i] > 0 ? x[i] : 0;
}
