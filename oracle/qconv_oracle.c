/*
 * qconv_oracle.c -- TEST INFRASTRUCTURE ONLY.
 *
 * A plain, slow, obviously correct CPU reference for reduced-precision
 * (4-bit / 8-bit) integer 2-D convolution with a per-channel requantising
 * epilogue and nibble packing.  Only the test suite, the smoke check and the
 * CPU-baseline leg of the benchmark load this code.  It shares nothing with
 * the GPU library (no headers, helpers or tables) and the GPU library never
 * loads it.
 *
 * Everything is exact integer arithmetic: products and sums are formed in
 * int64, so the result is the unique mathematical value of each definition.
 *
 * Definitions followed (paper "Learning from Distinctive Candidates to
 * Optimize Reduced-Precision Convolution Program on Tensor Cores"):
 *   - Sec. 2.1: a convolution over an N x H x W x I input with O filters of
 *     R x S is the product of the lowered (im2col) matrix (N*H*W, I*R*S) with
 *     the (I*R*S, O) filter matrix; every output element is one inner product
 *     of a lowered row with a filter column.  oracle_conv2d sums that inner
 *     product directly, tap by tap, without forming the lowered matrix.
 *   - Sec. 3.2.1: the accumulator of a reduced-precision product needs far
 *     fewer than 32 bits; oracle_conv2d checks |acc| < 2^31 for every output
 *     and reports a violation instead of wrapping.
 *   - Sec. 3.2.2: the epilogue runs on the wide accumulator, and only after
 *     it has finished is the value clipped to the low bit-width and packed.
 *     oracle_requant is that order: scale, round, ReLU, clamp.
 *   - Sec. 1 and Sec. 3.2.3: eight 4-bit values share one 32-bit word.
 *     oracle_pack4 / oracle_unpack4 fix the order used here: channel 8j+i of
 *     a pixel lives in bits [4i, 4i+3] of that pixel's word j.
 *
 * Readings where the paper is silent (each is also listed in the design
 * notes): cross-correlation (no filter flip); output size
 * P = floor((H + 2*pad_h - R) / stride_h) + 1 (likewise Q); zero padding;
 * two's-complement nibbles for signed 4-bit values; saturation of
 * out-of-range int8 inputs before packing; round-half-up (toward +inf) for
 * the requantiser, computed with an explicit floor so that negative values
 * do not depend on the behaviour of '>>' on signed integers.
 */
#include <stdint.h>
#include <stddef.h>
#include <stdlib.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#define ORACLE_OK 0
#define ORACLE_EINVAL -1
#define ORACLE_EOVERFLOW -5

/* Output extent of a strided, zero-padded window (a reading: see header). */
int64_t oracle_out_dim(int64_t in, int64_t window, int64_t stride, int64_t pad)
{
    int64_t span = in + 2 * pad - window;
    if (stride < 1 || pad < 0 || window < 1 || span < 0)
        return -1;
    return span / stride + 1;
}

/* Range of a b-bit integer, signed (two's complement) or unsigned. */
static int64_t range_lo(int bits, int is_signed) { return is_signed ? -((int64_t)1 << (bits - 1)) : 0; }
static int64_t range_hi(int bits, int is_signed)
{
    return is_signed ? ((int64_t)1 << (bits - 1)) - 1 : ((int64_t)1 << bits) - 1;
}

/* Saturate an integer into the b-bit range. */
int64_t oracle_saturate(int64_t v, int bits, int is_signed)
{
    int64_t lo = range_lo(bits, is_signed), hi = range_hi(bits, is_signed);
    if (v < lo) return lo;
    if (v > hi) return hi;
    return v;
}

/* Value of one 4-bit field. */
static int64_t nibble_value(uint32_t nib, int is_signed)
{
    if (is_signed && nib >= 8)
        return (int64_t)nib - 16;
    return (int64_t)nib;
}

/*
 * Unpack `count` 4-bit values (count a multiple of 8) from 32-bit words.
 * Value number v = 8*j + i is bits [4i, 4i+3] of word j.
 */
void oracle_unpack4(const uint32_t *words, int64_t count, int is_signed, int32_t *out)
{
    for (int64_t v = 0; v < count; ++v) {
        int64_t j = v / 8, i = v % 8;
        uint32_t nib = (words[j] >> (4 * i)) & 0xFu;
        out[v] = (int32_t)nibble_value(nib, is_signed);
    }
}

/*
 * Pack `count` integers (count a multiple of 8, each already inside the
 * signed or unsigned 4-bit range) into 32-bit words, value 8*j+i into bits
 * [4i, 4i+3] of word j.  Returns ORACLE_EINVAL if a value is out of range.
 */
int oracle_pack4(const int32_t *vals, int64_t count, int is_signed, uint32_t *words)
{
    for (int64_t j = 0; j < count / 8; ++j)
        words[j] = 0;
    for (int64_t v = 0; v < count; ++v) {
        int64_t x = vals[v];
        if (x < range_lo(4, is_signed) || x > range_hi(4, is_signed))
            return ORACLE_EINVAL;
        uint32_t nib = (uint32_t)(x < 0 ? x + 16 : x);
        words[v / 8] |= nib << (4 * (v % 8));
    }
    return ORACLE_OK;
}

/*
 * The relayout-and-pack step applied to activations entering the network and
 * to filters (Sec. 1: values are quantised and grouped eight to a 32-bit
 * word along the channel axis; Sec. 3.3: the packed tensor keeps channels
 * innermost so that the next layer reads it in the same layout).
 *
 * src is int8 in N x C x H x W order (filters: K x C x R x S).  Each value
 * is first saturated into the b-bit range.  dst is
 *   bits == 4: uint32 words, N x H x W x (C/8), channel c of a pixel in
 *              word c/8, bits [4*(c%8), 4*(c%8)+3];
 *   bits == 8: int8, N x H x W x C.
 */
int oracle_relayout_pack(const int8_t *src, int64_t n, int64_t c, int64_t h, int64_t w,
                         int bits, int is_signed, void *dst)
{
    if (n < 0 || c < 0 || h < 0 || w < 0)
        return ORACLE_EINVAL;
    if (bits == 4) {
        if (c % 8 != 0)
            return ORACLE_EINVAL;
        uint32_t *out = (uint32_t *)dst;
        for (int64_t i0 = 0; i0 < n; ++i0)
            for (int64_t y = 0; y < h; ++y)
                for (int64_t x = 0; x < w; ++x)
                    for (int64_t j = 0; j < c / 8; ++j) {
                        uint32_t word = 0;
                        for (int64_t i = 0; i < 8; ++i) {
                            int64_t ch = 8 * j + i;
                            int64_t v = oracle_saturate(src[((i0 * c + ch) * h + y) * w + x], 4, is_signed);
                            uint32_t nib = (uint32_t)(v < 0 ? v + 16 : v);
                            word |= nib << (4 * i);
                        }
                        out[((i0 * h + y) * w + x) * (c / 8) + j] = word;
                    }
        return ORACLE_OK;
    }
    if (bits == 8) {
        int8_t *out = (int8_t *)dst;
        for (int64_t i0 = 0; i0 < n; ++i0)
            for (int64_t y = 0; y < h; ++y)
                for (int64_t x = 0; x < w; ++x)
                    for (int64_t ch = 0; ch < c; ++ch) {
                        int64_t v = oracle_saturate(src[((i0 * c + ch) * h + y) * w + x], 8, is_signed);
                        out[((i0 * h + y) * w + x) * c + ch] = (int8_t)v;
                    }
        return ORACLE_OK;
    }
    return ORACLE_EINVAL;
}

/*
 * Direct convolution, the plain definition of Sec. 2.1:
 *
 *   acc[n,p,q,k] = sum_{r<R} sum_{s<S} sum_{c<C}
 *                    x[n, p*sh - ph + r, q*sw - pw + s, c] * w[k, r, s, c]
 *
 * with x taken as 0 outside the H x W image.  x is N x H x W x C (int32
 * values), w is K x R x S x C, acc is N x P x Q x K.  Sums are formed in
 * int64; if any |acc| >= 2^31 the function returns ORACLE_EOVERFLOW.
 *
 * Only output pixels listed in `pix` (flat indices n*P*Q + p*Q + q; NULL
 * means all of them, in order) are computed; with a list, acc holds
 * npix x K values in list order.  nthreads > 1 splits the pixel loop over
 * OpenMP threads; it changes nothing in the arithmetic.
 */
int oracle_conv2d(const int32_t *x, const int32_t *wt,
                  int64_t n, int64_t h, int64_t w, int64_t c, int64_t k, int64_t r, int64_t s,
                  int64_t sh, int64_t sw, int64_t ph, int64_t pw,
                  const int64_t *pix, int64_t npix, int32_t *acc, int nthreads)
{
    int64_t p_out = oracle_out_dim(h, r, sh, ph);
    int64_t q_out = oracle_out_dim(w, s, sw, pw);
    if (n < 0 || c < 1 || k < 1 || p_out < 1 || q_out < 1)
        return ORACLE_EINVAL;
    int64_t total = n * p_out * q_out;
    if (pix == NULL)
        npix = total;
    for (int64_t t = 0; t < npix; ++t)
        if (pix != NULL && (pix[t] < 0 || pix[t] >= total))
            return ORACLE_EINVAL;

    int overflow = 0;
#ifdef _OPENMP
    if (nthreads < 1)
        nthreads = 1;
#pragma omp parallel for num_threads(nthreads) schedule(static) reduction(| : overflow)
#endif
    for (int64_t t = 0; t < npix; ++t) {
        int64_t m = pix ? pix[t] : t;
        int64_t ni = m / (p_out * q_out);
        int64_t pi = (m / q_out) % p_out;
        int64_t qi = m % q_out;
        for (int64_t ko = 0; ko < k; ++ko) {
            int64_t sum = 0;
            for (int64_t ri = 0; ri < r; ++ri) {
                int64_t yi = pi * sh - ph + ri;
                if (yi < 0 || yi >= h)
                    continue;
                for (int64_t si = 0; si < s; ++si) {
                    int64_t xi = qi * sw - pw + si;
                    if (xi < 0 || xi >= w)
                        continue;
                    const int32_t *xp = x + ((ni * h + yi) * w + xi) * c;
                    const int32_t *wp = wt + ((ko * r + ri) * s + si) * c;
                    for (int64_t ci = 0; ci < c; ++ci)
                        sum += (int64_t)xp[ci] * (int64_t)wp[ci];
                }
            }
            if (sum >= ((int64_t)1 << 31) || sum < -((int64_t)1 << 31))
                overflow = 1;
            acc[t * k + ko] = (int32_t)sum;
        }
    }
    return overflow ? ORACLE_EOVERFLOW : ORACLE_OK;
}

/* floor(a / 2^sh) for any sign of a, without relying on signed '>>'. */
static int64_t floor_div_pow2(int64_t a, int sh)
{
    int64_t d = (int64_t)1 << sh;
    int64_t q = a / d; /* C division truncates toward zero */
    if (a % d != 0 && a < 0)
        q -= 1;
    return q;
}

/*
 * The requantising epilogue, applied element by element to acc (npix x k,
 * channels innermost), in the order of Sec. 3.2.2 (epilogue on the wide
 * value, then clip):
 *
 *   t = acc * mult[ch]                    (exact, int64)
 *   t = floor((t + 2^(shift-1)) / 2^shift) (round half up)
 *   t = max(t, 0)                          if relu
 *   t = min(max(t, lo), hi)
 *
 * shift must lie in [1, 62]; returns ORACLE_EINVAL otherwise.
 */
int oracle_requant(const int32_t *acc, int64_t npix, int64_t k, const int32_t *mult,
                   int shift, int relu, int64_t lo, int64_t hi, int32_t *out)
{
    if (shift < 1 || shift > 62 || lo > hi)
        return ORACLE_EINVAL;
    for (int64_t t = 0; t < npix; ++t)
        for (int64_t ko = 0; ko < k; ++ko) {
            int64_t v = (int64_t)acc[t * k + ko] * (int64_t)mult[ko];
            v = floor_div_pow2(v + ((int64_t)1 << (shift - 1)), shift);
            if (relu && v < 0)
                v = 0;
            if (v < lo) v = lo;
            if (v > hi) v = hi;
            out[t * k + ko] = (int32_t)v;
        }
    return ORACLE_OK;
}

/*
 * The epilogue with the two additions Sec. 3.2.2 and a residual network
 * need, element by element:
 *
 *   t = (acc + bias[ch]) * mult[ch]          (exact, int64; bias may be NULL = 0)
 *   t = floor((t + 2^(shift-1)) / 2^shift)   (round half up)
 *   t = t + res[i]                           (res may be NULL = 0)
 *   t = max(t, 0)                            if relu
 *   t = min(max(t, lo), hi)
 *
 * The bias is an offset in accumulator units (a folded batch norm's shift);
 * the residual is a tensor already in the output's quantised units (the
 * shortcut of a residual block), added before ReLU and clipping.  Returns
 * ORACLE_EINVAL for shift outside [1, 62] or lo > hi.
 */
int oracle_requant_ext(const int32_t *acc, int64_t npix, int64_t k, const int32_t *mult, const int32_t *bias,
                       int shift, const int32_t *res, int relu, int64_t lo, int64_t hi, int32_t *out)
{
    if (shift < 1 || shift > 62 || lo > hi)
        return ORACLE_EINVAL;
    for (int64_t t = 0; t < npix; ++t)
        for (int64_t ko = 0; ko < k; ++ko) {
            int64_t a = (int64_t)acc[t * k + ko] + (bias ? (int64_t)bias[ko] : 0);
            int64_t v = a * (int64_t)mult[ko];
            v = floor_div_pow2(v + ((int64_t)1 << (shift - 1)), shift);
            if (res)
                v += res[t * k + ko];
            if (relu && v < 0)
                v = 0;
            if (v < lo) v = lo;
            if (v > hi) v = hi;
            out[t * k + ko] = (int32_t)v;
        }
    return ORACLE_OK;
}

/* Threads OpenMP would use by default (1 without OpenMP). */
int oracle_max_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}
