// Host side of libqconv: argument validation, sizes, tile choice and launch.
// Validation and sizing touch no device and run on any machine; only the
// launch paths call the HIP runtime.
#include <hip/hip_runtime.h>
#include <stdarg.h>
#include <stdint.h>
#include <stdio.h>
#include <string.h>

#include <algorithm>
#include <initializer_list>
#include <map>
#include <mutex>
#include <string>
#include <tuple>
#include <set>
#include <unordered_map>

#include "qconv.h"
#include "qconv_internal.h"

using namespace qconv;

// Digest of the sources and flags this library was built from (set by the
// build; a build from elsewhere says "unknown").  It is also kept as a plain
// string in the file, so a caller can check a binary without loading it.
#ifndef QCONV_SOURCE_DIGEST
#define QCONV_SOURCE_DIGEST "unknown"
#endif
__attribute__((used)) static const char kDigestMarker[] = "QCONV_SOURCE_DIGEST=" QCONV_SOURCE_DIGEST;

namespace {

thread_local char g_err[256] = "";

// Geometry of the calling thread's most recent convolution launch.
struct LaunchGeometry {
    int64_t grid = 0, threads = 0, lds = 0;
    char kernel[96] = "";
};
thread_local LaunchGeometry g_last_launch;

int fail(int code, const char *fmt, ...) __attribute__((format(printf, 2, 3)));
int fail(int code, const char *fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_err, sizeof(g_err), fmt, ap);
    va_end(ap);
    return code;
}

constexpr int64_t kLdsBytes = 160 * 1024;   // LDS per workgroup on gfx950
constexpr int64_t kUnrollLdsBytes = 64 * 1024;   // LDS the unroll kernel may stage per row
constexpr int64_t kMaxBytes = (int64_t)1 << 31;

bool aligned16(const void *p) { return ((uintptr_t)p & 15u) == 0; }

int64_t out_dim(int64_t in, int64_t win, int64_t stride, int64_t pad) {
    int64_t span = in + 2 * pad - win;
    if (span < 0) return -1;
    return span / stride + 1;
}

// Product of non-negative factors, saturated at 2^62 so that a descriptor
// with huge dimensions cannot wrap its size checks.
int64_t mul_sat(std::initializer_list<int64_t> fs) {
    constexpr int64_t kCap = (int64_t)1 << 62;
    int64_t r = 1;
    for (int64_t f : fs) {
        if (f != 0 && r > kCap / f) return kCap;
        r *= f;
    }
    return r;
}

int64_t max_abs(int bits, int is_signed) {
    if (bits == 4) return is_signed ? 8 : 15;
    return is_signed ? 128 : 255;
}

// Full descriptor validation shared by every entry point.
int check_desc(const qconv_desc *d, qconv_layout_info *info) {
    if (!d) return fail(QCONV_EINVAL, "descriptor is NULL");
    if (d->n <= 0 || d->h <= 0 || d->w <= 0 || d->c <= 0 || d->k <= 0 || d->r <= 0 || d->s <= 0)
        return fail(QCONV_EINVAL, "sizes must be positive (n=%d h=%d w=%d c=%d k=%d r=%d s=%d)", d->n, d->h, d->w,
                    d->c, d->k, d->r, d->s);
    if (d->stride_h < 1 || d->stride_w < 1) return fail(QCONV_EINVAL, "strides must be >= 1");
    if (d->pad_h < 0 || d->pad_w < 0) return fail(QCONV_EINVAL, "padding must be >= 0");
    if ((d->x_signed != 0 && d->x_signed != 1) || (d->w_signed != 0 && d->w_signed != 1))
        return fail(QCONV_EINVAL, "x_signed and w_signed must be 0 or 1");
    if (d->nb < 0 || (d->nb > 1 && d->n % d->nb != 0))
        return fail(QCONV_EINVAL, "nb must be 0, 1 or a divisor of n (n=%d nb=%d)", d->n, d->nb);
    if (d->nb > 1 && d->stride_w != 1)
        return fail(QCONV_EUNSUPPORTED, "the batch-interleaved layout needs stride_w == 1 (got %d)", d->stride_w);
    int64_t p = out_dim(d->h, d->r, d->stride_h, d->pad_h);
    int64_t q = out_dim(d->w, d->s, d->stride_w, d->pad_w);
    if (p < 1 || q < 1) return fail(QCONV_EINVAL, "filter window larger than the padded input");
    if (d->bits != 4 && d->bits != 8) return fail(QCONV_EUNSUPPORTED, "bits must be 4 or 8 (got %d)", d->bits);
    if (d->bits == 4 && (d->c % 8 || d->k % 8))
        return fail(QCONV_EUNSUPPORTED, "4-bit needs c %% 8 == 0 and k %% 8 == 0 (c=%d k=%d)", d->c, d->k);
    if (d->bits == 8 && (d->c % 4 || d->k % 4))
        return fail(QCONV_EUNSUPPORTED, "8-bit needs c %% 4 == 0 and k %% 4 == 0 (c=%d k=%d)", d->c, d->k);
    if (d->bits == 8 && (!d->x_signed || !d->w_signed))
        return fail(QCONV_EUNSUPPORTED, "8-bit operands must be signed (the int8 MFMA is signed)");
    const int64_t bits = d->bits;
    const int64_t m = mul_sat({d->n, p, q});
    const int64_t x_bytes = mul_sat({d->n, d->h, d->w, d->c, bits}) / 8;
    const int64_t w_bytes = mul_sat({d->k, d->r, d->s, d->c, bits}) / 8;
    const int64_t y_raw = mul_sat({m, d->k, 4});
    if (x_bytes >= kMaxBytes || w_bytes >= kMaxBytes || y_raw >= kMaxBytes)
        return fail(QCONV_EUNSUPPORTED, "tensors must stay below 2 GiB (32-bit indexing)");
    // every product below is now far from overflowing
    const int64_t y_packed = m * d->k * bits / 8;
    const int64_t depth = (int64_t)d->c * d->r * d->s;
    const int64_t worst = depth * max_abs(d->bits, d->x_signed) * max_abs(d->bits, d->w_signed);
    if (worst >= ((int64_t)1 << 31))
        return fail(QCONV_EUNSUPPORTED, "worst-case accumulator %lld does not fit int32", (long long)worst);
    if (d->bits == 4) {
        int64_t scaled = worst << (4 * (d->x_signed + d->w_signed));
        if (scaled >= ((int64_t)1 << 31))
            return fail(QCONV_EUNSUPPORTED, "worst-case accumulator %lld times the widening factor does not fit int32",
                        (long long)worst);
    }
    if (info) {
        info->p = (int32_t)p;
        info->q = (int32_t)q;
        info->m = m;
        info->gemm_k = depth;
        info->macs = m * d->k * depth;
        info->x_bytes = x_bytes;
        info->w_bytes = w_bytes;
        info->y_raw_bytes = y_raw;
        info->y_packed_bytes = y_packed;
        info->workspace_bytes = 0;
        info->max_abs_acc = worst;
    }
    return QCONV_OK;
}

// Validates d and gives the geometry the kernels run.  The batch-interleaved
// layout (nb > 1) is plain NHWC of n/nb images nb times as wide, in which a
// filter's columns lie nb pixels apart: padding nb*pad_w, output width q*nb
// (stride_w is 1), and kd->nb is that tap spacing.  Otherwise kd = *d, nb 1.
int kernel_desc(const qconv_desc *d, qconv_desc *kd, qconv_layout_info *kli) {
    int rc = check_desc(d, kli);
    if (rc != QCONV_OK) return rc;
    *kd = *d;
    kd->nb = d->nb > 1 ? d->nb : 1;
    if (kd->nb > 1) {
        const int64_t w = (int64_t)d->w * kd->nb, pw = (int64_t)d->pad_w * kd->nb, q = (int64_t)kli->q * kd->nb;
        if (w + 2 * pw >= (1ll << 30) || q >= (1ll << 30))
            return fail(QCONV_EUNSUPPORTED, "interleaved rows of %lld padded pixels are too wide", (long long)(w + 2 * pw));
        kd->n = d->n / kd->nb;
        kd->w = (int32_t)w;
        kd->pad_w = (int32_t)pw;
        kli->q = (int32_t)q;
    }
    return QCONV_OK;
}

int check_epilogue(const qconv_desc *d, const qconv_epilogue *e) {
    if (e && e->mode == QCONV_OUT_RAW_I32 && (e->bias || e->residual))
        return fail(QCONV_EINVAL, "bias and residual apply to the requant epilogue only");
    if (!e || e->mode == QCONV_OUT_RAW_I32) return QCONV_OK;
    if (e->residual_signed != 0 && e->residual_signed != 1) return fail(QCONV_EINVAL, "residual_signed must be 0 or 1");
    if (e->residual && !aligned16(e->residual)) return fail(QCONV_EINVAL, "residual must be 16-byte aligned");
    if (e->mode != QCONV_OUT_REQUANT) return fail(QCONV_EINVAL, "unknown epilogue mode %d", e->mode);
    if (!e->mult) return fail(QCONV_EINVAL, "requant epilogue needs a multiplier array");
    if (e->shift < 1 || e->shift > 62) return fail(QCONV_EINVAL, "shift must be in [1, 62] (got %d)", e->shift);
    if (e->relu != 0 && e->relu != 1) return fail(QCONV_EINVAL, "relu must be 0 or 1");
    if (e->clamp_lo > e->clamp_hi) return fail(QCONV_EINVAL, "clamp_lo > clamp_hi");
    const int lo = e->clamp_lo, hi = e->clamp_hi;
    bool ok;
    if (d->bits == 4)
        ok = (lo >= 0 && hi <= 15) || (lo >= -8 && hi <= 7);
    else
        ok = lo >= -128 && hi <= 127;
    if (!ok) return fail(QCONV_EINVAL, "clamp range [%d, %d] does not fit the %d-bit output", lo, hi, d->bits);
    return QCONV_OK;
}

// Padded ("virtual") row of output pixel m's first tap.
int64_t vrow_of(const qconv_desc *d, int64_t p, int64_t q, int64_t m) {
    int64_t img = m / (p * q), rem = m % (p * q);
    return img * (d->h + 2 * d->pad_h) + (rem / q) * d->stride_h;
}

// Largest number of padded rows any workgroup of tile_p pixels touches.
int64_t band_rows(const qconv_desc *d, int64_t p, int64_t q, int64_t tile_p) {
    static std::mutex mu;
    static std::unordered_map<std::string, int64_t> cache;
    // keyed by everything the result depends on: the output extent (p, q)
    // follows from both axes' strides and paddings
    char key[192];
    snprintf(key, sizeof(key), "%d,%d,%d,%d,%d,%d,%d,%d,%d,%lld,%lld,%lld", d->n, d->h, d->w, d->r, d->s, d->stride_h,
             d->stride_w, d->pad_h, d->pad_w, (long long)p, (long long)q, (long long)tile_p);
    {
        std::lock_guard<std::mutex> g(mu);
        auto it = cache.find(key);
        if (it != cache.end()) return it->second;
    }
    const int64_t m = (int64_t)d->n * p * q;
    int64_t best = 0;
    for (int64_t m0 = 0; m0 < m; m0 += tile_p) {
        int64_t last = std::min(m0 + tile_p, m) - 1;
        best = std::max(best, vrow_of(d, p, q, last) + d->r - vrow_of(d, p, q, m0));
    }
    std::lock_guard<std::mutex> g(mu);
    if (cache.size() > 4096) cache.clear();
    cache[key] = best;
    return best;
}

int64_t pad_plane(int64_t bytes) { return (bytes + 255) / 256 * 256 + 128; }

constexpr int kNumCUs = 256;   // MI355X compute units
// staging rounds of an 8-bit wide tile's band: the first is prefetched during
// the previous stage's MFMAs, the rest are loaded and written in turn
constexpr int64_t kBandRounds = 4;

struct Plan {
    int64_t rows = 0, pstride_b = 0, pstride_w = 0, lds = 0;
    int64_t off_b0 = 0, off_b1 = 0, off_w0 = 0, off_w1 = 0, off_m = 0, off_e = 0;
    int64_t mtiles = 0, ktiles = 0, grid = 0;
    int64_t splits = 1, cps = 0;   // split-K: splits of the chunk range, chunks per split
    bool proj = false;             // a fused projection (its own accumulators and partial sums)
};

int64_t round_up(int64_t v, int64_t m) { return (v + m - 1) / m * m; }

// Workgroups of this tile that fit one CU, from LDS and wave slots only.
int64_t per_cu_estimate(const qconv_tile_info &t, int64_t lds) {
    const int64_t by_lds = lds > 0 ? kLdsBytes / lds : 16;
    const int64_t by_waves = 32 / (t.threads / 64);
    return std::max<int64_t>(1, std::min<int64_t>({by_lds, by_waves, 16}));
}

// per_cu: workgroups per CU to plan the persistent grid for (0 = estimate).
// splits: requested split-K factor (wide tiles); normalised so no split is empty.
// one_band: a persistent single-chunk plan keeps one LDS band buffer (the
// kernel then adds a barrier before restaging it), so that more workgroups fit
// a CU and their phases overlap.
// ablation: the techniques switched off (bit 0 lowered staging, bit 1 LDS
// epilogue), for the measurement instances of 3x3 layers.
// proj: the filter image carries a fused 1x1 projection as one more tap, and
// the projection's multipliers and biases sit beside the layer's.
int plan_tile(const qconv_desc *d, const qconv_layout_info &li, const qconv_tile_info &t, Plan *out,
              int64_t per_cu = 0, int64_t splits = 1, bool one_band = false, int ablation = 0, bool proj = false) {
    if (t.bits != d->bits)
        return fail(QCONV_EUNSUPPORTED, "tile %s is built for %d-bit operands", t.name, t.bits);
    if ((t.x_signed >= 0 && t.x_signed != d->x_signed) || (t.w_signed >= 0 && t.w_signed != d->w_signed))
        return fail(QCONV_EUNSUPPORTED, "tile %s is built for x_signed=%d, w_signed=%d", t.name, t.x_signed, t.w_signed);
    const int64_t ncols = d->w + 2 * d->pad_w;
    const int64_t nchunks = (d->c + t.chunk_c - 1) / t.chunk_c;
    Plan pl;
    pl.proj = proj;
    pl.rows = band_rows(d, li.p, li.q, t.tile_p);
    pl.mtiles = (li.m + t.tile_p - 1) / t.tile_p;
    pl.ktiles = (d->k + t.tile_k - 1) / t.tile_k;
    if (t.variant == QCONV_VARIANT_STAGED) {
        if (splits != 1) return fail(QCONV_EUNSUPPORTED, "tile %s has no split-K", t.name);
        if (d->nb > 1) return fail(QCONV_EUNSUPPORTED, "tile %s does not read the batch-interleaved layout", t.name);
        const int64_t gran = 2 * d->bits;
        pl.pstride_b = pad_plane(pl.rows * ncols * gran);
        pl.pstride_w = pad_plane((int64_t)d->r * d->s * t.tile_k * gran);
        pl.lds = (int64_t)(t.chunk_c / 16) * (pl.pstride_b + pl.pstride_w);
        pl.grid = pl.mtiles * pl.ktiles;
    } else {
        if ((d->c * d->bits) % 128 != 0)
            return fail(QCONV_EUNSUPPORTED, "tile %s needs c*bits %% 128 == 0 (whole 16-byte vectors)", t.name);
        const int64_t vpp = (int64_t)t.chunk_c * d->bits / 128;
        const int64_t pj = wide_band_pixels_per_thread(t.tile_p, t.threads, (int)vpp);
        const bool lowered = (ablation & 1) != 0, ldsepi = (ablation & 2) != 0, packed_lds = (ablation & 4) != 0;
        if (ablation && (d->r != 3 || d->s != 3 || splits != 1 || d->nb > 1))
            return fail(QCONV_EUNSUPPORTED, "ablation instances run 3x3 filters without a split, plain layout");
        if (packed_lds && d->bits != 4)
            return fail(QCONV_EUNSUPPORTED, "only 4-bit activations are kept packed in LDS");
        const int64_t bpix = packed_lds ? 8 : 16;   // band bytes per pixel and granule plane
        const int64_t rounds = d->bits == 8 ? kBandRounds : 1;
        if (!lowered && pl.rows * ncols > rounds * (int64_t)t.threads * pj)
            return fail(QCONV_EUNSUPPORTED, "tile %s: the input band of this shape exceeds %d staging round(s)", t.name,
                        (int)rounds);
        const int64_t planes = t.chunk_c / 16;
        // plane strides: multiples of 256 bytes keep the four 16-lane groups of a
        // 16-byte LDS read in distinct banks; filter planes are whole KiB so a
        // prepared filter block is copied with 1 KiB LDS-DMA instructions
        // (the lowered operand holds every tile pixel once per tap instead)
        pl.pstride_b = lowered ? round_up((int64_t)d->r * d->s * t.tile_p * bpix, 256)
                               : round_up(pl.rows * ncols * bpix, 256);
        pl.pstride_w = round_up(((int64_t)d->r * d->s + (proj ? 1 : 0)) * t.tile_k * 16, 1024);
        const int64_t bbuf = planes * pl.pstride_b, wbuf = planes * pl.pstride_w;
        // buffer loads take 32-bit offsets, and offset 2^31 marks padding
        if (li.x_bytes >= (1ll << 31) || pl.ktiles * nchunks * wbuf >= (1ll << 31))
            return fail(QCONV_EUNSUPPORTED, "tile %s addresses operands with 31-bit buffer offsets", t.name);
        // multipliers, biases, split-K flag (and the projection's multipliers and biases)
        const int64_t mbytes0 = proj ? (int64_t)t.tile_k * 16 + 16 : round_up((int64_t)t.tile_k * 8 + 4, 16);
        const int64_t mbytes = mbytes0 + (ldsepi ? (int64_t)t.tile_p * t.tile_k * 4 : 0);   // + int32 tile
        const int64_t single = bbuf + wbuf + mbytes;
        const int64_t tiles = pl.mtiles * pl.ktiles;
        if (splits < 1 || splits > nchunks)
            return fail(QCONV_EUNSUPPORTED, "split-K factor %lld outside 1..%lld (channel chunks of tile %s)",
                        (long long)splits, (long long)nchunks, t.name);
        pl.cps = (nchunks + splits - 1) / splits;
        pl.splits = (nchunks + pl.cps - 1) / pl.cps;
        if (pl.splits > 1) {
            // one output tile per workgroup, cps chunks each
            if (pl.cps == 1) {
                pl.off_b0 = pl.off_b1 = 0;
                pl.off_w0 = pl.off_w1 = bbuf;
                pl.off_m = bbuf + wbuf;
                pl.lds = single;
            } else {
                pl.off_b0 = 0;
                pl.off_b1 = bbuf;
                pl.off_w0 = 2 * bbuf;
                pl.off_w1 = pl.off_w0 + wbuf;
                pl.off_m = pl.off_w1 + wbuf;
                pl.lds = pl.off_m + mbytes;
            }
            pl.grid = tiles * pl.splits;
        } else if (nchunks == 1 && tiles <= kNumCUs * per_cu_estimate(t, single)) {
            // every workgroup gets exactly one stage: one band buffer suffices
            pl.off_b0 = pl.off_b1 = 0;
            pl.off_w0 = pl.off_w1 = bbuf;
            pl.off_m = bbuf + wbuf;
            pl.lds = single;
            pl.grid = tiles;
        } else {
            if (one_band && nchunks == 1) {
                pl.off_b0 = pl.off_b1 = 0;
                pl.off_w0 = pl.off_w1 = bbuf;
                pl.off_m = bbuf + wbuf;
                pl.lds = single;
            } else {
                pl.off_b0 = 0;
                pl.off_b1 = bbuf;
                pl.off_w0 = 2 * bbuf;
                pl.off_w1 = pl.off_w0 + (nchunks > 1 ? wbuf : 0);
                pl.off_m = pl.off_w1 + wbuf;
                pl.lds = pl.off_m + mbytes;
            }
            const int64_t pc = per_cu > 0 ? per_cu : per_cu_estimate(t, pl.lds);
            const int64_t gpk = std::min<int64_t>(pl.mtiles, std::max<int64_t>(1, (kNumCUs * pc + pl.ktiles - 1) / pl.ktiles));
            pl.grid = gpk * pl.ktiles;
        }
    }
    if (t.variant == QCONV_VARIANT_WIDE && pl.lds > kLdsBytes && pl.off_b1 != pl.off_b0) {
        // two band buffers do not fit: keep one (the kernel then waits for every
        // wave to finish reading it before restaging; filters stay double)
        const int64_t shift_b = pl.off_b1 - pl.off_b0;
        pl.off_b1 = pl.off_b0;
        pl.off_w0 -= shift_b;
        pl.off_w1 -= shift_b;
        pl.off_m -= shift_b;
        pl.lds -= shift_b;
    }
    if (t.variant == QCONV_VARIANT_WIDE && (ablation & 2)) pl.off_e = pl.off_m + round_up((int64_t)t.tile_k * 8 + 4, 16);
    if (pl.lds > kLdsBytes)
        return fail(QCONV_EUNSUPPORTED, "tile %s needs %lld bytes of LDS for this shape (limit %lld)", t.name,
                    (long long)pl.lds, (long long)kLdsBytes);
    if (pl.grid <= 0 || pl.grid >= (1ll << 31)) return fail(QCONV_EUNSUPPORTED, "grid size out of range");
    if (out) *out = pl;
    return QCONV_OK;
}

int pick_default(const qconv_desc *d, const qconv_layout_info &li) {
    // Static heuristic: favour 64x64 wave tiles (operand reuse), the pipelined
    // kernel where it applies, and enough workgroups to cover every CU; the
    // sweep harness measures the alternatives.
    const TileEntry *tab = tile_table();
    const int nt = tile_table_size();
    int best = -1;
    double best_score = -1.0;
    for (int i = 0; i < nt; ++i) {
        const qconv_tile_info &t = tab[i].info;
        if (t.bits != d->bits) continue;
        Plan pl;
        if (plan_tile(d, li, t, &pl) != QCONV_OK) continue;
        const double tiles = (double)pl.mtiles * pl.ktiles;
        const double util = (double)li.m * d->k / (tiles * t.tile_p * t.tile_k);
        const double waves = tiles * t.threads / 64.0;
        const double fill = std::min(1.0, waves / (4.0 * kNumCUs));
        const double reuse = 2.0 * t.frag_p * t.frag_k / (t.frag_p + t.frag_k);
        const double pipe = t.variant == QCONV_VARIANT_WIDE ? 1.5 : 1.0;
        const double chunk = t.chunk_c <= d->c ? 1.0 : 0.5;
        const double score = util * fill * reuse * pipe * chunk;
        if (score > best_score) {
            best_score = score;
            best = i;
        }
    }
    return best;
}

// The layer can carry a fused 1x1 projection: a 3x3 window with padding 1, so
// its centre tap reads pixel (p*stride_h, q*stride_w), the pixel a 1x1 filter
// at the same stride without padding reads.
bool proj_shape_ok(const qconv_desc *d) {
    return d->r == 3 && d->s == 3 && d->pad_h == 1 && d->pad_w == 1 && d->nb <= 1;
}

// The built-in tile for a layer with a fused projection: the static heuristic's
// score among the tiles that have a projection instance and fit the shape.
int pick_proj_default(const qconv_desc *d, const qconv_layout_info &li) {
    const TileEntry *tab = tile_table();
    int best = -1;
    double best_score = -1.0;
    for (int i = 0; i < tile_table_size(); ++i) {
        const qconv_tile_info &t = tab[i].info;
        if (t.bits != d->bits || !proj_instance(t.name)) continue;
        Plan pl;
        if (plan_tile(d, li, t, &pl, 0, 1, false, 0, true) != QCONV_OK) continue;
        const double tiles = (double)pl.mtiles * pl.ktiles;
        const double util = (double)li.m * d->k / (tiles * t.tile_p * t.tile_k);
        const double fill = std::min(1.0, tiles * t.threads / 64.0 / (4.0 * kNumCUs));
        const double score = util * fill * (2.0 * t.frag_p * t.frag_k / (t.frag_p + t.frag_k));
        if (score > best_score) {
            best_score = score;
            best = i;
        }
    }
    return best;
}

struct DevAttrCache {
    std::mutex mu;
    std::set<std::pair<int, const void *>> done;   // (device, kernel) whose max LDS attribute is set
    // resident workgroups per CU the runtime reports, per (device, kernel, threads, LDS bytes)
    std::map<std::tuple<int, const void *, int, int64_t>, int> occupancy;
};
DevAttrCache g_attr;

}  // namespace

// ---- the device scratch of qconv2d_prepared_noalloc: the split-K workspace
// for callers that cannot allocate.  One array per device (each GPU the
// library runs on holds its own copy until the process ends).  Layout: the
// arrival counters first, at a fixed place, then the partial sums.  The
// array's name is only a host-side stand-in: host code uses the address
// hipGetSymbolAddress gives for the current device, never the name itself.
constexpr int64_t kScratchBytes = 16ll << 20;
constexpr int64_t kScratchCounterBytes = 64ll << 10;   // up to 16384 output tiles
static __device__ __align__(256) uint8_t scratch[kScratchBytes];

__global__ void __launch_bounds__(256) clear_words(uint32_t *p, int32_t n) {
    const int32_t i = (int32_t)(blockIdx.x * 256 + threadIdx.x);
    if (i < n) p[i] = 0u;   // a vector store (no scalar-cache writes)
}

namespace {

struct ScratchCache {
    std::mutex mu;
    std::unordered_map<int, uint8_t *> ptr;   // device -> its copy of `scratch`
};
ScratchCache g_scratch;

// The current device's scratch address; on the first call on a device, also
// enqueues (on `stream`) the clearing of its arrival counters, which every
// split-K launch then leaves at zero again.
int scratch_for_current_device(hipStream_t stream, uint8_t **out) {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) return fail(QCONV_EHIP, "hipGetDevice failed");
    std::lock_guard<std::mutex> g(g_scratch.mu);
    auto it = g_scratch.ptr.find(dev);
    if (it != g_scratch.ptr.end()) {
        *out = it->second;
        return QCONV_OK;
    }
    void *p = nullptr;
    hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p)
        return fail(QCONV_EHIP, "hipGetSymbolAddress(scratch): %s", hipGetErrorString(e));
    const int32_t words = (int32_t)(kScratchCounterBytes / 4);
    hipLaunchKernelGGL(clear_words, dim3((unsigned)((words + 255) / 256)), dim3(256), 0, stream,
                       static_cast<uint32_t *>(p), words);
    e = hipGetLastError();
    if (e != hipSuccess) return fail(QCONV_EHIP, "scratch clear launch: %s", hipGetErrorString(e));
    g_scratch.ptr[dev] = static_cast<uint8_t *>(p);
    *out = static_cast<uint8_t *>(p);
    return QCONV_OK;
}

}  // namespace

extern "C" {

const char *qconv_build_digest(void) { return kDigestMarker + sizeof("QCONV_SOURCE_DIGEST=") - 1; }

const char *qconv_strerror(int status) {
    switch (status) {
        case QCONV_OK: return "ok";
        case QCONV_EINVAL: return "invalid argument";
        case QCONV_EUNSUPPORTED: return "unsupported configuration";
        case QCONV_EWORKSPACE: return "workspace too small";
        case QCONV_EHIP: return "HIP runtime error";
        default: return "unknown status";
    }
}

const char *qconv_last_error(void) { return g_err; }

int qconv_layout(const qconv_desc *d, qconv_layout_info *out) {
    g_err[0] = 0;
    return check_desc(d, out);
}

int qconv_tile_count(void) { return tile_table_size(); }

int qconv_tile_get(int32_t tile_id, qconv_tile_info *out) {
    if (!out || tile_id < 0 || tile_id >= tile_table_size()) return fail(QCONV_EINVAL, "unknown tile %d", tile_id);
    *out = tile_table()[tile_id].info;
    return QCONV_OK;
}

int qconv_tile_check(const qconv_desc *d, int32_t tile_id) {
    g_err[0] = 0;
    qconv_layout_info li;
    qconv_desc kd;
    int rc = kernel_desc(d, &kd, &li);
    if (rc) return rc;
    d = &kd;
    if (tile_id < 0 || tile_id >= tile_table_size()) return fail(QCONV_EINVAL, "unknown tile %d", tile_id);
    return plan_tile(d, li, tile_table()[tile_id].info, nullptr);
}

int qconv_default_tile(const qconv_desc *d) {
    g_err[0] = 0;
    qconv_layout_info li;
    qconv_desc kd;
    int rc = kernel_desc(d, &kd, &li);
    if (rc) return rc;
    d = &kd;
    int t = pick_default(d, li);
    if (t < 0) return fail(QCONV_EUNSUPPORTED, "no compiled tile fits this shape");
    return t;
}

int qconv_pack_interleaved(const int8_t *src, void *dst, int32_t n, int32_t c, int32_t h, int32_t w, int32_t bits,
                           int32_t is_signed, int32_t nb, void *stream) {
    g_err[0] = 0;
    if (n < 0 || c < 0 || h < 0 || w < 0) return fail(QCONV_EINVAL, "sizes must be non-negative");
    if (nb < 1 || n % nb != 0) return fail(QCONV_EINVAL, "nb must be >= 1 and divide n (n=%d nb=%d)", n, nb);
    if (is_signed != 0 && is_signed != 1) return fail(QCONV_EINVAL, "is_signed must be 0 or 1");
    if (bits != 4 && bits != 8) return fail(QCONV_EUNSUPPORTED, "bits must be 4 or 8 (got %d)", bits);
    if (bits == 4 && c % 8) return fail(QCONV_EUNSUPPORTED, "4-bit packing needs c %% 8 == 0 (c=%d)", c);
    if (bits == 8 && !is_signed) return fail(QCONV_EUNSUPPORTED, "8-bit values are signed");
    const int64_t count = mul_sat({n, c, h, w});
    if (count == 0) return QCONV_OK;
    if (count >= kMaxBytes) return fail(QCONV_EUNSUPPORTED, "tensor must stay below 2^31 values");
    if (!src || !dst) return fail(QCONV_EINVAL, "src and dst must be non-NULL");
    if (((uintptr_t)dst & 3u) != 0) return fail(QCONV_EINVAL, "dst must be 4-byte aligned");
    const uintptr_t s0 = (uintptr_t)src, s1 = s0 + count;
    const uintptr_t d0 = (uintptr_t)dst, d1 = d0 + count * bits / 8;
    if (s0 < d1 && d0 < s1) return fail(QCONV_EINVAL, "src and dst overlap");
    hipError_t e = launch_pack(src, dst, n, c, h, w, bits, is_signed, nb, (hipStream_t)stream);
    if (e != hipSuccess) return fail(QCONV_EHIP, "pack launch: %s", hipGetErrorString(e));
    return QCONV_OK;
}

int qconv_pack(const int8_t *src, void *dst, int32_t n, int32_t c, int32_t h, int32_t w, int32_t bits,
               int32_t is_signed, void *stream) {
    return qconv_pack_interleaved(src, dst, n, c, h, w, bits, is_signed, 1, stream);
}

}  // extern "C"

namespace {

int resolve_tile(const qconv_desc *d, const qconv_layout_info &li, int32_t tile_id) {
    if (tile_id == -1) {
        tile_id = pick_default(d, li);
        if (tile_id < 0) return fail(QCONV_EUNSUPPORTED, "no compiled tile fits this shape");
    }
    if (tile_id < 0 || tile_id >= tile_table_size()) return fail(QCONV_EINVAL, "unknown tile %d", tile_id);
    return tile_id;
}

// Bytes of the prepared filters of `tile` for this shape: the int8 image of
// every (channel tile, chunk) block for wide tiles, the packed KRSC filters
// themselves otherwise.
int64_t prepared_bytes(const qconv_desc *d, const qconv_layout_info &li, const qconv_tile_info &t, const Plan &pl) {
    if (t.variant != QCONV_VARIANT_WIDE) return li.w_bytes;
    const int64_t nchunks = (d->c + t.chunk_c - 1) / t.chunk_c;
    return pl.ktiles * nchunks * (t.chunk_c / 16) * pl.pstride_w;
}

// Split-K workspace: int32 partial sums of every (tile, split) block in the
// kernel's register order (a fused projection's after the layer's, in each
// block), then one arrival counter per output tile.
int64_t split_part_bytes(const qconv_tile_info &t, const Plan &pl) {
    return pl.splits > 1 ? round_up(pl.mtiles * pl.ktiles * pl.splits * (int64_t)t.tile_p * t.tile_k * 4 *
                                        (pl.proj ? 2 : 1), 256)
                         : 0;
}
int64_t split_workspace_bytes(const qconv_tile_info &t, const Plan &pl) {
    return pl.splits > 1 ? split_part_bytes(t, pl) + round_up(pl.mtiles * pl.ktiles * 4, 256) : 0;
}

void fill_args(ConvArgs &a, const qconv_desc *d, const qconv_layout_info &li, const TileEntry &te, const Plan &pl) {
    memset(&a, 0, sizeof(a));
    a.n = d->n; a.h = d->h; a.w = d->w; a.c = d->c; a.k = d->k; a.r = d->r; a.s = d->s;
    a.sh = d->stride_h; a.sw = d->stride_w; a.ph = d->pad_h; a.pw = d->pad_w;
    a.p = li.p; a.q = li.q;
    a.m = (int32_t)li.m;
    a.vh = d->h + 2 * d->pad_h;
    a.ncols = d->w + 2 * d->pad_w;
    a.tap_w = d->nb > 1 ? d->nb : 1;
    a.xpix = d->c * d->bits / 8;
    a.nchunks = (d->c + te.info.chunk_c - 1) / te.info.chunk_c;
    a.vec16 = (d->c * d->bits) % 128 == 0;
    a.band_rows = (int32_t)pl.rows;
    a.xbytes = (int32_t)li.x_bytes;
    a.wbytes = (int32_t)li.w_bytes;
    a.off_b0 = (int32_t)pl.off_b0;
    a.off_b1 = (int32_t)pl.off_b1;
    a.off_w0 = (int32_t)pl.off_w0;
    a.off_w1 = (int32_t)pl.off_w1;
    a.off_m = (int32_t)pl.off_m;
    a.off_e = (int32_t)pl.off_e;
    a.pstride_b = (int32_t)pl.pstride_b;
    a.pstride_w = (int32_t)pl.pstride_w;
    a.ktiles = (int32_t)pl.ktiles;
    a.mtiles = (int32_t)pl.mtiles;
    a.splits = (int32_t)pl.splits;
    a.cps = (int32_t)(pl.cps > 0 ? pl.cps : (d->c + te.info.chunk_c - 1) / te.info.chunk_c);
    a.gpk = (int32_t)(pl.splits > 1 ? pl.mtiles : std::max<int64_t>(pl.grid / std::max<int64_t>(pl.ktiles, 1), 1));
    a.div_splits = make_fastdiv((uint32_t)std::max<int64_t>(pl.splits, 1));
    a.div_ktiles = make_fastdiv((uint32_t)std::max<int64_t>(pl.ktiles, 1));
    a.div_gpk = make_fastdiv((uint32_t)a.gpk);
    a.div_pq = make_fastdiv((uint32_t)(li.p * li.q));
    a.div_q = make_fastdiv((uint32_t)li.q);
    a.div_vh = make_fastdiv((uint32_t)a.vh);
    a.div_ncols = make_fastdiv((uint32_t)a.ncols);
    a.div_rs = make_fastdiv((uint32_t)(d->r * d->s));
    a.div_s = make_fastdiv((uint32_t)d->s);
    a.div_w = make_fastdiv((uint32_t)d->w);
    a.div_wq = make_fastdiv((uint32_t)((d->w + 3) / 4));
    a.div_brows = make_fastdiv((uint32_t)std::max<int64_t>(pl.rows, 1));
    a.div_pad2 = make_fastdiv((uint32_t)std::max<int64_t>(2 * (int64_t)d->pad_w, 1));
    a.div_rb4 = make_fastdiv((uint32_t)((std::max<int64_t>(pl.rows, 1) + 3) & ~int64_t(3)));
    a.x_signed = d->x_signed;
    a.w_signed = d->w_signed;
    // widening: unsigned nibble -> low half of a byte; signed nibble -> high half (value * 16)
    a.xmask = d->x_signed ? 0xF0F0F0F0u : 0x0F0F0F0Fu;
    a.xsl = d->x_signed ? 4 : 0;
    a.xsr = d->x_signed ? 0 : 4;
    a.wmask = d->w_signed ? 0xF0F0F0F0u : 0x0F0F0F0Fu;
    a.wsl = d->w_signed ? 4 : 0;
    a.wsr = d->w_signed ? 0 : 4;
    a.acc_shift = d->bits == 4 ? 4 * (d->x_signed + d->w_signed) : 0;
}

// Kernels that stage more than 64 KiB of LDS must opt in, once per device.
// Workgroups of `kernel` (threads, dynamic LDS bytes) that fit one CU, as the
// runtime reports them; 0 if it cannot say.  Asked once per device and shape:
// eager launches of persistent plans would otherwise query it every call.
int occupancy_per_cu(const void *kernel, int threads, int64_t lds) {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) return 0;
    const auto key = std::make_tuple(dev, kernel, threads, lds);
    {
        std::lock_guard<std::mutex> g(g_attr.mu);
        const auto it = g_attr.occupancy.find(key);
        if (it != g_attr.occupancy.end()) return it->second;
    }
    int occ = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&occ, kernel, threads, (size_t)lds) != hipSuccess) return 0;
    std::lock_guard<std::mutex> g(g_attr.mu);
    g_attr.occupancy[key] = occ;
    return occ;
}

int ensure_lds_attribute(const void *kernel, int64_t lds) {
    if (lds <= 64 * 1024) return QCONV_OK;
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) return fail(QCONV_EHIP, "hipGetDevice failed");
    std::lock_guard<std::mutex> g(g_attr.mu);
    if (!g_attr.done.count({dev, kernel})) {
        hipError_t e = hipFuncSetAttribute(kernel, hipFuncAttributeMaxDynamicSharedMemorySize, (int)kLdsBytes);
        if (e != hipSuccess) return fail(QCONV_EHIP, "hipFuncSetAttribute: %s", hipGetErrorString(e));
        g_attr.done.insert({dev, kernel});
    }
    return QCONV_OK;
}

// The workgroup order of xcd_order -1 (the library's choice).  Each XCD has
// its own L2, so bytes are fetched once per XCD that reads them.  Ordered
// pixel tile by pixel tile, every XCD reads every channel tile's filters and
// an eighth of the input; ordered channel tile by channel tile, every XCD
// reads its channel tiles' filters and (with at least eight channel tiles)
// all of the input.  The order with fewer such bytes wins: channel tiles for
// deep layers, whose filters outweigh their input.
int auto_xcd_order(const qconv_layout_info &li, const Plan &pl, int64_t filter_bytes) {
    if (pl.ktiles < 2) return 1;
    const int64_t k = std::min<int64_t>(pl.ktiles, 8);
    const int64_t pixel_major = 8 * filter_bytes + li.x_bytes;
    const int64_t channel_major = filter_bytes + k * li.x_bytes;
    return channel_major < pixel_major ? 2 : 1;
}

// The convolution; w is packed KRSC filters (prepared == false) or the
// prepared filters of tile_id (prepared == true, w_bytes_given bytes).
// splits > 1 (prepared filters only): split-K over channel chunks with its
// workspace in `workspace`.
// wg_per_cu, band_buffers, xcd_order: the launch knobs of a qconv_schedule.
// x_nchw (then x is unused): int8 N x C x H x W activations, packed on the way
// by the tile's fused instance, which also writes the packed copy to x_packed
// when that is not null.
int run_conv(const qconv_desc *d, const void *x, const void *w, bool prepared, size_t w_bytes_given,
             const qconv_epilogue *epi, void *y, void *workspace, size_t workspace_bytes, int32_t tile_id,
             int32_t splits, void *stream, int32_t wg_per_cu = 0, int32_t band_buffers = 0,
             int32_t xcd_order = -1, int32_t ablation = 0, const int8_t *x_nchw = nullptr,
             void *x_packed = nullptr, bool noalloc = false, const qconv_epilogue *epi_proj = nullptr,
             void *y_proj = nullptr) {
    qconv_layout_info li;
    qconv_desc kd;
    int rc = kernel_desc(d, &kd, &li);
    if (rc) return rc;
    d = &kd;
    rc = check_epilogue(d, epi);
    if (rc) return rc;
    // the fused pack reads int8 NCHW activations (n*c*h*w bytes) instead of packed ones
    const bool fused = x_nchw != nullptr;
    if (fused) x = x_nchw;
    const int64_t xin_bytes = fused ? (int64_t)d->n * d->nb * d->c * d->h * (d->w / d->nb) : li.x_bytes;
    if (!x || !w || !y) return fail(QCONV_EINVAL, "x, w and y must be non-NULL");
    if (!aligned16(x) || !aligned16(w) || !aligned16(y)) return fail(QCONV_EINVAL, "x, w and y must be 16-byte aligned");
    if ((int64_t)workspace_bytes < li.workspace_bytes)
        return fail(QCONV_EWORKSPACE, "workspace of %zu bytes, need %lld", workspace_bytes,
                    (long long)li.workspace_bytes);
    // a fused 1x1 projection (y_proj): same input, stride, channels and mode, its own epilogue
    const bool proj = y_proj != nullptr;
    if (proj) {
        if (!proj_shape_ok(d))
            return fail(QCONV_EUNSUPPORTED, "a fused projection needs a 3x3 layer with padding 1 in the plain layout");
        rc = check_epilogue(d, epi_proj);
        if (rc) return rc;
        const int m1 = epi ? epi->mode : QCONV_OUT_RAW_I32, m2 = epi_proj ? epi_proj->mode : QCONV_OUT_RAW_I32;
        if (m1 != m2) return fail(QCONV_EINVAL, "the layer and its projection must use the same epilogue mode");
        if ((epi && epi->residual) || (epi_proj && epi_proj->residual))
            return fail(QCONV_EUNSUPPORTED, "a layer with a fused projection takes no residual");
        if (!prepared || ablation || x_nchw)
            return fail(QCONV_EUNSUPPORTED, "a fused projection runs from prepared filters, without ablation");
        if (!aligned16(y_proj)) return fail(QCONV_EINVAL, "y_proj must be 16-byte aligned");
        if (tile_id == -1) {
            tile_id = pick_proj_default(d, li);
            if (tile_id < 0) return fail(QCONV_EUNSUPPORTED, "no tile with a projection instance fits this shape");
        }
    }
    rc = resolve_tile(d, li, tile_id);
    if (rc < 0) return rc;
    tile_id = rc;
    const TileEntry &te = tile_table()[tile_id];
    Plan pl;
    if (ablation && (!prepared || te.info.variant != QCONV_VARIANT_WIDE || !ablation_instance(te.info.name, ablation)))
        return fail(QCONV_EUNSUPPORTED, "no ablation instance %d of tile %s", ablation, te.info.name);
    const ProjInstance *pi = proj ? proj_instance(te.info.name) : nullptr;
    if (proj && !pi) return fail(QCONV_EUNSUPPORTED, "tile %s has no projection instance", te.info.name);
    rc = plan_tile(d, li, te.info, &pl, 0, splits, false, ablation, proj);
    if (rc) return rc;
    int64_t wsb = split_workspace_bytes(te.info, pl);
    uint8_t *ws_cnt = nullptr;   // noalloc: the scratch's counters (its partial sums are `workspace`)
    if (noalloc && wsb > 0) {
        // the library's own scratch: counters at its start, partial sums after them
        const int64_t part = split_part_bytes(te.info, pl), tiles = pl.mtiles * pl.ktiles;
        if (tiles * 4 > kScratchCounterBytes || part > kScratchBytes - kScratchCounterBytes)
            return fail(QCONV_EWORKSPACE, "split-K of %lld tiles x %lld splits needs %lld bytes of partial sums and "
                        "%lld counters; the no-alloc scratch holds %lld bytes and %lld counters",
                        (long long)tiles, (long long)pl.splits, (long long)part, (long long)tiles,
                        (long long)(kScratchBytes - kScratchCounterBytes), (long long)(kScratchCounterBytes / 4));
        uint8_t *base = nullptr;
        rc = scratch_for_current_device((hipStream_t)stream, &base);
        if (rc) return rc;
        ws_cnt = base;
        workspace = base + kScratchCounterBytes;
        workspace_bytes = (size_t)part;
        wsb = part;
    }
    if (wsb > 0) {
        if (!workspace || (int64_t)workspace_bytes < wsb)
            return fail(QCONV_EWORKSPACE, "split-K workspace of %zu bytes, need %lld", workspace ? workspace_bytes : 0,
                        (long long)wsb);
        if (!aligned16(workspace)) return fail(QCONV_EINVAL, "workspace must be 16-byte aligned");
    }
    const int64_t wb = prepared ? prepared_bytes(d, li, te.info, pl) : li.w_bytes;
    if (prepared && (int64_t)w_bytes_given < wb)
        return fail(QCONV_EINVAL, "prepared filters of %zu bytes, tile %s needs %lld", w_bytes_given, te.info.name,
                    (long long)wb);
    if (wb >= kMaxBytes) return fail(QCONV_EUNSUPPORTED, "filter image must stay below 2 GiB");
    const bool requant = epi && epi->mode == QCONV_OUT_REQUANT;
    const int64_t ybytes = requant ? li.y_packed_bytes : li.y_raw_bytes;
    const uintptr_t y0 = (uintptr_t)y, y1 = y0 + ybytes;
    if (((uintptr_t)x < y1 && y0 < (uintptr_t)x + xin_bytes) || ((uintptr_t)w < y1 && y0 < (uintptr_t)w + wb))
        return fail(QCONV_EINVAL, "y overlaps x or w");
    if (wsb > 0) {
        const uintptr_t w0 = (uintptr_t)workspace, w1 = w0 + wsb;
        if ((w0 < y1 && y0 < w1) || ((uintptr_t)x < w1 && w0 < (uintptr_t)x + xin_bytes) ||
            ((uintptr_t)w < w1 && w0 < (uintptr_t)w + wb))
            return fail(QCONV_EINVAL, "workspace overlaps x, w or y");
    }
    if (proj) {
        const uintptr_t p0 = (uintptr_t)y_proj, p1 = p0 + ybytes;
        if ((p0 < y1 && y0 < p1) || ((uintptr_t)x < p1 && p0 < (uintptr_t)x + xin_bytes) ||
            ((uintptr_t)w < p1 && p0 < (uintptr_t)w + wb) ||
            (wsb > 0 && (uintptr_t)workspace < p1 && p0 < (uintptr_t)workspace + wsb))
            return fail(QCONV_EINVAL, "y_proj overlaps x, w, y or the workspace");
    }
    if (requant && epi->residual) {
        // each lane reads its own output words of the residual before storing
        // them, so y itself may be the residual; any other overlap may not
        const uintptr_t r0 = (uintptr_t)epi->residual, r1 = r0 + ybytes;
        if (r0 != y0 && r0 < y1 && y0 < r1) return fail(QCONV_EINVAL, "residual overlaps y without being y");
        if (((uintptr_t)x < r1 && r0 < (uintptr_t)x + xin_bytes) || ((uintptr_t)w < r1 && r0 < (uintptr_t)w + wb))
            return fail(QCONV_EINVAL, "residual overlaps x or w");
        if (wsb > 0 && (uintptr_t)workspace < r1 && r0 < (uintptr_t)workspace + wsb)
            return fail(QCONV_EINVAL, "residual overlaps the workspace");
    }
    // the epilogue flavour: bias and residual are compiled into separate kernels;
    // prepared filters of a 3x3 or 1x1 layer run the tile's fixed-size instance
    // (whose taps are one column apart: not for 3x3 in the interleaved layout)
    const bool ext = requant && (epi->bias || epi->residual || (proj && epi_proj->bias));
    if (ablation && ext) return fail(QCONV_EUNSUPPORTED, "ablation instances have no bias or residual epilogue");
    const KernelSet &ks = ext ? te.ext : te.plain;
    ConvLauncher launch = ks.launch;
    const void *kernel = ks.kernel;
    const FixedInstance *single = nullptr;   // the fixed-size instance whose single-stage copy may run
    if (prepared && te.info.variant == QCONV_VARIANT_WIDE)
        for (int i = 0; i < 2; ++i)
            if (ks.fixed[i].launch && ks.fixed[i].r == d->r && ks.fixed[i].s == d->s && (d->nb == 1 || d->s == 1)) {
                // several channel chunks per workgroup: the instance that spreads
                // the next chunk's filter copies over the MFMA loop
                const bool mc = pl.cps > 1 && ks.fixed[i].launch_mc;
                launch = mc ? ks.fixed[i].launch_mc : ks.fixed[i].launch;
                kernel = mc ? ks.fixed[i].kernel_mc : ks.fixed[i].kernel;
                single = mc ? nullptr : &ks.fixed[i];
            }
    if (pi) {
        const FixedInstance &fi = ext ? pi->ext : pi->plain;
        launch = fi.launch;
        kernel = fi.kernel;
        single = &fi;
    }
    if (ablation) {
        const AblationInstance *ai = ablation_instance(te.info.name, ablation);
        launch = ai->launch;
        kernel = ai->kernel;
        single = nullptr;
    }
    if (fused) {
        if (!prepared || !te.fused.launch || d->r != te.fused.r || d->s != te.fused.s || ext || ablation || d->nb != 1)
            return fail(QCONV_EUNSUPPORTED, "the fused pack runs %s's 3x3 instance from prepared filters, plain "
                        "layout, without bias, residual or ablation", te.info.name);
        if (xin_bytes >= kMaxBytes) return fail(QCONV_EUNSUPPORTED, "int8 activations must stay below 2 GiB");
        if (x_packed) {
            // every input row must lie in some tile's band (windows that touch,
            // reaching the last row) for the packed copy to be complete
            if (d->stride_h > d->r || (int64_t)(li.p - 1) * d->stride_h + d->r - d->pad_h < d->h)
                return fail(QCONV_EUNSUPPORTED, "the bands of this shape skip input rows: no packed copy");
            if (!aligned16(x_packed)) return fail(QCONV_EINVAL, "x_packed must be 16-byte aligned");
            const uintptr_t p0 = (uintptr_t)x_packed, p1 = p0 + li.x_bytes;
            auto hits = [&](const void *q, int64_t bytes) {
                return q && (uintptr_t)q < p1 && p0 < (uintptr_t)q + bytes;
            };
            if (hits(x, xin_bytes) || hits(w, wb) || hits(y, ybytes) || (wsb > 0 && hits(workspace, wsb)))
                return fail(QCONV_EINVAL, "x_packed overlaps another operand");
        }
        launch = te.fused.launch;
        kernel = te.fused.kernel;
        single = &te.fused;
    }
    if (te.info.variant == QCONV_VARIANT_WIDE && pl.splits == 1 && pl.off_b1 != pl.off_b0) {
        // persistent grid: size it by the occupancy the runtime reports for this kernel
        rc = ensure_lds_attribute(kernel, pl.lds);
        if (rc) return rc;
        const int occ = occupancy_per_cu(kernel, te.info.threads, pl.lds);
        // a single-chunk layer whose second band buffer is what keeps another
        // workgroup off the CU runs with one band buffer instead (automatic
        // choice; band_buffers forces either)
        Plan one;
        const bool one_ok =
            plan_tile(d, li, te.info, &one, 0, 1, true, ablation, proj) == QCONV_OK && one.lds < pl.lds;
        const int occ1 = one_ok ? occupancy_per_cu(kernel, te.info.threads, one.lds) : 0;
        const bool use_one = band_buffers == 1 ? one_ok : (band_buffers == 2 ? false : one_ok && occ > 0 && occ1 > occ);
        const int pc = wg_per_cu > 0 ? wg_per_cu : (use_one ? occ1 : occ);
        if (pc > 0 || use_one) {
            rc = plan_tile(d, li, te.info, &pl, pc > 0 ? pc : 0, 1, use_one, ablation, proj);
            if (rc) return rc;
        }
    }
    ConvArgs a;
    fill_args(a, d, li, te, pl);
    a.xptr = static_cast<const uint8_t *>(x);
    if (fused) {
        a.xsrc = x_nchw;
        a.xsrc_bytes = (int32_t)xin_bytes;
        a.xpk = static_cast<uint8_t *>(x_packed);
    }
    a.wptr = static_cast<const uint8_t *>(w);
    a.yptr = static_cast<uint8_t *>(y);
    a.mult = requant ? epi->mult : nullptr;
    a.w_image = (prepared && te.info.variant == QCONV_VARIANT_WIDE) ? 1 : 0;
    a.xcd_order = xcd_order >= 0 ? xcd_order : auto_xcd_order(li, pl, a.w_image ? wb : li.w_bytes);
    if (wsb > 0) {
        a.ws_part = static_cast<int32_t *>(workspace);
        a.ws_cnt = reinterpret_cast<uint32_t *>(ws_cnt ? ws_cnt
                                                       : static_cast<uint8_t *>(workspace) + split_part_bytes(te.info, pl));
    }
    if (a.w_image) a.wbytes = (int32_t)wb;
    a.mode = requant ? QCONV_OUT_REQUANT : QCONV_OUT_RAW_I32;
    if (requant) {
        a.bias = epi->bias;
        a.res = static_cast<const uint8_t *>(epi->residual);
        a.res_signed = epi->residual_signed;
        a.shift = epi->shift;
        a.lo = epi->relu ? std::max(epi->clamp_lo, 0) : epi->clamp_lo;
        a.hi = epi->clamp_hi;
        if (a.lo > a.hi) a.lo = a.hi;   // relu with an all-negative clamp range: every value is clamp_hi
    }
    if (proj) {
        a.yproj = static_cast<uint8_t *>(y_proj);
        if (requant) {
            a.mult2 = epi_proj->mult;
            a.bias2 = epi_proj->bias;
            a.shift2 = epi_proj->shift;
            a.lo2 = epi_proj->relu ? std::max(epi_proj->clamp_lo, 0) : epi_proj->clamp_lo;
            a.hi2 = epi_proj->clamp_hi;
            if (a.lo2 > a.hi2) a.lo2 = a.hi2;
        }
    }
    // every workgroup runs one stage (at most one tile, one chunk): the
    // instance's single-stage copy
    if (single && single->launch_one && pl.cps == 1 && (pl.splits > 1 || pl.grid >= pl.mtiles * pl.ktiles)) {
        const bool oct = fused && single->launch_one_oct && d->w % 8 == 0;
        launch = oct ? single->launch_one_oct : single->launch_one;
        kernel = oct ? single->kernel_one_oct : single->kernel_one;
    }
    rc = ensure_lds_attribute(kernel, pl.lds);
    if (rc) return rc;
    hipError_t e = launch(a, dim3((unsigned)pl.grid), (size_t)pl.lds, (hipStream_t)stream);
    if (e != hipSuccess) return fail(QCONV_EHIP, "conv launch (%s): %s", te.info.name, hipGetErrorString(e));
    g_last_launch.grid = pl.grid;
    g_last_launch.threads = te.info.threads;
    g_last_launch.lds = pl.lds;
    snprintf(g_last_launch.kernel, sizeof(g_last_launch.kernel), "%s", te.info.name);
    return QCONV_OK;
}

}  // namespace

extern "C" {

int qconv2d(const qconv_desc *d, const void *x, const void *w, const qconv_epilogue *epi, void *y, void *workspace,
            size_t workspace_bytes, int32_t tile_id, void *stream) {
    g_err[0] = 0;
    return run_conv(d, x, w, false, 0, epi, y, workspace, workspace_bytes, tile_id, 1, stream);
}

static int check_schedule_knobs(const qconv_schedule *s) {
    if (!s) return fail(QCONV_EINVAL, "schedule must be non-NULL");
    if (s->wg_per_cu < 0 || s->wg_per_cu > 16) return fail(QCONV_EINVAL, "wg_per_cu must be in [0, 16]");
    if (s->band_buffers < 0 || s->band_buffers > 2) return fail(QCONV_EINVAL, "band_buffers must be 0, 1 or 2");
    if (s->xcd_order < -1 || s->xcd_order > 2) return fail(QCONV_EINVAL, "xcd_order must be -1, 0, 1 or 2");
    if (s->ablation < 0 || s->ablation > 7) return fail(QCONV_EINVAL, "ablation must be in [0, 7]");
    if (s->splits < 1) return fail(QCONV_EUNSUPPORTED, "splits must be >= 1");
    return QCONV_OK;
}

int qconv_schedule_check(const qconv_desc *d, const qconv_schedule *s) {
    g_err[0] = 0;
    int rc = check_schedule_knobs(s);
    if (rc) return rc;
    qconv_layout_info li;
    qconv_desc kd;
    rc = kernel_desc(d, &kd, &li);
    if (rc) return rc;
    d = &kd;
    rc = resolve_tile(d, li, s->tile_id);
    if (rc < 0) return rc;
    const qconv_tile_info &t = tile_table()[rc].info;
    if (s->ablation && (t.variant != QCONV_VARIANT_WIDE || !ablation_instance(t.name, s->ablation)))
        return fail(QCONV_EUNSUPPORTED, "no ablation instance %d of tile %s", s->ablation, t.name);
    return plan_tile(d, li, t, nullptr, 0, s->splits, false, s->ablation);
}

int qconv2d_scheduled(const qconv_desc *d, const void *x, const void *w_prepared, size_t w_prepared_bytes,
                      const qconv_epilogue *epi, void *y, const qconv_schedule *s, void *workspace,
                      size_t workspace_bytes, void *stream) {
    g_err[0] = 0;
    int rc = check_schedule_knobs(s);
    if (rc) return rc;
    return run_conv(d, x, w_prepared, true, w_prepared_bytes, epi, y, workspace, workspace_bytes, s->tile_id,
                    s->splits, stream, s->wg_per_cu, s->band_buffers, s->xcd_order, s->ablation);
}

int qconv_workspace_bytes(const qconv_desc *d, int32_t tile_id, int32_t splits, size_t *bytes) {
    g_err[0] = 0;
    qconv_layout_info li;
    qconv_desc kd;
    int rc = kernel_desc(d, &kd, &li);
    if (rc) return rc;
    d = &kd;
    if (!bytes) return fail(QCONV_EINVAL, "bytes must be non-NULL");
    rc = resolve_tile(d, li, tile_id);
    if (rc < 0) return rc;
    Plan pl;
    const TileEntry &te = tile_table()[rc];
    int prc = plan_tile(d, li, te.info, &pl, 0, splits);
    if (prc) return prc;
    *bytes = (size_t)split_workspace_bytes(te.info, pl);
    return QCONV_OK;
}

int qconv_max_splits(const qconv_desc *d, int32_t tile_id) {
    g_err[0] = 0;
    qconv_layout_info li;
    qconv_desc kd;
    int rc = kernel_desc(d, &kd, &li);
    if (rc) return rc;
    d = &kd;
    rc = resolve_tile(d, li, tile_id);
    if (rc < 0) return rc;
    const qconv_tile_info &t = tile_table()[rc].info;
    if (t.variant != QCONV_VARIANT_WIDE) return 1;
    return (d->c + t.chunk_c - 1) / t.chunk_c;
}

int qconv_prepared_filter_bytes(const qconv_desc *d, int32_t tile_id, size_t *bytes) {
    g_err[0] = 0;
    qconv_layout_info li;
    qconv_desc kd;
    int rc = kernel_desc(d, &kd, &li);
    if (rc) return rc;
    d = &kd;
    if (!bytes) return fail(QCONV_EINVAL, "bytes must be non-NULL");
    rc = resolve_tile(d, li, tile_id);
    if (rc < 0) return rc;
    Plan pl;
    const TileEntry &te = tile_table()[rc];
    int prc = plan_tile(d, li, te.info, &pl);
    if (prc) return prc;
    *bytes = (size_t)prepared_bytes(d, li, te.info, pl);
    return QCONV_OK;
}

int qconv_prepare_filters(const qconv_desc *d, const void *w_packed, int32_t tile_id, void *w_prepared,
                          size_t bytes, void *stream) {
    g_err[0] = 0;
    qconv_layout_info li;
    qconv_desc kd;
    int rc = kernel_desc(d, &kd, &li);
    if (rc) return rc;
    d = &kd;
    if (!w_packed || !w_prepared) return fail(QCONV_EINVAL, "filter pointers must be non-NULL");
    if (!aligned16(w_packed) || !aligned16(w_prepared)) return fail(QCONV_EINVAL, "filters must be 16-byte aligned");
    rc = resolve_tile(d, li, tile_id);
    if (rc < 0) return rc;
    tile_id = rc;
    const TileEntry &te = tile_table()[tile_id];
    Plan pl;
    rc = plan_tile(d, li, te.info, &pl);
    if (rc) return rc;
    const int64_t need = prepared_bytes(d, li, te.info, pl);
    if ((int64_t)bytes < need)
        return fail(QCONV_EINVAL, "prepared filter buffer of %zu bytes, need %lld", bytes, (long long)need);
    const uintptr_t s0 = (uintptr_t)w_packed, s1 = s0 + li.w_bytes, d0 = (uintptr_t)w_prepared, d1 = d0 + need;
    if (s0 < d1 && d0 < s1) return fail(QCONV_EINVAL, "packed and prepared filters overlap");
    hipError_t e;
    if (te.info.variant == QCONV_VARIANT_WIDE) {
        ConvArgs a;
        fill_args(a, d, li, te, pl);
        a.wptr = static_cast<const uint8_t *>(w_packed);
        e = te.prep(a, static_cast<uint8_t *>(w_prepared), need / 16, nullptr, (hipStream_t)stream);
    } else {
        e = hipMemcpyAsync(w_prepared, w_packed, (size_t)li.w_bytes, hipMemcpyDeviceToDevice, (hipStream_t)stream);
    }
    if (e != hipSuccess) return fail(QCONV_EHIP, "prepare filters (%s): %s", te.info.name, hipGetErrorString(e));
    return QCONV_OK;
}

int qconv2d_prepared(const qconv_desc *d, const void *x, const void *w_prepared, size_t w_prepared_bytes,
                     const qconv_epilogue *epi, void *y, int32_t tile_id, int32_t splits, void *workspace,
                     size_t workspace_bytes, void *stream) {
    g_err[0] = 0;
    return run_conv(d, x, w_prepared, true, w_prepared_bytes, epi, y, workspace, workspace_bytes, tile_id, splits,
                    stream);
}

int qconv2d_prepared_noalloc(const qconv_desc *d, const void *x, const void *w_prepared, size_t w_prepared_bytes,
                             const qconv_epilogue *epi, void *y, int32_t tile_id, int32_t splits, void *stream) {
    g_err[0] = 0;
    return run_conv(d, x, w_prepared, true, w_prepared_bytes, epi, y, nullptr, 0, tile_id, splits, stream, 0, 0, -1, 0,
                    nullptr, nullptr, true);
}

// The tile a layer with a fused projection runs (tile_id, or the built-in
// choice for -1) and its plan; the descriptor is already the kernel's.
static int proj_tile_plan(const qconv_desc *d, const qconv_layout_info &li, int32_t tile_id, Plan *pl,
                          int32_t splits = 1) {
    if (!proj_shape_ok(d))
        return fail(QCONV_EUNSUPPORTED, "a fused projection needs a 3x3 layer with padding 1 in the plain layout");
    if (tile_id == -1) {
        tile_id = pick_proj_default(d, li);
        if (tile_id < 0) return fail(QCONV_EUNSUPPORTED, "no tile with a projection instance fits this shape");
    }
    if (tile_id < 0 || tile_id >= tile_table_size()) return fail(QCONV_EINVAL, "unknown tile %d", tile_id);
    const qconv_tile_info &t = tile_table()[tile_id].info;
    if (!proj_instance(t.name)) return fail(QCONV_EUNSUPPORTED, "tile %s has no projection instance", t.name);
    int rc = plan_tile(d, li, t, pl, 0, splits, false, 0, true);
    return rc ? rc : tile_id;
}

int qconv_proj_workspace_bytes(const qconv_desc *d, int32_t tile_id, int32_t splits, size_t *bytes) {
    g_err[0] = 0;
    qconv_layout_info li;
    qconv_desc kd;
    int rc = kernel_desc(d, &kd, &li);
    if (rc) return rc;
    if (!bytes) return fail(QCONV_EINVAL, "bytes must be non-NULL");
    Plan pl;
    rc = proj_tile_plan(&kd, li, tile_id, &pl, splits);
    if (rc < 0) return rc;
    *bytes = (size_t)split_workspace_bytes(tile_table()[rc].info, pl);
    return QCONV_OK;
}

int qconv_proj_default_tile(const qconv_desc *d) {
    g_err[0] = 0;
    qconv_layout_info li;
    qconv_desc kd;
    int rc = kernel_desc(d, &kd, &li);
    if (rc) return rc;
    Plan pl;
    return proj_tile_plan(&kd, li, -1, &pl);
}

int qconv_proj_tile_check(const qconv_desc *d, int32_t tile_id) {
    g_err[0] = 0;
    if (tile_id < 0) return fail(QCONV_EINVAL, "unknown tile %d", tile_id);
    qconv_layout_info li;
    qconv_desc kd;
    int rc = kernel_desc(d, &kd, &li);
    if (rc) return rc;
    Plan pl;
    rc = proj_tile_plan(&kd, li, tile_id, &pl);
    return rc < 0 ? rc : QCONV_OK;
}

int qconv_prepared_proj_filter_bytes(const qconv_desc *d, int32_t tile_id, size_t *bytes) {
    g_err[0] = 0;
    qconv_layout_info li;
    qconv_desc kd;
    int rc = kernel_desc(d, &kd, &li);
    if (rc) return rc;
    if (!bytes) return fail(QCONV_EINVAL, "bytes must be non-NULL");
    Plan pl;
    rc = proj_tile_plan(&kd, li, tile_id, &pl);
    if (rc < 0) return rc;
    *bytes = (size_t)prepared_bytes(&kd, li, tile_table()[rc].info, pl);
    return QCONV_OK;
}

int qconv_prepare_filters_proj(const qconv_desc *d, const void *w_packed, const void *w_proj_packed, int32_t tile_id,
                               void *w_prepared, size_t bytes, void *stream) {
    g_err[0] = 0;
    qconv_layout_info li;
    qconv_desc kd;
    int rc = kernel_desc(d, &kd, &li);
    if (rc) return rc;
    d = &kd;
    if (!w_packed || !w_proj_packed || !w_prepared) return fail(QCONV_EINVAL, "filter pointers must be non-NULL");
    if (!aligned16(w_packed) || !aligned16(w_proj_packed) || !aligned16(w_prepared))
        return fail(QCONV_EINVAL, "filters must be 16-byte aligned");
    Plan pl;
    rc = proj_tile_plan(d, li, tile_id, &pl);
    if (rc < 0) return rc;
    const TileEntry &te = tile_table()[rc];
    const int64_t need = prepared_bytes(d, li, te.info, pl);
    if ((int64_t)bytes < need)
        return fail(QCONV_EINVAL, "prepared filter buffer of %zu bytes, need %lld", bytes, (long long)need);
    const int64_t proj_bytes = li.w_bytes / (d->r * d->s);   // k x 1 x 1 x c packed
    const uintptr_t d0 = (uintptr_t)w_prepared, d1 = d0 + need;
    const uintptr_t s0 = (uintptr_t)w_packed, s1 = s0 + li.w_bytes;
    const uintptr_t p0 = (uintptr_t)w_proj_packed, p1 = p0 + proj_bytes;
    if ((s0 < d1 && d0 < s1) || (p0 < d1 && d0 < p1)) return fail(QCONV_EINVAL, "packed and prepared filters overlap");
    ConvArgs a;
    fill_args(a, d, li, te, pl);
    a.wptr = static_cast<const uint8_t *>(w_packed);
    hipError_t e = te.prep(a, static_cast<uint8_t *>(w_prepared), need / 16,
                           static_cast<const uint8_t *>(w_proj_packed), (hipStream_t)stream);
    if (e != hipSuccess) return fail(QCONV_EHIP, "prepare filters (%s): %s", te.info.name, hipGetErrorString(e));
    return QCONV_OK;
}

int qconv2d_proj(const qconv_desc *d, const void *x, const void *w_prepared, size_t w_prepared_bytes,
                 const qconv_epilogue *epi, void *y, const qconv_epilogue *epi_proj, void *y_proj, int32_t tile_id,
                 int32_t splits, void *workspace, size_t workspace_bytes, void *stream) {
    g_err[0] = 0;
    if (!y_proj) return fail(QCONV_EINVAL, "y_proj must be non-NULL");
    return run_conv(d, x, w_prepared, true, w_prepared_bytes, epi, y, workspace, workspace_bytes, tile_id, splits,
                    stream, 0, 0, -1, 0, nullptr, nullptr, false, epi_proj, y_proj);
}

int qconv_noalloc_limits(int64_t *scratch_bytes, int64_t *max_tiles) {
    g_err[0] = 0;
    if (scratch_bytes) *scratch_bytes = kScratchBytes - kScratchCounterBytes;
    if (max_tiles) *max_tiles = kScratchCounterBytes / 4;
    return QCONV_OK;
}

int qconv2d_packing(const qconv_desc *d, const int8_t *x_nchw, void *x_packed, const void *w_prepared,
                    size_t w_prepared_bytes, const qconv_epilogue *epi, void *y, int32_t tile_id, void *stream) {
    g_err[0] = 0;
    if (!x_nchw) return fail(QCONV_EINVAL, "x_nchw must be non-NULL");
    return run_conv(d, nullptr, w_prepared, true, w_prepared_bytes, epi, y, nullptr, 0, tile_id, 1, stream, 0, 0, -1,
                    0, x_nchw, x_packed);
}

int qconv_unroll(const int8_t *src, int8_t *dst, int32_t n, int32_t c, int32_t h, int32_t w, int32_t taps_h,
                 int32_t stride_h, int32_t pad_h, int32_t out_h, int32_t taps_w, int32_t stride_w, int32_t pad_w,
                 int32_t c_out, void *stream) {
    g_err[0] = 0;
    if (n < 0 || c < 0 || h < 0 || w < 0 || out_h < 0) return fail(QCONV_EINVAL, "sizes must be >= 0");
    if (taps_h < 1 || taps_w < 1 || stride_h < 1 || stride_w < 1 || pad_h < 0 || pad_w < 0)
        return fail(QCONV_EINVAL, "taps and strides must be >= 1, pads >= 0");
    if (c_out < 16 || c_out % 16 != 0) return fail(QCONV_EINVAL, "c_out must be a positive multiple of 16");
    const int64_t real = (int64_t)taps_h * taps_w * c;
    if (real > c_out) return fail(QCONV_EINVAL, "taps_h * taps_w * c (%lld) exceeds c_out (%d)", (long long)real, c_out);
    const int64_t span = (int64_t)w + 2 * pad_w - taps_w;
    if (span < 0) return fail(QCONV_EINVAL, "filter width larger than the padded input");
    const int64_t wout = span / stride_w + 1;
    const int64_t in_bytes = mul_sat({n, c, h, w}), out_bytes = mul_sat({n, out_h, wout, c_out});
    if (out_bytes == 0) return QCONV_OK;
    if (in_bytes >= ((int64_t)1 << 62) || out_bytes >= ((int64_t)1 << 62) ||
        (int64_t)out_h * stride_h + taps_h >= (1ll << 31) || (int64_t)w + 2ll * pad_w >= (1ll << 31))
        return fail(QCONV_EUNSUPPORTED, "unroll sizes out of range");
    if (!dst || (in_bytes > 0 && !src)) return fail(QCONV_EINVAL, "src and dst must be non-NULL");
    if (!aligned16(dst)) return fail(QCONV_EINVAL, "dst must be 16-byte aligned");
    if (in_bytes > 0 && (uintptr_t)src < (uintptr_t)dst + out_bytes && (uintptr_t)dst < (uintptr_t)src + in_bytes)
        return fail(QCONV_EINVAL, "src and dst overlap");
    const int64_t lw = (int64_t)w + 2 * pad_w, staged = 4ll * c_out + lw * c * taps_h;
    if (staged > kUnrollLdsBytes)
        return fail(QCONV_EUNSUPPORTED, "unroll stages %lld bytes per output row (limit %lld): meant for few channels",
                    (long long)staged, (long long)kUnrollLdsBytes);
    UnrollArgs a{n, c, h, w, taps_h, stride_h, pad_h, out_h, taps_w, stride_w, pad_w, (int32_t)wout, c_out,
                 (int32_t)lw};
    if ((int64_t)n * out_h >= (1ll << 31) || wout * (c_out / 16) >= (1ll << 31))
        return fail(QCONV_EUNSUPPORTED, "unroll grid out of range");
    hipError_t e = launch_unroll(src, dst, a, (hipStream_t)stream);
    if (e != hipSuccess) return fail(QCONV_EHIP, "unroll launch: %s", hipGetErrorString(e));
    return QCONV_OK;
}

int qconv_probe_mfma_i8_shape(int32_t shape, int32_t blocks, int32_t iters, int32_t *sink, uint64_t *stamps, int64_t *ops,
                              void *stream) {
    g_err[0] = 0;
    if (shape != 0 && shape != 1) return fail(QCONV_EINVAL, "shape must be 0 (16x16x64) or 1 (32x32x32), got %d", shape);
    if (blocks < 1 || blocks > (1 << 20) || iters < 1 || iters > (1 << 24))
        return fail(QCONV_EINVAL, "blocks must be in [1, 2^20] and iters in [1, 2^24] (got %d, %d)", blocks, iters);
    if (!sink || !stamps) return fail(QCONV_EINVAL, "sink and stamps must be device pointers");
    if (((uintptr_t)stamps & 7u) != 0 || ((uintptr_t)sink & 3u) != 0)
        return fail(QCONV_EINVAL, "stamps must be 8-byte and sink 4-byte aligned");
    if (ops) *ops = mfma_probe_ops(blocks, iters);
    hipError_t e = launch_mfma_probe(blocks, iters, shape == 1, sink, stamps, (hipStream_t)stream);
    if (e != hipSuccess) return fail(QCONV_EHIP, "probe launch: %s", hipGetErrorString(e));
    return QCONV_OK;
}

int qconv_probe_mfma_i8(int32_t blocks, int32_t iters, int32_t *sink, uint64_t *stamps, int64_t *ops, void *stream) {
    return qconv_probe_mfma_i8_shape(0, blocks, iters, sink, stamps, ops, stream);
}

int qconv_last_launch(int64_t *grid, int64_t *threads, int64_t *lds_bytes) {
    if (grid) *grid = g_last_launch.grid;
    if (threads) *threads = g_last_launch.threads;
    if (lds_bytes) *lds_bytes = g_last_launch.lds;
    return g_last_launch.grid > 0 ? QCONV_OK : fail(QCONV_EINVAL, "no convolution launched on this thread yet");
}

int qconv_probe_launch(int32_t blocks, int32_t threads, int32_t lds_bytes, void *stream) {
    g_err[0] = 0;
    if (blocks < 1 || blocks > (1 << 20) || threads < 64 || threads > 1024 || threads % 64 != 0 || lds_bytes < 0 ||
        lds_bytes > kLdsBytes)
        return fail(QCONV_EINVAL, "blocks in [1, 2^20], threads a multiple of 64 in [64, 1024], lds_bytes in [0, %lld]",
                    (long long)kLdsBytes);
    hipError_t e = launch_empty_probe(blocks, threads, lds_bytes, (hipStream_t)stream);
    if (e != hipSuccess) return fail(QCONV_EHIP, "empty probe launch: %s", hipGetErrorString(e));
    return QCONV_OK;
}

int qconv_probe_grid_meet(int32_t blocks, int32_t rounds, int32_t two_level, uint32_t *arrivals, int32_t *err,
                          void *stream) {
    g_err[0] = 0;
    if (blocks < 1 || rounds < 0 || rounds > 4096 || (two_level != 0 && two_level != 1))
        return fail(QCONV_EINVAL, "blocks must be positive, rounds in [0, 4096] and two_level 0 or 1 (got %d, %d, %d)",
                    blocks, rounds, two_level);
    if (!arrivals || !err || ((uintptr_t)arrivals & 3u) != 0 || ((uintptr_t)err & 3u) != 0)
        return fail(QCONV_EINVAL, "arrivals and err must be 4-byte aligned device pointers");
    int dev = 0, cus = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
        return fail(QCONV_EHIP, "no device to query");
    // one 256-thread workgroup per CU at most: the whole grid is resident at once
    if (blocks > cus) return fail(QCONV_EINVAL, "blocks must be at most %d (the CUs), got %d", cus, blocks);
    // a fraction of a second of polling (each poll is a device-scope load)
    // before a workgroup gives up
    constexpr int kSpinLimit = 1 << 17;
    hipError_t e = launch_meet_probe(blocks, rounds, two_level, kSpinLimit, arrivals, err, (hipStream_t)stream);
    if (e != hipSuccess) return fail(QCONV_EHIP, "meeting probe launch: %s", hipGetErrorString(e));
    return QCONV_OK;
}

// Host-only consistency checks of the helpers the kernels rely on; returns 0
// when they hold.  Exposed so CPU tests can run them without a device.
int qconv_selftest(void) {
    const uint32_t ds[] = {1, 2, 3, 5, 7, 9, 14, 28, 49, 56, 58, 196, 784, 3136, 12544, 65535, 100003};
    for (uint32_t dv : ds) {
        FastDiv f = make_fastdiv(dv);
        for (uint32_t n = 0; n < 200000; n += 7)
            if (fdiv(n, f) != n / dv) return 1;
        const uint32_t big[] = {0x7fffffffu, 0x7ffffffeu, 0x40000000u, 123456789u};
        for (uint32_t n : big)
            if (fdiv(n, f) != n / dv) return 2;
    }
    return 0;
}

}  // extern "C"
