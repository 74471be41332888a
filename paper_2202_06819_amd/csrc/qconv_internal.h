// Internal declarations shared by the host library and the HIP kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "qconv.h"

namespace qconv {

// Unsigned division by a run-time constant d >= 1, exact for numerators below
// 2^31: q = (umulhi(n, mul) + n) >> shr with shr = ceil(log2 d) and
// mul = floor(2^32 * (2^shr - d) / d) + 1 (Granlund & Montgomery, 1994).
struct FastDiv {
    uint32_t d;
    uint32_t mul;
    uint32_t shr;
};

inline FastDiv make_fastdiv(uint32_t d) {
    FastDiv f{d, 0u, 0u};
    uint32_t l = 0;
    while ((1ull << l) < d) ++l;
    f.shr = l;
    f.mul = (uint32_t)(((1ull << 32) * ((1ull << l) - d)) / d + 1);
    return f;
}

__host__ __device__ inline uint32_t fdiv(uint32_t n, FastDiv f) {
#if defined(__HIP_DEVICE_COMPILE__)
    uint32_t t = __umulhi(n, f.mul);
#else
    uint32_t t = (uint32_t)(((uint64_t)n * f.mul) >> 32);
#endif
    return (t + n) >> f.shr;
}

// Everything a convolution launch needs, passed by value as the kernel argument.
struct ConvArgs {
    const uint8_t *xptr;    // packed activations, N x H x W x C
    const uint8_t *wptr;    // packed filters, K x R x S x C
    uint8_t *yptr;          // output (raw int32 or packed)
    const int32_t *mult;    // per-channel multipliers (requant mode)
    int32_t n, h, w, c, k, r, s;
    int32_t sh, sw, ph, pw, p, q;
    int32_t m;              // n * p * q
    int32_t vh;             // h + 2*ph: rows of one zero-padded image
    int32_t ncols;          // w + 2*pw: columns of one zero-padded row
    int32_t tap_w;          // band columns between horizontal filter taps: 1, or nb (batch-interleaved)
    int32_t xpix;           // bytes per input pixel (and per filter tap)
    int32_t nchunks;        // channel chunks of the main loop
    int32_t vec16;          // 1: every 16-byte vector of a pixel is whole (C*bits % 128 == 0)
    int32_t band_rows;      // padded rows the band buffer holds
    int32_t xbytes;         // packed activation bytes (buffer-load range)
    int32_t wbytes;         // packed filter bytes (buffer-load range)
    int32_t off_b0, off_b1; // LDS byte offsets of the two band buffers (pipelined kernel)
    int32_t off_w0, off_w1; // LDS byte offsets of the two filter buffers (equal when one chunk)
    int32_t off_m;          // LDS byte offset of the workgroup's multipliers (wide kernel)
    int32_t off_e;          // LDS byte offset of the int32 accumulator tile (ablation: LDS epilogue)
    int32_t w_image;        // 1: wptr is a prepared filter image (wide kernel), 0: packed KRSC filters
    int32_t pstride_b;      // bytes per granule plane of the band buffer
    int32_t pstride_w;      // bytes per granule plane of the filter buffer
    int32_t ktiles;         // workgroup tiles along output channels
    int32_t mtiles;         // workgroup tiles along output pixels
    int32_t splits;         // split-K factor over channel chunks (1: none)
    int32_t cps;            // channel chunks per split
    int32_t gpk;            // wide kernel: workgroups per channel tile (mtiles with a split, grid / ktiles without)
    FastDiv div_splits, div_ktiles, div_gpk;   // by splits, ktiles and gpk
    int32_t xcd_order;      // 1, 2: renumber workgroups so consecutive tiles share an XCD (wide kernel);
                            // 2: consecutive tiles share a channel tile rather than pixels
    int32_t *ws_part;       // split-K partial sums (splits > 1)
    uint32_t *ws_cnt;       // split-K arrival counters, one per output tile, zero between calls
    FastDiv div_pq, div_q, div_vh, div_ncols, div_rs, div_s;
    int32_t x_signed, w_signed;
    // operand widening of 4-bit nibbles to int8 lanes (see widen4)
    uint32_t xmask, wmask;
    int32_t xsl, xsr, wsl, wsr;
    int32_t acc_shift;      // accumulators carry a factor 2^acc_shift from widening
    // epilogue
    int32_t mode;           // QCONV_OUT_RAW_I32 / QCONV_OUT_REQUANT
    int32_t shift;
    int32_t lo, hi;         // clamp bounds, ReLU already folded into lo
    const int32_t *bias;    // per-channel accumulator offsets, or null
    const uint8_t *res;     // residual in y's packed layout, or null
    int32_t res_signed;     // residual values are signed
    // the pack fused into the convolution (NCHW instances)
    const int8_t *xsrc;     // int8 N x C x H x W activations
    int32_t xsrc_bytes;
    uint8_t *xpk;           // packed copy of the input written on the way, or null
    FastDiv div_w, div_wq;  // by w and by its column quads
    FastDiv div_brows;      // by band_rows
    FastDiv div_pad2;       // by 2 pw, a band row's padding columns (1 if none)
    FastDiv div_rb4;        // by band_rows rounded up to a multiple of 4
    // a 1x1 projection at the same stride fused into a 3x3 launch (PROJ
    // instances): its filters are tap r*s of the prepared image, its input the
    // centre tap's pixels, its output and epilogue its own
    uint8_t *yproj;         // its output (raw int32 or packed, as yptr)
    const int32_t *mult2;   // its per-channel multipliers (requant mode)
    const int32_t *bias2;   // its per-channel accumulator offsets, or null
    int32_t shift2, lo2, hi2;
};

// Band pixels one thread of a wide tile stages per channel chunk: the 4
// packed 16-byte vectors every thread prefetches, or more for tiles whose
// pixel count reaches the thread count (their band of zero-padded rows can
// hold about three times as many pixels as the tile).
constexpr int wide_band_pixels_per_thread(int tile_p, int threads, int vecs_per_pixel) {
    const int base = 4 / vecs_per_pixel;
    const int need = (3 * tile_p + threads - 1) / threads;
    return base > need ? base : need;
}

using ConvLauncher = hipError_t (*)(const ConvArgs &, dim3 grid, size_t lds_bytes, hipStream_t);
// builds a prepared filter image; `wproj` (or null): packed K x 1 x 1 x C filters
// of a fused projection, placed as the image's last tap
using PrepLauncher = hipError_t (*)(const ConvArgs &, uint8_t *image, int64_t elems, const uint8_t *wproj,
                                    hipStream_t);

// A compiled instance of a tile for one fixed filter size (prepared filters).
struct FixedInstance {
    int r, s;
    ConvLauncher launch;
    const void *kernel;
    ConvLauncher launch_mc; // variant for plans with several channel chunks per workgroup, or null
    const void *kernel_mc;
    ConvLauncher launch_one;   // variant for plans whose workgroups each run one stage, or null
    const void *kernel_one;
    ConvLauncher launch_one_oct;   // the same for input rows of whole pixel octets (fused pack), or null
    const void *kernel_one_oct;
};

// The kernels of one tile for one epilogue flavour.
struct KernelSet {
    ConvLauncher launch;
    const void *kernel;     // for hipFuncSetAttribute
    FixedInstance fixed[2]; // wide tiles: 3x3 and 1x1 instances; empty (r == 0) otherwise
};

struct TileEntry {
    qconv_tile_info info;
    KernelSet plain;        // epilogue without bias and residual
    KernelSet ext;          // epilogue with bias and/or residual
    PrepLauncher prep;      // builds the filter image (wide tiles), else null
    FixedInstance fused;    // 3x3 instance reading int8 NCHW activations (the pack fused in), or empty
};

// A kernel with some of the techniques switched off (for measurement).
struct AblationInstance {
    const char *tile;       // the tile it is a variant of
    int mask;               // bits: 1 lowered staging, 2 LDS epilogue, 4 packed activations in LDS
    ConvLauncher launch;
    const void *kernel;
};

// A 3x3 instance of a tile with a 1x1 projection at the same stride fused in
// (prepared filters, no split).
struct ProjInstance {
    const char *tile;       // the tile it is a variant of
    FixedInstance plain;    // epilogues without bias
    FixedInstance ext;      // epilogues with per-channel biases
};

// Defined in qconv_conv.hip.
const TileEntry *tile_table();
int tile_table_size();

// Defined in qconv_tiles_abl.hip.
const AblationInstance *ablation_instance(const char *tile_name, int mask);

// Defined in qconv_tiles_proj.hip.
const ProjInstance *proj_instance(const char *tile_name);

// Defined in qconv_pack.hip.
hipError_t launch_pack(const int8_t *src, void *dst, int32_t n, int32_t c, int32_t h, int32_t w, int32_t bits,
                       int32_t is_signed, int32_t nb, hipStream_t stream);

// Patch unrolling (qconv_unroll): source n x c x h x w, destination
// n x out_h x wout x c_out; lw = w + 2 * pad_w is the staged row length.
struct UnrollArgs {
    int32_t n, c, h, w;
    int32_t taps_h, stride_h, pad_h, out_h;
    int32_t taps_w, stride_w, pad_w, wout;
    int32_t c_out, lw;
};

// Defined in qconv_unroll.hip.
int64_t unroll_lds_bytes(const UnrollArgs &a);
hipError_t launch_unroll(const int8_t *src, int8_t *dst, const UnrollArgs &a, hipStream_t stream);

// Defined in qconv_probe.hip (measurement aid).
int64_t mfma_probe_ops(int blocks, int iters);
hipError_t launch_mfma_probe(int blocks, int iters, bool wide, int32_t *sink, uint64_t *stamps, hipStream_t stream);
hipError_t launch_empty_probe(int blocks, int threads, int lds_bytes, hipStream_t stream);
// the meeting probe's counters: the top one, then one per XCD group, each on
// its own 64-byte line (uint32 elements kMeetStride apart)
constexpr int kMeetCounters = 9;
constexpr int kMeetStride = 16;
hipError_t launch_meet_probe(int blocks, int rounds, int two_level, int spin_limit, uint32_t *arrivals, int32_t *err,
                             hipStream_t stream);

}  // namespace qconv
