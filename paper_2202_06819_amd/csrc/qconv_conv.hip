// Implicit-GEMM quantised convolution for gfx950 (CDNA4), int8 MFMA with
// int32 accumulation.
//
// GEMM view (Sec. 2.1): rows = output pixels m = (n, p, q), columns = output
// channels, depth = (r, s, c).  The MFMA's A operand is the filter block
// (16 output channels x 64 depth values), B is the activation block (64 depth
// values x 16 pixels); D = A * B holds 16 channels x 16 pixels.
//
// Staging (the duplicate-aware load of Sec. 3.1 / Alg. 1, restated): a
// workgroup owns TP consecutive output pixels.  Instead of loading the
// lowered matrix -- where every input pixel appears up to R*S times -- it
// copies once per channel chunk the band of zero-padded input rows those
// pixels touch into LDS.  A lowered row is then pure address arithmetic: the
// pixel's base offset in the band plus a per-tap offset that is the same for
// every lane.  Padding rows and columns are materialised as zeros in the band,
// so no lane ever tests a border.
//
// LDS layout: channels are split into 16-channel granules (8 bytes packed
// 4-bit, 16 bytes int8).  Each granule index owns a plane; inside a plane a
// pixel's granule sits at (band_row * ncols + col) * granule_bytes.  MFMA
// lane l reads granule plane (l / 16) of pixel (l % 16): the 16 lanes of a
// plane read consecutive addresses, and planes are padded by 128 mod 256
// bytes so the four lane groups of a read fall into different banks.
//
// Operands stay packed in HBM and LDS; 4-bit values are widened to int8 in
// VGPRs right before the MFMA (see widen4).
//
// Output packing in registers (Sec. 3.2.3 and 3.3, restated for wave64): the
// MFMA result lane layout gives lane l the rows 4*(l/16)+v of the D tile.
// Filters are placed in A so that D row i of fragment tm is output channel
// (i/4)*4*FK + 4*tm + i%4 of the wave's channel block; then each lane ends
// with 4*FK consecutive channels of one pixel and packs them into whole
// 32-bit words without any cross-lane exchange.  The epilogue (requantise,
// ReLU, clamp, pack) runs on those registers and stores each pixel's
// channels as one contiguous run (Sec. 3.2.2: epilogue before the store).
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "qconv_internal.h"

namespace qconv {

typedef int v4i __attribute__((ext_vector_type(4)));

// 4-bit nibbles -> int8 lanes.  Each 32-bit word holds channels 0..7 of a
// group; lo keeps the even channels, hi the odd ones, one per byte:
//   unsigned: lo = v & 0x0F0F0F0F,        hi = (v >> 4) & 0x0F0F0F0F
//   signed:   lo = (v << 4) & 0xF0F0F0F0, hi = v & 0xF0F0F0F0   (value * 16)
// The signed form is exact: the nibble in the high half of a byte is the
// two's-complement int8 16*v.  Both operands use the same channel order, so
// the dot product is unchanged; the factor 16 is removed from the int32
// accumulator by an exact arithmetic shift.
__device__ __forceinline__ v4i widen4(uint2 v, uint32_t mask, int sl, int sr) {
    v4i o;
    o[0] = (int)((v.x << sl) & mask);
    o[1] = (int)((v.x >> sr) & mask);
    o[2] = (int)((v.y << sl) & mask);
    o[3] = (int)((v.y >> sr) & mask);
    return o;
}

template <int BITS>
struct Gran;
template <>
struct Gran<4> {
    using raw = uint2;
    __device__ static __forceinline__ v4i widen(raw v, uint32_t mask, int sl, int sr) { return widen4(v, mask, sl, sr); }
};
template <>
struct Gran<8> {
    using raw = uint4;
    __device__ static __forceinline__ v4i widen(raw v, uint32_t, int, int) {
        v4i o;
        o[0] = (int)v.x;
        o[1] = (int)v.y;
        o[2] = (int)v.z;
        o[3] = (int)v.w;
        return o;
    }
};

// Padded row ("virtual row") of output pixel m's first tap, and its column.
__device__ __forceinline__ void pixel_origin(const ConvArgs &a, int m, int &vrow, int &col) {
    int img = (int)fdiv((uint32_t)m, a.div_pq);
    int rem = m - img * (a.p * a.q);
    int pp = (int)fdiv((uint32_t)rem, a.div_q);
    int qq = rem - pp * a.q;
    vrow = img * a.vh + pp * a.sh;
    col = qq * a.sw;
}

template <int BITS, int WP, int WK, int FP, int FK, int CK>
__global__ void __launch_bounds__(WP * WK * 64) conv_igemm(ConvArgs a) {
    constexpr int NT = WP * WK * 64;
    constexpr int TP = WP * FP * 16;
    constexpr int TK = WK * FK * 16;
    constexpr int GRAN = 2 * BITS;          // bytes of a 16-channel granule
    constexpr int KSTEPS = CK / 64;         // MFMA depth steps per tap and chunk
    constexpr int VPP = CK * BITS / 128;    // 16-byte vectors per pixel and chunk
    constexpr int GPV = 16 / GRAN;          // granules per 16-byte vector
    constexpr int CPW = 32 / BITS;          // channels per 32-bit word
    static_assert(BITS == 8 || FK % 2 == 0, "4-bit output packs 8 channels per word: FK must be even");
    using G = Gran<BITS>;
    using Raw = typename G::raw;

    extern __shared__ __attribute__((aligned(16))) uint8_t smem[];
    uint8_t *band = smem;
    uint8_t *wlds = smem + (size_t)(CK / 16) * a.pstride_b;

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int wp = wave % WP;
    const int wk = wave / WP;
    const int l16 = lane & 15;
    const int gq = lane >> 4;

    const int bid = blockIdx.x;
    const int kt = bid % a.ktiles;
    const int mt = bid / a.ktiles;
    const int m0 = mt * TP;
    const int k0 = kt * TK;
    const int rs = a.r * a.s;

    // Band of padded rows this workgroup's pixels touch.
    int vlo, c_unused, vlast;
    pixel_origin(a, m0, vlo, c_unused);
    pixel_origin(a, min(m0 + TP, a.m) - 1, vlast, c_unused);
    const int nrows = vlast + a.r - vlo;   // <= a.band_rows (checked on the host)

    int pixoff[FP];
#pragma unroll
    for (int tn = 0; tn < FP; ++tn) {
        int m = min(m0 + wp * FP * 16 + tn * 16 + l16, a.m - 1);
        int vr, cl;
        pixel_origin(a, m, vr, cl);
        pixoff[tn] = ((vr - vlo) * a.ncols + cl) * GRAN;
    }

    v4i acc[FP][FK];
#pragma unroll
    for (int tn = 0; tn < FP; ++tn)
#pragma unroll
        for (int tm = 0; tm < FK; ++tm) acc[tn][tm] = v4i{0, 0, 0, 0};

    const int nvec_band = nrows * a.ncols * VPP;
    const int nvec_w = TK * rs * VPP;

    for (int chunk = 0; chunk < a.nchunks; ++chunk) {
        const int cbyte = chunk * (CK * BITS / 8);
        const int cbase = chunk * CK;
        __syncthreads();
        // ---- band: global -> LDS, every needed input pixel exactly once
        for (int idx = tid; idx < nvec_band; idx += NT) {
            const int part = idx % VPP;
            const int pix = idx / VPP;
            const int rowl = (int)fdiv((uint32_t)pix, a.div_ncols);
            const int col = pix - rowl * a.ncols;
            const int vrow = vlo + rowl;
            const int img = (int)fdiv((uint32_t)vrow, a.div_vh);
            const int hh = vrow - img * a.vh - a.ph;
            const int ww = col - a.pw;
            uint32_t d[4] = {0u, 0u, 0u, 0u};
            const bool inside = img < a.n && hh >= 0 && hh < a.h && ww >= 0 && ww < a.w;
            if (inside) {
                const int ch0 = cbase + part * (128 / BITS);
                const uint8_t *src =
                    a.xptr + ((size_t)(img * a.h + hh) * a.w + ww) * a.xpix + cbyte + part * 16;
                if (a.vec16 && ch0 + 128 / BITS <= a.c) {
                    uint4 v = *reinterpret_cast<const uint4 *>(src);
                    d[0] = v.x; d[1] = v.y; d[2] = v.z; d[3] = v.w;
                } else {
#pragma unroll
                    for (int e = 0; e < 4; ++e)
                        if (ch0 + e * CPW < a.c) d[e] = reinterpret_cast<const uint32_t *>(src)[e];
                }
            }
            const int off = pix * GRAN;
            if constexpr (BITS == 4) {
                *reinterpret_cast<uint2 *>(band + (size_t)(part * GPV) * a.pstride_b + off) = uint2{d[0], d[1]};
                *reinterpret_cast<uint2 *>(band + (size_t)(part * GPV + 1) * a.pstride_b + off) = uint2{d[2], d[3]};
            } else {
                *reinterpret_cast<uint4 *>(band + (size_t)part * a.pstride_b + off) = uint4{d[0], d[1], d[2], d[3]};
            }
        }
        // ---- filters: TK channels x R*S taps of this chunk, in MFMA row order
        for (int idx = tid; idx < nvec_w; idx += NT) {
            const int part = idx % VPP;
            const int t = idx / VPP;
            const int slot = (int)fdiv((uint32_t)t, a.div_rs);
            const int tap = t - slot * rs;
            // slot = wave_k * FK*16 + tm*16 + i  ->  channel (i/4)*4*FK + 4*tm + i%4 of that wave's block
            const int wkk = slot / (FK * 16);
            const int rem = slot % (FK * 16);
            const int tm = rem / 16;
            const int i = rem % 16;
            const int kk = k0 + wkk * FK * 16 + (i / 4) * (4 * FK) + 4 * tm + (i % 4);
            uint32_t d[4] = {0u, 0u, 0u, 0u};
            if (kk < a.k) {
                const int ch0 = cbase + part * (128 / BITS);
                const uint8_t *src = a.wptr + ((size_t)kk * rs + tap) * a.xpix + cbyte + part * 16;
                if (a.vec16 && ch0 + 128 / BITS <= a.c) {
                    uint4 v = *reinterpret_cast<const uint4 *>(src);
                    d[0] = v.x; d[1] = v.y; d[2] = v.z; d[3] = v.w;
                } else {
#pragma unroll
                    for (int e = 0; e < 4; ++e)
                        if (ch0 + e * CPW < a.c) d[e] = reinterpret_cast<const uint32_t *>(src)[e];
                }
            }
            const int off = (tap * TK + slot) * GRAN;
            if constexpr (BITS == 4) {
                *reinterpret_cast<uint2 *>(wlds + (size_t)(part * GPV) * a.pstride_w + off) = uint2{d[0], d[1]};
                *reinterpret_cast<uint2 *>(wlds + (size_t)(part * GPV + 1) * a.pstride_w + off) = uint2{d[2], d[3]};
            } else {
                *reinterpret_cast<uint4 *>(wlds + (size_t)part * a.pstride_w + off) = uint4{d[0], d[1], d[2], d[3]};
            }
        }
        __syncthreads();

        // ---- main loop over taps: LDS -> VGPR, widen, MFMA
        for (int tap = 0; tap < rs; ++tap) {
            const int rr = tap / a.s;
            const int ss = tap - rr * a.s;
            const int toff = (rr * a.ncols + ss) * GRAN;
#pragma unroll
            for (int ks = 0; ks < KSTEPS; ++ks) {
                const int g = ks * 4 + gq;
                const uint8_t *bp = band + (size_t)g * a.pstride_b + toff;
                const uint8_t *ap = wlds + (size_t)g * a.pstride_w + (tap * TK + wk * FK * 16 + l16) * GRAN;
                v4i A[FK], B[FP];
#pragma unroll
                for (int tm = 0; tm < FK; ++tm)
                    A[tm] = G::widen(*reinterpret_cast<const Raw *>(ap + tm * 16 * GRAN), a.wmask, a.wsl, a.wsr);
#pragma unroll
                for (int tn = 0; tn < FP; ++tn)
                    B[tn] = G::widen(*reinterpret_cast<const Raw *>(bp + pixoff[tn]), a.xmask, a.xsl, a.xsr);
#pragma unroll
                for (int tn = 0; tn < FP; ++tn)
#pragma unroll
                    for (int tm = 0; tm < FK; ++tm)
                        acc[tn][tm] = __builtin_amdgcn_mfma_i32_16x16x64_i8(A[tm], B[tn], acc[tn][tm], 0, 0, 0);
            }
        }
    }

    // ---- epilogue in registers: this lane holds channels cb .. cb + 4*FK - 1 of
    // pixel m for every pixel fragment tn.
    const int cb = k0 + wk * FK * 16 + gq * 4 * FK;
    if (a.mode == QCONV_OUT_RAW_I32) {
#pragma unroll
        for (int tn = 0; tn < FP; ++tn) {
            const int m = m0 + wp * FP * 16 + tn * 16 + l16;
            if (m >= a.m) continue;
            int32_t *yrow = reinterpret_cast<int32_t *>(a.yptr) + (size_t)m * a.k;
#pragma unroll
            for (int tm = 0; tm < FK; ++tm) {
                if (cb + 4 * tm < a.k) {
                    v4i v = acc[tn][tm];
                    int4 o{v[0] >> a.acc_shift, v[1] >> a.acc_shift, v[2] >> a.acc_shift, v[3] >> a.acc_shift};
                    *reinterpret_cast<int4 *>(yrow + cb + 4 * tm) = o;
                }
            }
        }
        return;
    }

    int32_t mul[4 * FK];
#pragma unroll
    for (int e = 0; e < 4 * FK; ++e) mul[e] = (cb + e < a.k) ? a.mult[cb + e] : 0;
    const int64_t rnd = (int64_t)1 << (a.shift - 1);
#pragma unroll
    for (int tn = 0; tn < FP; ++tn) {
        const int m = m0 + wp * FP * 16 + tn * 16 + l16;
        if (m >= a.m) continue;
        uint32_t words[4 * FK / CPW];
#pragma unroll
        for (int wd = 0; wd < 4 * FK / CPW; ++wd) words[wd] = 0u;
#pragma unroll
        for (int tm = 0; tm < FK; ++tm)
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                const int e = 4 * tm + v;   // channel cb + e
                int64_t t = (int64_t)(acc[tn][tm][v] >> a.acc_shift) * mul[e] + rnd;
                t >>= a.shift;              // arithmetic: floor
                t = t < a.lo ? a.lo : t;
                t = t > a.hi ? a.hi : t;
                words[e / CPW] |= ((uint32_t)t & ((1u << BITS) - 1u)) << (BITS * (e % CPW));
            }
        uint32_t *yw = reinterpret_cast<uint32_t *>(a.yptr + (size_t)m * (a.k * BITS / 8) + cb * BITS / 8);
#pragma unroll
        for (int wd = 0; wd < 4 * FK / CPW; ++wd)
            if (cb + wd * CPW < a.k) yw[wd] = words[wd];
    }
}

template <int BITS, int WP, int WK, int FP, int FK, int CK>
static hipError_t launch_conv(const ConvArgs &a, dim3 grid, size_t lds, hipStream_t stream) {
    hipLaunchKernelGGL((conv_igemm<BITS, WP, WK, FP, FK, CK>), grid, dim3(WP * WK * 64), lds, stream, a);
    return hipGetLastError();
}

// The compiled tile space: (bits, waves_p, waves_k, frag_p, frag_k, chunk_c).
#define QCONV_TILE_LIST(X)   \
    X(4, 4, 1, 4, 4, 64)     \
    X(4, 4, 1, 2, 4, 64)     \
    X(4, 4, 1, 1, 4, 64)     \
    X(4, 2, 2, 4, 4, 64)     \
    X(4, 2, 2, 2, 4, 64)     \
    X(4, 1, 4, 4, 4, 64)     \
    X(4, 4, 1, 4, 2, 64)     \
    X(4, 2, 2, 4, 2, 64)     \
    X(4, 4, 1, 4, 4, 128)    \
    X(4, 2, 2, 4, 4, 128)    \
    X(4, 2, 2, 2, 4, 128)    \
    X(4, 1, 4, 4, 4, 128)    \
    X(8, 4, 1, 4, 4, 64)     \
    X(8, 4, 1, 2, 4, 64)     \
    X(8, 2, 2, 4, 4, 64)     \
    X(8, 2, 2, 2, 4, 64)     \
    X(8, 1, 4, 4, 4, 64)     \
    X(8, 4, 1, 4, 2, 64)     \
    X(8, 2, 2, 4, 4, 128)

#define QCONV_TILE_ENTRY(B, WP, WK, FP, FK, CK)                                                              \
    {{0, B, WP, WK, FP, FK, CK, WP * FP * 16, WK * FK * 16, WP * WK * 64,                                    \
      "b" #B "_w" #WP "x" #WK "_f" #FP "x" #FK "_c" #CK},                                                    \
     &launch_conv<B, WP, WK, FP, FK, CK>,                                                                    \
     reinterpret_cast<const void *>(&conv_igemm<B, WP, WK, FP, FK, CK>)},

static TileEntry g_tiles[] = {QCONV_TILE_LIST(QCONV_TILE_ENTRY)};

const TileEntry *tile_table() {
    static bool numbered = [] {
        for (int i = 0; i < (int)(sizeof(g_tiles) / sizeof(g_tiles[0])); ++i) g_tiles[i].info.id = i;
        return true;
    }();
    (void)numbered;
    return g_tiles;
}

int tile_table_size() { return (int)(sizeof(g_tiles) / sizeof(g_tiles[0])); }

}  // namespace qconv
