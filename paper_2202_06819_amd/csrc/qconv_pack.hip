// Relayout-and-pack for gfx950: int8 N x C x H x W  ->  channel-packed
// N x H x W x C (Sec. 1: eight 4-bit values per 32-bit word along the channel
// axis; Sec. 3.3: channels innermost so consumers read it coalesced).
//
// The operation is a transpose of each image's C x (H*W) plane.  A workgroup
// of 128 threads owns a tile of 64 channels x 64 pixels (small tiles, so even
// a batch-8 56x56 tensor spreads over more than twice as many workgroups as
// there are CUs).  It reads the tile row by row (each channel's pixels are
// contiguous in NCHW: 32 bytes per lane, two lanes per 64-byte row segment),
// saturates every value into the target range and parks it in LDS; it then
// reads 8 channels x 4 pixels per lane as dwords, transposes the bytes in
// registers, packs nibbles and writes each pixel's words.  The LDS row pitch
// of 17 dwords keeps the column reads of a wave (8 channel groups x 8 pixel
// quads) free of bank conflicts.  The kernel is HBM-bound: every input byte
// is read once and every output byte written once.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "qconv_internal.h"

namespace qconv {

constexpr int PK_C = 64;          // channels per tile
constexpr int PK_P = 64;          // pixels per tile (64-byte segments of each channel row)
constexpr int PK_PITCH = 68;      // LDS row pitch in bytes (17 dwords: conflict-free column reads)
constexpr int PK_THREADS = 128;   // phase 2: 8 channel groups x 16 pixel quads

// Same renumbering as the convolution kernels: block b runs on XCD b % 8;
// give every XCD a contiguous range so neighbouring pixel tiles (which share
// cache lines at row ends) meet in one L2.
__device__ __forceinline__ int pack_xcd_block(int b, int g) {
    const int x = b % 8, i = b / 8, q = g / 8, r = g % 8;
    return (x < r ? x * (q + 1) : r * (q + 1) + (x - r) * q) + i;
}

__device__ __forceinline__ uint32_t byte_of(uint32_t v, int j) { return (v >> (8 * j)) & 0xFFu; }

// 4x4 byte transpose: byte k of result j is byte j of t[k].
__device__ __forceinline__ uint32_t gather_byte(const uint32_t (&t)[4], int j) {
    return byte_of(t[0], j) | (byte_of(t[1], j) << 8) | (byte_of(t[2], j) << 16) | (byte_of(t[3], j) << 24);
}

// (ptiles, ctiles, nb: the divisors of the block and image decompositions)
template <int BITS, bool SIGNED>
__global__ void __launch_bounds__(PK_THREADS)
    pack_nchw(const int8_t *__restrict__ src, uint8_t *__restrict__ dst, int c, int hw, FastDiv ptiles,
              FastDiv ctiles, FastDiv nb) {
    constexpr int LO = SIGNED ? -(1 << (BITS - 1)) : 0;
    constexpr int HI = SIGNED ? (1 << (BITS - 1)) - 1 : (1 << BITS) - 1;
    __shared__ __attribute__((aligned(16))) uint8_t tile[PK_C * PK_PITCH];
    const int tid = threadIdx.x;
    int bid = pack_xcd_block(blockIdx.x, gridDim.x);
    const int rest = (int)fdiv((uint32_t)bid, ptiles);
    const int pt = bid - rest * (int)ptiles.d;
    const int img = (int)fdiv((uint32_t)rest, ctiles);
    const int ct = rest - img * (int)ctiles.d;
    const int c0 = ct * PK_C;
    const int p0 = pt * PK_P;
    const int8_t *plane = src + (size_t)img * c * hw;
    // destination pixel of (img, pix): nb images interleaved per pixel
    // (nb = 1: plain N x H x W x C)
    const int ig = (int)fdiv((uint32_t)img, nb);
    const size_t obase = (size_t)ig * hw * nb.d + (img - ig * (int)nb.d);
    auto out_pixel = [&](int px) { return obase + (size_t)px * nb.d; };

    // ---- phase 1: 64 channel rows x 64 pixels; a lane reads 32 consecutive
    // pixels of one row, saturates them and parks them in LDS
    {
        const int row = tid >> 1;
        const int seg = (tid & 1) * 32;
        const int ch = c0 + row;
        uint32_t v[8];
        const int8_t *rp = plane + (size_t)ch * hw + p0 + seg;
        if (ch < c && p0 + seg + 32 <= hw && (reinterpret_cast<uintptr_t>(rp) & 15) == 0) {
            const uint4 a = *reinterpret_cast<const uint4 *>(rp);
            const uint4 b = *reinterpret_cast<const uint4 *>(rp + 16);
            v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
            v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
        } else {
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                uint32_t w = 0;
#pragma unroll
                for (int k = 0; k < 4; ++k) {
                    const int px = p0 + seg + 4 * e + k;
                    if (ch < c && px < hw) w |= (uint32_t)(uint8_t)rp[4 * e + k] << (8 * k);
                }
                v[e] = w;
            }
        }
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            uint32_t w = v[e];
            if constexpr (BITS == 4) {
                // byte-parallel range test (for signed values on v + 8, added per
                // byte without carries); only words with a byte out of range
                // take the per-byte clamp
                const uint32_t t = SIGNED ? (((w & 0x7F7F7F7Fu) + 0x08080808u) ^ (w & 0x80808080u)) : w;
                if ((t & 0xF0F0F0F0u) != 0u) {
                    uint32_t o = 0;
#pragma unroll
                    for (int k = 0; k < 4; ++k) {
                        const int x = (int)(int8_t)byte_of(w, k);
                        o |= ((uint32_t)(x < LO ? LO : (x > HI ? HI : x)) & 0xFFu) << (8 * k);
                    }
                    w = o;
                }
            }
            *reinterpret_cast<uint32_t *>(tile + row * PK_PITCH + seg + 4 * e) = w;
        }
    }
    __syncthreads();

    // ---- phase 2: a lane takes 8 channels (group g) x 4 pixels (quad q):
    // 8 dword reads, an in-register transpose, and one output word (4-bit) or
    // two (8-bit) per pixel
    const int g = tid & 7;
    const int q = tid >> 3;
    const int cg = c0 + 8 * g;
    if (cg >= c) return;
    uint32_t d[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) d[i] = *reinterpret_cast<const uint32_t *>(tile + (8 * g + i) * PK_PITCH + 4 * q);
    if constexpr (BITS == 4) {
        // byte j of t[k]: channel 8g+2k in the low nibble, 8g+2k+1 in the high one, of pixel j
        uint32_t t[4];
#pragma unroll
        for (int k = 0; k < 4; ++k) t[k] = (d[2 * k] & 0x0F0F0F0Fu) | ((d[2 * k + 1] << 4) & 0xF0F0F0F0u);
        uint32_t *out = reinterpret_cast<uint32_t *>(dst);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int pix = p0 + 4 * q + j;
            if (pix < hw) out[out_pixel(pix) * (c / 8) + cg / 8] = gather_byte(t, j);
        }
    } else {
        const uint32_t lo4[4] = {d[0], d[1], d[2], d[3]};
        const uint32_t hi4[4] = {d[4], d[5], d[6], d[7]};
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int pix = p0 + 4 * q + j;
            if (pix >= hw) continue;
            uint32_t *out = reinterpret_cast<uint32_t *>(dst + out_pixel(pix) * c + cg);   // c % 4 == 0
            out[0] = gather_byte(lo4, j);
            if (cg + 4 < c) out[1] = gather_byte(hi4, j);
        }
    }
}

hipError_t launch_pack(const int8_t *src, void *dst, int32_t n, int32_t c, int32_t h, int32_t w, int32_t bits,
                       int32_t is_signed, int32_t nb, hipStream_t stream) {
    const int hw = h * w;
    const int ptiles = (hw + PK_P - 1) / PK_P;
    const int ctiles = (c + PK_C - 1) / PK_C;
    const long long blocks = (long long)n * ptiles * ctiles;
    uint8_t *d = static_cast<uint8_t *>(dst);
    const dim3 grid((unsigned)blocks), block(PK_THREADS);
    const FastDiv dp = make_fastdiv((uint32_t)ptiles), dc = make_fastdiv((uint32_t)ctiles),
                  dn = make_fastdiv((uint32_t)(nb > 0 ? nb : 1));
    if (bits == 4 && is_signed)
        hipLaunchKernelGGL((pack_nchw<4, true>), grid, block, 0, stream, src, d, c, hw, dp, dc, dn);
    else if (bits == 4)
        hipLaunchKernelGGL((pack_nchw<4, false>), grid, block, 0, stream, src, d, c, hw, dp, dc, dn);
    else
        hipLaunchKernelGGL((pack_nchw<8, true>), grid, block, 0, stream, src, d, c, hw, dp, dc, dn);
    return hipGetLastError();
}

}  // namespace qconv
