// Relayout-and-pack for gfx950: int8 N x C x H x W  ->  channel-packed
// N x H x W x C (Sec. 1: eight 4-bit values per 32-bit word along the channel
// axis; Sec. 3.3: channels innermost so consumers read it coalesced).
//
// The operation is a transpose of each image's C x (H*W) plane.  A workgroup
// owns a tile of 64 channels x 64 pixels.  It reads the tile row by row
// (each channel's 64 pixels are contiguous in NCHW, 16 bytes per lane),
// saturates every value into the target range, and parks it in LDS; it then
// reads the tile column-wise (one pixel's channels), packs, and writes each
// pixel's run of channels contiguously.  Both HBM streams are therefore
// coalesced; the LDS tile row has a 4-byte pad so the column reads spread
// over banks.  The kernel is HBM-bound: every input byte is read once and
// every output byte written once.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "qconv_internal.h"

namespace qconv {

constexpr int PK_C = 64;          // channels per tile
constexpr int PK_P = 64;          // pixels per tile
constexpr int PK_ROW = PK_P + 4;  // LDS row pitch in bytes
constexpr int PK_THREADS = 256;

__device__ __forceinline__ int sat(int v, int lo, int hi) { return v < lo ? lo : (v > hi ? hi : v); }

template <int BITS>
__global__ void __launch_bounds__(PK_THREADS)
    pack_nchw(const int8_t *__restrict__ src, uint8_t *__restrict__ dst, int c, int hw, int ptiles, int ctiles,
              int lo, int hi) {
    __shared__ int8_t tile[PK_C * PK_ROW];
    const int tid = threadIdx.x;
    int bid = blockIdx.x;
    const int ct = bid % ctiles;
    bid /= ctiles;
    const int pt = bid % ptiles;
    const int img = bid / ptiles;
    const int c0 = ct * PK_C;
    const int p0 = pt * PK_P;
    const int8_t *plane = src + (size_t)img * c * hw;

    // ---- load: 64 channel rows x 64 pixels; lane covers 16 consecutive pixels of one row
    {
        const int row = tid >> 2;            // channel within tile
        const int seg = (tid & 3) * 16;      // first pixel of this lane's segment
        const int ch = c0 + row;
        int8_t vals[16];
        if (ch < c && p0 + seg + 16 <= hw && ((((size_t)img * c + ch) * hw + p0 + seg) & 15) == 0) {
            int4 v = *reinterpret_cast<const int4 *>(plane + (size_t)ch * hw + p0 + seg);
            const int8_t *b = reinterpret_cast<const int8_t *>(&v);
#pragma unroll
            for (int e = 0; e < 16; ++e) vals[e] = b[e];
        } else {
#pragma unroll
            for (int e = 0; e < 16; ++e) {
                const int px = p0 + seg + e;
                vals[e] = (ch < c && px < hw) ? plane[(size_t)ch * hw + px] : (int8_t)0;
            }
        }
#pragma unroll
        for (int e = 0; e < 16; ++e) tile[row * PK_ROW + seg + e] = (int8_t)sat(vals[e], lo, hi);
    }
    __syncthreads();

    // ---- store: one pixel's channel run per group of 4 lanes
    const int px = tid >> 2;                 // pixel within tile
    const int part = tid & 3;                // quarter of the 64 channels: 16 channels
    const int pix = p0 + px;
    if (pix >= hw) return;
    const int cq = c0 + part * 16;
    if (cq >= c) return;
    if constexpr (BITS == 4) {
        // 16 channels -> two 32-bit words; channel 8j+i in bits [4i, 4i+3] of word j
        uint32_t wv[2] = {0u, 0u};
#pragma unroll
        for (int e = 0; e < 16; ++e)
            wv[e >> 3] |= ((uint32_t)(uint8_t)tile[(part * 16 + e) * PK_ROW + px] & 0xFu) << (4 * (e & 7));
        uint32_t *out = reinterpret_cast<uint32_t *>(dst) + ((size_t)img * hw + pix) * (c / 8) + cq / 8;
        if (cq + 16 <= c) {
            out[0] = wv[0];
            out[1] = wv[1];
        } else {
            out[0] = wv[0];  // c % 8 == 0: the run holds exactly one more word
        }
    } else {
        uint8_t bv[16];
#pragma unroll
        for (int e = 0; e < 16; ++e) bv[e] = (uint8_t)tile[(part * 16 + e) * PK_ROW + px];
        uint8_t *out = dst + ((size_t)img * hw + pix) * c + cq;
        const int cnt = min(16, c - cq);
        if (cnt == 16 && (((size_t)img * hw + pix) * c + cq) % 16 == 0) {
            *reinterpret_cast<uint4 *>(out) = *reinterpret_cast<const uint4 *>(bv);
        } else {
            for (int e = 0; e < cnt; ++e) out[e] = bv[e];
        }
    }
}

hipError_t launch_pack(const int8_t *src, void *dst, int32_t n, int32_t c, int32_t h, int32_t w, int32_t bits,
                       int32_t is_signed, hipStream_t stream) {
    const int hw = h * w;
    const int ptiles = (hw + PK_P - 1) / PK_P;
    const int ctiles = (c + PK_C - 1) / PK_C;
    const long long blocks = (long long)n * ptiles * ctiles;
    const int lo = is_signed ? -(1 << (bits - 1)) : 0;
    const int hi = is_signed ? (1 << (bits - 1)) - 1 : (1 << bits) - 1;
    if (bits == 4)
        hipLaunchKernelGGL(pack_nchw<4>, dim3((unsigned)blocks), dim3(PK_THREADS), 0, stream, src,
                           static_cast<uint8_t *>(dst), c, hw, ptiles, ctiles, lo, hi);
    else
        hipLaunchKernelGGL(pack_nchw<8>, dim3((unsigned)blocks), dim3(PK_THREADS), 0, stream, src,
                           static_cast<uint8_t *>(dst), c, hw, ptiles, ctiles, lo, hi);
    return hipGetLastError();
}

}  // namespace qconv
