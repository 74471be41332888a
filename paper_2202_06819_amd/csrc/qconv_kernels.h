// Implicit-GEMM quantised convolution for gfx950 (CDNA4), int8 MFMA with
// int32 accumulation.
//
// GEMM view (Sec. 2.1): rows = output pixels m = (n, p, q), columns = output
// channels, depth = (r, s, c).  The MFMA's A operand is a filter block (16
// output channels x 64 depth values), B an activation block (64 depth values
// x 16 pixels); D = A * B holds 16 channels x 16 pixels.
//
// Staging (the duplicate-aware load of Sec. 3.1 / Alg. 1, restated): a
// workgroup owns TP consecutive output pixels.  Instead of loading the
// lowered matrix -- where every input pixel appears up to R*S times -- it
// copies once per channel chunk the band of zero-padded input rows those
// pixels touch into LDS.  A lowered row is then pure address arithmetic: the
// pixel's base offset in the band plus a per-tap offset that is the same for
// every lane.  Padding rows and columns are materialised as zeros in the band,
// so no lane tests a border in the main loop.
//
// Operands stay packed in HBM and LDS; 4-bit values are widened to int8 in
// VGPRs right before the MFMA (widen4).
//
// Output packing in registers (Sec. 3.2.3 and 3.3, restated for wave64): the
// MFMA result layout gives lane l the rows 4*(l/16)+v of the D tile.  Filters
// are placed in A so that D row i of fragment tm is output channel
// row_channel(tm, i) of the wave's block; each lane then ends with 4*FK
// consecutive channels of one pixel and packs whole 32-bit words without any
// cross-lane exchange.  The epilogue (requantise, ReLU, clamp, pack) runs on
// those registers and stores each pixel's channel run contiguously
// (Sec. 3.2.2: epilogue before the store).
//
// Two kernels share this design:
//   conv_staged  global -> VGPR -> LDS staging, one stage at a time; any
//                C that is a multiple of the packing word.
//   conv_wide    the packed operands of the next (tile, chunk) stage are
//                fetched into VGPRs while the MFMAs consume the current stage,
//                then widened once and written to LDS as int8, so the MFMA loop
//                itself carries no VALU work (widening inside that loop halves
//                MFMA throughput on gfx950); two stage buffers; a workgroup
//                walks several output tiles and keeps its filter block
//                resident in LDS when the whole depth fits one chunk.  Needs
//                every 16-byte vector of a pixel to be whole
//                (C*bits % 128 == 0).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>
#include <string.h>

#include <type_traits>

#include "qconv_device.h"
#include "qconv_internal.h"

namespace qconv {

// ============================================================== conv_staged

template <int BITS, int WP, int WK, int FP, int FK, int CK, bool EXT>
__global__ void __launch_bounds__(WP * WK * 64) conv_staged(ConvArgs a) {
    constexpr int NT = WP * WK * 64;
    constexpr int TP = WP * FP * 16;
    constexpr int TK = WK * FK * 16;
    constexpr int GRAN = 2 * BITS;          // bytes of a 16-channel granule
    constexpr int KSTEPS = CK / 64;         // MFMA depth steps per tap and chunk
    constexpr int VPP = CK * BITS / 128;    // 16-byte vectors per pixel and chunk
    constexpr int GPV = 16 / GRAN;          // granules per 16-byte vector
    constexpr int CPW = 32 / BITS;          // channels per 32-bit word
    constexpr int BATCH = 4;                // vectors in flight per thread while staging
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

    const int mt = (int)fdiv(blockIdx.x, a.div_ktiles);   // blockIdx.x / ktiles
    const int kt = (int)blockIdx.x - mt * a.ktiles;
    const int m0 = mt * TP;
    const int k0 = kt * TK;
    const int rs = a.r * a.s;

    int vlo, c_unused, vlast;
    pixel_origin(a, m0, vlo, c_unused);
    pixel_origin(a, min(m0 + TP, a.m) - 1, vlast, c_unused);
    const int nrows = vlast + a.r - vlo;   // <= a.band_rows (host-checked)

    int pixoff[FP];
#pragma unroll
    for (int tn = 0; tn < FP; ++tn) {
        int m = min(m0 + wp * FP * 16 + tn * 16 + l16, a.m - 1);
        int vr, cl;
        pixel_origin(a, m, vr, cl);
        pixoff[tn] = ((vr - vlo) * a.ncols + cl) * GRAN;
    }

    const int cb = k0 + wk * FK * 16 + gq * 4 * FK;
    v4i acc[FP][FK];
    if constexpr (EXT) {
        init_acc<FP, FK>(a, acc, a.bias ? a.bias + cb : nullptr, true, cb);
    } else {
#pragma unroll
        for (int tn = 0; tn < FP; ++tn)
#pragma unroll
            for (int tm = 0; tm < FK; ++tm) acc[tn][tm] = v4i{0, 0, 0, 0};
    }
    EpiParams<FK> ep;
    load_epilogue_params<FK>(a, cb, ep);

    const int nvec_band = nrows * a.ncols * VPP;
    const int nvec_w = TK * rs * VPP;

    for (int chunk = 0; chunk < a.nchunks; ++chunk) {
        const int cbyte = chunk * (CK * BITS / 8);
        const int cbase = chunk * CK;
        __syncthreads();
        // ---- band: global -> VGPR -> LDS; BATCH loads are issued before any is waited on
        for (int base = 0; base < nvec_band; base += NT * BATCH) {
            uint32_t d[BATCH][4];
#pragma unroll
            for (int u = 0; u < BATCH; ++u) {
                d[u][0] = d[u][1] = d[u][2] = d[u][3] = 0u;
                const int idx = base + u * NT + tid;
                if (idx >= nvec_band) continue;
                const int part = idx % VPP;
                const int pix = idx / VPP;
                const int rowl = (int)fdiv((uint32_t)pix, a.div_ncols);
                const int col = pix - rowl * a.ncols;
                const int vrow = vlo + rowl;
                const int img = (int)fdiv((uint32_t)vrow, a.div_vh);
                const int hh = vrow - img * a.vh - a.ph;
                const int ww = col - a.pw;
                if (img < a.n && hh >= 0 && hh < a.h && ww >= 0 && ww < a.w) {
                    const int ch0 = cbase + part * (128 / BITS);
                    const uint8_t *src = a.xptr + ((size_t)(img * a.h + hh) * a.w + ww) * a.xpix + cbyte + part * 16;
                    if (a.vec16 && ch0 + 128 / BITS <= a.c) {
                        uint4 v = *reinterpret_cast<const uint4 *>(src);
                        d[u][0] = v.x; d[u][1] = v.y; d[u][2] = v.z; d[u][3] = v.w;
                    } else {
#pragma unroll
                        for (int e = 0; e < 4; ++e)
                            if (ch0 + e * CPW < a.c) d[u][e] = reinterpret_cast<const uint32_t *>(src)[e];
                    }
                }
            }
#pragma unroll
            for (int u = 0; u < BATCH; ++u) {
                const int idx = base + u * NT + tid;
                if (idx >= nvec_band) continue;
                const int part = idx % VPP;
                const int off = (idx / VPP) * GRAN;
                if constexpr (BITS == 4) {
                    *reinterpret_cast<uint2 *>(band + (size_t)(part * GPV) * a.pstride_b + off) = uint2{d[u][0], d[u][1]};
                    *reinterpret_cast<uint2 *>(band + (size_t)(part * GPV + 1) * a.pstride_b + off) = uint2{d[u][2], d[u][3]};
                } else {
                    *reinterpret_cast<uint4 *>(band + (size_t)part * a.pstride_b + off) =
                        uint4{d[u][0], d[u][1], d[u][2], d[u][3]};
                }
            }
        }
        // ---- filters: TK channels x R*S taps of this chunk, in MFMA row order
        for (int base = 0; base < nvec_w; base += NT * BATCH) {
            uint32_t d[BATCH][4];
#pragma unroll
            for (int u = 0; u < BATCH; ++u) {
                d[u][0] = d[u][1] = d[u][2] = d[u][3] = 0u;
                const int idx = base + u * NT + tid;
                if (idx >= nvec_w) continue;
                const int part = idx % VPP;
                const int t = idx / VPP;
                const int slot = (int)fdiv((uint32_t)t, a.div_rs);
                const int tap = t - slot * rs;
                const int wkk = slot / (FK * 16);
                const int rem = slot % (FK * 16);
                const int kk = k0 + wkk * FK * 16 + row_channel<FK>(rem / 16, rem % 16);
                if (kk < a.k) {
                    const int ch0 = cbase + part * (128 / BITS);
                    const uint8_t *src = a.wptr + ((size_t)kk * rs + tap) * a.xpix + cbyte + part * 16;
                    if (a.vec16 && ch0 + 128 / BITS <= a.c) {
                        uint4 v = *reinterpret_cast<const uint4 *>(src);
                        d[u][0] = v.x; d[u][1] = v.y; d[u][2] = v.z; d[u][3] = v.w;
                    } else {
#pragma unroll
                        for (int e = 0; e < 4; ++e)
                            if (ch0 + e * CPW < a.c) d[u][e] = reinterpret_cast<const uint32_t *>(src)[e];
                    }
                }
            }
#pragma unroll
            for (int u = 0; u < BATCH; ++u) {
                const int idx = base + u * NT + tid;
                if (idx >= nvec_w) continue;
                const int part = idx % VPP;
                const int t = idx / VPP;
                const int slot = (int)fdiv((uint32_t)t, a.div_rs);
                const int tap = t - slot * rs;
                const int off = (tap * TK + slot) * GRAN;
                if constexpr (BITS == 4) {
                    *reinterpret_cast<uint2 *>(wlds + (size_t)(part * GPV) * a.pstride_w + off) = uint2{d[u][0], d[u][1]};
                    *reinterpret_cast<uint2 *>(wlds + (size_t)(part * GPV + 1) * a.pstride_w + off) = uint2{d[u][2], d[u][3]};
                } else {
                    *reinterpret_cast<uint4 *>(wlds + (size_t)part * a.pstride_w + off) =
                        uint4{d[u][0], d[u][1], d[u][2], d[u][3]};
                }
            }
        }
        __syncthreads();

        // ---- main loop over taps: LDS -> VGPR, widen, MFMA
        for (int rr = 0; rr < a.r; ++rr)
            for (int ss = 0; ss < a.s; ++ss) {
                const int tap = rr * a.s + ss;
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
    epilogue<BITS, FP, FK, EXT>(a, acc, m0 + wp * FP * 16, cb, l16, ep);
}

// ============================================================== conv_wide

// Widening of one packed 16-byte vector with the signedness fixed at compile
// time: 4-bit -> two 16-byte int8 granules (16 channels each, even channels
// then odd channels of every word, the same order for both operands), 8-bit ->
// itself.  3 VALU ops per packed 32-bit word.
template <int BITS, bool SIGNED>
__device__ __forceinline__ void widen_vec(uint4 v, uint4 &g0, uint4 &g1) {
    if constexpr (BITS == 8) {
        g0 = v;
        g1 = v;
    } else if constexpr (SIGNED) {
        g0 = uint4{(v.x << 4) & 0xF0F0F0F0u, v.x & 0xF0F0F0F0u, (v.y << 4) & 0xF0F0F0F0u, v.y & 0xF0F0F0F0u};
        g1 = uint4{(v.z << 4) & 0xF0F0F0F0u, v.z & 0xF0F0F0F0u, (v.w << 4) & 0xF0F0F0F0u, v.w & 0xF0F0F0F0u};
    } else {
        g0 = uint4{v.x & 0x0F0F0F0Fu, (v.x >> 4) & 0x0F0F0F0Fu, v.y & 0x0F0F0F0Fu, (v.y >> 4) & 0x0F0F0F0Fu};
        g1 = uint4{v.z & 0x0F0F0F0Fu, (v.z >> 4) & 0x0F0F0F0Fu, v.w & 0x0F0F0F0Fu, (v.w >> 4) & 0x0F0F0F0Fu};
    }
}

constexpr int kWideMaxV = 4;   // packed 16-byte filter vectors a thread gathers per batch
// MFMA steps whose LDS fragment reads are in flight ahead of the step being
// multiplied (fixed-size instances).  A wave's step of 2x2 fragments is 64
// MFMA cycles, well under an LDS read's latency with the CU's other waves
// reading too, so one step ahead leaves the wave waiting on LDS.
#ifndef QCONV_LDS_LOOKAHEAD
#define QCONV_LDS_LOOKAHEAD 2
#endif
constexpr int kLdsLookahead = QCONV_LDS_LOOKAHEAD;

// ---- the pack fused into the convolution (int8 N x C x H x W activations).
// Four int8 values of one channel -> the int8 MFMA operand bytes that
// widening the packed 4-bit values gives: saturated into [0, 15] (unsigned)
// or [-8, 7] and moved to the high nibble (signed, value * 16).  8-bit values
// pass unchanged.
template <int BITS, bool SIGNED>
__device__ __forceinline__ uint32_t saturate_operand(uint32_t x) {
    if constexpr (BITS == 8) {
        return x;
    } else if constexpr (!SIGNED) {
        if ((x & 0xF0F0F0F0u) == 0u) return x;                          // all in range
        const uint32_t neg = x & 0x80808080u;                           // negative bytes
        const uint32_t big = (((x & 0x7F7F7F7Fu) + 0x70707070u) & 0x80808080u) & ~neg;   // above 15
        uint32_t r = (x & 0x0F0F0F0Fu) | ((big >> 7) * 0x0Fu);
        return r & ~((neg >> 7) * 0xFFu);
    } else {
        uint32_t r = 0u;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int v = (int)(int8_t)(x >> (8 * i));
            const int c = v < -8 ? -8 : (v > 7 ? 7 : v);
            r |= ((uint32_t)(c << 4) & 0xF0u) << (8 * i);
        }
        return r;
    }
}

// 4x4 byte transpose: t[e] holds byte e of a0, a1, a2, a3 (in that order).
__device__ __forceinline__ void transpose4x4(uint32_t a0, uint32_t a1, uint32_t a2, uint32_t a3, uint32_t (&t)[4]) {
    const uint32_t lo01 = __builtin_amdgcn_perm(a1, a0, 0x05010400u);   // a0.b0 a1.b0 a0.b1 a1.b1
    const uint32_t hi01 = __builtin_amdgcn_perm(a1, a0, 0x07030602u);   // a0.b2 a1.b2 a0.b3 a1.b3
    const uint32_t lo23 = __builtin_amdgcn_perm(a3, a2, 0x05010400u);
    const uint32_t hi23 = __builtin_amdgcn_perm(a3, a2, 0x07030602u);
    t[0] = __builtin_amdgcn_perm(lo23, lo01, 0x05040100u);
    t[1] = __builtin_amdgcn_perm(lo23, lo01, 0x07060302u);
    t[2] = __builtin_amdgcn_perm(hi23, hi01, 0x05040100u);
    t[3] = __builtin_amdgcn_perm(hi23, hi01, 0x07060302u);
}

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef __attribute__((address_space(3))) void lds_void;
constexpr uint32_t kRsrcWord3 = 0x00020000u;   // raw buffer, dword data format (gfx9 family)

// Buffer resource for a read-only tensor of `bytes` bytes (wave-uniform).
// Loads at offsets >= bytes return zeros.
__device__ __forceinline__ u32x4 make_rsrc(const void *base, int32_t bytes) {
    const uint64_t b = (uint64_t)base;
    u32x4 r;
    r[0] = __builtin_amdgcn_readfirstlane((uint32_t)b);
    r[1] = __builtin_amdgcn_readfirstlane((uint32_t)(b >> 32));
    r[2] = __builtin_amdgcn_readfirstlane((uint32_t)bytes);
    r[3] = kRsrcWord3;
    return r;
}

constexpr uint32_t kOutOfRange = 0x80000000u;   // a buffer offset past every tensor: loads return 0
// Cache-policy operand of a buffer access that is coherent across the device
// (sc1): it is written through to, and read from, past the XCD's L2.
constexpr int kCoherentAux = 16;

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_brsrc(const void *base, int32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), (short)0, bytes, (int)kRsrcWord3);
}

__device__ __forceinline__ uint4 buffer_load16(__amdgpu_buffer_rsrc_t r, uint32_t off) {
    const auto v = __builtin_amdgcn_raw_buffer_load_b128(r, (int)off, 0, 0);
    return uint4{v[0], v[1], v[2], v[3]};
}

// Global memory straight into LDS (no VGPR round trip): lane i's 16 bytes
// (dma16) or 4 bytes (dma4) from buffer offset `voff` land at lds_dst + 16*i
// (or 4*i).  Inline assembly keeps the compiler from guarding later LDS reads
// with waits on these loads; the kernel waits explicitly.
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
__device__ __forceinline__ void dma16(const uint8_t *lds_dst, uint32_t voff, u32x4 rsrc) {
    const uint32_t m0v = __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)(lds_void *)lds_dst);
    asm volatile("s_mov_b32 m0, %0\n\tbuffer_load_dwordx4 %1, %2, 0 offen lds" : : "s"(m0v), "v"(voff), "s"(rsrc)
                 : "memory", "m0");
}
// dma16 with the LDS destination as a byte address, a scalar offset added to
// voff (one address register serves a run of copies), and the wave's lanes
// set to `lanes` (all or none) for the copy; exec is restored after it.  (A
// plain move, not an AND: the copy is a whole 1 KiB block either way, and no
// condition code is written behind the compiler's back.)
__device__ __forceinline__ void dma16m(uint32_t lds_addr, uint32_t voff, uint32_t soff, u32x4 rsrc,
                                       uint64_t lanes) {
    const uint32_t m0v = __builtin_amdgcn_readfirstlane(lds_addr);
    const uint32_t so = __builtin_amdgcn_readfirstlane(soff);
    const uint32_t half = __builtin_amdgcn_readfirstlane((uint32_t)lanes);   // all ones or zero
    const uint64_t mask = ((uint64_t)half << 32) | half;
    uint64_t saved;
    asm volatile(
        "s_mov_b64 %0, exec\n\t"
        "s_mov_b64 exec, %1\n\t"
        "s_mov_b32 m0, %2\n\t"
        "buffer_load_dwordx4 %3, %4, %5 offen lds\n\t"
        "s_mov_b64 exec, %0"
        : "=&s"(saved)
        : "s"(mask), "s"(m0v), "v"(voff), "s"(rsrc), "s"(so)
        : "memory", "m0");
}
__device__ __forceinline__ void dma4(const uint8_t *lds_dst, uint32_t voff, u32x4 rsrc) {
    const uint32_t m0v = __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)(lds_void *)lds_dst);
    asm volatile("s_mov_b32 m0, %0\n\tbuffer_load_dword %1, %2, 0 offen lds" : : "s"(m0v), "v"(voff), "s"(rsrc)
                 : "memory", "m0");
}
#pragma clang diagnostic pop

// Scheduling groups, in program order, for the instruction scheduler.
template <int N>
__device__ __forceinline__ void sched_lds_reads() { __builtin_amdgcn_sched_group_barrier(0x100, N, 0); }
template <int N>
__device__ __forceinline__ void sched_mfmas() { __builtin_amdgcn_sched_group_barrier(0x008, N, 0); }

// f(integral_constant<int, I>) for I = B .. E-1, unrolled at compile time (for
// scheduling-group counts that differ between steps).
template <int B, int E, typename F>
__device__ __forceinline__ void static_for(F &&f) {
    if constexpr (B < E) {
        f(std::integral_constant<int, B>{});
        static_for<B + 1, E>(f);
    }
}

// Workgroups are dispatched round-robin over the 8 XCDs, each with its own L2:
// block b runs on XCD b % 8.  Renumber them so that every XCD gets one
// contiguous range of logical blocks; neighbouring output tiles share halo
// rows, which then meet in the same L2.  A bijection for any grid size.
__device__ __forceinline__ int xcd_block(int b, int g) {
    constexpr int X = 8;
    const int x = b % X, i = b / X;
    const int q = g / X, r = g % X;
    return (x < r ? x * (q + 1) : r * (q + 1) + (x - r) * q) + i;
}

// RC, SC: filter height and width fixed at compile time (0: taken from the
// descriptor).  A fixed-size instance always reads prepared filters and runs a
// fully unrolled MFMA loop with immediate LDS offsets.
// ABL (ablation of the techniques, for measurement): bit 0 stages the lowered
// (im2col) operand instead of the band -- one copy of every pixel per filter
// tap, as without duplicate awareness; bit 1 sends the int32 accumulators
// through LDS to a separate requantise-and-pack pass instead of packing them
// in registers before the store; bit 2 (4-bit) keeps the staged activations
// packed in LDS and widens every fragment after its LDS read, inside the
// MFMA loop, instead of once when the band is written.
// PROJ: a 1x1 projection at the same stride is fused into a 3x3 instance (pad
// 1): its filter block is tap 9 of the prepared image, its input the centre
// tap's band pixels -- the fragments the 3x3 already reads -- and it keeps
// accumulators (split-K partial sums too), multipliers and an output of its
// own (no residual).
// ONE: the instance for plans whose workgroups each run a single stage (one
// tile, one chunk): it carries a copy of the stage compiled without the
// prefetch machinery (a workgroup with more stages still takes the general
// loop, so the instance is correct for any plan).
template <int BITS, int WP, int WK, int FP, int FK, int CK, bool XS, bool WS, int RC, int SC, bool EXT, int ABL = 0,
          bool MC = false, bool NCHW = false, bool PROJ = false, bool ONE = false, bool OCT = false>
__device__ __forceinline__ void wide_body(const ConvArgs &a) {
    constexpr bool FIXED = RC > 0 && SC > 0;
    constexpr bool LOWERED = (ABL & 1) != 0;
    constexpr bool LDSEPI = (ABL & 2) != 0;
    constexpr bool PACKEDLDS = (ABL & 4) != 0;
    constexpr int BPIX = PACKEDLDS ? 8 : 16;   // band bytes per pixel (or lowered entry) and granule plane
    static_assert(!PACKEDLDS || BITS == 4, "only 4-bit activations are packed");
    static_assert(!NCHW || (!LOWERED && !MC), "the fused pack stages the band itself");
    static_assert(ABL == 0 || (FIXED && !EXT), "ablation instances are fixed-size, without bias or residual");
    static_assert(!PROJ || (RC == 3 && SC == 3 && ABL == 0 && !MC && !NCHW), "the projection rides on a plain 3x3");
    static_assert(!ONE || (FIXED && !MC), "single-stage copies are made of the fixed-size instances");
    static_assert(!OCT || (NCHW && ONE), "the octet-rows copy is a single-stage fused-pack instance");
    constexpr int NW = WP * WK;
    constexpr int NT = NW * 64;
    constexpr int TP = WP * FP * 16;
    constexpr int TK = WK * FK * 16;
    constexpr int KSTEPS = CK / 64;
    constexpr int VPP = CK * BITS / 128;    // packed 16-byte vectors per pixel (or filter tap) and chunk
    constexpr int GPV = 16 / (2 * BITS);    // 16-channel int8 granules per packed vector
    constexpr int CPV = 128 / BITS;         // channels per packed vector
    // band pixels (lowered entries) a thread stages per chunk
    constexpr int PJ = LOWERED ? (RC * SC * TP + NT - 1) / NT : wide_band_pixels_per_thread(TP, NT, VPP);
    constexpr int MAXV = kWideMaxV;
    static_assert(BITS == 8 || FK % 2 == 0, "4-bit output packs 8 channels per word: FK must be even");
    static_assert(VPP >= 1 && 4 % VPP == 0, "a pixel's vectors must divide the per-thread budget");

    extern __shared__ __attribute__((aligned(16))) uint8_t smem[];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int wp = wave % WP;
    const int wk = wave / WP;
    const int l16 = lane & 15;
    const int gq = lane >> 4;

    // Work assignment.  Without a split, a workgroup walks output tiles j0,
    // j0 + gpk, ... of one channel tile over all channel chunks.  With a split
    // (a.splits > 1) it owns one output tile and the chunk range of its split;
    // the splits of a tile have consecutive logical numbers (one XCD).
    // Logical tiles lt are numbered channel tile fastest (xcd_order 0, 1:
    // consecutive workgroups share pixels, so an XCD reads its share of the
    // input and every channel tile's filters) or pixel tile fastest
    // (xcd_order 2: an XCD takes one channel tile's filters and the pixels).
    // (the divisions by launch constants use the host's multiply-shift divisors)
    const int lb = a.xcd_order ? xcd_block(blockIdx.x, gridDim.x) : (int)blockIdx.x;
    const int lt = (int)fdiv((uint32_t)lb, a.div_splits);   // lb / splits
    const int sp = lb - lt * a.splits;
    const int gpk = a.gpk;   // logical tiles per channel tile: workgroups sharing this channel tile
    const int ltk = (int)fdiv((uint32_t)lt, a.div_ktiles);   // lt / ktiles
    const int kt = a.xcd_order == 2 ? (int)fdiv((uint32_t)lt, a.div_gpk) : lt - ltk * a.ktiles;
    const int j0 = a.xcd_order == 2 ? lt - kt * gpk : ltk;
    const int my_tiles = (int)fdiv((uint32_t)(a.mtiles - j0 + gpk - 1), a.div_gpk);   // tiles j0, j0 + gpk, ...
    const int c_begin = sp * a.cps;                                     // chunks [c_begin, c_end)
    const int c_end = min(a.nchunks, c_begin + a.cps);
    const int nst = my_tiles * (c_end - c_begin);
    const int k0 = kt * TK;
    const int R = FIXED ? RC : a.r;
    const int S = FIXED ? SC : a.s;
    const int rs = R * S;
    const bool w_image = FIXED || a.w_image;

    const __amdgpu_buffer_rsrc_t rx = make_brsrc(a.xptr, a.xbytes);

    // ---- band staging.  The band of a tile is the run of zero-padded input
    // rows its pixels touch; thread tid stages band pixels tid, tid + NT, ...
    // Their byte offsets in x (or kOutOfRange for padding, which loads as
    // zeros) are computed once per tile and reused for every channel chunk.
    // Plane g of the LDS band holds granule g (channels 16g .. 16g+15 of the
    // chunk) of every band pixel, 16 bytes each: one write instruction fills
    // one plane contiguously.
    uint32_t poff[PJ];
    int npix = 0, band_vlo = 0;
    auto set_band = [&](int ti) {
        const int m0 = (j0 + ti * gpk) * TP;
        if constexpr (LOWERED) {
            // entry e = tap * TP + p: tile pixel p shifted by filter tap `tap`
            npix = RC * SC * TP;
#pragma unroll
            for (int j = 0; j < PJ; ++j) {
                const int e = j * NT + tid;
                const int tap = e / TP;
                const int p = e - tap * TP;
                int vr, cl;
                pixel_origin(a, min(m0 + p, a.m - 1), vr, cl);
                const int vrow = vr + tap / SC;
                const int col = cl + tap % SC;
                const int img = (int)fdiv((uint32_t)vrow, a.div_vh);
                const int hh = vrow - img * a.vh - a.ph;
                const int ww = col - a.pw;
                const bool in = e < npix && img < a.n && hh >= 0 && hh < a.h && ww >= 0 && ww < a.w;
                poff[j] = in ? (uint32_t)(((img * a.h + hh) * a.w + ww) * a.xpix) : kOutOfRange;
            }
            return;
        }
        int vlo, vlast, cu;
        pixel_origin(a, m0, vlo, cu);
        pixel_origin(a, min(m0 + TP, a.m) - 1, vlast, cu);
        npix = (vlast + R - vlo) * a.ncols;   // beyond NT * PJ: staged by band_rest
        band_vlo = vlo;
#pragma unroll
        for (int j = 0; j < PJ; ++j) {
            const int pix = j * NT + tid;
            const int rowl = (int)fdiv((uint32_t)pix, a.div_ncols);
            const int col = pix - rowl * a.ncols;
            const int vrow = vlo + rowl;
            const int img = (int)fdiv((uint32_t)vrow, a.div_vh);
            const int hh = vrow - img * a.vh - a.ph;
            const int ww = col - a.pw;
            const bool in = pix < npix && img < a.n && hh >= 0 && hh < a.h && ww >= 0 && ww < a.w;
            poff[j] = in ? (uint32_t)(((img * a.h + hh) * a.w + ww) * a.xpix) : kOutOfRange;
        }
    };
    struct Fetch {
        uint4 v[PJ][VPP];
    };
    auto band_fetch = [&](int c, Fetch &f) {
        const uint32_t cbyte = (uint32_t)c * (CK * BITS / 8);
        const int cbase = c * CK;
#pragma unroll
        for (int j = 0; j < PJ; ++j)
#pragma unroll
            for (int p = 0; p < VPP; ++p) {
                const bool ok = poff[j] != kOutOfRange && cbase + p * CPV < a.c;
                f.v[j][p] = buffer_load16(rx, ok ? poff[j] + cbyte + p * 16 : kOutOfRange);
            }
    };
    auto band_store = [&](const Fetch &f, int buf, int base = 0) {
        uint8_t *bb = smem + (buf ? a.off_b1 : a.off_b0);
#pragma unroll
        for (int j = 0; j < PJ; ++j) {
            const int pix = base + j * NT + tid;
            if (pix >= npix) continue;
#pragma unroll
            for (int p = 0; p < VPP; ++p) {
                if constexpr (PACKEDLDS) {
                    // each 16-channel granule stays two packed words (widened in the MFMA loop)
                    const uint4 v = f.v[j][p];
                    *reinterpret_cast<uint2 *>(bb + (size_t)(p * GPV) * a.pstride_b + pix * 8) = uint2{v.x, v.y};
                    *reinterpret_cast<uint2 *>(bb + (size_t)(p * GPV + 1) * a.pstride_b + pix * 8) = uint2{v.z, v.w};
                } else {
                    uint4 g0, g1;
                    widen_vec<BITS, XS>(f.v[j][p], g0, g1);
                    *reinterpret_cast<uint4 *>(bb + (size_t)(p * GPV) * a.pstride_b + pix * 16) = g0;
                    if constexpr (GPV == 2)
                        *reinterpret_cast<uint4 *>(bb + (size_t)(p * GPV + 1) * a.pstride_b + pix * 16) = g1;
                }
            }
        }
    };

    // Band pixels past the first NT * PJ (bands of strided layers can be
    // several times the tile): staged here in further rounds, each loaded and
    // written before the next, after the first round is in place.  8-bit
    // tiles only, whose per-thread budget is one pixel per round; compiled into
    // the 4-bit kernels the idle rounds cost 2-9 %, and their budget of two
    // pixels already covers the strided layers.
    auto band_rest = [&](int c, int buf) {
        if constexpr (!LOWERED && BITS == 8) {
            const uint32_t cbyte = (uint32_t)c * (CK * BITS / 8);
            const int cbase = c * CK;
            for (int base = NT * PJ; base < npix; base += NT * PJ) {
                Fetch f;
#pragma unroll
                for (int j = 0; j < PJ; ++j) {
                    const int pix = base + j * NT + tid;
                    const int rowl = (int)fdiv((uint32_t)pix, a.div_ncols);
                    const int col = pix - rowl * a.ncols;
                    const int vrow = band_vlo + rowl;
                    const int img = (int)fdiv((uint32_t)vrow, a.div_vh);
                    const int hh = vrow - img * a.vh - a.ph;
                    const int ww = col - a.pw;
                    const bool in = pix < npix && img < a.n && hh >= 0 && hh < a.h && ww >= 0 && ww < a.w;
                    const uint32_t off = in ? (uint32_t)(((img * a.h + hh) * a.w + ww) * a.xpix) : kOutOfRange;
#pragma unroll
                    for (int p = 0; p < VPP; ++p) {
                        const bool ok = off != kOutOfRange && cbase + p * CPV < a.c;
                        f.v[j][p] = buffer_load16(rx, ok ? off + cbyte + p * 16 : kOutOfRange);
                    }
                }
                band_store(f, buf, base);
            }
        }
    };

    // ---- band staging from int8 N x C x H x W (NCHW instances: the pack fused
    // into the convolution).  Item (band row, column quad, channel octet):
    // eight dwords -- 4 columns of one image row for each of 8 channels --
    // saturated like qconv_pack, transposed in registers into 4 pixels x 8
    // channels in the band's granule byte order, and written with one 8-byte
    // LDS store per pixel.  The granule of channels 16g .. 16g+15 keeps the
    // order the widening of packed values gives: 4-bit dwords hold channels
    // {0,2,4,6}, {1,3,5,7}, {8,10,..}, {9,11,..}; 8-bit ones 0..3, 4..7, ...
    // Padding columns are written as zeros; padding rows load as zeros.
    const __amdgpu_buffer_rsrc_t rsx = make_brsrc(a.xsrc, a.xsrc_bytes);
    auto band_rows_of = [&](int ti, int &vlo, int &nrows, int &vend_own) {
        const int m0 = (j0 + ti * gpk) * TP;
        int vlast, cu;
        pixel_origin(a, m0, vlo, cu);
        pixel_origin(a, min(m0 + TP, a.m) - 1, vlast, cu);
        nrows = vlast + R - vlo;
        // rows this tile writes to the packed copy: up to the next tile's first
        vend_own = vlast + R;
        if (m0 + TP < a.m) {
            int vnext;
            pixel_origin(a, m0 + TP, vnext, cu);
            vend_own = min(vend_own, vnext);
        }
    };
    // (`issued` runs once the first round's loads are out: the prologue puts
    // its filter and channel copies behind them)
    auto nchw_stage = [&](int ti, int c, int buf, auto &&issued) {
        uint8_t *bb = smem + (buf ? a.off_b1 : a.off_b0);
        int vlo, nrows, vend_own;
        band_rows_of(ti, vlo, nrows, vend_own);
        // the band rows' padding columns are zeros (stored while the first
        // round of loads is in flight)
        auto pad_zero = [&] {
            constexpr int NG = CK / 16;   // granule planes of a chunk
            const int npad = nrows * 2 * a.pw;
            for (int e = tid; e < npad * NG; e += NT) {
                const int g = e % NG, q = e / NG;
                const int rowl = (int)fdiv((uint32_t)q, a.div_pad2), side = q - rowl * 2 * a.pw;
                const int col = side < a.pw ? side : a.w + side;
                *reinterpret_cast<uint4 *>(bb + (size_t)g * a.pstride_b + (rowl * a.ncols + col) * 16) =
                    uint4{0u, 0u, 0u, 0u};
            }
        };
        constexpr int NCO = CK / 8;   // channel octets of a chunk
        constexpr int IB = 2;         // items a thread has in flight at once
        // items run column quad fastest, then band row, then channel octet:
        // a channel's band rows are contiguous in NCHW, so the lanes of one
        // load instruction read one contiguous run (rows up to band_rows, the
        // most any tile's band has; this tile's extra ones are skipped)
        const int nwq = (a.w + 3) >> 2;
        // (OCT instances run only for rows of whole pixel octets, and carry
        // no code for other widths: the smaller kernel launches faster)
        if (OCT || (a.w & 7) == 0) {
            // rows of whole pixel octets: an item is 8 channels x 8 pixels, one
            // 8-byte load per channel (half the load instructions of quads).
            // Items run channel-octet parity fastest, then band row (rows
            // rounded up to 4), then column octet, then octet pair: an item's
            // eight pixel stores lie 128 bytes apart per lane, so lanes that
            // differ in row and octet parity are what spreads one store
            // instruction over the LDS banks
            const int nwo = a.w >> 3;
            const int rb4 = (a.band_rows + 3) & ~3;
            const int items8 = NCO * rb4 * nwo;
            const int hw = a.h * a.w;
            for (int base = 0; base < items8; base += NT) {
                const int it = base + tid;
                const int q = it >> 1;
                const int rest = (int)fdiv((uint32_t)q, a.div_rb4), rowl = q - rest * rb4;
                const int cp = (int)fdiv((uint32_t)(2 * rest), a.div_wq);   // rest / nwo (nwq = 2 nwo)
                const int wo = rest - cp * nwo;
                const int co = 2 * cp + (it & 1);
                const bool in_band = it < items8 && rowl < nrows;
                const int vrow = vlo + rowl;
                const int img = (int)fdiv((uint32_t)vrow, a.div_vh);
                const int hh = vrow - img * a.vh - a.ph;
                const bool row_ok = in_band && img < a.n && hh >= 0 && hh < a.h;
                const int ww0 = wo * 8;
                const int ch0 = c * CK + co * 8;
                const int off0 = row_ok && ch0 < a.c ? (((img * a.c + ch0) * a.h + hh) * a.w) + ww0 : (int)kOutOfRange;
                u32x2 L[8];
#pragma unroll
                for (int k = 0; k < 8; ++k) L[k] = __builtin_amdgcn_raw_buffer_load_b64(rsx, off0, k * hw, 0);
                if (base == 0) {
                    issued();
                    pad_zero();
                }
                if (!in_band) continue;
                uint32_t any = 0u;
#pragma unroll
                for (int k = 0; k < 8; ++k) any |= L[k][0] | L[k][1];
                if (BITS == 8 || XS || (any & 0xF0F0F0F0u) != 0u) {
#pragma unroll
                    for (int k = 0; k < 8; ++k) {
                        L[k][0] = saturate_operand<BITS, XS>(L[k][0]);
                        L[k][1] = saturate_operand<BITS, XS>(L[k][1]);
                    }
                }
                uint8_t *dst = bb + (size_t)(co >> 1) * a.pstride_b + (rowl * a.ncols + a.pw + ww0) * 16 + (co & 1) * 8;
#pragma unroll
                for (int hf = 0; hf < 2; ++hf) {
                    uint32_t d0[4], d1[4];
                    if constexpr (BITS == 4) {
                        transpose4x4(L[0][hf], L[2][hf], L[4][hf], L[6][hf], d0);
                        transpose4x4(L[1][hf], L[3][hf], L[5][hf], L[7][hf], d1);
                    } else {
                        transpose4x4(L[0][hf], L[1][hf], L[2][hf], L[3][hf], d0);
                        transpose4x4(L[4][hf], L[5][hf], L[6][hf], L[7][hf], d1);
                    }
#pragma unroll
                    for (int e = 0; e < 4; ++e)
                        *reinterpret_cast<uint2 *>(dst + (hf * 4 + e) * 16) = uint2{d0[e], d1[e]};
                }
            }
            return;
        }
        if constexpr (OCT) return;
        const int items = NCO * a.band_rows * nwq;
        const bool dwords = (a.w & 3) == 0;
        for (int base = 0; base < items; base += NT * IB) {
            uint32_t L[IB][8];
            int pix0[IB], nvalid[IB], plane[IB], half[IB];
#pragma unroll
            for (int u = 0; u < IB; ++u) {
                const int it = base + u * NT + tid;
                const int t = (int)fdiv((uint32_t)it, a.div_wq);
                const int wq = it - t * nwq;
                const int co = (int)fdiv((uint32_t)t, a.div_brows), rowl = t - co * a.band_rows;
                const bool in_band = it < items && rowl < nrows;
                const int vrow = vlo + rowl;
                const int img = (int)fdiv((uint32_t)vrow, a.div_vh);
                const int hh = vrow - img * a.vh - a.ph;
                const bool row_ok = in_band && img < a.n && hh >= 0 && hh < a.h;
                const int ww0 = wq * 4;
                const int ch0 = c * CK + co * 8;
                pix0[u] = in_band ? rowl * a.ncols + a.pw + ww0 : -1;
                nvalid[u] = min(4, a.w - ww0);
                plane[u] = co >> 1;
                half[u] = (co & 1) * 8;
                // channel ch0 + k lies k planes on: one vector offset for the
                // octet, the plane step as the scalar offset (c is a multiple of
                // 8, so the octet is in range or out as a whole; an offset from
                // kOutOfRange stays past the tensor)
                const int off0 = row_ok && ch0 < a.c ? (((img * a.c + ch0) * a.h + hh) * a.w) + ww0 : (int)kOutOfRange;
#pragma unroll
                for (int k = 0; k < 8; ++k) {
                    const bool ok = row_ok && ch0 + k < a.c;
                    const uint32_t off = (uint32_t)((((img * a.c + ch0 + k) * a.h + hh) * a.w) + ww0);
                    if (dwords) {
                        L[u][k] = __builtin_amdgcn_raw_buffer_load_b32(rsx, off0, k * a.h * a.w, 0);
                    } else {
                        uint32_t v = 0u;
#pragma unroll
                        for (int e = 0; e < 4; ++e)
                            v |= (uint32_t)__builtin_amdgcn_raw_buffer_load_b8(
                                     rsx, ok && e < nvalid[u] ? (int)(off + e) : (int)kOutOfRange, 0, 0)
                                 << (8 * e);
                        L[u][k] = v;
                    }
                }
            }
            if (base == 0) {
                issued();
                pad_zero();
            }
#pragma unroll
            for (int u = 0; u < IB; ++u) {
                if (pix0[u] < 0) continue;
                // (4-bit unsigned: one test for the common case of an octet
                // already in range)
                uint32_t any = 0u;
#pragma unroll
                for (int k = 0; k < 8; ++k) any |= L[u][k];
                if (BITS == 8 || XS || (any & 0xF0F0F0F0u) != 0u) {
#pragma unroll
                    for (int k = 0; k < 8; ++k) L[u][k] = saturate_operand<BITS, XS>(L[u][k]);
                }
                uint32_t d0[4], d1[4];
                if constexpr (BITS == 4) {
                    transpose4x4(L[u][0], L[u][2], L[u][4], L[u][6], d0);
                    transpose4x4(L[u][1], L[u][3], L[u][5], L[u][7], d1);
                } else {
                    transpose4x4(L[u][0], L[u][1], L[u][2], L[u][3], d0);
                    transpose4x4(L[u][4], L[u][5], L[u][6], L[u][7], d1);
                }
                uint8_t *dst = bb + (size_t)plane[u] * a.pstride_b + pix0[u] * 16 + half[u];
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    if (e < nvalid[u]) *reinterpret_cast<uint2 *>(dst + e * 16) = uint2{d0[e], d1[e]};
            }
        }
    };
    // The packed copy of the input (qconv_pack's output), for the rows this
    // tile owns -- from its band's first row up to the next tile's -- and this
    // chunk's channels: each (pixel, granule) read back from the band and
    // repacked (the inverse of the widening).
    // (threads first, first + step, ... of the workgroup take the units)
    auto nchw_write_packed = [&](int ti, int c, int buf, int first, int step) {
        const uint8_t *bb = smem + (buf ? a.off_b1 : a.off_b0);
        int vlo, nrows, vend_own;
        band_rows_of(ti, vlo, nrows, vend_own);
        constexpr int NG = CK / 16;
        // a unit is one pixel's granules of this chunk: the lanes of a wave read
        // consecutive pixels of one plane (256 contiguous bytes per 16 lanes, no
        // bank conflicts) and write consecutive pixels' packed runs
        const int units = (vend_own - vlo) * a.w;
        const int ng = min(NG, (a.c - c * CK + 15) / 16);   // granules of this chunk inside c
        for (int t = first; t < units; t += step) {
            const int rowl = (int)fdiv((uint32_t)t, a.div_w), ww = t - rowl * a.w;
            const int vrow = vlo + rowl;
            const int img = (int)fdiv((uint32_t)vrow, a.div_vh);
            const int hh = vrow - img * a.vh - a.ph;
            if (img >= a.n || hh < 0 || hh >= a.h) continue;
            const uint8_t *src = bb + (rowl * a.ncols + a.pw + ww) * 16;
            const size_t pix = ((size_t)img * a.h + hh) * a.w + ww;
#pragma unroll
            for (int g = 0; g < NG; ++g) {
                if (g >= ng) break;
                const uint4 v = *reinterpret_cast<const uint4 *>(src + (size_t)g * a.pstride_b);
                const int ch0 = c * CK + g * 16;
                if constexpr (BITS == 4) {
                    uint2 w;
                    if constexpr (XS) {
                        w.x = ((v.x >> 4) & 0x0F0F0F0Fu) | (v.y & 0xF0F0F0F0u);
                        w.y = ((v.z >> 4) & 0x0F0F0F0Fu) | (v.w & 0xF0F0F0F0u);
                    } else {
                        w.x = (v.x & 0x0F0F0F0Fu) | ((v.y & 0x0F0F0F0Fu) << 4);
                        w.y = (v.z & 0x0F0F0F0Fu) | ((v.w & 0x0F0F0F0Fu) << 4);
                    }
                    *reinterpret_cast<uint2 *>(a.xpk + pix * (a.c / 2) + ch0 / 2) = w;
                } else {
                    *reinterpret_cast<uint4 *>(a.xpk + pix * a.c + ch0) = v;
                }
            }
        }
    };

    // ---- filter staging.  Prepared filters (a.w_image): the block of this
    // channel tile and chunk is already the LDS image (int8, MFMA row order,
    // planes of pstride_w bytes), copied with asynchronous LDS-DMA.  Otherwise
    // the packed KRSC filters are gathered, widened and written here; lanes run
    // along filter slots so LDS writes stay contiguous.
    const u32x4 rimg = make_rsrc(a.wptr, a.wbytes);
    auto w_dma = [&](int c, int buf) {
        uint8_t *wb = smem + (buf ? a.off_w1 : a.off_w0);
        const uint32_t base = (uint32_t)((kt * a.nchunks + c) * (CK / 16) * a.pstride_w);
        const int nkb = (CK / 16) * a.pstride_w / 1024;
        for (int i = wave; i < nkb; i += NW) dma16(wb + i * 1024, base + i * 1024 + lane * 16, rimg);
    };
    struct WFetch {
        uint4 v[MAXV];
    };
    auto w_gather = [&](int c, int base, WFetch &f) {
        const int n = TK * rs * VPP;
        const int cbyte = c * (CK * BITS / 8);
        const int cbase = c * CK;
#pragma unroll
        for (int u = 0; u < MAXV; ++u) {
            f.v[u] = uint4{0u, 0u, 0u, 0u};
            const int idx = base + u * NT + tid;
            if (idx >= n) continue;
            // idx = (part * rs + tap) * TK + slot
            const int slot = idx % TK;
            const int rest = idx / TK;
            const int pt = (int)fdiv((uint32_t)rest, a.div_rs);
            const int tap = rest - pt * rs;
            const int kk = k0 + (slot / (FK * 16)) * FK * 16 + row_channel<FK>((slot % (FK * 16)) / 16, slot % 16);
            if (kk < a.k && cbase + pt * CPV < a.c)
                f.v[u] = *reinterpret_cast<const uint4 *>(a.wptr + ((size_t)kk * rs + tap) * a.xpix + cbyte + pt * 16);
        }
    };
    auto w_gather_store = [&](const WFetch &f, int base, int buf) {
        const int n = TK * rs * VPP;
        uint8_t *wb = smem + (buf ? a.off_w1 : a.off_w0);
#pragma unroll
        for (int u = 0; u < MAXV; ++u) {
            const int idx = base + u * NT + tid;
            if (idx >= n) continue;
            const int slot = idx % TK;
            const int rest = idx / TK;
            const int pt = (int)fdiv((uint32_t)rest, a.div_rs);
            const int tap = rest - pt * rs;
            uint4 g0, g1;
            widen_vec<BITS, WS>(f.v[u], g0, g1);
            const int e = (tap * TK + slot) * 16;
            *reinterpret_cast<uint4 *>(wb + (size_t)(pt * GPV) * a.pstride_w + e) = g0;
            if constexpr (GPV == 2) *reinterpret_cast<uint4 *>(wb + (size_t)(pt * GPV + 1) * a.pstride_w + e) = g1;
        }
    };
    auto w_load_all = [&](int c, int buf) {
        if constexpr (!FIXED) {
            const int n = TK * rs * VPP;
            for (int base = 0; base < n; base += NT * MAXV) {
                WFetch f;
                w_gather(c, base, f);
                w_gather_store(f, base, buf);
            }
        }
    };

    const int lane_b = gq * a.pstride_b;
    const int lane_a = gq * a.pstride_w + (wk * FK * 16 + l16) * 16;
    int pixoff[FP];
    auto set_tile = [&](int ti) {
        const int m0 = (j0 + ti * gpk) * TP;
        if constexpr (LOWERED) {
#pragma unroll
            for (int tn = 0; tn < FP; ++tn) pixoff[tn] = (wp * FP * 16 + tn * 16 + l16) * BPIX + lane_b;
            return;
        }
        int vlo, cu;
        pixel_origin(a, m0, vlo, cu);
#pragma unroll
        for (int tn = 0; tn < FP; ++tn) {
            int m = min(m0 + wp * FP * 16 + tn * 16 + l16, a.m - 1);
            int vr, cl;
            pixel_origin(a, m, vr, cl);
            pixoff[tn] = ((vr - vlo) * a.ncols + cl) * BPIX + lane_b;
        }
    };

    v4i acc[FP][FK];
#pragma unroll
    for (int tn = 0; tn < FP; ++tn)
#pragma unroll
        for (int tm = 0; tm < FK; ++tm) acc[tn][tm] = v4i{0, 0, 0, 0};
    // the projection's accumulators (PROJ)
    v4i acc2[PROJ ? FP : 1][PROJ ? FK : 1];
#pragma unroll
    for (int tn = 0; tn < (PROJ ? FP : 1); ++tn)
#pragma unroll
        for (int tm = 0; tm < (PROJ ? FK : 1); ++tm) acc2[tn][tm] = v4i{0, 0, 0, 0};
    // the projection's epilogue reads the same fields as the main one
    ConvArgs ap = a;
    if constexpr (PROJ) {
        ap.yptr = a.yproj;
        ap.mult = a.mult2;
        ap.bias = a.bias2;
        ap.shift = a.shift2;
        ap.lo = a.lo2;
        ap.hi = a.hi2;
        ap.res = nullptr;
    }

    const int cb = k0 + wk * FK * 16 + gq * 4 * FK;
    // the workgroup's TK multipliers (and biases) go to LDS by DMA, read back
    // for the epilogue; channels past k repeat the last one and are never stored
    // (PROJ: the projection's follow at mlds2 = mlds + 2*TK + 4)
    int32_t *mlds = reinterpret_cast<int32_t *>(smem + a.off_m);
    int32_t *blds = mlds + TK;
    int32_t *mlds2 = mlds + 2 * TK + 4;
    int32_t *blds2 = mlds2 + TK;
    auto dma_channels = [&](int32_t *dst, const int32_t *src) {
        const u32x4 r = make_rsrc(src, 4 * a.k);
        for (int e = 0; e < TK; e += 64)
            if (e + lane < TK)   // TK may be 32: only the lanes of the buffer write
                dma4(reinterpret_cast<const uint8_t *>(dst + e), (uint32_t)min(k0 + e + lane, a.k - 1) * 4u, r);
    };
    auto channel_dmas = [&] {
        if (a.mode == QCONV_OUT_REQUANT && wave == 0) dma_channels(mlds, a.mult);
        if (EXT && a.mode == QCONV_OUT_REQUANT && a.bias && wave == (NW > 1 ? 1 : 0)) dma_channels(blds, a.bias);
        if constexpr (PROJ) {
            if (a.mode == QCONV_OUT_REQUANT && wave == (NW > 2 ? 2 : 0)) dma_channels(mlds2, a.mult2);
            if (EXT && a.mode == QCONV_OUT_REQUANT && a.bias2 && wave == (NW > 3 ? 3 : 0))
                dma_channels(blds2, a.bias2);
        }
    };

    // ---- prologue: stage 0 (every load in flight before the first wait).
    // The band's loads go out first: they come from HBM, while the filter
    // image and the channel parameters, read by every workgroup of the
    // channel tile, mostly come from L2.
    if (nst > 0) {
        if constexpr (NCHW) {
            nchw_stage(0, c_begin, 0, [&] {
                if (w_image) w_dma(c_begin, 0);
                channel_dmas();
            });
            __builtin_amdgcn_s_waitcnt(0);
        } else {
            set_band(0);
            Fetch fb;
            band_fetch(c_begin, fb);
            if (w_image) w_dma(c_begin, 0);
            channel_dmas();
            if (!w_image) w_load_all(c_begin, 0);
            __builtin_amdgcn_s_waitcnt(0);
            band_store(fb, 0);
            band_rest(c_begin, 0);
        }
    }
    set_tile(0);
    __syncthreads();

    // the workgroup keeps one channel tile: its epilogue multipliers are read
    // from LDS and prepared once
    EpiParams<FK> ep, ep2;
    auto lds_epilogue_params = [&](const ConvArgs &aa, const int32_t *ml, EpiParams<FK> &e2) {
        if (aa.mode == QCONV_OUT_REQUANT) {
            int32_t mraw[4 * FK];
#pragma unroll
            for (int e = 0; e < 4 * FK; e += 4) {
                const int4 q = *reinterpret_cast<const int4 *>(ml + cb - k0 + e);
                mraw[e] = q.x; mraw[e + 1] = q.y; mraw[e + 2] = q.z; mraw[e + 3] = q.w;
            }
            make_epilogue_params<FK>(aa, mraw, e2);
        } else {
            e2.fast = false;
        }
    };
    // accumulators start from the bias (in the first split of a tile only)
    const bool bias_here = EXT && a.mode == QCONV_OUT_REQUANT && a.bias && sp == 0;
    const bool bias2_here = PROJ && EXT && a.mode == QCONV_OUT_REQUANT && a.bias2 && sp == 0;
    if (!ONE || nst != 1) {
        lds_epilogue_params(a, mlds, ep);
        if constexpr (PROJ) lds_epilogue_params(ap, mlds2, ep2);
        if (bias_here) init_acc<FP, FK>(a, acc, blds + cb - k0, false, cb);
        if constexpr (PROJ)
            if (bias2_here) init_acc<FP, FK>(ap, acc2, blds2 + cb - k0, false, cb);
    }
    // (a single stage prepares them once its MFMAs are issued, and adds the
    // bias to the finished sums in the workgroup that runs the epilogue)

    const int nit = rs * KSTEPS;

    // Ablation: the tile's int32 accumulators go to LDS; then every thread takes
    // whole output words (pixel, CPW channels), requantises, packs and stores
    // them.  Two barriers per tile.
    auto lds_epilogue = [&](int ti) {
        int32_t *elds = reinterpret_cast<int32_t *>(smem + a.off_e);
        const int pl0 = wp * FP * 16 + l16;
#pragma unroll
        for (int tn = 0; tn < FP; ++tn)
#pragma unroll
            for (int tm = 0; tm < FK; ++tm) {
                const v4i v = acc[tn][tm];
                *reinterpret_cast<int4 *>(elds + (pl0 + tn * 16) * TK + (cb - k0) + 4 * tm) = int4{v[0], v[1], v[2], v[3]};
            }
        __syncthreads();
        const int m0 = (j0 + ti * gpk) * TP;
        if (a.mode == QCONV_OUT_RAW_I32) {
            for (int i = tid; i < TP * TK / 4; i += NT) {
                const int pl = i / (TK / 4), c4 = (i - pl * (TK / 4)) * 4;
                const int m = m0 + pl;
                if (m >= a.m || k0 + c4 >= a.k) continue;
                const int4 q = *reinterpret_cast<const int4 *>(elds + pl * TK + c4);
                *reinterpret_cast<int4 *>(reinterpret_cast<int32_t *>(a.yptr) + (size_t)m * a.k + k0 + c4) =
                    int4{q.x >> a.acc_shift, q.y >> a.acc_shift, q.z >> a.acc_shift, q.w >> a.acc_shift};
            }
        } else {
            constexpr int CPW = 32 / BITS;
            constexpr uint32_t VMASK = (1u << BITS) - 1u;
            const int e = 32 - a.shift - a.acc_shift;
            const int64_t rnd = (int64_t)1 << (a.shift - 1);
            for (int i = tid; i < TP * TK / CPW; i += NT) {
                const int pl = i / (TK / CPW), c0 = (i - pl * (TK / CPW)) * CPW;
                const int m = m0 + pl;
                if (m >= a.m || k0 + c0 >= a.k) continue;
                uint32_t word = 0u;
#pragma unroll
                for (int qv = 0; qv < CPW; ++qv) {
                    const int32_t v = elds[pl * TK + c0 + qv];
                    const int32_t mu = mlds[c0 + qv];
                    int64_t t;
                    if (e >= 0 && (e == 0 || (uint32_t)mu + (1u << (31 - e)) < (2u << (31 - e))))
                        t = ((int64_t)v * (int32_t)((uint32_t)mu << e) + ((int64_t)1 << 31)) >> 32;
                    else
                        t = ((int64_t)(v >> a.acc_shift) * mu + rnd) >> a.shift;
                    t = t < a.lo ? a.lo : (t > a.hi ? a.hi : t);
                    word |= ((uint32_t)(int32_t)t & VMASK) << (BITS * qv);
                }
                *reinterpret_cast<uint32_t *>(a.yptr + (size_t)m * (a.k * BITS / 8) + (k0 + c0) * BITS / 8) = word;
            }
        }
        __syncthreads();
    };

    // One stage: the MFMAs over the staged chunk (with the next stage's
    // operands in flight), then the tile's epilogue after its last chunk.  In
    // ONE instances a workgroup with a single stage (one tile, one chunk: most
    // single-chunk layers) runs a copy compiled without the prefetch
    // machinery, so none of its set-up -- which the compiler hoists ahead of
    // the loop -- sits between the first barrier and the first MFMA, and its
    // epilogue multipliers are prepared after the MFMAs are issued.  (Kept in
    // instances of their own: the second copy changes the general loop's
    // register allocation.)
    int ti = 0, c = c_begin;
    auto stage = [&](int st, auto single) {
        constexpr bool SINGLE = decltype(single)::value;
        int nti = ti, nc = c + 1;
        if (nc == c_end) {
            nc = c_begin;
            ++nti;
        }
        const int cur = SINGLE ? 0 : st & 1;
        const bool more = !SINGLE && st + 1 < nst;
        // prefetch the next stage; it lands while the MFMAs run
        Fetch fb;
        WFetch fw;
        if (more) {
            if constexpr (!NCHW) {
                if (nti != ti) set_band(nti);
                band_fetch(nc, fb);
            }
            if (c_end - c_begin > 1) {
                // (the multi-chunk instances issue their filter DMA inside the MFMA loop)
                if (w_image) {
                    if constexpr (!MC) w_dma(nc, cur ^ 1);
                } else if constexpr (!FIXED) {
                    w_gather(nc, 0, fw);
                }
            }
        }

        // ---- MFMA loop: int8 fragments straight from LDS, one step of lookahead
        if constexpr (NCHW && SINGLE) {
            // a single stage writes the packed copy before its MFMAs, from the
            // upper half of the waves only: each shares its SIMD with a
            // lower-half wave, whose MFMAs run meanwhile
            constexpr int WH = NW > 1 ? NW / 2 : 0;
            if (a.xpk && wave >= WH) nchw_write_packed(ti, c, cur, tid - WH * 64, NT - WH * 64);
        }
        const uint8_t *bb = smem + (cur ? a.off_b1 : a.off_b0);
        const uint8_t *wb = smem + ((c_end - c_begin > 1 && cur) ? a.off_w1 : a.off_w0) + lane_a;
        auto offs = [&](int it, int &ao, int &bo) {
            const int tap = it / KSTEPS;
            const int ks = it % KSTEPS;
            const int rr = (int)fdiv((uint32_t)tap, a.div_s);
            const int ss = tap - rr * a.s;
            ao = ks * 4 * a.pstride_w + tap * TK * 16;
            bo = ks * 4 * a.pstride_b + (rr * a.ncols + ss * a.tap_w) * 16;
        };
        if constexpr (FIXED) {
            // every step's LDS offsets are known: filter reads use immediate
            // offsets from one base; band reads from one base per (fragment,
            // filter row, depth step) plus the column as an immediate
            constexpr int TAPS_IMG = RC * SC + (PROJ ? 1 : 0);   // taps in the filter image
            constexpr int PSW = (TAPS_IMG * TK * 16 + 1023) / 1024 * 1024;   // filter plane stride
            constexpr int NIT = RC * SC * KSTEPS;
            constexpr int CT = (RC / 2) * SC + SC / 2;   // the centre tap (the projection's pixels)
            const uint8_t *wa = wb;
            const uint8_t *brow[FP][RC][KSTEPS];
#pragma unroll
            for (int tn = 0; tn < FP; ++tn)
#pragma unroll
                for (int rr = 0; rr < RC; ++rr)
#pragma unroll
                    for (int ks = 0; ks < KSTEPS; ++ks)
                        brow[tn][rr][ks] = bb + pixoff[tn] + (LOWERED ? rr * SC * TP : rr * a.ncols) * BPIX +
                                           ks * 4 * a.pstride_b;
            // LA steps of fragments in flight: register sets rotate over NS = LA + 1
            // (larger sets -- 4x4 fragments, or 2x4 with a projection -- keep
            // one: their steps are longer and their registers are spoken for)
            constexpr int LA0 = FK + FP + (PROJ ? FK : 0) <= 6 ? kLdsLookahead : 1;
            constexpr int LA = LA0 < NIT ? LA0 : NIT;
            constexpr int NS = LA + 1;
            v4i A[NS][FK], B[NS][FP];
            v4i Ap[NS][PROJ ? FK : 1];   // the projection's filter fragments at the centre tap
            // Multi-chunk instances (MC): the next chunk's filter block goes out
            // as 1 KiB LDS-DMA copies spread over the MFMA steps (about one per
            // step and wave); issued all at once before the loop they queue
            // behind each other in the address unit and hold the wave off its
            // MFMAs.  The last stage runs the same copies with no lanes enabled,
            // so no branch splits the loop's schedule.  A wave whose share is
            // one short repeats the last block: the same bytes to the same
            // place.  (Single-chunk layers keep the instances without them: the
            // copies constrain the loop's schedule even when idle.)
            constexpr int NKB = (CK / 16) * PSW / 1024;
            constexpr int DPW = (NKB + NW - 1) / NW;
            const uint64_t dma_lanes = (more && c_end - c_begin > 1) ? ~0ull : 0ull;
            const uint32_t wnext = (uint32_t)(uintptr_t)(lds_void *)smem + ((cur ^ 1) ? a.off_w1 : a.off_w0);
            const uint32_t wblk = (uint32_t)((kt * a.nchunks + nc) * (CK / 16) * PSW) + lane * 16;
            auto dma_step = [&](int it) {
#pragma unroll
                for (int j = it * DPW / NIT; j < (it + 1) * DPW / NIT; ++j) {
                    const int i = min(wave + j * NW, NKB - 1);
                    dma16m(wnext + (uint32_t)i * 1024u, wblk, (uint32_t)i * 1024u, rimg, dma_lanes);
                }
            };
            auto ld = [&](int it, int set) {
                const int tap = it / KSTEPS, ks = it % KSTEPS, rr = tap / SC, ss = tap % SC;
#pragma unroll
                for (int tm = 0; tm < FK; ++tm)
                    A[set][tm] = *reinterpret_cast<const v4i *>(wa + ks * 4 * PSW + tap * TK * 16 + tm * 256);
#pragma unroll
                for (int tn = 0; tn < FP; ++tn) {
                    const uint8_t *bp = brow[tn][rr][ks] + ss * (LOWERED ? TP : 1) * BPIX;
                    if constexpr (PACKEDLDS) {
                        const uint2 v = *reinterpret_cast<const uint2 *>(bp);
                        uint4 g0, g1;
                        widen_vec<BITS, XS>(uint4{v.x, v.y, 0u, 0u}, g0, g1);
                        B[set][tn] = v4i{(int)g0.x, (int)g0.y, (int)g0.z, (int)g0.w};
                    } else {
                        B[set][tn] = *reinterpret_cast<const v4i *>(bp);
                    }
                }
                if constexpr (PROJ) {
                    if (tap == CT) {
#pragma unroll
                        for (int tm = 0; tm < FK; ++tm)
                            Ap[set][tm] = *reinterpret_cast<const v4i *>(wa + ks * 4 * PSW + RC * SC * TK * 16 + tm * 256);
                    }
                }
            };
#pragma unroll
            for (int it = 0; it < LA; ++it) ld(it, it);
#pragma unroll
            for (int it = 0; it < NIT; ++it) {
                if constexpr (MC) dma_step(it);
                if (it + LA < NIT) ld(it + LA, (it + LA) % NS);
#pragma unroll
                for (int tn = 0; tn < FP; ++tn)
#pragma unroll
                    for (int tm = 0; tm < FK; ++tm)
                        acc[tn][tm] = __builtin_amdgcn_mfma_i32_16x16x64_i8(A[it % NS][tm], B[it % NS][tn], acc[tn][tm],
                                                                            0, 0, 0);
                if constexpr (PROJ) {
                    if (it / KSTEPS == CT) {
                        // the same activation fragments times the projection's filters
#pragma unroll
                        for (int tn = 0; tn < FP; ++tn)
#pragma unroll
                            for (int tm = 0; tm < FK; ++tm)
                                acc2[tn][tm] = __builtin_amdgcn_mfma_i32_16x16x64_i8(Ap[it % NS][tm], B[it % NS][tn],
                                                                                     acc2[tn][tm], 0, 0, 0);
                    }
                }
            }
            // Pin the issue order (the scheduler otherwise reuses one register
            // set and waits on every read): the LDS reads of step it+LA go out
            // before the MFMAs of step it.  (PROJ: the centre tap's steps read
            // and multiply the projection's fragments too.)
            constexpr auto centre = [](int it) { return PROJ && it / KSTEPS == CT; };
            static_for<0, LA>([&](auto J) { sched_lds_reads<FK + FP + (centre(decltype(J)::value) ? FK : 0)>(); });
            static_for<0, NIT>([&](auto I) {
                constexpr int it = decltype(I)::value;
                if constexpr (it + LA < NIT) sched_lds_reads<FK + FP + (centre(it + LA) ? FK : 0)>();
                sched_mfmas<FP * FK * (centre(it) ? 2 : 1)>();
            });
        } else {
            // three fragment sets in rotation: the LDS reads of step it+2 are in
            // flight while the MFMAs of step it run
            v4i A0[FK], B0[FP], A1[FK], B1[FP], A2[FK], B2[FP];
            auto ld = [&](int it, v4i(&A)[FK], v4i(&B)[FP]) {
                int ao, bo;
                offs(it, ao, bo);
    #pragma unroll
                for (int tm = 0; tm < FK; ++tm) A[tm] = *reinterpret_cast<const v4i *>(wb + ao + tm * 256);
    #pragma unroll
                for (int tn = 0; tn < FP; ++tn) B[tn] = *reinterpret_cast<const v4i *>(bb + bo + pixoff[tn]);
            };
            auto mm = [&](const v4i(&A)[FK], const v4i(&B)[FP]) {
    #pragma unroll
                for (int tn = 0; tn < FP; ++tn)
    #pragma unroll
                    for (int tm = 0; tm < FK; ++tm)
                        acc[tn][tm] = __builtin_amdgcn_mfma_i32_16x16x64_i8(A[tm], B[tn], acc[tn][tm], 0, 0, 0);
            };
            // clamped step indices: re-reading the last step is harmless
            ld(0, A0, B0);
            ld(min(1, nit - 1), A1, B1);
            int it = 0;
            for (; it + 3 <= nit; it += 3) {
                ld(min(it + 2, nit - 1), A2, B2);
                mm(A0, B0);
                ld(min(it + 3, nit - 1), A0, B0);
                mm(A1, B1);
                ld(min(it + 4, nit - 1), A1, B1);
                mm(A2, B2);
#pragma unroll
                for (int g = 0; g < 3; ++g) {
                    sched_lds_reads<FK + FP>();
                    sched_mfmas<FP * FK>();
                }
            }
            if (it < nit) mm(A0, B0);
            if (it + 1 < nit) mm(A1, B1);
        }

        // the packed copy of this stage's band rows: before the next stage is
        // staged when that reuses the one band buffer, else after it (its
        // loads are then waited for without these stores)
        if constexpr (NCHW && !SINGLE)
            if (a.xpk && a.off_b1 == a.off_b0) nchw_write_packed(ti, c, cur, tid, NT);

        // The next stage's operands (in flight during the MFMAs) are waited for
        // and staged before this stage's epilogue issues its stores: the wait
        // covers loads only, never the store acknowledgements.
        if (more) {
            // with a single band buffer every wave must be done reading it
            if (a.off_b1 == a.off_b0) __syncthreads();
            __builtin_amdgcn_s_waitcnt(0);   // prefetched band (and filter DMA) have landed
            if constexpr (NCHW) {
                nchw_stage(nti, nc, cur ^ 1, [] {});
            } else {
                band_store(fb, cur ^ 1);
                band_rest(nc, cur ^ 1);
            }
            if constexpr (!FIXED) if (c_end - c_begin > 1 && !w_image) {
                w_gather_store(fw, 0, cur ^ 1);
                for (int base = NT * MAXV; base < TK * rs * VPP; base += NT * MAXV) {
                    WFetch f2;
                    w_gather(nc, base, f2);
                    w_gather_store(f2, base, cur ^ 1);
                }
            }
        }
        if constexpr (NCHW && !SINGLE)
            if (a.xpk && a.off_b1 != a.off_b0) nchw_write_packed(ti, c, cur, tid, NT);
        if (c == c_end - 1) {
            if (a.splits > 1) {
                // split-K: publish this split's partial sums; the last split of the
                // tile to arrive adds the others and runs the epilogue.  Partial
                // sums move with device-coherent loads and stores (sc1, the form
                // of monotonic agent-scope atomics), so no L2 write-back or
                // invalidation is needed: the stores are complete (waited for)
                // before the arrival count is bumped, and the last arrival reads
                // them past the caches.  (A release/acquire pair would write back
                // and invalidate the whole L2 of the XCD in every workgroup.)
                // (PROJ: the projection's partial sums follow the layer's)
                const int tile = lt;
                constexpr int kFrag = 64 * 16;                      // one fragment of a wave: 64 lanes x int4
                constexpr int kAccBytes = NW * FP * FK * kFrag;      // one accumulator set of a tile
                constexpr int kSplitBytes = (PROJ ? 2 : 1) * kAccBytes;   // one split's partial sums of a tile
                const __amdgpu_buffer_rsrc_t rws = make_brsrc(
                    reinterpret_cast<const uint8_t *>(a.ws_part) + (size_t)tile * a.splits * kSplitBytes,
                    a.splits * kSplitBytes);
                const int lane_off = (wave * FP * FK) * kFrag + lane * 16;
#pragma unroll
                for (int tn = 0; tn < FP; ++tn)
#pragma unroll
                    for (int tm = 0; tm < FK; ++tm) {
                        const v4i v = acc[tn][tm];
                        __builtin_amdgcn_raw_buffer_store_b128(u32x4{(uint32_t)v[0], (uint32_t)v[1], (uint32_t)v[2], (uint32_t)v[3]},
                                                               rws, sp * kSplitBytes + lane_off + (tn * FK + tm) * kFrag, 0,
                                                               kCoherentAux);
                        if constexpr (PROJ) {
                            const v4i v2 = acc2[tn][tm];
                            __builtin_amdgcn_raw_buffer_store_b128(
                                u32x4{(uint32_t)v2[0], (uint32_t)v2[1], (uint32_t)v2[2], (uint32_t)v2[3]}, rws,
                                sp * kSplitBytes + kAccBytes + lane_off + (tn * FK + tm) * kFrag, 0, kCoherentAux);
                        }
                    }
                __builtin_amdgcn_s_waitcnt(0);   // every wave's partial stores are complete
                __syncthreads();
                uint32_t *flag = reinterpret_cast<uint32_t *>(smem + a.off_m) + 2 * TK;   // past multipliers and biases
                if (tid == 0)
                    *flag = __hip_atomic_fetch_add(a.ws_cnt + tile, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                __syncthreads();
                const bool last = *flag == (uint32_t)(a.splits - 1);
                if (!last) return;   // uniform over the workgroup
                for (int o = 0; o < a.splits; ++o) {
                    if (o == sp) continue;
#pragma unroll
                    for (int tn = 0; tn < FP; ++tn)
#pragma unroll
                        for (int tm = 0; tm < FK; ++tm) {
                            const u32x4 q = __builtin_amdgcn_raw_buffer_load_b128(
                                rws, o * kSplitBytes + lane_off + (tn * FK + tm) * kFrag, 0, kCoherentAux);
                            acc[tn][tm] += v4i{(int)q[0], (int)q[1], (int)q[2], (int)q[3]};
                            if constexpr (PROJ) {
                                const u32x4 q2 = __builtin_amdgcn_raw_buffer_load_b128(
                                    rws, o * kSplitBytes + kAccBytes + lane_off + (tn * FK + tm) * kFrag, 0, kCoherentAux);
                                acc2[tn][tm] += v4i{(int)q2[0], (int)q2[1], (int)q2[2], (int)q2[3]};
                            }
                        }
                }
                if (tid == 0)   // ready for the next call
                    __hip_atomic_store(a.ws_cnt + tile, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            }
            if constexpr (SINGLE) {
                lds_epilogue_params(a, mlds, ep);
                if constexpr (PROJ) lds_epilogue_params(ap, mlds2, ep2);
                if (EXT && a.mode == QCONV_OUT_REQUANT && a.bias) add_bias<FP, FK>(a, acc, blds + cb - k0);
                if constexpr (PROJ)
                    if (EXT && a.mode == QCONV_OUT_REQUANT && a.bias2) add_bias<FP, FK>(ap, acc2, blds2 + cb - k0);
            }
            if constexpr (LDSEPI)
                lds_epilogue(ti);
            else
                epilogue<BITS, FP, FK, EXT>(a, acc, (j0 + ti * gpk) * TP + wp * FP * 16, cb, l16, ep);
            if constexpr (!SINGLE) {   // the accumulators of the next tile
                if (bias_here) {
                    init_acc<FP, FK>(a, acc, blds + cb - k0, false, cb);
                } else {
#pragma unroll
                    for (int tn = 0; tn < FP; ++tn)
#pragma unroll
                        for (int tm = 0; tm < FK; ++tm) acc[tn][tm] = v4i{0, 0, 0, 0};
                }
            }
            if constexpr (PROJ) {
                epilogue<BITS, FP, FK, EXT>(ap, acc2, (j0 + ti * gpk) * TP + wp * FP * 16, cb, l16, ep2);
                if constexpr (!SINGLE) {
                    if (bias2_here) {
                        init_acc<FP, FK>(ap, acc2, blds2 + cb - k0, false, cb);
                    } else {
#pragma unroll
                        for (int tn = 0; tn < FP; ++tn)
#pragma unroll
                            for (int tm = 0; tm < FK; ++tm) acc2[tn][tm] = v4i{0, 0, 0, 0};
                    }
                }
            }
        }
        if (more) {
            __syncthreads();
            if (nti != ti) set_tile(nti);
        }
        ti = nti;
        c = nc;
    };
    if (ONE && nst == 1) {
        stage(0, std::bool_constant<ONE>{});
    } else {
        for (int st = 0; st < nst; ++st) stage(st, std::false_type{});
    }
}

// Build the filter image conv_wide stages directly: for channel tile kt and
// chunk c, plane g (channels 16g..16g+15 of the chunk), element tap*TK + slot
// holds the widened int8 granule of output channel row_channel(slot) at that
// tap -- the same bytes the gather path writes into LDS.  One thread per
// 16-byte element; padding elements are zero.
// With `wproj` (packed K x 1 x 1 x C filters of a fused projection) the image
// has one more tap, rs, holding those filters.
template <int BITS, int FK, bool WS>
__global__ void __launch_bounds__(256) build_filter_image(ConvArgs a, int TK, int CK, uint8_t *img, int64_t total,
                                                          const uint8_t *wproj) {
    const int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (e >= total) return;
    const int rs = a.r * a.s;
    const int taps = rs + (wproj ? 1 : 0);
    const int ng = CK / 16;
    const int64_t plane_elems = a.pstride_w / 16;
    const int64_t blk = e / (ng * plane_elems);
    const int64_t rem = e - blk * ng * plane_elems;
    const int g = (int)(rem / plane_elems);
    const int el = (int)(rem - (int64_t)g * plane_elems);
    const int kt = (int)(blk / a.nchunks);
    const int c = (int)(blk - (int64_t)kt * a.nchunks);
    uint4 out = uint4{0u, 0u, 0u, 0u};
    if (el < taps * TK) {
        const int tap = el / TK;
        const int slot = el - tap * TK;
        const int kk = kt * TK + (slot / (FK * 16)) * FK * 16 + row_channel<FK>((slot % (FK * 16)) / 16, slot % 16);
        const int ch = c * CK + 16 * g;
        if (kk < a.k && ch < a.c) {
            const uint8_t *src = tap < rs ? a.wptr + ((size_t)kk * rs + tap) * a.xpix + (size_t)ch * BITS / 8
                                          : wproj + (size_t)kk * a.xpix + (size_t)ch * BITS / 8;
            if constexpr (BITS == 4) {
                const uint2 v = *reinterpret_cast<const uint2 *>(src);
                uint4 g0, g1;
                widen_vec<4, WS>(uint4{v.x, v.y, 0u, 0u}, g0, g1);
                out = g0;
            } else {
                out = *reinterpret_cast<const uint4 *>(src);
            }
        }
    }
    *reinterpret_cast<uint4 *>(img + e * 16) = out;
}

// One operand signedness per kernel (the widening is compiled for it); 8-bit
// operands are always signed.
template <int BITS, int WP, int WK, int FP, int FK, int CK, bool XS, bool WS, int RC, int SC, bool EXT, int ABL = 0,
          bool MC = false, bool NCHW = false, bool PROJ = false, bool ONE = false, bool OCT = false>
__global__ void __launch_bounds__(WP * WK * 64) __attribute__((amdgpu_waves_per_eu(2))) conv_wide(ConvArgs a) {
    const ConvArgs args = warm_kernarg_lines(a);
    wide_body<BITS, WP, WK, FP, FK, CK, XS, WS, RC, SC, EXT, ABL, MC, NCHW, PROJ, ONE, OCT>(args);
}

// ============================================================== tile registry

template <int BITS, int WP, int WK, int FP, int FK, int CK, bool EXT>
static hipError_t launch_staged(const ConvArgs &a, dim3 grid, size_t lds, hipStream_t stream) {
    hipLaunchKernelGGL((conv_staged<BITS, WP, WK, FP, FK, CK, EXT>), grid, dim3(WP * WK * 64), lds, stream, a);
    return hipGetLastError();
}

template <int BITS, int WP, int WK, int FP, int FK, int CK, bool XS, bool WS, int RC, int SC, bool EXT, int ABL = 0,
          bool MC = false, bool NCHW = false, bool PROJ = false, bool ONE = false, bool OCT = false>
static hipError_t launch_wide(const ConvArgs &a, dim3 grid, size_t lds, hipStream_t stream) {
    hipLaunchKernelGGL((conv_wide<BITS, WP, WK, FP, FK, CK, XS, WS, RC, SC, EXT, ABL, MC, NCHW, PROJ, ONE, OCT>), grid,
                       dim3(WP * WK * 64), lds, stream, a);
    return hipGetLastError();
}

template <int BITS, int WK, int FK, int CK, bool WS>
static hipError_t launch_prep(const ConvArgs &a, uint8_t *img, int64_t elems, const uint8_t *wproj,
                              hipStream_t stream) {
    const int64_t blocks = (elems + 255) / 256;
    hipLaunchKernelGGL((build_filter_image<BITS, FK, WS>), dim3((unsigned)blocks), dim3(256), 0, stream, a, WK * FK * 16, CK,
                       img, elems, wproj);
    return hipGetLastError();
}

// The compiled tile space: (bits, waves_p, waves_k, frag_p, frag_k, chunk_c).
#define QCONV_STAGED_TILES(X) \
    X(4, 4, 1, 1, 4, 64)      \
    X(4, 4, 1, 2, 4, 64)      \
    X(4, 2, 2, 2, 4, 128)     \
    X(4, 4, 1, 4, 2, 64)      \
    X(4, 4, 1, 1, 2, 64)      \
    X(8, 4, 1, 1, 4, 64)      \
    X(8, 4, 1, 2, 4, 64)      \
    X(8, 4, 1, 4, 2, 64)      \
    X(8, 4, 1, 2, 1, 64)

// (in four groups, each compiled in a translation unit of its own)
#define QCONV_WIDE_TILES_A(X) \
    X(4, 4, 1, 1, 4, 64) \
    X(4, 4, 2, 2, 2, 64) \
    X(4, 2, 2, 2, 2, 64) \
    X(4, 4, 1, 2, 4, 64) \
    X(4, 4, 1, 4, 4, 64) \
    X(4, 8, 1, 1, 4, 64)
#define QCONV_WIDE_TILES_B(X) \
    X(4, 8, 1, 2, 4, 64) \
    X(4, 4, 2, 2, 4, 64) \
    X(4, 4, 2, 4, 4, 64) \
    X(4, 2, 2, 4, 4, 64) \
    X(4, 2, 4, 4, 4, 64) \
    X(4, 1, 4, 4, 4, 64)
#define QCONV_WIDE_TILES_C(X) \
    X(4, 4, 1, 4, 2, 64) \
    X(4, 8, 1, 4, 2, 64) \
    X(4, 4, 2, 4, 4, 128) \
    X(4, 2, 2, 4, 4, 128) \
    X(4, 2, 4, 2, 4, 128) \
    X(4, 1, 4, 4, 4, 128)
#define QCONV_WIDE_TILES_D(X) \
    X(8, 4, 1, 2, 4, 64) \
    X(8, 4, 2, 2, 2, 64) \
    X(8, 4, 1, 4, 4, 64) \
    X(8, 8, 1, 2, 4, 64) \
    X(8, 4, 2, 4, 4, 64) \
    X(8, 2, 2, 4, 4, 64) \
    X(8, 2, 4, 4, 4, 64) \
    X(8, 1, 4, 4, 4, 64) \
    X(4, 8, 1, 2, 4, 128) \
    X(4, 4, 2, 2, 2, 128)
#define QCONV_WIDE_TILES(X) QCONV_WIDE_TILES_A(X) QCONV_WIDE_TILES_B(X) QCONV_WIDE_TILES_C(X) QCONV_WIDE_TILES_D(X)
#define QCONV_TILE_INFO(V, PREFIX, B, WP, WK, FP, FK, CK, XS, WS)                                                 \
    {0, B, WP, WK, FP, FK, CK, WP * FP * 16, WK * FK * 16, WP * WK * 64, V, XS, WS,                              \
     PREFIX #B "_w" #WP "x" #WK "_f" #FP "x" #FK "_c" #CK}
#define QCONV_STAGED_SET(B, WP, WK, FP, FK, CK, EXT)                                                              \
    {&launch_staged<B, WP, WK, FP, FK, CK, EXT>,                                                                  \
     reinterpret_cast<const void *>(&conv_staged<B, WP, WK, FP, FK, CK, EXT>), {}}
#define QCONV_STAGED_ENTRY(B, WP, WK, FP, FK, CK)                                                                 \
    {QCONV_TILE_INFO(QCONV_VARIANT_STAGED, "staged_b", B, WP, WK, FP, FK, CK, -1, -1),                           \
     QCONV_STAGED_SET(B, WP, WK, FP, FK, CK, false), QCONV_STAGED_SET(B, WP, WK, FP, FK, CK, true), nullptr, {}},
// 4-bit: unsigned activations x signed filters; 8-bit: signed x signed.
// Each wide tile also has fixed-size instances for 3x3 and 1x1 filters, used
// with prepared filters.
#define QCONV_WIDE_INST(B, WP, WK, FP, FK, CK, R, S, EXT)                                                         \
    &launch_wide<B, WP, WK, FP, FK, CK, (B == 8), true, R, S, EXT>,                                               \
        reinterpret_cast<const void *>(&conv_wide<B, WP, WK, FP, FK, CK, (B == 8), true, R, S, EXT>)
#define QCONV_WIDE_MC(B, WP, WK, FP, FK, CK, R, S, EXT)                                                           \
    &launch_wide<B, WP, WK, FP, FK, CK, (B == 8), true, R, S, EXT, 0, true>,                                      \
        reinterpret_cast<const void *>(&conv_wide<B, WP, WK, FP, FK, CK, (B == 8), true, R, S, EXT, 0, true>)
#define QCONV_WIDE_ONE(B, WP, WK, FP, FK, CK, R, S, EXT)                                                          \
    &launch_wide<B, WP, WK, FP, FK, CK, (B == 8), true, R, S, EXT, 0, false, false, false, true>,                 \
        reinterpret_cast<const void *>(                                                                           \
            &conv_wide<B, WP, WK, FP, FK, CK, (B == 8), true, R, S, EXT, 0, false, false, false, true>)
#define QCONV_WIDE_SET(B, WP, WK, FP, FK, CK, EXT)                                                                \
    {QCONV_WIDE_INST(B, WP, WK, FP, FK, CK, 0, 0, EXT),                                                           \
     {{3, 3, QCONV_WIDE_INST(B, WP, WK, FP, FK, CK, 3, 3, EXT), QCONV_WIDE_MC(B, WP, WK, FP, FK, CK, 3, 3, EXT),  \
       QCONV_WIDE_ONE(B, WP, WK, FP, FK, CK, 3, 3, EXT)},                                                         \
      {1, 1, QCONV_WIDE_INST(B, WP, WK, FP, FK, CK, 1, 1, EXT), nullptr, nullptr,                                 \
       QCONV_WIDE_ONE(B, WP, WK, FP, FK, CK, 1, 1, EXT)}}}
#define QCONV_WIDE_FUSED(B, WP, WK, FP, FK, CK)                                                                   \
    {3, 3, &launch_wide<B, WP, WK, FP, FK, CK, (B == 8), true, 3, 3, false, 0, false, true>,                      \
     reinterpret_cast<const void *>(&conv_wide<B, WP, WK, FP, FK, CK, (B == 8), true, 3, 3, false, 0, false, true>), \
     nullptr, nullptr, &launch_wide<B, WP, WK, FP, FK, CK, (B == 8), true, 3, 3, false, 0, false, true, false, true>, \
     reinterpret_cast<const void *>(                                                                              \
         &conv_wide<B, WP, WK, FP, FK, CK, (B == 8), true, 3, 3, false, 0, false, true, false, true>),             \
     &launch_wide<B, WP, WK, FP, FK, CK, (B == 8), true, 3, 3, false, 0, false, true, false, true, true>,          \
     reinterpret_cast<const void *>(                                                                              \
         &conv_wide<B, WP, WK, FP, FK, CK, (B == 8), true, 3, 3, false, 0, false, true, false, true, true>)}
#define QCONV_PROJ_INST(B, WP, WK, FP, FK, CK, EXT)                                                               \
    {3, 3, &launch_wide<B, WP, WK, FP, FK, CK, (B == 8), true, 3, 3, EXT, 0, false, false, true>,                \
     reinterpret_cast<const void *>(&conv_wide<B, WP, WK, FP, FK, CK, (B == 8), true, 3, 3, EXT, 0, false, false, true>), \
     nullptr, nullptr, &launch_wide<B, WP, WK, FP, FK, CK, (B == 8), true, 3, 3, EXT, 0, false, false, true, true>, \
     reinterpret_cast<const void *>(                                                                              \
         &conv_wide<B, WP, WK, FP, FK, CK, (B == 8), true, 3, 3, EXT, 0, false, false, true, true>)}
#define QCONV_PROJ_ENTRY(B, WP, WK, FP, FK, CK)                                                                   \
    {"wide_b" #B "_w" #WP "x" #WK "_f" #FP "x" #FK "_c" #CK, QCONV_PROJ_INST(B, WP, WK, FP, FK, CK, false),         \
     QCONV_PROJ_INST(B, WP, WK, FP, FK, CK, true)},
#define QCONV_WIDE_ENTRY(B, WP, WK, FP, FK, CK)                                                                   \
    {QCONV_TILE_INFO(QCONV_VARIANT_WIDE, "wide_b", B, WP, WK, FP, FK, CK, (B == 8), 1),                         \
     QCONV_WIDE_SET(B, WP, WK, FP, FK, CK, false), QCONV_WIDE_SET(B, WP, WK, FP, FK, CK, true),                 \
     &launch_prep<B, WK, FK, CK, true>, QCONV_WIDE_FUSED(B, WP, WK, FP, FK, CK)},

}  // namespace qconv
