// Patch unrolling for convolutions with very few input channels (the 3-channel
// 7x7 stride-2 stem of a ResNet): filter taps are folded into the channel
// axis, so the layer runs on the channel-packed kernels at a useful MMA depth.
//
//   dst[n][u][q][(b*taps_w + s)*C + c] =
//       src[n][c][u*stride_h + b - pad_h][q*stride_w + s - pad_w]
//
// for b < taps_h, s < taps_w (0 outside the input, and 0 for channels from
// taps_h*taps_w*C to c_out).  Folding every filter row turns the layer into a
// 1x1 convolution; folding groups of stride_h rows turns a strided R-row
// filter into a ceil(R/stride_h)-row one at stride 1.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "qconv_internal.h"

namespace qconv {

namespace {

// One workgroup per output row (image, u).  The taps_h source rows of all C
// channels that the row reads are staged in LDS with their zero padding, and
// a table gives each output channel's LDS offset (-1 for a zero channel);
// the threads then assemble 16-byte output vectors from it, consecutive
// threads writing consecutive vectors of the row.  (Workgroups that loop over
// several rows were slower: every row's loads, barrier and stores form one
// latency chain, and one resident workgroup per row overlaps them best.)
__global__ void __launch_bounds__(256) unroll_patches(const int8_t *__restrict__ src, int8_t *__restrict__ dst,
                                                      UnrollArgs a) {
    extern __shared__ __attribute__((aligned(16))) uint8_t smem[];
    int32_t *table = reinterpret_cast<int32_t *>(smem);
    uint8_t *rows = smem + 4 * a.c_out;
    const int real = a.taps_h * a.taps_w * a.c;
    for (int ch = threadIdx.x; ch < a.c_out; ch += 256) {
        int off = -1;
        if (ch < real) {
            const int tap = ch / a.c, ci = ch - tap * a.c;
            const int b = tap / a.taps_w, s = tap - b * a.taps_w;
            off = (ci * a.taps_h + b) * a.lw + s;
        }
        table[ch] = off;
    }
    const int nrb = a.c * a.taps_h;
    const int vpp = a.c_out / 16;
    const int u = (int)(blockIdx.x % (unsigned)a.out_h);
    const int img = (int)(blockIdx.x / (unsigned)a.out_h);
    // staged row rb = ci * taps_h + b holds source row u*stride_h + b - pad_h
    // of channel ci; each thread takes one column of up to 8 rows at a time,
    // so that their loads are in flight together
    for (int x = threadIdx.x; x < a.lw; x += 256) {
        const int col = x - a.pad_w;
        const bool col_ok = col >= 0 && col < a.w;
        for (int rb0 = 0; rb0 < nrb; rb0 += 8) {
            uint8_t vals[8];
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                const int rb = rb0 + e;
                const int ci = rb / a.taps_h, b = rb - ci * a.taps_h;
                const int y = u * a.stride_h + b - a.pad_h;
                vals[e] = 0;
                if (rb < nrb && col_ok && y >= 0 && y < a.h)
                    vals[e] = (uint8_t)src[(((int64_t)img * a.c + ci) * a.h + y) * a.w + col];
            }
#pragma unroll
            for (int e = 0; e < 8; ++e)
                if (rb0 + e < nrb) rows[(rb0 + e) * a.lw + x] = vals[e];
        }
    }
    __syncthreads();
    int8_t *out = dst + ((int64_t)img * a.out_h + u) * a.wout * a.c_out;
    for (int v = threadIdx.x; v < a.wout * vpp; v += 256) {
        const int q = v / vpp, j = v - q * vpp;
        const int base = q * a.stride_w;
        const int4 *t4 = reinterpret_cast<const int4 *>(table + 16 * j);
        uint32_t words[4];
#pragma unroll
        for (int g = 0; g < 4; ++g) {
            const int4 o = t4[g];
            const int oo[4] = {o.x, o.y, o.z, o.w};
            uint32_t word = 0;
#pragma unroll
            for (int e = 0; e < 4; ++e)
                if (oo[e] >= 0) word |= (uint32_t)rows[oo[e] + base] << (8 * e);
            words[g] = word;
        }
        *reinterpret_cast<uint4 *>(out + (int64_t)v * 16) = uint4{words[0], words[1], words[2], words[3]};
    }
}

}  // namespace

int64_t unroll_lds_bytes(const UnrollArgs &a) { return 4ll * a.c_out + (int64_t)a.c * a.taps_h * a.lw; }

hipError_t launch_unroll(const int8_t *src, int8_t *dst, const UnrollArgs &a, hipStream_t stream) {
    const int64_t blocks = (int64_t)a.n * a.out_h;
    if (blocks == 0 || a.wout == 0) return hipSuccess;
    hipLaunchKernelGGL(unroll_patches, dim3((unsigned)blocks), dim3(256), (size_t)unroll_lds_bytes(a), stream, src,
                       dst, a);
    return hipGetLastError();
}

}  // namespace qconv
