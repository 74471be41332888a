// Width unrolling for convolutions with very few input channels (the 3-channel
// 7x7 stem of a ResNet): the S filter columns are folded into the channel
// axis, so the convolution becomes an R x 1 one over S*C (padded) channels,
// which the channel-packed kernels run at a useful MMA depth.
//
//   dst[n][h][q][s*C + c] = src[n][c][h][q*stride + s - pad]   (0 outside,
//                                                               and for
//                                                               channels >= S*C)
//
// A filter bank k x c x r x s unrolls the same way with stride 1 and pad 0
// (its one output column holds all S taps): it becomes k x r x 1 x (S*C).
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "qconv_internal.h"

namespace qconv {

namespace {

// One thread per output pixel (n, h, q): gathers its taps*c bytes from the
// NCHW planes and writes the c_out-byte channel run with 16-byte stores.
__global__ void __launch_bounds__(256) unroll_width(const int8_t *__restrict__ src, int8_t *__restrict__ dst,
                                                    int n, int c, int h, int w, int taps, int stride, int pad,
                                                    int wout, int c_out) {
    const int64_t pix = (int64_t)blockIdx.x * 256 + threadIdx.x;
    const int64_t total = (int64_t)n * h * wout;
    if (pix >= total) return;
    const int q = (int)(pix % wout);
    const int64_t nh = pix / wout;
    const int row = (int)(nh % h);
    const int img = (int)(nh / h);
    int8_t *out = dst + pix * c_out;
    for (int v = 0; v < c_out; v += 16) {
        uint32_t words[4] = {0u, 0u, 0u, 0u};
#pragma unroll
        for (int b = 0; b < 16; ++b) {
            const int ch = v + b;
            int8_t val = 0;
            if (ch < taps * c) {
                const int s = ch / c, ci = ch - s * c;
                const int col = q * stride + s - pad;
                if (col >= 0 && col < w) val = src[(((int64_t)img * c + ci) * h + row) * w + col];
            }
            words[b >> 2] |= (uint32_t)(uint8_t)val << (8 * (b & 3));
        }
        *reinterpret_cast<uint4 *>(out + v) = uint4{words[0], words[1], words[2], words[3]};
    }
}

}  // namespace

hipError_t launch_unroll(const int8_t *src, int8_t *dst, int32_t n, int32_t c, int32_t h, int32_t w, int32_t taps,
                         int32_t stride, int32_t pad, int32_t wout, int32_t c_out, hipStream_t stream) {
    const int64_t total = (int64_t)n * h * wout;
    if (total == 0) return hipSuccess;
    hipLaunchKernelGGL(unroll_width, dim3((unsigned)((total + 255) / 256)), dim3(256), 0, stream, src, dst, n, c, h,
                       w, taps, stride, pad, wout, c_out);
    return hipGetLastError();
}

}  // namespace qconv
