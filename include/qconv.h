/*
 * qconv.h -- C ABI of libqconv: reduced-precision (4-bit / 8-bit) integer 2-D
 * convolution on AMD Instinct MI355X (gfx950), run as an implicit GEMM on the
 * int8 matrix cores with int32 accumulation.
 *
 * The operation is the one the paper "Learning from Distinctive Candidates to
 * Optimize Reduced-Precision Convolution Program on Tensor Cores" schedules:
 *   - Sec. 2.1: a convolution of an N x H x W x C input with K filters of
 *     R x S is the GEMM (N*P*Q, C*R*S) x (C*R*S, K) of the lowered (im2col)
 *     input with the filters;
 *   - Sec. 1 and Sec. 3.3: operands are 4-bit values packed eight per 32-bit
 *     word along the channel axis, in a layout whose output is already the
 *     next layer's input layout;
 *   - Sec. 3.2.2: an epilogue on the wide accumulator followed by clipping
 *     to the low bit-width and packing.
 *
 * Conventions shared by every entry point
 *   - All tensor pointers are DEVICE pointers owned by the caller; the library
 *     never allocates, frees or retains them beyond the call.
 *   - Calls enqueue work on `stream` (a hipStream_t; NULL = the default
 *     stream) and return without waiting.  Argument errors are reported
 *     before anything is enqueued; faults during execution surface at the
 *     caller's next synchronisation.
 *   - Return value: QCONV_OK or a negative status; qconv_strerror() names it
 *     and qconv_last_error() gives the detail of the calling thread's most
 *     recent failure.
 *   - Mutable global state: per thread, the last error message and the
 *     last launch's geometry; per device, caches of kernel attributes and
 *     occupancy; a cache of band heights keyed by every shape field they
 *     depend on; and the no-alloc entry's scratch array.  The caches are
 *     locked, so calls on distinct streams may run concurrently from any
 *     threads, except that no-alloc calls that overlap on one device race
 *     on its scratch.
 *
 * Packed layouts (b = bits)
 *   activations  N x H x W x C, channels innermost
 *   filters      K x R x S x C, channels innermost
 *   b = 4: each pixel (or filter tap) is C/8 uint32 words; channel 8j+i is
 *          bits [4i, 4i+3] of word j; signed values are two's-complement
 *          nibbles.
 *   b = 8: each pixel is C int8 values.
 *   batch-interleaved (qconv_desc.nb > 1; the NHWCnc layout of Sec. 3.3.2
 *   with n = nb images and c = the whole channel run): N/nb x H x W x nb x C,
 *   i.e. image i's pixel (y, x) is pixel ((i/nb)*H + y)*W*nb + x*nb + i%nb
 *   of the plain layout; each pixel's channels are packed as above.  Nb
 *   consecutive pixels -- one MMA tile's rows -- then hold the same (y, x)
 *   of nb images, and a row of the tensor is contiguous for all of them.
 */
#ifndef QCONV_H
#define QCONV_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Status codes. */
#define QCONV_OK 0
#define QCONV_EINVAL (-1)      /* NULL, bad sizes, window larger than padded input, bad epilogue, misaligned */
#define QCONV_EUNSUPPORTED (-2) /* valid request outside what the kernels implement (bit-width, channel multiple,
                                   accumulator bound, tile not usable for the shape) */
#define QCONV_EWORKSPACE (-3)  /* workspace smaller than qconv_layout_info.workspace_bytes */
#define QCONV_EHIP (-4)        /* the HIP runtime rejected a launch or attribute call */

/* Epilogue modes. */
#define QCONV_OUT_RAW_I32 0    /* y = int32 accumulators, N x P x Q x K */
#define QCONV_OUT_REQUANT 1    /* y = requantised values, packed like the input (b-bit, N x P x Q x K) */

/*
 * One convolution.  n, h, w, c: input batch, height, width, channels;
 * k: output channels; r, s: filter height and width; stride and zero padding
 * per axis; bits: 4 or 8; x_signed / w_signed: 0 or 1 (8-bit needs both 1).
 * Output extent P = (h + 2*pad_h - r)/stride_h + 1, Q likewise (Sec. 2.1; no
 * dilation, no groups; cross-correlation, no filter flip).  nb: activation
 * layout, 0 or 1 for N x H x W x C, nb > 1 for the batch-interleaved layout
 * (input, output and residual alike); it needs n % nb == 0, and stride_w == 1
 * (else QCONV_EUNSUPPORTED).  The filters' layout does not change.
 */
typedef struct qconv_desc {
    int32_t n, h, w, c;
    int32_t k, r, s;
    int32_t stride_h, stride_w;
    int32_t pad_h, pad_w;
    int32_t bits;
    int32_t x_signed, w_signed;
    int32_t nb;
} qconv_desc;

/* Sizes derived from a qconv_desc (bytes unless stated). */
typedef struct qconv_layout_info {
    int32_t p, q;              /* output height and width */
    int64_t m;                 /* GEMM rows = n*p*q */
    int64_t gemm_k;            /* GEMM depth = c*r*s */
    int64_t macs;              /* n*p*q*k*c*r*s; effective ops = 2*macs */
    int64_t x_bytes;           /* packed input */
    int64_t w_bytes;           /* packed filters */
    int64_t y_raw_bytes;       /* int32 output */
    int64_t y_packed_bytes;    /* requantised packed output */
    int64_t workspace_bytes;   /* device scratch qconv2d needs (0 today) */
    int64_t max_abs_acc;       /* worst-case |accumulator| over all inputs of the declared ranges */
} qconv_layout_info;

/*
 * Epilogue (Sec. 3.2.2: the wide accumulator is processed first -- the bias
 * addition and batch-norm scaling the section names -- then clipped and
 * packed):
 *   t = (acc + bias[k]) * mult[k]             (exact, 64-bit; no bias = 0)
 *   t = floor((t + 2^(shift-1)) / 2^shift)    (round half up)
 *   t = t + residual[n, p, q, k]              (no residual = 0)
 *   t = max(t, 0) if relu
 *   t = min(max(t, clamp_lo), clamp_hi)
 * The clamp range must fit the output type: 4-bit [0,15] (unsigned output)
 * or [-8,7] (signed), 8-bit [-128,127].  The output is signed iff
 * clamp_lo < 0.
 *   mult      DEVICE pointer to k int32 values.
 *   bias      DEVICE pointer to k int32 values, or NULL: an offset in
 *             accumulator units (a folded batch norm's shift).  The sum
 *             accumulator + bias is formed in int32 (scaled by 2^acc_shift,
 *             acc_shift = 4 per signed 4-bit operand, else 0), so every value
 *             must keep |bias| <= (2^31 - 1) / 2^acc_shift - max_abs_acc
 *             (qconv_layout); outside that bound results wrap.
 *   residual  DEVICE pointer, or NULL: a tensor in y's packed layout and bit
 *             width (n x p x q x k; the shortcut of a residual block, e.g. an
 *             earlier layer's output), 16-byte aligned; its values are read
 *             as signed when residual_signed is 1, else unsigned.  It may be y
 *             itself (updated in place) but must not otherwise overlap y, and
 *             must not overlap x, w or the workspace.
 * In QCONV_OUT_RAW_I32 mode only `mode` is read, and bias and residual must
 * be NULL.
 */
typedef struct qconv_epilogue {
    int32_t mode;
    const int32_t *mult;
    int32_t shift;             /* 1 .. 62 */
    int32_t relu;              /* 0 or 1 */
    int32_t clamp_lo, clamp_hi;
    const int32_t *bias;       /* NULL = none */
    const void *residual;      /* NULL = none */
    int32_t residual_signed;   /* 0 or 1 */
} qconv_epilogue;

/*
 * A compile-time tile configuration of the convolution kernel: the paper's
 * schedule knobs (Sec. 4.1) restated for 64-wide waves and MFMA.
 *   waves_p, waves_k   waves of a workgroup along output pixels / channels
 *                      (BLK-ROW-WARPS, BLK-COL-WARPS)
 *   frag_p, frag_k     16x16 MFMA tiles per wave along pixels / channels
 *                      (WARP-ROW-TILES, WARP-COL-TILES)
 *   chunk_c            input channels staged per main-loop step (CHUNK)
 *   tile_p, tile_k     workgroup tile = 16*waves*frag along each axis
 *   bits               4 or 8: operand width the kernel is built for
 *   variant            QCONV_VARIANT_STAGED: global -> VGPR -> LDS staging, one
 *                      stage at a time, any channel count;
 *                      QCONV_VARIANT_WIDE: next stage prefetched into registers
 *                      during the MFMAs, operands widened once and staged in
 *                      LDS as int8, double buffered, persistent over output
 *                      tiles; needs c*bits % 128 == 0
 */
#define QCONV_VARIANT_STAGED 0
#define QCONV_VARIANT_WIDE 2

typedef struct qconv_tile_info {
    int32_t id;
    int32_t bits;
    int32_t waves_p, waves_k;
    int32_t frag_p, frag_k;
    int32_t chunk_c;
    int32_t tile_p, tile_k;
    int32_t threads;
    int32_t variant;
    int32_t x_signed, w_signed;   /* operand signedness the kernel is built for; -1 = any */
    char name[64];
} qconv_tile_info;

/*
 * qconv_layout -- host only, no device work.  Validates `d` exactly as
 * qconv2d does and fills `out` with the output extent and buffer sizes.
 *   p, q, m, gemm_k, macs   the GEMM view of Sec. 2.1: M = n*p*q lowered
 *                           rows (P, Q as in qconv_desc), depth c*r*s
 *   x_bytes, w_bytes,       the packed layouts above (Sec. 1: eight 4-bit
 *   y_*_bytes               values per 32-bit word)
 *   max_abs_acc             the largest |accumulator| any input of the
 *                           declared ranges can give, c*r*s*max|x|*max|w|;
 *                           Sec. 3.2.1 argues that 32-bit accumulators are
 *                           enough for reduced-precision products, and the
 *                           descriptor is rejected (QCONV_EUNSUPPORTED) when
 *                           this bound, times the widening factor of signed
 *                           4-bit operands, reaches 2^31
 * Returns QCONV_EINVAL / QCONV_EUNSUPPORTED for a descriptor qconv2d would
 * reject.  `out` may be NULL (validation only).
 */
int qconv_layout(const qconv_desc *d, qconv_layout_info *out);

/*
 * qconv_pack -- relayout and pack (Sec. 1: eight 4-bit values grouped per
 * 32-bit word along the channel axis; Sec. 3.3: channels innermost so the
 * tensor is read with coalesced accesses).
 *   src  DEVICE int8, n x c x h x w (activations) -- or k x c x r x s for
 *        filters, which gives the k x r x s x c filter layout
 *   dst  DEVICE, the packed layout above (bits 4: n*h*w*c/8 uint32;
 *        bits 8: n*h*w*c int8)
 * Each value is saturated into the b-bit range of `is_signed` before packing.
 * Needs c % 8 == 0 for bits 4; bits 8 needs is_signed == 1.  src and dst must
 * not overlap.  Errors: QCONV_EINVAL (NULL, negative sizes),
 * QCONV_EUNSUPPORTED (bits, channel multiple), QCONV_EHIP (launch).
 * Zero-sized tensors are a no-op returning QCONV_OK.
 */
int qconv_pack(const int8_t *src, void *dst, int32_t n, int32_t c, int32_t h, int32_t w,
               int32_t bits, int32_t is_signed, void *stream);

/*
 * qconv_pack_interleaved -- qconv_pack of activations into the
 * batch-interleaved layout (Sec. 3.3.2's NHWCnc, nb images per pixel): the
 * same values and packing, image i's pixel (y, x) stored at pixel
 * ((i/nb)*h + y)*w*nb + x*nb + i%nb.  nb = 1 is qconv_pack.  Needs
 * n % nb == 0 (QCONV_EINVAL otherwise); other rules and errors as qconv_pack.
 */
int qconv_pack_interleaved(const int8_t *src, void *dst, int32_t n, int32_t c, int32_t h, int32_t w,
                           int32_t bits, int32_t is_signed, int32_t nb, void *stream);

/*
 * qconv_unroll -- patch unrolling for layers with very few input channels
 * (e.g. the 3-channel 7x7 stride-2 stem of a ResNet): folds filter taps into
 * the channel axis so the layer runs on the channel-packed kernels with
 * taps_h*taps_w*c real values per MMA depth instead of c.
 *   src   DEVICE int8, n x c x h x w (NCHW); may be NULL when it is empty
 *   dst   DEVICE int8, n x out_h x wout x c_out, 16-byte aligned, not
 *         overlapping src; wout = (w + 2*pad_w - taps_w) / stride_w + 1
 *   dst[n][u][q][(b*taps_w + s)*c + ci] =
 *       src[n][ci][u*stride_h + b - pad_h][q*stride_w + s - pad_w]
 *   for b < taps_h, s < taps_w, ci < c (0 where the row or column is outside
 *   the input), and 0 for channels from taps_h*taps_w*c to c_out.
 * For a layer x (*) f with filters k x c x R x S, stride (sh, sw), padding
 * (ph, pw) and output P x Q, two foldings give the same result:
 *   - all rows:  unroll(x; R, sh, ph, P; S, sw, pw) (*) unroll(f; R, 1, 0, 1;
 *     S, 1, 0), a 1x1 convolution at stride 1;
 *   - row groups of sh:  unroll(x; sh, sh, ph, P + R' - 1; S, sw, pw) (*)
 *     unroll(f; sh, sh, 0, R'; S, 1, 0) with R' = ceil(R / sh), an R' x 1
 *     convolution at stride 1 without padding (filter rows beyond R are 0).
 * The unrolled operands are 8-bit (signed).  Needs taps_h*taps_w*c <= c_out,
 * c_out % 16 == 0, and 4*c_out + c*taps_h*(w + 2*pad_w) <= 65536 (bytes
 * staged per output row).  Errors: QCONV_EINVAL (NULL, sizes, overlap,
 * alignment), QCONV_EUNSUPPORTED (staging limit), QCONV_EHIP.  An empty
 * destination is a no-op.
 */
int qconv_unroll(const int8_t *src, int8_t *dst, int32_t n, int32_t c, int32_t h, int32_t w, int32_t taps_h,
                 int32_t stride_h, int32_t pad_h, int32_t out_h, int32_t taps_w, int32_t stride_w, int32_t pad_w,
                 int32_t c_out, void *stream);

/*
 * qconv2d -- the convolution (Sec. 2.1) as an implicit GEMM with the
 * epilogue of Sec. 3.2.2 fused into it.
 *   x          DEVICE, packed activations, 16-byte aligned
 *   w          DEVICE, packed filters, 16-byte aligned
 *   epi        host struct; NULL means QCONV_OUT_RAW_I32
 *   y          DEVICE output, 16-byte aligned: y_raw_bytes (raw mode) or
 *              y_packed_bytes (requant mode); must not overlap x or w
 *   workspace  DEVICE scratch of workspace_bytes (may be NULL when 0)
 *   tile_id    a tile from qconv_tile_get, or -1 for the built-in choice
 * Requirements beyond qconv_layout's: bits 4 needs c % 8 == 0 and
 * k % 8 == 0; bits 8 needs c % 4 == 0 and k % 4 == 0 and both operands
 * signed; the worst-case accumulator (max_abs_acc) must stay below 2^31
 * (Sec. 3.2.1).  Every tile gives byte-identical results.
 * Errors: QCONV_EINVAL, QCONV_EUNSUPPORTED, QCONV_EWORKSPACE, QCONV_EHIP.
 */
int qconv2d(const qconv_desc *d, const void *x, const void *w, const qconv_epilogue *epi, void *y,
            void *workspace, size_t workspace_bytes, int32_t tile_id, void *stream);

/*
 * Prepared filters.  Filters are constant across calls, so their layout work
 * can be done once, offline, like packing them (Sec. 3.3: keep operands in the
 * layout the kernel consumes).  For a wide tile the prepared form is the
 * int8 image of each (output-channel tile, channel chunk) block exactly as
 * the kernel stages it in LDS, so staging filters becomes a contiguous copy;
 * for other tiles it is the packed KRSC filters unchanged.
 *
 * qconv_prepared_filter_bytes -- host only: size of the prepared filters of
 *   `tile_id` (-1 = the built-in choice for `d`) for this shape.
 * qconv_prepare_filters -- device work on `stream`: w_packed (packed KRSC,
 *   16-byte aligned) -> w_prepared (`bytes` >= the size above, 16-byte
 *   aligned, not overlapping w_packed).  Errors: QCONV_EINVAL,
 *   QCONV_EUNSUPPORTED, QCONV_EHIP.
 * qconv2d_prepared -- qconv2d with prepared filters; `tile_id` must be the
 *   one they were prepared for (-1 resolves the same way for the same
 *   descriptor).  `splits` (1 = none) selects split-K, below; `workspace`
 *   may be NULL when splits == 1.  Results are identical to qconv2d.
 */
int qconv_prepared_filter_bytes(const qconv_desc *d, int32_t tile_id, size_t *bytes);
int qconv_prepare_filters(const qconv_desc *d, const void *w_packed, int32_t tile_id, void *w_prepared,
                          size_t bytes, void *stream);
int qconv2d_prepared(const qconv_desc *d, const void *x, const void *w_prepared, size_t w_prepared_bytes,
                     const qconv_epilogue *epi, void *y, int32_t tile_id, int32_t splits, void *workspace,
                     size_t workspace_bytes, void *stream);

/*
 * A 1x1 projection fused into a 3x3 layer.  A residual stage's first block
 * reads one input twice: its 3x3 convolution (stride s, padding 1) and the
 * 1x1 projection of its shortcut (stride s, no padding), whose output pixel
 * (p, q) reads input pixel (p*s, q*s) -- exactly the pixel the 3x3 window's
 * centre tap reads.  The fused launch stages the input band once (Sec. 3.1)
 * and runs the projection's products on the centre tap's fragments, so the
 * projection costs no launch and no second pass over the input; each output
 * gets its own epilogue before its store (Sec. 3.2.2) in the packed layout
 * the next layer reads (Sec. 3.3).  The two outputs equal qconv2d of the 3x3
 * layer and qconv2d of the projection (d with r = s = 1 and no
 * padding) on the same input.
 *   d          the 3x3 layer: r == s == 3, pad_h == pad_w == 1, plain layout;
 *              the projection has the same n, h, w, c, k, strides, bits and
 *              signedness
 * qconv_proj_default_tile -- host only: the built-in tile for such a layer, or
 *   an error (QCONV_EUNSUPPORTED when no tile with a projection instance fits).
 * qconv_proj_tile_check -- host only: QCONV_OK if `tile_id` can run it.
 * qconv_prepared_proj_filter_bytes -- host only: size of its prepared filters.
 * qconv_prepare_filters_proj -- device work on `stream`: packed KRSC 3x3
 *   filters `w_packed` and packed k x 1 x 1 x c projection filters
 *   `w_proj_packed` (16-byte aligned) -> one prepared image for `tile_id`
 *   (the projection is its tenth tap).  Errors as qconv_prepare_filters.
 * qconv_proj_workspace_bytes -- host only: split-K workspace of the fused
 *   launch for (tile_id, splits) (the projection's partial sums double it; 0
 *   when splits == 1); errors as qconv_workspace_bytes.
 * qconv2d_proj -- the fused launch.  `epi` and `epi_proj` must have the same
 *   mode: raw (both NULL or QCONV_OUT_RAW_I32: y and y_proj get int32
 *   accumulators) or requant (each with its own multipliers, shift, ReLU,
 *   clamp and optional bias; no residual).  y and y_proj (16-byte aligned,
 *   y_packed_bytes or y_raw_bytes each) must not overlap each other or any
 *   input.  `splits`, `workspace` and `workspace_bytes` as for split-K below
 *   (qconv_max_splits bounds `splits`; the workspace is
 *   qconv_proj_workspace_bytes long, under the same contract).  Errors as
 *   qconv2d_prepared.
 */
int qconv_proj_default_tile(const qconv_desc *d);
int qconv_proj_tile_check(const qconv_desc *d, int32_t tile_id);
int qconv_prepared_proj_filter_bytes(const qconv_desc *d, int32_t tile_id, size_t *bytes);
int qconv_prepare_filters_proj(const qconv_desc *d, const void *w_packed, const void *w_proj_packed, int32_t tile_id,
                               void *w_prepared, size_t bytes, void *stream);
int qconv_proj_workspace_bytes(const qconv_desc *d, int32_t tile_id, int32_t splits, size_t *bytes);
int qconv2d_proj(const qconv_desc *d, const void *x, const void *w_prepared, size_t w_prepared_bytes,
                 const qconv_epilogue *epi, void *y, const qconv_epilogue *epi_proj, void *y_proj, int32_t tile_id,
                 int32_t splits, void *workspace, size_t workspace_bytes, void *stream);

/*
 * qconv2d_packing -- qconv_pack of the activations fused into
 * qconv2d_prepared (Sec. 1 packing, Sec. 3.1 staging): the convolution reads
 * int8 activations and saturates each value into the b-bit range of
 * d->x_signed while it stages its input band, so y is exactly
 * qconv2d_prepared(qconv_pack(x_nchw)).  One launch instead of two, for a
 * network's first layer.
 *   x_nchw    DEVICE int8, n x c x h x w, 16-byte aligned
 *   x_packed  DEVICE, qconv_layout_info.x_bytes, 16-byte aligned, or NULL:
 *             also receives qconv_pack(x_nchw), each pixel written by the
 *             workgroup whose band's rows it starts (needs bands that cover
 *             every input row: stride_h <= r and the last window reaching the
 *             last row, else QCONV_EUNSUPPORTED)
 * Runs a wide tile's 3x3 instance (tile_id as for the prepared filters;
 * d->r == d->s == 3), plain layout, no split, no bias or residual; other
 * requests return QCONV_EUNSUPPORTED.  No operand may overlap another.
 * Errors as qconv2d_prepared.
 */
int qconv2d_packing(const qconv_desc *d, const int8_t *x_nchw, void *x_packed, const void *w_prepared,
                    size_t w_prepared_bytes, const qconv_epilogue *epi, void *y, int32_t tile_id, void *stream);

/*
 * Split-K over channel chunks (prepared filters, wide tiles).  The depth
 * C*R*S of the implicit GEMM (Sec. 2.1) is a sum over channel chunks of
 * `chunk_c` channels; with `splits` > 1 each output tile is computed by
 * `splits` workgroups, each summing its range of chunks into exact int32
 * partial sums.  The last workgroup of a tile to finish adds the others'
 * partial sums and applies the epilogue, so results are identical to
 * splits == 1 (integer addition is exact and associative).
 *
 * qconv_max_splits -- host only: number of channel chunks of `tile_id` for
 *   this shape (the largest useful `splits`; 1 for staged tiles), or an error.
 * qconv_workspace_bytes -- host only: workspace `qconv2d_prepared` needs for
 *   (tile_id, splits): 0 when splits == 1.  Requests past the chunk count are
 *   QCONV_EUNSUPPORTED; a request that would leave a split empty is reduced.
 * Workspace contract: caller-owned device memory, 16-byte aligned, not
 *   overlapping x, w or y, and ZERO-FILLED before its first use; every call
 *   leaves it ready for the next (its arrival counters return to zero).  Calls
 *   that use one workspace must not run concurrently.  QCONV_EWORKSPACE when it
 *   is missing or too small.
 */
int qconv_max_splits(const qconv_desc *d, int32_t tile_id);
int qconv_workspace_bytes(const qconv_desc *d, int32_t tile_id, int32_t splits, size_t *bytes);

/*
 * qconv2d_prepared_noalloc -- for callers that cannot allocate device memory
 * (code under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc): qconv2d_prepared without a workspace argument.  A split-K call
 * keeps its partial sums and arrival counters in a scratch array the library
 * holds in each GPU's memory (a static device array, present from the load of
 * the library to the end of the process), so nothing is allocated, freed or
 * memset by the call; the caller still passes x, the prepared filters and y.
 * Results are identical to qconv2d_prepared with the same tile and splits.
 *   Limit: the split-K partial sums (tiles x splits x tile_p x tile_k int32)
 *   must fit the scratch, and the output tiles its counters; qconv_noalloc_limits
 *   gives both (16 MiB minus 64 KiB, 16384 tiles).  Larger requests return
 *   QCONV_EWORKSPACE before anything is enqueued.  splits == 1 uses no scratch.
 *   Set-up: the first call on a device looks up that device's copy of the
 *   array and enqueues, on `stream`, the clearing of its counters (a small
 *   kernel, no memset); every split-K launch leaves them at zero again.
 *   Concurrency: all calls on one GPU share its scratch, which keeps the last
 *   call's contents; split-K calls that overlap in time on one GPU (other
 *   streams, other threads) race and give wrong results.  Serialise them.
 * Errors as qconv2d_prepared.
 */
int qconv2d_prepared_noalloc(const qconv_desc *d, const void *x, const void *w_prepared, size_t w_prepared_bytes,
                             const qconv_epilogue *epi, void *y, int32_t tile_id, int32_t splits, void *stream);

/* Host only: the no-alloc scratch's capacity for split-K partial sums (bytes) and
 * output tiles (counters); either pointer may be NULL.  Returns QCONV_OK. */
int qconv_noalloc_limits(int64_t *scratch_bytes, int64_t *max_tiles);

/*
 * Schedules.  The knobs of the schedule search space (Sec. 4.1: warps per
 * block along M and N, MMA tiles per warp along M and N, the input-channel
 * chunk -- here fixed per compiled tile -- and the loop order), as they exist
 * in this implementation, plus the launch knobs it adds.  Every valid
 * schedule computes the same bytes; only the time differs, which is what a
 * schedule search measures.
 *   tile_id       compiled tile (qconv_tile_get: waves and fragments per
 *                 workgroup along pixels and channels, chunk); -1 = the
 *                 built-in choice
 *   splits        split-K factor over channel chunks, 1 .. qconv_max_splits
 *                 (1 for staged tiles)
 *   wg_per_cu     workgroups per CU a persistent grid is sized for (1..16);
 *                 0 = the runtime's occupancy figure.  Ignored when every
 *                 workgroup gets a single stage or with a split.
 *   band_buffers  LDS band buffers of a persistent single-chunk plan: 1 (one
 *                 more barrier per stage, less LDS), 2, or 0 = whichever lets
 *                 more workgroups share a CU.  Ignored where it does not apply.
 *   xcd_order     1 = consecutive workgroup tiles are placed on one XCD,
 *                 pixel tiles outermost, so neighbouring tiles share its L2
 *                 (halo rows) while it reads every channel tile's filters;
 *                 2 = the same with channel tiles outermost, so an XCD reads
 *                 only its channel tiles' filters (deep layers, whose filters
 *                 outweigh their input); 0 = the hardware's round-robin
 *                 order; -1 = the library's choice (what qconv2d and
 *                 qconv2d_prepared use): the order whose bytes read into the
 *                 eight L2s, filters and input, are fewer
 *   ablation      0 for normal use.  For measuring the techniques (the
 *                 ablation of Sec. 4.4), a bit mask of techniques switched
 *                 off: 1 = duplicate-aware loading (Sec. 3.1) -- every tile
 *                 pixel is staged once per filter tap, as the lowered matrix;
 *                 2 = register-level packing (Sec. 3.2) -- the int32
 *                 accumulators pass through LDS to a separate requantise and
 *                 pack step; 4 = widening at staging -- the 4-bit activations
 *                 stay packed in LDS and every fragment is widened to int8
 *                 after its LDS read, inside the MFMA loop.  Every subset
 *                 (1 .. 7) is compiled for 4-bit 3x3 layers on the tiles
 *                 wide_b4_w4x1_f1x4_c64, wide_b4_w8x1_f1x4_c64 and
 *                 wide_b4_w4x1_f2x4_c64, without split, bias or residual;
 *                 QCONV_EUNSUPPORTED otherwise.  Results are identical.
 * qconv_schedule_check -- host only: QCONV_OK if the schedule can run `d`
 *   (QCONV_EINVAL for a knob out of range, else what the call would return).
 * qconv2d_scheduled -- qconv2d_prepared with every knob given; the prepared
 *   filters must be those of s->tile_id; `workspace` as for split-K above.
 *   qconv2d_prepared(..., tile_id, splits, ...) is the schedule
 *   {tile_id, splits, 0, 0, -1, 0}.
 */
typedef struct {
    int32_t tile_id;
    int32_t splits;
    int32_t wg_per_cu;
    int32_t band_buffers;
    int32_t xcd_order;
    int32_t ablation;
} qconv_schedule;

int qconv_schedule_check(const qconv_desc *d, const qconv_schedule *s);
int qconv2d_scheduled(const qconv_desc *d, const void *x, const void *w_prepared, size_t w_prepared_bytes,
                      const qconv_epilogue *epi, void *y, const qconv_schedule *s, void *workspace,
                      size_t workspace_bytes, void *stream);

/* Number of compiled tile configurations; ids are 0 .. count-1. */
int qconv_tile_count(void);

/* Describe tile `tile_id`.  QCONV_EINVAL for an unknown id or NULL `out`. */
int qconv_tile_get(int32_t tile_id, qconv_tile_info *out);

/*
 * qconv_tile_check -- host only: QCONV_OK if tile `tile_id` can run `d`
 * (bit-width matches, staging fits in LDS), else the status qconv2d would
 * return for it.
 */
int qconv_tile_check(const qconv_desc *d, int32_t tile_id);

/* The tile qconv2d uses for tile_id = -1 (a static per-shape heuristic). */
int qconv_default_tile(const qconv_desc *d);

/*
 * qconv_build_digest -- host only: a 16-hex-digit digest of the sources and
 * compile flags this library was built from (static string; "unknown" for a
 * build that did not set it).  Lets a caller check that the binary it loaded
 * is the one its sources describe.
 */
const char *qconv_build_digest(void);

/* Static text for a status code. */
const char *qconv_strerror(int status);

/* Detail of the calling thread's most recent failure ("" if none). */
const char *qconv_last_error(void);

/*
 * qconv_probe_mfma_i8 -- measurement aid, not part of the convolution: a
 * kernel that issues nothing but v_mfma_i32_16x16x64_i8 (four waves per
 * workgroup, eight independent accumulator chains per wave), so a caller can
 * time the int8 rate the matrix cores sustain on this device and report a
 * convolution kernel against it as well as against the nominal peak (the
 * evaluation of Sec. 4 rates kernels by their throughput).
 *   blocks  workgroups, 1 .. 2^20;  iters  rounds of eight MFMAs per wave, 1 .. 2^24
 *   sink    device int32[blocks * 256], 4-byte aligned: one sum per lane, written
 *           so the work stays live (its values mean nothing)
 *   stamps  device uint64[blocks * 4], 8-byte aligned: per workgroup, wave 0's
 *           shader-clock counter before and after its loop, then the 100 MHz
 *           constant counter before and after; their ratio is the shader clock
 *   ops     host, may be NULL: int8 operations one launch performs
 *           (blocks * 4 * iters * 8 * 32768)
 * QCONV_EINVAL for out-of-range sizes or NULL/misaligned buffers; QCONV_EHIP
 * if the launch is rejected.  Asynchronous on `stream`.
 */
int qconv_probe_mfma_i8(int32_t blocks, int32_t iters, int32_t *sink, uint64_t *stamps, int64_t *ops,
                        void *stream);

/*
 * qconv_probe_mfma_i8_shape -- the same probe with the MFMA shape chosen:
 * shape 0 is qconv_probe_mfma_i8 (eight chains of v_mfma_i32_16x16x64_i8 per
 * wave), shape 1 runs four chains of v_mfma_i32_32x32x32_i8 per wave -- the
 * same int8 operations per round, so *ops has the same closed form.  With
 * blocks = 256 or 512 (one or two waves per SIMD, the occupancy of the
 * convolution kernels) the two rates show what the instruction shape itself
 * costs.  Arguments, errors and asynchrony as for qconv_probe_mfma_i8;
 * QCONV_EINVAL also for a shape other than 0 or 1.
 */
int qconv_probe_mfma_i8_shape(int32_t shape, int32_t blocks, int32_t iters, int32_t *sink, uint64_t *stamps,
                              int64_t *ops, void *stream);

/*
 * qconv_last_launch -- host only: the grid (workgroups), workgroup size
 * (threads) and dynamic LDS bytes of the calling thread's most recent
 * convolution launch (any qconv2d* entry point that returned QCONV_OK); any
 * pointer may be NULL.  QCONV_EINVAL when the thread has launched none.
 */
int qconv_last_launch(int64_t *grid, int64_t *threads, int64_t *lds_bytes);

/*
 * qconv_probe_launch -- measurement aid, not part of the convolution: an
 * empty kernel over `blocks` workgroups of `threads` threads with `lds_bytes`
 * of dynamic LDS.  Its time per launch (back to back, or replayed from a
 * graph) is the fixed cost of dispatching and draining a grid of that shape,
 * the floor under any kernel launched once per layer.
 *   blocks 1 .. 2^20; threads a multiple of 64 in 64 .. 1024; lds_bytes
 *   0 .. 163840.  QCONV_EINVAL otherwise; QCONV_EHIP if the launch is
 *   rejected.  Asynchronous on `stream`.
 */
int qconv_probe_launch(int32_t blocks, int32_t threads, int32_t lds_bytes, void *stream);

/*
 * qconv_probe_grid_meet -- measurement aid, not part of the convolution: the
 * cost of a device-wide meeting inside one launch, the alternative to a launch
 * per layer when a chain of layers (Sec. 3.3: each layer's packed output is
 * the next one's input) runs as one persistent grid.  Enqueues a one-wave
 * kernel that zeroes the counters, then `blocks` workgroups of 256 threads
 * that meet `rounds` times: each workgroup releases its writes at device
 * scope, counts itself in, waits until the whole grid has arrived, then
 * acquires.  The time per launch at rounds R minus that at rounds 0, over R,
 * is the cost of one meeting.
 *   blocks    1 .. the device's CU count (the grid must be resident at once)
 *   rounds    0 .. 4096
 *   two_level 0: every workgroup adds 1 to one counter; 1: each adds 1 to its
 *             XCD group's counter (blockIdx mod 8) and the last of a group
 *             adds 1 to the top counter
 *   arrivals  device uint32[144], 4-byte aligned, owned by the caller: the top
 *             counter at [0], group g's at [16 (g + 1)]; on return (after the
 *             stream drains) [0] holds rounds x blocks (flat) or rounds x
 *             min(blocks, 8) (two-level)
 *   err       device int32, 4-byte aligned: left alone unless a workgroup gave
 *             up waiting (2^17 polls, a fraction of a second), which writes 1;
 *             the caller zeroes it first
 * QCONV_EINVAL for out-of-range arguments or NULL/misaligned pointers;
 * QCONV_EHIP if the device cannot be queried or a launch is rejected.
 * Asynchronous on `stream`; calls that overlap on one set of counters race.
 */
int qconv_probe_grid_meet(int32_t blocks, int32_t rounds, int32_t two_level, uint32_t *arrivals, int32_t *err,
                          void *stream);

/*
 * Host-only self-check of the index arithmetic the kernels use (run-time
 * constant division); touches no device.  Returns 0 when it holds.
 */
int qconv_selftest(void);

#ifdef __cplusplus
}
#endif

#endif /* QCONV_H */
