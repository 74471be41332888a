// Ablation instances (4-bit, 3x3, prepared filters; for measurement only):
// every subset of the three techniques switched off (mask bits: 1 lowered
// staging, 2 LDS-staged int32 epilogue, 4 packed activations in LDS widened
// in the MFMA loop), for three tiles.  In a translation unit of its own so the
// build compiles it in parallel.  They are single-stage instances, like the
// full kernel they are measured against on single-chunk layers.
#include <string.h>

#include "qconv_kernels.h"

namespace qconv {

#define QCONV_ABL(WP, WK, FP, FK, MASK)                                                                           \
    {"wide_b4_w" #WP "x" #WK "_f" #FP "x" #FK "_c64", MASK,                                                        \
     &launch_wide<4, WP, WK, FP, FK, 64, false, true, 3, 3, false, MASK, false, false, false, true>,              \
     reinterpret_cast<const void *>(                                                                              \
         &conv_wide<4, WP, WK, FP, FK, 64, false, true, 3, 3, false, MASK, false, false, false, true>)}
#define QCONV_ABL7(WP, WK, FP, FK)                                                                                \
    QCONV_ABL(WP, WK, FP, FK, 1), QCONV_ABL(WP, WK, FP, FK, 2), QCONV_ABL(WP, WK, FP, FK, 3),                     \
        QCONV_ABL(WP, WK, FP, FK, 4), QCONV_ABL(WP, WK, FP, FK, 5), QCONV_ABL(WP, WK, FP, FK, 6),                 \
        QCONV_ABL(WP, WK, FP, FK, 7)
static const AblationInstance g_ablation[] = {QCONV_ABL7(4, 1, 1, 4), QCONV_ABL7(8, 1, 1, 4), QCONV_ABL7(4, 1, 2, 4)};

const AblationInstance *ablation_instance(const char *tile_name, int mask) {
    for (const AblationInstance &e : g_ablation)
        if (e.mask == mask && strcmp(e.tile, tile_name) == 0) return &e;
    return nullptr;
}

}  // namespace qconv
