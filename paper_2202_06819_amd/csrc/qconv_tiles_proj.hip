// 3x3 instances with a 1x1 projection at the same stride fused in (the
// strided entry of a residual stage and its shortcut projection read the same
// block input), compiled for the tiles that run those layers.  In a
// translation unit of its own so the build compiles it in parallel.
#include <string.h>

#include "qconv_kernels.h"

namespace qconv {

#define QCONV_PROJ_TILES(X) \
    X(4, 4, 2, 2, 2, 64)    \
    X(4, 2, 2, 2, 2, 64)    \
    X(4, 4, 1, 2, 4, 64)    \
    X(4, 4, 2, 2, 2, 128)   \
    X(8, 4, 2, 2, 2, 64)    \
    X(8, 4, 1, 2, 4, 64)

static const ProjInstance g_proj[] = {QCONV_PROJ_TILES(QCONV_PROJ_ENTRY)};

const ProjInstance *proj_instance(const char *tile_name) {
    for (const ProjInstance &e : g_proj)
        if (strcmp(e.tile, tile_name) == 0) return &e;
    return nullptr;
}

}  // namespace qconv
