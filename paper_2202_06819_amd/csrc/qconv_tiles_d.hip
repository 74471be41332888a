// Wide tiles of group D (qconv_kernels.h), compiled in a translation unit
// of their own; qconv_conv.hip appends them to the tile registry.
#include "qconv_kernels.h"

namespace qconv {

TileEntry g_wide_tiles_d[] = {QCONV_WIDE_TILES_D(QCONV_WIDE_ENTRY)};
int g_wide_tiles_d_count = (int)(sizeof(g_wide_tiles_d) / sizeof(g_wide_tiles_d[0]));

}  // namespace qconv
