// Wide tiles of group B (qconv_kernels.h), compiled in a translation unit
// of their own; qconv_conv.hip appends them to the tile registry.
#include "qconv_kernels.h"

namespace qconv {

TileEntry g_wide_tiles_b[] = {QCONV_WIDE_TILES_B(QCONV_WIDE_ENTRY)};
int g_wide_tiles_b_count = (int)(sizeof(g_wide_tiles_b) / sizeof(g_wide_tiles_b[0]));

}  // namespace qconv
