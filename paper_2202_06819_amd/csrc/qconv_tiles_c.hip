// Wide tiles of group C (qconv_kernels.h), compiled in a translation unit
// of their own; qconv_conv.hip appends them to the tile registry.
#include "qconv_kernels.h"

namespace qconv {

TileEntry g_wide_tiles_c[] = {QCONV_WIDE_TILES_C(QCONV_WIDE_ENTRY)};
int g_wide_tiles_c_count = (int)(sizeof(g_wide_tiles_c) / sizeof(g_wide_tiles_c[0]));

}  // namespace qconv
