// Tile registry of the convolution kernels of qconv_kernels.h.  The staged
// tiles and the first group of wide tiles are compiled here; the other wide
// groups, the ablation instances and the projection instances each in a
// translation unit of its own (qconv_tiles_*.hip), so the build compiles them
// in parallel.  Tile ids
// follow the lists' order: staged tiles, then wide groups A to D.
#include <vector>

#include "qconv_kernels.h"

namespace qconv {

extern TileEntry g_wide_tiles_b[], g_wide_tiles_c[], g_wide_tiles_d[];   // (not const: a const array would also be emitted for the device)
extern int g_wide_tiles_b_count, g_wide_tiles_c_count, g_wide_tiles_d_count;

static TileEntry g_tiles_here[] = {QCONV_STAGED_TILES(QCONV_STAGED_ENTRY) QCONV_WIDE_TILES_A(QCONV_WIDE_ENTRY)};

static const std::vector<TileEntry> &all_tiles() {
    static const std::vector<TileEntry> all = [] {
        std::vector<TileEntry> v(std::begin(g_tiles_here), std::end(g_tiles_here));
        v.insert(v.end(), g_wide_tiles_b, g_wide_tiles_b + g_wide_tiles_b_count);
        v.insert(v.end(), g_wide_tiles_c, g_wide_tiles_c + g_wide_tiles_c_count);
        v.insert(v.end(), g_wide_tiles_d, g_wide_tiles_d + g_wide_tiles_d_count);
        for (int i = 0; i < (int)v.size(); ++i) v[i].info.id = i;
        return v;
    }();
    return all;
}

const TileEntry *tile_table() { return all_tiles().data(); }

int tile_table_size() { return (int)all_tiles().size(); }

}  // namespace qconv
