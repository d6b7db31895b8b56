// Kernel instantiations for A ROW-major, B ROW-major (one of the four
// layout specialisations of the Matmul Compute Decomposition section).  One
// translation unit per layout pair so the library builds in parallel.
#include "gba_tiles.hpp"

namespace gba {

#define GBA_VEC_ENTRY(id, BM, BN, WM, WN) \
    {&launch_gemm<BM, BN, WM, WN, ROW, ROW, false, true>, &launch_gemm<BM, BN, WM, WN, ROW, ROW, true, true>},

const LayoutTable &table_RR()
{
    static const LayoutTable t = {
        {GBA_TILE_LIST(GBA_VEC_ENTRY)},
        {&launch_gemm<64, 64, 2, 2, ROW, ROW, false, false>, &launch_gemm<64, 64, 2, 2, ROW, ROW, true, false>},
    };
    return t;
}

#undef GBA_VEC_ENTRY

static_assert(TILES[GENERIC_TILE].bm == 64 && TILES[GENERIC_TILE].bn == 64 &&
                  TILES[GENERIC_TILE].wm == 2 && TILES[GENERIC_TILE].wn == 2,
              "scalar entries are instantiated for the generic tile");

}  // namespace gba
