// Kernel instantiations for A COL-major, B COL-major (one of the four
// layout specialisations of the Matmul Compute Decomposition section).  One
// translation unit per layout pair so the library builds in parallel.
#include "gba_tiles.hpp"

namespace gba {

#define GBA_FAST_ENTRY(id, BM, BN, WM, WN, SK, NSTG) \
    {&launch_fast<BM, BN, WM, WN, SK, NSTG, COL, COL, false>, fast_acc16<BM, BN, WM, WN, SK, NSTG, COL, COL>()},

const LayoutTable &table_CC()
{
    static const LayoutTable t = {
        {GBA_TILE_LIST(GBA_FAST_ENTRY)},
        {&launch_generic<COL, COL, false>, &launch_generic<COL, COL, true>},
    };
    return t;
}

#undef GBA_FAST_ENTRY

}  // namespace gba
