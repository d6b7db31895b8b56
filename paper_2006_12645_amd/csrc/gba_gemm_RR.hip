// Kernel instantiations for A ROW-major, B ROW-major (one of the four
// layout specialisations of the Matmul Compute Decomposition section).  One
// translation unit per layout pair so the library builds in parallel.
#include "gba_tiles.hpp"

namespace gba {

#define GBA_FAST_ENTRY(id, BM, BN, WM, WN, SK, NSTG) \
    {&launch_fast<BM, BN, WM, WN, SK, NSTG, ROW, ROW, false>, fast_acc16<BM, BN, WM, WN, SK, NSTG, ROW, ROW>()},

const LayoutTable &table_RR()
{
    static const LayoutTable t = {
        {GBA_TILE_LIST(GBA_FAST_ENTRY)},
        {&launch_generic<ROW, ROW, false>, &launch_generic<ROW, ROW, true>},
    };
    return t;
}

#undef GBA_FAST_ENTRY

}  // namespace gba
