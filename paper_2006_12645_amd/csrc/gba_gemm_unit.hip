// Kernel instantiations for one operand-layout pair (one of the four layout
// specialisations of the Matmul Compute Decomposition section) and one
// kernel variant.  The build compiles this file once per combination, with
//   GBA_LA, GBA_LB  0 = row-major, 1 = column-major (A and B)
//   GBA_PRO         1 = ReLU prologue on the left operands
//   GBA_DUAL        1 = a second product P.Q accumulated with A.B
// so the library's kernels build in parallel.
#include "gba_tiles.hpp"

#if !defined(GBA_LA) || !defined(GBA_LB) || !defined(GBA_PRO) || !defined(GBA_DUAL)
#error "gba_gemm_unit.hip needs GBA_LA, GBA_LB, GBA_PRO and GBA_DUAL"
#endif

namespace gba {

constexpr int UNIT_LA = GBA_LA, UNIT_LB = GBA_LB;
constexpr bool UNIT_PRO = GBA_PRO != 0, UNIT_DUAL = GBA_DUAL != 0;

#define GBA_FAST_ENTRY(id, BM, BN, WM, WN, SK, NSTG)                                              \
    {&launch_fast<BM, BN, WM, WN, SK, NSTG, UNIT_LA, UNIT_LB, false, UNIT_PRO, UNIT_DUAL>,         \
     fast_acc16<BM, BN, WM, WN, SK, NSTG, UNIT_LA, UNIT_LB, UNIT_PRO, UNIT_DUAL>()},
#define GBA_SPLIT_ENTRY(id, BM, BN, WM, WN, SK, NSTG) \
    fast_split<BM, BN, WM, WN, SK, NSTG, UNIT_LA, UNIT_LB, UNIT_PRO, UNIT_DUAL>(),

template <>
const LayoutTable &layout_table<UNIT_LA, UNIT_LB, UNIT_PRO, UNIT_DUAL>()
{
    static const LayoutTable t = {
        {GBA_TILE_LIST(GBA_FAST_ENTRY)},
        {GBA_TILE_LIST(GBA_SPLIT_ENTRY)},
        {&launch_generic<UNIT_LA, UNIT_LB, false, UNIT_PRO, UNIT_DUAL>,
         &launch_generic<UNIT_LA, UNIT_LB, true, UNIT_PRO, UNIT_DUAL>},
    };
    return t;
}

#undef GBA_FAST_ENTRY
#undef GBA_SPLIT_ENTRY

}  // namespace gba
