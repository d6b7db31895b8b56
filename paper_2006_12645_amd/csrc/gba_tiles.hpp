// gba_tiles.hpp -- the tile configurations compiled into the library and the
// launch-table types shared by the per-layout instantiation units and the
// host entry points.
//
// The paper generated one kernel per block/warp tile choice and kept the
// best per problem size (Experimental Evaluation section); this table is the
// MI355X counterpart of that tile space.  Block tiles are sized for the
// 160 KB LDS of a gfx950 compute unit (two stages of (BM + BN) x 64 fp16)
// and warp tiles for its 512 registers per lane.
#pragma once

#include <hip/hip_runtime.h>

#include "gba_kernel.hpp"
#include "gba_kernel16.hpp"
#include "gba_kernel_generic.hpp"

namespace gba {

struct TileCfg {
    int bm, bn, wm, wn, sk, nstg;
};

// X(id, BM, BN, WM, WN, SK, NSTG): BM output rows x BN output columns per
// workgroup, WM x WN waves, each owning a (BM/WM) x (BN/WN) warp tile
// (multiples of 32 x 32, the MFMA block), times SK k-groups of waves that
// split each reduction step (intra-workgroup split-K; fp32 accumulation
// only); NSTG LDS stages.
#define GBA_TILE_LIST(X)         \
    X(0, 256, 256, 2, 2, 1, 2)   \
    X(1, 256, 256, 2, 4, 1, 2)   \
    X(2, 256, 128, 2, 2, 1, 2)   \
    X(3, 128, 256, 2, 2, 1, 2)   \
    X(4, 128, 128, 2, 2, 1, 2)   \
    X(5, 128, 64, 2, 2, 1, 2)    \
    X(6, 64, 64, 2, 2, 1, 2)     \
    X(7, 64, 128, 2, 2, 1, 2)    \
    X(8, 32, 64, 1, 2, 1, 2)     \
    X(9, 32, 32, 1, 1, 1, 2)     \
    X(10, 64, 64, 1, 1, 4, 2)    \
    X(11, 64, 64, 2, 2, 2, 4)    \
    X(12, 32, 64, 1, 1, 4, 2)    \
    X(13, 32, 32, 1, 1, 4, 4)    \
    X(14, 128, 128, 2, 2, 2, 2)  \
    X(15, 64, 128, 1, 2, 2, 2)   \
    X(16, 256, 128, 2, 4, 1, 2)  \
    X(17, 128, 256, 4, 2, 1, 2)  \
    X(18, 128, 128, 2, 4, 1, 2)  \
    X(19, 128, 64, 4, 2, 1, 2)   \
    X(20, 64, 128, 2, 4, 1, 2)   \
    X(21, 32, 64, 1, 2, 1, 4)    \
    X(22, 64, 64, 2, 2, 1, 4)    \
    X(23, 32, 32, 1, 1, 1, 4)    \
    X(24, 32, 128, 1, 2, 1, 4)   \
    X(25, 128, 32, 2, 1, 1, 4)

constexpr int NUM_TILES = 26;

#define GBA_TILE_CFG(id, BM, BN, WM, WN, SK, NSTG) TileCfg{BM, BN, WM, WN, SK, NSTG},
constexpr TileCfg TILES[NUM_TILES] = {GBA_TILE_LIST(GBA_TILE_CFG)};
#undef GBA_TILE_CFG

// Block tile of the general path (any size, leading dimension, alignment).
constexpr TileCfg GENERIC_TILE = {64, 64, 2, 2, 1, 2};

typedef hipError_t (*LaunchFn)(const GemmArgs &, hipStream_t);

// Tiles whose reduction can also be split across workgroups (fp32
// accumulation): one k-group and at most 128x128 outputs.  Larger tiles
// already fill the GPU with few output tiles.
constexpr bool tile_splits(const TileCfg &c) { return c.sk == 1 && c.bm * c.bn <= 128 * 128; }

// Per operand-layout pair and kernel variant: fast[tile][acc16] for the
// aligned fast path (null for fp16 accumulation with split-K), split[tile]
// for its reduction split across workgroups (null where tile_splits is
// false), generic[acc16] otherwise.
struct LayoutTable {
    LaunchFn fast[NUM_TILES][2];
    LaunchFn split[NUM_TILES];
    LaunchFn generic[2];
};

// Which tiles run the 16x16x32 kernel (gemm_bias_act_fast16): the ones
// with eight waves of one k-group, in every layout where an M- or
// N-contiguous operand tile has 128 or more elements per row (its
// conflict-free group permutation needs eight 16-element groups); and,
// without prologue and unless the reduction is split across workgroups,
// the four-stage small tiles (21-25) under the same layout condition (all
// of them in the layout where both operand tiles are reduction-contiguous,
// 32x128 with row-major B, 128x32 with column-major A), where the 16x16x32
// kernel adds waves that only issue copies (with fp16 accumulation its
// fp16 running sum also breaks the chain of dependent MFMAs).  With fp32
// accumulation that is 6-10% faster than these tiles on 32x32x16 without
// copy-only waves, and than the k-group tiles on 1024^3 in RC (6.66 against
// 7.33 us) and 1000^3 (6.99 against 7.75); in RR, 32x128 takes 1024^3 in
// 7.84 us against 8.78 on the k-group 64x64 tile.
constexpr bool use_fast16(int la, int lb, int bm, int bn, int wm, int wn, int sk, int nstg, bool acc16, bool pro,
                          bool split = false)
{
    const bool layouts = (bm >= 128 || la == ROW) && (bn >= 128 || lb == COL);
    if (wm * wn == 8) return layouts;
    return (acc16 || !split) && !pro && sk == 1 && nstg == 4 && layouts;
}

// hipGetLastError reports the last failure of any runtime call on the
// calling thread, not only of the launch before it: the launchers clear it
// first, so that an earlier, unrelated failure does not turn a kernel that
// was enqueued (and will run) into an error return.
inline void clear_last_error() { (void)hipGetLastError(); }

template <int BM, int BN, int WM, int WN, int SK, int NSTG, int LA, int LB, bool ACC16, bool PRO, bool DUAL,
          bool SPLIT = false>
hipError_t launch_fast(const GemmArgs &a, hipStream_t s)
{
    // one workgroup per output tile, times the splits of its reduction
    constexpr int NPW = use_fast16(LA, LB, BM, BN, WM, WN, SK, NSTG, ACC16, PRO, SPLIT)
                            ? copy_only_waves<WM, WN, SK, ACC16, PRO, SPLIT>() : 0;
    dim3 grid((unsigned)(a.tiles_m * a.tiles_n * (SPLIT ? a.splits : 1))), block(64 * (WM * WN * SK + NPW));
    // The 8-wave tiles (one k-group) run on 16x16x32 MFMAs, and so do the
    // four-stage small tiles where use_fast16 allows them;
    // everything else on 32x32x16 (measured per tile: the 16x16x32 kernels
    // of the 4-wave tiles were up to 20% slower with fp32 accumulation, and
    // the 4-wave 256x256 one does not fit its 64 accumulator blocks per wave
    // in registers)
    clear_last_error();
    if constexpr (use_fast16(LA, LB, BM, BN, WM, WN, SK, NSTG, ACC16, PRO, SPLIT))
        hipLaunchKernelGGL((gemm_bias_act_fast16<BM, BN, WM, WN, SK, NSTG, LA, LB, ACC16, PRO, DUAL, SPLIT>), grid,
                           block, 0, s, a);
    else
        hipLaunchKernelGGL((gemm_bias_act_fast<BM, BN, WM, WN, SK, NSTG, LA, LB, ACC16, PRO, DUAL, SPLIT>), grid,
                           block, 0, s, a);
    return hipGetLastError();
}

// Launch-table entry for fp16 accumulation: none with split-K.
template <int BM, int BN, int WM, int WN, int SK, int NSTG, int LA, int LB, bool PRO, bool DUAL>
constexpr LaunchFn fast_acc16()
{
    if constexpr (SK == 1) return &launch_fast<BM, BN, WM, WN, SK, NSTG, LA, LB, true, PRO, DUAL>;
    else return nullptr;
}

// Launch-table entry for a reduction split across workgroups.
template <int BM, int BN, int WM, int WN, int SK, int NSTG, int LA, int LB, bool PRO, bool DUAL>
constexpr LaunchFn fast_split()
{
    if constexpr (tile_splits(TileCfg{BM, BN, WM, WN, SK, NSTG}))
        return &launch_fast<BM, BN, WM, WN, SK, NSTG, LA, LB, false, PRO, DUAL, true>;
    else return nullptr;
}

template <int LA, int LB, bool ACC16, bool PRO, bool DUAL>
hipError_t launch_generic(const GemmArgs &a, hipStream_t s)
{
    constexpr TileCfg c = GENERIC_TILE;
    dim3 grid((unsigned)(a.tiles_m * a.tiles_n)), block(64 * c.wm * c.wn);
    clear_last_error();
    hipLaunchKernelGGL((gemm_bias_act_generic<c.bm, c.bn, c.wm, c.wn, LA, LB, ACC16, PRO, DUAL>),
                       grid, block, 0, s, a);
    return hipGetLastError();
}

// Host-side launch table of one layout pair (LA, LB) and variant: PRO = ReLU
// prologue on the left operands, DUAL = a second product.  Each
// specialisation is defined in its own instantiation unit
// (gba_gemm_unit.hip compiled once per combination).
template <int LA, int LB, bool PRO, bool DUAL>
const LayoutTable &layout_table();

}  // namespace gba
