// gba_tiles.hpp -- the tile configurations compiled into the library and the
// launch-table types shared by the per-layout instantiation units and the
// host entry points.
//
// The paper generated one kernel per block/warp tile choice and kept the
// best per problem size (Experimental Evaluation section); this table is the
// MI355X counterpart of that tile space.  Block tiles are sized for the
// 160 KB LDS of a gfx950 compute unit (two stages of (BM + BN) x 64 fp16)
// and wave tiles for its 512 registers per lane.
#pragma once

#include <hip/hip_runtime.h>

#include "gba_kernel.hpp"

namespace gba {

struct TileCfg {
    int bm, bn, wm, wn;
};

// X(id, BM, BN, WM, WN): BM output rows x BN output columns per workgroup,
// WM x WN waves, each owning a (BM/WM) x (BN/WN) sub-tile.
#define GBA_TILE_LIST(X)   \
    X(0, 256, 256, 2, 4)   \
    X(1, 256, 256, 2, 2)   \
    X(2, 128, 128, 2, 2)   \
    X(3, 256, 128, 2, 2)   \
    X(4, 128, 256, 2, 2)   \
    X(5, 64, 64, 2, 2)     \
    X(6, 32, 64, 1, 2)     \
    X(7, 64, 128, 2, 2)

constexpr int NUM_TILES = 8;
// The configuration used whenever an operand is not 16-byte aligned.
constexpr int GENERIC_TILE = 5;

#define GBA_TILE_CFG(id, BM, BN, WM, WN) TileCfg{BM, BN, WM, WN},
constexpr TileCfg TILES[NUM_TILES] = {GBA_TILE_LIST(GBA_TILE_CFG)};
#undef GBA_TILE_CFG

typedef hipError_t (*LaunchFn)(const GemmArgs &, hipStream_t);

// Per operand-layout pair: vec[tile][acc16] for 16-byte aligned operands,
// scalar[acc16] (GENERIC_TILE) otherwise.
struct LayoutTable {
    LaunchFn vec[NUM_TILES][2];
    LaunchFn scalar[2];
};

template <int BM, int BN, int WM, int WN, int LA, int LB, bool ACC16, bool VEC>
hipError_t launch_gemm(const GemmArgs &a, hipStream_t s)
{
    dim3 grid((unsigned)(a.tiles_m * a.tiles_n)), block(64 * WM * WN);
    hipLaunchKernelGGL((gemm_bias_act_kernel<BM, BN, WM, WN, LA, LB, ACC16, VEC>), grid, block, 0,
                       s, a);
    return hipGetLastError();
}

// Host-side launch tables, one per layout pair (defined in gba_gemm_<layout>.hip).
const LayoutTable &table_RR();
const LayoutTable &table_RC();
const LayoutTable &table_CR();
const LayoutTable &table_CC();

}  // namespace gba
