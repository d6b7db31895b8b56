// gba_common.hpp -- types and helpers shared by the fused GEMM + bias +
// activation kernels (fast path in gba_kernel.hpp, general path in
// gba_kernel_generic.hpp).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace gba {

typedef _Float16 h8 __attribute__((ext_vector_type(8)));
typedef float f4 __attribute__((ext_vector_type(4)));
typedef float f16v __attribute__((ext_vector_type(16)));
typedef int i4 __attribute__((ext_vector_type(4)));

enum { ROW = 0, COL = 1 };

// Kernel arguments: operands as the C ABI describes them (A(i,k), B(k,j) per
// layout, C row-major), the activation switch and the output tile grid.
struct GemmArgs {
    const _Float16 *A;
    const _Float16 *B;
    const _Float16 *bias;  // may be null
    _Float16 *C;
    int64_t lda, ldb, ldc;
    int M, N, K;
    int relu;
    int tiles_m, tiles_n;
};

__device__ __forceinline__ h8 zero_h8()
{
    h8 z;
#pragma unroll
    for (int e = 0; e < 8; ++e) z[e] = (_Float16)0.0f;
    return z;
}

// Map the hardware workgroup id to a (tile_m, tile_n) pair.  Workgroups are
// dispatched round-robin over the 8 XCDs, each with its own L2, so the
// linear order is first regrouped to give each XCD a contiguous range, and
// that range is walked in groups of GROUP_M tile rows so the workgroups that
// share an L2 also share A row panels and B column panels.
__device__ __forceinline__ void tile_coords(int bid, int nwg, int tiles_m, int &tm, int &tn)
{
    constexpr int NXCD = 8, GROUP_M = 4;
    int q = nwg / NXCD, rem = nwg % NXCD;
    int xcd = bid % NXCD, local = bid / NXCD;
    int lin = xcd < rem ? xcd * (q + 1) + local : rem * (q + 1) + (xcd - rem) * q + local;
    int tiles_n = nwg / tiles_m;
    int group = lin / (GROUP_M * tiles_n);
    int first_m = group * GROUP_M;
    int gm = tiles_m - first_m < GROUP_M ? tiles_m - first_m : GROUP_M;
    int in_group = lin - group * GROUP_M * tiles_n;
    tm = first_m + in_group % gm;
    tn = in_group / gm;
}

}  // namespace gba
