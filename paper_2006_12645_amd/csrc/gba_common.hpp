// gba_common.hpp -- types and helpers shared by the fused GEMM + bias +
// activation kernels (fast path in gba_kernel.hpp, general path in
// gba_kernel_generic.hpp).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace gba {

typedef _Float16 h8 __attribute__((ext_vector_type(8)));
typedef _Float16 h4 __attribute__((ext_vector_type(4)));
typedef float f4 __attribute__((ext_vector_type(4)));
typedef float f16v __attribute__((ext_vector_type(16)));
typedef int i4 __attribute__((ext_vector_type(4)));

enum { ROW = 0, COL = 1 };
enum { ACT_NONE = 0, ACT_RELU = 1, ACT_SIGMOID = 2, ACT_TANH = 3 };
enum { BIAS_NONE = 0, BIAS_ROW = 1, BIAS_FULL = 2 };

// Kernel arguments: operands as the C ABI describes them (A(i,k), B(k,j) per
// layout, C row-major), the optional second product P.Q (same layouts as A
// and B, reduction length K2; read only by kernels built for two products),
// the epilogue's bias and activation, and the output tile grid.
struct GemmArgs {
    const _Float16 *A;
    const _Float16 *B;
    const _Float16 *P;
    const _Float16 *Q;
    const _Float16 *bias;  // null when bias_kind == BIAS_NONE
    _Float16 *C;
    int64_t lda, ldb, ldp, ldq, ldc, ldbias;
    int M, N, K, K2;
    int act;               // ACT_*
    int bias_kind;         // BIAS_*: bias[j] or bias[i*ldbias + j]
    float bias_sign;       // +1: add the bias, -1: subtract it
    int sub;               // nonzero: C = A.B - P.Q instead of A.B + P.Q
    int tiles_m, tiles_n;
    // Reduction split across workgroups (splits > 1): workgroup b computes
    // split b % splits of output tile b / splits, i.e. reduction steps
    // [split * split_steps, (split + 1) * split_steps) of the steps of A.B
    // followed by those of P.Q; its fp32 partial tile goes to ws and the
    // last split of a tile to arrive (counted in counters, which start and
    // end at zero) sums them in split order and runs the epilogue.
    int splits, split_steps;
    float *ws;
    unsigned *counters;
};

__device__ __forceinline__ h8 zero_h8()
{
    h8 z;
#pragma unroll
    for (int e = 0; e < 8; ++e) z[e] = (_Float16)0.0f;
    return z;
}

typedef float f2v __attribute__((ext_vector_type(2)));
typedef _Float16 h2v __attribute__((ext_vector_type(2)));

// Two fp32 values rounded to the nearest fp16 (ties to even) and back.
__device__ __forceinline__ f2v round_f16x2(f2v x)
{
    return __builtin_convertvector(__builtin_convertvector(x, h2v), f2v);
}

typedef short s8 __attribute__((ext_vector_type(8)));

// max(x, 0) on eight fp16 values (the ReLU of a prologue), as a signed
// 16-bit integer max on the bit patterns: one v_pk_max_i16 per two values,
// where a floating-point max would first canonicalise its inputs.  Every
// finite fp16 with the sign bit set (and -0) becomes +0; positive values
// are unchanged.
__device__ __forceinline__ h8 relu_h8(h8 v)
{
    const s8 zero = {0, 0, 0, 0, 0, 0, 0, 0};
    return __builtin_bit_cast(h8, __builtin_elementwise_max(__builtin_bit_cast(s8, v), zero));
}

// tanh from its odd Taylor series near 0 (|x| < 1/16, where the next term
// is below 2^-28 relative) and from tanh|x| = (1 - e) / (1 + e),
// e = exp(-2|x|), elsewhere.
__device__ __forceinline__ float tanh_f32(float x)
{
    const float ax = __builtin_fabsf(x);
    const float x2 = x * x;
    const float series = x * (1.f + x2 * (-1.f / 3.f + x2 * (2.f / 15.f)));
    const float e = __expf(-2.f * ax);
    const float t = (1.f - e) * __builtin_amdgcn_rcpf(1.f + e);
    const float big = __builtin_copysignf(t, x);
    return ax < 0.0625f ? series : big;
}

// The epilogue's activation on NV values; act is uniform across the grid.
// Sigmoid is 1 / (1 + exp(-x)).
template <int NV>
__device__ __forceinline__ void activate(int act, float (&x)[NV])
{
    if (act == ACT_RELU) {
#pragma unroll
        for (int e = 0; e < NV; ++e) x[e] = x[e] > 0.f ? x[e] : 0.f;
    } else if (act == ACT_SIGMOID) {
#pragma unroll
        for (int e = 0; e < NV; ++e) x[e] = __builtin_amdgcn_rcpf(1.f + __expf(-x[e]));
    } else if (act == ACT_TANH) {
#pragma unroll
        for (int e = 0; e < NV; ++e) x[e] = tanh_f32(x[e]);
    }
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
