// gba_kernel.hpp -- the fast path of the fused fp16 GEMM + bias + activation
// for gfx950, used when every operand is 16-byte aligned, the leading
// dimensions are multiples of 8 and the contiguous extent of each operand is
// a multiple of 8 (so every 16-byte chunk is either wholly inside the matrix
// or wholly outside it).
//
// Structure (Matmul Compute Decomposition and Data Movement sections):
//   * A workgroup owns a BM x BN block tile of C, its WM x WN waves a
//     (BM/WM) x (BN/WN) warp tile each; the reduction runs in steps of
//     BK = 64 (strip-mining of the sequential dimension).
//   * Each step's A and B tiles go global -> registers -> LDS (the split copy
//     of the Global to Shared Memory subsection) through 16-byte buffer
//     loads; the next step's loads are in flight while the current step is
//     multiplied (Prefetching and Hiding Latency subsection) and LDS is
//     double-buffered, so one barrier per step suffices.
//   * The wave-level contraction is v_mfma_f32_32x32x16_f16: fp16 inputs,
//     fp32 accumulation, a 32x32 output block per instruction -- the CDNA4
//     counterpart of the paper's 32x32x8 macro-MMA.  A 16-deep slice of k is
//     one instruction per 32x32 block (the outer-product order of the
//     strip-mined warp MMA).
//   * After the last step the accumulators get the bias add, ReLU and fp16
//     conversion in registers, and each lane stores 16 contiguous outputs as
//     two 16-byte writes (Pointwise Operations in Epilogue subsection): the
//     matmul result never reaches global memory.
//
// Operand roles.  The MFMA "A" slot (rows = lane % 32) is fed with columns
// of B and the "B" slot (columns = lane % 32) with rows of A, so each
// instruction yields a block of C transposed: lane l's 16 accumulators are 16
// output columns of output row l % 32.  Inside each 32-column block the B
// columns are presented to the MFMA in the order jp32 so that those 16
// columns are consecutive -- the wide-store reordering that the paper does
// through shared memory, obtained here for free.
//
// LDS.  Both tiles are stored reduction-contiguous, one 128-byte row (64
// fp16 = 8 chunks of 16 bytes) per output row / column; chunk c of row r is
// kept at chunk position c ^ swz32(r) (Swizzled Shared Memory subsection).
// swz32 depends on r mod 32 only, so fragment addresses differ between
// blocks by constants, and it makes the fragment reads and the row-wise
// staging writes free of bank conflicts.
//
// Layouts.  A reduction-contiguous operand (row-major A, column-major B) is
// copied chunk by chunk.  For the other two cases a lane loads an 8 x 8
// block of fp16 as 8 chunks along M (or N), transposes it in registers and
// writes 8 reduction-contiguous chunks: the per-layout copy helpers.
//
// Edges.  Out-of-range chunks are fetched through a buffer resource with an
// offset beyond its size, which the hardware returns as zeros without a
// branch; out-of-range outputs are not stored.
#pragma once

#include "gba_common.hpp"

namespace gba {

// Raw (unswizzled, stride 0) buffer resource with range checking.
constexpr int RSRC_WORD3 = 0x00020000;
// Offset of a chunk that must read as zero: beyond every resource's size.
constexpr int OOB_OFFSET = (int)0x80000000u;
constexpr int MAX_RECORDS = 0x7fffffff;

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const _Float16 *base, int64_t bytes)
{
    int n = bytes > MAX_RECORDS ? MAX_RECORDS : (bytes < 0 ? 0 : (int)bytes);
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<_Float16 *>(base), (short)0, n, RSRC_WORD3);
}

__device__ __forceinline__ h8 buffer_load16(__amdgpu_buffer_rsrc_t r, int voff)
{
    return __builtin_bit_cast(h8, __builtin_amdgcn_raw_buffer_load_b128(r, voff, 0, 0));
}

// Chunk permutation of LDS row r (periodic in 32 rows).
__device__ __forceinline__ int swz32(int r)
{
    int b0 = ((r >> 2) ^ (r >> 4)) & 1;
    int b1 = (r ^ (r >> 2) ^ (r >> 3)) & 1;
    int b2 = (r >> 1) & 1;
    return b0 | (b1 << 1) | (b2 << 2);
}

// Column (inside a 32-column block of B) presented as MFMA row rho.  The
// MFMA returns row rho = 8*(r/4) + 4*(lane/32) + r%4 in accumulator r of a
// lane, which this maps to column 16*(lane/32) + r.
__device__ __forceinline__ int jp32(int rho) { return 16 * ((rho >> 2) & 1) + 4 * (rho >> 3) + (rho & 3); }

// One operand tile of R rows (output rows of A, or output columns of B) by
// 64 reduction indices: per-thread chunk offsets, staging registers, and the
// register -> LDS write.
//   KCONT: reduction-contiguous in global memory (row-major A, col-major B).
template <int R, int NT, bool KCONT>
struct FastStage {
    static constexpr int CHUNKS = R * 8;
    static constexpr int BLOCKS = R;  // 8 x 8 blocks when transposing
    static constexpr int PER = KCONT ? CHUNKS / NT : (BLOCKS + NT - 1) / NT;
    static constexpr int NREG = KCONT ? PER : PER * 8;
    static_assert(!KCONT || CHUNKS % NT == 0, "chunks must divide evenly among the threads");

    int voff[NREG];      // byte offset of each chunk from the tile origin (or OOB_OFFSET)
    int kchunk[KCONT ? PER : 1];  // reduction chunk index (KCONT tail masking)
    int lds_off[KCONT ? PER : PER * 8];  // LDS byte offset of each written chunk
    h8 v[NREG];

    __device__ __forceinline__ void init(int64_t ld, int r0, int rtot, int tid)
    {
        if constexpr (KCONT) {
#pragma unroll
            for (int p = 0; p < PER; ++p) {
                int idx = tid + p * NT;
                int r = idx >> 3, c = idx & 7;
                voff[p] = r0 + r < rtot ? (int)(((int64_t)r * ld + 8 * c) * 2) : OOB_OFFSET;
                kchunk[p] = c;
                lds_off[p] = (r * 8 + (c ^ swz32(r))) * 16;
            }
        } else {
#pragma unroll
            for (int p = 0; p < PER; ++p) {
                int idx = tid + p * NT;
                int rb = idx % (R / 8), kb = idx / (R / 8);
                bool live = idx < BLOCKS && r0 + 8 * rb < rtot;
#pragma unroll
                for (int q = 0; q < 8; ++q)
                    voff[p * 8 + q] = live ? (int)(((int64_t)(8 * kb + q) * ld + 8 * rb) * 2) : OOB_OFFSET;
#pragma unroll
                for (int rr = 0; rr < 8; ++rr) {
                    int r = 8 * rb + rr;
                    lds_off[p * 8 + rr] = idx < BLOCKS ? (r * 8 + (kb ^ swz32(r))) * 16 : -1;
                }
            }
        }
    }

    // Loads of a step whose 64 reduction indices are all below K.
    __device__ __forceinline__ void load(__amdgpu_buffer_rsrc_t rs)
    {
#pragma unroll
        for (int p = 0; p < NREG; ++p) v[p] = buffer_load16(rs, voff[p]);
    }

    // Loads of the last, partial step: reduction chunks at or beyond K read
    // as zeros (for the transposing layouts the resource size does that).
    __device__ __forceinline__ void load_tail(__amdgpu_buffer_rsrc_t rs, int kleft)
    {
        if constexpr (KCONT) {
#pragma unroll
            for (int p = 0; p < PER; ++p) v[p] = buffer_load16(rs, 8 * kchunk[p] < kleft ? voff[p] : OOB_OFFSET);
        } else {
            load(rs);
        }
    }

    __device__ __forceinline__ void store(char *lds) const
    {
        if constexpr (KCONT) {
#pragma unroll
            for (int p = 0; p < PER; ++p) *reinterpret_cast<h8 *>(lds + lds_off[p]) = v[p];
        } else {
#pragma unroll
            for (int p = 0; p < PER; ++p) {
                if (BLOCKS % NT == 0 || lds_off[p * 8] >= 0) {
#pragma unroll
                    for (int rr = 0; rr < 8; ++rr) {
                        h8 t;
#pragma unroll
                        for (int q = 0; q < 8; ++q) t[q] = v[p * 8 + q][rr];
                        *reinterpret_cast<h8 *>(lds + lds_off[p * 8 + rr]) = t;
                    }
                }
            }
        }
    }
};

template <int BM, int BN, int WM, int WN, int LA, int LB, bool ACC16>
__global__ void __launch_bounds__(64 * WM * WN) gemm_bias_act_fast(GemmArgs p)
{
    constexpr int NT = 64 * WM * WN;
    constexpr int BK = 64;
    constexpr int WTM = BM / WM, WTN = BN / WN;
    constexpr int TM = WTM / 32, TN = WTN / 32;
    constexpr int ROWB = BK * 2;              // bytes per LDS row
    constexpr int STAGE = (BM + BN) * ROWB;   // bytes per LDS stage
    static_assert(WTM % 32 == 0 && WTN % 32 == 0, "warp tile must be a multiple of 32x32");

    __shared__ __attribute__((aligned(16))) char lds[2 * STAGE];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int wm = wave % WM, wn = wave / WM;
    const int l32 = lane & 31, hi = lane >> 5;

    int tm, tn;
    tile_coords(blockIdx.x, gridDim.x, p.tiles_m, tm, tn);
    const int m0 = tm * BM, n0 = tn * BN;

    FastStage<BM, NT, LA == ROW> sa;
    FastStage<BN, NT, LB == COL> sb;
    sa.init(p.lda, m0, p.M, tid);
    sb.init(p.ldb, n0, p.N, tid);

    // Resource of the step starting at reduction index k0 for each operand.
    auto rsrc_a = [&](int k0) {
        if constexpr (LA == ROW) return make_rsrc(p.A + (int64_t)m0 * p.lda + k0, MAX_RECORDS);
        else return make_rsrc(p.A + (int64_t)k0 * p.lda + m0, (int64_t)(p.K - k0) * p.lda * 2);
    };
    auto rsrc_b = [&](int k0) {
        if constexpr (LB == COL) return make_rsrc(p.B + (int64_t)n0 * p.ldb + k0, MAX_RECORDS);
        else return make_rsrc(p.B + (int64_t)k0 * p.ldb + n0, (int64_t)(p.K - k0) * p.ldb * 2);
    };
    auto load_step = [&](int k0) {
        if (k0 + BK <= p.K) {
            sa.load(rsrc_a(k0));
            sb.load(rsrc_b(k0));
        } else {
            sa.load_tail(rsrc_a(k0), p.K - k0);
            sb.load_tail(rsrc_b(k0), p.K - k0);
        }
    };

    // Fragment byte offsets inside a stage for each 16-deep slice ks; blocks
    // further along differ by 32 rows = 4096 bytes.
    int offq[4], offp[4];
    {
        const int rq = wm * WTM + l32;
        const int rp = BM + wn * WTN + jp32(l32);
#pragma unroll
        for (int ks = 0; ks < 4; ++ks) {
            offq[ks] = rq * ROWB + (((2 * ks + hi) ^ swz32(l32)) * 16);
            offp[ks] = rp * ROWB + (((2 * ks + hi) ^ swz32(jp32(l32))) * 16);
        }
    }

    f16v acc[TN][TM];
#pragma unroll
    for (int t = 0; t < TN; ++t)
#pragma unroll
        for (int s = 0; s < TM; ++s)
#pragma unroll
            for (int e = 0; e < 16; ++e) acc[t][s][e] = 0.f;

    const int nk = (p.K + BK - 1) / BK;
    if (nk > 0) {
        load_step(0);
        sa.store(lds);
        sb.store(lds + BM * ROWB);
        __syncthreads();
    }

    for (int kt = 0; kt < nk; ++kt) {
        char *cur = lds + (kt & 1) * STAGE;
        char *nxt = lds + ((kt + 1) & 1) * STAGE;
        const bool more = kt + 1 < nk;
        if (more) load_step((kt + 1) * BK);
#pragma unroll
        for (int ks = 0; ks < 4; ++ks) {
            h8 fq[TM], fp[TN];
#pragma unroll
            for (int s = 0; s < TM; ++s) fq[s] = *reinterpret_cast<const h8 *>(cur + offq[ks] + s * 32 * ROWB);
#pragma unroll
            for (int t = 0; t < TN; ++t) fp[t] = *reinterpret_cast<const h8 *>(cur + offp[ks] + t * 32 * ROWB);
#pragma unroll
            for (int t = 0; t < TN; ++t)
#pragma unroll
                for (int s = 0; s < TM; ++s)
                    acc[t][s] = __builtin_amdgcn_mfma_f32_32x32x16_f16(fp[t], fq[s], acc[t][s], 0, 0, 0);
            if constexpr (ACC16) {
                if (ks & 1) {
                    // fp16 accumulation: round the running sum to fp16 at the
                    // end of every aligned 32-deep group of k.
#pragma unroll
                    for (int t = 0; t < TN; ++t)
#pragma unroll
                        for (int s = 0; s < TM; ++s)
#pragma unroll
                            for (int e = 0; e < 16; ++e) acc[t][s][e] = (float)(_Float16)acc[t][s][e];
                }
            }
        }
        if (more) {
            sa.store(nxt);
            sb.store(nxt + BM * ROWB);
        }
        __syncthreads();
    }

    // Epilogue on registers: + bias, ReLU, fp16, two 16-byte stores per lane
    // per 32x32 block.
#pragma unroll
    for (int t = 0; t < TN; ++t) {
        const int j = n0 + wn * WTN + 32 * t + 16 * hi;
        float b[16];
#pragma unroll
        for (int e = 0; e < 16; ++e) b[e] = 0.f;
        if (p.bias != nullptr && j < p.N) {
            h8 b0 = *reinterpret_cast<const h8 *>(p.bias + j);
            h8 b1 = j + 8 < p.N ? *reinterpret_cast<const h8 *>(p.bias + j + 8) : zero_h8();
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                b[e] = (float)b0[e];
                b[8 + e] = (float)b1[e];
            }
        }
#pragma unroll
        for (int s = 0; s < TM; ++s) {
            const int i = m0 + wm * WTM + 32 * s + l32;
            h8 o0, o1;
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                float x0 = acc[t][s][e] + b[e];
                float x1 = acc[t][s][8 + e] + b[8 + e];
                if (p.relu) {
                    x0 = x0 > 0.f ? x0 : 0.f;
                    x1 = x1 > 0.f ? x1 : 0.f;
                }
                o0[e] = (_Float16)x0;
                o1[e] = (_Float16)x1;
            }
            if (i < p.M && j < p.N) {
                _Float16 *dst = p.C + (int64_t)i * p.ldc + j;
                *reinterpret_cast<h8 *>(dst) = o0;
                if (j + 8 < p.N) *reinterpret_cast<h8 *>(dst + 8) = o1;
            }
        }
    }
}

}  // namespace gba
