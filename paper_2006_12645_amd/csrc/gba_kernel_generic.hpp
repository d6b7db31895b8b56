// gba_kernel_generic.hpp -- the general-case fused fp16 GEMM + bias +
// activation kernel for gfx950: any size, leading dimension and (2-byte)
// alignment.  The 16-byte aligned fast path is in gba_kernel.hpp.
//
// One workgroup computes one BM x BN tile of C (block tile, Tiling for Blocks
// and Warps subsection); its waves each own a WTM x WTN sub-tile (warp tile).
// The reduction dimension is walked in steps of BK = 64 (strip-mining of the
// sequential dimension), staged global -> registers -> LDS (Global to Shared
// Memory subsection) with the next step's global loads in flight while the
// current step is multiplied (Prefetching and Hiding Latency subsection).
// Each 32-deep slice of a step is one wave-wide v_mfma_f32_16x16x32_f16 per
// 16x16 output block: the CDNA4 matrix instruction plays the role of the
// paper's composed macro-MMA.  After the last step the bias add, ReLU and
// fp16 conversion run on the accumulator registers and each lane stores 8
// contiguous fp16 values (Pointwise Operations in Epilogue subsection): the
// matmul result never reaches global memory.
//
// Operand roles.  The MFMA "A" slot (rows indexed by lane % 16) is fed with
// columns of B, the "B" slot (columns indexed by lane % 16) with rows of A,
// so the instruction produces a block of C transposed: lane l holds four
// consecutive output COLUMNS of one output row.  A permutation of the B
// columns inside each 32-column pair of blocks (jperm below) makes those two
// groups of four adjacent, so every lane owns 8 contiguous fp16 outputs and
// stores them with one 16-byte write -- the role the paper gives to its
// reordering through shared memory, done here without any shared memory.
//
// LDS layout.  Both operand tiles are stored reduction-contiguous: a row of
// 64 fp16 (128 bytes = 8 chunks of 16 bytes) per output row or column, and
// chunk c of row r lives at chunk position c ^ swz16(r).  swz is a bijection on
// chunks per row chosen so that (a) 8 lanes writing one row, (b) lanes
// writing the same chunk of 8-row-strided rows (transposed staging), (c)
// 16 consecutive rows read at one chunk, and (d) the jperm-ordered reads of
// the B tile all touch distinct banks (Swizzled Shared Memory subsection).
//
// Layouts.  When an operand is stored reduction-contiguous in global memory
// (row-major A, column-major B) a lane copies 16-byte chunks straight through.
// Otherwise (column-major A, row-major B) a lane loads an 8 x 8 block as 8
// row chunks, transposes it in registers and writes 8 reduction-contiguous
// chunks: the four per-layout copy helpers of the Global to Shared Memory
// subsection.
//
// Edges.  Rows/columns beyond M or N and reduction indices beyond K are
// loaded as zeros and out-of-range outputs are not stored, so any size is
// handled in the kernel (the partial-tile case of the Tiling subsection).
#pragma once

#include "gba_common.hpp"

namespace gba {

// Bijective chunk permutation per LDS row (see header comment).
__device__ __forceinline__ int swz16(int r)
{
    int b0 = ((r >> 2) ^ (r >> 3)) & 1;
    int b1 = (r ^ (r >> 1) ^ (r >> 4)) & 1;
    int b2 = ((r >> 1) ^ (r >> 3) ^ (r >> 5)) & 1;
    return b0 | (b1 << 1) | (b2 << 2);
}

// Position of MFMA row rho of block t inside a wave's run of B columns: two
// neighbouring blocks share 32 columns so that a lane's 2 x 4 results are 8
// consecutive columns.
__device__ __forceinline__ int jperm(int t, int rho)
{
    return 32 * (t >> 1) + 8 * (rho >> 2) + 4 * (t & 1) + (rho & 3);
}

// Eight fp16 at any 2-byte alignment: gfx950 (with the unaligned access
// mode of its HSA runtime) serves a misaligned 16-byte load or store as one
// instruction, so these compile to single dwordx4 accesses.
typedef _Float16 h8u __attribute__((ext_vector_type(8), aligned(2)));

// Eight consecutive fp16 from p[0..7], the ones at index >= lim read as 0.
__device__ __forceinline__ h8 load8(const _Float16 *p, int lim)
{
    if (lim >= 8) return *reinterpret_cast<const h8u *>(p);
    h8 v;
#pragma unroll
    for (int e = 0; e < 8; ++e) v[e] = e < lim ? p[e] : (_Float16)0.0f;
    return v;
}

// Global -> register -> LDS copy of one operand tile of R rows (output rows
// for A, output columns for B) by BK reduction indices.
//   KCONT: the operand is reduction-contiguous in global memory.
//   RELU: the prologue's ReLU is applied to the values on their way from
//         the registers to LDS (Pointwise Operations in Prologue subsection).
// X points at the operand, ld is its leading dimension, r0/k0 the tile origin,
// rtot/ktot the extents.
template <int R, int BK, int NT, bool KCONT, bool RELU>
struct TileCopy16 {
    static constexpr int CHUNKS = R * BK / 8;                 // 16-byte chunks per tile
    static constexpr int KCH = BK / 8;                        // chunks per LDS row
    static constexpr int PER = KCONT ? (CHUNKS + NT - 1) / NT // chunks per thread
                                     : (CHUNKS / 8 + NT - 1) / NT;  // 8x8 blocks per thread
    static constexpr int NREG = KCONT ? PER : PER * 8;
    h8 v[NREG];

    __device__ __forceinline__ void load(const _Float16 *X, int64_t ld, int r0, int k0, int rtot,
                                         int ktot, int tid)
    {
        if constexpr (KCONT) {
#pragma unroll
            for (int p = 0; p < PER; ++p) {
                int idx = tid + p * NT;
                int r = idx / KCH, c = idx % KCH;
                int gr = r0 + r, gk = k0 + 8 * c;
                h8 x = zero_h8();
                if ((CHUNKS % NT == 0 || idx < CHUNKS) && gr < rtot && gk < ktot)
                    x = load8(X + (int64_t)gr * ld + gk, ktot - gk);
                v[p] = x;
            }
        } else {
            constexpr int RB = R / 8;
#pragma unroll
            for (int p = 0; p < PER; ++p) {
                int idx = tid + p * NT;
                int rb = idx % RB, kb = idx / RB;
                int gr = r0 + 8 * rb, gk0 = k0 + 8 * kb;
                bool live = (CHUNKS / 8) % NT == 0 || idx < CHUNKS / 8;
#pragma unroll
                for (int q = 0; q < 8; ++q) {
                    h8 x = zero_h8();
                    if (live && gk0 + q < ktot && gr < rtot)
                        x = load8(X + (int64_t)(gk0 + q) * ld + gr, rtot - gr);
                    v[p * 8 + q] = x;
                }
            }
        }
    }

    __device__ __forceinline__ void store(h8 *lds, int tid)
    {
        if constexpr (RELU) {
#pragma unroll
            for (int i = 0; i < NREG; ++i) v[i] = relu_h8(v[i]);
        }
        if constexpr (KCONT) {
#pragma unroll
            for (int p = 0; p < PER; ++p) {
                int idx = tid + p * NT;
                if (CHUNKS % NT == 0 || idx < CHUNKS) {
                    int r = idx / KCH, c = idx % KCH;
                    lds[r * KCH + (c ^ swz16(r))] = v[p];
                }
            }
        } else {
            constexpr int RB = R / 8;
#pragma unroll
            for (int p = 0; p < PER; ++p) {
                int idx = tid + p * NT;
                if ((CHUNKS / 8) % NT == 0 || idx < CHUNKS / 8) {
                    int rb = idx % RB, kb = idx / RB;
#pragma unroll
                    for (int rr = 0; rr < 8; ++rr) {
                        h8 t;
#pragma unroll
                        for (int q = 0; q < 8; ++q) t[q] = v[p * 8 + q][rr];
                        int r = 8 * rb + rr;
                        lds[r * KCH + (kb ^ swz16(r))] = t;
                    }
                }
            }
        }
    }
};

// PRO: ReLU prologue on the left operand of every product.  DUAL: a second
// product P.Q is accumulated into the same registers after A.B (Matmuls
// with Pointwise Epilogue subsection); C - R is formed as -((-C) + R).
template <int BM, int BN, int WM, int WN, int LA, int LB, bool ACC16, bool PRO, bool DUAL>
__global__ void __launch_bounds__(64 * WM * WN) gemm_bias_act_generic(GemmArgs p)
{
    constexpr int NT = 64 * WM * WN;
    constexpr int BK = 64;
    constexpr int KCH = BK / 8;
    constexpr int WTM = BM / WM, WTN = BN / WN;
    constexpr int TM = WTM / 16, TN = WTN / 16;
    static_assert(WTM % 16 == 0 && WTN % 32 == 0, "wave tile: 16-row, 32-column multiples");

    // Two stages of [A tile | B tile], in 16-byte chunks.
    __shared__ h8 lds[2][(BM + BN) * KCH];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int wm = wave % WM, wn = wave / WM;

    int tm, tn;
    tile_coords(blockIdx.x, gridDim.x, p.tiles_m, tm, tn);
    const int m0 = tm * BM, n0 = tn * BN;

    TileCopy16<BM, BK, NT, LA == ROW, PRO> ca;
    TileCopy16<BN, BK, NT, LB == COL, false> cb;

    f4 acc[TN][TM];
#pragma unroll
    for (int t = 0; t < TN; ++t)
#pragma unroll
        for (int s = 0; s < TM; ++s) acc[t][s] = f4{0.f, 0.f, 0.f, 0.f};
    auto negate_acc = [&]() {
#pragma unroll
        for (int t = 0; t < TN; ++t)
#pragma unroll
            for (int s = 0; s < TM; ++s) acc[t][s] = -acc[t][s];
    };

    // LDS read offsets (in chunks) of this lane's fragments, before the
    // k-chunk swizzle: row index and its swizzle value.
    const int kq = lane >> 4;  // which 8-wide k group of a 32-deep slice
    int rowA[TM], swA[TM], rowB[TN], swB[TN];
#pragma unroll
    for (int s = 0; s < TM; ++s) {
        int r = wm * WTM + 16 * s + (lane & 15);
        rowA[s] = r * KCH;
        swA[s] = swz16(r);
    }
#pragma unroll
    for (int t = 0; t < TN; ++t) {
        int r = wn * WTN + jperm(t, lane & 15);
        rowB[t] = (BM + r) * KCH;
        swB[t] = swz16(r);
    }

#pragma unroll 1
    for (int seg = 0; seg < (DUAL ? 2 : 1); ++seg) {
        const _Float16 *const X = seg == 0 ? p.A : p.P;
        const _Float16 *const Y = seg == 0 ? p.B : p.Q;
        const int64_t ldx = seg == 0 ? p.lda : p.ldp;
        const int64_t ldy = seg == 0 ? p.ldb : p.ldq;
        const int Kseg = seg == 0 ? p.K : p.K2;
        // (the last step of the previous pass ended with a barrier, so LDS
        // is free to refill)
        if (seg == 1 && p.sub) negate_acc();

        const int nk = (Kseg + BK - 1) / BK;
        if (nk > 0) {
            ca.load(X, ldx, m0, 0, p.M, Kseg, tid);
            cb.load(Y, ldy, n0, 0, p.N, Kseg, tid);
            ca.store(&lds[0][0], tid);
            cb.store(&lds[0][BM * KCH], tid);
            __syncthreads();
        }

        for (int kt = 0; kt < nk; ++kt) {
            const int cur = kt & 1;
            const bool more = kt + 1 < nk;
            if (more) {
                ca.load(X, ldx, m0, (kt + 1) * BK, p.M, Kseg, tid);
                cb.load(Y, ldy, n0, (kt + 1) * BK, p.N, Kseg, tid);
            }
            const h8 *L = &lds[cur][0];
#pragma unroll
            for (int ks = 0; ks < BK / 32; ++ks) {
                const int c = ks * 4 + kq;
                h8 fa[TM], fb[TN];
#pragma unroll
                for (int s = 0; s < TM; ++s) fa[s] = L[rowA[s] + (c ^ swA[s])];
#pragma unroll
                for (int t = 0; t < TN; ++t) fb[t] = L[rowB[t] + (c ^ swB[t])];
#pragma unroll
                for (int t = 0; t < TN; ++t)
#pragma unroll
                    for (int s = 0; s < TM; ++s)
                        acc[t][s] = __builtin_amdgcn_mfma_f32_16x16x32_f16(fb[t], fa[s], acc[t][s], 0, 0, 0);
                if constexpr (ACC16) {
                    // fp16 accumulation: the running sum is rounded to fp16 at
                    // the end of every aligned 32-deep group of k.
#pragma unroll
                    for (int t = 0; t < TN; ++t)
#pragma unroll
                        for (int s = 0; s < TM; ++s)
#pragma unroll
                            for (int e = 0; e < 4; e += 2) {
                                const f2v r = round_f16x2(f2v{acc[t][s][e], acc[t][s][e + 1]});
                                acc[t][s][e] = r[0];
                                acc[t][s][e + 1] = r[1];
                            }
                }
            }
            if (more) {
                ca.store(&lds[cur ^ 1][0], tid);
                cb.store(&lds[cur ^ 1][BM * KCH], tid);
            }
            __syncthreads();
        }
        if (seg == 1 && p.sub) negate_acc();
    }

    // Epilogue on registers: +/- bias, activation, fp16, one 16-byte store
    // per lane per pair of MFMA blocks.
#pragma unroll
    for (int pr = 0; pr < TN / 2; ++pr) {
        const int j = n0 + wn * WTN + 32 * pr + 8 * kq;
        float b[8];
        if (p.bias_kind == BIAS_ROW) {
            h8 bv = zero_h8();
            if (j < p.N) bv = load8(p.bias + j, p.N - j);
#pragma unroll
            for (int e = 0; e < 8; ++e) b[e] = p.bias_sign * (float)bv[e];
        } else {
#pragma unroll
            for (int e = 0; e < 8; ++e) b[e] = 0.f;
        }
#pragma unroll
        for (int s = 0; s < TM; ++s) {
            const int i = m0 + wm * WTM + 16 * s + (lane & 15);
            float x[8];
#pragma unroll
            for (int e = 0; e < 8; ++e) x[e] = (e < 4 ? acc[2 * pr][s][e] : acc[2 * pr + 1][s][e - 4]) + b[e];
            if (p.bias_kind == BIAS_FULL) {
                h8 bv = zero_h8();
                if (i < p.M && j < p.N) bv = load8(p.bias + (int64_t)i * p.ldbias + j, p.N - j);
#pragma unroll
                for (int e = 0; e < 8; ++e) x[e] += p.bias_sign * (float)bv[e];
            }
            activate(p.act, x);
            h8 o;
#pragma unroll
            for (int e = 0; e < 8; ++e) o[e] = (_Float16)x[e];
            if (i < p.M && j < p.N) {
                _Float16 *dst = p.C + (int64_t)i * p.ldc + j;
                if (j + 8 <= p.N) {
                    *reinterpret_cast<h8u *>(dst) = o;
                } else {
#pragma unroll
                    for (int e = 0; e < 8; ++e)
                        if (j + e < p.N) dst[e] = o[e];
                }
            }
        }
    }
}

}  // namespace gba
