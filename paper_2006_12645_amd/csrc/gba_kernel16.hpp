// gba_kernel16.hpp -- the fast path on v_mfma_f32_16x16x32_f16 (the 8-wave
// tiles, every operand layout; and the four-stage small tiles without the
// prologue: all of them when both operand tiles are reduction-contiguous,
// the 32x128 one with row-major B and the 128x32 one with column-major A,
// whose M- or N-contiguous operand tile has 128 elements per row).
//
// Same decomposition as gemm_bias_act_fast (block tile per workgroup, warp
// tiles per wave, 64-deep reduction steps through direct global -> LDS
// copies over NSTG stages, one barrier per step, epilogue in registers), with
// the wave-level contraction on 16x16 output blocks, 32 deep per
// instruction.  For the same work the 16x16x32 instruction reads and writes
// a quarter of the accumulator registers that 32x32x16 does per instruction
// (half per flop), and under the part's power limit this runs the MFMA pipes
// at a markedly higher clock (measured on a GEMM-shaped loop with LDS
// fragment reads: 1.70 against 1.44-1.52 PFLOP/s).
//
// Operand roles and store order.  As in the 32x32 path the MFMA "A" slot
// takes columns of B and the "B" slot rows of A, so lane l holds, for every
// 16x16 block, output row l % 16 and the four output columns presented as
// MFMA rows 4*(l/16) .. 4*(l/16)+3.  The B columns are presented in the
// order perm16: within each group of G blocks (16G columns), block t's MFMA
// row rho is column 4G*(rho/4) + 4*(t%G) + rho%4, so across the group's G
// blocks a lane holds 4G consecutive outputs of its row (16 for G = 4: two
// 16-byte stores).  An operand contiguous along N (row-major B) instead
// uses G = 1, the natural column order: its transposing fragment reads then
// touch 16 consecutive columns per row, which fT16 keeps free of bank
// conflicts (the grouped order would put four 8-byte reads of a row into
// four groups and conflict), and each lane stores 4 consecutive outputs.
//
// Layouts.  As in the 32x32 path each tile keeps its global layout in LDS:
// reduction-contiguous operands as 128-byte rows (chunk permutations swzA16
// / swzB16), M- or N-contiguous ones as 64 reduction rows whose 16-element
// groups are permuted by fT16 of the row, read with ds_read_b64_tr_b16 pairs
// (lanes 4j+c of a 16-lane group address row j at the 4-element chunk that
// result lanes 4c..4c+3 need, so each lane receives 8 consecutive k of one
// row or column, the same k slots as the 16-byte reads).
//
// Slices.  A 64-deep step is two 32-deep halves; each half is split into two
// slices over the A blocks of the warp tile (TM/2 each), so a step has four
// slices like the 32x32 path.  The A fragments of the next slice are read
// during the current one; the B fragments of a half are read during the
// slice before it (and used by both of its slices).
#pragma once

#include "gba_kernel.hpp"

namespace gba {

// Column (inside a warp tile's B columns) presented as MFMA row rho of
// 16-column block t, with G blocks per group of consecutive outputs.
template <int G>
__device__ __forceinline__ int perm16(int t, int rho)
{
    return 16 * G * (t / G) + 4 * G * (rho >> 2) + 4 * (t % G) + (rho & 3);
}

// Waves that only issue copies, added to the workgroups of the small tiles
// (one, two or four computing waves, latency-bound: with the copies on the
// computing waves each 64-deep step waits for their issue).  Four of them,
// with fp16 accumulation: 32 x 4096 x 1024 on the 32x32 tile 9.2 -> 6.8 us,
// 1024 x 1024 x 4096 on the 64x64 tile 28.2 -> 21.7 us (one or two gave
// less).  Not with the prologue, whose left tile is staged through the
// computing waves' registers.
template <int WM, int WN, int SK, bool ACC16, bool PRO, bool SPLIT>
constexpr int copy_only_waves()
{
    return (WM * WN < 8 && SK == 1 && !PRO && !SPLIT) ? 4 : 0;
}

template <int BM, int BN, int WM, int WN, int SK, int NSTG, int LA, int LB, bool ACC16, bool PRO, bool DUAL,
          bool SPLIT>
__global__ void __launch_bounds__(64 * (WM * WN * SK + copy_only_waves<WM, WN, SK, ACC16, PRO, SPLIT>()))
gemm_bias_act_fast16(GemmArgs p)
{
    constexpr int NTG = 64 * WM * WN;         // threads per k-group
    constexpr int NT = NTG * SK;              // threads that compute
    constexpr int NPW = copy_only_waves<WM, WN, SK, ACC16, PRO, SPLIT>();
    constexpr int BK = 64;
    constexpr int WTM = BM / WM, WTN = BN / WN;
    constexpr int TM = WTM / 16, TN = WTN / 16;   // 16x16 blocks of the warp tile
    constexpr int TMH = TM / 2;                    // A blocks per slice
    // Operands contiguous along the reduction use DmaCopy and 16-byte
    // fragment reads, the others (TA / TB) DmaCopyT and transposing reads.
    constexpr bool TA = LA == COL, TB = LB == ROW;
    constexpr int G = TB ? 1 : (TN < 4 ? TN : 4);  // B blocks per group of consecutive outputs
    constexpr int ROWB = BK * 2;                   // bytes per LDS row
    constexpr int SUB = (BM + BN) * ROWB;          // bytes per k-group sub-stage
    constexpr int STAGE = SK * SUB;                // bytes per LDS stage
    constexpr int NS = NSTG;
    static_assert((NS & (NS - 1)) == 0, "stage count must be a power of two");
    static_assert(WTM % 32 == 0 && WTN % 32 == 0, "warp tile must be a multiple of 32x32");
    static_assert(TN % G == 0 && (TB || G >= 2), "B blocks come in groups of two or four");
    static_assert(!(ACC16 && SK > 1), "fp16 accumulation is defined for a single running sum");
    static_assert(!SPLIT || (SK == 1 && !ACC16), "a split reduction needs one k-group and fp32 sums");
    constexpr int PADN = BN + 4;               // fp32 row pitch of the split-K partial tiles
    constexpr int RED = SK > 1 ? SK * BM * PADN * 4 : 0;
    constexpr int LDS_BYTES = NS * STAGE > RED ? NS * STAGE : RED;

    __shared__ __attribute__((aligned(16))) char lds[LDS_BYTES];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int grp = SK == 1 ? 0 : wave / (WM * WN);   // k-group
    const int gtid = tid - grp * NTG;         // thread index inside the k-group
    const int wm = (wave % (WM * WN)) % WM, wn = (wave % (WM * WN)) / WM;
    const int l16 = lane & 15, g4 = lane >> 4;

    int tile_id = blockIdx.x, kspl = 0;
    if constexpr (SPLIT) {
        tile_id = __builtin_amdgcn_readfirstlane((int)blockIdx.x / p.splits);
        kspl = __builtin_amdgcn_readfirstlane((int)blockIdx.x - tile_id * p.splits);
    }
    int tm, tn;
    tile_coords(tile_id, SPLIT ? p.tiles_m * p.tiles_n : (int)gridDim.x, p.tiles_m, tm, tn);
    const int m0 = tm * BM, n0 = tn * BN;
    const int mc = m0 + BM <= p.M ? m0 : p.M - BM;
    const int nc = n0 + BN <= p.N ? n0 : p.N - BN;

    // Which waves issue the copies.  Two waves share each SIMD; the hardware
    // issues from the older one whenever it can, so waves 0-3 run ahead and
    // wait at the step's barrier while waves 4-7 finish alone.  A direct
    // copy instruction holds its wave's issue for tens of cycles, so on the
    // one-product, single-k-group tiles the leading waves issue all of a
    // step's copies and the trailing ones only read fragments and multiply
    // (4096^3: 2853 -> 2688 cycles per step, measured with s_memtime; the
    // leading waves' wait at the barrier 1096 -> 442 cycles).  The 256x128
    // and 128x256 tiles were 1.5-3% slower that way and keep all eight
    // waves copying.  So do the two-product kernels (the 128x128 one grows
    // from 87 to 137 VGPRs, one workgroup per compute unit instead of two)
    // and the 256x256 tile with fp16 accumulation (its loops spill).
    // The prologue ReLU either on the A fragments as they are read (the left
    // tile then comes in by direct copies, and the copy split below applies)
    // or on the left tile staged through registers (where the tile is
    // written into LDS).  On the fragments each of the WN waves that read an
    // A block rectifies it again (one packed integer max per dword), which
    // measured: 4096^3 RC 109.5 -> 107.1 us (the kernel without prologue
    // 107.0), RR 117.5 -> 112.1, 8192x4096x1024 69.7 -> 67.1; the 8-wave
    // 128x64 / 64x128 tiles 7-9% faster; slower with column-major A (its
    // transposing fragment reads; 1.5-2%) and on the 128x128 tile (5-15%),
    // which keep the staged tile.
    constexpr bool PROF = PRO && LA == ROW && WM * WN == 8 && (BM * BN == 256 * 256 || BM * BN == 128 * 64);
    constexpr bool PROS = PRO && !PROF;            // register-staged left tile
    constexpr bool CH = !PROS && !DUAL && !SPLIT && SK == 1 && WM * WN == 8 && BM * BN != 256 * 128 &&
                        !(ACC16 && BM * BN > 128 * 128);
    constexpr int NTC = NPW ? 64 * NPW : CH ? NTG / 2 : NTG;   // threads that issue the copies
    using CopyA = std::conditional_t<TA, DmaCopyT<BM, NTC, 1>, DmaCopy<BM, NTC, 1>>;
    using CopyB = std::conditional_t<TB, DmaCopyT<BN, NTC, 1>, DmaCopy<BN, NTC, 2>>;
    const int rwave = __builtin_amdgcn_readfirstlane(wave);
    const bool copy_wave = NPW ? rwave >= WM * WN : (!CH || rwave < WM * WN / 2);
    const int ctid = NPW ? tid - NT : CH ? (gtid & (NTC - 1)) : gtid;   // thread index among the copiers
    CopyA ca;
    CopyB cb;

    // Fragment byte offsets inside a stage, per 32-deep half h: A block s is
    // 16 rows (2048 bytes) after block 0 (swzA16 has period 16); each B
    // block has its own rows.
    int offa[TA ? TM : 2], offb[TB ? 1 : 2][TN];
    {
        // transposing reads: lane 4j + c of group g4 addresses reduction row
        // 8*g4 + j (+ 32 per half, + 4 for the second read of a pair) at the
        // 4-element chunk 4c of the block's 16 elements
        const int kr = 8 * g4 + (l16 >> 2), c4 = 4 * (l16 & 3);
        if constexpr (TA) {
#pragma unroll
            for (int s = 0; s < TM; ++s)
                offa[s] = kr * (2 * BM) + 32 * (((wm * WTM) / 16 + s) ^ fT16(kr)) + 2 * c4;
        } else {
            const int ra = wm * WTM + l16;
#pragma unroll
            for (int h = 0; h < 2; ++h) offa[h] = ra * ROWB + (((4 * h + g4) ^ swzA16(l16)) * 16);
        }
#pragma unroll
        for (int t = 0; t < TN; ++t) {
            if constexpr (TB) {
                offb[0][t] = BM * ROWB + kr * (2 * BN) + 32 * (((wn * WTN) / 16 + t) ^ fT16(kr)) + 2 * c4;
            } else {
                const int rb = wn * WTN + perm16<G>(t, l16);
#pragma unroll
                for (int h = 0; h < 2; ++h)
                    offb[h][t] = (BM + rb) * ROWB + (((4 * h + g4) ^ swzB16(rb)) * 16);
            }
        }
    }

    f4 acc[TN][TM];
#pragma unroll
    for (int t = 0; t < TN; ++t)
#pragma unroll
        for (int s = 0; s < TM; ++s) acc[t][s] = f4{0.f, 0.f, 0.f, 0.f};

    // fp16 accumulation on tiles with at most one wave per SIMD: the running
    // sum is kept as fp16 (s16) and each MFMA computes its 32-deep group's
    // sum from zero, which is then added to the running sum with one fp32
    // add and one rounding to fp16 (v_fma_mix: the fp16 operand is widened
    // inside the instruction).  The MFMAs then no longer wait for the
    // previous group's rounding -- only the adds form a chain -- which is
    // what bounds the small memory-bound tiles; with two waves per SIMD the
    // other wave already hides that chain, and the extra hazard waits of
    // this form cost more than it saves.  Same result class as rounding the
    // fp32 accumulator in place: the fp32 sum of S and the group is rounded
    // once to fp16 (here the group's own sum is rounded to fp32 first).
    constexpr bool FOLD = ACC16 && WM * WN < 8;
    h4 s16[FOLD ? TN : 1][FOLD ? TM : 1];
    float one = 1.f;
    if constexpr (FOLD) {
        // an opaque 1.0 keeps fma(s, 1, g) an fma, which selects v_fma_mix
        // (with a literal 1.0 it is folded to a widening and an add)
        asm("v_mov_b32 %0, 1.0" : "=v"(one));
#pragma unroll
        for (int t = 0; t < TN; ++t)
#pragma unroll
            for (int s = 0; s < TM; ++s) s16[t][s] = h4{0, 0, 0, 0};
    }
    auto fold = [&](h4 sv, f4 g) {
        const h2v lo = {(_Float16)__builtin_fmaf((float)sv[0], one, g[0]),
                        (_Float16)__builtin_fmaf((float)sv[1], one, g[1])};
        const h2v hi = {(_Float16)__builtin_fmaf((float)sv[2], one, g[2]),
                        (_Float16)__builtin_fmaf((float)sv[3], one, g[3])};
        return __builtin_shufflevector(lo, hi, 0, 1, 2, 3);
    };

    // A fragments of two slices, B fragments of two halves.
    h8 fa[2][TMH], fb[2][TN];
    auto read_a = [&](int buf, const char *stage, int h, int q) {
#pragma unroll
        for (int s = 0; s < TMH; ++s) {
            if constexpr (TA) fa[buf][s] = read_frag_tr<BM>(stage + offa[q * TMH + s] + h * 32 * (2 * BM));
            else fa[buf][s] = *reinterpret_cast<const h8 *>(stage + offa[h] + (q * TMH + s) * 16 * ROWB);
            if constexpr (PROF) fa[buf][s] = relu_h8(fa[buf][s]);
        }
    };
    auto read_b = [&](int buf, const char *stage, int h) {
#pragma unroll
        for (int t = 0; t < TN; ++t) {
            if constexpr (TB) fb[buf][t] = read_frag_tr<BN>(stage + offb[0][t] + h * 32 * (2 * BN));
            else fb[buf][t] = *reinterpret_cast<const h8 *>(stage + offb[h][t]);
        }
    };
    // The slice's MFMAs: A blocks q*TMH .. q*TMH+TMH-1 of half `bbuf`.
    auto mfmas = [&](int abuf, int bbuf, int q) {
#pragma unroll
        for (int t = 0; t < TN; ++t)
#pragma unroll
            for (int s = 0; s < TMH; ++s) {
                if constexpr (FOLD) {
                    const f4 g = __builtin_amdgcn_mfma_f32_16x16x32_f16(fb[bbuf][t], fa[abuf][s],
                                                                        f4{0.f, 0.f, 0.f, 0.f}, 0, 0, 0);
                    s16[t][q * TMH + s] = fold(s16[t][q * TMH + s], g);
                } else {
                    acc[t][q * TMH + s] = __builtin_amdgcn_mfma_f32_16x16x32_f16(fb[bbuf][t], fa[abuf][s],
                                                                                 acc[t][q * TMH + s], 0, 0, 0);
                }
            }
    };
    auto round16 = [&]() {
        // fp16 accumulation: the running sum is rounded to fp16 at the end of
        // every aligned 32-deep group of k (after both slices of a half)
        if constexpr (ACC16 && !FOLD) {
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
    };
    auto negate_acc = [&]() {
#pragma unroll
        for (int t = 0; t < TN; ++t)
#pragma unroll
            for (int s = 0; s < TM; ++s) {
                if constexpr (FOLD) s16[t][s] = -s16[t][s];
                else acc[t][s] = -acc[t][s];
            }
    };

    constexpr int NM = TN * TMH;              // MFMAs per slice
    // fragment reads (DS instructions) of slices 0, 2 and of slices 1, 3
    constexpr int NRA = TMH * (TA ? 2 : 1), NRB = NRA + TN * (TB ? 2 : 1);
    constexpr int NL = CopyA::NLOAD + CopyB::NLOAD;
    // Loads still allowed in flight at a step's barrier: the copies of the
    // steps after the next one, and (prologue) the left tile of step kt+2,
    // whose register loads are issued just before the barrier.
    constexpr int VM_AT_BARRIER = (NS - 2) * NL + (PROS ? CopyA::NLOAD : 0);
    // Tiles that put two workgroups on a compute unit (by their LDS) raise
    // their waves' priority over the first three slices of a step (the
    // MFMA-only stretch), so a workgroup there is not held back by the
    // copies and barrier of the other: 2-5% on the 8-wave 128x128 tile; it
    // made the 256x256 tile (one workgroup per compute unit) 1-2% slower and
    // the 128x64 one (three) no faster, which do not use it.
    constexpr bool PRIO = NS * STAGE <= 80 * 1024 && NS * STAGE > 160 * 1024 / 3;
    char *const mine = lds + grp * SUB;

    // Prologue ReLU (Pointwise Operations in Prologue subsection), on the
    // tiles that do not rectify their A fragments (PROF) applied where the
    // paper applies it: the left operand's tile goes from global memory
    // into registers, through one packed max per dword, and into LDS, so
    // each element is rectified once (not once per wave that reads it).
    // The registers carry the next step's left tile across the step
    // boundary: written to LDS in the third slice of a step, then loaded
    // with the tile of the step after next right away, so the loads have a
    // whole step to land before they are written in turn.
    static_assert(!PROS || NS == 2, "the register-staged prologue assumes two LDS stages");
    i4 ra[PROS ? CopyA::NLOAD : 1];
    auto relu_store_a = [&](char *stage) {
        if constexpr (PROS) {
#pragma unroll
            for (int i = 0; i < CopyA::NLOAD; ++i)
                ra[i] = __builtin_bit_cast(i4, relu_h8(__builtin_bit_cast(h8, ra[i])));
            ca.store(stage, ra);
        }
    };

    // The row bias of this lane's output columns (4G consecutive per group
    // of G blocks), loaded before the reduction.
    constexpr int NGRP = TN / G;
    constexpr int NV = G >= 2 ? G / 2 : 1;    // 8-element chunks per group (G = 1: one 4-element chunk)
    h8 brow[SK == 1 ? NGRP : 1][NV];
    if constexpr (SK == 1) {
        if (p.bias_kind == BIAS_ROW) {
#pragma unroll
            for (int tg = 0; tg < NGRP; ++tg) {
                const _Float16 *bp = p.bias + nc + wn * WTN + 16 * G * tg + 4 * G * g4;
#pragma unroll
                for (int v = 0; v < NV; ++v) {
                    if constexpr (G >= 2) brow[tg][v] = *reinterpret_cast<const h8 *>(bp + 8 * v);
                    else {
                        const h4 b4 = *reinterpret_cast<const h4 *>(bp);
                        brow[tg][v] = h8{b4[0], b4[1], b4[2], b4[3], 0, 0, 0, 0};
                    }
                }
            }
        }
    }

#pragma unroll 1
    for (int seg = 0; seg < (DUAL ? 2 : 1); ++seg) {
        const _Float16 *const X = seg == 0 ? p.A : p.P;
        const _Float16 *const Y = seg == 0 ? p.B : p.Q;
        const int64_t ldx = seg == 0 ? p.lda : p.ldp;
        const int64_t ldy = seg == 0 ? p.ldb : p.ldq;
        const int Kseg = seg == 0 ? p.K : p.K2;
        if (seg == 1) {
            __syncthreads();
            if (p.sub) negate_acc();
        }
        ca.init(ldx, ctid);
        cb.init(ldy, ctid);

        auto rsrc_a = [&](int k0) {
            if constexpr (TA) return make_rsrc(X + (int64_t)k0 * ldx + mc, MAX_RECORDS);
            else return make_rsrc(X + (int64_t)mc * ldx + k0, MAX_RECORDS);
        };
        auto rsrc_b = [&](int k0) {
            if constexpr (TB) return make_rsrc(Y + (int64_t)k0 * ldy + nc, MAX_RECORDS);
            else return make_rsrc(Y + (int64_t)nc * ldy + k0, MAX_RECORDS);
        };
        const int nk_seg = (Kseg + SK * BK - 1) / (SK * BK);
        int s_lo = 0, s_hi = nk_seg;
        if constexpr (SPLIT) {
            const int off = seg == 0 ? 0 : (p.K + SK * BK - 1) / (SK * BK);
            const int lo = kspl * p.split_steps - off, hi = lo + p.split_steps;
            s_lo = __builtin_amdgcn_readfirstlane(lo < 0 ? 0 : (lo > nk_seg ? nk_seg : lo));
            s_hi = __builtin_amdgcn_readfirstlane(hi < 0 ? 0 : (hi > nk_seg ? nk_seg : hi));
        }
        const int nk = s_hi - s_lo;

        // Copies of step s: B straight into `stage`; A too, or (prologue)
        // into the registers ra (load_a, issued separately in the loop).
        auto step_k0 = [&](int s) {
            return __builtin_amdgcn_readfirstlane((((s < nk ? s : nk - 1) + s_lo) * SK + grp) * BK);
        };
        auto load_a = [&](int s) {
            if constexpr (PROS) {
                const int k0 = step_k0(s);
                ca.load(rsrc_a(k0), s < nk ? Kseg - k0 : 0, ra);
            }
        };
        auto copy_step = [&](int s, char *stage) {
            const int k0 = step_k0(s);
            const int kleft = s < nk ? Kseg - k0 : 0;
            if constexpr (!PROS) ca.dma(rsrc_a(k0), stage, kleft);
            cb.dma(rsrc_b(k0), stage + BM * ROWB, kleft);
        };

        if (nk > 0) {
#pragma unroll
            for (int s = 0; s < NS; ++s) {
                load_a(s);
                if (copy_wave) copy_step(s, mine + s * STAGE);
                // the prologue writes step 0's left tile now; step 1's stays
                // in registers until the first step's barrier
                if (PROS && s == 0) relu_store_a(mine);
            }
            __builtin_amdgcn_sched_barrier(0);
            wait_vm_lgkm0<(NS - 1) * NL>();
            __builtin_amdgcn_s_barrier();
            __builtin_amdgcn_sched_barrier(0);
            if (NPW == 0 || !copy_wave) {
                read_a(0, mine, 0, 0);
                read_b(0, mine, 0);
            }
        }
        if constexpr (NPW > 0) {
            // Copy-only waves: the barrier of every step, as the computing
            // waves (step kt+1 landed, step kt's stage released), then the
            // copies of step kt+NS into that stage.
            if (copy_wave) {
                for (int kt = 0; kt < nk; ++kt) {
                    char *cur = mine + (kt & (NS - 1)) * STAGE;
                    __builtin_amdgcn_sched_barrier(0);
                    wait_vm_lgkm0<VM_AT_BARRIER>();
                    __builtin_amdgcn_s_barrier();
                    __builtin_amdgcn_sched_barrier(0);
                    copy_step(kt + NS, cur);
                }
                __builtin_amdgcn_s_waitcnt(0);
                continue;
            }
        }

        // One reduction step.  On entry LDS stage `cur` holds step kt, steps
        // kt+1 .. kt+NS-1 are under way into the other stages, fa[0] holds
        // the A fragments of slice 0 and fb[0] the B fragments of half 0.
        // (two instances of the loop: with the copies, for the waves that
        // issue them, and without)
        auto run_loop = [&](auto with_copies) {
        constexpr bool WC = decltype(with_copies)::value;
        for (int kt = 0; kt < nk; ++kt) {
            char *cur = mine + (kt & (NS - 1)) * STAGE;
            char *nxt = mine + ((kt + 1) & (NS - 1)) * STAGE;
            // slice 0: half 0, first A blocks
            read_a(1, cur, 0, 1);
            if constexpr (PRIO) __builtin_amdgcn_s_setprio(1);
            mfmas(0, 0, 0);
            sched_slice<NM, NRA, 0, 0, false>();
            // slice 1: half 0, second A blocks (B fragments of half 1 in flight)
            read_a(0, cur, 1, 0);
            read_b(1, cur, 1);
            mfmas(1, 0, 1);
            round16();
            sched_slice<NM, NRB, 0, 0, false>();
            // slice 2: half 1, first A blocks (prologue: plus step kt+1's
            // rectified left tile into its stage, whose loads were issued
            // three slices ago; kept inside this slice so that the wait for
            // them is not hoisted to the top of the step)
            if constexpr (PROS) __builtin_amdgcn_sched_barrier(0);
            read_a(1, cur, 1, 1);
            relu_store_a(nxt);
            load_a(kt + NS);
            mfmas(0, 1, 0);
            if constexpr (PROS) sched_slice2<NM, NRA, 0x200, CopyA::NLOAD, 0x020, CopyA::NLOAD>();
            else sched_slice<NM, NRA, 0, 0, false>();
            if constexpr (PRIO) __builtin_amdgcn_s_setprio(0);
            // Step kt+1 complete in LDS for every wave; every read of `cur` done.
            if constexpr (VM_AT_BARRIER == 0) {
                __builtin_amdgcn_s_waitcnt(0);
                __syncthreads();
            } else {
                __builtin_amdgcn_sched_barrier(0);
                wait_vm_lgkm0<VM_AT_BARRIER>();
                __builtin_amdgcn_s_barrier();
                __builtin_amdgcn_sched_barrier(0);
            }
            // slice 3: half 1, second A blocks, plus the first fragments of
            // step kt+1 and the copies of step kt+NS (into `cur`, now free)
            read_a(0, nxt, 0, 0);
            read_b(0, nxt, 0);
            mfmas(1, 1, 1);
            round16();
            if constexpr (WC) copy_step(kt + NS, cur);
            sched_slice<NM, NRB, 0x020, WC ? NL : 0, false>();
        }
        };
        if (copy_wave) run_loop(std::true_type{});
        else run_loop(std::false_type{});

        __builtin_amdgcn_s_waitcnt(0);
        if (seg == 1 && p.sub) negate_acc();
    }
    // the copy-only waves are done (the epilogue has no barrier)
    if (NPW > 0 && copy_wave) return;
    if constexpr (FOLD) {
#pragma unroll
        for (int t = 0; t < TN; ++t)
#pragma unroll
            for (int s = 0; s < TM; ++s)
#pragma unroll
                for (int e = 0; e < 4; ++e) acc[t][s][e] = (float)s16[t][s][e];
    }

    if constexpr (SPLIT) {
        {
            // Partial tile of this split to the workspace, each thread's 4
            // accumulators of a 16x16 block as one 16-byte write.
            float *const part = p.ws + (size_t)tile_id * p.splits * (BM * BN);
#pragma unroll
            for (int t = 0; t < TN; ++t)
#pragma unroll
                for (int s = 0; s < TM; ++s)
                    *reinterpret_cast<f4 *>(part + (size_t)kspl * (BM * BN) + ((t * TM + s) * NT + tid) * 4) =
                        acc[t][s];
            __syncthreads();
            __shared__ int last_split;
            if (tid == 0) {
                const unsigned before = __hip_atomic_fetch_add(p.counters + tile_id, 1u, __ATOMIC_RELEASE,
                                                               __HIP_MEMORY_SCOPE_AGENT);
                last_split = before == (unsigned)(p.splits - 1);
                if (last_split) __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
            }
            __syncthreads();
            if (!__builtin_amdgcn_readfirstlane(last_split)) return;
#pragma unroll
            for (int t = 0; t < TN; ++t)
#pragma unroll
                for (int s = 0; s < TM; ++s) acc[t][s] = f4{0.f, 0.f, 0.f, 0.f};
            for (int j = 0; j < p.splits; ++j) {
#pragma unroll
                for (int t = 0; t < TN; ++t)
#pragma unroll
                    for (int s = 0; s < TM; ++s)
                        acc[t][s] += *reinterpret_cast<const f4 *>(part + (size_t)j * (BM * BN) +
                                                                   ((t * TM + s) * NT + tid) * 4);
            }
            // partials back to zero (see the 32x32 kernel)
            for (int j = 0; j < p.splits; ++j) {
#pragma unroll
                for (int t = 0; t < TN; ++t)
#pragma unroll
                    for (int s = 0; s < TM; ++s)
                        *reinterpret_cast<f4 *>(part + (size_t)j * (BM * BN) + ((t * TM + s) * NT + tid) * 4) =
                            f4{0.f, 0.f, 0.f, 0.f};
            }
            if (tid == 0)
                __hip_atomic_store(p.counters + tile_id, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
    }

    if constexpr (SK > 1) {
        // Split-K: every k-group writes its partial tile to LDS (fp32, rows
        // padded by 4 floats), then all threads sum the SK partials in group
        // order, apply the epilogue and store 8 contiguous outputs each.
        __syncthreads();
        float *part = reinterpret_cast<float *>(lds);
#pragma unroll
        for (int t = 0; t < TN; ++t)
#pragma unroll
            for (int s = 0; s < TM; ++s) {
                const int i = wm * WTM + 16 * s + l16;
                const int j = wn * WTN + 16 * G * (t / G) + 4 * G * g4 + 4 * (t % G);
                *reinterpret_cast<f4 *>(part + (grp * BM + i) * PADN + j) = acc[t][s];
            }
        __syncthreads();
        constexpr int CPR = BN / 8;
        for (int c = tid; c < BM * CPR; c += NT) {
            const int i = c / CPR, j = (c % CPR) * 8;
            float x[8];
#pragma unroll
            for (int e = 0; e < 8; ++e) x[e] = 0.f;
#pragma unroll
            for (int g = 0; g < SK; ++g) {
                const f4 *src = reinterpret_cast<const f4 *>(part + (g * BM + i) * PADN + j);
                const f4 a0 = src[0], a1 = src[1];
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    x[e] += a0[e];
                    x[4 + e] += a1[e];
                }
            }
            if (p.bias_kind != BIAS_NONE) {
                const _Float16 *bp = p.bias_kind == BIAS_ROW ? p.bias + nc + j
                                                             : p.bias + (int64_t)(mc + i) * p.ldbias + nc + j;
                const h8 bv = *reinterpret_cast<const h8 *>(bp);
#pragma unroll
                for (int e = 0; e < 8; ++e) x[e] += p.bias_sign * (float)bv[e];
            }
            activate(p.act, x);
            h8 o;
#pragma unroll
            for (int e = 0; e < 8; ++e) o[e] = (_Float16)x[e];
            if (mc + i >= m0 && nc + j >= n0)
                *reinterpret_cast<h8 *>(p.C + (int64_t)(mc + i) * p.ldc + nc + j) = o;
        }
        return;
    }

    // Epilogue on registers: per A block and group of G B blocks a lane
    // holds 4G consecutive outputs of one row: +/- bias, activation, fp16,
    // 16-byte stores (8-byte for G = 1; each guarded so an output shared
    // with a neighbouring tile is stored by its owner only).  Row blocks
    // outermost.
#pragma unroll
    for (int s = 0; s < TM; ++s) {
#pragma unroll
        for (int tg = 0; tg < NGRP; ++tg) {
            const int i = mc + wm * WTM + 16 * s + l16;
            const int j = nc + wn * WTN + 16 * G * tg + 4 * G * g4;
            float x[4 * G];
#pragma unroll
            for (int u = 0; u < G; ++u)
#pragma unroll
                for (int r = 0; r < 4; ++r) x[4 * u + r] = acc[tg * G + u][s][r];
            constexpr int W = G >= 2 ? 8 : 4;   // outputs per chunk
            if (p.bias_kind == BIAS_ROW) {
#pragma unroll
                for (int v = 0; v < NV; ++v)
#pragma unroll
                    for (int e = 0; e < W; ++e) x[W * v + e] += p.bias_sign * (float)brow[tg][v][e];
            } else if (p.bias_kind == BIAS_FULL) {
                const _Float16 *bp = p.bias + (int64_t)i * p.ldbias + j;
#pragma unroll
                for (int v = 0; v < NV; ++v) {
                    if constexpr (W == 8) {
                        const h8 bv = *reinterpret_cast<const h8 *>(bp + 8 * v);
#pragma unroll
                        for (int e = 0; e < 8; ++e) x[8 * v + e] += p.bias_sign * (float)bv[e];
                    } else {
                        const h4 bv = *reinterpret_cast<const h4 *>(bp);
#pragma unroll
                        for (int e = 0; e < 4; ++e) x[e] += p.bias_sign * (float)bv[e];
                    }
                }
            }
            activate(p.act, x);
            if (i >= m0) {
                _Float16 *dst = p.C + (int64_t)i * p.ldc + j;
#pragma unroll
                for (int v = 0; v < NV; ++v) {
                    if constexpr (W == 8) {
                        h8 o;
#pragma unroll
                        for (int e = 0; e < 8; ++e) o[e] = (_Float16)x[8 * v + e];
                        if (j + 8 * v >= n0) *reinterpret_cast<h8 *>(dst + 8 * v) = o;
                    } else {
                        h4 o;
#pragma unroll
                        for (int e = 0; e < 4; ++e) o[e] = (_Float16)x[e];
                        if (j >= n0) *reinterpret_cast<h4 *>(dst) = o;
                    }
                }
            }
        }
    }
}

}  // namespace gba
