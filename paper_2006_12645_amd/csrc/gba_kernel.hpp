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
//   * Each step's A and B tiles go from global memory straight into LDS
//     (gfx950's buffer loads with an LDS destination: the split copy of the
//     Global to Shared Memory subsection without the register stage), in
//     16-byte chunks; the copies of the next steps are in flight while the
//     current step is multiplied (Prefetching and Hiding Latency subsection)
//     over two or four LDS stages, with one barrier per step.
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
// LDS and layouts.  Each tile keeps the layout it has in global memory.  A
// reduction-contiguous operand (row-major A, column-major B) is stored as
// one 128-byte row (64 fp16 = 8 chunks of 16 bytes) per output row / column,
// chunk c of row r at chunk position c ^ swz32(r) (Swizzled Shared Memory
// subsection), and its MFMA fragments are 16-byte reads.  An operand
// contiguous along M or N (column-major A, row-major B) is stored as 64
// reduction rows, block-swizzled (bswT), and its fragments come from
// gfx950's transposing LDS reads (ds_read_b64_tr_b16), which turn four
// rows of four consecutive elements into four elements of one column per
// lane -- the transposition the paper's Volta kernels leave to the layout of
// shared memory.  Both swizzles keep the fragment reads free of bank
// conflicts; the copies write whole KB blocks of LDS.
//
// Edges.  A tile that would cross the last row or column of C is shifted
// back inside the matrix (this path needs M >= BM and N >= BN), so its loads
// never leave the operands; the outputs it shares with its neighbour are
// stored only by the tile that owns them.  Reduction indices at or beyond K
// (last step only) are fetched through a buffer offset beyond the resource's
// size, which the hardware returns as zeros without a branch.
#pragma once

#include <type_traits>

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

// Chunk permutation of LDS row r (periodic in 32 rows).
__device__ __forceinline__ int swz32(int r)
{
    int b0 = ((r >> 2) ^ (r >> 4)) & 1;
    int b1 = (r ^ (r >> 2) ^ (r >> 3)) & 1;
    int b2 = (r >> 1) & 1;
    return b0 | (b1 << 1) | (b2 << 2);
}

// Chunk permutations of the 16x16x32 path's LDS rows (conflict-free for
// its fragment reads: 16 rows of one 16-row block at one chunk for A, the
// permuted columns of perm16 for B).  swzA16 has period 16, so the A blocks
// of a warp tile sit at fixed offsets from each other.
__device__ __forceinline__ int swzA16(int r) { return ((r >> 1) & 3) | (((r ^ (r >> 3)) & 1) << 2); }
__device__ __forceinline__ int swzB16(int r)
{
    return ((r >> 1) & 1) | (((r ^ (r >> 4)) & 1) << 1) | (((r ^ (r >> 3) ^ (r >> 5)) & 1) << 2);
}

// Chunk permutation SW: 0 swz32 (32x32x16 path), 1 swzA16, 2 swzB16.
template <int SW>
__device__ __forceinline__ int swz_sel(int r)
{
    if constexpr (SW == 1) return swzA16(r);
    else if constexpr (SW == 2) return swzB16(r);
    else return swz32(r);
}

// Column (inside a 32-column block of B) presented as MFMA row rho.  The
// MFMA returns row rho = 8*(r/4) + 4*(lane/32) + r%4 in accumulator r of a
// lane, which this maps to column 16*(lane/32) + r.
__device__ __forceinline__ int jp32(int rho) { return 16 * ((rho >> 2) & 1) + 4 * (rho >> 3) + (rho & 3); }

typedef __attribute__((address_space(3))) void lds_void;

// s_waitcnt vmcnt(VM) lgkmcnt(0): all but the VM most recent global loads
// done, and every LDS access of this wave done.
template <int VM>
__device__ __forceinline__ void wait_vm_lgkm0()
{
    static_assert(VM >= 0 && VM < 64, "vmcnt field is 6 bits");
    __builtin_amdgcn_s_waitcnt((VM & 0xF) | ((VM >> 4) << 14) | (0x7 << 4));
}

// 16 bytes per lane from buffer `rs` straight into LDS at `lds` + 16 * lane.
__device__ __forceinline__ void buffer_load16_lds(__amdgpu_buffer_rsrc_t rs, char *lds, int voff, int soff)
{
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (lds_void *)lds, 16, voff, soff, 0, 0);
}

// Scheduling hints for one 16-deep slice of NM MFMAs: the NR fragment reads
// for the next slice go first (so they have the whole slice to land), then
// the MFMAs, each followed by its share of the CNT instructions of class
// MASK (global copies: 0x020), so those are spread evenly over the slice
// instead of queueing behind each other.  SPREAD: the reads are spread over
// the MFMAs as well (measured 2-4% faster with the twice as many transposing
// reads of the M-/N-contiguous layouts, 1-2% slower without them).
template <int NM, int NR, int MASK, int CNT, bool SPREAD, int I = 0>
__device__ __forceinline__ void sched_slice()
{
    constexpr int R0 = SPREAD ? 0 : NR;  // reads ahead of the first MFMA
    if constexpr (I == 0 && R0 > 0) __builtin_amdgcn_sched_group_barrier(0x100, R0, 0);
    if constexpr (I < NM) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        constexpr int r = ((NR - R0) * (I + 1)) / NM - ((NR - R0) * I) / NM;
        if constexpr (r > 0) __builtin_amdgcn_sched_group_barrier(0x100, r, 0);
        constexpr int c = (CNT * (I + 1)) / NM - (CNT * I) / NM;
        if constexpr (CNT > 0 && c > 0) __builtin_amdgcn_sched_group_barrier(MASK, c, 0);
        sched_slice<NM, NR, MASK, CNT, SPREAD, I + 1>();
    }
}

// As sched_slice, with two classes of instructions after the reads: NA of
// class MA spread over the first half of the slice's MFMAs, then NB of
// class MB over the second half (the prologue's LDS writes of the staged
// left tile, then the loads that refill its registers).
template <int NM, int NR, int MA, int NA, int MB, int NB, int I = 0>
__device__ __forceinline__ void sched_slice2()
{
    constexpr int H = NM / 2;
    if constexpr (I == 0 && NR > 0) __builtin_amdgcn_sched_group_barrier(0x100, NR, 0);
    if constexpr (I < NM) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        constexpr int J = I < H ? I : I - H;
        constexpr int CNT = I < H ? NA : NB;
        constexpr int MASK = I < H ? MA : MB;
        constexpr int c = (CNT * (J + 1)) / H - (CNT * J) / H;
        if constexpr (CNT > 0 && c > 0) __builtin_amdgcn_sched_group_barrier(MASK, c, 0);
        sched_slice2<NM, NR, MA, NA, MB, NB, I + 1>();
    }
}

// Direct global -> LDS copy of a reduction-contiguous operand tile with the
// gfx950 buffer_load_dwordx4 ... lds form: each instruction moves 64 chunks
// of 16 bytes into 1 KB of LDS in lane order (8 rows of 128 bytes), so lane
// l fetches the global chunk that the swizzle places at position l % 8 of
// row l / 8.  No registers hold the data and no LDS write instruction is
// issued.  Instruction i of wave w fills rows 8*(NW*i + w) .. +7.  A chunk
// at or beyond K is fetched with an out-of-range offset, for which the copy
// writes zeros.  SW selects the chunk permutation (swz_sel).
template <int R, int NT, int SW = 0>
struct DmaCopy {
    static constexpr int NW = NT / 64;
    static constexpr int NI = R / (8 * NW);                   // instructions per wave per step
    // rows of instructions NV apart differ by a multiple of the chunk
    // permutation's period, so they share lane offsets
    static constexpr int PER = SW == 2 ? 64 : 32;
    static constexpr int NV0 = (8 * NW) % PER == 0 ? 1 : PER / (8 * NW);
    static constexpr int NV = NV0 < NI ? NV0 : NI;            // distinct lane offsets
    static constexpr int NLOAD = NI;
    static_assert(R % (8 * NW) == 0, "rows must divide evenly among the waves");

    int voff[NV];  // lane byte offset from the instruction's first row
    int kq[NV];    // reduction index of the lane's chunk
    int w;         // wave index (uniform)
    int lb;        // 16 * lane: the lane's byte offset inside an instruction's KB
    int64_t ldb2;

    __device__ __forceinline__ void init(int64_t ld, int tid)
    {
        ldb2 = ld * 2;
        w = __builtin_amdgcn_readfirstlane(tid >> 6);
        const int l = tid & 63;
        lb = 16 * l;
#pragma unroll
        for (int v = 0; v < NV; ++v) {
            const int row = 8 * (NW * v + w) + (l >> 3);
            const int c = (l & 7) ^ swz_sel<SW>(row);
            voff[v] = (int)((l >> 3) * ldb2) + 16 * c;
            kq[v] = 8 * c;
        }
    }

    // Issue the step's copies into `stage`; chunks at or beyond kleft
    // (= K - step origin) become zeros.
    __device__ __forceinline__ void dma(__amdgpu_buffer_rsrc_t rs, char *stage, int kleft)
    {
#pragma unroll
        for (int i = 0; i < NI; ++i) {
            const int v = i % NV;
            const int row0 = 8 * (NW * i + w);
            buffer_load16_lds(rs, stage + row0 * 128, kq[v] < kleft ? voff[v] : OOB_OFFSET,
                              (int)(row0 * ldb2));
        }
    }

    // The same copy staged through registers, for a transform between the
    // global load and the LDS write (the prologue's ReLU): load() fetches
    // the lane's chunks, store() writes them where dma() would have put them.
    __device__ __forceinline__ void load(__amdgpu_buffer_rsrc_t rs, int kleft, i4 (&r)[NI]) const
    {
#pragma unroll
        for (int i = 0; i < NI; ++i) {
            const int v = i % NV;
            const int row0 = 8 * (NW * i + w);
            r[i] = __builtin_amdgcn_raw_buffer_load_b128(rs, kq[v] < kleft ? voff[v] : OOB_OFFSET,
                                                         (int)(row0 * ldb2), 0);
        }
    }
    __device__ __forceinline__ void store(char *stage, const i4 (&r)[NI]) const
    {
#pragma unroll
        for (int i = 0; i < NI; ++i)
            *reinterpret_cast<i4 *>(stage + 8 * (NW * i + w) * 128 + lb) = r[i];
    }
};

// LDS layout of an operand tile that is contiguous along M (column-major A)
// or N (row-major B): 64 reduction rows of R elements, row k at byte 2Rk of
// the tile, its 32-element block b kept at block position b ^ bswT<R>(k % 4).
// The transposing fragment reads (ds_read_b64_tr_b16) of a wave touch four
// consecutive rows and 4 x 16 bytes of one 32-element block per row half;
// the block swizzle spreads those over all banks.
template <int R>
__device__ __forceinline__ int bswT(int j)
{
    if constexpr (R >= 128) return j;
    else if constexpr (R == 64) return (j >> 1) & 1;
    else return 0;
}

// Direct global -> LDS copy of such a tile (the transposed counterpart of
// DmaCopy): instruction g = NW * i + w fills the g-th KB of the tile, i.e.
// rows RPI * g .. RPI * g + RPI - 1, lane l the 16-byte chunk at byte 16 l,
// fetched from the global chunk that the block swizzle puts there.  Rows at
// or beyond K are fetched with an out-of-range offset and become zeros.
// 16-element group permutation of reduction row k of an M- or N-contiguous
// tile on the 16x16x32 path: its fragment reads touch, per half-wave, 16
// consecutive elements of eight rows k0 + {0..3, 8..11}, which this spreads
// over eight distinct 32-byte bank groups.
__device__ __forceinline__ int fT16(int k) { return (k & 3) | (((k >> 3) & 1) << 2); }

template <int R, int NT, int SW = 0>
struct DmaCopyT {
    static constexpr int NW = NT / 64;
    static constexpr int CPR = R / 8;             // 16-byte chunks per row
    static constexpr int RPI = 1024 / (2 * R);    // rows per instruction
    static constexpr int NI = 64 / (RPI * NW);    // instructions per wave per step
    static constexpr int NLOAD = NI;
    static_assert(R >= 32 && R <= 512 && (R & (R - 1)) == 0, "rows of 32 to 512 elements");
    static_assert(SW == 0 || R >= 128, "the 16x16x32 permutation needs 8 or more groups per row");
    static_assert(64 % (RPI * NW) == 0, "rows must divide evenly among the waves");
    // A wave's consecutive instructions start RS rows apart; the chunk
    // permutation repeats every PER rows (fT16 every 16, bswT every 4), so
    // the lane offsets take NV distinct values.
    static constexpr int RS = RPI * NW;
    static constexpr int PER = SW ? 16 : 4;
    static constexpr int NV0 = RS % PER == 0 ? 1 : PER / RS;
    static constexpr int NV = NV0 < NI ? NV0 : NI;
    static_assert((RS & (RS - 1)) == 0, "a power-of-two row stride");

    int voff[NV];  // lane byte offset from the instruction's first row
    int krow;      // reduction row (inside the step) of the lane's chunk in instruction 0
    int w;         // wave index (uniform)
    int lb;        // 16 * lane: the lane's byte offset inside an instruction's KB
    int64_t ldb2;

    __device__ __forceinline__ void init(int64_t ld, int tid)
    {
        ldb2 = ld * 2;
        w = __builtin_amdgcn_readfirstlane(tid >> 6);
        const int l = tid & 63, rl = l / CPR, p = l % CPR;
        lb = 16 * l;
        krow = w * RPI + rl;
#pragma unroll
        for (int v = 0; v < NV; ++v) {
            const int r = krow + RS * v;
            const int col = SW ? 16 * ((p >> 1) ^ fT16(r)) + 8 * (p & 1)
                               : 32 * ((p >> 2) ^ bswT<R>(r & 3)) + 8 * (p & 3);
            voff[v] = (int)(rl * ldb2) + 2 * col;
        }
    }

    // Instruction i's chunk holds reduction row krow + RS i; the bound moves
    // to the uniform side so the comparison needs no per-instruction row.
    __device__ __forceinline__ void dma(__amdgpu_buffer_rsrc_t rs, char *stage, int kleft)
    {
#pragma unroll
        for (int i = 0; i < NI; ++i) {
            const int g = NW * i + w;
            buffer_load16_lds(rs, stage + g * 1024, krow < kleft - RS * i ? voff[i % NV] : OOB_OFFSET,
                              (int)(g * RPI * ldb2));
        }
    }

    // Register-staged form (as in DmaCopy).
    __device__ __forceinline__ void load(__amdgpu_buffer_rsrc_t rs, int kleft, i4 (&r)[NI]) const
    {
#pragma unroll
        for (int i = 0; i < NI; ++i) {
            const int g = NW * i + w;
            r[i] = __builtin_amdgcn_raw_buffer_load_b128(rs, krow < kleft - RS * i ? voff[i % NV] : OOB_OFFSET,
                                                         (int)(g * RPI * ldb2), 0);
        }
    }
    __device__ __forceinline__ void store(char *stage, const i4 (&r)[NI]) const
    {
#pragma unroll
        for (int i = 0; i < NI; ++i) *reinterpret_cast<i4 *>(stage + (NW * i + w) * 1024 + lb) = r[i];
    }
};

// Lane byte offset, inside such a tile, of the first transposing read of the
// fragment of 32-element block blk for the 16-deep slice at row 0 (add 32 R
// bytes per slice, 8 R for the second read of four more rows).  A
// ds_read_b64_tr_b16 gives lane 4c + d of every 16-lane group element d of
// the 4-element chunk addressed by lane 4j + c, for j = 0..3: so lane 4j + c
// addresses row j (plus 8 for the upper half-wave, which takes k 8..15 of
// the slice) at the 4-column group that its result lanes 4c..4c+3 need.
// PERM: the MFMA column order jp32 of the B operand (groups of four columns
// stay together under it), else the identity.
template <int R, bool PERM>
__device__ __forceinline__ int offT(int lane, int blk)
{
    const int i = lane & 15, q = (lane >> 4) & 1, hi = lane >> 5;
    const int j = i >> 2, c = i & 3;
    const int colb = PERM ? 16 * (c & 1) + 8 * q + 4 * (c >> 1) : 16 * q + 4 * c;
    return (8 * hi + j) * (2 * R) + 64 * (blk ^ bswT<R>(j)) + 16 * (colb >> 3) + 8 * ((colb >> 2) & 1);
}

typedef short s4v __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) s4v lds_s4v;

// The 8 fp16 of one fragment (rows k .. k+3 at p, k+4 .. k+7 at p + 8R).
template <int R>
__device__ __forceinline__ h8 read_frag_tr(const char *p)
{
    const s4v lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s4v *)p);
    const s4v hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s4v *)(p + 8 * R));
    return __builtin_bit_cast(h8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
}

// SK > 1: intra-workgroup split-K (Split-K subsection): the workgroup holds
// SK groups of WM x WN waves; in every step group g multiplies its own
// 64-deep slab of the reduction (SK slabs per step, each in its own LDS
// sub-stage), and after the last step the SK partial tiles are summed
// through LDS before the epilogue.
// NSTG (a power of two) LDS stages: the copies of a step are issued
// NSTG - 1 steps before the step is multiplied, so small tiles that cannot
// cover the memory latency with work hide it with depth.
// PRO: the prologue's ReLU on the left operand of every product (Pointwise
// Operations in Prologue subsection), applied to its MFMA fragments as they
// leave LDS, so LDS holds one copy of the operand.
// DUAL: a second product P.Q of the same output shape is accumulated into
// the same registers after A.B (Matmuls with Pointwise Epilogue
// subsection): the reduction runs over A.B's K steps and then over P.Q's K2
// steps, and only the sum (or difference) leaves the kernel.
// SPLIT: each output tile's reduction is split across p.splits workgroups
// (the grid holds p.splits workgroups per tile); every split writes its
// fp32 partial tile to p.ws and the last one of a tile to arrive sums them
// in split order and runs the epilogue.
template <int BM, int BN, int WM, int WN, int SK, int NSTG, int LA, int LB, bool ACC16, bool PRO, bool DUAL,
          bool SPLIT>
__global__ void __launch_bounds__(64 * WM * WN * SK) gemm_bias_act_fast(GemmArgs p)
{
    constexpr int NTG = 64 * WM * WN;         // threads per k-group
    constexpr int NT = NTG * SK;
    constexpr int BK = 64;
    constexpr int WTM = BM / WM, WTN = BN / WN;
    constexpr int TM = WTM / 32, TN = WTN / 32;
    constexpr int ROWB = BK * 2;              // bytes per LDS row
    constexpr int SUB = (BM + BN) * ROWB;     // bytes per k-group sub-stage
    constexpr int STAGE = SK * SUB;           // bytes per LDS stage
    // Operands contiguous along the reduction use DmaCopy and ds_read_b128
    // fragments, the others (TA / TB) DmaCopyT and transposing reads.
    constexpr bool TA = LA == COL, TB = LB == ROW;
    constexpr int NS = NSTG;                  // LDS stages
    static_assert((NS & (NS - 1)) == 0, "stage count must be a power of two");
    constexpr int PADN = BN + 4;              // fp32 row pitch of the split-K partial tiles
    constexpr int RED = SK > 1 ? SK * BM * PADN * 4 : 0;
    constexpr int LDS_BYTES = NS * STAGE > RED ? NS * STAGE : RED;
    static_assert(WTM % 32 == 0 && WTN % 32 == 0, "warp tile must be a multiple of 32x32");
    static_assert(!(ACC16 && SK > 1), "fp16 accumulation is defined for a single running sum");

    __shared__ __attribute__((aligned(16))) char lds[LDS_BYTES];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int grp = wave / (WM * WN);         // k-group
    const int gtid = tid - grp * NTG;         // thread index inside the k-group
    const int wm = (wave % (WM * WN)) % WM, wn = (wave % (WM * WN)) / WM;
    const int l32 = lane & 31, hi = lane >> 5;

    static_assert(!SPLIT || (SK == 1 && !ACC16), "a split reduction needs one k-group and fp32 sums");
    // This workgroup's output tile and, under a split reduction, its split
    // (readfirstlane: both are uniform, and in scalar registers every
    // address derived from them stays scalar).
    int tile_id = blockIdx.x, kspl = 0;
    if constexpr (SPLIT) {
        tile_id = __builtin_amdgcn_readfirstlane((int)blockIdx.x / p.splits);
        kspl = __builtin_amdgcn_readfirstlane((int)blockIdx.x - tile_id * p.splits);
    }
    int tm, tn;
    tile_coords(tile_id, SPLIT ? p.tiles_m * p.tiles_n : (int)gridDim.x, p.tiles_m, tm, tn);
    // Output tile origin, and the origin of the tile actually computed: an
    // edge tile is shifted back so that it lies inside the matrix (M >= BM
    // and N >= BN on this path); the rows/columns it shares with its
    // neighbour are computed twice but stored once.
    const int m0 = tm * BM, n0 = tn * BN;
    const int mc = m0 + BM <= p.M ? m0 : p.M - BM;
    const int nc = n0 + BN <= p.N ? n0 : p.N - BN;

    using CopyA = std::conditional_t<TA, DmaCopyT<BM, NTG>, DmaCopy<BM, NTG>>;
    using CopyB = std::conditional_t<TB, DmaCopyT<BN, NTG>, DmaCopy<BN, NTG>>;
    CopyA ca;
    CopyB cb;

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
    // Transposing reads: per 32-element block of the warp tile (the B tile
    // starts BM * ROWB bytes into the stage, as in the other layout).
    int offtq[TA ? TM : 1], offtp[TB ? TN : 1];
    if constexpr (TA) {
#pragma unroll
        for (int s = 0; s < TM; ++s) offtq[s] = offT<BM, false>(lane, wm * TM + s);
    }
    if constexpr (TB) {
#pragma unroll
        for (int t = 0; t < TN; ++t) offtp[t] = BM * ROWB + offT<BN, true>(lane, wn * TN + t);
    }

    f16v acc[TN][TM];
#pragma unroll
    for (int t = 0; t < TN; ++t)
#pragma unroll
        for (int s = 0; s < TM; ++s)
#pragma unroll
            for (int e = 0; e < 16; ++e) acc[t][s][e] = 0.f;

    // Fragments of two 16-deep slices: one being multiplied, one in flight.
    h8 fq[2][TM], fp[2][TN];
    auto read_frags = [&](int buf, const char *stage, int ks) {
#pragma unroll
        for (int s = 0; s < TM; ++s) {
            if constexpr (TA) fq[buf][s] = read_frag_tr<BM>(stage + offtq[s] + ks * 32 * BM);
            else fq[buf][s] = *reinterpret_cast<const h8 *>(stage + offq[ks] + s * 32 * ROWB);
        }
#pragma unroll
        for (int t = 0; t < TN; ++t) {
            if constexpr (TB) fp[buf][t] = read_frag_tr<BN>(stage + offtp[t] + ks * 32 * BN);
            else fp[buf][t] = *reinterpret_cast<const h8 *>(stage + offp[ks] + t * 32 * ROWB);
        }
    };
    auto mfmas = [&](int buf) {
        if constexpr (PRO) {
            // the prologue's ReLU, once per fragment, right before its use
            // (so the fragment read in flight is not waited for early)
#pragma unroll
            for (int s = 0; s < TM; ++s) fq[buf][s] = relu_h8(fq[buf][s]);
        }
#pragma unroll
        for (int t = 0; t < TN; ++t)
#pragma unroll
            for (int s = 0; s < TM; ++s)
                acc[t][s] = __builtin_amdgcn_mfma_f32_32x32x16_f16(fp[buf][t], fq[buf][s], acc[t][s], 0, 0, 0);
    };
    auto round16 = [&]() {
        // fp16 accumulation: the running sum is rounded to fp16 at the end of
        // every aligned 32-deep group of k (pairs: one v_cvt_pk_f16_f32 and
        // two v_cvt_f32_f16 per two values, against four single conversions).
        if constexpr (ACC16) {
#pragma unroll
            for (int t = 0; t < TN; ++t)
#pragma unroll
                for (int s = 0; s < TM; ++s)
#pragma unroll
                    for (int e = 0; e < 16; e += 2) {
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
            for (int s = 0; s < TM; ++s) acc[t][s] = -acc[t][s];
    };

    // Instruction interleaving hints for the scheduler: each MFMA is paired
    // with the fragment read (DS read) or global copy (VMEM read) that has
    // to overlap it.
    constexpr int NM = TN * TM;           // MFMAs per 16-deep slice
    constexpr int NR = TM * (TA ? 2 : 1) + TN * (TB ? 2 : 1);  // fragment reads per slice
    constexpr int NL = CopyA::NLOAD + CopyB::NLOAD;
    // Global loads still allowed in flight at the barrier of step kt: the
    // copies of steps kt+2 .. kt+NS-1; step kt+1 must have landed.
    constexpr int VM_AT_BARRIER = (NS - 2) * NL;
    char *const mine = lds + grp * SUB;   // this k-group's sub-stage of stage 0

    // The row bias of this lane's output columns, loaded before the
    // reduction so its latency is hidden behind it (the epilogue of the
    // single k-group tiles uses it from registers).
    h8 brow[SK == 1 ? TN : 1][2];
    if constexpr (SK == 1) {
        if (p.bias_kind == BIAS_ROW) {
#pragma unroll
            for (int t = 0; t < TN; ++t) {
                const _Float16 *bp = p.bias + nc + wn * WTN + 32 * t + 16 * hi;
                brow[t][0] = *reinterpret_cast<const h8 *>(bp);
                brow[t][1] = *reinterpret_cast<const h8 *>(bp + 8);
            }
        }
    }

    // One pass of the pipelined reduction per product: A.B, then (DUAL)
    // P.Q on top of it.  C - R is formed as -((-C) + R): negating the
    // running sum is exact and rounding is symmetric, so this equals
    // subtracting every product of R.
#pragma unroll 1
    for (int seg = 0; seg < (DUAL ? 2 : 1); ++seg) {
        const _Float16 *const X = seg == 0 ? p.A : p.P;
        const _Float16 *const Y = seg == 0 ? p.B : p.Q;
        const int64_t ldx = seg == 0 ? p.lda : p.ldp;
        const int64_t ldy = seg == 0 ? p.ldb : p.ldq;
        const int Kseg = seg == 0 ? p.K : p.K2;
        if (seg == 1) {
            // every wave is done with the first product's LDS stages (and
            // its trailing copies have landed) before they are refilled
            __syncthreads();
            if (p.sub) negate_acc();
        }
        ca.init(ldx, gtid);
        cb.init(ldy, gtid);

        // Resource of the step starting at reduction index k0 for each operand.
        auto rsrc_a = [&](int k0) {
            if constexpr (LA == ROW) return make_rsrc(X + (int64_t)mc * ldx + k0, MAX_RECORDS);
            else return make_rsrc(X + (int64_t)k0 * ldx + mc, MAX_RECORDS);
        };
        auto rsrc_b = [&](int k0) {
            if constexpr (LB == COL) return make_rsrc(Y + (int64_t)nc * ldy + k0, MAX_RECORDS);
            else return make_rsrc(Y + (int64_t)k0 * ldy + nc, MAX_RECORDS);
        };
        // Steps [s_lo, s_hi) of this product are this workgroup's: all of
        // them, or under a split its part of the split's range of the
        // concatenated steps of both products.
        const int nk_seg = (Kseg + SK * BK - 1) / (SK * BK);
        int s_lo = 0, s_hi = nk_seg;
        if constexpr (SPLIT) {
            const int off = seg == 0 ? 0 : (p.K + SK * BK - 1) / (SK * BK);
            const int lo = kspl * p.split_steps - off, hi = lo + p.split_steps;
            s_lo = __builtin_amdgcn_readfirstlane(lo < 0 ? 0 : (lo > nk_seg ? nk_seg : lo));
            s_hi = __builtin_amdgcn_readfirstlane(hi < 0 ? 0 : (hi > nk_seg ? nk_seg : hi));
        }
        const int nk = s_hi - s_lo;

        // Copies of step s (this k-group's slab) into `stage`.  Steps past
        // the last one are issued too, so every step of the loop below has
        // the same shape, but entirely with out-of-range offsets: they write
        // zeros into a stage nobody reads again without touching memory.  A
        // slab starting at or beyond K reads as zeros.
        auto copy_step = [&](int s, char *stage) {
            // wave-uniform; without readfirstlane the compiler may take it
            // (through the k-group index, from the thread index, or the
            // split range) for divergent and loop over the lanes of every
            // copy
            const int k0 = __builtin_amdgcn_readfirstlane((((s < nk ? s : nk - 1) + s_lo) * SK + grp) * BK);
            const int kleft = s < nk ? Kseg - k0 : 0;
            const auto ra = rsrc_a(k0);
            const auto rb = rsrc_b(k0);
            ca.dma(ra, stage, kleft);
            cb.dma(rb, stage + BM * ROWB, kleft);
        };

        // Prologue: steps 0 .. NS-1 into the LDS stages, then the first
        // fragments of step 0.
        if (nk > 0) {
#pragma unroll
            for (int s = 0; s < NS; ++s) copy_step(s, mine + s * STAGE);
            // step 0 landed for every wave (the later steps may still be in
            // flight: the loop's barriers wait for them)
            __builtin_amdgcn_sched_barrier(0);
            wait_vm_lgkm0<(NS - 1) * NL>();
            __builtin_amdgcn_s_barrier();
            __builtin_amdgcn_sched_barrier(0);
            read_frags(0, mine, 0);
        }

        // One reduction step.  On entry LDS stage `cur` holds step kt, steps
        // kt+1 .. kt+NS-1 are under way into the other stages and fq/fp[0]
        // hold slice 0 of step kt.
        for (int kt = 0; kt < nk; ++kt) {
            char *cur = mine + (kt & (NS - 1)) * STAGE;
            char *nxt = mine + ((kt + 1) & (NS - 1)) * STAGE;
            // slice 0 (fragments of slice 1 in flight)
            read_frags(1, cur, 1);
            mfmas(0);
            sched_slice<NM, NR, 0, 0, TA || TB>();
            // slice 1
            read_frags(0, cur, 2);
            mfmas(1);
            round16();
            sched_slice<NM, NR, 0, 0, TA || TB>();
            // slice 2
            read_frags(1, cur, 3);
            mfmas(0);
            sched_slice<NM, NR, 0, 0, TA || TB>();
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
            // slice 3, plus the first fragments of step kt+1 and the copies of
            // step kt+NS (into `cur`, now free)
            read_frags(0, nxt, 0);
            mfmas(1);
            round16();
            copy_step(kt + NS, cur);
            sched_slice<NM, NR, 0x020, NL, TA || TB>();
        }

        // Drain the trailing (unused) copies: nothing may still be writing LDS
        // when it is reused below or released.
        __builtin_amdgcn_s_waitcnt(0);
        if (seg == 1 && p.sub) negate_acc();
    }

    if constexpr (SPLIT) {
        {
            // Partial tile of this split to the workspace, each thread's
            // accumulators of a 32x32 block as 16 consecutive floats (a wave
            // writes 4 KB contiguously per block).
            float *const part = p.ws + (size_t)tile_id * p.splits * (BM * BN);
#pragma unroll
            for (int t = 0; t < TN; ++t)
#pragma unroll
                for (int s = 0; s < TM; ++s) {
                    f4 *dst = reinterpret_cast<f4 *>(part + (size_t)kspl * (BM * BN) + ((t * TM + s) * NT + tid) * 16);
#pragma unroll
                    for (int q = 0; q < 4; ++q)
                        dst[q] = f4{acc[t][s][4 * q], acc[t][s][4 * q + 1], acc[t][s][4 * q + 2], acc[t][s][4 * q + 3]};
                }
            // Count this split in, releasing the workgroup's partial (all of
            // its stores are done at the barrier) at device scope; the last
            // split to arrive acquires every other split's partial and goes
            // on, the others are done.  One release per workgroup and one
            // acquire per output tile: an acquire invalidates the cached
            // operands of every workgroup sharing the cache.
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
            // Sum of the partials in split order (independent of arrival
            // order, so the result is deterministic); the counter is reset
            // for the next call.
#pragma unroll
            for (int t = 0; t < TN; ++t)
#pragma unroll
                for (int s = 0; s < TM; ++s)
#pragma unroll
                    for (int e = 0; e < 16; ++e) acc[t][s][e] = 0.f;
            for (int j = 0; j < p.splits; ++j) {
#pragma unroll
                for (int t = 0; t < TN; ++t)
#pragma unroll
                    for (int s = 0; s < TM; ++s) {
                        const f4 *src =
                            reinterpret_cast<const f4 *>(part + (size_t)j * (BM * BN) + ((t * TM + s) * NT + tid) * 16);
#pragma unroll
                        for (int q = 0; q < 4; ++q) {
                            const f4 v = src[q];
#pragma unroll
                            for (int e = 0; e < 4; ++e) acc[t][s][4 * q + e] += v[e];
                        }
                    }
            }
            // The partials go back to zero like the counter: a later call
            // with more output tiles keeps counters where this call kept
            // partials, and the workspace contract is that every byte a
            // call uses is zero when it completes.
            for (int j = 0; j < p.splits; ++j) {
#pragma unroll
                for (int t = 0; t < TN; ++t)
#pragma unroll
                    for (int s = 0; s < TM; ++s) {
                        f4 *dst = reinterpret_cast<f4 *>(part + (size_t)j * (BM * BN) + ((t * TM + s) * NT + tid) * 16);
#pragma unroll
                        for (int q = 0; q < 4; ++q) dst[q] = f4{0.f, 0.f, 0.f, 0.f};
                    }
            }
            if (tid == 0)
                __hip_atomic_store(p.counters + tile_id, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
    }

    if constexpr (SK > 1) {
        // Split-K: every k-group writes its partial tile to LDS (fp32, rows
        // padded by 4 floats so the 32 rows a store touches hit distinct
        // banks), then all threads sum the SK partials in group order, apply
        // the epilogue and store 8 contiguous outputs each.
        __syncthreads();
        float *part = reinterpret_cast<float *>(lds);
#pragma unroll
        for (int t = 0; t < TN; ++t)
#pragma unroll
            for (int s = 0; s < TM; ++s) {
                const int i = wm * WTM + 32 * s + l32;
                const int j = wn * WTN + 32 * t + 16 * hi;
                f4 *dst = reinterpret_cast<f4 *>(part + (grp * BM + i) * PADN + j);
#pragma unroll
                for (int q = 0; q < 4; ++q)
                    dst[q] = f4{acc[t][s][4 * q], acc[t][s][4 * q + 1], acc[t][s][4 * q + 2], acc[t][s][4 * q + 3]};
            }
        __syncthreads();
        constexpr int CPR = BN / 8;   // 8-column chunks per row
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

    // Epilogue on registers: +/- bias, activation, fp16, two 16-byte stores
    // per lane per 32x32 block (each guarded so an output shared with a
    // neighbouring tile is stored by its owner only).  Row blocks outermost:
    // a wave's consecutive stores complete each row of its warp tile (up to
    // 128 bytes), so no cache line is written back to memory half-filled
    // while the whole grid stores at once.
    float b[TN][16];
#pragma unroll
    for (int t = 0; t < TN; ++t) {
        if (p.bias_kind == BIAS_ROW) {
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                b[t][e] = p.bias_sign * (float)brow[t][0][e];
                b[t][8 + e] = p.bias_sign * (float)brow[t][1][e];
            }
        } else {
#pragma unroll
            for (int e = 0; e < 16; ++e) b[t][e] = 0.f;
        }
    }
#pragma unroll
    for (int s = 0; s < TM; ++s) {
#pragma unroll
        for (int t = 0; t < TN; ++t) {
            const int j = nc + wn * WTN + 32 * t + 16 * hi;
            const int i = mc + wm * WTM + 32 * s + l32;
            float x[16];
#pragma unroll
            for (int e = 0; e < 16; ++e) x[e] = acc[t][s][e] + b[t][e];
            if (p.bias_kind == BIAS_FULL) {
                const _Float16 *bp = p.bias + (int64_t)i * p.ldbias + j;
                const h8 b0 = *reinterpret_cast<const h8 *>(bp);
                const h8 b1 = *reinterpret_cast<const h8 *>(bp + 8);
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    x[e] += p.bias_sign * (float)b0[e];
                    x[8 + e] += p.bias_sign * (float)b1[e];
                }
            }
            activate(p.act, x);
            h8 o0, o1;
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                o0[e] = (_Float16)x[e];
                o1[e] = (_Float16)x[8 + e];
            }
            if (i >= m0) {
                _Float16 *dst = p.C + (int64_t)i * p.ldc + j;
                if (j >= n0) *reinterpret_cast<h8 *>(dst) = o0;
                if (j + 8 >= n0) *reinterpret_cast<h8 *>(dst + 8) = o1;
            }
        }
    }
}

}  // namespace gba
