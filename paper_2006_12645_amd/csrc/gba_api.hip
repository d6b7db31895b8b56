// gba_api.hip -- the C entry points of libgba.so: argument validation, tile
// selection, launch on the caller's stream, and the unfused baseline's
// pointwise kernels.  Declarations and contracts are in include/gba.h.
#include <limits.h>
#include <stdint.h>

#include <mutex>

#include "gba.h"
#include "gba_tiles.hpp"

namespace gba {
namespace {

bool is_layout(int v) { return v == GBA_ROW_MAJOR || v == GBA_COL_MAJOR; }

bool aligned(const void *p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) & (a - 1)) == 0; }

int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

bool has_second(const gba_fused_desc &d) { return d.second != GBA_SECOND_NONE; }

// Host-side validation of a request (include/gba.h states the rules).
gba_status validate(const gba_fused_desc &d)
{
    if (!is_layout(d.layoutA) || !is_layout(d.layoutB)) return GBA_EINVAL;
    if (d.act < GBA_ACT_NONE || d.act > GBA_ACT_TANH) return GBA_EINVAL;
    if (d.accum != GBA_ACC_F32 && d.accum != GBA_ACC_F16) return GBA_EINVAL;
    if (d.prologue != GBA_PRO_NONE && d.prologue != GBA_PRO_RELU) return GBA_EINVAL;
    if (d.second < GBA_SECOND_NONE || d.second > GBA_SECOND_SUB) return GBA_EINVAL;
    if (d.bias_kind < GBA_BIAS_NONE || d.bias_kind > GBA_BIAS_FULL) return GBA_EINVAL;
    if (d.bias_op != GBA_OP_ADD && d.bias_op != GBA_OP_SUB) return GBA_EINVAL;
    if (d.tile_id >= NUM_TILES) return GBA_EINVAL;
    if (d.split_k < 0) return GBA_EINVAL;
    if (d.workspace != nullptr && !aligned(d.workspace, 256)) return GBA_EINVAL;
    const bool two = has_second(d);
    if (d.M < 0 || d.N < 0 || d.K < 0 || d.lda < 0 || d.ldb < 0 || d.ldc < 0) return GBA_EINVAL;
    if (two && (d.K2 < 0 || d.ldp < 0 || d.ldq < 0)) return GBA_EINVAL;
    if (d.bias_kind == GBA_BIAS_FULL && d.ldbias < 0) return GBA_EINVAL;
    if (d.M > INT_MAX || d.N > INT_MAX || d.K > INT_MAX || (two && d.K2 > INT_MAX))
        return GBA_EUNSUPPORTED;
    if (d.M == 0 || d.N == 0) return GBA_OK;
    if (d.C == nullptr || d.ldc < d.N) return GBA_EINVAL;
    const bool rowA = d.layoutA == GBA_ROW_MAJOR, rowB = d.layoutB == GBA_ROW_MAJOR;
    if (d.K > 0) {
        if (d.A == nullptr || d.B == nullptr) return GBA_EINVAL;
        if (d.lda < (rowA ? d.K : d.M) || d.ldb < (rowB ? d.N : d.K)) return GBA_EINVAL;
    }
    if (two && d.K2 > 0) {
        if (d.P == nullptr || d.Q == nullptr) return GBA_EINVAL;
        if (d.ldp < (rowA ? d.K2 : d.M) || d.ldq < (rowB ? d.N : d.K2)) return GBA_EINVAL;
    }
    if (d.bias_kind != GBA_BIAS_NONE && d.bias == nullptr) return GBA_EINVAL;
    if (d.bias_kind == GBA_BIAS_FULL && d.ldbias < d.N) return GBA_EINVAL;
    const bool with_bias = d.bias_kind != GBA_BIAS_NONE;
    if (!aligned(d.A, 2) || !aligned(d.B, 2) || !aligned(d.C, 2) || (with_bias && !aligned(d.bias, 2)) ||
        (two && (!aligned(d.P, 2) || !aligned(d.Q, 2))))
        return GBA_EUNSUPPORTED;
    return GBA_OK;
}

bool tile_fits(int tile, int64_t M, int64_t N) { return M >= TILES[tile].bm && N >= TILES[tile].bn; }

// Which small tiles the rule below the 256x256 cases may take (fp32
// accumulation): none, the RC set of four-stage tiles (21-23), or one tile
// id (24 in RR, 25 in CC); where no four-stage tile has copy-only waves
// (the prologue, and the CR layout) the k-group tiles instead, with the
// limits fitted in RC (SMALL_PRO_RC) or in the other layouts (SMALL_KGROUP).
constexpr int SMALL_NONE = -1, SMALL_RC = 0, SMALL_PRO_RC = -2, SMALL_KGROUP = -3;

int select_tile_rest(int64_t M, int64_t N, int64_t K, int accum, int small);

// Tile choice by problem shape (K is the total reduction length), the
// operand layouts, the accumulation and the prologue, tuned on MI355X over
// the workload shapes, random multiples of 128 and thin shapes (measured
// sweeps of every tile, warm and with operands from HBM).  The base rule
// (fitted in RC with fp32 accumulation; the layout-, accumulation- and
// prologue-specific branches are described where they are taken):
//   * the 256x256 tile (8 waves) as soon as it yields 136 workgroups: one
//     round over 53% or more of the 256 compute units beats two rounds of
//     a smaller tile; from 112 when 128x128 tiles (two per compute unit)
//     would not fit in one round;
//   * else 128x128 (two workgroups per compute unit) from 260 workgroups,
//     then 128x64 / 64x128 from 400: the 8-wave 128x64 tile on 16x16x32
//     MFMAs when B is reduction-contiguous, the 8-wave 64x128 one when only
//     A is, else the 4-wave tile with the long side along the longer output
//     side;
//   * a reduction of 1024 or more (fp32 accumulation only) whose 64x64
//     tiles fit in one round of 160 (from K = 2048: 88) to 256 workgroups
//     takes 64x64 with two k-groups of waves (intra-workgroup split-K) --
//     below 128 of them, 32x64 with four k-groups if that makes at most
//     256;
//     from K = 2048, with fewer
//     output tiles still, 64x64 with two k-groups while that makes more
//     than 64 workgroups, else 32x32 with four k-groups and four LDS
//     stages;
//   * else 64x64 from 160 workgroups (in RC, the four-stage 64x64 tile
//     instead for K >= 1792 over at most 512 of them), then 32x64 --
//     replaced, for fp32 accumulation and K >= 768, by 32x32 with four
//     k-groups when that makes at most 128 workgroups, else by 32x64 with
//     four k-groups when that makes at most 256 -- then 32x32.
// The 256x128 and 128x256 tiles (4 or 8 waves) were never clearly the
// fastest in those sweeps and are only used when asked for.  128x128 means
// the 8-wave tile on 16x16x32 MFMAs: with fp32 accumulation 3-6% faster
// than the 4-wave one over the shapes the rule gives it, except with
// column-major A and row-major B, where the two were within a few percent
// either way.  Over four sets of 51 shapes in RC (two of them held out from
// the fitting) the base rule is 0.35-0.5% slower in total than the
// per-shape best tile (1.3-1.5% before the 8-wave 128x64 / 64x128 tiles
// and the four-stage 64x64 one took the shapes above).  With fp16
// accumulation the 8-wave tiles are 25-40% faster than the 4-wave ones
// from 128x128 down and about 10% faster than 64x64 or 32x64 on the
// small-M inference shapes (measured in the RC layout), so they come first.
// Flops per byte of compulsory traffic (2MNK over 2(MK + KN + MN)) at the
// ridge point of the part (2500 TFLOP/s over 8 TB/s): below it a problem
// is bound by HBM when its operands come from there, and the four-stage
// tiles (21-25: copies three steps ahead of the MFMAs) beat the two-stage
// ones.
constexpr double RIDGE_AI = 315.0;

int select_tile(int64_t M, int64_t N, int64_t K, int accum, int la, int lb, bool pro)
{
    auto tiles = [&](int t) -> int64_t {
        return tile_fits(t, M, N) ? ceil_div(M, TILES[t].bm) * ceil_div(N, TILES[t].bn) : 0;
    };
    const double ai = (double)M * N * K / ((double)M * K + (double)K * N + (double)M * N + 1.0);
    // Short reductions (K <= 256) over 1024 or more rows and columns: two to
    // four 64-deep steps, where a large tile's pipeline fill and epilogue
    // outweigh its steps.  With column-major B (either accumulation): 256x256
    // from 208 workgroups, else 128x128 from 256, else the 8-wave tile with
    // its long side along the longer output side; with row-major B (fp32):
    // 256x256 from 256 workgroups, else the 4-wave 128x128 tile from 384,
    // else the 4-wave 128x64 / 64x128 one.  On 48 shapes (1024-4096 rows and
    // columns, K = 64-256) per layout, warm / with operands from HBM: RC
    // 1.9% / 1.8% and CC 1.7% / 1.5% over the per-shape best tile (fp32; fp16
    // 3.3% / 2.8% and 2.6% / 2.0%), RR 3.1% / 3.3% and CR 2.7% / 2.8%,
    // against 4.4% / 3.7%, 3.9% / 3.5% (fp16 4.2% / 3.4%, 3.3% / 2.5%), 15% /
    // 13% and 11% / 10% for the rule below (3072x3072x128 RR: 12.1 / 11.9 us
    // on 128x64 against 16.6 / 16.4 on 256x256).
    if (K <= 256 && M >= 1024 && N >= 1024) {
        if (lb == GBA_COL_MAJOR) {
            if (tiles(1) >= 208) return 1;
            if (tiles(18) >= 256) return 18;
            return N > M ? 20 : 19;
        }
        if (accum == GBA_ACC_F32) {
            if (tiles(1) >= 256) return 1;
            if (tiles(4) >= 384) return 4;
            return N > M ? 7 : 5;
        }
    }
    if (accum == GBA_ACC_F16) {
        // fp16 accumulation: the 256x256 tile (which then keeps every wave
        // issuing copies) only from 208 workgroups; below
        // that the 8-wave 128x128 / 128x64 / 64x128 tiles are 3-25% faster
        // in every layout (M x N = 4096 x 2304 to 4096 x 3072, K = 1024 and
        // 4096; from 224 workgroups the two are within a few percent, the
        // 256x256 one ahead for K = 4096)
        if (tiles(1) >= 208) return 1;
    } else {
        if (tiles(1) >= 136) return 1;
        if (tiles(1) >= 112 && tiles(4) > 512) return 1;  // 128x128 would need a second round
    }
    if (accum == GBA_ACC_F16) {
        // fp16 accumulation cannot split the reduction over k-groups (one
        // running sum).  In RC the small tiles run with copy-only waves
        // beside the computing ones, which keeps enough bytes in flight from
        // HBM: the 32x32 tile while it makes at most one round of 256
        // workgroups, else the 32x64 one, else the 64x64 one up to 640
        // workgroups (on 72 random RC shapes and 66 thin ones, warm and with
        // operands from HBM: 1.1% and 0.4% slower in total than the
        // per-shape best tile, against 4.9% and 16% for the rule before;
        // the 8-wave tiles keep two stages and pull less from HBM: 896 x
        // 1536 x 1024, 15.6 against 11.8 us cold).  The other layouts have
        // branches of their own below.  Larger problems then take the 8-wave
        // tiles on 16x16x32 MFMAs (their two waves per SIMD overlap one
        // wave's rounding with the other's MFMAs): 128x128 for one round of
        // short reductions (K <= 1024, 128-255 workgroups) and from 384
        // workgroups, else 64x128 or 128x64 -- with both operand tiles
        // reduction-contiguous 64x128.
        const bool rc = la == GBA_ROW_MAJOR && lb == GBA_COL_MAJOR;
        if (rc) {
            if (tile_fits(23, M, N) && tiles(23) <= 256) return 23;
            if (tile_fits(21, M, N) && tiles(21) <= 256) return 21;
            if (tile_fits(22, M, N) && tiles(22) <= 640) return 22;
        } else if (la == lb && !pro) {
            // RR and CC: the four-stage tile with its long side along the
            // operand's contiguous direction (32x128 in RR, 128x32 in CC)
            // up to one round of 256 workgroups, where it does not fit the
            // 32x64 tile on memory-bound thin shapes, else the 8-wave
            // tiles below (on 36 thin shapes per layout, warm and with
            // operands from HBM: 5.5% / 0% slower in total than the
            // per-shape best tile in RR and 3.0% / 0.5% in CC, against
            // 21% / 49% and 16% / 27% for the rule before)
            const int tn = la == GBA_ROW_MAJOR ? 24 : 25;
            if (tile_fits(tn, M, N) && tiles(tn) <= 256) return tn;
            if (ai < RIDGE_AI && (M <= 256 || N <= 256) && tile_fits(8, M, N) && tiles(8) <= 256) return 8;
        } else if (la == lb) {
            // RR and CC with the prologue, where those tiles have no
            // copy-only waves: the 8-wave tiles below (36 thin shapes per
            // layout: 1.1% / 0.8% slower in total than the per-shape best in
            // RR and 1.5% / 1.8% in CC, against 42% / 21% and 24% / 12% on
            // the four-stage tiles)
        } else {
            // CR, where no small tile has copy-only waves: thin memory-bound
            // shapes take the two-stage 32x32 tile (at most 512 workgroups,
            // at most 128 rows or columns), else 64x64 up to 512
            // workgroups; then 128x128 from 384 workgroups, else the 8-wave
            // tile with its long side along the longer output side (on 36
            // thin and 51 random shapes, warm / with operands from HBM:
            // 1.4% / 0.4% and 1.4% / 1.6% slower in total than the
            // per-shape best tile, against 6.3% / 2.5% and 4.6% / 5.0%; with
            // the prologue, thin: 1.2% / 0.5% against 11% / 5.5%)
            if (ai < RIDGE_AI && (M <= 256 || N <= 256)) {
                if (tile_fits(9, M, N) && tiles(9) <= 512 && (M < N ? M : N) <= 128) return 9;
                if (tile_fits(6, M, N) && tiles(6) <= 512) return 6;
            }
            if (tiles(18) >= 384) return 18;
            const int t8w = N > M ? 20 : 19;
            if (tile_fits(t8w, M, N)) return t8w;
            if (tiles(18) >= 128) return 18;
        }
        const int64_t t18 = tiles(18);
        if (t18 >= 384 || (t18 >= 128 && t18 < 256 && K <= 1024)) return 18;
        if (tile_fits(20, M, N) && la == GBA_ROW_MAJOR) return 20;
        if (tile_fits(19, M, N) && lb == GBA_COL_MAJOR) return 19;
        if (t18 >= 128) return 18;
    }
    const bool cr = la == GBA_COL_MAJOR && lb == GBA_ROW_MAJOR;
    const bool rc = la == GBA_ROW_MAJOR && lb == GBA_COL_MAJOR;
    int small = SMALL_NONE;
    if (accum == GBA_ACC_F32) {
        if (cr) small = SMALL_KGROUP;
        else small = pro ? (rc ? SMALL_PRO_RC : SMALL_KGROUP) : rc ? SMALL_RC : la == GBA_ROW_MAJOR ? 24 : 25;
    }
    const int t = select_tile_rest(M, N, K, accum, small);
    // RR / CC, long reductions over at most two rounds of 64x64 tiles: the
    // four-stage 32x128 / 128x32 tile (896 x 2304 x 3200 RR: 30.9 / 34.8 us
    // warm / from HBM against 33.2 / 42.8)
    if (t == 6 && small >= 24 && tile_fits(small, M, N) && tiles(small) <= 512 && K >= 1792) return small;
    // memory-bound: the four-stage 64x64 tile (M = 256 x 4096 x 1024 from
    // HBM: 8.4 against 13.7 us; about 4% slower with cache-resident operands);
    // not in CR or with the prologue in RR / CC, where it has no copy-only
    // waves and a transposed tile
    if (t == 6 && ai < RIDGE_AI && small != SMALL_KGROUP) return 22;
    // long reductions over at most two rounds of 64x64 tiles: the four-stage
    // tile again (RC only; its transposed copies lose in the other layouts)
    if (t == 6 && rc && tiles(6) <= 512 && K >= 1792) return 22;
    // 128x64 / 64x128: the 8-wave 128x64 tile on 16x16x32 MFMAs where B is
    // reduction-contiguous, the 8-wave 64x128 one where only A is
    if (t == 5 || t == 7) {
        if (lb == GBA_COL_MAJOR) return 19;
        if (la == GBA_ROW_MAJOR) return 20;
    }
    return t == 4 && (accum == GBA_ACC_F16 || !cr) ? 18 : t;
}

// The rule below the 256x256 cases.  `small` (fp32 accumulation only):
//   * SMALL_RC: in RC the four-stage small tiles run on 16x16x32 MFMAs with
//     copy-only waves and take what the rule would give to the k-group
//     tiles (except the 32x32 one with four k-groups, for long reductions
//     over few output tiles) and to the 64x64 / 32x64 tiles: the 32x32
//     tile while it makes at most one round of 256 workgroups, else the
//     32x64 one, else the 64x64 one up to 512 workgroups.  Over two sets of
//     51 shapes and 53 thin ones (warm and with operands from HBM) that is
//     0.6% and 0.9% slower in total than the per-shape best tile, against
//     1.8% and 3.1% for the rule without them.
//   * 24 (RR) / 25 (CC): the one four-stage tile that runs on 16x16x32
//     MFMAs with copy-only waves in that layout (32x128 / 128x32: the long
//     side along the direction in which the operand tile is contiguous)
//     takes 129 to 256 workgroups (65 to 256 from K = 2048); fewer output
//     tiles over a reduction of 512 or more take the k-group tiles, 32x32
//     with four k-groups up to 256 workgroups, else 32x64 with four.  Over
//     51 random shapes and 53 thin ones per layout (warm / with operands
//     from HBM) that is 1.9% / 1.8% and 1.3% / 0.5% slower in total than
//     the per-shape best tile in RR, 1.3% / 1.6% and 0.5% / 0.6% in CC,
//     against 2.9% / 4.7% and 17% / 19% (RR), 2.7% / 4.4% and 16% / 20%
//     (CC) for the rule without them.
int select_tile_rest(int64_t M, int64_t N, int64_t K, int accum, int small)
{
    auto tiles = [&](int t) -> int64_t {
        return tile_fits(t, M, N) ? ceil_div(M, TILES[t].bm) * ceil_div(N, TILES[t].bn) : 0;
    };
    if (tiles(4) >= 260) return 4;
    const int t57 = N > M ? 7 : 5;
    if (tiles(t57) >= 400) return t57;
    if (small == SMALL_PRO_RC || small == SMALL_KGROUP) {
        // With the prologue, and in CR, over a reduction of 512 or more,
        // few output tiles (fewer than 160 64x64 tiles in RC, 384 in the
        // other layouts) take the k-group tiles: 32x32, else 32x64, else
        // 64x64, each with four k-groups, while that makes at most 256
        // workgroups.  With the prologue, over 53 thin and 51 random shapes
        // per layout (warm / with operands from HBM) that is 0.7% / 0.7% and
        // 2.9% / 2.0% slower in total than the per-shape best tile in RC,
        // 1.3% / 1.2% and 3.5% / 2.1% in RR, 0.9% / 1.1% and 5.1% / 1.1% in
        // CC and 1.2% / 0.6% and 2.4% / 3.0% in CR, against 14% / 3.3% and
        // 5.3% / 1.5% (RC), 35% / 34% and 10% / 10% (RR), 28% / 33% and
        // 13% / 9.5% (CC), 9.8% / 14% and 2.8% / 3.6% (CR) on the tiles
        // chosen without it; CR without the prologue 1.0% / 0.5% and
        // 2.7% / 4.0%, against 8.6% / 14% and 3.0% / 4.6%.  Held out (51
        // random shapes, seed 4242, with the prologue): RC 2.8% / 2.1%, RR
        // 3.3% / 2.8%, CC 4.0% / 1.4%, against 4.1% / 1.7%, 9.1% / 9.3% and
        // 11% / 8.5% ignoring the prologue.
        if (K >= 512 && tiles(6) < (small == SMALL_PRO_RC ? 160 : 384)) {
            if (tile_fits(13, M, N) && tiles(13) <= 256) return 13;
            if (tile_fits(12, M, N) && tiles(12) <= 256) return 12;
            if (tile_fits(10, M, N) && tiles(10) <= 256) return 10;
        }
        return select_tile_rest(M, N, K, accum, SMALL_NONE);
    }
    if (small >= 24) {
        const int64_t n = tiles(small);
        if (n > (K >= 2048 ? 64 : 128) && n <= 256) return small;
        if (K >= 512 && tiles(6) < 160) {
            if (tile_fits(13, M, N) && tiles(13) <= 256) return 13;
            if (tile_fits(12, M, N) && tiles(12) <= 256) return 12;
        }
        return select_tile_rest(M, N, K, accum, SMALL_NONE);
    }
    const bool rcs = small == SMALL_RC;
    if (accum == GBA_ACC_F32 && K >= 1024) {
        const int64_t n11 = tiles(11), n8 = tiles(8);
        if (!rcs && n11 >= (K >= 2048 ? 88 : 160) && n11 <= 256)
            return n11 < 128 && tiles(12) <= 256 ? 12 : 11;
        // (in RC's small-tile branch from K = 2048 at exactly 128 32x64
        // tiles as well: 64 x 4096 x 2048 on 32x32 with four k-groups 7.58 /
        // 9.07 us warm / from HBM against 7.38 / 10.58 on the four-stage
        // 32x32 tile; the thin set's total from HBM 1.2% -> 0.4% over the
        // per-shape best, the random sets unchanged)
        if (K >= 2048 && (n8 < 128 || (n8 <= 128 && (K >= 4096 || rcs)))) {
            if (n11 > 64) {
                if (!rcs) return 11;
            } else if (tile_fits(13, M, N)) {
                return 13;
            }
        }
    }
    if (rcs) {
        if (tile_fits(23, M, N) && tiles(23) <= 256) return 23;
        if (tile_fits(21, M, N) && tiles(21) <= 256) return 21;
        if (tile_fits(22, M, N) && tiles(22) <= 512) return 22;
        return select_tile_rest(M, N, K, accum, SMALL_NONE);
    }
    if (tiles(6) >= 160) return 6;
    if (tile_fits(8, M, N)) {
        // few 32x64 tiles over a reduction of 768 or more: the k-group
        // tiles keep more waves busy per output tile
        if (accum == GBA_ACC_F32 && K >= 768) {
            if (tile_fits(13, M, N) && tiles(13) <= 128) return 13;
            if (tiles(12) <= 256) return 12;
        }
        return 8;
    }
    if (tile_fits(9, M, N)) return 9;
    return -1;  // smaller than the smallest tile: general path
}

// Largest leading dimension the fast path addresses with 32-bit offsets.
constexpr int64_t FAST_MAX_LD = int64_t(1) << 21;

// The fast path needs every 16-byte chunk of every operand wholly inside or
// wholly outside the matrix.
bool fast_path_ok(const gba_fused_desc &d)
{
    const bool two = has_second(d), rowA = d.layoutA == GBA_ROW_MAJOR, colB = d.layoutB == GBA_COL_MAJOR;
    if (!aligned(d.A, 16) || !aligned(d.B, 16) || !aligned(d.C, 16)) return false;
    if (d.bias_kind != GBA_BIAS_NONE && !aligned(d.bias, 16)) return false;
    if (d.lda % 8 || d.ldb % 8 || d.ldc % 8 || d.lda >= FAST_MAX_LD || d.ldb >= FAST_MAX_LD) return false;
    if (d.bias_kind == GBA_BIAS_FULL && d.ldbias % 8) return false;
    if (d.N % 8 || (rowA ? d.K : d.M) % 8 || (colB ? d.K : d.N) % 8) return false;
    if (two) {
        if (!aligned(d.P, 16) || !aligned(d.Q, 16)) return false;
        if (d.ldp % 8 || d.ldq % 8 || d.ldp >= FAST_MAX_LD || d.ldq >= FAST_MAX_LD) return false;
        if ((rowA ? d.K2 : d.M) % 8 || (colB ? d.K2 : d.N) % 8) return false;
    }
    return true;
}

template <int LA, int LB>
const LayoutTable &variant_table(bool pro, bool dual)
{
    if (pro) return dual ? layout_table<LA, LB, true, true>() : layout_table<LA, LB, true, false>();
    return dual ? layout_table<LA, LB, false, true>() : layout_table<LA, LB, false, false>();
}

const LayoutTable &table_for(int la, int lb, bool pro, bool dual)
{
    if (la == GBA_ROW_MAJOR)
        return lb == GBA_ROW_MAJOR ? variant_table<ROW, ROW>(pro, dual) : variant_table<ROW, COL>(pro, dual);
    return lb == GBA_ROW_MAJOR ? variant_table<COL, ROW>(pro, dual) : variant_table<COL, COL>(pro, dual);
}

// Most workgroups one output tile's reduction is split across.
constexpr int64_t MAX_SPLITS = 64;

// The library splits a reduction by itself (split_k == 0) only where that
// was measured to win: reductions of 16384 or more over so few outputs that
// the 64x64 tile makes at most 32 workgroups.  There the 64x64 tile with
// about 128 workgroups in all beats every unsplit tile 1.6-2.7x
// (64x512x32768: 30 us against 50; 128x128x65536: 35 against 94).  On
// shorter reductions the partial-tile traffic and the device-scope release
// of every split cost more than the extra workgroups gain.
constexpr int AUTO_SPLIT_TILE = 6;

int64_t auto_splits(int64_t M, int64_t N, int64_t ktot)
{
    const TileCfg &c = TILES[AUTO_SPLIT_TILE];
    if (ktot < 16384 || !tile_fits(AUTO_SPLIT_TILE, M, N)) return 1;
    const int64_t tiles = ceil_div(M, c.bm) * ceil_div(N, c.bn);
    return tiles <= 32 ? ceil_div(128, tiles) : 1;
}

// How a valid request runs: the tile (or the general path), the output tile
// grid, and the split of each tile's reduction across workgroups with the
// workspace it needs.
struct Plan {
    int tile;          // -1: general path
    TileCfg cfg;
    int64_t tiles_m, tiles_n;
    int64_t splits, split_steps;
    size_t ws_bytes;   // 0 when unsplit
};

size_t counter_bytes(int64_t tiles) { return (size_t)ceil_div(tiles * 4, 256) * 256; }

Plan make_plan(const gba_fused_desc &d, bool may_split)
{
    const bool two = has_second(d);
    const int64_t ktot = d.K + (two ? d.K2 : 0);
    Plan pl;
    // A requested tile that is larger than the problem is replaced by the
    // library's choice; problems smaller than every tile take the general path.
    const bool tile_ok = d.tile_id >= 0 && tile_fits(d.tile_id, d.M, d.N) &&
                         !(d.accum == GBA_ACC_F16 && TILES[d.tile_id].sk > 1);
    const bool fp32 = d.accum == GBA_ACC_F32;
    int64_t auto_s = 1;
    if (may_split && d.split_k == 0 && !tile_ok && fp32) auto_s = auto_splits(d.M, d.N, ktot);
    pl.tile = tile_ok ? d.tile_id
                      : (auto_s > 1 ? AUTO_SPLIT_TILE : select_tile(d.M, d.N, ktot, d.accum, d.layoutA, d.layoutB,
                                                                            d.prologue == GBA_PRO_RELU));
    if (pl.tile >= 0 && !fast_path_ok(d)) pl.tile = -1;
    pl.cfg = pl.tile >= 0 ? TILES[pl.tile] : GENERIC_TILE;
    pl.tiles_m = ceil_div(d.M, pl.cfg.bm);
    pl.tiles_n = ceil_div(d.N, pl.cfg.bn);
    pl.splits = 1;
    pl.split_steps = 0;
    pl.ws_bytes = 0;
    if (may_split && pl.tile >= 0 && tile_splits(pl.cfg) && fp32 && d.split_k != 1) {
        const int64_t tiles = pl.tiles_m * pl.tiles_n;
        const int64_t nk = ceil_div(d.K, 64) + (two ? ceil_div(d.K2, 64) : 0);
        int64_t want = d.split_k >= 2 ? d.split_k : auto_s;
        want = want < nk ? want : nk;
        want = want < MAX_SPLITS ? want : MAX_SPLITS;
        if (want >= 2) {
            // equal step ranges, none of them empty
            const int64_t steps = ceil_div(nk, want);
            const int64_t splits = ceil_div(nk, steps);
            if (splits >= 2 && tiles * splits <= INT_MAX) {
                pl.splits = splits;
                pl.split_steps = steps;
                pl.ws_bytes = counter_bytes(tiles) + (size_t)(splits * tiles) * pl.cfg.bm * pl.cfg.bn * sizeof(float);
            }
        }
    }
    return pl;
}

// The plan a validated request runs with, given the workspace it carries:
// without room for the split the plan is made again without one (the
// library's unsplit tile choice differs from its split one).
Plan plan_for(const gba_fused_desc &d)
{
    Plan pl = make_plan(d, true);
    if (pl.splits > 1 && (d.workspace == nullptr || d.workspace_bytes < pl.ws_bytes)) pl = make_plan(d, false);
    return pl;
}

gba_status run_fused(const gba_fused_desc &d, hipStream_t stream)
{
    gba_status st = validate(d);
    if (st != GBA_OK || d.M == 0 || d.N == 0) return st;
    const bool two = has_second(d);
    const Plan pl = plan_for(d);
    const int tile = pl.tile;
    const bool fast = tile >= 0;

    GemmArgs a;
    a.A = static_cast<const _Float16 *>(d.A);
    a.B = static_cast<const _Float16 *>(d.B);
    a.P = two ? static_cast<const _Float16 *>(d.P) : nullptr;
    a.Q = two ? static_cast<const _Float16 *>(d.Q) : nullptr;
    a.bias = d.bias_kind == GBA_BIAS_NONE ? nullptr : static_cast<const _Float16 *>(d.bias);
    a.C = static_cast<_Float16 *>(d.C);
    a.lda = d.lda;
    a.ldb = d.ldb;
    a.ldp = two ? d.ldp : 0;
    a.ldq = two ? d.ldq : 0;
    a.ldc = d.ldc;
    a.ldbias = d.bias_kind == GBA_BIAS_FULL ? d.ldbias : 0;
    a.M = (int)d.M;
    a.N = (int)d.N;
    a.K = (int)d.K;
    a.K2 = two ? (int)d.K2 : 0;
    a.act = d.act;
    a.bias_kind = d.bias_kind;
    a.bias_sign = d.bias_op == GBA_OP_SUB ? -1.f : 1.f;
    a.sub = d.second == GBA_SECOND_SUB;
    if (pl.tiles_m * pl.tiles_n > INT_MAX) return GBA_EUNSUPPORTED;
    a.tiles_m = (int)pl.tiles_m;
    a.tiles_n = (int)pl.tiles_n;
    a.splits = (int)pl.splits;
    a.split_steps = (int)pl.split_steps;
    a.counters = pl.splits > 1 ? static_cast<unsigned *>(d.workspace) : nullptr;
    a.ws = pl.splits > 1 ? reinterpret_cast<float *>(static_cast<char *>(d.workspace) +
                                                      counter_bytes(pl.tiles_m * pl.tiles_n))
                         : nullptr;

    const LayoutTable &tab = table_for(d.layoutA, d.layoutB, d.prologue == GBA_PRO_RELU, two);
    const int acc16 = d.accum == GBA_ACC_F16;
    LaunchFn fn = !fast ? tab.generic[acc16] : (pl.splits > 1 ? tab.split[tile] : tab.fast[tile][acc16]);
    return fn(a, stream) == hipSuccess ? GBA_OK : GBA_EHIP;
}

// The request of gemm_bias_act: one product, no prologue, row bias if any.
gba_fused_desc single_product(gba_layout la, gba_layout lb, int64_t M, int64_t N, int64_t K,
                              const void *A, int64_t lda, const void *B, int64_t ldb, const void *bias,
                              void *C, int64_t ldc, gba_act act, gba_acc accum, int tile_id)
{
    gba_fused_desc d;
    gba_fused_desc_init(&d);
    d.layoutA = la;
    d.layoutB = lb;
    d.M = M;
    d.N = N;
    d.K = K;
    d.A = A;
    d.lda = lda;
    d.B = B;
    d.ldb = ldb;
    d.bias_kind = bias ? GBA_BIAS_ROW : GBA_BIAS_NONE;
    d.bias = bias;
    d.act = act;
    d.accum = accum;
    d.C = C;
    d.ldc = ldc;
    d.tile_id = tile_id;
    return d;
}

// ---------------------------------------------------------------------------
// Unfused baseline: in-place bias add and ReLU over a row-major fp16 matrix.
// HBM-bound; each thread handles 16-byte chunks of a row.

template <bool VEC>
__global__ void __launch_bounds__(256) bias_add_kernel(_Float16 *C, int64_t ldc, const _Float16 *bias,
                                                       int M, int N)
{
    const int64_t nch = (N + 7) / 8;
    const int64_t total = (int64_t)M * nch;
    for (int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; idx < total;
         idx += (int64_t)gridDim.x * blockDim.x) {
        const int64_t i = idx / nch;
        const int j = (int)(idx - i * nch) * 8;
        _Float16 *row = C + i * ldc + j;
        if (VEC && j + 8 <= N) {
            h8 c = *reinterpret_cast<const h8 *>(row);
            h8 b = *reinterpret_cast<const h8 *>(bias + j);
#pragma unroll
            for (int e = 0; e < 8; ++e) c[e] = (_Float16)((float)c[e] + (float)b[e]);
            *reinterpret_cast<h8 *>(row) = c;
        } else {
            for (int e = 0; e < 8 && j + e < N; ++e)
                row[e] = (_Float16)((float)row[e] + (float)bias[j + e]);
        }
    }
}

// The two-launch baseline's second kernel: bias add and activation in one
// pass, C = fp16(act(C + bias)) in fp32.
template <bool VEC>
__global__ void __launch_bounds__(256) bias_act_kernel(_Float16 *C, int64_t ldc, const _Float16 *bias,
                                                       int act, int M, int N)
{
    const int64_t nch = (N + 7) / 8;
    const int64_t total = (int64_t)M * nch;
    for (int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; idx < total;
         idx += (int64_t)gridDim.x * blockDim.x) {
        const int64_t i = idx / nch;
        const int j = (int)(idx - i * nch) * 8;
        _Float16 *row = C + i * ldc + j;
        if (VEC && j + 8 <= N) {
            h8 c = *reinterpret_cast<const h8 *>(row);
            const h8 b = *reinterpret_cast<const h8 *>(bias + j);
            float x[8];
#pragma unroll
            for (int e = 0; e < 8; ++e) x[e] = (float)c[e] + (float)b[e];
            activate(act, x);
#pragma unroll
            for (int e = 0; e < 8; ++e) c[e] = (_Float16)x[e];
            *reinterpret_cast<h8 *>(row) = c;
        } else {
            for (int e = 0; e < 8 && j + e < N; ++e) {
                float x[1] = {(float)row[e] + (float)bias[j + e]};
                activate(act, x);
                row[e] = (_Float16)x[0];
            }
        }
    }
}

template <bool VEC>
__global__ void __launch_bounds__(256) relu_kernel(_Float16 *C, int64_t ldc, int M, int N)
{
    const int64_t nch = (N + 7) / 8;
    const int64_t total = (int64_t)M * nch;
    for (int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; idx < total;
         idx += (int64_t)gridDim.x * blockDim.x) {
        const int64_t i = idx / nch;
        const int j = (int)(idx - i * nch) * 8;
        _Float16 *row = C + i * ldc + j;
        if (VEC && j + 8 <= N) {
            h8 c = *reinterpret_cast<const h8 *>(row);
#pragma unroll
            for (int e = 0; e < 8; ++e) c[e] = c[e] > (_Float16)0.0f ? c[e] : (_Float16)0.0f;
            *reinterpret_cast<h8 *>(row) = c;
        } else {
            for (int e = 0; e < 8 && j + e < N; ++e)
                row[e] = row[e] > (_Float16)0.0f ? row[e] : (_Float16)0.0f;
        }
    }
}

template <bool VEC>
__global__ void __launch_bounds__(256) add_kernel(_Float16 *C, int64_t ldc, const _Float16 *X, int64_t ldx,
                                                  int M, int N)
{
    const int64_t nch = (N + 7) / 8;
    const int64_t total = (int64_t)M * nch;
    for (int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; idx < total;
         idx += (int64_t)gridDim.x * blockDim.x) {
        const int64_t i = idx / nch;
        const int j = (int)(idx - i * nch) * 8;
        _Float16 *row = C + i * ldc + j;
        const _Float16 *xrow = X + i * ldx + j;
        if (VEC && j + 8 <= N) {
            h8 c = *reinterpret_cast<const h8 *>(row);
            const h8 x = *reinterpret_cast<const h8 *>(xrow);
#pragma unroll
            for (int e = 0; e < 8; ++e) c[e] = (_Float16)((float)c[e] + (float)x[e]);
            *reinterpret_cast<h8 *>(row) = c;
        } else {
            for (int e = 0; e < 8 && j + e < N; ++e)
                row[e] = (_Float16)((float)row[e] + (float)xrow[e]);
        }
    }
}

unsigned pointwise_grid(int64_t M, int64_t N)
{
    int64_t chunks = M * ((N + 7) / 8);
    int64_t blocks = ceil_div(chunks, 256);
    return (unsigned)(blocks < 65536 ? (blocks > 0 ? blocks : 1) : 65536);
}

gba_status validate_pointwise(int64_t M, int64_t N, const void *C, int64_t ldc, const void *bias,
                              bool need_bias)
{
    if (M < 0 || N < 0 || ldc < 0) return GBA_EINVAL;
    if (M > INT_MAX || N > INT_MAX) return GBA_EUNSUPPORTED;
    if (M == 0 || N == 0) return GBA_OK;
    if (C == nullptr || ldc < N || (need_bias && bias == nullptr)) return GBA_EINVAL;
    if (!aligned(C, 2) || !aligned(bias, 2)) return GBA_EUNSUPPORTED;
    return GBA_OK;
}

// ---------------------------------------------------------------------------
// Library-held scratch of gba_fused_gemm_noalloc: the workspace of a
// reduction split across workgroups (per-tile arrival counters, then the
// fp32 partial tiles), for callers that cannot allocate.  One copy per GPU,
// at its own device address, held until the process ends.  In host code
// the array's name is only a host-side stand-in: kernels and copies get the
// device address from hipGetSymbolAddress, taken once per device.

constexpr size_t NOALLOC_SCRATCH_BYTES = GBA_NOALLOC_SCRATCH_BYTES;
static_assert(NOALLOC_SCRATCH_BYTES % 256 == 0, "scratch size keeps 256-byte alignment");

static __device__ __align__(256) char scratch[NOALLOC_SCRATCH_BYTES];

constexpr int MAX_DEVICES = 64;
std::once_flag scratch_once[MAX_DEVICES];
void *scratch_ptr[MAX_DEVICES];
hipError_t scratch_err[MAX_DEVICES];

// Device address of the current device's scratch (looked up on the first
// call per device, with that device current).
gba_status device_scratch(void **ptr)
{
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess) return GBA_EHIP;
    if (dev < 0 || dev >= MAX_DEVICES) return GBA_EUNSUPPORTED;
    std::call_once(scratch_once[dev], [dev] {
        void *p = nullptr;
        const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        scratch_err[dev] = e;
        scratch_ptr[dev] = e == hipSuccess ? p : nullptr;
    });
    if (scratch_err[dev] != hipSuccess || scratch_ptr[dev] == nullptr) return GBA_EHIP;
    *ptr = scratch_ptr[dev];
    return GBA_OK;
}

// Sets n 32-bit words to zero: the split counters are cleared with a kernel
// (a memset node in a captured graph is not reliable on this platform).
__global__ void __launch_bounds__(256) zero_words_kernel(unsigned *p, int n)
{
    const int i = (int)(blockIdx.x * blockDim.x + threadIdx.x);
    if (i < n) p[i] = 0u;
}

}  // namespace
}  // namespace gba

using namespace gba;

extern "C" void gba_fused_desc_init(gba_fused_desc *desc)
{
    if (desc == nullptr) return;
    *desc = gba_fused_desc{};
    desc->layoutA = GBA_ROW_MAJOR;
    desc->layoutB = GBA_ROW_MAJOR;
    desc->prologue = GBA_PRO_NONE;
    desc->second = GBA_SECOND_NONE;
    desc->bias_kind = GBA_BIAS_NONE;
    desc->bias_op = GBA_OP_ADD;
    desc->act = GBA_ACT_NONE;
    desc->accum = GBA_ACC_F32;
    desc->tile_id = -1;
}

extern "C" gba_status gba_fused_workspace_size(const gba_fused_desc *desc, size_t *bytes)
{
    if (desc == nullptr || bytes == nullptr) return GBA_EINVAL;
    *bytes = 0;
    const gba_status st = validate(*desc);
    if (st != GBA_OK || desc->M == 0 || desc->N == 0) return st;
    *bytes = make_plan(*desc, true).ws_bytes;
    return GBA_OK;
}

extern "C" gba_status gba_fused_tile(const gba_fused_desc *desc, int *tile)
{
    if (desc == nullptr || tile == nullptr) return GBA_EINVAL;
    *tile = -1;
    const gba_status st = validate(*desc);
    if (st != GBA_OK || desc->M == 0 || desc->N == 0) return st;
    *tile = plan_for(*desc).tile;
    return GBA_OK;
}

extern "C" gba_status gba_fused_gemm(const gba_fused_desc *desc, gba_stream_t stream)
{
    if (desc == nullptr) return GBA_EINVAL;
    return run_fused(*desc, reinterpret_cast<hipStream_t>(stream));
}

extern "C" gba_status gba_fused_gemm_noalloc(const gba_fused_desc *desc, gba_stream_t stream)
{
    if (desc == nullptr) return GBA_EINVAL;
    gba_fused_desc d = *desc;
    d.workspace = nullptr;  // the caller's workspace fields are ignored
    d.workspace_bytes = 0;
    gba_status st = validate(d);
    if (st != GBA_OK || d.M == 0 || d.N == 0) return st;
    const Plan pl = make_plan(d, true);
    if (pl.splits > 1) {
        if (pl.ws_bytes > NOALLOC_SCRATCH_BYTES) return GBA_ESCRATCH;
        void *ws = nullptr;
        st = device_scratch(&ws);
        if (st != GBA_OK) return st;
        // The counters must be zero when the split kernel starts, whatever an
        // earlier call left behind.
        const int64_t ntiles = pl.tiles_m * pl.tiles_n;
        hipStream_t s = reinterpret_cast<hipStream_t>(stream);
        clear_last_error();
        hipLaunchKernelGGL(zero_words_kernel, dim3((unsigned)ceil_div(ntiles, 256)), dim3(256), 0, s,
                           static_cast<unsigned *>(ws), (int)ntiles);
        if (hipGetLastError() != hipSuccess) return GBA_EHIP;
        d.workspace = ws;
        d.workspace_bytes = NOALLOC_SCRATCH_BYTES;
    }
    return run_fused(d, reinterpret_cast<hipStream_t>(stream));
}

extern "C" gba_status gemm_bias_act(gba_layout layoutA, gba_layout layoutB, int64_t M, int64_t N,
                                    int64_t K, const void *A, int64_t lda, const void *B, int64_t ldb,
                                    const void *bias, void *C, int64_t ldc, gba_act act,
                                    gba_acc accum, gba_stream_t stream)
{
    return run_fused(single_product(layoutA, layoutB, M, N, K, A, lda, B, ldb, bias, C, ldc, act, accum, -1),
                     reinterpret_cast<hipStream_t>(stream));
}

extern "C" gba_status gemm_bias_act_tile(gba_layout layoutA, gba_layout layoutB, int64_t M,
                                         int64_t N, int64_t K, const void *A, int64_t lda,
                                         const void *B, int64_t ldb, const void *bias, void *C,
                                         int64_t ldc, gba_act act, gba_acc accum, int tile_id,
                                         gba_stream_t stream)
{
    return run_fused(
        single_product(layoutA, layoutB, M, N, K, A, lda, B, ldb, bias, C, ldc, act, accum, tile_id),
        reinterpret_cast<hipStream_t>(stream));
}

extern "C" int gba_num_tiles(void) { return NUM_TILES; }

extern "C" gba_status gba_tile_info(int tile_id, int *bm, int *bn, int *bk, int *waves, int *split_k)
{
    if (tile_id < 0 || tile_id >= NUM_TILES) return GBA_EINVAL;
    const TileCfg &c = TILES[tile_id];
    if (bm) *bm = c.bm;
    if (bn) *bn = c.bn;
    if (bk) *bk = 64;
    if (waves) *waves = c.wm * c.wn * c.sk;
    if (split_k) *split_k = c.sk;
    return GBA_OK;
}

extern "C" int gba_select_tile(gba_layout layoutA, gba_layout layoutB, int64_t M, int64_t N, int64_t K,
                               gba_acc accum)
{
    if (!is_layout(layoutA) || !is_layout(layoutB)) return -1;
    if (accum != GBA_ACC_F32 && accum != GBA_ACC_F16) return -1;
    if (M < 0 || N < 0 || K < 0 || M > INT_MAX || N > INT_MAX || K > INT_MAX) return -1;
    return select_tile(M, N, K, accum, layoutA, layoutB, false);  // -1 also when the general path would run
}

extern "C" gba_status gba_bias_add_f16(int64_t M, int64_t N, void *C, int64_t ldc, const void *bias,
                                       gba_stream_t stream)
{
    gba_status st = validate_pointwise(M, N, C, ldc, bias, true);
    if (st != GBA_OK || M == 0 || N == 0) return st;
    const bool vec = aligned(C, 16) && aligned(bias, 16) && ldc % 8 == 0;
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    dim3 grid(pointwise_grid(M, N)), block(256);
    _Float16 *c = static_cast<_Float16 *>(C);
    const _Float16 *b = static_cast<const _Float16 *>(bias);
    clear_last_error();
    if (vec)
        hipLaunchKernelGGL(bias_add_kernel<true>, grid, block, 0, s, c, ldc, b, (int)M, (int)N);
    else
        hipLaunchKernelGGL(bias_add_kernel<false>, grid, block, 0, s, c, ldc, b, (int)M, (int)N);
    return hipGetLastError() == hipSuccess ? GBA_OK : GBA_EHIP;
}

extern "C" gba_status gba_bias_act_f16(int64_t M, int64_t N, void *C, int64_t ldc, const void *bias,
                                       gba_act act, gba_stream_t stream)
{
    if (act < GBA_ACT_NONE || act > GBA_ACT_TANH) return GBA_EINVAL;
    gba_status st = validate_pointwise(M, N, C, ldc, bias, true);
    if (st != GBA_OK || M == 0 || N == 0) return st;
    const bool vec = aligned(C, 16) && aligned(bias, 16) && ldc % 8 == 0;
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    dim3 grid(pointwise_grid(M, N)), block(256);
    _Float16 *c = static_cast<_Float16 *>(C);
    const _Float16 *b = static_cast<const _Float16 *>(bias);
    clear_last_error();
    if (vec)
        hipLaunchKernelGGL(bias_act_kernel<true>, grid, block, 0, s, c, ldc, b, (int)act, (int)M, (int)N);
    else
        hipLaunchKernelGGL(bias_act_kernel<false>, grid, block, 0, s, c, ldc, b, (int)act, (int)M, (int)N);
    return hipGetLastError() == hipSuccess ? GBA_OK : GBA_EHIP;
}

extern "C" gba_status gba_relu_f16(int64_t M, int64_t N, void *C, int64_t ldc, gba_stream_t stream)
{
    gba_status st = validate_pointwise(M, N, C, ldc, nullptr, false);
    if (st != GBA_OK || M == 0 || N == 0) return st;
    const bool vec = aligned(C, 16) && ldc % 8 == 0;
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    dim3 grid(pointwise_grid(M, N)), block(256);
    _Float16 *c = static_cast<_Float16 *>(C);
    clear_last_error();
    if (vec)
        hipLaunchKernelGGL(relu_kernel<true>, grid, block, 0, s, c, ldc, (int)M, (int)N);
    else
        hipLaunchKernelGGL(relu_kernel<false>, grid, block, 0, s, c, ldc, (int)M, (int)N);
    return hipGetLastError() == hipSuccess ? GBA_OK : GBA_EHIP;
}

extern "C" gba_status gba_add_f16(int64_t M, int64_t N, void *C, int64_t ldc, const void *X, int64_t ldx,
                                  gba_stream_t stream)
{
    gba_status st = validate_pointwise(M, N, C, ldc, X, true);
    if (st != GBA_OK || M == 0 || N == 0) return st;
    if (ldx < N) return GBA_EINVAL;
    const bool vec = aligned(C, 16) && aligned(X, 16) && ldc % 8 == 0 && ldx % 8 == 0;
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    dim3 grid(pointwise_grid(M, N)), block(256);
    _Float16 *c = static_cast<_Float16 *>(C);
    const _Float16 *x = static_cast<const _Float16 *>(X);
    clear_last_error();
    if (vec)
        hipLaunchKernelGGL(add_kernel<true>, grid, block, 0, s, c, ldc, x, ldx, (int)M, (int)N);
    else
        hipLaunchKernelGGL(add_kernel<false>, grid, block, 0, s, c, ldc, x, ldx, (int)M, (int)N);
    return hipGetLastError() == hipSuccess ? GBA_OK : GBA_EHIP;
}

extern "C" const char *gba_status_string(gba_status status)
{
    switch (status) {
    case GBA_OK: return "GBA_OK";
    case GBA_EINVAL: return "GBA_EINVAL: invalid argument";
    case GBA_EUNSUPPORTED: return "GBA_EUNSUPPORTED: unsupported argument";
    case GBA_EHIP: return "GBA_EHIP: HIP launch error";
    case GBA_ESCRATCH:
        return "GBA_ESCRATCH: the request's split reduction needs more than the library's static "
               "scratch (GBA_NOALLOC_SCRATCH_BYTES); use gba_fused_gemm with a workspace or fewer splits";
    }
    return "unknown gba_status";
}

extern "C" const char *gba_version(void) { return "gba 0.1.0 gfx950"; }
