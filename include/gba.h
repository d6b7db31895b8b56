/*
 * gba.h -- fused fp16 GEMM + bias + activation for AMD MI355X (gfx950).
 *
 * C ABI of libgba.so.  Plain pointers and sizes only; C99 compatible.
 *
 * The operation is the matmul followed by the pointwise ReLU-of-add
 * statement of the paper's Problem Statement section (Listing 1 and its
 * expression tree, whose root is ReLU over the add of the matmul result and
 * the bias), computed in ONE kernel so the matmul result never goes to
 * global memory (Kernel Fusion section, "Pointwise Operations in Epilogue").
 * Operands may be row- or column-major, the four layout specialisations of
 * the Matmul Compute Decomposition section.
 *
 * Common conventions for every entry point below:
 *   - All array pointers are DEVICE pointers (memory the caller allocated on
 *     the GPU that is current for `stream`).  fp16 means IEEE binary16.
 *   - The caller owns every buffer.  The library never allocates, frees or
 *     synchronises; it keeps no mutable global state and is thread-safe.
 *   - Calls are asynchronous: work is enqueued on `stream` (NULL = the null
 *     stream) and the function returns once the kernel is launched.
 *   - Arguments are validated on the host before anything is enqueued.  On
 *     any error nothing is launched and the output is left untouched.
 *   - Outputs must not alias inputs.
 */
#ifndef GBA_H
#define GBA_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ABI-identical to hipStream_t. */
typedef struct ihipStream_t *gba_stream_t;

typedef enum { GBA_ROW_MAJOR = 0, GBA_COL_MAJOR = 1 } gba_layout;
typedef enum { GBA_ACT_NONE = 0, GBA_ACT_RELU = 1 } gba_act;
typedef enum { GBA_ACC_F32 = 0, GBA_ACC_F16 = 1 } gba_acc;
typedef enum {
    GBA_OK = 0,
    GBA_EINVAL = 1,        /* malformed argument (negative size, ld too small, NULL, bad enum) */
    GBA_EUNSUPPORTED = 2,  /* well-formed but outside what the library implements */
    GBA_EHIP = 3           /* the HIP runtime reported an error at launch */
} gba_status;

/*
 * gemm_bias_act -- C = act(A*B + bias), fp16 in, fp16 out.
 *
 * Follows the Problem Statement section (Listing 1): for 0<=i<M, 0<=j<N
 *     pre(i,j) = sum_{k<K} A(i,k) * B(k,j) + (bias ? bias[j] : 0)
 *     C[i*ldc + j] = fp16( act == GBA_ACT_RELU ? max(pre, 0) : pre )
 * with products summed in fp32 (accum == GBA_ACC_F32; fp16 inputs and fp32
 * accumulation as in the Background section) or with the running sum rounded
 * to fp16 after every aligned group of 32 k values (accum == GBA_ACC_F16).
 * The bias add and ReLU are done in fp32 and rounded once to fp16 (RNE).
 *
 * Layout and leading dimensions (BLAS meaning):
 *     A(i,k) = layoutA == GBA_ROW_MAJOR ? A[i*lda + k] : A[k*lda + i]
 *              (lda >= K resp. lda >= M)
 *     B(k,j) = layoutB == GBA_ROW_MAJOR ? B[k*ldb + j] : B[j*ldb + k]
 *              (ldb >= N resp. ldb >= K)
 *     C is always row-major, ldc >= N.
 *     bias: fp16[N] broadcast over rows, or NULL for no bias.
 * Sizes that are not tile multiples are handled inside the kernel (masked
 * loads and stores); nothing outside the stated extents is read or written.
 * Pointers need only fp16 (2-byte) alignment; 16-byte aligned A, B, C, bias
 * with lda, ldb, ldc multiples of 8 take the vectorised fast path.
 *
 * Degenerate sizes: M == 0 or N == 0 -> GBA_OK, nothing launched.
 * K == 0 -> C = act(bias) (the empty sum is zero).
 * Errors: GBA_EINVAL for M, N or K < 0, a leading dimension below its
 * extent, a NULL A/B (when M,N,K > 0) or C (when M,N > 0), or a bad enum;
 * GBA_EUNSUPPORTED for M, N or K above 2^31-1 or pointers not 2-byte
 * aligned; GBA_EHIP if the launch fails.
 */
gba_status gemm_bias_act(gba_layout layoutA, gba_layout layoutB,
                         int64_t M, int64_t N, int64_t K,
                         const void *A, int64_t lda,
                         const void *B, int64_t ldb,
                         const void *bias, void *C, int64_t ldc,
                         gba_act act, gba_acc accum, gba_stream_t stream);

/*
 * gemm_bias_act_tile -- gemm_bias_act with the tile configuration forced.
 *
 * The paper generates kernels for several block/warp tile sizes and keeps
 * the fastest per problem size (Experimental Evaluation section); this entry
 * point exposes that choice for sweeps.  tile_id indexes the table reported
 * by gba_tile_info; tile_id < 0 means "let the library choose" (identical to
 * gemm_bias_act).  A tile larger than the problem (bm > M or bn > N) is
 * replaced by the library's choice, and operands that miss the fast path's
 * alignment conditions use the general kernel whatever tile_id says.  Errors
 * as gemm_bias_act, plus GBA_EINVAL for a tile_id at or beyond
 * gba_num_tiles().
 */
gba_status gemm_bias_act_tile(gba_layout layoutA, gba_layout layoutB,
                              int64_t M, int64_t N, int64_t K,
                              const void *A, int64_t lda,
                              const void *B, int64_t ldb,
                              const void *bias, void *C, int64_t ldc,
                              gba_act act, gba_acc accum, int tile_id,
                              gba_stream_t stream);

/* Number of tile configurations compiled into the library. */
int gba_num_tiles(void);

/*
 * gba_tile_info -- describe tile configuration tile_id (Tiling for Blocks
 * and Warps and Split-K subsections): block tile bm x bn x bk (output rows x
 * output columns x reduction depth per step), waves per workgroup and the
 * intra-workgroup split-K factor.  Any output pointer may be NULL.
 * Returns GBA_EINVAL for an unknown tile_id.
 */
gba_status gba_tile_info(int tile_id, int *bm, int *bn, int *bk, int *waves, int *split_k);

/*
 * gba_select_tile -- the tile configuration gemm_bias_act would use for this
 * problem on its aligned fast path (host-only computation, no GPU access).
 * Returns the tile id, or -1 if the arguments are invalid or the problem is
 * smaller than every tile (M < 32 or N < 32: general path).
 */
int gba_select_tile(gba_layout layoutA, gba_layout layoutB, int64_t M, int64_t N, int64_t K,
                    gba_acc accum);

/*
 * Unfused baseline pieces (the separate-kernel chain that the paper's
 * evaluation compares against: a GEMM, then a bias add, then an
 * activation).  Same conventions as above; C is row-major M x N with
 * leading dimension ldc >= N and is updated in place:
 *   gba_bias_add_f16: C[i*ldc+j] = fp16(C[i*ldc+j] + bias[j])  (fp32 add)
 *   gba_relu_f16:     C[i*ldc+j] = max(C[i*ldc+j], 0)
 * Errors: GBA_EINVAL for negative sizes, ldc < N, NULL C or bias when the
 * work is non-empty; GBA_EUNSUPPORTED for sizes above 2^31-1 or pointers
 * not 2-byte aligned; GBA_EHIP if the launch fails.
 */
gba_status gba_bias_add_f16(int64_t M, int64_t N, void *C, int64_t ldc, const void *bias,
                            gba_stream_t stream);
gba_status gba_relu_f16(int64_t M, int64_t N, void *C, int64_t ldc, gba_stream_t stream);

/* Static, human-readable name of a status code. */
const char *gba_status_string(gba_status status);

/* Library version string, e.g. "gba 0.1.0 gfx950". */
const char *gba_version(void);

#ifdef __cplusplus
}
#endif

#endif /* GBA_H */
