/*
 * gba.h -- fused fp16 GEMM + bias + activation for AMD MI355X (gfx950).
 *
 * C ABI of libgba.so.  Plain pointers and sizes only; C99 compatible.
 *
 * The headline operation is the matmul followed by the pointwise
 * ReLU-of-add statement of the paper's Problem Statement section (Listing 1
 * and its expression tree, whose root is ReLU over the add of the matmul
 * result and the bias), computed in ONE kernel so the matmul result never
 * goes to global memory (Kernel Fusion section, "Pointwise Operations in
 * Epilogue").  gba_fused_gemm adds the section's other idioms: a ReLU
 * prologue, a second matmul feeding the epilogue, a full or subtracted bias
 * and the Sigmoid and Tanh activations.
 * Operands may be row- or column-major, the four layout specialisations of
 * the Matmul Compute Decomposition section.
 *
 * Common conventions for every entry point below:
 *   - All array pointers are DEVICE pointers (memory the caller allocated on
 *     the GPU that is current for `stream`).  fp16 means IEEE binary16.
 *   - The caller owns every buffer.  The library never allocates, frees or
 *     synchronises; it keeps no mutable global state and is thread-safe.
 *     The one exception is gba_fused_gemm_noalloc, which uses a static
 *     device array of the library's own (see there).
 *   - Calls are asynchronous: work is enqueued on `stream` (NULL = the null
 *     stream) and the function returns once the kernel is launched.
 *   - Arguments are validated on the host before anything is enqueued.  On
 *     any error nothing is launched and the output is left untouched.
 *   - Outputs must not alias inputs.
 *   - Inputs are expected to be finite.  The outputs for NaN or infinite
 *     inputs, and for results beyond the fp16 range, are not specified.
 */
#ifndef GBA_H
#define GBA_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ABI-identical to hipStream_t. */
typedef struct ihipStream_t *gba_stream_t;

typedef enum { GBA_ROW_MAJOR = 0, GBA_COL_MAJOR = 1 } gba_layout;
/* Epilogue activation (the pointwise ops of the Introduction's scope):
 * identity, ReLU max(x, 0), Sigmoid 1 / (1 + exp(-x)), Tanh. */
typedef enum { GBA_ACT_NONE = 0, GBA_ACT_RELU = 1, GBA_ACT_SIGMOID = 2, GBA_ACT_TANH = 3 } gba_act;
typedef enum { GBA_ACC_F32 = 0, GBA_ACC_F16 = 1 } gba_acc;
typedef enum {
    GBA_OK = 0,
    GBA_EINVAL = 1,        /* malformed argument (negative size, ld too small, NULL, bad enum) */
    GBA_EUNSUPPORTED = 2,  /* well-formed but outside what the library implements */
    GBA_EHIP = 3,          /* the HIP runtime reported an error at launch */
    GBA_ESCRATCH = 4       /* gba_fused_gemm_noalloc: the request needs more scratch than
                              GBA_NOALLOC_SCRATCH_BYTES */
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
 * The bias add and activation are done in fp32 and rounded once to fp16
 * (RNE).  act may also be GBA_ACT_SIGMOID or GBA_ACT_TANH (see
 * gba_fused_gemm for their accuracy).
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

/* Left-operand prologue (Listing 4, ReLU + Matmul). */
typedef enum { GBA_PRO_NONE = 0, GBA_PRO_RELU = 1 } gba_prologue;
/* Second product (Listing 5, Sum of Matmuls): none, A.B + P.Q, A.B - P.Q. */
typedef enum { GBA_SECOND_NONE = 0, GBA_SECOND_ADD = 1, GBA_SECOND_SUB = 2 } gba_second;
/* Bias shape: none, fp16[N] broadcast over rows, or a full M x N fp16 tile. */
typedef enum { GBA_BIAS_NONE = 0, GBA_BIAS_ROW = 1, GBA_BIAS_FULL = 2 } gba_bias_kind;
/* Add or subtract the bias. */
typedef enum { GBA_OP_ADD = 0, GBA_OP_SUB = 1 } gba_op;

/*
 * gba_fused_desc -- one request of gba_fused_gemm.  Fill it with
 * gba_fused_desc_init first (which selects: row-major A and B, no prologue,
 * no second product, no bias, no activation, fp32 accumulation, library tile
 * choice), then set what the request needs.  Every pointer is a DEVICE
 * pointer; a field that the request does not use is ignored.
 */
typedef struct gba_fused_desc {
    gba_layout layoutA, layoutB;  /* also the layouts of P and Q */
    int64_t M, N, K;
    const void *A;                /* A(i,k): ROW A[i*lda+k] (lda >= K), COL A[k*lda+i] (lda >= M) */
    int64_t lda;
    const void *B;                /* B(k,j): ROW B[k*ldb+j] (ldb >= N), COL B[j*ldb+k] (ldb >= K) */
    int64_t ldb;
    gba_prologue prologue;        /* applied to A and, with a second product, to P */
    gba_second second;
    int64_t K2;                   /* reduction length of P.Q */
    const void *P;                /* M x K2, stored like A with leading dimension ldp */
    int64_t ldp;
    const void *Q;                /* K2 x N, stored like B with leading dimension ldq */
    int64_t ldq;
    gba_bias_kind bias_kind;
    gba_op bias_op;
    const void *bias;             /* ROW: bias[j]; FULL: bias[i*ldbias + j], ldbias >= N */
    int64_t ldbias;
    gba_act act;
    gba_acc accum;
    void *C;                      /* output, row-major: C[i*ldc + j], ldc >= N */
    int64_t ldc;
    int tile_id;                  /* < 0: library's choice; else as gemm_bias_act_tile */
    int split_k;                  /* 0: library's choice, 1: never, s >= 2: s-way (see below) */
    void *workspace;              /* device memory for a split reduction, or NULL */
    size_t workspace_bytes;
} gba_fused_desc;

/* Set *desc to the defaults listed above (tile_id = -1, split_k = 0, no
 * workspace, everything else zero / NONE / ADD / F32).  NULL is ignored. */
void gba_fused_desc_init(gba_fused_desc *desc);

/*
 * gba_fused_workspace_size -- bytes of workspace the request would use to
 * split its reduction across workgroups (0: it would not split).
 *
 * Splitting is an implementation choice of the fast path for fp32
 * accumulation (the paper partitions the reduction only inside a thread
 * block; this is the same partition across blocks): when an output has too
 * few tiles to occupy the GPU, or a long reduction, each output tile's
 * reduction steps (A.B's, then P.Q's) are divided among up to split_k
 * workgroups.  Each writes its fp32 partial tile to the workspace; the last
 * of a tile's splits to finish adds the partials in split order (the result
 * does not depend on which finishes last) and runs the epilogue.  Only the
 * summation order changes, not the tolerance; GBA_ACC_F16 never splits.
 *
 * Workspace contract (gba_fused_gemm): at least this many bytes, 256-byte
 * aligned, on the device the call runs on, and all zero when the call is
 * enqueued.  A call that splits uses it for one 32-bit counter per output
 * tile followed by the fp32 partial tiles, and leaves every byte it used
 * at zero again when it completes, so a workspace zero-filled once serves
 * any number of calls in stream order, whatever their shapes and tiles;
 * calls that may run at the same time need separate workspaces.  With a NULL or smaller workspace the
 * call runs unsplit.  split_k >= 2 asks for that many splits (fewer when
 * the reduction has fewer 64-deep steps); 0 lets the library decide.
 *
 * Errors: as gba_fused_gemm's validation; GBA_EINVAL also for bytes ==
 * NULL or split_k < 0.
 */
gba_status gba_fused_workspace_size(const gba_fused_desc *desc, size_t *bytes);

/*
 * gba_fused_tile -- the tile configuration gba_fused_gemm would run the
 * request on, given the workspace the descriptor carries (host-only
 * computation, no GPU access): *tile is the tile id (see gba_tile_info), or
 * -1 for the general path and for an empty output.  The library's choice
 * depends on the shape, the layouts, the accumulation and the prologue (see
 * gba_select_tile); a requested tile_id that fits is kept.
 *
 * Errors: as gba_fused_gemm's validation; GBA_EINVAL also for tile == NULL.
 */
gba_status gba_fused_tile(const gba_fused_desc *desc, int *tile);

/*
 * gba_fused_gemm -- the four computation idioms of the paper's scope
 * (Introduction) in one kernel: a matmul with a pointwise prologue
 * (Pointwise Operations in Prologue, Listing 4), with a pointwise epilogue
 * (Pointwise Operations in Epilogue, Listing 1), and two matmuls of the same
 * output shape feeding a pointwise op (Matmuls with Pointwise Epilogue,
 * Listing 5).  For 0<=i<M, 0<=j<N:
 *
 *     pro(x)   = prologue == GBA_PRO_RELU ? max(x, 0) : x
 *     Cp(i,j)  = sum_{k<K}  pro(A(i,k)) * B(k,j)
 *     R(i,j)   = sum_{k<K2} pro(P(i,k)) * Q(k,j)                 (second != NONE)
 *     Z(i,j)   = Cp + R (SECOND_ADD), Cp - R (SECOND_SUB), Cp (SECOND_NONE)
 *     pre(i,j) = Z +/- bias(i,j)   (bias_op; no term for GBA_BIAS_NONE)
 *     C[i*ldc + j] = fp16(act(pre))
 *
 * Neither Cp nor R ever reaches global memory: both products are summed in
 * ONE fp32 running sum per output (A.B's terms, then P.Q's, negated for
 * SECOND_SUB), so the P.Q operands may have a different reduction length
 * K2 as long as the output shape matches.  GBA_ACC_F16 rounds that running
 * sum to fp16 after every aligned group of 32 k values of each product.
 * The bias term and activation are evaluated in fp32 and the result rounded
 * once to fp16 (RNE).  Sigmoid and Tanh use the hardware exp2 and
 * reciprocal approximations (Tanh from its Taylor series for |x| < 1/16):
 * within a few fp32 ulps of the result, far below the fp16 rounding.
 *
 * Fast path: 16-byte aligned A, B, C and (if used) P, Q, bias; lda, ldb,
 * ldc (and ldp, ldq, ldbias when used) multiples of 8 and below 2^21 for
 * the operands; N and the contiguous extents of all operands multiples of 8.
 * Anything else takes the general kernel.  Outputs must not alias inputs.
 *
 * Degenerate sizes: M == 0 or N == 0 -> GBA_OK, nothing launched; K == 0
 * or K2 == 0 make that product's empty sum zero.
 * Reduction split across workgroups: see gba_fused_workspace_size.
 *
 * Errors: GBA_EINVAL for desc == NULL, a bad enum, a tile_id at or beyond
 * gba_num_tiles(), negative sizes or leading dimensions, a leading
 * dimension below its extent, a NULL pointer that the request reads
 * (A/B when K > 0, P/Q when K2 > 0, bias when bias_kind != NONE, C),
 * split_k < 0, or a workspace not 256-byte aligned;
 * GBA_EUNSUPPORTED for M, N, K or K2 above 2^31-1 or pointers not 2-byte
 * aligned; GBA_EHIP if the launch fails.  Nothing is launched on error.
 */
gba_status gba_fused_gemm(const gba_fused_desc *desc, gba_stream_t stream);

/*
 * gba_fused_gemm_noalloc -- gba_fused_gemm for callers that cannot allocate
 * device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc).  Same request, same result bits as
 * gba_fused_gemm given a workspace of at least gba_fused_workspace_size
 * bytes; desc->workspace and desc->workspace_bytes are ignored.
 *
 * When the request splits its reduction across workgroups, the split's
 * workspace is the library's own static device array of
 * GBA_NOALLOC_SCRATCH_BYTES bytes (one per GPU, created with the library's
 * code object and held until the process ends); its counters are cleared by
 * a small kernel on `stream` before the split kernel.  Requests that do not
 * split use no scratch.  The call allocates nothing (no hipMalloc, no
 * allocating library routine); its first call on a device looks up that
 * device's scratch address once, with the device current.
 *
 * Every call on one GPU shares that GPU's scratch, which keeps the last
 * call's contents: calls that may overlap on one GPU (different streams,
 * different host threads without ordering) race on it and give undefined
 * results.  Calls in one stream's order are safe.
 *
 * Errors: as gba_fused_gemm; GBA_ESCRATCH (nothing launched) when the split
 * the request asks for (or the library chooses) needs more than
 * GBA_NOALLOC_SCRATCH_BYTES; GBA_EUNSUPPORTED for a device index >= 64.
 */
#define GBA_NOALLOC_SCRATCH_BYTES ((size_t)16 << 20)
gba_status gba_fused_gemm_noalloc(const gba_fused_desc *desc, gba_stream_t stream);

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
 * gba_fused_gemm makes the same choice for requests without the prologue
 * (K being the total reduction length of both products); with the prologue
 * it may take another tile.  Returns the tile id, or -1 if the arguments
 * are invalid or the problem is smaller than every tile (M < 32 or N < 32:
 * general path).
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
 *   gba_add_f16:      C[i*ldc+j] = fp16(C[i*ldc+j] + X[i*ldx+j])  (fp32 add;
 *                     the separate add of two matmul results, Listing 5)
 *   gba_bias_act_f16: C[i*ldc+j] = fp16(act(C[i*ldc+j] + bias[j]))  (fp32;
 *                     the bias add and activation in one pass: the second
 *                     kernel of a two-launch chain, GEMM then bias+act)
 * Errors: GBA_EINVAL for negative sizes, ldc < N (or ldx < N), NULL C, bias
 * or X when the work is non-empty, a bad act; GBA_EUNSUPPORTED for sizes above 2^31-1
 * or pointers not 2-byte aligned; GBA_EHIP if the launch fails.
 */
gba_status gba_bias_add_f16(int64_t M, int64_t N, void *C, int64_t ldc, const void *bias,
                            gba_stream_t stream);
gba_status gba_relu_f16(int64_t M, int64_t N, void *C, int64_t ldc, gba_stream_t stream);
gba_status gba_bias_act_f16(int64_t M, int64_t N, void *C, int64_t ldc, const void *bias,
                            gba_act act, gba_stream_t stream);
gba_status gba_add_f16(int64_t M, int64_t N, void *C, int64_t ldc, const void *X, int64_t ldx,
                       gba_stream_t stream);

/* Static, human-readable name of a status code. */
const char *gba_status_string(gba_status status);

/* Library version string, e.g. "gba 0.1.0 gfx950". */
const char *gba_version(void);

#ifdef __cplusplus
}
#endif

#endif /* GBA_H */
