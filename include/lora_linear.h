/*
 * lora_linear.h -- C ABI of the LoRA-adapted linear layer for AMD MI355X (gfx950).
 *
 * The operation is Eq. 1 of JORA (arXiv 2403.11366, Section 3, "Model Transfer
 * API"): output = W0 x + b0 + B A x, where W0 is a frozen weight and the rank-r
 * factors B and A are the only trainable parameters.  This library evaluates it
 * row-major over m tokens, without bias, with the conventional LoRA scale
 * s = alpha / r (the configuration of Listing 3 carries LORA_R and LORA_ALPHA):
 *
 *     U  = X A^T                 [m, r]   (saved for the backward)
 *     Y  = X W^T + s U B^T       [m, n]
 *
 * and its chain-rule backward for an upstream gradient dY (W0 frozen: no dW):
 *
 *     dU = s dY B,  dX = dY W + dU A,  dB = s dY^T U,  dA = dU^T X.
 *
 * Conventions shared by every entry point:
 *   - Matrices are dense, row-major, leading dimension = row length.
 *   - Matrix pointers are DEVICE pointers (hipMalloc'd or from a framework's
 *     device allocator) and must be 16-byte aligned.  The caller owns every
 *     buffer, including the workspace; the library allocates nothing, frees
 *     nothing and never synchronises.
 *   - bfloat16 values are passed as raw 16-bit patterns (lora_bf16).
 *   - Shapes: m >= 1 (any value; tails are masked); n, k >= 8 and multiples of
 *     8 (rows must be 16-byte aligned); 1 <= r <= 64.
 *   - `stream` is a hipStream_t (NULL = the default stream).  Calls enqueue
 *     kernels on it and return; results are valid once the stream has been
 *     synchronised.  Calls that share buffers must be ordered by the caller.
 *   - Outputs are overwritten (no accumulation into existing contents).
 *   - All arguments are validated before anything is enqueued.  On an error
 *     nothing is launched and every output is left untouched, except when a
 *     launch itself fails (LORA_ERR_HIP): kernels of the call enqueued before
 *     it may run.  No C++ exception crosses this interface.
 *   - Arithmetic: bf16 operands, fp32 accumulation on the matrix cores, bf16
 *     outputs rounded to nearest-even.  The rank-r intermediates U and dU enter
 *     the matrix cores as a bf16 high part plus a bf16 low part, so they keep
 *     about 16 significant bits.  Reductions use a fixed order: repeated calls
 *     on the same inputs give bit-identical results.
 */
#ifndef LORA_LINEAR_H
#define LORA_LINEAR_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef uint16_t lora_bf16;

typedef enum {
  LORA_OK = 0,
  LORA_ERR_NULL = 1,        /* a required pointer is NULL */
  LORA_ERR_SHAPE = 2,       /* m < 1, n or k < 8 or not a multiple of 8, r < 1, merge sign not +-1 */
  LORA_ERR_ALIGN = 3,       /* a matrix pointer is not 16-byte aligned */
  LORA_ERR_UNSUPPORTED = 4, /* r > 64, or a dimension beyond the supported range */
  LORA_ERR_WORKSPACE = 5,   /* workspace missing or smaller than lora_linear_bwd_workspace_size() */
  LORA_ERR_ALIAS = 6,       /* an output overlaps an input or another output */
  LORA_ERR_HIP = 7          /* the HIP runtime reported an error at launch; also returned, before anything
                               is enqueued, while an error of an earlier HIP call is pending on the calling
                               thread (hipPeekAtLastError; it is left for the caller to read) */
} lora_status;

/*
 * Forward of Eq. 1 (Section 3): Y = X W^T + (alpha/r) (X A^T) B^T, and U = X A^T.
 *
 *   X  [m, k]  layer input (bf16), read only
 *   W  [n, k]  frozen weight W0, stored [out, in] (bf16), read only
 *   A  [r, k]  LoRA down projection (bf16), read only
 *   B  [n, r]  LoRA up projection (bf16), read only
 *   Y  [m, n]  output (bf16), written
 *   U  [m, r]  output (fp32), written: the unscaled X A^T, needed by the backward
 *   alpha      LoRA alpha; the scale is s = alpha / r, computed in fp32
 *
 * A bf16 matrix-core GEMM over k that streams each X tile through LDS once
 * for both W and A, then adds s U B^T to the accumulators in its epilogue
 * before rounding Y to bf16.  One launch for most shapes; where it fills the
 * compute units better, the output columns are split between two launches
 * of different tile sizes, and for r > 16 a pass computing U runs first.
 */
lora_status lora_linear_fwd(const lora_bf16* X, const lora_bf16* W, const lora_bf16* A,
                            const lora_bf16* B, lora_bf16* Y, float* U,
                            int64_t m, int64_t n, int64_t k, int64_t r, float alpha,
                            void* stream);

/*
 * Forward with LoRA dropout on the adapter input (the configuration of
 * Listing 3 carries LORA_DROPOUT = 0.05; the dropout acts on the input of A,
 * while the frozen W0 sees x unchanged):
 *
 *     D = keep * X / (1 - p),   U = D A^T,   Y = X W^T + (alpha/r) U B^T
 *
 *   keep  [m, k/8] bytes, device: bit (l % 8) of byte (i, l / 8) set keeps
 *         X[i][l] in D.  The mask is an input (the caller draws it, for
 *         instance from a Bernoulli(1 - p) source); the backward must be given
 *         the same mask.  16-byte aligned, read only.
 *   p     dropout rate, 0 <= p < 1 (else LORA_ERR_SHAPE)
 *   other arguments as in lora_linear_fwd; U is the dropped U = D A^T.
 * Requires k % 64 == 0 (LORA_ERR_SHAPE otherwise).  The mask zeroes X
 * elements of the U operand on the matrix cores; 1 / (1 - p) is applied to U
 * in fp32.
 */
lora_status lora_linear_fwd_dropout(const lora_bf16* X, const lora_bf16* W, const lora_bf16* A,
                                    const lora_bf16* B, const uint8_t* keep, float p, lora_bf16* Y, float* U,
                                    int64_t m, int64_t n, int64_t k, int64_t r, float alpha, void* stream);

/*
 * Keep mask for the *_dropout entry points, drawn on the device (Listing 3
 * carries LORA_DROPOUT; the mask is what the dropout of the adapter input
 * draws).  Writes keep [m, k/8] in the layout those entry points read: bit
 * (l % 8) of byte (i, l / 8) set keeps X[i][l].
 *
 * Generator: the counter-based Philox4x64-10 (Salmon, Moraes, Dror, Shaw,
 * "Parallel random numbers: as easy as 1, 2, 3", SC 2011), key (seed, 0).
 * Bytes 2t and 2t + 1 of the mask (byte b = i (k/8) + l/8 holds the bits of
 * elements l .. l + 7 of row i, l a multiple of 8) come from one generator
 * block at the 256-bit counter (offset + t as a 128-bit integer, 0, 0); its
 * four 64-bit output words give sixteen 16-bit values u_e (u_{4h+j} = bits
 * 16j .. 16j + 15 of word h), and bit e of the byte pair (e = 0..7 in byte
 * 2t, 8..15 in byte 2t + 1) is set iff u_e < floor((1 - p) 2^16 + 1/2)
 * (computed in double from the float p).  Every element is kept independently
 * with probability 1 - p up to that rounding (2^-16), exactly for p = 0.  The
 * call uses the counters offset .. offset + ceil(m k / 16) - 1: for a fresh
 * mask per step, advance offset by that count (or change the seed).
 *
 *   seed, offset  generator key word and first counter
 *   p             dropout rate, 0 <= p < 1 (else LORA_ERR_SHAPE)
 *   keep          DEVICE buffer of m * k / 8 bytes, 16-byte aligned, written
 *   m, k          rows and columns of the X the mask is for (k a multiple of 8)
 * The result depends only on (seed, offset, p, m, k).
 */
lora_status lora_dropout_keep_mask(uint64_t seed, uint64_t offset, float p, uint8_t* keep, int64_t m, int64_t k,
                                   void* stream);

/*
 * Bytes of device workspace lora_linear_bwd needs for this shape (0 on an
 * invalid shape).  The workspace holds transposed and split copies of the
 * rank-r operands and the fixed-order split-K partial sums of dA and dB.
 */
size_t lora_linear_bwd_workspace_size(int64_t m, int64_t n, int64_t k, int64_t r);

/*
 * Backward of Eq. 1 for the trainable A and B (Section 3: B and A are the
 * trainable weights; W0 is frozen, so no dW is formed).
 *
 *   dY [m, n]  upstream gradient (bf16), read only
 *   X  [m, k]  the forward's input (bf16), read only
 *   W, A, B    as in lora_linear_fwd, read only
 *   U  [m, r]  the forward's U output (fp32), read only
 *   dX [m, k]  output (bf16), written:  dY W + dU A, with dU = s dY B
 *   dA [r, k]  output (fp32), written:  dU^T X
 *   dB [n, r]  output (fp32), written:  s dY^T U
 *   workspace  device buffer of at least lora_linear_bwd_workspace_size(m,n,k,r)
 *              bytes, 16-byte aligned; contents on entry are ignored.  It must not
 *              be used concurrently by another call.
 */
lora_status lora_linear_bwd(const lora_bf16* dY, const lora_bf16* X, const lora_bf16* W,
                            const lora_bf16* A, const lora_bf16* B, const float* U,
                            lora_bf16* dX, float* dA, float* dB,
                            void* workspace, size_t workspace_bytes,
                            int64_t m, int64_t n, int64_t k, int64_t r, float alpha,
                            void* stream);

/*
 * lora_linear_bwd without a workspace argument, for callers that cannot
 * allocate device memory: code being captured into a HIP graph, tight
 * serving loops, harnesses that forbid allocation.  Same arguments (minus the
 * workspace), outputs, definitions and errors as lora_linear_bwd.
 *
 * The workspace is a fixed array of LORA_NOALLOC_SCRATCH_BYTES bytes inside
 * this library, one per GPU, kept until the process ends; its device address
 * is looked up on the first call on each device (with that device current).
 * The call allocates and frees nothing.  Shapes whose workspace
 * (lora_linear_bwd_workspace_size) exceeds LORA_NOALLOC_SCRATCH_BYTES return
 * LORA_ERR_WORKSPACE before anything is enqueued; every Llama-2 projection
 * shape of up to 8192 tokens fits.  All calls on one GPU share its array:
 * calls whose kernels may overlap in time on one GPU (other streams, other
 * threads) race on it and must be ordered by the caller; a call's result
 * depends only on its own arguments (no part of the array needs clearing).
 */
#define LORA_NOALLOC_SCRATCH_BYTES ((size_t)32 << 20)

lora_status lora_linear_bwd_noalloc(const lora_bf16* dY, const lora_bf16* X, const lora_bf16* W,
                                    const lora_bf16* A, const lora_bf16* B, const float* U,
                                    lora_bf16* dX, float* dA, float* dB,
                                    int64_t m, int64_t n, int64_t k, int64_t r, float alpha,
                                    void* stream);

/*
 * Bytes of device workspace lora_linear_bwd_fused needs for this shape (0 on
 * an invalid shape or r > 16): dU^T in bf16 high and low parts, the dB
 * partials of the dX launch (one per 128-token tile row) and the split-K
 * partials of dA.
 */
size_t lora_linear_bwd_fused_workspace_size(int64_t m, int64_t n, int64_t k, int64_t r);

/*
 * The same backward as lora_linear_bwd (same arguments, outputs and
 * definitions) with dU and dB formed inside the dX GEMM from the dY tiles it
 * already stages: the rank-r products dU = s dY B ride as extra matrix-core
 * products on the GEMM's k loop over n, and the dB = s dY^T U partials of
 * each 128-token tile row are formed at every tiles_n-th stage; a token
 * reduction for dA = dU^T X and a fixed-order finalize follow (three
 * launches, no separate pass over dY).  Results agree with lora_linear_bwd
 * to rounding (the sums run in a different fixed order) and are
 * bit-identical from run to run.
 *
 * Requires r <= 16 (LORA_ERR_UNSUPPORTED otherwise); the workspace is
 * lora_linear_bwd_fused_workspace_size(m, n, k, r) bytes, 16-byte aligned.
 * Other errors as in lora_linear_bwd.
 */
lora_status lora_linear_bwd_fused(const lora_bf16* dY, const lora_bf16* X, const lora_bf16* W,
                                  const lora_bf16* A, const lora_bf16* B, const float* U,
                                  lora_bf16* dX, float* dA, float* dB,
                                  void* workspace, size_t workspace_bytes,
                                  int64_t m, int64_t n, int64_t k, int64_t r, float alpha,
                                  void* stream);

/*
 * Backward of lora_linear_fwd_dropout for the same keep mask and rate:
 *
 *     dU = s dY B,  dX = dY W + keep * (dU A) / (1 - p),
 *     dB = s dY^T U,  dA = dU^T D  with  D = keep * X / (1 - p)
 *
 * Arguments as in lora_linear_bwd plus keep and p as in
 * lora_linear_fwd_dropout (U must be that forward's U).  The workspace size is
 * lora_linear_bwd_workspace_size(m, n, k, r).  Requires k % 64 == 0.
 */
lora_status lora_linear_bwd_dropout(const lora_bf16* dY, const lora_bf16* X, const lora_bf16* W,
                                    const lora_bf16* A, const lora_bf16* B, const float* U, const uint8_t* keep,
                                    float p, lora_bf16* dX, float* dA, float* dB, void* workspace,
                                    size_t workspace_bytes, int64_t m, int64_t n, int64_t k, int64_t r, float alpha,
                                    void* stream);

/*
 * Merge (sign = +1) or unmerge (sign = -1) of the adapter into the frozen
 * weight, following the second form of Eq. 1 (Section 3): W0 x + B A x =
 * (W0 + B A) x.  With the scale s = alpha / r:
 *
 *     W_out = W + sign * s * B A            [n, k]
 *
 *   W      [n, k]  frozen weight (bf16), read only
 *   A      [r, k]  LoRA down projection (bf16), read only
 *   B      [n, r]  LoRA up projection (bf16), read only
 *   W_out  [n, k]  output (bf16), written; it may be W itself (in-place merge),
 *                  but any other overlap with an input is LORA_ERR_ALIAS
 *   sign   +1 or -1 (anything else is LORA_ERR_SHAPE)
 *
 * The rank-r product runs on the matrix cores with fp32 accumulation; the sum
 * with W is formed in fp32 and rounded once to bf16 (nearest-even).  Because
 * of that rounding, unmerging a merged weight returns W only up to bf16
 * rounding.  The shape rules are those above with no m.
 */
lora_status lora_linear_merge(const lora_bf16* W, const lora_bf16* A, const lora_bf16* B, lora_bf16* W_out,
                              int64_t n, int64_t k, int64_t r, float alpha, int sign, void* stream);

/*
 * Grouped forward of projections that read one input (the query, key and value
 * projections of an attention block, or gate and up of an MLP; Section 3
 * adapts the query and value projections): for g = 0 .. group-1,
 *
 *     U_g = X A_g^T,   Y_g = X W_g^T + (alpha/r) U_g B_g^T
 *
 *   X       [m, k] device, shared input (bf16), read only
 *   group   number of projections, 1 .. 8 (0 or less: LORA_ERR_SHAPE; more than
 *           8: LORA_ERR_UNSUPPORTED)
 *   n       HOST array [group]: output features n_g of each projection (the
 *           shape rules above apply to each; their sum is at most 2^22)
 *   W, A, B HOST arrays [group] of device pointers: W_g [n_g, k], A_g [r, k],
 *           B_g [n_g, r] (bf16), read only
 *   Y, U    HOST arrays [group] of device pointers: Y_g [m, n_g] (bf16) and
 *           U_g [m, r] (fp32), written
 *   r, alpha  one rank and alpha for the group
 * One kernel launch: the output tiles of all projections form one grid, so the
 * group fills the chip as one problem of m x (sum of n_g) outputs.  Each Y_g,
 * U_g equals what lora_linear_fwd computes for projection g.  No output may
 * overlap any input or another output.
 */
lora_status lora_linear_group_fwd(const lora_bf16* X, int64_t group, const int64_t* n,
                                  const lora_bf16* const* W, const lora_bf16* const* A,
                                  const lora_bf16* const* B, lora_bf16* const* Y, float* const* U,
                                  int64_t m, int64_t k, int64_t r, float alpha, void* stream);

/*
 * Bytes of device workspace lora_linear_group_bwd needs (0 on invalid
 * arguments): the sum over the group of each projection's backward workspace.
 */
size_t lora_linear_group_bwd_workspace_size(int64_t group, const int64_t* n, int64_t m, int64_t k, int64_t r);

/*
 * Backward of lora_linear_group_fwd.  X feeds every projection, so its
 * gradient is the sum of their contributions:
 *
 *     dX = sum_g (dY_g W_g + dU_g A_g),   dU_g = s dY_g B_g,
 *     dB_g = s dY_g^T U_g,   dA_g = dU_g^T X
 *
 *   dY      HOST array [group] of device pointers dY_g [m, n_g] (bf16), read only
 *   X, group, n, W, A, B, r, alpha   as in lora_linear_group_fwd
 *   U       HOST array [group] of device pointers: the forward's U_g [m, r] (fp32)
 *   dX      [m, k] device (bf16), written: the summed input gradient
 *   dA, dB  HOST arrays [group] of device pointers dA_g [r, k], dB_g [n_g, r]
 *           (fp32), written
 *   workspace  at least lora_linear_group_bwd_workspace_size(...) bytes, 16-byte
 *              aligned, not used concurrently by another call
 * dX is one matrix-core GEMM over the concatenated contraction of all
 * projections (one bf16 rounding of the whole sum); dA_g and dB_g equal what
 * lora_linear_bwd computes for projection g.
 */
lora_status lora_linear_group_bwd(const lora_bf16* const* dY, const lora_bf16* X, int64_t group, const int64_t* n,
                                  const lora_bf16* const* W, const lora_bf16* const* A,
                                  const lora_bf16* const* B, const float* const* U, lora_bf16* dX,
                                  float* const* dA, float* const* dB, void* workspace, size_t workspace_bytes,
                                  int64_t m, int64_t k, int64_t r, float alpha, void* stream);

/*
 * Launch plan of a call (host only: no GPU, no HIP call, nothing enqueued).
 * Reports, in launch order, the kernels the entry point named by `op` would
 * launch for these shapes -- the same plan the entry point itself executes --
 * so that tools and tests can tell which kernel variant serves a shape.
 *
 *   op        which entry point (lora_op below)
 *   group, n  the output widths: for single-projection ops group = 1 and n
 *             points to n; for the grouped ops as in lora_linear_group_fwd
 *   m, k, r   as in the entry point (m is ignored for LORA_OP_MERGE)
 *   out       HOST array of `capacity` entries (may be NULL when capacity is 0)
 * Returns the number of launches (entries beyond `capacity` are not written),
 * or minus the lora_status the entry point would return for these shapes
 * (shape rules only: no pointer checks).
 */
typedef enum {
  LORA_OP_FWD = 0,          /* lora_linear_fwd */
  LORA_OP_FWD_DROPOUT = 1,  /* lora_linear_fwd_dropout */
  LORA_OP_BWD = 2,          /* lora_linear_bwd */
  LORA_OP_BWD_DROPOUT = 3,  /* lora_linear_bwd_dropout */
  LORA_OP_BWD_FUSED = 4,    /* lora_linear_bwd_fused */
  LORA_OP_MERGE = 5,        /* lora_linear_merge */
  LORA_OP_GROUP_FWD = 6,    /* lora_linear_group_fwd */
  LORA_OP_GROUP_BWD = 7,    /* lora_linear_group_bwd */
  LORA_OP_KEEP_MASK = 8     /* lora_dropout_keep_mask (m, k; n and r ignored) */
} lora_op;

typedef struct {
  char kernel[128];         /* the instantiation as profilers print it, e.g.
                               "lora::lora_bwd_dx_kernel<128, 256, 2, 4, 16, false, false, true>" */
  int64_t grid;             /* workgroups */
  int32_t block;            /* threads per workgroup */
  int32_t tile_m, tile_n;   /* GEMM output tile (tokens x features), 0 for other kernels */
  int32_t member;           /* grouped backward: projection served by a per-projection launch */
  int64_t col_begin;        /* GEMM output columns [col_begin, col_end) of a single projection */
  int64_t col_end;
} lora_launch_info;

int64_t lora_linear_plan(lora_op op, int64_t group, const int64_t* n, int64_t m, int64_t k, int64_t r,
                         lora_launch_info* out, int64_t capacity);

/* Static, human-readable name of a status code. */
const char* lora_status_string(lora_status s);

#ifdef __cplusplus
}
#endif

#endif /* LORA_LINEAR_H */
