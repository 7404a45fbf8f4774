/*
 * partir.h -- C ABI of libpartir: executing PartIR:Core loops on one MI355X.
 *
 * PartIR:Core (arXiv 2401.11202, Sec. 5) expresses a partitioned tensor
 * program with a pure loop over a mesh axis of size R whose action is either
 *   #tile<d>  -- the iteration results are concatenated along dim d, or
 *   #sum      -- the iteration results are summed,
 * and with `slice d x[r]`, the r-th of R equal contiguous chunks of x along
 * dim d (semantics: App. C, figure "Interpretation of PartIR:Core"; typing
 * rules TTile / TSum / TSlice in the figure "abstract syntax and typing
 * rules").  Every entry point below evaluates all R virtual shards of such a
 * loop nest on the calling GPU:
 *   - a slice is a zero-copy view (base pointer + offset, same leading dim);
 *   - a #tile result is written by each shard straight into its slice of the
 *     output (the all_gather of the SPMD lowering, Sec. 6.1, becomes an
 *     offset store);
 *   - a #sum is reduced on the device, in shard order r = 0..R-1, either in
 *     the MFMA accumulators of one output tile or through fp32 partials (the
 *     all_reduce of the lowering becomes an in-device reduction).
 *
 * Conventions shared by all entry points
 * --------------------------------------
 * Layout.  Every matrix is row-major with an explicit leading dimension
 *   (elements between consecutive rows).  The weights of partir_mlp_block,
 *   partir_attn_block, partir_decoder_layer and their training and backward
 *   calls are logical W [fan_in, fan_out], row-major: `slice 1 W[m]` is a
 *   block of its columns and `slice 0 W[m]` a block of its rows, both views,
 *   and the GEMMs read them in place (transposed LDS reads form the MFMA
 *   operand).  The device-local entry points (*_sharded) take their weight
 *   parts from W^T [fan_out, fan_in] instead, as each declaration states.
 * Memory.  All tensor pointers are device pointers owned by the caller, which
 *   also allocates the workspace (size from the matching *_workspace query;
 *   may be NULL when the query returns 0).  The library allocates no device
 *   memory in these calls and keeps no pointer after a call returns.
 * Alignment.  Base pointers and every row must be 16-byte aligned (leading
 *   dims multiple of 8 for bf16, of 4 for f32), and so must every shard view
 *   (the sliced extent times the element size is a multiple of 16 bytes).
 * Execution.  Work is enqueued on `stream` (a hipStream_t; NULL = the
 *   default stream) and the call returns without waiting.  Results of a
 *   #sum are deterministic: the same inputs give the same bits on every run.
 * Empty operands.  A size of 0 is legal wherever the method allows it: a
 *   zero-size dim slices into R empty shards (TSlice with n_d = 0), a #tile
 *   of empty shards is an empty result (nothing is launched), and a #sum over
 *   an empty contraction (K = 0, F = 0) is the empty sum, so the output is
 *   the epilogue applied to 0 (zeros, the bias, or the unchanged residual).
 *   A pointer may be NULL when its tensor holds no elements or is never read.
 * Errors.  Argument errors are detected before anything is enqueued; the
 *   call then returns the status and leaves every output untouched.  A failed
 *   launch returns PARTIR_E_HIP.  Faults during execution surface at the
 *   caller's next synchronisation.  partir_last_error() gives a thread-local
 *   message for the last failing call on this thread.  No C++ exception
 *   crosses this interface; the library's only mutable global state is that
 *   message, the trace buffer and a per-device property cache.
 */
#ifndef PARTIR_H
#define PARTIR_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum partir_status {
  PARTIR_OK = 0,
  PARTIR_E_NULL = 1,         /* a required pointer is NULL                       */
  PARTIR_E_SHAPE = 2,        /* a size is < 0 / too large, or sizes disagree     */
  PARTIR_E_DIVISIBILITY = 3, /* R does not divide the sliced dim (rule TSlice)   */
  PARTIR_E_AXIS = 4,         /* invalid axis, or one axis both tiled and summed  */
  PARTIR_E_DTYPE = 5,        /* unsupported dtype combination                    */
  PARTIR_E_LAYOUT = 6,       /* leading dim < cols, or 16-byte misalignment      */
  PARTIR_E_WORKSPACE = 7,    /* workspace smaller than the query returns         */
  PARTIR_E_HIP = 8,          /* a HIP runtime call or kernel launch failed       */
  PARTIR_E_UNSUPPORTED = 9   /* R < 1, or an option the library does not provide */
} partir_status;

typedef enum partir_dtype { PARTIR_F32 = 0, PARTIR_BF16 = 1 } partir_dtype;

/* Loop axes of a single matmul C[M,N] = A[M,K] B[K,N]. */
typedef enum partir_axis {
  PARTIR_AXIS_NONE = -1,
  PARTIR_AXIS_M = 0,   /* #tile<0>: slice 0 A[r], result rows concatenated    */
  PARTIR_AXIS_N = 1,   /* #tile<1>: slice 1 B[r], result columns concatenated */
  PARTIR_AXIS_K = 2    /* #sum: slice 1 A[r] and slice 0 B[r], results summed */
} partir_axis;

/* How B is stored for partir_loop_matmul. */
typedef enum partir_b_layout {
  PARTIR_B_KN = 0,     /* B as a row-major [K, N] array (leading dim ldb >= N)          */
  PARTIR_B_NK = 1      /* B given by its transpose, row-major [N, K] (ldb >= K)         */
} partir_b_layout;

/* Realisation of a #sum loop on the device. */
typedef enum partir_sum_impl {
  PARTIR_SUM_AUTO = 0,   /* chosen by the planner from the output tile count              */
  PARTIR_SUM_FUSED = 1,  /* shard K-ranges accumulate, r ascending, in one MFMA accumulator */
  PARTIR_SUM_SPLITK = 2  /* each shard writes an fp32 partial; an ordered reduce sums them  */
} partir_sum_impl;

typedef enum partir_act { PARTIR_ACT_NONE = 0, PARTIR_ACT_GELU_ERF = 1 } partir_act;

/* ------------------------------------------------------------------------ */
/* Single partitioned matmul: the three tile-mapping entries of matmul       */
/* (Sec. 5.2.1, figure matmul-examples).                                      */
/* ------------------------------------------------------------------------ */
/*
 * C[M,N] = A[M,K] @ B[K,N], written as a loop over R virtual shards:
 *   tile_axis = M  : loop [#tile<0>] { matmul(slice 0 A[r], B) }
 *   tile_axis = N  : loop [#tile<1>] { matmul(A, slice 1 B[r]) }
 *   sum_axis  = K  : loop [#sum]     { matmul(slice 1 A[r], slice 0 B[r]) }
 * With both set, the tile loop is outside and the sum loop inside, over two
 * distinct axes of size R each (nesting one axis twice is forbidden,
 * Sec. 5.2.3).  R = 1 is the unpartitioned product.
 *
 * A: [M, K] row-major, leading dim lda >= K.   B: per b_layout, leading dim ldb.
 * C: [M, N] row-major, leading dim ldc >= N, overwritten.
 * Both B layouts are read in place (no transposed copy); a bf16 B given as
 * [K, N] needs N and N/R (with a tile over N) multiples of 8.
 * ab_dtype: PARTIR_F32 or PARTIR_BF16 (A and B alike); c_dtype: PARTIR_F32,
 * or PARTIR_BF16 when ab_dtype is bf16.  Accumulation is fp32.
 * b_layout: partir_b_layout.  sum_impl: partir_sum_impl (ignored without a
 * #sum).  ws / ws_bytes: workspace of at least partir_loop_matmul_workspace().
 * M, N or K may be 0: M = 0 or N = 0 launches nothing; K = 0 writes zeros.
 * Limits: bf16 operands address each block of 64 rows (K-contiguous) or 64
 * K rows (B as [K, N]) through a 32-bit byte range, so lda and ldb are at
 * most 2^24 elements; the output tiles (64 x 64 counted per shard) times R
 * must stay below 2^31.
 * Errors: E_NULL (a non-empty A, B or C NULL, or ws NULL with ws_bytes
 * short), E_SHAPE (a size < 0 or above 2^30, or beyond the limits above),
 * E_DIVISIBILITY (R does not divide the tiled or summed dim), E_AXIS,
 * E_DTYPE, E_LAYOUT, E_WORKSPACE, E_UNSUPPORTED (R < 1), E_HIP.
 */
int partir_loop_matmul(const void* A, const void* B, void* C,
                       int64_t M, int64_t N, int64_t K,
                       int64_t lda, int64_t ldb, int64_t ldc,
                       int ab_dtype, int c_dtype, int b_layout,
                       int tile_axis, int sum_axis, int R, int sum_impl,
                       void* ws, size_t ws_bytes, void* stream);

/* Workspace bytes partir_loop_matmul needs for these arguments (0 if none);
 * returns (size_t)-1 if the arguments are invalid. */
size_t partir_loop_matmul_workspace(int64_t M, int64_t N, int64_t K,
                                    int ab_dtype, int c_dtype, int b_layout,
                                    int tile_axis, int sum_axis, int R, int sum_impl);

/* For callers that cannot allocate (code under HIP graph capture, tight
 * serving loops, harnesses that forbid hipMalloc): partir_loop_matmul with
 * the same arguments except the workspace, which is instead a 64 MiB array
 * in the library's device memory (one per GPU, held until the process
 * ends).  The call allocates nothing (no hipMalloc or hipFree; with kernel
 * tracing off it creates no events either).  A call whose
 * partir_loop_matmul_workspace exceeds 64 MiB returns PARTIR_E_WORKSPACE
 * before anything is enqueued; other errors as partir_loop_matmul.  Every
 * split-K partial and tail part is written in full before it is read, so
 * nothing is cleared between calls, but calls on one GPU share the array:
 * calls that overlap in time on that GPU (different streams, or different
 * host threads) race and must be ordered by the caller.  The current device
 * must be the one `stream` belongs to. */
int partir_loop_matmul_noalloc(const void* A, const void* B, void* C,
                               int64_t M, int64_t N, int64_t K,
                               int64_t lda, int64_t ldb, int64_t ldc,
                               int ab_dtype, int c_dtype, int b_layout,
                               int tile_axis, int sum_axis, int R, int sum_impl,
                               void* stream);

/* ------------------------------------------------------------------------ */
/* Megatron MLP block nested in a batch #tile (Sec. 5.2.2 final listing,      */
/* Sec. 2.3 on model parallelism).                                            */
/* ------------------------------------------------------------------------ */
/*
 * Y = loop b [#tile<0>](R_batch) {
 *       loop m [#sum](R_model) {
 *         act(slice 0 X[b] @ slice 1 W1[m] + slice 0 b1[m]) @ slice 0 W2[m] }
 *       + b2 }
 * X: [T, D] bf16 row-major (ld = D).  W1: [D, F] bf16 and W2: [F, D] bf16,
 * row-major [fan_in, fan_out] (slice 1 W1[m] is a column block, slice 0
 * W2[m] a row block; both are read in place).  b1: [F] f32 or NULL (tiled
 * with W1's columns).  b2: [D] f32 or NULL, added once after the #sum.
 * Y: [T, D], out_dtype F32 or BF16.
 * act: partir_act applied to the first product.  The intermediate
 * H = act(X W1 + b1) ([T, F], stored bf16) lives in the workspace; each model
 * shard m writes its columns [m F/R_model, (m+1) F/R_model) and the second
 * product sums the shards' K-ranges in order.  T = 0 or D = 0 launches
 * nothing; F = 0 (every model shard empty) gives Y = b2 (or 0).
 * Errors: E_NULL, E_SHAPE, E_DIVISIBILITY (R_batch does not divide T or
 * R_model does not divide F), E_DTYPE (in_dtype other than BF16), E_LAYOUT,
 * E_WORKSPACE, E_UNSUPPORTED (R < 1), E_HIP.
 */
int partir_mlp_block(const void* X, const void* W1, const void* b1,
                     const void* W2, const void* b2, void* Y,
                     int64_t T, int64_t D, int64_t F,
                     int in_dtype, int out_dtype, int act,
                     int R_batch, int R_model,
                     void* ws, size_t ws_bytes, void* stream);

/* The MLP block on device-local arrays: the lowered program of the schedule
 * BP + MP + Z3 (Sec. 3: batch tiling, Megatron, parameters sharded over the
 * batch axis) with the input and output activations also sharded over the
 * model axis (the remark after Sec. 3's FSDP chain), run for every device of
 * the mesh {B: R_batch, M: R_model} on this GPU.  Device (b, m) is part index
 * p = b * R_model + m; each part is its own array (any address):
 *   X_parts[p]   [T/(R_batch R_model), D] bf16: token rows p of X
 *   W1t_parts[p] [F/R_model, D/R_batch] bf16: W1t rows block m, cols block b
 *   W2t_parts[p] [D/R_batch, F/R_model] bf16: W2t rows block b, cols block m
 *   Y_parts[p]   [T/(R_batch R_model), D] out_dtype: token rows p of Y
 *   b1 [F], b2 [D] fp32 replicated, either may be NULL.
 * The collectives of the lowering (Sec. 6) are fused away: all_gather of X
 * over M and of W1, W2 over B become the GEMMs reading each part in place,
 * and the all_reduce over M with the all_slice after it (a reduce_scatter)
 * becomes the down-projection's in-accumulator #sum over m whose output rows
 * are stored by their owner.  Y equals partir_mlp_block on the concatenated
 * operands.  Arrays are host arrays of R_batch * R_model device pointers
 * (<= 64 devices).  Constraints: T/(R_batch R_model), D/R_batch and F/R_model
 * multiples of 64; 16-byte aligned parts.  Workspace: H [T, F] bf16.
 * Errors: E_NULL, E_SHAPE, E_DIVISIBILITY, E_LAYOUT, E_DTYPE, E_WORKSPACE,
 * E_UNSUPPORTED, E_HIP. */
int partir_mlp_block_sharded(const void* const* X_parts, const void* const* W1t_parts,
                             const void* b1, const void* const* W2t_parts, const void* b2,
                             void* const* Y_parts, int64_t T, int64_t D, int64_t F,
                             int out_dtype, int act, int R_batch, int R_model,
                             void* ws, size_t ws_bytes, void* stream);
size_t partir_mlp_block_sharded_workspace(int64_t T, int64_t D, int64_t F, int R_batch, int R_model);

/* The decoder layer on device-local arrays: BP + MP + Z3 with the residual
 * stream sharded over the model axis too, so the RMSNorms run on each
 * device's own tokens (sequence-parallel norms).  Device (b, m) of the mesh
 * {B: R_batch, M: R_model} is part p = b * R_model + m:
 *   x_parts[p]   [B*S/(R_batch R_model), D] fp32: token rows p of x, updated
 *                in place to the layer's output
 *   Wq|Wk|Wv|W1_parts[p]: W_t[rows block m, cols block b] bf16 (W_t = W^T
 *                [out, in]; blocks of out/R_model rows and D/R_batch columns)
 *   Wo|W2_parts[p]: W_t[rows block b, cols block m] (D/R_batch rows, in/R_model
 *                columns)
 *   g1, g2 [D] fp32 replicated (g2 may be NULL when F = 0).
 * Lowered program per device (Sec. 6 collectives, all fused): the norm of the
 * device's tokens is stored into the gathered activation buffer (all_gather
 * over M); the projections read the weight parts in place (all_gathers over
 * B); the attention-out and FFN-down #sums over m stay in the tile and each
 * row block is added into its owner's residual part (reduce_scatter).  The
 * result equals partir_decoder_layer on the concatenated x.  Constraints:
 * those of partir_decoder_layer, T/(R_batch R_model) a multiple of 16,
 * D/R_batch and F/R_model multiples of 64, at most 21 devices (the Q|K|V
 * projection reads three weights' blocks through one table of 64 parts).
 * Errors: E_NULL, E_SHAPE, E_DIVISIBILITY, E_LAYOUT, E_WORKSPACE,
 * E_UNSUPPORTED, E_HIP. */
int partir_decoder_layer_sharded(void* const* x_parts, const void* g1, const void* g2, float eps,
                                 const void* const* Wq_parts, const void* const* Wk_parts,
                                 const void* const* Wv_parts, const void* const* Wo_parts,
                                 const void* const* W1_parts, const void* const* W2_parts,
                                 int64_t B, int64_t S, int64_t D, int64_t n_heads, int64_t d_head,
                                 int64_t F, int R_batch, int R_model,
                                 void* ws, size_t ws_bytes, void* stream);
size_t partir_decoder_layer_sharded_workspace(int64_t B, int64_t S, int64_t D, int64_t n_heads,
                                              int64_t d_head, int64_t F, int R_batch, int R_model);

/* The forward of a training step: partir_mlp_block, and also the
 * pre-activation Z = X W1 + b1 [T, F] bf16 (row-major, caller-owned, written
 * by the same up-projection tiles) that partir_mlp_block_backward reads
 * instead of recomputing it.  Same workspace as partir_mlp_block.  Z must be
 * non-NULL when T, D and F are all non-zero; errors as partir_mlp_block. */
int partir_mlp_block_train(const void* X, const void* W1, const void* b1,
                           const void* W2, const void* b2, void* Y, void* Z,
                           int64_t T, int64_t D, int64_t F,
                           int in_dtype, int out_dtype, int act,
                           int R_batch, int R_model,
                           void* ws, size_t ws_bytes, void* stream);

size_t partir_mlp_block_workspace(int64_t T, int64_t D, int64_t F, int out_dtype,
                                  int R_batch, int R_model);

/* ------------------------------------------------------------------------ */
/* Backward pass of the MLP block (the evaluation trains, Sec. 7; gradient   */
/* reductions of batch and model parallelism, Sec. 2.3).                      */
/* ------------------------------------------------------------------------ */
/*
 * Given dY = dL/dY of partir_mlp_block's output (Z = X W1 + b1, H = act(Z),
 * Y = H W2 + b2), computes, with the same batch (R_batch) and model
 * (R_model) loops:
 *   dH  = dY W2^T      loop b [#tile<0>] { loop m [#tile<1>] }
 *   dZ  = dH * act'(Z) (Z recomputed)
 *   dW2 = H^T dY       loop m [#tile<0>] { loop b [#sum] }   the batch-parallel gradient sum
 *   dW1 = X^T dZ       loop m [#tile<1>] { loop b [#sum] }
 *   dX  = dZ W1^T      loop b [#tile<0>] { loop m [#sum] }   the model-parallel sum
 *   db1 = sum_t dZ, db2 = sum_t dY  (in fixed row-block order)
 * X, W1, W2, b1 as in partir_mlp_block; dY: [T, D] bf16.  Outputs fp32:
 * dX [T, D]; dW1 [D, F] and dW2 [F, D] (the weights' layout); db1 [F],
 * db2 [D] (either may be NULL: not computed).
 * Z: the pre-activation X W1 + b1 [T, F] bf16 kept by partir_mlp_block_train
 * (read only), or NULL: then it is recomputed into the workspace.
 * Intermediates Z (when recomputed), dH, dZ and H = act(Z) are bf16 in the
 * workspace; every operand is read in place (no transposed copies).  The
 * workspace query assumes Z is recomputed (an upper bound otherwise).  Constraints: D, F/R_model and T/R_batch multiples of 8.  A
 * size of 0 gives empty sums (zeros) for every non-empty gradient.
 * Errors: E_NULL, E_SHAPE, E_DIVISIBILITY, E_LAYOUT, E_WORKSPACE,
 * E_UNSUPPORTED (R < 1, unknown act), E_HIP.
 */
int partir_mlp_block_backward(const void* X, const void* W1, const void* b1,
                              const void* W2, const void* dY, const void* Z,
                              void* dX, void* dW1, void* db1, void* dW2, void* db2,
                              int64_t T, int64_t D, int64_t F, int act,
                              int R_batch, int R_model,
                              void* ws, size_t ws_bytes, void* stream);

/* with_bias_grads: nonzero if db1 / db2 will be requested. */
size_t partir_mlp_block_backward_workspace(int64_t T, int64_t D, int64_t F, int act,
                                           int with_bias_grads, int R_batch, int R_model);

/* ------------------------------------------------------------------------ */
/* Attention block: heads #tile inside a Megatron #sum, in a batch #tile     */
/* (Megatron model parallelism of attention, Sec. 2.3; the MP tactic shards   */
/* the QKV weights on their heads dim and the output weight on its rows,      */
/* Sec. 3; the batch tile of BP, Sec. 3; TMR matmul forms, Sec. 5.2.1).       */
/* ------------------------------------------------------------------------ */
/*
 * Y = loop b [#tile<0>](R_batch) {
 *       loop m [#sum](R_model) {
 *         (loop h [#tile<1>](n_heads/R_model) {
 *             attn(Q_h, K_h, V_h) }) @ slice 0 Wo[m] } }
 * with Q = slice 0 X[b] @ slice 1 Wq[m] (K, V likewise) and, per sequence
 * and head, attn = softmax(scale * Q K^T, keys j <= query i when causal) V.
 * X: [B*S, D] bf16, sequence-major (token t = s*S + position).  Wq, Wk, Wv,
 * Wo: [D, D] bf16 row-major [fan_in, fan_out], read in place; head h owns
 * columns [h*d_head, (h+1)*d_head) of Wq, Wk, Wv (so of Q, K and V) and rows
 * [h*d_head, (h+1)*d_head) of Wo.  Batch shards hold whole sequences.
 * scale <= 0 selects 1/sqrt(d_head).  Y: [B*S, D], out_dtype F32 or BF16.
 * The workspace holds Q, K, V and the attention output (bf16, [B*S, D] each).
 * Constraints: d_head == 128, S a multiple of 128, S*D*2 < 4 GiB (one
 * sequence's rows of an [S, D] bf16 array).  B = 0 or S = 0 (no tokens)
 * launches nothing.
 * Errors: E_NULL, E_SHAPE (n_heads*d_head != D, or d_head / S outside the
 * constraints), E_DIVISIBILITY (R_batch does not divide B or R_model does not
 * divide n_heads), E_DTYPE, E_LAYOUT, E_WORKSPACE, E_UNSUPPORTED, E_HIP.
 */
int partir_attn_block(const void* X, const void* Wq, const void* Wk,
                      const void* Wv, const void* Wo, void* Y,
                      int64_t B, int64_t S, int64_t D, int64_t n_heads, int64_t d_head,
                      int causal, float scale, int in_dtype, int out_dtype,
                      int R_batch, int R_model,
                      void* ws, size_t ws_bytes, void* stream);

size_t partir_attn_block_workspace(int64_t B, int64_t S, int64_t D, int64_t n_heads,
                                   int64_t d_head, int R_batch, int R_model);

/* The forward of a training step: partir_attn_block, and also Q, K, V, the
 * attention output A and the per-row lse kept in the caller's buffer `saved`
 * (partir_attn_block_saved_bytes bytes: Q | K | V | A, each [B*S, D] bf16 at
 * 256-byte aligned offsets, then lse [B*S, n_heads] fp32) for
 * partir_attn_block_backward.  Workspace: that of partir_attn_block minus the
 * Q, K, V, A it no longer holds (partir_attn_block_workspace is an upper
 * bound). */
int partir_attn_block_train(const void* X, const void* Wq, const void* Wk,
                            const void* Wv, const void* Wo, void* Y, void* saved,
                            int64_t B, int64_t S, int64_t D, int64_t n_heads, int64_t d_head,
                            int causal, float scale, int in_dtype, int out_dtype,
                            int R_batch, int R_model,
                            void* ws, size_t ws_bytes, void* stream);
size_t partir_attn_block_saved_bytes(int64_t B, int64_t S, int64_t D, int64_t n_heads);

/* Gradients of the attention block for dY [B*S, D] bf16 (the evaluation
 * trains, Sec. 7), with the forward's batch (R_batch) and heads (R_model)
 * loops:
 *   dA = dY Wo^T                   loop b [#tile<0>] { loop m [#tile<1>] }
 *   dQ, dK, dV = per-head attention gradients (partir_attention_backward)
 *   dX = dQ Wq^T + dK Wk^T + dV Wv^T   loop b [#tile<0>] { loop m [#sum] }, and
 *                                      the sum over the three projections
 *   dW{q,k,v} = X^T d{Q,K,V}       loop m [#tile<1>] { loop b [#sum] }
 *   dWo = A^T dY                   loop m [#tile<0>] { loop b [#sum] }
 * Weights as in partir_attn_block and their gradients in the same
 * [fan_in, fan_out] layout (dW* fp32 [D, D]); dX fp32 [B*S, D]; `saved` from
 * partir_attn_block_train.  The workspace holds dA, [dQ dK dV] and the
 * rowsums; every operand is read in place.  Constraints as
 * partir_attn_block.  Errors: E_NULL, E_SHAPE, E_DIVISIBILITY, E_LAYOUT,
 * E_WORKSPACE, E_UNSUPPORTED, E_HIP. */
int partir_attn_block_backward(const void* X, const void* Wq, const void* Wk,
                               const void* Wv, const void* Wo, const void* saved,
                               const void* dY, void* dX, void* dWq, void* dWk,
                               void* dWv, void* dWo,
                               int64_t B, int64_t S, int64_t D, int64_t n_heads, int64_t d_head,
                               int causal, float scale, int R_batch, int R_model,
                               void* ws, size_t ws_bytes, void* stream);
size_t partir_attn_block_backward_workspace(int64_t B, int64_t S, int64_t D, int64_t n_heads,
                                            int64_t d_head, int R_batch, int R_model);

/* ------------------------------------------------------------------------ */
/* Attention core alone, with the key axis as a loop whose reduction is a     */
/* custom associative #sum (Sec. 5.2.1 footnote: any associative reduction).  */
/* ------------------------------------------------------------------------ */
/*
 * O = loop h [#tile<1>](n_heads) {
 *       loop s [#sum softmax](R_kv) { partial(Q_h, slice 0 K_h[s], slice 0 V_h[s]) } }
 * The key positions of each sequence are split into R_kv contiguous shards.
 * A shard yields (m, l, o) for every query: m = max_j c s_j over its keys
 * (log2 domain, c = scale log2 e), l = sum_j 2^(c s_j - m), o = sum_j
 * 2^(c s_j - m) v_j.  The reduction is (m, l, o) (+) (m', l', o') =
 * (M, 2^(m-M) l + 2^(m'-M) l', 2^(m-M) o + 2^(m'-M) o'), M = max(m, m'),
 * which is associative and commutative; the shards are folded in order
 * s = 0..R_kv-1 and O = o / l.  With causal masking a query sees keys at
 * positions <= its own, so shards past it contribute (-inf, 0, 0) and are
 * skipped.  With a causal mask and a grid too small to fill the device several
 * times over, each shard of at least 2048 keys is evaluated as 2 or 4 ordered
 * parts of at least 1024 keys, folded in the same order (the plan text names
 * them).  R_kv = 1 is plain attention (no workspace).
 * Q, K, V, O: [B*S, n_heads*d_head] bf16 row-major (ld = n_heads*d_head),
 * sequence-major; head h owns columns [h*d_head, (h+1)*d_head).
 * scale <= 0 selects 1/sqrt(d_head).  Constraints: d_head == 128, S a
 * multiple of 128, S*n_heads*d_head*2 < 4 GiB, R_kv dividing S/64.
 * Workspace (R_kv > 1): the parts' fp32 o (P*B*S*n_heads*d_head) and m, l
 * (P*B*S*n_heads each), P = R_kv times the parts per shard;
 * partir_attention_workspace gives the size for a causal mask, which is also
 * enough without one.
 * Errors: E_NULL, E_SHAPE (also when (S/128)*B*n_heads*R_kv exceeds 2^29),
 * E_DIVISIBILITY (R_kv does not divide S/64), E_LAYOUT, E_WORKSPACE,
 * E_UNSUPPORTED (R_kv < 1), E_HIP.
 */
int partir_attention(const void* Q, const void* K, const void* V, void* O,
                     int64_t B, int64_t S, int64_t n_heads, int64_t d_head,
                     int causal, float scale, int R_kv,
                     void* ws, size_t ws_bytes, void* stream);

size_t partir_attention_workspace(int64_t B, int64_t S, int64_t n_heads, int64_t d_head, int R_kv);

/* The forward of a training step: partir_attention, and also the per-row
 * base-2 log-sum-exp of the scaled scores, lse[t][h] = log2 sum_j
 * 2^(c s_tj) (c = scale log2 e; equal to the natural log-sum-exp times
 * log2 e), lse: [B*S, n_heads] fp32, which partir_attention_backward reads
 * instead of recomputing the softmax denominators.  Same workspace as
 * partir_attention; lse must be non-NULL when B*S > 0. */
int partir_attention_train(const void* Q, const void* K, const void* V, void* O, float* lse,
                           int64_t B, int64_t S, int64_t n_heads, int64_t d_head,
                           int causal, float scale, int R_kv,
                           void* ws, size_t ws_bytes, void* stream);

/* Gradients of the attention core (the evaluation trains, Sec. 7).  With
 * P = softmax of the scaled (masked) scores:
 *   dV = P^T dO;  dS = P * (dO V^T - rowsum(dO * O));  dQ = scale dS K;
 *   dK = scale dS^T Q,
 * per head (the heads #tile carries over: every head's gradients are
 * independent).  Q, K, V, O, dO, dQ, dK, dV: [B*S, n_heads*d_head] bf16 as in
 * partir_attention; lse from partir_attention_train.  dQ is accumulated by
 * one workgroup per query block over the keys, dK and dV by one per key block
 * over the queries, in a fixed order: deterministic, no atomics.  Workspace:
 * the rowsums, B*S*n_heads fp32.  Constraints as partir_attention.
 * Errors: E_NULL, E_SHAPE, E_LAYOUT, E_WORKSPACE, E_HIP. */
int partir_attention_backward(const void* Q, const void* K, const void* V, const void* O,
                              const void* dO, const float* lse,
                              void* dQ, void* dK, void* dV,
                              int64_t B, int64_t S, int64_t n_heads, int64_t d_head,
                              int causal, float scale,
                              void* ws, size_t ws_bytes, void* stream);
size_t partir_attention_backward_workspace(int64_t B, int64_t S, int64_t n_heads, int64_t d_head);

/* ------------------------------------------------------------------------ */
/* Pre-norm decoder layer on an fp32 residual stream, in place: the          */
/* transformer layer the evaluation partitions (Sec. 7.1, with its           */
/* additional normalisation), under BP + MP (Sec. 3) as a batch #tile over   */
/* the attention and MLP nests above.                                         */
/* ------------------------------------------------------------------------ */
/*
 * x = loop b [#tile<0>](R_batch) { xb = slice 0 x[b];
 *       h  = xb + loop m [#sum](R_model) { attn_m(rmsnorm(xb, g1)) @ slice 0 Wo[m] };
 *       h  + loop m [#sum](R_model) { gelu(rmsnorm(h, g2) @ slice 1 W1[m]) @ slice 0 W2[m] } }
 * rmsnorm(x, g) = g * x / sqrt(mean(x^2) + eps) over the D features of a row;
 * attention is causal with scale 1/sqrt(d_head).
 * x: [B*S, D] f32, updated in place.  g1, g2: [D] f32.  Wq..Wo as in
 * partir_attn_block; W1: [D, F] bf16; W2: [F, D] bf16 ([fan_in, fan_out]).
 * Workspace: normalised activations, Q, K, V, attention output and the
 * [B*S, F] FFN intermediate, all bf16.
 * F = 0 leaves out the FFN half (it adds the empty sum); B = 0 or S = 0
 * launches nothing.
 * Errors: as partir_attn_block, plus E_DIVISIBILITY when R_model does not
 * divide F.
 */
int partir_decoder_layer(void* x, const void* g1, const void* g2, float eps,
                         const void* Wq, const void* Wk, const void* Wv,
                         const void* Wo, const void* W1, const void* W2,
                         int64_t B, int64_t S, int64_t D, int64_t n_heads,
                         int64_t d_head, int64_t F, int R_batch, int R_model,
                         void* ws, size_t ws_bytes, void* stream);

size_t partir_decoder_layer_workspace(int64_t B, int64_t S, int64_t D, int64_t n_heads,
                                      int64_t d_head, int64_t F, int R_batch, int R_model);

/* ------------------------------------------------------------------------ */
/* Plans: what a call will do, without doing it (host only, no GPU needed).  */
/* ------------------------------------------------------------------------ */
typedef struct partir_plan_info {
  int n_virtual_shards;     /* product of the loop sizes of the nest               */
  int n_tile_loops;         /* #tile loops in the nest (incl. the heads loop)       */
  int n_sum_loops;          /* #sum loops: the in-device stand-ins for all_reduce   */
  int n_sum_splitk;         /* of those, realised through fp32 partials in HBM      */
  int n_launches;           /* kernel launches the call enqueues                    */
  int reserved;
  size_t workspace_bytes;   /* what the matching *_workspace query returns          */
  double flops;             /* algorithmic FLOPs (causal attention: unmasked pairs)  */
} partir_plan_info;

/* Fill *info for the call with these arguments; returns a partir_status. */
int partir_plan_loop_matmul(int64_t M, int64_t N, int64_t K, int ab_dtype, int c_dtype,
                            int b_layout, int tile_axis, int sum_axis, int R, int sum_impl,
                            partir_plan_info* info);
int partir_plan_mlp_block(int64_t T, int64_t D, int64_t F, int out_dtype,
                          int R_batch, int R_model, partir_plan_info* info);
int partir_plan_attn_block(int64_t B, int64_t S, int64_t D, int64_t n_heads, int64_t d_head,
                           int R_batch, int R_model, partir_plan_info* info);
int partir_plan_attention(int64_t B, int64_t S, int64_t n_heads, int64_t d_head, int causal, int R_kv,
                          partir_plan_info* info);
int partir_plan_attention_backward(int64_t B, int64_t S, int64_t n_heads, int64_t d_head, int causal,
                                   partir_plan_info* info);
int partir_plan_attn_block_backward(int64_t B, int64_t S, int64_t D, int64_t n_heads, int64_t d_head,
                                    int causal, int R_batch, int R_model, partir_plan_info* info);
int partir_plan_mlp_block_backward(int64_t T, int64_t D, int64_t F, int act, int R_batch, int R_model,
                                   partir_plan_info* info);
int partir_plan_mlp_block_sharded(int64_t T, int64_t D, int64_t F, int act, int R_batch, int R_model,
                                  partir_plan_info* info);
int partir_plan_decoder_layer_sharded(int64_t B, int64_t S, int64_t D, int64_t n_heads, int64_t d_head,
                                      int64_t F, int R_batch, int R_model, partir_plan_info* info);
int partir_plan_decoder_layer(int64_t B, int64_t S, int64_t D, int64_t n_heads,
                              int64_t d_head, int64_t F, int R_batch, int R_model,
                              partir_plan_info* info);

/* Human-readable shard table of the last plan built on this thread
 * (views, offsets, tile grid and #sum realisation per launch).  The string is
 * owned by the library and valid until the next call on this thread. */
const char* partir_last_plan_text(void);

/* ------------------------------------------------------------------------ */
/* Planner: ManualPartition tactics, value tiling and propagation on the host */
/* (Sec. 3 schedules; Sec. 5.1 value tiling; Sec. 5.2 TMR, propagation,       */
/* inference and conflicts; App. A multi-axis nests).  No GPU needed.         */
/* ------------------------------------------------------------------------ */
/*
 * program: NUL-terminated text, one statement per line (or ';'), '#' comments:
 *   mesh <axis>=<size> ...            the mesh axes, in order
 *   arg <name> <rows>x<cols>          a 2-D function argument
 *   <name> = matmul <a> <b> | add <a> <b> | gelu <a> | rmsnorm <a>
 *   ret <name> ...
 * schedule: text, one tactic per line:
 *   partition <axis> <name>:<dim> ...   ManualPartition({name: dim, ...}, axis):
 *                                       value-tile each named value, then propagate
 *   tile <name> <dim> <axis>            a bare value-tiling action
 *   propagate                           a bare propagation action
 * TMR: matmul (#tile<0>,_) -> #tile<0>, (_,#tile<1>) -> #tile<1>,
 * (#tile<1>,#tile<0>) -> #sum; add (#tile<d>,#tile<d>) -> #tile<d>; gelu
 * #tile<d> -> #tile<d>; rmsnorm #tile<0> -> #tile<0>.  An op never gets a
 * second loop over an axis it is already nested in; several matching entries
 * are a conflict, reported and left alone.
 * out / out_len: caller buffer for the NUL-terminated report; *needed (if
 * non-NULL) receives its size.  Report lines:
 *   action <...>                          every action, each rewrite tagged
 *                                         (forward|backward|inference), conflicts
 *   loop <op> <kind> <axis>:<tile0|tile1|sum> ... | none   loop nest, outer first
 *   operand <op> <i> <value> <axis>:<dim> ...     how the op slices operand i
 *   gather|reshard <op> <value> <axis>    a tiled value used whole / along another dim
 *   value <name> <axis>:<dim> ... | replicated    tiling after the schedule
 *   call partir_loop_matmul <op> tile=<M|N|none> sum=<K|none> R=<n>
 *   call partir_mlp_block <op> R_batch=<n> R_model=<n> ops=<up>,<act>,<down>
 *   nest <op> (...)                       a nest no single entry point runs
 * Errors: E_NULL, E_SHAPE (parse error or shape mismatch), E_AXIS (unknown
 * axis or dim, or a value tiled along two dims on one axis), E_DIVISIBILITY
 * (TSlice), E_UNSUPPORTED (unknown op), E_WORKSPACE (out too small).
 */
int partir_propagate(const char* program, const char* schedule, char* out, size_t out_len,
                     size_t* needed);

/* ------------------------------------------------------------------------ */
/* Kernel trace: per-kernel GPU time measured with HIP events.                */
/* ------------------------------------------------------------------------ */
typedef struct partir_trace_entry {
  char name[48];            /* kernel family name                               */
  int64_t launches;         /* launches recorded since the last reset           */
  double total_ms;          /* summed GPU time between the events bracketing it */
} partir_trace_entry;

/* While enabled, every launch is bracketed by two events on its stream.
 * Enabling creates events (a host-side resource), so it is meant for
 * measurement runs, not for callers that must not allocate. */
int partir_trace_enable(int on);
/* Synchronises the recorded events and folds them into per-name totals;
 * writes up to max entries and returns how many kernel names exist (or a
 * negative status). */
int partir_trace_read(partir_trace_entry* out, int max);
void partir_trace_reset(void);

/* ------------------------------------------------------------------------ */
const char* partir_status_string(int status);
const char* partir_last_error(void);
const char* partir_version(void);

#ifdef __cplusplus
}
#endif

#endif /* PARTIR_H */
