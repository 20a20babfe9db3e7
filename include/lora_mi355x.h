/*
 * lora_mi355x.h -- C ABI of the MI355X (gfx950) LoRA-linear library.
 *
 * The operation (LoRA as described in the paper's background on
 * parameter-efficient fine-tuning: a frozen base weight W plus a trained
 * rank-r pair A, B; r and alpha from its hyperparameter table; the frozen-base
 * forward y = W x and input gradient dx = W^T dy, with no weight gradient,
 * from its algorithm "On-the-fly Dequantization"), with tokens as rows:
 *
 *   forward   u  = x A^T                      [T, r]   (fp32, kept for bwd)
 *             y  = x W^T + s u B^T            [T, d_out]
 *   backward  du = s dy B                     [T, r]
 *             dx = dy W + du A                [T, d_in]
 *             dA = du^T x                     [r, d_in]   (fp32)
 *             dB = s dy^T u                   [d_out, r]  (fp32)
 *   s = alpha / r.  W is frozen: dW = dy^T x is never formed or allocated.
 *
 * Layouts (all row-major, leading dimension = row length, no padding):
 *   x [T, d_in], W [d_out, d_in], A [r, d_in], B [d_out, r], y/dy [T, d_out],
 *   dx [T, d_in], u [T, r] fp32, dA [r, d_in] fp32, dB [d_out, r] fp32.
 *
 * Element types: x, W, A, B, dy, y, dx have the type `dt` (bf16 with fp32
 * accumulation, or fp32 end to end as a check mode); u, dA, dB are fp32.
 * In bf16 mode the products s*u and du are rounded to bf16 (round to nearest
 * even) before they enter the matrix cores; y and dx are rounded once, from
 * the fp32 accumulator.
 *
 * Ownership: every pointer is a device pointer owned by the caller.  The
 * library never allocates device memory (apart from the counter noted
 * below) and keeps no pointer after a call returns.  Scratch space comes
 * from the caller's workspace `ws` of `ws_bytes` bytes (size it with
 * lora_linear_workspace_bytes); its contents
 * on entry are ignored and on return are unspecified.
 *
 * Streams: all work is enqueued on `hip_stream` (a hipStream_t; NULL = the
 * null stream) and the call returns without synchronising.  Two calls that
 * share a workspace must be ordered on one stream.
 *
 * Errors: every entry point validates all arguments before enqueuing any
 * work, so nothing is written when it returns an error.  It returns
 *   LORA_EINVAL        a NULL required pointer, a pointer not 16-byte
 *                      aligned, a size < 1, r outside [0,128], a non-finite
 *                      scale, or an output overlapping an input or another
 *                      output;
 *   LORA_EUNSUPPORTED  d_in or d_out not a multiple of 8 or above 2^20, or a
 *                      matrix with 2^31 or more elements;
 *   LORA_EWORKSPACE    ws_bytes below the required size (or ws NULL when
 *                      the required size is non-zero);
 *   LORA_EHIP          a kernel launch failed (asynchronous device faults
 *                      surface at the caller's next stream synchronisation).
 * lora_last_error() returns a short text for the calling thread's last error.
 * No entry point prints, aborts or throws.
 *
 * Determinism: every reduction (over tokens, over the split feature axis of
 * the rank-r products, across waves) adds its parts in a fixed order, so
 * identical inputs give bitwise identical outputs.  Atomics appear only where
 * they cannot change a result: the counters of the fused hand-over (they
 * order work; see lora_handover_giveups); the part counts of the dA / dB
 * token reductions that run as token parts (they pick the part that adds
 * the parts' tiles, which it adds in ascending part order); and, in the
 * top-k table build, the reservation of candidate-list slots, whose order is
 * normalised by the selection (ties go to the smaller index).
 *
 * Device memory held by the library itself: one 4-byte counter per device
 * (lora_handover_giveups); everything else is the caller's.
 */
#ifndef LORA_MI355X_H
#define LORA_MI355X_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  LORA_OK = 0,
  LORA_EINVAL = 1,
  LORA_EUNSUPPORTED = 2,
  LORA_EWORKSPACE = 3,
  LORA_EHIP = 4
} lora_status_t;

typedef enum { LORA_BF16 = 0, LORA_F32 = 1 } lora_dtype_t;

typedef enum { LORA_OP_FWD = 0, LORA_OP_BWD = 1, LORA_OP_FROZEN_DX = 2 } lora_op_t;

/* Workspace bytes sufficient for any call of `op` with these sizes, whether
 * or not the optional u pointers are given.  Returns 0 when none is needed
 * and (size_t)-1 for sizes the entry point would reject.  Pure host logic. */
size_t lora_linear_workspace_bytes(lora_op_t op, int64_t T, int64_t d_in, int64_t d_out,
                                   int64_t r, lora_dtype_t dt);

/* LoRA forward (the definitions above): y = x W^T + s (x A^T) B^T.
 *   u_save  optional [T, r] fp32 output receiving u = x A^T (unscaled) for the
 *           backward pass; NULL keeps u in the workspace only.
 *   r = 0   gives the plain frozen linear y = x W^T; A, B, u_save are ignored
 *           and may be NULL.
 *   scale   s = alpha / r, any finite value. */
lora_status_t lora_linear_fwd(const void *x, const void *W, const void *A, const void *B,
                              void *y, float *u_save, int64_t T, int64_t d_in, int64_t d_out,
                              int64_t r, float scale, lora_dtype_t dt, void *ws,
                              size_t ws_bytes, void *hip_stream);

/* LoRA backward: dx = dy W + du A, dA = du^T x, dB = s dy^T u, du = s dy B.
 *   u_saved  [T, r] fp32 from lora_linear_fwd, or NULL to recompute u = x A^T
 *            (activation rematerialisation in place of storing it).
 *   dx       may be NULL when the input gradient is not needed.
 *   dA, dB   required when r > 0; ignored (may be NULL) when r = 0, in which
 *            case the call computes dx = dy W only.
 *   Outputs are overwritten, not accumulated. */
lora_status_t lora_linear_bwd(const void *x, const void *W, const void *A, const void *B,
                              const float *u_saved, const void *dy, void *dx, float *dA,
                              float *dB, int64_t T, int64_t d_in, int64_t d_out, int64_t r,
                              float scale, lora_dtype_t dt, void *ws, size_t ws_bytes,
                              void *hip_stream);

/* For callers that cannot allocate device memory -- code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc: the same
 * operation as lora_linear_bwd, with the workspace taken from a static
 * device array of the library (LORA_NOALLOC_SCRATCH_BYTES per GPU, held by
 * every GPU the library runs on until the process ends) instead of a caller
 * buffer.  Calls no allocating routine.  Arguments, outputs and errors as for
 * lora_linear_bwd, plus LORA_EWORKSPACE when the sizes need more workspace
 * than the static array holds, and LORA_EHIP if its address cannot be looked
 * up.  The array belongs to the current device (hip_stream must be one of
 * its streams) and keeps the last call's contents; calls that overlap on
 * one GPU (other streams, other threads) race on it and must not be issued. */
#define LORA_NOALLOC_SCRATCH_BYTES (16u << 20)
lora_status_t lora_linear_bwd_noalloc(const void *x, const void *W, const void *A, const void *B,
                                      const float *u_saved, const void *dy, void *dx, float *dA,
                                      float *dB, int64_t T, int64_t d_in, int64_t d_out, int64_t r,
                                      float scale, lora_dtype_t dt, void *hip_stream);

/* Rank-0 frozen linear input gradient, dx = dy W (the frozen LM head of the
 * paper's checkpointing scheme, whose backward needs only dx):
 *   dy [T, d_out], W [d_out, d_in], dx [T, d_in]. */
lora_status_t frozen_linear_bwd_dx(const void *dy, const void *W, void *dx, int64_t T,
                                   int64_t d_in, int64_t d_out, lora_dtype_t dt, void *ws,
                                   size_t ws_bytes, void *hip_stream);

/* ---- Quantized frozen base ------------------------------------------------
 * The same three operations with W stored quantized and dequantized on the
 * fly (the paper's algorithm "On-the-fly Dequantization": W = s * W_q + b,
 * rematerialised for the forward and again for the backward; its mixed
 * precision quantization keeps linear layers in INT4 and the output head in
 * INT8).  Here the dequantized W never exists in memory: each GEMM workgroup
 * expands the codes of its tile into bf16 in on-chip memory.
 *
 *   W_codes   [d_out][d_in * bits / 8] bytes of unsigned codes; bits = 8:
 *             one code per byte; bits = 4: two per byte, the code of the even
 *             input k in the low nibble, of k + 1 in the high nibble.
 *   W_scale,  [d_in / group][d_out] fp32, group-major: the weight of code q
 *   W_offset  in row n, input k is
 *               W_scale[k / group][n] * q + W_offset[k / group][n]
 *             (a GEMM stage reads one group's scales for many consecutive
 *             rows, which this layout keeps contiguous).
 *   group     a power of two >= 16 that divides d_in.
 * Everything else is as for the bf16 entry points, with dt = LORA_BF16
 * (x, A, B, y, dy, dx bf16) and rank r <= 64.  Errors as above, plus
 * LORA_EINVAL for bits not 4 or 8 or a NULL codes / scale / offset pointer,
 * and LORA_EUNSUPPORTED for a bad group or r > 64.  The workspace sizes are
 * those of the bf16 operations. */
lora_status_t lora_linear_fwd_q(const void *x, const void *W_codes, const float *W_scale,
                                const float *W_offset, int bits, int64_t group, const void *A,
                                const void *B, void *y, float *u_save, int64_t T, int64_t d_in,
                                int64_t d_out, int64_t r, float scale, void *ws, size_t ws_bytes,
                                void *hip_stream);
lora_status_t lora_linear_bwd_q(const void *x, const void *W_codes, const float *W_scale,
                                const float *W_offset, int bits, int64_t group, const void *A,
                                const void *B, const float *u_saved, const void *dy, void *dx,
                                float *dA, float *dB, int64_t T, int64_t d_in, int64_t d_out,
                                int64_t r, float scale, void *ws, size_t ws_bytes,
                                void *hip_stream);
lora_status_t frozen_linear_bwd_dx_q(const void *dy, const void *W_codes, const float *W_scale,
                                     const float *W_offset, int bits, int64_t group, void *dx,
                                     int64_t T, int64_t d_in, int64_t d_out, void *ws,
                                     size_t ws_bytes, void *hip_stream);

/* ---- Frozen LM head: reduced-vocabulary cross entropy with logits masking --
 * The paper's "Softmax Approximation" computes the logits only over a reduced
 * vocabulary J, the union of the first k entries of the similarity-table rows
 * of the targets, and its "Logits Masking" only for the trainable positions;
 * the masked causal-LM loss sums -log p_t over those positions.  With h
 * [T, D] the final hidden states, W [V, D] the frozen output embedding (row v
 * = token v), rows [nrows] the trainable positions (distinct) and y [T] the
 * targets:
 *   J          = sorted union over i of table[y[rows[i]]][0 .. k-1]
 *   z_i[j]     = h[rows[i]] . W[J[j]]                     (never stored)
 *   loss[i]    = logsumexp_j z_i[j] - z_i[tpos[i]],  tpos[i] = position of
 *                y[rows[i]] in J
 *   dh[rows[i]] = dscale (sum_j softmax(z_i)[j] W[J[j]] - W[y[rows[i]]]),
 *   dh[t] = 0 for positions t not listed.  W is frozen (no weight gradient).
 * The logits are reduced tile by tile to row maxima and sums of exponentials
 * inside the GEMM; the backward recomputes them in chunks of 8192 columns of
 * J, so neither the logits nor their gradient is ever held in full.
 *
 * Integer arrays are int32 device arrays.  Workspace sizes:
 * lm_head_workspace_bytes(op, T, V, D, nrows, nJ) with op LM_HEAD_OP_VOCAB
 * (for lm_head_build_vocab; nJ ignored), LM_HEAD_OP_LOSS (loss only) or
 * LM_HEAD_OP_LOSS_DH; (size_t)-1 for sizes the calls would reject. */
typedef enum { LM_HEAD_OP_VOCAB = 0, LM_HEAD_OP_LOSS = 1, LM_HEAD_OP_LOSS_DH = 2 } lm_head_op_t;
size_t lm_head_workspace_bytes(int op, int64_t T, int64_t V, int64_t D, int64_t nrows,
                               int64_t nJ);

/* J [V] (capacity) and tpos [nrows] from the similarity table [V, ldtab]
 * (its first k columns are used; row v should start with v itself, which
 * puts every target in J), the targets y [T] and the trainable positions
 * rows [nrows].  *nJ (host) receives |J|: this call waits for its stream to
 * finish.  Entries outside their ranges are skipped and give tpos = -1 (the
 * loss of such a position is NaN).  Errors: LORA_EINVAL for NULL or
 * misaligned pointers, bad sizes or overlapping outputs, LORA_EWORKSPACE. */
lora_status_t lm_head_build_vocab(const int32_t *table, int64_t V, int64_t ldtab, int64_t k,
                                  const int32_t *targets, int64_t T, const int32_t *rows,
                                  int64_t nrows, int32_t *J, int32_t *tpos, int64_t *nJ, void *ws,
                                  size_t ws_bytes, void *hip_stream);

/* loss_rows [nrows] fp32 per trainable position, loss_total (optional, one
 * fp32) their sum, and, when dh (bf16 [T, D]) is not NULL, the gradient of
 * dscale * sum(loss_rows) with respect to h.  h, W bf16; D a multiple of 8.
 * Errors as above, plus LORA_EUNSUPPORTED for D. */
lora_status_t lm_head_reduced_ce(const void *h, const void *W, int64_t T, int64_t V, int64_t D,
                                 const int32_t *rows, int64_t nrows, const int32_t *J, int64_t nJ,
                                 const int32_t *tpos, float *loss_rows, float *loss_total,
                                 void *dh, float dscale, void *ws, size_t ws_bytes,
                                 void *hip_stream);

/* ---- Top-k similarity table ------------------------------------------------
 * The lookup table of the reduced-vocabulary softmax (paper: "Softmax
 * Approximation"): for each token i of the frozen embedding matrix W [V, D]
 * (bf16, row v = token v) the k tokens of highest cosine similarity
 * C[i][j] = (w_i . w_j) / (|w_i| |w_j|), in descending order (the smaller
 * index first among equal similarities):
 *   table [V, k] int32, values [V, k] fp32 (optional, the similarities).
 * Row i starts with i itself when no other token points the same way.  The
 * V x V similarities are never stored: a GEMM over a batch of rows and a
 * chunk of columns appends the candidates above each row's running
 * threshold, and a per-row selection keeps the k best whenever a row's
 * candidate list might not hold another chunk.
 * Similarities are fp32 (bf16 products, fp32 sums): tokens within about
 * 1e-6 of each other may come out in either order.  Requires 1 <= k <=
 * min(V, 2048) and D a multiple of 8; workspace topk_table_workspace_bytes
 * ((size_t)-1 for rejected sizes).  Errors: LORA_EINVAL, LORA_EUNSUPPORTED
 * (D, sizes), LORA_EWORKSPACE, LORA_EHIP. */
size_t topk_table_workspace_bytes(int64_t V, int64_t D, int64_t k);
lora_status_t topk_table_build(const void *W, int64_t V, int64_t D, int64_t k, int32_t *table,
                               float *values, void *ws, size_t ws_bytes, void *hip_stream);

/* ---- Checkpointed step over a chain of LoRA linears -------------------------
 * The paper's algorithm "Memory-Efficient Checkpointing for LoRA Fine-tuning"
 * on one GPU, for a chain of nodes x_i = node_i(x_{i-1}) (node i a LoRA
 * linear, bf16): the forward keeps no LoRA activation and sends each node's
 * input to pinned host memory on `copy_stream` while the following nodes run
 * on `compute_stream`; the backward brings each input back one node ahead of
 * its use, recomputes u from it (as lora_linear_bwd with u_saved = NULL) and
 * backpropagates.  The loss node between the two (the paper's LM head) is
 * the caller's: it turns the forward's output x_n into g_n = dL/dx_n.
 * Device memory: two activation and two gradient buffers of the widest node
 * plus one LoRA workspace (lora_ckpt_workspace_bytes), whatever n is; host
 * memory: every node's input (lora_ckpt_host_bytes), which must be pinned
 * (hipHostMalloc) for the copies to run asynchronously.  Both calls return
 * once their work is enqueued; the host stash may be read or reused only
 * after the backward's work on both streams has completed.  The streams have
 * the default priority; one stream may serve as both.
 * Errors: LORA_EINVAL (n < 1, T < 1, a node's d_in not the previous d_out, a
 * missing pointer, a workspace not 256-byte aligned), LORA_EUNSUPPORTED (a
 * node's shape), LORA_EWORKSPACE (host or device scratch too small),
 * LORA_EHIP, and those of lora_linear_fwd / lora_linear_bwd. */
typedef struct {
  const void *W, *A, *B; /* bf16: W [d_out, d_in], A [r, d_in], B [d_out, r] */
  float *dA, *dB;        /* fp32 outputs [r, d_in], [d_out, r] (overwritten) */
  int64_t d_in, d_out, r;
  float scale;
} lora_node_t;
size_t lora_ckpt_workspace_bytes(const lora_node_t *nodes, int n, int64_t T);
size_t lora_ckpt_host_bytes(const lora_node_t *nodes, int n, int64_t T);
/* x0 [T, d_in of node 0] is only read; out [T, d_out of node n-1] receives x_n. */
lora_status_t lora_ckpt_forward(const lora_node_t *nodes, int n, int64_t T, const void *x0,
                                void *out, void *host_stash, size_t host_bytes, void *ws,
                                size_t ws_bytes, void *compute_stream, void *copy_stream);
/* g_n [T, d_out of node n-1]; dx0 [T, d_in of node 0] or NULL. */
lora_status_t lora_ckpt_backward(const lora_node_t *nodes, int n, int64_t T, const void *g_n,
                                 void *dx0, const void *host_stash, size_t host_bytes, void *ws,
                                 size_t ws_bytes, void *compute_stream, void *copy_stream);

/* ---- Plan and hand-over diagnostics -----------------------------------------
 * Which kernel configuration lora_linear_fwd / lora_linear_bwd run for these
 * sizes (host logic only, no GPU work): the output tile of the forward GEMM
 * (y, T x d_out) and of the dx GEMM (T x d_in); whether the rank-r pass runs
 * as producer workgroups inside that GEMM launch ("fused"); and otherwise
 * over how many partial sums of its reduction axis u = x A^T and
 * du = s dy B are computed; and over how many consecutive token ranges each
 * output block of the token reductions dA = du^T x and dB = s dy^T u runs
 * in the unfused dx launch (bwd_side_parts; 1 = all T in one workgroup).
 * Errors as for the entry points' size checks. */
typedef struct {
  int fwd_tile_m, fwd_tile_n, fwd_fused, fwd_u_parts;
  int bwd_tile_m, bwd_tile_n, bwd_fused, bwd_du_parts;
  int bwd_side_parts;
} lora_plan_t;
lora_status_t lora_linear_plan(int64_t T, int64_t d_in, int64_t d_out, int64_t r, lora_dtype_t dt,
                               lora_plan_t *plan);

/* A fused launch hands the rank-r rows from its producer workgroups to its
 * tiles through counters in the workspace; a wait for them gives up after a
 * bounded time (0.2 s) instead of hanging, and a launch whose wait gave up
 * may have used incomplete rows.  Every wave whose wait gave up adds one to
 * a counter of the current device; this call synchronises the device,
 * stores the count in *count and, if `reset`, sets it back to 0.  A caller
 * that needs certainty checks that the count stays 0.  Errors: LORA_EINVAL
 * (NULL), LORA_EHIP. */
lora_status_t lora_handover_giveups(uint64_t *count, int reset);

/* Test hook: with hold = 1, every tile's hand-over wait in the fused
 * launches enqueued afterwards (from any thread) gives up after its 0.2 s
 * budget instead of seeing the producers' count, so those launches' results
 * are invalid and lora_handover_giveups counts them; hold = 0 (the default)
 * restores normal operation.  Errors: LORA_EINVAL for other values. */
lora_status_t lora_debug_set_handover(int hold);

/* Static text for a status code. */
const char *lora_status_str(lora_status_t status);

/* Text describing the calling thread's most recent error ("" if none). */
const char *lora_last_error(void);

/* Benchmark timing hook.  While enabled, every launch of a library kernel is
 * bracketed by a pair of hipEvents recorded on the stream it runs on.
 * lora_profiler_read() waits for the recorded events of kernel `kernel_id`
 * (see lora_kernel_name) and returns their summed duration in milliseconds
 * and the number of launches; lora_profiler_reset() drops all records.
 * Returns LORA_EINVAL for an unknown id, LORA_EHIP on an event failure. */
lora_status_t lora_profiler_enable(int on);
lora_status_t lora_profiler_reset(void);
lora_status_t lora_profiler_read(int kernel_id, double *total_ms, int64_t *launches);

/* Name of library kernel `kernel_id` (0 .. lora_kernel_count()-1), NULL if
 * out of range. */
const char *lora_kernel_name(int kernel_id);
int lora_kernel_count(void);

#ifdef __cplusplus
}
#endif

#endif /* LORA_MI355X_H */
