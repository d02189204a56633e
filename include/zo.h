/*
 * zo.h -- C ABI of the SubZero+ hot path on AMD Instinct MI355X (gfx950).
 *
 * SubZero+ (arXiv 2608.15665) fine-tunes every weight matrix W_i (m x n, the
 * out x in layout of a linear layer) with zeroth-order estimates taken inside
 * a rank-r subspace spanned by column-orthonormal U_i (m x r) and V_i (n x r).
 * Three operations dominate its cost and are exported here:
 *
 *   zo_subspace_refresh      Haar-distributed U, V: thin QR of Gaussian panels
 *                            with column signs fixed so diag(R) > 0
 *                            (Eq. 11, Alg. 1).
 *   zo_perturbed_linear      the linear layer under the query perturbations
 *                            W +- eps U Z_j V^T (Eq. 4, Alg. 2, the forward of
 *                            Eq. 5) without forming the perturbed weight.
 *   zo_subspace_adam_update  aggregate the per-query estimates, run Adam on the
 *                            r x r state and apply W <- W - lr U S V^T
 *                            (Eqs. 6-10, tail of Alg. 3).
 *
 * plus small helpers for a squared-error loss and the central or forward
 * difference, and the network a query evaluates (the forward of Eq. 5): a
 * pre-LN decoder layer of the OPT family and a LLaMA-family layer with every
 * weight matrix perturbed, with their row norms, rotary positions and causal
 * attention as entry points of their own.
 *
 * Conventions (all entry points)
 *   - Every tensor argument is DEVICE memory owned by the caller; the library
 *     allocates nothing.  Scratch space comes from the caller's `workspace`
 *     (device memory, 256-byte aligned, size from the matching *_workspace()
 *     query).  Descriptor arrays (zo_panel, zo_update_item, blk_query,
 *     blk_sign) are HOST memory read during the call only.
 *   - Matrices are row-major and dense (leading dimension = number of
 *     columns).  bf16 tensors hold IEEE bfloat16 bit patterns (uint16_t).
 *     bf16 tensors must be 16-byte aligned; fp32 tensors 4-byte aligned.
 *   - Work is enqueued on `stream` (a hipStream_t; NULL = the default
 *     stream).  No call synchronises; results are ready when the stream is.
 *   - Return value: a zo_status.  Argument errors are detected on the host
 *     before anything is enqueued; the call then returns ZO_ERR_INVALID_ARG /
 *     ZO_ERR_UNSUPPORTED / ZO_ERR_WORKSPACE, launches nothing, and
 *     zo_last_error_detail() (thread-local) says what was wrong.  A failed
 *     launch returns ZO_ERR_HIP.
 *   - Results are deterministic: no atomics take part in any reduction.
 */
#ifndef ZO_H
#define ZO_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define ZO_ABI_VERSION 1
#define ZO_MAX_RANK 128   /* r limit of zo_perturbed_linear and the update   */
#define ZO_MAX_QR_RANK 128 /* r limit of zo_subspace_refresh                 */
#define ZO_MAX_BLOCKS 256 /* nblk limit of zo_perturbed_linear               */
#define ZO_MAX_QUERIES 256
#define ZO_MAX_GROUP 8    /* count limit of zo_perturbed_linear_prepare_group   */

/* ZO_ERR_RANK_DEFICIENT and ZO_ERR_NONFINITE are reserved: no call returns
 * them.  Both conditions arise on the device after the call has returned
 * (every call is asynchronous), so they are reported through device memory
 * instead: the refresh's info array and the update's nonfinite_flag. */
typedef enum {
  ZO_OK = 0,
  ZO_ERR_INVALID_ARG = 1,
  ZO_ERR_UNSUPPORTED = 2,
  ZO_ERR_RANK_DEFICIENT = 3,
  ZO_ERR_NONFINITE = 4,
  ZO_ERR_HIP = 5,
  ZO_ERR_WORKSPACE = 6
} zo_status;

typedef enum { ZO_F32 = 0, ZO_BF16 = 1, ZO_F16 = 2 } zo_dtype;
/* Epilogues fused into the perturbed linear's output (zo_perturbed_linear_apply_ex). */
typedef enum { ZO_EPI_NONE = 0, ZO_EPI_RELU = 1, ZO_EPI_RESIDUAL = 2, ZO_EPI_SILU_MUL = 3 } zo_epilogue;

int zo_abi_version(void);
const char* zo_status_str(int status);
/* Text of the last error raised on the calling thread ("" if none). */
const char* zo_last_error_detail(void);

/* ------------------------------------------------------------------------
 * Subspace refresh -- Eq. 11 and Alg. 1 (HaarProjMatrix).
 *
 * For each panel p (rows_p x r, rows_p >= r): Omega_p = Q_p R_p with
 * Q_p^T Q_p = I and R_p upper triangular with a POSITIVE diagonal, i.e. the
 * Q of any thin QR with each column multiplied by the sign of the matching
 * R diagonal entry.  This factor is unique, and for Gaussian Omega it is
 * Haar distributed.  Computed in float64 by CholeskyQR2 (R1 = chol(O^T O),
 * Q1 = O R1^-1, R2 = chol(Q1^T Q1), Q = Q1 R2^-1), whose Cholesky factors
 * have a positive diagonal, so the sign correction is built in; outputs
 * rounded once to float32.  Bitwise reproducible.  Accuracy: Q within 1e-5
 * of the exact factor (tested against a float64 Householder QR) on panels
 * whose columns are not nearly dependent -- column scaling does not matter
 * (tested to condition 1e9); nearly collinear columns are tested to
 * condition 2e7 - 4e7.  From condition ~1e8 of that kind the Cholesky pivots
 * fall to the rounding noise of the Gram matrix: a pivot that comes out not
 * positive is reported through info, one that comes out positive is not and
 * the result is then inaccurate.  Gaussian panels with rows >= 2 r (every
 * configuration here) reach such a condition with probability below 1e-30.
 *
 *   omega   device, rows x r fp32, row-major; read only.
 *   q       device, rows x r fp32 output; may alias omega.
 *   r_diag  device, r fp32 output (diag of the corrected R, > 0); nullable.
 *   info    device, `count` ints, nullable: info[p] = 0, or k+1 when the
 *           first Cholesky pivot that is not positive is at column k
 *           (Omega_p rank deficient, or numerically so; an exactly zero
 *           column gives this).
 *           R_kk is then reported as 0, the Q column is zero and the other
 *           columns are formed as if column k were absent.
 * Limits: 1 <= r <= ZO_MAX_QR_RANK, rows <= 2^26.  Panels of one call share
 * r; rows may differ.
 * ------------------------------------------------------------------------ */
typedef struct {
  int rows;
  const float* omega;
  float* q;
  float* r_diag;
} zo_panel;

size_t zo_subspace_refresh_workspace(int count, const zo_panel* panels, int r);
int zo_subspace_refresh(int count, const zo_panel* panels, int r, int* info,
                        void* workspace, size_t ws_bytes, void* stream);

/* zo_subspace_refresh without a workspace argument, for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc).  Same arguments, arithmetic, results
 * (bitwise) and errors as zo_subspace_refresh; its scratch is a static device
 * array of ZO_NOALLOC_SCRATCH_BYTES that each GPU the library runs on holds
 * until the process ends (its address is looked up on the first call on each
 * device, with that device current).  The call allocates nothing.
 *   - A call whose zo_subspace_refresh_workspace size exceeds
 *     ZO_NOALLOC_SCRATCH_BYTES returns ZO_ERR_WORKSPACE and launches nothing;
 *     split its panels over several calls.  (Each panel of r <= 64 needs about
 *     (ceil(rows / 2048) + 3) * 32 KiB; of 64 < r <= 128 about
 *     ceil(rows / 1024) * 66 KiB + 384 KiB; plus 72 bytes per panel for the
 *     call's descriptor table.)
 *   - Every call on one GPU uses the same scratch: calls that overlap on one
 *     GPU (on different streams, or from different threads without ordering)
 *     race and give wrong results.  Calls enqueued on one stream are ordered
 *     and safe.  Nothing the scratch holds from an earlier call is read. */
#define ZO_NOALLOC_SCRATCH_BYTES (64u << 20)
int zo_subspace_refresh_noalloc(int count, const zo_panel* panels, int r,
                                int* info, void* stream);

/* ------------------------------------------------------------------------
 * Perturbed linear -- Eq. 4 inside the forward of Eq. 5 (Alg. 2 + Alg. 3).
 *
 * For every block b = 0..nblk-1 (one query j = blk_query[b] with sign
 * s = blk_sign[b] in {+1, -1, 0}):
 *
 *     Y_b = X_b (W + s eps U Z_j V^T)^T
 *         = X_b W^T + (X_b V) (s eps U Z_j)^T
 *
 * computed in the second form: W is only read (bitwise unchanged), the
 * m x n perturbed weight is never formed.
 *
 *   T            rows (tokens) per block; m, n: W is m x n (out x in).
 *   X            device, block b starts at X + b * x_block_stride elements,
 *                each block T x n.  x_block_stride = 0: all blocks share one
 *                X (the first layer of a network); otherwise >= T*n.  With
 *                a shared X and nblk > 1, X W^T is computed once (into an
 *                fp32 T x m region of the workspace, which the workspace size
 *                includes) and each block adds its own rank-r term to it
 *                before the single rounding (plain and ReLU epilogues; the
 *                residual and gated ones compute every block in full).
 *   W            device, m x n.  in_dtype ZO_BF16, ZO_F16 or ZO_F32 for X
 *                and W.
 *   U, V         device fp32, m x r and n x r (column-orthonormal).
 *   Z            device fp32, q x r x r (Z_j row-major).
 *   blk_query    host, nblk ints in [0, q).
 *   blk_sign     host, nblk int8 in {+1, -1, 0}.
 *   Y            device, nblk blocks of T x m, contiguous; out_dtype is
 *                in_dtype or ZO_F32 (fp32 inputs require fp32 output).
 * Arithmetic: bf16 (fp16) inputs use bf16 (fp16) MFMA for X_b W^T with fp32
 * accumulation.  The rank-r term is added into the same accumulators with
 * its operands X_b V and s eps U Z_j each carried as a high + low pair of
 * bf16 (about 16 significant bits, and bf16's range: eps U Z_j entries sit
 * near fp16's smallest normal), so it is ~2^-16 accurate relative to its own
 * size.  X_b V itself is formed by the input type's MFMA from a high + low
 * split of V (for fp16, of 256 V, scaled back exactly).  Outputs rounded to
 * nearest even.  fp32 inputs use fp32 FMA throughout.
 * Limits: 1 <= r <= ZO_MAX_RANK, 1 <= q <= ZO_MAX_QUERIES, 1 <= nblk <=
 * ZO_MAX_BLOCKS; 16-bit inputs need m % 8 == 0 and n % 8 == 0; fp16 inputs
 * need |V| < 255 entrywise (a column-orthonormal V has |V| <= 1; larger
 * entries overflow the scaled split to infinity).
 * ------------------------------------------------------------------------ */
size_t zo_perturbed_linear_workspace(int T, int m, int n, int r, int q, int nblk,
                                     long long x_block_stride, int in_dtype);
int zo_perturbed_linear(int T, int m, int n, int r, int q, int nblk,
                        const int* blk_query, const int8_t* blk_sign, float eps,
                        int in_dtype, const void* X, long long x_block_stride,
                        const void* W, const float* U, const float* V,
                        const float* Z, int out_dtype, void* Y,
                        void* workspace, size_t ws_bytes, void* stream);

/* The same operation in two phases (zo_perturbed_linear = prepare + apply):
 *   prepare  forms the rank-r operands X_b V and s_b eps U Z_{j(b)} in the
 *            workspace (small launches; reads X once);
 *   apply    one GEMM launch: Y_b = X_b W^T plus the prepared rank-r term.
 * apply must be given the same dimensions, X and workspace as the prepare
 * it follows on the same stream, with the workspace untouched in between.
 * Arguments, limits and errors as for zo_perturbed_linear. */
int zo_perturbed_linear_prepare(int T, int m, int n, int r, int q, int nblk,
                                const int* blk_query, const int8_t* blk_sign,
                                float eps, int in_dtype, const void* X,
                                long long x_block_stride, const float* U,
                                const float* V, const float* Z, void* workspace,
                                size_t ws_bytes, void* stream);
int zo_perturbed_linear_apply(int T, int m, int n, int r, int q, int nblk,
                              int in_dtype, const void* X,
                              long long x_block_stride, const void* W,
                              int out_dtype, void* Y, void* workspace,
                              size_t ws_bytes, void* stream);

/* prepare for count perturbed linears that read the same X (a layer's q, k
 * and v): one projection pass reads X once for all of them, against their
 * stacked V factors.  Matrix i has m[i] rows, its own U[i], V[i], Z[i] and its
 * own workspace[i] (ws_bytes[i] bytes, as for zo_perturbed_linear_prepare);
 * T, n, r, q, nblk, the blocks, eps, in_dtype, X and x_block_stride are
 * shared.  group_ws: device scratch of zo_perturbed_linear_group_workspace
 * bytes (0 for fp32 inputs or count = 1, when the call runs the separate
 * prepares; group_ws may then be NULL).  The count workspaces and group_ws
 * must be pairwise disjoint (ZO_ERR_INVALID_ARG otherwise).  The prepared operands are bitwise
 * those of separate prepares; each matrix is then applied with
 * zo_perturbed_linear_apply(_ex) and its own workspace.
 * Limits: 1 <= count <= ZO_MAX_GROUP; those of zo_perturbed_linear. */
size_t zo_perturbed_linear_group_workspace(int count, int T, int n, int r, int q,
                                           int nblk, long long x_block_stride,
                                           int in_dtype);
int zo_perturbed_linear_prepare_group(int count, const int* m, int T, int n,
                                      int r, int q, int nblk,
                                      const int* blk_query,
                                      const int8_t* blk_sign, float eps,
                                      int in_dtype, const void* X,
                                      long long x_block_stride,
                                      const float* const* U,
                                      const float* const* V,
                                      const float* const* Z,
                                      void* const* workspace,
                                      const size_t* ws_bytes, void* group_ws,
                                      size_t group_ws_bytes, void* stream);

/* apply with a fused epilogue on the fp32 result, before its one rounding to
 * out_dtype -- the operations that follow a linear inside the decoder layer
 * of the network the queries evaluate (the forward of Eq. 5):
 *   ZO_EPI_NONE      Y_b = result (zo_perturbed_linear_apply);
 *   ZO_EPI_RELU      Y_b = max(result, 0);
 *   ZO_EPI_RESIDUAL  Y_b = R_b + result, R_b at R + b * r_block_stride
 *                    elements (0: one R for every block), out_dtype, T x m
 *                    rows of stride m.  R may be Y itself.
 *   ZO_EPI_SILU_MUL  Y_b = silu(R_b) * result, silu(x) = x / (1 + e^-x), R_b
 *                    laid out as for ZO_EPI_RESIDUAL (the gated MLP of the
 *                    LLaMA-family layer: R is the gate projection's output).
 * Limits as for zo_perturbed_linear_apply; with 16-bit outputs R is 16-byte
 * aligned and r_block_stride a multiple of 8 (0 or >= T*m). */
int zo_perturbed_linear_apply_ex(int T, int m, int n, int r, int q, int nblk,
                                 int in_dtype, const void* X,
                                 long long x_block_stride, const void* W,
                                 int out_dtype, void* Y, int epilogue,
                                 const void* R, long long r_block_stride,
                                 void* workspace, size_t ws_bytes, void* stream);

/* ------------------------------------------------------------------------
 * Perturbed linear of a LoRA-adapted layer -- Eq. 4 and Alg. 2 applied to
 * the two trainable adapter factors (the LoRA scheme of the experiments,
 * r_L = 8, alpha = 16), inside the forward of Eq. 5.
 *
 * The frozen base W (m x n) carries the adapter A (rl x n) and B (m x rl);
 * each factor has its own rank-r subspace and coefficients.  For every block
 * b (query j = blk_query[b], sign s = blk_sign[b]):
 *
 *     A'  = A + s eps U_A Z_A,j V_A^T          B' = B + s eps U_B Z_B,j V_B^T
 *     Y_b = X_b (W + scale B' A')^T            (scale = alpha / rl)
 *
 * computed without forming W + scale B' A' or A', as the frozen-base GEMM
 * plus a rank-(rl + r) term: X_b [A^T | V_A] times
 * scale [B' | s eps B' U_A Z_A,j] (the second factor is m x (rl + r) per
 * block).  W, A and B are only read.
 *
 *   T, m, n, q, nblk, blk_query, blk_sign, eps, in_dtype, X, x_block_stride,
 *   W, out_dtype, Y   as for zo_perturbed_linear.
 *   rl          adapter rank (rows of A, columns of B).
 *   r           subspace rank of each factor.
 *   scale       the adapter scaling alpha / rl.
 *   A, B        device fp32, rl x n and m x rl (row-major).
 *   U_A, V_A    device fp32, rl x r and n x r.
 *   U_B, V_B    device fp32, m x r and rl x r.
 *   Z_A, Z_B    device fp32, q x r x r each.
 * Arithmetic as for zo_perturbed_linear with rank rl + r (the adapter
 * operands enter the GEMM as high + low bf16 pairs; with fp16 inputs the
 * projection's right factor [A ; V_A^T] needs entries below 255 in
 * magnitude).
 * Limits: rl >= 1, r >= 1, rl + r <= ZO_MAX_RANK; the rest as for
 * zo_perturbed_linear.
 *
 * The two-phase form: zo_lora_perturbed_linear_prepare fills the workspace;
 * then zo_perturbed_linear_apply with rank rl + r (same T, m, n, q, nblk, X,
 * x_block_stride, in_dtype and workspace, on the same stream) adds the
 * frozen-base GEMM and writes Y.  Workspace size:
 * zo_lora_perturbed_linear_workspace (equal to the full-tuning size at rank
 * rl + r).
 * ------------------------------------------------------------------------ */
size_t zo_lora_perturbed_linear_workspace(int T, int m, int n, int rl, int r,
                                          int q, int nblk,
                                          long long x_block_stride,
                                          int in_dtype);
int zo_lora_perturbed_linear(int T, int m, int n, int rl, int r, int q,
                             int nblk, const int* blk_query,
                             const int8_t* blk_sign, float eps, float scale,
                             int in_dtype, const void* X,
                             long long x_block_stride, const void* W,
                             const float* A, const float* U_A,
                             const float* V_A, const float* Z_A,
                             const float* B, const float* U_B,
                             const float* V_B, const float* Z_B,
                             int out_dtype, void* Y, void* workspace,
                             size_t ws_bytes, void* stream);
int zo_lora_perturbed_linear_prepare(int T, int m, int n, int rl, int r, int q,
                                     int nblk, const int* blk_query,
                                     const int8_t* blk_sign, float eps,
                                     float scale, int in_dtype, const void* X,
                                     long long x_block_stride, const float* A,
                                     const float* U_A, const float* V_A,
                                     const float* Z_A, const float* B,
                                     const float* U_B, const float* V_B,
                                     const float* Z_B, void* workspace,
                                     size_t ws_bytes, void* stream);

/* ------------------------------------------------------------------------
 * The network a query evaluates -- the forward inside Eq. 5 (each query's
 * loss is that of the whole model with every matrix perturbed, Alg. 3), as a
 * pre-LN decoder layer of the OPT family:
 *
 *   A = LN1(H);   Q, K, V = A Wq'^T, A Wk'^T, A Wv'^T;   C = attention(Q, K, V)
 *   H2 = H + C Wo'^T;   F = relu(LN2(H2) W1'^T);   H_out = H2 + F W2'^T
 *
 * with each W' = W + s eps U Z_j V^T for block b's query j and sign s (Eq. 4;
 * each matrix has its own U, V, Z).  No biases (the perturbed parameters are
 * the weight matrices).
 * ------------------------------------------------------------------------ */

/* Row-wise layer normalisation: Y = (X - mean) / sqrt(var + eps_ln) * gamma +
 * beta per row of d elements, population variance, statistics in fp32.
 * X, Y: rows x d (dtype, may alias); gamma, beta: device fp32 [d].
 * Limits: d % 8 == 0; 16-byte aligned pointers. */
int zo_layernorm(long long rows, int d, int dtype, const void* X,
                 const float* gamma, const float* beta, float eps_ln, void* Y,
                 void* stream);

/* The same layer of the LLaMA family (pre-norm, RMS normalisation, rotary
 * positions on queries and keys, SwiGLU MLP, no biases):
 *
 *   A = RMS1(H);   Q = rope(A Wq'^T);   K = rope(A Wk'^T);   V = A Wv'^T
 *   C = attention(Q, K, V);   H2 = H + C Wo'^T;   A2 = RMS2(H2)
 *   H_out = H2 + (silu(A2 Wg'^T) * (A2 Wu'^T)) Wd'^T
 *
 * Row-wise RMS normalisation: Y = X / sqrt(mean(X^2) + eps) * gamma per row of d
 * elements, statistics in fp32.  X, Y: rows x d (dtype, may alias); gamma:
 * device fp32 [d]; eps finite and >= 0; rows = 0 launches nothing.
 * Limits: d % 8 == 0; 16-byte aligned pointers. */
int zo_rmsnorm(long long rows, int d, int dtype, const void* X,
               const float* gamma, float eps, void* Y, void* stream);

/* Rotary position embedding, in place: X is rows x d (bf16 or fp16) holding
 * sequences of seq_len rows one after another (a row's position p is its index
 * within its sequence); in each head (dh = d / heads columns) dimension
 * i < dh/2 and dimension i + dh/2 are rotated together by the angle
 * p * base^(-2i/dh): (a, b) -> (a cos - b sin, b cos + a sin).  The angle is
 * formed and reduced modulo 2 pi in fp64, its sine and cosine and the rotation
 * taken in fp32, one rounding to the dtype.  Limits: rows % seq_len == 0;
 * dh % 16 == 0; base > 1; 16-byte aligned X. */
int zo_rope(long long rows, int seq_len, int d, int heads, int dtype, void* X,
            float base, void* stream);

/* Multi-head causal self-attention.  Q, K, V, O: nblk blocks of T rows x d
 * (dtype bf16 or fp16, row-major, contiguous blocks); each block holds
 * T / seq_len sequences one after another; head h is columns h dh ..
 * (h+1) dh - 1 (dh = d / heads).  Query t of a sequence attends to its keys
 * t' <= t with weights softmax(q_t . k_t' / sqrt(dh)).  fp32 softmax; the
 * products run on the MFMA with P as a hi + lo 16-bit pair (~2^-16 relative
 * before the output's rounding to dtype).
 * Limits: T % seq_len == 0; dh = 64 or 128; 16-byte aligned pointers. */
int zo_causal_attention(int nblk, int T, int seq_len, int d, int heads,
                        int dtype, const void* Q, const void* K, const void* V,
                        void* O, void* stream);

/* The same with grouped key/value heads (the Qwen models of the experiments):
 * K and V are nblk blocks of T rows x kv_heads dh (dh = d / heads), and query
 * head h reads key/value head h / (heads / kv_heads).  zo_causal_attention is
 * this call with kv_heads = heads.  Limits: heads % kv_heads == 0; the rest as
 * for zo_causal_attention. */
int zo_causal_attention_gqa(int nblk, int T, int seq_len, int d, int heads,
                            int kv_heads, int dtype, const void* Q,
                            const void* K, const void* V, void* O,
                            void* stream);

/* One perturbed matrix: W (m x n, the layer's dtype), U (m x r), V (n x r)
 * and Z (q x r x r) fp32. */
typedef struct {
  const void* W;
  const float* U;
  const float* V;
  const float* Z;
} zo_matrix;

/* A decoder layer: q, k, v, o (d x d), fc1 (ffn x d), fc2 (d x ffn), and the
 * two layer norms' gamma / beta (device fp32 [d]). */
typedef struct {
  zo_matrix q, k, v, o, fc1, fc2;
  const float* ln1_gamma;
  const float* ln1_beta;
  const float* ln2_gamma;
  const float* ln2_beta;
} zo_decoder_layer;

/* The layer for all nblk blocks at once (block b: query blk_query[b], sign
 * blk_sign[b], as for zo_perturbed_linear).  H: the layer input, one T x d
 * for every block (h_block_stride = 0: the model's first layer) or nblk
 * contiguous blocks (h_block_stride = T*d); H_out: nblk blocks of T x d (may
 * alias H when h_block_stride = T*d).  The six products are perturbed
 * linears (zo_perturbed_linear_apply_ex: ReLU after fc1, the residuals fused
 * into o and fc2); intermediate activations are stored in dtype in the
 * workspace (zo_decoder_layer_workspace bytes).
 * Limits: dtype bf16 or fp16; those of zo_causal_attention and of
 * zo_perturbed_linear for each matrix. */
size_t zo_decoder_layer_workspace(int T, int seq_len, int d, int heads, int ffn,
                                  int r, int q, int nblk, int dtype);
int zo_decoder_layer_forward(int T, int seq_len, int d, int heads, int ffn,
                             int r, int q, int nblk, const int* blk_query,
                             const int8_t* blk_sign, float eps, float eps_ln,
                             int dtype, const void* H, long long h_block_stride,
                             const zo_decoder_layer* layer, void* H_out,
                             void* workspace, size_t ws_bytes, void* stream);

/* A LLaMA-family layer: q, k, v, o (d x d), gate, up (ffn x d), down
 * (d x ffn), and the two RMS norms' gamma (device fp32 [d]). */
typedef struct {
  zo_matrix q, k, v, o, gate, up, down;
  const float* rms1_gamma;
  const float* rms2_gamma;
} zo_llama_layer;

/* The LLaMA-family layer for all nblk blocks at once; arguments as for
 * zo_decoder_layer_forward, with eps_rms for the RMS norms and rope_base for
 * the rotary angles.  The seven products are perturbed linears (the residuals
 * fused into o and down, silu(gate) * up fused into up); intermediate
 * activations are stored in dtype in the workspace
 * (zo_llama_layer_workspace bytes).
 * Limits: dtype bf16 or fp16; those of zo_causal_attention, of zo_rope and of
 * zo_perturbed_linear for each matrix. */
size_t zo_llama_layer_workspace(int T, int seq_len, int d, int heads, int ffn,
                                int r, int q, int nblk, int dtype);
int zo_llama_layer_forward(int T, int seq_len, int d, int heads, int ffn,
                           int r, int q, int nblk, const int* blk_query,
                           const int8_t* blk_sign, float eps, float eps_rms,
                           float rope_base, int dtype, const void* H,
                           long long h_block_stride, const zo_llama_layer* layer,
                           void* H_out, void* workspace, size_t ws_bytes,
                           void* stream);

/* ------------------------------------------------------------------------
 * Subspace Adam update -- Eqs. 6-10 and the tail of Alg. 3.
 *
 * With q global estimates g_j (shared by every matrix, e.g. the central
 * differences (L+_j - L-_j) / (2 eps)), for each item:
 *
 *     Zbar = (1/q) sum_j g_j Z_j                          (r x r)
 *     M1  <- beta1 M1 + (1 - beta1) Zbar                  (Eq. 7)
 *     M2  <- beta2 M2 + (1 - beta2) Zbar * Zbar           (Eq. 8)
 *     S    = (M1 / (1 - beta1^t)) / (sqrt(M2 / (1 - beta2^t)) + eps_adam)
 *     W   <- W - lr U S V^T                               (Eq. 10)
 *
 * t >= 1 is the 1-based Adam step.  The r x r work is float64 inside; the
 * moments are stored fp32.  The m x n product is accumulated in fp32
 * (bf16 or fp16 W: MFMA on a hi+lo bf16 split of lr U S and V; fp32 W: fp32
 * FMA), added to W in fp32 and rounded to nearest even when W is bf16 or
 * fp16 (fp16 overflows to infinity, as IEEE rounding does).
 *
 *   W          device m x n (w_dtype), updated in place.
 *   U, V, Z    device fp32: m x r, n x r, q x r x r.
 *   M1, M2     device fp32 r x r, updated in place.
 *   zbar_out   device fp32 r x r, nullable: Zbar.
 *   w_f32_out  device fp32 m x n, nullable: the new W before its storage
 *              rounding (a check hook).
 *   g          device fp32, q values.
 *   nonfinite_flag  device int, nullable.  If Zbar or S of an item has a
 *              non-finite entry, that item's W, M1 and M2 are left untouched
 *              and *nonfinite_flag is set to 1 (never cleared here).
 * Limits: 1 <= r <= ZO_MAX_RANK, 1 <= q <= ZO_MAX_QUERIES; 16-bit W needs
 * n % 8 == 0 and n <= 2^20 (a 512-row tile of W and of w_f32_out must stay
 * under 2^31 bytes).
 * ------------------------------------------------------------------------ */
typedef struct {
  int m, n;
  void* W;
  const float* U;
  const float* V;
  const float* Z;
  float* M1;
  float* M2;
  float* zbar_out;
  float* w_f32_out;
} zo_update_item;

size_t zo_subspace_adam_update_workspace(int count, const zo_update_item* items,
                                         int r, int q, int w_dtype);
int zo_subspace_adam_update(int count, const zo_update_item* items, int w_dtype,
                            int r, int q, const float* g, int t, float lr,
                            float beta1, float beta2, float eps_adam,
                            int* nonfinite_flag, void* workspace,
                            size_t ws_bytes, void* stream);

/* ------------------------------------------------------------------------
 * Subspace SGD update -- the "SubZero+/SGD" variant of the experiments and,
 * with q = 1, SubZero's own update (Sec. "Preliminaries": W <- W - eta g
 * U Z V^T).  For each item:
 *
 *     Zbar = (1/q) sum_j g_j Z_j,     W <- W - lr U Zbar V^T
 *
 * Arguments, arithmetic, workspace rules and the non-finite guard as for
 * zo_subspace_adam_update; M1 and M2 are neither read nor written (may be
 * NULL).  zo_subspace_sgd_update_workspace gives the workspace size.
 * ------------------------------------------------------------------------ */
size_t zo_subspace_sgd_update_workspace(int count, const zo_update_item* items,
                                        int r, int q, int w_dtype);
int zo_subspace_sgd_update(int count, const zo_update_item* items, int w_dtype,
                           int r, int q, const float* g, float lr,
                           int* nonfinite_flag, void* workspace,
                           size_t ws_bytes, void* stream);

/* ------------------------------------------------------------------------
 * Squared-error loss per block (the loss of a one-layer regression model):
 * out[b] = 0.5 * sum((Y_b - Ystar)^2) / T, float64 accumulation in a fixed
 * order.  Y: nblk blocks of T x m (dtype: ZO_F32, ZO_BF16 or ZO_F16), Ystar:
 * T x m (same dtype), out: device float64 [nblk].
 * ------------------------------------------------------------------------ */
size_t zo_sq_loss_workspace(int nblk, int T, int m);
int zo_sq_loss(int nblk, int T, int m, int dtype, const void* Y,
               const void* Ystar, double* out, void* workspace,
               size_t ws_bytes, void* stream);

/* Central difference of Eq. 3 for every query:
 * g[j] = (L[2j] - L[2j+1]) / (2 eps), L device float64 [2q] (block 2j is the
 * + perturbation, 2j+1 the - one), g device fp32 [q]; float64 arithmetic. */
int zo_combine_central(int q, const double* L, float eps, float* g,
                       void* stream);

/* Forward difference of Eq. 6 (Alg. 3's estimator, one baseline and q
 * perturbed forwards): g[j] = (L[1 + j] - L[0]) / eps, L device float64
 * [q + 1] (block 0 is the unperturbed baseline, blk_sign 0; block 1 + j is
 * query j with sign +1), g device fp32 [q]; float64 arithmetic. */
int zo_combine_forward(int q, const double* L, float eps, float* g,
                       void* stream);

/* ------------------------------------------------------------------------
 * The LLaMA-family layer of the LoRA scheme (the Qwen models of the
 * experiments, Sec. "Experiments"; Eq. 4 / Alg. 2 on the adapter factors):
 * grouped key/value heads, a frozen base, and LoRA adapters on q and v whose
 * factors are the perturbed parameters:
 *
 *   A = RMS1(H);   Q = rope(A (Wq + scale B_q' A_q')^T);   K = rope(A Wk^T)
 *   V = A (Wv + scale B_v' A_v')^T;   C = attention(Q, K, V; kv_heads)
 *   H2 = H + C Wo^T;   A2 = RMS2(H2);   H_out = H2 + (silu(A2 Wg^T) * (A2 Wu^T)) Wd^T
 *
 * with A' and B' as for zo_lora_perturbed_linear (each factor in its own
 * subspace, block b's query and sign).  No biases.
 * ------------------------------------------------------------------------ */
/* An adapted matrix: the frozen W (m x n, the layer's dtype) and the adapter
 * factors with their subspaces and coefficients, as for
 * zo_lora_perturbed_linear (A rl x n, B m x rl, fp32). */
typedef struct {
  const void* W;
  const float* A;
  const float* U_A;
  const float* V_A;
  const float* Z_A;
  const float* B;
  const float* U_B;
  const float* V_B;
  const float* Z_B;
} zo_lora_matrix;

/* q (d x d) and v (kv_heads dh x d) adapted; the frozen k (kv_heads dh x d),
 * o (d x d), gate, up (ffn x d), down (d x ffn); the RMS norms' gamma. */
typedef struct {
  zo_lora_matrix q, v;
  const void* k;
  const void* o;
  const void* gate;
  const void* up;
  const void* down;
  const float* rms1_gamma;
  const float* rms2_gamma;
} zo_llama_lora_layer;

/* The layer for all nblk blocks at once; H, h_block_stride, H_out, eps_rms,
 * rope_base, dtype and the workspace as for zo_llama_layer_forward; rl, r,
 * scale as for zo_lora_perturbed_linear.  The frozen products run the fused
 * GEMM without a rank-r segment (the residuals fused into o and down,
 * silu(gate) * up into up); the adapted ones run it at rank rl + r.
 * Limits: those of zo_causal_attention_gqa, zo_rope and
 * zo_lora_perturbed_linear for q and v. */
size_t zo_llama_lora_layer_workspace(int T, int seq_len, int d, int heads,
                                     int kv_heads, int ffn, int rl, int r,
                                     int q, int nblk, int dtype);
int zo_llama_lora_layer_forward(int T, int seq_len, int d, int heads,
                                int kv_heads, int ffn, int rl, int r, int q,
                                int nblk, const int* blk_query,
                                const int8_t* blk_sign, float eps, float scale,
                                float eps_rms, float rope_base, int dtype,
                                const void* H, long long h_block_stride,
                                const zo_llama_lora_layer* layer, void* H_out,
                                void* workspace, size_t ws_bytes, void* stream);

#ifdef __cplusplus
}
#endif
#endif /* ZO_H */
