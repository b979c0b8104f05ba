/*
 * bt.h -- C ABI of libbt, an MI355X (gfx950) implementation of one FP32 GPT-2
 * training step on one GPU's data-parallel shard.
 *
 * The operations follow the paper's statement of the problem: the layer
 * definitions, every forward and backward operator and the AdamW step of a
 * GPT-2 decoder (Evaluation section: GPT-2 architecture figure caption and
 * the "Training hyperparameters" table), the per-kernel list of the
 * "Performance Benchmarks" appendix (attention, GELU, LayerNorm, sparse
 * cross-entropy, reduce-sum, AdamW), the dense projections served by the
 * native GEMM library ("Implementation", native GEMM library paragraph) and
 * the micro-step loop of Algorithm "Distributed Data Parallel Training Step".
 *
 * Conventions for every entry point
 *  - Pointers are DEVICE pointers unless a comment says "host".  All floating
 *    point tensors are FP32, row-major, contiguous unless a leading dimension
 *    is given.  Integer tensors are int32.
 *  - The caller owns every buffer.  libbt never allocates, frees or keeps
 *    device memory; scratch space is passed in as a workspace (ws) whose size
 *    is given by the matching *_ws_bytes query.
 *  - `stream` is a hipStream_t passed as void* (NULL = the null stream).  All
 *    work is enqueued asynchronously on it; only bt_gpt2_train_step blocks
 *    the host (once, to return the loss).
 *  - Arguments are validated before anything is launched.  On a violation a
 *    BT_E* code is returned, nothing is launched and bt_last_error() gives a
 *    thread-local detail string.  A failed launch returns BT_EHIP.
 *  - Alignment: every float pointer must be 16-byte aligned; leading
 *    dimensions and the dimensions named "vectorised" must be multiples of 4.
 *  - Results are deterministic: no floating-point atomics, fixed-order
 *    reductions, so identical calls give bitwise identical results.
 */
#ifndef BT_H
#define BT_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  BT_OK = 0,
  BT_EINVAL = 1,      /* NULL pointer or out-of-range scalar argument */
  BT_ESHAPE = 2,      /* inconsistent or unsupported shape */
  BT_EALIGN = 3,      /* pointer or leading dimension not suitably aligned */
  BT_EWORKSPACE = 4,  /* workspace missing or smaller than the query says */
  BT_EHIP = 5,        /* a HIP runtime call or kernel launch failed */
  BT_ENONFINITE = 6   /* non-finite gradient norm: the optimizer step was skipped */
} bt_status;

const char* bt_status_str(bt_status s);
/* Detail string and status of the last failure on this host thread.  Every
 * entry point that returns a bt_status (and bt_gpt2_train_step) clears both
 * when it starts, so after a successful call they are "" and BT_OK. */
const char* bt_last_error(void);
bt_status bt_last_status(void);
/* Library version, "major.minor.patch". */
const char* bt_version(void);

typedef enum { BT_OP_N = 0, BT_OP_T = 1 } bt_op;

typedef enum {
  BT_EPI_NONE = 0,      /* out = acc */
  BT_EPI_BIAS = 1,      /* out = acc + bias[n] */
  BT_EPI_BIAS_GELU = 2, /* pre = acc + bias[n]; optional preact_out = pre; out = gelu(pre) */
  BT_EPI_DGELU = 3      /* out = acc * gelu'(gelu_in[m, n])  (GELU backward fused) */
} bt_epi;

/*
 * Dense product (native GEMM library paragraph of "Implementation": QKV,
 * attention-output and MLP projections in forward and backward layouts).
 *
 *   C[m, n] = epi( sum_k op(A)[m, k] * op(B)[k, n] ) + residual[m, n] + beta * C[m, n]
 *
 * op(A) is A (M x K, lda >= K) for BT_OP_N or A^T with A stored K x M
 * (lda >= M) for BT_OP_T; likewise op(B) is B (K x N, ldb >= N) or B^T with
 * B stored N x K (ldb >= K).  C is M x N with ldc >= N.  beta is 0 or 1
 * (1 = accumulate into C, used for gradient accumulation).
 * bias [N] is required for BIAS / BIAS_GELU.  preact_out (M x N, ldc) is
 * optional for BIAS_GELU.  gelu_in (M x N, ldc) is required for DGELU.
 * residual (M x N, ldc) is optional and must not alias C.
 * M, N, K >= 0 (an empty product writes beta*C + residual with acc = 0; with
 * K = 0 the epilogue still applies).  M, N, K, lda, ldb, ldc must be
 * multiples of 4.  FP32 inputs, FP32 accumulation on the matrix cores.
 * colsum_B (optional, [N]) receives the column sums of op(B) over K,
 *   colsum_B[n] = beta * colsum_B[n] + sum_k op(B)[k, n],
 * i.e. the bias gradient sum_m dY[m, n] of a weight-gradient product
 * dW = X^T dY, computed from the dY tiles the product already reads.  It
 * requires opB = BT_OP_N, epi = BT_EPI_NONE and no residual.
 * ws may be NULL when bt_gemm_ws_bytes() returns 0 for the shape; otherwise
 * it must hold that many bytes (split-K partial products; any epilogue may
 * be split, which applies it in the fixed-order reduction of the partials).
 * Too small a workspace for a split shape: BT_EWORKSPACE, nothing launched.
 */
bt_status bt_gemm(bt_op opA, bt_op opB, int M, int N, int K,
                  const float* A, int lda, const float* B, int ldb,
                  float beta, float* C, int ldc,
                  const float* bias, bt_epi epi, float* preact_out, const float* gelu_in,
                  const float* residual, float* colsum_B, void* ws, size_t ws_bytes,
                  void* stream);
size_t bt_gemm_ws_bytes(bt_op opA, bt_op opB, int M, int N, int K, bt_epi epi);
/* The launch plan bt_gemm uses for a product, computed on the host (no
 * device work): *tile_depth, the k-depth of its 128 x 128 block tile (16 or
 * 32); *splits, the number of K ranges whose partial products are summed in
 * a fixed order (1 = not split; bt_gemm_ws_bytes() > 0 exactly when > 1);
 * *direct, 1 when its operand tiles are copied straight into LDS (every tile
 * full), 0 when they are staged with bounds checks.  The plan depends only on
 * (opA, opB, M, N, K) and the leading dimensions, not on the epilogue.
 * M, N, K positive multiples of 4, else BT_ESHAPE; NULL outputs BT_EINVAL. */
bt_status bt_gemm_plan(bt_op opA, bt_op opB, int M, int N, int K, int lda, int ldb, int* tile_depth,
                       int* splits, int* direct);

/*
 * bt_gemm for callers that cannot allocate device memory: code under HIP
 * graph capture, tight serving loops, harnesses that forbid hipMalloc.  Same
 * operation, arguments and results as bt_gemm (bitwise: the same kernels and
 * split), minus ws/ws_bytes: the split-K partials go to a static device
 * array of the library, bt_gemm_noalloc_max_ws_bytes() = 64 MiB, held by
 * every GPU the library runs on until the process ends (its device address
 * is looked up once per device on the first call there).  A product whose
 * bt_gemm_ws_bytes() exceeds that returns BT_EWORKSPACE before anything is
 * launched (at GPT-2 124M, B = 16: every per-layer product fits; the tied
 * LM head's input and weight gradients do not).  The call allocates nothing.
 * All calls on one GPU share the one array, which keeps the last call's
 * partials: calls that overlap on a GPU (several streams or host threads)
 * race and must be serialised by the caller.
 */
bt_status bt_gemm_noalloc(bt_op opA, bt_op opB, int M, int N, int K,
                          const float* A, int lda, const float* B, int ldb,
                          float beta, float* C, int ldc,
                          const float* bias, bt_epi epi, float* preact_out, const float* gelu_in,
                          const float* residual, float* colsum_B, void* stream);
size_t bt_gemm_noalloc_max_ws_bytes(void);

/*
 * Causal multi-head self-attention forward (GPT-2 architecture figure:
 * masked multi-head self-attention; appendix "Attention Forward", causal
 * case).  Per batch b and head h: S = Q K^T / sqrt(hd) with key j visible to
 * query i iff j <= i, P = softmax(S) row-wise, O = P V.
 *   qkv [B, T, 3, H, hd]   (the QKV projection output, [B*T, 3*H*hd])
 *   out [B, T, H, hd]      (written)
 *   lse [B, H, T]          (written; natural-log sum of exp of each score row)
 * hd a multiple of 4, at most 128 (zero-padded to 32, 64 or 128 inside the
 * kernels; 128 is the head dim of the 2.42B configuration).  T >= 1,
 * B, H >= 1.  qkv and out 16-byte aligned.  Otherwise BT_ESHAPE / BT_EALIGN.
 */
bt_status bt_attention_fwd(const float* qkv, float* out, float* lse,
                           int B, int T, int H, int hd, void* stream);

/*
 * Causal attention backward (appendix "Attention Backward").  From dout
 * [B, T, H, hd], qkv, out and lse of the forward it writes dqkv [B, T, 3, H,
 * hd] (overwritten).  P is recomputed from lse.  Deterministic (no atomics).
 * ws (16-byte aligned, caller-owned, contents scratch) selects the method:
 *  - ws_bytes >= bt_attention_bwd_ws_bytes(): the row sums D = rowsum(dout *
 *    out), then a key-major pass that accumulates dK, dV and stores
 *    dS / sqrt(hd) ([B, H, T, T] floats in ws), then dQ = dS K as one batched
 *    product.  Needs T % 4 == 0; for other T the size function returns the
 *    minimum and the second method runs.
 *  - bt_attention_bwd_ws_min_bytes() <= ws_bytes < that: a query-major pass
 *    (D and dQ, recomputing S and dP) and the key-major pass (dK, dV); no
 *    memory quadratic in T.
 * Smaller (or NULL) ws: BT_EWORKSPACE.
 */
bt_status bt_attention_bwd(const float* dout, const float* qkv, const float* out,
                           const float* lse, float* dqkv, void* ws, size_t ws_bytes,
                           int B, int T, int H, int hd, void* stream);
size_t bt_attention_bwd_ws_bytes(int B, int T, int H, int hd);
size_t bt_attention_bwd_ws_min_bytes(int B, int T, int H, int hd);

/*
 * ---- Context parallelism: one rank's share of ring attention ----
 * Section "Context Parallelism": the sequence is spread over W ranks; the
 * key/value shards travel around a ring; at each step a rank attends its
 * local queries to the shard it holds, giving a partial output and its
 * log-sum-exp, and folds them into its running (out, lse) with the
 * sigmoid-scaled update; the backward recomputes the scores shard by shard
 * and sends each shard's dK/dV around the ring with it.  Token chunks are
 * rearranged once where the data is loaded so that every rank carries the
 * same causal work: the sequence is cut into 2W equal chunks and rank r
 * holds chunks r and 2W-1-r.  These calls are the per-rank kernels; moving
 * the shards between GPUs is the caller's.
 *
 * Positions: a side's rows are n (1 or 2) contiguous segments of `seg`
 * tokens; segment i starts at global token position pos[i].  Key j is visible
 * to query i iff position(j) <= position(i).
 */
typedef struct {
  int seg;       /* tokens per segment: a positive multiple of 128 */
  int n_q, n_k;  /* segments of the query rows and of the key/value rows: 1 or 2 */
  int q_pos[2];  /* global position of each query segment's first token (multiple of 32, >= 0) */
  int k_pos[2];  /* same for the key/value segments */
} bt_cp_segments;

/*
 * Segments of rank `rank`'s queries and of the shard owned by rank `shard`
 * under the load-balanced split above (seg = T / (2W), two segments a side).
 * Host only; writes *out.  T must be a multiple of 2 W 128 (BT_ESHAPE);
 * ranks outside [0, W): BT_EINVAL.
 */
bt_status bt_cp_rank_segments(int T, int W, int rank, int shard, bt_cp_segments* out);

/*
 * The rearrangement at the data-loading boundary: local [B, T/W] (int32,
 * device, written) = rank `rank`'s two chunks of each row of tokens [B, T]
 * (int32, device), in order.  Same size rules as bt_cp_rank_segments.
 */
bt_status bt_cp_shard_tokens(const int32_t* tokens, int32_t* local, int B, int T, int W, int rank,
                             void* stream);

/*
 * Forward of one ring step.  Queries: the Q part of the rank's local qkv
 * [B, Tq, 3, H, hd] with Tq = n_q seg.  Keys and values of the shard: row t of
 * batch b at kv + (b Tk + t) kv_stride (K) and + H hd (V), Tk = n_k seg; a
 * view into the owner's qkv (kv = qkv + H hd, kv_stride = 3 H hd) or a packed
 * [B, Tk, 2, H, hd] buffer (kv_stride = 2 H hd) both fit.  kv_stride a
 * multiple of 4 and >= 2 H hd.
 *   merge = 0: out [B, Tq, H, hd] and lse [B, H, Tq] are written with this
 *              shard's attention; a query with no visible key gets a zero
 *              row and lse = -inf.
 *   merge = 1: (out, lse) hold the running state and are updated in place:
 *              out <- out - sigmoid(blse - lse) (out - bout),
 *              lse <- lse - log sigmoid(lse - blse); a row whose block is
 *              empty keeps its state, a row whose state is empty (lse = -inf)
 *              takes the block.
 * hd as bt_attention_fwd.  Errors: BT_ESHAPE (segments, sizes), BT_EALIGN
 * (qkv, out, kv not 16-byte aligned), BT_EINVAL (NULL, merge not 0/1).
 */
bt_status bt_attention_block_fwd(const float* qkv, const float* kv, long long kv_stride, float* out,
                                 float* lse, int merge, int B, int H, int hd,
                                 const bt_cp_segments* segs, void* stream);

/*
 * The sigmoid-scaled update on its own, for a partial result computed
 * elsewhere: out [B, T, H, hd], lse [B, H, T] updated in place by block_out,
 * block_lse of the same layout (rules as merge = 1 above).
 */
bt_status bt_attention_lse_merge(float* out, float* lse, const float* block_out, const float* block_lse,
                                 int B, int T, int H, int hd, void* stream);

/*
 * D = rowsum(dout o out) per head, D [B, H, T] (written), from the rank's
 * final output out and its gradient dout [B, T, H, hd].  Computed once per
 * rank before the backward ring.
 */
bt_status bt_attention_rowdot(const float* dout, const float* out, float* D, int B, int T, int H, int hd,
                              void* stream);

/*
 * Backward of one ring step, given the final lse [B, H, Tq] (after every
 * merge) and D: P = exp(S - lse) on visible entries, dV = P^T dO,
 * dS = P o (dO V^T - D), dQ = dS K / sqrt(hd), dK = dS^T Q / sqrt(hd).
 * dQ goes to the Q part of dqkv [B, Tq, 3, H, hd] (its K and V parts are not
 * touched); dK and dV of the shard go to dkv, laid out as kv (same
 * kv_stride).  accumulate: bit 0 adds into dQ, bit 1 adds into dK/dV (else
 * they are overwritten).  Deterministic.
 * ws (16-byte aligned, caller-owned scratch) selects the method:
 *  - ws_bytes >= bt_attention_block_bwd_ws_bytes() > 0: a key-major pass
 *    (dK, dV) that also stores dS / sqrt(hd) ([B, H, Tq, Tk] floats in ws),
 *    then dQ (+)= dS K as one batched matrix-core product over the visible
 *    key range of each 128-row tile.  Needs every segment position to be a
 *    multiple of 128 (the load-balanced split's are); otherwise the size
 *    function returns 0.
 *  - otherwise (ws may be NULL): a query-major pass recomputes S and dP for
 *    dQ and the key-major pass gives dK, dV; no workspace.
 * Errors as bt_attention_block_fwd; gradients must not alias inputs
 * (BT_EINVAL).
 */
bt_status bt_attention_block_bwd(const float* dout, const float* qkv, const float* kv, long long kv_stride,
                                 const float* lse, const float* D, float* dqkv, float* dkv,
                                 int accumulate, void* ws, size_t ws_bytes, int B, int H, int hd,
                                 const bt_cp_segments* segs, void* stream);
size_t bt_attention_block_bwd_ws_bytes(int B, int H, int hd, const bt_cp_segments* segs);

/*
 * LayerNorm forward over the last dimension (pre-normalised blocks of the
 * GPT-2 architecture figure; appendix "LayerNorm Forward"):
 *   mean = sum_c x / C, var = sum_c (x - mean)^2 / C, rstd = 1/sqrt(var + eps)
 *   y = gamma * (x - mean) * rstd + beta
 * x, y [M, C]; mean, rstd [M] (written, for the backward).  C multiple of 4,
 * C <= 4096, M >= 0 (M = 0 writes nothing).  y must not alias x.
 */
bt_status bt_layernorm_fwd(const float* x, const float* gamma, const float* beta,
                           float* y, float* mean, float* rstd, int M, int C, float eps,
                           void* stream);

/*
 * LayerNorm backward (appendix "LayerNorm Backward").  With
 * xhat = (x - mean) * rstd and g = dy * gamma:
 *   dx     = dx_beta * dx + rstd * (g - mean_c(g) - xhat * mean_c(g * xhat))
 *   dgamma = param_beta * dgamma + sum_m dy * xhat
 *   dbeta  = param_beta * dbeta  + sum_m dy
 * dx_beta, param_beta in {0, 1}.  dx may alias dy only when dx_beta == 0.
 * ws holds bt_layernorm_bwd_ws_bytes(M, C) bytes (per-block column partials,
 * reduced in a fixed order).  M = 0 (no rows): dx is not written and the
 * parameter gradients become param_beta times themselves (zeros at 0).
 */
bt_status bt_layernorm_bwd(const float* dy, const float* x, const float* gamma,
                           const float* mean, const float* rstd, float* dx, float* dgamma,
                           float* dbeta, float dx_beta, float param_beta, void* ws,
                           size_t ws_bytes, int M, int C, void* stream);
size_t bt_layernorm_bwd_ws_bytes(int M, int C);

/*
 * tanh-form GELU (GPT-2 figure: GELU feed-forward sublayer; appendix "GELU
 * Forward / Backward"):  gelu(x) = x/2 (1 + tanh(sqrt(2/pi)(x + 0.044715 x^3))).
 * bt_gelu_fwd: y = gelu(x).  bt_gelu_bwd: dx = dy * gelu'(x); dx may alias dy.
 * n must be a multiple of 4; n = 0 writes nothing.
 */
bt_status bt_gelu_fwd(const float* x, float* y, size_t n, void* stream);
bt_status bt_gelu_bwd(const float* x, const float* dy, float* dx, size_t n, void* stream);

/*
 * Sparse (integer-target) softmax cross-entropy over the first V of Vp
 * columns (Algorithm "Distributed Data Parallel Training Step": cross-entropy
 * of the forward against the target; appendix "Sparse Cross-Entropy Loss").
 *   lse[m]       = log sum_{j<V} exp(z[m, j])
 *   loss_rows[m] = lse[m] - z[m, targets[m]]
 * targets in [0, V).  Vp multiple of 4, V <= Vp, M >= 0 (M = 0 writes
 * nothing, in all three calls).  The targets live on the
 * device and are not checked on the host: a row whose target lies outside
 * [0, V) gets a NaN loss and (in the backward and fused calls) a NaN gradient
 * in its columns < V, so that a training step over it reports a non-finite
 * gradient norm and skips its update instead of training toward a wrong
 * class.
 */
bt_status bt_softmax_xent_fwd(const float* logits, const int32_t* targets, float* loss_rows,
                              float* lse, int M, int V, int Vp, void* stream);
/* dlogits[m, j] = (exp(z[m, j] - lse[m]) - [j == targets[m]]) * scale for j < V, 0 for
 * j >= V.  dlogits may alias logits (in place). */
bt_status bt_softmax_xent_bwd(const float* logits, const float* lse, const int32_t* targets,
                              float* dlogits, float scale, int M, int V, int Vp, void* stream);
/* Fused forward + backward in one pass over each row: writes loss_rows and lse
 * and overwrites logits with dlogits (scale as above). */
bt_status bt_softmax_xent_fused(float* logits, const int32_t* targets, float* loss_rows,
                                float* lse, float scale, int M, int V, int Vp, void* stream);

/*
 * AdamW over one flat arena, one launch ("Implementation: Horizontal Tensor
 * Fusion"; hyper-parameter table).  For every element i < n, with
 * c = *grad_scale (1 if grad_scale is NULL) and d = (i < n_decay):
 *   g = c * g[i];  m = b1 m + (1-b1) g;  v = b2 v + (1-b2) g^2
 *   p = p - lr*wd*d*p - lr * (m / (1-b1^t)) / (sqrt(v / (1-b2^t)) + eps)
 * If *grad_scale is not finite, nothing is written (p, m, v keep their
 * values): a non-finite gradient norm skips the step.
 * t >= 1.  n and n_decay multiples of 4, n_decay <= n (n = 0 writes
 * nothing).  The scalars are
 * host doubles: 1 - beta and the bias corrections are formed in double and
 * rounded to FP32 once (0.999 itself is not an FP32 number; 1 - 0.999f would
 * be off by 1.3e-5 relative).
 */
bt_status bt_adamw_step(float* p, const float* g, float* m, float* v, size_t n, size_t n_decay,
                        double lr, double beta1, double beta2, double eps, double weight_decay, int t,
                        const float* grad_scale, void* stream);

/*
 * Global gradient-norm clip (hyper-parameter table: gradient clip 1.0):
 *   norm = sqrt(sum_i g[i]^2);  coef = min(1, clip / (norm + 1e-6))  (coef = 1 if clip <= 0)
 * and coef = NaN whenever norm is not finite (a NaN or Inf gradient), with or
 * without clipping, so that bt_adamw_step given this coefficient skips the
 * update.  Writes the two device scalars out_norm[0], out_coef[0].
 * Fixed-order two-stage reduction.  ws holds bt_grad_norm_ws_bytes(n) bytes.
 * n multiple of 4; n = 0 is an empty sum (norm 0).
 */
bt_status bt_grad_norm_clip(const float* g, size_t n, float clip, float* out_norm,
                            float* out_coef, void* ws, size_t ws_bytes, void* stream);
size_t bt_grad_norm_ws_bytes(size_t n);

/*
 * Embeddings with learned positions and the token table tied to the LM head
 * (GPT-2 architecture figure).  tokens [B, T] int32 (values outside [0, Vp)
 * are clamped to that range).  C a multiple of 4, 0 < Vp <= 2^24, B, T >= 0,
 * B*T*C/4 < 2^31; otherwise BT_ESHAPE.  With B*T = 0 there are no
 * positions: x0 and dwte are not written, and the rows t < T of dwpe become
 * wpe_beta * dwpe (zeros at wpe_beta = 0).
 * fwd: x0[b, t, :] = wte[tokens[b, t], :] + wpe[t, :]            (x0 [B*T, C])
 * bwd: dwte[v, :] += sum over positions with token v of dx0       (always accumulates)
 *      dwpe[t, :]  = wpe_beta * dwpe[t, :] + sum_b dx0[b, t, :]    (rows t < T; wpe_beta 0 or 1)
 * The backward groups the positions by token on the device (a token index:
 * a stable sort of (token, position)) and adds each token's rows in position
 * order and each position's rows in batch order: deterministic, no
 * floating-point atomics.
 * bt_embedding_bwd builds the index itself in ws (bt_embedding_bwd_ws_bytes
 * bytes, 16-byte aligned, scratch): three launches.
 */
bt_status bt_embedding_fwd(const int32_t* tokens, const float* wte, const float* wpe, float* x0,
                           int B, int T, int C, int Vp, void* stream);
bt_status bt_embedding_bwd(const int32_t* tokens, const float* dx0, float* dwte, float* dwpe,
                           float wpe_beta, void* ws, size_t ws_bytes, int B, int T, int C, int Vp,
                           void* stream);
size_t bt_embedding_bwd_ws_bytes(int B, int T, int C, int Vp);
/*
 * The backward in two halves.  bt_embedding_index builds the token index of
 * tokens [B, T] (one workgroup: a stable radix sort of (token, position) and
 * the run boundaries of the sorted list) into `index`, a caller-owned device
 * buffer of bt_embedding_index_bytes(B, T) bytes, 16-byte aligned.  It only
 * reads the tokens, so it can run on another stream while the forward runs.
 * bt_embedding_bwd_indexed then sums dx0 as bt_embedding_bwd does (two
 * launches; ws holds bt_embedding_bwd_indexed_ws_bytes(B, T, C) bytes of
 * per-piece partial sums).  The index must stay unchanged until the backward
 * has run; it may serve several backward calls on the same tokens.  Results
 * equal bt_embedding_bwd bitwise.
 */
size_t bt_embedding_index_bytes(int B, int T);
bt_status bt_embedding_index(const int32_t* tokens, void* index, size_t index_bytes, int B, int T, int Vp,
                             void* stream);
bt_status bt_embedding_bwd_indexed(const void* index, size_t index_bytes, const float* dx0, float* dwte,
                                   float* dwpe, float wpe_beta, void* ws, size_t ws_bytes, int B, int T,
                                   int C, int Vp, void* stream);
size_t bt_embedding_bwd_indexed_ws_bytes(int B, int T, int C);

/*
 * Column sums ("reduce-sum" kernel of the appendix; bias gradients):
 *   out[n] = beta * out[n] + sum_m X[m, n]      (X [M, N], ldx >= N)
 * Fixed-order two-stage reduction.  ws holds bt_colsum_ws_bytes(M, N) bytes.
 * M >= 0: with no rows, out becomes beta * out (zeros at beta = 0).
 */
bt_status bt_colsum(const float* X, int M, int N, int ldx, float* out, float beta, void* ws,
                    size_t ws_bytes, void* stream);
size_t bt_colsum_ws_bytes(int M, int N);

/* ------------------------------------------------------------------------
 * Composed GPT-2 step.
 *
 * Flat parameter layout (also the layout of grads, m and v), decayed prefix
 * first:  wte [Vp, C], wpe [max_T, C], then for each layer l: Wqkv [C, 3C],
 * Wo [C, C], Wfc [C, 4C], Wfp [4C, C]  (linear weights stored [in, out]);
 * then, not decayed, for each layer: ln1g [C], ln1b [C], bqkv [3C], bo [C],
 * ln2g [C], ln2b [C], bfc [4C], bfp [C]; then lnfg [C], lnfb [C].
 * opt_state is [m | v], 2 * P floats.
 * ------------------------------------------------------------------------ */
typedef struct {
  int V;            /* real vocabulary (loss over columns < V) */
  int Vp;           /* padded rows of wte (multiple of 4) */
  int max_T;        /* rows of wpe */
  int L;            /* layers */
  int H;            /* heads; the head dim C / H a multiple of 4, at most 128 */
  int C;            /* model width, multiple of 4, at most 4096 */
  float ln_eps;     /* LayerNorm epsilon */
  double lr, beta1, beta2, adam_eps, weight_decay;  /* AdamW (host scalars) */
  double grad_clip; /* <= 0: no clipping */
} bt_gpt2_config;

typedef struct bt_gpt2_ctx bt_gpt2_ctx;

size_t bt_gpt2_num_params(const bt_gpt2_config* cfg);
size_t bt_gpt2_num_decay_params(const bt_gpt2_config* cfg);
/* offsets: host array of at least n_tensors+1 entries (call with offsets =
 * NULL to get *n_tensors); entry i is the element offset of tensor i in the
 * flat layout above, the last entry is P. */
bt_status bt_gpt2_param_offsets(const bt_gpt2_config* cfg, size_t* offsets, int* n_tensors);
/* Device workspace for activations and scratch of a step with up to
 * max_B x max_T tokens. */
size_t bt_gpt2_workspace_bytes(const bt_gpt2_config* cfg, int max_B, int max_T);
/* Creates a host-side context bound to the caller's workspace and stream
 * (no HIP call).  At its first step the context creates a second HIP stream
 * (default priority) and two events, released by bt_gpt2_destroy: each
 * micro-step builds the embedding backward's token index on that stream
 * while the forward runs on `stream`, forked after the work already enqueued
 * on `stream` and joined before the embedding backward.  The step counter t
 * starts at 0. */
bt_status bt_gpt2_create(const bt_gpt2_config* cfg, void* workspace, size_t ws_bytes, int max_B,
                         int max_T, void* stream, bt_gpt2_ctx** out);
/* Frees the host-side context only; never touches caller memory. */
void bt_gpt2_destroy(bt_gpt2_ctx* ctx);
/* Current step counter (number of optimizer steps taken). */
int bt_gpt2_step_count(const bt_gpt2_ctx* ctx);
void bt_gpt2_set_step_count(bt_gpt2_ctx* ctx, int t);

/*
 * Forward + backward of one micro-batch (Algorithm "Distributed Data Parallel
 * Training Step", one micro-step).  Gradients are those of
 * loss_scale * sum over the B*T positions of the per-position loss; they
 * overwrite grads (accumulate = 0) or are added to it (accumulate = 1).
 * d_loss (device scalar) receives loss_scale * sum of per-position losses,
 * added to its previous value when accumulate = 1.  For one plain step use
 * loss_scale = 1/(B*T); for k micro-steps 1/(B*T*k).  tokens, targets
 * [B, T]; B <= max_B, T <= max_T of the context and T <= cfg.max_T, B*T a
 * multiple of 4 (else BT_ESHAPE before any launch).
 * loss_rows (optional, device [B*T]) receives the unscaled per-position loss.
 */
bt_status bt_gpt2_fwd_bwd(bt_gpt2_ctx* ctx, const float* params, float* grads,
                          const int32_t* tokens, const int32_t* targets, int B, int T,
                          float loss_scale, int accumulate, float* d_loss, float* loss_rows);
/* Global gradient norm, clip (cfg.grad_clip > 0) and AdamW at step t with
 * learning rate lr.  The norm and clip coefficient stay on the device; when
 * the norm is not finite the AdamW launch writes nothing (read the norm with
 * bt_gpt2_read_scalars to detect it). */
bt_status bt_gpt2_optimizer_step(bt_gpt2_ctx* ctx, float* params, float* grads, float* opt_state,
                                 int t, double lr);
/* Waits for the context's stream, then copies to host out[3] the device
 * scalars [last loss written by bt_gpt2_train_step, gradient norm, clip
 * coefficient (1 without clipping, NaN for a non-finite norm)] of the last
 * step. */
bt_status bt_gpt2_read_scalars(const bt_gpt2_ctx* ctx, float* out);

/*
 * Step profiler (the paper's kernel-level profiler, reduced to what this
 * path needs).  When enabled, every kernel-class call made by
 * bt_gpt2_fwd_bwd and bt_gpt2_optimizer_step is bracketed by two HIP events
 * recorded on the context's stream; elapsed times and the algorithmic work
 * of each call accumulate per class until read.  Event creation happens at
 * enable time (host-side runtime objects; no device memory).
 */
enum {
  BT_PROF_GEMM = 0, BT_PROF_ATTN_FWD, BT_PROF_ATTN_BWD, BT_PROF_LN_FWD, BT_PROF_LN_BWD,
  BT_PROF_XENT, BT_PROF_EMB_FWD, BT_PROF_EMB_BWD, BT_PROF_COLSUM, BT_PROF_GRAD_NORM,
  BT_PROF_ADAMW, BT_PROF_OTHER, BT_PROF_NCLASSES
};
typedef struct {
  long long launches;  /* library calls of this class (one call may launch 2-3 kernels) */
  double ms;           /* summed GPU time between the bracketing events */
  double flops;        /* algorithmic floating-point operations */
  double bytes;        /* algorithmic HBM bytes (each operand read / written once) */
} bt_kernel_stat;
bt_status bt_gpt2_profile_enable(bt_gpt2_ctx* ctx, int enable);
/* Waits for the stream, then copies BT_PROF_NCLASSES entries to host out;
 * reset != 0 clears the totals afterwards. */
bt_status bt_gpt2_profile_read(bt_gpt2_ctx* ctx, bt_kernel_stat* out, int reset);

/*
 * One full training step: forward, backward, clip, AdamW (t = previous
 * count + 1, lr = cfg.lr).  Returns the mean loss over the B*T positions at
 * the pre-update parameters; NaN on error (bt_last_status() and
 * bt_last_error() say why).  A non-finite gradient norm (NaN or Inf in any
 * gradient) returns NaN with BT_ENONFINITE: parameters, moments and the step
 * counter are left unchanged.  Blocks until the step has finished.
 */
float bt_gpt2_train_step(bt_gpt2_ctx* ctx, float* params, float* grads, float* opt_state,
                         const int32_t* tokens, const int32_t* targets, int B, int T);

#ifdef __cplusplus
}
#endif
#endif /* BT_H */
