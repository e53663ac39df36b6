/*
 * estp.h - C ABI of libestp, the MI355X (gfx950) library for the scoring and
 * pooling path of ESTP, Entropy-and-Semantic Token Pooling (arXiv 2608.15592).
 *
 * ESTP predicts an LLM's output length from its prefill: every prompt token
 * gets a next-token entropy H_i (Eq. 2, Section 4.2) and an attention-based
 * semantic importance S_j (Eq. 1, Section 4.1); the two are fused into
 * T_i = lambda1 S_i + lambda2 H_i (Eq. 3), turned into pooling weights by a
 * temperature softmax over the prompt (Eq. 4), and the weighted sum of the
 * hidden states (Eq. 5) feeds a small MLP length head whose K-bin
 * distribution gives the expected length (Eq. 7, Section 4.3).  Predicted
 * lengths order requests shortest-job-first (Section 5.4).
 *
 * Conventions shared by every call
 * --------------------------------
 *  - Every tensor pointer is a DEVICE pointer (memory of the current HIP
 *    device), contiguous, row-major, with the shapes given per call.  The
 *    caller owns all memory; the library never allocates.  Scratch memory
 *    comes from the caller through (workspace, workspace_bytes); the
 *    matching *_workspace_size() call returns the bytes needed for a shape
 *    (0 means none; a NULL workspace is then allowed).  Workspace pointers
 *    must be 256-byte aligned.
 *  - Inputs are read-only.  Outputs are fully overwritten (no pre-zeroing).
 *  - Every call is asynchronous: it validates its arguments on the host,
 *    enqueues its kernels on `stream` (a hipStream_t; NULL = the default
 *    stream) and returns.  Results are visible after the caller synchronises
 *    the stream.  Calls on one stream run in order.
 *  - Argument validation happens before any device work: a failed check
 *    returns an error and enqueues nothing.  Shapes whose kernel grid would
 *    exceed one launch (2^32 - 1 work-items) return ESTP_ERR_UNSUPPORTED.  Device-resident values
 *    (cu_seqlens contents, NaN/Inf in tensors) are not inspected; a prompt of
 *    length 0 or a cu_seqlens array that is not non-decreasing from 0 to
 *    n_tok is invalid input with undefined results.  NaN/Inf propagate.
 *  - Packed variable-length batches: prompt b owns tokens
 *    [cu_seqlens[b], cu_seqlens[b+1]) of every [n_tok, ...] tensor;
 *    cu_seqlens is int32 [B+1] in device memory with cu_seqlens[0] = 0 and
 *    cu_seqlens[B] = n_tok; max_seqlen (host) bounds every prompt length.
 *  - bf16 tensors hold IEEE bfloat16; arithmetic is fp32 throughout.
 *  - The library keeps no global mutable state besides a per-thread error
 *    message (estp_last_error); calls are thread-safe.
 */
#ifndef ESTP_H_
#define ESTP_H_

#include <stddef.h>
#include <stdint.h>

#if defined(__GNUC__) || defined(__clang__)
#define ESTP_API __attribute__((visibility("default")))
#else
#define ESTP_API
#endif

#ifdef __cplusplus
extern "C" {
#endif

typedef enum estp_status {
  ESTP_OK = 0,
  ESTP_ERR_INVALID_ARG = 1, /* null pointer, bad size, bad alignment, bad hyperparameter */
  ESTP_ERR_UNSUPPORTED = 2, /* valid but not implemented (dtype, head_dim) */
  ESTP_ERR_WORKSPACE = 3,   /* workspace smaller than *_workspace_size() */
  ESTP_ERR_HIP = 4          /* a HIP runtime call or kernel launch failed */
} estp_status;

typedef enum estp_dtype { ESTP_BF16 = 0, ESTP_F32 = 1 } estp_dtype;

/* How S and H are scaled before Eq. 3.  NONE is Eq. 3 as printed; ZSCORE
 * replaces S and H by their per-prompt z-scores (population standard
 * deviation, (v - mean) / (std + 1e-6)) so that both terms are commensurate;
 * MINMAX by (v - min) / (max - min + 1e-6) per prompt. */
typedef enum estp_norm { ESTP_NORM_NONE = 0, ESTP_NORM_ZSCORE = 1, ESTP_NORM_MINMAX = 2 } estp_norm;

/* Hidden activation of the length head (the paper names an MLP predictor
 * without fixing its activation). */
typedef enum estp_act { ESTP_ACT_RELU = 0, ESTP_ACT_GELU_TANH = 1 } estp_act;

/* Library version, e.g. 200 for 0.2.0.  The version this header describes is
 * ESTP_VERSION; a library whose estp_version() differs has other signatures.
 * 0.2.0 added the vocab_argmax argument of estp_token_entropy. */
#define ESTP_VERSION 200
ESTP_API int estp_version(void);

/* Static text for a status code. */
ESTP_API const char* estp_status_string(int status);

/* Detail of the last failed call on this thread ("" if none). */
ESTP_API const char* estp_last_error(void);

/* 1 when the debug checks are on in this process, else 0.  They are switched
 * on by ESTP_DEBUG_CHECKS=1 in the environment (read once).  Every call that
 * takes cu_seqlens then copies it back and checks it before any kernel runs
 * (cu_seqlens[0] = 0, cu_seqlens[B] = n_tok, every prompt length in
 * [1, max_seqlen]; ESTP_ERR_INVALID_ARG otherwise), and every call that
 * builds a work list of live blocks or chunks on the device compares it with
 * its definition before the kernels that use it run (ESTP_ERR_HIP on a
 * mismatch).  The checks synchronise the stream: for testing, not for use
 * under graph capture. */
ESTP_API int estp_debug_checks(void);

/* ------------------------------------------------------------------------
 * Token entropy (Eq. 2, Section 4.2).
 *
 *   H[i] = - sum_v P_i(v) ln P_i(v),  P_i = softmax_v(z_i),  z_i = W x_i
 *
 * for every row i of X: the entropy, in nats, of the next-token distribution
 * the LM head assigns from token i's final-layer hidden state.  The logits
 * z_i (n_tok x V) never reach memory: a GEMM streams the vocabulary and
 * keeps a running max / exp-sum / sum(p*z) per row (bf16 inputs: matrix
 * cores with fp32 accumulation; fp32 inputs: fp32 FMAs throughout).
 *
 *   X  [n_tok, d]  hidden states (dtype), 16-byte aligned
 *   W  [V, d]      LM-head weight in nn.Linear layout (dtype), 16-byte aligned
 *   H  [n_tok]     float32 output
 *   vocab_argmax [n_tok]  int32 output, or NULL: the mode of the same
 *                  distribution, argmax_v P_i(v), i.e. the vocabulary index of
 *                  the largest logit z_i[v] as computed here (fp32
 *                  accumulation), the lowest index among equal largest logits.
 *                  Unspecified for rows whose logits are not all finite.
 *                  NULL skips the bookkeeping.
 *   dtype          ESTP_BF16 or ESTP_F32 (X and W alike)
 * Requires n_tok >= 1, V >= 1, d >= 8, d % 8 == 0; for ESTP_BF16 a d that is
 * not a multiple of 32 returns ESTP_ERR_UNSUPPORTED (the matrix-core k steps
 * are 32 deep); 512 d >= 2^32 returns it for either dtype.  The workspace
 * size does not depend on whether vocab_argmax is requested.
 * ------------------------------------------------------------------------ */
ESTP_API size_t estp_token_entropy_workspace_size(int64_t n_tok, int32_t d, int32_t V, int dtype);
ESTP_API int estp_token_entropy(const void* X, const void* W, int64_t n_tok, int32_t d, int32_t V, int dtype,
                       float* H, int32_t* vocab_argmax, void* workspace, size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------------------
 * Token entropy without allocation or workspace.
 *
 * For callers that cannot allocate device memory: code under HIP graph
 * capture, tight serving loops, harnesses that forbid allocation.  The same
 * computation and kernels as estp_token_entropy (same arguments, same
 * results bit for bit), but the per-slice partial states live in a device
 * array owned by the library: ESTP_NOALLOC_SCRATCH_BYTES (32 MiB) on every
 * GPU the library runs on, held until the process ends.  The call allocates
 * nothing; the caller still passes X, W and the outputs.
 *
 *   A shape whose estp_token_entropy_workspace_size() exceeds
 *   ESTP_NOALLOC_SCRATCH_BYTES returns ESTP_ERR_UNSUPPORTED before any device
 *   work (with V >= 4096: n_tok up to 104857 tokens fit).
 *   All calls on one GPU share its array, and it keeps the last call's
 *   contents: calls that can overlap on one GPU (several streams, several
 *   host threads) race and must be serialised by the caller.
 *   ESTP_ERR_HIP if the runtime cannot give the array's address on the
 *   current device.
 * ------------------------------------------------------------------------ */
#define ESTP_NOALLOC_SCRATCH_BYTES (32u << 20)
ESTP_API int estp_token_entropy_noalloc(const void* X, const void* W, int64_t n_tok, int32_t d, int32_t V, int dtype,
                               float* H, int32_t* vocab_argmax, void* stream);

/* ------------------------------------------------------------------------
 * Attention importance (Eq. 1, Section 4.1).
 *
 *   S[j] = sum_l (1/N_b) sum_{i>=j} (1/Hq) sum_h A^{l,h}_{ij}
 *   A^{l,h}_{ij} = exp(scale q^{l,h}_i . k^{l,g(h)}_j) / sum_{j'<=i} exp(scale q^{l,h}_i . k^{l,g(h)}_{j'})
 *
 * for each token j of prompt b (N_b tokens): the mean over the prompt's
 * queries of the causal attention it receives, averaged over the query heads,
 * summed over the L layers given.  The diagonal A_jj is included.  Query head
 * h reads key head g(h) = h / (Hq / Hkv).  The N x N attention never reaches
 * memory: pass 1 records each query row's log-sum-exp, pass 2 re-forms the
 * scores per key block and sums exp(s - lse) over the later queries.  Each
 * prompt's S sums to L.
 *
 *   Q  [L, n_tok, Hq, dh]   post-RoPE queries (dtype), 16-byte aligned
 *   K  [L, n_tok, Hkv, dh]  post-RoPE keys (dtype), 16-byte aligned
 *   cu_seqlens [B+1]        int32, device
 *   scale                   score scale, typically 1/sqrt(dh); finite, > 0
 *   S  [n_tok]              float32 output
 *   dtype                   ESTP_BF16 (matrix-core scores, fp32 accumulation) or
 *                           ESTP_F32 (fp32 FMAs throughout); Q and K alike
 * Requires Hq % Hkv == 0, dh in {32, 64, 128}, 1 <= max_seqlen.
 * ------------------------------------------------------------------------ */
ESTP_API size_t estp_attn_importance_workspace_size(int64_t n_tok, int32_t B, int32_t max_seqlen, int32_t L, int32_t Hq,
                                           int32_t Hkv, int32_t dh, int dtype);
ESTP_API int estp_attn_importance(const void* Q, const void* K, const int32_t* cu_seqlens, int32_t B, int32_t max_seqlen,
                         int64_t n_tok, int32_t L, int32_t Hq, int32_t Hkv, int32_t dh, float scale, int dtype,
                         float* S, void* workspace, size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------------------
 * Attention importance from a prefill's row normalisers (Eq. 1, Section 4.1).
 *
 * The same S as estp_attn_importance, with the first pass replaced by the
 * caller's per-row log partition sums, as a FlashAttention-style prefill
 * already returns them alongside its output:
 *
 *   lse [L, Hq, n_tok]  float32, natural log, device:
 *                       lse[l][h][i] = log sum_{j <= i, same prompt} exp(scale q^{l,h}_i . k^{l,g(h)}_j)
 *
 * Row i of head h is then normalised as exp(scale q.k - lse[l][h][i]); the
 * scores are formed once (the column-sum pass) instead of twice.  Values of
 * lse that are not the exact normalisers give the correspondingly scaled
 * rows (no renormalisation).  Other arguments, layouts and requirements are
 * those of estp_attn_importance; `lse` must be non-null.
 * ------------------------------------------------------------------------ */
ESTP_API size_t estp_attn_importance_from_lse_workspace_size(int64_t n_tok, int32_t B, int32_t max_seqlen, int32_t L,
                                                    int32_t Hq, int32_t Hkv, int32_t dh, int dtype);
ESTP_API int estp_attn_importance_from_lse(const void* Q, const void* K, const float* lse, const int32_t* cu_seqlens,
                                  int32_t B, int32_t max_seqlen, int64_t n_tok, int32_t L, int32_t Hq, int32_t Hkv,
                                  int32_t dh, float scale, int dtype, float* S, void* workspace,
                                  size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------------------
 * Attention importance, variants (Eq. 1, Section 4.1).
 *
 *   S[j] = sum_l w_l (1/N_b) sum_{i in I(j)} (1/Hq) sum_h A^{l,h}_{ij}
 *
 * with I(j) = {i >= j} (the diagonal included, as estp_attn_importance) or,
 * with ESTP_IMPORTANCE_EXCLUDE_SELF in `flags`, I(j) = {i > j}: each token's
 * attention to itself is left out of the column sums (the rows A^{l,h}_{i.}
 * are still the causal softmax over j <= i).  This is the other reading of
 * the paper's note on self-similarity.
 *
 *   lse            NULL: the row log-sum-exps are computed (two passes, as
 *                  estp_attn_importance); else the caller's natural-log
 *                  [L, Hq, n_tok] row normalisers (one pass, as
 *                  estp_attn_importance_from_lse)
 *   layer_weights  host float32 [L], finite, at most 64 layers; NULL = all 1
 *   flags          0 or ESTP_IMPORTANCE_EXCLUDE_SELF
 * Workspace: estp_attn_importance_ex_workspace_size(..., with_lse = lse != NULL).
 * Other arguments and requirements are those of estp_attn_importance.
 * ------------------------------------------------------------------------ */
#define ESTP_IMPORTANCE_EXCLUDE_SELF 1
ESTP_API size_t estp_attn_importance_ex_workspace_size(int64_t n_tok, int32_t B, int32_t max_seqlen, int32_t L, int32_t Hq,
                                              int32_t Hkv, int32_t dh, int dtype, int with_lse);
ESTP_API int estp_attn_importance_ex(const void* Q, const void* K, const float* lse, const int32_t* cu_seqlens, int32_t B,
                            int32_t max_seqlen, int64_t n_tok, int32_t L, int32_t Hq, int32_t Hkv, int32_t dh,
                            float scale, const float* layer_weights, int flags, int dtype, float* S, void* workspace,
                            size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------------------
 * Fusion and pooling (Eq. 3, Eq. 4, Eq. 5, Section 4.2).
 *
 *   T_i = lambda1 S_i + lambda2 H_i              (after `norm`, per prompt)
 *   e_i = exp(T_i / alpha) / sum_{j in prompt} exp(T_j / alpha)
 *   pooled[b] = sum_{i in prompt b} e_i x_i
 *
 *   X  [n_tok, d]    hidden states (dtype), 16-byte aligned
 *   S, H [n_tok]     float32 scores (from the two calls above or any source)
 *   alpha            temperature, finite, > 0
 *   pooled [B, d]    float32 output
 *   e   [n_tok]      float32 output of the weights, or NULL
 *   top [B]          int32 output: global index of each prompt's largest
 *                    weight (lowest index among equal maxima), or NULL
 *   dtype            ESTP_BF16 or ESTP_F32
 * Requires d >= 8, d % 8 == 0.  A prompt longer than 262144 tokens returns
 * ESTP_ERR_UNSUPPORTED.
 * ------------------------------------------------------------------------ */
ESTP_API size_t estp_combine_pool_workspace_size(int64_t n_tok, int32_t B, int32_t max_seqlen, int32_t d, int dtype);
ESTP_API int estp_combine_pool(const void* X, const float* S, const float* H, const int32_t* cu_seqlens, int32_t B,
                      int32_t max_seqlen, int64_t n_tok, int32_t d, float lambda1, float lambda2, float alpha,
                      int norm, int dtype, float* pooled, float* e, int32_t* top, void* workspace,
                      size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------------------
 * Length head (Section 4.3, Eq. 7) and shortest-job-first order (Section 5.4).
 *
 *   a = act(W1 pooled[b] + b1),   o = W2 a + b2
 *   K == 1: yhat[b] = o[0]                               (direct regression)
 *   K  > 1: p = softmax(o), yhat[b] = sum_k p_k centres[k], bin[b] = argmax_k p_k
 *   order: prompt indices sorted by ascending yhat, ties by index
 *
 *   pooled [B, d]       float32
 *   W1 [hidden, d], b1 [hidden] or NULL (zero), W2 [K, hidden], b2 [K] or NULL: float32
 *   centres [K]         float32 bin centres (required when K > 1, ignored when K == 1)
 *   yhat [B]            float32 output
 *   bin  [B]            int32 output or NULL (written only when K > 1)
 *   order [B]           int32 output or NULL
 * Requires B >= 1, d >= 1, hidden >= 1, 1 <= K <= 1024, B <= 65536.
 * ------------------------------------------------------------------------ */
ESTP_API size_t estp_predict_workspace_size(int32_t B, int32_t d, int32_t hidden, int32_t K);
ESTP_API int estp_predict(const float* pooled, int32_t B, int32_t d, const float* W1, const float* b1, int32_t hidden,
                 int act, const float* W2, const float* b2, int32_t K, const float* centres, float* yhat,
                 int32_t* bin, int32_t* order, void* workspace, size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------------------
 * One training step of the K-bin length head (Eq. 6, Eq. 7, Eq. 8,
 * Section 4.3; AdamW, Section 5.1).
 *
 *   z = W1 h + b1, a = act(z), o = W2 a + b2, p-hat = softmax(o),
 *   y-hat = sum_k p-hat_k c_k                                       (Eq. 7)
 *   i = bin of the true length y: [edges[i], edges[i+1]); below edges[0] -> 0,
 *       at or above edges[K] -> K-1
 *   p_j = exp(-|j - i|) / sum_k exp(-|k - i|)                        (Eq. 6)
 *   loss = lambda3 * mean_b CE(p, p-hat) + (1 - lambda3) * mean_b (y - y-hat)^2   (Eq. 8)
 *
 * then the gradient of the loss at the current parameters and one AdamW
 * update of every parameter (PyTorch's form: decoupled decay
 * theta *= 1 - lr*weight_decay, moments m, v, bias corrections 1 - beta^step).
 *
 *   pooled [B, d]   float32 features (the pooled vectors), 16-byte aligned
 *   y [B]           float32 true lengths
 *   edges [K+1]     float32 ascending bin edges;  centres [K] float32 bin centres
 *   theta           float32 parameters, updated in place, flat layout
 *                   [W1 (hidden x d) | b1 (hidden) | W2 (K x hidden) | b2 (K)];
 *                   pointers into it serve estp_predict directly
 *   m, v            float32 AdamW moments, same layout, updated in place
 *                   (zero before step 1)
 *   step            1-based step count (bias corrections)
 *   loss            float32 device scalar: the batch loss before the update, or NULL
 * Requires 2 <= K <= 1024, d % 4 == 0, lambda3 in [0, 1], betas in [0, 1),
 * eps > 0; theta, m, v 16-byte aligned.  Batch sums run in a fixed order.
 * ------------------------------------------------------------------------ */
ESTP_API size_t estp_head_train_step_workspace_size(int32_t B, int32_t d, int32_t hidden, int32_t K);
ESTP_API int estp_head_train_step(const float* pooled, const float* y, int32_t B, int32_t d, int32_t hidden, int32_t K,
                         int act, const float* edges, const float* centres, float* theta, float* m, float* v,
                         int32_t step, float lambda3, float lr, float beta1, float beta2, float eps,
                         float weight_decay, float* loss, void* workspace, size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------------------
 * Analyses on the path's outputs.
 *
 * estp_misalignment: the entropy / semantics split behind Fig. 1b
 * (Section 1).  Within each prompt (N tokens) the tokens are ranked by H and
 * by S (ascending; equal values by token index) and split into the lowest
 * floor(frac_low N) and the highest floor(frac_high N) (Fig. 1b compares
 * the top and bottom 40%: frac_low = frac_high = 0.4).
 *   H, S [n_tok]    float32, device;  cu_seqlens [B+1] int32, device
 *   counts [B, 4]   int32 output: #high-H, #high-H that are low-S,
 *                   #low-H, #low-H that are high-S
 * The two misalignment ratios are counts[.,1] / counts[.,0] and
 * counts[.,3] / counts[.,2].  Exact integer counts.
 *
 * estp_sjf_padding: static batches of `batch` requests taken in `order`
 * (e.g. the shortest-job-first order from estp_predict, Section 5.4; NULL =
 * as given); each batch runs for its longest true length, back to back.
 *   lengths [B]     int32 true output lengths, device
 *   order [B]       int32 permutation of 0..B-1, device, or NULL
 *   out [3]         int64 output, device: padded tokens
 *                   sum_batches (size * max - sum), useful tokens sum y,
 *                   sum over requests of start(batch) + y_i
 * Padding ratio = out[0] / out[1]; mean completion time = out[2] / B.
 * ------------------------------------------------------------------------ */
ESTP_API int estp_misalignment(const float* H, const float* S, const int32_t* cu_seqlens, int32_t B, float frac_low,
                      float frac_high, int32_t* counts, void* stream);
ESTP_API int estp_sjf_padding(const int32_t* lengths, const int32_t* order, int32_t B, int32_t batch, int64_t* out,
                     void* stream);

#ifdef __cplusplus
}
#endif

#endif /* ESTP_H_ */
