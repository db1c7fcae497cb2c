/*
 * libbpt — one Blockwise Parallel Transformer layer on AMD Instinct MI355X (gfx950).
 *
 * The layer is a pre-LayerNorm GPT block (the paper builds on the GPT
 * architecture; Section 4, "Model Configuration"):
 *
 *     U  = LN1(X);   Q = U Wq,  K = U Wk,  V = U Wv         (Algorithm 1, "project")
 *     O  = softmax(Q_h K_h^T / sqrt(dh) + mask) V_h, per head (eq. 1), computed
 *          blockwise with running max / sum rescaling (Section 3, eq. 3)
 *     Hd = X + O Wo
 *     Y  = Hd + act(LN2(Hd) W1 + b1) W2 + b2                  (eq. 2; act = GELU or ReLU)
 *
 * and, per Algorithm 1, the FFN and both residuals are applied to each group of
 * query blocks right after that group's attention, before the next group
 * starts, so that no S x S score matrix and no S x F FFN intermediate is ever
 * stored. The backward recomputes attention probabilities blockwise from the
 * saved log-sum-exp and the FFN intermediate per query-block group.
 *
 * Conventions (all entry points):
 *  - Every pointer argument of a compute call is a DEVICE pointer on the
 *    current HIP device, owned by the caller. The library never allocates or
 *    frees device memory; all scratch comes from the caller's workspace.
 *  - Matrices are row-major; y = x @ W with W[D_in, D_out]. Head h owns
 *    columns [h*dh, (h+1)*dh) of Wq, Wk, Wv and rows [h*dh, (h+1)*dh) of Wo.
 *  - X, dY, Wq..W2 and the saved activations are in cfg->dtype; Y and dX in
 *    cfg->out_dtype. LayerNorm gains/shifts and FFN biases are always fp32
 *    vectors and may be NULL (gain 1, shift 0, no bias). Weight gradients are
 *    fp32 and OVERWRITTEN; a NULL gradient pointer skips that output.
 *  - Every pointer must be 16-byte aligned. Y must not alias X; dX must not
 *    alias dY or X; outputs must not overlap inputs, saved or workspace.
 *  - Calls are asynchronous on `stream` (a hipStream_t; NULL = the default
 *    stream) and never synchronise. Arguments are validated before anything
 *    is launched, so on any error status nothing has been written. Faults
 *    inside kernels surface at the caller's next synchronisation.
 *  - Supported: dh = D/H in {64, 128}; D and F multiples of 64; B, S >= 1;
 *    1 <= Bq, Bkv <= S. Other shapes return BPT_ERR_UNSUPPORTED.
 *  - bpt_last_error() returns a thread-local message for the last failure.
 */
#ifndef LIBBPT_H
#define LIBBPT_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  BPT_OK = 0,
  BPT_ERR_INVALID_ARG = 1,  /* NULL pointer, non-positive size, D % H != 0, Bq > S ... */
  BPT_ERR_UNSUPPORTED = 2,  /* valid but not implemented (dh, D % 64, dtype)          */
  BPT_ERR_WORKSPACE = 3,    /* workspace smaller than bpt_workspace_bytes()            */
  BPT_ERR_HIP = 4           /* a kernel launch was rejected by the HIP runtime         */
} bpt_status;

typedef enum { BPT_F32 = 0, BPT_BF16 = 1 } bpt_dtype;

typedef struct {
  int64_t B, S, D, H, F;   /* batch, sequence length, model width, heads, FFN width        */
  int64_t Bq, Bkv;         /* query / key-value block LENGTHS in tokens (Section 3's      */
                           /* problem statement, Algorithm 1). Need not divide S. Bq is   */
                           /* the unit of FFN fusion (see group_blocks). Bkv is validated */
                           /* but does not change the GPU path: its kernels step through  */
                           /* keys in tiles of 64, their LDS / matrix-core tile, whatever */
                           /* Bkv is (bpt_describe reports the tiles). The method is      */
                           /* exact, so results depend on Bq and the tiles only through   */
                           /* rounding.                                                     */
  int32_t causal;          /* 1: query q sees key k iff k <= q, within one sequence        */
  int32_t dtype;           /* bpt_dtype of X, dY, weights and saved activations             */
  int32_t out_dtype;       /* bpt_dtype of Y and dX                                         */
  int32_t group_blocks;    /* query blocks per FFN group: at most group_blocks * Bq rows of */
                           /* the [., F] intermediate are live at once (a run of one         */
                           /* sequence, or several whole sequences when two or more fit);    */
                           /* 0 = automatic: max(16384, 2^27 / F) rows rounded up to whole  */
                           /* query blocks (a narrow FFN gets taller groups, its            */
                           /* intermediate staying at 2^27 elements)                        */
  float ln_eps;            /* LayerNorm epsilon (biased variance), e.g. 1e-5                */
  int32_t activation;      /* bpt_activation of the FFN                                     */
  float dropout;           /* rate p in [0, 1) of dropout on the two residual branches:     */
                           /* h = X + drop(O Wo), Y = h + drop(FFN(LN2 h)); 0 = none        */
  uint64_t dropout_seed;   /* key of the dropout masks: element (t, n) of branch k (0: O Wo,*/
                           /* 1: FFN) uses word n%4 of Philox4x32-10 at counter             */
                           /* (n/4, t, k, 0), t = b*S + s, key (seed low, seed high 32 bits);*/
                           /* kept iff the word >= floor(p 2^32), kept values scaled by     */
                           /* 1/(1 - p). Pass the same seed to bpt_layer_bwd.               */
} bpt_config;

/* FFN activation: the exact-erf GELU of GPT models (default) or eq. (2)'s ReLU,
 * max(0, z), whose derivative is taken as 0 at z = 0. */
typedef enum { BPT_GELU = 0, BPT_RELU = 1 } bpt_activation;

typedef struct {           /* device pointers; see the conventions above                    */
  const float *ln1_g, *ln1_b;              /* [D] fp32 or NULL                               */
  const void *Wq, *Wk, *Wv, *Wo;           /* [D, D] in cfg->dtype                           */
  const float *ln2_g, *ln2_b;              /* [D] fp32 or NULL                               */
  const void *W1;                          /* [D, F] in cfg->dtype                           */
  const float *b1;                         /* [F] fp32 or NULL                               */
  const void *W2;                          /* [F, D] in cfg->dtype                           */
  const float *b2;                         /* [D] fp32 or NULL                               */
} bpt_params;

typedef struct {           /* fp32 device pointers, overwritten; NULL = not wanted          */
  float *dln1_g, *dln1_b, *dWq, *dWk, *dWv, *dWo, *dln2_g, *dln2_b, *dW1, *db1, *dW2, *db2;
} bpt_grads;

/* Byte offsets of the tensors the forward saves for the backward, inside the
 * caller's `saved` buffer. E = element size of cfg->dtype; T = B*S tokens;
 * Sp = S rounded up to a multiple of 64.
 *   qkv  [T, 3D] E   Q in columns [0, D) (dtype BF16: multiplied by log2(e)/sqrt(D/H),
 *                    the base-2 score scale; F32: unscaled), K in [D, 2D), V in [2D, 3D)
 *   o    [T, D] E    attention output (heads concatenated), before Wo
 *   lse  [B, H, Sp] fp32  natural-log log-sum-exp of each query row's scores
 *   h    [T, D] fp32 residual stream after attention, X + O Wo
 *   mu1, rstd1, mu2, rstd2 [T] fp32  LayerNorm statistics                               */
typedef struct {
  size_t qkv, o, lse, h, mu1, rstd1, mu2, rstd2, total;
} bpt_saved_layout;

/* Host-only checks of a configuration; never touches a GPU. */
bpt_status bpt_validate(const bpt_config* cfg);

/* Rows of the [., F] FFN intermediate that are live at once: group_blocks * Bq clipped to
 * S, or, when that holds two or more whole sequences, the most whole sequences it holds
 * (at most B) times S. Returns -1 for an invalid configuration. Host-only. */
int64_t bpt_group_rows(const bpt_config* cfg);

/* Size of the `saved` buffer and the offsets inside it. Section 3.1's memory analysis
 * counts what a blockwise layer keeps for its backward: activations linear in the
 * sequence length, no S x S attention matrix and no S x F FFN intermediate. Here that
 * is O(B*S*D) (layout below). Returns 0 / a non-OK status for an invalid
 * configuration. Host-only. */
size_t bpt_saved_bytes(const bpt_config* cfg);
bpt_status bpt_saved_layout_of(const bpt_config* cfg, bpt_saved_layout* out);

/* Workspace needed by bpt_layer_fwd (backward = 0) or bpt_layer_bwd (backward = 1):
 * O(D^2 + D*F + B*S*D + group_rows*F). Section 3.1 bounds the live FFN intermediate of a
 * blockwise layer by one query block's [Bq, F]; here it is one group's [group_rows, F],
 * independent of S. Returns 0 for an invalid configuration. Host-only. */
size_t bpt_workspace_bytes(const bpt_config* cfg, int backward);

/* Forward of one layer (Algorithm 1). X, Y: [B, S, D]. `saved` (bpt_saved_bytes
 * bytes) receives the activations the backward needs. Y must not alias X. */
bpt_status bpt_layer_fwd(const bpt_config* cfg, const void* X, const bpt_params* params, void* Y,
                         void* saved, void* workspace, size_t workspace_bytes, void* stream);

/* bpt_layer_fwd for callers that cannot allocate device memory: code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc. It takes no workspace:
 * its kernels use the library's own static device array of BPT_NOALLOC_SCRATCH_BYTES
 * (64 MiB), one per GPU that runs it, held until the process ends. The caller still passes
 * X, Y and `saved` (bpt_saved_bytes bytes), as for bpt_layer_fwd, with which the results
 * are identical. A configuration whose bpt_workspace_bytes(cfg, 0) exceeds the array
 * returns BPT_ERR_WORKSPACE before anything is launched. Allocates nothing (no hipMalloc
 * or hipFree; its launches bypass the launch profiler). Every call on one GPU shares that
 * GPU's array: calls that overlap on one GPU (several streams or threads) race. */
#define BPT_NOALLOC_SCRATCH_BYTES ((size_t)64 << 20)
bpt_status bpt_layer_fwd_noalloc(const bpt_config* cfg, const void* X, const bpt_params* params, void* Y,
                                 void* saved, void* stream);

/* Backward of one layer given the forward's `saved` buffer and the upstream
 * gradient dY [B, S, D]. Writes dX [B, S, D] (out_dtype) and every non-NULL
 * gradient in `grads`. As in Section 3 (the checkpointed attention scan and the
 * rematerialised FFN of Fig. 3), nothing of size S x S or S x F was saved: attention
 * probabilities are rebuilt blockwise from the saved log-sum-exp, and the FFN
 * intermediate is recomputed per query-block group. Same conventions as the forward;
 * the workspace must be bpt_workspace_bytes(cfg, 1) bytes. */
bpt_status bpt_layer_bwd(const bpt_config* cfg, const void* X, const bpt_params* params,
                         const void* saved, const void* dY, void* dX, const bpt_grads* grads,
                         void* workspace, size_t workspace_bytes, void* stream);

/* Where bpt_layer_bwd leaves the gradients of the attention inputs inside its workspace,
 * for tests and tooling (the attention backward of Section 3 rebuilds the probabilities
 * blockwise and produces them on the way to dU and the projection weight gradients).
 * After the call has completed, the workspace bytes from *offset hold dQ, dK, dV
 * feature-major as one [3D, B*Sp] matrix in cfg->dtype, Sp = S rounded up to 64:
 * element (b, s, n) of dQ at row n, column b*Sp + s; dK in rows [D, 2D), dV in rows
 * [2D, 3D); columns b*Sp + s with s >= S hold zeros. dQ, dK, dV are the gradients of the
 * unscaled Q = U Wq, K, V (the base-2 scale of the stored query is undone). Host-only. */
bpt_status bpt_bwd_qkv_grad_offset(const bpt_config* cfg, size_t* offset);

const char* bpt_status_string(int status);
const char* bpt_last_error(void);

/* Human-readable description of the kernel tiling used for a configuration
 * (internal MFMA / LDS tiles, FFN group rows). Host-only. Returns bytes written. */
size_t bpt_describe(const bpt_config* cfg, char* buf, size_t buf_bytes);

/* Launch timing for tooling (benchmarks, roofline reports). bpt_profile_enable(1)
 * clears the record and brackets every later launch of bpt_layer_fwd / bpt_layer_bwd
 * with two HIP events on the launch stream, tagged with the call site's name and
 * its algorithmic flops and HBM bytes; bpt_profile_enable(0) stops recording.
 * After the caller has synchronised those streams, bpt_profile_report writes a
 * JSON object {name: {count, ms, flops, bytes}} into buf (NUL-terminated,
 * truncated to buf_bytes) and returns its full length. Process-wide; not meant to
 * be toggled while another thread is launching. */
bpt_status bpt_profile_enable(int on);
size_t bpt_profile_report(char* buf, size_t buf_bytes);

/* ---------------------------------------------------------------------------
 * Cross-entropy of a language-model head, blockwise over tokens. Section 3 of the
 * paper remarks that the blockwise scheme applies to the final cross-entropy loss
 * as well: here the [T, V] logits never exist at once, only those of block_rows
 * tokens, in the workspace.
 *
 *     logits = h W        h [T, D] and W [D, ldw] in cfg->dtype (row-major, y = x @ W);
 *                         the first V columns of W are the vocabulary
 *     lse_t  = log sum_{v < V} exp(logits[t, v])
 *     loss   = (1/T) sum_t (lse_t - logits[t, y_t])
 *
 * The backward recomputes each block's logits and forms G = (dloss / T)
 * (softmax - onehot(y)) in cfg->dtype (bf16: rounded to nearest even, like every
 * other matrix-multiply operand), then dh = G W^T and dW = h^T G with fp32
 * accumulation. Same conventions as the layer calls (device pointers owned by the
 * caller, 16-byte alignment, asynchronous on `stream`, validation before launch).
 */
typedef struct {
  int64_t T, D, V;       /* tokens, hidden width, vocabulary size                          */
  int64_t ldw;           /* columns of W as stored: >= V and a multiple of 64. Columns       */
                         /* V..ldw-1 are not logits, but must hold finite values (the        */
                         /* backward multiplies them by zero)                                */
  int64_t block_rows;    /* tokens whose logits are live at once; 0 = automatic (8192)       */
  int32_t dtype;         /* bpt_dtype of h, W and dh                                          */
  int32_t reserved;      /* must be 0                                                         */
} bpt_xent_config;

/* Host-only checks; D and ldw must be multiples of 64 (else BPT_ERR_UNSUPPORTED). */
bpt_status bpt_xent_validate(const bpt_xent_config* cfg);

/* Workspace of bpt_xent_fwd (backward = 0): block_rows * ldw fp32 logits + T floats;
 * of bpt_xent_bwd (backward = 1): ldw * block_rows (rounded up to 64) elements of
 * cfg->dtype (one block's logit gradient, vocabulary-major). Returns 0 for an invalid
 * configuration. Host-only. */
size_t bpt_xent_workspace_bytes(const bpt_xent_config* cfg, int backward);

/* Forward. targets: [T] int32 class indices; a target outside [0, V) makes that
 * token's loss, and so *loss, NaN. Writes loss (one float) and lse [T] (fp32, the
 * natural-log log-sum-exp of each token's logits, which the backward takes). */
bpt_status bpt_xent_fwd(const bpt_xent_config* cfg, const void* h, const void* W, const int32_t* targets,
                        float* loss, float* lse, void* workspace, size_t workspace_bytes, void* stream);

/* Backward for an upstream gradient dloss of the loss (host scalar). Writes dh [T, D]
 * in cfg->dtype and, unless dW is NULL, dW [D, ldw] fp32 (columns from V on get 0).
 * Both are OVERWRITTEN. A target outside [0, V) contributes no one-hot term. */
bpt_status bpt_xent_bwd(const bpt_xent_config* cfg, const void* h, const void* W, const int32_t* targets,
                        const float* lse, float dloss, void* dh, float* dW, void* workspace,
                        size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------------ GPT training step
 * Section 5 trains decoder-only GPT models (Table 1 shapes) made of the layer
 * above. The entry points below are the rest of such a model's training step:
 * the token and position embedding in front of the first layer, the final
 * LayerNorm before the LM head (bpt_xent_*), and the AdamW update (Adam with
 * decoupled weight decay; Section 5 trains with weight decay 0.1). Same
 * conventions as above: device pointers, 16-byte aligned, asynchronous on
 * `stream`, validated before any launch. */

typedef struct {
  int64_t B, S;          /* batch and sequence length: tokens [B, S], row t = b*S + s       */
  int64_t D;             /* width, a multiple of 8                                           */
  int64_t V;             /* vocabulary (rows of Wte)                                         */
  int32_t dtype;         /* bpt_dtype of Wte, Wpe and X                                      */
  int32_t grad_dtype;    /* bpt_dtype of the dX that bpt_embed_bwd reads                     */
} bpt_embed_config;

/* X[t] = Wte[tokens[t]] + Wpe[t mod S]. tokens: [B*S] int32; Wte [V, D]; Wpe [S, D]
 * or NULL (no position table); X [B*S, D]. A token outside [0, V) gives a NaN row. */
bpt_status bpt_embed_fwd(const bpt_embed_config* cfg, const int32_t* tokens, const void* Wte,
                         const void* Wpe, void* X, void* stream);

/* Gradients of the embedding for an upstream dX [B*S, D] (cfg->grad_dtype):
 * dWte [V, D] fp32 = per vocabulary row, the sum of dX over the tokens equal to it
 * (a token outside [0, V) adds nothing); dWpe [S, D] fp32 = sum over the batch.
 * Both are OVERWRITTEN; NULL skips. dWte's rows are summed with floating-point
 * atomics, so the order of the additions into a repeated token's row, and with it
 * the last bits of that row, may differ between runs. */
bpt_status bpt_embed_bwd(const bpt_embed_config* cfg, const int32_t* tokens, const void* dX, float* dWte,
                         float* dWpe, void* stream);

typedef struct {
  int64_t rows, D;       /* rows of width D, D a multiple of 4                              */
  float eps;             /* added to the biased variance                                    */
  int32_t in_dtype;      /* bpt_dtype of X and dX                                           */
  int32_t out_dtype;     /* bpt_dtype of Y and dY                                           */
  int32_t reserved;      /* 0                                                               */
} bpt_ln_config;

/* Workspace of bpt_ln_bwd in bytes (the column-sum partials of dg, db and, for a
 * bf16 dY, an fp32 copy of it). 0 for an invalid configuration. Host-only. */
size_t bpt_ln_workspace_bytes(const bpt_ln_config* cfg);

/* LayerNorm per row: Y = g (X - mean) rstd + b, rstd = 1/sqrt(var + eps), var the
 * biased variance; the same LayerNorm as the layer's LN1/LN2. g, b: fp32 [D] or
 * NULL (1, 0). mean, rstd: fp32 [rows], written for bpt_ln_bwd. */
bpt_status bpt_ln_fwd(const bpt_ln_config* cfg, const void* X, const float* g, const float* b, void* Y,
                      float* mean, float* rstd, void* stream);

/* Backward of bpt_ln_fwd: dX [rows, D] (in_dtype) from dY (out_dtype), X and the
 * saved mean/rstd; dg = sum_rows dY * xhat, db = sum_rows dY (fp32 [D], OVERWRITTEN;
 * both NULL skips them, exactly one NULL is an error). */
bpt_status bpt_ln_bwd(const bpt_ln_config* cfg, const void* X, const float* g, const float* mean,
                      const float* rstd, const void* dY, void* dX, float* dg, float* db, void* workspace,
                      size_t workspace_bytes, void* stream);

typedef struct {
  float lr, beta1, beta2, eps, weight_decay;
  int32_t lowp_dtype;    /* bpt_dtype of the rounded copy p_lowp                             */
  int64_t step;          /* 1-based step count, for the bias corrections                    */
} bpt_adamw_config;

/* One AdamW step on n fp32 elements, in place:
 *   m = beta1 m + (1 - beta1) g,   v = beta2 v + (1 - beta2) g^2,
 *   p = p - lr wd p - lr (m / (1 - beta1^step)) / (sqrt(v / (1 - beta2^step)) + eps)
 * and, unless p_lowp is NULL, p_lowp = p rounded to lowp_dtype (the copy the
 * layer's kernels read). */
bpt_status bpt_adamw_step(const bpt_adamw_config* cfg, int64_t n, float* p, const float* g, float* m, float* v,
                          void* p_lowp, void* stream);

#ifdef __cplusplus
}
#endif
#endif /* LIBBPT_H */
