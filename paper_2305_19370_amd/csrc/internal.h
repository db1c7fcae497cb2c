// Host-side launchers shared between libbpt's translation units (not part of the C ABI).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace bpt {

// F16 is used for one tensor only: GELU'(z) saved by the FFN recompute of the bf16 path.
enum Dt { F32 = 0, BF16 = 1, F16 = 2 };

// ---------------------------------------------------------------- GEMM
// C[M, N] = A[M, K] * B[N, K]^T ("NT": both operands K-contiguous), fp32 accumulation,
// optional batch (grid z) with element strides, followed by a fused epilogue.
enum Epi {
  EPI_STORE = 0,   // C = acc            (fp32 C may accumulate: C += acc)
  EPI_RESID = 1,   // C = acc + R[m, n] (+ bias[n])
  EPI_GELU = 2,    // z = acc (+ bias[n] or bias[m]); C = GELU(z); C2 = GELU'(z) if C2
  EPI_MUL = 3,     // C = acc * R[m, n]  (R fp32 or fp16)
  EPI_XENT = 4,    // cross-entropy gradient of logits acc: for n < nvalid
                   // C = alpha (exp(acc - rowv[m]) - [n == tgt[m]]), rowv the row's
                   // log-sum-exp; C = 0 for nvalid <= n
  EPI_RELU = 5,    // as EPI_GELU with max(0, z) and its derivative (0 at z = 0)
  EPI_XENT_T = 6,  // EPI_XENT on the transposed logits (rows m = vocabulary, columns n =
                   // tokens): for m < nvalid C = alpha (exp(acc - rowv[n]) - [m == tgt[n]]),
                   // C = 0 for nvalid <= m
};

struct GemmArgs {
  const void* A = nullptr;
  const void* B = nullptr;
  void* C = nullptr;
  const void* R = nullptr;     // residual (EPI_RESID) or multiplier (EPI_MUL)
  const float* bias = nullptr;
  void* C2 = nullptr;          // second output of EPI_GELU / EPI_RELU, element type c2t (F32 or F16)
  Dt c2t = F32;
  int64_t M = 0, N = 0, K = 0;
  int64_t Nstore = 0;          // columns [N, Nstore) of C (and C2) are written with 0
  int64_t lda = 0, ldb = 0, ldc = 0, ldr = 0, ldc2 = 0;
  int64_t sA = 0, sB = 0, sC = 0, sR = 0, sC2 = 0;   // batch strides in elements
  int batch = 1;
  int accumulate = 0;          // fp32 C only: C += acc
  float alpha = 1.0f;          // EPI_STORE: acc is multiplied by alpha before it is stored;
                               // EPI_XENT: the gradient's scale
  const float* rowv = nullptr; // EPI_XENT: per-row log-sum-exp (natural log), [M]; EPI_XENT_T: per column, [N]
  const int32_t* tgt = nullptr;// EPI_XENT: per-row target column, [M]; EPI_XENT_T: per-column target row, [N]
  int64_t nvalid = 0;          // EPI_XENT: columns from nvalid on are not logits; EPI_XENT_T: rows
  int bias_on_m = 0;           // EPI_GELU / EPI_RELU: bias indexed by row instead of column
  // Transposed operands (trans_b with any epilogue, trans_a with EPI_STORE, EPI_GELU, EPI_RELU or
  // EPI_XENT_T, both with EPI_STORE): trans_a means A is stored K-major, element
  // (m, k) at A[k * lda + m]; likewise trans_b for B (element (n, k) at B[k * ldb + n]).
  // For such an operand, x_rows is the number of k rows that may be read (rows from
  // x_rows up to K are not read, and the other operand must be zero at those k), and
  // x_cols the number of columns that may be read from the pointer (>= M or N; a
  // multiple of 8). 0 means K and M (or N).
  int trans_a = 0, trans_b = 0;
  int64_t a_rows = 0, b_rows = 0, a_cols = 0, b_cols = 0;
};

// ab: element type of A and B. ct: type of C; rt: type of R.
hipError_t gemm(Dt ab, Epi epi, Dt ct, Dt rt, const GemmArgs& a, hipStream_t s);

// ---------------------------------------------------------------- attention
// The bf16 kernels take Q multiplied by log2(e)/sqrt(dh), so that Q K^T are the scores in
// base-2 units (exp2 of them is the unnormalised probability); the fp32 kernels take Q
// as the projection produced it.
struct AttnArgs {
  // token-major tensors: token (b, s) is row b*S + s
  const void* q = nullptr;  int64_t ld_q = 0;    // pointer already at head 0's first column
  const void* k = nullptr;  int64_t ld_k = 0;
  const void* v = nullptr;  int64_t ld_v = 0;
  const void* dout = nullptr; int64_t ld_do = 0;
  void* o = nullptr;        int64_t ld_o = 0;
  // feature-major outputs: element (b, s, f) at row f, column b*Sp + s
  void* dqt = nullptr; void* dkt = nullptr; void* dvt = nullptr; int64_t ld_dt = 0;
  float* lse = nullptr;        // [B, H, Sp] natural log
  const float* ndelta = nullptr;// [B, H, Sp] -Delta, Delta = rowsum(dO * O)
  const float* nlse2 = nullptr;// [B, H, Sp] minus the log-sum-exp in base 2 (bf16 backward)
  int64_t S = 0, Sp = 0;
  int B = 0, H = 0, dh = 0;
  int causal = 0;
  int64_t q_begin = 0, q_end = 0;  // forward: query rows [q_begin, q_end) of batch b_begin
  int b_begin = 0, nb = 0;
};

hipError_t attn_fwd(Dt dt, const AttnArgs& a, hipStream_t s);
// backward: dK and dV (key-outer kernel), dQ (query-outer kernel)
hipError_t attn_bwd_dkdv(Dt dt, const AttnArgs& a, hipStream_t s);
hipError_t attn_bwd_dq(Dt dt, const AttnArgs& a, hipStream_t s);

// ---------------------------------------------------------------- row-wise / layout kernels
// LayerNorm over D per row. x: [rows, D] (ti); out [rows, D] (to).
// mode 0: compute and write mu/rstd; mode 1: use the given mu/rstd.
hipError_t layer_norm(Dt ti, Dt to, const void* x, int64_t ldx, const float* g, const float* b,
                      void* out, int64_t ldo, float* mu, float* rstd, int64_t rows, int64_t D,
                      float eps, int use_stats, hipStream_t s);

// out = resid + LN^T(dout), per row (resid may be null: 0); out2 (optional, type t2) gets
// the same values.
hipError_t layer_norm_bwd(Dt ti, const void* x, const float* mu, const float* rstd, const float* g,
                          const float* dout, Dt tr, const void* resid, Dt to, void* out,
                          Dt t2, void* out2, int64_t rows, int64_t D, hipStream_t s);

// dgamma[d] = sum_r dout[r,d] * xhat[r,d]; dbeta[d] = sum_r dout[r,d] (overwrite).
// `partial` is workspace of layer_norm_param_grad_ws(D) floats.
size_t layer_norm_param_grad_ws(int64_t D);
hipError_t layer_norm_param_grad(Dt ti, const void* x, const float* mu, const float* rstd,
                                 const float* dout, float* dgamma, float* dbeta, float* partial,
                                 int64_t rows, int64_t D, hipStream_t s);

// out[c, r] = in[r, c] for r < rows, 0 for rows <= r < rows_store; batched over z.
hipError_t transpose(Dt t, const void* in, int64_t ld_in, int64_t s_in, void* out, int64_t ld_out,
                     int64_t s_out, int64_t rows, int64_t cols, int64_t rows_store, int batch,
                     hipStream_t s);

// out[r, c] = in[r, c]
hipError_t copy2d(Dt t, const void* in, int64_t ld_in, void* out, int64_t ld_out, int64_t rows,
                  int64_t cols, hipStream_t s);

// out[c] (+)= sum_r in[r, c]  (in: [rows, cols] of type t)
hipError_t col_sum(Dt t, const void* in, int64_t ld, int64_t rows, int64_t cols, float* out,
                   int accumulate, float* partial, hipStream_t s);
// out[r] (+)= sum_c in[r, c]
hipError_t row_sum(Dt t, const void* in, int64_t ld, int64_t rows, int64_t cols, float* out,
                   int accumulate, hipStream_t s);

// ndelta[b, h, s] = -sum_d dO[b*S+s, h*dh+d] * O[b*S+s, h*dh+d]; nlse2 = -lse * log2(e);
// both are 0 for the padding positions s >= S
hipError_t attn_delta(Dt t, const void* dout, const void* o, int64_t ld, const float* lse, float* ndelta,
                      float* nlse2, int B, int64_t S, int64_t Sp, int H, int dh, hipStream_t s);

// ---------------------------------------------------------------- cross-entropy of an LM head
// Per row t of a block of fp32 logits z [rows, ld]: lse[t] over the first V columns and
// the token loss lse[t] - z[t, tgt[t]] (NaN for a target outside [0, V)).
hipError_t xent_rows(const float* z, int64_t ld, int64_t rows, int64_t V, const int32_t* tgt, float* lse,
                     float* tok, hipStream_t s);
// out[0] = mean of x[0..n), summed in a fixed order
hipError_t mean_of(const float* x, int64_t n, float* out, hipStream_t s);
// ---------------------------------------------------------------- GPT step pieces
// X[t] = Wte[tok[t]] + Wpe[t mod S] (Wpe may be null); NaN row for tok outside [0, V). D % 8 == 0.
hipError_t embed_fwd(Dt t, const int32_t* tok, const void* Wte, const void* Wpe, void* X, int64_t rows,
                     int64_t S, int64_t D, int64_t V, hipStream_t s);
// dWte = 0, then dWte[tok[t]] += dX[t] (fp32 atomics)
hipError_t embed_dwte(Dt t, const int32_t* tok, const void* dX, float* dWte, int64_t rows, int64_t D, int64_t V,
                      hipStream_t s);
// dWpe[s] = sum_b dX[b S + s] (overwrite)
hipError_t embed_dwpe(Dt t, const void* dX, float* dWpe, int64_t B, int64_t S, int64_t D, hipStream_t s);
// out[i] = in[i] (bf16 -> fp32), n % 8 == 0
hipError_t bf16_to_f32(const void* in, float* out, int64_t n, hipStream_t s);
// one AdamW step over n fp32 elements; pl (type tl) gets the updated p when not null
hipError_t adamw(Dt tl, float* p, const float* g, float* m, float* v, void* pl, int64_t n, float lr, float b1,
                 float b2, float eps, float wd, float c1, float c2, hipStream_t s);

// out[i] (+)= sum over z < nz of part[z n + i], added in slice order (n % 4 == 0)
hipError_t sum_slices(const float* part, int nz, int64_t n, float* out, int accumulate, hipStream_t s);
// ---------------------------------------------------------------- residual-branch dropout
// Element (t, n) of branch `site` is kept iff word n % 4 of Philox4x32-10 at counter
// (n / 4, t, site, 0), key (k0, k1), is >= threshold; kept values are multiplied by scale.
struct DropArgs {
  uint32_t k0 = 0, k1 = 0, site = 0, threshold = 0;
  float scale = 1.0f;
  int64_t row0 = 0;            // token index t of the first row passed
};
// out = R + f * (acc + bias) over rows x D (acc fp32 [rows, D]; bias fp32 [D] or null)
hipError_t dropout_add(const float* acc, Dt tr, const void* R, const float* bias, Dt to, void* out, int64_t rows,
                       int64_t D, const DropArgs& a, hipStream_t s);
// out = f * in over rows x D
hipError_t dropout_scale(Dt ti, const void* in, Dt to, void* out, int64_t rows, int64_t D, const DropArgs& a,
                         hipStream_t s);

// bytes (a multiple of 4) of zeros at p, by a kernel (no memset node in captured graphs)
hipError_t fill_zero(void* p, int64_t bytes, hipStream_t s);

}  // namespace bpt
