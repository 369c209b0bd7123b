/*
 * libchunk_ops — the individual steps of a decoder stage's Chunk F and
 * Chunk B, exposed one by one so each can be checked on its own. The stage
 * entry points in libchunk.h run exactly these operations.
 *
 * Piper's Chunk exec is the operator graph of the annotated region for F
 * and its autograd graph for B (Piper Section 4.1, "IR"); the paper does not
 * spell out the layer. The formulas below are the standard pre-norm decoder
 * layer of libchunk.h's lc_stage_desc.
 *
 * Conventions of libchunk.h apply (device pointers owned by the caller,
 * stream-ordered, no host synchronisation, no allocation, host-side
 * argument checks before anything is enqueued).
 *
 * Element types: `dtype` (lc_dtype) is the type of activations and weights;
 * accumulation is fp32 in every kernel; fp32 buffers are marked as such.
 * Leading dimensions are in elements and must be multiples of 8; the
 * contiguous extent of every bf16 operand must be a multiple of 8.
 */
#ifndef LIBCHUNK_OPS_H
#define LIBCHUNK_OPS_H

#include "libchunk.h"

#ifdef __cplusplus
extern "C" {
#endif

/* ------------------------------------------------------------------ GEMM
 * C(m, n) = sum_k A(m, k) * B(n, k), fp32 accumulation, with
 *   A(m, k) = a_kmajor ? A[m*lda + k] : A[k*lda + m]
 *   B(n, k) = b_kmajor ? B[n*ldb + k] : B[k*ldb + n]
 * which covers a projection's forward Y = X W^T (both k-major), its input
 * gradient dX = dY W (B not k-major) and its weight gradient dW = dY^T X
 * (neither k-major), followed by one of these epilogues:
 *
 *   LC_EPI_STORE      C[m*ldc+n] = acc                     (dtype)
 *   LC_EPI_STORE_F32  C[m*ldc+n] = acc                     (fp32 C)
 *   LC_EPI_ACCUM_F32  C[m*ldc+n] += acc, once per element  (fp32 C: the
 *                     gradient bucket; the addition happens after the full
 *                     K reduction, so the result equals C + (A.B^T) with
 *                     one fp32 rounding of the sum)
 *   LC_EPI_RESIDUAL   C[m*ldc+n] = R[m*ldr+n] + acc        (dtype)
 *   LC_EPI_ROPE       C = acc, then columns n < rope_cols (the q and k
 *                     blocks of a fused QKV projection) are rotated per
 *                     head of head_dim columns: pair (i, i+hd/2) at
 *                     position p = m mod rope_seq by angle table
 *                     cos/sin[p*hd/2 + i] (fp32 tables, [rope_seq, hd/2]).
 *                     head_dim must be 128 for bf16.
 *   LC_EPI_SWIGLU     gated FFN input projection: B holds W1 rows
 *                     [0, N) (gate) and W3 rows [N, 2N) (up) (B k-major,
 *                     2N rows); writes gate = acc_W1 to aux0 and
 *                     up = acc_W3 to aux1 ([M, N], leading dim ld_aux) and
 *                     silu(gate)*up to C ([M, N], ldc). N must be a
 *                     multiple of 64.
 *   LC_EPI_SWIGLU_BWD given da = acc ([M, N]) and gate/up read from
 *                     aux0/aux1 ([M, N], ld_aux), writes into C [M, 2N]:
 *                       C[m*ldc + n]     = da * up * s(g) (1 + g (1 - s(g)))
 *                       C[m*ldc + N + n] = da * silu(g)
 *                     (s = logistic sigmoid, g = gate).
 * Dimensions may be any positive size except as noted (edges are masked).
 */
typedef enum lc_gemm_epilogue {
  LC_EPI_STORE = 0,
  LC_EPI_STORE_F32 = 1,
  LC_EPI_ACCUM_F32 = 2,
  LC_EPI_RESIDUAL = 3,
  LC_EPI_ROPE = 4,
  LC_EPI_SWIGLU = 5,
  LC_EPI_SWIGLU_BWD = 6
} lc_gemm_epilogue;

typedef struct lc_gemm_args {
  int32_t dtype;        /* lc_dtype of A and B (and of C for non-F32 epilogues) */
  int32_t epilogue;     /* lc_gemm_epilogue */
  int64_t M, N, K;
  const void *A; int64_t lda; int32_t a_kmajor;
  int32_t b_kmajor; const void *B; int64_t ldb;
  void *C; int64_t ldc;
  const void *R; int64_t ldr;           /* LC_EPI_RESIDUAL */
  void *aux0; void *aux1; int64_t ld_aux; /* SWIGLU / SWIGLU_BWD */
  const float *rope_cos; const float *rope_sin; /* LC_EPI_ROPE */
  int32_t rope_seq; int32_t rope_cols; int32_t head_dim; int32_t reserved;
} lc_gemm_args;

lc_status lc_gemm(const lc_gemm_args *args, void *stream);

/* ------------------------------------------------------------------ RMSNorm
 * Forward over T rows of d: rstd[t] = 1/sqrt(mean_k x[t,k]^2 + eps) (fp32),
 * n[t,k] = x[t,k] * rstd[t] * g[k]. */
lc_status lc_rmsnorm_forward(int32_t dtype, int64_t T, int64_t d, const void *x,
                             const void *g, float eps, void *n, float *rstd, void *stream);

/* Backward: with xh = x*rstd and dxh = dn*g,
 *   dx[t,k] = dres[t,k] + rstd[t] * (dxh[t,k] - xh[t,k] * mean_k'(dxh*xh))
 * (dres nullable = 0), and dg_accum[k] += sum_t dn[t,k]*xh[t,k] (fp32, a
 * fixed-order reduction: per-block partials in `scratch`, then one ordered
 * sum; run-to-run deterministic). scratch: lc_rmsnorm_scratch_bytes. */
lc_status lc_rmsnorm_backward(int32_t dtype, int64_t T, int64_t d, const void *dn,
                              const void *x, const float *rstd, const void *g,
                              const void *dres, void *dx, float *dg_accum,
                              void *scratch, size_t scratch_bytes, void *stream);
size_t lc_rmsnorm_scratch_bytes(int64_t T, int64_t d);

/* ------------------------------------------------------------------ attention
 * Causal softmax attention per (batch row b, head h): for query i,
 *   o_i = sum_{j<=i} softmax_j(q_i.k_j / sqrt(hd)) v_j,
 * lse[b,h,i] = log sum_{j<=i} exp(q_i.k_j / sqrt(hd)) (fp32).
 * q, k, v, o are [B, S, H*hd] row blocks: element (b, s, h, e) of q sits at
 * q[(b*S + s)*ld_qkv + h*hd + e] (likewise k, v with ld_qkv, o with ld_o).
 * bf16 requires hd == 128; fp32 requires hd <= 128. */
lc_status lc_attention_forward(int32_t dtype, int32_t B, int32_t S, int32_t H, int32_t hd,
                               const void *q, const void *k, const void *v, int64_t ld_qkv,
                               void *o, int64_t ld_o, float *lse, void *stream);

/* Backward of the above given do (ld_o, like o): with P recomputed from lse,
 *   D_i = sum_e do_ie o_ie, dv_j = sum_i P_ij do_i,
 *   dS_ij = P_ij (do_i.v_j - D_i), dq_i = sum_j dS_ij k_j / sqrt(hd),
 *   dk_j = sum_i dS_ij q_i / sqrt(hd).
 * If rope_cos/rope_sin are non-NULL, dq and dk are then rotated back by
 * -angle (the transpose of the forward rotation, positions 0..S-1).
 * dq, dk, dv use ld_dqkv. scratch (fp32, lc_attention_scratch_bytes) holds
 * D. Deterministic: no atomics. */
lc_status lc_attention_backward(int32_t dtype, int32_t B, int32_t S, int32_t H, int32_t hd,
                                const void *q, const void *k, const void *v, int64_t ld_qkv,
                                const void *o, const void *dout, int64_t ld_o,
                                const float *lse, void *dq, void *dk, void *dv,
                                int64_t ld_dqkv, const float *rope_cos, const float *rope_sin,
                                void *scratch, size_t scratch_bytes, void *stream);
size_t lc_attention_scratch_bytes(int32_t B, int32_t S, int32_t H);

/* ------------------------------------------------------------------ casts */

/* out[i] = round-to-nearest-even bf16 of in[i] (NaN stays NaN, made quiet). */
lc_status lc_cast_bf16(const float *in, uint16_t *out, size_t n, void *stream);

#ifdef __cplusplus
}
#endif

#endif /* LIBCHUNK_OPS_H */
