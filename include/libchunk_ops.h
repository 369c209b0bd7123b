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
 * argument checks before anything is enqueued). Every tensor carries its
 * own element type (lc_dtype); accumulation is fp32 in every kernel.
 * Leading dimensions are in elements.
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
 * (neither k-major). A and B have type `dtype` (LC_BF16: matrix cores;
 * LC_FP32: the fp32 path). Then one epilogue, acc being the fp32 product:
 *
 *   LC_EPI_STORE      C[m*ldc+n] = acc                     (C: c_dtype)
 *   LC_EPI_STORE_F32  same with C fp32
 *   LC_EPI_ACCUM_F32  C[m*ldc+n] += acc, once per element  (C fp32: the
 *                     gradient bucket; the addition happens after the full
 *                     K reduction, so the result is C + (A.B^T) rounded once)
 *   LC_EPI_RESIDUAL   C[m*ldc+n] = R[m*ldr+n] + acc        (R: r_dtype, C: c_dtype)
 *   LC_EPI_ROPE       C = acc, then columns n < rope_cols (the q and k
 *                     blocks of a fused QKV projection) are rotated per
 *                     head of head_dim columns: pair (i, i+hd/2) at
 *                     position p = m mod rope_seq by angle table
 *                     cos/sin[p*hd/2 + i] (fp32 tables, [rope_seq, hd/2]);
 *                     C: c_dtype. head_dim must be 128 for bf16. With aux0
 *                     non-NULL the same values are also written to aux0
 *                     ([M, N], ld_aux, aux_dtype): a second copy in another
 *                     type (the attention backward's bf16 q, k, v).
 *   LC_EPI_SWIGLU     gated FFN input projection: B holds W1 rows
 *                     [0, N) (gate) and W3 rows [N, 2N) (up) (B k-major,
 *                     2N rows); writes gate = acc_W1 to aux0 and
 *                     up = acc_W3 to aux1 ([M, N], leading dim ld_aux,
 *                     aux_dtype) and silu(gate)*up to C ([M, N], ldc,
 *                     c_dtype). N must be a multiple of 64.
 *   LC_EPI_SWIGLU_BWD given da = acc ([M, N]) and gate/up read from
 *                     aux0/aux1 ([M, N], ld_aux, aux_dtype), writes into
 *                     C [M, 2N] (c_dtype):
 *                       C[m*ldc + n]     = da * up * s(g) (1 + g (1 - s(g)))
 *                       C[m*ldc + N + n] = da * silu(g)
 *                     (s = logistic sigmoid, g = gate).
 * Limits of the bf16 kernel: leading dimensions and N multiples of 8; K a
 * multiple of 8 when an operand is k-major; M a multiple of 8 when A is not
 * k-major; 16-byte aligned pointers. Other dimensions may be any positive
 * size (edges are masked).
 */
/* Grouped modes (n_groups groups; group_offsets is a device array of
 * n_groups + 1 nondecreasing offsets written by an earlier kernel, such as the
 * expert offsets of lc_moe_dispatch; values are clamped to [0, M] or [0, K]):
 *   LC_GROUP_NONE  one product as above.
 *   LC_GROUP_ROWS  rows [off[g], off[g+1]) of A and C are multiplied with
 *                  B_g = B + g * group_stride_b (an expert's weights); rows at
 *                  or beyond off[n_groups] are not written. M bounds the rows.
 *   LC_GROUP_K     C_g = C + g * group_stride_c receives the epilogue of
 *                  sum over k in [off[g], off[g+1]) of A(m, k) B(n, k) (an
 *                  expert's weight gradient over its routed rows); both
 *                  operands must not be k-major. K bounds the offsets.
 */
typedef enum lc_gemm_group { LC_GROUP_NONE = 0, LC_GROUP_ROWS = 1, LC_GROUP_K = 2 } lc_gemm_group;

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
  int32_t dtype;        /* lc_dtype of A and B */
  int32_t epilogue;     /* lc_gemm_epilogue */
  int32_t c_dtype;      /* type of C for STORE, RESIDUAL, ROPE, SWIGLU(_BWD) */
  int32_t r_dtype;      /* type of R (RESIDUAL) */
  int32_t aux_dtype;    /* type of aux0/aux1 (SWIGLU, SWIGLU_BWD) */
  int32_t reserved0;
  int64_t M, N, K;
  const void *A; int64_t lda; int32_t a_kmajor;
  int32_t b_kmajor; const void *B; int64_t ldb;
  void *C; int64_t ldc;
  const void *R; int64_t ldr;
  void *aux0; void *aux1; int64_t ld_aux;
  const float *rope_cos; const float *rope_sin;
  int32_t rope_seq; int32_t rope_cols; int32_t head_dim; int32_t reserved1;
  /* grouped products (the experts of a mixture-of-experts FFN); see below */
  int32_t group_mode;              /* lc_gemm_group */
  int32_t n_groups;                /* 1 .. 64 */
  const int32_t *group_offsets;    /* device, n_groups + 1 entries */
  int64_t group_stride_b;          /* LC_GROUP_ROWS: elements from B_g to B_(g+1) */
  int64_t group_stride_c;          /* LC_GROUP_K: elements from C_g to C_(g+1) */
} lc_gemm_args;

lc_status lc_gemm(const lc_gemm_args *args, void *stream);

/* ------------------------------------------------------------------ RMSNorm
 * Forward over T rows of d:
 *   rstd[t] = 1/sqrt(mean_k x[t,k]^2 + eps)   (fp32)
 *   n[t,k]  = x[t,k] * rstd[t] * g[k]
 * Backward, with xh = x*rstd and dxh = dn*g:
 *   dx[t,k] = dres[t,k] + rstd[t] * (dxh[t,k] - xh[t,k] * mean_k'(dxh*xh))
 *   dg_accum[k] += sum_t dn[t,k] * xh[t,k]
 * dres may be NULL (0); dx_copy, if non-NULL, receives dx again as bf16
 * (the operand copy a following bf16 matrix product needs). The gain
 * gradient is a fixed-order reduction (per-block partial sums in `scratch`,
 * lc_rmsnorm_scratch_bytes, then one ordered sum): run-to-run deterministic,
 * one fp32 addition into dg_accum per element. d must be a multiple of 8.
 */
typedef struct lc_norm_args {
  int64_t T, d;
  float eps;
  int32_t x_dtype;     /* x */
  int32_t w_dtype;     /* g */
  int32_t out_dtype;   /* n (forward) or dx (backward) */
  int32_t dn_dtype;    /* dn (backward) */
  int32_t dres_dtype;  /* dres (backward) */
  const void *x; const void *g; void *n; float *rstd;
  const void *dn; const void *dres; void *dx; void *dx_copy; float *dg_accum;
  void *scratch; size_t scratch_bytes;
} lc_norm_args;

lc_status lc_rmsnorm_forward(const lc_norm_args *args, void *stream);
lc_status lc_rmsnorm_backward(const lc_norm_args *args, void *stream);
size_t lc_rmsnorm_scratch_bytes(int64_t T, int64_t d);

/* lc_rmsnorm_backward for callers that cannot allocate device memory (code
 * under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc): the same kernels and results, bit for bit, but the gain
 * gradient's partial sums go to a fixed device array of
 * LC_RMSNORM_NOALLOC_SCRATCH_BYTES inside the library instead of
 * args->scratch (ignored; may be NULL). The call allocates nothing: on the
 * first call on a device it looks up that device's copy of the array
 * (hipGetSymbolAddress, with that device current) and keeps the address.
 * The caller still passes every input and output. Each partial sum is
 * written before it is read, so nothing needs clearing between calls. All
 * calls on one GPU share its array: calls that may overlap on one GPU
 * (different streams without ordering, or host threads) race and must be
 * serialised by the caller. Limit: ceil(T / 16) * d <= 4,194,304 partial
 * sums (for example T <= 16384 at d = 4096), else LC_ERR_WORKSPACE before
 * anything is enqueued. Without dg_accum no scratch is used. */
#define LC_RMSNORM_NOALLOC_SCRATCH_BYTES ((size_t)16 << 20)
lc_status lc_rmsnorm_backward_noalloc(const lc_norm_args *args, void *stream);

/* ------------------------------------------------------------------ attention
 * Causal softmax attention per (batch row b, head h): for query i,
 *   o_i = sum_{j<=i} softmax_j(q_i.k_j / sqrt(hd)) v_j,
 * lse[b,h,i] = log sum_{j<=i} exp(q_i.k_j / sqrt(hd)) (fp32 [B, H, S]).
 * q, k, v, o are [B, S, H*hd] row blocks: element (b, s, h, e) of q sits at
 * q[(b*S + s)*ld_qkv + h*hd + e] (likewise k, v with ld_qkv, o and dout
 * with ld_o, dq, dk, dv with ld_dqkv). Grouped-query attention: with
 * 0 < Hkv < H, k, v, dk, dv have Hkv heads and query head h uses key/value
 * head h / (H / Hkv); dk and dv sum over the query heads of their group
 * (in head order). Hkv = 0 means H.
 * Backward, given dout and P recomputed from lse:
 *   D_i = sum_e dout_ie o_ie, dv_j = sum_i P_ij dout_i,
 *   dS_ij = P_ij (dout_i.v_j - D_i), dq_i = sum_j dS_ij k_j / sqrt(hd),
 *   dk_j = sum_i dS_ij q_i / sqrt(hd);
 * if rope_cos/rope_sin are non-NULL, dq and dk are then rotated back by
 * -angle (the transpose of the forward rotation, positions 0..S-1).
 * Deterministic (no atomics); scratch (lc_attention_scratch_bytes) holds D
 * and -lse log2(e) per query (fp32 [B, H, S] each) and, for fp16 q/k/v, the
 * bf16 copies of q, k and v that the backward's
 * gradient products read. A caller that already holds those copies (the
 * projection's epilogue can write them, lc_gemm LC_EPI_ROPE with aux0) passes
 * them in qkv_bf16: bf16 [B*S, ...] rows of stride ld_qkv_bf16 with q at
 * column 0, k at column H*hd and v at column (H + Hkv)*hd, holding q, k, v
 * rounded to bf16 (from the fp16 values, or from the fp32 values those were
 * rounded from); the backward then reads them instead of writing its own
 * (NULL: it writes them into the scratch).
 * Types: matrix-core path: q, k, v LC_FP16 or LC_BF16 (`dtype`; forward
 * products in that type), o, dout, dq, dk, dv LC_BF16 (gradient products in
 * bf16), head_dim 128, S a multiple of 128. fp32 path: everything LC_FP32,
 * even head_dim <= 128.
 */
typedef struct lc_attn_args {
  int32_t dtype;       /* q, k, v */
  int32_t o_dtype;     /* o, dout, dq, dk, dv */
  int32_t B, S, H, hd;
  const void *q; const void *k; const void *v; int64_t ld_qkv;
  void *o; int64_t ld_o; float *lse;
  const void *dout; void *dq; void *dk; void *dv; int64_t ld_dqkv;
  const float *rope_cos; const float *rope_sin;
  void *scratch; size_t scratch_bytes;
  int32_t Hkv;         /* key/value heads (0 = H); divides H */
  int32_t reserved;
  const void *qkv_bf16; int64_t ld_qkv_bf16;  /* optional bf16 q|k|v copies (backward, fp16 q/k/v) */
} lc_attn_args;

lc_status lc_attention_forward(const lc_attn_args *args, void *stream);
lc_status lc_attention_backward(const lc_attn_args *args, void *stream);
size_t lc_attention_scratch_bytes(int32_t B, int32_t S, int32_t H);
/* The backward's scratch with Hkv key/value heads (grouped-query attention). */
size_t lc_attention_scratch_bytes_kv(int32_t B, int32_t S, int32_t H, int32_t Hkv);

/* ------------------------------------------------------------------ q/k norm
 * Qwen3-style per-head RMSNorm of q and k fused with RoPE, over T tokens of
 * a packed row qk[t] = [q heads 0..H-1 | k heads 0..Hkv-1] (hd values each,
 * row stride ld): for every head row x (hd values),
 *   r = 1/sqrt(mean(x^2) + eps), y = x * r * g   (g = gq for q, gk for k),
 * then rotate-half RoPE on y at position t % seq_len (angles as in the
 * stage: the fp32 tables cos, sin [seq_len, hd/2]).
 * Forward: reads raw x from qk (dtype x_dtype: LC_FP16 or LC_FP32), writes
 * the rotated y back in place, a copy of the raw rows to raw ([T, (H+Hkv)*hd],
 * same dtype) and r to rstd ([T, H+Hkv] fp32).
 * Backward: dqk holds the gradient with respect to y (attention's backward
 * has already undone the rotation) (dtype d_dtype:
 * LC_BF16 or LC_FP32, row stride ld_d); overwrites it in place with the
 * gradient with respect to x (xh = x*r, dxh = dy*g:
 * dx = r*(dxh - xh*mean(dxh*xh))), and adds sum over rows of dy*xh into
 * dgq / dgk (fp32 [hd]; stored instead when store_dg is 1). The gain sums
 * are deterministic: per-block partials in scratch
 * (lc_qk_norm_scratch_bytes), then one ordered sum. hd in {16, 32, 64,
 * 128}; g in w_dtype. */
typedef struct lc_qknorm_args {
  int64_t T;
  int32_t H, Hkv, hd, seq_len;
  float eps;
  int32_t x_dtype, w_dtype, d_dtype;
  void *qk; int64_t ld;
  void *raw; float *rstd;
  const void *gq; const void *gk;
  const float *rope_cos; const float *rope_sin;
  void *dqk; int64_t ld_d;
  float *dgq; float *dgk; int32_t store_dg; int32_t reserved;
  void *scratch; size_t scratch_bytes;
} lc_qknorm_args;

lc_status lc_qk_norm_rope_forward(const lc_qknorm_args *args, void *stream);
lc_status lc_qk_norm_rope_backward(const lc_qknorm_args *args, void *stream);
size_t lc_qk_norm_scratch_bytes(int64_t T, int32_t hd);

/* ------------------------------------------------------------------ MoE routing
 * Router and dispatch of a top-2 mixture-of-experts FFN over T tokens of d
 * features and E experts (2 <= E <= 64); the expert FFNs themselves are
 * grouped products (lc_gemm with LC_GROUP_ROWS / LC_GROUP_K).
 *
 * lc_moe_route reads n [T, d] and the router weights wr [E, d] (element types
 * n_dtype, w_dtype) and writes, per token t:
 *   l[t, e] = sum_i n[t, i] wr[e, i]                    (fp32 accumulation)
 *   sel[t, 0], sel[t, 1] = the two experts of largest softmax(l[t]); equal
 *                          probabilities go to the lower expert index; a NaN
 *                          logit ranks below every number
 *   w[t, k] = softmax(l[t])[sel_k] / (softmax(l[t])[sel_0] + softmax(l[t])[sel_1])
 *           (computed as w0 = 1 / (1 + exp(l1 - l0)), w1 = exp(l1 - l0) w0)
 * sel is int32 [T, 2] and w fp32 [T, 2], device.
 *
 * lc_moe_dispatch groups the 2T (token, expert) pairs of sel/w by expert with
 * a stable counting sort (expert-major, token-minor order; the same result on
 * every run) and writes (device, int32 unless noted):
 *   offsets[E + 1]  offsets[e] = number of pairs routed to experts below e
 *   perm[2T]        token of sorted row r
 *   wrow[2T]        fp32 gate weight w[perm[r], k] of sorted row r
 *   rowpos[T, 2]    sorted row of pair (t, sel[t, k])
 * A pair whose expert is outside [0, E), or repeats the token's first expert,
 * is not placed (rowpos -1); rows past offsets[E] then hold token 0 with
 * weight 0. One workgroup does the whole sort (tokens in chunks of 1024).
 */
typedef struct lc_moe_args {
  int64_t T;
  int32_t d;
  int32_t E;
  int32_t n_dtype;
  int32_t w_dtype;
  const void *n;          /* [T, d] */
  const void *wr;         /* [E, d] */
  int32_t *sel;           /* [T, 2] */
  float *w;               /* [T, 2] */
  int32_t *offsets;       /* [E + 1] */
  int32_t *perm;          /* [2T] */
  float *wrow;            /* [2T] */
  int32_t *rowpos;        /* [T, 2] */
} lc_moe_args;

lc_status lc_moe_route(const lc_moe_args *args, void *stream);
lc_status lc_moe_dispatch(const lc_moe_args *args, void *stream);

/* ------------------------------------------------------------------ casts */

/* out[i] = round-to-nearest-even bf16 of in[i] (NaN stays NaN, made quiet). */
lc_status lc_cast_bf16(const float *in, uint16_t *out, size_t n, void *stream);

#ifdef __cplusplus
}
#endif

#endif /* LIBCHUNK_OPS_H */
