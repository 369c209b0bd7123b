// Host-only core of libchunk: descriptor validation, the canonical parameter
// layout, Order generation/validation and the workspace plan. No HIP calls,
// so it builds with the plain host compiler and is testable without a GPU.
#pragma once

#include <stddef.h>
#include <stdint.h>

#include <vector>

#include "libchunk.h"

#define LC_TRY(expr)                 \
  do {                               \
    lc_status _st = (expr);          \
    if (_st != LC_OK) return _st;    \
  } while (0)

namespace lc {

lc_status fail(lc_status st, const char *fmt, ...) __attribute__((format(printf, 2, 3)));

// Rows per block of the RMSNorm backward's gain-gradient partial sums.
constexpr int kNormRowsPerBlock = 16;
size_t rmsnorm_scratch_size(int64_t T, int64_t d);
size_t attn_scratch_size(int64_t B, int64_t S, int64_t H, int64_t Hkv);
// byte offset of grouped-query attention's dk/dv shares in that scratch
size_t attn_share_offset(int64_t B, int64_t S, int64_t H, int64_t Hkv);
// Tokens per block of the per-head q/k RMSNorm's gain-gradient partial sums
// (each block writes 2 * head_dim floats: q gains, then k gains).
constexpr int kQkTokensPerBlock = 4;
size_t qknorm_scratch_size(int64_t T, int64_t hd);
inline int kv_heads(const lc_stage_desc &d) { return d.n_kv_heads > 0 ? d.n_kv_heads : d.n_heads; }
// Tokens per block of the MoE router weight gradient's partial sums.
constexpr int kRouterTokensPerBlock = 128;
size_t moe_router_scratch_size(int64_t T, int64_t d, int64_t E);

// An Order's entries as one sequence: the LC_ORDER_WITH_NEXT flag removed
// and every overlapped pair checked (LC_ERR_BAD_ORDER) and put with its
// acquiring entry (F, or Bi beside Bw) first.
lc_status flatten_order(const lc_order &order, std::vector<lc_order_entry> *flat);

// Validates a stage descriptor (shapes, dtype, the kernels' limits).
lc_status validate_desc(const lc_stage_desc *d);

// Per-layer sizes of the canonical flat bucket.
struct ParamPlan {
  size_t per_layer;                 // elements per layer
  size_t wq, wk, wv, wo, g1;        // offsets inside a layer
  size_t qn, kn;                    // per-head q/k norm gains (qk_norm)
  size_t w1, w3, w2;                // dense FFN
  size_t wr, expert0, expert_stride;  // MoE: router, first expert's W1, stride per expert
  size_t g2;
  size_t total;
};
ParamPlan param_plan(const lc_stage_desc &d);

// Where every stashed activation and scratch buffer lives in the caller's
// workspace. Offsets are bytes from the workspace base, 256-byte aligned.
// Element types of a stage's internal tensors (see lc_stage_desc's precision
// note): GEMM operands in the compute dtype, attention q/k/v in fp16 for bf16
// stages, residual stream / gate-up stash / norm inputs in fp32.
struct StageTypes {
  int op;    // GEMM operand activations and gradients (n1, o, n2, act, dgu, dqkv, ...)
  int att;   // attention q, k, v
  int res;   // residual stream, its gradient, gate/up stash, norm-input gradients
};
StageTypes stage_types(const lc_stage_desc &d);

struct StagePlan {
  size_t elem;          // bytes per GEMM-operand element (2 or 4)
  StageTypes ty;
  int64_t T;            // tokens per microbatch
  int64_t dkv;          // key/value width n_kv_heads * head_dim
  int64_t qkv_cols;     // d + 2 dkv: columns of the packed q|k|v
  // RoPE table: cos then sin, fp32 [seq_len, head_dim/2]
  size_t rope_cos, rope_sin;
  // stash: max_in_flight slots of n_layers layer blocks
  size_t slot0, slot_bytes, layer_bytes;
  // offsets inside one layer block
  size_t xin, rstd1, n1, qkv, o, lse, h, rstd2, n2, gate, up, act;
  // qk_norm: the projection's raw q|k [T, d + dkv] (att type) and the
  // per-head reciprocal RMS [T, n_heads + n_kv_heads] (fp32)
  size_t qkraw, rstdqk;
  // fp16 attention operands without qk_norm: the projection's bf16 copy of
  // q|k|v [T, qkv_cols] for the attention backward's gradient products (0: none)
  size_t qkvb;
  // weight-pass slots (split backward): max_w_pending slots of n_layers
  // blocks, each holding the gradient operands a backward-for-inputs pass
  // leaves for the backward-for-weights pass of the same microbatch: the
  // layer-output gradient dy [T, d], dgate|dup [T, 2f], dh [T, d] and
  // dq|dk|dv [T, 3d] (op type), and the fp32 gain-gradient partial sums of
  // both norms (rmsnorm_scratch_size each)
  int32_t w_slots;
  size_t wslot0, wslot_bytes, wlayer_bytes;
  size_t w_dy, w_da, w_dh, w_dqkv, w_p2, w_p1, w_pqk;
  size_t w_dys, w_dl, w_rpart;  // MoE layers: routed dy rows, router logit gradients, dWr partials
  // MoE per-layer extras (0 when dense): routing (sel, w [T, 2]), dispatch
  // (perm, wrow [2T], rowpos [T, 2], expert offsets [E + 1]), the gathered
  // expert inputs xp [2T, d] (op type) and expert outputs eo [2T, d] (fp32)
  size_t moe_sel, moe_w, moe_perm, moe_wrow, moe_rowpos, moe_off, moe_xp, moe_eo;
  // backward scratch (one set, reused by every microbatch)
  size_t s_dy0, s_dy1;  // residual-stream gradient ping-pong [T, d] (res type)
  size_t s_dy16;        // operand copy of the current layer's dy [T, d] (op type)
  size_t s_da;          // dgate|dup [T, 2f] (or MoE rows [2T, 2fe])
  size_t s_dn;          // [T, d] gradient at a norm output (res type)
  size_t s_do;          // [T, d] gradient at attention output
  size_t s_dqkv;        // [T, 3d]
  size_t s_dh;          // [T, d] (res type)
  size_t s_dh16;        // operand copy of dh [T, d] (op type)
  size_t s_attn, s_attn_bytes;  // attention backward scratch
  size_t s_norm, s_norm_bytes;  // RMSNorm backward scratch
  size_t s_qkn, s_qkn_bytes;    // q/k norm gain partial sums (qk_norm)
  // MoE backward: weighted expert-output gradients dys [2T, d] (op type),
  // expert-input gradients dns [2T, d] (fp32), gate-weight gradients dw [2T],
  // router-logit gradients dl [T, 2], router weight-gradient partial sums
  size_t s_moe_dys, s_moe_dns, s_moe_dw, s_moe_dl, s_moe_part, s_moe_part_bytes;
  size_t total;
};
lc_status stage_plan(const lc_stage_desc &d, int32_t max_in_flight, int32_t max_w_pending,
                     StagePlan *out);

}  // namespace lc
