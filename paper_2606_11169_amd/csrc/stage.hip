// Stage composer: Chunk F / Chunk B of a decoder pipeline stage as a sequence
// of kernel launches on the caller's stream, the activation stash, and the
// Order runner.
//
// Piper's worker runs the tasks of its sub-DAG in order on their streams,
// keeps a forward's outputs in local storage until the last consumer (the
// matching backward) has been scheduled, then frees them (Piper Section
// 4.3.2, scheduling loop and "Memory management"). Here one stage runs on one
// stream, so stream order alone makes reuse of a freed stash slot safe: a slot
// is taken by chunk_forward(mb) and returned by chunk_backward(mb) as soon as
// its launches are enqueued. Gradients of every backward are added into the
// bucket's flat fp32 buffer (Section 4.3.2; accumulated across microbatches,
// Section 6.2).
//
// Split backward (Section 4.1, PASS values Bi and Bw): the backward for the
// inputs runs every input-gradient launch of Chunk B and leaves the operands
// of the weight-gradient products (per layer: the layer-output gradient,
// dgate|dup, dh, dq|dk|dv, all in the operand type, and both norms' gain
// partial sums) in a weight-pass slot; the backward for the weights runs the
// weight-gradient products and the gain sums from there, then frees the
// weight-pass slot and the stash slot (the products also read n1, o, n2 and
// act from the stash). The same kernels in the same per-element order make
// the gradient bit-identical to Chunk B's.
//
// Tensor element types follow StageTypes: matrix-product operands in the
// compute dtype, attention q/k/v in fp16 for a bf16 stage, and the residual
// stream (inside and between layers), its gradient, the gate/up values kept
// for the backward and every norm input in fp32.
#include "common.hpp"

#include <math.h>
#include <stdlib.h>
#include <string.h>

#include <algorithm>
#include <new>
#include <vector>

struct lc_stage {
  lc_stage_desc d;
  lc::StagePlan plan;
  lc::ParamPlan pp;
  char *ws;
  int32_t slots;
  std::vector<int32_t> owner;      // microbatch stashed in each slot, -1 if free
  std::vector<const void *> xin0;  // the caller's X of that microbatch
  std::vector<int32_t> wowner;     // microbatch whose weight pass is pending, per weight-pass slot
  std::vector<hipEvent_t> events;  // cross-stream synchronisation of lc_run_order_overlap
  bool grad_store = false;         // backwards overwrite the gradient buffer (ZeRO runs, dense)
  std::vector<hipEvent_t> tev;     // weight-gradient product timing: start, stop per launch
  std::vector<double> tflop;       // algorithmic FLOP of each timed launch (size = capacity)
  int32_t tn = 0;                  // launches timed since the last read
  std::vector<float> rope_host;    // cos table then sin table (fp32)
};

namespace lc {

lc_status hip_fail(hipError_t e, const char *what) {
  return fail(LC_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

namespace {

struct LayerBufs {
  char *base;
  void *at(size_t off) const { return base + off; }
};

struct W {  // weight pointers of one layer (compute dtype) and grad pointers (fp32)
  const char *w;
  float *g;
  size_t es;
  const void *wp(size_t off) const { return w + off * es; }
  float *gp(size_t off) const { return g + off; }
};

lc_gemm_args gemm_base(int dtype, int epi, int64_t M, int64_t N, int64_t K) {
  lc_gemm_args a;
  memset(&a, 0, sizeof a);
  a.dtype = dtype;
  a.epilogue = epi;
  a.c_dtype = dtype;
  a.M = M;
  a.N = N;
  a.K = K;
  return a;
}

// A weight-gradient product (fp32 output into the gradient), bracketed by the
// stage's timing events on its stream while lc_stage_timer_enable has left
// capacity.
lc_status wgrad_launch(lc_stage *st, const lc_gemm_args &a, hipStream_t s) {
  const int32_t i = st->tn;
  const bool timed = i < (int32_t)st->tflop.size();
  if (timed) {
    const hipError_t e = hipEventRecord(st->tev[2 * i], s);
    if (e != hipSuccess) return hip_fail(e, "recording a timing event");
  }
  LC_TRY(gemm_launch(a, s));
  if (timed) {
    const hipError_t e = hipEventRecord(st->tev[2 * i + 1], s);
    if (e != hipSuccess) return hip_fail(e, "recording a timing event");
    st->tflop[i] = 2.0 * (double)a.M * (double)a.N * (double)a.K;
    st->tn = i + 1;
  }
  return LC_OK;
}

lc_norm_args norm_base(int64_t T, int64_t d, float eps) {
  lc_norm_args a;
  memset(&a, 0, sizeof a);
  a.T = T;
  a.d = d;
  a.eps = eps;
  return a;
}

}  // namespace

static LayerBufs layer_bufs(lc_stage *st, int slot, int l) {
  LayerBufs b;
  b.base = st->ws + st->plan.slot0 + (size_t)slot * st->plan.slot_bytes +
           (size_t)l * st->plan.layer_bytes;
  return b;
}

static LayerBufs wlayer_bufs(lc_stage *st, int wslot, int l) {
  LayerBufs b;
  b.base = st->ws + st->plan.wslot0 + (size_t)wslot * st->plan.wslot_bytes +
           (size_t)l * st->plan.wlayer_bytes;
  return b;
}

// MoE FFN of one layer (Chunk F): route, dispatch, gather, two grouped
// expert products, weighted combine with the residual h.
static lc_status moe_forward(lc_stage *st, const W &w, const LayerBufs &L, void *out, int out_dt,
                             hipStream_t s) {
  const lc_stage_desc &d = st->d;
  const StagePlan &P = st->plan;
  const ParamPlan &pp = st->pp;
  const int dt = d.compute_dtype;
  const StageTypes ty = P.ty;
  const int64_t T = P.T, D = d.d_model, FE = d.d_ff_expert, R = 2 * T;
  const int E = d.n_experts;
  lc_moe_args ma;
  memset(&ma, 0, sizeof ma);
  ma.T = T; ma.d = (int32_t)D; ma.E = E; ma.n_dtype = ty.op; ma.w_dtype = dt;
  ma.n = L.at(P.n2); ma.wr = w.wp(pp.wr);
  ma.sel = static_cast<int32_t *>(L.at(P.moe_sel));
  ma.w = static_cast<float *>(L.at(P.moe_w));
  ma.offsets = static_cast<int32_t *>(L.at(P.moe_off));
  ma.perm = static_cast<int32_t *>(L.at(P.moe_perm));
  ma.wrow = static_cast<float *>(L.at(P.moe_wrow));
  ma.rowpos = static_cast<int32_t *>(L.at(P.moe_rowpos));
  LC_TRY(moe_route_launch(ma, s));
  LC_TRY(moe_dispatch_launch(ma, s));
  LC_TRY(moe_gather_launch(L.at(P.n2), L.at(P.moe_xp), ma.perm, R, D * (int64_t)P.elem, s));
  // gate, up = xp [W1_e; W3_e]^T per expert; act = silu(gate) * up
  lc_gemm_args a = gemm_base(dt, LC_EPI_SWIGLU, R, FE, D);
  a.A = L.at(P.moe_xp); a.lda = D; a.a_kmajor = 1;
  a.B = w.wp(pp.expert0); a.ldb = D; a.b_kmajor = 1;
  a.C = L.at(P.act); a.ldc = FE; a.c_dtype = ty.op;
  a.aux0 = L.at(P.gate); a.aux1 = L.at(P.up); a.ld_aux = FE; a.aux_dtype = ty.res;
  a.group_mode = LC_GROUP_ROWS; a.n_groups = E; a.group_offsets = ma.offsets;
  a.group_stride_b = (int64_t)pp.expert_stride;
  LC_TRY(gemm_launch(a, s));
  // eo = act W2_e^T per expert (fp32)
  a = gemm_base(dt, LC_EPI_STORE_F32, R, D, FE);
  a.A = L.at(P.act); a.lda = FE; a.a_kmajor = 1;
  a.B = w.wp(pp.expert0 + 2 * FE * D); a.ldb = FE; a.b_kmajor = 1;
  a.C = L.at(P.moe_eo); a.ldc = D;
  a.group_mode = LC_GROUP_ROWS; a.n_groups = E; a.group_offsets = ma.offsets;
  a.group_stride_b = (int64_t)pp.expert_stride;
  LC_TRY(gemm_launch(a, s));
  // out = h + w0 eo[rowpos0] + w1 eo[rowpos1]
  return moe_combine_launch(L.at(P.h), ty.res, static_cast<const float *>(L.at(P.moe_eo)), ma.w,
                            ma.rowpos, out, out_dt, T, (int)D, s);
}

// G[W2_e] += dys_e^T act_e over each expert's rows
static lc_status moe_w2_grad(lc_stage *st, const W &w, const LayerBufs &L, const void *dys,
                             hipStream_t s) {
  const StagePlan &P = st->plan;
  const ParamPlan &pp = st->pp;
  const int64_t D = st->d.d_model, FE = st->d.d_ff_expert, R = 2 * P.T;
  lc_gemm_args a = gemm_base(st->d.compute_dtype, LC_EPI_ACCUM_F32, D, FE, R);
  a.A = dys; a.lda = D; a.a_kmajor = 0;
  a.B = L.at(P.act); a.ldb = FE; a.b_kmajor = 0;
  a.C = w.gp(pp.expert0 + 2 * FE * D); a.ldc = FE;
  a.group_mode = LC_GROUP_K; a.n_groups = st->d.n_experts;
  a.group_offsets = static_cast<const int32_t *>(L.at(P.moe_off));
  a.group_stride_c = (int64_t)pp.expert_stride;
  return wgrad_launch(st, a, s);
}

// G[W1_e; W3_e] += [dgate | dup]_e^T xp_e
static lc_status moe_w13_grad(lc_stage *st, const W &w, const LayerBufs &L, const void *da,
                              hipStream_t s) {
  const StagePlan &P = st->plan;
  const ParamPlan &pp = st->pp;
  const int64_t D = st->d.d_model, FE = st->d.d_ff_expert, R = 2 * P.T;
  lc_gemm_args a = gemm_base(st->d.compute_dtype, LC_EPI_ACCUM_F32, 2 * FE, D, R);
  a.A = da; a.lda = 2 * FE; a.a_kmajor = 0;
  a.B = L.at(P.moe_xp); a.ldb = D; a.b_kmajor = 0;
  a.C = w.gp(pp.expert0); a.ldc = D;
  a.group_mode = LC_GROUP_K; a.n_groups = st->d.n_experts;
  a.group_offsets = static_cast<const int32_t *>(L.at(P.moe_off));
  a.group_stride_c = (int64_t)pp.expert_stride;
  return wgrad_launch(st, a, s);
}

// MoE FFN of one layer (Chunk B): given dy (the gradient at the layer output),
// writes dn = dL/dn2 (fp32, P.s_dn) and adds the expert and router weight
// gradients into the bucket. With a weight-pass layer block WL (the backward
// for the inputs) the routed dy rows, [dgate | dup] and the router logit
// gradients go there instead, and moe_weight adds the weight gradients.
static lc_status moe_backward(lc_stage *st, const W &w, const LayerBufs &L, const void *dy,
                              int dy_dt, hipStream_t s, const LayerBufs *WL = nullptr) {
  const lc_stage_desc &d = st->d;
  const StagePlan &P = st->plan;
  const ParamPlan &pp = st->pp;
  const int dt = d.compute_dtype;
  const StageTypes ty = P.ty;
  const int64_t T = P.T, D = d.d_model, FE = d.d_ff_expert, R = 2 * T;
  const int E = d.n_experts;
  char *ws = st->ws;
  const int32_t *off = static_cast<const int32_t *>(L.at(P.moe_off));
  const float *eo = static_cast<const float *>(L.at(P.moe_eo));
  void *dys = WL ? WL->at(P.w_dys) : ws + P.s_moe_dys;
  float *dns = reinterpret_cast<float *>(ws + P.s_moe_dns);
  float *dw = reinterpret_cast<float *>(ws + P.s_moe_dw);
  float *dl = WL ? static_cast<float *>(WL->at(P.w_dl)) : reinterpret_cast<float *>(ws + P.s_moe_dl);
  void *da = WL ? WL->at(P.w_da) : ws + P.s_da;
  // dys[r] = wrow[r] dy[perm[r]], dw[r] = dy[perm[r]] . eo[r]
  LC_TRY(moe_bwd_gather_launch(dy, dy_dt, eo, static_cast<const int32_t *>(L.at(P.moe_perm)),
                               static_cast<const float *>(L.at(P.moe_wrow)), dys, ty.op, dw, R,
                               (int)D, s));
  // [dgate | dup] = SwiGLU'(dys W2_e) per expert
  lc_gemm_args a = gemm_base(dt, LC_EPI_SWIGLU_BWD, R, FE, D);
  a.A = dys; a.lda = D; a.a_kmajor = 1;
  a.B = w.wp(pp.expert0 + 2 * FE * D); a.ldb = FE; a.b_kmajor = 0;
  a.C = da; a.ldc = 2 * FE; a.c_dtype = ty.op;
  a.aux0 = L.at(P.gate); a.aux1 = L.at(P.up); a.ld_aux = FE; a.aux_dtype = ty.res;
  a.group_mode = LC_GROUP_ROWS; a.n_groups = E; a.group_offsets = off;
  a.group_stride_b = (int64_t)pp.expert_stride;
  LC_TRY(gemm_launch(a, s));
  if (!WL) LC_TRY(moe_w2_grad(st, w, L, dys, s));
  // dns = [dgate | dup] [W1_e; W3_e] per expert (fp32)
  a = gemm_base(dt, LC_EPI_STORE_F32, R, D, 2 * FE);
  a.A = da; a.lda = 2 * FE; a.a_kmajor = 1;
  a.B = w.wp(pp.expert0); a.ldb = D; a.b_kmajor = 0;
  a.C = dns; a.ldc = D;
  a.group_mode = LC_GROUP_ROWS; a.n_groups = E; a.group_offsets = off;
  a.group_stride_b = (int64_t)pp.expert_stride;
  LC_TRY(gemm_launch(a, s));
  if (!WL) LC_TRY(moe_w13_grad(st, w, L, da, s));
  // dn = dns[rowpos0] + dns[rowpos1] + dl Wr; then G[Wr] += dl^T n2
  const int32_t *sel = static_cast<const int32_t *>(L.at(P.moe_sel));
  LC_TRY(moe_bwd_combine_launch(dns, dw, static_cast<const float *>(L.at(P.moe_w)), sel,
                                static_cast<const int32_t *>(L.at(P.moe_rowpos)), w.wp(pp.wr), dt,
                                dl, reinterpret_cast<float *>(ws + P.s_dn), T, (int)D, s));
  if (WL) return LC_OK;
  return moe_router_grad_launch(L.at(P.n2), ty.op, sel, dl,
                                reinterpret_cast<float *>(ws + P.s_moe_part), P.s_moe_part_bytes,
                                w.gp(pp.wr), T, (int)D, E, s);
}

// The backward for the weights of a MoE FFN: the expert and router weight
// gradients from the operands moe_backward left in the weight-pass layer
// block WL (the router's partial sums go to WL too).
static lc_status moe_weight(lc_stage *st, const W &w, const LayerBufs &L, const LayerBufs &WL,
                            hipStream_t s) {
  const StagePlan &P = st->plan;
  LC_TRY(moe_w2_grad(st, w, L, WL.at(P.w_dys), s));
  LC_TRY(moe_w13_grad(st, w, L, WL.at(P.w_da), s));
  return moe_router_grad_launch(L.at(P.n2), P.ty.op, static_cast<const int32_t *>(L.at(P.moe_sel)),
                                static_cast<const float *>(WL.at(P.w_dl)),
                                static_cast<float *>(WL.at(P.w_rpart)),
                                moe_router_scratch_size(P.T, st->d.d_model, st->d.n_experts),
                                w.gp(st->pp.wr), P.T, st->d.d_model, st->d.n_experts, s);
}

// The per-head q/k norm arguments of one layer (q|k of the packed qkv rows).
static lc_qknorm_args qknorm_base(lc_stage *st, const W &w, const LayerBufs &L) {
  const lc_stage_desc &d = st->d;
  const StagePlan &P = st->plan;
  lc_qknorm_args q;
  memset(&q, 0, sizeof q);
  q.T = P.T;
  q.H = d.n_heads; q.Hkv = kv_heads(d); q.hd = d.head_dim; q.seq_len = d.seq_len;
  q.eps = d.rms_eps;
  q.x_dtype = P.ty.att; q.w_dtype = d.compute_dtype; q.d_dtype = P.ty.op;
  q.qk = L.at(P.qkv); q.ld = P.qkv_cols;
  q.raw = L.at(P.qkraw); q.rstd = static_cast<float *>(L.at(P.rstdqk));
  q.gq = w.wp(st->pp.qn); q.gk = w.wp(st->pp.kn);
  return q;
}

static lc_status forward_layers(lc_stage *st, const lc_param_bufs *pb, const void *x, void *y,
                                int slot, hipStream_t s) {
  const lc_stage_desc &d = st->d;
  const StagePlan &P = st->plan;
  const ParamPlan &pp = st->pp;
  const int dt = d.compute_dtype;
  const StageTypes ty = P.ty;
  const int64_t T = P.T, D = d.d_model, F = d.d_ff, Dkv = P.dkv, QC = P.qkv_cols;
  const size_t ea = dtype_size(ty.att);
  const float *rc = reinterpret_cast<const float *>(st->ws + P.rope_cos);
  const float *rs = reinterpret_cast<const float *>(st->ws + P.rope_sin);
  for (int l = 0; l < d.n_layers; ++l) {
    const LayerBufs L = layer_bufs(st, slot, l);
    const W w{static_cast<const char *>(pb->w) + (size_t)l * pp.per_layer * P.elem, nullptr, P.elem};
    const bool first = l == 0, last = l == d.n_layers - 1;
    const void *xin = first ? x : L.at(P.xin);
    const int x_dt = first ? dt : ty.res;
    void *out = last ? y : layer_bufs(st, slot, l + 1).at(P.xin);
    // n1 = RMSNorm(x; g1)
    lc_norm_args na = norm_base(T, D, d.rms_eps);
    na.x = xin; na.x_dtype = x_dt;
    na.g = w.wp(pp.g1); na.w_dtype = dt;
    na.n = L.at(P.n1); na.out_dtype = ty.op;
    na.rstd = static_cast<float *>(L.at(P.rstd1));
    LC_TRY(rmsnorm_fwd_launch(na, s));
    // [q|k|v] = n1 [Wq;Wk;Wv]^T, RoPE on q and k (after their per-head norm)
    lc_gemm_args a = gemm_base(dt, d.qk_norm ? LC_EPI_STORE : LC_EPI_ROPE, T, QC, D);
    a.A = L.at(P.n1); a.lda = D; a.a_kmajor = 1;
    a.B = w.wp(pp.wq); a.ldb = D; a.b_kmajor = 1;
    a.C = L.at(P.qkv); a.ldc = QC; a.c_dtype = ty.att;
    if (!d.qk_norm) {
      a.rope_cos = rc; a.rope_sin = rs; a.rope_seq = d.seq_len; a.rope_cols = (int)(D + Dkv);
      a.head_dim = d.head_dim;
      if (P.qkvb) {  // the bf16 copy the attention backward's gradient products read
        a.aux0 = L.at(P.qkvb); a.ld_aux = QC; a.aux_dtype = LC_BF16;
      }
    }
    LC_TRY(gemm_launch(a, s));
    if (d.qk_norm) {
      lc_qknorm_args qa = qknorm_base(st, w, L);
      qa.rope_cos = rc; qa.rope_sin = rs;
      LC_TRY(qknorm_fwd_launch(qa, s));
    }
    // o = causal attention
    char *qkv = static_cast<char *>(L.at(P.qkv));
    lc_attn_args at;
    memset(&at, 0, sizeof at);
    at.dtype = ty.att; at.o_dtype = ty.op;
    at.B = d.micro_batch; at.S = d.seq_len; at.H = d.n_heads; at.hd = d.head_dim;
    at.Hkv = kv_heads(d);
    at.q = qkv; at.k = qkv + D * ea; at.v = qkv + (D + Dkv) * ea; at.ld_qkv = QC;
    at.o = L.at(P.o); at.ld_o = D; at.lse = static_cast<float *>(L.at(P.lse));
    LC_TRY(attn_fwd_launch(at, s));
    // h = x + o Wo^T
    a = gemm_base(dt, LC_EPI_RESIDUAL, T, D, D);
    a.A = L.at(P.o); a.lda = D; a.a_kmajor = 1;
    a.B = w.wp(pp.wo); a.ldb = D; a.b_kmajor = 1;
    a.C = L.at(P.h); a.ldc = D; a.c_dtype = ty.res;
    a.R = xin; a.ldr = D; a.r_dtype = x_dt;
    LC_TRY(gemm_launch(a, s));
    // n2 = RMSNorm(h; g2)
    na.x = L.at(P.h); na.x_dtype = ty.res;
    na.g = w.wp(pp.g2);
    na.n = L.at(P.n2);
    na.rstd = static_cast<float *>(L.at(P.rstd2));
    LC_TRY(rmsnorm_fwd_launch(na, s));
    if (d.n_experts > 0) {
      LC_TRY(moe_forward(st, w, L, out, last ? dt : ty.res, s));
      continue;
    }
    // gate, up = n2 W1^T, n2 W3^T; act = silu(gate) * up
    a = gemm_base(dt, LC_EPI_SWIGLU, T, F, D);
    a.A = L.at(P.n2); a.lda = D; a.a_kmajor = 1;
    a.B = w.wp(pp.w1); a.ldb = D; a.b_kmajor = 1;
    a.C = L.at(P.act); a.ldc = F; a.c_dtype = ty.op;
    a.aux0 = L.at(P.gate); a.aux1 = L.at(P.up); a.ld_aux = F; a.aux_dtype = ty.res;
    LC_TRY(gemm_launch(a, s));
    // y = h + act W2^T
    a = gemm_base(dt, LC_EPI_RESIDUAL, T, D, F);
    a.A = L.at(P.act); a.lda = F; a.a_kmajor = 1;
    a.B = w.wp(pp.w2); a.ldb = F; a.b_kmajor = 1;
    a.C = out; a.ldc = D; a.c_dtype = last ? dt : ty.res;
    a.R = L.at(P.h); a.ldr = D; a.r_dtype = ty.res;
    LC_TRY(gemm_launch(a, s));
  }
  return LC_OK;
}

// Chunk B (wslot < 0), or the backward for the inputs (wslot >= 0: weight
// products skipped, their operands and the gain partial sums left in weight-
// pass slot wslot).
// RMSNorm backward of Chunk B with its gain gradient added into (or, for a
// stage writing fresh gradients, stored to) dg.
static lc_status norm_bwd_full(const lc_stage *st, lc_norm_args nb, float *dg, hipStream_t s) {
  if (!st->grad_store) {
    nb.dg_accum = dg;
    return rmsnorm_bwd_launch(nb, s);
  }
  LC_TRY(rmsnorm_bwd_partials_launch(nb, s));
  return rmsnorm_dg_final_launch(static_cast<const float *>(nb.scratch), dg, nb.T, nb.d, s, true);
}

static lc_status backward_layers(lc_stage *st, const lc_param_bufs *pb, const void *x0,
                                 const void *dy_in, void *dx_out, int slot, int wslot,
                                 hipStream_t s) {
  const lc_stage_desc &d = st->d;
  const StagePlan &P = st->plan;
  const ParamPlan &pp = st->pp;
  const int dt = d.compute_dtype;
  const StageTypes ty = P.ty;
  const bool copies = ty.op != ty.res;  // bf16 operand copies of fp32 gradients
  const bool split = wslot >= 0;
  // the weight products overwrite their gradient instead of adding into it
  const int gepi = st->grad_store ? LC_EPI_STORE_F32 : LC_EPI_ACCUM_F32;
  const int64_t T = P.T, D = d.d_model, F = d.d_ff, Dkv = P.dkv, QC = P.qkv_cols;
  const size_t ea = dtype_size(ty.att), es = P.elem;
  const float *rc = reinterpret_cast<const float *>(st->ws + P.rope_cos);
  const float *rs = reinterpret_cast<const float *>(st->ws + P.rope_sin);
  char *ws = st->ws;
  // gradient flowing into the current layer: residual version and operand version
  const void *dy_res = dy_in, *dy_op = dy_in;
  int dy_dt = dt;
  if (split) {
    // the weight pass reads the top layer's dy after the caller may have reused it
    void *top = wlayer_bufs(st, wslot, d.n_layers - 1).at(P.w_dy);
    hipError_t e = hipMemcpyAsync(top, dy_in, (size_t)T * D * es, hipMemcpyDeviceToDevice, s);
    if (e != hipSuccess) return hip_fail(e, "saving dy for the weight pass");
    dy_op = top;
  }
  for (int l = d.n_layers - 1; l >= 0; --l) {
    const LayerBufs L = layer_bufs(st, slot, l);
    const LayerBufs WL = split ? wlayer_bufs(st, wslot, l) : LayerBufs{nullptr};
    const size_t lw = (size_t)l * pp.per_layer;
    const W w{static_cast<const char *>(pb->w) + lw * P.elem, split ? nullptr : pb->grad + lw,
              P.elem};
    const bool first = l == 0;
    const void *xin = first ? x0 : L.at(P.xin);
    const int x_dt = first ? dt : ty.res;
    // operand copy of the gradient handed to layer l - 1
    void *dy_next_op = first ? nullptr
                       : split ? wlayer_bufs(st, wslot, l - 1).at(P.w_dy)
                               : ws + P.s_dy16;
    void *dx = first ? dx_out
               : (split && !copies) ? dy_next_op
                                    : ws + ((d.n_layers - 1 - l) % 2 == 0 ? P.s_dy0 : P.s_dy1);
    void *dn = ws + P.s_dn, *dO = ws + P.s_do;
    void *da = split ? WL.at(P.w_da) : ws + P.s_da;
    void *dh = (split && !copies) ? WL.at(P.w_dh) : ws + P.s_dh;
    void *dh_op = !copies ? dh : split ? WL.at(P.w_dh) : ws + P.s_dh16;
    char *dqkv = split ? static_cast<char *>(WL.at(P.w_dqkv)) : ws + P.s_dqkv;
    lc_gemm_args a;
    if (d.n_experts > 0) {
      LC_TRY(moe_backward(st, w, L, dy_res, dy_dt, s, split ? &WL : nullptr));
    } else {
    // [dgate | dup] = SwiGLU'(dy W2)
    a = gemm_base(dt, LC_EPI_SWIGLU_BWD, T, F, D);
    a.A = dy_op; a.lda = D; a.a_kmajor = 1;
    a.B = w.wp(pp.w2); a.ldb = F; a.b_kmajor = 0;
    a.C = da; a.ldc = 2 * F; a.c_dtype = ty.op;
    a.aux0 = L.at(P.gate); a.aux1 = L.at(P.up); a.ld_aux = F; a.aux_dtype = ty.res;
    LC_TRY(gemm_launch(a, s));
    // G[W2] += dy^T act
    if (!split) {
      a = gemm_base(dt, gepi, D, F, T);
      a.A = dy_op; a.lda = D; a.a_kmajor = 0;
      a.B = L.at(P.act); a.ldb = F; a.b_kmajor = 0;
      a.C = w.gp(pp.w2); a.ldc = F;
      LC_TRY(wgrad_launch(st, a, s));
    }
    // dn2 = [dgate | dup] [W1; W3]
    a = gemm_base(dt, LC_EPI_STORE, T, D, 2 * F);
    a.A = da; a.lda = 2 * F; a.a_kmajor = 1;
    a.B = w.wp(pp.w1); a.ldb = D; a.b_kmajor = 0;
    a.C = dn; a.ldc = D; a.c_dtype = ty.res;
    LC_TRY(gemm_launch(a, s));
    // G[W1; W3] += [dgate | dup]^T n2
    if (!split) {
      a = gemm_base(dt, gepi, 2 * F, D, T);
      a.A = da; a.lda = 2 * F; a.a_kmajor = 0;
      a.B = L.at(P.n2); a.ldb = D; a.b_kmajor = 0;
      a.C = w.gp(pp.w1); a.ldc = D;
      LC_TRY(wgrad_launch(st, a, s));
    }
    }
    // dh = dy + RMSNorm2'(dn2); G[g2] += ... (or its partial sums)
    lc_norm_args nb = norm_base(T, D, d.rms_eps);
    nb.dn = dn; nb.dn_dtype = ty.res;
    nb.x = L.at(P.h); nb.x_dtype = ty.res;
    nb.rstd = static_cast<float *>(L.at(P.rstd2));
    nb.g = w.wp(pp.g2); nb.w_dtype = dt;
    nb.dres = dy_res; nb.dres_dtype = dy_dt;
    nb.dx = dh; nb.out_dtype = ty.res;
    nb.dx_copy = copies ? dh_op : nullptr;
    if (split) {
      nb.scratch = WL.at(P.w_p2); nb.scratch_bytes = rmsnorm_scratch_size(T, D);
      LC_TRY(rmsnorm_bwd_partials_launch(nb, s));
    } else {
      nb.scratch = ws + P.s_norm; nb.scratch_bytes = P.s_norm_bytes;
      LC_TRY(norm_bwd_full(st, nb, w.gp(pp.g2), s));
    }
    // do = dh Wo
    a = gemm_base(dt, LC_EPI_STORE, T, D, D);
    a.A = dh_op; a.lda = D; a.a_kmajor = 1;
    a.B = w.wp(pp.wo); a.ldb = D; a.b_kmajor = 0;
    a.C = dO; a.ldc = D; a.c_dtype = ty.op;
    LC_TRY(gemm_launch(a, s));
    // G[Wo] += dh^T o
    if (!split) {
      a = gemm_base(dt, gepi, D, D, T);
      a.A = dh_op; a.lda = D; a.a_kmajor = 0;
      a.B = L.at(P.o); a.ldb = D; a.b_kmajor = 0;
      a.C = w.gp(pp.wo); a.ldc = D;
      LC_TRY(wgrad_launch(st, a, s));
    }
    // dq, dk, dv (dq, dk rotated back)
    char *qkv = static_cast<char *>(L.at(P.qkv));
    lc_attn_args at;
    memset(&at, 0, sizeof at);
    at.dtype = ty.att; at.o_dtype = ty.op;
    at.B = d.micro_batch; at.S = d.seq_len; at.H = d.n_heads; at.hd = d.head_dim;
    at.Hkv = kv_heads(d);
    at.q = qkv; at.k = qkv + D * ea; at.v = qkv + (D + Dkv) * ea; at.ld_qkv = QC;
    at.o = L.at(P.o); at.ld_o = D; at.lse = static_cast<float *>(L.at(P.lse));
    at.dout = dO;
    at.dq = dqkv; at.dk = dqkv + D * es; at.dv = dqkv + (D + Dkv) * es; at.ld_dqkv = QC;
    at.rope_cos = rc; at.rope_sin = rs;
    at.scratch = ws + P.s_attn; at.scratch_bytes = P.s_attn_bytes;
    if (P.qkvb) {
      at.qkv_bf16 = L.at(P.qkvb); at.ld_qkv_bf16 = QC;
    }
    LC_TRY(attn_bwd_launch(at, s));
    // dq, dk through the per-head norms (in place); G[qn], G[kn] += ...
    if (d.qk_norm) {
      lc_qknorm_args qa = qknorm_base(st, w, L);
      qa.dqk = dqkv; qa.ld_d = QC;
      if (split) {
        qa.scratch = WL.at(P.w_pqk); qa.scratch_bytes = qknorm_scratch_size(T, d.head_dim);
        LC_TRY(qknorm_bwd_partials_launch(qa, s));
      } else {
        qa.scratch = ws + P.s_qkn; qa.scratch_bytes = P.s_qkn_bytes;
        LC_TRY(qknorm_bwd_partials_launch(qa, s));
        LC_TRY(qknorm_dg_final_launch(static_cast<const float *>(qa.scratch), w.gp(pp.qn),
                                      w.gp(pp.kn), T, d.head_dim, st->grad_store, s));
      }
    }
    // dn1 = [dq|dk|dv] [Wq;Wk;Wv]
    a = gemm_base(dt, LC_EPI_STORE, T, D, QC);
    a.A = dqkv; a.lda = QC; a.a_kmajor = 1;
    a.B = w.wp(pp.wq); a.ldb = D; a.b_kmajor = 0;
    a.C = dn; a.ldc = D; a.c_dtype = ty.res;
    LC_TRY(gemm_launch(a, s));
    // G[Wq;Wk;Wv] += [dq|dk|dv]^T n1
    if (!split) {
      a = gemm_base(dt, gepi, QC, D, T);
      a.A = dqkv; a.lda = QC; a.a_kmajor = 0;
      a.B = L.at(P.n1); a.ldb = D; a.b_kmajor = 0;
      a.C = w.gp(pp.wq); a.ldc = D;
      LC_TRY(wgrad_launch(st, a, s));
    }
    // dx = dh + RMSNorm1'(dn1); G[g1] += ... (or its partial sums)
    nb.dn = dn; nb.dn_dtype = ty.res;
    nb.x = xin; nb.x_dtype = x_dt;
    nb.rstd = static_cast<float *>(L.at(P.rstd1));
    nb.g = w.wp(pp.g1);
    nb.dres = dh; nb.dres_dtype = ty.res;
    nb.dx = dx; nb.out_dtype = first ? dt : ty.res;
    nb.dx_copy = (copies && !first) ? dy_next_op : nullptr;
    if (split) {
      nb.scratch = WL.at(P.w_p1); nb.scratch_bytes = rmsnorm_scratch_size(T, D);
      LC_TRY(rmsnorm_bwd_partials_launch(nb, s));
    } else {
      LC_TRY(norm_bwd_full(st, nb, w.gp(pp.g1), s));
    }
    dy_res = dx;
    dy_op = copies ? dy_next_op : dx;
    dy_dt = ty.res;
  }
  return LC_OK;
}

// The backward for the weights: every weight-gradient product and gain sum of
// Chunk B, from the operands the backward for the inputs left in weight-pass
// slot wslot and the activations in stash slot `slot`.
static lc_status weight_layers(lc_stage *st, const lc_param_bufs *pb, int slot, int wslot,
                               hipStream_t s) {
  const lc_stage_desc &d = st->d;
  const StagePlan &P = st->plan;
  const ParamPlan &pp = st->pp;
  const int dt = d.compute_dtype;
  const int64_t T = P.T, D = d.d_model, F = d.d_ff, QC = P.qkv_cols;
  const int gepi = st->grad_store ? LC_EPI_STORE_F32 : LC_EPI_ACCUM_F32;
  for (int l = d.n_layers - 1; l >= 0; --l) {
    const LayerBufs L = layer_bufs(st, slot, l);
    const LayerBufs WL = wlayer_bufs(st, wslot, l);
    const size_t lw = (size_t)l * pp.per_layer;
    const W w{static_cast<const char *>(pb->w) + lw * P.elem, pb->grad + lw, P.elem};
    lc_gemm_args a;
    if (d.n_experts > 0) {
      LC_TRY(moe_weight(st, w, L, WL, s));
    } else {
    // G[W2] += dy^T act
    a = gemm_base(dt, gepi, D, F, T);
    a.A = WL.at(P.w_dy); a.lda = D; a.a_kmajor = 0;
    a.B = L.at(P.act); a.ldb = F; a.b_kmajor = 0;
    a.C = w.gp(pp.w2); a.ldc = F;
    LC_TRY(wgrad_launch(st, a, s));
    // G[W1; W3] += [dgate | dup]^T n2
    a = gemm_base(dt, gepi, 2 * F, D, T);
    a.A = WL.at(P.w_da); a.lda = 2 * F; a.a_kmajor = 0;
    a.B = L.at(P.n2); a.ldb = D; a.b_kmajor = 0;
    a.C = w.gp(pp.w1); a.ldc = D;
    LC_TRY(wgrad_launch(st, a, s));
    }
    LC_TRY(rmsnorm_dg_final_launch(static_cast<const float *>(WL.at(P.w_p2)), w.gp(pp.g2), T, D, s,
                                   st->grad_store));
    // G[Wo] += dh^T o
    a = gemm_base(dt, gepi, D, D, T);
    a.A = WL.at(P.w_dh); a.lda = D; a.a_kmajor = 0;
    a.B = L.at(P.o); a.ldb = D; a.b_kmajor = 0;
    a.C = w.gp(pp.wo); a.ldc = D;
    LC_TRY(wgrad_launch(st, a, s));
    // G[Wq;Wk;Wv] += [dq|dk|dv]^T n1
    a = gemm_base(dt, gepi, QC, D, T);
    a.A = WL.at(P.w_dqkv); a.lda = QC; a.a_kmajor = 0;
    a.B = L.at(P.n1); a.ldb = D; a.b_kmajor = 0;
    a.C = w.gp(pp.wq); a.ldc = D;
    LC_TRY(wgrad_launch(st, a, s));
    LC_TRY(rmsnorm_dg_final_launch(static_cast<const float *>(WL.at(P.w_p1)), w.gp(pp.g1), T, D, s,
                                   st->grad_store));
    if (d.qk_norm)
      LC_TRY(qknorm_dg_final_launch(static_cast<const float *>(WL.at(P.w_pqk)), w.gp(pp.qn),
                                    w.gp(pp.kn), T, d.head_dim, st->grad_store, s));
  }
  return LC_OK;
}

static lc_status check_params(const lc_stage *st, const lc_param_bufs *pb, bool need_grad) {
  if (!st) return fail(LC_ERR_INVALID_ARG, "null stage");
  if (!pb || !pb->w) return fail(LC_ERR_INVALID_ARG, "null parameter buffers");
  if (!aligned16(pb->w)) return fail(LC_ERR_INVALID_ARG, "weights must be 16-byte aligned");
  if (need_grad && (!pb->grad || !aligned16(pb->grad)))
    return fail(LC_ERR_INVALID_ARG, "gradient buffer must be non-null and 16-byte aligned");
  return LC_OK;
}

static lc_status check_mb(const lc_microbatch_desc *mb, bool fwd) {
  if (!mb) return fail(LC_ERR_INVALID_ARG, "null microbatch descriptor");
  if (fwd) {
    if (!mb->x || !mb->y || !aligned16(mb->x) || !aligned16(mb->y))
      return fail(LC_ERR_INVALID_ARG, "microbatch %d: x and y must be non-null and aligned", mb->mb);
  } else {
    if (!mb->dy || !mb->dx || !aligned16(mb->dy) || !aligned16(mb->dx))
      return fail(LC_ERR_INVALID_ARG, "microbatch %d: dy and dx must be non-null and aligned",
                  mb->mb);
  }
  return LC_OK;
}

static int find_slot(const lc_stage *st, int32_t mb) {
  for (int i = 0; i < st->slots; ++i)
    if (st->owner[i] == mb) return i;
  return -1;
}

static int find_wslot(const lc_stage *st, int32_t mb) {
  for (int i = 0; i < (int)st->wowner.size(); ++i)
    if (st->wowner[i] == mb) return i;
  return -1;
}

static lc_status do_forward(lc_stage *st, const lc_param_bufs *pb, const lc_microbatch_desc *mb,
                            hipStream_t s) {
  int slot = find_slot(st, -1);
  st->owner[slot] = mb->mb;
  st->xin0[slot] = mb->x;
  return forward_layers(st, pb, mb->x, mb->y, slot, s);
}

static void release(lc_stage *st, int slot) {
  st->owner[slot] = -1;
  st->xin0[slot] = nullptr;
}

static lc_status do_backward(lc_stage *st, const lc_param_bufs *pb, const lc_microbatch_desc *mb,
                             hipStream_t s) {
  const int slot = find_slot(st, mb->mb);
  lc_status r = backward_layers(st, pb, st->xin0[slot], mb->dy, mb->dx, slot, -1, s);
  release(st, slot);
  return r;
}

static lc_status do_backward_input(lc_stage *st, const lc_param_bufs *pb,
                                   const lc_microbatch_desc *mb, hipStream_t s) {
  const int slot = find_slot(st, mb->mb), wslot = find_wslot(st, -1);
  st->wowner[wslot] = mb->mb;
  return backward_layers(st, pb, st->xin0[slot], mb->dy, mb->dx, slot, wslot, s);
}

static lc_status do_backward_weight(lc_stage *st, const lc_param_bufs *pb, int32_t mb,
                                    hipStream_t s) {
  const int slot = find_slot(st, mb), wslot = find_wslot(st, mb);
  lc_status r = weight_layers(st, pb, slot, wslot, s);
  st->wowner[wslot] = -1;
  release(st, slot);
  return r;
}

}  // namespace lc

using namespace lc;

extern "C" {

lc_status lc_stage_create_split(const lc_stage_desc *desc, void *workspace, size_t ws_bytes,
                                int32_t max_in_flight, int32_t max_w_pending, void *stream,
                                lc_stage **out) {
  if (!out) return fail(LC_ERR_INVALID_ARG, "null output handle");
  *out = nullptr;
  StagePlan plan;
  LC_TRY(validate_desc(desc));
  LC_TRY(stage_plan(*desc, max_in_flight, max_w_pending, &plan));
  if (!workspace) return fail(LC_ERR_INVALID_ARG, "null workspace");
  if (reinterpret_cast<uintptr_t>(workspace) & 255u)
    return fail(LC_ERR_INVALID_ARG, "workspace must be 256-byte aligned");
  if (ws_bytes < plan.total)
    return fail(LC_ERR_WORKSPACE, "workspace of %zu bytes < %zu needed", ws_bytes, plan.total);
  lc_stage *st = new (std::nothrow) lc_stage();
  if (!st) return fail(LC_ERR_INVALID_ARG, "out of host memory");
  st->d = *desc;
  st->plan = plan;
  st->pp = param_plan(*desc);
  st->ws = static_cast<char *>(workspace);
  st->slots = max_in_flight;
  st->owner.assign((size_t)max_in_flight, -1);
  st->xin0.assign((size_t)max_in_flight, nullptr);
  st->wowner.assign((size_t)max_w_pending, -1);
  // RoPE angles p * base^(-2i/hd) in double, tables rounded once to float
  const int half = desc->head_dim / 2, S = desc->seq_len;
  st->rope_host.resize((size_t)2 * S * half);
  for (int pos = 0; pos < S; ++pos)
    for (int i = 0; i < half; ++i) {
      const double theta = pow((double)desc->rope_base, -2.0 * i / (double)desc->head_dim);
      const double ang = (double)pos * theta;
      st->rope_host[(size_t)pos * half + i] = (float)cos(ang);
      st->rope_host[(size_t)S * half + (size_t)pos * half + i] = (float)sin(ang);
    }
  const size_t tb = (size_t)S * half * sizeof(float);
  hipStream_t s = static_cast<hipStream_t>(stream);
  hipError_t e = hipMemcpyAsync(st->ws + plan.rope_cos, st->rope_host.data(), tb,
                                hipMemcpyHostToDevice, s);
  if (e == hipSuccess)
    e = hipMemcpyAsync(st->ws + plan.rope_sin, st->rope_host.data() + (size_t)S * half, tb,
                       hipMemcpyHostToDevice, s);
  if (e != hipSuccess) {
    delete st;
    return hip_fail(e, "uploading the RoPE table");
  }
  *out = st;
  return LC_OK;
}

lc_status lc_stage_create(const lc_stage_desc *desc, void *workspace, size_t ws_bytes,
                          int32_t max_in_flight, void *stream, lc_stage **out) {
  return lc_stage_create_split(desc, workspace, ws_bytes, max_in_flight, 0, stream, out);
}

lc_status lc_stage_destroy(lc_stage *stage) {
  if (stage) {
    for (hipEvent_t e : stage->events) hipEventDestroy(e);
    for (hipEvent_t e : stage->tev) hipEventDestroy(e);
  }
  delete stage;
  return LC_OK;
}

lc_status chunk_forward(lc_stage *stage, const lc_param_bufs *params, const lc_microbatch_desc *mb,
                        void *stream) {
  LC_TRY(check_params(stage, params, false));
  LC_TRY(check_mb(mb, true));
  if (find_slot(stage, mb->mb) >= 0)
    return fail(LC_ERR_STATE, "microbatch %d is already stashed", mb->mb);
  if (mb->mb < 0) return fail(LC_ERR_INVALID_ARG, "negative microbatch index");
  if (find_slot(stage, -1) < 0)
    return fail(LC_ERR_STASH_FULL, "all %d stash slots are in use", stage->slots);
  return do_forward(stage, params, mb, static_cast<hipStream_t>(stream));
}

lc_status chunk_backward(lc_stage *stage, const lc_param_bufs *params, const lc_microbatch_desc *mb,
                         void *stream) {
  LC_TRY(check_params(stage, params, true));
  LC_TRY(check_mb(mb, false));
  if (mb->mb < 0 || find_slot(stage, mb->mb) < 0)
    return fail(LC_ERR_STATE, "microbatch %d has no stashed forward", mb->mb);
  if (find_wslot(stage, mb->mb) >= 0)
    return fail(LC_ERR_STATE, "microbatch %d already ran its backward for the inputs", mb->mb);
  return do_backward(stage, params, mb, static_cast<hipStream_t>(stream));
}

lc_status chunk_backward_input(lc_stage *stage, const lc_param_bufs *params,
                               const lc_microbatch_desc *mb, void *stream) {
  LC_TRY(check_params(stage, params, false));
  LC_TRY(check_mb(mb, false));
  if (mb->mb < 0 || find_slot(stage, mb->mb) < 0)
    return fail(LC_ERR_STATE, "microbatch %d has no stashed forward", mb->mb);
  if (find_wslot(stage, mb->mb) >= 0)
    return fail(LC_ERR_STATE, "microbatch %d already ran its backward for the inputs", mb->mb);
  if (find_wslot(stage, -1) < 0)
    return fail(LC_ERR_STASH_FULL, "all %d weight-pass slots are in use",
                (int)stage->wowner.size());
  return do_backward_input(stage, params, mb, static_cast<hipStream_t>(stream));
}

lc_status chunk_backward_weight(lc_stage *stage, const lc_param_bufs *params,
                                const lc_microbatch_desc *mb, void *stream) {
  LC_TRY(check_params(stage, params, true));
  if (!mb) return fail(LC_ERR_INVALID_ARG, "null microbatch descriptor");
  if (mb->mb < 0 || find_wslot(stage, mb->mb) < 0)
    return fail(LC_ERR_STATE, "microbatch %d has no pending weight pass", mb->mb);
  return do_backward_weight(stage, params, mb->mb, static_cast<hipStream_t>(stream));
}

lc_status lc_stage_timer_enable(lc_stage *stage, int32_t max_launches) {
  if (!stage || max_launches < 0 || max_launches > (1 << 20))
    return fail(LC_ERR_INVALID_ARG, "null stage or launch capacity outside [0, 2^20]");
  for (hipEvent_t e : stage->tev) hipEventDestroy(e);
  stage->tev.clear();
  stage->tflop.clear();
  stage->tn = 0;
  for (int64_t i = 0; i < 2 * (int64_t)max_launches; ++i) {
    hipEvent_t e;
    const hipError_t r = hipEventCreate(&e);
    if (r != hipSuccess) {
      for (hipEvent_t x : stage->tev) hipEventDestroy(x);
      stage->tev.clear();
      return hip_fail(r, "creating timing events");
    }
    stage->tev.push_back(e);
  }
  stage->tflop.assign(max_launches, 0.0);
  return LC_OK;
}

lc_status lc_stage_timer_read(lc_stage *stage, float *ms, double *flop, int32_t cap, int32_t *n) {
  if (!stage || !n || cap < 0 || (cap > 0 && (!ms || !flop)))
    return fail(LC_ERR_INVALID_ARG, "null stage, count or output arrays, or negative capacity");
  const int32_t k = stage->tn < cap ? stage->tn : cap;
  for (int32_t i = 0; i < k; ++i) {
    hipError_t e = hipEventSynchronize(stage->tev[2 * i + 1]);
    if (e == hipSuccess) e = hipEventElapsedTime(&ms[i], stage->tev[2 * i], stage->tev[2 * i + 1]);
    if (e != hipSuccess) return hip_fail(e, "reading a timing event");
    flop[i] = stage->tflop[i];
  }
  *n = stage->tn;
  stage->tn = 0;
  return LC_OK;
}

lc_status lc_stage_moe_routing(lc_stage *stage, int32_t mb, int32_t layer, int32_t *sel_out,
                               void *stream) {
  if (!stage || !sel_out) return fail(LC_ERR_INVALID_ARG, "null stage or output");
  if (stage->d.n_experts <= 0) return fail(LC_ERR_INVALID_ARG, "dense stage has no routing");
  if (layer < 0 || layer >= stage->d.n_layers) return fail(LC_ERR_INVALID_ARG, "layer out of range");
  const int slot = mb < 0 ? -1 : find_slot(stage, mb);
  if (slot < 0) return fail(LC_ERR_STATE, "microbatch %d is not stashed", mb);
  const LayerBufs L = layer_bufs(stage, slot, layer);
  const size_t bytes = (size_t)stage->plan.T * 2 * sizeof(int32_t);
  hipError_t e = hipMemcpyAsync(sel_out, L.at(stage->plan.moe_sel), bytes, hipMemcpyDeviceToDevice,
                                static_cast<hipStream_t>(stream));
  return e == hipSuccess ? LC_OK : hip_fail(e, "copying the routing");
}

}  // extern "C"

namespace lc {
namespace {

// Last enqueue that touched a resource: stream index (0 = main, 1 = aux) and
// the event recorded after it (-1: nothing recorded in this call, i.e.
// ordered before the call on the main stream).
struct LastUse {
  int stream = 0;
  int ev = -1;
};

lc_status ensure_events(lc_stage *st, size_t n) {
  while (st->events.size() < n) {
    hipEvent_t e;
    hipError_t r = hipEventCreateWithFlags(&e, hipEventDisableTiming);
    if (r != hipSuccess) return hip_fail(r, "creating an event");
    st->events.push_back(e);
  }
  return LC_OK;
}

bool uses_scratch(int pass) { return pass == LC_PASS_B || pass == LC_PASS_BI; }
bool writes_grad(int pass) { return pass == LC_PASS_B || pass == LC_PASS_BW; }

// Number of later entries of the Order that depend on entry i (the later
// passes of the same microbatch): the dispatch priority within a pair.
int downstream(const std::vector<lc_order_entry> &flat, size_t i) {
  int n = 0;
  for (size_t j = i + 1; j < flat.size(); ++j) n += flat[j].mb == flat[i].mb;
  return n;
}

// ZeRO-3: the weight shards concatenated into the temporary full buffer.
lc_status gather_weights(const lc_stage *st, const lc_zero_bufs &z, hipStream_t s) {
  char *dst = static_cast<char *>(z.w_full);
  for (int i = 0; i < z.n_w_shards; ++i) {
    const size_t bytes = z.w_shard_lens[i] * st->plan.elem;
    if (bytes && z.w_shards[i] != dst) {
      hipError_t e = hipMemcpyAsync(dst, z.w_shards[i], bytes, hipMemcpyDeviceToDevice, s);
      if (e != hipSuccess) return hip_fail(e, "gathering the weight shards");
    }
    dst += bytes;
  }
  return LC_OK;
}

lc_status run_entries(lc_stage *st, const lc_param_bufs *pb_in, const lc_order &order,
                      const lc_microbatch_desc *mbs, hipStream_t s_main, hipStream_t s_aux,
                      const lc_zero_bufs *z = nullptr) {
  lc_param_bufs zb = *pb_in;
  if (z) {
    zb.grad = z->grad_full;
    if (z->level == 3) zb.w = z->w_full;
  }
  const lc_param_bufs *pb = &zb;
  std::vector<lc_order_entry> flat;
  LC_TRY(flatten_order(order, &flat));
  const bool two = s_aux != s_main;
  const hipStream_t strm[2] = {s_main, s_aux};
  std::vector<LastUse> mb_use((size_t)order.num_microbatches), slot_use((size_t)st->slots),
      wslot_use(st->wowner.size());
  LastUse scratch_use, grad_use;
  int nev = 0;
  if (two) {
    LC_TRY(ensure_events(st, flat.size() + 2));
    // aux starts after everything already enqueued on main (the RoPE upload,
    // the caller's zeroing of the gradient, ...)
    hipError_t r = hipEventRecord(st->events[(size_t)nev], s_main);
    if (r == hipSuccess) r = hipStreamWaitEvent(s_aux, st->events[(size_t)nev], 0);
    if (r != hipSuccess) return hip_fail(r, "joining the auxiliary stream");
    ++nev;
  }
  // flat keeps each pair's two entries adjacent; walk the original entries to
  // know which ones are paired
  size_t fi = 0;
  for (int32_t i = 0; i < order.n_entries; ++i) {
    const bool pair = (order.entries[i].pass & LC_ORDER_WITH_NEXT) != 0;
    size_t idx[2] = {fi, fi + 1};
    const int n = pair ? 2 : 1;
    int on[2] = {0, 0};
    if (pair) {
      // the backward that uses the working buffers (B, Bi) or, for {Bi, Bw},
      // the Bi stays on the main stream; the other entry goes to aux
      const int p0 = flat[fi].pass, p1 = flat[fi + 1].pass;
      const bool first_main = uses_scratch(p0) || (p0 != LC_PASS_F && p1 == LC_PASS_F);
      on[0] = first_main ? 0 : 1;
      on[1] = 1 - on[0];
      if (downstream(flat, fi + 1) > downstream(flat, fi)) {
        std::swap(idx[0], idx[1]);
        std::swap(on[0], on[1]);
      }
      ++i;
    }
    for (int k = 0; k < n; ++k) {
      const lc_order_entry e = flat[idx[k]];
      const int si = two ? on[k] : 0;
      const lc_microbatch_desc *mb = &mbs[e.mb];
      int slot = -1, wslot = -1;
      switch (e.pass) {
        case LC_PASS_F: slot = find_slot(st, -1); break;
        case LC_PASS_BI: slot = find_slot(st, e.mb); wslot = find_wslot(st, -1); break;
        case LC_PASS_BW: slot = find_slot(st, e.mb); wslot = find_wslot(st, e.mb); break;
        default: slot = find_slot(st, e.mb); break;
      }
      if (slot < 0 || (e.pass == LC_PASS_BI || e.pass == LC_PASS_BW) == (wslot < 0))
        return fail(LC_ERR_STATE, "internal: no slot for entry of microbatch %d", e.mb);
      if (two) {
        LastUse *deps[5] = {&mb_use[(size_t)e.mb], &slot_use[(size_t)slot],
                            wslot >= 0 ? &wslot_use[(size_t)wslot] : nullptr,
                            uses_scratch(e.pass) ? &scratch_use : nullptr,
                            writes_grad(e.pass) ? &grad_use : nullptr};
        int waited[5], nw = 0;
        for (LastUse *d : deps) {
          if (!d || d->ev < 0 || d->stream == si) continue;
          bool dup = false;
          for (int w = 0; w < nw; ++w) dup |= waited[w] == d->ev;
          if (dup) continue;
          hipError_t r = hipStreamWaitEvent(strm[si], st->events[(size_t)d->ev], 0);
          if (r != hipSuccess) return hip_fail(r, "waiting on the other stream");
          waited[nw++] = d->ev;
        }
      }
      if (z && z->level == 3) LC_TRY(gather_weights(st, *z, strm[si]));
      // a dense stage's backward writes every gradient element once, so it
      // stores into the temporary gradient; a mixture-of-experts stage adds
      // into a zeroed one (an expert may receive no rows)
      if (z && writes_grad(e.pass) && st->d.n_experts > 0)
        LC_TRY(zero_fill_launch(z->grad_full, st->pp.total, strm[si]));
      st->grad_store = z && st->d.n_experts == 0;
      lc_status r;
      switch (e.pass) {
        case LC_PASS_F: r = do_forward(st, pb, mb, strm[si]); break;
        case LC_PASS_B: r = do_backward(st, pb, mb, strm[si]); break;
        case LC_PASS_BI: r = do_backward_input(st, pb, mb, strm[si]); break;
        default: r = do_backward_weight(st, pb, e.mb, strm[si]); break;
      }
      st->grad_store = false;
      if (r != LC_OK) return r;
      // this rank's share of the reduce-scatter
      if (z && writes_grad(e.pass))
        LC_TRY(accumulate_launch(z->grad_shard, z->grad_full + z->shard_offset, LC_FP32,
                                 z->shard_len, strm[si]));
      if (two) {
        hipError_t er = hipEventRecord(st->events[(size_t)nev], strm[si]);
        if (er != hipSuccess) return hip_fail(er, "recording an event");
        const LastUse u{si, nev++};
        mb_use[(size_t)e.mb] = u;
        slot_use[(size_t)slot] = u;
        if (wslot >= 0) wslot_use[(size_t)wslot] = u;
        if (uses_scratch(e.pass)) scratch_use = u;
        if (writes_grad(e.pass)) grad_use = u;
      }
    }
    fi += (size_t)n;
  }
  if (two) {
    // main continues after everything enqueued on aux
    hipError_t r = hipEventRecord(st->events[(size_t)nev], s_aux);
    if (r == hipSuccess) r = hipStreamWaitEvent(s_main, st->events[(size_t)nev], 0);
    if (r != hipSuccess) return hip_fail(r, "joining the main stream");
  }
  return LC_OK;
}

lc_status check_run(lc_stage *stage, const lc_param_bufs *params, const lc_order *order,
                    const lc_microbatch_desc *mbs) {
  LC_TRY(check_params(stage, params, true));
  LC_TRY(lc_order_validate_split(order, stage->slots, (int32_t)stage->wowner.size(), nullptr,
                                 nullptr));
  if (!mbs) return fail(LC_ERR_INVALID_ARG, "null microbatch array");
  for (int i = 0; i < order->num_microbatches; ++i) {
    if (mbs[i].mb != i) return fail(LC_ERR_INVALID_ARG, "mbs[%d].mb = %d, expected %d", i, mbs[i].mb, i);
    LC_TRY(check_mb(&mbs[i], true));
    LC_TRY(check_mb(&mbs[i], false));
  }
  for (int i = 0; i < stage->slots; ++i)
    if (stage->owner[i] != -1)
      return fail(LC_ERR_STATE, "lc_run_order needs an empty stash (microbatch %d is stashed)",
                  stage->owner[i]);
  for (size_t i = 0; i < stage->wowner.size(); ++i)
    if (stage->wowner[i] != -1)
      return fail(LC_ERR_STATE, "lc_run_order needs no pending weight pass (microbatch %d)",
                  stage->wowner[i]);
  return LC_OK;
}

// The lc_run_order* calls start from an empty stash (check_run); if an entry
// fails after others were enqueued, the stash returns to that empty state so
// the stage stays usable (the outputs of the failed run are undefined).
lc_status run_or_reset(lc_stage *st, const lc_param_bufs *pb, const lc_order &order,
                       const lc_microbatch_desc *mbs, hipStream_t s_main, hipStream_t s_aux,
                       const lc_zero_bufs *z = nullptr) {
  const lc_status r = run_entries(st, pb, order, mbs, s_main, s_aux, z);
  if (r != LC_OK) {
    std::fill(st->owner.begin(), st->owner.end(), -1);
    std::fill(st->wowner.begin(), st->wowner.end(), -1);
  }
  return r;
}

bool ranges_overlap(const void *a, size_t a_bytes, const void *b, size_t b_bytes) {
  const char *x = static_cast<const char *>(a), *y = static_cast<const char *>(b);
  return a_bytes && b_bytes && x < y + b_bytes && y < x + a_bytes;
}

}  // namespace
}  // namespace lc

extern "C" {

lc_status lc_run_order(lc_stage *stage, const lc_param_bufs *params, const lc_order *order,
                       const lc_microbatch_desc *mbs, void *stream) {
  LC_TRY(check_run(stage, params, order, mbs));
  hipStream_t s = static_cast<hipStream_t>(stream);
  return run_or_reset(stage, params, *order, mbs, s, s);
}

lc_status lc_run_order_zero(lc_stage *stage, const lc_param_bufs *params, const lc_zero_bufs *zero,
                            const lc_order *order, const lc_microbatch_desc *mbs, void *stream) {
  if (!zero) return fail(LC_ERR_INVALID_ARG, "null ZeRO buffers");
  if (!params) return fail(LC_ERR_INVALID_ARG, "null parameter buffers");
  const lc_zero_bufs &z = *zero;
  if (z.level != 2 && z.level != 3) return fail(LC_ERR_INVALID_ARG, "ZeRO level must be 2 or 3");
  if (!stage) return fail(LC_ERR_INVALID_ARG, "null stage");
  const size_t n = stage->pp.total;
  if (!z.grad_shard || !z.grad_full || !aligned16(z.grad_shard) || !aligned16(z.grad_full))
    return fail(LC_ERR_INVALID_ARG, "ZeRO gradient buffers must be non-null and 16-byte aligned");
  if (z.shard_offset % 4 || z.shard_offset > n || z.shard_len > n - z.shard_offset)
    return fail(LC_ERR_INVALID_ARG, "gradient shard [%zu, +%zu) is not a 4-aligned slice of %zu",
                z.shard_offset, z.shard_len, n);
  if (ranges_overlap(z.grad_shard, z.shard_len * 4, z.grad_full, n * 4))
    return fail(LC_ERR_INVALID_ARG, "the gradient shard overlaps the temporary full gradient");
  lc_param_bufs pb = *params;
  pb.grad = z.grad_full;
  if (z.level == 3) {
    if (z.n_w_shards < 1 || z.n_w_shards > 1024 || !z.w_shards || !z.w_shard_lens)
      return fail(LC_ERR_INVALID_ARG, "ZeRO-3 needs 1..1024 weight shards");
    if (!z.w_full || !aligned16(z.w_full))
      return fail(LC_ERR_INVALID_ARG, "ZeRO-3 temporary weights must be non-null and 16-byte aligned");
    const size_t esz = stage->plan.elem;
    size_t tot = 0;
    for (int i = 0; i < z.n_w_shards; ++i) {
      if (!z.w_shards[i] && z.w_shard_lens[i])
        return fail(LC_ERR_INVALID_ARG, "weight shard %d is null", i);
      if (z.w_shard_lens[i] > n - std::min(tot, n))
        return fail(LC_ERR_INVALID_ARG, "weight shards hold more than the bucket's %zu elements", n);
      // a shard may already sit at its own place in the temporary buffer (an
      // in-place gather: its copy is skipped); any other overlap would let
      // one shard's copy overwrite another before it is read
      const char *own = static_cast<const char *>(z.w_full) + tot * esz;
      if (z.w_shards[i] != own &&
          ranges_overlap(z.w_shards[i], z.w_shard_lens[i] * esz, z.w_full, n * esz))
        return fail(LC_ERR_INVALID_ARG, "weight shard %d overlaps the temporary full weights "
                    "away from its own place", i);
      tot += z.w_shard_lens[i];
    }
    if (tot != n)
      return fail(LC_ERR_INVALID_ARG, "weight shards hold %zu elements, the bucket %zu", tot, n);
    pb.w = z.w_full;
  }
  LC_TRY(check_run(stage, &pb, order, mbs));
  hipStream_t s = static_cast<hipStream_t>(stream);
  return run_or_reset(stage, params, *order, mbs, s, s, zero);
}

lc_status lc_run_order_overlap(lc_stage *stage, const lc_param_bufs *params,
                               const lc_order *order, const lc_microbatch_desc *mbs,
                               void *stream, void *aux_stream) {
  LC_TRY(check_run(stage, params, order, mbs));
  return run_or_reset(stage, params, *order, mbs, static_cast<hipStream_t>(stream),
                      static_cast<hipStream_t>(aux_stream));
}

}  // extern "C"
