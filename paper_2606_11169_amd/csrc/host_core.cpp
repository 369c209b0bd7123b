// Host-only core of libchunk (see host_core.hpp). Built with the host C++
// compiler; makes no HIP call.
#include "host_core.hpp"

#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <vector>

namespace lc {

static thread_local char g_err[512] = "";

lc_status fail(lc_status st, const char *fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof g_err, fmt, ap);
  va_end(ap);
  return st;
}

static inline size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

lc_status validate_desc(const lc_stage_desc *d) {
  if (!d) return fail(LC_ERR_INVALID_ARG, "null stage descriptor");
  if (d->n_layers <= 0 || d->d_model <= 0 || d->n_heads <= 0 || d->head_dim <= 0 ||
      d->seq_len <= 0 || d->micro_batch <= 0)
    return fail(LC_ERR_INVALID_ARG, "stage dimensions must be positive");
  if (d->n_kv_heads < 0 || (d->n_kv_heads > 0 && d->n_heads % d->n_kv_heads != 0))
    return fail(LC_ERR_INVALID_ARG, "n_kv_heads (%d) must be 0 or divide n_heads (%d)",
                d->n_kv_heads, d->n_heads);
  if (d->qk_norm != 0 && d->qk_norm != 1) return fail(LC_ERR_INVALID_ARG, "qk_norm must be 0 or 1");
  if (d->qk_norm && (d->head_dim < 16 || d->head_dim > 128 || (d->head_dim & (d->head_dim - 1))))
    return fail(LC_ERR_UNSUPPORTED, "the q/k norm kernels need head_dim in {16, 32, 64, 128}");
  if ((int64_t)d->n_heads * d->head_dim != d->d_model)
    return fail(LC_ERR_INVALID_ARG, "d_model (%d) != n_heads (%d) * head_dim (%d)", d->d_model,
                d->n_heads, d->head_dim);
  if (d->head_dim % 2 != 0) return fail(LC_ERR_INVALID_ARG, "head_dim must be even");
  if (d->causal != 1) return fail(LC_ERR_UNSUPPORTED, "only causal attention is implemented");
  if (!(d->rms_eps >= 0.0f) || !(d->rope_base > 0.0f))
    return fail(LC_ERR_INVALID_ARG, "rms_eps must be >= 0 and rope_base > 0");
  if (d->compute_dtype != LC_FP32 && d->compute_dtype != LC_BF16)
    return fail(LC_ERR_INVALID_ARG, "compute_dtype must be LC_FP32 or LC_BF16");
  if (d->n_experts < 0) return fail(LC_ERR_INVALID_ARG, "n_experts must be >= 0");
  if (d->n_experts == 0) {
    if (d->d_ff <= 0) return fail(LC_ERR_INVALID_ARG, "d_ff must be positive");
  } else {
    if (d->top_k != 2) return fail(LC_ERR_UNSUPPORTED, "MoE stages route to top_k == 2 experts");
    if (d->n_experts < 2) return fail(LC_ERR_INVALID_ARG, "MoE needs at least 2 experts");
    if (d->d_ff_expert <= 0) return fail(LC_ERR_INVALID_ARG, "d_ff_expert must be positive");
    if (d->compute_dtype != LC_BF16)
      return fail(LC_ERR_UNSUPPORTED, "MoE stages need compute_dtype LC_BF16 (grouped matrix-core products)");
  }
  // limits of the kernels
  if (d->compute_dtype == LC_BF16) {
    if (d->head_dim != 128)
      return fail(LC_ERR_UNSUPPORTED, "bf16 attention kernels need head_dim == 128");
    if (d->d_model % 64 != 0) return fail(LC_ERR_UNSUPPORTED, "bf16 needs d_model %% 64 == 0");
    int64_t f = d->n_experts ? d->d_ff_expert : d->d_ff;
    if (f % 64 != 0) return fail(LC_ERR_UNSUPPORTED, "bf16 needs the FFN width %% 64 == 0");
    if (d->seq_len % 128 != 0) return fail(LC_ERR_UNSUPPORTED, "bf16 needs seq_len %% 128 == 0");
  } else {
    if (d->head_dim > 128) return fail(LC_ERR_UNSUPPORTED, "fp32 attention needs head_dim <= 128");
    if (d->d_model % 4 != 0) return fail(LC_ERR_UNSUPPORTED, "fp32 needs d_model %% 4 == 0");
  }
  if (d->n_experts > 64) return fail(LC_ERR_UNSUPPORTED, "at most 64 experts");
  return LC_OK;
}

ParamPlan param_plan(const lc_stage_desc &d) {
  ParamPlan p{};
  const size_t D = (size_t)d.d_model;
  size_t off = 0;
  const size_t Dkv = (size_t)kv_heads(d) * (size_t)d.head_dim;
  p.wq = off; off += D * D;
  p.wk = off; off += Dkv * D;
  p.wv = off; off += Dkv * D;
  p.wo = off; off += D * D;
  p.g1 = off; off += D;
  if (d.qk_norm) {
    p.qn = off; off += (size_t)d.head_dim;
    p.kn = off; off += (size_t)d.head_dim;
  }
  if (d.n_experts == 0) {
    const size_t F = (size_t)d.d_ff;
    p.w1 = off; off += F * D;
    p.w3 = off; off += F * D;
    p.w2 = off; off += D * F;
  } else {
    const size_t FE = (size_t)d.d_ff_expert, E = (size_t)d.n_experts;
    p.wr = off; off += E * D;
    p.expert0 = off;
    p.expert_stride = 3 * FE * D;
    off += E * p.expert_stride;
  }
  p.g2 = off; off += D;
  p.per_layer = off;
  p.total = off * (size_t)d.n_layers;
  return p;
}

StageTypes stage_types(const lc_stage_desc &d) {
  StageTypes t;
  if (d.compute_dtype == LC_BF16) {
    t.op = LC_BF16;
    t.att = LC_FP16;
    t.res = LC_FP32;
  } else {
    t.op = t.att = t.res = LC_FP32;
  }
  return t;
}

static size_t bytes_of(int dt) { return dt == LC_FP32 ? 4 : 2; }

lc_status stage_plan(const lc_stage_desc &d, int32_t max_in_flight, int32_t max_w_pending,
                     StagePlan *out) {
  lc_status st = validate_desc(&d);
  if (st != LC_OK) return st;
  if (max_in_flight <= 0) return fail(LC_ERR_INVALID_ARG, "max_in_flight must be positive");
  if (max_w_pending < 0 || max_w_pending > max_in_flight)
    return fail(LC_ERR_INVALID_ARG, "max_w_pending must be in [0, max_in_flight]");
  StagePlan p{};
  p.ty = stage_types(d);
  const size_t es = bytes_of(p.ty.op), ea = bytes_of(p.ty.att), er = bytes_of(p.ty.res);
  const int64_t T = (int64_t)d.micro_batch * d.seq_len;
  const size_t D = (size_t)d.d_model, H = (size_t)d.n_heads;
  const bool moe = d.n_experts > 0;
  const size_t F = moe ? (size_t)d.d_ff_expert : (size_t)d.d_ff;
  const size_t R = moe ? 2 * (size_t)T : (size_t)T;  // FFN rows (routed rows for MoE)
  p.elem = es;
  p.T = T;
  const size_t Hkv = (size_t)kv_heads(d);
  p.dkv = (int64_t)(Hkv * (size_t)d.head_dim);
  p.qkv_cols = (int64_t)D + 2 * p.dkv;
  const size_t QC = (size_t)p.qkv_cols;
  size_t off = 0;
  const size_t half = (size_t)d.head_dim / 2;
  p.rope_cos = off; off = align256(off + (size_t)d.seq_len * half * 4);
  p.rope_sin = off; off = align256(off + (size_t)d.seq_len * half * 4);

  // one layer block of the stash
  size_t lo = 0;
  auto take = [&](size_t bytes) { size_t r = lo; lo = align256(lo + bytes); return r; };
  p.xin = take((size_t)T * D * er);
  p.rstd1 = take((size_t)T * 4);
  p.n1 = take((size_t)T * D * es);
  p.qkv = take((size_t)T * QC * ea);
  p.qkvb = (p.ty.att == LC_FP16 && !d.qk_norm) ? take((size_t)T * QC * 2) : 0;
  if (d.qk_norm) {
    p.qkraw = take((size_t)T * (D + (size_t)p.dkv) * ea);
    p.rstdqk = take((size_t)T * (H + Hkv) * 4);
  }
  p.o = take((size_t)T * D * es);
  p.lse = take((size_t)T * H * 4);
  p.h = take((size_t)T * D * er);
  p.rstd2 = take((size_t)T * 4);
  p.n2 = take((size_t)T * D * es);
  p.gate = take(R * F * er);
  p.up = take(R * F * er);
  p.act = take(R * F * es);
  if (moe) {
    const size_t E = (size_t)d.n_experts;
    p.moe_sel = take((size_t)T * 2 * 4);
    p.moe_w = take((size_t)T * 2 * 4);
    p.moe_perm = take(R * 4);
    p.moe_wrow = take(R * 4);
    p.moe_rowpos = take((size_t)T * 2 * 4);
    p.moe_off = take((E + 1) * 4);
    p.moe_xp = take(R * D * es);
    p.moe_eo = take(R * D * 4);
  }
  p.layer_bytes = lo;
  p.slot_bytes = lo * (size_t)d.n_layers;
  p.slot0 = off;
  off = align256(off + p.slot_bytes * (size_t)max_in_flight);

  // one layer block of a weight-pass slot
  size_t wo = 0;
  auto wtake = [&](size_t bytes) { size_t r = wo; wo = align256(wo + bytes); return r; };
  p.w_dy = wtake((size_t)T * D * es);
  p.w_da = wtake(R * 2 * F * es);
  p.w_dh = wtake((size_t)T * D * es);
  p.w_dqkv = wtake((size_t)T * QC * es);
  p.w_p2 = wtake(rmsnorm_scratch_size(T, d.d_model));
  p.w_p1 = wtake(rmsnorm_scratch_size(T, d.d_model));
  p.w_pqk = d.qk_norm ? wtake(qknorm_scratch_size(T, d.head_dim)) : 0;
  if (moe) {
    p.w_dys = wtake(R * D * es);
    p.w_dl = wtake((size_t)T * 2 * 4);
    p.w_rpart = wtake(moe_router_scratch_size(T, d.d_model, d.n_experts));
  }
  p.wlayer_bytes = wo;
  p.wslot_bytes = wo * (size_t)d.n_layers;
  p.w_slots = max_w_pending;
  p.wslot0 = off;
  off = align256(off + p.wslot_bytes * (size_t)max_w_pending);

  auto stake = [&](size_t bytes) { size_t r = off; off = align256(off + bytes); return r; };
  p.s_dy0 = stake((size_t)T * D * er);
  p.s_dy1 = stake((size_t)T * D * er);
  p.s_dy16 = stake((size_t)T * D * es);
  p.s_da = stake(R * 2 * F * es);
  p.s_dn = stake((size_t)T * D * er);
  p.s_do = stake((size_t)T * D * es);
  p.s_dqkv = stake((size_t)T * QC * es);
  p.s_dh = stake((size_t)T * D * er);
  p.s_dh16 = stake((size_t)T * D * es);
  p.s_attn_bytes = attn_scratch_size(d.micro_batch, d.seq_len, d.n_heads, (int64_t)Hkv);
  p.s_attn = stake(p.s_attn_bytes);
  p.s_norm_bytes = rmsnorm_scratch_size(T, d.d_model);
  p.s_norm = stake(p.s_norm_bytes);
  if (d.qk_norm) {
    p.s_qkn_bytes = qknorm_scratch_size(T, d.head_dim);
    p.s_qkn = stake(p.s_qkn_bytes);
  }
  if (moe) {
    p.s_moe_dys = stake(R * D * es);
    p.s_moe_dns = stake(R * D * 4);
    p.s_moe_dw = stake(R * 4);
    p.s_moe_dl = stake((size_t)T * 2 * 4);
    p.s_moe_part_bytes = moe_router_scratch_size(T, d.d_model, d.n_experts);
    p.s_moe_part = stake(p.s_moe_part_bytes);
  }
  p.total = off;
  *out = p;
  return LC_OK;
}

size_t rmsnorm_scratch_size(int64_t T, int64_t d) {
  const int64_t blocks = (T + kNormRowsPerBlock - 1) / kNormRowsPerBlock;
  return (size_t)(blocks * d) * sizeof(float);
}

size_t moe_router_scratch_size(int64_t T, int64_t d, int64_t E) {
  const int64_t nblk = (T + kRouterTokensPerBlock - 1) / kRouterTokensPerBlock;
  return (size_t)(nblk * E * d) * sizeof(float);
}

size_t attn_share_offset(int64_t B, int64_t S, int64_t H, int64_t Hkv) {
  // D and -lse log2(e) (fp32 [B, H, S] each), then for the matrix-core
  // backward of fp16 inputs bf16 rows of v ([B*S, Hkv*128]), q ([B*S, H*128])
  // and k ([B*S, Hkv*128])
  const size_t dbytes = ((size_t)(B * S * H) * 2 * sizeof(float) + 255) / 256 * 256;
  return align256(dbytes + (size_t)(B * S) * (size_t)(H + 2 * Hkv) * 128 * 2);
}

size_t attn_scratch_size(int64_t B, int64_t S, int64_t H, int64_t Hkv) {
  // with grouped-query attention, then each query head's fp32 share of dk
  // and dv ([B*S, H*128] each)
  const size_t shares = Hkv < H ? (size_t)(B * S) * (size_t)H * 128 * 4 * 2 : 0;
  return attn_share_offset(B, S, H, Hkv) + shares;
}

size_t qknorm_scratch_size(int64_t T, int64_t hd) {
  const int64_t nblk = (T + kQkTokensPerBlock - 1) / kQkTokensPerBlock;
  return (size_t)(nblk * 2 * hd) * sizeof(float);
}

lc_status flatten_order(const lc_order &order, std::vector<lc_order_entry> *flat) {
  flat->clear();
  flat->reserve((size_t)order.n_entries);
  for (int32_t i = 0; i < order.n_entries; ++i) {
    lc_order_entry e = order.entries[i];
    if (!(e.pass & LC_ORDER_WITH_NEXT)) {
      flat->push_back(e);
      continue;
    }
    if (i + 1 >= order.n_entries)
      return fail(LC_ERR_BAD_ORDER, "entry %d: overlapped with a next entry that does not exist", i);
    lc_order_entry f = order.entries[i + 1];
    if (f.pass & LC_ORDER_WITH_NEXT)
      return fail(LC_ERR_BAD_ORDER, "entries %d-%d: an overlapped group holds two entries", i,
                  i + 2);
    e.pass &= ~LC_ORDER_WITH_NEXT;
    const int a = e.pass, b = f.pass;
    const bool kinds =
        (a == LC_PASS_F && (b == LC_PASS_B || b == LC_PASS_BI || b == LC_PASS_BW)) ||
        (b == LC_PASS_F && (a == LC_PASS_B || a == LC_PASS_BI || a == LC_PASS_BW)) ||
        (a == LC_PASS_BI && b == LC_PASS_BW) || (a == LC_PASS_BW && b == LC_PASS_BI);
    if (!kinds || e.mb == f.mb)
      return fail(LC_ERR_BAD_ORDER,
                  "entries %d, %d: an overlapped pair is F with B, Bi or Bw, or Bi with Bw, of "
                  "two different microbatches",
                  i, i + 1);
    // the acquiring entry (F, Bi) first
    if (b == LC_PASS_F || (b == LC_PASS_BI && a == LC_PASS_BW)) std::swap(e, f);
    flat->push_back(e);
    flat->push_back(f);
    ++i;
  }
  return LC_OK;
}

}  // namespace lc

using namespace lc;

extern "C" {

const char *lc_last_error(void) { return g_err; }

lc_status lc_param_count(const lc_stage_desc *desc, size_t *n_elems) {
  lc_status st = validate_desc(desc);
  if (st != LC_OK) return st;
  if (!n_elems) return fail(LC_ERR_INVALID_ARG, "null output pointer");
  *n_elems = param_plan(*desc).total;
  return LC_OK;
}

lc_status lc_param_offset(const lc_stage_desc *desc, int32_t layer, int32_t tensor_id,
                          int32_t expert, size_t *offset, int64_t shape[2]) {
  lc_status st = validate_desc(desc);
  if (st != LC_OK) return st;
  if (!offset || !shape) return fail(LC_ERR_INVALID_ARG, "null output pointer");
  if (layer < 0 || layer >= desc->n_layers) return fail(LC_ERR_INVALID_ARG, "layer out of range");
  const ParamPlan p = param_plan(*desc);
  const int64_t D = desc->d_model;
  const bool moe = desc->n_experts > 0;
  size_t base = (size_t)layer * p.per_layer, o = 0;
  int64_t r = 0, c = 1;
  if (tensor_id != LC_T_W1 && tensor_id != LC_T_W3 && tensor_id != LC_T_W2 && expert != 0)
    return fail(LC_ERR_INVALID_ARG, "expert index only applies to W1/W3/W2");
  switch (tensor_id) {
    case LC_T_WQ: o = p.wq; r = D; c = D; break;
    case LC_T_WK: o = p.wk; r = (int64_t)kv_heads(*desc) * desc->head_dim; c = D; break;
    case LC_T_WV: o = p.wv; r = (int64_t)kv_heads(*desc) * desc->head_dim; c = D; break;
    case LC_T_QN: case LC_T_KN:
      if (!desc->qk_norm) return fail(LC_ERR_INVALID_ARG, "stage has no q/k norm gains");
      o = tensor_id == LC_T_QN ? p.qn : p.kn; r = desc->head_dim; break;
    case LC_T_WO: o = p.wo; r = D; c = D; break;
    case LC_T_G1: o = p.g1; r = D; break;
    case LC_T_G2: o = p.g2; r = D; break;
    case LC_T_WR:
      if (!moe) return fail(LC_ERR_INVALID_ARG, "dense stage has no router");
      o = p.wr; r = desc->n_experts; c = D; break;
    case LC_T_W1: case LC_T_W3: case LC_T_W2: {
      if (!moe) {
        if (expert != 0) return fail(LC_ERR_INVALID_ARG, "dense stage has no experts");
        const int64_t F = desc->d_ff;
        if (tensor_id == LC_T_W1) { o = p.w1; r = F; c = D; }
        if (tensor_id == LC_T_W3) { o = p.w3; r = F; c = D; }
        if (tensor_id == LC_T_W2) { o = p.w2; r = D; c = F; }
      } else {
        if (expert < 0 || expert >= desc->n_experts)
          return fail(LC_ERR_INVALID_ARG, "expert out of range");
        const int64_t FE = desc->d_ff_expert;
        size_t e0 = p.expert0 + (size_t)expert * p.expert_stride;
        if (tensor_id == LC_T_W1) { o = e0; r = FE; c = D; }
        if (tensor_id == LC_T_W3) { o = e0 + (size_t)(FE * D); r = FE; c = D; }
        if (tensor_id == LC_T_W2) { o = e0 + (size_t)(2 * FE * D); r = D; c = FE; }
      }
      break;
    }
    default: return fail(LC_ERR_INVALID_ARG, "unknown tensor id %d", tensor_id);
  }
  *offset = base + o;
  shape[0] = r;
  shape[1] = c;
  return LC_OK;
}

lc_status lc_order_1f1b(int32_t M, int32_t P, int32_t s, lc_order_entry *out, int32_t capacity,
                        int32_t *n) {
  if (M <= 0 || P <= 0 || s < 0 || s >= P)
    return fail(LC_ERR_INVALID_ARG, "need M > 0, P > 0 and 0 <= s < P");
  if (!out || !n) return fail(LC_ERR_INVALID_ARG, "null output pointer");
  if (capacity < 2 * M) return fail(LC_ERR_INVALID_ARG, "capacity %d < 2M = %d", capacity, 2 * M);
  const int32_t W = (P - s - 1) < M ? (P - s - 1) : M;
  int32_t k = 0;
  for (int32_t i = 0; i < W; ++i) out[k++] = lc_order_entry{i, LC_PASS_F};
  for (int32_t i = 0; i < M - W; ++i) {
    out[k++] = lc_order_entry{W + i, LC_PASS_F};
    out[k++] = lc_order_entry{i, LC_PASS_B};
  }
  for (int32_t i = M - W; i < M; ++i) out[k++] = lc_order_entry{i, LC_PASS_B};
  *n = k;
  return LC_OK;
}

lc_status lc_order_1f1b_overlap(int32_t M, int32_t P, int32_t s, lc_order_entry *out,
                                int32_t capacity, int32_t *n) {
  LC_TRY(lc_order_1f1b(M, P, s, out, capacity, n));
  // the steady state: entries W + 2i, W + 2i + 1 for i < M - W
  const int32_t W = (P - s - 1) < M ? (P - s - 1) : M;
  // (none without warm-up: each pair would be one microbatch's F and B)
  for (int32_t i = 0; W > 0 && i < M - W; ++i) out[W + 2 * i].pass |= LC_ORDER_WITH_NEXT;
  return LC_OK;
}

lc_status lc_order_1f1b_split(int32_t M, int32_t P, int32_t s, int32_t w_delay,
                              lc_order_entry *out, int32_t capacity, int32_t *n) {
  if (w_delay < 0) return fail(LC_ERR_INVALID_ARG, "w_delay must be >= 0");
  if (!out || !n) return fail(LC_ERR_INVALID_ARG, "null output pointer");
  if (M > 0 && capacity < 3 * M)
    return fail(LC_ERR_INVALID_ARG, "capacity %d < 3M = %d", capacity, 3 * M);
  std::vector<lc_order_entry> base((size_t)(M > 0 ? 2 * M : 0));
  int32_t nb = 0;
  lc_status st = lc_order_1f1b(M, P, s, base.data(), 2 * M, &nb);
  if (st != LC_OK) return st;
  int32_t k = 0, oldest = 0;  // Bw entries leave in microbatch order
  for (int32_t i = 0; i < nb; ++i) {
    const lc_order_entry e = base[(size_t)i];
    if (e.pass == LC_PASS_F) {
      out[k++] = e;
      continue;
    }
    out[k++] = lc_order_entry{e.mb, LC_PASS_BI};
    if (e.mb - oldest >= w_delay) out[k++] = lc_order_entry{oldest++, LC_PASS_BW};
  }
  while (oldest < M) out[k++] = lc_order_entry{oldest++, LC_PASS_BW};
  *n = k;
  return LC_OK;
}

lc_status lc_order_1f1b_split_overlap(int32_t M, int32_t P, int32_t s, int32_t w_delay,
                                      lc_order_entry *out, int32_t capacity, int32_t *n) {
  LC_TRY(lc_order_1f1b_split(M, P, s, w_delay, out, capacity, n));
  // each Bi with another microbatch's Bw right after it becomes a pair (an
  // entry belongs to at most one pair)
  for (int32_t i = 0; i + 1 < *n; ++i)
    if (out[i].pass == LC_PASS_BI && out[i + 1].pass == LC_PASS_BW && out[i].mb != out[i + 1].mb) {
      out[i].pass |= LC_ORDER_WITH_NEXT;
      ++i;
    }
  return LC_OK;
}

lc_status lc_order_validate_split(const lc_order *order, int32_t max_in_flight,
                                  int32_t max_w_pending, int32_t *peak, int32_t *peak_w) {
  if (peak) *peak = 0;
  if (peak_w) *peak_w = 0;
  if (!order) return fail(LC_ERR_INVALID_ARG, "null order");
  if (max_in_flight <= 0) return fail(LC_ERR_INVALID_ARG, "max_in_flight must be positive");
  if (max_w_pending < 0) return fail(LC_ERR_INVALID_ARG, "max_w_pending must be >= 0");
  const int32_t M = order->num_microbatches;
  if (M <= 0) return fail(LC_ERR_BAD_ORDER, "num_microbatches must be positive");
  if (order->n_entries < 2 * M || (int64_t)order->n_entries > 3 * (int64_t)M)
    return fail(LC_ERR_BAD_ORDER, "an Order over %d microbatches has %d entries, not 2M to 3M", M,
                order->n_entries);
  if (!order->entries) return fail(LC_ERR_INVALID_ARG, "null entries");
  std::vector<lc_order_entry> flat;
  LC_TRY(flatten_order(*order, &flat));
  // seen[mb] bit p: pass p of mb has appeared
  std::vector<uint8_t> seen((size_t)M, 0);
  static const char *const kName[4] = {"F", "B", "Bi", "Bw"};
  int32_t last_f = -1, last_b = -1, live = 0, pk = 0, wlive = 0, pkw = 0;
  lc_status res = LC_OK;
  for (int32_t i = 0; i < order->n_entries && res == LC_OK; ++i) {
    const lc_order_entry e = flat[(size_t)i];
    if (e.mb < 0 || e.mb >= M) {
      res = fail(LC_ERR_BAD_ORDER, "entry %d: microbatch %d out of range", i, e.mb);
      break;
    }
    if (e.pass < LC_PASS_F || e.pass > LC_PASS_BW) {
      res = fail(LC_ERR_BAD_ORDER, "entry %d: unknown pass %d", i, e.pass);
      break;
    }
    uint8_t &sn = seen[(size_t)e.mb];
    const uint8_t bit = (uint8_t)(1u << e.pass);
    if (sn & bit) {
      res = fail(LC_ERR_BAD_ORDER, "entry %d: %s%d appears twice", i, kName[e.pass], e.mb);
      break;
    }
    switch (e.pass) {
      case LC_PASS_F:
        if (e.mb <= last_f) {
          res = fail(LC_ERR_BAD_ORDER, "entry %d: F%d after F%d (forwards must be in order)", i,
                     e.mb, last_f);
          break;
        }
        last_f = e.mb;
        if (++live > pk) pk = live;
        if (live > max_in_flight)
          res = fail(LC_ERR_STASH_FULL, "entry %d: %d microbatches in flight > %d slots", i, live,
                     max_in_flight);
        break;
      case LC_PASS_B:
      case LC_PASS_BI:
        if (!(sn & (1u << LC_PASS_F))) {
          res = fail(LC_ERR_BAD_ORDER, "entry %d: %s%d before F%d", i, kName[e.pass], e.mb, e.mb);
          break;
        }
        if (e.mb <= last_b || (sn & ((1u << LC_PASS_B) | (1u << LC_PASS_BI)))) {
          res = fail(LC_ERR_BAD_ORDER,
                     "entry %d: %s%d after the backward of microbatch %d (B and Bi entries "
                     "must be in order, one per microbatch)",
                     i, kName[e.pass], e.mb, last_b);
          break;
        }
        last_b = e.mb;
        if (e.pass == LC_PASS_B) {
          --live;
        } else {
          if (++wlive > pkw) pkw = wlive;
          if (wlive > max_w_pending)
            res = fail(LC_ERR_STASH_FULL, "entry %d: %d weight passes pending > %d slots", i,
                       wlive, max_w_pending);
        }
        break;
      default:  // LC_PASS_BW
        if (!(sn & (1u << LC_PASS_BI))) {
          res = fail(LC_ERR_BAD_ORDER, "entry %d: Bw%d before Bi%d", i, e.mb, e.mb);
          break;
        }
        --live;
        --wlive;
        break;
    }
    sn |= bit;
  }
  if (peak) *peak = pk;
  if (peak_w) *peak_w = pkw;
  if (res != LC_OK) return res;
  for (int32_t mb = 0; mb < M; ++mb) {
    const uint8_t sn = seen[(size_t)mb];
    const bool has_b = sn & (1u << LC_PASS_B), has_bw = sn & (1u << LC_PASS_BW);
    if (!(sn & (1u << LC_PASS_F)) || has_b == has_bw)
      return fail(LC_ERR_BAD_ORDER, "microbatch %d lacks its F, or its B (or Bi and Bw)", mb);
  }
  return LC_OK;
}

lc_status lc_order_validate(const lc_order *order, int32_t max_in_flight, int32_t *peak) {
  return lc_order_validate_split(order, max_in_flight, max_in_flight, peak, nullptr);
}

lc_status lc_workspace_bytes_split(const lc_stage_desc *desc, int32_t max_in_flight,
                                   int32_t max_w_pending, size_t *bytes) {
  if (!bytes) return fail(LC_ERR_INVALID_ARG, "null output pointer");
  StagePlan p;
  lc_status st = validate_desc(desc);
  if (st != LC_OK) return st;
  st = stage_plan(*desc, max_in_flight, max_w_pending, &p);
  if (st != LC_OK) return st;
  *bytes = p.total;
  return LC_OK;
}

lc_status lc_workspace_bytes(const lc_stage_desc *desc, int32_t max_in_flight, size_t *bytes) {
  return lc_workspace_bytes_split(desc, max_in_flight, 0, bytes);
}

size_t lc_rmsnorm_scratch_bytes(int64_t T, int64_t d) { return rmsnorm_scratch_size(T, d); }
size_t lc_attention_scratch_bytes(int32_t B, int32_t S, int32_t H) {
  return attn_scratch_size(B, S, H, H);
}
size_t lc_attention_scratch_bytes_kv(int32_t B, int32_t S, int32_t H, int32_t Hkv) {
  return attn_scratch_size(B, S, H, Hkv > 0 ? Hkv : H);
}
size_t lc_qk_norm_scratch_bytes(int64_t T, int32_t hd) { return qknorm_scratch_size(T, hd); }

}  // extern "C"
