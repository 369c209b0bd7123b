// Qwen3-style per-head RMSNorm of q and k fused with RoPE (HBM-bound row
// kernels over the packed q|k head rows of T tokens).
//
//   forward:  r = 1/sqrt(mean(x^2) + eps), y = x * r * g, then rotate-half
//             RoPE of y at the token's position
//   backward: given dy (gradient at y, the rotation already undone by the
//             attention backward), xh = x * r, dxh = dy * g:
//             dx = r * (dxh - xh * mean(dxh * xh)), dg += sum over rows dy * xh
//
// A head row of hd values is held by hd / 8 consecutive lanes, 8 values each
// (16- or 32-byte accesses), so a wave covers 512 / hd rows at once. Row
// sums are shuffles inside each row's lane group. RoPE pairs value i with
// i + hd/2: the partner sits in the lane hd/16 positions away.
//
// The gain gradient is deterministic: a backward workgroup handles
// kQkTokensPerBlock tokens in a fixed row order, sums each lane's rows, then
// the row slots of a wave in a fixed shuffle tree, then the waves in order,
// and writes partial[blk][0, hd) (q gains) and [hd, 2 hd) (k gains); the
// final kernel adds the partials of each column in block order (sixteen
// slices of consecutive blocks, then the slices in order).
#include "common.hpp"

namespace lc {
namespace {

constexpr int NTH = 256;

struct QkP {
  int64_t T;
  int H, NH, hd, lpr, seq_len;  // NH = H + Hkv heads per token; lpr = hd / 8 lanes per row
  float eps;
  int x_dt, w_dt, d_dt;
  void *qk;
  int64_t ld;
  void *raw;
  float *rstd;
  const void *gq, *gk;
  const float *rcos, *rsin;
  void *dqk;
  int64_t ld_d;
  float *partial;
  float *dgq, *dgk;
  int store_dg, nblk;
};

// sum over the lpr lanes of a row (lanes aligned to lpr, lpr a power of two)
__device__ __forceinline__ float row_sum(float v, int lpr) {
  for (int o = 1; o < lpr; o <<= 1) v += __shfl_xor(v, o, 64);
  return v;
}

template <int XD, int WD>  // element types of q|k and the gains (compile-time)
__global__ __launch_bounds__(NTH) void qk_norm_rope_fwd_kernel(QkP p) {
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  const int rpw = 64 / p.lpr, l = lane % p.lpr;
  const int64_t row = ((int64_t)blockIdx.x * 4 + wv) * rpw + lane / p.lpr;
  if (row >= p.T * p.NH) return;  // whole row groups leave together
  const int64_t t = row / p.NH;
  const int j = (int)(row % p.NH);
  const bool isq = j < p.H;
  const int64_t col = (int64_t)j * p.hd + 8 * l;  // q heads then k heads
  float x[8];
  ld8<XD>(p.qk, t * p.ld + col, p.x_dt, x);
  st8<XD>(p.raw, row * p.hd + 8 * l, p.x_dt, x);
  float ss = 0.0f;
#pragma unroll
  for (int e = 0; e < 8; ++e) ss += x[e] * x[e];
  ss = row_sum(ss, p.lpr);
  const float r = 1.0f / sqrtf(ss / (float)p.hd + p.eps);
  if (l == 0) p.rstd[row] = r;
  float g[8];
  ld8<WD>(isq ? p.gq : p.gk, 8 * l, p.w_dt, g);
  float y[8], z[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) y[e] = x[e] * r * g[e];
  // rotate-half: lanes l < lpr/2 hold values i, lanes l + lpr/2 values i + hd/2
  const int half = p.hd / 2;
  const bool first = l < p.lpr / 2;
  const int i0 = 8 * l - (first ? 0 : half);
  const int pos = (int)(t % p.seq_len);
  const float *cs = p.rcos + (int64_t)pos * half + i0;
  const float *sn = p.rsin + (int64_t)pos * half + i0;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const float other = __shfl_xor(y[e], p.lpr / 2, 64);
    const float c = cs[e], s = sn[e];
    // first half: a c - b s; second half: a s + b c (a = value i, b = value i + hd/2)
    z[e] = first ? y[e] * c - other * s : other * s + y[e] * c;
  }
  st8<XD>(p.qk, t * p.ld + col, p.x_dt, z);
}

template <int XD, int WD, int DD>  // element types of raw q|k, the gains and the gradient
__global__ __launch_bounds__(NTH) void qk_norm_bwd_kernel(QkP p) {
  __shared__ float red[2][128];
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  const int rpw = 64 / p.lpr, l = lane % p.lpr, slot = lane / p.lpr;
  const int64_t r0 = (int64_t)blockIdx.x * kQkTokensPerBlock * p.NH;
  const int64_t r1 = min(p.T * p.NH, r0 + (int64_t)kQkTokensPerBlock * p.NH);
  float aq[8], ak[8], gq[8], gk[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) aq[e] = ak[e] = 0.0f;
  ld8<WD>(p.gq, 8 * l, p.w_dt, gq);
  ld8<WD>(p.gk, 8 * l, p.w_dt, gk);
  // iteration it: rows r0 + (4 it + wv) rpw + slot
  for (int64_t base = r0 + (int64_t)wv * rpw; base < r1; base += 4 * rpw) {
    const int64_t row = base + slot;
    const bool ok = row < r1;
    const int64_t rr = ok ? row : r0;
    const int64_t t = rr / p.NH;
    const int j = (int)(rr % p.NH);
    const bool isq = j < p.H;
    const int64_t col = (int64_t)j * p.hd + 8 * l;
    float a[8], b[8];
    ld8<DD>(p.dqk, t * p.ld_d + col, p.d_dt, a);
    ld8<XD>(p.raw, rr * p.hd + 8 * l, p.x_dt, b);
    const float r = p.rstd[rr];
    float dot = 0.0f;  // sum dy * g * x
#pragma unroll
    for (int e = 0; e < 8; ++e) dot += a[e] * (isq ? gq[e] : gk[e]) * b[e];
    dot = row_sum(dot, p.lpr);
    const float mean = dot * r / (float)p.hd;
    const float r2m = r * mean;
    if (!ok) continue;  // row groups past the block's end (lane-group uniform)
    float o[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const float gv = isq ? gq[e] : gk[e];
      o[e] = r * (a[e] * gv - b[e] * r2m);
      const float term = a[e] * (b[e] * r);
      if (isq) aq[e] += term;
      else ak[e] += term;
    }
    st8<DD>(p.dqk, t * p.ld_d + col, p.d_dt, o);
  }
  // the wave's row slots: fixed shuffle tree (slot 0 ends with the sum)
  for (int o = p.lpr; o < 64; o <<= 1) {
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      aq[e] += __shfl_xor(aq[e], o, 64);
      ak[e] += __shfl_xor(ak[e], o, 64);
    }
  }
  // the waves in order
#pragma unroll 1
  for (int w = 0; w < 4; ++w) {
    if (wv == w && slot == 0) {
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        red[0][8 * l + e] = (w == 0 ? 0.0f : red[0][8 * l + e]) + aq[e];
        red[1][8 * l + e] = (w == 0 ? 0.0f : red[1][8 * l + e]) + ak[e];
      }
    }
    __syncthreads();
  }
  const int t = threadIdx.x;
  if (t < 2 * p.hd)
    p.partial[(int64_t)blockIdx.x * 2 * p.hd + t] = t < p.hd ? red[0][t] : red[1][t - p.hd];
}

constexpr int SLICES = 16;
// column k < 2 hd: the q (k < hd) or k gain gradient gets the sum over blocks
__global__ __launch_bounds__(1024) void qk_norm_dg_final_kernel(QkP p) {
  __shared__ float sl[SLICES][64];
  const int t = threadIdx.x, sidx = t >> 6, kc = t & 63;
  const int k = blockIdx.x * 64 + kc, width = 2 * p.hd;
  const int per = (p.nblk + SLICES - 1) / SLICES;
  const int b0 = sidx * per, b1 = min(p.nblk, b0 + per);
  float s = 0.0f;
  if (k < width)
    for (int b = b0; b < b1; ++b) s += p.partial[(int64_t)b * width + k];
  sl[sidx][kc] = s;
  __syncthreads();
  if (sidx == 0 && k < width) {
    float tot = sl[0][kc];
#pragma unroll
    for (int i = 1; i < SLICES; ++i) tot += sl[i][kc];
    float *dg = k < p.hd ? p.dgq + k : p.dgk + (k - p.hd);
    *dg = p.store_dg ? tot : *dg + tot;
  }
}

lc_status check(const lc_qknorm_args &a, bool bwd) {
  if (a.T <= 0 || a.H <= 0 || a.Hkv <= 0 || a.seq_len <= 0)
    return fail(LC_ERR_INVALID_ARG, "q/k norm: sizes must be positive");
  if (a.hd != 16 && a.hd != 32 && a.hd != 64 && a.hd != 128)
    return fail(LC_ERR_UNSUPPORTED, "q/k norm: head_dim must be 16, 32, 64 or 128");
  if (a.x_dtype != LC_FP16 && a.x_dtype != LC_FP32)
    return fail(LC_ERR_INVALID_ARG, "q/k norm: x_dtype must be LC_FP16 or LC_FP32");
  if (!valid_dtype(a.w_dtype)) return fail(LC_ERR_INVALID_ARG, "q/k norm: unknown w_dtype");
  const int64_t width = (int64_t)(a.H + a.Hkv) * a.hd;
  if (!a.raw || !a.rstd || !a.gq || !a.gk || !aligned16(a.raw) || !aligned16(a.gq) || !aligned16(a.gk))
    return fail(LC_ERR_INVALID_ARG, "q/k norm: null or unaligned pointer");
  if (!bwd) {
    if (!a.qk || !aligned16(a.qk) || a.ld < width || a.ld % 8)
      return fail(LC_ERR_INVALID_ARG, "q/k norm: bad qk pointer or ld");
    if (!a.rope_cos || !a.rope_sin) return fail(LC_ERR_INVALID_ARG, "q/k norm: null RoPE table");
  } else {
    if (a.d_dtype != LC_BF16 && a.d_dtype != LC_FP32)
      return fail(LC_ERR_INVALID_ARG, "q/k norm: d_dtype must be LC_BF16 or LC_FP32");
    if (!a.dqk || !aligned16(a.dqk) || a.ld_d < width || a.ld_d % 8)
      return fail(LC_ERR_INVALID_ARG, "q/k norm: bad dqk pointer or ld_d");
    if (!a.scratch || a.scratch_bytes < qknorm_scratch_size(a.T, a.hd))
      return fail(LC_ERR_WORKSPACE, "q/k norm: scratch smaller than lc_qk_norm_scratch_bytes");
  }
  return LC_OK;
}

QkP make(const lc_qknorm_args &a) {
  QkP p{};
  p.T = a.T;
  p.H = a.H;
  p.NH = a.H + a.Hkv;
  p.hd = a.hd;
  p.lpr = a.hd / 8;
  p.seq_len = a.seq_len;
  p.eps = a.eps;
  p.x_dt = a.x_dtype;
  p.w_dt = a.w_dtype;
  p.d_dt = a.d_dtype;
  p.qk = a.qk;
  p.ld = a.ld;
  p.raw = a.raw;
  p.rstd = a.rstd;
  p.gq = a.gq;
  p.gk = a.gk;
  p.rcos = a.rope_cos;
  p.rsin = a.rope_sin;
  p.dqk = a.dqk;
  p.ld_d = a.ld_d;
  p.partial = static_cast<float *>(a.scratch);
  p.dgq = a.dgq;
  p.dgk = a.dgk;
  p.store_dg = a.store_dg;
  p.nblk = (int)((a.T + kQkTokensPerBlock - 1) / kQkTokensPerBlock);
  return p;
}

}  // namespace

lc_status qknorm_fwd_launch(const lc_qknorm_args &a, hipStream_t s) {
  LC_TRY(check(a, false));
  const QkP p = make(a);
  const int64_t rows = a.T * p.NH, per_block = 4 * (64 / p.lpr);
  const dim3 grid((unsigned)((rows + per_block - 1) / per_block));
  with_dtype(p.x_dt, [&](auto xd) {
    with_dtype(p.w_dt, [&](auto wd) {
      hipLaunchKernelGGL((qk_norm_rope_fwd_kernel<decltype(xd)::value, decltype(wd)::value>), grid,
                         dim3(NTH), 0, s, p);
    });
  });
  return check_launch("qk_norm_rope_fwd_kernel");
}

lc_status qknorm_bwd_partials_launch(const lc_qknorm_args &a, hipStream_t s) {
  LC_TRY(check(a, true));
  const QkP p = make(a);
  with_dtype(p.x_dt, [&](auto xd) {
    with_dtype(p.w_dt, [&](auto wd) {
      with_dtype(p.d_dt, [&](auto dd) {
        hipLaunchKernelGGL((qk_norm_bwd_kernel<decltype(xd)::value, decltype(wd)::value,
                                               decltype(dd)::value>),
                           dim3((unsigned)p.nblk), dim3(NTH), 0, s, p);
      });
    });
  });
  return check_launch("qk_norm_bwd_kernel");
}

lc_status qknorm_dg_final_launch(const float *partial, float *dgq, float *dgk, int64_t T, int hd,
                                 bool store, hipStream_t s) {
  if (!partial || !dgq || !dgk || T <= 0 || hd <= 0 || hd > 128)
    return fail(LC_ERR_INVALID_ARG, "q/k norm: bad gain-gradient sum arguments");
  QkP p{};
  p.partial = const_cast<float *>(partial);
  p.dgq = dgq;
  p.dgk = dgk;
  p.hd = hd;
  p.store_dg = store;
  p.nblk = (int)((T + kQkTokensPerBlock - 1) / kQkTokensPerBlock);
  hipLaunchKernelGGL(qk_norm_dg_final_kernel, dim3((unsigned)((2 * hd + 63) / 64)), dim3(1024), 0,
                     s, p);
  return check_launch("qk_norm_dg_final_kernel");
}

lc_status qknorm_bwd_launch(const lc_qknorm_args &a, hipStream_t s) {
  if (!a.dgq || !a.dgk) return fail(LC_ERR_INVALID_ARG, "q/k norm: null gain gradient");
  LC_TRY(qknorm_bwd_partials_launch(a, s));
  return qknorm_dg_final_launch(static_cast<const float *>(a.scratch), a.dgq, a.dgk, a.T, a.hd,
                                a.store_dg != 0, s);
}

}  // namespace lc

extern "C" {

lc_status lc_qk_norm_rope_forward(const lc_qknorm_args *args, void *stream) {
  if (!args) return lc::fail(LC_ERR_INVALID_ARG, "q/k norm: null args");
  return lc::qknorm_fwd_launch(*args, static_cast<hipStream_t>(stream));
}

lc_status lc_qk_norm_rope_backward(const lc_qknorm_args *args, void *stream) {
  if (!args) return lc::fail(LC_ERR_INVALID_ARG, "q/k norm: null args");
  return lc::qknorm_bwd_launch(*args, static_cast<hipStream_t>(stream));
}

}  // extern "C"
