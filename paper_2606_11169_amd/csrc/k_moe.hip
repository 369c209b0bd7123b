// Mixture-of-experts routing, dispatch and combine for a top-2 MoE FFN
// (gfx950). The expert products themselves are grouped GEMMs (k_gemm.hip).
//
// Forward, per layer, on the normalised activations n [T, d]:
//   route:    l[t, e] = n[t] . Wr[e] (fp32), top-2 experts by softmax(l[t])
//             (ties to the lower index), weights renormalised over the pair:
//             w0 = 1 / (1 + exp(l1 - l0)), w1 = 1 - w0 in exact arithmetic
//             (the full softmax's normaliser cancels in the ratio).
//   dispatch: stable counting sort of the 2T (token, expert) pairs by expert:
//             offsets[E + 1], perm[r] (token of sorted row r), wrow[r] (its
//             gate weight), rowpos[t, k] (sorted row of token t's k-th pair).
//             Ranks come from wave ballots and prefix sums of integer counts,
//             so the permutation is the same on every run.
//   gather:   xs[r] = n[perm[r]] (the grouped GEMMs read contiguous rows).
//   combine:  y[t] = h[t] + w[t, 0] eo[rowpos[t, 0]] + w[t, 1] eo[rowpos[t, 1]]
//             (fixed order, fp32).
// Backward:
//   bwd gather:  dys[r] = wrow[r] dy[perm[r]] (operand of the expert
//                products), dw[r] = dy[perm[r]] . eo[r] (gate-weight gradient).
//   bwd combine: dl_k = w_k (dw_k - sum_j w_j dw_j) for the two selected
//                logits; dn[t] = dns[rowpos[t, 0]] + dns[rowpos[t, 1]]
//                + dl_0 Wr[e_0] + dl_1 Wr[e_1].
//   router weight gradient: dWr[e] += sum_t dl[t, e] n[t] as per-block partial
//                sums over 128-token blocks, added in block order.
#include "common.hpp"

#include <math.h>

namespace lc {
namespace {

// ------------------------------------------------------------------ route
struct RouteP {
  const void *n, *wr;
  int32_t *sel;
  float *w;
  int64_t T;
  int d, E, n_dt, w_dt;
};

// one wave per token, 4 tokens per workgroup
template <int ND, int WD>  // element types of n and Wr (compile-time)
__global__ __launch_bounds__(256) void moe_route_kernel(RouteP p) {
  const int lane = threadIdx.x & 63;
  const int64_t t = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (t >= p.T) return;
  // running top-2 over the logits in expert order; strict comparisons keep
  // the lower index on ties, and a NaN logit ranks below every number, so
  // the two selected experts are always distinct
  float l0 = -INFINITY, l1 = -INFINITY;
  int e0 = 0, e1 = 1;
  for (int e = 0; e < p.E; ++e) {
    float s = 0.0f;
    for (int c = lane * 8; c < p.d; c += 64 * 8) {
      float a[8], b[8];
      ld8<ND>(p.n, t * p.d + c, p.n_dt, a);
      ld8<WD>(p.wr, (int64_t)e * p.d + c, p.w_dt, b);
#pragma unroll
      for (int i = 0; i < 8; ++i) s += a[i] * b[i];
    }
    float l = wave_sum(s);
    if (l != l) l = -INFINITY;
    if (e == 0) {
      l0 = l;
      e0 = 0;
    } else if (e == 1) {
      if (l > l0) {
        l1 = l0; e1 = 0;
        l0 = l; e0 = 1;
      } else {
        l1 = l; e1 = 1;
      }
    } else if (l > l0) {
      l1 = l0; e1 = e0;
      l0 = l; e0 = e;
    } else if (l > l1) {
      l1 = l; e1 = e;
    }
  }
  if (lane == 0) {
    const float z = expf(l1 - l0);  // pi_1 / pi_0 <= 1
    const float w0 = 1.0f / (1.0f + z);
    p.sel[2 * t] = e0;
    p.sel[2 * t + 1] = e1;
    p.w[2 * t] = w0;
    p.w[2 * t + 1] = z * w0;
  }
}

// ------------------------------------------------------------------ dispatch
struct DispatchP {
  const int32_t *sel;
  const float *w;
  int32_t *offsets, *perm, *rowpos;
  float *wrow;
  int T, E;
};

constexpr int kDispatchThreads = 1024;

__global__ __launch_bounds__(kDispatchThreads) void moe_dispatch_kernel(DispatchP p) {
  __shared__ int cnt[65], run[64];
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  if (tid < 65) cnt[tid] = 0;
  __syncthreads();
  // a pair is placed when its expert is in range (and differs from the
  // token's first expert); other pairs get rowpos -1 and no row
  for (int t = tid; t < p.T; t += kDispatchThreads) {
    const int a = p.sel[2 * t], b = p.sel[2 * t + 1];
    const bool ok_a = a >= 0 && a < p.E, ok_b = b >= 0 && b < p.E && b != a;
    if (ok_a) atomicAdd(&cnt[a], 1);  // integer counts: order-independent
    if (ok_b) atomicAdd(&cnt[b], 1);
    if (!ok_a) p.rowpos[2 * t] = -1;
    if (!ok_b) p.rowpos[2 * t + 1] = -1;
  }
  __syncthreads();
  if (tid == 0) {
    int acc = 0;
    for (int e = 0; e < p.E; ++e) {
      const int c = cnt[e];
      p.offsets[e] = acc;
      run[e] = acc;
      acc += c;
    }
    p.offsets[p.E] = acc;
    cnt[64] = acc;
  }
  __syncthreads();
  // rows past the last placed pair (only when some pair was not placed) read
  // token 0 with weight 0
  for (int r = cnt[64] + tid; r < 2 * p.T; r += kDispatchThreads) {
    p.perm[r] = 0;
    p.wrow[r] = 0.0f;
  }
  // pairs in token order, kDispatchThreads tokens at a time: each wave counts
  // its pairs of every expert with one ballot per expert (no barrier between
  // experts), then each thread places its (at most two) pairs after the
  // earlier waves' and lanes' pairs of the same expert
  __shared__ int wcnt[64][kDispatchThreads / 64];
  const unsigned long long below = (1ull << lane) - 1ull;
  for (int base = 0; base < p.T; base += kDispatchThreads) {
    const int t = base + tid;
    const bool valid = t < p.T;
    const int a = valid ? p.sel[2 * t] : -1, b0 = valid ? p.sel[2 * t + 1] : -1;
    const int b = b0 == a ? -1 : b0;
    unsigned long long bal_a = 0, bal_b = 0;
    for (int e = 0; e < p.E; ++e) {
      const unsigned long long bal = __ballot(valid && (a == e || b == e));
      if (lane == 0) wcnt[e][wv] = __popcll(bal);
      if (a == e) bal_a = bal;
      if (b == e) bal_b = bal;
    }
    __syncthreads();
#pragma unroll
    for (int k = 0; k < 2; ++k) {
      const int e = k == 0 ? a : b;
      if (valid && e >= 0 && e < p.E) {
        int pre = 0;
        for (int i = 0; i < wv; ++i) pre += wcnt[e][i];
        const int pos = run[e] + pre + __popcll((k == 0 ? bal_a : bal_b) & below);
        p.perm[pos] = t;
        p.wrow[pos] = p.w[2 * t + k];
        p.rowpos[2 * t + k] = pos;
      }
    }
    __syncthreads();
    if (tid < p.E) {
      int tot = 0;
      for (int i = 0; i < kDispatchThreads / 64; ++i) tot += wcnt[tid][i];
      run[tid] += tot;
    }
    __syncthreads();
  }
}

// ------------------------------------------------------------------ row gather
struct GatherP {
  const char *src;
  char *dst;
  const int32_t *idx;
  int64_t rows;
  int row_bytes;  // multiple of 16
};

// one wave per row: dst[r] = src[idx[r]] (raw bytes)
__global__ __launch_bounds__(256) void moe_gather_kernel(GatherP p) {
  const int lane = threadIdx.x & 63;
  const int64_t r = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (r >= p.rows) return;
  const int64_t s = p.idx[r];
  const uint4 *src = reinterpret_cast<const uint4 *>(p.src + s * p.row_bytes);
  uint4 *dst = reinterpret_cast<uint4 *>(p.dst + r * p.row_bytes);
  for (int c = lane; c < p.row_bytes / 16; c += 64) dst[c] = src[c];
}

// ------------------------------------------------------------------ combine
struct CombineP {
  const void *h;      // residual input [T, d]
  const float *eo;    // expert outputs in sorted order [2T, d]
  const float *w;     // [T, 2]
  const int32_t *rowpos;
  void *out;
  int64_t T;
  int d, h_dt, out_dt;
};

template <int HD, int OD>  // element types of h and out
__global__ __launch_bounds__(256) void moe_combine_kernel(CombineP p) {
  const int lane = threadIdx.x & 63;
  const int64_t t = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (t >= p.T) return;
  const int64_t q0 = p.rowpos[2 * t], q1 = p.rowpos[2 * t + 1];
  // an unplaced pair (rowpos -1) contributes nothing
  const float w0 = q0 >= 0 ? p.w[2 * t] : 0.0f, w1 = q1 >= 0 ? p.w[2 * t + 1] : 0.0f;
  const int64_t r0 = q0 >= 0 ? q0 : 0, r1 = q1 >= 0 ? q1 : 0;
  for (int c = lane * 8; c < p.d; c += 64 * 8) {
    float x[8], a[8], b[8];
    ld8<HD>(p.h, t * p.d + c, p.h_dt, x);
    ld8<LC_FP32>(p.eo, r0 * p.d + c, LC_FP32, a);
    ld8<LC_FP32>(p.eo, r1 * p.d + c, LC_FP32, b);
#pragma unroll
    for (int i = 0; i < 8; ++i) x[i] = (x[i] + w0 * a[i]) + w1 * b[i];
    st8<OD>(p.out, t * p.d + c, p.out_dt, x);
  }
}

// ------------------------------------------------------------------ backward
struct BwdGatherP {
  const void *dy;     // [T, d]
  const float *eo;    // [2T, d]
  const int32_t *perm;
  const float *wrow;
  void *dys;          // [2T, d], dys_dt
  float *dw;          // [2T]
  int64_t rows;
  int d, dy_dt, dys_dt;
};

template <int GD, int SD>  // element types of dy and dys
__global__ __launch_bounds__(256) void moe_bwd_gather_kernel(BwdGatherP p) {
  const int lane = threadIdx.x & 63;
  const int64_t r = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (r >= p.rows) return;
  const int64_t t = p.perm[r];
  const float wr = p.wrow[r];
  float dot = 0.0f;
  for (int c = lane * 8; c < p.d; c += 64 * 8) {
    float g[8], e[8];
    ld8<GD>(p.dy, t * p.d + c, p.dy_dt, g);
    ld8<LC_FP32>(p.eo, r * p.d + c, LC_FP32, e);
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      dot += g[i] * e[i];
      g[i] *= wr;
    }
    st8<SD>(p.dys, r * p.d + c, p.dys_dt, g);
  }
  dot = wave_sum(dot);
  if (lane == 0) p.dw[r] = dot;
}

struct BwdCombineP {
  const float *dns;   // [2T, d] fp32
  const float *dw;    // [2T]
  const float *w;     // [T, 2]
  const int32_t *sel, *rowpos;
  const void *wr;     // [E, d]
  float *dl;          // [T, 2]
  float *dn;          // [T, d]
  int64_t T;
  int d, w_dt;
};

template <int WD>  // element type of Wr
__global__ __launch_bounds__(256) void moe_bwd_combine_kernel(BwdCombineP p) {
  const int lane = threadIdx.x & 63;
  const int64_t t = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (t >= p.T) return;
  const int64_t q0 = p.rowpos[2 * t], q1 = p.rowpos[2 * t + 1];
  const bool ok0 = q0 >= 0, ok1 = q1 >= 0;  // unplaced pairs carry no gradient
  const int64_t r0 = ok0 ? q0 : 0, r1 = ok1 ? q1 : 0;
  const int e0 = ok0 ? p.sel[2 * t] : 0, e1 = ok1 ? p.sel[2 * t + 1] : 0;
  const float w0 = ok0 ? p.w[2 * t] : 0.0f, w1 = ok1 ? p.w[2 * t + 1] : 0.0f;
  const float dw0 = ok0 ? p.dw[r0] : 0.0f, dw1 = ok1 ? p.dw[r1] : 0.0f;
  const float inner = w0 * dw0 + w1 * dw1;
  const float dl0 = w0 * (dw0 - inner), dl1 = w1 * (dw1 - inner);
  const float s0 = ok0 ? 1.0f : 0.0f, s1 = ok1 ? 1.0f : 0.0f;
  if (lane == 0) {
    p.dl[2 * t] = dl0;
    p.dl[2 * t + 1] = dl1;
  }
  for (int c = lane * 8; c < p.d; c += 64 * 8) {
    float a[8], b[8], g0[8], g1[8];
    ld8<LC_FP32>(p.dns, r0 * p.d + c, LC_FP32, a);
    ld8<LC_FP32>(p.dns, r1 * p.d + c, LC_FP32, b);
    ld8<WD>(p.wr, (int64_t)e0 * p.d + c, p.w_dt, g0);
    ld8<WD>(p.wr, (int64_t)e1 * p.d + c, p.w_dt, g1);
#pragma unroll
    for (int i = 0; i < 8; ++i) a[i] = ((s0 * a[i] + s1 * b[i]) + dl0 * g0[i]) + dl1 * g1[i];
    st8<LC_FP32>(p.dn, t * p.d + c, LC_FP32, a);
  }
}

struct RouterGradP {
  const void *n;          // [T, d]
  const int32_t *sel;     // [T, 2]
  const float *dl;        // [T, 2]
  float *partial;         // [nblk][E][d]
  float *g;               // [E, d] gradient bucket
  int64_t T;
  int d, E, n_dt, nblk;
};

// partial[blk][e][i] = sum over the block's tokens of dl(t, e) n[t, i]. A
// thread owns column i for a group of up to 8 experts (grid z), so each n
// value is read once per group rather than once per expert; every sum runs
// over the block's tokens in order.
constexpr int kRouterExpertsPerPass = 8;
template <int ND>  // element type of n
__global__ __launch_bounds__(256) void moe_router_partial_kernel(RouterGradP p) {
  const int i = blockIdx.x * 256 + threadIdx.x;
  const int blk = blockIdx.y, eg = blockIdx.z * kRouterExpertsPerPass;
  const int64_t t0 = (int64_t)blk * kRouterTokensPerBlock;
  const int64_t t1 = min(p.T, t0 + kRouterTokensPerBlock);
  float s[kRouterExpertsPerPass];
#pragma unroll
  for (int k = 0; k < kRouterExpertsPerPass; ++k) s[k] = 0.0f;
  // the block's selections and logit gradients staged in LDS once
  __shared__ int32_t ssel[2 * kRouterTokensPerBlock];
  __shared__ float sdl[2 * kRouterTokensPerBlock];
  for (int j = threadIdx.x; j < 2 * (int)(t1 - t0); j += 256) {
    ssel[j] = p.sel[2 * t0 + j];
    sdl[j] = p.dl[2 * t0 + j];
  }
  __syncthreads();
  if (i >= p.d) return;
#pragma unroll 4
  for (int64_t t = t0; t < t1; ++t) {
    const int tl = (int)(t - t0);
    const int e0 = ssel[2 * tl] - eg, e1 = ssel[2 * tl + 1] - eg;  // (the pair's experts differ)
    const float d0 = sdl[2 * tl], d1 = sdl[2 * tl + 1];
    float x;
    if constexpr (ND == LC_FP32) x = static_cast<const float *>(p.n)[t * p.d + i];
    else if constexpr (ND == LC_BF16) x = (float)static_cast<const __bf16 *>(p.n)[t * p.d + i];
    else x = (float)static_cast<const _Float16 *>(p.n)[t * p.d + i];
#pragma unroll
    for (int k = 0; k < kRouterExpertsPerPass; ++k) {
      const float c = k == e0 ? d0 : (k == e1 ? d1 : 0.0f);
      s[k] += c * x;
    }
  }
#pragma unroll
  for (int k = 0; k < kRouterExpertsPerPass; ++k)
    if (eg + k < p.E) p.partial[((int64_t)blk * p.E + eg + k) * p.d + i] = s[k];
}

__global__ __launch_bounds__(256) void moe_router_final_kernel(RouterGradP p) {
  const int64_t j = (int64_t)blockIdx.x * 256 + threadIdx.x;  // e * d + i
  if (j >= (int64_t)p.E * p.d) return;
  float s = 0.0f;
  for (int b = 0; b < p.nblk; ++b) s += p.partial[(int64_t)b * p.E * p.d + j];
  p.g[j] = p.g[j] + s;
}

unsigned rows_grid(int64_t rows) { return (unsigned)((rows + 3) / 4); }

}  // namespace

static lc_status check_route_args(const lc_moe_args &a) {
  if (a.T <= 0 || a.d <= 0 || a.E < 2 || a.E > 64)
    return fail(LC_ERR_INVALID_ARG, "moe: need T > 0, d > 0 and 2 <= E <= 64");
  if (a.T > INT32_MAX / 2) return fail(LC_ERR_UNSUPPORTED, "moe: too many tokens");
  if (a.d % 8) return fail(LC_ERR_UNSUPPORTED, "moe: d %% 8 != 0");
  return LC_OK;
}

lc_status moe_route_launch(const lc_moe_args &a, hipStream_t s) {
  LC_TRY(check_route_args(a));
  if (!a.n || !a.wr || !a.sel || !a.w || !aligned16(a.n) || !aligned16(a.wr))
    return fail(LC_ERR_INVALID_ARG, "moe route: null or unaligned pointer");
  if (!valid_dtype(a.n_dtype) || !valid_dtype(a.w_dtype))
    return fail(LC_ERR_INVALID_ARG, "moe route: unknown dtype");
  RouteP p{a.n, a.wr, a.sel, a.w, a.T, a.d, a.E, a.n_dtype, a.w_dtype};
  with_dtype(a.n_dtype, [&](auto nd) {
    with_dtype(a.w_dtype, [&](auto wd) {
      hipLaunchKernelGGL((moe_route_kernel<decltype(nd)::value, decltype(wd)::value>),
                         dim3(rows_grid(a.T)), dim3(256), 0, s, p);
    });
  });
  return check_launch("moe_route_kernel");
}

lc_status moe_dispatch_launch(const lc_moe_args &a, hipStream_t s) {
  LC_TRY(check_route_args(a));
  if (!a.sel || !a.w || !a.offsets || !a.perm || !a.wrow || !a.rowpos)
    return fail(LC_ERR_INVALID_ARG, "moe dispatch: null pointer");
  DispatchP p{a.sel, a.w, a.offsets, a.perm, a.rowpos, a.wrow, (int)a.T, a.E};
  hipLaunchKernelGGL(moe_dispatch_kernel, dim3(1), dim3(kDispatchThreads), 0, s, p);
  return check_launch("moe_dispatch_kernel");
}

lc_status moe_gather_launch(const void *src, void *dst, const int32_t *idx, int64_t rows,
                            int64_t row_bytes, hipStream_t s) {
  if (rows <= 0) return LC_OK;
  if (row_bytes % 16 || row_bytes > INT32_MAX || !aligned16(src) || !aligned16(dst))
    return fail(LC_ERR_INVALID_ARG, "moe gather: rows must be 16-byte multiples, aligned");
  GatherP p{static_cast<const char *>(src), static_cast<char *>(dst), idx, rows, (int)row_bytes};
  hipLaunchKernelGGL(moe_gather_kernel, dim3(rows_grid(rows)), dim3(256), 0, s, p);
  return check_launch("moe_gather_kernel");
}

lc_status moe_combine_launch(const void *h, int h_dt, const float *eo, const float *w,
                             const int32_t *rowpos, void *out, int out_dt, int64_t T, int d,
                             hipStream_t s) {
  CombineP p{h, eo, w, rowpos, out, T, d, h_dt, out_dt};
  with_dtype(h_dt, [&](auto hd) {
    with_dtype(out_dt, [&](auto od) {
      hipLaunchKernelGGL((moe_combine_kernel<decltype(hd)::value, decltype(od)::value>),
                         dim3(rows_grid(T)), dim3(256), 0, s, p);
    });
  });
  return check_launch("moe_combine_kernel");
}

lc_status moe_bwd_gather_launch(const void *dy, int dy_dt, const float *eo, const int32_t *perm,
                                const float *wrow, void *dys, int dys_dt, float *dw,
                                int64_t rows, int d, hipStream_t s) {
  BwdGatherP p{dy, eo, perm, wrow, dys, dw, rows, d, dy_dt, dys_dt};
  with_dtype(dy_dt, [&](auto gd) {
    with_dtype(dys_dt, [&](auto sd) {
      hipLaunchKernelGGL((moe_bwd_gather_kernel<decltype(gd)::value, decltype(sd)::value>),
                         dim3(rows_grid(rows)), dim3(256), 0, s, p);
    });
  });
  return check_launch("moe_bwd_gather_kernel");
}

lc_status moe_bwd_combine_launch(const float *dns, const float *dw, const float *w,
                                 const int32_t *sel, const int32_t *rowpos, const void *wr,
                                 int w_dt, float *dl, float *dn, int64_t T, int d,
                                 hipStream_t s) {
  BwdCombineP p{dns, dw, w, sel, rowpos, wr, dl, dn, T, d, w_dt};
  with_dtype(w_dt, [&](auto wd) {
    hipLaunchKernelGGL((moe_bwd_combine_kernel<decltype(wd)::value>), dim3(rows_grid(T)), dim3(256),
                       0, s, p);
  });
  return check_launch("moe_bwd_combine_kernel");
}

lc_status moe_router_grad_launch(const void *n, int n_dt, const int32_t *sel, const float *dl,
                                 float *scratch, size_t scratch_bytes, float *g, int64_t T,
                                 int d, int E, hipStream_t s) {
  const int nblk = (int)((T + kRouterTokensPerBlock - 1) / kRouterTokensPerBlock);
  if (scratch_bytes < moe_router_scratch_size(T, d, E))
    return fail(LC_ERR_WORKSPACE, "moe router gradient: scratch too small");
  RouterGradP p{n, sel, dl, scratch, g, T, d, E, n_dt, nblk};
  with_dtype(n_dt, [&](auto nd) {
    hipLaunchKernelGGL((moe_router_partial_kernel<decltype(nd)::value>),
                       dim3((unsigned)((d + 255) / 256), (unsigned)nblk,
                            (unsigned)((E + kRouterExpertsPerPass - 1) / kRouterExpertsPerPass)),
                       dim3(256), 0, s, p);
  });
  LC_TRY(check_launch("moe_router_partial_kernel"));
  hipLaunchKernelGGL(moe_router_final_kernel, dim3((unsigned)(((int64_t)E * d + 255) / 256)),
                     dim3(256), 0, s, p);
  return check_launch("moe_router_final_kernel");
}

}  // namespace lc

extern "C" {

lc_status lc_moe_route(const lc_moe_args *args, void *stream) {
  if (!args) return lc::fail(LC_ERR_INVALID_ARG, "moe: null args");
  return lc::moe_route_launch(*args, static_cast<hipStream_t>(stream));
}

lc_status lc_moe_dispatch(const lc_moe_args *args, void *stream) {
  if (!args) return lc::fail(LC_ERR_INVALID_ARG, "moe: null args");
  return lc::moe_dispatch_launch(*args, static_cast<hipStream_t>(stream));
}

}  // extern "C"
