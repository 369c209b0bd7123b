// RMSNorm forward and backward (HBM-bound row kernels).
//
//   forward:  rstd_t = 1/sqrt(mean_k x_tk^2 + eps),  n_tk = x_tk * rstd_t * g_k
//   backward: xh = x*rstd, dxh = dn*g,
//             dx_tk = dres_tk + rstd_t (dxh_tk - xh_tk * mean_k(dxh*xh)),
//             dg_k += sum_t dn_tk xh_tk
//
// Row kernels: one wave per row, 16-byte vector accesses (8 bf16 or 4 fp32
// per lane per step); a row is read once for its reduction and again for the
// write (the second read hits L2). The gain gradient is a column reduction over
// rows: blocks of kNormRowsPerBlock rows write fp32 partial sums, then one
// thread per column adds the partials in block order into dg — the same
// order on every run, no atomics.
#include "common.hpp"

namespace lc {
namespace {

template <typename T> struct Vec;  // 16 bytes of T, as floats
template <> struct Vec<bf16_t> {
  static constexpr int N = 8;
  __device__ static void load(const bf16_t *p, float (&x)[8]) {
    const uint4 a = *reinterpret_cast<const uint4 *>(p);
    const uint32_t w[4] = {a.x, a.y, a.z, a.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      x[2 * i] = __uint_as_float(w[i] << 16);
      x[2 * i + 1] = __uint_as_float(w[i] & 0xFFFF0000u);
    }
  }
  __device__ static void store(bf16_t *p, const float (&x)[8]) {
    uint4 a;
    a.x = pack_bf2(x[0], x[1]);
    a.y = pack_bf2(x[2], x[3]);
    a.z = pack_bf2(x[4], x[5]);
    a.w = pack_bf2(x[6], x[7]);
    *reinterpret_cast<uint4 *>(p) = a;
  }
};
template <> struct Vec<float> {
  static constexpr int N = 4;
  __device__ static void load(const float *p, float (&x)[4]) {
    const float4 a = *reinterpret_cast<const float4 *>(p);
    x[0] = a.x; x[1] = a.y; x[2] = a.z; x[3] = a.w;
  }
  __device__ static void store(float *p, const float (&x)[4]) {
    *reinterpret_cast<float4 *>(p) = make_float4(x[0], x[1], x[2], x[3]);
  }
};

constexpr int ROWS_PER_BLOCK = 4;  // one wave per row

template <typename T>
__global__ __launch_bounds__(256) void rmsnorm_fwd_kernel(const T *__restrict__ x,
                                                          const T *__restrict__ g, float eps,
                                                          T *__restrict__ n, float *__restrict__ rstd,
                                                          int64_t rows, int d) {
  constexpr int V = Vec<T>::N;
  const int lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * ROWS_PER_BLOCK + (threadIdx.x >> 6);
  if (row >= rows) return;
  const T *xr = x + row * d;
  float ss = 0.0f;
  for (int c = lane * V; c < d; c += 64 * V) {
    float v[V];
    Vec<T>::load(xr + c, v);
#pragma unroll
    for (int e = 0; e < V; ++e) ss += v[e] * v[e];
  }
  ss = wave_sum(ss);
  const float r = 1.0f / sqrtf(ss / (float)d + eps);
  if (lane == 0) rstd[row] = r;
  T *nr = n + row * d;
  for (int c = lane * V; c < d; c += 64 * V) {
    float v[V], gv[V];
    Vec<T>::load(xr + c, v);
    Vec<T>::load(g + c, gv);
#pragma unroll
    for (int e = 0; e < V; ++e) v[e] = v[e] * r * gv[e];
    Vec<T>::store(nr + c, v);
  }
}

template <typename T>
__global__ __launch_bounds__(256) void rmsnorm_bwd_rows_kernel(
    const T *__restrict__ dn, const T *__restrict__ x, const float *__restrict__ rstd,
    const T *__restrict__ g, const T *__restrict__ dres, T *__restrict__ dx, int64_t rows, int d) {
  constexpr int V = Vec<T>::N;
  const int lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * ROWS_PER_BLOCK + (threadIdx.x >> 6);
  if (row >= rows) return;
  const T *dnr = dn + row * d;
  const T *xr = x + row * d;
  const float r = rstd[row];
  float dot = 0.0f;  // sum_k dn*g*x
  for (int c = lane * V; c < d; c += 64 * V) {
    float a[V], b[V], gv[V];
    Vec<T>::load(dnr + c, a);
    Vec<T>::load(xr + c, b);
    Vec<T>::load(g + c, gv);
#pragma unroll
    for (int e = 0; e < V; ++e) dot += a[e] * gv[e] * b[e];
  }
  dot = wave_sum(dot);
  const float mean = dot * r / (float)d;  // mean_k(dxh * xh)
  const float r2m = r * mean;
  T *dxr = dx + row * d;
  for (int c = lane * V; c < d; c += 64 * V) {
    float a[V], b[V], gv[V], o[V];
    Vec<T>::load(dnr + c, a);
    Vec<T>::load(xr + c, b);
    Vec<T>::load(g + c, gv);
    if (dres) {
      Vec<T>::load(dres + row * d + c, o);
    } else {
#pragma unroll
      for (int e = 0; e < V; ++e) o[e] = 0.0f;
    }
#pragma unroll
    for (int e = 0; e < V; ++e) o[e] += r * (a[e] * gv[e] - b[e] * r2m);
    Vec<T>::store(dxr + c, o);
  }
}

// partial[blk][k] = sum over rows of block blk of dn[t,k] * x[t,k] * rstd[t]
template <typename T>
__global__ __launch_bounds__(256) void rmsnorm_dg_partial_kernel(const T *__restrict__ dn,
                                                                 const T *__restrict__ x,
                                                                 const float *__restrict__ rstd,
                                                                 float *__restrict__ partial,
                                                                 int64_t rows, int d) {
  const int k = blockIdx.x * 256 + threadIdx.x;
  if (k >= d) return;
  const int64_t r0 = (int64_t)blockIdx.y * kNormRowsPerBlock;
  const int64_t r1 = min(rows, r0 + kNormRowsPerBlock);
  float s = 0.0f;
  for (int64_t t = r0; t < r1; ++t) s += ld_elem(dn + t * d + k) * (ld_elem(x + t * d + k) * rstd[t]);
  partial[(int64_t)blockIdx.y * d + k] = s;
}

__global__ __launch_bounds__(256) void rmsnorm_dg_final_kernel(const float *__restrict__ partial,
                                                               int nblk, int d,
                                                               float *__restrict__ dg) {
  const int k = blockIdx.x * 256 + threadIdx.x;
  if (k >= d) return;
  float s = 0.0f;
  for (int b = 0; b < nblk; ++b) s += partial[(int64_t)b * d + k];
  dg[k] = dg[k] + s;
}

}  // namespace

lc_status rmsnorm_fwd_launch(int dtype, int64_t T, int64_t d, const void *x, const void *g,
                             float eps, void *n, float *rstd, hipStream_t s) {
  if (T <= 0 || d <= 0) return fail(LC_ERR_INVALID_ARG, "rmsnorm: T and d must be positive");
  if (!x || !g || !n || !rstd) return fail(LC_ERR_INVALID_ARG, "rmsnorm: null pointer");
  if (!aligned16(x) || !aligned16(g) || !aligned16(n))
    return fail(LC_ERR_INVALID_ARG, "rmsnorm: unaligned pointer");
  const int vec = dtype == LC_BF16 ? 8 : 4;
  if (d % vec) return fail(LC_ERR_UNSUPPORTED, "rmsnorm: d %% %d != 0", vec);
  if (d > INT32_MAX) return fail(LC_ERR_UNSUPPORTED, "rmsnorm: d too large");
  const dim3 grid((unsigned)((T + ROWS_PER_BLOCK - 1) / ROWS_PER_BLOCK));
  if (dtype == LC_BF16) {
    hipLaunchKernelGGL(rmsnorm_fwd_kernel<bf16_t>, grid, dim3(256), 0, s,
                       static_cast<const bf16_t *>(x), static_cast<const bf16_t *>(g), eps,
                       static_cast<bf16_t *>(n), rstd, T, (int)d);
  } else if (dtype == LC_FP32) {
    hipLaunchKernelGGL(rmsnorm_fwd_kernel<float>, grid, dim3(256), 0, s,
                       static_cast<const float *>(x), static_cast<const float *>(g), eps,
                       static_cast<float *>(n), rstd, T, (int)d);
  } else {
    return fail(LC_ERR_INVALID_ARG, "rmsnorm: unknown dtype");
  }
  return check_launch("rmsnorm_fwd_kernel");
}

lc_status rmsnorm_bwd_launch(int dtype, int64_t T, int64_t d, const void *dn, const void *x,
                             const float *rstd, const void *g, const void *dres, void *dx,
                             float *dg_accum, void *scratch, size_t scratch_bytes, hipStream_t s) {
  if (T <= 0 || d <= 0) return fail(LC_ERR_INVALID_ARG, "rmsnorm: T and d must be positive");
  if (!dn || !x || !rstd || !g || !dx) return fail(LC_ERR_INVALID_ARG, "rmsnorm: null pointer");
  if (!aligned16(dn) || !aligned16(x) || !aligned16(g) || !aligned16(dx) ||
      (dres && !aligned16(dres)))
    return fail(LC_ERR_INVALID_ARG, "rmsnorm: unaligned pointer");
  const int vec = dtype == LC_BF16 ? 8 : 4;
  if (d % vec) return fail(LC_ERR_UNSUPPORTED, "rmsnorm: d %% %d != 0", vec);
  if (d > INT32_MAX) return fail(LC_ERR_UNSUPPORTED, "rmsnorm: d too large");
  if (dg_accum && (!scratch || scratch_bytes < rmsnorm_scratch_size(T, d)))
    return fail(LC_ERR_WORKSPACE, "rmsnorm: scratch smaller than lc_rmsnorm_scratch_bytes");
  const dim3 grid((unsigned)((T + ROWS_PER_BLOCK - 1) / ROWS_PER_BLOCK));
  const int nblk = (int)((T + kNormRowsPerBlock - 1) / kNormRowsPerBlock);
  const dim3 pgrid((unsigned)((d + 255) / 256), (unsigned)nblk);
  float *partial = static_cast<float *>(scratch);
  if (dtype == LC_BF16) {
    hipLaunchKernelGGL(rmsnorm_bwd_rows_kernel<bf16_t>, grid, dim3(256), 0, s,
                       static_cast<const bf16_t *>(dn), static_cast<const bf16_t *>(x), rstd,
                       static_cast<const bf16_t *>(g), static_cast<const bf16_t *>(dres),
                       static_cast<bf16_t *>(dx), T, (int)d);
    LC_TRY(check_launch("rmsnorm_bwd_rows_kernel"));
    if (dg_accum)
      hipLaunchKernelGGL(rmsnorm_dg_partial_kernel<bf16_t>, pgrid, dim3(256), 0, s,
                         static_cast<const bf16_t *>(dn), static_cast<const bf16_t *>(x), rstd,
                         partial, T, (int)d);
  } else if (dtype == LC_FP32) {
    hipLaunchKernelGGL(rmsnorm_bwd_rows_kernel<float>, grid, dim3(256), 0, s,
                       static_cast<const float *>(dn), static_cast<const float *>(x), rstd,
                       static_cast<const float *>(g), static_cast<const float *>(dres),
                       static_cast<float *>(dx), T, (int)d);
    LC_TRY(check_launch("rmsnorm_bwd_rows_kernel"));
    if (dg_accum)
      hipLaunchKernelGGL(rmsnorm_dg_partial_kernel<float>, pgrid, dim3(256), 0, s,
                         static_cast<const float *>(dn), static_cast<const float *>(x), rstd,
                         partial, T, (int)d);
  } else {
    return fail(LC_ERR_INVALID_ARG, "rmsnorm: unknown dtype");
  }
  if (!dg_accum) return LC_OK;
  LC_TRY(check_launch("rmsnorm_dg_partial_kernel"));
  hipLaunchKernelGGL(rmsnorm_dg_final_kernel, dim3((unsigned)((d + 255) / 256)), dim3(256), 0, s,
                     partial, nblk, (int)d, dg_accum);
  return check_launch("rmsnorm_dg_final_kernel");
}

}  // namespace lc

extern "C" {

lc_status lc_rmsnorm_forward(int32_t dtype, int64_t T, int64_t d, const void *x, const void *g,
                             float eps, void *n, float *rstd, void *stream) {
  return lc::rmsnorm_fwd_launch(dtype, T, d, x, g, eps, n, rstd, static_cast<hipStream_t>(stream));
}

lc_status lc_rmsnorm_backward(int32_t dtype, int64_t T, int64_t d, const void *dn, const void *x,
                              const float *rstd, const void *g, const void *dres, void *dx,
                              float *dg_accum, void *scratch, size_t scratch_bytes, void *stream) {
  return lc::rmsnorm_bwd_launch(dtype, T, d, dn, x, rstd, g, dres, dx, dg_accum, scratch,
                                scratch_bytes, static_cast<hipStream_t>(stream));
}

}  // extern "C"
