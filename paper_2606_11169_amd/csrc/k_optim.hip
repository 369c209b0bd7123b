// Bandwidth-bound kernels over flat buffers: gradient accumulation into the
// bucket, the fused AdamW shard step with its bf16 cast, and the plain cast.
//
// Piper keeps one flat gradient buffer per bucket and accumulates microbatch
// gradients into it; under ZeRO-1 each rank steps the optimizer state of its
// own shard (Piper Section 4.3.2 "Memory management", Section 6.2).
//
// Every element is read and written exactly once per call. Each thread
// handles 8 consecutive elements with 16-byte loads/stores (two float4 per
// fp32 stream, one uint4 per bf16 stream); threads of the first workgroup
// also take the n % 8 tail one element each. This file is compiled with
// -ffp-contract=off: every multiply and add below is its own IEEE fp32
// operation, the divide is the correctly rounded one and the square root is
// made correctly rounded by sqrt_rn, so the results are bitwise those of the
// written-out operation sequence.
#include "common.hpp"

#include <math.h>

namespace lc {
namespace {

constexpr int VEC = 8;
constexpr int NTH = 256;

__device__ __forceinline__ void load8(const float *p, float (&x)[8]) {
  const float4 a = reinterpret_cast<const float4 *>(p)[0];
  const float4 b = reinterpret_cast<const float4 *>(p)[1];
  x[0] = a.x; x[1] = a.y; x[2] = a.z; x[3] = a.w;
  x[4] = b.x; x[5] = b.y; x[6] = b.z; x[7] = b.w;
}
__device__ __forceinline__ void load8(const bf16_t *p, float (&x)[8]) {
  const uint4 a = *reinterpret_cast<const uint4 *>(p);
  const uint32_t w[4] = {a.x, a.y, a.z, a.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    x[2 * i] = __uint_as_float(w[i] << 16);
    x[2 * i + 1] = __uint_as_float(w[i] & 0xFFFF0000u);
  }
}
__device__ __forceinline__ void store8(float *p, const float (&x)[8]) {
  reinterpret_cast<float4 *>(p)[0] = make_float4(x[0], x[1], x[2], x[3]);
  reinterpret_cast<float4 *>(p)[1] = make_float4(x[4], x[5], x[6], x[7]);
}
__device__ __forceinline__ void store8_bf16(bf16_t *p, const float (&x)[8]) {
  uint4 a;
  a.x = pack_bf2(x[0], x[1]);
  a.y = pack_bf2(x[2], x[3]);
  a.z = pack_bf2(x[4], x[5]);
  a.w = pack_bf2(x[6], x[7]);
  *reinterpret_cast<uint4 *>(p) = a;
}

template <typename G>
__global__ __launch_bounds__(NTH) void accumulate_kernel(float *__restrict__ acc,
                                                         const G *__restrict__ g, size_t n) {
  const size_t nv = n / VEC;
  const size_t i = (size_t)blockIdx.x * NTH + threadIdx.x;
  if (i < nv) {
    float a[8], b[8];
    load8(acc + i * VEC, a);
    load8(g + i * VEC, b);
#pragma unroll
    for (int e = 0; e < 8; ++e) a[e] = a[e] + b[e];
    store8(acc + i * VEC, a);
  }
  if (blockIdx.x == 0 && threadIdx.x < n - nv * VEC) {
    const size_t t = nv * VEC + threadIdx.x;
    acc[t] = acc[t] + ld_elem(g + t);
  }
}

__global__ __launch_bounds__(NTH) void fill_zero_kernel(float *__restrict__ p, size_t n) {
  const size_t nv = n / VEC;
  const size_t i = (size_t)blockIdx.x * NTH + threadIdx.x;
  if (i < nv) {
    const float z[8] = {0.0f, 0.0f, 0.0f, 0.0f, 0.0f, 0.0f, 0.0f, 0.0f};
    store8(p + i * VEC, z);
  }
  if (blockIdx.x == 0 && threadIdx.x < n - nv * VEC) p[nv * VEC + threadIdx.x] = 0.0f;
}

struct AdamS {
  float c_wd, b1, b2, omb1, omb2, step_size, bc2s, eps;
};

// Correctly rounded fp32 square root. The hardware estimate s (v_sqrt_f32,
// within 1 ulp) is compared with its two neighbours s-, s+ through exact fma
// residuals: sqrt(x) lies below the midpoint of (s-, s) iff x - s- * s <= 0,
// and above the midpoint of (s, s+) iff x - s+ * s > 0 (x - s+- * s is an
// integer multiple of ulp(s)^2, so it can never fall strictly between 0 and
// the midpoint gap). Inputs below 2^-64 are scaled by 2^64 first so that the
// residuals stay normal; the result is scaled back by 2^-32 exactly.
__device__ __forceinline__ float sqrt_rn(float x) {
  const bool tiny = x < 0x1.0p-64f;
  const float xs = tiny ? x * 0x1.0p+64f : x;
  float s = __builtin_amdgcn_sqrtf(xs);
  if (xs > 0.0f && xs < INFINITY) {
    const float dn = __int_as_float(__float_as_int(s) - 1);
    const float up = __int_as_float(__float_as_int(s) + 1);
    const float rdn = __builtin_fmaf(-dn, s, xs);
    const float rup = __builtin_fmaf(-up, s, xs);
    if (rdn <= 0.0f) s = dn;
    if (rup > 0.0f) s = up;
  }
  return tiny ? s * 0x1.0p-32f : s;
}

__device__ __forceinline__ void adam_elem(float &p, float &m, float &v, float g, const AdamS &s) {
  p = p * s.c_wd;
  const float m1 = s.b1 * m;
  const float m2 = s.omb1 * g;
  m = m1 + m2;
  const float gg = g * g;
  const float v1 = s.b2 * v;
  const float v2 = s.omb2 * gg;
  v = v1 + v2;
  const float den = __fadd_rn(__fdiv_rn(sqrt_rn(v), s.bc2s), s.eps);
  const float upd = s.step_size * __fdiv_rn(m, den);
  p = p - upd;
}

template <typename G, bool CAST>
__global__ __launch_bounds__(NTH) void adam_kernel(float *__restrict__ P, float *__restrict__ Mo,
                                                   float *__restrict__ V,
                                                   const G *__restrict__ Gr,
                                                   bf16_t *__restrict__ out, size_t n, AdamS s) {
  const size_t nv = n / VEC;
  const size_t i = (size_t)blockIdx.x * NTH + threadIdx.x;
  if (i < nv) {
    float p[8], m[8], v[8], g[8];
    load8(P + i * VEC, p);
    load8(Mo + i * VEC, m);
    load8(V + i * VEC, v);
    load8(Gr + i * VEC, g);
#pragma unroll
    for (int e = 0; e < 8; ++e) adam_elem(p[e], m[e], v[e], g[e], s);
    store8(P + i * VEC, p);
    store8(Mo + i * VEC, m);
    store8(V + i * VEC, v);
    if (CAST) store8_bf16(out + i * VEC, p);
  }
  if (blockIdx.x == 0 && threadIdx.x < n - nv * VEC) {
    const size_t t = nv * VEC + threadIdx.x;
    float p = P[t], m = Mo[t], v = V[t];
    adam_elem(p, m, v, ld_elem(Gr + t), s);
    P[t] = p;
    Mo[t] = m;
    V[t] = v;
    if (CAST) out[t] = f2bf(p);
  }
}

__global__ __launch_bounds__(NTH) void cast_kernel(const float *__restrict__ in,
                                                   bf16_t *__restrict__ out, size_t n) {
  const size_t nv = n / VEC;
  const size_t i = (size_t)blockIdx.x * NTH + threadIdx.x;
  if (i < nv) {
    float x[8];
    load8(in + i * VEC, x);
    store8_bf16(out + i * VEC, x);
  }
  if (blockIdx.x == 0 && threadIdx.x < n - nv * VEC) out[nv * VEC + threadIdx.x] = f2bf(in[nv * VEC + threadIdx.x]);
}

// One pass: one 8-element block per thread (a measured 9% more bandwidth than
// a grid-stride loop over resident workgroups); the first workgroup also
// covers the n % 8 tail.
unsigned stream_grid(size_t n) {
  const size_t want = (n / VEC + NTH - 1) / NTH;
  return (unsigned)(want < 1 ? 1 : want);
}

// a dispatch counts work-items in 32 bits: at most 2^32 - 1 threads
lc_status check_n(size_t n, const char *what) {
  if ((n / VEC + NTH) >= (size_t)0xFFFFFFFFu)
    return fail(LC_ERR_UNSUPPORTED, "%s: n = %zu exceeds one dispatch (8 * (2^32 - 256) elements)", what, n);
  return LC_OK;
}

}  // namespace

lc_status accumulate_launch(float *acc, const void *g, int g_dtype, size_t n, hipStream_t s) {
  if (n == 0) return LC_OK;
  if (!acc || !g) return fail(LC_ERR_INVALID_ARG, "accumulate: null pointer");
  if (!aligned16(acc) || !aligned16(g)) return fail(LC_ERR_INVALID_ARG, "accumulate: unaligned");
  LC_TRY(check_n(n, "accumulate"));
  const size_t gb = g_dtype == LC_BF16 ? 2 : 4;
  const char *a0 = reinterpret_cast<const char *>(acc), *g0 = static_cast<const char *>(g);
  if (a0 < g0 + n * gb && g0 < a0 + n * 4)
    return fail(LC_ERR_INVALID_ARG, "accumulate: accum and g overlap");
  if (g_dtype == LC_FP32) {
    hipLaunchKernelGGL(accumulate_kernel<float>, dim3(stream_grid(n)), dim3(NTH), 0, s, acc,
                       static_cast<const float *>(g), n);
  } else if (g_dtype == LC_BF16) {
    hipLaunchKernelGGL(accumulate_kernel<bf16_t>, dim3(stream_grid(n)), dim3(NTH), 0, s, acc,
                       static_cast<const bf16_t *>(g), n);
  } else {
    return fail(LC_ERR_INVALID_ARG, "accumulate: unknown dtype %d", g_dtype);
  }
  return check_launch("accumulate_kernel");
}

lc_status zero_fill_launch(float *buf, size_t n, hipStream_t s) {
  if (n == 0) return LC_OK;
  if (!buf || !aligned16(buf)) return fail(LC_ERR_INVALID_ARG, "zero fill: null or unaligned buffer");
  LC_TRY(check_n(n, "zero fill"));
  hipLaunchKernelGGL(fill_zero_kernel, dim3(stream_grid(n)), dim3(NTH), 0, s, buf, n);
  return check_launch("fill_zero_kernel");
}

lc_status adam_launch(float *p, float *m, float *v, const void *g, int g_dtype, uint16_t *out,
                      size_t n, const lc_adam_hparams &hp, hipStream_t s) {
  if (n == 0) return LC_OK;
  if (!p || !m || !v || !g) return fail(LC_ERR_INVALID_ARG, "adam: null pointer");
  if (!aligned16(p) || !aligned16(m) || !aligned16(v) || !aligned16(g) || (out && !aligned16(out)))
    return fail(LC_ERR_INVALID_ARG, "adam: pointers must be 16-byte aligned");
  if (hp.step < 1) return fail(LC_ERR_INVALID_ARG, "adam: step must be >= 1");
  LC_TRY(check_n(n, "adam"));
  if (g_dtype != LC_FP32 && g_dtype != LC_BF16)
    return fail(LC_ERR_INVALID_ARG, "adam: unknown grad dtype %d", g_dtype);
  // host scalars: double precision from the float hyper-parameters, rounded once
  const double lr = hp.lr, b1 = hp.beta1, b2 = hp.beta2, wd = hp.weight_decay;
  const double t = (double)hp.step;
  AdamS sc;
  sc.c_wd = (float)(1.0 - lr * wd);
  sc.b1 = hp.beta1;
  sc.b2 = hp.beta2;
  sc.omb1 = (float)(1.0 - b1);
  sc.omb2 = (float)(1.0 - b2);
  sc.step_size = (float)(lr / (1.0 - pow(b1, t)));
  sc.bc2s = (float)sqrt(1.0 - pow(b2, t));
  sc.eps = hp.eps;
  const dim3 grid(stream_grid(n)), block(NTH);
  if (g_dtype == LC_FP32) {
    const float *gp = static_cast<const float *>(g);
    if (out) hipLaunchKernelGGL((adam_kernel<float, true>), grid, block, 0, s, p, m, v, gp, out, n, sc);
    else hipLaunchKernelGGL((adam_kernel<float, false>), grid, block, 0, s, p, m, v, gp, out, n, sc);
  } else {
    const bf16_t *gp = static_cast<const bf16_t *>(g);
    if (out) hipLaunchKernelGGL((adam_kernel<bf16_t, true>), grid, block, 0, s, p, m, v, gp, out, n, sc);
    else hipLaunchKernelGGL((adam_kernel<bf16_t, false>), grid, block, 0, s, p, m, v, gp, out, n, sc);
  }
  return check_launch("adam_kernel");
}

lc_status cast_bf16_launch(const float *in, uint16_t *out, size_t n, hipStream_t s) {
  if (n == 0) return LC_OK;
  if (!in || !out || !aligned16(in) || !aligned16(out))
    return fail(LC_ERR_INVALID_ARG, "cast: null or unaligned pointer");
  LC_TRY(check_n(n, "cast"));
  hipLaunchKernelGGL(cast_kernel, dim3(stream_grid(n)), dim3(NTH), 0, s, in, out, n);
  return check_launch("cast_kernel");
}

}  // namespace lc

extern "C" {

lc_status chunk_accumulate_grad(float *accum, const void *g, int32_t g_dtype, size_t n,
                                void *stream) {
  return lc::accumulate_launch(accum, g, g_dtype, n, static_cast<hipStream_t>(stream));
}

lc_status lc_zero_fill_f32(float *buf, size_t n, void *stream) {
  return lc::zero_fill_launch(buf, n, static_cast<hipStream_t>(stream));
}

lc_status shard_adam_step(float *master, float *m, float *v, const void *grad, int32_t grad_dtype,
                          uint16_t *out_bf16, size_t n, const lc_adam_hparams *hp, void *stream) {
  if (!hp) return lc::fail(LC_ERR_INVALID_ARG, "adam: null hyper-parameters");
  return lc::adam_launch(master, m, v, grad, grad_dtype, out_bf16, n, *hp,
                         static_cast<hipStream_t>(stream));
}

lc_status lc_cast_bf16(const float *in, uint16_t *out, size_t n, void *stream) {
  return lc::cast_bf16_launch(in, out, n, static_cast<hipStream_t>(stream));
}

}  // extern "C"
