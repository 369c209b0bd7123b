// Shared device/host helpers for libchunk's HIP kernels (gfx950 / CDNA4).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>
#include <stddef.h>

#include "libchunk.h"

#include <type_traits>
#include "libchunk_ops.h"
#include "host_core.hpp"

namespace lc {

// ------------------------------------------------------------------ errors
lc_status hip_fail(hipError_t e, const char *what);
inline lc_status check_launch(const char *what) {
  hipError_t e = hipGetLastError();
  return e == hipSuccess ? LC_OK : hip_fail(e, what);
}
inline bool aligned16(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }
inline size_t dtype_size(int dt) { return dt == LC_FP32 ? 4 : 2; }
inline bool valid_dtype(int dt) { return dt == LC_FP32 || dt == LC_BF16 || dt == LC_FP16; }

// ------------------------------------------------------------------ types
typedef uint16_t bf16_t;  // storage of a bfloat16 value (bit-exact paths)
typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8_v;     // MFMA operand
typedef __attribute__((ext_vector_type(8))) _Float16 f16x8_v;    // MFMA operand
typedef __attribute__((ext_vector_type(4))) __bf16 bf16x4_v;
typedef __attribute__((ext_vector_type(4))) _Float16 f16x4_v;
typedef __attribute__((ext_vector_type(16))) float f32x16_v;     // 32x32 MFMA accumulator
typedef __attribute__((ext_vector_type(4))) float f32x4_v;

__device__ __forceinline__ float bf2f(bf16_t b) { return __uint_as_float(uint32_t(b) << 16); }

// float -> bf16, round to nearest even; NaN keeps sign and high payload and is
// made quiet. Written out on the bit pattern: the bit-exact kernels (AdamW's
// cast, lc_cast_bf16) use this one.
__device__ __forceinline__ bf16_t f2bf(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7FFFFFFFu) > 0x7F800000u) return bf16_t((u >> 16) | 0x0040u);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return bf16_t(u >> 16);
}

__device__ __forceinline__ uint32_t pack_bf2(float lo, float hi) {
  return uint32_t(f2bf(lo)) | (uint32_t(f2bf(hi)) << 16);
}

// element access generic over the storage type (float or bf16_t)
template <typename T> __device__ __forceinline__ float ld_elem(const T *p);
template <> __device__ __forceinline__ float ld_elem<float>(const float *p) { return *p; }
template <> __device__ __forceinline__ float ld_elem<bf16_t>(const bf16_t *p) { return bf2f(*p); }
template <typename T> __device__ __forceinline__ void st_elem(T *p, float v);
template <> __device__ __forceinline__ void st_elem<float>(float *p, float v) { *p = v; }
template <> __device__ __forceinline__ void st_elem<bf16_t>(bf16_t *p, float v) { *p = f2bf(v); }

// Four consecutive elements of a tensor whose type is known at run time
// (uniform across the wave): 8 bytes for bf16/fp16 (hardware round-to-nearest-
// even conversions), 16 bytes for fp32.
__device__ __forceinline__ void store4_dt(void *base, int64_t idx, int dt, float a, float b,
                                          float c, float d) {
  if (dt == LC_FP32) {
    *reinterpret_cast<float4 *>(static_cast<float *>(base) + idx) = make_float4(a, b, c, d);
  } else if (dt == LC_BF16) {
    bf16x4_v v = {(__bf16)a, (__bf16)b, (__bf16)c, (__bf16)d};
    *reinterpret_cast<bf16x4_v *>(static_cast<__bf16 *>(base) + idx) = v;
  } else {
    f16x4_v v = {(_Float16)a, (_Float16)b, (_Float16)c, (_Float16)d};
    *reinterpret_cast<f16x4_v *>(static_cast<_Float16 *>(base) + idx) = v;
  }
}

__device__ __forceinline__ float4 load4_dt(const void *base, int64_t idx, int dt) {
  if (dt == LC_FP32) return *reinterpret_cast<const float4 *>(static_cast<const float *>(base) + idx);
  if (dt == LC_BF16) {
    const bf16x4_v v = *reinterpret_cast<const bf16x4_v *>(static_cast<const __bf16 *>(base) + idx);
    return make_float4((float)v[0], (float)v[1], (float)v[2], (float)v[3]);
  }
  const f16x4_v v = *reinterpret_cast<const f16x4_v *>(static_cast<const _Float16 *>(base) + idx);
  return make_float4((float)v[0], (float)v[1], (float)v[2], (float)v[3]);
}

// Eight consecutive elements as floats / from floats (16 or 32 bytes).
__device__ __forceinline__ void load8_dt(const void *base, int64_t idx, int dt, float (&x)[8]) {
  const float4 a = load4_dt(base, idx, dt), b = load4_dt(base, idx + 4, dt);
  x[0] = a.x; x[1] = a.y; x[2] = a.z; x[3] = a.w;
  x[4] = b.x; x[5] = b.y; x[6] = b.z; x[7] = b.w;
}
__device__ __forceinline__ void store8_dt(void *base, int64_t idx, int dt, const float (&x)[8]) {
  store4_dt(base, idx, dt, x[0], x[1], x[2], x[3]);
  store4_dt(base, idx + 4, dt, x[4], x[5], x[6], x[7]);
}

// 8 consecutive values of a tensor whose element type is the template
// argument DT, or the run-time value rt when DT < 0: with a compile-time type
// the accesses are straight-line code, which lets the compiler keep several
// loads in flight instead of waiting at the type branches
template <int DT>
__device__ __forceinline__ void ld8(const void *base, int64_t idx, int rt, float (&x)[8]) {
  load8_dt(base, idx, DT < 0 ? rt : DT, x);
}
template <int DT>
__device__ __forceinline__ void st8(void *base, int64_t idx, int rt, const float (&x)[8]) {
  store8_dt(base, idx, DT < 0 ? rt : DT, x);
}

// Calls f with the element type dt as a compile-time constant
// (std::integral_constant<int, dt>); dt must be a valid lc_dtype.
template <typename F>
inline void with_dtype(int dt, F f) {
  if (dt == LC_FP32) f(std::integral_constant<int, LC_FP32>{});
  else if (dt == LC_BF16) f(std::integral_constant<int, LC_BF16>{});
  else f(std::integral_constant<int, LC_FP16>{});
}

// logistic sigmoid with the hardware reciprocal (about 1 ulp); used in
// activation epilogues whose results are rounded to bf16 or checked at 1e-4
__device__ __forceinline__ float sigmoidf_(float z) {
  return __builtin_amdgcn_rcpf(1.0f + __expf(-z));
}

// wave-wide reductions (64 lanes)
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

inline unsigned ceil_div(size_t a, size_t b) { return unsigned((a + b - 1) / b); }

// ------------------------------------------------------------------ internal launchers
// Defined in the kernel translation units; used by the stage composer.
lc_status gemm_launch(const lc_gemm_args &a, hipStream_t s);
lc_status zero_fill_launch(float *buf, size_t n, hipStream_t s);
lc_status rmsnorm_fwd_launch(const lc_norm_args &a, hipStream_t s);
lc_status rmsnorm_bwd_launch(const lc_norm_args &a, hipStream_t s);
// The backward's row pass only: dx (and dx_copy) and the gain-gradient
// partial sums in a.scratch (a.dg_accum is ignored) ...
lc_status rmsnorm_bwd_partials_launch(const lc_norm_args &a, hipStream_t s);
// ... and, later, dg[k] += the sum of those partials in the order
// rmsnorm_bwd_launch uses, for the same T and d (dg[k] = the sum if store).
lc_status rmsnorm_dg_final_launch(const float *partial, float *dg, int64_t T, int64_t d,
                                  hipStream_t s, bool store = false);
lc_status qknorm_fwd_launch(const lc_qknorm_args &a, hipStream_t s);
// the backward's rows and gain partial sums (a.dgq, a.dgk unused) ...
lc_status qknorm_bwd_partials_launch(const lc_qknorm_args &a, hipStream_t s);
// ... and the ordered sum of those partials into (or, with store, onto) dgq, dgk
lc_status qknorm_dg_final_launch(const float *partial, float *dgq, float *dgk, int64_t T, int hd,
                                 bool store, hipStream_t s);
lc_status attn_fwd_launch(const lc_attn_args &a, hipStream_t s);
lc_status attn_bwd_launch(const lc_attn_args &a, hipStream_t s);
lc_status accumulate_launch(float *acc, const void *g, int g_dtype, size_t n, hipStream_t s);
lc_status adam_launch(float *p, float *m, float *v, const void *g, int g_dtype, uint16_t *out,
                      size_t n, const lc_adam_hparams &hp, hipStream_t s);
lc_status cast_bf16_launch(const float *in, uint16_t *out, size_t n, hipStream_t s);
lc_status moe_route_launch(const lc_moe_args &a, hipStream_t s);
lc_status moe_dispatch_launch(const lc_moe_args &a, hipStream_t s);
lc_status moe_gather_launch(const void *src, void *dst, const int32_t *idx, int64_t rows,
                            int64_t row_bytes, hipStream_t s);
lc_status moe_combine_launch(const void *h, int h_dt, const float *eo, const float *w,
                             const int32_t *rowpos, void *out, int out_dt, int64_t T, int d,
                             hipStream_t s);
lc_status moe_bwd_gather_launch(const void *dy, int dy_dt, const float *eo, const int32_t *perm,
                                const float *wrow, void *dys, int dys_dt, float *dw,
                                int64_t rows, int d, hipStream_t s);
lc_status moe_bwd_combine_launch(const float *dns, const float *dw, const float *w,
                                 const int32_t *sel, const int32_t *rowpos, const void *wr,
                                 int w_dt, float *dl, float *dn, int64_t T, int d,
                                 hipStream_t s);
lc_status moe_router_grad_launch(const void *n, int n_dt, const int32_t *sel, const float *dl,
                                 float *scratch, size_t scratch_bytes, float *g, int64_t T,
                                 int d, int E, hipStream_t s);

}  // namespace lc
