// Shared device/host helpers for libchunk's HIP kernels (gfx950 / CDNA4).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>
#include <stddef.h>

#include "libchunk.h"
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

#define LC_TRY(expr)                 \
  do {                               \
    lc_status _st = (expr);          \
    if (_st != LC_OK) return _st;    \
  } while (0)

// ------------------------------------------------------------------ types
typedef uint16_t bf16_t;  // storage of a bfloat16 value
typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8_v;   // MFMA operand
typedef __attribute__((ext_vector_type(16))) float f32x16_v;   // 32x32 MFMA accumulator
typedef __attribute__((ext_vector_type(4))) float f32x4_v;

__device__ __forceinline__ float bf2f(bf16_t b) { return __uint_as_float(uint32_t(b) << 16); }

// float -> bf16, round to nearest even; NaN keeps sign and high payload and is
// made quiet. Written out on the bit pattern so that every caller gets the same
// rounding on every target.
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
lc_status rmsnorm_fwd_launch(int dtype, int64_t T, int64_t d, const void *x, const void *g,
                             float eps, void *n, float *rstd, hipStream_t s);
lc_status rmsnorm_bwd_launch(int dtype, int64_t T, int64_t d, const void *dn, const void *x,
                             const float *rstd, const void *g, const void *dres, void *dx,
                             float *dg_accum, void *scratch, size_t scratch_bytes, hipStream_t s);
lc_status attn_fwd_launch(int dtype, int B, int S, int H, int hd, const void *q, const void *k,
                          const void *v, int64_t ld_qkv, void *o, int64_t ld_o, float *lse,
                          hipStream_t s);
lc_status attn_bwd_launch(int dtype, int B, int S, int H, int hd, const void *q, const void *k,
                          const void *v, int64_t ld_qkv, const void *o, const void *dout,
                          int64_t ld_o, const float *lse, void *dq, void *dk, void *dv,
                          int64_t ld_dqkv, const float *rcos, const float *rsin, void *scratch,
                          size_t scratch_bytes, hipStream_t s);
lc_status accumulate_launch(float *acc, const void *g, int g_dtype, size_t n, hipStream_t s);
lc_status adam_launch(float *p, float *m, float *v, const void *g, int g_dtype, uint16_t *out,
                      size_t n, const lc_adam_hparams &hp, hipStream_t s);
lc_status cast_bf16_launch(const float *in, uint16_t *out, size_t n, hipStream_t s);

}  // namespace lc
