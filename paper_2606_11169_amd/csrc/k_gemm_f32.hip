// fp32 GEMM path (fp32-compute stages): LDS-tiled FMA kernel, 64 x 64 tile,
// 256 threads with 4 x 4 outputs each, with the same operand layouts and
// epilogues as the bf16 matrix-core kernel. RoPE and the SwiGLU gate are
// applied by small elementwise kernels after the product (these stages are
// tiny and launch-bound; none of this path is on the bf16 hot path).
#include "common.hpp"

namespace lc {
namespace {

constexpr int TM = 64, TN = 64, TK = 16;

struct F32P {
  const float *A;
  const float *B;
  float *C;
  const float *R;
  const float *aux0;
  const float *aux1;
  int64_t lda, ldb, ldc, ldr, ld_aux;
  int M, N, K;
  int a_k, b_k;
  int epi;
};

__global__ __launch_bounds__(256) void gemm_f32_kernel(F32P p) {
  __shared__ float As[TK][TM + 4];
  __shared__ float Bs[TK][TN + 4];
  const int tid = threadIdx.x;
  const int tx = tid & 15, ty = tid >> 4;
  const int m0 = blockIdx.y * TM, n0 = blockIdx.x * TN;
  float acc[4][4] = {};
  for (int k0 = 0; k0 < p.K; k0 += TK) {
    for (int e = tid; e < TM * TK; e += 256) {
      int mm, kk;
      if (p.a_k) { mm = e / TK; kk = e % TK; } else { kk = e / TM; mm = e % TM; }
      const int gm = m0 + mm, gk = k0 + kk;
      float v = 0.0f;
      if (gm < p.M && gk < p.K) v = p.a_k ? p.A[(int64_t)gm * p.lda + gk] : p.A[(int64_t)gk * p.lda + gm];
      As[kk][mm] = v;
    }
    for (int e = tid; e < TN * TK; e += 256) {
      int nn, kk;
      if (p.b_k) { nn = e / TK; kk = e % TK; } else { kk = e / TN; nn = e % TN; }
      const int gn = n0 + nn, gk = k0 + kk;
      float v = 0.0f;
      if (gn < p.N && gk < p.K) v = p.b_k ? p.B[(int64_t)gn * p.ldb + gk] : p.B[(int64_t)gk * p.ldb + gn];
      Bs[kk][nn] = v;
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < TK; ++kk) {
      float a[4], b[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) a[i] = As[kk][ty * 4 + i];
#pragma unroll
      for (int j = 0; j < 4; ++j) b[j] = Bs[kk][tx * 4 + j];
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(a[i], b[j], acc[i][j]);
    }
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int m = m0 + ty * 4 + i;
    if (m >= p.M) continue;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int n = n0 + tx * 4 + j;
      if (n >= p.N) continue;
      const float v = acc[i][j];
      float *c = p.C + (int64_t)m * p.ldc + n;
      switch (p.epi) {
        case LC_EPI_ACCUM_F32: *c = *c + v; break;
        case LC_EPI_RESIDUAL: *c = p.R[(int64_t)m * p.ldr + n] + v; break;
        case LC_EPI_SWIGLU_BWD: {
          const float g = p.aux0[(int64_t)m * p.ld_aux + n];
          const float u = p.aux1[(int64_t)m * p.ld_aux + n];
          const float s = sigmoidf_(g);
          c[0] = v * u * s * (1.0f + g * (1.0f - s));
          c[p.N] = v * g * s;
          break;
        }
        default: *c = v; break;
      }
    }
  }
}

// rotate column pairs (i, i + hd/2) of every head below rope_cols
__global__ void rope_f32_kernel(float *C, int64_t ldc, int M, int rope_cols, int hd,
                                const float *rcos, const float *rsin, int rope_seq) {
  const int half = hd / 2;
  const int64_t total = (int64_t)M * (rope_cols / 2);
  for (int64_t e = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; e < total;
       e += (int64_t)gridDim.x * blockDim.x) {
    const int m = (int)(e / (rope_cols / 2));
    const int r = (int)(e % (rope_cols / 2));
    const int head = r / half, i = r % half;
    const int pos = m % rope_seq;
    float *row = C + (int64_t)m * ldc + head * hd;
    const float a = row[i], b = row[i + half];
    const float cs = rcos[pos * half + i], sn = rsin[pos * half + i];
    row[i] = a * cs - b * sn;
    row[i + half] = a * sn + b * cs;
  }
}

__global__ void swiglu_act_f32_kernel(const float *g, const float *u, int64_t ld_aux, float *C,
                                      int64_t ldc, int M, int N) {
  const int64_t total = (int64_t)M * N;
  for (int64_t e = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; e < total;
       e += (int64_t)gridDim.x * blockDim.x) {
    const int m = (int)(e / N), n = (int)(e % N);
    const float gv = g[(int64_t)m * ld_aux + n];
    C[(int64_t)m * ldc + n] = gv * sigmoidf_(gv) * u[(int64_t)m * ld_aux + n];
  }
}

lc_status run_f32(F32P p, hipStream_t s) {
  dim3 grid((unsigned)((p.N + TN - 1) / TN), (unsigned)((p.M + TM - 1) / TM));
  hipLaunchKernelGGL(gemm_f32_kernel, grid, dim3(256), 0, s, p);
  return check_launch("gemm_f32_kernel");
}

}  // namespace

lc_status gemm_f32_launch(const lc_gemm_args &a, hipStream_t s) {
  F32P p{};
  p.A = static_cast<const float *>(a.A);
  p.B = static_cast<const float *>(a.B);
  p.C = static_cast<float *>(a.C);
  p.R = static_cast<const float *>(a.R);
  p.aux0 = static_cast<const float *>(a.aux0);
  p.aux1 = static_cast<const float *>(a.aux1);
  p.lda = a.lda;
  p.ldb = a.ldb;
  p.ldc = a.ldc;
  p.ldr = a.ldr;
  p.ld_aux = a.ld_aux;
  p.M = (int)a.M;
  p.N = (int)a.N;
  p.K = (int)a.K;
  p.a_k = a.a_kmajor != 0;
  p.b_k = a.b_kmajor != 0;
  p.epi = a.epilogue;
  if (a.epilogue == LC_EPI_SWIGLU) {
    if (!a.b_kmajor) return fail(LC_ERR_UNSUPPORTED, "gemm fp32: SwiGLU needs k-major B");
    F32P q = p;
    q.epi = LC_EPI_STORE;
    q.C = static_cast<float *>(a.aux0);
    q.ldc = a.ld_aux;
    LC_TRY(run_f32(q, s));  // gate = A W1^T
    q.B = p.B + (int64_t)a.N * a.ldb;
    q.C = static_cast<float *>(a.aux1);
    LC_TRY(run_f32(q, s));  // up = A W3^T
    const int64_t total = a.M * a.N;
    hipLaunchKernelGGL(swiglu_act_f32_kernel, dim3((unsigned)std::min<int64_t>((total + 255) / 256, 65535)),
                       dim3(256), 0, s, static_cast<const float *>(a.aux0),
                       static_cast<const float *>(a.aux1), a.ld_aux, p.C, a.ldc, p.M, p.N);
    return check_launch("swiglu_act_f32_kernel");
  }
  if (a.epilogue == LC_EPI_ROPE) {
    F32P q = p;
    q.epi = LC_EPI_STORE;
    LC_TRY(run_f32(q, s));
    if (a.rope_cols > 0) {
      const int64_t total = a.M * (a.rope_cols / 2);
      hipLaunchKernelGGL(rope_f32_kernel, dim3((unsigned)std::min<int64_t>((total + 255) / 256, 65535)),
                         dim3(256), 0, s, p.C, a.ldc, p.M, a.rope_cols, a.head_dim, a.rope_cos,
                         a.rope_sin, a.rope_seq);
      return check_launch("rope_f32_kernel");
    }
    return LC_OK;
  }
  return run_f32(p, s);
}

}  // namespace lc
