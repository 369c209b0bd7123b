// bf16 GEMM on CDNA4 matrix cores (v_mfma_f32_32x32x16_bf16), fp32 accumulation,
// with the fused epilogues of a decoder layer's projections.
//
//   C(m, n) = sum_k A(m, k) B(n, k)
//   A(m, k) = A_K ? A[m*lda + k] : A[k*lda + m]      (A_K: k is contiguous)
//   B(n, k) = B_K ? B[n*ldb + k] : B[k*ldb + n]
//
// Tile: 256 x 256 x 64 per workgroup of 256 threads (4 waves, 2 x 2), each wave
// owns 128 x 128 = 4 x 4 MFMA blocks of 32 x 32. Operand tiles live in LDS as
// [row][64 k] bf16 rows of 128 bytes whose eight 16-byte chunks are XOR-swizzled
// by (row & 7), so that the MFMA fragment reads (16 bytes per lane, 32 rows at
// the same k-chunk) and the tile writes are bank-conflict free. Two LDS stages:
// the global loads of k-tile t+1 are in flight while tile t is multiplied.
//
// An operand whose k is not contiguous in memory (a weight read as dX = dY W,
// or both operands of a weight gradient dW = dY^T X) is loaded as 8 x 8 blocks
// (eight 16-byte rows along m, one per k) and transposed in registers, so the
// LDS image and the MFMA path are identical for every layout and no transposed
// copy is ever materialised in HBM.
//
// The MFMA is issued with B's fragment in the instruction's first operand and
// A's in the second, which leaves lane l holding output row m = l % 32 and four
// runs of four consecutive columns n = 8g + 4(l / 32) + e: epilogues store 8 or
// 16 contiguous bytes per lane, and the column pairs (c, c + 64) that RoPE and
// SwiGLU combine sit in the same lane (blocks j and j + 2 of a 128-wide wave).
// Output, residual and gate/up element types are run-time values (uniform
// branches in the epilogue only).
#include "common.hpp"

namespace lc {
namespace {

constexpr int BM = 256, BN = 256, BK = 64;
constexpr int NT = 256;            // threads per workgroup
constexpr int WM = 128, WN = 128;  // wave tile
constexpr int FM = WM / 32, FN = WN / 32;
constexpr int TILE_BYTES = BM * BK * 2;  // one operand tile in LDS (32 KiB)

struct GemmP {
  const bf16_t *A;
  const bf16_t *B;
  void *C;
  const void *R;
  void *aux0;
  void *aux1;
  const float *rcos;
  const float *rsin;
  int64_t lda, ldb, ldc, ldr, ld_aux;
  int M, N, K;  // N: output columns (SwiGLU: gate/up width)
  int tiles_m, tiles_n;
  int rope_seq, rope_cols;
  int c_dt, r_dt, aux_dt;
};

__device__ __forceinline__ int lds_off(int row, int chunk) {
  return row * 128 + ((chunk ^ (row & 7)) << 4);
}

// 8x8 transpose of bf16 held as 8 rows of uint4 (row r = 8 consecutive m at k r)
// into 8 rows of uint4 (row mm = 8 consecutive k at m mm).
__device__ __forceinline__ void transpose8x8(const uint4 (&r)[8], uint4 (&t)[8]) {
  const uint32_t *rw = reinterpret_cast<const uint32_t *>(r);
  uint32_t *tw = reinterpret_cast<uint32_t *>(t);
#pragma unroll
  for (int p = 0; p < 4; ++p) {      // m pair (2p, 2p+1) = dword p of every row
#pragma unroll
    for (int q = 0; q < 4; ++q) {    // k pair (2q, 2q+1) = dword q of the output
      const uint32_t lo = rw[(2 * q) * 4 + p];
      const uint32_t hi = rw[(2 * q + 1) * 4 + p];
      tw[(2 * p) * 4 + q] = (lo & 0xFFFFu) | (hi << 16);
      tw[(2 * p + 1) * 4 + q] = (lo >> 16) | (hi & 0xFFFF0000u);
    }
  }
}

// Loads of one 256 x 64 operand tile into registers.
// KMAJ: thread t covers rows (t>>3) + 32i, chunk t&7, i < 8.
// !KMAJ: thread t covers the 8x8 block (m-block t&31, k-block t>>5).
template <bool KMAJ, int ROWMAP>
struct TileLoader {
  uint4 v[8];

  // ROWMAP 0: tile row r -> operand row base + r (valid below lim)
  // ROWMAP 1 (SwiGLU B rows): tile row r -> gate row ob + (r>>7)*64 + (r&63) for
  //           (r&127) < 64, else up row N + ob + (r>>7)*64 + (r&63); valid while
  //           the output column ob + (r>>7)*64 + (r&63) < N.
  __device__ __forceinline__ void load(const bf16_t *__restrict__ X, int64_t ld, int base,
                                       int lim, int k0, int K, int tid) {
    if constexpr (KMAJ) {
      const int ch = tid & 7;
      const int gk = k0 + ch * 8;
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const int r = (tid >> 3) + 32 * i;
        int grow;
        bool ok;
        if constexpr (ROWMAP == 0) {
          grow = base + r;
          ok = grow < lim;
        } else {
          const int oc = base + (r >> 7) * 64 + (r & 63);
          ok = oc < lim;
          grow = ((r & 127) < 64) ? oc : lim + oc;
        }
        ok = ok && (gk < K);
        if (ok) {
          v[i] = *reinterpret_cast<const uint4 *>(X + (int64_t)grow * ld + gk);
        } else {
          v[i] = make_uint4(0, 0, 0, 0);
        }
      }
    } else {
      static_assert(ROWMAP == 0, "row remap needs a k-major operand");
      const int mb = tid & 31, kb = tid >> 5;
      const int gm = base + mb * 8;
      const bool mok = gm < lim;
#pragma unroll
      for (int kk = 0; kk < 8; ++kk) {
        const int gk = k0 + kb * 8 + kk;
        if (mok && gk < K) {
          v[kk] = *reinterpret_cast<const uint4 *>(X + (int64_t)gk * ld + gm);
        } else {
          v[kk] = make_uint4(0, 0, 0, 0);
        }
      }
    }
  }

  __device__ __forceinline__ void store(char *lds, int tid) const {
    if constexpr (KMAJ) {
      const int ch = tid & 7;
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const int r = (tid >> 3) + 32 * i;
        *reinterpret_cast<uint4 *>(lds + lds_off(r, ch)) = v[i];
      }
    } else {
      const int mb = tid & 31, kb = tid >> 5;
      uint4 t[8];
      transpose8x8(v, t);
#pragma unroll
      for (int mm = 0; mm < 8; ++mm) {
        *reinterpret_cast<uint4 *>(lds + lds_off(mb * 8 + mm, kb)) = t[mm];
      }
    }
  }
};

template <bool A_K, bool B_K, int EPI>
__global__ __launch_bounds__(NT) void gemm_bf16_kernel(GemmP p) {
  extern __shared__ __align__(16) char smem[];
  // LDS: A stage 0, A stage 1, B stage 0, B stage 1
  auto ldsA = [&](int st) { return smem + st * TILE_BYTES; };
  auto ldsB = [&](int st) { return smem + (2 + st) * TILE_BYTES; };

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;

  // Workgroups are dispatched round-robin over the 8 XCDs; give each XCD a
  // contiguous run of tiles, then walk tiles in groups of 8 tile-rows so that
  // neighbouring workgroups share A rows and B columns in the XCD's L2.
  int wg = blockIdx.x;
  const int nwg = gridDim.x;
  if ((nwg & 7) == 0) wg = (wg & 7) * (nwg >> 3) + (wg >> 3);
  constexpr int GROUP = 8;
  const int per_group = GROUP * p.tiles_n;
  const int first_m = (wg / per_group) * GROUP;
  const int gsz = min(p.tiles_m - first_m, GROUP);
  const int tm = first_m + (wg % per_group) % gsz;
  const int tn = (wg % per_group) / gsz;
  const int m0 = tm * BM;
  constexpr bool SWI = (EPI == LC_EPI_SWIGLU);
  const int n0 = SWI ? tn * (BN / 2) : tn * BN;  // first output column

  TileLoader<A_K, 0> la;
  TileLoader<B_K, SWI ? 1 : 0> lb;

  f32x16_v acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

  const int nk = (p.K + BK - 1) / BK;
  la.load(p.A, p.lda, m0, p.M, 0, p.K, tid);
  lb.load(p.B, p.ldb, n0, p.N, 0, p.K, tid);
  la.store(ldsA(0), tid);
  lb.store(ldsB(0), tid);
  __syncthreads();

  const int frow = lane & 31;
  const int fhalf = lane >> 5;
  for (int kt = 0; kt < nk; ++kt) {
    const int cur = kt & 1;
    const bool more = kt + 1 < nk;
    if (more) {
      la.load(p.A, p.lda, m0, p.M, (kt + 1) * BK, p.K, tid);
      lb.load(p.B, p.ldb, n0, p.N, (kt + 1) * BK, p.K, tid);
    }
    const char *sa = ldsA(cur);
    const char *sb = ldsB(cur);
#pragma unroll
    for (int s = 0; s < BK / 16; ++s) {
      const int ch = s * 2 + fhalf;
      bf16x8_v af[FM], bfr[FN];
#pragma unroll
      for (int i = 0; i < FM; ++i)
        af[i] = *reinterpret_cast<const bf16x8_v *>(sa + lds_off(wm * WM + i * 32 + frow, ch));
#pragma unroll
      for (int j = 0; j < FN; ++j)
        bfr[j] = *reinterpret_cast<const bf16x8_v *>(sb + lds_off(wn * WN + j * 32 + frow, ch));
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(bfr[j], af[i], acc[i][j], 0, 0, 0);
    }
    if (more) {
      la.store(ldsA(cur ^ 1), tid);
      lb.store(ldsB(cur ^ 1), tid);
    }
    __syncthreads();
  }

  // ------------------------------------------------------------ epilogue
  const int h4 = 4 * fhalf;
#pragma unroll
  for (int i = 0; i < FM; ++i) {
    const int m = m0 + wm * WM + i * 32 + frow;
    if (m >= p.M) continue;
    if constexpr (EPI == LC_EPI_SWIGLU) {
#pragma unroll
      for (int j = 0; j < 2; ++j) {
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const int n = n0 + wn * 64 + j * 32 + 8 * g + h4;
          if (n >= p.N) continue;
          float gt[4], up[4], a[4];
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            gt[e] = acc[i][j][4 * g + e];
            up[e] = acc[i][j + 2][4 * g + e];
            a[e] = gt[e] * sigmoidf_(gt[e]) * up[e];
          }
          const int64_t oa = (int64_t)m * p.ld_aux + n;
          store4_dt(p.aux0, oa, p.aux_dt, gt[0], gt[1], gt[2], gt[3]);
          store4_dt(p.aux1, oa, p.aux_dt, up[0], up[1], up[2], up[3]);
          store4_dt(p.C, (int64_t)m * p.ldc + n, p.c_dt, a[0], a[1], a[2], a[3]);
        }
      }
    } else if constexpr (EPI == LC_EPI_ROPE) {
      const int hbase = n0 + wn * WN;  // first column of this wave's head (head_dim 128)
      if (hbase >= p.N) continue;
      const bool rot = hbase < p.rope_cols;
      const int pos = m % p.rope_seq;
#pragma unroll
      for (int j = 0; j < 2; ++j) {
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const int c = j * 32 + 8 * g + h4;  // column inside the head, < 64
          float x1[4], x2[4];
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            x1[e] = acc[i][j][4 * g + e];
            x2[e] = acc[i][j + 2][4 * g + e];
          }
          if (rot) {
            const float4 cs = *reinterpret_cast<const float4 *>(p.rcos + (int64_t)pos * 64 + c);
            const float4 sn = *reinterpret_cast<const float4 *>(p.rsin + (int64_t)pos * 64 + c);
            const float cv[4] = {cs.x, cs.y, cs.z, cs.w};
            const float sv[4] = {sn.x, sn.y, sn.z, sn.w};
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              const float a = x1[e], b = x2[e];
              x1[e] = a * cv[e] - b * sv[e];
              x2[e] = a * sv[e] + b * cv[e];
            }
          }
          const int64_t row = (int64_t)m * p.ldc + hbase;
          store4_dt(p.C, row + c, p.c_dt, x1[0], x1[1], x1[2], x1[3]);
          store4_dt(p.C, row + c + 64, p.c_dt, x2[0], x2[1], x2[2], x2[3]);
        }
      }
    } else {
#pragma unroll
      for (int j = 0; j < FN; ++j) {
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const int n = n0 + wn * WN + j * 32 + 8 * g + h4;
          if (n >= p.N) continue;
          float v0 = acc[i][j][4 * g + 0], v1 = acc[i][j][4 * g + 1];
          float v2 = acc[i][j][4 * g + 2], v3 = acc[i][j][4 * g + 3];
          const int64_t oc = (int64_t)m * p.ldc + n;
          if constexpr (EPI == LC_EPI_STORE) {
            store4_dt(p.C, oc, p.c_dt, v0, v1, v2, v3);
          } else if constexpr (EPI == LC_EPI_RESIDUAL) {
            const float4 r = load4_dt(p.R, (int64_t)m * p.ldr + n, p.r_dt);
            store4_dt(p.C, oc, p.c_dt, r.x + v0, r.y + v1, r.z + v2, r.w + v3);
          } else if constexpr (EPI == LC_EPI_ACCUM_F32) {
            float4 *cp = reinterpret_cast<float4 *>(static_cast<float *>(p.C) + oc);
            float4 c = *cp;
            c.x += v0;
            c.y += v1;
            c.z += v2;
            c.w += v3;
            *cp = c;
          } else if constexpr (EPI == LC_EPI_SWIGLU_BWD) {
            const int64_t oa = (int64_t)m * p.ld_aux + n;
            const float4 gt = load4_dt(p.aux0, oa, p.aux_dt);
            const float4 up = load4_dt(p.aux1, oa, p.aux_dt);
            const float gv[4] = {gt.x, gt.y, gt.z, gt.w};
            const float uv[4] = {up.x, up.y, up.z, up.w};
            const float dv[4] = {v0, v1, v2, v3};
            float dg[4], du[4];
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              const float s = sigmoidf_(gv[e]);
              dg[e] = dv[e] * uv[e] * s * (1.0f + gv[e] * (1.0f - s));
              du[e] = dv[e] * gv[e] * s;
            }
            store4_dt(p.C, oc, p.c_dt, dg[0], dg[1], dg[2], dg[3]);
            store4_dt(p.C, oc + p.N, p.c_dt, du[0], du[1], du[2], du[3]);
          }
        }
      }
    }
  }
}

template <bool A_K, bool B_K, int EPI>
lc_status launch_t(const GemmP &p, hipStream_t s) {
  const unsigned grid = (unsigned)p.tiles_m * (unsigned)p.tiles_n;
  const size_t lds = 4 * TILE_BYTES;
  static bool attr_set = false;
  if (!attr_set) {
    hipError_t e = hipFuncSetAttribute((const void *)gemm_bf16_kernel<A_K, B_K, EPI>,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return hip_fail(e, "gemm: setting the LDS size");
    attr_set = true;
  }
  hipLaunchKernelGGL((gemm_bf16_kernel<A_K, B_K, EPI>), dim3(grid), dim3(NT), lds, s, p);
  return check_launch("gemm_bf16_kernel");
}

}  // namespace

lc_status gemm_f32_launch(const lc_gemm_args &a, hipStream_t s);  // k_gemm_f32.hip

// the epilogue types this call uses (STORE_F32 and ACCUM_F32 imply fp32 C)
static int c_type(const lc_gemm_args &a) {
  return (a.epilogue == LC_EPI_STORE_F32 || a.epilogue == LC_EPI_ACCUM_F32) ? LC_FP32 : a.c_dtype;
}

static lc_status check_gemm_args(const lc_gemm_args &a) {
  if (a.M <= 0 || a.N <= 0 || a.K <= 0) return fail(LC_ERR_INVALID_ARG, "gemm: M, N, K must be > 0");
  if (a.M > INT32_MAX / 2 || a.N > INT32_MAX / 4 || a.K > INT32_MAX / 2)
    return fail(LC_ERR_UNSUPPORTED, "gemm: dimension too large");
  if (!a.A || !a.B || !a.C) return fail(LC_ERR_INVALID_ARG, "gemm: null operand");
  if (!aligned16(a.A) || !aligned16(a.B) || !aligned16(a.C))
    return fail(LC_ERR_INVALID_ARG, "gemm: operands must be 16-byte aligned");
  if (a.epilogue < LC_EPI_STORE || a.epilogue > LC_EPI_SWIGLU_BWD)
    return fail(LC_ERR_INVALID_ARG, "gemm: unknown epilogue %d", a.epilogue);
  if (!valid_dtype(c_type(a))) return fail(LC_ERR_INVALID_ARG, "gemm: unknown c_dtype");
  const bool bf = a.dtype == LC_BF16;
  if (bf && (a.lda % 8 || a.ldb % 8 || a.ldc % 8))
    return fail(LC_ERR_INVALID_ARG, "gemm: ld %% 8 != 0");
  const int64_t acols = a.a_kmajor ? a.K : a.M;
  const int64_t brows = a.epilogue == LC_EPI_SWIGLU ? 2 * a.N : a.N;
  const int64_t bcols = a.b_kmajor ? a.K : brows;
  if (a.lda < acols || a.ldb < bcols) return fail(LC_ERR_INVALID_ARG, "gemm: ld too small");
  if (a.epilogue == LC_EPI_RESIDUAL) {
    if (!a.R || !aligned16(a.R) || (bf && a.ldr % 8) || a.ldr < a.N || !valid_dtype(a.r_dtype))
      return fail(LC_ERR_INVALID_ARG, "gemm: bad residual operand");
  }
  if (a.epilogue == LC_EPI_SWIGLU || a.epilogue == LC_EPI_SWIGLU_BWD) {
    if (!a.aux0 || !a.aux1 || !aligned16(a.aux0) || !aligned16(a.aux1) ||
        (bf && a.ld_aux % 8) || a.ld_aux < a.N || !valid_dtype(a.aux_dtype))
      return fail(LC_ERR_INVALID_ARG, "gemm: bad gate/up operands");
    if (a.epilogue == LC_EPI_SWIGLU_BWD && a.ldc < 2 * a.N)
      return fail(LC_ERR_INVALID_ARG, "gemm: ldc < 2N for SWIGLU_BWD");
  } else if (a.ldc < a.N) {
    return fail(LC_ERR_INVALID_ARG, "gemm: ldc < N");
  }
  if (a.epilogue == LC_EPI_ROPE) {
    if (!a.rope_cos || !a.rope_sin || a.rope_seq <= 0 || a.rope_cols < 0 ||
        a.head_dim <= 0 || a.head_dim % 2 || a.rope_cols % a.head_dim || a.N % a.head_dim)
      return fail(LC_ERR_INVALID_ARG, "gemm: bad RoPE arguments");
  }
  return LC_OK;
}

lc_status gemm_launch(const lc_gemm_args &a, hipStream_t s) {
  LC_TRY(check_gemm_args(a));
  if (a.dtype == LC_FP32) {
    if (c_type(a) != LC_FP32 || (a.epilogue == LC_EPI_RESIDUAL && a.r_dtype != LC_FP32) ||
        ((a.epilogue == LC_EPI_SWIGLU || a.epilogue == LC_EPI_SWIGLU_BWD) &&
         a.aux_dtype != LC_FP32))
      return fail(LC_ERR_UNSUPPORTED, "gemm fp32: every tensor must be fp32");
    return gemm_f32_launch(a, s);
  }
  if (a.dtype != LC_BF16) return fail(LC_ERR_INVALID_ARG, "gemm: A/B dtype must be fp32 or bf16");
  // layout limits of the bf16 kernel: 16-byte rows along every contiguous extent
  if (a.N % 8) return fail(LC_ERR_UNSUPPORTED, "gemm bf16: N %% 8 != 0");
  if ((a.a_kmajor || a.b_kmajor) && a.K % 8) return fail(LC_ERR_UNSUPPORTED, "gemm bf16: K %% 8 != 0");
  if (!a.a_kmajor && a.M % 8) return fail(LC_ERR_UNSUPPORTED, "gemm bf16: M %% 8 != 0 (A not k-major)");
  if (a.epilogue == LC_EPI_ROPE && a.head_dim != 128)
    return fail(LC_ERR_UNSUPPORTED, "gemm bf16: RoPE epilogue needs head_dim 128");
  if (a.epilogue == LC_EPI_SWIGLU && (a.N % 64 || !a.b_kmajor))
    return fail(LC_ERR_UNSUPPORTED, "gemm bf16: SwiGLU needs N %% 64 == 0 and k-major B");
  if (a.epilogue == LC_EPI_ROPE && (!aligned16(a.rope_cos) || !aligned16(a.rope_sin)))
    return fail(LC_ERR_INVALID_ARG, "gemm: RoPE tables must be 16-byte aligned");

  GemmP p{};
  p.A = static_cast<const bf16_t *>(a.A);
  p.B = static_cast<const bf16_t *>(a.B);
  p.C = a.C;
  p.R = a.R;
  p.aux0 = a.aux0;
  p.aux1 = a.aux1;
  p.rcos = a.rope_cos;
  p.rsin = a.rope_sin;
  p.lda = a.lda;
  p.ldb = a.ldb;
  p.ldc = a.ldc;
  p.ldr = a.ldr;
  p.ld_aux = a.ld_aux;
  p.M = (int)a.M;
  p.N = (int)a.N;
  p.K = (int)a.K;
  p.tiles_m = (int)((a.M + BM - 1) / BM);
  p.tiles_n = a.epilogue == LC_EPI_SWIGLU ? (int)((a.N + BN / 2 - 1) / (BN / 2))
                                          : (int)((a.N + BN - 1) / BN);
  p.rope_seq = a.rope_seq;
  p.rope_cols = a.rope_cols;
  p.c_dt = c_type(a);
  p.r_dt = a.r_dtype;
  p.aux_dt = a.aux_dtype;

  const bool ak = a.a_kmajor != 0, bk = a.b_kmajor != 0;
  switch (a.epilogue) {
    case LC_EPI_STORE:
    case LC_EPI_STORE_F32:
      if (ak && bk) return launch_t<true, true, LC_EPI_STORE>(p, s);
      if (ak && !bk) return launch_t<true, false, LC_EPI_STORE>(p, s);
      if (!ak && !bk) return launch_t<false, false, LC_EPI_STORE>(p, s);
      break;
    case LC_EPI_ACCUM_F32:
      if (ak && bk) return launch_t<true, true, LC_EPI_ACCUM_F32>(p, s);
      if (!ak && !bk) return launch_t<false, false, LC_EPI_ACCUM_F32>(p, s);
      break;
    case LC_EPI_RESIDUAL:
      if (ak && bk) return launch_t<true, true, LC_EPI_RESIDUAL>(p, s);
      break;
    case LC_EPI_ROPE:
      if (ak && bk) return launch_t<true, true, LC_EPI_ROPE>(p, s);
      break;
    case LC_EPI_SWIGLU:
      if (ak && bk) return launch_t<true, true, LC_EPI_SWIGLU>(p, s);
      break;
    case LC_EPI_SWIGLU_BWD:
      if (ak && !bk) return launch_t<true, false, LC_EPI_SWIGLU_BWD>(p, s);
      if (ak && bk) return launch_t<true, true, LC_EPI_SWIGLU_BWD>(p, s);
      break;
  }
  return fail(LC_ERR_UNSUPPORTED, "gemm bf16: layout (a_kmajor=%d, b_kmajor=%d) not built for "
              "epilogue %d", (int)ak, (int)bk, a.epilogue);
}

}  // namespace lc

extern "C" lc_status lc_gemm(const lc_gemm_args *args, void *stream) {
  if (!args) return lc::fail(LC_ERR_INVALID_ARG, "gemm: null args");
  return lc::gemm_launch(*args, static_cast<hipStream_t>(stream));
}
