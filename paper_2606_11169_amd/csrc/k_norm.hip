// RMSNorm forward and backward (HBM-bound row kernels).
//
//   forward:  rstd_t = 1/sqrt(mean_k x_tk^2 + eps),  n_tk = x_tk * rstd_t * g_k
//   backward: xh = x*rstd, dxh = dn*g,
//             dx_tk = dres_tk + rstd_t (dxh_tk - xh_tk * mean_k(dxh*xh)),
//             dg_k += sum_t dn_tk xh_tk
//
// Forward: one wave per row, 8 elements per lane per step (16- or 32-byte
// accesses); rows of up to 4096 elements stay in registers between the row's
// reduction and its write (one read), longer rows are read twice (the second
// read hits L2). Backward: rows of up to 4096 elements are split over four
// waves (so that a workgroup of 16 waves keeps four rows in registers at
// once and the chip holds enough waves to cover memory latency); longer rows
// go one per wave, read twice. Every tensor's element type is a run-time
// value (uniform branches), except in the instantiations for the decoder
// stage's own type mix, where the types are template arguments (straight-line
// loads: 20-25% faster forward, 9% faster backward rows). The gain gradient is a column reduction over
// rows: each backward workgroup handles kNormRowsPerBlock rows and writes
// the fp32 partial sums of its rows in a fixed order, then the final kernel
// adds the partials of each column: sixteen slices of consecutive blocks,
// each summed in block order, then the slices in order — the same order on
// every run, no atomics.
#include "common.hpp"

#include <mutex>

namespace lc {
namespace {

constexpr int ROWS_PER_BLOCK = 4;  // forward: one wave per row
constexpr int MAXU = 8;            // 8-element chunks per lane held in registers
constexpr int MAXD = 64 * 8 * MAXU;

struct NormP {
  const void *x, *g, *dn, *dres;
  void *n, *dx, *dx_copy;
  float *rstd;
  float *partial, *dg;
  int part;      // write the gain-gradient partial sums
  int dg_store;  // the final sum overwrites dg instead of adding into it
  int64_t rows;
  int d;
  float eps;
  int x_dt, w_dt, out_dt, dn_dt, dres_dt;
  int nblk;
};

template <int XDT, int WDT, int ODT>
__global__ __launch_bounds__(256) void rmsnorm_fwd_kernel(NormP p) {
  const int lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * ROWS_PER_BLOCK + (threadIdx.x >> 6);
  if (row >= p.rows) return;
  const int64_t base = row * p.d;
  float ss = 0.0f;
  if (p.d <= MAXD) {
    float v[MAXU][8];
#pragma unroll
    for (int u = 0; u < MAXU; ++u) {
      const int c = lane * 8 + 512 * u;
      if (c < p.d) {
        ld8<XDT>(p.x, base + c, p.x_dt, v[u]);
#pragma unroll
        for (int e = 0; e < 8; ++e) ss += v[u][e] * v[u][e];
      }
    }
    ss = wave_sum(ss);
    const float r = 1.0f / sqrtf(ss / (float)p.d + p.eps);
    if (lane == 0) p.rstd[row] = r;
#pragma unroll
    for (int u = 0; u < MAXU; ++u) {
      const int c = lane * 8 + 512 * u;
      if (c < p.d) {
        float gv[8];
        ld8<WDT>(p.g, c, p.w_dt, gv);
#pragma unroll
        for (int e = 0; e < 8; ++e) v[u][e] = v[u][e] * r * gv[e];
        st8<ODT>(p.n, base + c, p.out_dt, v[u]);
      }
    }
    return;
  }
  for (int c = lane * 8; c < p.d; c += 64 * 8) {
    float v[8];
    load8_dt(p.x, base + c, p.x_dt, v);
#pragma unroll
    for (int e = 0; e < 8; ++e) ss += v[e] * v[e];
  }
  ss = wave_sum(ss);
  const float r = 1.0f / sqrtf(ss / (float)p.d + p.eps);
  if (lane == 0) p.rstd[row] = r;
  for (int c = lane * 8; c < p.d; c += 64 * 8) {
    float v[8], gv[8];
    load8_dt(p.x, base + c, p.x_dt, v);
    load8_dt(p.g, c, p.w_dt, gv);
#pragma unroll
    for (int e = 0; e < 8; ++e) v[e] = v[e] * r * gv[e];
    store8_dt(p.n, base + c, p.out_dt, v);
  }
}

// rows longer than MAXD: the row is read twice, the gain gradient is not formed here
__device__ __forceinline__ void bwd_row_long(const NormP &p, int64_t row, int lane) {
  const int64_t base = row * p.d;
  const float r = p.rstd[row];
  float dot = 0.0f;
  for (int c = lane * 8; c < p.d; c += 64 * 8) {
    float a[8], b[8], gv[8];
    load8_dt(p.dn, base + c, p.dn_dt, a);
    load8_dt(p.x, base + c, p.x_dt, b);
    load8_dt(p.g, c, p.w_dt, gv);
#pragma unroll
    for (int e = 0; e < 8; ++e) dot += a[e] * gv[e] * b[e];
  }
  dot = wave_sum(dot);
  const float mean = dot * r / (float)p.d;
  const float r2m = r * mean;
  for (int c = lane * 8; c < p.d; c += 64 * 8) {
    float a[8], b[8], gv[8], o[8];
    load8_dt(p.dn, base + c, p.dn_dt, a);
    load8_dt(p.x, base + c, p.x_dt, b);
    load8_dt(p.g, c, p.w_dt, gv);
    if (p.dres) {
      load8_dt(p.dres, base + c, p.dres_dt, o);
    } else {
#pragma unroll
      for (int e = 0; e < 8; ++e) o[e] = 0.0f;
    }
#pragma unroll
    for (int e = 0; e < 8; ++e) o[e] += r * (a[e] * gv[e] - b[e] * r2m);
    store8_dt(p.dx, base + c, p.out_dt, o);
    if (p.dx_copy) store8_dt(p.dx_copy, base + c, LC_BF16, o);
  }
}

// Rows of up to MAXD values: one workgroup of 16 waves per kNormRowsPerBlock
// rows, 4 waves per row (lane l of wave w of a row holds the 8-value chunks
// starting at 8 (64 w + l) and 8 (64 w + l) + 2048), four rows at a time:
// iteration i takes rows 4 i + s (s = wave / 4). A row's dot product is the
// sum of its four waves' shares in wave order (through LDS); the gain
// gradient's partial sums: each lane's rows in order, then the four row
// slots in order, into partial[blk][k].
constexpr int BW_THREADS = 1024;
constexpr int BW_CHUNKS = MAXD / 2048;  // 8-value chunks per lane
template <int DNDT, int XDT, int WDT, int RDT, int ODT>
__global__ __launch_bounds__(BW_THREADS) void rmsnorm_bwd_rows_kernel(NormP p) {
  __shared__ float red[MAXD];
  __shared__ float dots[2][4][4];  // [iteration parity][row slot][wave of the row]
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  const int slot = wv >> 2, wr = wv & 3;
  const int rl = wr * 64 + lane;
  const int64_t r0 = (int64_t)blockIdx.x * kNormRowsPerBlock;
  const int64_t r1 = min(p.rows, r0 + kNormRowsPerBlock);
  float acc[BW_CHUNKS][8];
#pragma unroll
  for (int u = 0; u < BW_CHUNKS; ++u)
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[u][e] = 0.0f;
#pragma unroll 1
  for (int i = 0; i < kNormRowsPerBlock / 4; ++i) {
    const int64_t row = r0 + 4 * i + slot;
    const bool ok = row < r1;  // wave-uniform
    const int64_t base = row * p.d;
    float a[BW_CHUNKS][8], b[BW_CHUNKS][8];
    float dot = 0.0f;  // this wave's share of sum_k dn*g*x
    const float r = ok ? p.rstd[row] : 0.0f;
#pragma unroll
    for (int u = 0; u < BW_CHUNKS; ++u) {
      const int c = 8 * rl + 2048 * u;
      if (ok && c < p.d) {
        float gv[8];
        ld8<DNDT>(p.dn, base + c, p.dn_dt, a[u]);
        ld8<XDT>(p.x, base + c, p.x_dt, b[u]);
        ld8<WDT>(p.g, c, p.w_dt, gv);
#pragma unroll
        for (int e = 0; e < 8; ++e) dot += a[u][e] * gv[e] * b[u][e];
      }
    }
    dot = wave_sum(dot);
    if (lane == 0) dots[i & 1][slot][wr] = dot;
    __syncthreads();
    if (!ok) continue;
    const float tot = dots[i & 1][slot][0] + dots[i & 1][slot][1] + dots[i & 1][slot][2] +
                      dots[i & 1][slot][3];
    const float mean = tot * r / (float)p.d;  // mean_k(dxh * xh)
    const float r2m = r * mean;
#pragma unroll
    for (int u = 0; u < BW_CHUNKS; ++u) {
      const int c = 8 * rl + 2048 * u;
      if (c < p.d) {
        float o[8], gv[8];
        ld8<WDT>(p.g, c, p.w_dt, gv);
        if (p.dres) {
          ld8<RDT>(p.dres, base + c, p.dres_dt, o);
        } else {
#pragma unroll
          for (int e = 0; e < 8; ++e) o[e] = 0.0f;
        }
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          o[e] += r * (a[u][e] * gv[e] - b[u][e] * r2m);
          acc[u][e] += a[u][e] * (b[u][e] * r);
        }
        st8<ODT>(p.dx, base + c, p.out_dt, o);
        if (p.dx_copy) st8<LC_BF16>(p.dx_copy, base + c, LC_BF16, o);
      }
    }
  }
  if (!p.part) return;  // uniform: no gain gradient requested
#pragma unroll 1
  for (int s = 0; s < 4; ++s) {
    if (slot == s) {
#pragma unroll
      for (int u = 0; u < BW_CHUNKS; ++u) {
        const int c = 8 * rl + 2048 * u;
        if (c < p.d) {
#pragma unroll
          for (int e = 0; e < 8; ++e) red[c + e] = (s == 0 ? 0.0f : red[c + e]) + acc[u][e];
        }
      }
    }
    __syncthreads();
  }
  for (int k = threadIdx.x; k < p.d; k += BW_THREADS) p.partial[(int64_t)blockIdx.x * p.d + k] = red[k];
}

// Rows longer than MAXD: one workgroup of 4 waves per kNormRowsPerBlock rows
// (wave w: rows w, w + 4, ...), each row read twice; the gain gradient's
// partial sums come from rmsnorm_dg_partial_kernel.
__global__ __launch_bounds__(256) void rmsnorm_bwd_long_kernel(NormP p) {
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  const int64_t r0 = (int64_t)blockIdx.x * kNormRowsPerBlock;
  const int64_t r1 = min(p.rows, r0 + kNormRowsPerBlock);
  for (int64_t row = r0 + wv; row < r1; row += 4) bwd_row_long(p, row, lane);
}

__device__ __forceinline__ float ld1_dt(const void *base, int64_t i, int dt) {
  if (dt == LC_FP32) return static_cast<const float *>(base)[i];
  if (dt == LC_BF16) return (float)static_cast<const __bf16 *>(base)[i];
  return (float)static_cast<const _Float16 *>(base)[i];
}

// rows longer than MAXD: partial[blk][k] = sum over rows of block blk of dn[t,k] * x[t,k] * rstd[t]
__global__ __launch_bounds__(256) void rmsnorm_dg_partial_kernel(NormP p) {
  const int k = blockIdx.x * 256 + threadIdx.x;
  if (k >= p.d) return;
  const int64_t r0 = (int64_t)blockIdx.y * kNormRowsPerBlock;
  const int64_t r1 = min(p.rows, r0 + kNormRowsPerBlock);
  float s = 0.0f;
  for (int64_t t = r0; t < r1; ++t)
    s += ld1_dt(p.dn, t * p.d + k, p.dn_dt) * (ld1_dt(p.x, t * p.d + k, p.x_dt) * p.rstd[t]);
  p.partial[(int64_t)blockIdx.y * p.d + k] = s;
}

// dg[k] += sum of partial[b][k] over blocks b: sixteen slices of consecutive
// blocks (each summed in block order), then the slices in order
constexpr int DG_SLICES = 16;
__global__ __launch_bounds__(1024) void rmsnorm_dg_final_kernel(NormP p) {
  __shared__ float sl[DG_SLICES][64];
  const int t = threadIdx.x, sidx = t >> 6, kc = t & 63;
  const int k = blockIdx.x * 64 + kc;
  const int per = (p.nblk + DG_SLICES - 1) / DG_SLICES;
  const int b0 = sidx * per, b1 = min(p.nblk, b0 + per);
  float s = 0.0f;
  if (k < p.d) {
    int b = b0;
    for (; b + 8 <= b1; b += 8) {
      float v[8];
#pragma unroll
      for (int i = 0; i < 8; ++i) v[i] = p.partial[(int64_t)(b + i) * p.d + k];
#pragma unroll
      for (int i = 0; i < 8; ++i) s += v[i];
    }
    for (; b < b1; ++b) s += p.partial[(int64_t)b * p.d + k];
  }
  sl[sidx][kc] = s;
  __syncthreads();
  if (sidx == 0 && k < p.d) {
    float tot = sl[0][kc];
#pragma unroll
    for (int i = 1; i < DG_SLICES; ++i) tot += sl[i][kc];
    p.dg[k] = p.dg_store ? tot : p.dg[k] + tot;
  }
}

lc_status check_common(const lc_norm_args &a, bool bwd) {
  if (a.T <= 0 || a.d <= 0) return fail(LC_ERR_INVALID_ARG, "rmsnorm: T and d must be positive");
  if (a.d % 8) return fail(LC_ERR_UNSUPPORTED, "rmsnorm: d %% 8 != 0");
  if (a.d > INT32_MAX) return fail(LC_ERR_UNSUPPORTED, "rmsnorm: d too large");
  if (!valid_dtype(a.x_dtype) || !valid_dtype(a.w_dtype) || !valid_dtype(a.out_dtype))
    return fail(LC_ERR_INVALID_ARG, "rmsnorm: unknown dtype");
  if (!a.x || !a.g || !a.rstd) return fail(LC_ERR_INVALID_ARG, "rmsnorm: null pointer");
  if (!aligned16(a.x) || !aligned16(a.g)) return fail(LC_ERR_INVALID_ARG, "rmsnorm: unaligned pointer");
  if (!bwd) {
    if (!a.n || !aligned16(a.n)) return fail(LC_ERR_INVALID_ARG, "rmsnorm: bad output pointer");
  } else {
    if (!valid_dtype(a.dn_dtype) || (a.dres && !valid_dtype(a.dres_dtype)))
      return fail(LC_ERR_INVALID_ARG, "rmsnorm: unknown dtype");
    if (!a.dn || !a.dx || !aligned16(a.dn) || !aligned16(a.dx) || (a.dres && !aligned16(a.dres)) ||
        (a.dx_copy && !aligned16(a.dx_copy)))
      return fail(LC_ERR_INVALID_ARG, "rmsnorm: bad backward pointer");
    if (a.dg_accum && (!a.scratch || a.scratch_bytes < rmsnorm_scratch_size(a.T, a.d)))
      return fail(LC_ERR_WORKSPACE, "rmsnorm: scratch smaller than lc_rmsnorm_scratch_bytes");
  }
  return LC_OK;
}

NormP make_params(const lc_norm_args &a) {
  NormP p{};
  p.x = a.x;
  p.g = a.g;
  p.dn = a.dn;
  p.dres = a.dres;
  p.n = a.n;
  p.dx = a.dx;
  p.dx_copy = a.dx_copy;
  p.rstd = a.rstd;
  p.partial = static_cast<float *>(a.scratch);
  p.dg = a.dg_accum;
  p.part = a.dg_accum != nullptr;
  p.rows = a.T;
  p.d = (int)a.d;
  p.eps = a.eps;
  p.x_dt = a.x_dtype;
  p.w_dt = a.w_dtype;
  p.out_dt = a.out_dtype;
  p.dn_dt = a.dn_dtype;
  p.dres_dt = a.dres_dtype;
  p.nblk = (int)((a.T + kNormRowsPerBlock - 1) / kNormRowsPerBlock);
  return p;
}

}  // namespace

lc_status rmsnorm_fwd_launch(const lc_norm_args &a, hipStream_t s) {
  LC_TRY(check_common(a, false));
  const NormP p = make_params(a);
  const dim3 grid((unsigned)((a.T + ROWS_PER_BLOCK - 1) / ROWS_PER_BLOCK));
  // the decoder stage's type mix (fp32 residual rows, bf16 gain and output)
  // has its own instantiation; every other mix takes the generic kernel
  if (p.x_dt == LC_FP32 && p.w_dt == LC_BF16 && p.out_dt == LC_BF16)
    hipLaunchKernelGGL((rmsnorm_fwd_kernel<LC_FP32, LC_BF16, LC_BF16>), grid, dim3(256), 0, s, p);
  else
    hipLaunchKernelGGL((rmsnorm_fwd_kernel<-1, -1, -1>), grid, dim3(256), 0, s, p);
  return check_launch("rmsnorm_fwd_kernel");
}

namespace {

// Row kernel, plus the separate partial-sum kernel for rows longer than MAXD
// when p.part is set.
lc_status bwd_rows(const NormP &p, hipStream_t s) {
  if (p.d <= MAXD) {
    // the decoder stage's type mix (fp32 dn, x, residual gradient and dx, bf16
    // gain) has its own instantiation; every other mix takes the generic kernel
    if (p.dn_dt == LC_FP32 && p.x_dt == LC_FP32 && p.w_dt == LC_BF16 && p.out_dt == LC_FP32 &&
        (!p.dres || p.dres_dt == LC_FP32))
      hipLaunchKernelGGL((rmsnorm_bwd_rows_kernel<LC_FP32, LC_FP32, LC_BF16, LC_FP32, LC_FP32>),
                         dim3((unsigned)p.nblk), dim3(BW_THREADS), 0, s, p);
    else
      hipLaunchKernelGGL((rmsnorm_bwd_rows_kernel<-1, -1, -1, -1, -1>), dim3((unsigned)p.nblk),
                         dim3(BW_THREADS), 0, s, p);
    return check_launch("rmsnorm_bwd_rows_kernel");
  }
  hipLaunchKernelGGL(rmsnorm_bwd_long_kernel, dim3((unsigned)p.nblk), dim3(256), 0, s, p);
  LC_TRY(check_launch("rmsnorm_bwd_long_kernel"));
  if (!p.part) return LC_OK;
  hipLaunchKernelGGL(rmsnorm_dg_partial_kernel, dim3((unsigned)((p.d + 255) / 256), (unsigned)p.nblk),
                     dim3(256), 0, s, p);
  return check_launch("rmsnorm_dg_partial_kernel");
}

lc_status dg_final(const NormP &p, hipStream_t s) {
  hipLaunchKernelGGL(rmsnorm_dg_final_kernel, dim3((unsigned)((p.d + 63) / 64)), dim3(1024), 0, s, p);
  return check_launch("rmsnorm_dg_final_kernel");
}

}  // namespace

lc_status rmsnorm_bwd_launch(const lc_norm_args &a, hipStream_t s) {
  LC_TRY(check_common(a, true));
  const NormP p = make_params(a);
  LC_TRY(bwd_rows(p, s));
  return a.dg_accum ? dg_final(p, s) : LC_OK;
}

lc_status rmsnorm_bwd_partials_launch(const lc_norm_args &a, hipStream_t s) {
  lc_norm_args b = a;
  b.dg_accum = nullptr;
  LC_TRY(check_common(b, true));
  if (!a.scratch || a.scratch_bytes < rmsnorm_scratch_size(a.T, a.d))
    return fail(LC_ERR_WORKSPACE, "rmsnorm: scratch smaller than lc_rmsnorm_scratch_bytes");
  NormP p = make_params(b);
  p.part = 1;
  return bwd_rows(p, s);
}

lc_status rmsnorm_dg_final_launch(const float *partial, float *dg, int64_t T, int64_t d,
                                  hipStream_t s, bool store) {
  if (!partial || !dg || T <= 0 || d <= 0 || d > INT32_MAX)
    return fail(LC_ERR_INVALID_ARG, "rmsnorm: bad gain-gradient sum arguments");
  NormP p{};
  p.partial = const_cast<float *>(partial);
  p.dg = dg;
  p.rows = T;
  p.d = (int)d;
  p.nblk = (int)((T + kNormRowsPerBlock - 1) / kNormRowsPerBlock);
  p.dg_store = store;
  return dg_final(p, s);
}

// ---------------------------------------------------------------- no allocation
// lc_rmsnorm_backward_noalloc keeps the gain gradient's partial sums in this
// fixed device array instead of a caller's scratch. Each GPU the library runs
// on holds its own copy (module memory, until the process ends). The array's
// name is a host-side stand-in: host code uses only the address that
// hipGetSymbolAddress returns for the current device.
static __device__ __align__(256) float scratch[LC_RMSNORM_NOALLOC_SCRATCH_BYTES / sizeof(float)];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void *g_scratch_ptr[kMaxDevices] = {};

// Device address of the current device's copy of `scratch`, looked up on
// the first call on that device (with it current) and kept.
lc_status noalloc_scratch(void **out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "rmsnorm (no allocation): hipGetDevice");
  if (dev < 0 || dev >= kMaxDevices)
    return fail(LC_ERR_UNSUPPORTED, "rmsnorm (no allocation): device %d beyond %d", dev, kMaxDevices);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void *p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return hip_fail(e, "rmsnorm (no allocation): hipGetSymbolAddress");
    if (!p) return fail(LC_ERR_HIP, "rmsnorm (no allocation): null scratch address");
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return LC_OK;
}

}  // namespace

lc_status rmsnorm_bwd_noalloc_launch(const lc_norm_args &in, hipStream_t s) {
  lc_norm_args a = in;
  a.scratch = nullptr;
  a.scratch_bytes = 0;
  if (a.dg_accum) {
    if (a.T <= 0 || a.d <= 0 || a.d > INT32_MAX)
      return fail(LC_ERR_INVALID_ARG, "rmsnorm: T and d must be positive (d < 2^31)");
    // ceil(T / 16) * d * 4 bytes of partial sums, compared without overflow
    const uint64_t blocks = ((uint64_t)a.T + kNormRowsPerBlock - 1) / kNormRowsPerBlock;
    const uint64_t cap = LC_RMSNORM_NOALLOC_SCRATCH_BYTES / sizeof(float);
    if (blocks > cap / (uint64_t)a.d)
      return fail(LC_ERR_WORKSPACE,
                  "rmsnorm (no allocation): T = %lld, d = %lld need %llu bytes of partial sums, "
                  "more than the fixed %zu (ceil(T / 16) * d * 4 must fit)",
                  (long long)a.T, (long long)a.d,
                  (unsigned long long)(blocks * (uint64_t)a.d * sizeof(float)),
                  (size_t)LC_RMSNORM_NOALLOC_SCRATCH_BYTES);
    LC_TRY(noalloc_scratch(&a.scratch));
    a.scratch_bytes = LC_RMSNORM_NOALLOC_SCRATCH_BYTES;
  }
  return rmsnorm_bwd_launch(a, s);
}

}  // namespace lc

extern "C" {

lc_status lc_rmsnorm_backward_noalloc(const lc_norm_args *args, void *stream) {
  if (!args) return lc::fail(LC_ERR_INVALID_ARG, "rmsnorm: null args");
  return lc::rmsnorm_bwd_noalloc_launch(*args, static_cast<hipStream_t>(stream));
}

lc_status lc_rmsnorm_forward(const lc_norm_args *args, void *stream) {
  if (!args) return lc::fail(LC_ERR_INVALID_ARG, "rmsnorm: null args");
  return lc::rmsnorm_fwd_launch(*args, static_cast<hipStream_t>(stream));
}

lc_status lc_rmsnorm_backward(const lc_norm_args *args, void *stream) {
  if (!args) return lc::fail(LC_ERR_INVALID_ARG, "rmsnorm: null args");
  return lc::rmsnorm_bwd_launch(*args, static_cast<hipStream_t>(stream));
}

}  // extern "C"
