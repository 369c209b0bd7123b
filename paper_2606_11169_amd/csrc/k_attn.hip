// Causal softmax attention on CDNA4 matrix cores (head_dim 128, fp16 or bf16
// q/k/v operands, fp32 softmax and accumulation), plus a plain fp32 path.
//
// Forward (written from the FlashAttention-2 algorithm of Dao, 2023): a
// workgroup owns 128 queries of one (batch row, head); each of its 4 waves owns
// 32 queries and walks the visible keys in blocks of 64 staged in LDS, keeping
// a running row maximum and row sum (online softmax) and the output
// accumulator in registers. The score block is computed transposed,
// S^T = K Q^T, so each lane holds one query's scores: the row max and row
// sum need only lane-local work plus one swap with the partner lane
// (lane ^ 32) that holds the other half of the keys. The output is likewise
// accumulated transposed, O^T += V^T P^T, so the per-query rescale factor is a
// lane-local scalar, and the P^T accumulator registers are fed straight back
// as the MFMA B operand: the keys a lane holds define the k-slots, and the
// V^T fragment is read from LDS in the same key order. Products use the q/k/v
// element type (P is rounded to it too).
//
// Backward (deterministic, no atomics): D = rowsum(dO * O) first; then one
// kernel per query block recomputes P^T from the saved log-sum-exp (with the
// forward's q/k type, so P matches the forward) and accumulates
// dQ^T = K^T dS^T over keys, and one kernel per key block accumulates
// dV^T = dO^T P and dK^T = Q^T dS over queries (S computed untransposed there
// so the key is the lane index). Every gradient product is bf16 x bf16 (q, k,
// v are converted while they are staged). RoPE's inverse rotation of dq/dk is
// applied in the epilogue. LDS tiles are filled from 8 x 8 blocks read once
// from HBM and written both row-major and transposed.
#include "common.hpp"

#include <math.h>

#include <type_traits>

namespace lc {
namespace {

constexpr int HD = 128;
constexpr int QB = 128;  // queries (or keys) per workgroup
constexpr int KB = 64;   // keys (or queries) per inner step
constexpr float LOG2E = 1.4426950408889634f;
constexpr float LN2 = 0.6931471805599453f;
constexpr int TILE = KB * HD * 2;  // 16 KiB: one [64][128] tile of 2-byte elements

typedef __attribute__((ext_vector_type(4))) unsigned u32x4_v;

template <typename E> struct V8;
template <> struct V8<__bf16> { typedef bf16x8_v type; };
template <> struct V8<_Float16> { typedef f16x8_v type; };

__device__ __forceinline__ f32x16_v mfma(bf16x8_v a, bf16x8_v b, f32x16_v c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ f32x16_v mfma(f16x8_v a, f16x8_v b, f32x16_v c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b, c, 0, 0, 0);
}

// 8 elements of type E (16 bytes) -> 8 bf16
template <typename E>
__device__ __forceinline__ uint4 to_bf16(uint4 v) {
  if constexpr (std::is_same<E, __bf16>::value) {
    return v;
  } else {
    const f16x8_v h = __builtin_bit_cast(f16x8_v, v);
    bf16x8_v b;
#pragma unroll
    for (int e = 0; e < 8; ++e) b[e] = (__bf16)(float)h[e];
    return __builtin_bit_cast(uint4, b);
  }
}

// [64 rows][128 cols] tile: 256-byte rows of 16 chunks, chunk XOR (row & 7)
__device__ __forceinline__ int rowt(int row, int c) { return row * 256 + ((c ^ (row & 7)) << 4); }
// [128 rows][64 cols] tile: 128-byte rows of 8 chunks, chunk XOR (row & 7)
__device__ __forceinline__ int colt(int row, int c) { return row * 128 + ((c ^ (row & 7)) << 4); }

__device__ __forceinline__ void transpose8x8(const uint4 (&r)[8], uint4 (&t)[8]) {
  const uint32_t *rw = reinterpret_cast<const uint32_t *>(r);
  uint32_t *tw = reinterpret_cast<uint32_t *>(t);
#pragma unroll
  for (int p = 0; p < 4; ++p) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const uint32_t lo = rw[(2 * q) * 4 + p];
      const uint32_t hi = rw[(2 * q + 1) * 4 + p];
      tw[(2 * p) * 4 + q] = (lo & 0xFFFFu) | (hi << 16);
      tw[(2 * p + 1) * 4 + q] = (lo >> 16) | (hi & 0xFFFF0000u);
    }
  }
}

// One 8 x 8 block of a [64][128] tile of 2-byte elements: rows rb*8 .. +7,
// columns eb*8 .. +7; stored row-major or transposed, optionally converted
// from element type E to bf16 on the way.
struct Blk {
  uint4 v[8];
  __device__ __forceinline__ void load(const void *base, int64_t ld, int64_t row0, int rb,
                                       int eb) {
    const uint16_t *b = static_cast<const uint16_t *>(base);
#pragma unroll
    for (int kk = 0; kk < 8; ++kk)
      v[kk] = *reinterpret_cast<const uint4 *>(b + (row0 + rb * 8 + kk) * ld + eb * 8);
  }
  template <typename E>
  __device__ __forceinline__ void store_rows(char *t, int rb, int eb, bool to_bf) const {
#pragma unroll
    for (int kk = 0; kk < 8; ++kk)
      *reinterpret_cast<uint4 *>(t + rowt(rb * 8 + kk, eb)) = to_bf ? to_bf16<E>(v[kk]) : v[kk];
  }
  template <typename E>
  __device__ __forceinline__ void store_cols(char *t, int rb, int eb, bool to_bf) const {
    uint4 tr[8];
    transpose8x8(v, tr);
#pragma unroll
    for (int ee = 0; ee < 8; ++ee)
      *reinterpret_cast<uint4 *>(t + colt(eb * 8 + ee, rb)) = to_bf ? to_bf16<E>(tr[ee]) : tr[ee];
  }
};

// fragment of 8 elements from a [128][64] transposed tile: columns c..c+3 and
// c+8..c+11 of row `row` (c = 16*step + 4*half, so both runs sit in adjacent chunks)
template <typename VT>
__device__ __forceinline__ VT frag_cols(const char *t, int row, int c) {
  const uint2 lo = *reinterpret_cast<const uint2 *>(t + colt(row, c >> 3) + (c & 7) * 2);
  const uint2 hi = *reinterpret_cast<const uint2 *>(t + colt(row, (c >> 3) + 1) + (c & 7) * 2);
  const u32x4_v w = {lo.x, lo.y, hi.x, hi.y};
  return __builtin_bit_cast(VT, w);
}

template <typename VT>
__device__ __forceinline__ VT frag_rows(const char *t, int row, int chunk) {
  return *reinterpret_cast<const VT *>(t + rowt(row, chunk));
}

template <typename E>
__device__ __forceinline__ typename V8<E>::type pack8(const f32x16_v &a, int base) {
  typename V8<E>::type r;
#pragma unroll
  for (int e = 0; e < 8; ++e) r[e] = (E)a[base + e];
  return r;
}

// row index inside a 32-row MFMA output block held by register r of a lane in half hf
__device__ __forceinline__ int out_row(int r, int hf) { return (r & 3) + 8 * (r >> 2) + 4 * hf; }

struct AttnP {
  const void *q, *k, *v;   // q/k/v element type (template)
  __bf16 *o;
  float *lse;
  const __bf16 *dout;
  __bf16 *dq, *dk, *dv;
  float *D;
  const float *rcos, *rsin;
  int64_t ld_qkv, ld_o, ld_d;
  int S, H;
  float scale;  // 1/sqrt(hd)
};

// ---------------------------------------------------------------- forward
template <typename QE>
__global__ __launch_bounds__(256) void attn_fwd_kernel(AttnP p) {
  typedef typename V8<QE>::type QV;
  extern __shared__ __align__(16) char smem[];  // 2 stages x (K rows | V^T)
  const int nqb = p.S / QB;
  const int qb = nqb - 1 - (int)blockIdx.x;  // heaviest blocks first
  const int h = blockIdx.y, b = blockIdx.z;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int l32 = lane & 31, hf = lane >> 5;
  const int64_t row0 = (int64_t)b * p.S;
  const QE *Q = static_cast<const QE *>(p.q) + h * HD;
  const QE *K = static_cast<const QE *>(p.k) + h * HD;
  const QE *V = static_cast<const QE *>(p.v) + h * HD;
  const int q0 = qb * QB + w * 32;
  const int myq = q0 + l32;
  const float sc = p.scale * LOG2E;

  QV qf[8];
#pragma unroll
  for (int es = 0; es < 8; ++es)
    qf[es] = *reinterpret_cast<const QV *>(Q + (row0 + myq) * p.ld_qkv + es * 16 + hf * 8);

  f32x16_v o[4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int r = 0; r < 16; ++r) o[i][r] = 0.0f;
  float m = -1e30f, l = 0.0f;

  const bool isK = tid < 128;
  const int bt = tid & 127, rb = bt >> 4, eb = bt & 15;
  Blk blk;
  const int nkb = (qb + 1) * QB / KB;
  blk.load(isK ? (const void *)K : (const void *)V, p.ld_qkv, row0, rb, eb);
  if (isK) blk.store_rows<QE>(smem, rb, eb, false); else blk.store_cols<QE>(smem + TILE, rb, eb, false);
  __syncthreads();

  for (int kb = 0; kb < nkb; ++kb) {
    const int cur = kb & 1;
    const bool more = kb + 1 < nkb;
    if (more) blk.load(isK ? (const void *)K : (const void *)V, p.ld_qkv, row0 + (kb + 1) * KB, rb, eb);
    const char *sK = smem + cur * 2 * TILE;
    const char *sVt = sK + TILE;
    const int k0 = kb * KB;
    if (k0 <= q0 + 31) {
      f32x16_v s[2];
#pragma unroll
      for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r) s[j][r] = 0.0f;
#pragma unroll
      for (int es = 0; es < 8; ++es)
#pragma unroll
        for (int j = 0; j < 2; ++j)
          s[j] = mfma(frag_rows<QV>(sK, j * 32 + l32, es * 2 + hf), qf[es], s[j]);
      const bool diag = k0 + KB - 1 > q0;
      float mx = -INFINITY;
#pragma unroll
      for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          float v = s[j][r] * sc;
          if (diag && k0 + j * 32 + out_row(r, hf) > myq) v = -INFINITY;
          s[j][r] = v;
          mx = fmaxf(mx, v);
        }
      mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
      const float mn = fmaxf(m, mx);
      const float alpha = exp2f(m - mn);
      m = mn;
      float ls = 0.0f;
#pragma unroll
      for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const float pv = exp2f(s[j][r] - mn);
          s[j][r] = pv;
          ls += pv;
        }
      l = l * alpha + ls;
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int r = 0; r < 16; ++r) o[i][r] *= alpha;
#pragma unroll
      for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int t = 0; t < 2; ++t) {
          const QV pf = pack8<QE>(s[j], 8 * t);
          const int kc = j * 32 + 16 * t + 4 * hf;
#pragma unroll
          for (int i = 0; i < 4; ++i) o[i] = mfma(frag_cols<QV>(sVt, i * 32 + l32, kc), pf, o[i]);
        }
    }
    if (more) {
      char *nb = smem + (cur ^ 1) * 2 * TILE;
      if (isK) blk.store_rows<QE>(nb, rb, eb, false); else blk.store_cols<QE>(nb + TILE, rb, eb, false);
    }
    __syncthreads();
  }

  const float lt = l + __shfl_xor(l, 32, 64);
  const float inv = 1.0f / lt;
  __bf16 *orow = p.o + (row0 + myq) * p.ld_o + h * HD;
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      bf16x4_v wv = {(__bf16)(o[i][4 * g] * inv), (__bf16)(o[i][4 * g + 1] * inv),
                     (__bf16)(o[i][4 * g + 2] * inv), (__bf16)(o[i][4 * g + 3] * inv)};
      *reinterpret_cast<bf16x4_v *>(orow + i * 32 + 8 * g + 4 * hf) = wv;
    }
  if (hf == 0) p.lse[((int64_t)b * p.H + h) * p.S + myq] = (m + log2f(lt)) * LN2;
}

// ---------------------------------------------------------------- backward
// D[b,h,i] = sum_e dO[i,e] O[i,e]; one workgroup per token row, 16 lanes per head
__global__ __launch_bounds__(256) void attn_bwd_prep_kernel(AttnP p, int d) {
  const int64_t row = blockIdx.x;  // b*S + s
  const int b = (int)(row / p.S), s = (int)(row % p.S);
  for (int c = threadIdx.x * 8; c < d; c += 256 * 8) {
    const bf16x8_v a = *reinterpret_cast<const bf16x8_v *>(p.dout + row * p.ld_o + c);
    const bf16x8_v o = *reinterpret_cast<const bf16x8_v *>(p.o + row * p.ld_o + c);
    float acc = 0.0f;
#pragma unroll
    for (int i = 0; i < 8; ++i) acc += (float)a[i] * (float)o[i];
#pragma unroll
    for (int o2 = 8; o2 > 0; o2 >>= 1) acc += __shfl_xor(acc, o2, 64);
    if ((threadIdx.x & 15) == 0) p.D[((int64_t)b * p.H + c / HD) * p.S + s] = acc;
  }
}

__device__ __forceinline__ void rope_inverse_pairs(f32x16_v (&acc)[4], const float *rcos,
                                                   const float *rsin, int pos, int hf) {
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int e = i * 32 + out_row(r, hf);  // < 64; partner column e + 64
      const float c = rcos[pos * 64 + e], sn = rsin[pos * 64 + e];
      const float a = acc[i][r], bb = acc[i + 2][r];
      acc[i][r] = a * c + bb * sn;
      acc[i + 2][r] = bb * c - a * sn;
    }
}

// lane holds acc^T[e][token] for its own token; store that token's row (bf16)
__device__ __forceinline__ void store_row_t(__bf16 *row, const f32x16_v (&acc)[4], float mul, int hf) {
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      bf16x4_v wv = {(__bf16)(acc[i][4 * g] * mul), (__bf16)(acc[i][4 * g + 1] * mul),
                     (__bf16)(acc[i][4 * g + 2] * mul), (__bf16)(acc[i][4 * g + 3] * mul)};
      *reinterpret_cast<bf16x4_v *>(row + i * 32 + 8 * g + 4 * hf) = wv;
    }
}

// dQ: one workgroup per 128 queries; LDS stage = K rows (QE) | K^T (bf16) | V rows (bf16)
template <typename QE>
__global__ __launch_bounds__(256) void attn_bwd_dq_kernel(AttnP p) {
  typedef typename V8<QE>::type QV;
  extern __shared__ __align__(16) char smem[];
  const int nqb = p.S / QB;
  const int qb = nqb - 1 - (int)blockIdx.x;
  const int h = blockIdx.y, b = blockIdx.z;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int l32 = lane & 31, hf = lane >> 5;
  const int64_t row0 = (int64_t)b * p.S;
  const QE *K = static_cast<const QE *>(p.k) + h * HD;
  const QE *V = static_cast<const QE *>(p.v) + h * HD;
  const int q0 = qb * QB + w * 32;
  const int myq = q0 + l32;
  const float sc = p.scale * LOG2E;

  QV qf[8];
  bf16x8_v df[8];
#pragma unroll
  for (int es = 0; es < 8; ++es) {
    qf[es] = *reinterpret_cast<const QV *>(static_cast<const QE *>(p.q) + h * HD +
                                           (row0 + myq) * p.ld_qkv + es * 16 + hf * 8);
    df[es] = *reinterpret_cast<const bf16x8_v *>(p.dout + h * HD + (row0 + myq) * p.ld_o +
                                                 es * 16 + hf * 8);
  }
  const int64_t si = ((int64_t)b * p.H + h) * p.S + myq;
  const float lse2 = p.lse[si] * LOG2E;
  const float Dq = p.D[si];

  f32x16_v acc[4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[i][r] = 0.0f;

  const bool isK = tid < 128;
  const int bt = tid & 127, rb = bt >> 4, eb = bt & 15;
  constexpr int STAGE = 3 * TILE;
  Blk blk;
  const int nkb = (qb + 1) * QB / KB;
  auto put = [&](char *st) {
    if (isK) {
      blk.store_rows<QE>(st, rb, eb, false);
      blk.store_cols<QE>(st + TILE, rb, eb, true);
    } else {
      blk.store_rows<QE>(st + 2 * TILE, rb, eb, true);
    }
  };
  blk.load(isK ? (const void *)K : (const void *)V, p.ld_qkv, row0, rb, eb);
  put(smem);
  __syncthreads();
  for (int kb = 0; kb < nkb; ++kb) {
    const int cur = kb & 1;
    const bool more = kb + 1 < nkb;
    if (more) blk.load(isK ? (const void *)K : (const void *)V, p.ld_qkv, row0 + (kb + 1) * KB, rb, eb);
    const char *sK = smem + cur * STAGE, *sKt = sK + TILE, *sV = sK + 2 * TILE;
    const int k0 = kb * KB;
    if (k0 <= q0 + 31) {
      f32x16_v s[2], dp[2];
#pragma unroll
      for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r) s[j][r] = dp[j][r] = 0.0f;
#pragma unroll
      for (int es = 0; es < 8; ++es)
#pragma unroll
        for (int j = 0; j < 2; ++j) {
          s[j] = mfma(frag_rows<QV>(sK, j * 32 + l32, es * 2 + hf), qf[es], s[j]);
          dp[j] = mfma(frag_rows<bf16x8_v>(sV, j * 32 + l32, es * 2 + hf), df[es], dp[j]);
        }
      const bool diag = k0 + KB - 1 > q0;
#pragma unroll
      for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          float pv = exp2f(s[j][r] * sc - lse2);
          if (diag && k0 + j * 32 + out_row(r, hf) > myq) pv = 0.0f;
          dp[j][r] = pv * (dp[j][r] - Dq);
        }
#pragma unroll
      for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int t = 0; t < 2; ++t) {
          const bf16x8_v pf = pack8<__bf16>(dp[j], 8 * t);
          const int kc = j * 32 + 16 * t + 4 * hf;
#pragma unroll
          for (int i = 0; i < 4; ++i)
            acc[i] = mfma(frag_cols<bf16x8_v>(sKt, i * 32 + l32, kc), pf, acc[i]);
        }
    }
    if (more) put(smem + (cur ^ 1) * STAGE);
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[i][r] *= p.scale;
  if (p.rcos) rope_inverse_pairs(acc, p.rcos, p.rsin, myq, hf);
  store_row_t(p.dq + h * HD + (row0 + myq) * p.ld_d, acc, 1.0f, hf);
}

// dK, dV: one workgroup per 128 keys; LDS stage = Q rows (QE) | Q^T (bf16) |
// dO rows | dO^T | lse | D
template <typename QE>
__global__ __launch_bounds__(256) void attn_bwd_dkdv_kernel(AttnP p) {
  typedef typename V8<QE>::type QV;
  extern __shared__ __align__(16) char smem[];
  const int kblk = blockIdx.x;
  const int h = blockIdx.y, b = blockIdx.z;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int l32 = lane & 31, hf = lane >> 5;
  const int64_t row0 = (int64_t)b * p.S;
  const QE *Q = static_cast<const QE *>(p.q) + h * HD;
  const __bf16 *dO = p.dout + h * HD;
  const int k0w = kblk * QB + w * 32;
  const int myk = k0w + l32;
  const float sc = p.scale * LOG2E;

  QV kf[8];
  bf16x8_v vf[8];
#pragma unroll
  for (int es = 0; es < 8; ++es) {
    const int64_t off = h * HD + (row0 + myk) * p.ld_qkv + es * 16 + hf * 8;
    kf[es] = *reinterpret_cast<const QV *>(static_cast<const QE *>(p.k) + off);
    const uint4 raw = *reinterpret_cast<const uint4 *>(static_cast<const QE *>(p.v) + off);
    vf[es] = __builtin_bit_cast(bf16x8_v, to_bf16<QE>(raw));
  }
  f32x16_v dk[4], dv[4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int r = 0; r < 16; ++r) dk[i][r] = dv[i][r] = 0.0f;

  const bool isQ = tid < 128;
  const int bt = tid & 127, rb = bt >> 4, eb = bt & 15;
  constexpr int STAGE = 4 * TILE + 512;
  const int64_t sbase = ((int64_t)b * p.H + h) * p.S;
  Blk blk;
  float sv = 0.0f;  // lse (threads 0..63) or D (threads 64..127) of the staged block
  auto fetch = [&](int qbi) {
    blk.load(isQ ? (const void *)Q : (const void *)dO, isQ ? p.ld_qkv : p.ld_o, row0 + qbi * KB, rb, eb);
    if (tid < 64) sv = p.lse[sbase + qbi * KB + tid] * LOG2E;
    else if (tid < 128) sv = p.D[sbase + qbi * KB + tid - 64];
  };
  auto put = [&](char *st) {
    if (isQ) {
      blk.store_rows<QE>(st, rb, eb, false);
      blk.store_cols<QE>(st + TILE, rb, eb, true);
    } else {
      blk.store_rows<__bf16>(st + 2 * TILE, rb, eb, false);
      blk.store_cols<__bf16>(st + 3 * TILE, rb, eb, false);
    }
    if (tid < 128) reinterpret_cast<float *>(st + 4 * TILE)[tid] = sv;
  };
  const int qfirst = kblk * QB / KB, nqblk = p.S / KB;
  fetch(qfirst);
  put(smem);
  __syncthreads();
  for (int qbi = qfirst; qbi < nqblk; ++qbi) {
    const int cur = (qbi - qfirst) & 1;
    const bool more = qbi + 1 < nqblk;
    if (more) fetch(qbi + 1);
    const char *sQ = smem + cur * STAGE, *sQt = sQ + TILE, *sD = sQ + 2 * TILE, *sDt = sQ + 3 * TILE;
    const float *sL = reinterpret_cast<const float *>(sQ + 4 * TILE);
    const int q0 = qbi * KB;
    if (q0 + KB - 1 >= k0w) {
      f32x16_v s[2], dp[2];
#pragma unroll
      for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r) s[j][r] = dp[j][r] = 0.0f;
#pragma unroll
      for (int es = 0; es < 8; ++es)
#pragma unroll
        for (int j = 0; j < 2; ++j) {
          s[j] = mfma(frag_rows<QV>(sQ, j * 32 + l32, es * 2 + hf), kf[es], s[j]);
          dp[j] = mfma(frag_rows<bf16x8_v>(sD, j * 32 + l32, es * 2 + hf), vf[es], dp[j]);
        }
      const bool diag = q0 < k0w + 31;
#pragma unroll
      for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int qi = j * 32 + out_row(r, hf);
          float pv = exp2f(s[j][r] * sc - sL[qi]);
          if (diag && q0 + qi < myk) pv = 0.0f;
          s[j][r] = pv;
          dp[j][r] = pv * (dp[j][r] - sL[64 + qi]);
        }
#pragma unroll
      for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int t = 0; t < 2; ++t) {
          const bf16x8_v pf = pack8<__bf16>(s[j], 8 * t);
          const bf16x8_v sf = pack8<__bf16>(dp[j], 8 * t);
          const int qc = j * 32 + 16 * t + 4 * hf;
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            dv[i] = mfma(frag_cols<bf16x8_v>(sDt, i * 32 + l32, qc), pf, dv[i]);
            dk[i] = mfma(frag_cols<bf16x8_v>(sQt, i * 32 + l32, qc), sf, dk[i]);
          }
        }
    }
    if (more) put(smem + (cur ^ 1) * STAGE);
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int r = 0; r < 16; ++r) dk[i][r] *= p.scale;
  if (p.rcos) rope_inverse_pairs(dk, p.rcos, p.rsin, myk, hf);
  store_row_t(p.dk + h * HD + (row0 + myk) * p.ld_d, dk, 1.0f, hf);
  store_row_t(p.dv + h * HD + (row0 + myk) * p.ld_d, dv, 1.0f, hf);
}

// ---------------------------------------------------------------- fp32 path
// Plain kernels: one thread per (batch row, head, query) or (..., key).
struct AttnF {
  const float *q, *k, *v;
  float *o;
  float *lse;
  const float *dout;
  float *dq, *dk, *dv;
  float *D;
  const float *rcos, *rsin;
  int64_t ld_qkv, ld_o, ld_d;
  int B, S, H, hd;
  float scale;
};

constexpr int MAXHD = 128;

__global__ void attn_fwd_f32_kernel(AttnF p) {
  const int64_t id = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
  if (id >= (int64_t)p.B * p.H * p.S) return;
  const int i = (int)(id % p.S), h = (int)((id / p.S) % p.H), b = (int)(id / ((int64_t)p.S * p.H));
  const int64_t r0 = (int64_t)b * p.S;
  const float *qi = p.q + (r0 + i) * p.ld_qkv + h * p.hd;
  float acc[MAXHD];
  for (int e = 0; e < p.hd; ++e) acc[e] = 0.0f;
  float m = -INFINITY, l = 0.0f;
  for (int j = 0; j <= i; ++j) {
    const float *kj = p.k + (r0 + j) * p.ld_qkv + h * p.hd;
    float s = 0.0f;
    for (int e = 0; e < p.hd; ++e) s += qi[e] * kj[e];
    s *= p.scale;
    const float mn = fmaxf(m, s);
    const float a = expf(m - mn), w = expf(s - mn);
    l = l * a + w;
    const float *vj = p.v + (r0 + j) * p.ld_qkv + h * p.hd;
    for (int e = 0; e < p.hd; ++e) acc[e] = acc[e] * a + w * vj[e];
    m = mn;
  }
  float *oi = p.o + (r0 + i) * p.ld_o + h * p.hd;
  for (int e = 0; e < p.hd; ++e) oi[e] = acc[e] / l;
  p.lse[((int64_t)b * p.H + h) * p.S + i] = m + logf(l);
}

__device__ void rope_inv_vec(float *x, int hd, int pos, const float *rc, const float *rs) {
  const int half = hd / 2;
  for (int e = 0; e < half; ++e) {
    const float c = rc[pos * half + e], s = rs[pos * half + e];
    const float a = x[e], bb = x[e + half];
    x[e] = a * c + bb * s;
    x[e + half] = bb * c - a * s;
  }
}

// per query: D_i and dq_i
__global__ void attn_bwd_q_f32_kernel(AttnF p) {
  const int64_t id = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
  if (id >= (int64_t)p.B * p.H * p.S) return;
  const int i = (int)(id % p.S), h = (int)((id / p.S) % p.H), b = (int)(id / ((int64_t)p.S * p.H));
  const int64_t r0 = (int64_t)b * p.S;
  const float *qi = p.q + (r0 + i) * p.ld_qkv + h * p.hd;
  const float *doi = p.dout + (r0 + i) * p.ld_o + h * p.hd;
  const float *oi = p.o + (r0 + i) * p.ld_o + h * p.hd;
  float Di = 0.0f;
  for (int e = 0; e < p.hd; ++e) Di += doi[e] * oi[e];
  const int64_t si = ((int64_t)b * p.H + h) * p.S + i;
  p.D[si] = Di;
  const float L = p.lse[si];
  float acc[MAXHD];
  for (int e = 0; e < p.hd; ++e) acc[e] = 0.0f;
  for (int j = 0; j <= i; ++j) {
    const float *kj = p.k + (r0 + j) * p.ld_qkv + h * p.hd;
    const float *vj = p.v + (r0 + j) * p.ld_qkv + h * p.hd;
    float s = 0.0f, dp = 0.0f;
    for (int e = 0; e < p.hd; ++e) {
      s += qi[e] * kj[e];
      dp += doi[e] * vj[e];
    }
    const float P = expf(s * p.scale - L);
    const float dS = P * (dp - Di);
    for (int e = 0; e < p.hd; ++e) acc[e] += dS * kj[e];
  }
  for (int e = 0; e < p.hd; ++e) acc[e] *= p.scale;
  if (p.rcos) rope_inv_vec(acc, p.hd, i, p.rcos, p.rsin);
  float *dqi = p.dq + (r0 + i) * p.ld_d + h * p.hd;
  for (int e = 0; e < p.hd; ++e) dqi[e] = acc[e];
}

// per key: dk_j and dv_j (needs D from the kernel above)
__global__ void attn_bwd_kv_f32_kernel(AttnF p) {
  const int64_t id = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
  if (id >= (int64_t)p.B * p.H * p.S) return;
  const int j = (int)(id % p.S), h = (int)((id / p.S) % p.H), b = (int)(id / ((int64_t)p.S * p.H));
  const int64_t r0 = (int64_t)b * p.S;
  const float *kj = p.k + (r0 + j) * p.ld_qkv + h * p.hd;
  const float *vj = p.v + (r0 + j) * p.ld_qkv + h * p.hd;
  float ak[MAXHD], av[MAXHD];
  for (int e = 0; e < p.hd; ++e) ak[e] = av[e] = 0.0f;
  for (int i = j; i < p.S; ++i) {
    const float *qi = p.q + (r0 + i) * p.ld_qkv + h * p.hd;
    const float *doi = p.dout + (r0 + i) * p.ld_o + h * p.hd;
    float s = 0.0f, dp = 0.0f;
    for (int e = 0; e < p.hd; ++e) {
      s += qi[e] * kj[e];
      dp += doi[e] * vj[e];
    }
    const int64_t si = ((int64_t)b * p.H + h) * p.S + i;
    const float P = expf(s * p.scale - p.lse[si]);
    const float dS = P * (dp - p.D[si]);
    for (int e = 0; e < p.hd; ++e) {
      av[e] += P * doi[e];
      ak[e] += dS * qi[e];
    }
  }
  for (int e = 0; e < p.hd; ++e) ak[e] *= p.scale;
  if (p.rcos) rope_inv_vec(ak, p.hd, j, p.rcos, p.rsin);
  float *dkj = p.dk + (r0 + j) * p.ld_d + h * p.hd;
  float *dvj = p.dv + (r0 + j) * p.ld_d + h * p.hd;
  for (int e = 0; e < p.hd; ++e) {
    dkj[e] = ak[e];
    dvj[e] = av[e];
  }
}

lc_status set_lds(const void *fn, size_t bytes) {
  hipError_t e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)bytes);
  return e == hipSuccess ? LC_OK : hip_fail(e, "attention: setting the LDS size");
}

lc_status check_common(const lc_attn_args &a, bool bwd) {
  if (a.B <= 0 || a.S <= 0 || a.H <= 0 || a.hd <= 0)
    return fail(LC_ERR_INVALID_ARG, "attention: dimensions must be positive");
  if (a.ld_qkv < (int64_t)a.H * a.hd || a.ld_o < (int64_t)a.H * a.hd)
    return fail(LC_ERR_INVALID_ARG, "attention: leading dimension smaller than H*hd");
  if (!a.q || !a.k || !a.v || !a.o || !a.lse) return fail(LC_ERR_INVALID_ARG, "attention: null pointer");
  if (!aligned16(a.q) || !aligned16(a.k) || !aligned16(a.v) || !aligned16(a.o))
    return fail(LC_ERR_INVALID_ARG, "attention: unaligned pointer");
  if (bwd) {
    if (!a.dout || !a.dq || !a.dk || !a.dv) return fail(LC_ERR_INVALID_ARG, "attention: null pointer");
    if (!aligned16(a.dout) || !aligned16(a.dq) || !aligned16(a.dk) || !aligned16(a.dv))
      return fail(LC_ERR_INVALID_ARG, "attention: unaligned pointer");
    if (a.ld_dqkv < (int64_t)a.H * a.hd) return fail(LC_ERR_INVALID_ARG, "attention: ld_dqkv too small");
    if ((a.rope_cos == nullptr) != (a.rope_sin == nullptr))
      return fail(LC_ERR_INVALID_ARG, "attention: give both RoPE tables or neither");
    if (!a.scratch || a.scratch_bytes < attn_scratch_size(a.B, a.S, a.H))
      return fail(LC_ERR_WORKSPACE, "attention backward: scratch too small");
  }
  if (a.dtype == LC_BF16 || a.dtype == LC_FP16) {
    if (a.o_dtype != LC_BF16) return fail(LC_ERR_UNSUPPORTED, "attention: o/gradients must be bf16");
    if (a.hd != HD) return fail(LC_ERR_UNSUPPORTED, "attention (matrix cores): head_dim must be 128");
    if (a.S % QB) return fail(LC_ERR_UNSUPPORTED, "attention (matrix cores): seq_len %% 128 != 0");
    if (a.ld_qkv % 8 || a.ld_o % 8 || (bwd && a.ld_dqkv % 8))
      return fail(LC_ERR_INVALID_ARG, "attention: ld %% 8 != 0");
    if (bwd && a.rope_cos && (!aligned16(a.rope_cos) || !aligned16(a.rope_sin)))
      return fail(LC_ERR_INVALID_ARG, "attention: unaligned RoPE table");
  } else if (a.dtype == LC_FP32) {
    if (a.o_dtype != LC_FP32) return fail(LC_ERR_UNSUPPORTED, "attention fp32: o must be fp32");
    if (a.hd > MAXHD || a.hd % 2) return fail(LC_ERR_UNSUPPORTED, "attention fp32: even head_dim <= 128");
  } else {
    return fail(LC_ERR_INVALID_ARG, "attention: unknown dtype");
  }
  return LC_OK;
}

AttnP mc_params(const lc_attn_args &a) {
  AttnP p{};
  p.q = a.q;
  p.k = a.k;
  p.v = a.v;
  p.o = static_cast<__bf16 *>(a.o);
  p.lse = a.lse;
  p.dout = static_cast<const __bf16 *>(a.dout);
  p.dq = static_cast<__bf16 *>(a.dq);
  p.dk = static_cast<__bf16 *>(a.dk);
  p.dv = static_cast<__bf16 *>(a.dv);
  p.D = static_cast<float *>(a.scratch);
  p.rcos = a.rope_cos;
  p.rsin = a.rope_sin;
  p.ld_qkv = a.ld_qkv;
  p.ld_o = a.ld_o;
  p.ld_d = a.ld_dqkv;
  p.S = a.S;
  p.H = a.H;
  p.scale = 1.0f / sqrtf((float)a.hd);
  return p;
}

AttnF f32_params(const lc_attn_args &a) {
  AttnF p{};
  p.q = static_cast<const float *>(a.q);
  p.k = static_cast<const float *>(a.k);
  p.v = static_cast<const float *>(a.v);
  p.o = static_cast<float *>(a.o);
  p.lse = a.lse;
  p.dout = static_cast<const float *>(a.dout);
  p.dq = static_cast<float *>(a.dq);
  p.dk = static_cast<float *>(a.dk);
  p.dv = static_cast<float *>(a.dv);
  p.D = static_cast<float *>(a.scratch);
  p.rcos = a.rope_cos;
  p.rsin = a.rope_sin;
  p.ld_qkv = a.ld_qkv;
  p.ld_o = a.ld_o;
  p.ld_d = a.ld_dqkv;
  p.B = a.B; p.S = a.S; p.H = a.H; p.hd = a.hd;
  p.scale = 1.0f / sqrtf((float)a.hd);
  return p;
}

template <typename QE>
lc_status fwd_mc(const lc_attn_args &a, hipStream_t s) {
  const size_t lds = 2 * 2 * TILE;
  static bool once = false;
  if (!once) { LC_TRY(set_lds((const void *)attn_fwd_kernel<QE>, lds)); once = true; }
  hipLaunchKernelGGL(attn_fwd_kernel<QE>, dim3(a.S / QB, a.H, a.B), dim3(256), lds, s, mc_params(a));
  return check_launch("attn_fwd_kernel");
}

template <typename QE>
lc_status bwd_mc(const lc_attn_args &a, hipStream_t s) {
  const AttnP p = mc_params(a);
  hipLaunchKernelGGL(attn_bwd_prep_kernel, dim3((unsigned)((int64_t)a.B * a.S)), dim3(256), 0, s, p,
                     a.H * HD);
  LC_TRY(check_launch("attn_bwd_prep_kernel"));
  const size_t lds_dq = 2 * 3 * TILE, lds_kv = 2 * (4 * TILE + 512);
  static bool once = false;
  if (!once) {
    LC_TRY(set_lds((const void *)attn_bwd_dq_kernel<QE>, lds_dq));
    LC_TRY(set_lds((const void *)attn_bwd_dkdv_kernel<QE>, lds_kv));
    once = true;
  }
  hipLaunchKernelGGL(attn_bwd_dkdv_kernel<QE>, dim3(a.S / QB, a.H, a.B), dim3(256), lds_kv, s, p);
  LC_TRY(check_launch("attn_bwd_dkdv_kernel"));
  hipLaunchKernelGGL(attn_bwd_dq_kernel<QE>, dim3(a.S / QB, a.H, a.B), dim3(256), lds_dq, s, p);
  return check_launch("attn_bwd_dq_kernel");
}

}  // namespace

lc_status attn_fwd_launch(const lc_attn_args &a, hipStream_t s) {
  LC_TRY(check_common(a, false));
  if (a.dtype == LC_FP16) return fwd_mc<_Float16>(a, s);
  if (a.dtype == LC_BF16) return fwd_mc<__bf16>(a, s);
  const AttnF p = f32_params(a);
  const int64_t n = (int64_t)a.B * a.H * a.S;
  hipLaunchKernelGGL(attn_fwd_f32_kernel, dim3((unsigned)((n + 127) / 128)), dim3(128), 0, s, p);
  return check_launch("attn_fwd_f32_kernel");
}

lc_status attn_bwd_launch(const lc_attn_args &a, hipStream_t s) {
  LC_TRY(check_common(a, true));
  if (a.dtype == LC_FP16) return bwd_mc<_Float16>(a, s);
  if (a.dtype == LC_BF16) return bwd_mc<__bf16>(a, s);
  const AttnF p = f32_params(a);
  const int64_t n = (int64_t)a.B * a.H * a.S;
  const dim3 grid((unsigned)((n + 127) / 128));
  hipLaunchKernelGGL(attn_bwd_q_f32_kernel, grid, dim3(128), 0, s, p);
  LC_TRY(check_launch("attn_bwd_q_f32_kernel"));
  hipLaunchKernelGGL(attn_bwd_kv_f32_kernel, grid, dim3(128), 0, s, p);
  return check_launch("attn_bwd_kv_f32_kernel");
}

}  // namespace lc

extern "C" {

lc_status lc_attention_forward(const lc_attn_args *args, void *stream) {
  if (!args) return lc::fail(LC_ERR_INVALID_ARG, "attention: null args");
  return lc::attn_fwd_launch(*args, static_cast<hipStream_t>(stream));
}

lc_status lc_attention_backward(const lc_attn_args *args, void *stream) {
  if (!args) return lc::fail(LC_ERR_INVALID_ARG, "attention: null args");
  return lc::attn_bwd_launch(*args, static_cast<hipStream_t>(stream));
}

}  // extern "C"
