// Causal softmax attention on CDNA4 matrix cores (head_dim 128, bf16 operands,
// fp32 softmax and accumulation), plus a plain fp32 path.
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
// V^T fragment is read from LDS in the same key order.
//
// Backward (deterministic, no atomics): D = rowsum(dO * O) first; then one
// kernel per query block recomputes P^T from the saved log-sum-exp and
// accumulates dQ^T = K^T dS^T over keys, and one kernel per key block
// accumulates dV^T = dO^T P and dK^T = Q^T dS over queries (S computed
// untransposed there so the key is the lane index). RoPE's inverse rotation
// of dq/dk is applied in the epilogue. LDS tiles are filled from 8 x 8
// blocks read once from HBM and written both row-major and transposed.
#include "common.hpp"

#include <math.h>

namespace lc {
namespace {

constexpr int HD = 128;
constexpr int QB = 128;  // queries (or keys) per workgroup
constexpr int KB = 64;   // keys (or queries) per inner step
constexpr float LOG2E = 1.4426950408889634f;
constexpr float LN2 = 0.6931471805599453f;
constexpr int TILE = KB * HD * 2;  // 16 KiB: one [64][128] bf16 tile

typedef __attribute__((ext_vector_type(4))) unsigned u32x4_v;

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

// One 8 x 8 block of a [64][128] tile: rows rb*8 .. +7, columns eb*8 .. +7.
struct Blk {
  uint4 v[8];
  __device__ __forceinline__ void load(const bf16_t *base, int64_t ld, int64_t row0, int rb,
                                       int eb) {
#pragma unroll
    for (int kk = 0; kk < 8; ++kk)
      v[kk] = *reinterpret_cast<const uint4 *>(base + (row0 + rb * 8 + kk) * ld + eb * 8);
  }
  __device__ __forceinline__ void store_rows(char *t, int rb, int eb) const {
#pragma unroll
    for (int kk = 0; kk < 8; ++kk) *reinterpret_cast<uint4 *>(t + rowt(rb * 8 + kk, eb)) = v[kk];
  }
  __device__ __forceinline__ void store_cols(char *t, int rb, int eb) const {
    uint4 tr[8];
    transpose8x8(v, tr);
#pragma unroll
    for (int ee = 0; ee < 8; ++ee) *reinterpret_cast<uint4 *>(t + colt(eb * 8 + ee, rb)) = tr[ee];
  }
};

// B/A fragment of 8 bf16 from a [128][64] transposed tile: columns c..c+3 and
// c+8..c+11 of row `row` (c = 16*step + 4*half, so both runs sit in adjacent chunks).
__device__ __forceinline__ bf16x8_v frag_cols(const char *t, int row, int c) {
  const uint2 lo = *reinterpret_cast<const uint2 *>(t + colt(row, c >> 3) + (c & 7) * 2);
  const uint2 hi = *reinterpret_cast<const uint2 *>(t + colt(row, (c >> 3) + 1) + (c & 7) * 2);
  const u32x4_v w = {lo.x, lo.y, hi.x, hi.y};
  return __builtin_bit_cast(bf16x8_v, w);
}

__device__ __forceinline__ bf16x8_v frag_rows(const char *t, int row, int chunk) {
  return *reinterpret_cast<const bf16x8_v *>(t + rowt(row, chunk));
}

__device__ __forceinline__ bf16x8_v pack8(const f32x16_v &a, int base) {
  bf16x8_v r;
#pragma unroll
  for (int e = 0; e < 8; ++e) r[e] = (__bf16)a[base + e];
  return r;
}

__device__ __forceinline__ f32x16_v mfma(bf16x8_v a, bf16x8_v b, f32x16_v c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

// row index inside a 32-row MFMA output block held by register r of a lane in half hf
__device__ __forceinline__ int out_row(int r, int hf) { return (r & 3) + 8 * (r >> 2) + 4 * hf; }

struct AttnP {
  const bf16_t *q, *k, *v;
  bf16_t *o;
  float *lse;
  const bf16_t *dout;
  bf16_t *dq, *dk, *dv;
  const float *D;
  const float *rcos, *rsin;
  int64_t ld_qkv, ld_o, ld_d;
  int S, H;
  float scale;  // 1/sqrt(hd)
};

// ---------------------------------------------------------------- forward
__global__ __launch_bounds__(256) void attn_fwd_kernel(AttnP p) {
  extern __shared__ __align__(16) char smem[];  // 2 stages x (K rows | V^T)
  const int nqb = p.S / QB;
  const int qb = nqb - 1 - (int)blockIdx.x;  // heaviest blocks first
  const int h = blockIdx.y, b = blockIdx.z;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int l32 = lane & 31, hf = lane >> 5;
  const int64_t row0 = (int64_t)b * p.S;
  const bf16_t *Q = p.q + h * HD, *K = p.k + h * HD, *V = p.v + h * HD;
  const int q0 = qb * QB + w * 32;
  const int myq = q0 + l32;
  const float sc = p.scale * LOG2E;

  bf16x8_v qf[8];
#pragma unroll
  for (int es = 0; es < 8; ++es)
    qf[es] = *reinterpret_cast<const bf16x8_v *>(Q + (row0 + myq) * p.ld_qkv + es * 16 + hf * 8);

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
  blk.load(isK ? K : V, p.ld_qkv, row0, rb, eb);
  if (isK) blk.store_rows(smem, rb, eb); else blk.store_cols(smem + TILE, rb, eb);
  __syncthreads();

  for (int kb = 0; kb < nkb; ++kb) {
    const int cur = kb & 1;
    const bool more = kb + 1 < nkb;
    if (more) blk.load(isK ? K : V, p.ld_qkv, row0 + (kb + 1) * KB, rb, eb);
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
        for (int j = 0; j < 2; ++j) s[j] = mfma(frag_rows(sK, j * 32 + l32, es * 2 + hf), qf[es], s[j]);
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
          const bf16x8_v pf = pack8(s[j], 8 * t);
          const int kc = j * 32 + 16 * t + 4 * hf;
#pragma unroll
          for (int i = 0; i < 4; ++i) o[i] = mfma(frag_cols(sVt, i * 32 + l32, kc), pf, o[i]);
        }
    }
    if (more) {
      char *nb = smem + (cur ^ 1) * 2 * TILE;
      if (isK) blk.store_rows(nb, rb, eb); else blk.store_cols(nb + TILE, rb, eb);
    }
    __syncthreads();
  }

  const float lt = l + __shfl_xor(l, 32, 64);
  const float inv = 1.0f / lt;
  bf16_t *orow = p.o + (row0 + myq) * p.ld_o + h * HD;
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      uint2 wv;
      wv.x = pack_bf2(o[i][4 * g] * inv, o[i][4 * g + 1] * inv);
      wv.y = pack_bf2(o[i][4 * g + 2] * inv, o[i][4 * g + 3] * inv);
      *reinterpret_cast<uint2 *>(orow + i * 32 + 8 * g + 4 * hf) = wv;
    }
  if (hf == 0) p.lse[((int64_t)b * p.H + h) * p.S + myq] = (m + log2f(lt)) * LN2;
}

// ---------------------------------------------------------------- backward
// D[b,h,i] = sum_e dO[i,e] O[i,e]; one workgroup per token row, 16 lanes per head
__global__ __launch_bounds__(256) void attn_bwd_prep_kernel(AttnP p, int d) {
  const int64_t row = blockIdx.x;  // b*S + s
  const int b = (int)(row / p.S), s = (int)(row % p.S);
  for (int c = threadIdx.x * 8; c < d; c += 256 * 8) {
    const uint4 a = *reinterpret_cast<const uint4 *>(p.dout + row * p.ld_o + c);
    const uint4 o = *reinterpret_cast<const uint4 *>(p.o + row * p.ld_o + c);
    const uint32_t aw[4] = {a.x, a.y, a.z, a.w}, ow[4] = {o.x, o.y, o.z, o.w};
    float acc = 0.0f;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      acc += __uint_as_float(aw[i] << 16) * __uint_as_float(ow[i] << 16);
      acc += __uint_as_float(aw[i] & 0xFFFF0000u) * __uint_as_float(ow[i] & 0xFFFF0000u);
    }
#pragma unroll
    for (int o2 = 8; o2 > 0; o2 >>= 1) acc += __shfl_xor(acc, o2, 64);
    if ((threadIdx.x & 15) == 0) {
      const int h = c / HD;
      const_cast<float *>(p.D)[((int64_t)b * p.H + h) * p.S + s] = acc;
    }
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

// lane holds acc^T[e][token] for token = its own; store the token's row
__device__ __forceinline__ void store_row_t(bf16_t *row, const f32x16_v (&acc)[4], float mul, int hf) {
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      uint2 wv;
      wv.x = pack_bf2(acc[i][4 * g] * mul, acc[i][4 * g + 1] * mul);
      wv.y = pack_bf2(acc[i][4 * g + 2] * mul, acc[i][4 * g + 3] * mul);
      *reinterpret_cast<uint2 *>(row + i * 32 + 8 * g + 4 * hf) = wv;
    }
}

// dQ: one workgroup per 128 queries; LDS stage = K rows | K^T | V rows
__global__ __launch_bounds__(256) void attn_bwd_dq_kernel(AttnP p) {
  extern __shared__ __align__(16) char smem[];
  const int nqb = p.S / QB;
  const int qb = nqb - 1 - (int)blockIdx.x;
  const int h = blockIdx.y, b = blockIdx.z;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int l32 = lane & 31, hf = lane >> 5;
  const int64_t row0 = (int64_t)b * p.S;
  const bf16_t *K = p.k + h * HD, *V = p.v + h * HD;
  const int q0 = qb * QB + w * 32;
  const int myq = q0 + l32;
  const float sc = p.scale * LOG2E;

  bf16x8_v qf[8], df[8];
#pragma unroll
  for (int es = 0; es < 8; ++es) {
    qf[es] = *reinterpret_cast<const bf16x8_v *>(p.q + h * HD + (row0 + myq) * p.ld_qkv + es * 16 + hf * 8);
    df[es] = *reinterpret_cast<const bf16x8_v *>(p.dout + h * HD + (row0 + myq) * p.ld_o + es * 16 + hf * 8);
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
      blk.store_rows(st, rb, eb);
      blk.store_cols(st + TILE, rb, eb);
    } else {
      blk.store_rows(st + 2 * TILE, rb, eb);
    }
  };
  blk.load(isK ? K : V, p.ld_qkv, row0, rb, eb);
  put(smem);
  __syncthreads();
  for (int kb = 0; kb < nkb; ++kb) {
    const int cur = kb & 1;
    const bool more = kb + 1 < nkb;
    if (more) blk.load(isK ? K : V, p.ld_qkv, row0 + (kb + 1) * KB, rb, eb);
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
          s[j] = mfma(frag_rows(sK, j * 32 + l32, es * 2 + hf), qf[es], s[j]);
          dp[j] = mfma(frag_rows(sV, j * 32 + l32, es * 2 + hf), df[es], dp[j]);
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
          const bf16x8_v pf = pack8(dp[j], 8 * t);
          const int kc = j * 32 + 16 * t + 4 * hf;
#pragma unroll
          for (int i = 0; i < 4; ++i) acc[i] = mfma(frag_cols(sKt, i * 32 + l32, kc), pf, acc[i]);
        }
    }
    if (more) put(smem + (cur ^ 1) * STAGE);
    __syncthreads();
  }
  if (p.rcos) {
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][r] *= p.scale;
    rope_inverse_pairs(acc, p.rcos, p.rsin, myq, hf);
    store_row_t(p.dq + h * HD + (row0 + myq) * p.ld_d, acc, 1.0f, hf);
  } else {
    store_row_t(p.dq + h * HD + (row0 + myq) * p.ld_d, acc, p.scale, hf);
  }
}

// dK, dV: one workgroup per 128 keys; LDS stage = Q rows | Q^T | dO rows | dO^T | lse | D
__global__ __launch_bounds__(256) void attn_bwd_dkdv_kernel(AttnP p) {
  extern __shared__ __align__(16) char smem[];
  const int kblk = blockIdx.x;
  const int h = blockIdx.y, b = blockIdx.z;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int l32 = lane & 31, hf = lane >> 5;
  const int64_t row0 = (int64_t)b * p.S;
  const bf16_t *Q = p.q + h * HD, *dO = p.dout + h * HD;
  const int k0w = kblk * QB + w * 32;
  const int myk = k0w + l32;
  const float sc = p.scale * LOG2E;

  bf16x8_v kf[8], vf[8];
#pragma unroll
  for (int es = 0; es < 8; ++es) {
    kf[es] = *reinterpret_cast<const bf16x8_v *>(p.k + h * HD + (row0 + myk) * p.ld_qkv + es * 16 + hf * 8);
    vf[es] = *reinterpret_cast<const bf16x8_v *>(p.v + h * HD + (row0 + myk) * p.ld_qkv + es * 16 + hf * 8);
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
    blk.load(isQ ? Q : dO, isQ ? p.ld_qkv : p.ld_o, row0 + qbi * KB, rb, eb);
    if (tid < 64) sv = p.lse[sbase + qbi * KB + tid] * LOG2E;
    else if (tid < 128) sv = p.D[sbase + qbi * KB + tid - 64];
  };
  auto put = [&](char *st) {
    char *t = isQ ? st : st + 2 * TILE;
    blk.store_rows(t, rb, eb);
    blk.store_cols(t + TILE, rb, eb);
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
          s[j] = mfma(frag_rows(sQ, j * 32 + l32, es * 2 + hf), kf[es], s[j]);
          dp[j] = mfma(frag_rows(sD, j * 32 + l32, es * 2 + hf), vf[es], dp[j]);
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
          const bf16x8_v pf = pack8(s[j], 8 * t);
          const bf16x8_v sf = pack8(dp[j], 8 * t);
          const int qc = j * 32 + 16 * t + 4 * hf;
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            dv[i] = mfma(frag_cols(sDt, i * 32 + l32, qc), pf, dv[i]);
            dk[i] = mfma(frag_cols(sQt, i * 32 + l32, qc), sf, dk[i]);
          }
        }
    }
    if (more) put(smem + (cur ^ 1) * STAGE);
    __syncthreads();
  }
  const int pos = myk;
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int r = 0; r < 16; ++r) dk[i][r] *= p.scale;
  if (p.rcos) rope_inverse_pairs(dk, p.rcos, p.rsin, pos, hf);
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

lc_status check_common(int dtype, int B, int S, int H, int hd, int64_t ld_qkv, int64_t ld_o) {
  if (B <= 0 || S <= 0 || H <= 0 || hd <= 0)
    return fail(LC_ERR_INVALID_ARG, "attention: dimensions must be positive");
  if (ld_qkv < (int64_t)H * hd || ld_o < (int64_t)H * hd)
    return fail(LC_ERR_INVALID_ARG, "attention: leading dimension smaller than H*hd");
  if (dtype == LC_BF16) {
    if (hd != HD) return fail(LC_ERR_UNSUPPORTED, "attention bf16: head_dim must be 128");
    if (S % QB) return fail(LC_ERR_UNSUPPORTED, "attention bf16: seq_len %% 128 != 0");
    if (ld_qkv % 8 || ld_o % 8) return fail(LC_ERR_INVALID_ARG, "attention: ld %% 8 != 0");
  } else if (dtype == LC_FP32) {
    if (hd > MAXHD || hd % 2) return fail(LC_ERR_UNSUPPORTED, "attention fp32: even head_dim <= 128");
  } else {
    return fail(LC_ERR_INVALID_ARG, "attention: unknown dtype");
  }
  return LC_OK;
}

}  // namespace

lc_status attn_fwd_launch(int dtype, int B, int S, int H, int hd, const void *q, const void *k,
                          const void *v, int64_t ld_qkv, void *o, int64_t ld_o, float *lse,
                          hipStream_t s) {
  LC_TRY(check_common(dtype, B, S, H, hd, ld_qkv, ld_o));
  if (!q || !k || !v || !o || !lse) return fail(LC_ERR_INVALID_ARG, "attention: null pointer");
  if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(o))
    return fail(LC_ERR_INVALID_ARG, "attention: unaligned pointer");
  if (dtype == LC_BF16) {
    AttnP p{};
    p.q = static_cast<const bf16_t *>(q);
    p.k = static_cast<const bf16_t *>(k);
    p.v = static_cast<const bf16_t *>(v);
    p.o = static_cast<bf16_t *>(o);
    p.lse = lse;
    p.ld_qkv = ld_qkv;
    p.ld_o = ld_o;
    p.S = S;
    p.H = H;
    p.scale = 1.0f / sqrtf((float)hd);
    const size_t lds = 2 * 2 * TILE;
    static bool once = false;
    if (!once) { LC_TRY(set_lds((const void *)attn_fwd_kernel, lds)); once = true; }
    hipLaunchKernelGGL(attn_fwd_kernel, dim3(S / QB, H, B), dim3(256), lds, s, p);
    return check_launch("attn_fwd_kernel");
  }
  AttnF p{};
  p.q = static_cast<const float *>(q);
  p.k = static_cast<const float *>(k);
  p.v = static_cast<const float *>(v);
  p.o = static_cast<float *>(o);
  p.lse = lse;
  p.ld_qkv = ld_qkv;
  p.ld_o = ld_o;
  p.B = B; p.S = S; p.H = H; p.hd = hd;
  p.scale = 1.0f / sqrtf((float)hd);
  const int64_t n = (int64_t)B * H * S;
  hipLaunchKernelGGL(attn_fwd_f32_kernel, dim3((unsigned)((n + 127) / 128)), dim3(128), 0, s, p);
  return check_launch("attn_fwd_f32_kernel");
}

lc_status attn_bwd_launch(int dtype, int B, int S, int H, int hd, const void *q, const void *k,
                          const void *v, int64_t ld_qkv, const void *o, const void *dout,
                          int64_t ld_o, const float *lse, void *dq, void *dk, void *dv,
                          int64_t ld_dqkv, const float *rcos, const float *rsin, void *scratch,
                          size_t scratch_bytes, hipStream_t s) {
  LC_TRY(check_common(dtype, B, S, H, hd, ld_qkv, ld_o));
  if (!q || !k || !v || !o || !dout || !lse || !dq || !dk || !dv)
    return fail(LC_ERR_INVALID_ARG, "attention backward: null pointer");
  if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(o) || !aligned16(dout) ||
      !aligned16(dq) || !aligned16(dk) || !aligned16(dv))
    return fail(LC_ERR_INVALID_ARG, "attention backward: unaligned pointer");
  if (ld_dqkv < (int64_t)H * hd) return fail(LC_ERR_INVALID_ARG, "attention: ld_dqkv too small");
  if ((rcos == nullptr) != (rsin == nullptr))
    return fail(LC_ERR_INVALID_ARG, "attention: give both RoPE tables or neither");
  if (!scratch || scratch_bytes < attn_scratch_size(B, S, H))
    return fail(LC_ERR_WORKSPACE, "attention backward: scratch too small");
  if (dtype == LC_BF16) {
    if (ld_dqkv % 8) return fail(LC_ERR_INVALID_ARG, "attention: ld_dqkv %% 8 != 0");
    if (rcos && !aligned16(rcos)) return fail(LC_ERR_INVALID_ARG, "attention: unaligned RoPE table");
    AttnP p{};
    p.q = static_cast<const bf16_t *>(q);
    p.k = static_cast<const bf16_t *>(k);
    p.v = static_cast<const bf16_t *>(v);
    p.o = const_cast<bf16_t *>(static_cast<const bf16_t *>(o));
    p.lse = const_cast<float *>(lse);
    p.dout = static_cast<const bf16_t *>(dout);
    p.dq = static_cast<bf16_t *>(dq);
    p.dk = static_cast<bf16_t *>(dk);
    p.dv = static_cast<bf16_t *>(dv);
    p.D = static_cast<const float *>(scratch);
    p.rcos = rcos;
    p.rsin = rsin;
    p.ld_qkv = ld_qkv;
    p.ld_o = ld_o;
    p.ld_d = ld_dqkv;
    p.S = S;
    p.H = H;
    p.scale = 1.0f / sqrtf((float)hd);
    hipLaunchKernelGGL(attn_bwd_prep_kernel, dim3((unsigned)((int64_t)B * S)), dim3(256), 0, s, p,
                       H * HD);
    LC_TRY(check_launch("attn_bwd_prep_kernel"));
    const size_t lds_dq = 2 * 3 * TILE, lds_kv = 2 * (4 * TILE + 512);
    static bool once = false;
    if (!once) {
      LC_TRY(set_lds((const void *)attn_bwd_dq_kernel, lds_dq));
      LC_TRY(set_lds((const void *)attn_bwd_dkdv_kernel, lds_kv));
      once = true;
    }
    hipLaunchKernelGGL(attn_bwd_dkdv_kernel, dim3(S / QB, H, B), dim3(256), lds_kv, s, p);
    LC_TRY(check_launch("attn_bwd_dkdv_kernel"));
    hipLaunchKernelGGL(attn_bwd_dq_kernel, dim3(S / QB, H, B), dim3(256), lds_dq, s, p);
    return check_launch("attn_bwd_dq_kernel");
  }
  AttnF p{};
  p.q = static_cast<const float *>(q);
  p.k = static_cast<const float *>(k);
  p.v = static_cast<const float *>(v);
  p.o = const_cast<float *>(static_cast<const float *>(o));
  p.lse = const_cast<float *>(lse);
  p.dout = static_cast<const float *>(dout);
  p.dq = static_cast<float *>(dq);
  p.dk = static_cast<float *>(dk);
  p.dv = static_cast<float *>(dv);
  p.D = static_cast<float *>(scratch);
  p.rcos = rcos;
  p.rsin = rsin;
  p.ld_qkv = ld_qkv;
  p.ld_o = ld_o;
  p.ld_d = ld_dqkv;
  p.B = B; p.S = S; p.H = H; p.hd = hd;
  p.scale = 1.0f / sqrtf((float)hd);
  const int64_t n = (int64_t)B * H * S;
  const dim3 grid((unsigned)((n + 127) / 128));
  hipLaunchKernelGGL(attn_bwd_q_f32_kernel, grid, dim3(128), 0, s, p);
  LC_TRY(check_launch("attn_bwd_q_f32_kernel"));
  hipLaunchKernelGGL(attn_bwd_kv_f32_kernel, grid, dim3(128), 0, s, p);
  return check_launch("attn_bwd_kv_f32_kernel");
}

}  // namespace lc

extern "C" {

lc_status lc_attention_forward(int32_t dtype, int32_t B, int32_t S, int32_t H, int32_t hd,
                               const void *q, const void *k, const void *v, int64_t ld_qkv,
                               void *o, int64_t ld_o, float *lse, void *stream) {
  return lc::attn_fwd_launch(dtype, B, S, H, hd, q, k, v, ld_qkv, o, ld_o, lse,
                             static_cast<hipStream_t>(stream));
}

lc_status lc_attention_backward(int32_t dtype, int32_t B, int32_t S, int32_t H, int32_t hd,
                                const void *q, const void *k, const void *v, int64_t ld_qkv,
                                const void *o, const void *dout, int64_t ld_o, const float *lse,
                                void *dq, void *dk, void *dv, int64_t ld_dqkv,
                                const float *rope_cos, const float *rope_sin, void *scratch,
                                size_t scratch_bytes, void *stream) {
  return lc::attn_bwd_launch(dtype, B, S, H, hd, q, k, v, ld_qkv, o, dout, ld_o, lse, dq, dk, dv,
                             ld_dqkv, rope_cos, rope_sin, scratch, scratch_bytes,
                             static_cast<hipStream_t>(stream));
}

}  // extern "C"
