// Causal softmax attention on CDNA4 matrix cores (head_dim 128, fp16 or bf16
// q/k/v operands, fp32 softmax and accumulation), plus a plain fp32 path.
//
// Forward (written from the FlashAttention-2 algorithm of Dao, 2023): a
// workgroup of 8 waves owns 256 queries of one (batch row, head); each wave
// owns 32 queries and walks the visible keys in blocks of 64, keeping a
// running row maximum and row sum (online softmax) and the output in
// registers. K and V blocks stream from HBM straight into a two-stage LDS ring
// (buffer_load_dwordx4 ... lds, one 1 KiB run of 4 rows per wave
// instruction, each row's 256 bytes read in address order). The score block is computed transposed, S^T = K Q^T, so each
// lane holds one query's scores: the row max and row sum need lane-local work
// plus one swap with the partner lane (lane ^ 32). The output is accumulated
// transposed, O^T += V^T P^T, so the rescale is a lane-local scalar (done
// only when some query's score exceeds its reference maximum by more than
// 2^8), and the P^T accumulator registers feed the
// MFMA directly: the keys a lane holds define the k slots, and the V^T
// fragment is read in that key order with the transposing LDS load
// ds_read_b64_tr_b16 from V's key-major rows. Forward products use the q/k/v
// element type (P is rounded to it too).
//
// Backward (deterministic, no atomics): one kernel per 256 queries forms
// D = rowsum(dO*O) of its queries (written out for the next kernel) and
// accumulates dQ^T = K^T dS^T over the visible key blocks; then one kernel per
// 128 keys accumulates dV^T = dO^T P and dK^T = Q^T dS over the query blocks
// at or after the diagonal. Both recompute P from the forward's log-sum-exp
// with the forward's q/k element type (so P matches the forward) and take
// every gradient product in bf16; for fp16 inputs they read bf16 rows of q,
// k and v that the caller passes (the QKV projection's epilogue writes them)
// or that a copy pass writes first. The gradient products read
// their K^T, Q^T and dO^T operands from the same row tiles as the score
// products, with transposing LDS reads in the accumulator's key (or query)
// order, so no transposed copy is ever written. RoPE's inverse rotation of
// dq/dk is applied in the epilogues.
//
// Row tiles are [64 rows][128 columns] of 2-byte elements (256-byte rows of 16
// chunks) in 16 load runs 1040 bytes apart: run q holds rows f(q) + 16 p
// (p = 0..3) with f(r) = ((r & 3) << 2) | ((r >> 2) & 3), so row r sits at
// f(r % 16) * 1040 + (r / 16) * 256. A 128-bit fragment read (16 consecutive
// rows, one chunk) and a transposing read (4 consecutive rows, four chunks)
// both touch every bank once per phase, and every fragment address is a
// per-lane base plus an immediate offset (no per-read address arithmetic). An
// earlier layout XOR-swizzled the chunks of each row across the lanes of a
// load, which needed an XOR and an add per transposing read.
#include "common.hpp"

#include <math.h>

#include <type_traits>

namespace lc {
namespace {

constexpr int HD = 128;
constexpr int QB = 128;    // granularity of seq_len accepted by the matrix-core path
constexpr int ROWS = 256;  // queries (or keys) per workgroup: 8 waves x 32
constexpr int KB = 64;     // keys (or queries) per inner block
constexpr int NT = 512;
constexpr float LOG2E = 1.4426950408889634f;

// 2^x by the hardware instruction (v_exp_f32): no range reduction for results
// below the normal range, which only ever go into softmax weights that are
// rounded to 16 bits (where they are zero anyway); 2^-inf = 0.
__device__ __forceinline__ float ex2(float x) { return __builtin_amdgcn_exp2f(x); }
constexpr float LN2 = 0.6931471805599453f;
// one [64][128] tile of 2-byte elements: 16 load runs of 1 KiB, 16 bytes apart
constexpr int RUNB = 1024 + 16;
constexpr int TILE = 16 * RUNB;

typedef __attribute__((ext_vector_type(4))) int i32x4_v;
typedef __attribute__((ext_vector_type(4))) short s16x4_v;
typedef __attribute__((address_space(3))) char lds_t;
#define LDS_AS(T, ptr) ((__attribute__((address_space(3))) T *)(ptr))

template <typename E> struct V8;
template <> struct V8<__bf16> { typedef bf16x8_v type; };
template <> struct V8<_Float16> { typedef f16x8_v type; };

__device__ __forceinline__ f32x16_v mfma(bf16x8_v a, bf16x8_v b, f32x16_v c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ f32x16_v mfma(f16x8_v a, f16x8_v b, f32x16_v c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b, c, 0, 0, 0);
}

// ---------------------------------------------------------------- tiles
// load run of tile row r (an involution on 0..15: run q holds rows swz(q) + 16 p)
__device__ __forceinline__ int swz(int r) { return ((r & 3) << 2) | ((r >> 2) & 3); }
__device__ __forceinline__ int tile_off(int r, int c) { return swz(r & 15) * RUNB + (r >> 4) * 256 + c * 16; }

__device__ __forceinline__ i32x4_v make_rsrc(const void *base, uint32_t bytes) {
  const uint64_t a = reinterpret_cast<uint64_t>(base);
  i32x4_v r;
  r[0] = __builtin_amdgcn_readfirstlane((int)(uint32_t)a);
  r[1] = __builtin_amdgcn_readfirstlane((int)((uint32_t)(a >> 32) & 0xFFFFu));
  r[2] = __builtin_amdgcn_readfirstlane((int)bytes);
  r[3] = 0x00020000;
  return r;
}

// 16 bytes per lane from byte offset `off` of the buffer into LDS at
// lds + 16 * lane (inline assembly: the compiler does not track it; the
// block loop's explicit wait before its barrier orders it)
__device__ __forceinline__ void dma16(i32x4_v rs, lds_t *lds, uint32_t off) {
  const uint32_t m0 = __builtin_amdgcn_readfirstlane((uint32_t) reinterpret_cast<uintptr_t>(lds));
  asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tbuffer_load_dwordx4 %0, %1, 0 offen lds"
               :
               : "v"(off), "s"(rs), "s"(m0)
               : "memory", "m0");
}
// the same with a wave-uniform part of the offset in the instruction's scalar
// offset (every access in range: the callers' tiles lie inside their buffers)
__device__ __forceinline__ void dma16s(i32x4_v rs, lds_t *lds, uint32_t voff, uint32_t soff) {
  const uint32_t m0 = __builtin_amdgcn_readfirstlane((uint32_t) reinterpret_cast<uintptr_t>(lds));
  asm volatile("s_mov_b32 m0, %3\n\ts_nop 0\n\tbuffer_load_dwordx4 %0, %1, %2 offen lds"
               :
               : "v"(voff), "s"(rs), "s"(__builtin_amdgcn_readfirstlane(soff)), "s"(m0)
               : "memory", "m0");
}
// 4 bytes per lane into lds + 4 * lane
__device__ __forceinline__ void dma4(i32x4_v rs, lds_t *lds, uint32_t off) {
  const uint32_t m0 = __builtin_amdgcn_readfirstlane((uint32_t) reinterpret_cast<uintptr_t>(lds));
  asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tbuffer_load_dword %0, %1, 0 offen lds"
               :
               : "v"(off), "s"(rs), "s"(m0)
               : "memory", "m0");
}

// Run `run` (0..15) of a [64][128] tile: rows swz(run) + 16 p (p = 0..3) of a
// block of 64 rows, each 16-lane group reading one row's 256 bytes in address
// order. run_lane is the per-lane part of the byte offset (row 16 (lane / 16)
// after row0, chunk lane % 16 after col0, with `ld` elements per row);
// tile_run_s loads run `run` of block kb, the block's and the run's first row
// in the instruction's scalar offset (every access in range: the callers'
// tiles lie inside their buffers).
__device__ __forceinline__ uint32_t run_lane(int64_t row0, int64_t ld, int col0, int lane) {
  return (uint32_t)(((row0 + 16 * (lane >> 4)) * ld + col0 + 8 * (lane & 15)) * 2);
}
__device__ __forceinline__ void tile_run_s(i32x4_v rs, lds_t *tile, int run, int kb, uint32_t vo,
                                           uint32_t row_bytes) {
  dma16s(rs, tile + run * RUNB, vo, (uint32_t)(kb * KB + swz(run)) * row_bytes);
}

__device__ __forceinline__ void wait_vm0() { __builtin_amdgcn_s_waitcnt(0x0F70); }

// MFMA operand of 32 tile rows row0 .. row0+31 at columns 16 s + 8 (lane / 32) + [0, 8)
// (row0 a multiple of 32): rows_lane(lane) plus an immediate offset
__device__ __forceinline__ uint32_t rows_lane(int lane) {
  return (uint32_t)(swz(lane & 15) * RUNB + ((lane >> 4) & 1) * 256 + (lane >> 5) * 16);
}
template <typename VT>
__device__ __forceinline__ VT frag_rows(const lds_t *t, int row0, int s, int lane) {
  return *reinterpret_cast<const __attribute__((address_space(3))) VT *>(
      t + rows_lane(lane) + (row0 >> 4) * 256 + 32 * s);
}

// MFMA operand of 32 tile columns col0 .. col0+31 (lane l: column col0 + l % 32)
// whose 8 k values are tile rows c .. c+3 and c+8 .. c+11, c = kbase + 4 (lane / 32):
// the key (or query) order of a 32 x 32 accumulator's registers 8t .. 8t+7
// (rows 16t + 4 hf + [0, 4) and 16t + 8 + 4 hf + [0, 4)), kbase = 32 j + 16 t.
// Two transposing reads: rows c .. c+3 sit in runs swz(c % 16 ..), 64 bytes
// apart in the banks, and rows c+8 .. c+11 two runs further (swz(x + 8) =
// swz(x) + 2 for x < 8), so every address is cols_lane(lane) plus an immediate.
__device__ __forceinline__ uint32_t cols_lane(int lane) {
  const int i16 = lane & 15, hf = lane >> 5, b4 = (lane >> 4) & 1;
  return (uint32_t)(swz(4 * hf + (i16 >> 2)) * RUNB + (16 * b4 + 4 * (i16 & 3)) * 2);
}
template <typename VT>
__device__ __forceinline__ VT frag_cols_x(uint32_t a, int i, int kbase) {
  typedef __attribute__((address_space(3))) s16x4_v lds_v4;
  const uint32_t lo = a + 64u * i + 16u * kbase;
  const s16x4_v v[2] = {__builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4 *)(uintptr_t)lo),
                        __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4 *)(uintptr_t)(lo + 2 * RUNB))};
  return __builtin_bit_cast(VT, v);
}
// the same from a tile pointer (kbase a multiple of 16)
template <typename VT>
__device__ __forceinline__ VT frag_cols(const lds_t *t, int col0, int kbase, int lane) {
  return frag_cols_x<VT>((uint32_t)(uintptr_t)t + cols_lane(lane), col0 >> 5, kbase);
}

// max / sum of a lane's value and lane (l ^ 32)'s, in every lane
// (v_permlane32_swap: the upper half of one register trades places with the
// lower half of the other; with both registers holding x, the results hold the
// lower and the upper half of x in both halves)
__device__ __forceinline__ float max_with_partner(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float sum_with_partner(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
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

__device__ __forceinline__ f32x16_v zero16() {
  f32x16_v z;
#pragma unroll
  for (int r = 0; r < 16; ++r) z[r] = 0.0f;
  return z;
}

// 8 elements of type E (16 bytes) as 8 bf16
template <typename E>
__device__ __forceinline__ bf16x8_v to_bf16x8(uint4 v) {
  if constexpr (std::is_same<E, __bf16>::value) {
    return __builtin_bit_cast(bf16x8_v, v);
  } else {
    const f16x8_v h = __builtin_bit_cast(f16x8_v, v);
    bf16x8_v b;
#pragma unroll
    for (int e = 0; e < 8; ++e) b[e] = (__bf16)(float)h[e];
    return b;
  }
}

struct AttnP {
  const void *q, *k, *v;   // q/k/v element type (template)
  __bf16 *o;
  float *lse;
  const __bf16 *dout;
  __bf16 *dq, *dk, *dv;
  float *D;
  float *nl2;  // -lse log2(e) of every query, written by the dQ kernel for dK/dV
  // backward: bf16 rows of q, k and v for the gradient products (p.q, p.k,
  // p.v themselves for bf16 inputs; for fp16 inputs copies in the scratch,
  // written through the _w pointers)
  const __bf16 *qb, *kb, *vb;
  __bf16 *qb_w, *kb_w, *vb_w;
  // grouped-query attention: fp32 partial dk, dv per query head [B*S, H*128]
  float *dkp, *dvp;
  const float *rcos, *rsin;
  int64_t ld_qkv, ld_o, ld_d, ld_qb, ld_kb, ld_vb;
  uint32_t qkv_bytes, o_bytes, qb_bytes, kb_bytes, vb_bytes, lse_bytes;  // buffer extents (q/k/v from p.q)
  int S, H, B;
  int Hkv, G;   // key/value heads; query heads per key/value head
  float scale;  // 1/sqrt(hd)
};

// ---------------------------------------------------------------- forward
// Query block, head and batch row of this workgroup (forward and dQ grids):
// the blocks in decreasing order of work (a causal block's work grows with its
// index), the (batch row, head) pairs fastest. Workgroups are handed to the 8
// XCDs round-robin, so each XCD receives blocks of every size; with the block
// index fastest instead, one XCD would receive only the heaviest and the
// middle blocks of every head (twice the mean work).
__device__ __forceinline__ void query_block_of(const AttnP &p, int nqb, int &qb, int &h, int &b) {
  const int nbh = p.H * p.B, i = (int)blockIdx.x;
  qb = nqb - 1 - i / nbh;
  h = (i % nbh) % p.H;
  b = (i % nbh) / p.H;
}

template <typename QE>
__global__ __launch_bounds__(NT) void attn_fwd_kernel(AttnP p) {
  typedef typename V8<QE>::type QV;
  __shared__ __align__(16) char smem[2 * 2 * TILE];  // stage s: K tile | V tile
  lds_t *const L = LDS_AS(char, smem);
  const int nqb = (p.S + ROWS - 1) / ROWS;
  int qb, h, b;
  query_block_of(p, nqb, qb, h, b);
  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int l32 = lane & 31, hf = lane >> 5;
  const int64_t row0 = (int64_t)b * p.S;
  const int q0 = qb * ROWS + w * 32;
  const bool active = q0 < p.S;
  const int myq = q0 + l32;
  const float sc = p.scale * LOG2E;
  const QE *Q = static_cast<const QE *>(p.q) + h * HD;
  const int kvh = h / p.G;

  QV qf[8];
#pragma unroll
  for (int es = 0; es < 8; ++es) {
    if (active) qf[es] = *reinterpret_cast<const QV *>(Q + (row0 + myq) * p.ld_qkv + es * 16 + hf * 8);
    else qf[es] = QV{};
  }
  f32x16_v o[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) o[i] = zero16();
  float m = -INFINITY, l = 0.0f;

  // waves 0-3 stream K (runs 4 (w & 3) .. + 3), waves 4-7 stream V
  const bool isK = w < 4;
  const i32x4_v rs = make_rsrc(isK ? p.k : p.v, p.qkv_bytes);
  const uint32_t vo = run_lane(row0, p.ld_qkv, kvh * HD, lane), rowb = (uint32_t)(p.ld_qkv * 2);
  auto load = [&](int kb, lds_t *st) {
#pragma unroll
    for (int t = 0; t < 4; ++t) tile_run_s(rs, st + (isK ? 0 : TILE), 4 * (w & 3) + t, kb, vo, rowb);
  };
  const int nkb = min(p.S, (qb + 1) * ROWS) / KB;
  load(0, L);
  wait_vm0();
  __syncthreads();
  for (int kb = 0; kb < nkb; ++kb) {
    const lds_t *cur = L + (kb & 1) * 2 * TILE;
    if (kb + 1 < nkb) load(kb + 1, L + ((kb + 1) & 1) * 2 * TILE);
    const int k0 = kb * KB;
    if (active && k0 <= q0 + 31) {
      f32x16_v s[2] = {zero16(), zero16()};
      // K fragments are read one k-step ahead of the products that use them
      QV kf[2][2];
      kf[0][0] = frag_rows<QV>(cur, 0, 0, lane);
      kf[0][1] = frag_rows<QV>(cur, 32, 0, lane);
#pragma unroll
      for (int es = 0; es < 8; ++es) {
        if (es + 1 < 8) {
          kf[(es + 1) & 1][0] = frag_rows<QV>(cur, 0, es + 1, lane);
          kf[(es + 1) & 1][1] = frag_rows<QV>(cur, 32, es + 1, lane);
        }
        __builtin_amdgcn_sched_barrier(0);  // (keeps the reads ahead of the products)
        s[0] = mfma(kf[es & 1][0], qf[es], s[0]);
        s[1] = mfma(kf[es & 1][1], qf[es], s[1]);
        __builtin_amdgcn_sched_barrier(0);
      }
      if (k0 + KB - 1 > q0) {  // diagonal block (wave-uniform): mask keys after the query
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
          for (int r = 0; r < 16; ++r)
            if (k0 + j * 32 + out_row(r, hf) > myq) s[j][r] = -INFINITY;
      }
      float mx0 = -INFINITY, mx1 = -INFINITY;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        mx0 = fmaxf(mx0, s[0][r]);
        mx1 = fmaxf(mx1, s[1][r]);
      }
      const float mx = max_with_partner(fmaxf(mx0, mx1)) * sc;
      // The reference maximum m only moves when a score exceeds it by more
      // than 8 (base-2 exponent units): softmax weights stay <= 2^8, exact in
      // the fp16/bf16 P and far from fp32 overflow, and most blocks skip the
      // rescale of the output.
      if (__any(mx > m + 8.0f)) {
        const float mn = fmaxf(m, mx);
        const float alpha = mn > m ? ex2(m - mn) : 1.0f;
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
          for (int r = 0; r < 16; ++r) o[i][r] *= alpha;
        l *= alpha;
        m = mn;
      }
      float ls[4] = {0.0f, 0.0f, 0.0f, 0.0f};  // four independent chains
#pragma unroll
      for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const float pv = ex2(__builtin_fmaf(s[j][r], sc, -m));
          s[j][r] = pv;
          ls[2 * j + (r & 1)] += pv;
        }
      l += (ls[0] + ls[1]) + (ls[2] + ls[3]);
      // V^T fragments of step n = 2 j + t (keys 32 j + 16 t ..) read while
      // step n - 1 multiplies
      const uint32_t av = (uint32_t)(uintptr_t)(cur + TILE) + cols_lane(lane);
      QV vfr[2][4];
#pragma unroll
      for (int i = 0; i < 4; ++i) vfr[0][i] = frag_cols_x<QV>(av, i, 0);
#pragma unroll
      for (int n = 0; n < 4; ++n) {
        const int j = n >> 1, t = n & 1;
        if (n + 1 < 4) {
#pragma unroll
          for (int i = 0; i < 4; ++i)
            vfr[(n + 1) & 1][i] = frag_cols_x<QV>(av, i, 32 * ((n + 1) >> 1) + 16 * ((n + 1) & 1));
        }
        const QV pf = pack8<QE>(s[j], 8 * t);
        __builtin_amdgcn_sched_barrier(0);  // (keeps the reads ahead of the products)
#pragma unroll
        for (int i = 0; i < 4; ++i) o[i] = mfma(vfr[n & 1][i], pf, o[i]);
        __builtin_amdgcn_sched_barrier(0);
      }
    }
    wait_vm0();
    __syncthreads();
  }
  if (!active) return;
  const float lt = sum_with_partner(l);
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
// fp16 inputs: bf16 rows of q, k and v for the gradient products, one
// 16-byte chunk (8 elements) per thread, consecutive threads on consecutive
// chunks of the [B*S, H*128] (q) and [B*S, Hkv*128] (k, v) matrices.
__global__ __launch_bounds__(256) void attn_bwd_copy_kernel(AttnP p) {
  const int64_t rows = (int64_t)p.B * p.S;
  const int cq = p.H * HD / 8, ck = p.Hkv * HD / 8;  // chunks per row
  int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  int src = 0, cpr = cq;
  if (i >= rows * cq) {
    i -= rows * cq;
    src = 1 + (int)(i / (rows * ck));
    i -= (src - 1) * rows * ck;
    cpr = ck;
  }
  if (src > 2) return;
  const int64_t r = i / cpr, c = 8 * (i % cpr);
  const _Float16 *const x = static_cast<const _Float16 *>(src == 0 ? p.q : src == 1 ? p.k : p.v);
  __bf16 *const y = src == 0 ? p.qb_w : src == 1 ? p.kb_w : p.vb_w;
  const int64_t ldy = src == 0 ? p.ld_qb : src == 1 ? p.ld_kb : p.ld_vb;
  *reinterpret_cast<bf16x8_v *>(y + r * ldy + c) =
      to_bf16x8<_Float16>(*reinterpret_cast<const uint4 *>(x + r * p.ld_qkv + c));
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

// lane holds acc^T[e][token] for its own token; store that token's row (fp32)
__device__ __forceinline__ void store_row_f32(float *row, const f32x16_v (&acc)[4], int hf) {
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int g = 0; g < 4; ++g)
      *reinterpret_cast<float4 *>(row + i * 32 + 8 * g + 4 * hf) =
          make_float4(acc[i][4 * g], acc[i][4 * g + 1], acc[i][4 * g + 2], acc[i][4 * g + 3]);
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

// dQ: one workgroup per 256 queries; LDS stage = K (QE) | V (bf16), plus the
// bf16 rows of K for fp16 inputs. Each query's D = dO.O is formed here from
// the dO row the lane pair holds and written out for the dK/dV kernel.
template <typename QE>
__global__ __launch_bounds__(NT) void attn_bwd_dq_kernel(AttnP p) {
  typedef typename V8<QE>::type QV;
  constexpr bool SEP = !std::is_same<QE, __bf16>::value;  // separate bf16 K tile
  constexpr int NTQ = SEP ? 3 : 2;                          // tiles per stage
  __shared__ __align__(16) char smem[2 * NTQ * TILE];
  lds_t *const L = LDS_AS(char, smem);
  const int nqb = (p.S + ROWS - 1) / ROWS;
  int qb, h, b;
  query_block_of(p, nqb, qb, h, b);
  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int l32 = lane & 31, hf = lane >> 5;
  const int64_t row0 = (int64_t)b * p.S;
  const int q0 = qb * ROWS + w * 32;
  const bool active = q0 < p.S;
  const int myq = q0 + l32;
  const float sc = p.scale * LOG2E;
  const int kvh = h / p.G;

  QV qf[8];
  bf16x8_v df[8];
#pragma unroll
  for (int es = 0; es < 8; ++es) {
    if (active) {
      qf[es] = *reinterpret_cast<const QV *>(static_cast<const QE *>(p.q) + h * HD +
                                             (row0 + myq) * p.ld_qkv + es * 16 + hf * 8);
      df[es] = *reinterpret_cast<const bf16x8_v *>(p.dout + h * HD + (row0 + myq) * p.ld_o +
                                                   es * 16 + hf * 8);
    } else {
      qf[es] = QV{};
      df[es] = bf16x8_v{};
    }
  }
  const int64_t si = ((int64_t)b * p.H + h) * p.S + (active ? myq : 0);
  const float lse2 = p.lse[si] * LOG2E;
  f32x16_v acc[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) acc[i] = zero16();

  // 16 NTQ runs per block: K (QE) runs 0-15, V (bf16) 16-31, bf16 K 32-47;
  // 2 NTQ per wave
  const i32x4_v rk = make_rsrc(p.k, p.qkv_bytes);
  const i32x4_v rvb = make_rsrc(p.vb, p.vb_bytes);
  const i32x4_v rkb = make_rsrc(p.kb, p.kb_bytes);
  const uint32_t vok = run_lane(row0, p.ld_qkv, kvh * HD, lane), vov = run_lane(row0, p.ld_vb, kvh * HD, lane),
                 vokb = run_lane(row0, p.ld_kb, kvh * HD, lane);
  const uint32_t rbk = (uint32_t)(p.ld_qkv * 2), rbv = (uint32_t)(p.ld_vb * 2), rbkb = (uint32_t)(p.ld_kb * 2);
  auto load = [&](int kb, lds_t *st) {
#pragma unroll
    for (int t = 0; t < 2 * NTQ; ++t) {
      const int run = 2 * NTQ * w + t, which = run >> 4;  // (wave-uniform)
      if (which == 0) tile_run_s(rk, st, run & 15, kb, vok, rbk);
      else if (which == 1) tile_run_s(rvb, st + TILE, run & 15, kb, vov, rbv);
      else tile_run_s(rkb, st + 2 * TILE, run & 15, kb, vokb, rbkb);
    }
  };
  const int nkb = min(p.S, (qb + 1) * ROWS) / KB;
  load(0, L);
  // D of this query (its O row read while the first block streams in): the
  // lane's 64 products, then its partner's (lane ^ 32)
  float Dq = 0.0f;
  if (active) {
#pragma unroll
    for (int es = 0; es < 8; ++es) {
      const bf16x8_v o8 = *reinterpret_cast<const bf16x8_v *>(p.o + h * HD + (row0 + myq) * p.ld_o +
                                                              es * 16 + hf * 8);
#pragma unroll
      for (int e = 0; e < 8; ++e) Dq += (float)df[es][e] * (float)o8[e];
    }
  }
  Dq = sum_with_partner(Dq);
  if (active && hf == 0) {
    p.D[si] = Dq;
    p.nl2[si] = -lse2;
  }
  wait_vm0();
  __syncthreads();
  for (int kb = 0; kb < nkb; ++kb) {
    const lds_t *cur = L + (kb & 1) * NTQ * TILE;
    if (kb + 1 < nkb) load(kb + 1, L + ((kb + 1) & 1) * NTQ * TILE);
    const int k0 = kb * KB;
    if (active && k0 <= q0 + 31) {
      f32x16_v s[2] = {zero16(), zero16()}, dp[2] = {zero16(), zero16()};
      // K fragments are read one k-step ahead of their products, V fragments
      // two products ahead of theirs (registers allow no more)
      QV kf[2][2];
#pragma unroll
      for (int j = 0; j < 2; ++j) kf[0][j] = frag_rows<QV>(cur, j * 32, 0, lane);
#pragma unroll
      for (int es = 0; es < 8; ++es) {
        bf16x8_v vf[2];
#pragma unroll
        for (int j = 0; j < 2; ++j) vf[j] = frag_rows<bf16x8_v>(cur + TILE, j * 32, es, lane);
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int j = 0; j < 2; ++j) s[j] = mfma(kf[es & 1][j], qf[es], s[j]);
        if (es + 1 < 8) {
#pragma unroll
          for (int j = 0; j < 2; ++j) kf[(es + 1) & 1][j] = frag_rows<QV>(cur, j * 32, es + 1, lane);
        }
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int j = 0; j < 2; ++j) dp[j] = mfma(vf[j], df[es], dp[j]);
        __builtin_amdgcn_sched_barrier(0);
      }
      if (k0 + KB - 1 > q0) {  // diagonal block (wave-uniform): P = 0 for keys after the query
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
          for (int r = 0; r < 16; ++r)
            if (k0 + j * 32 + out_row(r, hf) > myq) s[j][r] = -INFINITY;
      }
#pragma unroll
      for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const float pv = ex2(__builtin_fmaf(s[j][r], sc, -lse2));
          dp[j][r] = pv * (dp[j][r] - Dq);
        }
      // K^T fragments: transposing reads of the bf16 K rows in dS's key order
      uint32_t cl = cols_lane(lane);
      asm volatile("" : "+v"(cl));  // recomputed each block, not held across the loop
      const uint32_t ak = (uint32_t)(uintptr_t)cur + cl + (SEP ? 2 * TILE : 0);
#pragma unroll
      for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int t = 0; t < 2; ++t) {
          const bf16x8_v sf = pack8<__bf16>(dp[j], 8 * t);
#pragma unroll
          for (int i = 0; i < 4; ++i)
            acc[i] = mfma(frag_cols_x<bf16x8_v>(ak, i, j * 32 + 16 * t), sf, acc[i]);
        }
    }
    wait_vm0();
    __syncthreads();
  }
  if (!active) return;
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[i][r] *= p.scale;
  if (p.rcos) rope_inverse_pairs(acc, p.rcos, p.rsin, myq, hf);
  store_row_t(p.dq + h * HD + (row0 + myq) * p.ld_d, acc, 1.0f, hf);
}

// dK, dV: one workgroup of 8 waves per 128 keys and query head. Waves w and
// w + 4 own the same 32 keys (their K and V fragments stay in registers) and
// take the first and the second 32 queries of every 64-query block at or
// after the diagonal; at the end wave w + 4 hands its partial dK, dV to wave w
// through LDS, which adds them (fixed order: deterministic). LDS stage (two
// of them) = Q (QE) | dO | (fp16 inputs: bf16 Q) | -lse log2(e) | D of one 64-query
// block. With
// grouped-query attention the workgroup writes its query head's share of the
// key/value head's dK, dV as fp32 rows; attn_gqa_sum_kernel adds the shares.
constexpr int KV_ROWS = 128;
template <typename QE>
__global__ __launch_bounds__(NT) void attn_bwd_dkdv_kernel(AttnP p) {
  typedef typename V8<QE>::type QV;
  constexpr bool SEP = !std::is_same<QE, __bf16>::value;  // separate bf16 Q tile
  constexpr int NTK = SEP ? 3 : 2;                          // row tiles per stage
  constexpr int RPW = SEP ? 8 : 4;                          // tile runs per wave
  constexpr int STAGE = NTK * TILE + 512;
  // two stages (256-byte aligned for frag_cols_x), reused at the end for the
  // partial dK, dV that waves 4-7 hand over (4 x 128 rows x 64 lanes fp32)
  constexpr int HANDOFF = 4 * 128 * 64 * 4;
  __shared__ __align__(256) char smem[2 * STAGE > HANDOFF ? 2 * STAGE : HANDOFF];
  lds_t *const L = LDS_AS(char, smem);
  const int kblk = (int)blockIdx.x / p.H, h = (int)blockIdx.x % p.H;  // earliest (heaviest) keys first
  const int kvh = h / p.G;
  const int b = blockIdx.y;
  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int pw = w & 3, hq = w >> 2;  // key block of the pair, query half
  const int l32 = lane & 31, hf = lane >> 5;
  const int64_t row0 = (int64_t)b * p.S;
  const int k0w = kblk * KV_ROWS + pw * 32;
  const int myk = k0w + l32;
  const float sc = p.scale * LOG2E;

  QV kf[8];
  bf16x8_v vf[8];
#pragma unroll
  for (int es = 0; es < 8; ++es) {
    const int64_t off = kvh * HD + (row0 + myk) * p.ld_qkv + es * 16 + hf * 8;
    kf[es] = *reinterpret_cast<const QV *>(static_cast<const QE *>(p.k) + off);
    vf[es] = to_bf16x8<QE>(*reinterpret_cast<const uint4 *>(static_cast<const QE *>(p.v) + off));
  }
  f32x16_v dk[4], dv[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) dk[i] = dv[i] = zero16();

  // 16 NTK runs per block: wave w brings runs RPW sub .. + RPW - 1 of tile tl
  // (Q (QE), dO, bf16 Q; with three tiles waves 6 and 7 bring none); the last
  // wave also brings -lse log2(e) and D (64 floats each)
  const int tl = SEP ? (w >> 1) : (w >> 2), sub = SEP ? (w & 1) : (w & 3);
  const bool brings = tl < NTK;  // wave-uniform
  const i32x4_v rs = tl == 0 ? make_rsrc(p.q, p.qkv_bytes)
                   : tl == 1 ? make_rsrc(p.dout, p.o_bytes)
                             : make_rsrc(p.qb, p.qb_bytes);
  const i32x4_v rl = make_rsrc(p.nl2, p.lse_bytes);  // -lse log2(e), from the dQ kernel
  const i32x4_v rd = make_rsrc(p.D, p.lse_bytes);
  const int64_t sbase = ((int64_t)b * p.H + h) * p.S;
  // Byte offset of run q of block qbi: the lane's row 16 (lane / 16) and
  // column chunk lane % 16 (one per-lane offset), plus the block's and the
  // run's first row swz(q) in the instruction's scalar offset
  const int64_t ld = tl == 0 ? p.ld_qkv : tl == 1 ? p.ld_o : p.ld_qb;
  const uint32_t vo = (uint32_t)(((row0 + 16 * (lane >> 4)) * ld + h * HD + 8 * (lane & 15)) * 2);
  const uint32_t urow = (uint32_t)(ld * 2), ublk = (uint32_t)(KB * ld * 2);
  auto load = [&](int qbi, lds_t *st) {
    lds_t *const tile = st + tl * TILE;
    if (brings) {
#pragma unroll
      for (int t = 0; t < RPW; ++t) {
        const int q = RPW * sub + t;
        dma16s(rs, tile + q * RUNB, vo, ublk * (uint32_t)qbi + urow * (uint32_t)swz(q));
      }
    }
    if (w == NT / 64 - 1) {
      const uint32_t off = (uint32_t)((sbase + (int64_t)qbi * KB + lane) * 4);
      dma4(rl, st + NTK * TILE, off);
      dma4(rd, st + NTK * TILE + 256, off);
    }
  };
  const int qfirst = kblk * KV_ROWS / KB, nqblk = p.S / KB;
  load(qfirst, L);
  wait_vm0();
  __syncthreads();
  for (int qbi = qfirst; qbi < nqblk; ++qbi) {
    const int cur_i = (qbi - qfirst) & 1;
    const lds_t *cur = L + cur_i * STAGE;
    if (qbi + 1 < nqblk) load(qbi + 1, L + (cur_i ^ 1) * STAGE);
    const float *sL = reinterpret_cast<const float *>(smem + cur_i * STAGE + NTK * TILE) + 32 * hq;
    const int q0 = qbi * KB + 32 * hq;  // this wave's 32 queries
    if (q0 + 31 >= k0w) {
      f32x16_v s = zero16(), dp = zero16();
      // fragment rows of this wave's 32 queries: a per-lane base, made opaque
      // each block (so that it is not held across the loop), plus immediates
      uint32_t rl_ = rows_lane(lane) + 2 * hq * 256;
      asm volatile("" : "+v"(rl_));
      const lds_t *qrow = cur + rl_;
      typedef __attribute__((address_space(3))) QV lds_q;
      typedef __attribute__((address_space(3))) bf16x8_v lds_b;
      // each fragment is read one product ahead of the product that uses it
      QV qa = *reinterpret_cast<const lds_q *>(qrow);
      bf16x8_v da = *reinterpret_cast<const lds_b *>(qrow + TILE);
#pragma unroll
      for (int es = 0; es < 8; ++es) {
        const int offn = 32 * (es + 1);
        QV qn{};
        bf16x8_v dn{};
        if (es + 1 < 8) qn = *reinterpret_cast<const lds_q *>(qrow + offn);
        __builtin_amdgcn_sched_barrier(0);
        s = mfma(qa, kf[es], s);
        if (es + 1 < 8) dn = *reinterpret_cast<const lds_b *>(qrow + TILE + offn);
        __builtin_amdgcn_sched_barrier(0);
        dp = mfma(da, vf[es], dp);
        __builtin_amdgcn_sched_barrier(0);
        qa = qn;
        da = dn;
      }
      if (q0 < k0w + 31) {  // diagonal block (wave-uniform): P = 0 for queries before the key
#pragma unroll
        for (int r = 0; r < 16; ++r)
          if (q0 + out_row(r, hf) < myk) s[r] = -INFINITY;
      }
      // four rows at a time: their -lse log2(e) and D are 4 consecutive floats each
      // (rows 8 g + 4 hf + [0, 4) of the half), read one group ahead
      typedef __attribute__((ext_vector_type(4))) float f4_t;
      const f4_t *const lseq = reinterpret_cast<const f4_t *>(sL + 4 * hf);
      f4_t lc = lseq[0], dc = lseq[16];
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        f4_t ln{}, dn{};
        if (g + 1 < 4) {
          ln = lseq[2 * (g + 1)];
          dn = lseq[16 + 2 * (g + 1)];
        }
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int r = 4 * g + e;  // out_row(r, hf) = 8 g + 4 hf + e
          const float pv = ex2(__builtin_fmaf(s[r], sc, lc[e]));
          s[r] = pv;
          dp[r] = pv * (dp[r] - dc[e]);
        }
        __builtin_amdgcn_sched_barrier(0);
        lc = ln;
        dc = dn;
      }
      // P and dS rounded to bf16 before the gradient products, so that the
      // fp32 score registers are free while those run
      const bf16x8_v pf[2] = {pack8<__bf16>(s, 0), pack8<__bf16>(s, 8)};
      const bf16x8_v sf[2] = {pack8<__bf16>(dp, 0), pack8<__bf16>(dp, 8)};
      __builtin_amdgcn_sched_barrier(0);
      // dO^T and Q^T fragments: transposing reads of the dO and bf16 Q rows
      // in P's query order (queries 32 hq + 16 t + 4 hf + [0, 4), + 8 + [0, 4))
      uint32_t cl = cols_lane(lane);
      asm volatile("" : "+v"(cl));  // recomputed each block, not held across the loop
      // (the wave's query half, rows 32 hq .., in the base: compile-time offsets)
      const uint32_t aq = (uint32_t)(uintptr_t)cur + cl + 512 * hq + (SEP ? 2 * TILE : 0),
                     ao = aq + (SEP ? -TILE : TILE);
      // steps n = 4 t + i; the dO^T and Q^T fragments of step n + 1 are read
      // while step n multiplies
      bf16x8_v fo[2], fq[2];
      fo[0] = frag_cols_x<bf16x8_v>(ao, 0, 0);
      fq[0] = frag_cols_x<bf16x8_v>(aq, 0, 0);
#pragma unroll
      for (int n = 0; n < 8; ++n) {
        const int t = n >> 2, i = n & 3;
        if (n + 1 < 8) {
          const int i1 = (n + 1) & 3, k1 = 16 * ((n + 1) >> 2);
          fo[(n + 1) & 1] = frag_cols_x<bf16x8_v>(ao, i1, k1);
          fq[(n + 1) & 1] = frag_cols_x<bf16x8_v>(aq, i1, k1);
        }
        __builtin_amdgcn_sched_barrier(0);
        dv[i] = mfma(fo[n & 1], pf[t], dv[i]);
        dk[i] = mfma(fq[n & 1], sf[t], dk[i]);
        __builtin_amdgcn_sched_barrier(0);
      }
    }
    wait_vm0();
    __syncthreads();
  }
  // waves 4-7 hand their partial sums to waves 0-3 (the stages are free now)
  typedef __attribute__((address_space(3))) float lds_f;
  lds_f *const red = reinterpret_cast<lds_f *>(L) + pw * (128 * 64) + lane;
  if (hq == 1) {
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        red[(i * 16 + r) * 64] = dk[i][r];
        red[(64 + i * 16 + r) * 64] = dv[i][r];
      }
  }
  __syncthreads();
  if (hq == 1) return;
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      dk[i][r] = (dk[i][r] + red[(i * 16 + r) * 64]) * p.scale;
      dv[i][r] += red[(64 + i * 16 + r) * 64];
    }
  if (p.rcos) rope_inverse_pairs(dk, p.rcos, p.rsin, myk, hf);
  if (p.G == 1) {
    store_row_t(p.dk + h * HD + (row0 + myk) * p.ld_d, dk, 1.0f, hf);
    store_row_t(p.dv + h * HD + (row0 + myk) * p.ld_d, dv, 1.0f, hf);
  } else {
    const int64_t prow = (row0 + myk) * (int64_t)p.H * HD + h * HD;
    store_row_f32(p.dkp + prow, dk, hf);
    store_row_f32(p.dvp + prow, dv, hf);
  }
}

// Grouped-query attention: dk, dv of key/value head kvh = the sum, in head
// order, of the fp32 shares of its G query heads (8 elements per thread)
__global__ __launch_bounds__(256) void attn_gqa_sum_kernel(AttnP p) {
  const int64_t n8 = (int64_t)p.B * p.S * p.Hkv * HD / 8;
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= n8) return;
  const int64_t e0 = 8 * i;
  const int64_t row = e0 / ((int64_t)p.Hkv * HD);
  const int c = (int)(e0 % ((int64_t)p.Hkv * HD));  // kvh * HD + e
  const int kvh = c / HD, e = c % HD;
#pragma unroll
  for (int which = 0; which < 2; ++which) {
    const float *src = (which == 0 ? p.dkp : p.dvp) + row * (int64_t)p.H * HD + (int64_t)kvh * p.G * HD + e;
    float acc[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) acc[u] = 0.0f;
    for (int g = 0; g < p.G; ++g) {
      const float4 a = *reinterpret_cast<const float4 *>(src + g * HD);
      const float4 b = *reinterpret_cast<const float4 *>(src + g * HD + 4);
      acc[0] += a.x; acc[1] += a.y; acc[2] += a.z; acc[3] += a.w;
      acc[4] += b.x; acc[5] += b.y; acc[6] += b.z; acc[7] += b.w;
    }
    bf16x8_v v;
#pragma unroll
    for (int u = 0; u < 8; ++u) v[u] = (__bf16)acc[u];
    __bf16 *dst = (which == 0 ? p.dk : p.dv) + row * p.ld_d + c;
    *reinterpret_cast<bf16x8_v *>(dst) = v;
  }
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
  int Hkv, G;  // key/value heads; query heads per key/value head
  float scale;
};

constexpr int MAXHD = 128;

__global__ void attn_fwd_f32_kernel(AttnF p) {
  const int64_t id = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
  if (id >= (int64_t)p.B * p.H * p.S) return;
  const int i = (int)(id % p.S), h = (int)((id / p.S) % p.H), b = (int)(id / ((int64_t)p.S * p.H));
  const int64_t r0 = (int64_t)b * p.S;
  const float *qi = p.q + (r0 + i) * p.ld_qkv + h * p.hd;
  const int kvh = h / p.G;
  float acc[MAXHD];
  for (int e = 0; e < p.hd; ++e) acc[e] = 0.0f;
  float m = -INFINITY, l = 0.0f;
  for (int j = 0; j <= i; ++j) {
    const float *kj = p.k + (r0 + j) * p.ld_qkv + kvh * p.hd;
    float s = 0.0f;
    for (int e = 0; e < p.hd; ++e) s += qi[e] * kj[e];
    s *= p.scale;
    const float mn = fmaxf(m, s);
    const float a = expf(m - mn), w = expf(s - mn);
    l = l * a + w;
    const float *vj = p.v + (r0 + j) * p.ld_qkv + kvh * p.hd;
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
  const int kvh = h / p.G;
  float acc[MAXHD];
  for (int e = 0; e < p.hd; ++e) acc[e] = 0.0f;
  for (int j = 0; j <= i; ++j) {
    const float *kj = p.k + (r0 + j) * p.ld_qkv + kvh * p.hd;
    const float *vj = p.v + (r0 + j) * p.ld_qkv + kvh * p.hd;
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

// per key and key/value head: dk_j and dv_j summed over the head's query
// heads in order (needs D from the kernel above)
__global__ void attn_bwd_kv_f32_kernel(AttnF p) {
  const int64_t id = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
  if (id >= (int64_t)p.B * p.Hkv * p.S) return;
  const int j = (int)(id % p.S), kvh = (int)((id / p.S) % p.Hkv);
  const int b = (int)(id / ((int64_t)p.S * p.Hkv));
  const int64_t r0 = (int64_t)b * p.S;
  const float *kj = p.k + (r0 + j) * p.ld_qkv + kvh * p.hd;
  const float *vj = p.v + (r0 + j) * p.ld_qkv + kvh * p.hd;
  float ak[MAXHD], av[MAXHD];
  for (int e = 0; e < p.hd; ++e) ak[e] = av[e] = 0.0f;
  for (int h = kvh * p.G; h < (kvh + 1) * p.G; ++h)
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
  float *dkj = p.dk + (r0 + j) * p.ld_d + kvh * p.hd;
  float *dvj = p.dv + (r0 + j) * p.ld_d + kvh * p.hd;
  for (int e = 0; e < p.hd; ++e) {
    dkj[e] = ak[e];
    dvj[e] = av[e];
  }
}

int kv_of(const lc_attn_args &a) { return a.Hkv > 0 ? a.Hkv : a.H; }
size_t attn_scratch_bytes_of(const lc_attn_args &a) {
  return attn_scratch_size(a.B, a.S, a.H, kv_of(a));
}

lc_status check_common(const lc_attn_args &a, bool bwd) {
  if (a.B <= 0 || a.S <= 0 || a.H <= 0 || a.hd <= 0)
    return fail(LC_ERR_INVALID_ARG, "attention: dimensions must be positive");
  if (a.Hkv < 0 || a.H % kv_of(a) != 0)
    return fail(LC_ERR_INVALID_ARG, "attention: Hkv (%d) must be 0 or divide H (%d)", a.Hkv, a.H);
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
    if (!a.scratch || a.scratch_bytes < attn_scratch_bytes_of(a))
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
  const int64_t rows = (int64_t)a.B * a.S, d = (int64_t)a.H * HD;
  const int Hkv = kv_of(a);
  const int64_t dkv = (int64_t)Hkv * HD;
  // scratch: D, then -lse log2(e) (fp32 [B, H, S] each; 256-byte aligned
  // together), then for fp16 inputs bf16 rows of v ([rows, dkv]), q ([rows, d])
  // and k ([rows, dkv]), then (grouped-query attention) the fp32 dk, dv shares
  if (p.D) p.nl2 = p.D + rows * a.H;
  const size_t dbytes = ((size_t)rows * a.H * 2 * sizeof(float) + 255) / 256 * 256;
  __bf16 *const cp = a.scratch ? reinterpret_cast<__bf16 *>(static_cast<char *>(a.scratch) + dbytes) : nullptr;
  const bool bf = a.dtype == LC_BF16;
  if (!bf && a.qkv_bf16) {  // the caller's bf16 copies: no copy pass
    const __bf16 *c = static_cast<const __bf16 *>(a.qkv_bf16);
    p.qb = c;
    p.kb = c + d;
    p.vb = c + d + dkv;
    p.ld_qb = p.ld_kb = p.ld_vb = a.ld_qkv_bf16;
  } else {
    p.vb_w = bf ? nullptr : cp;
    p.qb_w = bf || !cp ? nullptr : cp + rows * dkv;
    p.kb_w = bf || !cp ? nullptr : cp + rows * (dkv + d);
    p.vb = bf ? static_cast<const __bf16 *>(a.v) : p.vb_w;
    p.qb = bf ? static_cast<const __bf16 *>(a.q) : p.qb_w;
    p.kb = bf ? static_cast<const __bf16 *>(a.k) : p.kb_w;
    p.ld_vb = bf ? a.ld_qkv : dkv;
    p.ld_qb = bf ? a.ld_qkv : d;
    p.ld_kb = bf ? a.ld_qkv : dkv;
  }
  if (a.scratch && Hkv < a.H) {
    char *sh = static_cast<char *>(a.scratch) + attn_share_offset(a.B, a.S, a.H, Hkv);
    p.dkp = reinterpret_cast<float *>(sh);
    p.dvp = p.dkp + rows * d;
  }
  p.rcos = a.rope_cos;
  p.rsin = a.rope_sin;
  p.ld_qkv = a.ld_qkv;
  p.ld_o = a.ld_o;
  p.ld_d = a.ld_dqkv;
  p.qkv_bytes = (uint32_t)(((rows - 1) * a.ld_qkv + d) * 2);
  p.o_bytes = (uint32_t)(((rows - 1) * a.ld_o + d) * 2);
  p.vb_bytes = (uint32_t)(((rows - 1) * p.ld_vb + dkv) * 2);
  p.qb_bytes = (uint32_t)(((rows - 1) * p.ld_qb + d) * 2);
  p.kb_bytes = (uint32_t)(((rows - 1) * p.ld_kb + dkv) * 2);
  p.lse_bytes = (uint32_t)(rows * a.H * sizeof(float));
  p.S = a.S;
  p.H = a.H;
  p.B = a.B;
  p.Hkv = Hkv;
  p.G = a.H / Hkv;
  p.scale = 1.0f / sqrtf((float)a.hd);
  return p;
}

// buffer offsets are 32-bit: every matrix the kernels stream must span less than 2 GiB
lc_status check_extents(const lc_attn_args &a) {
  const int64_t rows = (int64_t)a.B * a.S, d = (int64_t)a.H * HD;
  const int64_t lim = (int64_t)1 << 31;
  if (((rows - 1) * a.ld_qkv + d) * 2 >= lim || ((rows - 1) * a.ld_o + d) * 2 >= lim ||
      rows * d * 2 >= lim)
    return fail(LC_ERR_UNSUPPORTED, "attention: a q/k/v/o matrix spans 2 GiB or more");
  if (a.qkv_bf16 && a.dtype == LC_FP16) {
    const int64_t cols = d + 2 * (int64_t)kv_of(a) * HD;
    if (!aligned16(a.qkv_bf16) || a.ld_qkv_bf16 < cols || a.ld_qkv_bf16 % 8)
      return fail(LC_ERR_INVALID_ARG, "attention: qkv_bf16 must be 16-byte aligned with ld_qkv_bf16 >= "
                  "(H + 2 Hkv) * 128, a multiple of 8");
    if (((rows - 1) * a.ld_qkv_bf16 + cols) * 2 >= lim)
      return fail(LC_ERR_UNSUPPORTED, "attention: the bf16 q/k/v copies span 2 GiB or more");
  }
  return LC_OK;
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
  p.Hkv = kv_of(a);
  p.G = a.H / p.Hkv;
  p.scale = 1.0f / sqrtf((float)a.hd);
  return p;
}

template <typename QE>
lc_status fwd_mc(const lc_attn_args &a, hipStream_t s) {
  LC_TRY(check_extents(a));
  const unsigned nqb = (unsigned)((a.S + ROWS - 1) / ROWS);
  hipLaunchKernelGGL(attn_fwd_kernel<QE>, dim3(nqb * (unsigned)(a.H * a.B)), dim3(NT), 0, s,
                     mc_params(a));
  return check_launch("attn_fwd_kernel");
}

template <typename QE>
lc_status bwd_mc(const lc_attn_args &a, hipStream_t s) {
  LC_TRY(check_extents(a));
  const AttnP p = mc_params(a);
  if (!std::is_same<QE, __bf16>::value && !a.qkv_bf16) {
    const int64_t chunks = (int64_t)a.B * a.S * (a.H + 2 * p.Hkv) * HD / 8;
    hipLaunchKernelGGL(attn_bwd_copy_kernel, dim3((unsigned)((chunks + 255) / 256)), dim3(256), 0, s, p);
    LC_TRY(check_launch("attn_bwd_copy_kernel"));
  }
  // dQ first: it writes D, which the dK/dV kernel reads
  const unsigned nb = (unsigned)((a.S + ROWS - 1) / ROWS);
  hipLaunchKernelGGL(attn_bwd_dq_kernel<QE>, dim3(nb * (unsigned)(a.H * a.B)), dim3(NT), 0, s, p);
  LC_TRY(check_launch("attn_bwd_dq_kernel"));
  hipLaunchKernelGGL(attn_bwd_dkdv_kernel<QE>, dim3((unsigned)(a.S / KV_ROWS * a.H), a.B), dim3(NT), 0,
                     s, p);
  LC_TRY(check_launch("attn_bwd_dkdv_kernel"));
  if (p.G > 1) {
    const int64_t n8 = (int64_t)a.B * a.S * p.Hkv * HD / 8;
    hipLaunchKernelGGL(attn_gqa_sum_kernel, dim3((unsigned)((n8 + 255) / 256)), dim3(256), 0, s, p);
    LC_TRY(check_launch("attn_gqa_sum_kernel"));
  }
  return LC_OK;
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
  const int64_t nkv = (int64_t)a.B * p.Hkv * a.S;
  hipLaunchKernelGGL(attn_bwd_kv_f32_kernel, dim3((unsigned)((nkv + 127) / 128)), dim3(128), 0, s, p);
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
