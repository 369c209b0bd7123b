// bf16 GEMM on CDNA4 matrix cores (v_mfma_f32_32x32x16_bf16), fp32 accumulation,
// with the fused epilogues of a decoder layer's projections.
//
//   C(m, n) = sum_k A(m, k) B(n, k)
//   A(m, k) = A_K ? A[m*lda + k] : A[k*lda + m]      (A_K: k is contiguous)
//   B(n, k) = B_K ? B[n*ldb + k] : B[k*ldb + n]
//
// Tile: 256 x 256 per workgroup of 512 threads (8 waves, 4 along m x 2 along
// n); each wave owns 64 x 128 = 2 x 4 MFMA blocks of 32 x 32. K is walked in
// stages of 64: LDS holds two 64 KiB stages (A 256 x 64 | B 256 x 64); while
// the waves multiply stage s, stage s + 1 streams in from HBM/L2, and one
// barrier per stage both publishes the new stage and frees the old one.
// Waves 0-3 stream A, waves 4-7 stream B (8 loads of 1 KiB per wave per
// stage). A stage is multiplied in two halves of k = 32 (fragments of one
// half in registers at a time).
//
// Operand tiles go from HBM straight into LDS (buffer_load_dwordx4 ... lds:
// lane l of a wave's load fills bytes [16 l, 16 l + 16) of a 1 KiB LDS run),
// so no register staging is needed; the lanes of a load read global memory in
// address order, and padding between runs keeps fragment reads free of LDS
// bank conflicts. Buffer
// descriptors make out-of-range lanes (matrix edges, K tail) read zeros.
//   k-major operand: LDS rows of 64 k (128 B, one full cache line of the
//     operand row per 8-lane group, lanes in address order). Load run q
//     (0..31) holds tile rows q, q + 32, ..., q + 224, and runs sit 1040 bytes
//     apart, so tile row 32 p + q is at q * 1040 + 128 p. A fragment (32 rows
//     at one k chunk, 16 bytes per lane) is one ds_read_b128 of 32 runs at one
//     position, and the 16-byte run padding makes every 16 lanes touch all 64
//     banks once. (An earlier layout kept runs of 8 consecutive rows and
//     XOR-swizzled the 16-byte chunks of each cache line across the lanes of
//     a load, and the m/n-major one below XOR-swizzled 64-byte blocks: both
//     conflict-free too, but every product ran 3-6% slower with them. Rows of
//     32 k, i.e. half cache lines per load, cost a third of the throughput of
//     the global->LDS path.)
//   m/n-major operand (a weight read as dX = dY W, both operands of a weight
//     gradient dW = dY^T X): LDS rows of one k and 256 m (512 B, lanes in
//     address order); run q holds k rows q and q + 32, runs sit 1088 bytes
//     apart, so the four k rows one transposing read spans fall on different
//     banks. The fragment is read with the CDNA4
//     transposing load ds_read_b64_tr_b16: in each group of 16 lanes, lane j
//     receives element j % 4 of the 8 bytes addressed by lane 4e + j / 4 as its
//     element e, so lanes addressing four consecutive k rows at four 4-element
//     column runs receive one column's four k values each. Two such loads
//     give the 8 k values of the MFMA operand; no transposed copy exists in
//     HBM and no register shuffles are spent.
//
// The MFMA is issued with B's fragment in the instruction's first operand and
// A's in the second, which leaves lane l holding output row m = l % 32 and four
// runs of four consecutive columns n = 8g + 4(l / 32) + e: epilogues store 8 or
// 16 contiguous bytes per lane, and the column pairs (c, c + 64) that RoPE and
// SwiGLU combine sit in the same lane (blocks j and j + 2 of a 128-wide wave).
// Output, residual and gate/up element types are run-time values (uniform
// branches in the epilogue only), except in the instantiations for the decoder
// stage's own type mix (EpiTypes below), where they are compile-time constants.
#include "common.hpp"

#include <type_traits>

namespace lc {
namespace {

constexpr int BM = 256, BN = 256;
constexpr int KS = 64;             // k per stage
constexpr int NT = 512;            // threads per workgroup (8 waves)
constexpr int WM = 64, WN = 128;   // wave tile
constexpr int FM = WM / 32, FN = WN / 32;
// LDS-DMA runs: one 1 KiB load per wave instruction, with 16 bytes of padding
// after each run of a k-major operand and 64 after each run of an m/n-major one.
constexpr int RUN_K = 1024 + 16;
constexpr int RUN_MN = 1024 + 64;
constexpr int OPND_BYTES = 32 * RUN_MN;       // one operand's stage in LDS (32 runs)
constexpr int STAGE_BYTES = 2 * OPND_BYTES;   // A | B
constexpr uint32_t OOB = 0x80000000u;    // buffer offset beyond every operand: reads 0

typedef __attribute__((ext_vector_type(4))) short s16x4_v;
// LDS addresses stay 32-bit LDS-space pointers throughout (no generic pointers)
typedef __attribute__((address_space(3))) char lds_t;
typedef __attribute__((address_space(3))) bf16x8_v lds_v8;
typedef __attribute__((address_space(3))) s16x4_v lds_v4;
#define LDS_AS(T, ptr) ((__attribute__((address_space(3))) T *)(ptr))

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
  uint32_t a_bytes, b_bytes;  // byte extent of each operand (< 2^31)
  int M, N, K;  // N: output columns (SwiGLU: gate/up width)
  int tiles_m, tiles_n;
  int group;  // tile-rows per group of the tile walk
  int gmode, ngroups;
  const int32_t *goff;
  int64_t gstride_b, gstride_c;
  int rope_seq, rope_cols;
  int c_dt, r_dt, aux_dt;
};

typedef __attribute__((ext_vector_type(4))) int i32x4_v;

// Raw buffer descriptor (CDNA: dword3 = 0x00020000, stride 0): offsets past
// `bytes` read as zero.
__device__ __forceinline__ i32x4_v make_rsrc(const void *base, uint32_t bytes) {
  const uint64_t a = reinterpret_cast<uint64_t>(base);
  i32x4_v r;
  r[0] = __builtin_amdgcn_readfirstlane((int)(uint32_t)a);
  r[1] = __builtin_amdgcn_readfirstlane((int)((uint32_t)(a >> 32) & 0xFFFFu));
  r[2] = __builtin_amdgcn_readfirstlane((int)bytes);
  r[3] = 0x00020000;
  return r;
}

// 16 bytes per lane from the buffer at byte offset `off` into LDS at
// lds + 16 * lane. Issued as inline assembly: the compiler then does not track
// the load, so it inserts no wait for it before LDS reads of the other stage;
// the step's explicit wait before its barrier is what orders it.
__device__ __forceinline__ void dma16(i32x4_v rs, lds_t *lds, uint32_t off) {
  const uint32_t m0 = __builtin_amdgcn_readfirstlane((uint32_t) reinterpret_cast<uintptr_t>(lds));
  asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tbuffer_load_dwordx4 %0, %1, 0 offen lds"
               :
               : "v"(off), "s"(rs), "s"(m0)
               : "memory", "m0");
}

// The same with a wave-uniform part of the offset in the instruction's scalar
// offset. The hardware checks only the per-lane offset against the buffer's
// size, so callers use it where every lane's whole offset is inside the
// operand or the lane's own offset is OOB.
__device__ __forceinline__ void dma16s(i32x4_v rs, lds_t *lds, uint32_t voff, uint32_t soff) {
  const uint32_t m0 = __builtin_amdgcn_readfirstlane((uint32_t) reinterpret_cast<uintptr_t>(lds));
  asm volatile("s_mov_b32 m0, %3\n\ts_nop 0\n\tbuffer_load_dwordx4 %0, %1, %2 offen lds"
               :
               : "v"(voff), "s"(rs), "s"(__builtin_amdgcn_readfirstlane(soff)), "s"(m0)
               : "memory", "m0");
}

// One wave's share of an operand's loads: 8 of the 32 1-KiB LDS runs of a
// 256 x 64 stage (the four waves of a group load one operand).
//   k-major: run q = tile rows q + 32 p (p = 0..7); lane l -> position l/8,
//     global k chunk l%8.
//     ROWMAP 0: tile row r -> operand row base + r (valid below lim)
//     ROWMAP 1 (SwiGLU B rows): tile row r -> gate row ob + (r>>7)*64 + (r&63)
//       for (r&127) < 64, else up row lim + ob + (r>>7)*64 + (r&63); valid
//       while the output column ob + (r>>7)*64 + (r&63) < lim.
//   m/n-major: run q = k rows q and q + 32; lane l -> k row q + 32 (l/32),
//     global columns 8 (l%32) .. +7.
// Run t of wave w is q = 8w + t: consecutive runs are one row (k-major) or one
// k row (m/n-major) apart in the operand. The per-lane state is a row offset,
// an in-row offset, a validity mask and a k position; everything else is
// wave-uniform.
template <bool KMAJ, int ROWMAP>
struct Stream {
  uint32_t base;     // byte offset of run 0's row (k-major) or k row (m/n-major)
  uint32_t col[2];   // byte offset inside the row for even / odd runs
  uint32_t run;      // byte distance between consecutive runs
  uint32_t kb;       // bytes per unit of k
  uint32_t rows;     // bit t set when run t's row / columns are inside the operand
  int kl[2];         // k-major: first k of this lane's chunk; m/n-major: k row
                     // of run 0 (both entries equal)

  __device__ __forceinline__ void init(int64_t ld, int base_row, int lim, int wave, int lane) {
    if constexpr (KMAJ) {
      const int pos = lane >> 3;  // the lane's row position inside each run
      kl[0] = kl[1] = 8 * (lane & 7);
      int grow0, oc0;
      if constexpr (ROWMAP == 0) {
        grow0 = base_row + 8 * wave + 32 * pos;
        oc0 = grow0;
      } else {
        // tile row r = q + 32 pos: a gate row while (pos & 2) == 0, else an up
        // row, of output column base_row + (pos >> 2) 64 + 32 (pos & 1) + q
        oc0 = base_row + (pos >> 2) * 64 + 32 * (pos & 1) + 8 * wave;
        grow0 = (pos & 2) ? lim + oc0 : oc0;
      }
      rows = 0;
#pragma unroll
      for (int t = 0; t < 8; ++t) rows |= (oc0 + t < lim ? 1u : 0u) << t;
      base = rows ? (uint32_t)((int64_t)grow0 * ld * 2) : 0u;
      col[0] = col[1] = (uint32_t)(kl[0] * 2);
      run = (uint32_t)(ld * 2);
      kb = 2;
    } else {
      static_assert(ROWMAP == 0, "row remap needs a k-major operand");
      const int kr0 = 8 * wave + 32 * (lane >> 5);  // k row of run 0
      const int gm = base_row + 8 * (lane & 31);    // first of the lane's 8 columns
      kl[0] = kl[1] = kr0;
      rows = gm < lim ? 0xFFu : 0u;
      base = (uint32_t)((int64_t)kr0 * ld * 2);
      col[0] = col[1] = gm < lim ? (uint32_t)(gm * 2) : 0u;
      run = (uint32_t)(ld * 2);
      kb = (uint32_t)(ld * 2);
    }
  }

  // each run's per-lane byte offset at k = k0 (OOB for lanes outside the
  // operand's rows or columns); valid for stages that end at or before K
  __device__ __forceinline__ void offsets(uint32_t vo[8], int k0) const {
#pragma unroll
    for (int t = 0; t < 8; ++t)
      vo[t] = (rows >> t) & 1u ? base + t * run + col[t & 1] + (uint32_t)k0 * kb : OOB;
  }
  // run t of the wave's 8 runs of the stage starting at k0, into `lds` (the
  // operand's stage), every lane checked against K
  __device__ __forceinline__ void load1(i32x4_v rs, lds_t *lds, int wave, int k0, int K, int t) const {
    bool ok = (rows >> t) & 1u;
    if constexpr (KMAJ) ok = ok && k0 + kl[t & 1] < K;
    else ok = ok && k0 + kl[0] + t < K;
    const uint32_t off = ok ? base + t * run + col[t & 1] + (uint32_t)k0 * kb : OOB;
    dma16(rs, lds + (8 * wave + t) * (KMAJ ? RUN_K : RUN_MN), off);
  }
  __device__ __forceinline__ void load(i32x4_v rs, lds_t *lds, int wave, int k0, int K) const {
#pragma unroll
    for (int t = 0; t < 8; ++t) load1(rs, lds, wave, k0, K, t);
  }
};

// MFMA operand of 32 rows (row0 .. row0+31) at k = 16 s + 8 (lane / 32) + [0, 8)
// of the stage stored at t (s = 0 .. 3)
template <bool KMAJ>
__device__ __forceinline__ bf16x8_v frag(const lds_t *t, int row0, int s, int lane) {
  if constexpr (KMAJ) {
    // tile row row0 + i (row0 a multiple of 32) is position row0 / 32 of run i
    const int c = 2 * s + (lane >> 5);
    return *reinterpret_cast<const lds_v8 *>(t + (lane & 31) * RUN_K + (row0 >> 5) * 128 + c * 16);
  } else {
    // k row k is position k / 32 of run k % 32
    const int i16 = lane & 15, g = lane >> 4;
    const int m = row0 + 16 * (g & 1) + 4 * (i16 & 3);
    const int k = 16 * s + 8 * (g >> 1) + (i16 >> 2);
    const lds_t *p0 = t + (k & 31) * RUN_MN + (k >> 5) * 512 + m * 2;
    const s16x4_v lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4 *)(p0));
    const s16x4_v hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4 *)(p0 + 4 * RUN_MN));
    const s16x4_v v[2] = {lo, hi};
    return __builtin_bit_cast(bf16x8_v, v);
  }
}

// Scheduling pattern for one k-step: the NRD LDS reads of the next k-step
// spread over the NMF MFMAs of this one (reads first, as evenly as possible).
template <int NRD, int NMF, int I = 0>
__device__ __forceinline__ void interleave_steps() {
  if constexpr (I < NMF) {
    constexpr int r = NRD / NMF + (I < NRD % NMF ? 1 : 0);
    if constexpr (r > 0) __builtin_amdgcn_sched_group_barrier(0x100, r, 0);  // LDS reads
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);                       // one MFMA
    interleave_steps<NRD, NMF, I + 1>();
  }
}

// Element types of an epilogue's tensors: TM = 0 takes them from the run-time
// values in GemmP (uniform branches around every access); TM = 1 fixes them to
// the decoder stage's own mix for EPI (the branch-free accesses let the
// compiler keep the epilogue's loads in flight instead of waiting at each
// branch): residual add fp32 R and C, SwiGLU and its backward fp32 gate/up and
// bf16 C, RoPE fp16 C and bf16 copy. The host takes TM = 1 when the call's
// types are exactly that mix.
template <int EPI, int TM>
struct EpiTypes {
  static constexpr bool RES = EPI == LC_EPI_RESIDUAL, SWI = EPI == LC_EPI_SWIGLU || EPI == LC_EPI_SWIGLU_BWD;
  static constexpr bool ROPE = EPI == LC_EPI_ROPE;
  static constexpr int C = TM == 0 ? -1 : RES ? LC_FP32 : SWI ? LC_BF16 : ROPE ? LC_FP16 : -1;
  static constexpr int R = TM == 0 ? -1 : RES ? LC_FP32 : -1;
  static constexpr int X = TM == 0 ? -1 : SWI ? LC_FP32 : ROPE ? LC_BF16 : -1;
};

template <bool A_K, bool B_K, int EPI, int TM>
__global__ __launch_bounds__(NT) void gemm_bf16_kernel(GemmP p) {
  __shared__ __align__(16) char ring[2 * STAGE_BYTES];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform
  const int grp = wave >> 2, w4 = wave & 3;
  const int wm = w4, wn = grp;  // group g owns output columns [128 g, 128 g + 128)

  // Workgroups are dispatched round-robin over the 8 XCDs; give each XCD a
  // contiguous run of tiles, then walk tiles in groups of p.group tile-rows
  // (chosen by the host) so that neighbouring workgroups share A rows
  // and B columns in the XCD's L2.
  int wg = blockIdx.x;
  const int nwg = gridDim.x;
  if ((nwg & 7) == 0) wg = (wg & 7) * (nwg >> 3) + (wg >> 3);
  constexpr bool SWI = (EPI == LC_EPI_SWIGLU);
  int m0, tn, m_lim = p.M, kbeg = 0, kend = p.K;
  const bf16_t *Bp = p.B;
  void *Cp = p.C;
  if (p.gmode == LC_GROUP_ROWS) {
    // tile slot wg / tiles_n walks the groups' row tiles in order; slots past
    // the last group's tiles have nothing to do (the grid is an upper bound)
    tn = wg % p.tiles_n;
    int slot = wg / p.tiles_n, g = 0, lo = 0, hi = 0;
    for (; g < p.ngroups; ++g) {
      lo = min(max(p.goff[g], 0), p.M);
      hi = min(max(p.goff[g + 1], lo), p.M);
      const int nt = (hi - lo + BM - 1) / BM;
      if (slot < nt) break;
      slot -= nt;
    }
    if (g == p.ngroups) return;  // uniform across the workgroup, before any barrier
    m0 = lo + slot * BM;
    m_lim = hi;
    Bp = p.B + (int64_t)g * p.gstride_b;
  } else {
    int t = wg;
    if (p.gmode == LC_GROUP_K) {
      const int per = p.tiles_m * p.tiles_n, g = t / per;
      t -= g * per;
      kbeg = min(max(p.goff[g], 0), p.K);
      kend = min(max(p.goff[g + 1], kbeg), p.K);
      Cp = static_cast<char *>(p.C) + (int64_t)g * p.gstride_c * (p.c_dt == LC_FP32 ? 4 : 2);
    }
    const int per_group = p.group * p.tiles_n;
    const int first_m = (t / per_group) * p.group;
    const int gsz = min(p.tiles_m - first_m, p.group);
    m0 = (first_m + (t % per_group) % gsz) * BM;
    tn = (t % per_group) / gsz;
  }
  const int n0 = SWI ? tn * (BN / 2) : tn * BN;  // first output column

  f32x16_v acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

  lds_t *const R0 = LDS_AS(char, ring);
  const int ns = (kend - kbeg + KS - 1) / KS;  // stages
  // group 0 streams A, group 1 streams B
  const i32x4_v rs = grp == 0 ? make_rsrc(p.A, p.a_bytes) : make_rsrc(Bp, p.b_bytes);
  Stream<A_K, 0> sa_;
  Stream<B_K, SWI ? 1 : 0> sb_;
  if (grp == 0) sa_.init(p.lda, m0, m_lim, w4, lane);
  else sb_.init(p.ldb, n0, p.N, w4, lane);
  // Full stages use offsets computed once: run t's per-lane offset at kbeg,
  // plus the stage's k advance in the scalar offset (the same code for both
  // groups). A last stage that ends past K takes the per-lane K check.
  uint32_t vo[8];
  if (grp == 0) sa_.offsets(vo, kbeg);
  else sb_.offsets(vo, kbeg);
  const bool gk = grp == 0 ? A_K : B_K;
  const uint32_t kbw = gk ? 2u : (uint32_t)((grp == 0 ? p.lda : p.ldb) * 2);
  const int runb = gk ? RUN_K : RUN_MN;
  lds_t *const dst0 = R0 + grp * OPND_BYTES + 8 * w4 * runb;
  const bool ragged = (kend - kbeg) % KS != 0;
  auto load = [&](int st) {  // this group's operand of stage st
    if (ragged && st == ns - 1) {
      lds_t *stage = R0 + (st & 1) * STAGE_BYTES;
      if (grp == 0) sa_.load(rs, stage, w4, kbeg + st * KS, kend);
      else sb_.load(rs, stage + OPND_BYTES, w4, kbeg + st * KS, kend);
      return;
    }
    lds_t *d = dst0 + (st & 1) * STAGE_BYTES;
    const uint32_t so = (uint32_t)(st * KS) * kbw;
#pragma unroll
    for (int t = 0; t < 8; ++t) dma16s(rs, d + t * runb, vo[t], so);
  };

  typedef bf16x8_v FragA[FM];
  typedef bf16x8_v FragB[FN];
  // fragments of k-step q (k 16q .. 16q + 15) of stage st
  auto read_step = [&](int st, int q, FragA &af, FragB &bfr) {
    const lds_t *stage = R0 + (st & 1) * STAGE_BYTES;
#pragma unroll
    for (int i = 0; i < FM; ++i) af[i] = frag<A_K>(stage, wm * WM + i * 32, q, lane);
#pragma unroll
    for (int jj = 0; jj < FN; ++jj) bfr[jj] = frag<B_K>(stage + OPND_BYTES, wn * WN + jj * 32, q, lane);
  };
  auto multiply = [&](const FragA &af, const FragB &bfr) {
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int jj = 0; jj < FN; ++jj)
        acc[i][jj] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(bfr[jj], af[i], acc[i][jj], 0, 0, 0);
  };
  // LDS reads of one k-step: one per k-major fragment, two per m/n-major one
  constexpr int NRD = (A_K ? FM : 2 * FM) + (B_K ? FN : 2 * FN);
  constexpr int NMF = FM * FN;
  auto interleave = [&]() {
    interleave_steps<NRD, NMF>();
    __builtin_amdgcn_sched_barrier(0);
  };

  // Software pipeline over k-steps: the fragments of step q + 1 are read
  // while step q multiplies (two fragment sets in registers). Stage s + 1 goes
  // into the buffer of stage s - 1, whose last fragments every wave has read
  // before the barrier that published stage s. The barrier that publishes
  // stage s + 1 (after each wave's wait for its own loads and reads) sits
  // before the last k-step of stage s, so the first reads of stage s + 1
  // overlap that k-step's MFMAs.
  FragA fa[2];
  FragB fb[2];
  if (ns > 0) load(0);
  __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0)
  __syncthreads();
  if (ns > 0) read_step(0, 0, fa[0], fb[0]);
  for (int st = 0; st < ns; ++st) {
    if (st + 1 < ns) load(st + 1);
#pragma unroll
    for (int q = 0; q < 3; ++q) {
      read_step(st, q + 1, fa[(q + 1) & 1], fb[(q + 1) & 1]);
      multiply(fa[q & 1], fb[q & 1]);
      interleave();
    }
    __builtin_amdgcn_s_waitcnt(0x0070);  // vmcnt(0) lgkmcnt(0)
    __syncthreads();
    // (after the last stage this reads the other buffer's stale data, unused)
    read_step(st + 1, 0, fa[0], fb[0]);
    multiply(fa[1], fb[1]);
    interleave();
  }

  // ------------------------------------------------------------ epilogue
  // Each wave stages its 64 x 128 fp32 results through its own 16 KiB of the
  // (now idle) LDS ring, one 32-row block at a time: written in the MFMA
  // layout (lane = row, registers = columns), read back row-contiguous (16-byte
  // chunk c of row r at chunk c ^ (r & 15): both directions conflict-free), so
  // that every global access of the epilogue covers whole cache lines (two
  // rows of 128 columns, or four rows of two 64-column halves, per
  // instruction). Loads of a group of rows are issued before its stores.
  __syncthreads();  // every wave's last fragment reads are done
  const int frow = lane & 31, fhalf = lane >> 5;
  lds_t *const E = R0 + wave * 16384;
  typedef EpiTypes<EPI, TM> ET;
  const int c_dt = ET::C >= 0 ? ET::C : p.c_dt, r_dt = ET::R >= 0 ? ET::R : p.r_dt,
            aux_dt = ET::X >= 0 ? ET::X : p.aux_dt;
  typedef __attribute__((ext_vector_type(4))) float f32x4_t;
  typedef __attribute__((address_space(3))) f32x4_t lds_f4;
  const int ncol0 = n0 + wn * WN;  // first of the wave's 128 accumulator columns (non-SwiGLU)
  // 32-row block i of the wave's results into its LDS staging area
  auto stage_block = [&](int i) {
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int c = 8 * j + 2 * g + fhalf;
        const f32x4_t w = {acc[i][j][4 * g], acc[i][j][4 * g + 1], acc[i][j][4 * g + 2], acc[i][j][4 * g + 3]};
        *reinterpret_cast<lds_f4 *>(E + frow * 512 + ((c ^ (frow & 15)) << 4)) = w;
      }
  };
  auto chunk = [&](int r, int c) -> float4 {
    const f32x4_t v = *reinterpret_cast<const lds_f4 *>(E + r * 512 + ((c ^ (r & 15)) << 4));
    return make_float4(v[0], v[1], v[2], v[3]);
  };
  if constexpr (EPI == LC_EPI_ROPE || EPI == LC_EPI_SWIGLU) {
#pragma unroll
    for (int i = 0; i < FM; ++i) {
      const int mrow0 = m0 + wm * WM + i * 32;
      stage_block(i);
      {
        // lane: row 4 s + lane / 16, column quads q and q + 16 (columns 4q and 64 + 4q)
        const int q = lane & 15;
#pragma unroll
        for (int s0 = 0; s0 < 8; s0 += 4) {
          float4 x1[4], x2[4], cs[4], sn[4];
#pragma unroll
          for (int u = 0; u < 4; ++u) {
            const int rl = 4 * (s0 + u) + (lane >> 4);
            x1[u] = chunk(rl, q);
            x2[u] = chunk(rl, q + 16);
            if constexpr (EPI == LC_EPI_ROPE) {
              const int m = min(mrow0 + rl, m_lim - 1);
              const int pos = m % p.rope_seq;
              cs[u] = *reinterpret_cast<const float4 *>(p.rcos + (int64_t)pos * 64 + 4 * q);
              sn[u] = *reinterpret_cast<const float4 *>(p.rsin + (int64_t)pos * 64 + 4 * q);
            }
          }
#pragma unroll
          for (int u = 0; u < 4; ++u) {
            const int rl = 4 * (s0 + u) + (lane >> 4);
            const int m = mrow0 + rl;
            if (m >= m_lim) continue;
            float a[4] = {x1[u].x, x1[u].y, x1[u].z, x1[u].w};
            float b[4] = {x2[u].x, x2[u].y, x2[u].z, x2[u].w};
            if constexpr (EPI == LC_EPI_ROPE) {
              if (ncol0 >= p.N) continue;  // head past the output (uniform)
              if (ncol0 < p.rope_cols) {
                const float cv[4] = {cs[u].x, cs[u].y, cs[u].z, cs[u].w};
                const float sv[4] = {sn[u].x, sn[u].y, sn[u].z, sn[u].w};
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                  const float x = a[e], y = b[e];
                  a[e] = x * cv[e] - y * sv[e];
                  b[e] = x * sv[e] + y * cv[e];
                }
              }
              const int64_t row = (int64_t)m * p.ldc + ncol0 + 4 * q;
              store4_dt(Cp, row, c_dt, a[0], a[1], a[2], a[3]);
              store4_dt(Cp, row + 64, c_dt, b[0], b[1], b[2], b[3]);
              if (p.aux0) {  // a second copy in aux_dt
                const int64_t ra = (int64_t)m * p.ld_aux + ncol0 + 4 * q;
                store4_dt(p.aux0, ra, aux_dt, a[0], a[1], a[2], a[3]);
                store4_dt(p.aux0, ra + 64, aux_dt, b[0], b[1], b[2], b[3]);
              }
            } else {
              const int n = n0 + wn * 64 + 4 * q;  // output column of the gate/up pair
              if (n >= p.N) continue;
              float act[4];
#pragma unroll
              for (int e = 0; e < 4; ++e) act[e] = a[e] * sigmoidf_(a[e]) * b[e];
              const int64_t oa = (int64_t)m * p.ld_aux + n;
              store4_dt(p.aux0, oa, aux_dt, a[0], a[1], a[2], a[3]);
              store4_dt(p.aux1, oa, aux_dt, b[0], b[1], b[2], b[3]);
              store4_dt(Cp, (int64_t)m * p.ldc + n, c_dt, act[0], act[1], act[2], act[3]);
            }
          }
        }
      }
    }
  } else {
    // lane: row 2 s + lane / 32, column quad lane % 32. Pass t covers PU
    // values of s (2 PU rows) of 32-row block t / PPB. Epilogues that read a
    // tensor (residual, gradient bucket, gate/up) keep two passes of loads in
    // flight and issue pass t + 2's loads before pass t's stores: a wave's
    // loads and stores retire in issue order, so a wait for a load then never
    // waits for an earlier store.
    constexpr bool LD = EPI == LC_EPI_RESIDUAL || EPI == LC_EPI_ACCUM_F32 || EPI == LC_EPI_SWIGLU_BWD;
    constexpr int PU = 4, PPB = 16 / PU, NP = FM * PPB;
    const int q = lane & 31;
    const int n = ncol0 + 4 * q;
    const int ncl = n < p.N ? n : p.N - 4;  // loads of columns past N read valid data (unused)
    auto row_of = [&](int t, int u) { return 2 * ((t % PPB) * PU + u) + (lane >> 5); };
    float4 xa[2][PU], ya[2][PU];
    auto issue = [&](int t, float4 (&x)[PU], float4 (&y)[PU]) {
      const int mrow0 = m0 + wm * WM + (t / PPB) * 32;
#pragma unroll
      for (int u = 0; u < PU; ++u) {
        const int mc = min(mrow0 + row_of(t, u), m_lim - 1);
        if constexpr (EPI == LC_EPI_RESIDUAL) x[u] = load4_dt(p.R, (int64_t)mc * p.ldr + ncl, r_dt);
        if constexpr (EPI == LC_EPI_ACCUM_F32)
          x[u] = *reinterpret_cast<const float4 *>(static_cast<const float *>(Cp) + (int64_t)mc * p.ldc + ncl);
        if constexpr (EPI == LC_EPI_SWIGLU_BWD) {
          x[u] = load4_dt(p.aux0, (int64_t)mc * p.ld_aux + ncl, aux_dt);
          y[u] = load4_dt(p.aux1, (int64_t)mc * p.ld_aux + ncl, aux_dt);
        }
      }
    };
    stage_block(0);
    if constexpr (LD) {
      issue(0, xa[0], ya[0]);
      issue(1, xa[1], ya[1]);
    }
#pragma unroll
    for (int t = 0; t < NP; ++t) {
      if (t > 0 && t % PPB == 0) stage_block(t / PPB);  // after pass t - 1's LDS reads
      const int mrow0 = m0 + wm * WM + (t / PPB) * 32;
      float4 ra[PU], rb[PU];  // pass t's results (rb: SwiGLU backward's du)
#pragma unroll
      for (int u = 0; u < PU; ++u) {
        const float4 v = chunk(row_of(t, u), q);
        const float4 x = xa[t & 1][u], y = ya[t & 1][u];
        if constexpr (EPI == LC_EPI_SWIGLU_BWD) {
          const float o[4] = {v.x, v.y, v.z, v.w};
          const float gv[4] = {x.x, x.y, x.z, x.w};
          const float uv[4] = {y.x, y.y, y.z, y.w};
          float dg[4], du[4];
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const float sg = sigmoidf_(gv[e]);
            dg[e] = o[e] * uv[e] * sg * (1.0f + gv[e] * (1.0f - sg));
            du[e] = o[e] * gv[e] * sg;
          }
          ra[u] = make_float4(dg[0], dg[1], dg[2], dg[3]);
          rb[u] = make_float4(du[0], du[1], du[2], du[3]);
        } else if constexpr (LD) {
          ra[u] = make_float4(x.x + v.x, x.y + v.y, x.z + v.z, x.w + v.w);
        } else {
          ra[u] = v;
        }
      }
      if constexpr (LD) {
        if (t + 2 < NP) issue(t + 2, xa[t & 1], ya[t & 1]);
      }
#pragma unroll
      for (int u = 0; u < PU; ++u) {
        const int m = mrow0 + row_of(t, u);
        if (m >= m_lim || n >= p.N) continue;
        const int64_t oc = (int64_t)m * p.ldc + n;
        if constexpr (EPI == LC_EPI_ACCUM_F32) {
          *reinterpret_cast<float4 *>(static_cast<float *>(Cp) + oc) = ra[u];
        } else {
          store4_dt(Cp, oc, c_dt, ra[u].x, ra[u].y, ra[u].z, ra[u].w);
          if constexpr (EPI == LC_EPI_SWIGLU_BWD)
            store4_dt(Cp, oc + p.N, c_dt, rb[u].x, rb[u].y, rb[u].z, rb[u].w);
        }
      }
    }
  }
}

template <bool A_K, bool B_K, int EPI, int TM = 0>
lc_status launch_t(const GemmP &p, hipStream_t s) {
  // LC_GROUP_ROWS: an upper bound on the groups' row tiles (each group adds at
  // most one partial tile); LC_GROUP_K: every group has the full output grid
  unsigned grid = (unsigned)p.tiles_m * (unsigned)p.tiles_n;
  if (p.gmode == LC_GROUP_ROWS) grid = (unsigned)(p.tiles_m + p.ngroups) * (unsigned)p.tiles_n;
  if (p.gmode == LC_GROUP_K) grid *= (unsigned)p.ngroups;
  hipLaunchKernelGGL((gemm_bf16_kernel<A_K, B_K, EPI, TM>), dim3(grid), dim3(NT), 0, s, p);
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
  if (a.group_mode != LC_GROUP_NONE) {
    if (a.group_mode != LC_GROUP_ROWS && a.group_mode != LC_GROUP_K)
      return fail(LC_ERR_INVALID_ARG, "gemm: unknown group mode %d", a.group_mode);
    if (a.n_groups < 1 || a.n_groups > 64) return fail(LC_ERR_INVALID_ARG, "gemm: n_groups must be 1..64");
    if (!a.group_offsets || (reinterpret_cast<uintptr_t>(a.group_offsets) & 3))
      return fail(LC_ERR_INVALID_ARG, "gemm: group offsets must be a 4-byte aligned device array");
    if (a.epilogue == LC_EPI_ROPE || a.epilogue == LC_EPI_RESIDUAL)
      return fail(LC_ERR_UNSUPPORTED, "gemm: grouped products take STORE, ACCUM or SwiGLU epilogues");
    if (a.group_mode == LC_GROUP_ROWS && a.group_stride_b < 0)
      return fail(LC_ERR_INVALID_ARG, "gemm: negative group_stride_b");
    if (a.group_mode == LC_GROUP_K && (a.a_kmajor || a.b_kmajor || a.group_stride_c < 0))
      return fail(LC_ERR_UNSUPPORTED, "gemm: LC_GROUP_K needs m/n-major operands and group_stride_c >= 0");
  }
  if (a.epilogue == LC_EPI_ROPE && a.aux0) {
    if (!aligned16(a.aux0) || (bf && a.ld_aux % 8) || a.ld_aux < a.N || !valid_dtype(a.aux_dtype))
      return fail(LC_ERR_INVALID_ARG, "gemm: bad RoPE copy operand");
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
  if (a.dtype == LC_FP32 && a.group_mode != LC_GROUP_NONE)
    return fail(LC_ERR_UNSUPPORTED, "gemm fp32: grouped products need bf16 operands");
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
  // byte extents for the buffer descriptors (offsets are 32-bit)
  const int64_t brows = a.epilogue == LC_EPI_SWIGLU ? 2 * a.N : a.N;
  const int64_t a_ext = a.a_kmajor ? (a.M - 1) * a.lda + a.K : (a.K - 1) * a.lda + a.M;
  const int64_t b_ext = a.b_kmajor ? (brows - 1) * a.ldb + a.K : (a.K - 1) * a.ldb + brows;
  if (a_ext * 2 >= (int64_t)OOB || b_ext * 2 >= (int64_t)OOB)
    return fail(LC_ERR_UNSUPPORTED, "gemm bf16: an operand spans 2 GiB or more");
  p.a_bytes = (uint32_t)(a_ext * 2);
  p.b_bytes = (uint32_t)(b_ext * 2);
  p.tiles_m = (int)((a.M + BM - 1) / BM);
  p.tiles_n = a.epilogue == LC_EPI_SWIGLU ? (int)((a.N + BN / 2 - 1) / (BN / 2))
                                          : (int)((a.N + BN - 1) / BN);
  // 4 tile-rows per group, 3 when the grid has an odd number of tile-columns:
  // the fastest walk measured over the stage's shapes among groups of 2 to 8
  // and 16 (4 against 8: 1-2% faster on the 16-column dn2, dn1 and dW13
  // products, equal on the rest; 3 against 4 on the 43-column SwiGLU backward
  // and dW2 products: 1.5% and 3% faster)
  p.group = (p.tiles_n & 1) ? 3 : 4;
  p.gmode = a.group_mode;
  p.ngroups = a.group_mode == LC_GROUP_NONE ? 1 : a.n_groups;
  p.goff = a.group_offsets;
  p.gstride_b = a.group_stride_b;
  p.gstride_c = a.group_stride_c;
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
      if (ak && bk && p.c_dt == LC_FP32 && p.r_dt == LC_FP32)
        return launch_t<true, true, LC_EPI_RESIDUAL, 1>(p, s);
      if (ak && bk) return launch_t<true, true, LC_EPI_RESIDUAL>(p, s);
      break;
    case LC_EPI_ROPE:
      if (ak && bk && p.c_dt == LC_FP16 && (!p.aux0 || p.aux_dt == LC_BF16))
        return launch_t<true, true, LC_EPI_ROPE, 1>(p, s);
      if (ak && bk) return launch_t<true, true, LC_EPI_ROPE>(p, s);
      break;
    case LC_EPI_SWIGLU:
      if (ak && bk && p.c_dt == LC_BF16 && p.aux_dt == LC_FP32)
        return launch_t<true, true, LC_EPI_SWIGLU, 1>(p, s);
      if (ak && bk) return launch_t<true, true, LC_EPI_SWIGLU>(p, s);
      break;
    case LC_EPI_SWIGLU_BWD:
      if (ak && !bk && p.c_dt == LC_BF16 && p.aux_dt == LC_FP32)
        return launch_t<true, false, LC_EPI_SWIGLU_BWD, 1>(p, s);
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
