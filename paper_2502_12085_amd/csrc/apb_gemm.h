// Shared by apb_layer.hip and apb_scorer.hip (device code; each file that
// includes it instantiates its own kernels).
//
// The library's bf16 matrix products on gfx950, out[t][f] = sum_k x[t][k]
// W[f][k] (tokens t, output features f, weights row-major [f][k]): the
// layer's projections (apb_layer.hip) and the first layer of the retaining
// head (apb_scorer.hip).  One kernel template covers them: bf16 MFMA
// 16x16x32 with fp32 accumulation, output features on the MFMA M side (the
// weights are the A operand) and tokens on the N side, a 256 x 256
// workgroup tile of 4 waves (2 x 2, each 128 features x 128 tokens in 64
// 16 x 16 blocks, one wave per SIMD, accumulators in AGPRs), K steps of 64
// whose weight and token slabs are copied HBM -> LDS by
// global_load_lds_dwordx4 into XOR-swizzled tiles in two stages.  (16x16x32
// rather than 32x32x16: the same LDS bytes per flop and half the
// accumulator traffic, which this power-limited chip turns into clock.)
// Neither a copy nor an operand read spends a vector instruction on its
// address: a copy is a scalar base plus a fixed per-lane offset, a read one
// XOR of a per-lane base plus an instruction offset.  The step boundary is
// software-pipelined: at its last 32-deep substep a wave waits
// for its copies of the next step, passes the barrier, and issues that
// substep's MFMAs with the next step's first operand reads and the copies of
// the step after it (into the stage just finished) spread among them (for
// long K loops the copies start earlier, behind a second barrier that marks
// the stage free); the last two steps are peeled so the steady-state loop
// has no branches (the compiler can then count outstanding LDS reads
// exactly).
// The token operand is read row-major [t][k], head-major [k / dh][t][dh]
// (the attention output, whose heads are the O projection's K dimension), or
// from the head-major Q, K and V tensors as one [Q heads; K heads; V heads]
// feature row (the retaining head's input), so no transpose or
// concatenation is ever materialised.  Epilogues:
//  * row-major bf16 store, plus a residual in fp32 before the rounding;
//  * head-major Q/K/V store of the QKV projection (feature f is dim f % dh
//    of head f / dh: Q heads, then K heads, then V heads);
//  * SwiGLU: each wave's 128 weight rows are 64 gate rows and the 64 up
//    rows of the same features, so gate and up of one feature sit in the
//    same lane and register slot and SiLU(gate) * up is formed in registers;
//  * retaining head: bias, SiLU and the workgroup's share of the second
//    layer, one fp32 partial score per feature block, token and KV head.
#ifndef APB_GEMM_H_
#define APB_GEMM_H_

#include <math.h>

#include <type_traits>

#include "apb_internal.h"

namespace apb {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) bf16x8 lds_bf16x8;

constexpr int kBF = 256;        // weight rows (output features) per workgroup
constexpr int kBT = 256;        // tokens per workgroup
constexpr int kBK = 64;         // K per step
constexpr int kGemmThreads = 256;
constexpr int kPieces = 8;      // 1 KiB copy pieces per slab per wave per step
constexpr int kTileElems = kBF * kBK;  // = kBT * kBK

enum XMode { kXRowMajor = 0, kXHeadMajor = 1, kXQkv = 2 };
enum WMode { kWPlain = 0, kWGateUp = 1 };
enum Epi { kEpiRowMajor = 0, kEpiQkv = 1, kEpiSwiglu = 2, kEpiScorer = 3 };
constexpr int kScorerMaxKv = 8;  // scores per token the kEpiScorer epilogue forms

struct GemmParams {
  const uint16_t* x;      // tokens: [T][K], [K / dh][T][dh], or Q of kXQkv
  const uint16_t* w;      // [F][K]; the gate matrix for kWGateUp
  const uint16_t* w_up;   // [F][K] for kWGateUp
  const uint16_t* resid;  // [T][F] or null (kEpiRowMajor)
  uint16_t* out;          // [T][F] (kEpiRowMajor, kEpiSwiglu); Q for kEpiQkv
  uint16_t* out_k;        // kEpiQkv: K [n_kv][T][dh]
  uint16_t* out_v;        // kEpiQkv: V [n_kv][T][dh]
  int T, K, F;            // F: output features (I for kWGateUp)
  int dh;                 // head dim of a head-major operand or output
  int n_q, n_kv;          // kEpiQkv, kXQkv
  // kXQkv: the token operand is [Q heads; K heads; V heads] of the
  // head-major tensors x (Q, [n_q][x_rows][dh]), x_k and x_v ([n_kv][x_rows]
  // [dh]), at rows x_row0 + t
  const uint16_t* x_k;
  const uint16_t* x_v;
  int x_rows, x_row0;
  // kEpiScorer: bias, SiLU and the second layer of the retaining head
  const float* b1;        // [F]
  const float* w2;        // [n_kv][F]
  float* part;            // [F / kBF][n_kv][T] fp32 partial scores per feature block
  // tile grid (set by launch_gemm): token tiles, feature tiles, 8-tile blocks along tokens
  int ntx, nfy, nbt;
};

__device__ __forceinline__ uint32_t lds_offset(const void* p) {
  return (uint32_t)(uintptr_t)(__attribute__((address_space(3))) const void*)p;
}

// 16-byte chunk c of tile row r (128 bytes) sits at chunk c ^ ((r >> 1) & 7):
// any 16 consecutive rows, which one 16-lane pass of ds_read_b128 touches,
// land on 16 distinct 16-byte slots of the 256 bank bytes.
__device__ __forceinline__ int swz(int r) { return (r >> 1) & 7; }

// EARLY: the two-barrier step (long K loops), else one barrier per step.
template <int XM, int WM, int EPI, bool EARLY>
__global__ void __launch_bounds__(kGemmThreads, 1) gemm_kernel(GemmParams p) {
  // 256-byte aligned: operand addresses XOR step bits into the low byte of
  // a stage base plus lane offset
  __shared__ __attribute__((aligned(256))) uint16_t a_lds[2][kTileElems];  // weight slab
  __shared__ __attribute__((aligned(256))) uint16_t b_lds[2][kTileElems];  // token slab

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave & 1, wn = wave >> 1;  // feature half, token half
  // Blocked, XCD-aware tile order: workgroup b runs on XCD b % 8, and the 32
  // consecutive workgroups of one XCD take one block of 4 feature x 8 token
  // tiles, starting and finishing together, so per K step the XCD's L2
  // fetches 4 weight and 8 token slabs for 32 workgroups (with the tiles
  // dealt in grid order the same L2 fetched 1.2-3x the bytes).
  const int bid = blockIdx.x, xcd = bid & 7, slot = bid >> 3;
  const int blk = (slot >> 5) * 8 + xcd, sb = slot & 31;
  const int ftile = (blk / p.nbt) * 4 + (sb >> 3), ttile = (blk % p.nbt) * 8 + (sb & 7);
  if (ftile >= p.nfy || ttile >= p.ntx) return;  // past the grid's edge
  const int t0 = ttile * kBT;
  const int f0 = ftile * (WM == kWGateUp ? kBF / 2 : kBF);
  const int nk = p.K / kBK;

  // ---- copies: piece j (8 rows x 128 bytes) of each slab; wave w copies
  // pieces 8w .. 8w+7.  Lane l takes row l/8 of the piece and fetches the
  // chunk that belongs at slot l%8.  Rows past the last feature or token
  // repeat it (their results are never stored).  A copy is a scalar base (the
  // operand's first row for this workgroup, advanced by the K step in scalar
  // registers) plus a fixed per-lane byte offset: no vector instruction.
  const int cp_row = lane >> 3, cp_slot = lane & 7;
  const int x_ld = XM == kXRowMajor ? p.K : p.dh;  // elements between token rows
  // head-major operands: head dims are a power of two (64 or 128)
  const int dh_shift = XM == kXRowMajor ? 0 : 31 - __builtin_clz((unsigned)p.dh);
  uint32_t w_off[kPieces], x_off[kPieces];
#pragma unroll
  for (int i = 0; i < kPieces; ++i) {
    const int rho = 8 * (kPieces * wave + i) + cp_row;  // slab row 0..255
    const int chunk = 8 * (cp_slot ^ swz(rho));
    int fr = WM == kWGateUp ? f0 + 64 * (rho >> 7) + (rho & 63) : f0 + rho;
    fr = min(fr, p.F - 1);
    w_off[i] = 2u * (uint32_t)((fr - f0) * p.K + chunk);
    const int tr = min(t0 + rho, p.T - 1);
    x_off[i] = 2u * (uint32_t)((tr - t0) * x_ld + chunk);
  }
  const uint16_t* const w_first = p.w + (size_t)f0 * p.K;
  const uint16_t* const w_up_first = (WM == kWGateUp ? p.w_up : p.w) + (size_t)f0 * p.K;
  const uint16_t* const x_first = p.x + (size_t)t0 * x_ld;
  // copy q (0..15) of step kk into stage st: q < 8 weight pieces, else token pieces
  auto copy = [&](int kk, int st, int q) __attribute__((always_inline)) {
    const int k0 = kk * kBK;
    const int i = q & 7;
    const int j = kPieces * wave + i;
    if (q < 8) {
      // gate/up: rows 64..127 of either 128-row half are up-projection rows
      const uint16_t* base =
          (WM == kWGateUp && ((kPieces * wave + i) & 15) >= 8 ? w_up_first : w_first) + k0;
      const uint32_t d = __builtin_amdgcn_readfirstlane(lds_offset(&a_lds[st][j * 512]));
      asm volatile("s_mov_b32 m0, %2\n\tglobal_load_lds_dwordx4 %0, %1" ::"v"(w_off[i]), "s"(base),
                   "s"(d)
                   : "memory");
    } else {
      const uint16_t* base;
      if constexpr (XM == kXRowMajor) {
        base = x_first + k0;
      } else {
        // head-major tokens: K element k0 is column k0 % dh of head k0 / dh
        const int head = k0 >> dh_shift, j0 = k0 - (head << dh_shift);
        if constexpr (XM == kXQkv) {
          const uint16_t* src = head < p.n_q ? p.x : head < p.n_q + p.n_kv ? p.x_k : p.x_v;
          const int hh = head < p.n_q ? head
                         : head < p.n_q + p.n_kv ? head - p.n_q
                                                 : head - p.n_q - p.n_kv;
          base = src + ((size_t)hh * p.x_rows + p.x_row0 + t0) * p.dh + j0;
        } else {
          base = x_first + (size_t)head * p.T * p.dh + j0;
        }
      }
      const uint32_t d = __builtin_amdgcn_readfirstlane(lds_offset(&b_lds[st][j * 512]));
      asm volatile("s_mov_b32 m0, %2\n\tglobal_load_lds_dwordx4 %0, %1" ::"v"(x_off[i]), "s"(base),
                   "s"(d)
                   : "memory");
    }
  };

  // ---- operands (16x16x32 MFMAs): lane (li, lg) of a 16-row block reads
  // slab row 16*blk + li, K elements 32*kc + 8*lg .. +7, i.e. chunk
  // 4*kc + lg of that row, stored at slot (4*kc + lg) ^ swz(row).
  // swz(row) = (li >> 1) & 7 for every block, so the address is (lane base
  // ^ 64*kc) plus a constant for stage and block.  The 16 rows one 16-lane
  // pass of ds_read_b128 touches land on 16 distinct bank slots.
  const int li = lane & 15, lg = lane >> 4;
  const int sw = (li >> 1) & 7;
  const uint32_t lane_chunk = (uint32_t)(16 * (lg ^ sw));
  const uint32_t a_lane = (uint32_t)((128 * wm + li) * 128) + lane_chunk;
  const uint32_t b_lane = (uint32_t)((128 * wn + li) * 128) + lane_chunk;
  // stage st's row bases (the stages are 32 KiB apart, so the XOR with 64*kc
  // below touches only the chunk bits)
  auto a_base = [&](int st) __attribute__((always_inline)) { return lds_offset(a_lds[st]) + a_lane; };
  auto b_base = [&](int st) __attribute__((always_inline)) { return lds_offset(b_lds[st]) + b_lane; };
  auto read = [](uint32_t base, int blk, int kc) __attribute__((always_inline)) -> bf16x8 {
    return *(const lds_bf16x8*)(uintptr_t)((base ^ (64u * (uint32_t)kc)) + 2048u * (uint32_t)blk);
  };

  // acc[mb][nb]: 16 features x 16 tokens; lane (li, lg) holds features
  // 4*lg .. 4*lg+3 of token li
  f32x4 acc[8][8];
#pragma unroll
  for (int mb = 0; mb < 8; ++mb)
#pragma unroll
    for (int nb = 0; nb < 8; ++nb)
#pragma unroll
      for (int r = 0; r < 4; ++r) acc[mb][nb][r] = 0.f;
  bf16x8 av[2][8], bv[2][8];

  // prologue: step 0 copied and visible, step 1's copies in flight, step 0's
  // first operands read
#pragma unroll
  for (int q = 0; q < 16; ++q) copy(0, 0, q);
  asm volatile("s_waitcnt vmcnt(0)\n\ts_barrier" ::: "memory");
  if (nk > 1) {
#pragma unroll
    for (int q = 0; q < 16; ++q) copy(1, 1, q);
  }
#pragma unroll
  for (int mb = 0; mb < 8; ++mb) av[0][mb] = read(a_base(0), mb, 0);
#pragma unroll
  for (int nb = 0; nb < 8; ++nb) bv[0][nb] = read(b_base(0), nb, 0);

  // One K step in two substeps of 64 MFMAs; the odd MFMAs among the first 32
  // of a substep each carry one of the next substep's 16 operand reads.
  // NEXT: step kk+1 exists (at the last substep: wait for its copies,
  // barrier B, read its first operands); COPY: step kk+2 exists.  Its 16
  // copies go into the stage this step reads, each on its own MFMA four
  // apart (issued back to back they stall the wave, and the matrix core with
  // it, for hundreds of cycles).  That stage is free once every wave has read
  // the last substep's operands from it.  EARLY marks that point with barrier
  // A, at MFMA 48 of the first substep, and starts the copies there (4 in
  // the first substep, 12 in the second), giving them a quarter step more to
  // land: worth 5% on K loops of hundreds of steps, 1-2% slower on short
  // ones.  Otherwise the copies start after barrier B, on every fourth MFMA
  // of the second substep.
  auto step = [&](int kk, auto next_t, auto copy_t) __attribute__((always_inline)) {
    constexpr bool NEXT = decltype(next_t)::value, COPY = decltype(copy_t)::value;
    const int st = kk & 1;
    const uint32_t ab = a_base(st), bb = b_base(st), ab1 = a_base(st ^ 1), bb1 = b_base(st ^ 1);
#pragma unroll
    for (int kc = 0; kc < 2; ++kc) {
      const int cur = kc, nxt = kc ^ 1;
      const bool boundary = kc == 1;
      if (boundary && NEXT) {
        // barrier B: this wave's copies of step kk+1 have landed (only the
        // four copies of step kk+2 issued since barrier A may be
        // outstanding; copies complete in order); after the barrier every
        // wave's have
        if constexpr (EARLY && COPY) asm volatile("s_waitcnt vmcnt(4)\n\ts_barrier" ::: "memory");
        else if constexpr (EARLY) asm volatile("s_waitcnt vmcnt(0)\n\ts_barrier" ::: "memory");
        else asm volatile("s_waitcnt vmcnt(0)\n\ts_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
      }
#pragma unroll
      for (int i = 0; i < 64; ++i) {
        const int mb = i >> 3, nb = i & 7;
        if (EARLY && !boundary && COPY && i == 48) {
          // barrier A: every wave's reads of stage st are done
          asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
        }
        acc[mb][nb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av[cur][mb], bv[cur][nb],
                                                              acc[mb][nb], 0, 0, 0);
        if (i < 32 && (i & 1) == 1) {
          const int j = i >> 1;
          if (!boundary) {
            if (j < 8) av[nxt][j] = read(ab, j, 1);
            else bv[nxt][j - 8] = read(bb, j - 8, 1);
          } else if (NEXT) {
            if (j < 8) av[nxt][j] = read(ab1, j, 0);
            else bv[nxt][j - 8] = read(bb1, j - 8, 0);
          }
        }
        if (COPY && (i & 3) == 0) {
          if constexpr (EARLY) {
            if (!boundary && i >= 48) copy(kk + 2, st, (i - 48) >> 2);
            else if (boundary && i < 48) copy(kk + 2, st, 4 + (i >> 2));
          } else if (boundary) {
            copy(kk + 2, st, i >> 2);
          }
        }
        __builtin_amdgcn_sched_barrier(0);
      }
    }
  };
  const std::true_type yes{};
  const std::false_type no{};
  int kk = 0;
  for (; kk + 2 < nk; ++kk) step(kk, yes, yes);
  if (kk + 1 < nk) step(kk++, yes, no);
  step(kk, no, no);

  // ---- epilogue.  Lane (li, lg), block (mb, nb), element r holds slab row
  // 128*wm + 16*mb + 4*lg + r of token t0 + 128*wn + 16*nb + li: four
  // consecutive features (one 8-byte store).
  if constexpr (EPI == kEpiScorer) {
    // bias, SiLU and this workgroup's share of the second layer: for each of
    // its 256 tokens and each KV head, the sum over its 256 features of
    // SiLU(acc + b1) * w2, one fp32 partial per feature block
    __syncthreads();  // every wave is done with the LDS stages
    float* const w2_lds = reinterpret_cast<float*>(&a_lds[0][0]);  // [kBF][kScorerMaxKv]
    float* const b1_lds = w2_lds + kBF * kScorerMaxKv;              // [kBF]
    float* const red = reinterpret_cast<float*>(&b_lds[0][0]);     // [2][kScorerMaxKv][kBT]
    for (int i = tid; i < kBF * kScorerMaxKv; i += kGemmThreads) {
      const int u = i / kScorerMaxKv, kv = i % kScorerMaxKv;
      w2_lds[i] = kv < p.n_kv ? p.w2[(size_t)kv * p.F + f0 + u] : 0.f;
    }
    for (int i = tid; i < kBF; i += kGemmThreads) b1_lds[i] = p.b1[f0 + i];
    __syncthreads();
    float part[8][kScorerMaxKv];
#pragma unroll
    for (int nb = 0; nb < 8; ++nb)
#pragma unroll
      for (int kv = 0; kv < kScorerMaxKv; ++kv) part[nb][kv] = 0.f;
#pragma unroll
    for (int mb = 0; mb < 8; ++mb)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int u = 128 * wm + 16 * mb + 4 * lg + r;
        const f32x4 wa = *reinterpret_cast<const f32x4*>(&w2_lds[u * kScorerMaxKv]);
        const f32x4 wb = *reinterpret_cast<const f32x4*>(&w2_lds[u * kScorerMaxKv + 4]);
        const float bias = b1_lds[u];
#pragma unroll
        for (int nb = 0; nb < 8; ++nb) {
          // SiLU with the hardware reciprocal (within 1 ulp) instead of an
          // IEEE division, about ten instructions per element
          const float z = acc[mb][nb][r] + bias;
          const float a = z * __builtin_amdgcn_rcpf(1.f + __expf(-z));
#pragma unroll
          for (int kv = 0; kv < 4; ++kv) {
            part[nb][kv] = fmaf(a, wa[kv], part[nb][kv]);
            part[nb][4 + kv] = fmaf(a, wb[kv], part[nb][4 + kv]);
          }
        }
      }
    // the four lane groups hold the same tokens' other features
#pragma unroll
    for (int nb = 0; nb < 8; ++nb)
#pragma unroll
      for (int kv = 0; kv < kScorerMaxKv; ++kv) {
        float x = part[nb][kv];
        x += __shfl_xor(x, 16);
        part[nb][kv] = x + __shfl_xor(x, 32);
      }
    // the two feature halves (wm = 0, 1) of each token half meet in LDS
    if (lg == 0) {
#pragma unroll
      for (int nb = 0; nb < 8; ++nb)
#pragma unroll
        for (int kv = 0; kv < kScorerMaxKv; ++kv)
          red[(wm * kScorerMaxKv + kv) * kBT + 128 * wn + 16 * nb + li] = part[nb][kv];
    }
    __syncthreads();
    for (int i = tid; i < kScorerMaxKv * kBT; i += kGemmThreads) {
      const int kv = i / kBT, tl = i % kBT;
      const int t = t0 + tl;
      if (kv < p.n_kv && t < p.T)
        p.part[((size_t)ftile * p.n_kv + kv) * p.T + t] =
            red[kv * kBT + tl] + red[(kScorerMaxKv + kv) * kBT + tl];
    }
    return;
  }
#pragma unroll
  for (int nb = 0; nb < 8; ++nb) {
    const int t = t0 + 128 * wn + 16 * nb + li;
    if (t >= p.T) continue;
    if constexpr (EPI == kEpiSwiglu) {
#pragma unroll
      for (int mb = 0; mb < 4; ++mb) {
        const int f = f0 + 64 * wm + 16 * mb + 4 * lg;
        if (f >= p.F) continue;
        bf16x4 o;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const float gt = acc[mb][nb][i], up = acc[mb + 4][nb][i];
          o[i] = (__bf16)(gt * __builtin_amdgcn_rcpf(1.f + __expf(-gt)) * up);  // SiLU(gate) * up
        }
        *reinterpret_cast<bf16x4*>(p.out + (size_t)t * p.F + f) = o;
      }
    } else {
#pragma unroll
      for (int mb = 0; mb < 8; ++mb) {
        const int f = f0 + 128 * wm + 16 * mb + 4 * lg;
        if (f >= p.F) continue;
        float v[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) v[i] = acc[mb][nb][i];
        uint16_t* dst;
        if constexpr (EPI == kEpiQkv) {
          const int head = f / p.dh, j = f - head * p.dh;
          if (head < p.n_q)
            dst = p.out + ((size_t)head * p.T + t) * p.dh + j;
          else if (head < p.n_q + p.n_kv)
            dst = p.out_k + ((size_t)(head - p.n_q) * p.T + t) * p.dh + j;
          else
            dst = p.out_v + ((size_t)(head - p.n_q - p.n_kv) * p.T + t) * p.dh + j;
        } else {
          dst = p.out + (size_t)t * p.F + f;
          if (p.resid) {
            const bf16x4 rr = *reinterpret_cast<const bf16x4*>(p.resid + (size_t)t * p.F + f);
#pragma unroll
            for (int i = 0; i < 4; ++i) v[i] += (float)rr[i];
          }
        }
        bf16x4 o;
#pragma unroll
        for (int i = 0; i < 4; ++i) o[i] = (__bf16)v[i];
        *reinterpret_cast<bf16x4*>(dst) = o;
      }
    }
  }
}

template <int XM, int WM, int EPI>
hipError_t launch_gemm(GemmParams p, hipStream_t stream) {
  const int per_wg = WM == kWGateUp ? kBF / 2 : kBF;
  p.ntx = (p.T + kBT - 1) / kBT;
  p.nfy = (p.F + per_wg - 1) / per_wg;
  p.nbt = (p.ntx + 7) / 8;
  const int nblocks = ((p.nfy + 3) / 4) * p.nbt;  // blocks of 4 x 8 tiles
  const dim3 grid((unsigned)(256 * ((nblocks + 7) / 8)));
  if (p.K >= 8192)
    hipLaunchKernelGGL((gemm_kernel<XM, WM, EPI, true>), grid, dim3(kGemmThreads), 0, stream, p);
  else
    hipLaunchKernelGGL((gemm_kernel<XM, WM, EPI, false>), grid, dim3(kGemmThreads), 0, stream, p);
  return hipGetLastError();
}

}  // namespace
}  // namespace apb

#endif  // APB_GEMM_H_
