// Modified-mask attention of one APB host (Sec. 3.6, Eq. 2; Alg. 2,
// attention step) for gfx950 (CDNA4).
//
// Queries are the host's anchor and local rows [A; B]; keys and values are
// the concatenation [A; P; B], P being the earlier hosts' compressed blocks
// in host order.  Under the mask M' a query row r sees the concatenated keys
// 0 .. pos(r), pos(r) = r for anchor rows and r + Lp for local rows (causal
// attention over [A; P; B] without the passing block's query rows).  The
// concatenation is never materialised: key rows are fetched segment by
// segment from the anchor/local tensor and from the rank-major passing slots.
//
// Kernel design (one workgroup = 8 waves = 256 query rows of one query head,
// one workgroup per CU):
//  * Each wave owns 32 query rows (two 16-query blocks) and computes S^T =
//    K Q^T with v_mfma_f32_16x16x32_bf16 (keys on the M side, queries on the
//    N side); every K operand read feeds both query blocks.  The 16x16x32
//    shape accumulates 32 products per output per instruction (the 32x32x16
//    shape 16), so it moves half the fp32 accumulator data per flop; under
//    this chip's power limit a bf16 matrix load holds a higher clock with it
//    (measured: 1.87 vs 1.70 GHz on random operands).  In its accumulator
//    layout a lane holds 4 keys of each 16-key block for one query of each
//    block, so the softmax row statistics are lane-local up to an exchange
//    between four lanes (only on the rare max path and at the end), and the
//    probabilities are already laid out as the B operand of O^T = V^T P^T: no
//    LDS round trip for P.
//  * Ping-pong: the waves form two groups of four (one wave of each per
//    SIMD) that alternate between an MFMA phase (S of the next 128-key tile
//    and the PV product of the previous one, interleaved) and a softmax
//    phase, the phases separated by workgroup barriers.  On every SIMD one
//    wave feeds the matrix core while the other runs its exp/FMA work; a
//    single wave cannot overlap the two on gfx950.  A phase carries a fixed
//    cost (barrier, the first operand reads, the wait for the last MFMA
//    results), so the tiles are as long as registers and LDS allow.
//  * K and V tiles (128 keys) are copied HBM -> LDS by global_load_lds_dwordx4
//    (no register staging) into two-stage rings: group B copies K at the
//    start of its softmax phases, group A copies V early in its MFMA phases
//    (behind the phase's first operand reads), each with two phases to land.
//  * LDS tiles are row-major with an XOR swizzle of their 16-byte chunks: the
//    K operand reads (ds_read_b128) are free of bank conflicts, the
//    transposing V operand reads (ds_read_b64_tr_b16) two-way conflicted on
//    purpose (see the layout note below), and each read address is one XOR
//    of a per-lane base plus an immediate.
//  * Online softmax in fp32 registers in base 2 (scale*log2(e) folded into one
//    FMA), probabilities rounded to bf16 for the PV product, fp32 accumulate,
//    taken one 32-key block at a time (few live temporaries).  The running
//    max moves lazily: probabilities are formed against the current max and
//    the tile max is only computed when a tile's row sum exceeds 2^13, so
//    the max pass and the O rescale are off the common path.
//  * Tiles crossing a row's visible end are masked element-wise; tiles past
//    every row of the workgroup are not visited.
//  * Grid order puts the query tiles with the longest key prefix first, and
//    keeps a GQA group's workgroups on one XCD (one L2) when n_kv % 8 == 0.
#include <math.h>

#include "apb_internal.h"

namespace apb {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) i16x4 lds_i16x4;
typedef __attribute__((address_space(3))) bf16x8 lds_bf16x8;

constexpr int kGroupWaves = 4;                     // one wave per SIMD per group
constexpr int kWaves = 2 * kGroupWaves;     // ping-pong groups A and B
constexpr int kThreads = 64 * kWaves;
constexpr int kRowsPerWave = 32;
constexpr int kBM = kRowsPerWave * kWaves;  // query rows per workgroup
constexpr int kBN = 128;                           // keys per tile
constexpr int kKB = kBN / 16;                      // 16-key MFMA blocks per tile
constexpr int kNPC = kBN / 32;                     // 32-key chunks per tile (PV k-steps)
constexpr int kStages = 2;                         // LDS ring depth for K and V tiles
constexpr int kPD = 2;                             // LDS operand read-ahead (MFMA steps)
constexpr int kXcds = 8;                    // MI355X: 8 XCDs, workgroups dealt round-robin
constexpr float kSumLimit = 8192.f;         // lazy rescale: largest tile row-half sum against a stale max

struct Params {
  const uint16_t* q;
  const uint16_t* k;
  const uint16_t* v;
  const uint16_t* kp;
  const uint16_t* vp;
  uint16_t* o;
  float* lse;
  int La, Lb, lp, Lp, M, Ktot;
  int n_q, n_kv, group, n_qtiles;
  int xcd_map;  // 1: every XCD serves whole KV-head groups (n_kv % 8 == 0)
  float scale_log2;
};

__device__ __forceinline__ int vis_end(int r, int La, int Lp) {
  return (r < La ? r : r + Lp) + 1;
}

// Workgroup -> (query head, query tile).  Tiles with the longest key prefix
// go first.  With xcd_map, consecutive workgroup ids land on different XCDs,
// so the id is split into (xcd, slot) and XCD x serves KV heads x, x+8, ...:
// the query heads of one GQA group at neighbouring tiles share one L2.
__device__ __forceinline__ void map_block(const Params& p, int bid, int& head, int& qtile) {
  if (p.xcd_map) {
    const int xcd = bid % kXcds, slot = bid / kXcds;
    const int per_tile = p.group * (p.n_kv / kXcds);
    qtile = p.n_qtiles - 1 - slot / per_tile;
    const int rem = slot - (slot / per_tile) * per_tile;
    const int kv_local = rem / p.group;
    head = (xcd + kXcds * kv_local) * p.group + (rem - kv_local * p.group);
  } else {
    head = bid % p.n_q;
    qtile = p.n_qtiles - 1 - bid / p.n_q;
  }
}

// Address of concatenated key row c (0 <= c < Ktot) of KV head kvh, with
// per-lane selects instead of branches (the lanes of one copy may fall into
// different segments).
template <int D>
__device__ __forceinline__ const uint16_t* key_row_sel(const Params& p, const uint16_t* loc,
                                                       const uint16_t* pass, int kvh, int c) {
  const bool in_pass = c >= p.La && c < p.La + p.Lp;
  const int t = in_pass ? c - p.La : 0;
  const int s = t / p.lp;
  const int r = t - s * p.lp;
  const size_t pass_row = ((size_t)s * p.n_kv + kvh) * p.lp + r;
  const size_t loc_row = (size_t)kvh * p.M + (c < p.La ? c : c - p.Lp);
  return in_pass ? pass + pass_row * D : loc + loc_row * D;
}

// LDS tile layouts: row-major [kBN][D] bf16, 16-byte chunk c of row r stored
// at chunk position c ^ swz(r).  The LDS has 64 four-byte banks; a
// ds_read_b128 serves 16 lanes per clock, a ds_read_b64_tr_b16 32 lanes.
//  K: swz = r mod (D/8): the 16 rows one ds_read_b128 clock touches hit 16
//     different chunk positions (no bank conflicts).
//  V: swz = 4 * (r mod 4) (D = 128): the 16 lanes of one row group of a
//     transposing read touch 4 rows x 32 bytes on 4 different bank groups;
//     the 32 lanes of one clock cover rows r and r + 4 on the same banks, a
//     two-way conflict.  It is kept on purpose: a swizzle free of conflicts
//     (2 * (r mod 8)) gave bit-identical results but a 1.5-1.8% longer
//     launch, the softmax waves losing issue slots to an MFMA wave that no
//     longer stalls on its V reads.
template <int D>
__device__ __forceinline__ int k_swz(int r) { return r & (D / 8 - 1); }
template <int D>
__device__ __forceinline__ int v_swz(int r) { return (4 * (r & 3)) & (D / 8 - 1); }

// A wave-uniform 64-bit value in scalar registers (the copies take their
// base address and M0 from SGPRs).
__device__ __forceinline__ uint64_t uniform64(uint64_t x) {
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)x);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(x >> 32));
  return ((uint64_t)hi << 32) | lo;
}

// Byte offset of an LDS location, as M0 and LDS instructions address it.
__device__ __forceinline__ uint32_t lds_offset(const uint16_t* p) {
  return (uint32_t)(uintptr_t)(__attribute__((address_space(3))) const uint16_t*)p;
}

// Wait for this wave's outstanding LDS reads, then the workgroup barrier.
// Outstanding HBM -> LDS copies are not waited for here: each copying wave
// waits for its own copies (vmcnt) before the barrier that precedes their
// first reader.
__device__ __forceinline__ void phase_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

template <int D>
__global__ void __launch_bounds__(kThreads, 1)
attn_fwd_kernel(Params p) {
  constexpr int PIECE_ELEMS = 512;               // one 1 KiB DMA piece, in bf16
  constexpr int ROWS_PER_PIECE = PIECE_ELEMS / D;
  constexpr int PIECES = kBN * D / PIECE_ELEMS;  // pieces per tile per tensor
  constexpr int WP = PIECES / kGroupWaves;       // pieces per wave per tile
  constexpr int KCH = D / 8;                     // 16-byte chunks per key row
  constexpr int NKD = D / 32;                    // MFMA k-steps over head_dim (QK)
  constexpr int NDB = D / 16;                    // 16-wide blocks of head_dim in O^T
  constexpr int NPC = kNPC;                      // 32-key chunks of P (PV k-steps)
  constexpr int NQK = kKB * NKD;                 // QK operand reads per tile (two MFMAs each)
  constexpr int NPV = NPC * NDB;                 // PV operand reads per tile (two MFMAs each)
  constexpr int PD = kPD;
  static_assert(PIECES * PIECE_ELEMS == kBN * D && WP * kGroupWaves == PIECES, "tile split");
  static_assert(WP == 4 || WP == 8, "copy groups of four pieces");
  static_assert(NQK == NPV, "QK and PV step counts match for d in {64, 128}");

  // 256-byte aligned: operand addresses XOR step bits into the low byte of
  // a stage base plus lane offset
  __shared__ __attribute__((aligned(256))) uint16_t k_lds[kStages][kBN * D];
  __shared__ __attribute__((aligned(256))) uint16_t v_lds[kStages][kBN * D];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  // Wave index in a scalar register: every per-wave quantity below (group,
  // row range, tile counts) is uniform and its branches are scalar branches.
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int grp = wave / kGroupWaves;  // 0: group A, 1: group B
  const int wig = wave % kGroupWaves;  // wave in group

  int head, qtile;
  map_block(p, blockIdx.x, head, qtile);
  const int kvh = head / p.group;
  const int r0 = qtile * kBM;
  const int r_last = min(r0 + kBM, p.M) - 1;
  const int ntiles = (vis_end(r_last, p.La, p.Lp) + kBN - 1) / kBN;

  // Schedule, in phases separated by workgroup barriers.  Group A runs the
  // MFMA step of tile t, {S(t) = K(t) Q^T, O += P(t-1) V(t-1)}, in phase 2t
  // and the softmax of S(t) in phase 2t+1; group B runs the same one phase
  // later, so on every SIMD one wave issues MFMAs while the other runs its
  // exp/FMA work.  K(t) is read in phases 2t and 2t+1, V(t) in 2t+2 and
  // 2t+3.  Copies, into ring stage T % 2:
  //  - group B copies K(T) at the start of phase 2T-2 (its softmax phase; the
  //    stage's previous tile K(T-2) was last read in phase 2T-3) and waits
  //    for it at the end of phase 2T-1 (its MFMA phase);
  //  - group A copies V(T) at the start of phase 2T (its MFMA phase; V(T-2)
  //    was last read in phase 2T-1) and waits for it at the end of phase
  //    2T+1 (its softmax phase).
  // The barrier after each wait makes the tile visible to the phase that
  // first reads it.

  // Copy lanes: global_load_lds_dwordx4 puts lane l's 16 bytes at M0 +
  // inst_offset + 16*l and reads them from saddr + voffset + inst_offset, so
  // one M0 serves four of the wave's pieces (1 KiB apart in LDS and, inside
  // one segment, in HBM) and every lane fetches the chunk that belongs at its
  // swizzled slot.  The copies are inline asm so the compiler does not order
  // the LDS operand reads behind them.
  const bool copies_v = grp == 0;
  const uint16_t* cp_loc = copies_v ? p.v : p.k;
  const uint16_t* cp_pass = copies_v ? p.vp : p.kp;
  uint32_t cp_off[WP];  // per-lane byte offset of piece j, less (j % 4) KiB
#pragma unroll
  for (int j = 0; j < WP; ++j) {
    const int row = (wig * WP + j) * ROWS_PER_PIECE + lane / KCH;
    const int slot = lane % KCH;
    const int swz = copies_v ? v_swz<D>(row) : k_swz<D>(row);
    cp_off[j] = 2u * (uint32_t)(row * D + 8 * (slot ^ swz)) - 1024u * (j % 4);
  }
  // Segment cursor: concatenated key rows c in [.., seg_end) sit at byte
  // address seg_base + 2*D*c.  Tiles are copied in increasing order, so the
  // cursor moves only when a tile starts at or past seg_end.
  uint64_t seg_base = 0;
  int seg_end = 0;
  auto seek = [&](int c0) __attribute__((always_inline)) {
    if (c0 < p.La) {
      seg_end = p.La;
      seg_base = (uint64_t)cp_loc + (uint64_t)(2 * D) * ((uint64_t)kvh * p.M);
    } else if (c0 < p.La + p.Lp) {
      const int sl = (c0 - p.La) / p.lp;
      seg_end = p.La + (sl + 1) * p.lp;
      seg_base = (uint64_t)cp_pass +
                 (uint64_t)(2 * D) * (uint64_t)((int64_t)(sl * p.n_kv + kvh) * p.lp -
                                                (p.La + (int64_t)sl * p.lp));
    } else {
      seg_end = p.Ktot;
      seg_base = (uint64_t)cp_loc + (uint64_t)(2 * D) * (uint64_t)((int64_t)kvh * p.M - p.Lp);
    }
  };
  auto issue = [&](int T) __attribute__((always_inline)) {
    const int c0 = T * kBN;
    if (c0 >= seg_end) seek(c0);
    uint16_t* stage = copies_v ? v_lds[T % kStages] : k_lds[T % kStages];
    if (c0 + kBN <= seg_end) {
#pragma unroll
      for (int g = 0; g < WP / 4; ++g) {
        const uint64_t base = uniform64(seg_base + (uint64_t)(2 * D) * (uint32_t)c0);
        const uint32_t dst = __builtin_amdgcn_readfirstlane(
            lds_offset(&stage[(wig * WP + 4 * g) * PIECE_ELEMS]));
        asm volatile(
            "s_mov_b32 m0, %5\n\t"
            "global_load_lds_dwordx4 %0, %4\n\t"
            "global_load_lds_dwordx4 %1, %4 offset:1024\n\t"
            "global_load_lds_dwordx4 %2, %4 offset:2048\n\t"
            "global_load_lds_dwordx4 %3, %4 offset:3072" ::"v"(cp_off[4 * g]),
            "v"(cp_off[4 * g + 1]), "v"(cp_off[4 * g + 2]), "v"(cp_off[4 * g + 3]), "s"(base),
            "s"(dst)
            : "memory");
      }
    } else {
      // tile straddles a segment end (or the end of the keys): rows are
      // looked up one by one, rows past the end repeat the last key
#pragma unroll
      for (int j = 0; j < WP; ++j) {
        const uint32_t dst = lds_offset(&stage[(wig * WP + j) * PIECE_ELEMS]);
        const int row = (wig * WP + j) * ROWS_PER_PIECE + lane / KCH;
        const int slot = lane % KCH;
        const int c = min(c0 + row, p.Ktot - 1);
        const int swz = copies_v ? v_swz<D>(row) : k_swz<D>(row);
        const uint16_t* src = key_row_sel<D>(p, cp_loc, cp_pass, kvh, c) + 8 * (slot ^ swz);
        asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dwordx4 %0, off" ::"v"(src), "s"(dst)
                     : "memory");
      }
    }
  };
  // Every wave has at most one tile's copies in flight when it waits.
  auto land = []() __attribute__((always_inline)) { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); };

  const int w_first = r0 + kRowsPerWave * wave;
  const bool w_valid = w_first < p.M;
  const int w_lo = vis_end(w_first, p.La, p.Lp);  // shortest visible prefix in the wave
  // 16x16x32 MFMAs: lane (li, lg) is column li of a 16-wide block and holds
  // rows 4*lg .. 4*lg+3 of its accumulator; a wave's 32 queries are two
  // 16-query blocks qb.
  const int li = lane & 15, lg = lane >> 4;
  int rq[2], rq_end[2];
#pragma unroll
  for (int qb = 0; qb < 2; ++qb) {
    rq[qb] = w_first + 16 * qb + li;
    rq_end[qb] = vis_end(rq[qb], p.La, p.Lp);
  }

  // Q^T operand (B of S^T = K Q^T): query block qb, d-step kd holds query
  // rq[qb], dims 32*kd + 8*lg .. +7.
  bf16x8 qreg[2][NKD];
#pragma unroll
  for (int qb = 0; qb < 2; ++qb) {
    const uint16_t* qrow = p.q + ((size_t)head * p.M + min(rq[qb], p.M - 1)) * D;
    const unsigned keep = rq[qb] < p.M ? ~0u : 0u;  // rows past the end multiply by zero
#pragma unroll
    for (int kd = 0; kd < NKD; ++kd) {
      u32x4 raw = *reinterpret_cast<const u32x4*>(qrow + 32 * kd + 8 * lg);
      qreg[qb][kd] = __builtin_bit_cast(bf16x8, raw & keep);
    }
  }

  f32x4 oacc[NDB][2];  // O^T: 16-dim block db x query block qb
#pragma unroll
  for (int db = 0; db < NDB; ++db)
#pragma unroll
    for (int qb = 0; qb < 2; ++qb)
#pragma unroll
      for (int r = 0; r < 4; ++r) oacc[db][qb][r] = 0.f;
  f32x4 s[kKB][2];    // S^T of the current tile: 16-key block kb x query block qb
  bf16x8 pb[NPC][2];  // P of the previous tile: 32-key chunk x query block (B operands)
  float m_run[2] = {-INFINITY, -INFINITY};  // running max of scaled logits (base-2 units)
  float l_run[2] = {0.f, 0.f};              // this lane's share of the running sums

  // LDS operands, addressed as (stage base + lane base) ^ (step bits) +
  // immediate, so no per-step address registers stay live across tiles.
  //  QK step i: d-step kd = i / kKB, key block kb = i % kKB; the A operand
  //  (16 keys x 32 dims) has lane (li, lg) hold key 16*kb + li, chunk
  //  4*kd + lg, stored at chunk (4*kd + lg) ^ (li & (KCH-1)): byte
  //  16*(lg ^ (li & (KCH-1))) xor 64*kd of the row; kb is the immediate.
  //  PV step i: 32-key chunk kc = i / NDB, dim block db = i % NDB; the B
  //  operand pb[kc][qb] has lane group lg hold keys 32*kc + 4*lg + 0..3 and
  //  32*kc + 16 + 4*lg + 0..3 (its S^T accumulator rows, in that order as
  //  k = 8*lg .. 8*lg + 7), and the A operand (16 dims x 32 keys) comes from
  //  two transposing reads rd = 0, 1 of those two key runs: in the 16-lane
  //  group lg, source lane li addresses key row 32*kc + 16*rd + 4*lg + li/4
  //  at dims 16*db + 4*(li%4) .. +3 (result lane li, slot j gets element
  //  li%4 of source lane 4j + li/4).  With the V swizzle the dim block lands
  //  at byte 32*db xor the lane's fixed chunk offset; (kc, rd) is the
  //  immediate.
  const uint32_t k_lane = (uint32_t)(li * 2 * D + 16 * (lg ^ (li & (KCH - 1))));
  uint32_t v_lane;
  {
    const int row = 4 * lg + (li >> 2);
    const int vs = v_swz<D>(row);
    v_lane = (uint32_t)(row * 2 * D + 16 * (((li & 3) >> 1) ^ vs) + 8 * (li & 1));
  }
  auto k_operand = [&](uint32_t kb, int i) __attribute__((always_inline)) -> bf16x8 {
    const uint32_t a = (kb ^ (64u * (uint32_t)(i / kKB))) + (uint32_t)(16 * 2 * D * (i % kKB));
    return *(const lds_bf16x8*)(uintptr_t)a;
  };
  auto v_operand = [&](uint32_t vb, int i) __attribute__((always_inline)) -> bf16x8 {
    const int kc = i / NDB, db = i % NDB;
    const uint32_t x = vb ^ (32u * (uint32_t)db);
    i16x4 part[2];
#pragma unroll
    for (int rd = 0; rd < 2; ++rd)
      part[rd] = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
          (lds_i16x4*)(uintptr_t)(x + (uint32_t)((32 * kc + 16 * rd) * 2 * D)));
    return __builtin_bit_cast(
        bf16x8, __builtin_shufflevector(part[0], part[1], 0, 1, 2, 3, 4, 5, 6, 7));
  };
  auto pv_step = [&](const bf16x8& a, int i) __attribute__((always_inline)) {
    const int kc = i / NDB, db = i % NDB;
#pragma unroll
    for (int qb = 0; qb < 2; ++qb)
      oacc[db][qb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, pb[kc][qb], oacc[db][qb], 0, 0, 0);
  };
  auto qk_step = [&](const bf16x8& a, int i) __attribute__((always_inline)) {
    const int kd = i / kKB, kb = i % kKB;
    const f32x4 zero4 = {};
#pragma unroll
    for (int qb = 0; qb < 2; ++qb)
      s[kb][qb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, qreg[qb][kd],
                                                          kd == 0 ? zero4 : s[kb][qb], 0, 0, 0);
  };

  // MFMA steps.  qk_pv(t) computes S(t) = K(t) Q^T and O += P(t-1) V(t-1),
  // the two streams interleaved step by step with their LDS operands read PD
  // steps ahead into rotating registers; qk_only and pv_only are the first
  // and last tiles.  Every step is two MFMAs per stream (the two query
  // blocks share the operand read).  The scheduling barriers keep the
  // read-ahead distance.
  auto k_stage = [&](int t) __attribute__((always_inline)) { return lds_offset(k_lds[t % kStages]) + k_lane; };
  auto v_stage = [&](int t) __attribute__((always_inline)) { return lds_offset(v_lds[t % kStages]) + v_lane; };
  // copy_v: group A's V(t) copies, issued behind the phase's first operand
  // reads while the matrix core waits for them.
  auto qk_pv = [&](int t, bool copy_v) __attribute__((always_inline)) {
    const uint32_t kl = k_stage(t), vl = v_stage(t - 1);
    bf16x8 ka[PD + 1], va[PD + 1];
#pragma unroll
    for (int i = 0; i < PD; ++i) {
      ka[i] = k_operand(kl, i);
      va[i] = v_operand(vl, i);
    }
    if (copy_v) issue(t);
#pragma unroll
    for (int i = 0; i < NQK; ++i) {
      if (i + PD < NQK) {
        ka[(i + PD) % (PD + 1)] = k_operand(kl, i + PD);
        va[(i + PD) % (PD + 1)] = v_operand(vl, i + PD);
      }
      qk_step(ka[i % (PD + 1)], i);
      pv_step(va[i % (PD + 1)], i);
      __builtin_amdgcn_sched_barrier(0);
    }
  };
  auto qk_only = [&](int t, bool copy_v) __attribute__((always_inline)) {
    const uint32_t kl = k_stage(t);
    bf16x8 ka[PD + 1];
#pragma unroll
    for (int i = 0; i < PD; ++i) ka[i] = k_operand(kl, i);
    if (copy_v) issue(t);
#pragma unroll
    for (int i = 0; i < NQK; ++i) {
      if (i + PD < NQK) ka[(i + PD) % (PD + 1)] = k_operand(kl, i + PD);
      qk_step(ka[i % (PD + 1)], i);
      __builtin_amdgcn_sched_barrier(0);
    }
  };
  auto pv_only = [&](int t) __attribute__((always_inline)) {
    const uint32_t vl = v_stage(t);
    bf16x8 va[PD + 1];
#pragma unroll
    for (int i = 0; i < PD; ++i) va[i] = v_operand(vl, i);
#pragma unroll
    for (int i = 0; i < NPV; ++i) {
      if (i + PD < NPV) va[(i + PD) % (PD + 1)] = v_operand(vl, i + PD);
      pv_step(va[i % (PD + 1)], i);
      __builtin_amdgcn_sched_barrier(0);
    }
  };

  // Row statistics: a query's keys of a tile are spread over the four lane
  // groups (lanes li, li+16, li+32, li+48); the groups' values meet by
  // cross-lane exchanges, on the rare max path and once at the end.
  auto row_sum = [](float x) __attribute__((always_inline)) {
    x += __shfl_xor(x, 16);
    return x + __shfl_xor(x, 32);
  };
  auto row_max = [](float x) __attribute__((always_inline)) {
    x = fmaxf(x, __shfl_xor(x, 16));
    return fmaxf(x, __shfl_xor(x, 32));
  };

  // Softmax of tile t: mask, running max, exp2, row sums, P -> bf16.
  auto softmax = [&](int t) __attribute__((always_inline)) {
    const int c0 = t * kBN;
    if (c0 + kBN > w_lo) {  // tile crosses some row's visible end
#pragma unroll
      for (int kb = 0; kb < kKB; ++kb)
#pragma unroll
        for (int qb = 0; qb < 2; ++qb)
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const int c = c0 + 16 * kb + 4 * lg + r;
            if (c >= rq_end[qb]) s[kb][qb][r] = -INFINITY;
          }
    }
    // Lazy running max without a max pass on the common path: the
    // probabilities are taken against the current (possibly stale) m_run,
    // and only when some lane's tile sum of a row exceeds kSumLimit (a logit
    // far above m_run, or the first tile, where m_run = -inf) does the wave
    // find the rows' tile max, move m_run up to it, rescale O and l, and
    // redo the tile.  O and l share one m_run per row (the four lanes of a
    // row agree on it), and O / l and m_run*ln2 + ln(l) do not depend on its
    // value.  Each 32-key chunk is processed in three batches (its FMAs, its
    // exp2, then its sums and bf16 packing), so that no instruction waits on
    // the latency of the one before it.
    float rs[2][2];
    auto exp_tile = [&]() __attribute__((always_inline)) {
#pragma unroll
      for (int qb = 0; qb < 2; ++qb) rs[qb][0] = rs[qb][1] = 0.f;
#pragma unroll
      for (int kc = 0; kc < NPC; ++kc) {
        f32x4 e[2][2];  // [key block 2kc + h][query block]
#pragma unroll
        for (int h = 0; h < 2; ++h)
#pragma unroll
          for (int qb = 0; qb < 2; ++qb)
#pragma unroll
            for (int r = 0; r < 4; ++r)
              e[h][qb][r] = fmaf(s[2 * kc + h][qb][r], p.scale_log2, -m_run[qb]);
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int h = 0; h < 2; ++h)
#pragma unroll
          for (int qb = 0; qb < 2; ++qb)
#pragma unroll
            for (int r = 0; r < 4; ++r) e[h][qb][r] = __builtin_amdgcn_exp2f(e[h][qb][r]);
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int qb = 0; qb < 2; ++qb) {
#pragma unroll
          for (int h = 0; h < 2; ++h)
            rs[qb][h] += (e[h][qb][0] + e[h][qb][1]) + (e[h][qb][2] + e[h][qb][3]);
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            pb[kc][qb][r] = (__bf16)e[0][qb][r];
            pb[kc][qb][4 + r] = (__bf16)e[1][qb][r];
          }
        }
      }
    };
    exp_tile();
    const float l0 = rs[0][0] + rs[0][1], l1 = rs[1][0] + rs[1][1];
    if (__any(!(l0 <= kSumLimit) || !(l1 <= kSumLimit))) {
#pragma unroll
      for (int qb = 0; qb < 2; ++qb) {
        float mq[2] = {s[0][qb][0], s[1][qb][0]};  // two independent max chains
#pragma unroll
        for (int kb = 0; kb < kKB; ++kb)
#pragma unroll
          for (int r = 0; r < 4; ++r) mq[kb & 1] = fmaxf(mq[kb & 1], s[kb][qb][r]);
        const float mx = row_max(fmaxf(mq[0], mq[1]));
        const float m_new = fmaxf(m_run[qb], mx * p.scale_log2);
        const float alpha = m_new == -INFINITY ? 1.f : __builtin_amdgcn_exp2f(m_run[qb] - m_new);
        m_run[qb] = m_new;
        l_run[qb] *= alpha;
#pragma unroll
        for (int db = 0; db < NDB; ++db)
#pragma unroll
          for (int r = 0; r < 4; ++r) oacc[db][qb][r] *= alpha;
      }
      exp_tile();
    }
#pragma unroll
    for (int qb = 0; qb < 2; ++qb) l_run[qb] += rs[qb][0] + rs[qb][1];
  };

  // Tiles a wave's rows cannot see need no branch: the mask sets their
  // logits to -inf, so their probabilities are 0 and the running max does
  // not move.  The MFMA priority lets the MFMA wave win issue arbitration
  // over the softmax wave sharing its SIMD.
  auto mfma_prio = []() __attribute__((always_inline)) { __builtin_amdgcn_s_setprio(1); };
  auto base_prio = []() __attribute__((always_inline)) { __builtin_amdgcn_s_setprio(0); };
  // Both groups pass the same number of barriers: one after the prologue,
  // then two per tile, then two for the last PV products.
  if (grp == 0) {
    // group A: copies V; MFMA(t) in phase 2t, softmax(t) in phase 2t+1
    phase_barrier();  // K(0) landed (copied by group B)
    mfma_prio();
    qk_only(0, true);
    base_prio();
    phase_barrier();
    softmax(0);
    land();  // V(0)
    phase_barrier();
    for (int t = 1; t < ntiles; ++t) {
      mfma_prio();
      qk_pv(t, true);
      base_prio();
      phase_barrier();
      softmax(t);
      land();  // V(t)
      phase_barrier();
    }
    mfma_prio();
    pv_only(ntiles - 1);
    base_prio();
    phase_barrier();
    phase_barrier();
  } else {
    // group B: copies K; MFMA(t) in phase 2t+1, softmax(t) in phase 2t+2
    issue(0);
    land();  // K(0)
    phase_barrier();
    if (1 < ntiles) issue(1);
    phase_barrier();
    mfma_prio();
    qk_only(0, false);
    base_prio();
    land();  // K(1)
    phase_barrier();
    for (int t = 1; t < ntiles; ++t) {
      if (t + 1 < ntiles) issue(t + 1);
      softmax(t - 1);
      phase_barrier();
      mfma_prio();
      qk_pv(t, false);
      base_prio();
      land();  // K(t+1)
      phase_barrier();
    }
    softmax(ntiles - 1);
    phase_barrier();
    mfma_prio();
    pv_only(ntiles - 1);
    base_prio();
    phase_barrier();
  }

  if (!w_valid) return;
  float l_tot[2];
#pragma unroll
  for (int qb = 0; qb < 2; ++qb) l_tot[qb] = row_sum(l_run[qb]);  // every lane takes part
#pragma unroll
  for (int qb = 0; qb < 2; ++qb) {
    if (rq[qb] >= p.M) continue;
    const float inv = 1.f / l_tot[qb];
    uint16_t* orow = p.o + ((size_t)head * p.M + rq[qb]) * D;
#pragma unroll
    for (int db = 0; db < NDB; ++db) {
      bf16x4 w;
#pragma unroll
      for (int r = 0; r < 4; ++r) w[r] = (__bf16)(oacc[db][qb][r] * inv);
      *reinterpret_cast<bf16x4*>(orow + 16 * db + 4 * lg) = w;
    }
    if (p.lse && lg == 0)
      p.lse[(size_t)head * p.M + rq[qb]] = m_run[qb] * 0.69314718055994531f + logf(l_tot[qb]);
  }
}

}  // namespace

int attention_tile_rows() { return kBM; }

hipError_t launch_attention(const AttnArgs& a, hipStream_t stream) {
  Params p;
  p.q = a.q; p.k = a.k; p.v = a.v; p.kp = a.kp; p.vp = a.vp; p.o = a.o; p.lse = a.lse;
  p.La = a.La; p.Lb = a.Lb; p.lp = a.lp; p.Lp = a.Lp;
  p.M = a.La + a.Lb;
  p.Ktot = a.La + a.Lp + a.Lb;
  p.n_q = a.n_q; p.n_kv = a.n_kv; p.group = a.n_q / a.n_kv;
  p.n_qtiles = (p.M + kBM - 1) / kBM;
  p.xcd_map = (p.n_kv % kXcds) == 0;
  p.scale_log2 = a.scale_log2;
  const dim3 grid((unsigned)(p.n_qtiles * p.n_q));
  if (a.head_dim == 128)
    hipLaunchKernelGGL(attn_fwd_kernel<128>, grid, dim3(kThreads), 0, stream, p);
  else
    hipLaunchKernelGGL(attn_fwd_kernel<64>, grid, dim3(kThreads), 0, stream, p);
  return hipGetLastError();
}

}  // namespace apb
