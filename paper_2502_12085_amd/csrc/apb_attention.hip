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
// Kernel design (one workgroup = 4 waves = 128 query rows of one query head,
// two workgroups per CU, so two independent waves share each SIMD):
//  * Each wave owns 32 query rows and computes S^T = K Q^T with
//    v_mfma_f32_32x32x16_bf16 (keys on the M side, queries on the N side).
//    In that accumulator layout a lane holds one query and 16 keys, so the
//    softmax row statistics are lane-local up to one v_permlane32_swap, and
//    the probabilities are already laid out as the B operand of
//    O^T = V^T P^T: no LDS round trip for P.
//  * In-wave software pipeline over 32-key units: while the VALU runs the
//    softmax of unit u, the same wave's MFMAs compute the logits of unit u+1
//    and the PV product of unit u-1, the three streams interleaved step by
//    step.  Logits and probabilities are double-buffered in registers.  On
//    gfx950 one wave issues VALU work far slower than its MFMA pipe retires
//    32x32x16 products, so the exp/FMA work has to overlap MFMAs inside the
//    wave, not only across waves.
//  * K and V tiles (32 keys) sit row-major in LDS with an XOR swizzle of
//    their 16-byte chunks: the K operand reads (ds_read_b128) and the
//    transposing V operand reads (ds_read_b64_tr_b16) are both free of bank
//    conflicts.  Tiles are double-buffered and staged through registers: the
//    global loads of a unit's successors are issued at its start and stored
//    at its end, one barrier per unit.
//  * Online softmax in fp32 registers in base 2 (scale*log2(e) folded into one
//    FMA), probabilities rounded to bf16 for the PV product, fp32 accumulate.
//    The running max moves lazily (only when it grows by more than 2^8), so
//    the O rescale is off the common path.
//  * Unit classes per wave: units wholly visible to all 32 rows run with no
//    mask, units crossing the diagonal are masked element-wise, units beyond
//    every row's visible prefix are skipped.
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
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) i16x4 lds_i16x4;

constexpr int kWaves = 4;                   // one wave per SIMD; two workgroups per CU
constexpr int kThreads = 64 * kWaves;
#ifndef APB_ROW_BLOCKS
#define APB_ROW_BLOCKS 1
#endif
constexpr int kRB = APB_ROW_BLOCKS;         // 32-row blocks per wave
constexpr int kRowsPerWave = 32 * kRB;
constexpr int kBM = kRowsPerWave * kWaves;  // query rows per workgroup
constexpr int kBN = 32;                     // keys per tile
#ifndef APB_WAVES_PER_SIMD
#define APB_WAVES_PER_SIMD (APB_ROW_BLOCKS == 1 ? 2 : 1)
#endif
#ifndef APB_STAGES
#define APB_STAGES 3
#endif
constexpr int kWavesPerSimd = APB_WAVES_PER_SIMD;  // occupancy target (VGPR budget)
constexpr int kStages = APB_STAGES;                // LDS ring depth for K and V tiles
constexpr int kAhead = kStages - 1;                // tiles in flight ahead of the one computed
constexpr int kXcds = 8;                    // MI355X: 8 XCDs, workgroups dealt round-robin
constexpr float kRescaleSlack = 8.f;        // lazy rescale threshold, base-2 units

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

// Address of concatenated key row c (0 <= c < Ktot) of KV head kvh.
template <int D>
__device__ __forceinline__ const uint16_t* key_row(const Params& p, const uint16_t* loc,
                                                   const uint16_t* pass, int kvh, int c) {
  if (c < p.La) return loc + ((size_t)kvh * p.M + c) * D;
  if (c < p.La + p.Lp) {
    const int t = c - p.La;
    const int s = t / p.lp;
    const int r = t - s * p.lp;
    return pass + (((size_t)s * p.n_kv + kvh) * p.lp + r) * D;
  }
  return loc + ((size_t)kvh * p.M + (c - p.Lp)) * D;
}

// Base address of key tile [c0, c0 + kBN) when it lies inside one segment
// (anchor, one passing slot, or the local block) and below Ktot; nullptr
// when the tile straddles a boundary and rows must be looked up one by one.
template <int D>
__device__ __forceinline__ const uint16_t* tile_base(const Params& p, const uint16_t* loc,
                                                     const uint16_t* pass, int kvh, int c0) {
  if (c0 + kBN > p.Ktot) return nullptr;
  if (c0 + kBN <= p.La) return loc + ((size_t)kvh * p.M + c0) * D;
  if (c0 >= p.La + p.Lp) return loc + ((size_t)kvh * p.M + (c0 - p.Lp)) * D;
  if (c0 >= p.La && c0 + kBN <= p.La + p.Lp) {
    const int t = c0 - p.La;
    const int s = t / p.lp;
    const int r = t - s * p.lp;
    if (r + kBN <= p.lp) return pass + (((size_t)s * p.n_kv + kvh) * p.lp + r) * D;
  }
  return nullptr;
}

// Value held by the lane 32 apart (the other half of the wave holds the
// other 16 keys of the same query in the 32x32 accumulator layout).
__device__ __forceinline__ float half_swap(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false,
                                                  false);
  const int lane = threadIdx.x & 63;
  return __uint_as_float(lane < 32 ? r[1] : r[0]);
}

// LDS tile layouts: row-major [kBN][D] bf16, 16-byte chunk c of row r stored
// at chunk position c ^ swz(r).
//  K: swz = r mod (D/8): the 16 rows one ds_read_b128 pass touches hit 16
//     different chunk positions.
//  V: swz = 4 * (r mod 4) (D = 128): a transposing read touches 4 rows x 4
//     chunks, which land on 16 different chunk positions.
template <int D>
__device__ __forceinline__ int k_swz(int r) { return r & (D / 8 - 1); }
template <int D>
__device__ __forceinline__ int v_swz(int r) { return (4 * (r & 3)) & (D / 8 - 1); }

// Byte offset of an LDS location, as M0 and LDS instructions address it.
__device__ __forceinline__ uint32_t lds_offset(const uint16_t* p) {
  return (uint32_t)(uintptr_t)(__attribute__((address_space(3))) const uint16_t*)p;
}

// Wait for this wave's outstanding LDS operations, then the workgroup
// barrier.  Outstanding global loads are not waited for: the staged
// registers carry their own dependency into the LDS stores.
__device__ __forceinline__ void phase_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

template <int D>
__global__ void __launch_bounds__(kThreads, kWavesPerSimd)
attn_fwd_kernel(Params p) {
  constexpr int KCH = D / 8;                     // 16-byte chunks per key row
  constexpr int PIECE_ELEMS = 512;               // one 1 KiB DMA piece, in bf16
  constexpr int ROWS_PER_PIECE = PIECE_ELEMS / D;
  constexpr int DMA_PER_WAVE = kBN * D / PIECE_ELEMS / kWaves;  // pieces per wave per tensor
  constexpr int NKC = D / 16;                    // QK MFMA steps per tile (k over head_dim)
  constexpr int NDB = D / 32;                    // 32-wide blocks of head_dim in O^T
  static_assert(DMA_PER_WAVE * kWaves * PIECE_ELEMS == kBN * D, "tile split");
  static_assert(DMA_PER_WAVE == 1 || DMA_PER_WAVE == 2, "vmcnt immediates below");

  __shared__ __attribute__((aligned(16))) uint16_t k_lds[kStages][kBN * D];
  __shared__ __attribute__((aligned(16))) uint16_t v_lds[kStages][kBN * D];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  // Wave index in a scalar register: every per-wave quantity below (row
  // range, tile counts) is uniform and its branches are scalar branches.
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int n = lane & 31, h = lane >> 5;

  int head, qtile;
  map_block(p, blockIdx.x, head, qtile);
  const int kvh = head / p.group;
  const int r0 = qtile * kBM;
  const int r_last = min(r0 + kBM, p.M) - 1;
  const int ntiles = (vis_end(r_last, p.La, p.Lp) + kBN - 1) / kBN;

  const int w_first = r0 + kRowsPerWave * wave;
  const bool w_valid = w_first < p.M;
  const int w_lo = vis_end(w_first, p.La, p.Lp);
  const int w_hi = vis_end(min(w_first + kRowsPerWave - 1, p.M - 1), p.La, p.Lp);
  const int w_tiles = w_valid ? (w_hi + kBN - 1) / kBN : 0;
  // Row block b of this wave covers rows w_first + 32*b .. +31; lane n of
  // the S^T / O^T accumulators holds row w_first + 32*b + n.
  int rq[kRB], rq_end[kRB];
#pragma unroll
  for (int b = 0; b < kRB; ++b) {
    rq[b] = w_first + 32 * b + n;
    rq_end[b] = vis_end(rq[b], p.La, p.Lp);
  }

  // Q^T operands: query rq[b], head_dim slice 16*kc + 8*h .. +7.
  bf16x8 qreg[kRB][NKC];
#pragma unroll
  for (int b = 0; b < kRB; ++b) {
    const uint16_t* qrow = p.q + ((size_t)head * p.M + min(rq[b], p.M - 1)) * D;
#pragma unroll
    for (int kc = 0; kc < NKC; ++kc) {
      u32x4 raw = rq[b] < p.M ? *reinterpret_cast<const u32x4*>(qrow + 16 * kc + 8 * h)
                              : u32x4{0u, 0u, 0u, 0u};
      qreg[b][kc] = __builtin_bit_cast(bf16x8, raw);
    }
  }

  f32x16 oacc[kRB][NDB];
#pragma unroll
  for (int b = 0; b < kRB; ++b)
#pragma unroll
    for (int db = 0; db < NDB; ++db)
#pragma unroll
      for (int r = 0; r < 16; ++r) oacc[b][db][r] = 0.f;
  float m_run[kRB], l_run[kRB];  // running max (base-2 units) and lane-half row sum
#pragma unroll
  for (int b = 0; b < kRB; ++b) {
    m_run[b] = -INFINITY;
    l_run[b] = 0.f;
  }

  // HBM -> LDS copies of key tile t (K and V) straight into LDS stage st,
  // without registers: global_load_lds_dwordx4 writes the 16 bytes of lane
  // l to LDS address M0 + 16*l, so each instruction fills one 1 KiB piece of
  // the swizzled tile and every lane fetches the chunk that belongs at its
  // slot.  Each wave issues DMA_PER_WAVE such instructions per tensor.  For a
  // tile inside one segment the per-lane byte offsets within the tile are
  // fixed (precomputed below) and only the tile base, a scalar, changes.
  // Rows past Ktot repeat row Ktot-1: they are masked for every query.
  uint32_t koff[DMA_PER_WAVE], voff[DMA_PER_WAVE];
#pragma unroll
  for (int j = 0; j < DMA_PER_WAVE; ++j) {
    const int row = (wave * DMA_PER_WAVE + j) * ROWS_PER_PIECE + lane / KCH;
    const int slot = lane % KCH;
    koff[j] = 2u * (uint32_t)(row * D + 8 * (slot ^ k_swz<D>(row)));
    voff[j] = 2u * (uint32_t)(row * D + 8 * (slot ^ v_swz<D>(row)));
  }
  auto dma_tile = [&](int t, int st) {
    const int c0 = t * kBN;
    const uint16_t* kb = tile_base<D>(p, p.k, p.kp, kvh, c0);
    const uint16_t* vb = tile_base<D>(p, p.v, p.vp, kvh, c0);
    if (kb != nullptr) {
#pragma unroll
      for (int j = 0; j < DMA_PER_WAVE; ++j) {
        const int piece = wave * DMA_PER_WAVE + j;
        const uint32_t kdst = lds_offset(&k_lds[st][piece * PIECE_ELEMS]);
        const uint32_t vdst = lds_offset(&v_lds[st][piece * PIECE_ELEMS]);
        asm volatile("s_mov_b32 m0, %2\n\tglobal_load_lds_dwordx4 %0, %1" ::"v"(koff[j]),
                     "s"(kb), "s"(kdst)
                     : "memory");
        asm volatile("s_mov_b32 m0, %2\n\tglobal_load_lds_dwordx4 %0, %1" ::"v"(voff[j]),
                     "s"(vb), "s"(vdst)
                     : "memory");
      }
      return;
    }
#pragma unroll
    for (int j = 0; j < DMA_PER_WAVE; ++j) {
      const int piece = wave * DMA_PER_WAVE + j;
      const int row = piece * ROWS_PER_PIECE + lane / KCH;
      const int slot = lane % KCH;
      const int c = min(c0 + row, p.Ktot - 1);
      const uint16_t* ksrc = key_row<D>(p, p.k, p.kp, kvh, c) + 8 * (slot ^ k_swz<D>(row));
      const uint16_t* vsrc = key_row<D>(p, p.v, p.vp, kvh, c) + 8 * (slot ^ v_swz<D>(row));
      const uint32_t kdst = lds_offset(&k_lds[st][piece * PIECE_ELEMS]);
      const uint32_t vdst = lds_offset(&v_lds[st][piece * PIECE_ELEMS]);
      asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dwordx4 %0, off" ::"v"(ksrc), "s"(kdst)
                   : "memory");
      asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dwordx4 %0, off" ::"v"(vsrc), "s"(vdst)
                   : "memory");
    }
  };
  // Wait until this wave's copies of the tile issued before the most recent
  // one have landed (`newer_issued`: whether a later tile's copies follow).
  // `newer` = number of later tiles whose copies are already in flight.
  auto dma_wait = [&](int newer) {
    const int n = newer * 2 * DMA_PER_WAVE;
    if (n >= 8) asm volatile("s_waitcnt vmcnt(8)" ::: "memory");
    else if (n >= 6) asm volatile("s_waitcnt vmcnt(6)" ::: "memory");
    else if (n >= 4) asm volatile("s_waitcnt vmcnt(4)" ::: "memory");
    else if (n >= 2) asm volatile("s_waitcnt vmcnt(2)" ::: "memory");
    else asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  };

  // LDS operands.  QK step i (k over head_dim 16i .. 16i+15): A = K rows
  // (lane n holds key n of the tile).  PV step i: 16-key group c = i / NDB,
  // dim block db = i % NDB; pb[c] slot j of lane half hh holds key
  // 16c + 8*(j/4) + 4*hh + j%4 (the S^T accumulator layout), and the A operand
  // (dims x keys) comes from two transposing reads of 4 keys each: in a
  // 16-lane group g, source lane sl addresses key row 16c + 8*rd + 4*(g/2) +
  // sl/4 at dims 32*db + 16*(g%2) + 4*(sl%4) .. +3, and result lane i, slot j
  // gets element i%4 of source lane 4j + i/4.
  auto k_operand = [&](const uint16_t* kl, int i) -> bf16x8 {
    return *reinterpret_cast<const bf16x8*>(&kl[n * D + 8 * ((2 * i + h) ^ k_swz<D>(n))]);
  };
  auto v_operand = [&](const uint16_t* vl, int i) -> bf16x8 {
    const int c = i / NDB, db = i % NDB;
    const int g = lane >> 4, sl = lane & 15;
    i16x4 part[2];
#pragma unroll
    for (int rd = 0; rd < 2; ++rd) {
      const int row = 16 * c + 8 * rd + 4 * (g >> 1) + (sl >> 2);
      const int dim = 32 * db + 16 * (g & 1) + 4 * (sl & 3);
      const uint16_t* addr = &vl[row * D + 8 * ((dim >> 3) ^ v_swz<D>(row)) + (dim & 7)];
      part[rd] = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)addr);
    }
    return __builtin_bit_cast(
        bf16x8, __builtin_shufflevector(part[0], part[1], 0, 1, 2, 3, 4, 5, 6, 7));
  };

  // Ring of kStages LDS stages: tile t lives in stage t % kStages; the copies
  // of tile t+kAhead are issued at the start of tile t into the stage of
  // tile t-1 (every wave has passed the barrier that ended tile t-1), and
  // tile t+1 must have landed before the barrier that ends tile t.
#pragma unroll
  for (int a = 0; a < kAhead; ++a)
    if (a < ntiles) dma_tile(a, a);
  dma_wait(min(ntiles, kAhead) - 1);
  phase_barrier();

  int st = 0;  // stage of tile t
  for (int t = 0; t < ntiles; ++t) {
    if (t + kAhead < ntiles) dma_tile(t + kAhead, st == 0 ? kStages - 1 : st - 1);
    if (t < w_tiles) {
      const uint16_t* kl = k_lds[st];
      const uint16_t* vl = v_lds[st];
      // S^T = K(t) Q^T per row block: lane (n, h) holds keys
      // 8*(r/4) + 4*h + r%4 of query n.  Every K operand feeds kRB MFMAs.
      f32x16 s[kRB];
#pragma unroll
      for (int b = 0; b < kRB; ++b)
#pragma unroll
        for (int r = 0; r < 16; ++r) s[b][r] = 0.f;
#pragma unroll
      for (int i = 0; i < NKC; ++i) {
        const bf16x8 a = k_operand(kl, i);
#pragma unroll
        for (int b = 0; b < kRB; ++b)
          s[b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qreg[b][i], s[b], 0, 0, 0);
      }
      const int c0 = t * kBN;
      if (c0 + kBN > w_lo) {  // tile crosses some row's visible end
#pragma unroll
        for (int b = 0; b < kRB; ++b)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int c = c0 + 8 * (r >> 2) + 4 * h + (r & 3);
            if (c >= rq_end[b]) s[b][r] = -INFINITY;
          }
      }
      float m_blk[kRB];
      bool grow = false;
#pragma unroll
      for (int b = 0; b < kRB; ++b) {
        float mq[4];  // four independent max chains
#pragma unroll
        for (int j = 0; j < 4; ++j) mq[j] = fmaxf(s[b][j], s[b][j + 4]);
#pragma unroll
        for (int r = 8; r < 16; r += 4)
#pragma unroll
          for (int j = 0; j < 4; ++j) mq[j] = fmaxf(mq[j], s[b][r + j]);
        float mx = fmaxf(fmaxf(mq[0], mq[1]), fmaxf(mq[2], mq[3]));
        mx = fmaxf(mx, half_swap(mx));
        m_blk[b] = mx * p.scale_log2;
        grow = grow || (m_blk[b] > m_run[b] + kRescaleSlack);
      }
      // Lazy rescale: m_run only moves when some row's tile max exceeds it
      // by more than 2^kRescaleSlack, so exp2 arguments stay <= kRescaleSlack
      // and O and l share the same (possibly stale) m_run; O / l and
      // m_run*ln2 + ln(l) do not depend on the choice.
      if (__any(grow)) {
#pragma unroll
        for (int b = 0; b < kRB; ++b) {
          const float m_new = fmaxf(m_run[b], m_blk[b]);
          const float alpha =
              m_new == -INFINITY ? 1.f : __builtin_amdgcn_exp2f(m_run[b] - m_new);
          m_run[b] = m_new;
          l_run[b] *= alpha;
#pragma unroll
          for (int db = 0; db < NDB; ++db)
#pragma unroll
            for (int r = 0; r < 16; ++r) oacc[b][db][r] *= alpha;
        }
      }
      bf16x8 pb[kRB][2];
#pragma unroll
      for (int b = 0; b < kRB; ++b) {
        float rs[4] = {0.f, 0.f, 0.f, 0.f};  // four independent sum chains
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const float e = __builtin_amdgcn_exp2f(fmaf(s[b][r], p.scale_log2, -m_run[b]));
          rs[r & 3] += e;
          pb[b][r >> 3][r & 7] = (__bf16)e;
        }
        l_run[b] += (rs[0] + rs[1]) + (rs[2] + rs[3]);
      }
#pragma unroll
      for (int i = 0; i < 2 * NDB; ++i) {  // every V operand feeds kRB MFMAs
        const bf16x8 a = v_operand(vl, i);
#pragma unroll
        for (int b = 0; b < kRB; ++b)
          oacc[b][i % NDB] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, pb[b][i / NDB],
                                                                    oacc[b][i % NDB], 0, 0, 0);
      }
    }
    dma_wait(min(ntiles - 1 - (t + 1), kAhead - 1) < 0 ? 0 : min(ntiles - 1 - (t + 1), kAhead - 1));
    phase_barrier();
    st = st == kStages - 1 ? 0 : st + 1;
  }

  if (!w_valid) return;
#pragma unroll
  for (int b = 0; b < kRB; ++b) {
    const float l_tot = l_run[b] + half_swap(l_run[b]);
    if (rq[b] >= p.M) continue;
    const float inv = 1.f / l_tot;
    uint16_t* orow = p.o + ((size_t)head * p.M + rq[b]) * D;
#pragma unroll
    for (int db = 0; db < NDB; ++db)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        bf16x4 w;
#pragma unroll
        for (int i = 0; i < 4; ++i) w[i] = (__bf16)(oacc[b][db][4 * g + i] * inv);
        *reinterpret_cast<bf16x4*>(orow + 32 * db + 8 * g + 4 * h) = w;
      }
    if (p.lse && h == 0)
      p.lse[(size_t)head * p.M + rq[b]] = m_run[b] * 0.69314718055994531f + logf(l_tot);
  }
}

}  // namespace

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
