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
constexpr int kRowsPerWave = 32;
constexpr int kBM = kRowsPerWave * kWaves;  // query rows per workgroup
constexpr int kBN = 32;                     // keys per pipeline unit (one LDS tile)
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

// Wait for this wave's outstanding LDS operations, then the workgroup
// barrier.  Outstanding global loads are not waited for: the staged
// registers carry their own dependency into the LDS stores.
__device__ __forceinline__ void phase_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

template <int N>
struct Slot {
  static constexpr int value = N;
};

template <int D>
__global__ void __launch_bounds__(kThreads, 2)
attn_fwd_kernel(Params p) {
  constexpr int KCH = D / 8;                     // 16-byte chunks per key row
  constexpr int TILE_CHUNKS = kBN * KCH;
  constexpr int LOADS = TILE_CHUNKS / kThreads;  // per thread per tensor
  constexpr int NKC = D / 16;                    // QK MFMA steps per unit (k over head_dim)
  constexpr int NDB = D / 32;                    // 32-wide blocks of head_dim in O^T
  constexpr int NPV = 2 * NDB;                   // PV MFMA steps per unit (2 x 16 keys)
  constexpr int EPS = 16 / NKC;                  // softmax elements per interleaved step
  static_assert(LOADS * kThreads == TILE_CHUNKS, "tile split");
  static_assert(NKC == NPV, "QK and PV step counts match for d in {64, 128}");

  __shared__ __attribute__((aligned(16))) uint16_t k_lds[2][kBN * D];
  __shared__ __attribute__((aligned(16))) uint16_t v_lds[2][kBN * D];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  // Wave index in a scalar register: every per-wave quantity below (row
  // range, tile counts, the pipeline's stage predicates) is then uniform and
  // its branches are scalar branches, not exec-masked ones.
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
  const int rq = w_first + n;  // this lane's query row
  const int rq_end = rq < p.M ? vis_end(rq, p.La, p.Lp) : 0;  // rows past M see nothing

  // Q^T operand: query rq, head_dim slice 16*kc + 8*h .. +7.
  bf16x8 qreg[NKC];
  {
    const uint16_t* qrow = p.q + ((size_t)head * p.M + min(rq, p.M - 1)) * D;
#pragma unroll
    for (int kc = 0; kc < NKC; ++kc) {
      u32x4 raw = rq < p.M ? *reinterpret_cast<const u32x4*>(qrow + 16 * kc + 8 * h)
                           : u32x4{0u, 0u, 0u, 0u};
      qreg[kc] = __builtin_bit_cast(bf16x8, raw);
    }
  }

  f32x16 oacc[NDB];
#pragma unroll
  for (int db = 0; db < NDB; ++db)
#pragma unroll
    for (int r = 0; r < 16; ++r) oacc[db][r] = 0.f;
  f32x16 s[2];        // logits of units u (slot u&1) and u+1
  bf16x8 pbuf[2][2];  // probabilities of units u (slot u&1) and u-1
  float m_run = -INFINITY;  // running max of scaled logits (base-2 units)
  float l_run = 0.f;        // this lane-half's share of the running sum

  // Staged 16-byte chunks of upcoming tiles, two sets: the set loaded in unit
  // u is stored to LDS at the end of unit u+1, so a global load has a whole
  // unit of work to arrive.
  u32x4 kbuf[2][LOADS], vbuf[2][LOADS];

  // Global -> register staging of this thread's chunks of key tile t of K
  // or V.  Rows past Ktot repeat row Ktot-1: they are masked for every query.
  auto row_ptr = [&](const uint16_t* base, const uint16_t* loc, const uint16_t* pass, int c0,
                     int row) -> const uint16_t* {
    return base != nullptr ? base + (size_t)row * D
                           : key_row<D>(p, loc, pass, kvh, min(c0 + row, p.Ktot - 1));
  };
  auto load_k = [&](int t, auto set) {
    constexpr int ST = decltype(set)::value;
    const int c0 = t * kBN;
    const uint16_t* base = tile_base<D>(p, p.k, p.kp, kvh, c0);
#pragma unroll
    for (int i = 0; i < LOADS; ++i) {
      const int e = tid + i * kThreads;
      const int row = e / KCH, ch = e - row * KCH;
      kbuf[ST][i] = *reinterpret_cast<const u32x4*>(row_ptr(base, p.k, p.kp, c0, row) + 8 * ch);
    }
  };
  auto load_v = [&](int t, auto set) {
    constexpr int ST = decltype(set)::value;
    const int c0 = t * kBN;
    const uint16_t* base = tile_base<D>(p, p.v, p.vp, kvh, c0);
#pragma unroll
    for (int i = 0; i < LOADS; ++i) {
      const int e = tid + i * kThreads;
      const int row = e / KCH, ch = e - row * KCH;
      vbuf[ST][i] = *reinterpret_cast<const u32x4*>(row_ptr(base, p.v, p.vp, c0, row) + 8 * ch);
    }
  };
  auto store_k = [&](int buf, auto set) {
    constexpr int ST = decltype(set)::value;
#pragma unroll
    for (int i = 0; i < LOADS; ++i) {
      const int e = tid + i * kThreads;
      const int row = e / KCH, ch = e - row * KCH;
      *reinterpret_cast<u32x4*>(&k_lds[buf][row * D + 8 * (ch ^ k_swz<D>(row))]) = kbuf[ST][i];
    }
  };
  auto store_v = [&](int buf, auto set) {
    constexpr int ST = decltype(set)::value;
#pragma unroll
    for (int i = 0; i < LOADS; ++i) {
      const int e = tid + i * kThreads;
      const int row = e / KCH, ch = e - row * KCH;
      *reinterpret_cast<u32x4*>(&v_lds[buf][row * D + 8 * (ch ^ v_swz<D>(row))]) = vbuf[ST][i];
    }
  };

  // LDS operands.  QK step i (k over head_dim 16i .. 16i+15): A = K rows
  // (lane n holds key n of the unit).  PV step i: 16-key group c = i / NDB,
  // dim block db = i % NDB; pbuf[.][c] slot j of lane half hh holds key
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

  // One 32-key unit u of the pipeline: softmax of S_u (slot SL) interleaved
  // with QK_{u+1} (into slot SL^1, K tile u+1) and, when WITH_PV, PV_{u-1}
  // (probabilities in slot SL^1, V tile u-1).  Every stage runs for every
  // unit: units past a wave's visible range are fully masked and contribute
  // zeros, which keeps the body one straight-line block for the scheduler.
  auto unit = [&](int u, auto slot, auto with_pv) {
    constexpr int SL = decltype(slot)::value;
    constexpr bool PV = decltype(with_pv)::value != 0;
    if (u + 3 < ntiles) load_k(u + 3, Slot<SL>());
    if (u + 1 < ntiles) load_v(u + 1, Slot<SL>());
    const uint16_t* kl = k_lds[(u + 1) & 1];
    const uint16_t* vl = v_lds[(u + 1) & 1];  // V tile u-1
    // The first half of QK_{u+1} does not depend on this unit's softmax: its
    // MFMAs run while the row max and the rescale test below are computed.
    constexpr int NEARLY = NKC / 2;
#pragma unroll
    for (int r = 0; r < 16; ++r) s[SL ^ 1][r] = 0.f;
#pragma unroll
    for (int i = 0; i < NEARLY; ++i)
      s[SL ^ 1] =
          __builtin_amdgcn_mfma_f32_32x32x16_bf16(k_operand(kl, i), qreg[i], s[SL ^ 1], 0, 0, 0);
    const int c0 = u * kBN;
    if (c0 + kBN > w_lo) {  // unit crosses some row's visible end
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int c = c0 + 8 * (r >> 2) + 4 * h + (r & 3);
        if (c >= rq_end) s[SL][r] = -INFINITY;
      }
    }
    float mq[4];  // four independent max chains
#pragma unroll
    for (int j = 0; j < 4; ++j) mq[j] = fmaxf(s[SL][j], s[SL][j + 4]);
#pragma unroll
    for (int r = 8; r < 16; r += 4)
#pragma unroll
      for (int j = 0; j < 4; ++j) mq[j] = fmaxf(mq[j], s[SL][r + j]);
    float mx = fmaxf(fmaxf(mq[0], mq[1]), fmaxf(mq[2], mq[3]));
    mx = fmaxf(mx, half_swap(mx));
    const float m_blk = mx * p.scale_log2;
    // Lazy rescale: m_run only moves when some row's unit max exceeds it by
    // more than 2^kRescaleSlack, so exp2 arguments stay <= kRescaleSlack and
    // O, l and the pending P_{u-1} share the same (possibly stale) m_run;
    // O / l and m_run*ln2 + ln(l) do not depend on the choice.
    if (__any(m_blk > m_run + kRescaleSlack)) {
      const float m_new = fmaxf(m_run, m_blk);
      const float alpha = m_new == -INFINITY ? 1.f : __builtin_amdgcn_exp2f(m_run - m_new);
      m_run = m_new;
      l_run *= alpha;
#pragma unroll
      for (int db = 0; db < NDB; ++db)
#pragma unroll
        for (int r = 0; r < 16; ++r) oacc[db][r] *= alpha;
      if (PV) {
#pragma unroll
        for (int c = 0; c < 2; ++c)
#pragma unroll
          for (int j = 0; j < 8; ++j)
            pbuf[SL ^ 1][c][j] = (__bf16)((float)pbuf[SL ^ 1][c][j] * alpha);
      }
    }
    float rs[4] = {0.f, 0.f, 0.f, 0.f};  // four independent sum chains
    // Remaining QK steps, PV steps and softmax steps interleaved; LDS
    // operands two steps ahead in rotating registers.
    bf16x8 ka[3], va[3];
    ka[0] = k_operand(kl, NEARLY);
    ka[1] = k_operand(kl, NEARLY + 1);
    if (PV) {
      va[0] = v_operand(vl, 0);
      va[1] = v_operand(vl, 1);
    }
#pragma unroll
    for (int i = 0; i < NKC; ++i) {
      if (i + 2 < NKC) {
        if (NEARLY + i + 2 < NKC) ka[(i + 2) % 3] = k_operand(kl, NEARLY + i + 2);
        if (PV) va[(i + 2) % 3] = v_operand(vl, i + 2);
      }
      if (NEARLY + i < NKC)
        s[SL ^ 1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka[i % 3], qreg[NEARLY + i],
                                                             s[SL ^ 1], 0, 0, 0);
#pragma unroll
      for (int x = 0; x < EPS; ++x) {  // softmax elements EPS*i .. EPS*i + EPS-1
        const int r = EPS * i + x;
        const float e = __builtin_amdgcn_exp2f(fmaf(s[SL][r], p.scale_log2, -m_run));
        rs[r & 3] += e;
        pbuf[SL][r >> 3][r & 7] = (__bf16)e;
      }
      if (PV)
        oacc[i % NDB] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
            va[i % 3], pbuf[SL ^ 1][i / NDB], oacc[i % NDB], 0, 0, 0);
    }
    l_run += (rs[0] + rs[1]) + (rs[2] + rs[3]);
    // The set loaded in unit u-1 holds K(u+2) and V(u).  K(u+2) replaces
    // K(u) (last read by QK_u in unit u-1); V(u) replaces V(u-2) (last read
    // by PV_{u-2} in unit u-1).
    if (u + 2 < ntiles) store_k(u & 1, Slot<SL ^ 1>());
    if (u < ntiles) store_v(u & 1, Slot<SL ^ 1>());
    phase_barrier();
  };

  // Prologue: K tiles 0 and 1 in LDS, K(2) and V(0) staged in set 1 for
  // unit 0, S_0 = K(0) Q^T.
  load_k(0, Slot<0>());
  store_k(0, Slot<0>());
  if (ntiles > 1) {
    load_k(1, Slot<0>());
    store_k(1, Slot<0>());
  }
  if (ntiles > 2) load_k(2, Slot<1>());
  load_v(0, Slot<1>());
  phase_barrier();
#pragma unroll
  for (int r = 0; r < 16; ++r) s[0][r] = 0.f;
#pragma unroll
  for (int i = 0; i < NKC; ++i)
    s[0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(k_operand(k_lds[0], i), qreg[i], s[0], 0, 0,
                                                   0);
  phase_barrier();  // unit 0 overwrites K(0)
  // Units 0 .. ntiles: unit 0 has no PV yet, unit ntiles only finishes the
  // last PV.
  unit(0, Slot<0>(), Slot<0>());
  int u = 1;
  for (; u + 1 <= ntiles; u += 2) {
    unit(u, Slot<1>(), Slot<1>());
    unit(u + 1, Slot<0>(), Slot<1>());
  }
  if (u <= ntiles) unit(u, Slot<1>(), Slot<1>());

  if (!w_valid || rq >= p.M) return;
  const float l_tot = l_run + half_swap(l_run);
  const float inv = 1.f / l_tot;
  uint16_t* orow = p.o + ((size_t)head * p.M + rq) * D;
#pragma unroll
  for (int db = 0; db < NDB; ++db)
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      bf16x4 w;
#pragma unroll
      for (int i = 0; i < 4; ++i) w[i] = (__bf16)(oacc[db][4 * g + i] * inv);
      *reinterpret_cast<bf16x4*>(orow + 32 * db + 8 * g + 4 * h) = w;
    }
  if (p.lse && h == 0) p.lse[(size_t)head * p.M + rq] = m_run * 0.69314718055994531f + logf(l_tot);
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
