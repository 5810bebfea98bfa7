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
// Kernel design (one workgroup = 8 waves = 256 query rows of one query head):
//  * Each wave owns 32 query rows and computes S^T = K Q^T with
//    v_mfma_f32_32x32x16_bf16 (keys on the M side, queries on the N side).
//    In that accumulator layout a lane holds one query and 16 keys, so the
//    softmax row statistics are lane-local up to one v_permlane32_swap, and
//    the probabilities are already laid out as the B operand of
//    O^T = V^T P^T: no LDS round trip for P.
//  * Ping-pong: waves 0-3 (group A) and 4-7 (group B) put one wave on each
//    SIMD.  The key loop runs in phases separated by workgroup barriers; in
//    every phase one group issues its MFMAs (S(t) = K(t) Q^T and
//    O += P(t-1) V(t-1)) while the other group runs the softmax of its last
//    tile on the VALU, and the groups swap roles each phase, so each SIMD's
//    MFMA pipe is fed by one wave while the other wave's exp/FMA work
//    overlaps it.
//  * K and V tiles (64 keys) sit row-major in LDS with an XOR swizzle of
//    their 16-byte chunks: the K operand reads (ds_read_b128) and the
//    transposing V operand reads (ds_read_b64_tr_b16) are both free of bank
//    conflicts.  Tiles are double-buffered; all 8 waves stage the next tile
//    through a few registers, loaded one phase before they are stored.
//  * Online softmax in fp32 registers in base 2 (scale*log2(e) folded into one
//    FMA), probabilities rounded to bf16 for the PV product, fp32 accumulate.
//    The running max moves lazily (only when it grows by more than 2^8), so
//    the O rescale is off the common path.
//  * Tile classes per wave: key tiles wholly visible to all 32 rows run with
//    no mask, tiles crossing the diagonal are masked element-wise, tiles
//    beyond every row's visible prefix are skipped.
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

constexpr int kWaves = 8;                   // two groups of one wave per SIMD
constexpr int kThreads = 64 * kWaves;
constexpr int kRowsPerWave = 32;
constexpr int kBM = kRowsPerWave * kWaves;  // query rows per workgroup
constexpr int kBN = 64;                     // keys per tile
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

template <int D>
__global__ void __launch_bounds__(kThreads)
attn_fwd_kernel(Params p) {
  constexpr int KCH = D / 8;                    // 16-byte chunks per key row
  constexpr int TILE_CHUNKS = kBN * KCH;
  constexpr int LOADS = TILE_CHUNKS / kThreads;  // per thread per tensor
  constexpr int NKC = D / 16;                   // MFMA k-steps over head_dim
  constexpr int NDB = D / 32;                   // 32-wide blocks of head_dim in O^T
  static_assert(LOADS * kThreads == TILE_CHUNKS, "tile split");

  __shared__ __attribute__((aligned(16))) uint16_t k_lds[2][kBN * D];
  __shared__ __attribute__((aligned(16))) uint16_t v_lds[2][kBN * D];

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int n = lane & 31, h = lane >> 5;
  const int grp = wave >> 2;  // 0: group A, 1: group B

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
  const int rq_end = vis_end(rq, p.La, p.Lp);

  // Q^T operand: query rq, head_dim slice 16*kc + 8*h .. +7.
  bf16x8 qreg[NKC];
  {
    const uint16_t* qrow = p.q + ((size_t)head * p.M + min(rq, p.M - 1)) * D;
#pragma unroll
    for (int kc = 0; kc < NKC; ++kc) {
      uint4 raw = rq < p.M ? *reinterpret_cast<const uint4*>(qrow + 16 * kc + 8 * h)
                           : make_uint4(0u, 0u, 0u, 0u);
      qreg[kc] = __builtin_bit_cast(bf16x8, raw);
    }
  }

  f32x16 oacc[NDB];
#pragma unroll
  for (int db = 0; db < NDB; ++db)
#pragma unroll
    for (int r = 0; r < 16; ++r) oacc[db][r] = 0.f;
  f32x16 s[2];
  bf16x8 pb[4];
  float m_run = -INFINITY;  // running max of scaled logits (base-2 units)
  float l_run = 0.f;        // this lane-half's share of the running sum

  u32x4 kbuf[LOADS], vbuf[LOADS];  // staged 16-byte chunks of the next tiles

  // Global -> register staging of this thread's chunks of key tile t of K
  // (kbuf) or V (vbuf).  Rows past Ktot repeat row Ktot-1: they are masked
  // for every query.
  auto row_ptr = [&](const uint16_t* base, const uint16_t* loc, const uint16_t* pass, int c0,
                     int row) -> const uint16_t* {
    return base != nullptr ? base + (size_t)row * D
                           : key_row<D>(p, loc, pass, kvh, min(c0 + row, p.Ktot - 1));
  };
  auto load_k = [&](int t) {
    const int c0 = t * kBN;
    const uint16_t* base = tile_base<D>(p, p.k, p.kp, kvh, c0);
#pragma unroll
    for (int i = 0; i < LOADS; ++i) {
      const int e = tid + i * kThreads;
      const int row = e / KCH, ch = e - row * KCH;
      kbuf[i] = *reinterpret_cast<const u32x4*>(row_ptr(base, p.k, p.kp, c0, row) + 8 * ch);
    }
  };
  auto load_v = [&](int t) {
    const int c0 = t * kBN;
    const uint16_t* base = tile_base<D>(p, p.v, p.vp, kvh, c0);
#pragma unroll
    for (int i = 0; i < LOADS; ++i) {
      const int e = tid + i * kThreads;
      const int row = e / KCH, ch = e - row * KCH;
      vbuf[i] = *reinterpret_cast<const u32x4*>(row_ptr(base, p.v, p.vp, c0, row) + 8 * ch);
    }
  };
  auto store_k = [&](int buf) {
#pragma unroll
    for (int i = 0; i < LOADS; ++i) {
      const int e = tid + i * kThreads;
      const int row = e / KCH, ch = e - row * KCH;
      *reinterpret_cast<u32x4*>(&k_lds[buf][row * D + 8 * (ch ^ k_swz<D>(row))]) = kbuf[i];
    }
  };
  auto store_v = [&](int buf) {
#pragma unroll
    for (int i = 0; i < LOADS; ++i) {
      const int e = tid + i * kThreads;
      const int row = e / KCH, ch = e - row * KCH;
      *reinterpret_cast<u32x4*>(&v_lds[buf][row * D + 8 * (ch ^ v_swz<D>(row))]) = vbuf[i];
    }
  };

  // MFMA phase of tile t: S(t) = K(t) Q^T (QK steps i = 0..2*NKC-1: k-step
  // i/2, key block i%2) and O^T += V(t-1)^T P(t-1)^T (PV steps i: 16-key
  // group i/NDB, dim block i%NDB).  Both streams are interleaved step by
  // step and their LDS operands are read two steps ahead into rotating
  // registers, so the LDS latency hides behind the MFMAs.
  //
  // PV operands: MFMA step c contracts the 16 keys whose probabilities pb[c]
  // holds: lane half hh, slot j <-> key 16c + 8*(j/4) + 4*hh + j%4 (the S^T
  // accumulator layout).  The A operand (dims x keys) comes from two
  // transposing reads of 4 keys each: in a 16-lane group g, source lane sl
  // addresses key row 16c + 8*rd + 4*(g/2) + sl/4 at dims
  // 32*db + 16*(g%2) + 4*(sl%4) .. +3, and result lane i, slot j gets element
  // i%4 of source lane 4j + i/4.
  constexpr int NQK = 2 * NKC;   // QK MFMA steps per tile
  constexpr int NPV = 4 * NDB;   // PV MFMA steps per tile
  auto k_operand = [&](const uint16_t* kl, int i) -> bf16x8 {
    const int kc = i >> 1, row = 32 * (i & 1) + n;
    return *reinterpret_cast<const bf16x8*>(&kl[row * D + 8 * ((2 * kc + h) ^ k_swz<D>(row))]);
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
  auto qk_step = [&](const bf16x8& a, int i) {
    s[i & 1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qreg[i >> 1], s[i & 1], 0, 0, 0);
  };
  auto pv_step = [&](const bf16x8& a, int i) {
    oacc[i % NDB] =
        __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, pb[i / NDB], oacc[i % NDB], 0, 0, 0);
  };
  auto mfma_phase = [&](int t, bool do_qk, bool do_pv) {
    const uint16_t* kl = k_lds[t & 1];
    const uint16_t* vl = v_lds[(t + 1) & 1];  // V(t-1)
    if (do_qk) {
#pragma unroll
      for (int sb = 0; sb < 2; ++sb)
#pragma unroll
        for (int r = 0; r < 16; ++r) s[sb][r] = 0.f;
    }
    if (do_qk && do_pv) {
      static_assert(NQK == NPV, "QK and PV step counts match for d in {64, 128}");
      bf16x8 ka[3], va[3];
      ka[0] = k_operand(kl, 0); va[0] = v_operand(vl, 0);
      ka[1] = k_operand(kl, 1); va[1] = v_operand(vl, 1);
#pragma unroll
      for (int i = 0; i < NQK; ++i) {
        if (i + 2 < NQK) {
          ka[(i + 2) % 3] = k_operand(kl, i + 2);
          va[(i + 2) % 3] = v_operand(vl, i + 2);
        }
        qk_step(ka[i % 3], i);
        pv_step(va[i % 3], i);
      }
    } else if (do_qk) {
      bf16x8 ka[3];
      ka[0] = k_operand(kl, 0);
      ka[1] = k_operand(kl, 1);
#pragma unroll
      for (int i = 0; i < NQK; ++i) {
        if (i + 2 < NQK) ka[(i + 2) % 3] = k_operand(kl, i + 2);
        qk_step(ka[i % 3], i);
      }
    } else if (do_pv) {
      bf16x8 va[3];
      va[0] = v_operand(vl, 0);
      va[1] = v_operand(vl, 1);
#pragma unroll
      for (int i = 0; i < NPV; ++i) {
        if (i + 2 < NPV) va[(i + 2) % 3] = v_operand(vl, i + 2);
        pv_step(va[i % 3], i);
      }
    }
  };

  // Softmax of tile t: mask, running max, exp2, row sums, P -> bf16.
  auto softmax = [&](int t) {
    const int c0 = t * kBN;
    if (c0 + kBN > w_lo) {  // tile crosses some row's visible end
#pragma unroll
      for (int sb = 0; sb < 2; ++sb)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int c = c0 + 32 * sb + 8 * (r >> 2) + 4 * h + (r & 3);
          if (c >= rq_end) s[sb][r] = -INFINITY;
        }
    }
    float mq[4];  // four independent max chains
#pragma unroll
    for (int j = 0; j < 4; ++j) mq[j] = fmaxf(s[j >> 1][8 * (j & 1)], s[j >> 1][8 * (j & 1) + 1]);
#pragma unroll
    for (int r = 2; r < 8; ++r)
#pragma unroll
      for (int j = 0; j < 4; ++j) mq[j] = fmaxf(mq[j], s[j >> 1][8 * (j & 1) + r]);
    float mx = fmaxf(fmaxf(mq[0], mq[1]), fmaxf(mq[2], mq[3]));
    mx = fmaxf(mx, half_swap(mx));
    const float m_tile = mx * p.scale_log2;
    // Lazy rescale: m_run only moves when some row's tile max exceeds it by
    // more than 2^kRescaleSlack, so exp2 arguments stay <= kRescaleSlack and
    // O and l share the same (possibly stale) m_run; O / l and
    // m_run*ln2 + ln(l) do not depend on the choice of m_run.
    if (__any(m_tile > m_run + kRescaleSlack)) {
      const float m_new = fmaxf(m_run, m_tile);
      const float alpha = m_new == -INFINITY ? 1.f : __builtin_amdgcn_exp2f(m_run - m_new);
      m_run = m_new;
      l_run *= alpha;
#pragma unroll
      for (int db = 0; db < NDB; ++db)
#pragma unroll
        for (int r = 0; r < 16; ++r) oacc[db][r] *= alpha;
    }
    float rs[4] = {0.f, 0.f, 0.f, 0.f};  // four independent sum chains
#pragma unroll
    for (int sb = 0; sb < 2; ++sb)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const float e = __builtin_amdgcn_exp2f(fmaf(s[sb][r], p.scale_log2, -m_run));
        rs[r & 3] += e;
        pb[2 * sb + (r >> 3)][r & 7] = (__bf16)e;
      }
    l_run += (rs[0] + rs[1]) + (rs[2] + rs[3]);
  };

  // Prologue: K(0) in LDS.
  load_k(0);
  store_k(0);
  phase_barrier();

  // Phase ph.  Loads: in phase 2t (t < ntiles) this thread's share of K(t+1)
  // and V(t) goes to registers; at the end of phase 2t+1 it is stored into
  // k_lds[(t+1)&1] (last read in phase 2t-1) and v_lds[t&1] (last read in
  // phase 2t-1).  Compute: group A runs MFMA(t) = {QK(t), PV(t-1)} in phase
  // 2t and softmax(t) in phase 2t+1; group B runs the same one phase later.
  const int nphase = 2 * ntiles + 2;
  for (int ph = 0; ph < nphase; ++ph) {
    const int lt = ph >> 1;  // tile whose V (and the next K) this phase pair stages
    if ((ph & 1) == 0 && lt < ntiles) {
      if (lt + 1 < ntiles) load_k(lt + 1);
      load_v(lt);
    }
    const int my = ph - grp;
    if (my >= 0) {
      const int t = my >> 1;
      if ((my & 1) == 0) {
        // MFMA issue of this wave wins arbitration over the softmax wave
        // sharing its SIMD.
        __builtin_amdgcn_s_setprio(1);
        mfma_phase(t, t < w_tiles, t >= 1 && t - 1 < w_tiles);
        __builtin_amdgcn_s_setprio(0);
      } else if (t < w_tiles) {
        softmax(t);
      }
    }
    if ((ph & 1) == 1 && lt < ntiles) {
      if (lt + 1 < ntiles) store_k((lt + 1) & 1);
      store_v(lt & 1);
    }
    phase_barrier();
  }

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
