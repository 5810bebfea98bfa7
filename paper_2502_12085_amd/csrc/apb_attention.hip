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
// Kernel design (one workgroup = 4 waves = 128 query rows of one query head):
//  * Each wave owns 32 query rows and computes S^T = K Q^T with
//    v_mfma_f32_32x32x16_bf16 (keys on the M side, queries on the N side).
//    In that accumulator layout a lane holds one query and 16 keys, so the
//    softmax row statistics are lane-local up to one exchange with the lane
//    32 apart, and the probabilities are already laid out as the B operand of
//    O^T = V^T P^T: no LDS round trip for P.
//  * Q stays in registers for the whole key loop; K tiles (64 keys) are stored
//    row-major in LDS, V tiles transposed, with the 64 keys of a tile permuted
//    so that the 8 keys one lane contracts are contiguous (one 16-byte LDS
//    read per MFMA operand).  Both tiles are double-buffered: the global loads
//    of tile t+1 are in flight while tile t is computed.
//  * Online softmax in fp32 registers in base 2 (scale*log2(e) folded into one
//    FMA), probabilities rounded to bf16 for the PV product, fp32 accumulate.
//  * Tile classes per wave: key tiles wholly visible to all 32 rows run with
//    no mask, tiles crossing the diagonal are masked element-wise, tiles
//    beyond every row's visible prefix are skipped.
//  * Running max updated lazily (only when it grows by more than 2^8), so
//    the O rescale is off the common path.
//  * Grid order puts the query tiles with the longest key prefix first, and
//    keeps a GQA group's workgroups on one XCD (one L2) when n_kv % 8 == 0.
//  * __launch_bounds__(256, 2): at most 256 VGPRs, two waves per SIMD, so one
//    wave's softmax overlaps the other wave's MFMAs.
#include <math.h>

#include "apb_internal.h"

namespace apb {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int kBM = 128;         // query rows per workgroup
constexpr int kBN = 64;          // keys per tile
constexpr int kThreads = 256;    // 4 waves

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

constexpr int kXcds = 8;           // MI355X: 8 XCDs, workgroups dealt round-robin
constexpr float kRescaleSlack = 8.f;  // lazy rescale threshold, base-2 units

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

__device__ __forceinline__ int vis_end(int r, int La, int Lp) {
  return (r < La ? r : r + Lp) + 1;
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

// Value held by the lane 32 apart (the other half of the wave holds the
// other 16 keys of the same query in the 32x32 accumulator layout).
__device__ __forceinline__ float half_swap(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false,
                                                  false);
  const int lane = threadIdx.x & 63;
  return __uint_as_float(lane < 32 ? r[1] : r[0]);
}

// Position of key kk (0..63) of a tile inside a transposed V row: the keys a
// lane-half contracts in one 16-key MFMA step become 8 contiguous entries.
__device__ __forceinline__ int vt_pos(int kk) {
  const int sb = kk >> 5, qq = (kk >> 3) & 3, hh = (kk >> 2) & 1, i = kk & 3;
  return 32 * sb + 16 * (qq >> 1) + 8 * hh + 4 * (qq & 1) + i;
}

template <int D>
__global__ void __launch_bounds__(kThreads, 2)
attn_fwd_kernel(Params p) {
  constexpr int KST = D + 8;            // K tile row stride (bf16 elements)
  constexpr int VST = kBN + 8;          // V^T tile row stride
  constexpr int KCH = D / 8;            // 16-byte pieces per key row
  constexpr int K_LOADS = kBN * KCH / kThreads;          // per thread
  // V is staged in (4 keys x 8 dims) groups; consecutive lanes take
  // consecutive key groups of one 8-dim chunk, so the transposed 8-byte LDS
  // stores of 16 lanes hit 16 different bank pairs.
  constexpr int V_GROUPS = (kBN / 4) * KCH;
  constexpr int V_LOADS = (V_GROUPS + kThreads - 1) / kThreads;
  constexpr int NKC = D / 16;           // MFMA k-steps over head_dim
  constexpr int NDB = D / 32;           // 32-wide blocks of head_dim in O^T
  static_assert(K_LOADS * kThreads == kBN * KCH, "K tile split");

  __shared__ __attribute__((aligned(16))) uint16_t k_lds[2][kBN * KST];
  __shared__ __attribute__((aligned(16))) uint16_t vt_lds[2][D * VST];

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int n = lane & 31, h = lane >> 5;

  int head, qtile;
  map_block(p, blockIdx.x, head, qtile);
  const int kvh = head / p.group;
  const int r0 = qtile * kBM;
  const int r_last = min(r0 + kBM, p.M) - 1;
  const int ntiles = (vis_end(r_last, p.La, p.Lp) + kBN - 1) / kBN;

  const int w_first = r0 + 32 * wave;
  const bool w_valid = w_first < p.M;
  const int w_lo = vis_end(w_first, p.La, p.Lp);
  const int w_hi = vis_end(min(w_first + 31, p.M - 1), p.La, p.Lp);
  const int rq = w_first + n;                       // this lane's query row
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
  float m_run = -INFINITY;  // running max of scaled logits (base-2 units)
  float l_run = 0.f;        // this lane-half's share of the running sum

  uint4 kbuf[K_LOADS];
  uint4 vbuf[V_LOADS][4];

  // Global -> register staging of key tile t.  A tile that lies inside one
  // segment (anchor, one passing slot, or local block) and below Ktot takes a
  // single base address; tiles straddling a boundary fall back to per-row
  // segment lookup.
  auto load_tile = [&](int t) {
    const int c0 = t * kBN;
    const uint16_t* kbase = nullptr;
    const uint16_t* vbase = nullptr;
    if (c0 + kBN <= p.Ktot) {
      if (c0 + kBN <= p.La) {
        const size_t off = ((size_t)kvh * p.M + c0) * D;
        kbase = p.k + off; vbase = p.v + off;
      } else if (c0 >= p.La + p.Lp) {
        const size_t off = ((size_t)kvh * p.M + (c0 - p.Lp)) * D;
        kbase = p.k + off; vbase = p.v + off;
      } else if (c0 >= p.La && c0 + kBN <= p.La + p.Lp) {
        const int tt = c0 - p.La;
        const int sl = tt / p.lp;
        const int r = tt - sl * p.lp;
        if (r + kBN <= p.lp) {
          const size_t off = (((size_t)sl * p.n_kv + kvh) * p.lp + r) * D;
          kbase = p.kp + off; vbase = p.vp + off;
        }
      }
    }
    if (kbase != nullptr) {
      #pragma unroll
      for (int i = 0; i < K_LOADS; ++i) {
        const int e = tid + i * kThreads;
        const int row = e / KCH, ch = e - row * KCH;
        kbuf[i] = *reinterpret_cast<const uint4*>(kbase + (size_t)row * D + 8 * ch);
      }
      #pragma unroll
      for (int i = 0; i < V_LOADS; ++i) {
        const int e = tid + i * kThreads;
        if (e < V_GROUPS) {
          const int g = e % (kBN / 4), ch = e / (kBN / 4);
          #pragma unroll
          for (int j = 0; j < 4; ++j)
            vbuf[i][j] = *reinterpret_cast<const uint4*>(vbase + (size_t)(4 * g + j) * D + 8 * ch);
        }
      }
      return;
    }
    #pragma unroll
    for (int i = 0; i < K_LOADS; ++i) {
      const int e = tid + i * kThreads;
      const int row = e / KCH, ch = e - row * KCH;
      const int c = c0 + row;
      kbuf[i] = c < p.Ktot
                    ? *reinterpret_cast<const uint4*>(key_row<D>(p, p.k, p.kp, kvh, c) + 8 * ch)
                    : make_uint4(0u, 0u, 0u, 0u);
    }
    #pragma unroll
    for (int i = 0; i < V_LOADS; ++i) {
      const int e = tid + i * kThreads;
      if (e < V_GROUPS) {
        const int g = e % (kBN / 4), ch = e / (kBN / 4);
        #pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int c = c0 + 4 * g + j;
          vbuf[i][j] = c < p.Ktot
                           ? *reinterpret_cast<const uint4*>(key_row<D>(p, p.v, p.vp, kvh, c) + 8 * ch)
                           : make_uint4(0u, 0u, 0u, 0u);
        }
      }
    }
  };

  auto store_tile = [&](int buf) {
    #pragma unroll
    for (int i = 0; i < K_LOADS; ++i) {
      const int e = tid + i * kThreads;
      const int row = e / KCH, ch = e - row * KCH;
      *reinterpret_cast<uint4*>(&k_lds[buf][row * KST + 8 * ch]) = kbuf[i];
    }
    #pragma unroll
    for (int i = 0; i < V_LOADS; ++i) {
      const int e = tid + i * kThreads;
      if (e < V_GROUPS) {
        const int g = e % (kBN / 4), ch = e / (kBN / 4);
        const int pos = vt_pos(4 * g);
        const uint32_t* w0 = reinterpret_cast<const uint32_t*>(&vbuf[i][0]);
        const uint32_t* w1 = reinterpret_cast<const uint32_t*>(&vbuf[i][1]);
        const uint32_t* w2 = reinterpret_cast<const uint32_t*>(&vbuf[i][2]);
        const uint32_t* w3 = reinterpret_cast<const uint32_t*>(&vbuf[i][3]);
        #pragma unroll
        for (int d2 = 0; d2 < 4; ++d2) {
          // dims 8*ch + 2*d2 (low halves) and 8*ch + 2*d2 + 1 (high halves)
          const uint32_t a0 = w0[d2], a1 = w1[d2], a2 = w2[d2], a3 = w3[d2];
          uint2 lo, hi;
          lo.x = __builtin_amdgcn_perm(a1, a0, 0x05040100u);
          lo.y = __builtin_amdgcn_perm(a3, a2, 0x05040100u);
          hi.x = __builtin_amdgcn_perm(a1, a0, 0x07060302u);
          hi.y = __builtin_amdgcn_perm(a3, a2, 0x07060302u);
          *reinterpret_cast<uint2*>(&vt_lds[buf][(8 * ch + 2 * d2) * VST + pos]) = lo;
          *reinterpret_cast<uint2*>(&vt_lds[buf][(8 * ch + 2 * d2 + 1) * VST + pos]) = hi;
        }
      }
    }
  };

  load_tile(0);
  store_tile(0);
  __syncthreads();

  for (int t = 0; t < ntiles; ++t) {
    const int buf = t & 1;
    if (t + 1 < ntiles) load_tile(t + 1);
    const int c0 = t * kBN;
    if (w_valid && c0 < w_hi) {
      const uint16_t* kl = k_lds[buf];
      const uint16_t* vl = vt_lds[buf];
      f32x16 s[2];
      #pragma unroll
      for (int sb = 0; sb < 2; ++sb)
        #pragma unroll
        for (int r = 0; r < 16; ++r) s[sb][r] = 0.f;
      #pragma unroll
      for (int kc = 0; kc < NKC; ++kc) {
        #pragma unroll
        for (int sb = 0; sb < 2; ++sb) {
          const bf16x8 a =
              *reinterpret_cast<const bf16x8*>(&kl[(32 * sb + n) * KST + 16 * kc + 8 * h]);
          s[sb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qreg[kc], s[sb], 0, 0, 0);
        }
      }
      if (c0 + kBN > w_lo) {  // tile crosses some row's visible end
        #pragma unroll
        for (int sb = 0; sb < 2; ++sb)
          #pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int c = c0 + 32 * sb + 8 * (r >> 2) + 4 * h + (r & 3);
            if (c >= rq_end) s[sb][r] = -INFINITY;
          }
      }
      float mx = -INFINITY;
      #pragma unroll
      for (int sb = 0; sb < 2; ++sb)
        #pragma unroll
        for (int r = 0; r < 16; ++r) mx = fmaxf(mx, s[sb][r]);
      mx = fmaxf(mx, half_swap(mx));
      const float m_tile = mx * p.scale_log2;
      // Lazy rescale: the running max m_run only moves when some row's tile
      // max exceeds it by more than 2^kRescaleSlack, so exp2 arguments stay
      // <= kRescaleSlack and O and l share the same (possibly stale) m_run;
      // O / l and m_run*ln2 + ln(l) are unchanged by the choice of m_run.
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
      float rs = 0.f;
      bf16x8 pb[4];
      #pragma unroll
      for (int sb = 0; sb < 2; ++sb)
        #pragma unroll
        for (int r = 0; r < 16; ++r) {
          const float e = __builtin_amdgcn_exp2f(fmaf(s[sb][r], p.scale_log2, -m_run));
          rs += e;
          pb[2 * sb + (r >> 3)][r & 7] = (__bf16)e;
        }
      l_run += rs;
      #pragma unroll
      for (int c = 0; c < 4; ++c)
        #pragma unroll
        for (int db = 0; db < NDB; ++db) {
          const bf16x8 a =
              *reinterpret_cast<const bf16x8*>(&vl[(32 * db + n) * VST + 16 * c + 8 * h]);
          oacc[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, pb[c], oacc[db], 0, 0, 0);
        }
    }
    if (t + 1 < ntiles) store_tile(buf ^ 1);
    __syncthreads();
  }

  if (!w_valid || rq >= p.M) return;
  const float l_tot = l_run + half_swap(l_run);
  const float inv = 1.f / l_tot;
  uint16_t* orow = p.o + ((size_t)head * p.M + rq) * D;
  #pragma unroll
  for (int db = 0; db < NDB; ++db)
    #pragma unroll
    for (int g = 0; g < 4; ++g) {
      typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
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
