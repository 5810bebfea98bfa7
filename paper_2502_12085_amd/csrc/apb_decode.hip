// Decoding stage of APB (stage 2, Alg. 3) for gfx950: one host's exact
// attention of the new tokens against its KV cache, returned with the
// per-row LSE, and MergeScore, the exact combination of such partial results.
//
// Partial attention.  Rows are (query head, new token) pairs; the rows of one
// GQA group are contiguous ([n_q][n_new] order), so a 32-row block of one KV
// head shares every key.  Keys are the host's cache followed, on the last
// host, by the new tokens' own keys (new token j sees the cache and new
// tokens 0..j).  The work is memory-bound (every cached key/value is read
// once and used by at most g * n_new rows), so the key range is split over
// many workgroups (flash-decoding): workgroup (s, kv, rb) runs an online
// softmax over its share of the keys for its rows and writes its normalised
// partial (O / l, lse) to a caller-provided workspace; the merge kernel then
// combines the splits into the host's partial.  One-wave workgroups write the
// partial O in fp32; eight-wave ones, whose 256 rows per split make the
// partials a third of the step's bytes, write it in fp16 against a per-row
// power-of-two scale (every value within 2^-11 of the row's largest).  Few rows per KV
// head (one generated token): one-wave workgroups of one 32-row block each.
// Many rows (the question tokens): eight-wave workgroups that share each
// 128-key K/V tile among 256 rows and alternate MFMA and softmax phases
// between two wave groups, on the prefill kernel's schedule.
//  * S^T = K Q^T on v_mfma_f32_32x32x16_bf16 (32 keys on M, 32 rows on N).
//  * K and V are copied HBM -> LDS with global_load_lds_dwordx4 into
//    XOR-swizzled row-major tiles while earlier ones are computed (32-key
//    blocks through a three-stage ring for one wave; 128-key tiles through
//    two-stage rings, K and V copied in different phases, for eight).  K is
//    read back with
//    ds_read_b128 as the A operand of S^T; V is read back transposed with
//    ds_read_b64_tr_b16 as the A operand of O^T = V^T P^T, and P comes
//    straight from the S^T accumulator layout.
//  * Online softmax in base 2 in fp32 with a lazily moved running max (the
//    max pass and the O rescale only when a block sum passes 2^13), P
//    rounded to bf16 for the PV MFMA.
//
// MergeScore.  lse = m + ln sum_p exp(lse_p - m), A = sum_p exp(lse_p - lse)
// A_p with m the largest lse_p; parts with lse = -inf add nothing; a row
// with no part left gets A = 0, lse = -inf.
#include <math.h>

#include <mutex>

#include "apb_internal.h"

namespace apb {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef _Float16 f16x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) i16x4 lds_i16x4;
typedef __attribute__((address_space(3))) bf16x8 lds_bf16x8;

constexpr int kRows = 32;   // rows per workgroup (the MFMA N side)
constexpr int kKeys = 32;   // keys per MFMA block (the MFMA M side)
constexpr int kWgPerCu = 3; // one-wave workgroups per CU (LDS: 3 x 48 KiB at d = 128)
constexpr int kRing = 3;    // LDS stages of K and V blocks per workgroup
constexpr float kSumLimit = 8192.f;  // lazy rescale: largest block row-half sum against a stale max

struct DecParams {
  const uint16_t* q;
  const uint16_t* kc;
  const uint16_t* vc;
  const uint16_t* kn;
  const uint16_t* vn;
  float* part_o;        // [n_split][n_q * n_new][d] fp32 (one-wave kernel)
  uint16_t* part_h;     // [n_split][n_q * n_new][d] fp16 (eight-wave kernel)
  float* part_scale;    // [n_split][n_q * n_new]: part_h row r is O / part_scale[r]
  float* part_lse;      // [n_split][n_q * n_new]
  int Lc, n_new, append, n_kv, R, rows_total, blocks_per_split;
  float scale_log2;
};

__device__ __forceinline__ float half_swap(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false,
                                                  false);
  return __uint_as_float((threadIdx.x & 63) < 32 ? r[1] : r[0]);
}

// LDS tile swizzles: 16-byte chunk c of key row r sits at chunk c ^ swz(r).
// K: the 32 rows one ds_read_b128 pass touches hit distinct chunk slots;
// V: the transposing reads of 4 rows x 4 chunks hit 16 distinct slots: the
// 32 lanes one clock of such a read serves cover 4 rows x 64 bytes on 4
// different 64-byte bank groups, so these reads are free of bank conflicts.
template <int D>
__device__ __forceinline__ int k_swz(int r) { return r & (D / 8 - 1); }
template <int D>
__device__ __forceinline__ int v_swz(int r) { return (4 * (r & 3)) & (D / 8 - 1); }

__device__ __forceinline__ uint32_t lds_offset(const uint16_t* p) {
  return (uint32_t)(uintptr_t)(__attribute__((address_space(3))) const uint16_t*)p;
}

// s_waitcnt vmcnt(N) for a compile-time N (at most 63).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

// Wait until at most `later` (0 <= later <= MAXN) blocks of CPW copies each
// are outstanding.
template <int CPW, int MAXN>
__device__ __forceinline__ void wait_blocks(int later) {
  if constexpr (MAXN > 0) {
    if (later < MAXN) {
      wait_blocks<CPW, MAXN - 1>(later);
      return;
    }
  }
  wait_vmcnt<CPW * MAXN>();
}

// Key / value row c of the concatenation [cache; new] of KV head kvh.  The
// two bases are pinned in scalar registers: left to itself the compiler turns
// the per-lane choice into a per-lane load of the pointer from the kernel
// arguments, whose wait would also wait for every copy in flight.
template <int D>
__device__ __forceinline__ const uint16_t* kv_row(const DecParams& p, const uint16_t* cache,
                                                  const uint16_t* fresh, int kvh, int c) {
  asm volatile("" : "+s"(cache), "+s"(fresh));
  return c < p.Lc ? cache + ((size_t)kvh * p.Lc + c) * D
                  : fresh + ((size_t)kvh * p.n_new + (c - p.Lc)) * D;
}

// Keys per tile of the eight-wave kernel: four 32-key MFMA blocks, so that a
// phase holds 64 MFMAs (the most the registers allow, as in the prefill
// kernel) and its QK products run as four independent accumulator chains.
constexpr int kPingPongKB = 4;

// Few rows per KV head (one generated token): a one-wave workgroup owns the
// 32-row block blockIdx.z (kWgPerCu of them share a CU's LDS) and streams
// its split's 32-key blocks through its own ring.
template <int D>
__global__ void __launch_bounds__(64) decode_partial_kernel(DecParams p) {
  constexpr int BK = kKeys;                  // keys per ring block
  constexpr int NKC = D / 16;                // MFMA k-steps over head_dim
  constexpr int NDB = D / 32;                // 32-dim blocks of O^T
  constexpr int KCH = D / 8;                 // 16-byte chunks per row
  constexpr int PIECES = BK * D / 512;       // 1 KiB copies per K or V tile
  static_assert(PIECES == 4 || PIECES == 8, "copy unrolling below");
  constexpr int ROWS_PER_PIECE = 512 / D;
  constexpr int CPW = 2 * PIECES;            // copies per block
  // 256-byte aligned: operand addresses XOR step bits into the low byte of
  // a stage base plus lane offset
  __shared__ __attribute__((aligned(256))) uint16_t k_lds[kRing][BK * D];
  __shared__ __attribute__((aligned(256))) uint16_t v_lds[kRing][BK * D];

  const int lane = threadIdx.x & 63, n = lane & 31, h = lane >> 5;
  const int split = blockIdx.x, kvh = blockIdx.y, rb = blockIdx.z;
  const int Ltot = p.Lc + (p.append ? p.n_new : 0);
  const int nblk = (Ltot + BK - 1) / BK;
  const int b0 = split * p.blocks_per_split;
  const int b1 = min(b0 + p.blocks_per_split, nblk);

  // this lane's row (MFMA column n): query head kvh*g + rho / n_new, token rho % n_new
  const int rho = rb * kRows + n;
  const bool row_ok = rho < p.R;
  const int tok = row_ok ? rho % p.n_new : 0;
  const int vis = p.Lc + (p.append ? tok + 1 : 0);  // keys this row sees
  const size_t grow = (size_t)kvh * p.R + (row_ok ? rho : 0);  // row in [n_q * n_new]

  bf16x8 qreg[NKC];  // Q^T operand: row rho, dims 16*kc + 8*h .. +7
  {
    const unsigned keep = row_ok ? ~0u : 0u;
    const uint16_t* qrow = p.q + grow * D;
#pragma unroll
    for (int kc = 0; kc < NKC; ++kc) {
      const u32x4 raw = *reinterpret_cast<const u32x4*>(qrow + 16 * kc + 8 * h);
      qreg[kc] = __builtin_bit_cast(bf16x8, raw & keep);
    }
  }

  // per-lane copy slots: piece j (1 KiB) covers key rows j*ROWS_PER_PIECE ..
  // + ROWS_PER_PIECE-1 (lane / KCH picks the row, lane % KCH the chunk slot)
  const int cp_row0 = lane / KCH, cp_slot = lane % KCH;
  // K operand lane offset: key row n, chunk (2*kc + h) ^ k_swz(n) sits at
  // k_lane ^ (32*kc) (see the prefill kernel)
  const uint32_t k_lane = (uint32_t)(n * 2 * D + 16 * ((h ^ n) & 1) + 16 * (n & (KCH - 2)));
  // transposing-read lane base (see the prefill kernel for the derivation)
  uint32_t v_lane;
  {
    const int g = lane >> 4, sl = lane & 15;
    const int row = 4 * (g >> 1) + (sl >> 2);
    v_lane = (uint32_t)(row * 2 * D + 64 * (row & (NDB - 1)) +
                        16 * (2 * (g & 1) + ((sl & 3) >> 1)) + 8 * (sl & 1));
  }

  // K and V tiles of block b -> LDS buffer buf.  global_load_lds_dwordx4
  // puts lane l's 16 bytes at M0 + inst_offset + 16*l and reads them from
  // saddr + voffset + inst_offset, so a block inside one segment (cache or
  // new rows) takes one scalar base and one M0 per tile; lane offsets
  // (less the piece's KiB) are fixed per lane.  A block that straddles the
  // cache end or the last key looks its rows up one by one (rows past the
  // last key repeat it and are masked).
  uint32_t k_off[PIECES], v_off[PIECES];
#pragma unroll
  for (int j = 0; j < PIECES; ++j) {
    const int row = j * ROWS_PER_PIECE + cp_row0;
    // the instruction offset is 13-bit signed: pieces 4..7 use M0 + 4 KiB
    k_off[j] = 2u * (uint32_t)(row * D + 8 * (cp_slot ^ k_swz<D>(row))) - 1024u * (j & 3);
    v_off[j] = 2u * (uint32_t)(row * D + 8 * (cp_slot ^ v_swz<D>(row))) - 1024u * (j & 3);
  }
  auto load_block = [&](int b, int buf) __attribute__((always_inline)) {
    const int c0 = b * BK;
    const uint32_t kd = __builtin_amdgcn_readfirstlane(lds_offset(k_lds[buf]));
    const uint32_t vd = __builtin_amdgcn_readfirstlane(lds_offset(v_lds[buf]));
    const bool in_cache = c0 + BK <= p.Lc;
    const bool in_new = c0 >= p.Lc && c0 + BK <= Ltot;
    if (in_cache || in_new) {
      const size_t r0 = in_cache ? (size_t)kvh * p.Lc + c0 : (size_t)kvh * p.n_new + (c0 - p.Lc);
      const uint16_t* kb = (in_cache ? p.kc : p.kn) + r0 * D;
      const uint16_t* vb = (in_cache ? p.vc : p.vn) + r0 * D;
#define APB_DEC_PIECE(J, OFFS, BASE)                                                     \
  asm volatile("global_load_lds_dwordx4 %0, %1 offset:" #J ::"v"(OFFS[(J) / 1024 + q4]), \
               "s"(BASE)                                                                 \
               : "memory")
#pragma unroll
      for (int q4 = 0; q4 < PIECES; q4 += 4) {
        asm volatile("s_mov_b32 m0, %0" ::"s"(kd + 1024u * q4) : "memory");
        APB_DEC_PIECE(0, k_off, kb);
        APB_DEC_PIECE(1024, k_off, kb);
        APB_DEC_PIECE(2048, k_off, kb);
        APB_DEC_PIECE(3072, k_off, kb);
        asm volatile("s_mov_b32 m0, %0" ::"s"(vd + 1024u * q4) : "memory");
        APB_DEC_PIECE(0, v_off, vb);
        APB_DEC_PIECE(1024, v_off, vb);
        APB_DEC_PIECE(2048, v_off, vb);
        APB_DEC_PIECE(3072, v_off, vb);
      }
#undef APB_DEC_PIECE
    } else {
#pragma unroll
      for (int j = 0; j < PIECES; ++j) {
        const int row = j * ROWS_PER_PIECE + cp_row0;
        const int c = min(c0 + row, Ltot - 1);
        const uint16_t* ks = kv_row<D>(p, p.kc, p.kn, kvh, c) + 8 * (cp_slot ^ k_swz<D>(row));
        const uint16_t* vs = kv_row<D>(p, p.vc, p.vn, kvh, c) + 8 * (cp_slot ^ v_swz<D>(row));
        asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dwordx4 %0, off" ::"v"(ks),
                     "s"(kd + 1024u * j)
                     : "memory");
        asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dwordx4 %0, off" ::"v"(vs),
                     "s"(vd + 1024u * j)
                     : "memory");
      }
    }
  };

  f32x16 oacc[NDB];
#pragma unroll
  for (int db = 0; db < NDB; ++db)
#pragma unroll
    for (int r = 0; r < 16; ++r) oacc[db][r] = 0.f;
  float m_run = -INFINITY, l_run = 0.f;

  // three-stage ring: blocks b+1 and b+2 fly while block b is computed
#pragma unroll
  for (int i = 0; i < kRing - 1; ++i)
    if (b0 + i < b1) load_block(b0 + i, i);
  static_assert(CPW * (kRing - 2) <= 63, "vmcnt immediate range");
  for (int b = b0; b < b1; ++b) {
    const int buf = (b - b0) % kRing;
    // block b has landed once only the blocks issued after it are outstanding
    wait_blocks<CPW, kRing - 2>(min(b1 - 1 - b, kRing - 2));
    // block b+kRing-1 reuses the stage of block b-1, whose reads are done
    if (b + kRing - 1 < b1) load_block(b + kRing - 1, (b - b0 + kRing - 1) % kRing);
    // The operand reads of each product are issued together ahead of its
    // MFMAs (the scheduling barriers stop the compiler from re-serialising
    // read, wait, MFMA): the K operands, the QK MFMAs, the V operands (read
    // now, so that they land during the softmax), then the PV MFMAs.
    const uint32_t kl = lds_offset(k_lds[buf]);
    bf16x8 kop[NKC];
#pragma unroll
    for (int kc = 0; kc < NKC; ++kc)
      kop[kc] = *(const lds_bf16x8*)(uintptr_t)(kl + (k_lane ^ (32u * (uint32_t)kc)));
    __builtin_amdgcn_sched_barrier(0);
    f32x16 s;
#pragma unroll
    for (int r = 0; r < 16; ++r) s[r] = 0.f;
#pragma unroll
    for (int kc = 0; kc < NKC; ++kc)
      s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kop[kc], qreg[kc], s, 0, 0, 0);
    __builtin_amdgcn_sched_barrier(0);
    // V operands, one per 16-key group of the block and 32-dim block of O^T
    const uint32_t vb = lds_offset(v_lds[buf]);
    bf16x8 vop[2][NDB];
#pragma unroll
    for (int cst = 0; cst < 2; ++cst)
#pragma unroll
      for (int db = 0; db < NDB; ++db) {
        const uint32_t x = vb + (v_lane ^ (64u * (uint32_t)db));
        i16x4 part[2];
#pragma unroll
        for (int rd = 0; rd < 2; ++rd)
          part[rd] = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
              (lds_i16x4*)(uintptr_t)(x + (uint32_t)((16 * cst + 8 * rd) * 2 * D)));
        vop[cst][db] = __builtin_bit_cast(
            bf16x8, __builtin_shufflevector(part[0], part[1], 0, 1, 2, 3, 4, 5, 6, 7));
      }
    __builtin_amdgcn_sched_barrier(0);
    // mask: element r of this lane is key b*BK + 8*(r/4) + 4*h + r%4 of row
    // rho; only blocks that reach past the cache can hide keys
    const int c0 = b * BK;
    if (c0 + BK > p.Lc) {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int c = c0 + 8 * (r >> 2) + 4 * h + (r & 3);
        if (c >= vis) s[r] = -INFINITY;
      }
    }
    // Lazy running max (as in the prefill kernel): the probabilities are
    // formed against the current m_run, and only when some row-half's block
    // sum exceeds kSumLimit (a logit far above m_run, or a row's first
    // visible block, where m_run = -inf and the sum is not finite) does the
    // wave take the block max, raise m_run, rescale O and l and redo the
    // block.  A row that sees no key yet keeps m_run = -inf and P = 0.
    bf16x8 pb[2];
    float rs;
    auto exp_block = [&]() __attribute__((always_inline)) {
      float e[16];
#pragma unroll
      for (int r = 0; r < 16; ++r) e[r] = __builtin_amdgcn_exp2f(fmaf(s[r], p.scale_log2, -m_run));
      float r4[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) r4[j] = (e[j] + e[4 + j]) + (e[8 + j] + e[12 + j]);
#pragma unroll
      for (int r = 0; r < 16; ++r) pb[r >> 3][r & 7] = (__bf16)e[r];
      rs = (r4[0] + r4[1]) + (r4[2] + r4[3]);
    };
    exp_block();
    if (__any(!(rs <= kSumLimit))) {
      float mx = s[0];
#pragma unroll
      for (int r = 0; r < 16; ++r) mx = fmaxf(mx, s[r]);
      mx = fmaxf(mx, half_swap(mx));
      const float m_new = fmaxf(m_run, mx * p.scale_log2);
      if (m_new == -INFINITY) {  // nothing visible yet in this row
        rs = 0.f;
#pragma unroll
        for (int g = 0; g < 2; ++g)
#pragma unroll
          for (int j = 0; j < 8; ++j) pb[g][j] = (__bf16)0.f;
      } else {
        const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);  // m_run = -inf gives 0
        m_run = m_new;
        l_run *= alpha;
#pragma unroll
        for (int db = 0; db < NDB; ++db)
#pragma unroll
          for (int r = 0; r < 16; ++r) oacc[db][r] *= alpha;
        exp_block();
      }
    }
    l_run += rs;
    // O^T += V^T P^T
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int cst = 0; cst < 2; ++cst)
#pragma unroll
      for (int db = 0; db < NDB; ++db)
        oacc[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vop[cst][db], pb[cst], oacc[db], 0, 0, 0);
    // every lane's LDS reads of this buffer are done before it is refilled
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
  }

  if (!row_ok) return;
  const float l_tot = l_run + half_swap(l_run);
  const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
  float* orow = p.part_o + ((size_t)split * p.rows_total + grow) * D;
#pragma unroll
  for (int db = 0; db < NDB; ++db)
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      f32x4 w;
#pragma unroll
      for (int i = 0; i < 4; ++i) w[i] = oacc[db][4 * g + i] * inv;
      *reinterpret_cast<f32x4*>(orow + 32 * db + 8 * g + 4 * h) = w;
    }
  if (h == 0)
    p.part_lse[(size_t)split * p.rows_total + grow] =
        l_tot > 0.f ? m_run * 0.69314718055994531f + logf(l_tot) : -INFINITY;
}

// Many rows per KV head (the question tokens): eight waves, each owning a
// 32-row block, share every 128-key K/V tile of the split, on the prefill
// kernel's schedule.  The waves form two groups of four (one wave of each per
// SIMD) that alternate between an MFMA phase {S(t) = K(t) Q^T, O += P(t-1)
// V(t-1)} and a softmax phase one phase apart: on every SIMD one wave feeds
// the matrix core while the other runs its softmax, and a phase is 64 MFMAs
// long, so its fixed cost (barrier, first operand reads, drain) is spread
// over as much work as the registers allow.  K and V tiles go through
// two-stage rings (128 KiB): group B copies K(T) at the start of phase 2T-2
// (its softmax phase; K(T-2) was last read in phase 2T-3) and waits for it at
// the end of phase 2T-1; group A copies V(T) behind the first operand reads
// of phase 2T (its MFMA phase; V(T-2) was last read in phase 2T-1) and waits
// for it at the end of phase 2T+1.  Tile indices are relative to the split.
template <int D>
__global__ void __launch_bounds__(512) decode_pingpong_kernel(DecParams p) {
  constexpr int W = 8;
  constexpr int GW = W / 2;                  // waves per group
  constexpr int KB = kPingPongKB;            // 32-key MFMA blocks per tile
  constexpr int BK = KB * kKeys;             // keys per tile
  constexpr int NKC = D / 16;                // MFMA k-steps over head_dim
  constexpr int NDB = D / 32;                // 32-dim blocks of O^T
  constexpr int KCH = D / 8;                 // 16-byte chunks per row
  constexpr int PIECES = BK * D / 512;       // 1 KiB copies per K or V tile
  constexpr int ROWS_PER_PIECE = 512 / D;
  constexpr int WP = PIECES / GW;            // copies per wave per tile (one tensor)
  constexpr int NQK = KB * NKC;              // QK MFMAs per tile
  constexpr int NPG = BK / 16;               // 16-key groups of P (PV k-steps)
  constexpr int NPV = NPG * NDB;             // PV MFMAs per tile
  constexpr int PD = 2;                      // operand read-ahead (MFMA steps)
  static_assert(WP * GW == PIECES && WP % 4 == 0 && NQK == NPV, "tile split");
  __shared__ __attribute__((aligned(256))) uint16_t k_lds[2][BK * D];
  __shared__ __attribute__((aligned(256))) uint16_t v_lds[2][BK * D];

  const int lane = threadIdx.x & 63, n = lane & 31, h = lane >> 5;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int grp = wave / GW, wig = wave % GW;
  const int split = blockIdx.x, kvh = blockIdx.y, rb = blockIdx.z * W + wave;
  const int Ltot = p.Lc + (p.append ? p.n_new : 0);
  const int nblk = (Ltot + BK - 1) / BK;
  const int b0 = split * p.blocks_per_split;
  const int nb = max(0, min(b0 + p.blocks_per_split, nblk) - b0);

  // this lane's row (MFMA column n): query head kvh*g + rho / n_new, token rho % n_new
  const int rho = rb * kRows + n;
  const bool row_ok = rho < p.R;
  const int tok = row_ok ? rho % p.n_new : 0;
  const int vis = p.Lc + (p.append ? tok + 1 : 0);  // keys this row sees
  const size_t grow = (size_t)kvh * p.R + (row_ok ? rho : 0);  // row in [n_q * n_new]

  bf16x8 qreg[NKC];  // Q^T operand: row rho, dims 16*kc + 8*h .. +7
  {
    const unsigned keep = row_ok ? ~0u : 0u;
    const uint16_t* qrow = p.q + grow * D;
#pragma unroll
    for (int kc = 0; kc < NKC; ++kc) {
      const u32x4 raw = *reinterpret_cast<const u32x4*>(qrow + 16 * kc + 8 * h);
      qreg[kc] = __builtin_bit_cast(bf16x8, raw & keep);
    }
  }

  // Copies of tile T (keys (b0 + T) * BK ..): group A copies V, group B K;
  // wave wig of a group copies pieces wig*WP .. +WP-1 of the tile.  Inside one
  // segment (cache or new rows) one M0 serves four pieces: the instruction
  // offset moves the LDS destination and the source by the same 1 KiB, the
  // per-lane offsets carry the rest.  A tile that straddles the cache end or
  // the last key looks its rows up one by one (rows past the last key repeat
  // it and are masked).
  const bool copies_v = grp == 0;
  const uint16_t* cp_cache = copies_v ? p.vc : p.kc;
  const uint16_t* cp_new = copies_v ? p.vn : p.kn;
  uint32_t cp_off[WP];  // per-lane byte offset of piece j, less (j % 4) KiB
#pragma unroll
  for (int j = 0; j < WP; ++j) {
    const int row = (wig * WP + j) * ROWS_PER_PIECE + lane / KCH;
    const int slot = lane % KCH;
    const int swz = copies_v ? v_swz<D>(row) : k_swz<D>(row);
    cp_off[j] = 2u * (uint32_t)(row * D + 8 * (slot ^ swz)) - 1024u * (j % 4);
  }
  auto issue = [&](int T) __attribute__((always_inline)) {
    const int c0 = (b0 + T) * BK;
    uint16_t* stage = copies_v ? v_lds[T % 2] : k_lds[T % 2];
    const bool in_cache = c0 + BK <= p.Lc;
    const bool in_new = c0 >= p.Lc && c0 + BK <= Ltot;
    if (in_cache || in_new) {
      const uint16_t* base = in_cache ? cp_cache + ((size_t)kvh * p.Lc + c0) * D
                                      : cp_new + ((size_t)kvh * p.n_new + (c0 - p.Lc)) * D;
#pragma unroll
      for (int g = 0; g < WP / 4; ++g) {
        const uint32_t dst =
            __builtin_amdgcn_readfirstlane(lds_offset(&stage[(wig * WP + 4 * g) * 512]));
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
#pragma unroll
      for (int j = 0; j < WP; ++j) {
        const uint32_t dst = lds_offset(&stage[(wig * WP + j) * 512]);
        const int row = (wig * WP + j) * ROWS_PER_PIECE + lane / KCH;
        const int slot = lane % KCH;
        const int c = min(c0 + row, Ltot - 1);
        const int swz = copies_v ? v_swz<D>(row) : k_swz<D>(row);
        const uint16_t* src = kv_row<D>(p, cp_cache, cp_new, kvh, c) + 8 * (slot ^ swz);
        asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dwordx4 %0, off" ::"v"(src), "s"(dst)
                     : "memory");
      }
    }
  };
  // every wave has at most one tile's copies in flight when it waits
  auto land = []() __attribute__((always_inline)) { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); };
  auto barrier = []() __attribute__((always_inline)) {
    asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
  };

  // operands (the prefill kernel's layouts): QK step i is k-step i / KB of
  // 32-key block i % KB; PV step i is 16-key group i / NDB, dim block i % NDB
  const uint32_t k_lane = (uint32_t)(n * 2 * D + 16 * ((h ^ n) & 1) + 16 * (n & (KCH - 2)));
  uint32_t v_lane;
  {
    const int g = lane >> 4, sl = lane & 15;
    const int row = 4 * (g >> 1) + (sl >> 2);
    v_lane = (uint32_t)(row * 2 * D + 64 * (row & (NDB - 1)) +
                        16 * (2 * (g & 1) + ((sl & 3) >> 1)) + 8 * (sl & 1));
  }
  auto k_operand = [&](uint32_t kb, int i) __attribute__((always_inline)) -> bf16x8 {
    const uint32_t a = (kb ^ (32u * (uint32_t)(i / KB))) + (uint32_t)(kKeys * 2 * D * (i % KB));
    return *(const lds_bf16x8*)(uintptr_t)a;
  };
  auto v_operand = [&](uint32_t vb, int i) __attribute__((always_inline)) -> bf16x8 {
    const int c = i / NDB, db = i % NDB;
    const uint32_t x = vb ^ (64u * (uint32_t)db);
    i16x4 part[2];
#pragma unroll
    for (int rd = 0; rd < 2; ++rd)
      part[rd] = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
          (lds_i16x4*)(uintptr_t)(x + (uint32_t)((16 * c + 8 * rd) * 2 * D)));
    return __builtin_bit_cast(
        bf16x8, __builtin_shufflevector(part[0], part[1], 0, 1, 2, 3, 4, 5, 6, 7));
  };

  f32x16 oacc[NDB];
#pragma unroll
  for (int db = 0; db < NDB; ++db)
#pragma unroll
    for (int r = 0; r < 16; ++r) oacc[db][r] = 0.f;
  f32x16 s[KB];
  bf16x8 pb[NPG];
  float m_run = -INFINITY, l_run = 0.f;

  auto qk_step = [&](const bf16x8& a, int i) __attribute__((always_inline)) {
    const f32x16 zero16 = {};
    s[i % KB] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qreg[i / KB], i < KB ? zero16 : s[i % KB],
                                                        0, 0, 0);
  };
  auto pv_step = [&](const bf16x8& a, int i) __attribute__((always_inline)) {
    oacc[i % NDB] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, pb[i / NDB], oacc[i % NDB], 0, 0, 0);
  };
  auto k_stage = [&](int t) __attribute__((always_inline)) { return lds_offset(k_lds[t % 2]) + k_lane; };
  auto v_stage = [&](int t) __attribute__((always_inline)) { return lds_offset(v_lds[t % 2]) + v_lane; };
  // S of tile t with O += P V of tile t-1, interleaved; copy_v: group A's
  // V(t) copies, issued behind the phase's first operand reads
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
  // Softmax of tile t: mask, lazy running max, exp2, row sums, P -> bf16,
  // one 32-key block at a time in three batches (its FMAs, its exp2, its sums
  // and packing).  A row that sees no key of the split yet keeps m_run = -inf
  // and P = 0.
  auto softmax = [&](int t) __attribute__((always_inline)) {
    const int c0 = (b0 + t) * BK;
    if (c0 + BK > p.Lc) {  // only tiles that reach past the cache can hide keys
#pragma unroll
      for (int b = 0; b < KB; ++b)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int c = c0 + 32 * b + 8 * (r >> 2) + 4 * h + (r & 3);
          if (c >= vis) s[b][r] = -INFINITY;
        }
    }
    float rs[4];
    auto exp_tile = [&]() __attribute__((always_inline)) {
#pragma unroll
      for (int j = 0; j < 4; ++j) rs[j] = 0.f;
#pragma unroll
      for (int b = 0; b < KB; ++b) {
        f32x16 e;
#pragma unroll
        for (int r = 0; r < 16; ++r) e[r] = fmaf(s[b][r], p.scale_log2, -m_run);
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int r = 0; r < 16; ++r) e[r] = __builtin_amdgcn_exp2f(e[r]);
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int k = 0; k < 4; ++k)
#pragma unroll
          for (int j = 0; j < 4; ++j) rs[j] += e[4 * j + k];
#pragma unroll
        for (int r = 0; r < 16; ++r) pb[2 * b + (r >> 3)][r & 7] = (__bf16)e[r];
      }
    };
    exp_tile();
    if (__any(!((rs[0] + rs[1]) + (rs[2] + rs[3]) <= kSumLimit))) {
      float mx = s[0][0];
#pragma unroll
      for (int b = 0; b < KB; ++b)
#pragma unroll
        for (int r = 0; r < 16; ++r) mx = fmaxf(mx, s[b][r]);
      mx = fmaxf(mx, half_swap(mx));
      const float m_new = fmaxf(m_run, mx * p.scale_log2);
      if (m_new == -INFINITY) {  // nothing visible yet in this row
#pragma unroll
        for (int j = 0; j < 4; ++j) rs[j] = 0.f;
#pragma unroll
        for (int g = 0; g < NPG; ++g)
#pragma unroll
          for (int j = 0; j < 8; ++j) pb[g][j] = (__bf16)0.f;
      } else {
        const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);  // m_run = -inf gives 0
        m_run = m_new;
        l_run *= alpha;
#pragma unroll
        for (int db = 0; db < NDB; ++db)
#pragma unroll
          for (int r = 0; r < 16; ++r) oacc[db][r] *= alpha;
        exp_tile();
      }
    }
    l_run += (rs[0] + rs[1]) + (rs[2] + rs[3]);
  };
  auto mfma_prio = []() __attribute__((always_inline)) { __builtin_amdgcn_s_setprio(1); };
  auto base_prio = []() __attribute__((always_inline)) { __builtin_amdgcn_s_setprio(0); };

  // Both groups pass 2*nb + 3 barriers (a split owns at least one tile
  // unless there are no keys at all, when nobody enters).
  if (nb > 0) {
    if (grp == 0) {
      // group A: copies V; MFMA(t) in phase 2t, softmax(t) in phase 2t+1
      barrier();  // K(0) landed (copied by group B)
      mfma_prio();
      qk_only(0, true);
      base_prio();
      barrier();
      softmax(0);
      land();  // V(0)
      barrier();
      for (int t = 1; t < nb; ++t) {
        mfma_prio();
        qk_pv(t, true);
        base_prio();
        barrier();
        softmax(t);
        land();  // V(t)
        barrier();
      }
      mfma_prio();
      pv_only(nb - 1);
      base_prio();
      barrier();
      barrier();
    } else {
      // group B: copies K; MFMA(t) in phase 2t+1, softmax(t) in phase 2t+2
      issue(0);
      land();  // K(0)
      barrier();
      if (1 < nb) issue(1);
      barrier();
      mfma_prio();
      qk_only(0, false);
      base_prio();
      land();  // K(1)
      barrier();
      for (int t = 1; t < nb; ++t) {
        if (t + 1 < nb) issue(t + 1);
        softmax(t - 1);
        barrier();
        mfma_prio();
        qk_pv(t, false);
        base_prio();
        land();  // K(t+1)
        barrier();
      }
      softmax(nb - 1);
      barrier();
      mfma_prio();
      pv_only(nb - 1);
      base_prio();
      barrier();
    }
  }

  if (!row_ok) return;
  const float l_tot = l_run + half_swap(l_run);
  const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
  // fp16 partial: the row's values (this lane and its partner in the other
  // half hold 64 dims each) divided by 2^e, e the exponent of the row's
  // largest magnitude, so every scaled value lies in (-1, 1); the division is
  // exact and the rounding to fp16 is within 2^-11 of the largest value
  float mx = 0.f;
#pragma unroll
  for (int db = 0; db < NDB; ++db)
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      oacc[db][j] *= inv;
      mx = fmaxf(mx, fabsf(oacc[db][j]));
    }
  mx = fmaxf(mx, half_swap(mx));
  const int e = __builtin_amdgcn_frexp_expf(mx);  // 0 for an all-zero row
  uint16_t* hrow = p.part_h + ((size_t)split * p.rows_total + grow) * D;
#pragma unroll
  for (int db = 0; db < NDB; ++db)
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      f16x4 w;
#pragma unroll
      for (int i = 0; i < 4; ++i) w[i] = (_Float16)__builtin_amdgcn_ldexpf(oacc[db][4 * g + i], -e);
      *reinterpret_cast<f16x4*>(hrow + 32 * db + 8 * g + 4 * h) = w;
    }
  if (h == 0) {
    const size_t r = (size_t)split * p.rows_total + grow;
    p.part_lse[r] = l_tot > 0.f ? m_run * 0.69314718055994531f + logf(l_tot) : -INFINITY;
    p.part_scale[r] = __builtin_amdgcn_ldexpf(1.f, e);
  }
}

// MergeScore over n_parts partial results of `rows` rows: one workgroup per
// row.  The d/4 threads of a group cover the row's d outputs (four each) and
// the THREADS/(d/4) groups split the parts among themselves, so both many
// parts (the splits of one decode call) and few parts with many rows (the
// hosts of a decoding step) keep loads in flight; the groups' sums meet in
// LDS.  THREADS = 1024 when there are few rows and many parts.
// Four consecutive values of a part's row as fp32.
__device__ __forceinline__ f32x4 load_part4(const float* q) {
  return *reinterpret_cast<const f32x4*>(q);
}
__device__ __forceinline__ f32x4 load_part4(const uint16_t* q) {  // fp16 bits
  const f16x4 v = *reinterpret_cast<const f16x4*>(q);
  return f32x4{(float)v[0], (float)v[1], (float)v[2], (float)v[3]};
}

// PartT: float parts, or uint16_t parts holding the bits of fp16 values,
// whose row r of part q is O divided by scale_parts[q * rows + r].
template <typename OutT, int THREADS, typename PartT>
__global__ void __launch_bounds__(THREADS) merge_kernel(int n_parts, int rows, int d,
                                                        const PartT* __restrict__ o_parts,
                                                        const float* __restrict__ scale_parts,
                                                        const float* __restrict__ lse_parts,
                                                        OutT* __restrict__ o, float* __restrict__ lse) {
  constexpr bool kScaled = sizeof(PartT) == 2;
  constexpr int NW = THREADS / 64;
  __shared__ float red[NW];
  __shared__ __attribute__((aligned(16))) float acc_lds[THREADS * 4];
  __shared__ float tot_lds[THREADS / 16];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int row = blockIdx.x;
  const int tpr = d / 4, G = THREADS / tpr;
  const int grp = tid / tpr, c = (tid % tpr) * 4;
  const float* lrow = lse_parts + row;

  // 1. m = max over the parts' lse
  float m = -INFINITY;
  for (int q = tid; q < n_parts; q += THREADS) m = fmaxf(m, lrow[(size_t)q * rows]);
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) m = fmaxf(m, __shfl_xor(m, off));
  if (lane == 0) red[wave] = m;
  __syncthreads();
  m = red[0];
#pragma unroll
  for (int w = 1; w < NW; ++w) m = fmaxf(m, red[w]);

  // 2. this group's parts, four loads in flight per thread
  f32x4 acc = {0.f, 0.f, 0.f, 0.f};
  float tot = 0.f;
  if (m != -INFINITY) {
    int q = grp;
    for (; q + 3 * G < n_parts; q += 4 * G) {
      float w[4], sc[4];
      f32x4 x[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const size_t pr = (size_t)(q + u * G) * rows + row;
        w[u] = lse_parts[pr];
        sc[u] = kScaled ? scale_parts[pr] : 1.f;
        x[u] = load_part4(o_parts + pr * d + c);
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const float e = __expf(w[u] - m);  // 0 for an empty part (lse = -inf)
        acc += (kScaled ? e * sc[u] : e) * x[u];
        tot += e;
      }
    }
    for (; q < n_parts; q += G) {
      const size_t pr = (size_t)q * rows + row;
      const float e = __expf(lse_parts[pr] - m);
      acc += (kScaled ? e * scale_parts[pr] : e) * load_part4(o_parts + pr * d + c);
      tot += e;
    }
  }
  // 3. sum over groups
  *reinterpret_cast<f32x4*>(&acc_lds[4 * tid]) = acc;
  if (tid % tpr == 0) tot_lds[grp] = tot;
  __syncthreads();
  if (grp != 0) return;
  for (int g2 = 1; g2 < G; ++g2) {
    acc += *reinterpret_cast<const f32x4*>(&acc_lds[4 * (g2 * tpr + tid)]);
    tot += tot_lds[g2];
  }
  const float inv = tot > 0.f ? 1.f / tot : 0.f;
  if constexpr (sizeof(OutT) == 4) {
    *reinterpret_cast<f32x4*>(reinterpret_cast<float*>(o) + (size_t)row * d + c) = acc * inv;
  } else {
    typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
    bf16x4 w;
#pragma unroll
    for (int i = 0; i < 4; ++i) w[i] = (__bf16)(acc[i] * inv);
    *reinterpret_cast<bf16x4*>(reinterpret_cast<uint16_t*>(o) + (size_t)row * d + c) = w;
  }
  if (lse && tid == 0) lse[row] = tot > 0.f ? m + logf(tot) : -INFINITY;
}

template <typename OutT, typename PartT>
hipError_t launch_merge_t(int n_parts, int rows, int d, const PartT* o_parts,
                          const float* scale_parts, const float* lse_parts, OutT* o, float* lse,
                          hipStream_t stream) {
  if (rows == 0) return hipSuccess;
  // few rows, many parts (the key splits of one generated token): spread
  // each row's parts over 1024 threads so every thread has few loads to wait
  // for; otherwise 256 threads per row
  if (rows < 256 && n_parts >= 16)
    hipLaunchKernelGGL((merge_kernel<OutT, 1024, PartT>), dim3((unsigned)rows), dim3(1024), 0,
                       stream, n_parts, rows, d, o_parts, scale_parts, lse_parts, o, lse);
  else
    hipLaunchKernelGGL((merge_kernel<OutT, 256, PartT>), dim3((unsigned)rows), dim3(256), 0,
                       stream, n_parts, rows, d, o_parts, scale_parts, lse_parts, o, lse);
  return hipGetLastError();
}

}  // namespace

DecodePlan plan_decode(const DecodeArgs& a, uint64_t max_workspace_bytes) {
  DecodePlan pl;
  const int64_t keys = (int64_t)a.Lc + (a.append ? a.n_new : 0);
  const int64_t R = (int64_t)(a.n_q / a.n_kv) * a.n_new;
  // a GQA group of at least four 32-row blocks shares each K/V block among
  // the 8 waves of a workgroup (one workgroup per CU: its registers), else
  // one wave per workgroup (kWgPerCu per CU: their LDS)
  pl.waves = R >= 4 * kRows ? 8 : 1;
  const int64_t bk = pl.waves == 8 ? kPingPongKB * kKeys : kKeys;
  const int64_t nblk = (keys + bk - 1) / bk;
  const int64_t n_rb = (R + kRows * pl.waves - 1) / (kRows * pl.waves);
  // one round of workgroups, at least two key blocks each
  const int64_t target = pl.waves == 1 ? 256 * kWgPerCu : 256;
  int64_t n_split = target / (a.n_kv * n_rb);
  if (n_split > nblk / 2) n_split = nblk / 2;
  if (n_split < 1) n_split = 1;
  int64_t bps = nblk > 0 ? (nblk + n_split - 1) / n_split : 0;
  if (bps > 0) n_split = (nblk + bps - 1) / bps;
  // a workspace limit caps the splits (longer splits, the same kernels)
  const int64_t rows_total = (int64_t)a.n_q * a.n_new;
  // per (split, row): fp32 O and LSE, or fp16 O, its scale and the LSE
  const uint64_t per_row = pl.waves == 8 ? (uint64_t)a.head_dim * 2 + 8 : (uint64_t)(a.head_dim + 1) * 4;
  const uint64_t per_split = (uint64_t)rows_total * per_row;
  if ((uint64_t)n_split * per_split > max_workspace_bytes) {
    const int64_t cap = (int64_t)(max_workspace_bytes / per_split);
    if (cap < 1) {
      pl.n_split = 0;  // does not fit
      pl.blocks_per_split = 0;
      pl.row_blocks = (int)n_rb;
      pl.workspace_bytes = per_split;
      return pl;
    }
    bps = (nblk + cap - 1) / cap;
    n_split = (nblk + bps - 1) / bps;
  }
  pl.n_split = (int)n_split;
  pl.blocks_per_split = (int)bps;
  pl.row_blocks = (int)n_rb;
  pl.workspace_bytes = (uint64_t)n_split * per_split;
  return pl;
}

// Device scratch of the no-allocation entry point: one array per GPU (each
// device holds its own copy of a __device__ variable), found once per device
// by its symbol.  In host code `scratch` names a host-side stand-in, never the
// device memory: only the address from hipGetSymbolAddress is handed to
// kernels.
static __device__ __align__(256) float scratch[kDecodeScratchBytes / sizeof(float)];

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};
}  // namespace

hipError_t decode_scratch(void** ptr) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* addr = nullptr;
    e = hipGetSymbolAddress(&addr, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!addr) return hipErrorInvalidSymbol;
    g_scratch_ptr[dev] = addr;
  }
  *ptr = g_scratch_ptr[dev];
  return hipSuccess;
}

hipError_t launch_decode(const DecodeArgs& a, const DecodePlan& pl, hipStream_t stream) {
  DecParams p;
  p.q = a.q; p.kc = a.kc; p.vc = a.vc; p.kn = a.kn; p.vn = a.vn;
  const int64_t rows_total = (int64_t)a.n_q * a.n_new;
  const size_t parts = (size_t)pl.n_split * rows_total;  // (split, row) pairs
  if (pl.waves == 8) {
    // fp16 O, then the scales, then the LSEs
    p.part_o = nullptr;
    p.part_h = reinterpret_cast<uint16_t*>(a.workspace);
    p.part_scale = reinterpret_cast<float*>(p.part_h + parts * a.head_dim);
    p.part_lse = p.part_scale + parts;
  } else {
    // fp32 O, then the LSEs
    p.part_o = a.workspace;
    p.part_h = nullptr;
    p.part_scale = nullptr;
    p.part_lse = a.workspace + parts * a.head_dim;
  }
  p.Lc = a.Lc; p.n_new = a.n_new; p.append = a.append; p.n_kv = a.n_kv;
  p.R = (a.n_q / a.n_kv) * a.n_new;
  p.rows_total = (int)rows_total;
  p.blocks_per_split = pl.blocks_per_split;
  p.scale_log2 = a.scale_log2;
  const dim3 grid((unsigned)pl.n_split, (unsigned)a.n_kv, (unsigned)pl.row_blocks);
  const dim3 block((unsigned)(64 * pl.waves));
  if (a.head_dim == 128) {
    if (pl.waves == 8) hipLaunchKernelGGL((decode_pingpong_kernel<128>), grid, block, 0, stream, p);
    else hipLaunchKernelGGL((decode_partial_kernel<128>), grid, block, 0, stream, p);
  } else {
    if (pl.waves == 8) hipLaunchKernelGGL((decode_pingpong_kernel<64>), grid, block, 0, stream, p);
    else hipLaunchKernelGGL((decode_partial_kernel<64>), grid, block, 0, stream, p);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (pl.waves == 8)
    return launch_merge_t(pl.n_split, (int)rows_total, a.head_dim,
                          static_cast<const uint16_t*>(p.part_h), p.part_scale, p.part_lse,
                          a.o, a.lse, stream);
  return launch_merge_t(pl.n_split, (int)rows_total, a.head_dim, p.part_o,
                        static_cast<const float*>(nullptr), p.part_lse, a.o, a.lse, stream);
}

hipError_t launch_merge(const MergeArgs& a, hipStream_t stream) {
  return launch_merge_t<uint16_t, float>(a.n_parts, a.rows, a.head_dim, a.o_parts, nullptr,
                                         a.lse_parts, a.o, a.lse, stream);
}

}  // namespace apb
