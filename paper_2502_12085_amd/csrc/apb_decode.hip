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
// partial (O / l, lse) in fp32 to a caller-provided workspace; the merge
// kernel then combines the splits into the host's partial.  Few rows per KV
// head (one generated token): one-wave workgroups of one 32-row block each.
// Many rows (the question tokens): eight-wave workgroups that share each K/V
// block among 256 rows and alternate MFMA and softmax phases between two
// wave groups.
//  * S^T = K Q^T on v_mfma_f32_32x32x16_bf16 (32 keys on M, 32 rows on N).
//  * K and V blocks are copied HBM -> LDS with global_load_lds_dwordx4 into
//    XOR-swizzled row-major tiles, a three-stage ring, so the copies of
//    later blocks fly while block b is computed.  K is read back with
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

#include "apb_internal.h"

namespace apb {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
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
  float* part_o;    // [n_split][n_q * n_new][d]
  float* part_lse;  // [n_split][n_q * n_new]
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
// V: the transposing reads of 4 rows x 4 chunks hit 16 distinct slots.
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

// Keys per ring block of the eight-wave kernel: two 32-key MFMA blocks, so
// that a block's wait and barriers are paid once per 64 keys and its QK
// products run as two independent accumulator chains.
constexpr int kPingPongKB = 2;

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
  __shared__ __attribute__((aligned(16))) uint16_t k_lds[kRing][BK * D];
  __shared__ __attribute__((aligned(16))) uint16_t v_lds[kRing][BK * D];

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
// 32-row block, share every 64-key K/V block of a three-stage LDS ring, and
// work as two groups of four (one wave of each per SIMD) that alternate
// between an MFMA phase {S(b) = K(b) Q^T, O += P(b-1) V(b-1)} and a softmax
// phase one phase apart, as in the prefill kernel: on every SIMD one wave
// feeds the matrix core while the other runs its softmax.  Group A runs the
// MFMA step of block k in phase 2k and its softmax in phase 2k+1, group B one
// phase later; every wave copies its share of block k+1 at the start of
// phase 2k and waits for it at the end of phase 2k+1 (a barrier ends every
// phase).  Block k+1 goes into the stage of block k-2, whose last reader (the
// PV product of group B) ran in phase 2k-1.
template <int D>
__global__ void __launch_bounds__(512) decode_pingpong_kernel(DecParams p) {
  constexpr int W = 8;
  constexpr int KB = kPingPongKB;            // 32-key MFMA blocks per ring block
  constexpr int BK = KB * kKeys;             // keys per ring block
  constexpr int NKC = D / 16;                // MFMA k-steps over head_dim
  constexpr int NDB = D / 32;                // 32-dim blocks of O^T
  constexpr int KCH = D / 8;                 // 16-byte chunks per row
  constexpr int PIECES = BK * D / 512;       // 1 KiB copies per K or V tile
  constexpr int ROWS_PER_PIECE = 512 / D;
  constexpr int CPW = 2 * PIECES / W;        // copies per wave per block
  constexpr int NQK = KB * NKC;              // QK MFMAs per block
  constexpr int NPG = BK / 16;               // 16-key groups of P (PV k-steps)
  constexpr int NPV = NPG * NDB;             // PV MFMAs per block
  constexpr int PD = 2;                      // operand read-ahead (MFMA steps)
  static_assert(CPW * W == 2 * PIECES && NQK == NPV, "tile split");
  __shared__ __attribute__((aligned(16))) uint16_t k_lds[kRing][BK * D];
  __shared__ __attribute__((aligned(16))) uint16_t v_lds[kRing][BK * D];

  const int lane = threadIdx.x & 63, n = lane & 31, h = lane >> 5;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int grp = wave / 4;
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

  // copies: this wave's share, piece q = wave + W*i of the 2*PIECES pieces
  // (K pieces first, then V); a block inside one segment (cache or new
  // rows) takes one scalar base and one M0 per piece, a block straddling the
  // cache end or the last key looks its rows up one by one
  auto load_share = [&](int b, int buf) __attribute__((always_inline)) {
    const int c0 = b * BK;
    const bool in_cache = c0 + BK <= p.Lc;
    const bool in_new = c0 >= p.Lc && c0 + BK <= Ltot;
    // the lane's copy slot is recomputed here (the opaque copy of the lane
    // index keeps the compiler from holding four offsets live across the
    // block loop, where they would be spilled)
    int lane_c = lane;
    asm volatile("" : "+v"(lane_c));
    const int cp_row0 = lane_c / KCH, cp_slot = lane_c % KCH;
#pragma unroll
    for (int i = 0; i < CPW; ++i) {
      const int q = wave + W * i;
      const bool is_v = q >= PIECES;
      const int j = is_v ? q - PIECES : q;
      const int row = j * ROWS_PER_PIECE + cp_row0;
      const int swz = is_v ? v_swz<D>(row) : k_swz<D>(row);
      const uint32_t dst = __builtin_amdgcn_readfirstlane(
          lds_offset(is_v ? &v_lds[buf][j * 512] : &k_lds[buf][j * 512]));
      if (in_cache || in_new) {
        const size_t r0 = in_cache ? (size_t)kvh * p.Lc + c0 : (size_t)kvh * p.n_new + (c0 - p.Lc);
        const uint16_t* base = (is_v ? (in_cache ? p.vc : p.vn) : (in_cache ? p.kc : p.kn)) + r0 * D;
        const uint32_t off = 2u * (uint32_t)(row * D + 8 * (cp_slot ^ swz));
        asm volatile("s_mov_b32 m0, %2\n\tglobal_load_lds_dwordx4 %0, %1" ::"v"(off), "s"(base),
                     "s"(dst)
                     : "memory");
      } else {
        const int c = min(c0 + row, Ltot - 1);
        const uint16_t* src = kv_row<D>(p, is_v ? p.vc : p.kc, is_v ? p.vn : p.kn, kvh, c) +
                              8 * (cp_slot ^ swz);
        asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dwordx4 %0, off" ::"v"(src), "s"(dst)
                     : "memory");
      }
    }
  };
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
  auto k_stage = [&](int k) __attribute__((always_inline)) { return lds_offset(k_lds[k % kRing]) + k_lane; };
  auto v_stage = [&](int k) __attribute__((always_inline)) { return lds_offset(v_lds[k % kRing]) + v_lane; };
  // S of block k (ring index) with O += P V of block k-1, interleaved
  auto qk_pv = [&](int k) __attribute__((always_inline)) {
    const uint32_t kl = k_stage(k), vl = v_stage(k - 1);
    bf16x8 ka[PD + 1], va[PD + 1];
#pragma unroll
    for (int i = 0; i < PD; ++i) {
      ka[i] = k_operand(kl, i);
      va[i] = v_operand(vl, i);
    }
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
  auto qk_only = [&](int k) __attribute__((always_inline)) {
    const uint32_t kl = k_stage(k);
    bf16x8 ka[PD + 1];
#pragma unroll
    for (int i = 0; i < PD; ++i) ka[i] = k_operand(kl, i);
#pragma unroll
    for (int i = 0; i < NQK; ++i) {
      if (i + PD < NQK) ka[(i + PD) % (PD + 1)] = k_operand(kl, i + PD);
      qk_step(ka[i % (PD + 1)], i);
      __builtin_amdgcn_sched_barrier(0);
    }
  };
  auto pv_only = [&](int k) __attribute__((always_inline)) {
    const uint32_t vl = v_stage(k);
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
  // softmax of block b0+k: mask, lazy running max, exp2, row sums, P -> bf16
  auto softmax = [&](int k) __attribute__((always_inline)) {
    const int c0 = (b0 + k) * BK;
    if (c0 + BK > p.Lc) {  // only blocks that reach past the cache can hide keys
#pragma unroll
      for (int sb = 0; sb < KB; ++sb)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int c = c0 + 32 * sb + 8 * (r >> 2) + 4 * h + (r & 3);
          if (c >= vis) s[sb][r] = -INFINITY;
        }
    }
    float rs;
    auto exp_block = [&]() __attribute__((always_inline)) {
      float r4[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int sb = 0; sb < KB; ++sb) {
        float e[16];
#pragma unroll
        for (int r = 0; r < 16; ++r) e[r] = fmaf(s[sb][r], p.scale_log2, -m_run);
#pragma unroll
        for (int r = 0; r < 16; ++r) e[r] = __builtin_amdgcn_exp2f(e[r]);
#pragma unroll
        for (int j = 0; j < 4; ++j) r4[j] += (e[j] + e[4 + j]) + (e[8 + j] + e[12 + j]);
#pragma unroll
        for (int r = 0; r < 16; ++r) pb[2 * sb + (r >> 3)][r & 7] = (__bf16)e[r];
      }
      rs = (r4[0] + r4[1]) + (r4[2] + r4[3]);
    };
    exp_block();
    if (__any(!(rs <= kSumLimit))) {
      float mx = s[0][0];
#pragma unroll
      for (int sb = 0; sb < KB; ++sb)
#pragma unroll
        for (int r = 0; r < 16; ++r) mx = fmaxf(mx, s[sb][r]);
      mx = fmaxf(mx, half_swap(mx));
      const float m_new = fmaxf(m_run, mx * p.scale_log2);
      if (m_new == -INFINITY) {  // nothing visible yet in this row
        rs = 0.f;
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
        exp_block();
      }
    }
    l_run += rs;
  };
  auto mfma_prio = []() __attribute__((always_inline)) { __builtin_amdgcn_s_setprio(1); };
  auto base_prio = []() __attribute__((always_inline)) { __builtin_amdgcn_s_setprio(0); };

  // Both groups pass 2*nb + 3 barriers (a split always owns at least one
  // block unless there are no keys at all, when nobody enters).
  if (nb > 0) {
    load_share(b0, 0);
    land();
    // Q is taken into registers here, where its loads have landed with block
    // 0 (left to itself, the compiler waits for them at their first use,
    // after later copies have been issued, and so also for those copies)
#pragma unroll
    for (int kc = 0; kc < NKC; ++kc) asm volatile("" : "+v"(qreg[kc]));
    barrier();
    if (grp == 0) {
      for (int k = 0; k < nb; ++k) {
        if (k + 1 < nb) load_share(b0 + k + 1, (k + 1) % kRing);
        mfma_prio();
        if (k == 0) qk_only(0);
        else qk_pv(k);
        base_prio();
        barrier();
        softmax(k);
        if (k + 1 < nb) land();
        barrier();
      }
      mfma_prio();
      pv_only(nb - 1);
      base_prio();
      barrier();
      barrier();
    } else {
      if (1 < nb) load_share(b0 + 1, 1);
      barrier();
      for (int k = 0; k < nb; ++k) {
        mfma_prio();
        if (k == 0) qk_only(0);
        else qk_pv(k);
        base_prio();
        if (k + 1 < nb) land();
        barrier();
        if (k + 2 < nb) load_share(b0 + k + 2, (k + 2) % kRing);
        softmax(k);
        barrier();
      }
      mfma_prio();
      pv_only(nb - 1);
      base_prio();
      barrier();
    }
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

// MergeScore over n_parts partial results of `rows` rows: one workgroup per
// row.  The d/4 threads of a group cover the row's d outputs (four each) and
// the THREADS/(d/4) groups split the parts among themselves, so both many
// parts (the splits of one decode call) and few parts with many rows (the
// hosts of a decoding step) keep loads in flight; the groups' sums meet in
// LDS.  THREADS = 1024 when there are few rows and many parts.
template <typename OutT, int THREADS>
__global__ void __launch_bounds__(THREADS) merge_kernel(int n_parts, int rows, int d,
                                                        const float* __restrict__ o_parts,
                                                        const float* __restrict__ lse_parts,
                                                        OutT* __restrict__ o, float* __restrict__ lse) {
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
      float w[4];
      f32x4 x[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        w[u] = lrow[(size_t)(q + u * G) * rows];
        x[u] = *reinterpret_cast<const f32x4*>(o_parts + ((size_t)(q + u * G) * rows + row) * d + c);
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const float e = __expf(w[u] - m);  // 0 for an empty part (lse = -inf)
        acc += e * x[u];
        tot += e;
      }
    }
    for (; q < n_parts; q += G) {
      const float e = __expf(lrow[(size_t)q * rows] - m);
      acc += e * *reinterpret_cast<const f32x4*>(o_parts + ((size_t)q * rows + row) * d + c);
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

template <typename OutT>
hipError_t launch_merge_t(int n_parts, int rows, int d, const float* o_parts,
                          const float* lse_parts, OutT* o, float* lse, hipStream_t stream) {
  if (rows == 0) return hipSuccess;
  // few rows, many parts (the key splits of one generated token): spread
  // each row's parts over 1024 threads so every thread has few loads to wait
  // for; otherwise 256 threads per row
  if (rows < 256 && n_parts >= 16)
    hipLaunchKernelGGL((merge_kernel<OutT, 1024>), dim3((unsigned)rows), dim3(1024), 0, stream,
                       n_parts, rows, d, o_parts, lse_parts, o, lse);
  else
    hipLaunchKernelGGL((merge_kernel<OutT, 256>), dim3((unsigned)rows), dim3(256), 0, stream,
                       n_parts, rows, d, o_parts, lse_parts, o, lse);
  return hipGetLastError();
}

}  // namespace

DecodePlan plan_decode(const DecodeArgs& a) {
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
  pl.n_split = (int)n_split;
  pl.blocks_per_split = (int)bps;
  pl.row_blocks = (int)n_rb;
  const int64_t rows_total = (int64_t)a.n_q * a.n_new;
  pl.workspace_bytes = (uint64_t)n_split * rows_total * (a.head_dim + 1) * 4;
  return pl;
}

hipError_t launch_decode(const DecodeArgs& a, hipStream_t stream) {
  const DecodePlan pl = plan_decode(a);
  DecParams p;
  p.q = a.q; p.kc = a.kc; p.vc = a.vc; p.kn = a.kn; p.vn = a.vn;
  const int64_t rows_total = (int64_t)a.n_q * a.n_new;
  p.part_o = a.workspace;
  p.part_lse = a.workspace + (size_t)pl.n_split * rows_total * a.head_dim;
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
  return launch_merge_t<float>(pl.n_split, (int)rows_total, a.head_dim, p.part_o, p.part_lse,
                               a.o, a.lse, stream);
}

hipError_t launch_merge(const MergeArgs& a, hipStream_t stream) {
  return launch_merge_t<uint16_t>(a.n_parts, a.rows, a.head_dim, a.o_parts, a.lse_parts, a.o,
                                  a.lse, stream);
}

}  // namespace apb
