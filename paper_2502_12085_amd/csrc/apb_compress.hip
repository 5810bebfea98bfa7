// Compressor of one APB host (Sec. 3.4; Alg. 2, compression step) for gfx950:
// ArgTop-l_p of the retaining-head scores of every KV head, then the gather
// K^C = K_h[idx], V^C = V_h[idx].
//
// Design.  A grid of (S, n_kv) workgroups; workgroup (c, h) owns the local
// index range chunk c of KV head h.  Every workgroup of a head first finds
// the same selection threshold by an MSB-first radix select over all Lb
// scores (digits of an order-preserving 32-bit key: four of 8 bits here, three
// of 11, 11 and 10 bits in the register-resident kernel below; the scores of
// one head are a few hundred KB at most and stay in L2), so no scratch memory,
// atomics across workgroups or second launch are needed.  It then counts
// what was selected before its chunk and compacts its chunk in index order
// (wave ballot + mbcnt prefix counts, a 4-wave LDS scan), which yields the
// ascending output order and the lower-index-wins tie rule directly.  The
// selected rows are copied with 16-byte vector loads and stores.
#include "apb_internal.h"

namespace apb {
namespace {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / 64;

// Order-preserving map of an fp32 score to an unsigned key: a larger score
// gives a larger key, -0 maps with +0, NaN maps to 0 (below -inf, whose key
// is 0x007fffff).
__device__ __forceinline__ uint32_t score_key(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return 0u;
  if (u == 0x80000000u) u = 0u;
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// Exclusive prefix count of `pred` over the 256 threads of the block, in
// thread order; also returns the block total.  Uses `scan` (kWaves words).
__device__ __forceinline__ uint32_t block_exclusive_count(bool pred, uint32_t* scan,
                                                          uint32_t* total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const unsigned long long bal = __ballot(pred);
  const uint32_t in_wave = __builtin_amdgcn_mbcnt_hi(
      (uint32_t)(bal >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)bal, 0u));
  if (lane == 0) scan[wave] = (uint32_t)__popcll(bal);
  __syncthreads();
  uint32_t before = 0, all = 0;
  for (int w = 0; w < kWaves; ++w) {
    const uint32_t c = scan[w];
    before += (w < wave) ? c : 0u;
    all += c;
  }
  __syncthreads();
  *total = all;
  return before + in_wave;
}

__global__ void __launch_bounds__(kThreads)
topk_gather_kernel(const float* __restrict__ scores, const uint16_t* __restrict__ k,
                   const uint16_t* __restrict__ v, int32_t* __restrict__ out_idx,
                   uint16_t* __restrict__ out_k, uint16_t* __restrict__ out_v,
                   int La, int Lb, int lp, int head_dim, int chunk) {
  __shared__ uint32_t hist[256];
  __shared__ uint32_t scan[kWaves];
  __shared__ uint32_t sel_digit, sel_above;
  __shared__ int32_t list_src[kThreads];
  __shared__ int32_t list_dst[kThreads];

  const int tid = threadIdx.x, lane = tid & 63;
  const int head = blockIdx.y;
  const float* s = scores + (size_t)head * Lb;

  // ---- 1. radix select: key T of the lp-th largest score, and how many of
  //         the scores equal to T are selected (`need`, >= 1).
  uint32_t prefix = 0u, prefix_mask = 0u, remaining = (uint32_t)lp;
  for (int pass = 0; pass < 4; ++pass) {
    const int shift = 24 - 8 * pass;
    hist[tid] = 0u;
    __syncthreads();
    for (int i = tid; i < Lb; i += kThreads) {
      const uint32_t key = score_key(s[i]);
      if ((key & prefix_mask) == prefix) atomicAdd(&hist[(key >> shift) & 255u], 1u);
    }
    __syncthreads();
    if (tid < 64) {
      // lane L owns bins 4L..4L+3; suffix sums over lanes find the bin
      // holding the remaining-th largest key.
      uint32_t c[4], own = 0u;
      for (int j = 0; j < 4; ++j) { c[j] = hist[4 * lane + j]; own += c[j]; }
      uint32_t incl = own;  // inclusive suffix sum over lanes >= lane
      for (int off = 1; off < 64; off <<= 1) {
        const uint32_t o = __shfl_down(incl, off);
        if (lane + off < 64) incl += o;
      }
      const uint32_t above_lane = incl - own;
      if (above_lane < remaining && remaining <= incl) {
        uint32_t above = above_lane;
        for (int j = 3; j >= 0; --j) {
          if (remaining <= above + c[j]) {
            sel_digit = (uint32_t)(4 * lane + j);
            sel_above = above;
            break;
          }
          above += c[j];
        }
      }
    }
    __syncthreads();
    prefix |= sel_digit << shift;
    prefix_mask |= 255u << shift;
    remaining -= sel_above;
    __syncthreads();
  }
  const uint32_t T = prefix;
  const uint32_t need = remaining;

  // ---- 2. selected elements before this workgroup's chunk.
  const int c0 = blockIdx.x * chunk;
  const int c1 = min(Lb, c0 + chunk);
  if (c0 >= c1) return;
  uint32_t gt_before = 0u, eq_before = 0u;
  for (int base = 0; base < c0; base += kThreads) {
    const int i = base + tid;
    const uint32_t key = (i < c0) ? score_key(s[i]) : 0u;
    uint32_t tg, te;
    block_exclusive_count(i < c0 && key > T, scan, &tg);
    block_exclusive_count(i < c0 && key == T, scan, &te);
    gt_before += tg;
    eq_before += te;
  }

  // ---- 3. compaction of the chunk in index order + row gather.
  const int row_chunks = head_dim / 8;  // 16-byte pieces per row
  const size_t M = (size_t)La + Lb;
  const uint4* ksrc = reinterpret_cast<const uint4*>(k + (size_t)head * M * head_dim);
  const uint4* vsrc = reinterpret_cast<const uint4*>(v + (size_t)head * M * head_dim);
  uint4* kdst = reinterpret_cast<uint4*>(out_k + (size_t)head * lp * head_dim);
  uint4* vdst = reinterpret_cast<uint4*>(out_v + (size_t)head * lp * head_dim);
  for (int base = c0; base < c1; base += kThreads) {
    const int i = base + tid;
    const uint32_t key = (i < c1) ? score_key(s[i]) : 0u;
    const bool gt = i < c1 && key > T;
    const bool eq = i < c1 && key == T;
    uint32_t tg, te;
    const uint32_t gx = gt_before + block_exclusive_count(gt, scan, &tg);
    const uint32_t ex = eq_before + block_exclusive_count(eq, scan, &te);
    const uint32_t pos = gx + min(ex, need);
    // pos < lp holds by construction (exactly lp elements are selected); the
    // test keeps every store in bounds regardless.
    const bool sel = (gt || (eq && ex < need)) && pos < (uint32_t)lp;
    uint32_t nsel;
    const uint32_t slot = block_exclusive_count(sel, scan, &nsel);
    if (sel) {
      if (out_idx) out_idx[(size_t)head * lp + pos] = i;
      list_src[slot] = i;
      list_dst[slot] = (int32_t)pos;
    }
    __syncthreads();
    const int pieces = (int)nsel * row_chunks;
    for (int e = tid; e < 2 * pieces; e += kThreads) {
      const int which = e >= pieces;  // 0: K, 1: V
      const int ee = e - which * pieces;
      const int r = ee / row_chunks, ch = ee - r * row_chunks;
      const size_t src = ((size_t)La + list_src[r]) * row_chunks + ch;
      const size_t dst = (size_t)list_dst[r] * row_chunks + ch;
      if (which) vdst[dst] = vsrc[src];
      else kdst[dst] = ksrc[src];
    }
    gt_before += tg;
    eq_before += te;
    __syncthreads();
  }
}

// ---------------------------------------------------------------------------
// Register-resident variant for Lb <= 1024 * KPT (up to 32 keys per thread
// stay in registers without spills; with KPT = 64 the other 32 are staged in
// LDS, 128 KiB, index-major so that a wave's reads are conflict-free; longer
// local blocks use the kernel above).  1024 threads; thread t holds the keys
// of local indices KPT*t .. KPT*t + KPT-1, loaded once with 16-byte vector
// loads.  The radix select takes three digits of 11, 11 and 10 bits, each
// counted into one shared 2048-bin histogram (wider digits spread the keys
// of one wave's atomics over more addresses and save a pass); the selected
// counts before each thread's range come from a block scan.  Workgroup c of a head then gathers the selected rows whose
// output positions fall in its share [c*lp/S, (c+1)*lp/S).  Same threshold,
// same tie rule, same output as the kernel above.
constexpr int kRegThreads = 1024;
constexpr int kRegWaves = kRegThreads / 64;
constexpr int kSelBins = 2 * kRegThreads;  // 11-bit digits, two bins per thread

// Inclusive prefix sum over the 64 lanes of a wave: shifts inside each
// 16-lane row through DPP, then the three row totals taken by readlane.
__device__ __forceinline__ uint32_t wave_prefix_sum(uint32_t x) {
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x111, 0xf, 0xf, false);  // row_shr:1
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x112, 0xf, 0xf, false);  // row_shr:2
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x114, 0xf, 0xf, false);  // row_shr:4
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x118, 0xf, 0xf, false);  // row_shr:8
  const uint32_t r0 = (uint32_t)__builtin_amdgcn_readlane((int)x, 15);
  const uint32_t r1 = (uint32_t)__builtin_amdgcn_readlane((int)x, 31);
  const uint32_t r2 = (uint32_t)__builtin_amdgcn_readlane((int)x, 47);
  const int row = (threadIdx.x & 63) >> 4;
  return x + (row >= 1 ? r0 : 0u) + (row >= 2 ? r1 : 0u) + (row >= 3 ? r2 : 0u);
}

template <int KPT>
__global__ void __launch_bounds__(kRegThreads)
topk_gather_reg_kernel(const float* __restrict__ scores, const uint16_t* __restrict__ k,
                       const uint16_t* __restrict__ v, int32_t* __restrict__ out_idx,
                       uint16_t* __restrict__ out_k, uint16_t* __restrict__ out_v, int La,
                       int Lb, int lp, int head_dim, int share) {
  constexpr int KREG = KPT < 32 ? KPT : 32;  // keys per thread in registers
  constexpr int KLDS = KPT - KREG;           // keys per thread in LDS
  __shared__ uint32_t hist[kSelBins];
  __shared__ uint32_t wtot[kRegWaves];
  __shared__ uint32_t wsum_gt[kRegWaves], wsum_eq[kRegWaves];
  __shared__ uint32_t sel_digit, sel_above;
  __shared__ int32_t list_src[1024];
  __shared__ uint32_t lds_key[KLDS > 0 ? KLDS * kRegThreads : 1];  // [j - KREG][thread]

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int head = blockIdx.y;
  const float* s = scores + (size_t)head * Lb;
  const int i0 = KPT * tid;

  // ---- keys in registers (and LDS); indices past Lb are marked invalid
  uint32_t key[KREG];
  auto put = [&](int j, uint32_t kv) __attribute__((always_inline)) {
    if (j < KREG) key[j] = kv;
    else lds_key[(j - KREG) * kRegThreads + tid] = kv;
  };
  if (i0 + KPT <= Lb && ((uintptr_t)s & 15u) == 0) {
#pragma unroll
    for (int j = 0; j < KPT; j += 4) {
      const float4 f = *reinterpret_cast<const float4*>(s + i0 + j);
      put(j, score_key(f.x)); put(j + 1, score_key(f.y));
      put(j + 2, score_key(f.z)); put(j + 3, score_key(f.w));
    }
  } else {
#pragma unroll
    for (int j = 0; j < KPT; ++j) put(j, i0 + j < Lb ? score_key(s[i0 + j]) : 0u);
  }
  // key j of this thread (each thread reads back only its own LDS slots)
  auto get = [&](int j) __attribute__((always_inline)) -> uint32_t {
    return j < KREG ? key[j] : lds_key[(j - KREG) * kRegThreads + tid];
  };
  const int n_valid = max(0, min(KPT, Lb - i0));

  // every share slot is filled below (exactly lp distinct positions are
  // selected); -1 marks a slot as empty for the gather regardless
  list_src[tid] = -1;

  // ---- 1. radix select: key T of the lp-th largest score and `need`
  // three digits of 11, 11 and 10 bits into one shared 2048-bin histogram;
  // thread t owns bins 2t and 2t+1, reads and clears them after the counts
  for (int b = tid; b < kSelBins; b += kRegThreads) hist[b] = 0u;
  __syncthreads();
  uint32_t prefix = 0u, prefix_mask = 0u, remaining = (uint32_t)lp;
#pragma unroll
  for (int pass = 0; pass < 3; ++pass) {
    const int shift = pass == 0 ? 21 : (pass == 1 ? 10 : 0);
    const uint32_t dmask = pass == 2 ? 1023u : 2047u;
#pragma unroll
    for (int j = 0; j < KPT; ++j) {
      const uint32_t kj = get(j);
      if (j < n_valid && (kj & prefix_mask) == prefix) atomicAdd(&hist[(kj >> shift) & dmask], 1u);
    }
    __syncthreads();
    const uint32_t c0 = hist[2 * tid], c1 = hist[2 * tid + 1];
    hist[2 * tid] = 0u;
    hist[2 * tid + 1] = 0u;
    const uint32_t own = c0 + c1;
    const uint32_t pre = wave_prefix_sum(own);  // bins of the lanes <= lane
    const uint32_t wt = (uint32_t)__builtin_amdgcn_readlane((int)pre, 63);
    uint32_t incl = wt - pre + own;  // inclusive suffix sum over the lanes >= lane
    if (lane == 0) wtot[wave] = wt;
    __syncthreads();
#pragma unroll
    for (int w = 1; w < kRegWaves; ++w) incl += w > wave ? wtot[w] : 0u;
    const uint32_t above_t = incl - own;  // keys in the bins above 2t+1
    if (above_t < remaining && remaining <= incl) {
      if (remaining <= above_t + c1) {
        sel_digit = (uint32_t)(2 * tid + 1);
        sel_above = above_t;
      } else {
        sel_digit = (uint32_t)(2 * tid);
        sel_above = above_t + c1;
      }
    }
    __syncthreads();
    prefix |= sel_digit << shift;
    prefix_mask |= dmask << shift;
    remaining -= sel_above;
  }
  const uint32_t T = prefix;
  const uint32_t need = remaining;

  // ---- 2. counts above / equal to T before this thread's range (block scan)
  uint32_t n_gt = 0u, n_eq = 0u;
#pragma unroll
  for (int j = 0; j < KPT; ++j) {
    const uint32_t kj = get(j);
    n_gt += (j < n_valid && kj > T) ? 1u : 0u;
    n_eq += (j < n_valid && kj == T) ? 1u : 0u;
  }
  const uint32_t x_gt = wave_prefix_sum(n_gt), x_eq = wave_prefix_sum(n_eq);  // inclusive
  if (lane == 63) { wsum_gt[wave] = x_gt; wsum_eq[wave] = x_eq; }
  __syncthreads();
  uint32_t gt_before = x_gt - n_gt, eq_before = x_eq - n_eq;
#pragma unroll
  for (int w = 0; w < kRegWaves - 1; ++w) {
    gt_before += w < wave ? wsum_gt[w] : 0u;
    eq_before += w < wave ? wsum_eq[w] : 0u;
  }

  // ---- 3. this workgroup's share of output positions: its list in LDS
  const int p0 = blockIdx.x * share, p1 = min(lp, p0 + share);
#pragma unroll
  for (int j = 0; j < KPT; ++j) {
    const uint32_t kj = get(j);
    const bool gt = j < n_valid && kj > T;
    const bool eq = j < n_valid && kj == T;
    const uint32_t pos = gt_before + min(eq_before, need);
    const bool sel = gt || (eq && eq_before < need);
    if (sel && (int)pos >= p0 && (int)pos < p1) {
      list_src[pos - p0] = i0 + j;
      if (out_idx) out_idx[(size_t)head * lp + pos] = i0 + j;
    }
    gt_before += gt ? 1u : 0u;
    eq_before += eq ? 1u : 0u;
  }
  __syncthreads();

  // ---- 4. gather the share's rows with 16-byte copies
  const int row_chunks = head_dim / 8;
  const size_t M = (size_t)La + Lb;
  const uint4* ksrc = reinterpret_cast<const uint4*>(k + (size_t)head * M * head_dim);
  const uint4* vsrc = reinterpret_cast<const uint4*>(v + (size_t)head * M * head_dim);
  uint4* kdst = reinterpret_cast<uint4*>(out_k + (size_t)head * lp * head_dim);
  uint4* vdst = reinterpret_cast<uint4*>(out_v + (size_t)head * lp * head_dim);
  const int pieces = (p1 - p0) * row_chunks;
  for (int e = tid; e < 2 * pieces; e += kRegThreads) {
    const int which = e >= pieces;  // 0: K, 1: V
    const int ee = e - which * pieces;
    const int r = ee / row_chunks, ch = ee - r * row_chunks;
    const int li = list_src[r];
    if (li < 0 || li >= Lb) continue;
    const size_t src = ((size_t)La + li) * row_chunks + ch;
    const size_t dst = (size_t)(p0 + r) * row_chunks + ch;
    if (which) vdst[dst] = vsrc[src];
    else kdst[dst] = ksrc[src];
  }
}

}  // namespace

hipError_t launch_compress(const CompressArgs& a, hipStream_t stream) {
  if (a.lp == 0) return hipSuccess;
  if (a.Lb <= kRegThreads * 64) {
    // a share of at most 1024 output rows per workgroup, about 64 rows each
    // for the gather, at most 32 workgroups per head
    int groups = (a.lp + 63) / 64;
    groups = groups < 1 ? 1 : (groups > 32 ? 32 : groups);
    int share = (a.lp + groups - 1) / groups;
    if (share > 1024) {
      share = 1024;
      groups = (a.lp + share - 1) / share;
    }
    const dim3 grid(groups, a.n_kv);
    if (a.Lb <= kRegThreads * 4)
      hipLaunchKernelGGL(topk_gather_reg_kernel<4>, grid, dim3(kRegThreads), 0, stream, a.scores,
                         a.k, a.v, a.idx, a.out_k, a.out_v, a.La, a.Lb, a.lp, a.head_dim, share);
    else if (a.Lb <= kRegThreads * 16)
      hipLaunchKernelGGL(topk_gather_reg_kernel<16>, grid, dim3(kRegThreads), 0, stream, a.scores,
                         a.k, a.v, a.idx, a.out_k, a.out_v, a.La, a.Lb, a.lp, a.head_dim, share);
    else if (a.Lb <= kRegThreads * 32)
      hipLaunchKernelGGL(topk_gather_reg_kernel<32>, grid, dim3(kRegThreads), 0, stream, a.scores,
                         a.k, a.v, a.idx, a.out_k, a.out_v, a.La, a.Lb, a.lp, a.head_dim, share);
    else
      hipLaunchKernelGGL(topk_gather_reg_kernel<64>, grid, dim3(kRegThreads), 0, stream, a.scores,
                         a.k, a.v, a.idx, a.out_k, a.out_v, a.La, a.Lb, a.lp, a.head_dim, share);
    return hipGetLastError();
  }
  // Enough workgroups per head to spread the gather over the chip, each
  // owning at least 1024 local indices.
  int splits = a.Lb / 1024;
  splits = splits < 1 ? 1 : (splits > 32 ? 32 : splits);
  const int chunk = (a.Lb + splits - 1) / splits;
  dim3 grid(splits, a.n_kv);
  hipLaunchKernelGGL(topk_gather_kernel, grid, dim3(kThreads), 0, stream, a.scores, a.k, a.v,
                     a.idx, a.out_k, a.out_v, a.La, a.Lb, a.lp, a.head_dim, chunk);
  return hipGetLastError();
}

}  // namespace apb
