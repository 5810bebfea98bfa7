// One host's whole APB layer (Alg. 2 with the model's layer around the
// attention) for gfx950: RMSNorm, the QKV projection, RoPE, the retaining
// head, top-l_p selection and gather, the modified-mask attention, the O
// projection with its residual, RMSNorm, and the SwiGLU FFN with its
// residual.  The retaining head, the compressor and the attention are the
// library's own kernels; this file adds the layer's norms, rotary embedding
// and matrix products, and sequences the whole layer on one stream.
//
// Matrix products.  Every projection is out[t][f] = sum_k x[t][k] W[f][k]
// (tokens t, output features f, weights row-major [f][k]).  One kernel
// template covers them: bf16 MFMA 16x16x32 with fp32 accumulation, output
// features on the MFMA M side (the weights are the A operand) and tokens on
// the N side, a 256 x 256 workgroup tile of 4 waves (2 x 2, each 128
// features x 128 tokens in 64 16 x 16 blocks, one wave per SIMD,
// accumulators in AGPRs), K steps of 64 whose weight and token slabs are
// copied HBM -> LDS by global_load_lds_dwordx4 into XOR-swizzled tiles in
// two stages.  (16x16x32 rather than 32x32x16: the same LDS bytes per flop
// and half the accumulator traffic, which this power-limited chip turns
// into clock.)  Neither a
// copy nor an operand read spends a vector instruction on its address: a
// copy is a scalar base plus a fixed per-lane offset, a read one XOR of a
// per-lane base plus an instruction offset.  The step
// boundary is software-pipelined: at its last 32-deep substep a wave waits
// for its copies of the next step, passes the barrier, and issues that
// substep's MFMAs with the next step's first operand reads and the copies of
// the step after it (into the stage just finished) spread among them; the
// last two steps are peeled so the steady-state loop has no branches (the
// compiler can then count outstanding LDS reads exactly).
// The token operand is read either row-major [t][k] or head-major
// [k / dh][t][dh] (the attention output, whose heads are the O projection's
// K dimension), so no transpose is ever materialised.  Epilogues:
//  * row-major bf16 store, plus a residual in fp32 before the rounding;
//  * head-major Q/K/V store of the QKV projection (feature f is dim f % dh
//    of head f / dh: Q heads, then K heads, then V heads);
//  * SwiGLU: each wave's 128 weight rows are 64 gate rows and the 64 up
//    rows of the same features, so gate and up of one feature sit in the
//    same lane and register slot and SiLU(gate) * up is formed in registers.
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

enum XMode { kXRowMajor = 0, kXHeadMajor = 1 };
enum WMode { kWPlain = 0, kWGateUp = 1 };
enum Epi { kEpiRowMajor = 0, kEpiQkv = 1, kEpiSwiglu = 2 };

struct GemmParams {
  const uint16_t* x;      // tokens: [T][K] or [K / dh][T][dh]
  const uint16_t* w;      // [F][K]; the gate matrix for kWGateUp
  const uint16_t* w_up;   // [F][K] for kWGateUp
  const uint16_t* resid;  // [T][F] or null (kEpiRowMajor)
  uint16_t* out;          // [T][F] (kEpiRowMajor, kEpiSwiglu); Q for kEpiQkv
  uint16_t* out_k;        // kEpiQkv: K [n_kv][T][dh]
  uint16_t* out_v;        // kEpiQkv: V [n_kv][T][dh]
  int T, K, F;            // F: output features (I for kWGateUp)
  int dh;                 // head dim of a head-major operand or output
  int n_q, n_kv;          // kEpiQkv
};

__device__ __forceinline__ uint32_t lds_offset(const void* p) {
  return (uint32_t)(uintptr_t)(__attribute__((address_space(3))) const void*)p;
}

// 16-byte chunk c of tile row r (128 bytes) sits at chunk c ^ ((r >> 1) & 7):
// any 16 consecutive rows, which one 16-lane pass of ds_read_b128 touches,
// land on 16 distinct 16-byte slots of the 256 bank bytes.
__device__ __forceinline__ int swz(int r) { return (r >> 1) & 7; }

template <int XM, int WM, int EPI>
__global__ void __launch_bounds__(kGemmThreads, 1) gemm_kernel(GemmParams p) {
  __shared__ __attribute__((aligned(16))) uint16_t a_lds[2][kTileElems];  // weight slab
  __shared__ __attribute__((aligned(16))) uint16_t b_lds[2][kTileElems];  // token slab

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave & 1, wn = wave >> 1;  // feature half, token half
  const int n = lane & 31, h = lane >> 5;
  const int t0 = blockIdx.x * kBT;
  const int f0 = blockIdx.y * (WM == kWGateUp ? kBF / 2 : kBF);
  const int nk = p.K / kBK;

  // ---- copies: piece j (8 rows x 128 bytes) of each slab; wave w copies
  // pieces 8w .. 8w+7.  Lane l takes row l/8 of the piece and fetches the
  // chunk that belongs at slot l%8.  Rows past the last feature or token
  // repeat it (their results are never stored).  A copy is a scalar base (the
  // operand's first row for this workgroup, advanced by the K step in scalar
  // registers) plus a fixed per-lane byte offset: no vector instruction.
  const int cp_row = lane >> 3, cp_slot = lane & 7;
  const int x_ld = XM == kXHeadMajor ? p.dh : p.K;  // elements between token rows
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
      // head-major tokens: K element k0 is column k0 % dh of head k0 / dh
      const size_t xoff = XM == kXHeadMajor ? (size_t)(k0 / p.dh) * p.T * p.dh + (k0 % p.dh) : (size_t)k0;
      const uint16_t* base = x_first + xoff;
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
  // barrier, read its first operands); COPY: step kk+2 exists (its 16
  // copies, into the stage this step used, ride on every fourth MFMA of the
  // last substep: issued back to back they stall the wave, and the matrix
  // core with it, for hundreds of cycles).
  auto step = [&](int kk, auto next_t, auto copy_t) __attribute__((always_inline)) {
    constexpr bool NEXT = decltype(next_t)::value, COPY = decltype(copy_t)::value;
    const int st = kk & 1;
    const uint32_t ab = a_base(st), bb = b_base(st), ab1 = a_base(st ^ 1), bb1 = b_base(st ^ 1);
#pragma unroll
    for (int kc = 0; kc < 2; ++kc) {
      const int cur = kc, nxt = kc ^ 1;
      const bool boundary = kc == 1;
      if (boundary && NEXT) {
        // this wave's copies of step kk+1 have landed and its reads of stage
        // st are done; after the barrier every wave's are
        asm volatile("s_waitcnt vmcnt(0)\n\ts_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
      }
#pragma unroll
      for (int i = 0; i < 64; ++i) {
        const int mb = i >> 3, nb = i & 7;
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
        if (boundary && COPY && ((i & 3) == 0)) copy(kk + 2, st, i >> 2);
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
          o[i] = (__bf16)(gt / (1.f + __expf(-gt)) * up);
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

// RMSNorm of one row per workgroup: out = in / sqrt(mean(in^2) + eps) * gain,
// fp32 arithmetic, bf16 in and out.  D % 8 == 0.
__global__ void __launch_bounds__(256) rmsnorm_kernel(const uint16_t* __restrict__ in,
                                                      const uint16_t* __restrict__ gain,
                                                      uint16_t* __restrict__ out, int D,
                                                      float eps) {
  __shared__ float red[4];
  const int tid = threadIdx.x;
  const uint16_t* row = in + (size_t)blockIdx.x * D;
  float ss = 0.f;
  for (int c = 8 * tid; c < D; c += 8 * 256) {
    const bf16x8 x = *reinterpret_cast<const bf16x8*>(row + c);
#pragma unroll
    for (int i = 0; i < 8; ++i) ss += (float)x[i] * (float)x[i];
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) ss += __shfl_xor(ss, off);
  if ((tid & 63) == 0) red[tid >> 6] = ss;
  __syncthreads();
  const float inv = 1.f / sqrtf((red[0] + red[1] + red[2] + red[3]) / (float)D + eps);
  uint16_t* orow = out + (size_t)blockIdx.x * D;
  for (int c = 8 * tid; c < D; c += 8 * 256) {
    const bf16x8 x = *reinterpret_cast<const bf16x8*>(row + c);
    const bf16x8 g = *reinterpret_cast<const bf16x8*>(gain + c);
    bf16x8 y;
#pragma unroll
    for (int i = 0; i < 8; ++i) y[i] = (__bf16)((float)x[i] * inv * (float)g[i]);
    *reinterpret_cast<bf16x8*>(orow + c) = y;
  }
}

// RoPE in place on head-major Q [n_q][T][dh] and K [n_kv][T][dh]: the pair
// (j, j + dh/2) of every head rotated by pos[t] * theta^(-2j/dh).  The angle
// and its cosine and sine are computed in fp64 (positions reach 10^5 and
// beyond, where an fp32 angle would lose its fraction), the rotation in fp32.
// One thread per (token, j); it walks all heads with one cos/sin pair.
__global__ void __launch_bounds__(256) rope_kernel(uint16_t* __restrict__ q,
                                                   uint16_t* __restrict__ k,
                                                   const int32_t* __restrict__ pos, int T,
                                                   int n_q, int n_kv, int dh, double log_theta) {
  const int half = dh / 2;
  const int rows_per_block = 256 / half;
  const int t = blockIdx.x * rows_per_block + threadIdx.x / half;
  const int j = threadIdx.x % half;
  if (t >= T) return;
  const double ang = (double)pos[t] * exp(-2.0 * j / dh * log_theta);
  const float c = (float)cos(ang), s = (float)sin(ang);
  for (int hd = 0; hd < n_q + n_kv; ++hd) {
    uint16_t* base = hd < n_q ? q + ((size_t)hd * T + t) * dh : k + ((size_t)(hd - n_q) * T + t) * dh;
    __bf16* x = reinterpret_cast<__bf16*>(base);
    const float lo = (float)x[j], hi = (float)x[j + half];
    x[j] = (__bf16)(lo * c - hi * s);
    x[j + half] = (__bf16)(hi * c + lo * s);
  }
}

template <int XM, int WM, int EPI>
hipError_t launch_gemm(const GemmParams& p, hipStream_t stream) {
  const int per_wg = WM == kWGateUp ? kBF / 2 : kBF;
  const dim3 grid((unsigned)((p.T + kBT - 1) / kBT), (unsigned)((p.F + per_wg - 1) / per_wg));
  hipLaunchKernelGGL((gemm_kernel<XM, WM, EPI>), grid, dim3(kGemmThreads), 0, stream, p);
  return hipGetLastError();
}

// Workspace carve-up (256-byte aligned pieces).
struct LayerPlan {
  uint64_t x, q, attn, h1, act, scorer, scores, idx, total;
};

uint64_t align256(uint64_t b) { return (b + 255) & ~uint64_t(255); }

LayerPlan plan_layer(const LayerArgs& a) {
  LayerPlan pl;
  const uint64_t T = (uint64_t)a.La + a.Lb;
  uint64_t off = 0;
  auto take = [&](uint64_t bytes) {
    const uint64_t o = off;
    off += align256(bytes);
    return o;
  };
  pl.x = take(T * a.D * 2);
  pl.q = take((uint64_t)a.n_q * T * a.head_dim * 2);
  pl.attn = take((uint64_t)a.n_q * T * a.head_dim * 2);
  pl.h1 = take(T * a.D * 2);
  pl.act = take(T * a.I * 2);
  ScorerArgs sa{};
  sa.La = a.La; sa.Lb = a.Lb; sa.n_q = a.n_q; sa.n_kv = a.n_kv; sa.head_dim = a.head_dim;
  sa.hidden = a.scorer_hidden;
  pl.scorer = take(scorer_workspace_bytes(sa));
  pl.scores = take((uint64_t)a.n_kv * a.Lb * 4);
  pl.idx = take((uint64_t)a.n_kv * (a.lp > 0 ? a.lp : 1) * 4);
  pl.total = off;
  return pl;
}

}  // namespace

uint64_t layer_workspace_bytes(const LayerArgs& a) { return plan_layer(a).total; }

hipError_t launch_layer(const LayerArgs& a, hipStream_t stream) {
  const LayerPlan pl = plan_layer(a);
  uint8_t* ws = static_cast<uint8_t*>(a.workspace);
  uint16_t* x = reinterpret_cast<uint16_t*>(ws + pl.x);
  uint16_t* q = reinterpret_cast<uint16_t*>(ws + pl.q);
  uint16_t* attn = reinterpret_cast<uint16_t*>(ws + pl.attn);
  uint16_t* h1 = reinterpret_cast<uint16_t*>(ws + pl.h1);
  uint16_t* act = reinterpret_cast<uint16_t*>(ws + pl.act);
  float* scores = reinterpret_cast<float*>(ws + pl.scores);
  int32_t* idx = reinterpret_cast<int32_t*>(ws + pl.idx);
  const int T = a.La + a.Lb, d = a.head_dim;
  hipError_t e;

  // 1. x = RMSNorm(H; g1)
  hipLaunchKernelGGL(rmsnorm_kernel, dim3((unsigned)T), dim3(256), 0, stream, a.hidden, a.ln1, x,
                     a.D, a.eps);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  // 2. Q, K, V = x W_qkv^T (head-major), then RoPE on Q and K
  GemmParams g{};
  g.x = x; g.w = a.w_qkv; g.out = q; g.out_k = a.k_cache; g.out_v = a.v_cache;
  g.T = T; g.K = a.D; g.F = (a.n_q + 2 * a.n_kv) * d; g.dh = d; g.n_q = a.n_q; g.n_kv = a.n_kv;
  if ((e = launch_gemm<kXRowMajor, kWPlain, kEpiQkv>(g, stream)) != hipSuccess) return e;
  {
    const int rpb = 256 / (d / 2);
    hipLaunchKernelGGL(rope_kernel, dim3((unsigned)((T + rpb - 1) / rpb)), dim3(256), 0, stream, q,
                       a.k_cache, a.pos, T, a.n_q, a.n_kv, d, log((double)a.theta));
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  // 3. retaining-head scores of the local block, ArgTop-l_p and gather into
  //    this host's slot of the passing buffer
  {
    ScorerArgs sa{};
    sa.q = q; sa.k = a.k_cache; sa.v = a.v_cache; sa.w1 = a.r_w1; sa.b1 = a.r_b1; sa.w2 = a.r_w2;
    sa.b2 = a.r_b2; sa.scores = scores; sa.workspace = reinterpret_cast<float*>(ws + pl.scorer);
    sa.La = a.La; sa.Lb = a.Lb; sa.n_q = a.n_q; sa.n_kv = a.n_kv; sa.head_dim = d;
    sa.hidden = a.scorer_hidden;
    if ((e = launch_scorer(sa, stream)) != hipSuccess) return e;
  }
  if (a.lp > 0) {
    const size_t slot = (size_t)a.host_idx * a.n_kv * a.lp * d;
    CompressArgs ca;
    ca.scores = scores; ca.k = a.k_cache; ca.v = a.v_cache; ca.idx = idx;
    ca.out_k = a.pass_k + slot; ca.out_v = a.pass_v + slot;
    ca.La = a.La; ca.Lb = a.Lb; ca.lp = a.lp; ca.n_kv = a.n_kv; ca.head_dim = d;
    if ((e = launch_compress(ca, stream)) != hipSuccess) return e;
  }
  // 4. attention over [A; P; B] reading the earlier hosts' slots in place
  {
    AttnArgs aa;
    const int Lp = a.host_idx * a.lp;
    aa.q = q; aa.k = a.k_cache; aa.v = a.v_cache;
    aa.kp = Lp > 0 ? a.pass_k : nullptr;
    aa.vp = Lp > 0 ? a.pass_v : nullptr;
    aa.o = attn; aa.lse = nullptr;
    aa.La = a.La; aa.Lb = a.Lb; aa.lp = a.lp; aa.Lp = Lp;
    aa.n_q = a.n_q; aa.n_kv = a.n_kv; aa.head_dim = d;
    aa.scale_log2 = 1.4426950408889634f / sqrtf((float)d);
    if ((e = launch_attention(aa, stream)) != hipSuccess) return e;
  }
  // 5. H1 = H + concat_heads(A) W_o^T
  g = GemmParams{};
  g.x = attn; g.w = a.w_o; g.resid = a.hidden; g.out = h1;
  g.T = T; g.K = a.n_q * d; g.F = a.D; g.dh = d;
  if ((e = launch_gemm<kXHeadMajor, kWPlain, kEpiRowMajor>(g, stream)) != hipSuccess) return e;
  // 6. y = RMSNorm(H1; g2) (into the x buffer)
  hipLaunchKernelGGL(rmsnorm_kernel, dim3((unsigned)T), dim3(256), 0, stream, h1, a.ln2, x, a.D,
                     a.eps);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  // 7. act = SiLU(y W_gate^T) * (y W_up^T)
  g = GemmParams{};
  g.x = x; g.w = a.w_gate; g.w_up = a.w_up; g.out = act; g.T = T; g.K = a.D; g.F = a.I;
  if ((e = launch_gemm<kXRowMajor, kWGateUp, kEpiSwiglu>(g, stream)) != hipSuccess) return e;
  // 8. out = H1 + act W_down^T
  g = GemmParams{};
  g.x = act; g.w = a.w_down; g.resid = h1; g.out = a.hidden_out; g.T = T; g.K = a.I; g.F = a.D;
  return launch_gemm<kXRowMajor, kWPlain, kEpiRowMajor>(g, stream);
}

}  // namespace apb
