// Retaining-head scorer R of one APB host (Sec. 3.4; Alg. 2, compression
// step; App. B) for gfx950, with synthetic weights:
//   x_t = [Q_0[t] .. Q_{n_q-1}[t], K_0[t] .. K_{n_kv-1}[t], V_0[t] .. V_{n_kv-1}[t]]
//   s_t = W2 SiLU(W1 x_t + b1) + b2            (one score per KV head)
// for every local token t.  The architecture beyond "small MLP over [Q, K,
// V] with intermediate size 1024" is a reading (two linear layers with
// biases, SiLU between).
//
// Design.  The first layer is a bf16 GEMM H^T = W1 X^T (hidden units on the
// MFMA M side, tokens on the N side, fp32 accumulation) read straight from
// the head-major Q/K/V tensors: a 64-feature slice of x is one head's 64
// dims, so every K step of the GEMM copies a [tokens x 64] slab of one head
// and a [hidden x 64] slab of W1.  Workgroup tile 256 hidden x 256 tokens,
// 8 waves each owning 128 x 64, 32x32x16 bf16 MFMAs, K/V-style XOR-swizzled
// LDS tiles filled by global_load_lds_dwordx4 (two stages, the next K step
// in flight while the current one is multiplied).  The epilogue fuses the
// rest: bias, SiLU, and the workgroup's share of the second layer (its 256
// hidden units times W2), written as one fp32 partial score per hidden
// block; a small kernel adds the partials and b2 in a fixed order, so the
// scores are deterministic.
#include <math.h>

#include "apb_internal.h"

namespace apb {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) bf16x8 lds_bf16x8;

constexpr int kBH = 256;      // hidden units per workgroup (MFMA M side)
constexpr int kBT = 256;      // tokens per workgroup (MFMA N side)
constexpr int kBK = 64;       // features per K step (one head's 64 dims)
constexpr int kWaves = 8;     // 2 (hidden halves) x 4 (token quarters)
constexpr int kThreads = 64 * kWaves;
constexpr int kMaxKv = 8;     // KV heads the fused second layer supports
constexpr int kTile = kBH * kBK;  // bf16 elements per operand tile (= kBT * kBK)

struct ScorerParams {
  const uint16_t* q;
  const uint16_t* k;
  const uint16_t* v;
  const uint16_t* w1;   // [hidden][F]
  const float* b1;      // [hidden]
  const float* w2;      // [n_kv][hidden]
  float* part;          // [hidden / kBH][n_kv][Lb]
  int La, Lb, M;        // M = La + Lb rows of the Q/K/V tensors
  int n_q, n_kv, d, F, hidden;
};

__device__ __forceinline__ uint32_t lds_offset(const void* p) {
  return (uint32_t)(uintptr_t)(__attribute__((address_space(3))) const void*)p;
}

// Tiles are [rows][64] bf16, 128-byte rows; 16-byte chunk c of row r sits at
// chunk c ^ (r & 7), so the 8 rows one ds_read_b128 pass touches hit 8
// different chunk slots.
__device__ __forceinline__ int swz(int r) { return r & 7; }

__global__ void __launch_bounds__(kThreads, 1) scorer_gemm_kernel(ScorerParams p) {
  __shared__ __attribute__((aligned(16))) uint16_t a_lds[2][kTile];  // W1 slab
  __shared__ __attribute__((aligned(16))) uint16_t b_lds[2][kTile];  // token slab

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave & 1, wn = wave >> 1;  // hidden half, token quarter
  const int n = lane & 31, h = lane >> 5;
  const int hb = blockIdx.y;                 // hidden block
  const int t0 = blockIdx.x * kBT;           // first token of the tile
  const int n0 = hb * kBH;                   // first hidden unit
  const int nk = p.F / kBK;

  // ---- copies: piece j of a tile = 8 rows x 128 bytes; wave w copies
  // pieces 4w .. 4w+3 of the W1 tile and of the token tile.  Lane l takes
  // row l/8 of the piece and fetches the chunk that belongs at slot l%8.
  const int cp_row = lane >> 3, cp_slot = lane & 7;
  const uint32_t w_lane = (uint32_t)(cp_row * 2 * p.F + 16 * (cp_slot ^ cp_row));
  const uint32_t x_lane = (uint32_t)(cp_row * 2 * p.d + 16 * (cp_slot ^ cp_row));
  const bool full_tile = t0 + kBT <= p.Lb;
  auto issue = [&](int kk, int st) __attribute__((always_inline)) {
    const int f0 = kk * kBK;
    const int head = f0 / p.d, j0 = f0 - head * p.d;
    const uint16_t* src;
    int hh;
    if (head < p.n_q) { src = p.q; hh = head; }
    else if (head < p.n_q + p.n_kv) { src = p.k; hh = head - p.n_q; }
    else { src = p.v; hh = head - p.n_q - p.n_kv; }
    // tokens La + t0 .. of head hh, dims j0 .. j0+63
    const uint16_t* xbase = src + ((size_t)hh * p.M + p.La + t0) * p.d + j0;
    const uint16_t* wbase = p.w1 + (size_t)n0 * p.F + f0;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int j = 4 * wave + i;  // piece: rows 8j .. 8j+7
      const uint32_t wd = __builtin_amdgcn_readfirstlane(lds_offset(&a_lds[st][j * 512]));
      const uint32_t xd = __builtin_amdgcn_readfirstlane(lds_offset(&b_lds[st][j * 512]));
      const uint16_t* wb = wbase + (size_t)(8 * j) * p.F;
      asm volatile("s_mov_b32 m0, %2\n\tglobal_load_lds_dwordx4 %0, %1" ::"v"(w_lane), "s"(wb),
                   "s"(wd)
                   : "memory");
      if (full_tile) {
        const uint16_t* xb = xbase + (size_t)(8 * j) * p.d;
        asm volatile("s_mov_b32 m0, %2\n\tglobal_load_lds_dwordx4 %0, %1" ::"v"(x_lane),
                     "s"(xb), "s"(xd)
                     : "memory");
      } else {
        // ragged last tile: rows past the last token repeat it
        const int row = 8 * j + cp_row;
        const int t = min(t0 + row, p.Lb - 1) - t0;
        const uint16_t* xs = xbase + (size_t)t * p.d + 8 * (cp_slot ^ swz(row));
        asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dwordx4 %0, off" ::"v"(xs), "s"(xd)
                     : "memory");
      }
    }
  };

  // ---- operands: lane (n, h) of an MFMA block reads row 32*blk + n,
  // features 16*kc + 8*h .. +7, i.e. chunk 2*kc + h of that row
  auto a_read = [&](int st, int mb, int kc) __attribute__((always_inline)) -> bf16x8 {
    const int row = 128 * wm + 32 * mb + n;
    return *(const lds_bf16x8*)(uintptr_t)(lds_offset(a_lds[st]) + row * 128 +
                                            16 * ((2 * kc + h) ^ swz(row)));
  };
  auto b_read = [&](int st, int nb, int kc) __attribute__((always_inline)) -> bf16x8 {
    const int row = 64 * wn + 32 * nb + n;
    return *(const lds_bf16x8*)(uintptr_t)(lds_offset(b_lds[st]) + row * 128 +
                                            16 * ((2 * kc + h) ^ swz(row)));
  };

  f32x16 acc[4][2];
#pragma unroll
  for (int mb = 0; mb < 4; ++mb)
#pragma unroll
    for (int nb = 0; nb < 2; ++nb)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[mb][nb][r] = 0.f;

  issue(0, 0);
  for (int kk = 0; kk < nk; ++kk) {
    const int st = kk & 1;
    // this wave's copies of step kk have landed; after the barrier every
    // wave's have, and every wave is done reading the other stage
    asm volatile("s_waitcnt vmcnt(0)\n\ts_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
    if (kk + 1 < nk) issue(kk + 1, st ^ 1);
    bf16x8 av[2][4], bv[2][2];
#pragma unroll
    for (int mb = 0; mb < 4; ++mb) av[0][mb] = a_read(st, mb, 0);
#pragma unroll
    for (int nb = 0; nb < 2; ++nb) bv[0][nb] = b_read(st, nb, 0);
#pragma unroll
    for (int kc = 0; kc < 4; ++kc) {
      const int cur = kc & 1;
      if (kc + 1 < 4) {
#pragma unroll
        for (int mb = 0; mb < 4; ++mb) av[cur ^ 1][mb] = a_read(st, mb, kc + 1);
#pragma unroll
        for (int nb = 0; nb < 2; ++nb) bv[cur ^ 1][nb] = b_read(st, nb, kc + 1);
      }
#pragma unroll
      for (int mb = 0; mb < 4; ++mb)
#pragma unroll
        for (int nb = 0; nb < 2; ++nb)
          acc[mb][nb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av[cur][mb], bv[cur][nb],
                                                                acc[mb][nb], 0, 0, 0);
      __builtin_amdgcn_sched_barrier(0);
    }
  }

  // ---- epilogue: bias, SiLU, and this block's share of the second layer.
  // Lane (n, h), block (mb, nb), element r holds hidden unit
  // n0 + 128*wm + 32*mb + 8*(r/4) + 4*h + r%4 of token t0 + 64*wn + 32*nb + n.
  __syncthreads();  // the LDS stages are reused below
  float* w2_lds = reinterpret_cast<float*>(&a_lds[0][0]);     // [kBH][kMaxKv]
  float* b1_lds = w2_lds + kBH * kMaxKv;                        // [kBH]
  float* red = reinterpret_cast<float*>(&b_lds[0][0]);          // [2][kMaxKv][kBT]
  for (int i = tid; i < kBH * kMaxKv; i += kThreads) {
    const int u = i / kMaxKv, kv = i % kMaxKv;
    w2_lds[i] = kv < p.n_kv ? p.w2[(size_t)kv * p.hidden + n0 + u] : 0.f;
  }
  for (int i = tid; i < kBH; i += kThreads) b1_lds[i] = p.b1[n0 + i];
  __syncthreads();
  float part[2][kMaxKv];
#pragma unroll
  for (int nb = 0; nb < 2; ++nb)
#pragma unroll
    for (int kv = 0; kv < kMaxKv; ++kv) part[nb][kv] = 0.f;
#pragma unroll
  for (int mb = 0; mb < 4; ++mb)
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int u = 128 * wm + 32 * mb + 8 * (r >> 2) + 4 * h + (r & 3);
      const f32x4 wa = *reinterpret_cast<const f32x4*>(&w2_lds[u * kMaxKv]);
      const f32x4 wb = *reinterpret_cast<const f32x4*>(&w2_lds[u * kMaxKv + 4]);
      const float bias = b1_lds[u];
#pragma unroll
      for (int nb = 0; nb < 2; ++nb) {
        const float z = acc[mb][nb][r] + bias;
        const float a = z / (1.f + __expf(-z));
#pragma unroll
        for (int kv = 0; kv < 4; ++kv) {
          part[nb][kv] = fmaf(a, wa[kv], part[nb][kv]);
          part[nb][4 + kv] = fmaf(a, wb[kv], part[nb][4 + kv]);
        }
      }
    }
  // the two lane halves hold the same tokens' other hidden units
#pragma unroll
  for (int nb = 0; nb < 2; ++nb)
#pragma unroll
    for (int kv = 0; kv < kMaxKv; ++kv) {
      const float x = part[nb][kv];
      const auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x),
                                                       false, false);
      part[nb][kv] = x + __uint_as_float(h ? sw[0] : sw[1]);
    }
  // the two hidden halves (wm = 0, 1) of each token quarter meet in LDS
  if (h == 0) {
#pragma unroll
    for (int nb = 0; nb < 2; ++nb)
#pragma unroll
      for (int kv = 0; kv < kMaxKv; ++kv)
        red[(wm * kMaxKv + kv) * kBT + 64 * wn + 32 * nb + n] = part[nb][kv];
  }
  __syncthreads();
  for (int i = tid; i < kMaxKv * kBT; i += kThreads) {
    const int kv = i / kBT, tl = i % kBT;
    const int t = t0 + tl;
    if (kv < p.n_kv && t < p.Lb)
      p.part[((size_t)hb * p.n_kv + kv) * p.Lb + t] = red[kv * kBT + tl] + red[(kMaxKv + kv) * kBT + tl];
  }
}

// scores[kv][t] = b2[kv] + sum over hidden blocks, in block order
__global__ void __launch_bounds__(256) scorer_reduce_kernel(const float* __restrict__ part,
                                                            const float* __restrict__ b2,
                                                            float* __restrict__ scores, int nblk,
                                                            int n_kv, int Lb) {
  const size_t i = (size_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= (size_t)n_kv * Lb) return;
  const int kv = (int)(i / Lb);
  float s = 0.f;
  for (int b = 0; b < nblk; ++b) s += part[(size_t)b * n_kv * Lb + i];
  scores[i] = s + b2[kv];
}

}  // namespace

uint64_t scorer_workspace_bytes(const ScorerArgs& a) {
  return (uint64_t)(a.hidden / kBH) * a.n_kv * a.Lb * 4;
}

hipError_t launch_scorer(const ScorerArgs& a, hipStream_t stream) {
  ScorerParams p;
  p.q = a.q; p.k = a.k; p.v = a.v; p.w1 = a.w1; p.b1 = a.b1; p.w2 = a.w2;
  p.part = a.workspace;
  p.La = a.La; p.Lb = a.Lb; p.M = a.La + a.Lb;
  p.n_q = a.n_q; p.n_kv = a.n_kv; p.d = a.head_dim;
  p.F = (a.n_q + 2 * a.n_kv) * a.head_dim;
  p.hidden = a.hidden;
  const dim3 grid((unsigned)((a.Lb + kBT - 1) / kBT), (unsigned)(a.hidden / kBH));
  hipLaunchKernelGGL(scorer_gemm_kernel, grid, dim3(kThreads), 0, stream, p);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const size_t total = (size_t)a.n_kv * a.Lb;
  hipLaunchKernelGGL(scorer_reduce_kernel, dim3((unsigned)((total + 255) / 256)), dim3(256), 0,
                     stream, a.workspace, a.b2, a.scores, a.hidden / kBH, a.n_kv, a.Lb);
  return hipGetLastError();
}

int scorer_hidden_block() { return kBH; }
int scorer_max_kv() { return kMaxKv; }

}  // namespace apb
