// One host's whole APB layer (Alg. 2 with the model's layer around the
// attention) for gfx950: RMSNorm, the QKV projection, RoPE, the retaining
// head, top-l_p selection and gather, the modified-mask attention, the O
// projection with its residual, RMSNorm, and the SwiGLU FFN with its
// residual.  The retaining head, the compressor and the attention are the
// library's own kernels; this file adds the layer's norms, rotary embedding
// and matrix products, and sequences the whole layer on one stream.
//
// Matrix products: the GEMM kernel template of apb_gemm.h.
#include <math.h>

#include <type_traits>

#include "apb_gemm.h"
#include "apb_internal.h"

namespace apb {
namespace {

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
