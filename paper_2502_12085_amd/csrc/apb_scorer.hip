// Retaining-head scorer R of one APB host (Sec. 3.4; Alg. 2, compression
// step; App. B) for gfx950, with synthetic weights:
//   x_t = [Q_0[t] .. Q_{n_q-1}[t], K_0[t] .. K_{n_kv-1}[t], V_0[t] .. V_{n_kv-1}[t]]
//   s_t = W2 SiLU(W1 x_t + b1) + b2            (one score per KV head)
// for every local token t.  The architecture beyond "small MLP over [Q, K,
// V] with intermediate size 1024" is a reading (two linear layers with
// biases, SiLU between).
//
// Design.  The first layer is a bf16 GEMM H^T = W1 X^T (hidden units on the
// MFMA M side, tokens on the N side, fp32 accumulation) on the library's
// matrix-product kernel (apb_gemm.h): its token operand is read straight
// from the head-major Q/K/V tensors (a 64-feature K step is one head's 64
// dims, so no [tokens x features] matrix is ever built), and its epilogue
// fuses the rest: bias, SiLU, and the workgroup's share of the second layer
// (its 256 hidden units times W2), written as one fp32 partial score per
// hidden block; a small kernel adds the partials and b2 in a fixed order, so
// the scores are deterministic.
#include <math.h>

#include "apb_gemm.h"
#include "apb_internal.h"

namespace apb {
namespace {

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
  return (uint64_t)(a.hidden / kBF) * a.n_kv * a.Lb * 4;
}

hipError_t launch_scorer(const ScorerArgs& a, hipStream_t stream) {
  GemmParams p{};
  p.x = a.q; p.x_k = a.k; p.x_v = a.v;
  p.x_rows = a.La + a.Lb;
  p.x_row0 = a.La;
  p.w = a.w1; p.w_up = a.w1;
  p.T = a.Lb;
  p.K = (a.n_q + 2 * a.n_kv) * a.head_dim;
  p.F = a.hidden;
  p.dh = a.head_dim;
  p.n_q = a.n_q; p.n_kv = a.n_kv;
  p.b1 = a.b1; p.w2 = a.w2; p.part = a.workspace;
  hipError_t e = launch_gemm<kXQkv, kWPlain, kEpiScorer>(p, stream);
  if (e != hipSuccess) return e;
  const size_t total = (size_t)a.n_kv * a.Lb;
  hipLaunchKernelGGL(scorer_reduce_kernel, dim3((unsigned)((total + 255) / 256)), dim3(256), 0,
                     stream, a.workspace, a.b2, a.scores, a.hidden / kBF, a.n_kv, a.Lb);
  return hipGetLastError();
}

int scorer_hidden_block() { return kBF; }
int scorer_max_kv() { return kScorerMaxKv; }

}  // namespace apb
