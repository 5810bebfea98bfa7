// Internal launch interface between the C-ABI layer (apb_api.hip) and the
// gfx950 kernels (apb_attention.hip, apb_compress.hip, apb_decode.hip,
// apb_scorer.hip, apb_layer.hip).
// Not installed.
#ifndef APB_INTERNAL_H_
#define APB_INTERNAL_H_

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace apb {

// One host share, already validated.  Row counts are the paper's:
// La anchor rows, Lb local rows, lp rows per earlier host, Lp = host_idx*lp.
struct AttnArgs {
  const uint16_t* q;
  const uint16_t* k;
  const uint16_t* v;
  const uint16_t* kp;  // [host_idx][n_kv][lp][d], may be null when Lp == 0
  const uint16_t* vp;
  uint16_t* o;
  float* lse;          // may be null
  int32_t La, Lb, lp, Lp;
  int32_t n_q, n_kv, head_dim;
  float scale_log2;    // softmax scale * log2(e)
};

struct CompressArgs {
  const float* scores;
  const uint16_t* k;
  const uint16_t* v;
  int32_t* idx;        // may be null
  uint16_t* out_k;
  uint16_t* out_v;
  int32_t La, Lb, lp;
  int32_t n_kv, head_dim;
};

// One host's decoding-stage attention (Alg. 3), already validated.
struct DecodeArgs {
  const uint16_t* q;   // [n_q][n_new][d]
  const uint16_t* kc;  // [n_kv][Lc][d], may be null when Lc == 0
  const uint16_t* vc;
  const uint16_t* kn;  // [n_kv][n_new][d], used when append
  const uint16_t* vn;
  float* o;            // [n_q][n_new][d]
  float* lse;          // [n_q][n_new]
  float* workspace;    // DecodePlan::workspace_bytes, 16-byte aligned
  int32_t Lc, n_new, append;
  int32_t n_q, n_kv, head_dim;
  float scale_log2;
};

// How a decode call splits its keys; the workspace holds one partial per
// split and row: fp32 O and LSE (one-wave workgroups), or fp16 O with a
// per-row power-of-two scale and the LSE (eight-wave workgroups).
struct DecodePlan {
  int n_split;
  int blocks_per_split;
  int row_blocks;      // workgroups along the rows (each waves * 32 rows)
  int waves;           // waves per workgroup sharing one K/V ring (1 or 8)
  uint64_t workspace_bytes;
};

struct MergeArgs {
  const float* o_parts;    // [n_parts][rows][d]
  const float* lse_parts;  // [n_parts][rows]
  uint16_t* o;             // [rows][d] bf16
  float* lse;              // [rows], may be null
  int32_t n_parts, rows, head_dim;
};

// Retaining-head scores of one host's local block, already validated.
struct ScorerArgs {
  const uint16_t* q;   // [n_q][La+Lb][d]
  const uint16_t* k;   // [n_kv][La+Lb][d]
  const uint16_t* v;
  const uint16_t* w1;  // [hidden][(n_q + 2 n_kv) d] bf16
  const float* b1;     // [hidden]
  const float* w2;     // [n_kv][hidden]
  const float* b2;     // [n_kv]
  float* scores;       // [n_kv][Lb]
  float* workspace;    // scorer_workspace_bytes()
  int32_t La, Lb, n_q, n_kv, head_dim, hidden;
};

// One host's whole layer (Alg. 2 with the model's layer), already validated.
struct LayerArgs {
  const uint16_t* hidden;    // [T][D], T = La + Lb
  const int32_t* pos;        // [T]
  const uint16_t* ln1;       // [D]
  const uint16_t* w_qkv;     // [(n_q + 2 n_kv) d][D]
  const uint16_t* w_o;       // [D][n_q d]
  const uint16_t* ln2;       // [D]
  const uint16_t* w_gate;    // [I][D]
  const uint16_t* w_up;      // [I][D]
  const uint16_t* w_down;    // [D][I]
  const uint16_t* r_w1;      // retaining head, as ScorerArgs
  const float* r_b1;
  const float* r_w2;
  const float* r_b2;
  uint16_t* k_cache;         // out [n_kv][T][d] (post-RoPE)
  uint16_t* v_cache;         // out [n_kv][T][d]
  uint16_t* pass_k;          // [H][n_kv][lp][d]: slots < host_idx read, slot host_idx written
  uint16_t* pass_v;
  uint16_t* hidden_out;      // out [T][D]
  void* workspace;           // layer_workspace_bytes()
  int32_t host_idx, La, Lb, lp;
  int32_t n_q, n_kv, head_dim, D, I, scorer_hidden;
  float eps, theta;
};

hipError_t launch_attention(const AttnArgs& a, hipStream_t stream);
int attention_tile_rows();   // query rows per attention workgroup (one grid entry each)
hipError_t launch_compress(const CompressArgs& a, hipStream_t stream);
// max_workspace_bytes caps the splits; a plan with n_split == 0 does not fit.
DecodePlan plan_decode(const DecodeArgs& a, uint64_t max_workspace_bytes = ~0ull);
hipError_t launch_decode(const DecodeArgs& a, const DecodePlan& pl, hipStream_t stream);
// The no-allocation decode call's device scratch on the current device (its
// address, looked up once per device), kDecodeScratchBytes long.
constexpr uint64_t kDecodeScratchBytes = uint64_t(16) << 20;
hipError_t decode_scratch(void** ptr);
hipError_t launch_merge(const MergeArgs& a, hipStream_t stream);
uint64_t scorer_workspace_bytes(const ScorerArgs& a);
hipError_t launch_scorer(const ScorerArgs& a, hipStream_t stream);
int scorer_hidden_block();  // hidden must be a multiple of this
int scorer_max_kv();        // largest n_kv the fused second layer takes
uint64_t layer_workspace_bytes(const LayerArgs& a);
hipError_t launch_layer(const LayerArgs& a, hipStream_t stream);

}  // namespace apb

#endif  // APB_INTERNAL_H_
