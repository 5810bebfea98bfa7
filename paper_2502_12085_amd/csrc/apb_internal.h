// Internal launch interface between the C-ABI layer (apb_api.hip) and the
// gfx950 kernels (apb_attention.hip, apb_compress.hip).  Not installed.
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

hipError_t launch_attention(const AttnArgs& a, hipStream_t stream);
hipError_t launch_compress(const CompressArgs& a, hipStream_t stream);

}  // namespace apb

#endif  // APB_INTERNAL_H_
