// C-ABI layer of the APB host-share library: argument validation (host only,
// before any HIP call), status strings, the FLOP count, and dispatch to the
// gfx950 kernels.
#include <math.h>
#include <stddef.h>
#include <stdint.h>

#include "../../include/apb.h"
#include "apb_internal.h"

static_assert(APB_DECODE_NOALLOC_SCRATCH_BYTES == apb::kDecodeScratchBytes,
              "the header states the scratch size the library holds");

namespace {

thread_local char g_last_error[256] = "";

void set_last_error(hipError_t e) {
  const char* msg = hipGetErrorString(e);
  size_t i = 0;
  for (; msg && msg[i] && i + 1 < sizeof(g_last_error); ++i) g_last_error[i] = msg[i];
  g_last_error[i] = '\0';
}

constexpr int64_t kMaxRows = int64_t(1) << 30;

struct Range {
  uintptr_t lo, hi;  // [lo, hi)
};

Range range_of(const void* ptr, int64_t bytes) {
  const uintptr_t lo = reinterpret_cast<uintptr_t>(ptr);
  return Range{lo, lo + static_cast<uintptr_t>(bytes)};
}

bool overlaps(Range a, Range b) {
  if (a.lo == a.hi || b.lo == b.hi || a.lo == 0 || b.lo == 0) return false;
  return a.lo < b.hi && b.lo < a.hi;
}

bool aligned(const void* ptr, uintptr_t a) { return (reinterpret_cast<uintptr_t>(ptr) % a) == 0; }

}  // namespace

extern "C" {

int apb_abi_version(void) { return APB_ABI_VERSION; }

const char* apb_last_error(void) { return g_last_error; }

const char* apb_status_string(int status) {
  switch (status) {
    case APB_OK: return "ok";
    case APB_ERR_NULL_POINTER: return "a required pointer is NULL";
    case APB_ERR_BAD_SHAPE: return "a size violates the problem constraints";
    case APB_ERR_UNSUPPORTED: return "unsupported configuration (head_dim must be 64 or 128)";
    case APB_ERR_MISALIGNED: return "a pointer is not aligned (bf16: 16 bytes, fp32/int32: 4 bytes)";
    case APB_ERR_HIP: return "the HIP runtime reported an error";
    case APB_ERR_ALIAS: return "an output overlaps an input";
    case APB_ERR_SCRATCH:
      return "the call needs more device scratch than the no-allocation entry point holds "
             "(APB_DECODE_NOALLOC_SCRATCH_BYTES)";
    default: return "unknown status";
  }
}

apb_status_t apb_validate_problem(const apb_problem_t* p) {
  if (!p) return APB_ERR_NULL_POINTER;
  if (p->n_hosts < 1 || p->host_idx < 0 || p->host_idx >= p->n_hosts) return APB_ERR_BAD_SHAPE;
  if (p->anchor_len < 0 || p->local_len < 1) return APB_ERR_BAD_SHAPE;
  if (p->pass_len < 0 || p->pass_len > p->local_len) return APB_ERR_BAD_SHAPE;
  if (p->n_kv_heads < 1 || p->n_q_heads < 1 || p->n_q_heads % p->n_kv_heads != 0)
    return APB_ERR_BAD_SHAPE;
  if (p->head_dim < 1) return APB_ERR_BAD_SHAPE;
  const int64_t rows = (int64_t)p->anchor_len + (int64_t)p->host_idx * p->pass_len +
                       (int64_t)p->local_len;
  if (rows > kMaxRows) return APB_ERR_BAD_SHAPE;
  // Grid size: the attention kernel's query tiles times the query heads must
  // fit its 1-D grid.
  const int64_t tile = apb::attention_tile_rows();
  const int64_t tiles = ((int64_t)p->anchor_len + p->local_len + tile - 1) / tile * p->n_q_heads;
  if (tiles >= (int64_t(1) << 31)) return APB_ERR_BAD_SHAPE;
  if (p->head_dim != 64 && p->head_dim != 128) return APB_ERR_UNSUPPORTED;
  return APB_OK;
}

double apb_attention_flops(const apb_problem_t* p) {
  if (apb_validate_problem(p) != APB_OK) return -1.0;
  const double la = p->anchor_len, lb = p->local_len;
  const double lp = (double)p->host_idx * p->pass_len;
  const double pairs = la * (la + 1) / 2 + lb * (la + lp) + lb * (lb + 1) / 2;
  return 4.0 * p->head_dim * p->n_q_heads * pairs;
}

apb_status_t apb_compress_select(const apb_problem_t* p, const float* scores, const uint16_t* k,
                                 const uint16_t* v, int32_t* out_idx, uint16_t* out_k,
                                 uint16_t* out_v, void* stream) {
  const apb_status_t st = apb_validate_problem(p);
  if (st != APB_OK) return st;
  if (!scores || !k || !v || !out_k || !out_v) return APB_ERR_NULL_POINTER;
  if (!aligned(scores, 4) || !aligned(k, 16) || !aligned(v, 16) || !aligned(out_k, 16) ||
      !aligned(out_v, 16) || (out_idx && !aligned(out_idx, 4)))
    return APB_ERR_MISALIGNED;
  const int64_t d = p->head_dim, nkv = p->n_kv_heads, lp = p->pass_len;
  const int64_t kv_bytes = nkv * ((int64_t)p->anchor_len + p->local_len) * d * 2;
  const Range in[3] = {range_of(scores, nkv * p->local_len * 4), range_of(k, kv_bytes),
                       range_of(v, kv_bytes)};
  const Range out[3] = {range_of(out_idx, out_idx ? nkv * lp * 4 : 0),
                        range_of(out_k, nkv * lp * d * 2), range_of(out_v, nkv * lp * d * 2)};
  for (const Range& o : out) {
    for (const Range& i : in)
      if (overlaps(o, i)) return APB_ERR_ALIAS;
  }
  if (overlaps(out[0], out[1]) || overlaps(out[0], out[2]) || overlaps(out[1], out[2]))
    return APB_ERR_ALIAS;
  if (lp == 0) return APB_OK;

  apb::CompressArgs a;
  a.scores = scores; a.k = k; a.v = v; a.idx = out_idx; a.out_k = out_k; a.out_v = out_v;
  a.La = p->anchor_len; a.Lb = p->local_len; a.lp = p->pass_len;
  a.n_kv = p->n_kv_heads; a.head_dim = p->head_dim;
  const hipError_t e = apb::launch_compress(a, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) {
    set_last_error(e);
    return APB_ERR_HIP;
  }
  return APB_OK;
}

apb_status_t apb_attention_fwd(const apb_problem_t* p, const uint16_t* q, const uint16_t* k,
                               const uint16_t* v, const uint16_t* k_pass,
                               const uint16_t* v_pass, uint16_t* o, float* lse,
                               float softmax_scale, void* stream) {
  const apb_status_t st = apb_validate_problem(p);
  if (st != APB_OK) return st;
  const int64_t Lp = (int64_t)p->host_idx * p->pass_len;
  if (!q || !k || !v || !o) return APB_ERR_NULL_POINTER;
  if (Lp > 0 && (!k_pass || !v_pass)) return APB_ERR_NULL_POINTER;
  if (!aligned(q, 16) || !aligned(k, 16) || !aligned(v, 16) || !aligned(o, 16) ||
      (lse && !aligned(lse, 4)))
    return APB_ERR_MISALIGNED;
  if (Lp > 0 && (!aligned(k_pass, 16) || !aligned(v_pass, 16))) return APB_ERR_MISALIGNED;
  const int64_t d = p->head_dim, M = (int64_t)p->anchor_len + p->local_len;
  const int64_t q_bytes = (int64_t)p->n_q_heads * M * d * 2;
  const int64_t kv_bytes = (int64_t)p->n_kv_heads * M * d * 2;
  const int64_t pass_bytes = Lp > 0 ? Lp * p->n_kv_heads * d * 2 : 0;
  const Range in[5] = {range_of(q, q_bytes), range_of(k, kv_bytes), range_of(v, kv_bytes),
                       range_of(Lp > 0 ? k_pass : nullptr, pass_bytes),
                       range_of(Lp > 0 ? v_pass : nullptr, pass_bytes)};
  const Range out[2] = {range_of(o, q_bytes),
                        range_of(lse, lse ? (int64_t)p->n_q_heads * M * 4 : 0)};
  for (const Range& r : out)
    for (const Range& i : in)
      if (overlaps(r, i)) return APB_ERR_ALIAS;
  if (overlaps(out[0], out[1])) return APB_ERR_ALIAS;

  float scale = softmax_scale;
  if (!(scale > 0.f) || !isfinite(scale)) scale = 1.f / sqrtf((float)p->head_dim);
  apb::AttnArgs a;
  a.q = q; a.k = k; a.v = v;
  a.kp = Lp > 0 ? k_pass : nullptr;
  a.vp = Lp > 0 ? v_pass : nullptr;
  a.o = o; a.lse = lse;
  a.La = p->anchor_len; a.Lb = p->local_len; a.lp = p->pass_len; a.Lp = (int32_t)Lp;
  a.n_q = p->n_q_heads; a.n_kv = p->n_kv_heads; a.head_dim = p->head_dim;
  a.scale_log2 = scale * 1.4426950408889634f;
  const hipError_t e = apb::launch_attention(a, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) {
    set_last_error(e);
    return APB_ERR_HIP;
  }
  return APB_OK;
}

apb_status_t apb_validate_scorer(const apb_scorer_problem_t* p) {
  if (!p) return APB_ERR_NULL_POINTER;
  if (p->anchor_len < 0 || p->local_len < 1) return APB_ERR_BAD_SHAPE;
  if (p->n_kv_heads < 1 || p->n_q_heads < 1 || p->n_q_heads % p->n_kv_heads != 0)
    return APB_ERR_BAD_SHAPE;
  if (p->head_dim < 1 || p->hidden < 1) return APB_ERR_BAD_SHAPE;
  if ((int64_t)p->anchor_len + p->local_len > kMaxRows) return APB_ERR_BAD_SHAPE;
  if ((int64_t)(p->n_q_heads + 2 * p->n_kv_heads) * p->head_dim > (int64_t(1) << 20))
    return APB_ERR_BAD_SHAPE;
  if (p->head_dim != 64 && p->head_dim != 128) return APB_ERR_UNSUPPORTED;
  if (p->n_kv_heads > apb::scorer_max_kv()) return APB_ERR_UNSUPPORTED;
  if (p->hidden % apb::scorer_hidden_block() != 0) return APB_ERR_UNSUPPORTED;
  return APB_OK;
}

static apb::ScorerArgs scorer_args(const apb_scorer_problem_t* p) {
  apb::ScorerArgs a{};
  a.La = p->anchor_len; a.Lb = p->local_len; a.n_q = p->n_q_heads; a.n_kv = p->n_kv_heads;
  a.head_dim = p->head_dim; a.hidden = p->hidden;
  return a;
}

apb_status_t apb_scorer_workspace_size(const apb_scorer_problem_t* p, uint64_t* bytes) {
  const apb_status_t st = apb_validate_scorer(p);
  if (st != APB_OK) return st;
  if (!bytes) return APB_ERR_NULL_POINTER;
  *bytes = apb::scorer_workspace_bytes(scorer_args(p));
  return APB_OK;
}

apb_status_t apb_retaining_scores(const apb_scorer_problem_t* p, const uint16_t* q,
                                  const uint16_t* k, const uint16_t* v, const uint16_t* w1,
                                  const float* b1, const float* w2, const float* b2,
                                  float* scores, void* workspace, uint64_t workspace_bytes,
                                  void* stream) {
  const apb_status_t st = apb_validate_scorer(p);
  if (st != APB_OK) return st;
  if (!q || !k || !v || !w1 || !b1 || !w2 || !b2 || !scores || !workspace)
    return APB_ERR_NULL_POINTER;
  if (!aligned(q, 16) || !aligned(k, 16) || !aligned(v, 16) || !aligned(w1, 16) ||
      !aligned(b1, 4) || !aligned(w2, 4) || !aligned(b2, 4) || !aligned(scores, 4) ||
      !aligned(workspace, 16))
    return APB_ERR_MISALIGNED;
  apb::ScorerArgs a = scorer_args(p);
  const uint64_t need = apb::scorer_workspace_bytes(a);
  if (workspace_bytes < need) return APB_ERR_BAD_SHAPE;
  const int64_t d = p->head_dim, M = (int64_t)p->anchor_len + p->local_len;
  const int64_t F = (int64_t)(p->n_q_heads + 2 * p->n_kv_heads) * d;
  const Range in[7] = {range_of(q, (int64_t)p->n_q_heads * M * d * 2),
                       range_of(k, (int64_t)p->n_kv_heads * M * d * 2),
                       range_of(v, (int64_t)p->n_kv_heads * M * d * 2),
                       range_of(w1, (int64_t)p->hidden * F * 2), range_of(b1, (int64_t)p->hidden * 4),
                       range_of(w2, (int64_t)p->n_kv_heads * p->hidden * 4),
                       range_of(b2, (int64_t)p->n_kv_heads * 4)};
  const Range out[2] = {range_of(scores, (int64_t)p->n_kv_heads * p->local_len * 4),
                        range_of(workspace, (int64_t)need)};
  for (const Range& r : out)
    for (const Range& i : in)
      if (overlaps(r, i)) return APB_ERR_ALIAS;
  if (overlaps(out[0], out[1])) return APB_ERR_ALIAS;
  a.q = q; a.k = k; a.v = v; a.w1 = w1; a.b1 = b1; a.w2 = w2; a.b2 = b2; a.scores = scores;
  a.workspace = static_cast<float*>(workspace);
  const hipError_t e = apb::launch_scorer(a, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) {
    set_last_error(e);
    return APB_ERR_HIP;
  }
  return APB_OK;
}

static apb_scorer_problem_t layer_scorer_problem(const apb_layer_problem_t* p) {
  apb_scorer_problem_t s;
  s.anchor_len = p->attn.anchor_len; s.local_len = p->attn.local_len;
  s.n_q_heads = p->attn.n_q_heads; s.n_kv_heads = p->attn.n_kv_heads;
  s.head_dim = p->attn.head_dim; s.hidden = p->scorer_hidden;
  return s;
}

apb_status_t apb_validate_layer(const apb_layer_problem_t* p) {
  if (!p) return APB_ERR_NULL_POINTER;
  apb_status_t st = apb_validate_problem(&p->attn);
  if (st != APB_OK) return st;
  const apb_scorer_problem_t sp = layer_scorer_problem(p);
  st = apb_validate_scorer(&sp);
  if (st != APB_OK) return st;
  if (p->hidden < 64 || p->hidden % 64 != 0 || p->intermediate < 64 || p->intermediate % 64 != 0)
    return APB_ERR_BAD_SHAPE;
  if (p->hidden > (1 << 20) || p->intermediate > (1 << 20)) return APB_ERR_BAD_SHAPE;
  if (!(p->rms_eps > 0.f) || !isfinite(p->rms_eps) || !(p->rope_theta > 1.f) ||
      !isfinite(p->rope_theta))
    return APB_ERR_BAD_SHAPE;
  return APB_OK;
}

static apb::LayerArgs layer_args(const apb_layer_problem_t* p) {
  apb::LayerArgs a{};
  a.host_idx = p->attn.host_idx; a.La = p->attn.anchor_len; a.Lb = p->attn.local_len;
  a.lp = p->attn.pass_len; a.n_q = p->attn.n_q_heads; a.n_kv = p->attn.n_kv_heads;
  a.head_dim = p->attn.head_dim; a.D = p->hidden; a.I = p->intermediate;
  a.scorer_hidden = p->scorer_hidden; a.eps = p->rms_eps; a.theta = p->rope_theta;
  return a;
}

apb_status_t apb_layer_workspace_size(const apb_layer_problem_t* p, uint64_t* bytes) {
  const apb_status_t st = apb_validate_layer(p);
  if (st != APB_OK) return st;
  if (!bytes) return APB_ERR_NULL_POINTER;
  *bytes = apb::layer_workspace_bytes(layer_args(p));
  return APB_OK;
}

double apb_layer_flops(const apb_layer_problem_t* p) {
  if (apb_validate_layer(p) != APB_OK) return -1.0;
  const double T = (double)p->attn.anchor_len + p->attn.local_len;
  const double D = p->hidden, I = p->intermediate, d = p->attn.head_dim;
  const double nq = p->attn.n_q_heads, nkv = p->attn.n_kv_heads;
  const double Fr = (nq + 2 * nkv) * d, hr = p->scorer_hidden, Lb = p->attn.local_len;
  return 2 * T * D * (nq + 2 * nkv) * d + 2 * T * nq * d * D + 6 * T * D * I +
         2 * Lb * Fr * hr + 2 * Lb * hr * nkv + apb_attention_flops(&p->attn);
}

apb_status_t apb_layer_fwd(const apb_layer_problem_t* p, const apb_layer_weights_t* w,
                           const uint16_t* hidden_in, const int32_t* positions,
                           uint16_t* k_cache, uint16_t* v_cache, uint16_t* pass_k,
                           uint16_t* pass_v, uint16_t* hidden_out, void* workspace,
                           uint64_t workspace_bytes, void* stream) {
  const apb_status_t st = apb_validate_layer(p);
  if (st != APB_OK) return st;
  if (!w || !hidden_in || !positions || !k_cache || !v_cache || !hidden_out || !workspace)
    return APB_ERR_NULL_POINTER;
  if (!w->ln1 || !w->w_qkv || !w->w_o || !w->ln2 || !w->w_gate || !w->w_up || !w->w_down ||
      !w->r_w1 || !w->r_b1 || !w->r_w2 || !w->r_b2)
    return APB_ERR_NULL_POINTER;
  const apb_problem_t& ap = p->attn;
  if (ap.pass_len > 0 && (!pass_k || !pass_v)) return APB_ERR_NULL_POINTER;
  const void* b16[] = {w->ln1, w->w_qkv, w->w_o, w->ln2, w->w_gate, w->w_up, w->w_down, w->r_w1,
                       hidden_in, k_cache, v_cache, hidden_out, workspace};
  for (const void* ptr : b16)
    if (!aligned(ptr, 16)) return APB_ERR_MISALIGNED;
  if (!aligned(w->r_b1, 4) || !aligned(w->r_w2, 4) || !aligned(w->r_b2, 4) ||
      !aligned(positions, 4))
    return APB_ERR_MISALIGNED;
  if (ap.pass_len > 0 && (!aligned(pass_k, 16) || !aligned(pass_v, 16))) return APB_ERR_MISALIGNED;
  apb::LayerArgs a = layer_args(p);
  const uint64_t need = apb::layer_workspace_bytes(a);
  if (workspace_bytes < need) return APB_ERR_BAD_SHAPE;

  const int64_t T = (int64_t)ap.anchor_len + ap.local_len, D = p->hidden, I = p->intermediate;
  const int64_t d = ap.head_dim, nq = ap.n_q_heads, nkv = ap.n_kv_heads;
  const int64_t Fr = (nq + 2 * nkv) * d, hr = p->scorer_hidden;
  const int64_t slot = nkv * (int64_t)ap.pass_len * d * 2;  // bytes of one passing slot
  const bool pass = ap.pass_len > 0;
  const Range in[15] = {
      range_of(hidden_in, T * D * 2), range_of(positions, T * 4), range_of(w->ln1, D * 2),
      range_of(w->w_qkv, Fr * D * 2), range_of(w->w_o, D * nq * d * 2), range_of(w->ln2, D * 2),
      range_of(w->w_gate, I * D * 2), range_of(w->w_up, I * D * 2), range_of(w->w_down, D * I * 2),
      range_of(w->r_w1, hr * Fr * 2), range_of(w->r_b1, hr * 4), range_of(w->r_w2, nkv * hr * 4),
      range_of(w->r_b2, nkv * 4), range_of(pass ? pass_k : nullptr, ap.host_idx * slot),
      range_of(pass ? pass_v : nullptr, ap.host_idx * slot)};
  const Range out[6] = {range_of(k_cache, nkv * T * d * 2), range_of(v_cache, nkv * T * d * 2),
                        range_of(hidden_out, T * D * 2), range_of(workspace, (int64_t)need),
                        range_of(pass ? (const uint8_t*)pass_k + ap.host_idx * slot : nullptr, slot),
                        range_of(pass ? (const uint8_t*)pass_v + ap.host_idx * slot : nullptr, slot)};
  for (const Range& r : out)
    for (const Range& i : in)
      if (overlaps(r, i)) return APB_ERR_ALIAS;
  for (int i = 0; i < 6; ++i)
    for (int j = i + 1; j < 6; ++j)
      if (overlaps(out[i], out[j])) return APB_ERR_ALIAS;

  a.hidden = hidden_in; a.pos = positions;
  a.ln1 = w->ln1; a.w_qkv = w->w_qkv; a.w_o = w->w_o; a.ln2 = w->ln2; a.w_gate = w->w_gate;
  a.w_up = w->w_up; a.w_down = w->w_down; a.r_w1 = w->r_w1; a.r_b1 = w->r_b1; a.r_w2 = w->r_w2;
  a.r_b2 = w->r_b2; a.k_cache = k_cache; a.v_cache = v_cache;
  a.pass_k = pass ? pass_k : nullptr; a.pass_v = pass ? pass_v : nullptr;
  a.hidden_out = hidden_out; a.workspace = workspace;
  const hipError_t e = apb::launch_layer(a, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) {
    set_last_error(e);
    return APB_ERR_HIP;
  }
  return APB_OK;
}

apb_status_t apb_validate_decode(const apb_decode_problem_t* p) {
  if (!p) return APB_ERR_NULL_POINTER;
  if (p->n_kv_heads < 1 || p->n_q_heads < 1 || p->n_q_heads % p->n_kv_heads != 0)
    return APB_ERR_BAD_SHAPE;
  if (p->cache_len < 0 || p->n_new < 1 || (p->append_new != 0 && p->append_new != 1))
    return APB_ERR_BAD_SHAPE;
  if (p->head_dim < 1) return APB_ERR_BAD_SHAPE;
  if ((int64_t)p->cache_len + p->n_new > kMaxRows) return APB_ERR_BAD_SHAPE;
  // rows of one GQA group and of the whole call stay well inside int32
  if ((int64_t)p->n_q_heads * p->n_new > kMaxRows) return APB_ERR_BAD_SHAPE;
  if (p->head_dim != 64 && p->head_dim != 128) return APB_ERR_UNSUPPORTED;
  return APB_OK;
}

static apb::DecodeArgs decode_args(const apb_decode_problem_t* p) {
  apb::DecodeArgs a{};
  a.Lc = p->cache_len; a.n_new = p->n_new; a.append = p->append_new;
  a.n_q = p->n_q_heads; a.n_kv = p->n_kv_heads; a.head_dim = p->head_dim;
  return a;
}

apb_status_t apb_decode_workspace_size(const apb_decode_problem_t* p, uint64_t* bytes) {
  const apb_status_t st = apb_validate_decode(p);
  if (st != APB_OK) return st;
  if (!bytes) return APB_ERR_NULL_POINTER;
  *bytes = apb::plan_decode(decode_args(p)).workspace_bytes;
  return APB_OK;
}

// Checks shared by the two decode entry points (everything but the
// workspace), and the kernel arguments of a valid call.
static apb_status_t decode_checks(const apb_decode_problem_t* p, const uint16_t* q,
                                  const uint16_t* k_cache, const uint16_t* v_cache,
                                  const uint16_t* k_new, const uint16_t* v_new, float* o_part,
                                  float* lse_part, float softmax_scale, apb::DecodeArgs* a) {
  const apb_status_t st = apb_validate_decode(p);
  if (st != APB_OK) return st;
  const bool has_cache = p->cache_len > 0, app = p->append_new == 1;
  if (!q || !o_part || !lse_part) return APB_ERR_NULL_POINTER;
  if (has_cache && (!k_cache || !v_cache)) return APB_ERR_NULL_POINTER;
  if (app && (!k_new || !v_new)) return APB_ERR_NULL_POINTER;
  if (!aligned(q, 16) || !aligned(o_part, 16) || !aligned(lse_part, 4)) return APB_ERR_MISALIGNED;
  if (has_cache && (!aligned(k_cache, 16) || !aligned(v_cache, 16))) return APB_ERR_MISALIGNED;
  if (app && (!aligned(k_new, 16) || !aligned(v_new, 16))) return APB_ERR_MISALIGNED;
  const int64_t d = p->head_dim, rows = (int64_t)p->n_q_heads * p->n_new;
  const int64_t cache_bytes = has_cache ? (int64_t)p->n_kv_heads * p->cache_len * d * 2 : 0;
  const int64_t new_bytes = app ? (int64_t)p->n_kv_heads * p->n_new * d * 2 : 0;
  const Range in[5] = {range_of(q, rows * d * 2), range_of(has_cache ? k_cache : nullptr, cache_bytes),
                       range_of(has_cache ? v_cache : nullptr, cache_bytes),
                       range_of(app ? k_new : nullptr, new_bytes),
                       range_of(app ? v_new : nullptr, new_bytes)};
  const Range out[2] = {range_of(o_part, rows * d * 4), range_of(lse_part, rows * 4)};
  for (const Range& r : out)
    for (const Range& i : in)
      if (overlaps(r, i)) return APB_ERR_ALIAS;
  if (overlaps(out[0], out[1])) return APB_ERR_ALIAS;

  *a = decode_args(p);
  float scale = softmax_scale;
  if (!(scale > 0.f) || !isfinite(scale)) scale = 1.f / sqrtf((float)p->head_dim);
  a->q = q;
  a->kc = has_cache ? k_cache : nullptr;
  a->vc = has_cache ? v_cache : nullptr;
  a->kn = app ? k_new : nullptr;
  a->vn = app ? v_new : nullptr;
  a->o = o_part; a->lse = lse_part;
  a->scale_log2 = scale * 1.4426950408889634f;
  return APB_OK;
}

apb_status_t apb_decode_attention(const apb_decode_problem_t* p, const uint16_t* q,
                                  const uint16_t* k_cache, const uint16_t* v_cache,
                                  const uint16_t* k_new, const uint16_t* v_new, float* o_part,
                                  float* lse_part, float softmax_scale, void* workspace,
                                  uint64_t workspace_bytes, void* stream) {
  apb::DecodeArgs a;
  const apb_status_t st =
      decode_checks(p, q, k_cache, v_cache, k_new, v_new, o_part, lse_part, softmax_scale, &a);
  if (st != APB_OK) return st;
  if (!workspace) return APB_ERR_NULL_POINTER;
  if (!aligned(workspace, 16)) return APB_ERR_MISALIGNED;
  const apb::DecodePlan pl = apb::plan_decode(a);
  if (workspace_bytes < pl.workspace_bytes) return APB_ERR_BAD_SHAPE;
  const int64_t d = p->head_dim, rows = (int64_t)p->n_q_heads * p->n_new;
  const bool has_cache = p->cache_len > 0, app = p->append_new == 1;
  const int64_t cache_bytes = has_cache ? (int64_t)p->n_kv_heads * p->cache_len * d * 2 : 0;
  const int64_t new_bytes = app ? (int64_t)p->n_kv_heads * p->n_new * d * 2 : 0;
  const Range ws = range_of(workspace, (int64_t)pl.workspace_bytes);
  const Range others[7] = {range_of(q, rows * d * 2), range_of(a.kc, cache_bytes),
                           range_of(a.vc, cache_bytes), range_of(a.kn, new_bytes),
                           range_of(a.vn, new_bytes), range_of(o_part, rows * d * 4),
                           range_of(lse_part, rows * 4)};
  for (const Range& r : others)
    if (overlaps(ws, r)) return APB_ERR_ALIAS;
  a.workspace = static_cast<float*>(workspace);
  const hipError_t e = apb::launch_decode(a, pl, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) {
    set_last_error(e);
    return APB_ERR_HIP;
  }
  return APB_OK;
}

apb_status_t apb_decode_attention_noalloc(const apb_decode_problem_t* p, const uint16_t* q,
                                          const uint16_t* k_cache, const uint16_t* v_cache,
                                          const uint16_t* k_new, const uint16_t* v_new,
                                          float* o_part, float* lse_part, float softmax_scale,
                                          void* stream) {
  apb::DecodeArgs a;
  const apb_status_t st =
      decode_checks(p, q, k_cache, v_cache, k_new, v_new, o_part, lse_part, softmax_scale, &a);
  if (st != APB_OK) return st;
  // the split partials must fit the library's scratch: fewer, longer splits
  // when the default plan does not, an error when one split does not
  const apb::DecodePlan pl = apb::plan_decode(a, APB_DECODE_NOALLOC_SCRATCH_BYTES);
  if (pl.n_split < 1) return APB_ERR_SCRATCH;
  void* scratch = nullptr;
  hipError_t e = apb::decode_scratch(&scratch);
  if (e == hipSuccess) {
    a.workspace = static_cast<float*>(scratch);
    e = apb::launch_decode(a, pl, static_cast<hipStream_t>(stream));
  }
  if (e != hipSuccess) {
    set_last_error(e);
    return APB_ERR_HIP;
  }
  return APB_OK;
}

apb_status_t apb_merge_partials(int32_t n_parts, int32_t rows, int32_t head_dim,
                                const float* o_parts, const float* lse_parts, uint16_t* o,
                                float* lse, void* stream) {
  if (n_parts < 1 || rows < 0 || head_dim < 1) return APB_ERR_BAD_SHAPE;
  if ((int64_t)n_parts * rows > kMaxRows) return APB_ERR_BAD_SHAPE;
  if (head_dim != 64 && head_dim != 128) return APB_ERR_UNSUPPORTED;
  if (rows == 0) return APB_OK;
  if (!o_parts || !lse_parts || !o) return APB_ERR_NULL_POINTER;
  if (!aligned(o_parts, 16) || !aligned(lse_parts, 4) || !aligned(o, 16) ||
      (lse && !aligned(lse, 4)))
    return APB_ERR_MISALIGNED;
  const int64_t d = head_dim;
  const Range in[2] = {range_of(o_parts, (int64_t)n_parts * rows * d * 4),
                       range_of(lse_parts, (int64_t)n_parts * rows * 4)};
  const Range out[2] = {range_of(o, (int64_t)rows * d * 2), range_of(lse, lse ? (int64_t)rows * 4 : 0)};
  for (const Range& r : out)
    for (const Range& i : in)
      if (overlaps(r, i)) return APB_ERR_ALIAS;
  if (overlaps(out[0], out[1])) return APB_ERR_ALIAS;
  apb::MergeArgs a;
  a.o_parts = o_parts; a.lse_parts = lse_parts; a.o = o; a.lse = lse;
  a.n_parts = n_parts; a.rows = rows; a.head_dim = head_dim;
  const hipError_t e = apb::launch_merge(a, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) {
    set_last_error(e);
    return APB_ERR_HIP;
  }
  return APB_OK;
}

}  // extern "C"
