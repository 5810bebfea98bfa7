/*
 * apb.h -- C ABI of one host's share of APB attention on MI355X: the prefill
 * hot path and the decoding stage.
 *
 * APB (Accelerating distributed long-context inference by Passing compressed
 * context Blocks) splits a long document across H hosts.  Host h holds an
 * anchor block A (query tokens plus the first document tokens, Sec. 3.3), its
 * local block B_h (Sec. 3.3), and receives from every earlier host a
 * compressed block of l_p key/value rows chosen by a compressor (Sec. 3.4),
 * which together form the passing block P (Sec. 3.5).  Attention then runs
 * over queries [A; B_h] and keys/values [A; P; B_h] under a modified mask
 * (Sec. 3.6, Eq. 2).
 *
 * This library exports the kernels of that host share:
 *   apb_compress_select  ArgTop-l_p of the local block's scores + gather of
 *                        the selected K/V rows (Sec. 3.4; Alg. 2, compression
 *                        step);
 *   apb_attention_fwd    the modified-mask attention (Eq. 2; Alg. 2,
 *                        attention step);
 *   apb_retaining_scores the compressor's scores from a retaining head
 *                        (Sec. 3.4) with caller-supplied weights;
 *   apb_layer_fwd        the whole layer of one host around these kernels
 *                        (Alg. 2: projections, norms, RoPE, FFN);
 * and the decoding stage that follows the prefill (Alg. 3):
 *   apb_decode_attention one host's exact attention of the new tokens over
 *                        its KV cache, with the LSE;
 *   apb_merge_partials   MergeScore of the hosts' partial results;
 * plus apb_decode_attention_noalloc, the decode call for callers that cannot
 * allocate (its scratch is the library's own).
 *
 * Conventions shared by every entry point
 *   - All tensor pointers are caller-owned DEVICE memory on the current HIP
 *     device.  The library never allocates, frees or keeps them.
 *   - bf16 tensors are passed as uint16_t bit patterns.  Layouts are
 *     head-major, row-major, head_dim contiguous, densely packed.  bf16
 *     tensors must be 16-byte aligned; fp32 and int32 tensors 4-byte aligned.
 *   - Calls are asynchronous on `stream` (a hipStream_t passed as void*; NULL
 *     is the default stream), stateless and re-entrant (except
 *     apb_decode_attention_noalloc, whose calls on one GPU share its scratch).
 *     No host sync.
 *   - Every argument is validated on the host BEFORE any HIP call; a call
 *     that returns an error has launched nothing and written nothing.
 *   - Index arithmetic is 64-bit; a problem must satisfy
 *     La + host_idx*l_p + Lb <= 2^30 rows.
 *   - Outputs must not overlap inputs (checked: APB_ERR_ALIAS).
 */
#ifndef APB_H_
#define APB_H_

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define APB_ABI_VERSION 5

typedef enum {
  APB_OK = 0,
  APB_ERR_NULL_POINTER = 1, /* a required pointer is NULL                    */
  APB_ERR_BAD_SHAPE = 2,    /* a size violates the constraints below         */
  APB_ERR_UNSUPPORTED = 3,  /* valid in the paper, not built here (head_dim) */
  APB_ERR_MISALIGNED = 4,   /* a pointer breaks the alignment rule           */
  APB_ERR_HIP = 5,          /* the HIP runtime reported a launch error       */
  APB_ERR_ALIAS = 6,        /* an output overlaps an input                   */
  APB_ERR_SCRATCH = 7       /* a no-allocation call needs more scratch than
                               the library holds                             */
} apb_status_t;

/* One host's share of one attention layer: the inputs of Alg. 2 (l_p, h, H)
 * and of Alg. 1 (l_a, l_p, h, H), plus the attention head geometry. */
typedef struct {
  int32_t n_hosts;    /* H >= 1: hosts the document is split over (Sec. 3.3) */
  int32_t host_idx;   /* 0 <= host_idx < H, 0-based; equals the number of
                         previous hosts (the paper's h is host_idx + 1)      */
  int32_t anchor_len; /* La = l_q + l_a >= 0 anchor rows (Sec. 3.3); 0 for
                         the first host or the no-anchor ablation           */
  int32_t local_len;  /* Lb = l_b >= 1 rows of the local block (Sec. 3.3)   */
  int32_t pass_len;   /* 0 <= l_p <= Lb rows each host passes on (Sec. 3.4) */
  int32_t n_q_heads;  /* n_q >= 1, a multiple of n_kv                       */
  int32_t n_kv_heads; /* n_kv >= 1; query head i reads KV head i / (n_q/n_kv) */
  int32_t head_dim;   /* d, in {64, 128}                                     */
} apb_problem_t;

/*
 * apb_compress_select -- the compressor C of Sec. 3.4 given the retaining
 * heads' scores: ArgTop-l_p per KV head, then K^C = K_h[idx], V^C = V_h[idx]
 * (Alg. 2, compression step).
 *
 *   scores  fp32 [n_kv][Lb]       importance of each local KV pair.
 *   k, v    bf16 [n_kv][La+Lb][d] this host's keys/values; the local block
 *                                 starts at row La.
 *   out_idx int32 [n_kv][l_p]     selected local indices (0..Lb-1), ascending;
 *                                 may be NULL.
 *   out_k, out_v bf16 [n_kv][l_p][d]  bit copies of rows La+idx; typically
 *                                 slot host_idx of a rank-major passing
 *                                 buffer [H][n_kv][l_p][d].
 * Selection: the l_p largest scores; equal scores (-0 equal to +0) go to the
 * lower index; NaN ranks below -inf.  The result is unique, so it is
 * bit-exact and deterministic.  l_p == 0 launches nothing and returns APB_OK.
 */
apb_status_t apb_compress_select(const apb_problem_t* p, const float* scores,
                                 const uint16_t* k, const uint16_t* v,
                                 int32_t* out_idx, uint16_t* out_k,
                                 uint16_t* out_v, void* stream);

/*
 * apb_attention_fwd -- the modified-mask attention of Eq. 2 (Sec. 3.6):
 * queries [A; B_h], keys/values [A; P; B_h] with P the earlier hosts'
 * compressed blocks in host order (Sec. 3.5).  Mask M': causal attention over
 * the concatenation [A; P; B_h] with the query rows of P removed, i.e. query
 * row r sees concatenated keys 0..pos(r) where pos(r) = r for anchor rows
 * (r < La) and r + host_idx*l_p for local rows.
 *
 *   q       bf16 [n_q][La+Lb][d]
 *   k, v    bf16 [n_kv][La+Lb][d]            anchor rows then local rows.
 *   k_pass, v_pass bf16 [host_idx][n_kv][l_p][d]  rank-major slots 0..host_idx-1
 *                                 of the all-gathered compressed blocks
 *                                 (Alg. 2, communication step); required
 *                                 when host_idx*l_p > 0, ignored otherwise.
 *   o       bf16 [n_q][La+Lb][d]  softmax-weighted values, rounded to nearest
 *                                 even.
 *   lse     fp32 [n_q][La+Lb]     natural log of the sum of exp(scaled
 *                                 logits) per row, the quantity an LSE merge
 *                                 of partial results needs (Alg. 3); may be
 *                                 NULL.
 *   softmax_scale  multiplier of Q.K; <= 0, NaN or inf selects 1/sqrt(d)
 *                  (Eq. 1, d_m = head_dim).
 * Arithmetic: bf16 inputs, fp32 dot products and softmax, probabilities
 * rounded to bf16 for the value product, fp32 accumulation.
 */
apb_status_t apb_attention_fwd(const apb_problem_t* p, const uint16_t* q,
                               const uint16_t* k, const uint16_t* v,
                               const uint16_t* k_pass, const uint16_t* v_pass,
                               uint16_t* o, float* lse, float softmax_scale,
                               void* stream);

/* ------------------------------------------------------------------------
 * Retaining-head scorer R (Sec. 3.4; Alg. 2, compression step; App. B): the
 * importance of every local-block cache unit, the input of
 * apb_compress_select.  The paper fixes only a small MLP over [Q, K, V] with
 * intermediate size 1024; this library reads it as two linear layers with a
 * SiLU between:
 *   x_t = [Q_0[t] .. Q_{n_q-1}[t], K_0[t] .. K_{n_kv-1}[t], V_0[t] .. V_{n_kv-1}[t]]
 *   scores[kv][t] = (W2 SiLU(W1 x_t + b1) + b2)[kv]
 * ------------------------------------------------------------------------ */
typedef struct {
  int32_t anchor_len; /* La >= 0: rows of Q/K/V before the local block      */
  int32_t local_len;  /* Lb >= 1: local tokens to score                      */
  int32_t n_q_heads;  /* n_q >= 1, a multiple of n_kv                        */
  int32_t n_kv_heads; /* 1 <= n_kv <= 8 (one score per KV head)              */
  int32_t head_dim;   /* d, in {64, 128}                                     */
  int32_t hidden;     /* hidden units, a positive multiple of 256 (1024 in
                         the paper)                                          */
} apb_scorer_problem_t;

/* Host-only checks of a scorer problem (no HIP call). */
apb_status_t apb_validate_scorer(const apb_scorer_problem_t* p);

/* Bytes of device workspace apb_retaining_scores needs (host only). */
apb_status_t apb_scorer_workspace_size(const apb_scorer_problem_t* p, uint64_t* bytes);

/*
 * apb_retaining_scores -- the scores s_1..s_lb of Alg. 2 for one host.
 *
 *   q       bf16 [n_q][La+Lb][d]     k, v bf16 [n_kv][La+Lb][d]  (only rows
 *                                    La.. are read)
 *   w1      bf16 [hidden][(n_q + 2 n_kv) d]  first layer (out x in)
 *   b1      fp32 [hidden]
 *   w2      fp32 [n_kv][hidden]      second layer
 *   b2      fp32 [n_kv]
 *   scores  fp32 [n_kv][Lb]          the layout apb_compress_select takes
 *   workspace, workspace_bytes  caller-owned device scratch of at least
 *                   apb_scorer_workspace_size() bytes, 16-byte aligned.
 * Arithmetic: bf16 products with fp32 accumulation for the first layer, fp32
 * bias, SiLU and second layer; deterministic (fixed summation order).
 */
apb_status_t apb_retaining_scores(const apb_scorer_problem_t* p, const uint16_t* q,
                                  const uint16_t* k, const uint16_t* v, const uint16_t* w1,
                                  const float* b1, const float* w2, const float* b2,
                                  float* scores, void* workspace, uint64_t workspace_bytes,
                                  void* stream);

/* ------------------------------------------------------------------------
 * Decoding stage (stage 2, Alg. 3).  Every host attends the new tokens'
 * queries to its own KV cache (its local block; Alg. 1 keeps K_h, V_h), the
 * last host after appending the new tokens' own K/V; the hosts' partial
 * outputs are then gathered and merged by their LSE (MergeScore).
 * ------------------------------------------------------------------------ */
typedef struct {
  int32_t n_q_heads;  /* n_q >= 1, a multiple of n_kv                        */
  int32_t n_kv_heads; /* n_kv >= 1; query head i reads KV head i / (n_q/n_kv) */
  int32_t head_dim;   /* d, in {64, 128}                                     */
  int32_t cache_len;  /* Lc >= 0 rows in this host's KV cache                */
  int32_t n_new;      /* >= 1 new tokens (the question tokens at the first
                         decoding step, one generated token afterwards)     */
  int32_t append_new; /* 1 on the last host: the new tokens' K/V follow the
                         cache and new token j sees new tokens 0..j (causal);
                         0: the cache only                                   */
} apb_decode_problem_t;

/* Host-only checks of a decode problem (no HIP call). */
apb_status_t apb_validate_decode(const apb_decode_problem_t* p);

/* Bytes of device workspace apb_decode_attention needs for `p` (host only;
 * depends on the shapes only). */
apb_status_t apb_decode_workspace_size(const apb_decode_problem_t* p, uint64_t* bytes);

/*
 * apb_decode_attention -- one host's partial attention of a decoding step
 * (Alg. 3, the attention lines), exact softmax over the visible keys.
 *
 *   q        bf16 [n_q][n_new][d]   the new tokens' queries.
 *   k_cache, v_cache bf16 [n_kv][Lc][d]  this host's cache; ignored (may be
 *                                   NULL) when Lc == 0.
 *   k_new, v_new bf16 [n_kv][n_new][d]  the new tokens' keys/values; required
 *                                   when append_new, ignored otherwise.
 *   o_part   fp32 [n_q][n_new][d]   this host's partial output A_h.
 *   lse_part fp32 [n_q][n_new]      its natural-log LSE (what Gather and
 *                                   MergeScore need); a row with no visible
 *                                   key gets o = 0, lse = -inf.
 *   softmax_scale  as in apb_attention_fwd.
 *   workspace, workspace_bytes  caller-owned device scratch of at least
 *                   apb_decode_workspace_size() bytes, 16-byte aligned; the
 *                   call overwrites it (calls that overlap in time must not
 *                   share one).  The library allocates nothing.
 * Arithmetic: bf16 inputs, fp32 dot products and softmax, probabilities
 * rounded to bf16 for the value product, fp32 accumulation and output.  The
 * key range is split over workgroups whose normalised partials the call
 * merges: in fp32, or, when a KV head has 128 or more rows, in fp16 scaled
 * per row by a power of two (each value within 2^-11 of its row's largest).
 */
apb_status_t apb_decode_attention(const apb_decode_problem_t* p, const uint16_t* q,
                                  const uint16_t* k_cache, const uint16_t* v_cache,
                                  const uint16_t* k_new, const uint16_t* v_new,
                                  float* o_part, float* lse_part, float softmax_scale,
                                  void* workspace, uint64_t workspace_bytes, void* stream);

/*
 * apb_decode_attention_noalloc -- apb_decode_attention for callers that
 * cannot allocate device memory: code under HIP graph capture, tight serving
 * loops, harnesses that forbid allocation.  Same arguments, result and
 * arithmetic, minus the workspace: the split partials live in a device array
 * of APB_DECODE_NOALLOC_SCRATCH_BYTES that the library holds on every GPU it
 * runs on (from the first call on that GPU until the process ends).  The
 * call allocates nothing and frees nothing.
 *
 *   Limit: when the default split plan's partials exceed the array, the
 *   keys are split into fewer, longer parts (results then differ from
 *   apb_decode_attention's by rounding only); when even one part does not
 *   fit, the call returns APB_ERR_SCRATCH and launches nothing.  A part is
 *   n_q * n_new rows of (d + 1) * 4 bytes, or of 2 * d + 8 bytes when a KV
 *   head has 128 or more rows ((n_q / n_kv) * n_new >= 128).
 *   Races: every call on one GPU shares that GPU's array; calls that overlap
 *   in time on one GPU (other streams, other host threads) race and give
 *   undefined results.  Calls in one stream are ordered and safe.  The array
 *   keeps the last call's partials; nothing in it needs to start at zero.
 */
#define APB_DECODE_NOALLOC_SCRATCH_BYTES (16ull << 20)
apb_status_t apb_decode_attention_noalloc(const apb_decode_problem_t* p, const uint16_t* q,
                                          const uint16_t* k_cache, const uint16_t* v_cache,
                                          const uint16_t* k_new, const uint16_t* v_new,
                                          float* o_part, float* lse_part, float softmax_scale,
                                          void* stream);

/*
 * apb_merge_partials -- MergeScore of Alg. 3: given P partial results
 * (A_p, lse_p) of the same rows over disjoint key sets, the result over all
 * the keys: lse = ln sum_p exp(lse_p), A = sum_p exp(lse_p - lse) A_p.
 *
 *   o_parts   fp32 [n_parts][rows][d]   (e.g. the gathered o_part of H hosts)
 *   lse_parts fp32 [n_parts][rows]
 *   o         bf16 [rows][d]            rounded to nearest even.
 *   lse       fp32 [rows]               may be NULL.
 * n_parts >= 1, rows >= 0, d in {64, 128}.  A part with lse = -inf adds
 * nothing; a row whose parts are all -inf gets o = 0, lse = -inf.
 */
apb_status_t apb_merge_partials(int32_t n_parts, int32_t rows, int32_t head_dim,
                                const float* o_parts, const float* lse_parts, uint16_t* o,
                                float* lse, void* stream);

/* ------------------------------------------------------------------------
 * One host's whole layer (Alg. 2): the QKV projection of the anchor and
 * local hidden states, the retaining head R over the local block, ArgTop-l_p
 * and gather into this host's passing slot, attention over [A; P; B] with
 * the earlier hosts' slots, and the FFN.  The layer around attention is the
 * model's own; the paper does not restate it, and this library reads it as a
 * Llama-style pre-norm block:
 *   x = RMSNorm(H; ln1);  Q, K, V = heads of x W_qkv^T;  Q, K = RoPE(Q, K, pos)
 *   scores = R([Q_B, K_B, V_B]);  slot host_idx = K_B, V_B rows ArgTop-l_p
 *   A = apb_attention_fwd(Q, K, V, slots 0..host_idx-1)
 *   H1 = H + concat_heads(A) W_o^T;  y = RMSNorm(H1; ln2)
 *   out = H1 + (SiLU(y W_gate^T) * (y W_up^T)) W_down^T
 * RMSNorm(h)_c = h_c / sqrt(mean(h^2) + eps) * ln_c.  RoPE rotates the pair
 * (j, j + d/2) of every Q and K head by pos[t] * theta^(-2j/d).
 * ------------------------------------------------------------------------ */
typedef struct {
  apb_problem_t attn;     /* the host share (H, host_idx, La, Lb, l_p, heads) */
  int32_t hidden;         /* D >= 64, a multiple of 64                       */
  int32_t intermediate;   /* I >= 64, a multiple of 64 (FFN)                 */
  int32_t scorer_hidden;  /* retaining head's hidden units, as for
                             apb_retaining_scores (1024 in the paper)         */
  float rms_eps;          /* > 0                                             */
  float rope_theta;       /* > 1                                             */
} apb_layer_problem_t;

/* Weights of one layer, all caller-owned device memory, bf16 row-major
 * (rows = outputs) unless noted. */
typedef struct {
  const uint16_t* ln1;     /* [D]                                            */
  const uint16_t* w_qkv;   /* [(n_q + 2 n_kv) d][D]: Q heads, K heads, V heads */
  const uint16_t* w_o;     /* [D][n_q d]                                     */
  const uint16_t* ln2;     /* [D]                                            */
  const uint16_t* w_gate;  /* [I][D]                                         */
  const uint16_t* w_up;    /* [I][D]                                         */
  const uint16_t* w_down;  /* [D][I]                                         */
  const uint16_t* r_w1;    /* retaining head W1 bf16 [hidden_r][(n_q + 2 n_kv) d] */
  const float* r_b1;       /* fp32 [hidden_r]                                */
  const float* r_w2;       /* fp32 [n_kv][hidden_r]                          */
  const float* r_b2;       /* fp32 [n_kv]                                    */
} apb_layer_weights_t;

/* Host-only checks of a layer problem (no HIP call): the host share as in
 * apb_validate_problem, the retaining head as in apb_validate_scorer, D and
 * I multiples of 64, eps > 0, theta > 1. */
apb_status_t apb_validate_layer(const apb_layer_problem_t* p);

/* Bytes of device workspace apb_layer_fwd needs (host only). */
apb_status_t apb_layer_workspace_size(const apb_layer_problem_t* p, uint64_t* bytes);

/* Matrix-product FLOPs of one apb_layer_fwd call: the QKV, O and three FFN
 * products (2 flops per multiply-add), the retaining head's two layers and
 * the unmasked attention (apb_attention_flops).  Host-only; -1 if invalid. */
double apb_layer_flops(const apb_layer_problem_t* p);

/*
 * apb_layer_fwd -- one host's layer (Alg. 2).  T = La + Lb rows.
 *
 *   w           weights (above); every pointer required.
 *   hidden_in   bf16 [T][D]    anchor rows then local rows.
 *   positions   int32 [T]      RoPE position of every row.
 *   k_cache, v_cache  bf16 [n_kv][T][d]  out: the layer's KV cache (Alg. 2
 *                              returns it), K after RoPE.
 *   pass_k, pass_v    bf16 [H][n_kv][l_p][d] rank-major passing buffer:
 *                              slots 0..host_idx-1 are read (the earlier
 *                              hosts' blocks, already rotated), slot
 *                              host_idx is written (this host's block).
 *                              May be NULL only when l_p == 0.
 *   hidden_out  bf16 [T][D]    out.
 *   workspace   >= apb_layer_workspace_size() bytes, 16-byte aligned.
 * Arithmetic: bf16 operands and intermediates (x, Q/K/V, A, H1, y and the
 * SwiGLU product are stored in bf16), fp32 accumulation, norms, RoPE angles
 * in fp64 with fp32 rotation, residual sums in fp32 before rounding.
 */
apb_status_t apb_layer_fwd(const apb_layer_problem_t* p, const apb_layer_weights_t* w,
                           const uint16_t* hidden_in, const int32_t* positions,
                           uint16_t* k_cache, uint16_t* v_cache, uint16_t* pass_k,
                           uint16_t* pass_v, uint16_t* hidden_out, void* workspace,
                           uint64_t workspace_bytes, void* stream);

/* Host-only checks of a problem description (no HIP call). */
apb_status_t apb_validate_problem(const apb_problem_t* p);

/* Unmasked attention FLOPs of one call: 4*d per visible (query, key) pair
 * per query head, visible pairs La(La+1)/2 + Lb(La+Lp) + Lb(Lb+1)/2 with
 * Lp = host_idx*l_p.  Host-only; returns -1 for an invalid problem. */
double apb_attention_flops(const apb_problem_t* p);

/* Static text for a status code (never NULL). */
const char* apb_status_string(int status);

/* Text of the last HIP error seen by this thread ("" if none). */
const char* apb_last_error(void);

/* APB_ABI_VERSION of the built library. */
int apb_abi_version(void);

#ifdef __cplusplus
}
#endif

#endif /* APB_H_ */
