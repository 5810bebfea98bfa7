"""fp64 CPU oracle for one host's whole APB transformer layer (Alg. 2).

TEST INFRASTRUCTURE ONLY, like the rest of ``oracle/``: only ``tests/``,
``__graft_entry__.smoke()`` and the CPU-baseline leg of ``bench.py`` may use
it, and it shares no code with the HIP path.

Alg. 2 runs, per layer and host: the QKV projection of the anchor and local
hidden states, the retaining head R over the local block's [Q, K, V], the
top-l_p selection and gather of the compressed block, the all-gather (here:
the earlier hosts' blocks are given), attention over [A; P; B] under M', and
the FFN.  The layer around attention is the model's own (Llama-style, the
models of Sec. 4.1); the paper does not restate it, so this oracle adopts a
reading, written out as plain definitions:

    x   = RMSNorm(H; g1)                         g1, g2 per-channel gains
    Q, K, V = split(x W_qkv^T) into heads        head-major [heads, rows, d]
    Q, K = RoPE(Q, pos), RoPE(K, pos)            rotate-half pairs (j, j+d/2)
    s   = R([Q_B, K_B, V_B])                     retaining head, local rows
    idx = ArgTop-l_p(s); K^C, V^C = K_B[idx], V_B[idx]
    A   = Attention(Q, [K_A; K_P; K_B], [V_A; V_P; V_B])   (Eq. 2)
    H1  = H + concat_heads(A) W_o^T
    y   = RMSNorm(H1; g2)
    out = H1 + (SiLU(y W_gate^T) * (y W_up^T)) W_down^T

RMSNorm(h)_c = h_c / sqrt(mean_c(h_c^2) + eps) * g_c.  RoPE rotates the pair
(x_j, x_{j+d/2}) of every head by the angle pos * theta^(-2j/d), j < d/2.
The retaining head sees the same post-RoPE Q/K that attention and the KV
cache use.  The passing rows arrive already rotated (each keeps its source
position).
"""
from __future__ import annotations

import numpy as np

from .apb_oracle import attention_ref, bf16_to_f64, topk_ref
from .scorer_oracle import retaining_scores_ref, silu


def rmsnorm_ref(h, gain, eps):
    """Row-wise RMSNorm in fp64: h [rows, D], gain [D] (bf16 bits or floats)."""
    h = bf16_to_f64(h)
    ms = np.mean(h * h, axis=-1, keepdims=True)
    return h / np.sqrt(ms + eps) * bf16_to_f64(gain)[None, :]


def rope_ref(x, pos, theta):
    """Rotary embedding of head-major x [heads, rows, d] (fp64) at integer
    positions pos [rows]: pair (j, j + d/2) rotated by pos * theta^(-2j/d)."""
    x = np.asarray(x, dtype=np.float64)
    d = x.shape[-1]
    half = d // 2
    inv_freq = theta ** (-2.0 * np.arange(half) / d)
    ang = np.asarray(pos, dtype=np.float64)[:, None] * inv_freq[None, :]  # [rows, d/2]
    c, s = np.cos(ang)[None], np.sin(ang)[None]
    lo, hi = x[..., :half], x[..., half:]
    return np.concatenate([lo * c - hi * s, hi * c + lo * s], axis=-1)


def swiglu_ffn_ref(y, w_gate, w_up, w_down):
    """(SiLU(y W_gate^T) * (y W_up^T)) W_down^T in fp64; y [rows, D]."""
    g = y @ bf16_to_f64(w_gate).T
    u = y @ bf16_to_f64(w_up).T
    return (silu(g) * u) @ bf16_to_f64(w_down).T


def qkv_ref(x, w_qkv, n_q, n_kv, head_dim):
    """Projection x W_qkv^T split into head-major Q [n_q, rows, d], K, V
    [n_kv, rows, d]; output features are ordered Q heads, K heads, V heads."""
    y = x @ bf16_to_f64(w_qkv).T  # [rows, (n_q + 2 n_kv) d]
    rows = y.shape[0]
    heads = y.reshape(rows, n_q + 2 * n_kv, head_dim).transpose(1, 0, 2)
    return heads[:n_q], heads[n_q:n_q + n_kv], heads[n_q + n_kv:]


def layer_ref(hidden, pos, w, k_pass, v_pass, *, anchor_len, pass_len, n_q, n_kv, head_dim,
              eps, theta, rows=None):
    """One host's APB layer in fp64.

    hidden [La+Lb, D] bf16 bits; pos [La+Lb] ints; ``w`` a dict of weights
    (bf16 bits: ln1, w_qkv, w_o, ln2, w_gate, w_up, w_down, scorer w1;
    floats: scorer b1, w2, b2); k_pass/v_pass [host_idx, n_kv, l_p, d] bf16
    bits (already rotated).  ``rows`` restricts the attention and everything
    after it to a subset of rows (Q/K/V, scores and the selection are always
    computed for every row).  Returns a dict: q, k, v (post-RoPE, fp64), scores
    [n_kv, Lb], idx [n_kv, l_p], attn [n_q, len(rows), d], h1 and out
    [len(rows), D]."""
    h = bf16_to_f64(hidden)
    x = rmsnorm_ref(h, w["ln1"], eps)
    q, k, v = qkv_ref(x, w["w_qkv"], n_q, n_kv, head_dim)
    q = rope_ref(q, pos, theta)
    k = rope_ref(k, pos, theta)
    scores = retaining_scores_ref(q, k, v, w["w1"], w["b1"], w["w2"], w["b2"],
                                  anchor_len=anchor_len)
    idx = topk_ref(scores.astype(np.float32), pass_len)
    sel = np.arange(h.shape[0]) if rows is None else np.asarray(rows)
    attn, _ = attention_ref(q, k, v, k_pass, v_pass, anchor_len=anchor_len, rows=sel)
    a_flat = attn.transpose(1, 0, 2).reshape(len(sel), n_q * head_dim)
    h1 = h[sel] + a_flat @ bf16_to_f64(w["w_o"]).T
    y = rmsnorm_ref(h1, w["ln2"], eps)
    out = h1 + swiglu_ffn_ref(y, w["w_gate"], w["w_up"], w["w_down"])
    return dict(q=q, k=k, v=v, scores=scores, idx=idx, attn=attn, h1=h1, out=out)


def layer_flops(rows, hidden, intermediate, n_q, n_kv, head_dim, attn_flops, scorer_flops=0.0):
    """Matrix-multiply FLOPs of one host's layer: QKV and O projections, the
    three FFN products, attention (given, unmasked pairs) and the retaining
    head (given).  Norms, RoPE and activations are not counted, as in the
    paper's FLOPs table."""
    qkv = 2.0 * rows * hidden * (n_q + 2 * n_kv) * head_dim
    o = 2.0 * rows * n_q * head_dim * hidden
    ffn = 3 * 2.0 * rows * hidden * intermediate
    return qkv + o + ffn + attn_flops + scorer_flops


def apb_table_flops_per_layer(n, d_model, g, intermediate, n_hosts, l_a, l_p):
    """The paper's FLOPs-per-forward count for APB (App. C, FLOPs table) for
    one layer (L = 1), summed over all H hosts, restated so that the layer's
    own per-host count can be compared with it term by term: host 1 projects
    and runs the FFN on its n/H block, every later host on its block plus the
    anchor, attention is counted as causal over those rows, and the passing
    rows add the last term."""
    H = n_hosts
    blk = n / H
    first = 4 * (1 + 1 / g + 0.5 * n / (H * d_model) + 1.5 * intermediate / d_model) * blk * d_model ** 2
    rest = 4 * (H - 1) * (1 + 1 / g + 0.5 * (blk + l_a) / d_model + 1.5 * intermediate / d_model) \
        * (blk + l_a) * d_model ** 2
    passing = l_p * H * (H - 1) * (blk + l_a) * d_model
    return first + rest + passing

