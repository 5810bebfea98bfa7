"""fp64 CPU oracle for the retaining-head scorer R (Sec. 3.4; Alg. 2,
compression step; App. B).

TEST INFRASTRUCTURE ONLY, like the rest of ``oracle/``: only ``tests/``,
``__graft_entry__.smoke()`` and the CPU-baseline leg of ``bench.py`` may use
it, and it shares no code with the HIP path.

The paper gives the compressor as Locret's retaining heads: small MLPs that
take [Q, K, V] of every local-block cache unit and return its importance
(Sec. 3.4), with intermediate size 1024 (App. B).  The architecture is not
restated, so this oracle adopts a reading: for local token t,

    x_t = [Q_0[t], ..., Q_{n_q-1}[t], K_0[t], ..., K_{n_kv-1}[t],
           V_0[t], ..., V_{n_kv-1}[t]]            ((n_q + 2 n_kv) * d features)
    h_t = SiLU(W1 x_t + b1)                        (hidden units, 1024 in the paper)
    s_t = W2 h_t + b2                              (one score per KV head)

with SiLU(z) = z / (1 + exp(-z)), W1 [hidden][features], W2 [n_kv][hidden]
and biases b1 [hidden], b2 [n_kv].  Only local rows are scored (the anchor is
not compressed).  The trained weights are not available; the weights are
synthetic and the result is pinned at kernel level only.
"""
from __future__ import annotations

import numpy as np

from .apb_oracle import bf16_to_f64


def scorer_features(q, k, v, *, anchor_len):
    """x_t for every local token, fp64 [Lb, (n_q + 2 n_kv) d]."""
    parts = [bf16_to_f64(t)[:, anchor_len:] for t in (q, k, v)]  # [heads, Lb, d] each
    x = np.concatenate(parts, axis=0)                             # [n_q + 2 n_kv, Lb, d]
    return np.ascontiguousarray(x.transpose(1, 0, 2).reshape(x.shape[1], -1))


def silu(z):
    return z / (1.0 + np.exp(-z))


def retaining_scores_ref(q, k, v, w1, b1, w2, b2, *, anchor_len):
    """Scores fp64 [n_kv, Lb].  q [n_q, La+Lb, d], k/v [n_kv, La+Lb, d] bf16
    bits; w1 bf16 bits [hidden, features]; w2 [n_kv, hidden] and the biases
    as floats (fp32 on the device)."""
    x = scorer_features(q, k, v, anchor_len=anchor_len)
    h = silu(x @ bf16_to_f64(w1).T + np.asarray(b1, np.float64)[None, :])
    s = h @ np.asarray(w2, np.float64).T + np.asarray(b2, np.float64)[None, :]
    return np.ascontiguousarray(s.T)


def scorer_flops(n_q, n_kv, head_dim, local_len, hidden) -> float:
    """Multiply-adds x 2 of both layers (the activation is not counted)."""
    feats = (n_q + 2 * n_kv) * head_dim
    return 2.0 * local_len * feats * hidden + 2.0 * local_len * hidden * n_kv
