"""fp64 CPU oracle for the decoding stage of APB (stage 2, Alg. 3).

TEST INFRASTRUCTURE ONLY, like the rest of ``oracle/``: only ``tests/``,
``__graft_entry__.smoke()`` and the CPU-baseline leg of ``bench.py`` may use
it, and it shares no code with the HIP path.

What it computes, written as the plain definitions:

* ``decode_attention_ref`` -- one host's exact attention for the new tokens
  of a decoding step (Alg. 3, the two attention lines): every host attends
  the new tokens' queries to its own KV cache (its local block, Alg. 1 keeps
  K_h, V_h); the last host first appends the new tokens' own K/V to its cache.
  Reading (the paper does not spell it out): when several new tokens are
  processed at once (the question tokens at the first step), new token j
  sees the whole cache and new tokens 0..j, i.e. causal attention among the
  new tokens.  Returns the host's partial output A_h and its natural-log
  LSE per (query head, new token), the pair that Gather collects.
* ``merge_ref`` -- MergeScore (Alg. 3): the exact combination of partial
  softmax results, lse = ln sum_h exp(lse_h) and
  A = sum_h exp(lse_h - lse) A_h; a part with lse = -inf (no keys) adds
  nothing.
* ``stage2_ref`` -- the whole decoding-stage attention over H hosts on one
  machine: every host's partial, then the merge.

Scale defaults to 1/sqrt(d) (Eq. 1).  GQA maps query head i to KV head
i // (n_q / n_kv).  Every function is pinned by ``tests/test_decode_pins.py``.
"""
from __future__ import annotations

import math

import numpy as np

from .apb_oracle import bf16_to_f64


def decode_attention_ref(q, k_cache, v_cache, k_new=None, v_new=None, *, scale=None):
    """One host's stage-2 attention, fp64.

    q [n_q, n_new, d]; k_cache/v_cache [n_kv, Lc, d]; k_new/v_new [n_kv,
    n_new, d] or None (only the last host appends them); all bf16 bits (or
    floats for hand-written cases).  Returns (A [n_q, n_new, d], lse [n_q,
    n_new]); rows that see no key get A = 0 and lse = -inf."""
    n_q, n_new, d = q.shape
    n_kv, lc, _ = k_cache.shape
    if n_q % n_kv:
        raise ValueError("n_q must be a multiple of n_kv")
    if (k_new is None) != (v_new is None):
        raise ValueError("k_new and v_new go together")
    g = n_q // n_kv
    if scale is None:
        scale = 1.0 / math.sqrt(d)
    kc, vc = bf16_to_f64(k_cache), bf16_to_f64(v_cache)
    if k_new is not None:
        kc = np.concatenate([kc, bf16_to_f64(k_new)], axis=1)
        vc = np.concatenate([vc, bf16_to_f64(v_new)], axis=1)
    # keys visible to new token j: the cache, plus new tokens 0..j if appended
    ends = lc + (np.arange(n_new) + 1 if k_new is not None else np.zeros(n_new, np.int64))
    out = np.zeros((n_q, n_new, d))
    lse = np.full((n_q, n_new), -np.inf)
    for h in range(n_q):
        kv = h // g
        qh = bf16_to_f64(q[h])
        z = (qh @ kc[kv].T) * scale
        z[np.arange(kc.shape[1])[None, :] >= ends[:, None]] = -np.inf
        for j in range(n_new):
            if ends[j] == 0:
                continue
            m = z[j].max()
            p = np.exp(z[j] - m)
            l = p.sum()
            out[h, j] = (p @ vc[kv]) / l
            lse[h, j] = m + math.log(l)
    return out, lse


def merge_ref(a_parts, lse_parts):
    """MergeScore (Alg. 3).  a_parts [P, ..., d], lse_parts [P, ...] (fp64 or
    fp32).  Returns (A [..., d], lse [...]) in fp64."""
    a = np.asarray(a_parts, dtype=np.float64)
    l = np.asarray(lse_parts, dtype=np.float64)
    m = l.max(axis=0)
    safe_m = np.where(np.isfinite(m), m, 0.0)
    w = np.exp(l - safe_m[None])  # exp(-inf) = 0 drops empty parts
    tot = w.sum(axis=0)
    with np.errstate(invalid="ignore", divide="ignore"):
        out = (w[..., None] * a).sum(axis=0) / tot[..., None]
        lse = safe_m + np.log(tot)
    out = np.where(tot[..., None] > 0, out, 0.0)
    lse = np.where(tot > 0, lse, -np.inf)
    return out, lse


def stage2_ref(q, caches, k_new, v_new, *, scale=None):
    """Decoding-stage attention over H hosts (Alg. 3): ``caches`` is a list
    (host order) of (k_cache, v_cache); the last host also attends the new
    tokens' K/V.  Returns the merged (A, lse) and the per-host partials."""
    parts = []
    for h, (kc, vc) in enumerate(caches):
        last = h == len(caches) - 1
        parts.append(decode_attention_ref(q, kc, vc, k_new if last else None,
                                          v_new if last else None, scale=scale))
    a, lse = merge_ref(np.stack([p[0] for p in parts]), np.stack([p[1] for p in parts]))
    return a, lse, parts

