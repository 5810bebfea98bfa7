"""fp64 CPU oracle for one host's share of APB prefill attention.

TEST INFRASTRUCTURE ONLY: this module is the checker.  Only ``tests/``,
``__graft_entry__.smoke()`` and the CPU-baseline leg of ``bench.py`` may use
it.  It shares no code with the HIP path (no kernels, no headers, no tables,
no pre- or post-processing); the only thing both sides share is the seeded
input generator, which holds none of the method's arithmetic.

What it computes, written as the plain definitions from the paper:

* ``attention_ref`` -- the modified-mask attention of Eq. 2 (Sec. 3.6): the
  queries are the anchor and local rows [A; B], the keys and values are the
  anchor, passing and local rows [A; P; B] in that order, softmax over the
  scaled dot products (Eq. 1, scale 1/sqrt(d_m) with d_m the per-head size)
  under the mask M'.  Reading of M' (the framework figure is not available):
  causal attention over the concatenation [A; P; B] with the query rows of P
  removed -- anchor rows see the anchor causally, local rows see all of A, all
  of P and B causally.  Masked entries leave the softmax (additive -inf).
  Also returns the natural-log LSE of every row, the quantity the decode-stage
  merge of partial results needs (Alg. 3).
* ``topk_ref`` -- ArgTop-l_p of the retaining-head scores (Sec. 3.4; Alg. 2,
  compression step): per KV head the l_p largest fp32 scores, ties broken
  toward the lower index, -0 equal to +0, NaN below -inf, returned in
  ascending index order.
* ``gather_ref`` -- the compressed block K^C = K_h[idx], V^C = V_h[idx]
  (Sec. 3.4) as bit copies.
* ``simulate_hosts_ref`` -- Alg. 2 across hosts on one machine: every earlier
  host compresses its local block, the blocks are concatenated in host order
  into the passing block (Sec. 3.5), then the current host's attention runs.

Notation: ``host_idx`` is 0-based (= number of previous hosts; the paper's h
is host_idx + 1), La anchor rows, Lb local rows, l_p rows per previous host,
Lp = host_idx * l_p, GQA maps query head i to KV head i // (n_q / n_kv).

Every function here is pinned by the CPU tests against brute force, a
library special case, closed forms, hand-worked toys and invariants.
"""
from __future__ import annotations

import math

import numpy as np


def bf16_to_f64(bits: np.ndarray) -> np.ndarray:
    """Exact value of bf16 bit patterns: the 16 bits are the top half of an
    IEEE fp32 word, so widening to fp32 and then fp64 is exact.  Arrays that
    are already floating point (hand-written toy cases) pass through as fp64."""
    a = np.asarray(bits)
    if a.dtype.kind == "f":
        return a.astype(np.float64)
    u32 = a.astype(np.uint16).astype(np.uint32) << np.uint32(16)
    return u32.view(np.float32).astype(np.float64)


def visible_end(r: np.ndarray | int, anchor_len: int, passing_rows: int):
    """One past the last key a query row sees (Eq. 2 under M').

    Row r < La is anchor token r at concatenated position r; row r >= La is
    local token r - La at concatenated position r + Lp (after A and P).
    Causal attention over [A; P; B] lets a row see every key up to and
    including its own position."""
    r = np.asarray(r)
    return np.where(r < anchor_len, r, r + passing_rows) + 1


def assemble_kv(x_local: np.ndarray, x_pass: np.ndarray, anchor_len: int) -> np.ndarray:
    """Concatenate [A; P; B] per KV head (Eq. 2 key/value order; the passing
    block is the earlier hosts' compressed blocks in host order, Sec. 3.5).

    x_local [n_kv, La+Lb, d] (anchor rows first), x_pass [host_idx, n_kv, l_p, d].
    Returns fp64 [n_kv, La+Lp+Lb, d]."""
    loc = bf16_to_f64(x_local)
    parts = [loc[:, :anchor_len]]
    for s in range(x_pass.shape[0]):
        parts.append(bf16_to_f64(x_pass[s]))
    parts.append(loc[:, anchor_len:])
    return np.concatenate(parts, axis=1)


def attention_ref(q, k, v, k_pass, v_pass, *, anchor_len, scale=None,
                  heads=None, rows=None, row_block=256):
    """Modified-mask attention of one host share, in fp64 (Eq. 1, Eq. 2).

    q [n_q, La+Lb, d], k/v [n_kv, La+Lb, d], k_pass/v_pass
    [host_idx, n_kv, l_p, d], all bf16 bits.  ``scale`` defaults to
    1/sqrt(d).  ``heads``/``rows`` restrict the output to a subset (the rest
    of the result is not computed; returned arrays are indexed by the
    subset).  Returns (O [len(heads), len(rows), d], LSE [len(heads),
    len(rows)]) in fp64, LSE in natural log."""
    n_q, m_rows, d = q.shape
    n_kv = k.shape[0]
    if n_q % n_kv:
        raise ValueError("n_q must be a multiple of n_kv")
    g = n_q // n_kv
    lp = k_pass.shape[0] * k_pass.shape[2]
    if scale is None:
        scale = 1.0 / math.sqrt(d)
    heads = np.arange(n_q) if heads is None else np.asarray(heads)
    rows = np.arange(m_rows) if rows is None else np.asarray(rows)
    out = np.empty((len(heads), len(rows), d))
    lse = np.empty((len(heads), len(rows)))
    kc_cache = {}
    for hi, h in enumerate(heads):
        kv = int(h) // g
        if kv not in kc_cache:
            kc_cache = {kv: (assemble_kv(k[kv:kv + 1], k_pass[:, kv:kv + 1], anchor_len)[0],
                             assemble_kv(v[kv:kv + 1], v_pass[:, kv:kv + 1], anchor_len)[0])}
        kc, vc = kc_cache[kv]
        qh = bf16_to_f64(q[h])
        if qh.shape[-1] != kc.shape[-1]:
            raise ValueError("head_dim mismatch")
        for b0 in range(0, len(rows), row_block):
            rb = rows[b0:b0 + row_block]
            ends = visible_end(rb, anchor_len, lp)
            n_vis = int(ends.max())
            z = (qh[rb] @ kc[:n_vis].T) * scale
            z[np.arange(n_vis)[None, :] >= ends[:, None]] = -np.inf
            mx = z.max(axis=1, keepdims=True)
            p = np.exp(z - mx)
            l = p.sum(axis=1, keepdims=True)
            out[hi, b0:b0 + len(rb)] = (p @ vc[:n_vis]) / l
            lse[hi, b0:b0 + len(rb)] = (mx + np.log(l))[:, 0]
    return out, lse


def topk_ref(scores: np.ndarray, l_p: int) -> np.ndarray:
    """ArgTop-l_p per KV head (Sec. 3.4; Alg. 2).

    scores fp32 [n_kv, Lb].  Ranking: larger score first; equal scores (with
    -0 equal to +0) go to the lower index; NaN ranks below every number,
    -inf included.  Returns int32 [n_kv, l_p] in ascending index order."""
    scores = np.asarray(scores, dtype=np.float32)
    n_kv, lb = scores.shape
    if not 0 <= l_p <= lb:
        raise ValueError("need 0 <= l_p <= Lb")
    out = np.empty((n_kv, l_p), dtype=np.int32)
    idx = np.arange(lb)
    for h in range(n_kv):
        s = scores[h].astype(np.float64)
        nan = np.isnan(s)
        neg = np.where(nan, 0.0, -s)  # the sort compares values: -0 == +0
        order = np.lexsort((idx, neg, nan))  # last key is the primary one
        out[h] = np.sort(order[:l_p])
    return out


def gather_ref(x_local: np.ndarray, idx: np.ndarray, anchor_len: int) -> np.ndarray:
    """Compressed block rows x_h[idx] (Sec. 3.4): bit copies of the selected
    local rows.  x_local [n_kv, La+Lb, d] bf16 bits, idx [n_kv, l_p] local
    indices.  Returns [n_kv, l_p, d] bf16 bits."""
    n_kv = x_local.shape[0]
    return np.stack([x_local[h, anchor_len + idx[h]] for h in range(n_kv)])


def compress_ref(scores, k, v, l_p, anchor_len):
    """The compressor C on one host: top-l_p selection, then the gather."""
    idx = topk_ref(scores, l_p)
    return idx, gather_ref(k, idx, anchor_len), gather_ref(v, idx, anchor_len)


def simulate_hosts_ref(q, k, v, scores, earlier_hosts, *, anchor_len, l_p,
                       heads=None, rows=None):
    """Alg. 2 over hosts 0..host_idx on one machine.

    ``earlier_hosts`` is a list (host order) of dicts with that host's local
    ``k``, ``v`` [n_kv, La+Lb, d] and ``scores`` [n_kv, Lb].  Each earlier host
    compresses its block; the results, concatenated in host order, form the
    passing block (the all-gather keeps only previous hosts, Sec. 3.5).  The
    current host compresses too (its block would go to later hosts) and then
    runs the modified attention.  Returns (O, LSE, own idx, own K^C, own V^C,
    k_pass, v_pass)."""
    n_kv, _, d = k.shape
    kp = np.empty((len(earlier_hosts), n_kv, l_p, d), np.uint16)
    vp = np.empty_like(kp)
    for j, hb in enumerate(earlier_hosts):
        _, kp[j], vp[j] = compress_ref(hb["scores"], hb["k"], hb["v"], l_p, anchor_len)
    idx, kc, vc = compress_ref(scores, k, v, l_p, anchor_len)
    o, lse = attention_ref(q, k, v, kp, vp, anchor_len=anchor_len, heads=heads, rows=rows)
    return o, lse, idx, kc, vc, kp, vp


def attention_flops(n_q, head_dim, anchor_len, local_len, passing_rows) -> float:
    """Unmasked attention FLOPs: 4*d per visible (query, key) pair per query
    head (2*d for Q.K, 2*d for P.V).  Visible pairs per head: the anchor
    triangle, every local row against all of A and P, and the local
    triangle."""
    la, lb, lp = anchor_len, local_len, passing_rows
    pairs = la * (la + 1) // 2 + lb * (la + lp) + lb * (lb + 1) // 2
    return 4.0 * head_dim * n_q * pairs
