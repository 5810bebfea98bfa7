"""Seeded synthetic workloads for one host's share of APB prefill attention.

This module is shared by the GPU path, the oracle-based tests and the bench.
It draws random numbers and rounds them to the storage formats; it holds none
of the method's arithmetic (no attention, no selection, no masking).

Shapes follow the paper's problem statement: a host holds an anchor block of
La rows (query tokens plus the first l_a document tokens, Sec. 3.3), a local
block of Lb = l_b rows (Sec. 3.3), and receives l_p compressed rows from each
previous host (Sec. 3.4-3.5).  ``host_idx`` is 0-based and equals the number
of previous hosts, so the passing block holds Lp = host_idx * l_p rows.

Every tensor is head-major ``[heads, rows, d]`` with d contiguous, stored as
bf16 bit patterns (``uint16``).  Scores are fp32 ``[n_kv, Lb]``.
"""
from __future__ import annotations

import dataclasses
import math

import numpy as np


@dataclasses.dataclass(frozen=True)
class Problem:
    """One host's share of one attention layer (Alg. 2 inputs)."""

    n_hosts: int
    host_idx: int
    anchor_len: int
    local_len: int
    pass_len: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int

    @property
    def rows(self) -> int:
        """Query rows on this host: anchor then local block (Eq. 2)."""
        return self.anchor_len + self.local_len

    @property
    def passing_rows(self) -> int:
        """Lp: compressed rows received from the host_idx previous hosts."""
        return self.host_idx * self.pass_len

    @property
    def key_rows(self) -> int:
        return self.anchor_len + self.passing_rows + self.local_len

    @property
    def group(self) -> int:
        return self.n_q_heads // self.n_kv_heads


@dataclasses.dataclass(frozen=True)
class Workload:
    """A named problem plus the value distributions used to fill it."""

    name: str
    problem: Problem
    outlier_k: bool = False  # 2% of K channels scaled x8
    zipf_scores: bool = False  # scores ~ Zipf(1.5) instead of N(0, 1)


# The five workloads: a tiny case, and layers shaped like Llama-3.1-8B,
# Qwen-2.5-14B and Yi-34B at the context lengths and l_a / l_p / l_b the
# paper uses (App. B, Table of sequence hyperparameters; Sec. 4.1 model list).
WORKLOADS = {
    "tiny": Workload(
        "tiny", Problem(4, 2, 128, 512, 32, 4, 1, 64)),
    "llama8b_32k": Workload(
        "llama8b_32k", Problem(4, 3, 2048, 8192, 1024, 32, 8, 128)),
    "llama8b_128k": Workload(
        "llama8b_128k", Problem(8, 7, 4096, 16384, 2048, 32, 8, 128),
        outlier_k=True),
    "qwen14b_256k": Workload(
        "qwen14b_256k", Problem(8, 7, 4096, 32768, 4096, 40, 8, 128)),
    "yi34b_512k": Workload(
        "yi34b_512k", Problem(8, 7, 8192, 65536, 8192, 56, 8, 128),
        zipf_scores=True),
}


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round fp32 to bf16 (round to nearest, ties to even); return uint16 bits."""
    b = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    rounded = b + np.uint32(0x7FFF) + ((b >> np.uint32(16)) & np.uint32(1))
    return (rounded >> np.uint32(16)).astype(np.uint16)


def bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    """Exact widening of bf16 bit patterns to fp32 (used only for display
    and by generators that post-scale values; never by the oracle)."""
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def _normal_bf16(rng: np.random.Generator, shape, scale_cols=None) -> np.ndarray:
    """N(0,1) fp32 draws rounded to bf16, drawn head by head so that a
    prefix of heads never depends on how many heads follow."""
    out = np.empty(shape, dtype=np.uint16)
    for h in range(shape[0]):
        x = rng.standard_normal(shape[1:], dtype=np.float32)
        if scale_cols is not None:
            x[..., scale_cols[h]] *= np.float32(8.0)
        out[h] = f32_to_bf16_bits(x)
    return out


def outlier_channels(prob: Problem, seed: int) -> np.ndarray:
    """ceil(2% of d) K channels per KV head, chosen by a seeded RNG."""
    n_out = math.ceil(0.02 * prob.head_dim)
    rng = np.random.default_rng(np.random.SeedSequence(seed).spawn(7)[6])
    return np.stack([np.sort(rng.choice(prob.head_dim, n_out, replace=False))
                     for _ in range(prob.n_kv_heads)])


def make_inputs(wl: Workload, seed: int = 0) -> dict:
    """Generate every input of one host share.

    Per-tensor streams come from ``SeedSequence(seed).spawn(7)`` in the order
    Q, K, V, K_pass, V_pass, scores, outlier channels.  Returns a dict with
    ``q`` [n_q, La+Lb, d], ``k``/``v`` [n_kv, La+Lb, d] (local rows start at
    La), ``k_pass``/``v_pass`` [host_idx, n_kv, l_p, d] (rank-major slots of
    the earlier hosts' compressed blocks), all bf16 bits, and ``scores``
    fp32 [n_kv, Lb].
    """
    p = wl.problem
    ss = np.random.SeedSequence(seed).spawn(7)
    cols = outlier_channels(p, seed) if wl.outlier_k else None
    q = _normal_bf16(np.random.default_rng(ss[0]), (p.n_q_heads, p.rows, p.head_dim))
    k = _normal_bf16(np.random.default_rng(ss[1]), (p.n_kv_heads, p.rows, p.head_dim), cols)
    v = _normal_bf16(np.random.default_rng(ss[2]), (p.n_kv_heads, p.rows, p.head_dim))
    kp_rng = np.random.default_rng(ss[3])
    vp_rng = np.random.default_rng(ss[4])
    k_pass = np.empty((p.host_idx, p.n_kv_heads, p.pass_len, p.head_dim), np.uint16)
    v_pass = np.empty_like(k_pass)
    for s in range(p.host_idx):
        k_pass[s] = _normal_bf16(kp_rng, k_pass.shape[1:], cols)
        v_pass[s] = _normal_bf16(vp_rng, v_pass.shape[1:])
    s_rng = np.random.default_rng(ss[5])
    if wl.zipf_scores:
        scores = s_rng.zipf(1.5, size=(p.n_kv_heads, p.local_len)).astype(np.float32)
    else:
        scores = s_rng.standard_normal((p.n_kv_heads, p.local_len), dtype=np.float32)
    return dict(q=q, k=k, v=v, k_pass=k_pass, v_pass=v_pass, scores=scores,
                outlier_cols=cols)


def make_host_blocks(wl: Workload, seed: int = 0) -> list:
    """Synthetic local blocks of every earlier host (for the multi-host
    simulation): for host j < host_idx, K/V [n_kv, La+Lb, d] and scores
    [n_kv, Lb].  Stream ``SeedSequence(seed + 1000 + j)``."""
    p = wl.problem
    cols = outlier_channels(p, seed) if wl.outlier_k else None
    out = []
    for j in range(p.host_idx):
        ss = np.random.SeedSequence(seed + 1000 + j).spawn(3)
        k = _normal_bf16(np.random.default_rng(ss[0]), (p.n_kv_heads, p.rows, p.head_dim), cols)
        v = _normal_bf16(np.random.default_rng(ss[1]), (p.n_kv_heads, p.rows, p.head_dim))
        rng = np.random.default_rng(ss[2])
        if wl.zipf_scores:
            sc = rng.zipf(1.5, size=(p.n_kv_heads, p.local_len)).astype(np.float32)
        else:
            sc = rng.standard_normal((p.n_kv_heads, p.local_len), dtype=np.float32)
        out.append(dict(k=k, v=v, scores=sc))
    return out


# ----------------------------------------------------------- decoding stage
@dataclasses.dataclass(frozen=True)
class DecodeWorkload:
    """One decoding step (Alg. 3) over H hosts: every host's cache is its
    local block (Alg. 1 keeps K_h, V_h), the last host also appends the new
    tokens' K/V."""

    name: str
    n_hosts: int
    cache_len: int  # rows per host cache (the local block length l_b)
    n_new: int      # new tokens this step
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    outlier_k: bool = False

    @property
    def rows(self) -> int:
        return self.n_q_heads * self.n_new


# The 128K Llama-8B-shaped layer after its prefill (H = 8 hosts of 16384
# cached rows): one generated token, and the first step that feeds the
# question tokens (64 of them here).
DECODE_WORKLOADS = {
    "tiny_decode": DecodeWorkload("tiny_decode", 4, 512, 3, 4, 1, 64),
    "llama8b_128k_decode": DecodeWorkload("llama8b_128k_decode", 8, 16384, 1, 32, 8, 128,
                                          outlier_k=True),
    "llama8b_128k_question": DecodeWorkload("llama8b_128k_question", 8, 16384, 64, 32, 8, 128,
                                            outlier_k=True),
}


def make_decode_case(n_q: int, n_kv: int, d: int, cache_lens, n_new: int, seed: int = 0,
                     outlier_k: bool = False) -> dict:
    """Inputs of one decoding step over len(cache_lens) hosts.

    Streams: ``SeedSequence(seed).spawn(4 + 2*H)`` in the order Q, K_new,
    V_new, outlier channels, then K and V of host 0, 1, ...  Returns ``q``
    [n_q, n_new, d], ``k_new``/``v_new`` [n_kv, n_new, d], ``caches`` (list of
    (k, v), each [n_kv, Lc_h, d]), all bf16 bits."""
    H = len(cache_lens)
    ss = np.random.SeedSequence(seed).spawn(4 + 2 * H)
    cols = None
    if outlier_k:
        n_out = math.ceil(0.02 * d)
        rng = np.random.default_rng(ss[3])
        cols = np.stack([np.sort(rng.choice(d, n_out, replace=False)) for _ in range(n_kv)])
    q = _normal_bf16(np.random.default_rng(ss[0]), (n_q, n_new, d))
    k_new = _normal_bf16(np.random.default_rng(ss[1]), (n_kv, n_new, d), cols)
    v_new = _normal_bf16(np.random.default_rng(ss[2]), (n_kv, n_new, d))
    caches = []
    for h, lc in enumerate(cache_lens):
        kc = _normal_bf16(np.random.default_rng(ss[4 + 2 * h]), (n_kv, lc, d), cols)
        vc = _normal_bf16(np.random.default_rng(ss[5 + 2 * h]), (n_kv, lc, d))
        caches.append((kc, vc))
    return dict(q=q, k_new=k_new, v_new=v_new, caches=caches)


def make_decode_inputs(wl: DecodeWorkload, seed: int = 0, hosts=None) -> dict:
    """``make_decode_case`` for a named workload; ``hosts`` limits how many
    host caches are drawn (the first ones), e.g. 1 for the last host alone."""
    h = wl.n_hosts if hosts is None else hosts
    return make_decode_case(wl.n_q_heads, wl.n_kv_heads, wl.head_dim, [wl.cache_len] * h,
                            wl.n_new, seed, wl.outlier_k)


# ----------------------------------------------------- retaining-head scorer
SCORER_HIDDEN = 1024  # intermediate size of the retaining heads (App. B)


def make_scorer_weights(n_q: int, n_kv: int, head_dim: int, hidden: int = SCORER_HIDDEN,
                        seed: int = 0) -> dict:
    """Synthetic retaining-head weights (the trained ones are not available).

    Streams ``SeedSequence(seed + 2000).spawn(4)``: W1 bf16 bits [hidden,
    (n_q + 2 n_kv) d] ~ N(0, 1/features), b1 fp32 [hidden] ~ N(0, 0.1^2),
    W2 fp32 [n_kv, hidden] ~ N(0, 1/hidden), b2 fp32 [n_kv] ~ N(0, 0.1^2),
    so that with N(0, 1) inputs the hidden pre-activations and the scores
    are of order one."""
    feats = (n_q + 2 * n_kv) * head_dim
    ss = np.random.SeedSequence(seed + 2000).spawn(4)
    r = [np.random.default_rng(s) for s in ss]
    w1 = np.empty((hidden, feats), np.uint16)
    for j in range(hidden):
        w1[j] = f32_to_bf16_bits(r[0].standard_normal(feats, dtype=np.float32)
                                 * np.float32(1.0 / math.sqrt(feats)))
    b1 = (r[1].standard_normal(hidden, dtype=np.float32) * np.float32(0.1))
    w2 = (r[2].standard_normal((n_kv, hidden), dtype=np.float32)
          * np.float32(1.0 / math.sqrt(hidden)))
    b2 = (r[3].standard_normal(n_kv, dtype=np.float32) * np.float32(0.1))
    return dict(w1=w1, b1=b1, w2=w2, b2=b2)


# ------------------------------------------------------------ whole layer
@dataclasses.dataclass(frozen=True)
class LayerWorkload:
    """One host's whole transformer layer around the host share (Alg. 2):
    the attention problem plus the model's hidden size D, FFN intermediate
    size I, the retaining head's hidden size, RMSNorm eps and RoPE base."""

    name: str
    attn: Workload
    hidden: int
    intermediate: int
    scorer_hidden: int
    eps: float = 1e-5
    theta: float = 500000.0

    @property
    def problem(self) -> Problem:
        return self.attn.problem


# Llama-3.1-8B: D = 4096, I = 14336, 32/8 heads of 128; the tiny layer keeps
# the tiny host share with D = n_q * d = 256.
LAYER_WORKLOADS = {
    "tiny_layer": LayerWorkload("tiny_layer", WORKLOADS["tiny"], 256, 512, 256),
    "llama8b_32k_layer": LayerWorkload("llama8b_32k_layer", WORKLOADS["llama8b_32k"],
                                       4096, 14336, SCORER_HIDDEN),
    "llama8b_128k_layer": LayerWorkload("llama8b_128k_layer", WORKLOADS["llama8b_128k"],
                                        4096, 14336, SCORER_HIDDEN),
}


def layer_positions(p: Problem) -> np.ndarray:
    """Token positions of one host's rows (the RoPE input): anchor row r sits
    at position r; local row i of host h at La + h*Lb + i, i.e. the local
    blocks follow the anchor in document order."""
    pos = np.empty(p.rows, np.int32)
    pos[:p.anchor_len] = np.arange(p.anchor_len)
    pos[p.anchor_len:] = p.anchor_len + p.host_idx * p.local_len + np.arange(p.local_len)
    return pos


def _normal_matrix_bf16(rng: np.random.Generator, rows: int, cols: int, std: float) -> np.ndarray:
    out = np.empty((rows, cols), np.uint16)
    step = max(1, (1 << 22) // max(cols, 1))
    for r0 in range(0, rows, step):
        r1 = min(rows, r0 + step)
        out[r0:r1] = f32_to_bf16_bits(rng.standard_normal((r1 - r0, cols), dtype=np.float32)
                                      * np.float32(std))
    return out


def make_layer_inputs(lw: LayerWorkload, seed: int = 0) -> dict:
    """Inputs and synthetic weights of one host's layer.

    Streams ``SeedSequence(seed + 3000).spawn(11)`` in the order hidden,
    K_pass, V_pass, ln1, W_qkv, W_o, ln2, W_gate, W_up, W_down, (unused);
    the retaining head from ``make_scorer_weights(..., seed=seed)``.
    hidden [La+Lb, D] ~ N(0, 1); norm gains ~ 1 + N(0, 0.1^2); W_qkv, W_gate,
    W_up ~ N(0, 1/D); W_o ~ N(0, 1/(n_q d)); W_down ~ N(0, 1/I); passing
    K/V [host_idx, n_kv, l_p, d] ~ N(0, 1) (rows already rotated at their
    source positions).  All bf16 bits except the retaining head's fp32
    b1/w2/b2.  ``pos`` from ``layer_positions``."""
    p = lw.problem
    D, I = lw.hidden, lw.intermediate
    nqkv = (p.n_q_heads + 2 * p.n_kv_heads) * p.head_dim
    ss = np.random.SeedSequence(seed + 3000).spawn(11)
    r = [np.random.default_rng(s) for s in ss]
    hidden = _normal_matrix_bf16(r[0], p.rows, D, 1.0)
    k_pass = np.empty((p.host_idx, p.n_kv_heads, p.pass_len, p.head_dim), np.uint16)
    v_pass = np.empty_like(k_pass)
    for s in range(p.host_idx):
        k_pass[s] = _normal_bf16(r[1], k_pass.shape[1:])
        v_pass[s] = _normal_bf16(r[2], v_pass.shape[1:])
    gain = lambda rng: f32_to_bf16_bits(np.float32(1.0) + rng.standard_normal(D, dtype=np.float32)  # noqa: E731
                                        * np.float32(0.1))
    w = dict(
        ln1=gain(r[3]),
        w_qkv=_normal_matrix_bf16(r[4], nqkv, D, 1.0 / math.sqrt(D)),
        w_o=_normal_matrix_bf16(r[5], D, p.n_q_heads * p.head_dim,
                                1.0 / math.sqrt(p.n_q_heads * p.head_dim)),
        ln2=gain(r[6]),
        w_gate=_normal_matrix_bf16(r[7], I, D, 1.0 / math.sqrt(D)),
        w_up=_normal_matrix_bf16(r[8], I, D, 1.0 / math.sqrt(D)),
        w_down=_normal_matrix_bf16(r[9], D, I, 1.0 / math.sqrt(I)),
    )
    w.update(make_scorer_weights(p.n_q_heads, p.n_kv_heads, p.head_dim, lw.scorer_hidden,
                                 seed=seed))
    return dict(hidden=hidden, pos=layer_positions(p), k_pass=k_pass, v_pass=v_pass, w=w)
