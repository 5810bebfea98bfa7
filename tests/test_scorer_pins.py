"""Pins of the retaining-head scorer oracle (Sec. 3.4; App. B).

Checked against a hand-worked toy (``tests/golden/toy_scorer.json``),
one-hot weight probes that read back single entries of Q, K and V (which fix
the feature order head by head), pure-Python brute force, and structural
properties (anchor rows are never scored, constant output for W1 = 0,
linearity in the output layer).
"""
import json
import math
import os

import numpy as np
import pytest

import oracle
from paper_2502_12085_amd import inputs

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _rand_bf16(rng, shape, scale=1.0):
    return inputs.f32_to_bf16_bits(rng.standard_normal(shape).astype(np.float32) * scale)


def test_scorer_golden():
    t = json.load(open(os.path.join(GOLDEN, "toy_scorer.json")))
    s = oracle.retaining_scores_ref(np.array(t["q"]), np.array(t["k"]), np.array(t["v"]),
                                    np.array(t["w1"]), np.array(t["b1"]), np.array(t["w2"]),
                                    np.array(t["b2"]), anchor_len=t["anchor_len"])
    np.testing.assert_allclose(s, t["expect"], atol=1e-14)


def test_silu_closed_form():
    z = np.array([0.0, math.log(3), -math.log(3), 30.0, -30.0])
    np.testing.assert_allclose(oracle.silu(z), [0.0, 0.75 * math.log(3), -0.25 * math.log(3),
                                                30.0 / (1 + math.exp(-30)), -30.0 / (1 + math.exp(30))],
                               rtol=1e-15)


@pytest.mark.parametrize("which,head,dim", [("q", 0, 0), ("q", 2, 5), ("k", 0, 7), ("k", 1, 1),
                                            ("v", 1, 6), ("v", 0, 3)])
def test_one_hot_probe_reads_the_right_entry(which, head, dim):
    # W1 row 0 selects one feature, W2 reads hidden unit 0 for KV head 1: the
    # score is then SiLU(entry) for every local token
    rng = np.random.default_rng(7)
    n_q, n_kv, d, la, lb = 3, 2, 8, 4, 6
    q = _rand_bf16(rng, (n_q, la + lb, d))
    k = _rand_bf16(rng, (n_kv, la + lb, d))
    v = _rand_bf16(rng, (n_kv, la + lb, d))
    feats = (n_q + 2 * n_kv) * d
    off = {"q": 0, "k": n_q * d, "v": (n_q + n_kv) * d}[which] + head * d + dim
    hidden = 4
    w1 = np.zeros((hidden, feats))
    w1[0, off] = 1.0
    w2 = np.zeros((n_kv, hidden))
    w2[1, 0] = 1.0
    s = oracle.retaining_scores_ref(q, k, v, w1, np.zeros(hidden), w2, np.zeros(n_kv), anchor_len=la)
    src = {"q": q, "k": k, "v": v}[which]
    x = oracle.bf16_to_f64(src[head, la:, dim])
    np.testing.assert_allclose(s[1], x / (1 + np.exp(-x)), rtol=1e-15)
    np.testing.assert_allclose(s[0], 0.0, atol=0)


def test_brute_force_python():
    rng = np.random.default_rng(8)
    n_q, n_kv, d, la, lb, hidden = 2, 1, 2, 1, 3, 3
    q, k, v = (_rand_bf16(rng, (n, la + lb, d)) for n in (n_q, n_kv, n_kv))
    feats = (n_q + 2 * n_kv) * d
    w1 = rng.standard_normal((hidden, feats))
    b1 = rng.standard_normal(hidden)
    w2 = rng.standard_normal((n_kv, hidden))
    b2 = rng.standard_normal(n_kv)
    s = oracle.retaining_scores_ref(q, k, v, w1, b1, w2, b2, anchor_len=la)
    f = oracle.bf16_to_f64
    for t in range(lb):
        x = []
        for h in range(n_q):
            x += list(f(q[h, la + t]))
        for h in range(n_kv):
            x += list(f(k[h, la + t]))
        for h in range(n_kv):
            x += list(f(v[h, la + t]))
        hid = []
        for j in range(hidden):
            z = sum(w1[j][i] * x[i] for i in range(feats)) + b1[j]
            hid.append(z / (1 + math.exp(-z)))
        for kv in range(n_kv):
            exp = sum(w2[kv][j] * hid[j] for j in range(hidden)) + b2[kv]
            assert abs(s[kv, t] - exp) < 1e-12


def test_anchor_rows_are_not_scored_and_structure():
    rng = np.random.default_rng(9)
    n_q, n_kv, d, la, lb, hidden = 4, 2, 8, 5, 7, 16
    q, k, v = (_rand_bf16(rng, (n, la + lb, d)) for n in (n_q, n_kv, n_kv))
    feats = (n_q + 2 * n_kv) * d
    w1 = rng.standard_normal((hidden, feats)) / math.sqrt(feats)
    b1, w2, b2 = rng.standard_normal(hidden), rng.standard_normal((n_kv, hidden)), rng.standard_normal(n_kv)
    s = oracle.retaining_scores_ref(q, k, v, w1, b1, w2, b2, anchor_len=la)
    assert s.shape == (n_kv, lb)
    q2 = q.copy()
    q2[:, :la] = _rand_bf16(rng, (n_q, la, d))   # anchor rows do not matter
    np.testing.assert_array_equal(s, oracle.retaining_scores_ref(q2, k, v, w1, b1, w2, b2, anchor_len=la))
    s0 = oracle.retaining_scores_ref(q, k, v, np.zeros_like(w1), b1, w2, b2, anchor_len=la)
    const = w2 @ oracle.silu(b1) + b2
    np.testing.assert_allclose(s0, np.repeat(const[:, None], lb, axis=1), rtol=1e-14)
    s3 = oracle.retaining_scores_ref(q, k, v, w1, b1, 3 * w2, 3 * b2, anchor_len=la)
    np.testing.assert_allclose(s3, 3 * s, rtol=1e-13)


def _brute_force_multiply_adds(n_q, n_kv, d, lb, hidden):
    """Multiply-adds of scoring ``lb`` local tokens, counted one by one while
    the two layers are evaluated in plain Python loops (features gathered
    head by head, as in the brute-force test above)."""
    rng = np.random.default_rng(10)
    feats = (n_q + 2 * n_kv) * d
    x = rng.standard_normal((lb, feats))
    w1 = rng.standard_normal((hidden, feats))
    w2 = rng.standard_normal((n_kv, hidden))
    count = 0
    for t in range(lb):
        hid = []
        for j in range(hidden):
            z = 0.0
            for i in range(feats):
                z += w1[j][i] * x[t][i]
                count += 1
            hid.append(z / (1 + math.exp(-z)))
        for kv in range(n_kv):
            acc = 0.0
            for j in range(hidden):
                acc += w2[kv][j] * hid[j]
                count += 1
    return count


@pytest.mark.parametrize("shape", [(2, 1, 2, 3, 3), (4, 2, 8, 5, 16), (3, 3, 4, 1, 7)])
def test_flops_counted_by_brute_force(shape):
    # two flops per multiply-add, counted in the loops rather than restated
    assert oracle.scorer_flops(*shape) == 2.0 * _brute_force_multiply_adds(*shape)
