"""Pins of the whole-layer oracle (``oracle/layer_oracle.py``; Alg. 2 with
the model's layer around attention).  Each check is fixed by something other
than the oracle's own formulas: hand-worked values, closed forms,
invariants of RMSNorm and RoPE, a loop-by-loop brute force of one tiny layer,
and the paper's FLOPs table (App. C)."""
import math

import numpy as np
import pytest

import oracle
from paper_2502_12085_amd import inputs

RNG = np.random.default_rng(7)


# ------------------------------------------------------------------ RMSNorm
def test_rmsnorm_constant_rows_and_unit_rms():
    h = np.array([[3.0] * 8, [-0.5] * 8])
    g = np.full(8, 2.0)
    out = oracle.rmsnorm_ref(h, g, 0.0)
    np.testing.assert_allclose(out, [[2.0] * 8, [-2.0] * 8], rtol=1e-15)
    x = RNG.standard_normal((5, 32))
    y = oracle.rmsnorm_ref(x, np.ones(32), 0.0)
    np.testing.assert_allclose(np.sqrt(np.mean(y * y, axis=1)), 1.0, rtol=1e-13)


def test_rmsnorm_scale_invariance_and_eps():
    x = RNG.standard_normal((4, 16))
    g = RNG.standard_normal(16)
    np.testing.assert_allclose(oracle.rmsnorm_ref(7.5 * x, g, 0.0), oracle.rmsnorm_ref(x, g, 0.0),
                               rtol=1e-13)
    # eps enters under the square root: one element, value 1, eps 3 -> 1/2
    np.testing.assert_allclose(oracle.rmsnorm_ref(np.array([[1.0]]), np.array([1.0]), 3.0),
                               [[0.5]], rtol=1e-15)


def test_rmsnorm_brute_force():
    x = RNG.standard_normal((3, 6))
    g = RNG.standard_normal(6)
    ref = np.empty_like(x)
    for r in range(3):
        ss = 0.0
        for c in range(6):
            ss += x[r, c] * x[r, c]
        inv = 1.0 / math.sqrt(ss / 6 + 1e-5)
        for c in range(6):
            ref[r, c] = x[r, c] * inv * g[c]
    np.testing.assert_allclose(oracle.rmsnorm_ref(x, g, 1e-5), ref, rtol=1e-13)


# --------------------------------------------------------------------- RoPE
def test_rope_hand_values():
    # d = 4: pairs (0, 2) at frequency 1 and (1, 3) at theta^(-1/2) = 0.1
    x = np.array([[[0.0, 1.0, 0.0, 0.0]]])
    out = oracle.rope_ref(x, np.array([1]), 100.0)
    np.testing.assert_allclose(out[0, 0], [0.0, math.cos(0.1), 0.0, math.sin(0.1)], atol=1e-15)
    x = np.array([[[1.0, 0.0, 0.0, 0.0]]])
    out = oracle.rope_ref(x, np.array([2]), 100.0)
    np.testing.assert_allclose(out[0, 0], [math.cos(2.0), 0.0, math.sin(2.0), 0.0], atol=1e-15)
    # the second element of a pair rotates the other way into the first
    x = np.array([[[0.0, 0.0, 1.0, 0.0]]])
    out = oracle.rope_ref(x, np.array([1]), 100.0)
    np.testing.assert_allclose(out[0, 0], [-math.sin(1.0), 0.0, math.cos(1.0), 0.0], atol=1e-15)


def test_rope_position_zero_norms_and_relative_positions():
    x = RNG.standard_normal((2, 5, 16))
    np.testing.assert_array_equal(oracle.rope_ref(x, np.zeros(5, np.int64), 1e4), x)
    pos = RNG.integers(0, 5000, 5)
    y = oracle.rope_ref(x, pos, 1e4)
    n_x = x[..., :8] ** 2 + x[..., 8:] ** 2
    n_y = y[..., :8] ** 2 + y[..., 8:] ** 2
    np.testing.assert_allclose(n_y, n_x, rtol=1e-12)
    # <R(q, m), R(k, n)> depends on m - n only
    q = RNG.standard_normal((1, 1, 16))
    k = RNG.standard_normal((1, 1, 16))
    for m, n, c in [(5, 2, 100), (0, 7, 31), (1000, 999, 12345)]:
        a = np.sum(oracle.rope_ref(q, [m], 1e4) * oracle.rope_ref(k, [n], 1e4))
        b = np.sum(oracle.rope_ref(q, [m + c], 1e4) * oracle.rope_ref(k, [n + c], 1e4))
        assert abs(a - b) < 1e-10


def test_rope_brute_force_rotation_matrices():
    d, theta = 8, 500.0
    x = RNG.standard_normal((1, 3, d))
    pos = np.array([3, 17, 250])
    ref = np.empty_like(x)
    for r in range(3):
        for j in range(d // 2):
            a = pos[r] * theta ** (-2.0 * j / d)
            rot = np.array([[math.cos(a), -math.sin(a)], [math.sin(a), math.cos(a)]])
            ref[0, r, [j, j + d // 2]] = rot @ x[0, r, [j, j + d // 2]]
    np.testing.assert_allclose(oracle.rope_ref(x, pos, theta), ref, rtol=1e-12, atol=1e-14)


# ------------------------------------------------------------------ SwiGLU
def test_swiglu_scalar_toy_and_zero_gate():
    y = np.array([[2.0]])
    out = oracle.swiglu_ffn_ref(y, np.array([[1.0]]), np.array([[3.0]]), np.array([[0.5]]))
    np.testing.assert_allclose(out, [[3.0 * 2.0 / (1.0 + math.exp(-2.0))]], rtol=1e-15)
    y = RNG.standard_normal((4, 6))
    wu, wd = RNG.standard_normal((5, 6)), RNG.standard_normal((6, 5))
    np.testing.assert_array_equal(oracle.swiglu_ffn_ref(y, np.zeros((5, 6)), wu, wd), 0.0)


def test_qkv_feature_order():
    n_q, n_kv, d = 2, 1, 3
    D = (n_q + 2 * n_kv) * d
    x = RNG.standard_normal((4, D))
    q, k, v = oracle.qkv_ref(x, np.eye(D), n_q, n_kv, d)
    np.testing.assert_array_equal(q[1], x[:, 3:6])
    np.testing.assert_array_equal(k[0], x[:, 6:9])
    np.testing.assert_array_equal(v[0], x[:, 9:12])


# ------------------------------------------------------------ whole layer
def _tiny_layer(seed=0, host_idx=1, l_p=2):
    """A hand-sized layer: D = 8, 2 query heads and 1 KV head of d = 4,
    I = 8, La = 3, Lb = 5; weights as floats."""
    r = np.random.default_rng(seed)
    La, Lb, n_q, n_kv, d, D, I = 3, 5, 2, 1, 4, 8, 8
    w = dict(ln1=1 + 0.1 * r.standard_normal(D), w_qkv=r.standard_normal((16, D)) / 3,
             w_o=r.standard_normal((D, 8)) / 3, ln2=1 + 0.1 * r.standard_normal(D),
             w_gate=r.standard_normal((I, D)) / 3, w_up=r.standard_normal((I, D)) / 3,
             w_down=r.standard_normal((D, I)) / 3, w1=r.standard_normal((6, 16)) / 4,
             b1=r.standard_normal(6) * 0.1, w2=r.standard_normal((1, 6)) / 2,
             b2=np.array([0.05]))
    hidden = r.standard_normal((La + Lb, D))
    kp = r.standard_normal((host_idx, n_kv, l_p, d))
    vp = r.standard_normal((host_idx, n_kv, l_p, d))
    pos = np.array([0, 1, 2, 13, 14, 15, 16, 17])
    kw = dict(anchor_len=La, pass_len=l_p, n_q=n_q, n_kv=n_kv, head_dim=d, eps=1e-5, theta=50.0)
    return hidden, pos, w, kp, vp, kw


def _brute_layer(hidden, pos, w, kp, vp, anchor_len, n_q, n_kv, head_dim, eps, theta, **_):
    """The same layer, element by element with Python loops."""
    R, D = hidden.shape
    d, g = head_dim, n_q // n_kv

    def norm(vec, gain):
        ms = sum(t * t for t in vec) / len(vec)
        return [vec[c] / math.sqrt(ms + eps) * gain[c] for c in range(len(vec))]

    def matvec(W, vec):
        return [sum(W[o][c] * vec[c] for c in range(len(vec))) for o in range(len(W))]

    def rot(vec, p):
        out = list(vec)
        for j in range(d // 2):
            a = p * theta ** (-2.0 * j / d)
            out[j] = vec[j] * math.cos(a) - vec[j + d // 2] * math.sin(a)
            out[j + d // 2] = vec[j + d // 2] * math.cos(a) + vec[j] * math.sin(a)
        return out

    Q = [[None] * R for _ in range(n_q)]
    K = [[None] * R for _ in range(n_kv)]
    V = [[None] * R for _ in range(n_kv)]
    for r in range(R):
        y = matvec(w["w_qkv"], norm(hidden[r], w["ln1"]))
        for h in range(n_q):
            Q[h][r] = rot(y[h * d:(h + 1) * d], pos[r])
        for h in range(n_kv):
            K[h][r] = rot(y[(n_q + h) * d:(n_q + h + 1) * d], pos[r])
            V[h][r] = y[(n_q + n_kv + h) * d:(n_q + n_kv + h + 1) * d]
    out = []
    for r in range(R):
        a_flat = []
        for h in range(n_q):
            kv = h // g
            keys = [K[kv][j] for j in range(anchor_len)]
            vals = [V[kv][j] for j in range(anchor_len)]
            for s in range(kp.shape[0]):
                keys += [list(kp[s, kv, t]) for t in range(kp.shape[2])]
                vals += [list(vp[s, kv, t]) for t in range(vp.shape[2])]
            keys += [K[kv][j] for j in range(anchor_len, R)]
            vals += [V[kv][j] for j in range(anchor_len, R)]
            lp = kp.shape[0] * kp.shape[2]
            last = r if r < anchor_len else r + lp  # causal over [A; P; B]
            z = [sum(Q[h][r][c] * keys[j][c] for c in range(d)) / math.sqrt(d)
                 for j in range(last + 1)]
            m = max(z)
            e = [math.exp(t - m) for t in z]
            a_flat += [sum(e[j] * vals[j][c] for j in range(last + 1)) / sum(e) for c in range(d)]
        h1 = [hidden[r][c] + t for c, t in enumerate(matvec(w["w_o"], a_flat))]
        y = norm(h1, w["ln2"])
        gt, up = matvec(w["w_gate"], y), matvec(w["w_up"], y)
        act = [gt[i] / (1 + math.exp(-gt[i])) * up[i] for i in range(len(gt))]
        out.append([h1[c] + t for c, t in enumerate(matvec(w["w_down"], act))])
    return np.array(out)


def test_layer_matches_loop_brute_force():
    hidden, pos, w, kp, vp, kw = _tiny_layer()
    ref = oracle.layer_ref(hidden, pos, w, kp, vp, **kw)
    np.testing.assert_allclose(ref["out"], _brute_layer(hidden, pos, w, kp, vp, **kw),
                               rtol=1e-12, atol=1e-12)
    sub = oracle.layer_ref(hidden, pos, w, kp, vp, rows=[0, 4, 7], **kw)
    np.testing.assert_allclose(sub["out"], ref["out"][[0, 4, 7]], rtol=1e-13, atol=1e-13)


def test_layer_residual_path_only():
    hidden, pos, w, kp, vp, kw = _tiny_layer(1)
    w = dict(w, w_o=np.zeros_like(w["w_o"]), w_down=np.zeros_like(w["w_down"]))
    ref = oracle.layer_ref(hidden, pos, w, kp, vp, **kw)
    np.testing.assert_array_equal(ref["h1"], hidden)
    np.testing.assert_array_equal(ref["out"], hidden)


def test_layer_position_shift_invariance_without_passing_rows():
    hidden, pos, w, kp, vp, kw = _tiny_layer(2, host_idx=0)
    a = oracle.layer_ref(hidden, pos, w, kp, vp, **kw)["out"]
    b = oracle.layer_ref(hidden, pos + 1000, w, kp, vp, **kw)["out"]
    np.testing.assert_allclose(a, b, rtol=1e-10, atol=1e-10)
    c = oracle.layer_ref(hidden, pos + np.array([0, 0, 0, 1, 1, 1, 1, 1]), w, kp, vp, **kw)["out"]
    assert np.abs(a - c).max() > 1e-6  # moving only the local block relative to the anchor matters


def test_layer_selection_is_topk_of_its_scores():
    hidden, pos, w, kp, vp, kw = _tiny_layer(3)
    ref = oracle.layer_ref(hidden, pos, w, kp, vp, **kw)
    s = ref["scores"][0]
    assert ref["idx"].shape == (1, 2)
    chosen = set(ref["idx"][0].tolist())
    assert min(s[list(chosen)]) >= max(s[[i for i in range(5) if i not in chosen]])


def test_layer_flops_against_the_papers_table():
    """Summed over hosts, the per-host count equals the FLOPs table's APB row
    except for the two documented differences: causal pair counts include the
    diagonal (n(n+1)/2, not n^2/2), and the passing term is counted as
    4 d_model per (local query, passing key) pair, twice the table's
    coefficient over the local rows only."""
    lw = inputs.LAYER_WORKLOADS["llama8b_128k_layer"]
    p = lw.problem
    H, La, Lb, lp = p.n_hosts, p.anchor_len, p.local_len, p.pass_len
    D, I, g = lw.hidden, lw.intermediate, p.group
    ours = 0.0
    diag = 0.0
    pass_ours = 0.0
    for h in range(H):
        la = 0 if h == 0 else La  # the first host has no anchor in the table's count
        attn = oracle.attention_flops(p.n_q_heads, p.head_dim, la, Lb, h * lp)
        ours += oracle.layer_flops(la + Lb, D, I, p.n_q_heads, p.n_kv_heads, p.head_dim, attn)
        diag += 2.0 * (la + Lb) * D  # the diagonal half-pairs of the causal triangles
        pass_ours += 4.0 * D * Lb * h * lp
    n = H * Lb
    table = oracle.apb_table_flops_per_layer(n, D, g, I, H, La, lp)
    table_pass = lp * H * (H - 1) * (n / H + La) * D
    assert abs((ours - diag - pass_ours) - (table - table_pass)) / table < 1e-12
    assert abs(pass_ours / (table_pass * Lb / (Lb + La)) - 2.0) < 1e-12
