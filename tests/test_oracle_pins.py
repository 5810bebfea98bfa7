"""Pins of the fp64 oracle against what the paper and mathematics fix.

Each test checks the oracle against something other than itself: hand-worked
toy values, a brute-force dense mask written from the block rules, PyTorch's
causal scaled-dot-product attention over the concatenated sequence, closed
forms, invariants, and brute-force subset search for the selection.
"""
import itertools
import json
import math
import os

import numpy as np
import pytest
import torch
from scipy.special import logsumexp

import oracle
from paper_2502_12085_amd import inputs

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _rand_bf16(rng, shape, scale=1.0):
    return inputs.f32_to_bf16_bits(rng.standard_normal(shape).astype(np.float32) * scale)


def _case(rng, n_q, n_kv, d, la, lb, lp, host_idx):
    q = _rand_bf16(rng, (n_q, la + lb, d))
    k = _rand_bf16(rng, (n_kv, la + lb, d))
    v = _rand_bf16(rng, (n_kv, la + lb, d))
    kp = _rand_bf16(rng, (host_idx, n_kv, lp, d))
    vp = _rand_bf16(rng, (host_idx, n_kv, lp, d))
    return q, k, v, kp, vp


# ---------------------------------------------------------------- toys
def test_toy_attention_golden():
    spec = json.load(open(os.path.join(GOLDEN, "toy_attention.json")))
    for c in spec["cases"]:
        q = np.array(c["q_rows"], dtype=np.float64)[None]
        k = np.array(c["k_anchor"] + c["k_local"], dtype=np.float64)[None]
        v = np.array(c["v_anchor"] + c["v_local"], dtype=np.float64)[None]
        kp = np.array(c["k_pass"], dtype=np.float64)[None, None]
        vp = np.array(c["v_pass"], dtype=np.float64)[None, None]
        o, lse = oracle.attention_ref(q, k, v, kp, vp, anchor_len=c["anchor_len"],
                                      scale=c["scale"])
        np.testing.assert_allclose(o[0], np.array(c["expect_o"]), atol=1e-12, err_msg=c["name"])
        np.testing.assert_allclose(lse[0], np.array(c["expect_lse"]), atol=1e-12, err_msg=c["name"])


def test_toy_topk_golden():
    spec = json.load(open(os.path.join(GOLDEN, "toy_topk.json")))
    for c in spec["cases"]:
        s = np.array([float(x) for x in c["scores"]], dtype=np.float32)[None]
        got = oracle.topk_ref(s, c["l_p"])[0]
        assert got.tolist() == c["expect"], c


# ------------------------------------------------- brute-force dense mask
def _dense_mask_from_blocks(la, lb, lp_per_host, host_idx):
    """Visibility matrix written from the block rules of M' (one loop per
    block pair), independently of the oracle's position formula."""
    n_pass = lp_per_host * host_idx
    mask = np.zeros((la + lb, la + n_pass + lb), dtype=bool)
    for a in range(la):               # anchor rows: anchor block, causal
        for j in range(a + 1):
            mask[a, j] = True
    for b in range(lb):               # local rows
        row = la + b
        for j in range(la):           # whole anchor block
            mask[row, j] = True
        for s in range(host_idx):     # every earlier host's compressed block
            for t in range(lp_per_host):
                mask[row, la + s * lp_per_host + t] = True
        for j in range(b + 1):        # own block, causal
            mask[row, la + n_pass + j] = True
    return mask


def _key_rows_by_source(x_local, x_pass, la, kv):
    rows = []
    for j in range(la):
        rows.append(x_local[kv, j])
    for s in range(x_pass.shape[0]):
        for t in range(x_pass.shape[2]):
            rows.append(x_pass[s, kv, t])
    for j in range(la, x_local.shape[1]):
        rows.append(x_local[kv, j])
    return oracle.bf16_to_f64(np.stack(rows))


@pytest.mark.parametrize("shape", [
    # n_q, n_kv, d, La, Lb, l_p, host_idx
    (4, 2, 8, 5, 7, 3, 2),
    (3, 1, 4, 0, 9, 4, 3),    # no anchor (ablation), first rows see only P
    (2, 2, 6, 6, 5, 2, 0),    # first host: no passing block
    (2, 1, 4, 4, 6, 0, 3),    # l_p = 0: passing block empty
    (6, 3, 16, 13, 17, 5, 1),
])
def test_oracle_vs_bruteforce(shape):
    n_q, n_kv, d, la, lb, lp, hidx = shape
    rng = np.random.default_rng(sum(shape))
    q, k, v, kp, vp = _case(rng, n_q, n_kv, d, la, lb, lp, hidx)
    o, lse = oracle.attention_ref(q, k, v, kp, vp, anchor_len=la)
    mask = _dense_mask_from_blocks(la, lb, lp, hidx)
    g = n_q // n_kv
    for h in range(n_q):
        kc = _key_rows_by_source(k, kp, la, h // g)
        vc = _key_rows_by_source(v, vp, la, h // g)
        z = oracle.bf16_to_f64(q[h]) @ kc.T / math.sqrt(d)
        z = np.where(mask, z, -np.inf)
        ref_lse = logsumexp(z, axis=1)
        w = np.exp(z - ref_lse[:, None])
        np.testing.assert_allclose(o[h], w @ vc, atol=1e-12, rtol=1e-12)
        np.testing.assert_allclose(lse[h], ref_lse, atol=1e-12, rtol=1e-12)


def test_flops_matches_mask_count():
    for (la, lb, lp, hidx) in [(5, 7, 3, 2), (0, 9, 4, 3), (6, 5, 2, 0), (13, 17, 5, 1)]:
        pairs = int(_dense_mask_from_blocks(la, lb, lp, hidx).sum())
        assert oracle.attention_flops(3, 64, la, lb, lp * hidx) == 4.0 * 64 * 3 * pairs


# ------------------------------------------- library special case (SDPA)
@pytest.mark.parametrize("shape", [(4, 2, 16, 8, 12, 3, 2), (2, 1, 8, 0, 10, 5, 1), (2, 2, 8, 7, 9, 2, 3)])
def test_oracle_vs_torch_causal_sdpa(shape):
    """M' read as causal attention over [A; P; B] with the P query rows
    dropped: run PyTorch's causal SDPA over the full concatenation with dummy
    queries at the P positions and keep the A and B rows."""
    n_q, n_kv, d, la, lb, lp, hidx = shape
    rng = np.random.default_rng(7 + sum(shape))
    q, k, v, kp, vp = _case(rng, n_q, n_kv, d, la, lb, lp, hidx)
    o, _ = oracle.attention_ref(q, k, v, kp, vp, anchor_len=la)
    g = n_q // n_kv
    n_pass = lp * hidx
    qf = oracle.bf16_to_f64(q)
    qfull = np.concatenate([qf[:, :la], np.ones((n_q, n_pass, d)), qf[:, la:]], axis=1)
    kf = np.stack([_key_rows_by_source(k, kp, la, h // g) for h in range(n_q)])
    vf = np.stack([_key_rows_by_source(v, vp, la, h // g) for h in range(n_q)])
    ref = torch.nn.functional.scaled_dot_product_attention(
        torch.from_numpy(qfull), torch.from_numpy(kf), torch.from_numpy(vf), is_causal=True).numpy()
    keep = np.r_[0:la, la + n_pass:la + n_pass + lb]
    np.testing.assert_allclose(o, ref[:, keep], atol=1e-12, rtol=1e-12)


# ------------------------------------------------------------ closed forms
def test_q_zero_uniform_closed_form():
    rng = np.random.default_rng(3)
    n_q, n_kv, d, la, lb, lp, hidx = 4, 2, 8, 6, 10, 3, 3
    _, k, v, kp, vp = _case(rng, n_q, n_kv, d, la, lb, lp, hidx)
    q = np.zeros((n_q, la + lb, d), np.uint16)
    o, lse = oracle.attention_ref(q, k, v, kp, vp, anchor_len=la)
    vf = oracle.bf16_to_f64(v)
    vpf = oracle.bf16_to_f64(vp)
    for h in range(n_q):
        kv = h // 2
        for r in range(la + lb):
            if r < la:
                vis = [vf[kv, j] for j in range(r + 1)]
            else:
                vis = [vf[kv, j] for j in range(la)]
                vis += [vpf[s, kv, t] for s in range(hidx) for t in range(lp)]
                vis += [vf[kv, j] for j in range(la, r + 1)]
            np.testing.assert_allclose(o[h, r], np.mean(vis, axis=0), atol=1e-13)
            assert abs(lse[h, r] - math.log(len(vis))) < 1e-13


# --------------------------------------------------------------- invariants
def test_rows_sum_to_one_via_constant_v():
    rng = np.random.default_rng(4)
    q, k, _, kp, _ = _case(rng, 4, 2, 16, 9, 11, 4, 2)
    one = inputs.f32_to_bf16_bits(np.ones((2, 20, 16), np.float32))
    onep = inputs.f32_to_bf16_bits(np.ones((2, 2, 4, 16), np.float32))
    o, _ = oracle.attention_ref(q, k, one, kp, onep, anchor_len=9)
    np.testing.assert_allclose(o, 1.0, atol=1e-13)


def test_anchor_rows_ignore_passing_and_local_contents():
    rng = np.random.default_rng(5)
    la, lb = 7, 9
    q, k, v, kp, vp = _case(rng, 2, 1, 8, la, lb, 3, 2)
    o1, l1 = oracle.attention_ref(q, k, v, kp, vp, anchor_len=la)
    k2, v2 = k.copy(), v.copy()
    k2[:, la:] = _rand_bf16(rng, k2[:, la:].shape)
    v2[:, la:] = _rand_bf16(rng, v2[:, la:].shape)
    o2, l2 = oracle.attention_ref(q, k2, v2, _rand_bf16(rng, kp.shape), _rand_bf16(rng, vp.shape),
                                  anchor_len=la)
    np.testing.assert_array_equal(o1[:, :la], o2[:, :la])
    np.testing.assert_array_equal(l1[:, :la], l2[:, :la])
    assert not np.allclose(o1[:, la:], o2[:, la:])


def _causal_numpy(qf, kf, vf, scale):
    n = qf.shape[0]
    z = qf @ kf.T * scale
    z[np.triu_indices(n, 1)] = -np.inf
    lse = logsumexp(z, axis=1)
    return np.exp(z - lse[:, None]) @ vf, lse


def test_no_passing_reduces_to_causal():
    """Lp = 0 (first host, or l_p = 0): plain causal attention over [A; B]."""
    rng = np.random.default_rng(6)
    la, lb, d = 5, 11, 8
    for hidx, lp in [(0, 4), (3, 0)]:
        q, k, v, kp, vp = _case(rng, 2, 1, d, la, lb, lp, hidx)
        o, lse = oracle.attention_ref(q, k, v, kp, vp, anchor_len=la)
        for h in range(2):
            ro, rl = _causal_numpy(oracle.bf16_to_f64(q[h]), oracle.bf16_to_f64(k[0]),
                                   oracle.bf16_to_f64(v[0]), 1 / math.sqrt(d))
            np.testing.assert_allclose(o[h], ro, atol=1e-12)
            np.testing.assert_allclose(lse[h], rl, atol=1e-12)


def test_full_passing_equals_full_attention():
    """La = 0 and l_p = l_b with every index kept: the local rows of host 1
    equal the matching rows of causal attention over the whole document
    [B_0; B_1] (APB degenerates to full attention)."""
    rng = np.random.default_rng(8)
    lb, d = 9, 8
    q_all = _rand_bf16(rng, (1, 2 * lb, d))
    k_all = _rand_bf16(rng, (1, 2 * lb, d))
    v_all = _rand_bf16(rng, (1, 2 * lb, d))
    scores = rng.standard_normal((1, lb)).astype(np.float32)
    idx, kc, vc = oracle.compress_ref(scores, k_all[:, :lb], v_all[:, :lb], lb, 0)
    assert idx[0].tolist() == list(range(lb))
    o, lse = oracle.attention_ref(q_all[:, lb:], k_all[:, lb:], v_all[:, lb:], kc[None], vc[None],
                                  anchor_len=0)
    ro, rl = _causal_numpy(oracle.bf16_to_f64(q_all[0]), oracle.bf16_to_f64(k_all[0]),
                           oracle.bf16_to_f64(v_all[0]), 1 / math.sqrt(d))
    np.testing.assert_allclose(o[0], ro[lb:], atol=1e-12)
    np.testing.assert_allclose(lse[0], rl[lb:], atol=1e-12)


def test_passing_row_permutation_invariance():
    rng = np.random.default_rng(9)
    q, k, v, kp, vp = _case(rng, 2, 1, 8, 4, 6, 3, 3)
    o1, l1 = oracle.attention_ref(q, k, v, kp, vp, anchor_len=4)
    flat_k = kp.reshape(9, 1, 8)[::-1]  # reverse all passing rows (hosts and rows)
    flat_v = vp.reshape(9, 1, 8)[::-1]
    kp2 = np.ascontiguousarray(flat_k.reshape(3, 3, 1, 8).transpose(0, 2, 1, 3))
    vp2 = np.ascontiguousarray(flat_v.reshape(3, 3, 1, 8).transpose(0, 2, 1, 3))
    o2, l2 = oracle.attention_ref(q, k, v, kp2, vp2, anchor_len=4)
    np.testing.assert_allclose(o1, o2, atol=1e-13)
    np.testing.assert_allclose(l1, l2, atol=1e-13)


def test_scale_equals_scaled_queries():
    rng = np.random.default_rng(10)
    qf = rng.standard_normal((2, 10, 4))
    kf = rng.standard_normal((1, 10, 4))
    vf = rng.standard_normal((1, 10, 4))
    kpf = rng.standard_normal((2, 1, 2, 4))
    vpf = rng.standard_normal((2, 1, 2, 4))
    o1, l1 = oracle.attention_ref(qf, kf, vf, kpf, vpf, anchor_len=3, scale=1.0)
    o2, l2 = oracle.attention_ref(2 * qf, kf, vf, kpf, vpf, anchor_len=3, scale=0.5)
    np.testing.assert_allclose(o1, o2, atol=1e-12)
    np.testing.assert_allclose(l1, l2, atol=1e-12)
    o3, _ = oracle.attention_ref(qf, kf, vf, kpf, vpf, anchor_len=3)  # default 1/sqrt(d)
    o4, _ = oracle.attention_ref(qf, kf, vf, kpf, vpf, anchor_len=3, scale=0.5)
    np.testing.assert_allclose(o3, o4, atol=1e-12)


def test_gqa_equals_repeated_kv():
    rng = np.random.default_rng(11)
    q, k, v, kp, vp = _case(rng, 6, 2, 8, 4, 7, 2, 2)
    o1, l1 = oracle.attention_ref(q, k, v, kp, vp, anchor_len=4)
    rep = lambda x, ax: np.repeat(x, 3, axis=ax)
    o2, l2 = oracle.attention_ref(q, rep(k, 0), rep(v, 0), rep(kp, 1), rep(vp, 1), anchor_len=4)
    np.testing.assert_array_equal(o1, o2)
    np.testing.assert_array_equal(l1, l2)


def test_row_and_head_subsets_match_full():
    rng = np.random.default_rng(12)
    q, k, v, kp, vp = _case(rng, 4, 2, 8, 6, 10, 3, 2)
    o, lse = oracle.attention_ref(q, k, v, kp, vp, anchor_len=6, row_block=4)
    rows = np.array([0, 5, 6, 7, 15])
    heads = np.array([3, 1])
    os_, ls = oracle.attention_ref(q, k, v, kp, vp, anchor_len=6, heads=heads, rows=rows)
    np.testing.assert_allclose(os_, o[heads][:, rows], atol=1e-14)
    np.testing.assert_allclose(ls, lse[heads][:, rows], atol=1e-14)


# ------------------------------------------------------------------- top-k
def _bruteforce_topk(s, l_p):
    """The unique subset S (|S| = l_p) such that every member outranks every
    non-member, with 'i outranks j' meaning s_i > s_j, or equal scores and
    i < j (NaN below everything)."""
    n = len(s)

    def outranks(i, j):
        si, sj = s[i], s[j]
        if math.isnan(si):
            return math.isnan(sj) and i < j
        if math.isnan(sj):
            return True
        return si > sj or (si == sj and i < j)

    hits = [sub for sub in itertools.combinations(range(n), l_p)
            if all(outranks(i, j) for i in sub for j in range(n) if j not in sub)]
    assert len(hits) == 1
    return list(hits[0])


def test_topk_bruteforce_small():
    rng = np.random.default_rng(13)
    pool = np.array([-2.0, -0.0, 0.0, 1.0, 1.0, np.inf, -np.inf, np.nan, 3.5], np.float32)
    for trial in range(60):
        n = int(rng.integers(1, 10))
        s = rng.choice(pool, n) if trial % 2 else rng.standard_normal(n).astype(np.float32)
        for l_p in range(n + 1):
            assert oracle.topk_ref(s[None], l_p)[0].tolist() == _bruteforce_topk(s.tolist(), l_p)


def test_topk_matches_stable_argsort_and_special_cases():
    rng = np.random.default_rng(14)
    s = rng.standard_normal((3, 500)).astype(np.float32)
    s[1] = np.round(s[1] * 2) / 2  # many ties
    for l_p in [0, 1, 37, 250, 500]:
        got = oracle.topk_ref(s, l_p)
        for h in range(3):
            ref = np.sort(np.argsort(-s[h], kind="stable")[:l_p])
            assert got[h].tolist() == ref.tolist()
    eq = np.full((1, 20), 0.25, np.float32)
    assert oracle.topk_ref(eq, 6)[0].tolist() == list(range(6))
    inc = np.arange(20, dtype=np.float32)[None]
    assert oracle.topk_ref(inc, 5)[0].tolist() == list(range(15, 20))


def test_gather_is_bit_copy():
    rng = np.random.default_rng(15)
    la, lb, d = 3, 12, 8
    k = rng.integers(0, 65536, (2, la + lb, d), dtype=np.uint16)
    v = rng.integers(0, 65536, (2, la + lb, d), dtype=np.uint16)
    scores = rng.standard_normal((2, lb)).astype(np.float32)
    idx, kc, vc = oracle.compress_ref(scores, k, v, 4, la)
    for h in range(2):
        for t in range(4):
            assert kc[h, t].tobytes() == k[h, la + idx[h, t]].tobytes()
            assert vc[h, t].tobytes() == v[h, la + idx[h, t]].tobytes()


def test_simulated_hosts_build_passing_block_in_host_order():
    wl = inputs.Workload("t", inputs.Problem(4, 2, 4, 16, 3, 2, 1, 8))
    inp = inputs.make_inputs(wl, 0)
    hosts = inputs.make_host_blocks(wl, 0)
    o, lse, idx, kc, vc, kp, vp = oracle.simulate_hosts_ref(
        inp["q"], inp["k"], inp["v"], inp["scores"], hosts, anchor_len=4, l_p=3)
    for j, hb in enumerate(hosts):
        sel = np.sort(np.argsort(-hb["scores"][0], kind="stable")[:3])
        assert kp[j, 0].tobytes() == hb["k"][0, 4 + sel].tobytes()
        assert vp[j, 0].tobytes() == hb["v"][0, 4 + sel].tobytes()
    o2, _ = oracle.attention_ref(inp["q"], inp["k"], inp["v"], kp, vp, anchor_len=4)
    np.testing.assert_array_equal(o, o2)


# ----------------------------------------------------------- input recipe
def test_bf16_rounding_matches_torch():
    rng = np.random.default_rng(16)
    x = np.concatenate([rng.standard_normal(10000).astype(np.float32) * 10.0 ** rng.integers(-3, 4, 10000),
                        np.array([1.00390625, 1.01171875, -1.00390625], np.float32)])  # exact ties
    ours = inputs.f32_to_bf16_bits(x)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    np.testing.assert_array_equal(ours, ref)


def test_inputs_are_seeded_and_shaped():
    wl = inputs.WORKLOADS["tiny"]
    a = inputs.make_inputs(wl, 0)
    b = inputs.make_inputs(wl, 0)
    p = wl.problem
    assert a["q"].shape == (4, 640, 64) and a["k"].shape == (1, 640, 64)
    assert a["k_pass"].shape == (2, 1, 32, 64) and a["scores"].shape == (1, 512)
    for key in ("q", "k", "v", "k_pass", "v_pass", "scores"):
        np.testing.assert_array_equal(a[key], b[key])
    assert p.passing_rows == 64 and p.key_rows == 704


def test_outlier_channels_scale_k():
    wl = inputs.Workload("o", inputs.Problem(2, 1, 16, 64, 8, 4, 2, 128), outlier_k=True)
    inp = inputs.make_inputs(wl, 0)
    cols = inp["outlier_cols"]
    assert cols.shape == (2, 3)
    kf = inputs.bf16_bits_to_f32(inp["k"])
    for h in range(2):
        big = np.abs(kf[h][:, cols[h]]).mean()
        rest = np.abs(np.delete(kf[h], cols[h], axis=1)).mean()
        assert 5 < big / rest < 11
