"""Pins of the stage-2 (decoding) oracle: per-host partial attention and
MergeScore (Alg. 3).

Checked against: hand-worked values (``tests/golden/toy_merge.json``), the
prefill oracle (itself pinned in ``test_oracle_pins.py``) for the last host,
pure-Python brute force, the q = 0 closed form, and the exact identity that
merging the partial results of any split of the keys equals one softmax over
all of them.
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


def _case(rng, n_q=4, n_kv=2, d=16, lc=23, n_new=5):
    q = _rand_bf16(rng, (n_q, n_new, d))
    kc = _rand_bf16(rng, (n_kv, lc, d))
    vc = _rand_bf16(rng, (n_kv, lc, d))
    kn = _rand_bf16(rng, (n_kv, n_new, d))
    vn = _rand_bf16(rng, (n_kv, n_new, d))
    return q, kc, vc, kn, vn


def test_merge_golden():
    spec = json.load(open(os.path.join(GOLDEN, "toy_merge.json")))
    for c in spec["cases"]:
        lse = np.array([float(x) for x in c["lse_parts"]])
        a, l = oracle.merge_ref(np.array(c["a_parts"]), lse)
        np.testing.assert_allclose(a, c["expect_a"], atol=1e-15, err_msg=c["name"])
        assert abs(l - c["expect_lse"]) < 1e-15, c["name"]


def test_decode_golden_two_hosts():
    t = json.load(open(os.path.join(GOLDEN, "toy_merge.json")))["decode_toy"]
    q = np.array(t["q"])[None]  # one head, one new token
    caches = [(np.array(k)[None], np.array(v)[None]) for k, v in zip(t["caches_k"], t["caches_v"])]
    kn, vn = np.array(t["k_new"])[None], np.array(t["v_new"])[None]
    a, lse, parts = oracle.stage2_ref(q, caches, kn, vn)
    for h, (pa, pl) in enumerate(parts):
        np.testing.assert_allclose(pa[0, 0], t["expect_parts_a"][h], atol=1e-15)
        assert abs(pl[0, 0] - t["expect_parts_lse"][h]) < 1e-15
    np.testing.assert_allclose(a[0, 0], t["expect_a"], atol=1e-15)
    assert abs(lse[0, 0] - t["expect_lse"]) < 1e-15


def test_last_host_equals_prefill_oracle():
    # the last host's step is the prefill mask with no anchor, the cache as a
    # single passing slot and the new tokens as the local block
    rng = np.random.default_rng(1)
    q, kc, vc, kn, vn = _case(rng, n_q=6, n_kv=2, d=32, lc=37, n_new=9)
    a, lse = oracle.decode_attention_ref(q, kc, vc, kn, vn)
    o, l = oracle.attention_ref(q, kn, vn, kc[None], vc[None], anchor_len=0)
    np.testing.assert_allclose(a, o, atol=1e-12)
    np.testing.assert_allclose(lse, l, atol=1e-12)


def test_brute_force_python():
    # pure-Python softmax per (head, token), other host (no new K/V) and last host
    rng = np.random.default_rng(2)
    q, kc, vc, kn, vn = _case(rng, n_q=2, n_kv=1, d=4, lc=5, n_new=3)
    f = oracle.bf16_to_f64
    for with_new in (False, True):
        a, lse = oracle.decode_attention_ref(q, kc, vc, kn if with_new else None,
                                             vn if with_new else None)
        for h in range(2):
            for j in range(3):
                keys = [f(kc[0, i]) for i in range(5)]
                vals = [f(vc[0, i]) for i in range(5)]
                if with_new:
                    keys += [f(kn[0, i]) for i in range(j + 1)]
                    vals += [f(vn[0, i]) for i in range(j + 1)]
                z = [sum(f(q[h, j])[c] * kk[c] for c in range(4)) / 2.0 for kk in keys]
                m = max(z)
                w = [math.exp(x - m) for x in z]
                s = sum(w)
                exp_o = [sum(w[i] * vals[i][c] for i in range(len(w))) / s for c in range(4)]
                np.testing.assert_allclose(a[h, j], exp_o, atol=1e-12)
                assert abs(lse[h, j] - (m + math.log(s))) < 1e-12


def test_zero_query_closed_form():
    rng = np.random.default_rng(3)
    _, kc, vc, kn, vn = _case(rng, n_q=4, n_kv=2, d=8, lc=11, n_new=4)
    q = np.zeros((4, 4, 8))
    a, lse = oracle.decode_attention_ref(q, kc, vc, kn, vn)
    f = oracle.bf16_to_f64
    for h in range(4):
        kv = h // 2
        allv = np.concatenate([f(vc[kv]), f(vn[kv])])
        for j in range(4):
            n = 11 + j + 1
            np.testing.assert_allclose(a[h, j], allv[:n].mean(axis=0), atol=1e-12)
            assert abs(lse[h, j] - math.log(n)) < 1e-12
    a0, lse0 = oracle.decode_attention_ref(q, kc, vc)
    np.testing.assert_allclose(lse0, math.log(11), atol=1e-12)


@pytest.mark.parametrize("cuts", [[0, 40], [0, 7, 40], [0, 1, 2, 30, 40], [0, 0, 13, 40]])
def test_merge_of_any_split_equals_one_softmax(cuts):
    # hosts holding consecutive pieces of one cache (an empty piece included),
    # the last host appending the new tokens: merging their partials must
    # equal one softmax over everything (Alg. 3)
    rng = np.random.default_rng(4)
    q, kc, vc, kn, vn = _case(rng, n_q=4, n_kv=2, d=16, lc=40, n_new=3)
    caches = [(kc[:, a:b], vc[:, a:b]) for a, b in zip(cuts[:-1], cuts[1:])]
    a, lse, _ = oracle.stage2_ref(q, caches, kn, vn)
    a1, lse1 = oracle.decode_attention_ref(q, kc, vc, kn, vn)
    np.testing.assert_allclose(a, a1, atol=1e-12)
    np.testing.assert_allclose(lse, lse1, atol=1e-12)


def test_gqa_equals_repeated_kv():
    rng = np.random.default_rng(5)
    q, kc, vc, kn, vn = _case(rng, n_q=6, n_kv=2, d=8, lc=9, n_new=2)
    a, lse = oracle.decode_attention_ref(q, kc, vc, kn, vn)
    rep = lambda x: np.repeat(x, 3, axis=0)  # noqa: E731
    a2, lse2 = oracle.decode_attention_ref(q, rep(kc), rep(vc), rep(kn), rep(vn))
    np.testing.assert_allclose(a, a2, atol=1e-13)
    np.testing.assert_allclose(lse, lse2, atol=1e-13)


def test_scale_is_scaled_query():
    rng = np.random.default_rng(6)
    q = rng.standard_normal((2, 3, 8))
    kc, vc = rng.standard_normal((1, 7, 8)), rng.standard_normal((1, 7, 8))
    a, lse = oracle.decode_attention_ref(q, kc, vc, scale=0.7)
    a2, lse2 = oracle.decode_attention_ref(q * 0.7 * math.sqrt(8), kc, vc)
    np.testing.assert_allclose(a, a2, atol=1e-12)
    np.testing.assert_allclose(lse, lse2, atol=1e-12)


def test_empty_cache_rows():
    # a host with an empty cache and no new K/V has nothing to attend to:
    # A = 0, lse = -inf, and the merge drops it
    q = np.ones((1, 2, 4))
    a, lse = oracle.decode_attention_ref(q, np.zeros((1, 0, 4)), np.zeros((1, 0, 4)))
    assert np.all(a == 0) and np.all(np.isneginf(lse))
    a2, l2 = oracle.merge_ref(np.stack([a, np.full_like(a, 2.0)]), np.stack([lse, np.zeros_like(lse)]))
    np.testing.assert_allclose(a2, 2.0)
    np.testing.assert_allclose(l2, 0.0)
