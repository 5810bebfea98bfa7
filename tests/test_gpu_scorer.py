"""GPU parity of the retaining-head scorer (Sec. 3.4; App. B) through the C
ABI against the fp64 oracle, with synthetic weights.

Bar: scores within max-abs 1e-4.  The first layer accumulates bf16
products of magnitude ~1/sqrt(features) in fp32 and the rest is fp32, so the
expected error is ~1e-6 (measured); 1e-4 leaves room for the fast fp32 exp of SiLU.  The
selection made from GPU scores is checked to be a valid top-l_p of the
oracle's scores up to that tolerance (ties within it may go either way).
"""
import numpy as np
import pytest

import oracle
from paper_2502_12085_amd import inputs
from gpu_util import dev_bf16, need_gpu, say, run_compress

pytestmark = pytest.mark.gpu
SCORE_MAX_ABS = 1e-4


def _run(n_q, n_kv, d, la, lb, hidden, seed=0):
    torch = need_gpu()
    from paper_2502_12085_amd import apb
    rng = np.random.default_rng(seed)
    q, k, v = (inputs.f32_to_bf16_bits(rng.standard_normal((n, la + lb, d)).astype(np.float32))
               for n in (n_q, n_kv, n_kv))
    w = inputs.make_scorer_weights(n_q, n_kv, d, hidden, seed)
    p = apb.ScorerProblem(la, lb, n_q, n_kv, d, hidden)
    ws = torch.empty(apb.scorer_workspace_size(p), dtype=torch.uint8, device="cuda")
    s = torch.full((n_kv, lb), float("nan"), dtype=torch.float32, device="cuda")
    f = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()  # noqa: E731
    dq, dk, dv = dev_bf16(q), dev_bf16(k), dev_bf16(v)
    apb.retaining_scores(p, dq, dk, dv, dev_bf16(w["w1"]), f(w["b1"]), f(w["w2"]), f(w["b2"]), s, ws)
    torch.cuda.synchronize()
    ref = oracle.retaining_scores_ref(q, k, v, w["w1"], w["b1"], w["w2"], w["b2"], anchor_len=la)
    return s.cpu().numpy().astype(np.float64), ref, (dk, dv)


@pytest.mark.parametrize("shape", [
    # n_q, n_kv, d, La, Lb, hidden
    (4, 1, 64, 128, 512, 1024),     # tiny layer
    (4, 1, 64, 0, 300, 256),        # ragged tokens, no anchor, one hidden block
    (6, 2, 128, 77, 1000, 512),     # ragged, GQA 3
    (32, 8, 128, 64, 257, 1024),    # Llama-shaped features, ragged last tile
    (56, 8, 128, 0, 256, 256),      # Yi-shaped features
])
def test_scorer_matches_oracle(shape):
    say(f"[scorer] {shape}")
    got, ref, _ = _run(*shape)
    err = np.abs(got - ref)
    say(f"  max {err.max():.3e} mean {err.mean():.3e} (scores rms {np.sqrt((ref**2).mean()):.3f})")
    assert np.isfinite(got).all()
    assert err.max() <= SCORE_MAX_ABS


def test_scorer_deterministic():
    a, _, _ = _run(6, 2, 128, 10, 700, 512, seed=3)
    b, _, _ = _run(6, 2, 128, 10, 700, 512, seed=3)
    assert np.array_equal(a, b)


def test_scorer_then_compressor_selects_a_valid_top_lp():
    # GPU scores feed the compressor; every selected unit must rank in the
    # oracle's top l_p up to the score tolerance
    torch = need_gpu()
    n_q, n_kv, d, la, lb, hidden, lp = 8, 2, 128, 64, 2048, 1024, 256
    got, ref, (dk, dv) = _run(n_q, n_kv, d, la, lb, hidden, seed=5)
    prob = inputs.Problem(2, 1, la, lb, lp, n_q, n_kv, d)
    idx, _, _ = run_compress(prob, torch.from_numpy(got.astype(np.float32)).cuda(), dk, dv)
    idx = idx.cpu().numpy()
    for h in range(n_kv):
        thr = np.sort(ref[h])[::-1][lp - 1]  # l_p-th largest oracle score
        sel = np.zeros(lb, bool)
        sel[idx[h]] = True
        assert sel.sum() == lp
        assert (ref[h][sel] >= thr - 2 * SCORE_MAX_ABS).all()
        assert (ref[h][~sel] <= thr + 2 * SCORE_MAX_ABS).all()


def test_scorer_full_size_sampled():
    # the 128K Llama-8B-shaped host share: 16384 local tokens, 6144 features
    torch = need_gpu()
    from paper_2502_12085_amd import apb
    wl = inputs.WORKLOADS["llama8b_128k"]
    p = wl.problem
    say("[scorer] llama8b_128k full size")
    inp = inputs.make_inputs(wl, 0)
    w = inputs.make_scorer_weights(p.n_q_heads, p.n_kv_heads, p.head_dim, seed=0)
    sp = apb.ScorerProblem(p.anchor_len, p.local_len, p.n_q_heads, p.n_kv_heads, p.head_dim,
                           inputs.SCORER_HIDDEN)
    ws = torch.empty(apb.scorer_workspace_size(sp), dtype=torch.uint8, device="cuda")
    s = torch.empty((p.n_kv_heads, p.local_len), dtype=torch.float32, device="cuda")
    f = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()  # noqa: E731
    apb.retaining_scores(sp, dev_bf16(inp["q"]), dev_bf16(inp["k"]), dev_bf16(inp["v"]),
                         dev_bf16(w["w1"]), f(w["b1"]), f(w["w2"]), f(w["b2"]), s, ws)
    torch.cuda.synchronize()
    got = s.cpu().numpy().astype(np.float64)
    # sampled tokens: tile edges, the last token, random ones
    rng = np.random.default_rng(0)
    toks = np.unique(np.concatenate([[0, 1, 255, 256, 257, 8191, 8192, p.local_len - 1],
                                     rng.integers(0, p.local_len, 48)]))
    la = p.anchor_len
    sel = lambda t: t[:, la + toks]  # noqa: E731
    ref = oracle.retaining_scores_ref(np.concatenate([inp["q"][:, :la], sel(inp["q"])], axis=1),
                                      np.concatenate([inp["k"][:, :la], sel(inp["k"])], axis=1),
                                      np.concatenate([inp["v"][:, :la], sel(inp["v"])], axis=1),
                                      w["w1"], w["b1"], w["w2"], w["b2"], anchor_len=la)
    err = np.abs(got[:, toks] - ref)
    say(f"  max {err.max():.3e} mean {err.mean():.3e}")
    assert np.isfinite(got).all()
    assert err.max() <= SCORE_MAX_ABS
