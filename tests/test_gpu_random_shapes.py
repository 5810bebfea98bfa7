"""GPU parity on seeded random shapes, through the C ABI, against the fp64
oracle: the modified-mask attention with its LSE (Sec. 3.6, Eq. 2), the
ArgTop-l_p selection and gather (Sec. 3.4), the decoding step (Alg. 3) and
the retaining-head scorer (Sec. 3.4), each at the bar of its dedicated test.

The shapes are drawn from a fixed seed, so every run checks the same cases:
any host index, anchor and local lengths that are no tile multiple, l_p from
0 to Lb, GQA ratios 1-8 and both head sizes, sized so that the oracle
finishes each case in a few seconds.
"""
import numpy as np
import pytest

import oracle
from paper_2502_12085_amd import inputs
from gpu_util import (assert_attention_close, dev_bf16, host_bf16_to_f64, host_bits, need_gpu,
                      run_attention, run_compress, say, upload)

pytestmark = pytest.mark.gpu


def _attention_shapes(n=24, seed=20261202):
    rng = np.random.default_rng(seed)
    shapes = []
    for _ in range(n):
        hosts = int(rng.integers(1, 7))
        host_idx = int(rng.integers(0, hosts))
        la = 0 if rng.random() < 0.25 else int(rng.integers(1, 400))
        lb = int(rng.integers(1, 1000))
        lp = int(rng.integers(0, min(lb, 300) + 1))
        n_kv = int(rng.choice([1, 2]))
        g = int(rng.choice([1, 2, 3, 4]))
        d = int(rng.choice([64, 128]))
        shapes.append((hosts, host_idx, la, lb, lp, n_kv * g, n_kv, d))
    return shapes


ATTN_SHAPES = _attention_shapes()


@pytest.mark.parametrize("shape", ATTN_SHAPES, ids=[str(s) for s in ATTN_SHAPES])
def test_random_attention_and_selection(shape):
    need_gpu()
    p = inputs.Problem(*shape)
    wl = inputs.Workload("random", p)
    say(f"[random attention] {p}")
    inp = inputs.make_inputs(wl, seed=sum(shape))
    dv = upload(inp)
    o, lse = run_attention(p, dv)
    o_ref, lse_ref = oracle.attention_ref(inp["q"], inp["k"], inp["v"], inp["k_pass"],
                                          inp["v_pass"], anchor_len=p.anchor_len)
    assert_attention_close(host_bf16_to_f64(o), lse.cpu().numpy(), o_ref, lse_ref, str(shape))
    if p.pass_len > 0:
        idx, ok, ov = run_compress(p, dv["scores"], dv["k"], dv["v"])
        ridx, rk, rv = oracle.compress_ref(inp["scores"], inp["k"], inp["v"], p.pass_len,
                                           p.anchor_len)
        assert np.array_equal(idx.cpu().numpy(), ridx)
        assert np.array_equal(host_bits(ok), rk) and np.array_equal(host_bits(ov), rv)


def _decode_shapes(n=24, seed=20261203):
    rng = np.random.default_rng(seed)
    shapes = []
    for _ in range(n):
        n_kv = int(rng.choice([1, 2, 4]))
        g = int(rng.choice([1, 2, 4, 5, 7, 8]))
        d = int(rng.choice([64, 128]))
        lc = 0 if rng.random() < 0.1 else int(rng.integers(1, 3000))
        n_new = int(rng.choice([1, 1, 2, int(rng.integers(3, 70))]))
        append = int(rng.integers(0, 2)) if lc > 0 else 1
        shapes.append((n_kv * g, n_kv, d, lc, n_new, append))
    return shapes


DECODE_SHAPES = _decode_shapes()


@pytest.mark.parametrize("shape", DECODE_SHAPES, ids=[str(s) for s in DECODE_SHAPES])
def test_random_decode(shape):
    torch = need_gpu()
    from paper_2502_12085_amd import apb
    n_q, n_kv, d, lc, n_new, app = shape
    say(f"[random decode] {shape}")
    case = inputs.make_decode_case(n_q, n_kv, d, [lc], n_new, seed=sum(shape))
    kc, vc = case["caches"][0]
    kn = case["k_new"] if app else None
    vn = case["v_new"] if app else None
    p = apb.DecodeProblem(n_q, n_kv, d, lc, n_new, app)
    ws = torch.empty(max(apb.decode_workspace_size(p), 16), dtype=torch.uint8, device="cuda")
    o = torch.full((n_q, n_new, d), float("nan"), dtype=torch.float32, device="cuda")
    lse = torch.full((n_q, n_new), float("nan"), dtype=torch.float32, device="cuda")
    apb.decode_attention(p, dev_bf16(case["q"]), dev_bf16(kc) if lc > 0 else None,
                         dev_bf16(vc) if lc > 0 else None, dev_bf16(kn) if app else None,
                         dev_bf16(vn) if app else None, o, lse, ws)
    torch.cuda.synchronize()
    o_ref, lse_ref = oracle.decode_attention_ref(case["q"], kc, vc, kn, vn)
    assert_attention_close(o.cpu().numpy().astype(np.float64),
                           lse.cpu().numpy().astype(np.float64), o_ref, lse_ref, str(shape))


def _scorer_shapes(n=10, seed=20261204):
    rng = np.random.default_rng(seed)
    shapes = []
    for _ in range(n):
        n_kv = int(rng.choice([1, 2, 4, 8]))
        g = int(rng.choice([1, 2, 4]))
        d = int(rng.choice([64, 128]))
        la = int(rng.integers(0, 300))
        lb = int(rng.integers(1, 900))
        hidden = int(rng.choice([256, 512]))
        shapes.append((n_kv * g, n_kv, d, la, lb, hidden))
    return shapes


SCORER_SHAPES = _scorer_shapes()


@pytest.mark.parametrize("shape", SCORER_SHAPES, ids=[str(s) for s in SCORER_SHAPES])
def test_random_scorer(shape):
    from test_gpu_scorer import SCORE_MAX_ABS, _run
    say(f"[random scorer] {shape}")
    got, ref, _ = _run(*shape, seed=sum(shape))
    assert np.isfinite(got).all()
    assert np.abs(got - ref).max() <= SCORE_MAX_ABS
