"""GPU parity of the decoding stage (Alg. 3) through the C ABI against the
fp64 oracle: one host's partial attention (fp32 output, LSE) and MergeScore.

Bar: the attention bar (output max-abs 2e-2, mean-abs 2e-3; LSE max-abs
1e-3).  Cases span several 32-key blocks and splits with ragged tails, both
head sizes, an empty cache, more rows than one 32-row block, every host of a
simulated decoding step, GQA groups of 128 rows and more (where eight waves
share each K/V block), and the full-size 128K Llama-8B-shaped steps (every
row: a decoding step has only n_q * n_new rows).
"""
import numpy as np
import pytest

import oracle
from paper_2502_12085_amd import inputs
from gpu_util import assert_attention_close, dev_bf16, host_bf16_to_f64, need_gpu, say
import rescale_cases as rc

pytestmark = pytest.mark.gpu


def _run_decode(q, kc, vc, kn, vn, n_q, n_kv, d, scale=0.0):
    torch = need_gpu()
    from paper_2502_12085_amd import apb
    n_new = q.shape[1]
    lc = kc.shape[1]
    p = apb.DecodeProblem(n_q, n_kv, d, lc, n_new, 1 if kn is not None else 0)
    ws = torch.empty(apb.decode_workspace_size(p), dtype=torch.uint8, device="cuda")
    o = torch.full((n_q, n_new, d), float("nan"), dtype=torch.float32, device="cuda")
    lse = torch.full((n_q, n_new), float("nan"), dtype=torch.float32, device="cuda")
    dk = dev_bf16(kc) if lc > 0 else None
    dvv = dev_bf16(vc) if lc > 0 else None
    apb.decode_attention(p, dev_bf16(q), dk, dvv, dev_bf16(kn) if kn is not None else None,
                         dev_bf16(vn) if vn is not None else None, o, lse, ws, scale)
    torch.cuda.synchronize()
    return o.cpu().numpy().astype(np.float64), lse.cpu().numpy().astype(np.float64)


@pytest.mark.parametrize("shape", [
    # n_q, n_kv, d, Lc, n_new, append
    (4, 1, 64, 512, 3, 1),        # tiny decode: last host
    (4, 1, 64, 512, 3, 0),        # tiny decode: another host
    (8, 2, 128, 1000, 1, 1),      # ragged cache, one new token
    (8, 2, 128, 33, 5, 1),        # just over one block
    (6, 2, 128, 31, 2, 0),        # under one block
    (8, 2, 128, 0, 4, 1),         # empty cache: the new tokens alone
    (12, 2, 128, 777, 17, 1),     # 102 rows per KV head: four 32-row blocks
    (7, 7, 64, 3000, 40, 0),      # no GQA, 40 rows
    (56, 8, 128, 4100, 2, 1),     # Yi-shaped group of 7
    # >= 128 rows per KV head: 8 waves share each K/V block
    (8, 2, 64, 1000, 40, 1),      # 160 rows: one partly filled 256-row group, d = 64
    (16, 2, 128, 2000, 40, 1),    # 320 rows: two row groups, the second ragged
    (4, 4, 128, 513, 130, 1),     # no GQA, 130 causal new tokens over a ragged cache
    (8, 2, 128, 0, 64, 1),        # empty cache, 256 rows of new tokens alone
    (56, 8, 128, 100, 20, 0),     # few keys (four blocks), 140 rows, no append
    # eight-wave path, 128-key tiles: cache ends on, just past and just before
    # a tile edge, one-tile splits, one cached key, row groups past 256
    (15, 3, 128, 129, 50, 0),     # 250 rows, cache one key past a tile edge, no append
    (10, 2, 64, 1, 67, 1),        # one cached key, then 67 causal new tokens
    (1, 1, 64, 1000, 391, 1),     # no GQA, 391 rows (two row groups), long new block
    (6, 3, 128, 255, 116, 1),     # cache one key short of two tiles
    (10, 2, 128, 128, 77, 0),     # cache exactly one tile, 385 rows, no append
    (7, 1, 64, 4100, 39, 1),      # group of 7, many splits
])
def test_decode_matches_oracle(shape):
    n_q, n_kv, d, lc, n_new, app = shape
    say(f"[decode] {shape}")
    case = inputs.make_decode_case(n_q, n_kv, d, [lc], n_new, seed=11)
    kc, vc = case["caches"][0]
    kn = case["k_new"] if app else None
    vn = case["v_new"] if app else None
    o, lse = _run_decode(case["q"], kc, vc, kn, vn, n_q, n_kv, d)
    o_ref, lse_ref = oracle.decode_attention_ref(case["q"], kc, vc, kn, vn)
    assert_attention_close(o, lse, o_ref, lse_ref, f"decode {shape}")


def _scale_bf16(bits, k):
    """bf16 bits of the values times 2**k (exact while nothing overflows)."""
    x = inputs.bf16_bits_to_f32(bits).astype(np.float64) * 2.0 ** k
    out = inputs.f32_to_bf16_bits(x.astype(np.float32))
    assert np.array_equal(inputs.bf16_bits_to_f32(out).astype(np.float64), x)
    return out


@pytest.mark.parametrize("shape", [(8, 2, 128, 1000, 64, 1), (4, 1, 64, 300, 200, 0)])
def test_decode_split_partials_follow_the_scale_of_v(shape):
    """The eight-wave path (256 rows per KV head) keeps its split partials in
    fp16 against a per-row power-of-two scale: every step is then exact under
    V -> 2^k V, so O scales bit for bit and the LSE does not move, for values
    far outside fp16's range (2^16 times N(0,1)) and deep in its subnormals
    (2^-24 times)."""
    n_q, n_kv, d, lc, n_new, app = shape
    assert (n_q // n_kv) * n_new >= 128
    say(f"[decode V scale] {shape}")
    case = inputs.make_decode_case(n_q, n_kv, d, [lc], n_new, seed=23)
    kc, vc = case["caches"][0]
    kn = case["k_new"] if app else None
    vn = case["v_new"] if app else None
    o, lse = _run_decode(case["q"], kc, vc, kn, vn, n_q, n_kv, d)
    o_ref, lse_ref = oracle.decode_attention_ref(case["q"], kc, vc, kn, vn)
    assert_attention_close(o, lse, o_ref, lse_ref, f"decode V scale {shape}")
    for k in (16, -24):
        o_k, lse_k = _run_decode(case["q"], kc, _scale_bf16(vc, k), kn,
                                 _scale_bf16(vn, k) if app else None, n_q, n_kv, d)
        assert np.array_equal(o_k, o * 2.0 ** k), k
        assert np.array_equal(lse_k, lse), k


def test_decode_no_keys_rows():
    # no cache and nothing appended: every row sees nothing -> o = 0, lse = -inf
    case = inputs.make_decode_case(4, 2, 128, [0], 2, seed=3)
    kc, vc = case["caches"][0]
    o, lse = _run_decode(case["q"], kc, vc, None, None, 4, 2, 128)
    assert np.all(o == 0) and np.all(np.isneginf(lse))


def test_decode_custom_scale_and_determinism():
    case = inputs.make_decode_case(8, 2, 128, [2500], 3, seed=5)
    kc, vc = case["caches"][0]
    args = (case["q"], kc, vc, case["k_new"], case["v_new"], 8, 2, 128)
    o1, l1 = _run_decode(*args, scale=0.05)
    o2, l2 = _run_decode(*args, scale=0.05)
    assert np.array_equal(o1, o2) and np.array_equal(l1, l2)
    o_ref, lse_ref = oracle.decode_attention_ref(case["q"], kc, vc, case["k_new"], case["v_new"],
                                                 scale=0.05)
    assert_attention_close(o1, l1, o_ref, lse_ref, "decode scale 0.05")


@pytest.mark.parametrize("shape", [rc.DECODE_ONE_SPLIT["one_wave"][0],
                                   rc.DECODE_ONE_SPLIT["eight_wave"][0], rc.DECODE_MANY_SPLITS])
def test_decode_late_max_raise_scale_one(shape):
    """softmax_scale = 1.0: the running max moves after a split's first block
    and rescales a non-zero accumulator (CPU replay of the kernels' decision:
    tests/test_lazy_max_coverage.py); one-wave and eight-wave kernels."""
    n_q, n_kv, d, lc, n_new, app = shape
    say(f"[decode scale 1.0] {shape}")
    q, kc, vc, kn, vn = rc.decode_inputs(shape)
    o, lse = _run_decode(q, kc, vc, kn, vn, n_q, n_kv, d, scale=rc.SCALE)
    o_ref, lse_ref = oracle.decode_attention_ref(q, kc, vc, kn, vn, scale=rc.SCALE)
    assert_attention_close(o, lse, o_ref, lse_ref, f"decode scale 1.0 {shape}")


def _run_merge(o_parts, lse_parts):
    torch = need_gpu()
    from paper_2502_12085_amd import apb
    P, rows, d = o_parts.shape
    o = torch.full((rows, d), float("nan"), dtype=torch.bfloat16, device="cuda")
    lse = torch.full((rows,), float("nan"), dtype=torch.float32, device="cuda")
    apb.merge_partials(torch.from_numpy(np.ascontiguousarray(o_parts, np.float32)).cuda(),
                       torch.from_numpy(np.ascontiguousarray(lse_parts, np.float32)).cuda(), o, lse)
    torch.cuda.synchronize()
    return host_bf16_to_f64(o), lse.cpu().numpy().astype(np.float64)


@pytest.mark.parametrize("P,rows,d", [(1, 5, 64), (8, 32, 128), (3, 1000, 128), (64, 7, 64)])
def test_merge_matches_oracle(P, rows, d):
    rng = np.random.default_rng(P * 1000 + rows)
    o_parts = rng.standard_normal((P, rows, d)).astype(np.float32)
    lse_parts = (rng.standard_normal((P, rows)) * 5).astype(np.float32)
    if P > 1:
        lse_parts[0, ::3] = -np.inf  # empty parts are dropped
        o_parts[0, ::3] = 0.0
    o, lse = _run_merge(o_parts, lse_parts)
    o_ref, lse_ref = oracle.merge_ref(o_parts, lse_parts)
    assert_attention_close(o, lse, o_ref, lse_ref, f"merge P={P} rows={rows} d={d}")


def test_merge_all_parts_empty():
    o_parts = np.zeros((3, 4, 128), np.float32)
    lse_parts = np.full((3, 4), -np.inf, np.float32)
    o, lse = _run_merge(o_parts, lse_parts)
    assert np.all(o == 0) and np.all(np.isneginf(lse))


def _stage2(wl, seed=0):
    """Every host's partial on the GPU, then the GPU merge, against one
    softmax over all hosts' caches plus the new tokens."""
    torch = need_gpu()
    from paper_2502_12085_amd import apb
    case = inputs.make_decode_inputs(wl, seed)
    H = len(case["caches"])
    n_q, n_kv, d, n_new = wl.n_q_heads, wl.n_kv_heads, wl.head_dim, wl.n_new
    parts_o = torch.empty((H, n_q * n_new, d), dtype=torch.float32, device="cuda")
    parts_l = torch.empty((H, n_q * n_new), dtype=torch.float32, device="cuda")
    dq = dev_bf16(case["q"])
    for h, (kc, vc) in enumerate(case["caches"]):
        last = h == H - 1
        p = apb.DecodeProblem(n_q, n_kv, d, kc.shape[1], n_new, 1 if last else 0)
        ws = torch.empty(apb.decode_workspace_size(p), dtype=torch.uint8, device="cuda")
        apb.decode_attention(p, dq, dev_bf16(kc), dev_bf16(vc),
                             dev_bf16(case["k_new"]) if last else None,
                             dev_bf16(case["v_new"]) if last else None,
                             parts_o[h].view(n_q, n_new, d), parts_l[h].view(n_q, n_new), ws)
    o = torch.empty((n_q * n_new, d), dtype=torch.bfloat16, device="cuda")
    lse = torch.empty((n_q * n_new,), dtype=torch.float32, device="cuda")
    apb.merge_partials(parts_o, parts_l, o, lse)
    torch.cuda.synchronize()
    kc_all = np.concatenate([c[0] for c in case["caches"]], axis=1)
    vc_all = np.concatenate([c[1] for c in case["caches"]], axis=1)
    o_ref, lse_ref = oracle.decode_attention_ref(case["q"], kc_all, vc_all, case["k_new"],
                                                 case["v_new"])
    og = host_bf16_to_f64(o).reshape(n_q, n_new, d)
    assert_attention_close(og, lse.cpu().numpy().reshape(n_q, n_new), o_ref, lse_ref,
                           f"stage-2 {wl.name}")


def test_stage2_tiny_all_hosts():
    _stage2(inputs.DECODE_WORKLOADS["tiny_decode"])


@pytest.mark.parametrize("name", ["llama8b_128k_decode", "llama8b_128k_question"])
def test_stage2_full_size(name):
    say(f"[stage-2] {name}")
    _stage2(inputs.DECODE_WORKLOADS[name])
