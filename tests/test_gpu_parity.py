"""GPU parity: the HIP path through the C ABI against the fp64 oracle.

Attention: output within max-abs 2e-2 / mean-abs 2e-3, LSE within 1e-3.
Selection and gather: bit-exact.  Small problems are compared element by
element; the full-size workloads on sampled rows (segment boundaries, tile
edges, the last row, random rows) that the oracle computes one by one.
"""
import dataclasses
import json
import math
import os
import zlib

import numpy as np
import pytest

import oracle
from paper_2502_12085_amd import inputs
from gpu_util import (O_REL_PEAKED, assert_attention_close, host_bf16_to_f64, host_bits,
                      need_gpu, run_attention, run_compress, say, upload, dev_bf16)
import rescale_cases as rc

pytestmark = pytest.mark.gpu
GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _wl(name, **kw):
    wl = inputs.WORKLOADS[name]
    if kw:
        wl = dataclasses.replace(wl, problem=dataclasses.replace(wl.problem, **kw))
    return wl


def _full_check(wl, seed=0, heads=None):
    torch = need_gpu()
    p = wl.problem
    say(f"[attention] {wl.name} {p}")
    inp = inputs.make_inputs(wl, seed)
    dv = upload(inp)
    o, lse = run_attention(p, dv)
    o_ref, lse_ref = oracle.attention_ref(inp["q"], inp["k"], inp["v"], inp["k_pass"],
                                          inp["v_pass"], anchor_len=p.anchor_len, heads=heads)
    og = host_bf16_to_f64(o)
    lg = lse.cpu().numpy()
    if heads is not None:
        og, lg = og[heads], lg[heads]
    assert_attention_close(og, lg, o_ref, lse_ref, wl.name)
    return o, lse


@pytest.mark.parametrize("host_idx", [0, 1, 2, 3])
def test_tiny_every_host(host_idx):
    _full_check(_wl("tiny", host_idx=host_idx))


@pytest.mark.parametrize("shape", [
    # n_hosts, host_idx, La, Lb, l_p, n_q, n_kv, d   (ragged: not tile multiples)
    (4, 2, 100, 333, 17, 6, 2, 128),
    (4, 2, 100, 333, 17, 6, 2, 64),
    (8, 5, 0, 300, 40, 4, 4, 128),       # no anchor
    (2, 0, 77, 200, 50, 2, 1, 128),      # first host: no passing block
    (4, 3, 64, 256, 0, 3, 1, 64),        # l_p = 0
    (3, 1, 1, 1, 1, 1, 1, 128),          # one anchor row, one local row
    (4, 3, 130, 129, 129, 5, 5, 128),    # l_p = Lb, MHA
    (8, 7, 200, 700, 33, 7, 1, 128),     # GQA ratio 7
    (1, 0, 0, 1000, 0, 4, 2, 128),       # one host, no anchor: plain causal attention over B
    (4, 0, 0, 300, 300, 2, 1, 64),       # first host, no anchor, l_p = Lb (nothing passed in)
])
def test_ragged_shapes(shape):
    wl = inputs.Workload("ragged", inputs.Problem(*shape))
    _full_check(wl, seed=sum(shape))


def test_toy_golden_on_gpu():
    """The hand-worked uniform toy (Q = 0), head_dim padded to 64 with zeros."""
    torch = need_gpu()
    spec = json.load(open(os.path.join(GOLDEN, "toy_attention.json")))
    c = spec["cases"][0]
    d = 64
    pad = lambda rows: np.pad(np.array(rows, np.float32), ((0, 0), (0, d - len(rows[0]))))
    p = inputs.Problem(2, 1, 1, 2, 1, 1, 1, d)
    dv = {
        "q": dev_bf16(inputs.f32_to_bf16_bits(pad(c["q_rows"]))[None]),
        "k": dev_bf16(inputs.f32_to_bf16_bits(pad(c["k_anchor"] + c["k_local"]))[None]),
        "v": dev_bf16(inputs.f32_to_bf16_bits(pad(c["v_anchor"] + c["v_local"]))[None]),
        "k_pass": dev_bf16(inputs.f32_to_bf16_bits(pad(c["k_pass"]))[None, None]),
        "v_pass": dev_bf16(inputs.f32_to_bf16_bits(pad(c["v_pass"]))[None, None]),
    }
    o, lse = run_attention(p, dv)
    og = host_bf16_to_f64(o)[0, :, :2]
    np.testing.assert_allclose(og, np.array(c["expect_o"]), atol=1e-2)
    np.testing.assert_allclose(lse.cpu().numpy()[0], np.array(c["expect_lse"]), atol=1e-5)


def test_constant_v_gives_one():
    """Rows sum to one: with V = 1 every output is 1."""
    torch = need_gpu()
    wl = _wl("tiny")
    p = wl.problem
    inp = inputs.make_inputs(wl, 3)
    dv = upload(inp)
    dv["v"] = torch.ones_like(dv["v"])
    dv["v_pass"] = torch.ones_like(dv["v_pass"])
    o, _ = run_attention(p, dv)
    assert (o.float() == 1.0).all()


def test_softmax_scale_argument():
    torch = need_gpu()
    wl = _wl("tiny")
    p = wl.problem
    inp = inputs.make_inputs(wl, 4)
    dv = upload(inp)
    o, lse = run_attention(p, dv, softmax_scale=0.05)
    o_ref, lse_ref = oracle.attention_ref(inp["q"], inp["k"], inp["v"], inp["k_pass"],
                                          inp["v_pass"], anchor_len=p.anchor_len, scale=0.05)
    assert_attention_close(host_bf16_to_f64(o), lse.cpu().numpy(), o_ref, lse_ref, "scale 0.05")


@pytest.mark.parametrize("name", list(rc.ATTENTION))
def test_late_max_raise_scale_one(name):
    """softmax_scale = 1.0: the running max moves after the first tile and a
    non-zero O accumulator is rescaled (CPU replay of the kernel's decision:
    tests/test_lazy_max_coverage.py), every row against the oracle.  The
    softmax is peaked, so |O| approaches max|V| and the O bar adds the
    arithmetic's rounding bound (gpu_util.O_REL_PEAKED)."""
    need_gpu()
    p, inp = rc.attention_inputs(name)
    say(f"[attention scale 1.0] {name} {p}")
    o, lse = run_attention(p, upload(inp), softmax_scale=rc.SCALE)
    o_ref, lse_ref = oracle.attention_ref(inp["q"], inp["k"], inp["v"], inp["k_pass"],
                                          inp["v_pass"], anchor_len=p.anchor_len, scale=rc.SCALE)
    assert_attention_close(host_bf16_to_f64(o), lse.cpu().numpy(), o_ref, lse_ref,
                           f"{name} scale 1.0", o_rel=O_REL_PEAKED)


def test_planted_late_key_default_scale():
    """A key planted three tiles in along one query: that query's wave raises
    its max late at the default scale too."""
    need_gpu()
    p, inp = rc.attention_inputs("ragged_d128_planted")
    o, lse = run_attention(p, upload(inp))
    o_ref, lse_ref = oracle.attention_ref(inp["q"], inp["k"], inp["v"], inp["k_pass"],
                                          inp["v_pass"], anchor_len=p.anchor_len)
    assert_attention_close(host_bf16_to_f64(o), lse.cpu().numpy(), o_ref, lse_ref,
                           "planted late key", o_rel=O_REL_PEAKED)


def test_deterministic_and_fully_written():
    torch = need_gpu()
    wl = _wl("llama8b_32k", n_q_heads=8, n_kv_heads=2)
    p = wl.problem
    dv = upload(inputs.make_inputs(wl, 5))
    o1, l1 = run_attention(p, dv, fill=float("nan"))
    o2, l2 = run_attention(p, dv, fill=0.0)
    assert not torch.isnan(o1.float()).any() and not torch.isnan(l1).any()
    assert torch.equal(o1.view(torch.int16), o2.view(torch.int16))
    assert torch.equal(l1.view(torch.int32), l2.view(torch.int32))


def test_unaligned_to_256_bytes_and_no_lse():
    """Operands and outputs 16 bytes (the ABI's minimum) past a 256-byte
    boundary, and lse = NULL: the same output bits as aligned buffers."""
    torch = need_gpu()
    from paper_2502_12085_amd import apb
    wl = _wl("tiny", host_idx=3)
    p = wl.problem
    inp = inputs.make_inputs(wl, 8)
    dv = upload(inp)
    o_ref, lse_ref = run_attention(p, dv)

    def shifted(t):
        flat = torch.empty(t.numel() + 8, dtype=t.dtype, device="cuda")
        view = flat[8:].view(t.shape)  # 16 bytes past the allocation's start
        view.copy_(t)
        return view

    sq, sk, sv = shifted(dv["q"]), shifted(dv["k"]), shifted(dv["v"])
    skp, svp = shifted(dv["k_pass"]), shifted(dv["v_pass"])
    assert all(t.data_ptr() % 256 == 16 for t in (sq, sk, sv, skp, svp))
    o = shifted(torch.full_like(o_ref, float("nan")))
    apb.attention_fwd(p, sq, sk, sv, skp, svp, o, None)
    torch.cuda.synchronize()
    assert torch.equal(o.view(torch.int16), o_ref.view(torch.int16))
    assert_attention_close(host_bf16_to_f64(o), lse_ref.cpu().numpy(),
                           *oracle.attention_ref(inp["q"], inp["k"], inp["v"], inp["k_pass"],
                                                 inp["v_pass"], anchor_len=p.anchor_len),
                           "16-byte aligned, no LSE")


def test_guard_bands_untouched():
    torch = need_gpu()
    from paper_2502_12085_amd import apb
    wl = _wl("tiny", host_idx=3)
    p = wl.problem
    dv = upload(inputs.make_inputs(wl, 6))
    n_o = p.n_q_heads * p.rows * p.head_dim
    n_l = p.n_q_heads * p.rows
    g = 4096
    obuf = torch.full((n_o + 2 * g,), 1234.0, dtype=torch.bfloat16, device="cuda")
    lbuf = torch.full((n_l + 2 * g,), 1234.0, dtype=torch.float32, device="cuda")
    o = obuf[g:g + n_o]
    lse = lbuf[g:g + n_l]
    apb.attention_fwd(p, dv["q"], dv["k"], dv["v"], dv["k_pass"], dv["v_pass"], o, lse)
    torch.cuda.synchronize()
    assert (obuf[:g] == 1234.0).all() and (obuf[g + n_o:] == 1234.0).all()
    assert (lbuf[:g] == 1234.0).all() and (lbuf[g + n_l:] == 1234.0).all()


def test_llama8b_32k_heads_subset_full_rows():
    """The 32K Llama-8B-shaped share: every row of one query head per KV
    group compared element by element."""
    _full_check(_wl("llama8b_32k"), heads=np.array([0, 5, 10, 15, 16, 22, 27, 31]))


def test_llama8b_128k_heads_subset_full_rows():
    """The 128K Llama-8B-shaped share (outlier K channels): every row of one
    query head per KV group, element by element."""
    _full_check(_wl("llama8b_128k"), heads=np.array([0, 5, 10, 15, 16, 22, 27, 31]))


def test_d64_many_tiles_full_rows():
    """head_dim 64 over many key and query tiles (26 key tiles of 128, ten
    query tiles, GQA 4, a ragged passing block), every row of every head."""
    _full_check(inputs.Workload("d64_mid", inputs.Problem(4, 3, 512, 2048, 250, 8, 2, 64)))


def _sample_rows(p, rng, n_random=24):
    M = p.rows
    fixed = {0, 1, 63, 64, 127, 128, 255, 256, 511, 512, p.anchor_len - 1, p.anchor_len,
             p.anchor_len + 1,
             p.anchor_len + 127, p.anchor_len + 128, M - 129, M - 128, M - 2, M - 1}
    fixed = {r for r in fixed if 0 <= r < M}
    return np.array(sorted(fixed | set(rng.integers(0, M, n_random).tolist())))


@pytest.mark.parametrize("name", ["llama8b_32k", "llama8b_128k", "qwen14b_256k", "yi34b_512k"])
def test_full_size_sampled_rows(name):
    """Sampled rows of several heads (segment boundaries, tile edges, the
    last rows, random rows); at 256K and 512K also every row of the last
    query head."""
    torch = need_gpu()
    wl = inputs.WORKLOADS[name]
    p = wl.problem
    say(f"[attention full size] {name}")
    inp = inputs.make_inputs(wl, 0)
    dv = upload(inp)
    o, lse = run_attention(p, dv)
    assert not torch.isnan(o.float()).any() and not torch.isnan(lse).any()
    rng = np.random.default_rng(1)
    heads = np.array(sorted({0, p.n_q_heads - 1} | set(rng.integers(0, p.n_q_heads, 4).tolist())))
    rows = _sample_rows(p, rng)
    o_ref, lse_ref = oracle.attention_ref(inp["q"], inp["k"], inp["v"], inp["k_pass"],
                                          inp["v_pass"], anchor_len=p.anchor_len,
                                          heads=heads, rows=rows)
    og = host_bf16_to_f64(o[torch.as_tensor(heads).cuda()][:, torch.as_tensor(rows).cuda()])
    lg = lse[torch.as_tensor(heads).cuda()][:, torch.as_tensor(rows).cuda()].cpu().numpy()
    assert_attention_close(og, lg, o_ref, lse_ref, name)
    if name in ("qwen14b_256k", "yi34b_512k"):
        # and every row of the last query head (the last KV group)
        last = np.array([p.n_q_heads - 1])
        say(f"  {name}: every row of query head {last[0]}")
        o_ref, lse_ref = oracle.attention_ref(inp["q"], inp["k"], inp["v"], inp["k_pass"],
                                              inp["v_pass"], anchor_len=p.anchor_len, heads=last)
        assert_attention_close(host_bf16_to_f64(o[last[0]])[None], lse[last[0]].cpu().numpy()[None],
                               o_ref, lse_ref, f"{name} head {last[0]}")


# ------------------------------------------------------------- compressor
def _check_compress(p, inp, what):
    dv = upload(inp)
    idx, kc, vc = run_compress(p, dv["scores"], dv["k"], dv["v"])
    ridx, rk, rv = oracle.compress_ref(inp["scores"], inp["k"], inp["v"], p.pass_len, p.anchor_len)
    gi = idx.cpu().numpy()
    bad = int((gi != ridx).sum())
    say(f"  {what}: idx mismatches {bad}")
    np.testing.assert_array_equal(gi, ridx)
    np.testing.assert_array_equal(host_bits(kc), rk)
    np.testing.assert_array_equal(host_bits(vc), rv)


@pytest.mark.parametrize("name", list(inputs.WORKLOADS))
def test_compress_bit_exact(name):
    need_gpu()
    wl = inputs.WORKLOADS[name]
    say(f"[compress] {name}")
    _check_compress(wl.problem, inputs.make_inputs(wl, 0), name)


@pytest.mark.parametrize("case", ["ties", "signed_zero_nan_inf", "all_equal", "increasing",
                                  "lp_eq_lb", "lp_one", "ragged"])
def test_compress_edge_cases(case):
    need_gpu()
    rng = np.random.default_rng(zlib.crc32(case.encode()))
    lb, lp, d, n_kv, la = 3000, 700, 128, 3, 40
    s = rng.standard_normal((n_kv, lb)).astype(np.float32)
    if case == "ties":
        s = np.round(s * 2).astype(np.float32)
    elif case == "signed_zero_nan_inf":
        pool = np.array([0.0, -0.0, np.nan, np.inf, -np.inf, 1.0, -1.0], np.float32)
        s = rng.choice(pool, (n_kv, lb)).astype(np.float32)
    elif case == "all_equal":
        s[:] = 0.5
    elif case == "increasing":
        s = np.tile(np.arange(lb, dtype=np.float32), (n_kv, 1))
    elif case == "lp_eq_lb":
        lp = lb
    elif case == "lp_one":
        lp = 1
    elif case == "ragged":
        lb, lp, d, la = 1037, 333, 64, 7
        s = np.round(rng.standard_normal((n_kv, lb)) * 3).astype(np.float32)
    p = inputs.Problem(4, 1, la, lb, lp, n_kv, n_kv, d)
    inp = dict(scores=s, k=rng.integers(0, 65536, (n_kv, la + lb, d), dtype=np.uint16),
               v=rng.integers(0, 65536, (n_kv, la + lb, d), dtype=np.uint16),
               q=np.zeros((1, 1, 8), np.uint16), k_pass=np.zeros((1, 8), np.uint16),
               v_pass=np.zeros((1, 8), np.uint16))
    _check_compress(p, inp, case)


@pytest.mark.parametrize("case", ["normal_131072", "zipf_131072", "ties_nan_inf_ragged",
                                  "lp_near_lb", "lp_one"])
def test_compress_long_local_blocks(case):
    """Local blocks past 65536 rows (the paper's 1024K prefill setting over 8
    hosts has l_b = 131072): the multi-pass selection kernel, bit-exact."""
    need_gpu()
    rng = np.random.default_rng(zlib.crc32(case.encode()))
    n_kv, la, d = 2, 16, 128
    lb, lp = 131072, 2048
    if case == "normal_131072":
        s = rng.standard_normal((n_kv, lb)).astype(np.float32)
    elif case == "zipf_131072":
        s = rng.zipf(1.5, (n_kv, lb)).astype(np.float32)
    else:
        lb, d = 65536 + 1234, 64
        pool = np.array([0.0, -0.0, np.nan, np.inf, -np.inf, 1.0, -1.0, 2.5], np.float32)
        s = np.round(rng.standard_normal((n_kv, lb)) * 2).astype(np.float32)
        mask = rng.random((n_kv, lb)) < 0.2
        s[mask] = rng.choice(pool, int(mask.sum()))
        lp = {"ties_nan_inf_ragged": 20011, "lp_near_lb": lb - 3, "lp_one": 1}[case]
    p = inputs.Problem(4, 1, la, lb, lp, n_kv, n_kv, d)
    say(f"[compress long] {case}: Lb {lb} l_p {lp} d {d}")
    inp = dict(scores=s, k=rng.integers(0, 65536, (n_kv, la + lb, d), dtype=np.uint16),
               v=rng.integers(0, 65536, (n_kv, la + lb, d), dtype=np.uint16),
               q=np.zeros((1, 1, 8), np.uint16), k_pass=np.zeros((1, 8), np.uint16),
               v_pass=np.zeros((1, 8), np.uint16))
    _check_compress(p, inp, case)


def test_compress_without_indices():
    """out_idx = NULL: the gathered rows are the same bits."""
    torch = need_gpu()
    from paper_2502_12085_amd import apb
    wl = inputs.WORKLOADS["llama8b_32k"]
    p = wl.problem
    inp = inputs.make_inputs(wl, 9)
    dv = upload(inp)
    _, kc, vc = run_compress(p, dv["scores"], dv["k"], dv["v"])
    k2 = torch.zeros_like(kc)
    v2 = torch.zeros_like(vc)
    apb.compress_select(p, dv["scores"], dv["k"], dv["v"], None, k2, v2)
    torch.cuda.synchronize()
    assert torch.equal(k2.view(torch.int16), kc.view(torch.int16))
    assert torch.equal(v2.view(torch.int16), vc.view(torch.int16))


@pytest.mark.parametrize("case", ["misaligned_scores", "big_tie_groups"])
def test_compress_layouts(case):
    """Scores whose base is 4- but not 16-byte aligned (the vector loads step
    aside), and a long local block of integer scores with selections of
    thousands of rows per head (shares near the 1024-row limit)."""
    torch = need_gpu()
    from paper_2502_12085_amd import apb
    rng = np.random.default_rng(7)
    if case == "misaligned_scores":
        lb, lp, d, n_kv, la = 5000, 1500, 128, 2, 16
        s = rng.standard_normal((n_kv, lb)).astype(np.float32)
    else:
        lb, lp, d, n_kv, la = 30000, 29000, 64, 2, 0
        s = rng.zipf(1.5, (n_kv, lb)).astype(np.float32)
    p = inputs.Problem(4, 1, la, lb, lp, n_kv, n_kv, d)
    k = rng.integers(0, 65536, (n_kv, la + lb, d), dtype=np.uint16)
    v = rng.integers(0, 65536, (n_kv, la + lb, d), dtype=np.uint16)
    flat = torch.zeros(n_kv * lb + 1, dtype=torch.float32, device="cuda")
    ds = flat[1:].view(n_kv, lb)  # 4-byte aligned, never 16
    ds.copy_(torch.from_numpy(s))
    if case != "misaligned_scores":
        ds = torch.from_numpy(s).cuda()
    idx = torch.full((n_kv, lp), -1, dtype=torch.int32, device="cuda")
    ok = torch.zeros((n_kv, lp, d), dtype=torch.bfloat16, device="cuda")
    ov = torch.zeros_like(ok)
    apb.compress_select(p, ds, dev_bf16(k), dev_bf16(v), idx, ok, ov)
    torch.cuda.synchronize()
    ridx, rk, rv = oracle.compress_ref(s, k, v, lp, la)
    np.testing.assert_array_equal(idx.cpu().numpy(), ridx)
    np.testing.assert_array_equal(host_bits(ok), rk)
    np.testing.assert_array_equal(host_bits(ov), rv)
    say(f"  {case}: bit-exact")


def test_simulated_hosts_end_to_end():
    """Alg. 2 on one GPU: every earlier host's compressor writes its slot of
    a rank-major passing buffer, then the last host's attention reads it."""
    torch = need_gpu()
    for name in ("tiny", "llama8b_32k"):
        wl = inputs.WORKLOADS[name] if name == "tiny" else _wl(name, n_q_heads=8, n_kv_heads=2)
        p = wl.problem
        say(f"[host simulation] {name}")
        inp = inputs.make_inputs(wl, 0)
        hosts = inputs.make_host_blocks(wl, 0)
        dv = upload(inp)
        H = p.n_hosts
        kbuf = torch.zeros((H, p.n_kv_heads, p.pass_len, p.head_dim), dtype=torch.bfloat16,
                           device="cuda")
        vbuf = torch.zeros_like(kbuf)
        for j, hb in enumerate(hosts):
            run_compress(p, torch.from_numpy(hb["scores"]).cuda(), dev_bf16(hb["k"]),
                         dev_bf16(hb["v"]), kbuf[j], vbuf[j])
        run_compress(p, dv["scores"], dv["k"], dv["v"], kbuf[p.host_idx], vbuf[p.host_idx])
        dv["k_pass"], dv["v_pass"] = kbuf, vbuf
        o, lse = run_attention(p, dv)
        heads = np.arange(min(p.n_q_heads, 4))
        ro, rl, ridx, rkc, rvc, rkp, rvp = oracle.simulate_hosts_ref(
            inp["q"], inp["k"], inp["v"], inp["scores"], hosts, anchor_len=p.anchor_len,
            l_p=p.pass_len, heads=heads)
        np.testing.assert_array_equal(host_bits(kbuf[:p.host_idx]), rkp)
        np.testing.assert_array_equal(host_bits(vbuf[p.host_idx]), rvc)
        assert_attention_close(host_bf16_to_f64(o)[heads], lse.cpu().numpy()[heads], ro, rl, name)


def test_compressor_and_attention_concurrent_on_two_streams():
    """One host's compressor writes slot host_idx of the rank-major passing
    buffer while its attention reads slots [0, host_idx) of the same buffer
    (bench.py --overlap): run on two streams at once, in both launch orders,
    every output matches the serial run bit for bit (both kernels are
    deterministic, and neither touches what the other writes)."""
    torch = need_gpu()
    from paper_2502_12085_amd import apb
    wl = _wl("llama8b_32k", n_q_heads=16, n_kv_heads=4)
    p = wl.problem
    say(f"[two streams] {p}")
    inp = inputs.make_inputs(wl, 5)
    dv = upload(inp)
    H, n_kv, lp, d = p.n_hosts, p.n_kv_heads, p.pass_len, p.head_dim
    kbuf = torch.zeros((H, n_kv, lp, d), dtype=torch.bfloat16, device="cuda")
    vbuf = torch.zeros_like(kbuf)
    kbuf[:p.host_idx] = dv["k_pass"]
    vbuf[:p.host_idx] = dv["v_pass"]

    def run(order, s_att, s_cmp):
        kbuf[p.host_idx].zero_()
        vbuf[p.host_idx].zero_()
        idx = torch.full((n_kv, lp), -1, dtype=torch.int32, device="cuda")
        o = torch.full((p.n_q_heads, p.rows, d), float("nan"), dtype=torch.bfloat16, device="cuda")
        lse = torch.full((p.n_q_heads, p.rows), float("nan"), dtype=torch.float32, device="cuda")
        torch.cuda.synchronize()
        calls = {
            "att": lambda: apb.attention_fwd(p, dv["q"], dv["k"], dv["v"], kbuf, vbuf, o, lse,
                                             0.0, s_att),
            "cmp": lambda: apb.compress_select(p, dv["scores"], dv["k"], dv["v"], idx,
                                               kbuf[p.host_idx], vbuf[p.host_idx], s_cmp),
        }
        for name in order:
            calls[name]()
        torch.cuda.synchronize()
        return (host_bits(o), lse.cpu().numpy(), idx.cpu().numpy(), host_bits(kbuf[p.host_idx]),
                host_bits(vbuf[p.host_idx]))

    main = torch.cuda.current_stream()
    ref = run(("cmp", "att"), main, main)  # serial, one stream
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()  # default priority
    for order in (("att", "cmp"), ("cmp", "att")):
        got = run(order, s1, s2)
        for a, b in zip(got, ref):
            assert np.array_equal(a, b), order
    assert np.all(ref[2] >= 0)
