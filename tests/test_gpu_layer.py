"""GPU parity of one host's whole layer (``apb_layer_fwd``: Alg. 2 with the
model's layer around attention) through the C ABI against the fp64 layer
oracle.

Bar, derived from where the kernel rounds: x, Q/K/V, the attention output,
H1, y, the SwiGLU product and the output are stored in bf16, each with a
relative rounding error of at most 2^-8 (8 significant bits).  The output is
H1 + FFN(y): its own rounding and that of H1 carry through the residual
unchanged (<= 2^-8 |out| + 2^-8 |H1|), while the roundings inside the
products enter as sums of many independent terms and stay far smaller.
Hence per element |gpu - ref| <= 0.02 + 0.01 |ref| and mean-abs <= 4e-3 on
the output, the same on the KV cache (one rounding after the projection and
one after RoPE).  The selection is made from scores computed on the GPU's
bf16 Q/K/V, so it must be a valid top-l_p of the oracle's scores up to 0.05
(near-ties may go either way) and is otherwise checked bit for bit: the
written slot holds exactly the GPU KV cache rows it names, in ascending
order, and the earlier hosts' slots are untouched.
"""
import dataclasses

import numpy as np
import pytest

import oracle
from paper_2502_12085_amd import inputs
from gpu_util import dev_bf16, host_bf16_to_f64, host_bits, need_gpu, say

pytestmark = pytest.mark.gpu
ATOL, RTOL, MEAN_ABS = 0.02, 0.01, 4e-3
SCORE_TOL = 0.05


def _run_layer(lw, seed=0):
    torch = need_gpu()
    from paper_2502_12085_amd import apb
    p = lw.problem
    inp = inputs.make_layer_inputs(lw, seed)
    T, d, nkv = p.rows, p.head_dim, p.n_kv_heads
    w = {}
    for name, key in (("ln1", "ln1"), ("w_qkv", "w_qkv"), ("w_o", "w_o"), ("ln2", "ln2"),
                      ("w_gate", "w_gate"), ("w_up", "w_up"), ("w_down", "w_down"),
                      ("r_w1", "w1")):
        w[name] = dev_bf16(inp["w"][key])
    for name, key in (("r_b1", "b1"), ("r_w2", "w2"), ("r_b2", "b2")):
        w[name] = torch.from_numpy(np.ascontiguousarray(inp["w"][key])).cuda()
    hidden = dev_bf16(inp["hidden"])
    pos = torch.from_numpy(inp["pos"]).cuda()
    # rank-major passing buffers; the slots from host_idx on start as a NaN guard
    pk = torch.full((p.n_hosts, nkv, p.pass_len, d), float("nan"), dtype=torch.bfloat16,
                    device="cuda")
    pv = torch.full_like(pk, float("nan"))
    if p.host_idx > 0 and p.pass_len > 0:
        pk[:p.host_idx] = dev_bf16(inp["k_pass"])
        pv[:p.host_idx] = dev_bf16(inp["v_pass"])
    kc = torch.full((nkv, T, d), float("nan"), dtype=torch.bfloat16, device="cuda")
    vc = torch.full_like(kc, float("nan"))
    out = torch.full((T, lw.hidden), float("nan"), dtype=torch.bfloat16, device="cuda")
    ws = torch.empty(apb.layer_workspace_size(lw), dtype=torch.uint8, device="cuda")
    apb.layer_fwd(lw, w, hidden, pos, kc, vc, pk, pv, out, ws)
    torch.cuda.synchronize()
    return inp, dict(out=out, k=kc, v=vc, pk=pk, pv=pv)


def _oracle(lw, inp, rows=None):
    p = lw.problem
    return oracle.layer_ref(inp["hidden"], inp["pos"], inp["w"], inp["k_pass"], inp["v_pass"],
                            anchor_len=p.anchor_len, pass_len=p.pass_len, n_q=p.n_q_heads,
                            n_kv=p.n_kv_heads, head_dim=p.head_dim, eps=lw.eps, theta=lw.theta,
                            rows=rows)


def _close(got, ref, what):
    got = np.asarray(got, np.float64)
    assert np.isfinite(got).all(), f"{what}: non-finite values"
    err = np.abs(got - ref)
    bound = ATOL + RTOL * np.abs(ref)
    say(f"  {what}: max {err.max():.3e} mean {err.mean():.3e} worst err/bound "
        f"{(err / bound).max():.3f}")
    assert (err <= bound).all(), f"{what}: max err {err.max()}"
    assert err.mean() <= MEAN_ABS, f"{what}: mean err {err.mean()}"


def _check_selection(lw, inp, got, ref):
    """The written slot names a valid top-l_p of the oracle's scores (up to
    SCORE_TOL), in ascending order, copied bit for bit from the GPU cache;
    earlier slots are untouched."""
    p = lw.problem
    h, lp, La = p.host_idx, p.pass_len, p.anchor_len
    if lp == 0:
        return
    kc, vc = host_bits(got["k"]), host_bits(got["v"])
    slot_k, slot_v = host_bits(got["pk"][h]), host_bits(got["pv"][h])
    if h > 0:
        assert np.array_equal(host_bits(got["pk"][:h]), inp["k_pass"])
        assert np.array_equal(host_bits(got["pv"][:h]), inp["v_pass"])
    for kv in range(p.n_kv_heads):
        where = {kc[kv, La + i].tobytes(): i for i in range(p.local_len)}
        idx = np.array([where[slot_k[kv, t].tobytes()] for t in range(lp)])
        assert (np.diff(idx) > 0).all(), "selected rows must be ascending"
        assert np.array_equal(slot_v[kv], vc[kv, La + idx])
        s = ref["scores"][kv]
        thr = np.sort(s)[::-1][lp - 1]
        chosen = np.zeros(p.local_len, bool)
        chosen[idx] = True
        assert (s[chosen] >= thr - SCORE_TOL).all()
        if (~chosen).any():
            assert (s[~chosen] <= thr + SCORE_TOL).all()
        say(f"  selection kv {kv}: {np.sum(~np.isin(idx, ref['idx'][kv]))} of {lp} differ "
            "from the oracle's (within the score tolerance)")


def _tiny_variant(name, **kw):
    base = inputs.LAYER_WORKLOADS["tiny_layer"]
    prob = dataclasses.replace(base.problem, **{k: v for k, v in kw.items()
                                                if k in inputs.Problem.__dataclass_fields__})
    rest = {k: v for k, v in kw.items() if k not in inputs.Problem.__dataclass_fields__}
    return dataclasses.replace(base, name=name, attn=inputs.Workload(name, prob), **rest)


@pytest.mark.parametrize("lw", [
    inputs.LAYER_WORKLOADS["tiny_layer"],
    _tiny_variant("first_host", host_idx=0),
    _tiny_variant("no_passing", pass_len=0),
    _tiny_variant("ragged", n_hosts=5, host_idx=3, anchor_len=77, local_len=300, pass_len=20,
                  n_q_heads=6, n_kv_heads=2, hidden=384, intermediate=320),
    _tiny_variant("d128_gqa4", n_q_heads=8, n_kv_heads=2, head_dim=128, hidden=1024,
                  intermediate=704, anchor_len=0, host_idx=1),
    # an FFN long enough (K = 8320 in the down product) for the GEMM's
    # long-K schedule, 65 feature tiles (a partial block of 4) and ragged tokens
    _tiny_variant("long_ffn", anchor_len=77, local_len=300, intermediate=8320),
], ids=lambda lw: lw.name)
def test_layer_matches_oracle_every_row(lw):
    say(f"[layer] {lw.name}: {lw.problem}, D={lw.hidden}, I={lw.intermediate}")
    inp, got = _run_layer(lw)
    ref = _oracle(lw, inp)
    _close(host_bf16_to_f64(got["out"]), ref["out"], "hidden_out")
    _close(host_bf16_to_f64(got["k"]), ref["k"], "K cache (post-RoPE)")
    _close(host_bf16_to_f64(got["v"]), ref["v"], "V cache")
    _check_selection(lw, inp, got, ref)


def test_layer_deterministic():
    lw = inputs.LAYER_WORKLOADS["tiny_layer"]
    _, a = _run_layer(lw, seed=5)
    _, b = _run_layer(lw, seed=5)
    for key in ("out", "k", "v", "pk", "pv"):
        assert np.array_equal(host_bits(a[key]), host_bits(b[key])), key


def test_llama8b_128k_layer_sampled_rows():
    """The bench's layer (Llama-3.1-8B shapes, 128K context over 8 hosts, the
    last host) on sampled rows: segment edges, tile edges and random rows;
    the KV cache on every row."""
    lw = inputs.LAYER_WORKLOADS["llama8b_128k_layer"]
    p = lw.problem
    say(f"[layer] {lw.name}: generating inputs and running")
    inp, got = _run_layer(lw)
    rng = np.random.default_rng(11)
    rows = np.unique(np.concatenate([
        [0, 1, 255, 256, p.anchor_len - 1, p.anchor_len, p.anchor_len + 1, p.rows - 257,
         p.rows - 256, p.rows - 1], rng.integers(0, p.rows, 14)]))
    say(f"  oracle on {len(rows)} rows")
    ref = _oracle(lw, inp, rows=rows)
    _close(host_bf16_to_f64(got["out"])[rows], ref["out"], "hidden_out (sampled rows)")
    _close(host_bf16_to_f64(got["k"]), ref["k"], "K cache (post-RoPE)")
    _close(host_bf16_to_f64(got["v"]), ref["v"], "V cache")
    _check_selection(lw, inp, got, ref)
