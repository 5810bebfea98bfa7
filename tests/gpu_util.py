"""Helpers shared by the GPU tests: device upload of the seeded inputs,
calls through the C ABI, and the parity bar."""
import sys

import numpy as np
import pytest

# Parity bar for attention (bf16 in, fp32 accumulate): output max-abs 2e-2,
# mean-abs 2e-3; LSE (natural log) max-abs 1e-3.
O_MAX_ABS = 2e-2
O_MEAN_ABS = 2e-3
LSE_MAX_ABS = 1e-3


def say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def need_gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch


def dev_bf16(a):
    import torch
    t = torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16)
    return t.cuda()


def host_bf16_to_f64(t):
    import torch
    bits = t.detach().view(torch.int16).cpu().numpy().view(np.uint16)
    return (bits.astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)


def host_bits(t):
    import torch
    return t.detach().view(torch.int16).cpu().numpy().view(np.uint16)


def upload(inp):
    import torch
    d = {k: dev_bf16(inp[k]) for k in ("q", "k", "v", "k_pass", "v_pass")}
    d["scores"] = torch.from_numpy(np.ascontiguousarray(inp["scores"])).cuda()
    return d


def run_attention(prob, dv, softmax_scale=0.0, fill=float("nan")):
    import torch
    from paper_2502_12085_amd import apb
    o = torch.full((prob.n_q_heads, prob.rows, prob.head_dim), fill, dtype=torch.bfloat16,
                   device="cuda")
    lse = torch.full((prob.n_q_heads, prob.rows), fill, dtype=torch.float32, device="cuda")
    kp = dv["k_pass"] if prob.passing_rows > 0 else None
    vp = dv["v_pass"] if prob.passing_rows > 0 else None
    apb.attention_fwd(prob, dv["q"], dv["k"], dv["v"], kp, vp, o, lse, softmax_scale)
    torch.cuda.synchronize()
    return o, lse


def run_compress(prob, scores, k, v, out_k=None, out_v=None):
    import torch
    from paper_2502_12085_amd import apb
    n_kv, lp, d = prob.n_kv_heads, prob.pass_len, prob.head_dim
    idx = torch.full((n_kv, lp), -1, dtype=torch.int32, device="cuda")
    if out_k is None:
        out_k = torch.zeros((n_kv, lp, d), dtype=torch.bfloat16, device="cuda")
        out_v = torch.zeros((n_kv, lp, d), dtype=torch.bfloat16, device="cuda")
    apb.compress_select(prob, scores, k, v, idx, out_k, out_v)
    torch.cuda.synchronize()
    return idx, out_k, out_v


# Peaked softmax (a test's softmax_scale of 1.0): an output row is then close
# to a single value row, |O| reaches max|V| (about 5 for N(0, 1) values), and
# the arithmetic's own rounding grows with it: O rounded to bf16 (up to 2^-9
# |O|) plus the probabilities rounded to bf16 for the value product (up to
# 2^-9 of the weighted |V|, about |O| when one key dominates).  The bar for
# such cases adds that bound, 2^-8 |O_ref|, to the absolute 2e-2 per element.
O_REL_PEAKED = 2.0 ** -8


def assert_attention_close(o_gpu, lse_gpu, o_ref, lse_ref, what="", o_rel=0.0):
    o_gpu = np.asarray(o_gpu, dtype=np.float64)
    assert np.isfinite(o_gpu).all(), f"{what}: non-finite output"
    err = np.abs(o_gpu - o_ref)
    lerr = np.abs(np.asarray(lse_gpu, dtype=np.float64) - lse_ref)
    say(f"  {what}: O max {err.max():.3e} mean {err.mean():.3e}  LSE max {lerr.max():.3e}")
    if o_rel:
        excess = err - (O_MAX_ABS + o_rel * np.abs(o_ref))
        say(f"  {what}: largest O error over 2e-2 + {o_rel:.3g}|O_ref|: {excess.max():.3e}")
        assert excess.max() <= 0, f"{what}: O error {err.max()} past 2e-2 + {o_rel}|O_ref|"
    else:
        assert err.max() <= O_MAX_ABS, f"{what}: O max-abs {err.max()}"
    assert err.mean() <= O_MEAN_ABS, f"{what}: O mean-abs {err.mean()}"
    assert lerr.max() <= LSE_MAX_ABS, f"{what}: LSE max-abs {lerr.max()}"
