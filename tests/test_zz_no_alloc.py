"""The no-allocation decode entry point against the workspace one.

``apb_decode_attention_noalloc`` keeps the split partials in the library's
own per-GPU scratch.  Calls in a row share that array (the later ones with
smaller problems, so stale partials of an earlier call sit past what a later
call reads), and each result must match ``apb_decode_attention`` on the same
inputs: bit for bit when the split plan fits the scratch (same kernels, same
splits), within the attention bar (output max-abs 2e-2, mean-abs 2e-3; LSE
max-abs 1e-3) when the scratch caps the plan to fewer, longer splits.  The
capped case is also checked against the fp64 oracle.
"""
import numpy as np
import pytest

import oracle
from paper_2502_12085_amd import inputs
from gpu_util import assert_attention_close, dev_bf16, need_gpu, say

pytestmark = pytest.mark.gpu

# n_q, n_kv, d, Lc, n_new, append, capped: the first problem's default plan
# needs 8 splits of 8192 rows (eight-wave path, fp16 partials: 17.3 MB > the
# 16 MiB scratch) and runs with 7; the second is the 128K Llama-8B-shaped
# question step (14.1 MB, fits); the third a small one-wave problem.
CALLS = [
    (64, 8, 128, 16384, 128, 1, True),
    (32, 8, 128, 16384, 64, 1, False),
    (8, 2, 64, 1000, 3, 1, False),
]


def _plan_bytes(n_q, n_kv, d, lc, n_new, app):
    from paper_2502_12085_amd import apb
    return apb.decode_workspace_size(apb.DecodeProblem(n_q, n_kv, d, lc, n_new, app))


def _run_both(case, shape):
    torch = need_gpu()
    from paper_2502_12085_amd import apb
    n_q, n_kv, d, lc, n_new, app, _ = shape
    p = apb.DecodeProblem(n_q, n_kv, d, lc, n_new, app)
    kc, vc = case["caches"][0]
    q, dkc, dvc = dev_bf16(case["q"]), dev_bf16(kc), dev_bf16(vc)
    kn = dev_bf16(case["k_new"]) if app else None
    vn = dev_bf16(case["v_new"]) if app else None
    ws = torch.empty(apb.decode_workspace_size(p), dtype=torch.uint8, device="cuda")
    out = []
    for noalloc in (False, True):
        o = torch.full((n_q, n_new, d), float("nan"), dtype=torch.float32, device="cuda")
        lse = torch.full((n_q, n_new), float("nan"), dtype=torch.float32, device="cuda")
        if noalloc:
            apb.decode_attention_noalloc(p, q, dkc, dvc, kn, vn, o, lse)
        else:
            apb.decode_attention(p, q, dkc, dvc, kn, vn, o, lse, ws)
        torch.cuda.synchronize()
        out.append((o.cpu().numpy().astype(np.float64), lse.cpu().numpy().astype(np.float64)))
    return out


def test_noalloc_matches_workspace_entry_point_over_calls_in_a_row():
    from paper_2502_12085_amd import apb
    need_gpu()
    sizes = []
    for i, shape in enumerate(CALLS):
        n_q, n_kv, d, lc, n_new, app, capped = shape
        need = _plan_bytes(n_q, n_kv, d, lc, n_new, app)
        assert (need > apb.NOALLOC_SCRATCH_BYTES) == capped, (shape, need)
        sizes.append(n_q * n_new * d)
        say(f"[decode noalloc] call {i}: {shape[:6]} default-plan partials {need} B")
        case = inputs.make_decode_case(n_q, n_kv, d, [lc], n_new, seed=40 + i)
        (o_ws, l_ws), (o_na, l_na) = _run_both(case, shape)
        assert np.isfinite(o_na).all() and np.isfinite(l_na).all()
        if capped:
            assert_attention_close(o_na, l_na, o_ws, l_ws, f"noalloc vs workspace {shape[:6]}")
            kc, vc = case["caches"][0]
            o_ref, lse_ref = oracle.decode_attention_ref(case["q"], kc, vc, case["k_new"],
                                                         case["v_new"])
            assert_attention_close(o_na, l_na, o_ref, lse_ref, f"noalloc vs oracle {shape[:6]}")
        else:
            assert np.array_equal(o_na, o_ws) and np.array_equal(l_na, l_ws), shape
            say(f"  bit-identical to apb_decode_attention")
    assert sizes == sorted(sizes, reverse=True)  # each call smaller than the one before
