"""The C-ABI library loads and exports every symbol ``include/apb.h``
declares, and every validation error is raised on the host before any HIP
call (fake device addresses are never dereferenced)."""
import ctypes
import os
import re

import pytest

import oracle
from paper_2502_12085_amd import apb, inputs

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared_functions():
    text = open(os.path.join(ROOT, "include", "apb.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(apb_\w+)\s*\(", text)))


def test_library_exports_every_declared_symbol():
    L = apb.lib()
    declared = _declared_functions()
    assert set(declared) == set(apb.EXPORTED)
    for name in declared:
        assert hasattr(L, name), name
    assert apb.abi_version() == 5


def _prob(**kw):
    base = dict(n_hosts=4, host_idx=2, anchor_len=128, local_len=512, pass_len=32,
                n_q_heads=4, n_kv_heads=1, head_dim=64)
    base.update(kw)
    return apb.Problem(**base)


@pytest.mark.parametrize("kw,code", [
    (dict(), 0),
    (dict(n_hosts=0, host_idx=0), 2),
    (dict(host_idx=4), 2),
    (dict(host_idx=-1), 2),
    (dict(anchor_len=-1), 2),
    (dict(local_len=0), 2),
    (dict(pass_len=513), 2),
    (dict(pass_len=-1), 2),
    (dict(n_q_heads=6, n_kv_heads=4), 2),
    (dict(n_kv_heads=0), 2),
    (dict(head_dim=96), 3),
    (dict(head_dim=256), 3),
    (dict(anchor_len=0, host_idx=0), 0),
    (dict(pass_len=0), 0),
    (dict(anchor_len=1 << 29, local_len=1 << 29, pass_len=1, host_idx=3), 2),
])
def test_validate_problem(kw, code):
    assert apb.lib().apb_validate_problem(ctypes.byref(_prob(**kw))) == code


@pytest.mark.parametrize("rows,n_q,code", [
    # the attention grid is one workgroup per 256-row query tile per query
    # head and must stay below 2^31 entries
    ((1 << 30) - 256, 512, 0),  # (2^22 - 1) tiles x 512 heads = 2^31 - 512
    (1 << 30, 512, 2),          # 2^22 tiles x 512 heads = 2^31
    ((1 << 30) - 255, 512, 2),  # one row more rounds up to 2^22 tiles
    ((1 << 30) - 256, 513, 2),
])
def test_validate_problem_grid_boundary(rows, n_q, code):
    p = _prob(n_hosts=1, host_idx=0, anchor_len=0, local_len=rows, pass_len=0,
              n_q_heads=n_q, n_kv_heads=1, head_dim=128)
    assert apb.lib().apb_validate_problem(ctypes.byref(p)) == code


def test_flops_match_oracle_closed_form():
    for wl in inputs.WORKLOADS.values():
        p = wl.problem
        ref = oracle.attention_flops(p.n_q_heads, p.head_dim, p.anchor_len, p.local_len,
                                     p.passing_rows)
        assert apb.attention_flops(p) == pytest.approx(ref, rel=1e-12)
    assert apb.lib().apb_attention_flops(ctypes.byref(_prob(head_dim=96))) == -1.0
    # the 128K Llama-8B-shaped host share: 7.284e12 unmasked FLOPs
    assert apb.attention_flops(inputs.WORKLOADS["llama8b_128k"].problem) == pytest.approx(7.284e12, rel=1e-3)


def test_status_strings():
    L = apb.lib()
    for s in range(8):
        assert L.apb_status_string(s)
    assert L.apb_status_string(99) == b"unknown status"


# Fake, well-separated device addresses: validation must reject every call
# below before touching them.
A = 0x7F0000000000
Q, K, V, KP, VP, O, LSE, SC, IDX, OK_, OV = (A + i * (1 << 36) for i in range(11))


def _attn(p, q=Q, k=K, v=V, kp=KP, vp=VP, o=O, lse=LSE):
    return apb.lib().apb_attention_fwd(ctypes.byref(p), q, k, v, kp, vp, o, lse, 0.0, None)


def _comp(p, sc=SC, k=K, v=V, idx=IDX, ok=OK_, ov=OV):
    return apb.lib().apb_compress_select(ctypes.byref(p), sc, k, v, idx, ok, ov, None)


def test_attention_error_paths():
    p = _prob()
    assert apb.lib().apb_attention_fwd(None, Q, K, V, KP, VP, O, LSE, 0.0, None) == 1
    assert _attn(p, q=None) == 1
    assert _attn(p, o=None) == 1
    assert _attn(p, kp=None) == 1           # passing block required when Lp > 0
    assert _attn(p, q=Q + 8) == 4           # bf16 needs 16-byte alignment
    assert _attn(p, kp=KP + 2) == 4
    assert _attn(p, lse=LSE + 2) == 4
    assert _attn(p, o=Q) == 6               # output aliases an input
    assert _attn(p, o=K + 64) == 6
    assert _attn(p, lse=V + 16) == 6
    assert _attn(p, lse=O + 16) == 6        # outputs overlap each other
    assert _attn(_prob(head_dim=96)) == 3
    assert _attn(_prob(pass_len=600)) == 2


def test_compress_error_paths():
    p = _prob()
    assert apb.lib().apb_compress_select(None, SC, K, V, IDX, OK_, OV, None) == 1
    assert _comp(p, sc=None) == 1
    assert _comp(p, ok=None) == 1
    assert _comp(p, sc=SC + 2) == 4
    assert _comp(p, ok=OK_ + 8) == 4
    assert _comp(p, idx=IDX + 1) == 4
    assert _comp(p, ok=K) == 6
    assert _comp(p, idx=SC) == 6
    assert _comp(p, ov=OK_ + 32) == 6
    assert _comp(_prob(n_q_heads=3, n_kv_heads=2)) == 2
    # l_p = 0 is valid and launches nothing
    assert _comp(_prob(pass_len=0)) == 0


def test_binding_raises_without_the_library(monkeypatch, tmp_path):
    # no fallback: with libapb.so absent every call raises instead of
    # computing anything elsewhere
    monkeypatch.setattr(apb, "LIB_PATH", str(tmp_path / "libapb.so"))
    monkeypatch.setattr(apb, "_lib", None)
    with pytest.raises(RuntimeError, match="is missing"):
        apb.lib()
    with pytest.raises(RuntimeError, match="is missing"):
        apb.attention_flops(inputs.WORKLOADS["tiny"].problem)
    with pytest.raises(RuntimeError, match="is missing"):
        apb.validate_problem(inputs.WORKLOADS["tiny"].problem)


def test_binding_rejects_host_tensors():
    import torch
    x = torch.zeros(4, dtype=torch.bfloat16)
    with pytest.raises(ValueError):
        apb.attention_fwd(inputs.WORKLOADS["tiny"].problem, x, x, x, x, x, x)


# ------------------------------------------------------- decoding stage
def _dprob(**kw):
    base = dict(n_q_heads=8, n_kv_heads=2, head_dim=128, cache_len=1000, n_new=3, append_new=1)
    base.update(kw)
    return apb.DecodeProblem(**base)


@pytest.mark.parametrize("kw,code", [
    (dict(), 0),
    (dict(append_new=0), 0),
    (dict(cache_len=0), 0),
    (dict(cache_len=-1), 2),
    (dict(n_new=0), 2),
    (dict(append_new=2), 2),
    (dict(n_q_heads=6, n_kv_heads=4), 2),
    (dict(n_kv_heads=0), 2),
    (dict(head_dim=80), 3),
    (dict(cache_len=1 << 30), 2),
])
def test_validate_decode(kw, code):
    assert apb.validate_decode(_dprob(**kw)) == code


def test_decode_workspace_size_is_shape_only():
    # one fp32 partial (O and LSE) per split and row on the one-wave path (few
    # rows per KV head); more keys never need less scratch per row
    rows = 8 * 3
    sizes = []
    for lc in (0, 1, 31, 32, 1000, 16384, 65536):
        n = apb.decode_workspace_size(_dprob(cache_len=lc))
        assert n > 0 and n % (rows * 129 * 4) == 0
        sizes.append(n // (rows * 129 * 4))
    assert sizes == sorted(sizes) and sizes[0] == 1
    # 256 rows per KV head: the eight-wave path, fp16 O + scale + LSE per row
    rows = 32 * 64
    for lc in (0, 100, 16384):
        n = apb.decode_workspace_size(_dprob(n_q_heads=32, n_kv_heads=8, n_new=64, cache_len=lc))
        assert n > 0 and n % (rows * (2 * 128 + 8)) == 0
    with pytest.raises(apb.ApbError):
        apb.decode_workspace_size(_dprob(head_dim=80))
    assert apb.lib().apb_decode_workspace_size(ctypes.byref(_dprob()), None) == 1


DQ, DKC, DVC, DKN, DVN, DO, DL, WS = (A + i * (1 << 36) for i in range(8))


def _dec(p, q=DQ, kc=DKC, vc=DVC, kn=DKN, vn=DVN, o=DO, lse=DL, ws=WS, ws_bytes=1 << 30):
    return apb.lib().apb_decode_attention(ctypes.byref(p), q, kc, vc, kn, vn, o, lse, 0.0, ws,
                                          ws_bytes, None)


def test_decode_error_paths():
    p = _dprob()
    assert apb.lib().apb_decode_attention(None, DQ, DKC, DVC, DKN, DVN, DO, DL, 0.0, WS, 1 << 30,
                                          None) == 1
    assert _dec(p, q=None) == 1
    assert _dec(p, lse=None) == 1            # MergeScore needs the LSE
    assert _dec(p, ws=None) == 1
    assert _dec(p, kc=None) == 1             # cache required when Lc > 0
    assert _dec(p, kn=None) == 1             # new K/V required on the last host
    # optional pointers: validation gets past them and stops at the (too
    # small) workspace, so nothing is launched on the fake addresses
    assert _dec(_dprob(append_new=0), kn=None, vn=None, ws_bytes=16) == 2
    assert _dec(_dprob(cache_len=0), kc=None, vc=None, ws_bytes=16) == 2
    assert _dec(p, ws_bytes=16) == 2         # workspace too small
    assert _dec(p, q=DQ + 8) == 4
    assert _dec(p, o=DO + 4) == 4
    assert _dec(p, ws=WS + 4) == 4
    assert _dec(p, o=DQ) == 6
    assert _dec(p, ws=DKC + 64) == 6
    assert _dec(p, lse=DO + 16) == 6
    assert _dec(_dprob(head_dim=80)) == 3


def _dec_na(p, q=DQ, kc=DKC, vc=DVC, kn=DKN, vn=DVN, o=DO, lse=DL):
    return apb.lib().apb_decode_attention_noalloc(ctypes.byref(p), q, kc, vc, kn, vn, o, lse, 0.0,
                                                  None)


def test_decode_noalloc_error_paths():
    # every check runs on the host before any HIP call; the calls below all
    # fail, so nothing is launched on the fake addresses
    p = _dprob()
    assert apb.lib().apb_decode_attention_noalloc(None, DQ, DKC, DVC, DKN, DVN, DO, DL, 0.0,
                                                  None) == 1
    assert _dec_na(p, q=None) == 1
    assert _dec_na(p, lse=None) == 1
    assert _dec_na(p, kc=None) == 1
    assert _dec_na(p, kn=None) == 1
    assert _dec_na(p, q=DQ + 8) == 4
    assert _dec_na(p, o=DO + 4) == 4
    assert _dec_na(p, o=DQ) == 6
    assert _dec_na(p, lse=DO + 16) == 6
    assert _dec_na(_dprob(head_dim=80)) == 3
    assert _dec_na(_dprob(n_new=0)) == 2
    # one split's partials beyond the scratch: 256 or more rows per KV head
    # take the eight-wave path, whose partial per row is fp16 O (2d bytes),
    # its scale and the LSE
    rows_max = apb.NOALLOC_SCRATCH_BYTES // (2 * 128 + 8)
    big = _dprob(n_q_heads=8, n_kv_heads=8, n_new=rows_max // 8 + 1)
    assert _dec_na(big) == 7
    assert apb.lib().apb_status_string(7).startswith(b"the call needs more device scratch")


def test_decode_noalloc_scratch_constant_matches_header():
    text = open(os.path.join(ROOT, "include", "apb.h")).read()
    m = re.search(r"#define APB_DECODE_NOALLOC_SCRATCH_BYTES \((\d+)ull << (\d+)\)", text)
    assert m and int(m.group(1)) << int(m.group(2)) == apb.NOALLOC_SCRATCH_BYTES


def test_merge_error_paths():
    L = apb.lib()
    assert L.apb_merge_partials(0, 4, 128, DO, DL, DQ, WS, None) == 2
    assert L.apb_merge_partials(2, -1, 128, DO, DL, DQ, WS, None) == 2
    assert L.apb_merge_partials(2, 4, 96, DO, DL, DQ, WS, None) == 3
    assert L.apb_merge_partials(2, 0, 128, None, None, None, None, None) == 0  # nothing to do
    assert L.apb_merge_partials(2, 4, 128, None, DL, DQ, WS, None) == 1
    assert L.apb_merge_partials(2, 4, 128, DO, DL, None, WS, None) == 1
    assert L.apb_merge_partials(2, 4, 128, DO + 4, DL, DQ, WS, None) == 4
    assert L.apb_merge_partials(2, 4, 128, DO, DL, DQ + 2, WS, None) == 4
    assert L.apb_merge_partials(2, 4, 128, DO, DL, DO + 64, WS, None) == 6
    assert L.apb_merge_partials(2, 4, 128, DO, DL, DQ, DL + 4, None) == 6


# ---------------------------------------------------- retaining-head scorer
def _sprob(**kw):
    base = dict(anchor_len=128, local_len=512, n_q_heads=4, n_kv_heads=1, head_dim=64, hidden=1024)
    base.update(kw)
    return apb.ScorerProblem(**base)


@pytest.mark.parametrize("kw,code", [
    (dict(), 0),
    (dict(anchor_len=0), 0),
    (dict(local_len=0), 2),
    (dict(anchor_len=-1), 2),
    (dict(n_q_heads=6, n_kv_heads=4), 2),
    (dict(hidden=0), 2),
    (dict(head_dim=96), 3),
    (dict(n_q_heads=36, n_kv_heads=9), 3),   # more KV heads than the fused second layer takes
    (dict(hidden=1000), 3),                  # not a multiple of 256
])
def test_validate_scorer(kw, code):
    assert apb.validate_scorer(_sprob(**kw)) == code


def test_scorer_workspace_size():
    # one fp32 partial per 256 hidden units, KV head and local token
    assert apb.scorer_workspace_size(_sprob()) == 4 * 1 * 512 * 4
    assert apb.scorer_workspace_size(_sprob(n_q_heads=32, n_kv_heads=8, local_len=16384)) == 4 * 8 * 16384 * 4


SQ_, SK_, SV_, SW1, SB1, SW2, SB2, SS, SWS = (A + i * (1 << 36) for i in range(9))


def _score(p, q=SQ_, k=SK_, v=SV_, w1=SW1, b1=SB1, w2=SW2, b2=SB2, s=SS, ws=SWS, ws_bytes=1 << 30):
    return apb.lib().apb_retaining_scores(ctypes.byref(p), q, k, v, w1, b1, w2, b2, s, ws,
                                          ws_bytes, None)


def test_scorer_error_paths():
    p = _sprob()
    assert _score(p, q=None) == 1
    assert _score(p, w1=None) == 1
    assert _score(p, b2=None) == 1
    assert _score(p, ws=None) == 1
    assert _score(p, ws_bytes=100) == 2
    assert _score(p, w1=SW1 + 8) == 4
    assert _score(p, b1=SB1 + 2) == 4
    assert _score(p, ws=SWS + 4) == 4
    assert _score(p, s=SQ_ + 64) == 6
    assert _score(p, s=SW2) == 6
    assert _score(p, ws=SS + 16) == 6
    assert _score(_sprob(hidden=1000)) == 3


def test_probe_library_exports_and_validates():
    """libapb_probe.so exports what include/apb_probe.h declares and rejects
    bad arguments on the host (fake addresses are never dereferenced)."""
    from paper_2502_12085_amd import probe
    text = open(os.path.join(ROOT, "include", "apb_probe.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    declared = sorted(set(re.findall(r"\b(apb_\w+)\s*\(", text)))
    assert set(declared) == set(probe.EXPORTED)
    L = probe.lib()
    for name in declared:
        assert hasattr(L, name), name
    assert probe.mfma_flops(256, 8) == 256 * 8 * 4 * 8 * 2 * 32 * 32 * 16
    fake = 1 << 40
    for args in [(None, fake, 1, 8), (fake, None, 1, 8), (fake, fake, 0, 8), (fake, fake, 1, 0),
                 (fake, fake, 1, 12), (fake + 8, fake, 1, 8), (fake, fake, 1, (1 << 20) + 8)]:
        assert L.apb_probe_mfma_bf16(*args, None) == 1, args


# ------------------------------------------------------------ whole layer
def _lprob(**kw):
    lw = inputs.LAYER_WORKLOADS["tiny_layer"]
    base = dict(hidden=lw.hidden, intermediate=lw.intermediate, scorer_hidden=lw.scorer_hidden,
                rms_eps=lw.eps, rope_theta=lw.theta)
    attn = {k: kw.pop(k) for k in list(kw) if k in dict(apb.Problem._fields_)}
    base.update(kw)
    return apb.LayerProblem(_prob(**attn), **base)


@pytest.mark.parametrize("kw,code", [
    (dict(), 0),
    (dict(hidden=96), 2),
    (dict(hidden=0), 2),
    (dict(intermediate=100), 2),
    (dict(rms_eps=0.0), 2),
    (dict(rms_eps=float("nan")), 2),
    (dict(rope_theta=1.0), 2),
    (dict(rope_theta=float("inf")), 2),
    (dict(scorer_hidden=100), 3),          # the retaining head's hidden block
    (dict(head_dim=96), 3),
    (dict(pass_len=600), 2),
    (dict(n_q_heads=18, n_kv_heads=9), 3),  # more KV heads than the fused scorer takes
])
def test_validate_layer(kw, code):
    assert apb.validate_layer(_lprob(**kw)) == code


def test_layer_flops_and_workspace():
    for lw in inputs.LAYER_WORKLOADS.values():
        p = lw.problem
        attn = oracle.attention_flops(p.n_q_heads, p.head_dim, p.anchor_len, p.local_len,
                                      p.passing_rows)
        sc = oracle.scorer_flops(p.n_q_heads, p.n_kv_heads, p.head_dim, p.local_len,
                                 lw.scorer_hidden)
        ref = oracle.layer_flops(p.rows, lw.hidden, lw.intermediate, p.n_q_heads, p.n_kv_heads,
                                 p.head_dim, attn, sc)
        assert apb.layer_flops(lw) == pytest.approx(ref, rel=1e-12)
        ws = apb.layer_workspace_size(lw)
        # at least x, Q, A, H1 (bf16) and the SwiGLU product
        T, D = p.rows, lw.hidden
        assert ws >= 2 * (2 * T * D + 2 * p.n_q_heads * T * p.head_dim + T * lw.intermediate)
    assert apb.lib().apb_layer_flops(ctypes.byref(_lprob(hidden=96))) == -1.0


LW = {n: A + (11 + i) * (1 << 36) for i, n in enumerate(
    ("ln1", "w_qkv", "w_o", "ln2", "w_gate", "w_up", "w_down", "r_w1", "r_b1", "r_w2", "r_b2"))}
HIN, POS, KC, VC, PK, PV, HOUT, WS = (A + (22 + i) * (1 << 36) for i in range(8))


def _layer(p, ws_bytes=1 << 40, w=None, **kw):
    args = dict(hin=HIN, pos=POS, kc=KC, vc=VC, pk=PK, pv=PV, hout=HOUT, ws=WS)
    args.update(kw)
    ww = apb.LayerWeights(**(w or LW))
    return apb.lib().apb_layer_fwd(ctypes.byref(p), ctypes.byref(ww), args["hin"], args["pos"],
                                   args["kc"], args["vc"], args["pk"], args["pv"], args["hout"],
                                   args["ws"], ws_bytes, None)


def test_layer_error_paths():
    p = _lprob()
    ww = apb.LayerWeights(**LW)
    assert apb.lib().apb_layer_fwd(None, ctypes.byref(ww), HIN, POS, KC, VC, PK, PV, HOUT, WS,
                                   1 << 40, None) == 1
    assert _layer(p, hin=None) == 1
    assert _layer(p, pk=None) == 1                    # l_p > 0 needs the passing buffers
    assert _layer(p, w=dict(LW, w_up=None)) == 1
    assert _layer(p, w=dict(LW, r_b2=None)) == 1
    assert _layer(p, hout=HOUT + 8) == 4
    assert _layer(p, w=dict(LW, w_down=LW["w_down"] + 2)) == 4
    assert _layer(p, pos=POS + 2) == 4
    assert _layer(p, ws_bytes=16) == 2                # workspace too small
    assert _layer(p, hout=HIN) == 6                   # output over an input
    assert _layer(p, kc=LW["w_qkv"] + 256) == 6
    assert _layer(p, vc=KC + 64) == 6                 # outputs over each other
    assert _layer(p, ws=HOUT + 16) == 6
    # this host's slot (host_idx = 2) is written; the earlier slots are read
    slot = 1 * 32 * 64 * 2
    assert _layer(p, kc=PK + slot) == 6               # the KV cache over a read slot
    assert _layer(p, hout=PK + 2 * slot) == 6         # an output over the written slot
    assert _layer(_lprob(head_dim=96)) == 3
