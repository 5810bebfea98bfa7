"""Python binding of the APB host-share C ABI (``include/apb.h``).

Argument marshalling only: every step of the path runs in the HIP kernels of
``libapb.so``.  PyTorch supplies device memory and streams.  The names match
the C entry points without the ``apb_`` prefix.  If the library is missing,
every call raises: there is no fallback.
"""
from __future__ import annotations

import ctypes
import os

PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG, "libapb.so")

APB_OK = 0
NOALLOC_SCRATCH_BYTES = 16 << 20  # APB_DECODE_NOALLOC_SCRATCH_BYTES
STATUS_NAMES = {0: "APB_OK", 1: "APB_ERR_NULL_POINTER", 2: "APB_ERR_BAD_SHAPE",
                3: "APB_ERR_UNSUPPORTED", 4: "APB_ERR_MISALIGNED", 5: "APB_ERR_HIP",
                6: "APB_ERR_ALIAS", 7: "APB_ERR_SCRATCH"}
EXPORTED = ("apb_compress_select", "apb_attention_fwd", "apb_validate_problem",
            "apb_attention_flops", "apb_status_string", "apb_last_error", "apb_abi_version",
            "apb_validate_decode", "apb_decode_workspace_size", "apb_decode_attention",
            "apb_decode_attention_noalloc",
            "apb_merge_partials", "apb_validate_scorer", "apb_scorer_workspace_size",
            "apb_retaining_scores", "apb_validate_layer", "apb_layer_workspace_size",
            "apb_layer_flops", "apb_layer_fwd")


class ApbError(RuntimeError):
    def __init__(self, status: int, where: str, detail: str = ""):
        self.status = status
        msg = f"{where}: {STATUS_NAMES.get(status, status)}"
        if detail:
            msg += f" ({detail})"
        super().__init__(msg)


class Problem(ctypes.Structure):
    """``apb_problem_t``: one host's share of one attention layer."""

    _fields_ = [("n_hosts", ctypes.c_int32), ("host_idx", ctypes.c_int32),
                ("anchor_len", ctypes.c_int32), ("local_len", ctypes.c_int32),
                ("pass_len", ctypes.c_int32), ("n_q_heads", ctypes.c_int32),
                ("n_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32)]

    @classmethod
    def of(cls, p) -> "Problem":
        """From any object with the same field names (e.g. inputs.Problem)."""
        return cls(*(int(getattr(p, f)) for f, _ in cls._fields_))


class DecodeProblem(ctypes.Structure):
    """``apb_decode_problem_t``: one host's decoding step (Alg. 3)."""

    _fields_ = [("n_q_heads", ctypes.c_int32), ("n_kv_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("cache_len", ctypes.c_int32),
                ("n_new", ctypes.c_int32), ("append_new", ctypes.c_int32)]

    @classmethod
    def of(cls, p) -> "DecodeProblem":
        if isinstance(p, cls):
            return p
        return cls(*(int(getattr(p, f)) for f, _ in cls._fields_))


class ScorerProblem(ctypes.Structure):
    """``apb_scorer_problem_t``: one host's retaining-head scoring."""

    _fields_ = [("anchor_len", ctypes.c_int32), ("local_len", ctypes.c_int32),
                ("n_q_heads", ctypes.c_int32), ("n_kv_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("hidden", ctypes.c_int32)]


class LayerProblem(ctypes.Structure):
    """``apb_layer_problem_t``: one host's whole layer (Alg. 2)."""

    _fields_ = [("attn", Problem), ("hidden", ctypes.c_int32), ("intermediate", ctypes.c_int32),
                ("scorer_hidden", ctypes.c_int32), ("rms_eps", ctypes.c_float),
                ("rope_theta", ctypes.c_float)]

    @classmethod
    def of(cls, lw) -> "LayerProblem":
        """From an object with ``problem``, ``hidden``, ``intermediate``,
        ``scorer_hidden``, ``eps`` and ``theta`` (e.g. inputs.LayerWorkload)."""
        if isinstance(lw, cls):
            return lw
        return cls(Problem.of(lw.problem), int(lw.hidden), int(lw.intermediate),
                   int(lw.scorer_hidden), float(lw.eps), float(lw.theta))


class LayerWeights(ctypes.Structure):
    """``apb_layer_weights_t``: device pointers of one layer's weights."""

    _fields_ = [(n, ctypes.c_void_p) for n in ("ln1", "w_qkv", "w_o", "ln2", "w_gate", "w_up",
                                               "w_down", "r_w1", "r_b1", "r_w2", "r_b2")]


_lib = None


def lib() -> ctypes.CDLL:
    """Load ``libapb.so`` (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with "
                               "`python -m paper_2502_12085_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        vp, i32p = ctypes.c_void_p, ctypes.POINTER(Problem)
        L.apb_compress_select.argtypes = [i32p, vp, vp, vp, vp, vp, vp, vp]
        L.apb_compress_select.restype = ctypes.c_int
        L.apb_attention_fwd.argtypes = [i32p, vp, vp, vp, vp, vp, vp, vp, ctypes.c_float, vp]
        L.apb_attention_fwd.restype = ctypes.c_int
        L.apb_validate_problem.argtypes = [i32p]
        L.apb_validate_problem.restype = ctypes.c_int
        L.apb_attention_flops.argtypes = [i32p]
        L.apb_attention_flops.restype = ctypes.c_double
        L.apb_status_string.argtypes = [ctypes.c_int]
        L.apb_status_string.restype = ctypes.c_char_p
        L.apb_last_error.argtypes = []
        L.apb_last_error.restype = ctypes.c_char_p
        L.apb_abi_version.argtypes = []
        L.apb_abi_version.restype = ctypes.c_int
        dp = ctypes.POINTER(DecodeProblem)
        L.apb_validate_decode.argtypes = [dp]
        L.apb_validate_decode.restype = ctypes.c_int
        L.apb_decode_workspace_size.argtypes = [dp, ctypes.POINTER(ctypes.c_uint64)]
        L.apb_decode_workspace_size.restype = ctypes.c_int
        L.apb_decode_attention.argtypes = [dp, vp, vp, vp, vp, vp, vp, vp, ctypes.c_float, vp,
                                           ctypes.c_uint64, vp]
        L.apb_decode_attention.restype = ctypes.c_int
        L.apb_decode_attention_noalloc.argtypes = [dp, vp, vp, vp, vp, vp, vp, vp, ctypes.c_float,
                                                   vp]
        L.apb_decode_attention_noalloc.restype = ctypes.c_int
        L.apb_merge_partials.argtypes = [ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, vp, vp,
                                         vp, vp, vp]
        L.apb_merge_partials.restype = ctypes.c_int
        sp = ctypes.POINTER(ScorerProblem)
        L.apb_validate_scorer.argtypes = [sp]
        L.apb_validate_scorer.restype = ctypes.c_int
        L.apb_scorer_workspace_size.argtypes = [sp, ctypes.POINTER(ctypes.c_uint64)]
        L.apb_scorer_workspace_size.restype = ctypes.c_int
        L.apb_retaining_scores.argtypes = [sp, vp, vp, vp, vp, vp, vp, vp, vp, vp, ctypes.c_uint64,
                                           vp]
        L.apb_retaining_scores.restype = ctypes.c_int
        lp_ = ctypes.POINTER(LayerProblem)
        L.apb_validate_layer.argtypes = [lp_]
        L.apb_validate_layer.restype = ctypes.c_int
        L.apb_layer_workspace_size.argtypes = [lp_, ctypes.POINTER(ctypes.c_uint64)]
        L.apb_layer_workspace_size.restype = ctypes.c_int
        L.apb_layer_flops.argtypes = [lp_]
        L.apb_layer_flops.restype = ctypes.c_double
        L.apb_layer_fwd.argtypes = [lp_, ctypes.POINTER(LayerWeights), vp, vp, vp, vp, vp, vp, vp,
                                    vp, ctypes.c_uint64, vp]
        L.apb_layer_fwd.restype = ctypes.c_int
        _lib = L
    return _lib


def _ptr(t, name, dtypes):
    """Device pointer of a contiguous CUDA/HIP tensor, or None."""
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if t.dtype not in dtypes:
        raise ValueError(f"{name} has dtype {t.dtype}, expected one of {dtypes}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return t.data_ptr()


def _stream(stream):
    import torch
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def _check(status, where):
    if status != APB_OK:
        detail = lib().apb_status_string(status).decode()
        if status == 5:
            detail += ": " + lib().apb_last_error().decode()
        raise ApbError(status, where, detail)


def _bf16_types():
    import torch
    return (torch.bfloat16, torch.int16, torch.uint16)


def compress_select(problem, scores, k, v, out_idx, out_k, out_v, stream=None):
    """``apb_compress_select``: top-l_p of ``scores`` [n_kv, Lb] (fp32) per KV
    head and gather of K/V rows La+idx into ``out_k``/``out_v`` [n_kv, l_p, d]."""
    import torch
    b = _bf16_types()
    st = lib().apb_compress_select(
        ctypes.byref(Problem.of(problem)), _ptr(scores, "scores", (torch.float32,)),
        _ptr(k, "k", b), _ptr(v, "v", b), _ptr(out_idx, "out_idx", (torch.int32,)),
        _ptr(out_k, "out_k", b), _ptr(out_v, "out_v", b), _stream(stream))
    _check(st, "apb_compress_select")


def attention_fwd(problem, q, k, v, k_pass, v_pass, o, lse=None, softmax_scale=0.0,
                  stream=None):
    """``apb_attention_fwd``: modified-mask attention of one host share."""
    import torch
    b = _bf16_types()
    st = lib().apb_attention_fwd(
        ctypes.byref(Problem.of(problem)), _ptr(q, "q", b), _ptr(k, "k", b), _ptr(v, "v", b),
        _ptr(k_pass, "k_pass", b), _ptr(v_pass, "v_pass", b), _ptr(o, "o", b),
        _ptr(lse, "lse", (torch.float32,)), float(softmax_scale), _stream(stream))
    _check(st, "apb_attention_fwd")


def validate_problem(problem) -> int:
    return lib().apb_validate_problem(ctypes.byref(Problem.of(problem)))


def attention_flops(problem) -> float:
    return lib().apb_attention_flops(ctypes.byref(Problem.of(problem)))


def abi_version() -> int:
    return lib().apb_abi_version()


def validate_decode(problem) -> int:
    return lib().apb_validate_decode(ctypes.byref(DecodeProblem.of(problem)))


def decode_workspace_size(problem) -> int:
    """``apb_decode_workspace_size``: device scratch bytes a decode call needs."""
    n = ctypes.c_uint64(0)
    _check(lib().apb_decode_workspace_size(ctypes.byref(DecodeProblem.of(problem)),
                                           ctypes.byref(n)), "apb_decode_workspace_size")
    return int(n.value)


def decode_attention(problem, q, k_cache, v_cache, k_new, v_new, o_part, lse_part, workspace,
                     softmax_scale=0.0, stream=None):
    """``apb_decode_attention``: one host's stage-2 partial attention (Alg. 3).
    ``workspace`` is a device tensor of at least ``decode_workspace_size``
    bytes (any dtype)."""
    import torch
    b = _bf16_types()
    f = (torch.float32,)
    if workspace is None or not workspace.is_cuda or not workspace.is_contiguous():
        raise ValueError("workspace must be a contiguous device tensor")
    st = lib().apb_decode_attention(
        ctypes.byref(DecodeProblem.of(problem)), _ptr(q, "q", b), _ptr(k_cache, "k_cache", b),
        _ptr(v_cache, "v_cache", b), _ptr(k_new, "k_new", b), _ptr(v_new, "v_new", b),
        _ptr(o_part, "o_part", f), _ptr(lse_part, "lse_part", f), float(softmax_scale),
        workspace.data_ptr(), workspace.numel() * workspace.element_size(), _stream(stream))
    _check(st, "apb_decode_attention")


def decode_attention_noalloc(problem, q, k_cache, v_cache, k_new, v_new, o_part, lse_part,
                             softmax_scale=0.0, stream=None):
    """``apb_decode_attention_noalloc``: ``decode_attention`` without a
    workspace; the library's own per-GPU scratch holds the split partials
    (``NOALLOC_SCRATCH_BYTES``).  Calls that overlap on one GPU race."""
    import torch
    b = _bf16_types()
    f = (torch.float32,)
    st = lib().apb_decode_attention_noalloc(
        ctypes.byref(DecodeProblem.of(problem)), _ptr(q, "q", b), _ptr(k_cache, "k_cache", b),
        _ptr(v_cache, "v_cache", b), _ptr(k_new, "k_new", b), _ptr(v_new, "v_new", b),
        _ptr(o_part, "o_part", f), _ptr(lse_part, "lse_part", f), float(softmax_scale),
        _stream(stream))
    _check(st, "apb_decode_attention_noalloc")


def merge_partials(o_parts, lse_parts, o, lse=None, stream=None):
    """``apb_merge_partials``: MergeScore (Alg. 3) of ``o_parts`` [P, rows, d]
    (fp32) with ``lse_parts`` [P, rows] into ``o`` [rows, d] (bf16)."""
    import torch
    f = (torch.float32,)
    n_parts, rows, d = o_parts.shape
    st = lib().apb_merge_partials(
        int(n_parts), int(rows), int(d), _ptr(o_parts, "o_parts", f),
        _ptr(lse_parts, "lse_parts", f), _ptr(o, "o", _bf16_types()), _ptr(lse, "lse", f),
        _stream(stream))
    _check(st, "apb_merge_partials")


def validate_scorer(problem) -> int:
    return lib().apb_validate_scorer(ctypes.byref(problem))


def scorer_workspace_size(problem) -> int:
    """``apb_scorer_workspace_size``: device scratch bytes a scorer call needs."""
    n = ctypes.c_uint64(0)
    _check(lib().apb_scorer_workspace_size(ctypes.byref(problem), ctypes.byref(n)),
           "apb_scorer_workspace_size")
    return int(n.value)


def retaining_scores(problem, q, k, v, w1, b1, w2, b2, scores, workspace, stream=None):
    """``apb_retaining_scores``: retaining-head scores [n_kv, Lb] (fp32) of the
    local rows of ``q``/``k``/``v`` with weights ``w1`` (bf16 [hidden, F]),
    ``b1``, ``w2`` [n_kv, hidden], ``b2`` (fp32)."""
    import torch
    b = _bf16_types()
    f = (torch.float32,)
    if workspace is None or not workspace.is_cuda or not workspace.is_contiguous():
        raise ValueError("workspace must be a contiguous device tensor")
    st = lib().apb_retaining_scores(
        ctypes.byref(problem), _ptr(q, "q", b), _ptr(k, "k", b), _ptr(v, "v", b),
        _ptr(w1, "w1", b), _ptr(b1, "b1", f), _ptr(w2, "w2", f), _ptr(b2, "b2", f),
        _ptr(scores, "scores", f), workspace.data_ptr(),
        workspace.numel() * workspace.element_size(), _stream(stream))
    _check(st, "apb_retaining_scores")


def validate_layer(problem) -> int:
    return lib().apb_validate_layer(ctypes.byref(LayerProblem.of(problem)))


def layer_workspace_size(problem) -> int:
    """``apb_layer_workspace_size``: device scratch bytes a layer call needs."""
    n = ctypes.c_uint64(0)
    _check(lib().apb_layer_workspace_size(ctypes.byref(LayerProblem.of(problem)), ctypes.byref(n)),
           "apb_layer_workspace_size")
    return int(n.value)


def layer_flops(problem) -> float:
    return lib().apb_layer_flops(ctypes.byref(LayerProblem.of(problem)))


def layer_fwd(problem, weights: dict, hidden_in, positions, k_cache, v_cache, pass_k, pass_v,
              hidden_out, workspace, stream=None):
    """``apb_layer_fwd``: one host's whole layer (Alg. 2).  ``weights`` maps the
    ``apb_layer_weights_t`` field names to device tensors (bf16, the
    retaining head's r_b1/r_w2/r_b2 fp32); ``pass_k``/``pass_v`` are the
    rank-major [H, n_kv, l_p, d] passing buffers (slots < host_idx read, slot
    host_idx written)."""
    import torch
    b = _bf16_types()
    f = (torch.float32,)
    w = LayerWeights()
    for name, _ in LayerWeights._fields_:
        setattr(w, name, _ptr(weights[name], name, f if name in ("r_b1", "r_w2", "r_b2") else b))
    if workspace is None or not workspace.is_cuda or not workspace.is_contiguous():
        raise ValueError("workspace must be a contiguous device tensor")
    st = lib().apb_layer_fwd(
        ctypes.byref(LayerProblem.of(problem)), ctypes.byref(w), _ptr(hidden_in, "hidden_in", b),
        _ptr(positions, "positions", (torch.int32,)), _ptr(k_cache, "k_cache", b),
        _ptr(v_cache, "v_cache", b), _ptr(pass_k, "pass_k", b), _ptr(pass_v, "pass_v", b),
        _ptr(hidden_out, "hidden_out", b), workspace.data_ptr(),
        workspace.numel() * workspace.element_size(), _stream(stream))
    _check(st, "apb_layer_fwd")
