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
STATUS_NAMES = {0: "APB_OK", 1: "APB_ERR_NULL_POINTER", 2: "APB_ERR_BAD_SHAPE",
                3: "APB_ERR_UNSUPPORTED", 4: "APB_ERR_MISALIGNED", 5: "APB_ERR_HIP",
                6: "APB_ERR_ALIAS"}
EXPORTED = ("apb_compress_select", "apb_attention_fwd", "apb_validate_problem",
            "apb_attention_flops", "apb_status_string", "apb_last_error", "apb_abi_version")


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
