"""Binding of the matrix-core ceiling probe (``include/apb_probe.h``,
``libapb_probe.so``): measurement infrastructure for the benchmark, not a
step of the attention path.  Raises if the library has not been built."""
from __future__ import annotations

import ctypes
import os

PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG, "libapb_probe.so")
EXPORTED = ("apb_probe_mfma_bf16", "apb_probe_mfma_flops")

_lib = None


def lib() -> ctypes.CDLL:
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with "
                               "`python -m paper_2502_12085_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        vp = ctypes.c_void_p
        L.apb_probe_mfma_bf16.argtypes = [vp, vp, ctypes.c_int32, ctypes.c_int32, vp]
        L.apb_probe_mfma_bf16.restype = ctypes.c_int32
        L.apb_probe_mfma_flops.argtypes = [ctypes.c_int32, ctypes.c_int32]
        L.apb_probe_mfma_flops.restype = ctypes.c_double
        _lib = L
    return _lib


def mfma_bf16(operands, sink, n_workgroups: int, iters: int, stream) -> None:
    """Launch the MFMA loop: ``operands`` a device bf16 tensor of >= 8192
    elements, ``sink`` a device fp32 tensor of >= n_workgroups*512."""
    import torch
    if not (operands.is_cuda and sink.is_cuda):
        raise ValueError("operands and sink must be device tensors")
    if operands.dtype != torch.bfloat16 or operands.numel() < 8192:
        raise ValueError("operands: bf16, at least 8192 elements")
    if sink.dtype != torch.float32 or sink.numel() < n_workgroups * 512:
        raise ValueError("sink: fp32, at least n_workgroups*512 elements")
    st = lib().apb_probe_mfma_bf16(operands.data_ptr(), sink.data_ptr(), int(n_workgroups),
                                   int(iters), stream.cuda_stream)
    if st != 0:
        raise RuntimeError(f"apb_probe_mfma_bf16 returned {st}")


def mfma_flops(n_workgroups: int, iters: int) -> float:
    return lib().apb_probe_mfma_flops(int(n_workgroups), int(iters))
