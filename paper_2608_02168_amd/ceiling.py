"""ctypes binding of libhg_ceiling.so: the random-row gather ceiling that the
benchmark measures beside the SpMM kernels (see csrc/hg_ceiling.hip)."""
from __future__ import annotations

import ctypes as C
import os

import torch

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libhg_ceiling.so")
_lib = None


def lib() -> C.CDLL:
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is not built: run python -m paper_2608_02168_amd.build")
        L = C.CDLL(LIB_PATH)
        L.hgc_random_rows.argtypes = [C.c_void_p, C.c_int64, C.c_int64, C.c_uint64, C.c_void_p]
        L.hgc_random_rows.restype = C.c_int
        L.hgc_gather.argtypes = [C.c_void_p, C.c_int64, C.c_int32, C.c_void_p, C.c_int64, C.c_int32,
                                 C.c_void_p, C.c_int32, C.c_void_p]
        L.hgc_gather.restype = C.c_int
        _lib = L
    return _lib


def _stream() -> C.c_void_p:
    return C.c_void_p(torch.cuda.current_stream().cuda_stream)


def random_rows(idx: torch.Tensor, n_rows: int, seed: int) -> None:
    assert idx.dtype == torch.int32 and idx.is_cuda and idx.is_contiguous()
    rc = lib().hgc_random_rows(C.c_void_p(idx.data_ptr()), idx.numel(), n_rows, seed & (2**64 - 1), _stream())
    if rc != 0:
        raise RuntimeError(f"hgc_random_rows failed ({rc})")


def gather(table: torch.Tensor, idx: torch.Tensor, group: int, out: torch.Tensor, write: bool) -> None:
    assert table.dtype == torch.float32 and table.dim() == 2 and table.is_contiguous() and table.is_cuda
    assert idx.dtype == torch.int32 and idx.is_cuda and idx.is_contiguous()
    d = table.shape[1]
    need = (idx.numel() // group) if write else 1
    assert out.dtype == torch.float32 and out.is_contiguous() and out.numel() >= need * d
    rc = lib().hgc_gather(C.c_void_p(table.data_ptr()), table.shape[0], d, C.c_void_p(idx.data_ptr()), idx.numel(),
                          group, C.c_void_p(out.data_ptr()), 1 if write else 0, _stream())
    if rc != 0:
        raise RuntimeError(f"hgc_gather failed ({rc})")
