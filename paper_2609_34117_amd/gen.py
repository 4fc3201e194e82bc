"""ctypes binding of libswgen.so (``include/swgen.h``): device draws of
synthetic expert weights from the counter-based stream that
``inputs.philox_normal_bf16`` draws on the host.  Argument marshalling only;
importing raises if the library is not built."""
from __future__ import annotations

import ctypes
import os

import numpy as np
import torch

_LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libswgen.so")


def _load() -> ctypes.CDLL:
    if not os.path.exists(_LIB_PATH):
        raise ImportError(f"{_LIB_PATH} is not built: run `python -m paper_2609_34117_amd.build`")
    lib = ctypes.CDLL(_LIB_PATH)
    P, U64 = ctypes.c_void_p, ctypes.c_uint64
    sig = {
        "swg_philox_normal_bf16": ([P, U64, U64, U64, U64, ctypes.c_float, P], ctypes.c_int),
    }
    for name, (args, res) in sig.items():
        f = getattr(lib, name)
        f.argtypes = args
        f.restype = res
    lib.signatures = sig
    return lib


LIB = _load()


def philox_normal_bf16(dst: torch.Tensor, key: np.ndarray, start: int, std: float, stream=None):
    """Fills the device tensor `dst` (bf16 bits, any 2-byte dtype) with
    elements start .. start + dst.numel() - 1 of the tensor keyed `key`."""
    if not dst.is_cuda or not dst.is_contiguous() or dst.element_size() != 2:
        raise ValueError("dst must be a contiguous device tensor of 2-byte elements")
    s = torch.cuda.current_stream() if stream is None else stream
    rc = LIB.swg_philox_normal_bf16(dst.data_ptr(), dst.numel(), int(key[0]), int(key[1]), start,
                                    std, s.cuda_stream)
    if rc != 0:
        raise RuntimeError(f"swg_philox_normal_bf16 failed ({rc})")
    return dst
