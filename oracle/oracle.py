"""ctypes wrapper of the C oracle (``slimwise_oracle.c``).

TEST INFRASTRUCTURE ONLY.  A plain, slow, single-threaded CPU definition of
the SlimWise batched-decode MoE layer (arXiv 2609.34117, Sections 2.1 and
3.1), used to check the HIP library.  Arrays are numpy, bf16 tensors are
passed as their uint16 bit patterns.  Nothing here imports or calls the HIP
library.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "slimwise_oracle.c")
_LIB = os.environ.get("SWO_LIB") or os.path.join(_HERE, "libswo.so")
CFLAGS = ["-O2", "-std=c11", "-ffp-contract=off", "-fno-fast-math", "-fPIC", "-shared"]

_lib = None


def lib_path() -> str:
    return _LIB


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (single-threaded, no FMA contraction)."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", *CFLAGS, "-o", tmp, _SRC, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build(force=False)
        lib = ctypes.CDLL(_LIB)
        P = ctypes.c_void_p
        I = ctypes.c_int
        lib.swo_prune_compact.argtypes = [I, I, I, I, P, I, P, P, P, P, P, P, P, P, P, P, P]
        lib.swo_route.argtypes = [I, I, I, P, I, P, P, P, P, P, P, P]
        lib.swo_dispatch.argtypes = [I, I, P, I, P, P, P, P, P]
        lib.swo_forward.argtypes = [I, I, I, I, P, I, P, P, P, P, P]
        lib.swo_forward_f64.argtypes = [I, I, I, I, P, I, P, P, P, P, P]
        lib.swo_shared_expert.argtypes = [I, I, P, I, P, P, P, P]
        lib.swo_routing_mass.argtypes = [I, I, I, P, I, P, P, P, P, P]
        for f in (lib.swo_prune_compact, lib.swo_route, lib.swo_dispatch,
                  lib.swo_forward, lib.swo_forward_f64):
            f.restype = ctypes.c_int
        _lib = lib
    return _lib


def _p(a):
    return None if a is None else a.ctypes.data


def _c(a, dtype):
    if a is None:
        return None
    a = np.ascontiguousarray(a)
    if a.dtype != dtype:
        raise TypeError(f"expected {dtype}, got {a.dtype}")
    return a


def _check(rc: int, what: str):
    if rc != 0:
        raise ValueError(f"oracle {what}: invalid arguments")


def prune_compact(importance, n_keep, top_k, w13=None, w2=None, wr=None, bias=None):
    """Section 3.1: retain the top ``n_keep`` experts by importance.

    Returns ``(kept, remap, keep_mask, w13_c, w2_c, wr_c, bias_c)``; the
    compacted arrays are None where the input was None."""
    lib = _load()
    importance = _c(importance, np.float32)
    m = importance.shape[0]
    hidden = inter = 1
    if w13 is not None:
        w13 = _c(w13, np.uint16)
        _, two_i, hidden = w13.shape
        inter = two_i // 2
    if w2 is not None:
        w2 = _c(w2, np.uint16)
        _, hidden, inter = w2.shape
    if wr is not None:
        wr = _c(wr, np.float32)
        hidden = wr.shape[1]
    bias = _c(bias, np.float32)
    kept = np.empty(max(n_keep, 0), np.int32)
    remap = np.empty(m, np.int32)
    mask = np.empty(m, np.uint8)
    w13_c = None if w13 is None else np.empty((n_keep, 2 * inter, hidden), np.uint16)
    w2_c = None if w2 is None else np.empty((n_keep, hidden, inter), np.uint16)
    wr_c = None if wr is None else np.empty((n_keep, hidden), np.float32)
    bias_c = None if bias is None else np.empty(n_keep, np.float32)
    rc = lib.swo_prune_compact(hidden, inter, m, top_k, _p(importance), n_keep,
                               _p(w13), _p(w2), _p(wr), _p(bias), _p(kept), _p(remap),
                               _p(mask), _p(w13_c), _p(w2_c), _p(wr_c), _p(bias_c))
    _check(rc, "prune_compact")
    return kept, remap, mask, w13_c, w2_c, wr_c, bias_c


def route(x, wr, top_k, keep_mask=None, bias=None, want_logits=False):
    """Section 3.1, Eq. 2: masked top-k routing with renormalised gates.

    Returns ``(topk_ids, topk_w, gap)`` (+ ``logits`` if asked)."""
    lib = _load()
    x = _c(x, np.uint16)
    wr = _c(wr, np.float32)
    t, hidden = x.shape
    m = wr.shape[0]
    keep_mask = _c(keep_mask, np.uint8)
    bias = _c(bias, np.float32)
    ids = np.empty((t, top_k), np.int32)
    w = np.empty((t, top_k), np.float32)
    gap = np.empty(t, np.float32)
    logits = np.empty((t, m), np.float32) if want_logits else None
    rc = lib.swo_route(hidden, m, top_k, _p(x), t, _p(wr), _p(bias), _p(keep_mask),
                       _p(ids), _p(w), _p(gap), _p(logits))
    _check(rc, "route")
    return (ids, w, gap, logits) if want_logits else (ids, w, gap)


def dispatch(topk_ids, n_experts):
    """Section 2.1: expert histogram, offsets, stable permutation, active set.

    Returns ``(counts, offsets, perm, active[:n_active], n_active)``."""
    lib = _load()
    topk_ids = _c(topk_ids, np.int32)
    t, k = topk_ids.shape
    counts = np.empty(n_experts, np.int32)
    offsets = np.empty(n_experts + 1, np.int32)
    perm = np.empty(t * k, np.int32)
    active = np.empty(n_experts, np.int32)
    na = np.zeros(1, np.int32)
    rc = lib.swo_dispatch(n_experts, k, _p(topk_ids), t, _p(counts), _p(offsets),
                          _p(perm), _p(active), _p(na))
    _check(rc, "dispatch")
    n = int(na[0])
    return counts, offsets, perm, active[:n].copy(), n


def _forward(fn, out_dtype, x, w13, w2, topk_ids, topk_w):
    x = _c(x, np.uint16)
    w13 = _c(w13, np.uint16)
    w2 = _c(w2, np.uint16)
    topk_ids = _c(topk_ids, np.int32)
    topk_w = _c(topk_w, np.float32)
    t, hidden = x.shape
    m, two_i, h2 = w13.shape
    inter = two_i // 2
    if h2 != hidden or w2.shape != (m, hidden, inter):
        raise ValueError("oracle forward: shape mismatch")
    k = topk_ids.shape[1]
    out = np.empty((t, hidden), out_dtype)
    rc = fn(hidden, inter, m, k, _p(x), t, _p(w13), _p(w2), _p(topk_ids), _p(topk_w), _p(out))
    _check(rc, "forward")
    return out


def forward(x, w13, w2, topk_ids, topk_w):
    """The layer output with fp32 accumulation (the parity reference)."""
    return _forward(_load().swo_forward, np.float32, x, w13, w2, topk_ids, topk_w)


def forward_f64(x, w13, w2, topk_ids, topk_w):
    """The same computation accumulated in fp64 (error shadow)."""
    return _forward(_load().swo_forward_f64, np.float64, x, w13, w2, topk_ids, topk_w)


def shared_expert(x, w13s, w2s, gate_w, out=None):
    """Section 3.3: out + sigmoid(gate_w . x) * SwiGLU_s(x) per token (out
    defaults to zeros); returns the new output."""
    lib = _load()
    x = _c(x, np.uint16)
    w13s = _c(w13s, np.uint16)
    w2s = _c(w2s, np.uint16)
    gate_w = _c(gate_w, np.float32)
    t, hidden = x.shape
    inter = w2s.shape[-1]
    res = np.zeros((t, hidden), np.float32) if out is None else np.array(out, np.float32, copy=True)
    rc = lib.swo_shared_expert(hidden, inter, _p(x), t, _p(w13s), _p(w2s), _p(gate_w), _p(res))
    _check(rc, "shared_expert")
    return res


def routing_mass(x, wr, top_k, keep_mask=None, bias=None, mass=None):
    """Section 2.3: (mass_softmax, mass_topk) accumulated over the tokens of
    x, onto `mass` (a pair of [m] arrays) if given."""
    lib = _load()
    x = _c(x, np.uint16)
    wr = _c(wr, np.float32)
    t, hidden = x.shape
    m = wr.shape[0]
    keep_mask = _c(keep_mask, np.uint8)
    bias = _c(bias, np.float32)
    ms, mt = ((np.zeros(m, np.float32), np.zeros(m, np.float32)) if mass is None else
              (np.array(mass[0], np.float32, copy=True), np.array(mass[1], np.float32, copy=True)))
    rc = lib.swo_routing_mass(hidden, m, top_k, _p(x), t, _p(wr), _p(bias), _p(keep_mask),
                              _p(ms), _p(mt))
    _check(rc, "routing_mass")
    return ms, mt


def layer(x, wr, w13, w2, top_k, keep_mask=None, bias=None):
    """Route, dispatch and forward of one MoE layer; returns a dict."""
    ids, w, gap = route(x, wr, top_k, keep_mask=keep_mask, bias=bias)
    counts, offsets, perm, active, n_active = dispatch(ids, wr.shape[0])
    out = forward(x, w13, w2, ids, w)
    return dict(topk_ids=ids, topk_w=w, gap=gap, counts=counts, offsets=offsets,
                perm=perm, active=active, n_active=n_active, out=out)
