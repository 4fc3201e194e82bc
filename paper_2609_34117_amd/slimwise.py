"""Thin ctypes binding of libslimwise (the C ABI in ``include/slimwise.h``).

Argument marshalling only: every step of the layer runs in the HIP kernels of
``libslimwise.so``.  torch supplies device memory and the current stream.
bf16 tensors may be ``torch.bfloat16`` or ``torch.uint16``/``torch.int16``
bit patterns.  Importing this module loads the library and raises if it is
not built -- there is no fallback.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass
from typing import Optional

import torch

_LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libslimwise.so")

SW_OK = 0


class SlimwiseError(RuntimeError):
    pass


class Dims(ctypes.Structure):
    _fields_ = [("hidden", ctypes.c_int32), ("inter", ctypes.c_int32),
                ("n_experts", ctypes.c_int32), ("top_k", ctypes.c_int32)]


def _load() -> ctypes.CDLL:
    if not os.path.exists(_LIB_PATH):
        raise ImportError(f"{_LIB_PATH} is not built: run `python -m paper_2609_34117_amd.build`")
    lib = ctypes.CDLL(_LIB_PATH)
    P, I32, SZ = ctypes.c_void_p, ctypes.c_int32, ctypes.c_size_t
    D = ctypes.POINTER(Dims)
    sig = {
        "sw_status_str": ([ctypes.c_int], ctypes.c_char_p),
        "sw_abi_version": ([], I32),
        "sw_moe_prune_compact": ([D, P, I32, P, P, P, P, P, P, P, P, P, P, P, P], ctypes.c_int),
        "sw_moe_route_workspace_bytes": ([D, I32], SZ),
        "sw_moe_route": ([D, P, I32, P, P, P, P, P, P, P, SZ, P], ctypes.c_int),
        "sw_moe_dispatch": ([D, P, I32, P, P, P, P, P, P], ctypes.c_int),
        "sw_moe_route_dispatch": ([D, P, I32, P, P, P, P, P, P, P, P, P, P, P, P, SZ, P],
                                  ctypes.c_int),
        "sw_moe_route_shared_workspace_bytes": ([D, I32, I32, I32], SZ),
        "sw_moe_route_dispatch_shared": ([D, P, I32, P, P, P, I32, I32, P, P, P, P, P, P, P, P, P,
                                          SZ, P],
                                         ctypes.c_int),
        "sw_moe_forward_workspace_bytes": ([D, I32], SZ),
        "sw_moe_forward_kernels": ([D, I32, I32, P, P], ctypes.c_int),
        "sw_moe_pack_experts": ([D, P, P, P, P, P], ctypes.c_int),
        "sw_moe_forward": ([D, P, I32, P, P, I32, P, P, P, P, P, P, P, P, SZ, P], ctypes.c_int),
        "sw_moe_forward_no_alloc": ([D, P, I32, P, P, I32, P, P, P, P, P, P, P, P], ctypes.c_int),
        "sw_moe_forward_gate_up": ([D, P, I32, P, I32, P, P, P, P, P, P, SZ, P], ctypes.c_int),
        "sw_moe_forward_down": ([D, I32, P, I32, P, P, P, P, P, P, SZ, P], ctypes.c_int),
        "sw_moe_forward_combine": ([D, I32, P, P, P, P, SZ, P], ctypes.c_int),
        "sw_moe_shared_workspace_bytes": ([D, I32], SZ),
        "sw_moe_routing_mass_workspace_bytes": ([D, I32], SZ),
        "sw_moe_routing_mass": ([D, P, I32, P, P, P, P, P, P, SZ, P], ctypes.c_int),
        "sw_moe_shared_expert": ([D, P, I32, P, P, I32, P, P, P, SZ, P], ctypes.c_int),
        "sw_moe_layer_workspace_bytes": ([D, I32, I32, I32], SZ),
        "sw_moe_gate_up_builds_plan": ([D, I32, I32], I32),
        "sw_moe_forward_gate_up_plan": ([D, P, I32, P, I32, P, P, P, P, P, P, P, SZ, P],
                                        ctypes.c_int),
        "sw_moe_layer": ([D, P, I32, P, P, P, I32, I32, P, P, I32, P, P, P, P, P, P, P, P, P, P,
                          SZ, P], ctypes.c_int),
        "sw_moe_layer_phase": ([I32, D, P, I32, P, P, P, I32, I32, P, P, I32, P, P, P, P, P, P, P,
                                P, P, P, SZ, P], ctypes.c_int),
    }
    for name, (args, res) in sig.items():
        f = getattr(lib, name)
        f.argtypes = args
        f.restype = res
    lib.signatures = sig
    return lib


LIB = _load()
ABI_VERSION = 10
NO_ALLOC_SCRATCH_BYTES = 32 << 20
ROW_MAJOR, TILED = 0, 1
# sw_kernel_family values
KERNEL_FAMILIES = {0: "none", 1: "prefill", 2: "split_k", 3: "wave", 4: "generic"}
if LIB.sw_abi_version() != ABI_VERSION:
    raise ImportError(f"libslimwise ABI {LIB.sw_abi_version()} != binding ABI {ABI_VERSION}")

_BF16 = (torch.bfloat16, torch.uint16, torch.int16)


def _check(st: int, what: str):
    if st != SW_OK:
        raise SlimwiseError(f"{what}: {LIB.sw_status_str(st).decode()}")


def _ptr(t: Optional[torch.Tensor], dtypes=None, name="tensor"):
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if dtypes is not None and t.dtype not in dtypes:
        raise TypeError(f"{name}: dtype {t.dtype} not in {dtypes}")
    return t.data_ptr()


def _stream(stream) -> Optional[int]:
    if stream is None:
        stream = torch.cuda.current_stream()
    return stream.cuda_stream


def dims(hidden: int, inter: int, n_experts: int, top_k: int) -> Dims:
    return Dims(hidden, inter, n_experts, top_k)


def _empty(shape, dtype, device):
    return torch.empty(shape, dtype=dtype, device=device)


def sw_moe_route_workspace_bytes(d: Dims, n_tokens: int) -> int:
    return LIB.sw_moe_route_workspace_bytes(ctypes.byref(d), n_tokens)


def sw_moe_forward_workspace_bytes(d: Dims, n_tokens: int) -> int:
    return LIB.sw_moe_forward_workspace_bytes(ctypes.byref(d), n_tokens)


def sw_moe_forward_kernels(d: Dims, n_tokens: int, layout: int = TILED) -> tuple:
    """The kernel families (names of ``KERNEL_FAMILIES``) that serve the
    gate/up and the down projection of ``n_tokens`` tokens of this shape."""
    gu, dn = ctypes.c_int32(), ctypes.c_int32()
    _check(LIB.sw_moe_forward_kernels(ctypes.byref(d), n_tokens, layout, ctypes.byref(gu),
                                      ctypes.byref(dn)), "sw_moe_forward_kernels")
    return KERNEL_FAMILIES[gu.value], KERNEL_FAMILIES[dn.value]


def workspace(nbytes: int, device) -> torch.Tensor:
    """A 256-byte-aligned byte buffer (torch's caching allocator aligns to 512)."""
    return torch.empty(max(nbytes, 1), dtype=torch.uint8, device=device)


def sw_moe_prune_compact(importance: torch.Tensor, n_keep: int, top_k: int, *, hidden: int = 8,
                         inter: int = 8, w13=None, w2=None, wr=None, bias=None, compact=True,
                         stream=None) -> dict:
    """Section 3.1: kept set, remap, mask and (if ``compact``) the compacted pool."""
    dev = importance.device
    m = importance.shape[0]
    if w13 is not None:
        inter, hidden = w13.shape[1] // 2, w13.shape[2]
    elif wr is not None:
        hidden = wr.shape[1]
    d = Dims(hidden, inter, m, top_k)
    kept = _empty(max(n_keep, 0), torch.int32, dev)
    remap = _empty(m, torch.int32, dev)
    mask = _empty(m, torch.uint8, dev)
    w13_c = _empty((n_keep, 2 * inter, hidden), w13.dtype, dev) if compact and w13 is not None else None
    w2_c = _empty((n_keep, hidden, inter), w2.dtype, dev) if compact and w2 is not None else None
    wr_c = _empty((n_keep, hidden), torch.float32, dev) if compact and wr is not None else None
    bias_c = _empty(n_keep, torch.float32, dev) if compact and bias is not None else None
    st = LIB.sw_moe_prune_compact(
        ctypes.byref(d), _ptr(importance, (torch.float32,), "importance"), n_keep,
        _ptr(w13, _BF16, "w13"), _ptr(w2, _BF16, "w2"), _ptr(wr, (torch.float32,), "wr"),
        _ptr(bias, (torch.float32,), "bias"), _ptr(kept), _ptr(remap), _ptr(mask),
        _ptr(w13_c), _ptr(w2_c), _ptr(wr_c), _ptr(bias_c), _stream(stream))
    _check(st, "sw_moe_prune_compact")
    return dict(kept=kept, remap=remap, keep_mask=mask, w13=w13_c, w2=w2_c, wr=wr_c, bias=bias_c)


def sw_moe_pack_experts(w13=None, w2=None, *, top_k: int = 1, stream=None):
    """Re-lay expert pools out in the tiled (fragment-major) device layout.

    Returns ``(w13_tiled, w2_tiled)`` (None where the input was None)."""
    ref = w13 if w13 is not None else w2
    if w13 is not None:
        m, two_i, hidden = w13.shape
        inter = two_i // 2
    else:
        m, hidden, inter = w2.shape
    d = Dims(hidden, inter, m, min(top_k, m))
    w13_t = torch.empty_like(w13) if w13 is not None else None
    w2_t = torch.empty_like(w2) if w2 is not None else None
    st = LIB.sw_moe_pack_experts(ctypes.byref(d), _ptr(w13, _BF16, "w13"), _ptr(w2, _BF16, "w2"),
                                 _ptr(w13_t), _ptr(w2_t), _stream(stream))
    _check(st, "sw_moe_pack_experts")
    del ref
    return w13_t, w2_t


def sw_moe_route(x: torch.Tensor, wr: torch.Tensor, top_k: int, *, keep_mask=None, bias=None,
                 want_gap=True, out=None, ws=None, stream=None):
    """Section 3.1, Eq. 2: masked top-k and renormalised gates.

    Returns ``(topk_ids, topk_w, gap)``; ``out`` may supply that tuple."""
    t, hidden = x.shape
    m = wr.shape[0]
    d = Dims(hidden, 8, m, top_k)
    if out is None:
        out = (_empty((t, top_k), torch.int32, x.device), _empty((t, top_k), torch.float32, x.device),
               _empty(t, torch.float32, x.device) if want_gap else None)
    ids, w, gap = out
    nbytes = sw_moe_route_workspace_bytes(d, t)
    if ws is None:
        ws = workspace(nbytes, x.device)
    st = LIB.sw_moe_route(ctypes.byref(d), _ptr(x, _BF16, "x"), t, _ptr(wr, (torch.float32,), "wr"),
                          _ptr(bias, (torch.float32,), "bias"), _ptr(keep_mask, (torch.uint8,), "keep_mask"),
                          _ptr(ids), _ptr(w), _ptr(gap), _ptr(ws), ws.numel(), _stream(stream))
    _check(st, "sw_moe_route")
    return ids, w, gap


@dataclass
class Plan:
    """Dispatch plan of one step (device tensors)."""
    counts: torch.Tensor
    offsets: torch.Tensor
    perm: torch.Tensor
    active: torch.Tensor
    n_active: torch.Tensor


def alloc_plan(n_tokens: int, n_experts: int, top_k: int, device) -> Plan:
    return Plan(_empty(n_experts, torch.int32, device), _empty(n_experts + 1, torch.int32, device),
                _empty(max(n_tokens * top_k, 1), torch.int32, device),
                _empty(n_experts, torch.int32, device), _empty(1, torch.int32, device))


def sw_moe_dispatch(topk_ids: torch.Tensor, n_experts: int, *, plan: Optional[Plan] = None,
                    stream=None) -> Plan:
    """Section 2.1: histogram, offsets, stable permutation, active set."""
    t, k = topk_ids.shape
    d = Dims(8, 8, n_experts, k)
    if plan is None:
        plan = alloc_plan(t, n_experts, k, topk_ids.device)
    st = LIB.sw_moe_dispatch(ctypes.byref(d), _ptr(topk_ids, (torch.int32,), "topk_ids"), t,
                             _ptr(plan.counts), _ptr(plan.offsets), _ptr(plan.perm),
                             _ptr(plan.active), _ptr(plan.n_active), _stream(stream))
    _check(st, "sw_moe_dispatch")
    return plan


def sw_moe_route_dispatch(x: torch.Tensor, wr: torch.Tensor, top_k: int, *, keep_mask=None,
                          bias=None, want_gap=True, out=None, plan: Optional[Plan] = None, ws=None,
                          stream=None):
    """Section 3.1, Eq. 2 then Section 2.1, Eq. 1: ``sw_moe_route`` followed by
    ``sw_moe_dispatch`` in one call (bitwise the same results).

    Returns ``(topk_ids, topk_w, gap, plan)``."""
    t, hidden = x.shape
    m = wr.shape[0]
    d = Dims(hidden, 8, m, top_k)
    if out is None:
        out = (_empty((t, top_k), torch.int32, x.device), _empty((t, top_k), torch.float32, x.device),
               _empty(t, torch.float32, x.device) if want_gap else None)
    ids, w, gap = out
    if plan is None:
        plan = alloc_plan(t, m, top_k, x.device)
    nbytes = sw_moe_route_workspace_bytes(d, t)
    if ws is None:
        ws = workspace(nbytes, x.device)
    st = LIB.sw_moe_route_dispatch(
        ctypes.byref(d), _ptr(x, _BF16, "x"), t, _ptr(wr, (torch.float32,), "wr"),
        _ptr(bias, (torch.float32,), "bias"), _ptr(keep_mask, (torch.uint8,), "keep_mask"),
        _ptr(ids), _ptr(w), _ptr(gap), _ptr(plan.counts), _ptr(plan.offsets), _ptr(plan.perm),
        _ptr(plan.active), _ptr(plan.n_active), _ptr(ws), ws.numel(), _stream(stream))
    _check(st, "sw_moe_route_dispatch")
    return ids, w, gap, plan


def sw_moe_route_shared_workspace_bytes(d: Dims, n_tokens: int, n_shared: int,
                                        n_groups: int = 1) -> int:
    return LIB.sw_moe_route_shared_workspace_bytes(ctypes.byref(d), n_tokens, n_shared, n_groups)


def sw_moe_route_dispatch_shared(x: torch.Tensor, wr: torch.Tensor, top_k: int, n_shared: int, *,
                                 n_groups: int = 1, keep_mask=None, bias=None, want_gap=True,
                                 out=None, plan: Optional[Plan] = None, ws=None, stream=None):
    """Section 3.3: route + dispatch with the shared expert folded into the
    plan.  ``wr`` is [m + 1, H] (the router rows, then the shared gate row);
    the pool holds ``n_groups`` copies of the ``n_shared`` parts, and token
    t gets ``n_shared`` more slots, ids m + g * n_shared + s with
    g = t * n_groups // T, with the sigmoid of the shared gate logit.

    Returns ``(topk_ids [T, k + n_shared], topk_w, gap, plan over
    m + n_groups * n_shared)``."""
    t, hidden = x.shape
    m = wr.shape[0] - 1
    kout = top_k + n_shared
    d = Dims(hidden, 8, m, top_k)
    if out is None:
        out = (_empty((t, kout), torch.int32, x.device), _empty((t, kout), torch.float32, x.device),
               _empty(t, torch.float32, x.device) if want_gap else None)
    ids, w, gap = out
    if plan is None:
        plan = alloc_plan(t, m + n_groups * n_shared, kout, x.device)
    if ws is None:
        ws = workspace(sw_moe_route_shared_workspace_bytes(d, t, n_shared, n_groups), x.device)
    st = LIB.sw_moe_route_dispatch_shared(
        ctypes.byref(d), _ptr(x, _BF16, "x"), t, _ptr(wr, (torch.float32,), "wr"),
        _ptr(bias, (torch.float32,), "bias"), _ptr(keep_mask, (torch.uint8,), "keep_mask"),
        n_shared, n_groups, _ptr(ids), _ptr(w), _ptr(gap), _ptr(plan.counts), _ptr(plan.offsets),
        _ptr(plan.perm), _ptr(plan.active), _ptr(plan.n_active), _ptr(ws), ws.numel(),
        _stream(stream))
    _check(st, "sw_moe_route_dispatch_shared")
    return ids, w, gap, plan


def _fwd_dims(x_or_t, w13_or_w2, top_k, which="w13"):
    if which == "w13":
        m, two_i, hidden = w13_or_w2.shape
        return Dims(hidden, two_i // 2, m, top_k)
    m, hidden, inter = w13_or_w2.shape
    return Dims(hidden, inter, m, top_k)


def sw_moe_forward(x: torch.Tensor, w13: torch.Tensor, w2: torch.Tensor, topk_w: torch.Tensor,
                   plan: Plan, *, layout: int = ROW_MAJOR, out=None, ws=None,
                   stream=None) -> torch.Tensor:
    """Expert SwiGLU FFNs of every routed pair and the gate-weighted combine.

    ``layout``: ROW_MAJOR or TILED (weights from sw_moe_pack_experts)."""
    t = x.shape[0]
    d = _fwd_dims(x, w13, topk_w.shape[1])
    if out is None:
        out = _empty((t, d.hidden), torch.float32, x.device)
    if ws is None:
        ws = workspace(sw_moe_forward_workspace_bytes(d, t), x.device)
    st = LIB.sw_moe_forward(ctypes.byref(d), _ptr(x, _BF16, "x"), t, _ptr(w13, _BF16, "w13"),
                            _ptr(w2, _BF16, "w2"), layout, _ptr(topk_w, (torch.float32,), "topk_w"),
                            _ptr(plan.counts), _ptr(plan.offsets), _ptr(plan.perm),
                            _ptr(plan.active), _ptr(plan.n_active), _ptr(out, (torch.float32,), "out"),
                            _ptr(ws), ws.numel(), _stream(stream))
    _check(st, "sw_moe_forward")
    return out


def sw_moe_forward_no_alloc(x: torch.Tensor, w13: torch.Tensor, w2: torch.Tensor,
                            topk_w: torch.Tensor, plan: Plan, *, layout: int = ROW_MAJOR, out=None,
                            stream=None) -> torch.Tensor:
    """``sw_moe_forward`` on the library's static scratch: no workspace
    argument and no device allocation inside the call (``out`` may be
    passed in so that the caller allocates nothing either)."""
    t = x.shape[0]
    d = _fwd_dims(x, w13, topk_w.shape[1])
    if out is None:
        out = _empty((t, d.hidden), torch.float32, x.device)
    st = LIB.sw_moe_forward_no_alloc(ctypes.byref(d), _ptr(x, _BF16, "x"), t, _ptr(w13, _BF16, "w13"),
                                     _ptr(w2, _BF16, "w2"), layout,
                                     _ptr(topk_w, (torch.float32,), "topk_w"), _ptr(plan.counts),
                                     _ptr(plan.offsets), _ptr(plan.perm), _ptr(plan.active),
                                     _ptr(plan.n_active), _ptr(out, (torch.float32,), "out"),
                                     _stream(stream))
    _check(st, "sw_moe_forward_no_alloc")
    return out


def sw_moe_forward_gate_up(x, w13, top_k, plan: Plan, ws, *, layout: int = ROW_MAJOR, stream=None):
    t = x.shape[0]
    d = _fwd_dims(x, w13, top_k)
    st = LIB.sw_moe_forward_gate_up(ctypes.byref(d), _ptr(x, _BF16, "x"), t, _ptr(w13, _BF16, "w13"),
                                    layout,
                                    _ptr(plan.counts), _ptr(plan.offsets), _ptr(plan.perm),
                                    _ptr(plan.active), _ptr(plan.n_active), _ptr(ws), ws.numel(),
                                    _stream(stream))
    _check(st, "sw_moe_forward_gate_up")


def sw_moe_gate_up_builds_plan(d: Dims, n_tokens: int, layout: int = ROW_MAJOR) -> bool:
    return bool(LIB.sw_moe_gate_up_builds_plan(ctypes.byref(d), n_tokens, layout))


def sw_moe_forward_gate_up_plan(x, w13, topk_ids, plan: Plan, ws, *, layout: int = ROW_MAJOR,
                                stream=None):
    """The gate/up phase that builds ``plan`` from ``topk_ids`` (Section 2.1)
    on the way, for the decode batches ``sw_moe_gate_up_builds_plan`` names."""
    t = x.shape[0]
    d = _fwd_dims(x, w13, topk_ids.shape[1])
    st = LIB.sw_moe_forward_gate_up_plan(
        ctypes.byref(d), _ptr(x, _BF16, "x"), t, _ptr(w13, _BF16, "w13"), layout,
        _ptr(topk_ids, (torch.int32,), "topk_ids"), _ptr(plan.counts), _ptr(plan.offsets),
        _ptr(plan.perm), _ptr(plan.active), _ptr(plan.n_active), _ptr(ws), ws.numel(),
        _stream(stream))
    _check(st, "sw_moe_forward_gate_up_plan")


def sw_moe_forward_down(n_tokens, w2, top_k, plan: Plan, ws, *, layout: int = ROW_MAJOR,
                        stream=None):
    d = _fwd_dims(n_tokens, w2, top_k, which="w2")
    st = LIB.sw_moe_forward_down(ctypes.byref(d), n_tokens, _ptr(w2, _BF16, "w2"), layout,
                                 _ptr(plan.counts), _ptr(plan.offsets), _ptr(plan.perm),
                                 _ptr(plan.active), _ptr(plan.n_active), _ptr(ws), ws.numel(),
                                 _stream(stream))
    _check(st, "sw_moe_forward_down")


def sw_moe_forward_combine(topk_w, hidden, inter, n_experts, plan: Plan, out, ws, stream=None):
    t, k = topk_w.shape
    d = Dims(hidden, inter, n_experts, k)
    st = LIB.sw_moe_forward_combine(ctypes.byref(d), t, _ptr(topk_w, (torch.float32,), "topk_w"),
                                    _ptr(plan.n_active), _ptr(out, (torch.float32,), "out"),
                                    _ptr(ws), ws.numel(), _stream(stream))
    _check(st, "sw_moe_forward_combine")


def sw_moe_routing_mass(x: torch.Tensor, wr: torch.Tensor, top_k: int, *, keep_mask=None,
                        bias=None, mass=None, ws=None, stream=None):
    """Section 2.3: routing-mass statistics of the tokens of x, accumulated
    onto `mass` = (mass_softmax, mass_topk) (fp32 [m] device tensors, created
    as zeros if None); returns the pair."""
    t, hidden = x.shape
    m = wr.shape[0]
    d = Dims(hidden, 8, m, top_k)
    if mass is None:
        mass = (torch.zeros(m, dtype=torch.float32, device=x.device),
                torch.zeros(m, dtype=torch.float32, device=x.device))
    if ws is None:
        ws = workspace(LIB.sw_moe_routing_mass_workspace_bytes(ctypes.byref(d), t), x.device)
    st = LIB.sw_moe_routing_mass(ctypes.byref(d), _ptr(x, _BF16, "x"), t,
                                 _ptr(wr, (torch.float32,), "wr"), _ptr(bias, (torch.float32,), "bias"),
                                 _ptr(keep_mask, (torch.uint8,), "keep_mask"),
                                 _ptr(mass[0], (torch.float32,), "mass_softmax"),
                                 _ptr(mass[1], (torch.float32,), "mass_topk"), _ptr(ws), ws.numel(),
                                 _stream(stream))
    _check(st, "sw_moe_routing_mass")
    return mass


def sw_moe_shared_workspace_bytes(d: Dims, n_tokens: int) -> int:
    return LIB.sw_moe_shared_workspace_bytes(ctypes.byref(d), n_tokens)


def sw_moe_shared_expert(x: torch.Tensor, w13: torch.Tensor, w2: torch.Tensor,
                         gate_w: torch.Tensor, out: torch.Tensor, *, layout: int = ROW_MAJOR,
                         ws=None, stream=None) -> torch.Tensor:
    """Section 3.3: out += sigmoid(gate_w . x) * SwiGLU_s(x) (in place)."""
    t, hidden = x.shape
    two_i = w13.shape[-2]
    d = Dims(hidden, two_i // 2, 1, 1)
    if ws is None:
        ws = workspace(sw_moe_shared_workspace_bytes(d, t), x.device)
    st = LIB.sw_moe_shared_expert(ctypes.byref(d), _ptr(x, _BF16, "x"), t, _ptr(w13, _BF16, "w13"),
                                  _ptr(w2, _BF16, "w2"), layout,
                                  _ptr(gate_w, (torch.float32,), "gate_w"),
                                  _ptr(out, (torch.float32,), "out"), _ptr(ws), ws.numel(),
                                  _stream(stream))
    _check(st, "sw_moe_shared_expert")
    return out


def sw_moe_layer_workspace_bytes(d: Dims, n_tokens: int, n_shared: int = 0,
                                 n_groups: int = 1) -> int:
    return LIB.sw_moe_layer_workspace_bytes(ctypes.byref(d), n_tokens, n_shared, n_groups)


def sw_moe_layer(x: torch.Tensor, wr: torch.Tensor, top_k: int, w13: torch.Tensor,
                 w2: torch.Tensor, *, layout: int = ROW_MAJOR, n_shared: int = 0,
                 n_groups: int = 1, keep_mask=None, bias=None, want_gap=True, route_out=None,
                 plan: Optional[Plan] = None, out=None, ws=None, stream=None, phase=None):
    """Route, dispatch plan, expert FFNs and combine of one layer in one call
    (Section 3.1, Eq. 2; Section 2.1, Eq. 1): bitwise what
    ``sw_moe_route_dispatch`` (or ``sw_moe_route_dispatch_shared`` when
    ``n_shared`` > 0, ``wr`` then holding the shared gate row last) followed
    by ``sw_moe_forward`` give.  ``w13``/``w2`` hold the pool of
    m + n_groups * n_shared experts.

    ``phase`` (0-3) runs one phase of the call (``sw_moe_layer_phase``).

    Returns ``(topk_ids, topk_w, gap, plan, out)``."""
    t, hidden = x.shape
    m = wr.shape[0] - (1 if n_shared else 0)
    kout = top_k + n_shared
    pool = _fwd_dims(x, w13, kout)
    m_pool = m + (n_groups * n_shared if n_shared else 0)
    if pool.n_experts != m_pool:
        raise ValueError(f"w13 holds {pool.n_experts} experts, the layer's pool is {m_pool}")
    d = Dims(hidden, pool.inter, m, top_k)
    if route_out is None:
        route_out = (_empty((t, kout), torch.int32, x.device),
                     _empty((t, kout), torch.float32, x.device),
                     _empty(t, torch.float32, x.device) if want_gap else None)
    ids, w, gap = route_out
    if plan is None:
        plan = alloc_plan(t, m_pool, kout, x.device)
    if out is None:
        out = _empty((t, hidden), torch.float32, x.device)
    if ws is None:
        ws = workspace(sw_moe_layer_workspace_bytes(d, t, n_shared, n_groups), x.device)
    args = (ctypes.byref(d), _ptr(x, _BF16, "x"), t, _ptr(wr, (torch.float32,), "wr"),
            _ptr(bias, (torch.float32,), "bias"), _ptr(keep_mask, (torch.uint8,), "keep_mask"),
            n_shared, n_groups, _ptr(w13, _BF16, "w13"), _ptr(w2, _BF16, "w2"), layout, _ptr(ids),
            _ptr(w), _ptr(gap), _ptr(plan.counts), _ptr(plan.offsets), _ptr(plan.perm),
            _ptr(plan.active), _ptr(plan.n_active), _ptr(out, (torch.float32,), "out"), _ptr(ws),
            ws.numel(), _stream(stream))
    if phase is None:
        _check(LIB.sw_moe_layer(*args), "sw_moe_layer")
    else:
        _check(LIB.sw_moe_layer_phase(phase, *args), "sw_moe_layer_phase")
    return ids, w, gap, plan, out


def moe_layer(x, wr, w13, w2, top_k, *, keep_mask=None, bias=None, layout: int = ROW_MAJOR,
              stream=None) -> dict:
    """One layer through ``sw_moe_layer`` (allocating convenience wrapper)."""
    ids, w, gap, plan, out = sw_moe_layer(x, wr, top_k, w13, w2, layout=layout,
                                          keep_mask=keep_mask, bias=bias, stream=stream)
    return dict(topk_ids=ids, topk_w=w, gap=gap, plan=plan, out=out)
