"""CPU checks of the C ABI: the libraries load, export every symbol their
headers declare, and reject bad arguments before touching the device (so
these calls need no GPU and launch nothing)."""
import ctypes
import os
import re
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "slimwise.h")
LIB_PATH = os.path.join(ROOT, "paper_2609_34117_amd", "libslimwise.so")

SW_OK, SW_ERR_NULL, SW_ERR_SHAPE, SW_ERR_ALIGN, SW_ERR_UNSUPPORTED, SW_ERR_WORKSPACE = range(6)


class Dims(ctypes.Structure):
    _fields_ = [("hidden", ctypes.c_int32), ("inter", ctypes.c_int32),
                ("n_experts", ctypes.c_int32), ("top_k", ctypes.c_int32)]


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(sw_\w+)\s*\(", text)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(LIB_PATH):
        from paper_2609_34117_amd import build
        build.build()
    return ctypes.CDLL(LIB_PATH)


def test_header_declares_the_four_calls():
    names = declared_functions()
    for n in ("sw_moe_prune_compact", "sw_moe_route", "sw_moe_dispatch", "sw_moe_forward"):
        assert n in names


def test_library_exports_every_declared_symbol(lib):
    out = subprocess.run(["nm", "-D", "--defined-only", LIB_PATH], capture_output=True, text=True,
                         check=True).stdout
    exported = set(line.split()[-1] for line in out.splitlines() if line.strip())
    missing = [n for n in declared_functions() if n not in exported]
    assert not missing, missing
    for n in declared_functions():
        getattr(lib, n)


def test_status_strings_and_version(lib):
    lib.sw_status_str.restype = ctypes.c_char_p
    for s in range(7):
        assert lib.sw_status_str(s).startswith(b"SW_")
    assert lib.sw_abi_version() == 10


def _route(lib, d, x=16, t=4, wr=16, ids=16, w=16, ws=16, nbytes=1 << 20):
    f = lib.sw_moe_route
    P = ctypes.c_void_p
    f.argtypes = [ctypes.POINTER(Dims), P, ctypes.c_int32, P, P, P, P, P, P, P, ctypes.c_size_t, P]
    return f(ctypes.byref(d) if d is not None else None, x, t, wr, None, None, ids, w, None, ws,
             nbytes, None)


def test_route_validation_precedes_any_launch(lib):
    ok = Dims(64, 32, 8, 2)
    assert _route(lib, None) == SW_ERR_NULL
    assert _route(lib, Dims(0, 32, 8, 2)) == SW_ERR_SHAPE
    assert _route(lib, Dims(64, 32, 8, 9)) == SW_ERR_SHAPE        # k > m
    assert _route(lib, Dims(60, 32, 8, 2)) == SW_ERR_ALIGN        # H % 8
    assert _route(lib, Dims(64, 32, 2048, 2)) == SW_ERR_UNSUPPORTED
    assert _route(lib, Dims(64, 32, 64, 33)) == SW_ERR_UNSUPPORTED
    assert _route(lib, ok, t=-1) == SW_ERR_SHAPE
    assert _route(lib, ok, x=None) == SW_ERR_NULL
    assert _route(lib, ok, x=24) == SW_ERR_ALIGN                 # not 16-byte aligned
    assert _route(lib, ok, ids=18) == SW_ERR_ALIGN
    assert _route(lib, ok, nbytes=16) == SW_ERR_WORKSPACE
    assert _route(lib, ok, t=0, x=None, wr=None) == SW_OK         # empty batch: nothing to do
    assert _route(lib, Dims(64, 32, 8, 8), t=(1 << 28)) == SW_ERR_UNSUPPORTED  # T*k >= 2^31


def test_workspace_queries(lib):
    P = ctypes.POINTER(Dims)
    for name in ("sw_moe_route_workspace_bytes", "sw_moe_forward_workspace_bytes",
                 "sw_moe_shared_workspace_bytes", "sw_moe_routing_mass_workspace_bytes"):
        f = getattr(lib, name)
        f.argtypes = [P, ctypes.c_int32]
        f.restype = ctypes.c_size_t
        assert f(ctypes.byref(Dims(2048, 512, 256, 8)), 0) == 0
        assert f(None, 8) == 0
    f = lib.sw_moe_forward_workspace_bytes
    # h hi/lo (2 x T*k*I bf16) + y (T*k*H fp32)
    assert f(ctypes.byref(Dims(2048, 512, 256, 8)), 64) == 2 * 512 * 512 * 2 + 512 * 2048 * 4
    # router logits in up to 4 slices of H: a decode batch (few 16 x 16 tiles)
    # keeps 4 partial planes
    assert lib.sw_moe_route_workspace_bytes(ctypes.byref(Dims(2048, 512, 256, 8)), 64) == 4 * 64 * 256 * 4
    # prefill: two planes (64x64 tiles over slices of at least 8 chunks of
    # 128 columns of H), then the chunked dispatch's scratch: 32 chunks of
    # 1024 pairs (a histogram and a flag each)
    assert lib.sw_moe_route_workspace_bytes(ctypes.byref(Dims(2048, 512, 256, 8)), 4096) == (
        2 * 4096 * 256 * 4 + 32 * 256 * 4 + 256)
    assert lib.sw_moe_route_workspace_bytes(ctypes.byref(Dims(256, 128, 16, 2)), 8) == 8 * 16 * 4


def test_prune_and_dispatch_validation(lib):
    P = ctypes.c_void_p
    pc = lib.sw_moe_prune_compact
    pc.argtypes = [ctypes.POINTER(Dims)] + [P, ctypes.c_int32] + [P] * 11 + [P]
    d = Dims(64, 32, 16, 4)
    assert pc(ctypes.byref(d), 16, 3, None, None, None, None, 16, 16, 16, None, None, None, None, None) == SW_ERR_SHAPE
    assert pc(ctypes.byref(d), 16, 17, None, None, None, None, 16, 16, 16, None, None, None, None, None) == SW_ERR_SHAPE
    assert pc(ctypes.byref(d), None, 8, None, None, None, None, 16, 16, 16, None, None, None, None, None) == SW_ERR_NULL
    # a compacted output needs its source
    assert pc(ctypes.byref(d), 16, 8, None, None, None, None, 16, 16, 16, 16, None, None, None, None) == SW_ERR_NULL
    assert pc(ctypes.byref(d), 16, 8, 16, None, None, None, 16, 16, 16, 24, None, None, None, None) == SW_ERR_ALIGN
    dp = lib.sw_moe_dispatch
    dp.argtypes = [ctypes.POINTER(Dims), P, ctypes.c_int32, P, P, P, P, P, P]
    assert dp(ctypes.byref(d), 16, 4, None, 16, 16, 16, 16, None) == SW_ERR_NULL
    assert dp(ctypes.byref(d), None, 4, 16, 16, 16, 16, 16, None) == SW_ERR_NULL
    assert dp(ctypes.byref(d), 16, 4, 18, 16, 16, 16, 16, None) == SW_ERR_ALIGN


def test_route_dispatch_validation(lib):
    P = ctypes.c_void_p
    f = lib.sw_moe_route_dispatch
    f.argtypes = [ctypes.POINTER(Dims), P, ctypes.c_int32, P, P, P, P, P, P, P, P, P, P, P, P,
                  ctypes.c_size_t, P]
    d = Dims(64, 32, 8, 2)
    args = dict(x=16, wr=16, ids=16, w=16, c=16, o=16, p=16, a=16, na=16, ws=16)

    def call(dims=d, t=4, nbytes=1 << 20, **kw):
        a = dict(args, **kw)
        return f(ctypes.byref(dims) if dims is not None else None, a["x"], t, a["wr"], None, None,
                 a["ids"], a["w"], None, a["c"], a["o"], a["p"], a["a"], a["na"], a["ws"], nbytes, None)

    assert call(dims=None) == SW_ERR_NULL
    assert call(dims=Dims(64, 32, 8, 9)) == SW_ERR_SHAPE
    assert call(t=-1) == SW_ERR_SHAPE
    assert call(c=None) == SW_ERR_NULL
    assert call(x=None) == SW_ERR_NULL
    assert call(p=None) == SW_ERR_NULL
    assert call(x=24) == SW_ERR_ALIGN
    assert call(p=18) == SW_ERR_ALIGN
    assert call(na=2) == SW_ERR_ALIGN
    assert call(nbytes=16) == SW_ERR_WORKSPACE


def test_routing_mass_validation(lib):
    P = ctypes.c_void_p
    f = lib.sw_moe_routing_mass
    f.argtypes = [ctypes.POINTER(Dims), P, ctypes.c_int32, P, P, P, P, P, P, ctypes.c_size_t, P]
    d = Dims(64, 8, 8, 2)

    def call(dims=d, t=4, nbytes=1 << 20, **kw):
        a = dict(dict(x=16, wr=16, ms=16, mt=16, ws=16), **kw)
        return f(ctypes.byref(dims), a["x"], t, a["wr"], None, None, a["ms"], a["mt"], a["ws"],
                 nbytes, None)

    assert call(dims=Dims(64, 8, 8, 9)) == SW_ERR_SHAPE
    assert call(ms=None, mt=None, x=None) == SW_OK      # nothing to accumulate
    assert call(x=None) == SW_ERR_NULL
    assert call(wr=24) == SW_ERR_ALIGN
    assert call(mt=18) == SW_ERR_ALIGN
    assert call(nbytes=16) == SW_ERR_WORKSPACE


def test_shared_expert_validation(lib):
    P = ctypes.c_void_p
    f = lib.sw_moe_shared_expert
    f.argtypes = [ctypes.POINTER(Dims), P, ctypes.c_int32, P, P, ctypes.c_int32, P, P, P,
                  ctypes.c_size_t, P]
    d = Dims(64, 32, 1, 1)
    q = lib.sw_moe_shared_workspace_bytes
    q.argtypes = [ctypes.POINTER(Dims), ctypes.c_int32]
    q.restype = ctypes.c_size_t
    need = q(ctypes.byref(d), 4)
    assert need > 0

    def call(dims=d, nbytes=need, lay=0, **kw):
        a = dict(dict(x=16, w13=16, w2=16, g=16, out=16, ws=16), **kw)
        return f(ctypes.byref(dims), a["x"], 4, a["w13"], a["w2"], lay, a["g"], a["out"], a["ws"],
                 nbytes, None)

    assert call(dims=Dims(64, 32, 2, 1)) == SW_ERR_SHAPE   # one expert, top-1
    assert call(dims=Dims(64, 32, 1, 2)) == SW_ERR_SHAPE
    assert call(g=None) == SW_ERR_NULL
    assert call(out=None) == SW_ERR_NULL
    assert call(g=24) == SW_ERR_ALIGN
    assert call(nbytes=need - 1) == SW_ERR_WORKSPACE
    assert call(lay=3) == SW_ERR_SHAPE


def test_forward_validation(lib):
    P = ctypes.c_void_p
    f = lib.sw_moe_forward
    f.argtypes = [ctypes.POINTER(Dims), P, ctypes.c_int32, P, P, ctypes.c_int32, P, P, P, P, P, P,
                  P, P, ctypes.c_size_t, P]
    d = Dims(64, 32, 8, 2)
    q = lib.sw_moe_forward_workspace_bytes
    q.argtypes = [ctypes.POINTER(Dims), ctypes.c_int32]
    q.restype = ctypes.c_size_t
    need = q(ctypes.byref(d), 4)
    args = dict(x=16, w13=16, w2=16, lay=0, tw=16, c=16, o=16, p=16, a=16, na=16, out=16, ws=16)

    def call(nbytes=need, **kw):
        a = dict(args, **kw)
        return f(ctypes.byref(d), a["x"], 4, a["w13"], a["w2"], a["lay"], a["tw"], a["c"], a["o"],
                 a["p"], a["a"], a["na"], a["out"], a["ws"], nbytes, None)

    assert call(nbytes=need - 1) == SW_ERR_WORKSPACE
    assert call(w2=None) == SW_ERR_NULL
    assert call(na=None) == SW_ERR_NULL
    assert call(out=20) == SW_ERR_ALIGN
    assert call(ws=8) == SW_ERR_ALIGN
    assert call(lay=2) == SW_ERR_SHAPE           # unknown layout
    d.hidden, d.inter = 72, 40                   # tiled layout needs multiples of 32
    need2 = q(ctypes.byref(d), 4)
    assert call(nbytes=need2, lay=1) == SW_ERR_UNSUPPORTED


def test_layer_call_validation_and_plan_query(lib):
    # every rejection happens before the device is touched (no GPU here)
    P, I32, SZ, D = ctypes.c_void_p, ctypes.c_int32, ctypes.c_size_t, ctypes.POINTER(Dims)
    q = lib.sw_moe_layer_workspace_bytes
    q.argtypes, q.restype = [D, I32, I32, I32], SZ
    rq = lib.sw_moe_route_workspace_bytes
    rq.argtypes, rq.restype = [D, I32], SZ
    sq = lib.sw_moe_route_shared_workspace_bytes
    sq.argtypes, sq.restype = [D, I32, I32, I32], SZ
    fq = lib.sw_moe_forward_workspace_bytes
    fq.argtypes, fq.restype = [D, I32], SZ
    d = Dims(2048, 768, 64, 8)
    up = lambda v: (v + 255) // 256 * 256
    # the routing's workspace, then the forward's (on the pool of the routed
    # experts and the shared expert's parts)
    assert q(ctypes.byref(d), 64, 0, 1) == up(rq(ctypes.byref(d), 64)) + fq(ctypes.byref(d), 64)
    assert q(ctypes.byref(d), 64, 2, 3) == (up(sq(ctypes.byref(d), 64, 2, 3)) +
                                            fq(ctypes.byref(Dims(2048, 768, 70, 10)), 64))
    assert q(ctypes.byref(d), 0, 0, 1) == 0
    assert q(None, 8, 0, 1) == 0
    assert q(ctypes.byref(d), 8, -1, 1) == 0
    assert q(ctypes.byref(d), 8, 2, 0) == 0
    need = q(ctypes.byref(d), 4, 0, 1)
    f = lib.sw_moe_layer
    f.argtypes = [D, P, I32, P, P, P, I32, I32, P, P, I32, P, P, P, P, P, P, P, P, P, P, SZ, P]
    args = dict(x=16, T=4, wr=16, bias=None, keep=None, S=0, R=1, w13=16, w2=16, lay=1, ids=16,
                w=16, gap=None, c=16, o=16, p=16, a=16, na=16, out=16, ws=16)

    def call(nbytes=need, **kw):
        a = dict(args, **kw)
        return f(ctypes.byref(d), a["x"], a["T"], a["wr"], a["bias"], a["keep"], a["S"], a["R"],
                 a["w13"], a["w2"], a["lay"], a["ids"], a["w"], a["gap"], a["c"], a["o"], a["p"],
                 a["a"], a["na"], a["out"], a["ws"], nbytes, None)

    assert call(nbytes=need - 1) == SW_ERR_WORKSPACE
    for name in ("x", "wr", "w13", "w2", "ids", "w", "c", "p", "na", "out", "ws"):
        assert call(**{name: None}) == SW_ERR_NULL, name
    assert call(out=20) == SW_ERR_ALIGN
    assert call(wr=8) == SW_ERR_ALIGN
    assert call(p=18) == SW_ERR_ALIGN
    assert call(lay=2) == SW_ERR_SHAPE
    assert call(T=-1) == SW_ERR_SHAPE
    assert call(S=-1) == SW_ERR_SHAPE
    assert call(S=2, R=0) == SW_ERR_SHAPE
    assert call(S=2, R=600) == SW_ERR_UNSUPPORTED          # 64 + 1200 experts
    assert call(S=30) == SW_ERR_UNSUPPORTED                # 38 slots a token
    ph = lib.sw_moe_layer_phase
    ph.argtypes = [I32] + f.argtypes
    for bad_phase in (-1, 4):
        assert ph(bad_phase, ctypes.byref(d), 16, 4, 16, None, None, 0, 1, 16, 16, 1, 16, 16, None,
                  16, 16, 16, 16, 16, 16, 16, need, None) == SW_ERR_SHAPE
    assert ph(1, ctypes.byref(d), 16, 4, 16, None, None, 0, 1, 16, 16, 1, 16, 16, None, 16, 16,
              16, 16, 16, 16, 16, need - 1, None) == SW_ERR_WORKSPACE
    # which shapes build the plan in the gate/up launch (host logic only)
    b = lib.sw_moe_gate_up_builds_plan
    b.argtypes, b.restype = [D, I32, I32], I32
    built = lambda dd, T, lay=1: b(ctypes.byref(dd), T, lay)
    assert built(d, 64) == 1 and built(d, 3) == 1 and built(d, 64, 0) == 1
    assert built(d, 65) == 0                               # the 128-token variants
    assert built(d, 2) == 0                                # split-K kernels
    assert built(d, 0) == 0 and b(None, 8, 1) == 0
    assert built(Dims(2048, 512, 512, 8), 48) == 1         # 1922 plan words
    assert built(Dims(2048, 512, 512, 16), 64) == 0        # 2562 plan words: too many
    assert built(Dims(2048, 512, 600, 8), 8) == 0          # more experts than threads
    assert built(Dims(256, 128, 480, 16), 63) == 1         # 2450 plan words
    assert built(Dims(256, 128, 480, 16), 64) == 0         # 2466
    assert built(Dims(40, 40, 16, 2), 8, 0) == 0           # the generic kernels
    # the phase that builds it rejects other shapes before any launch
    g = lib.sw_moe_forward_gate_up_plan
    g.argtypes = [D, P, I32, P, I32, P, P, P, P, P, P, P, SZ, P]
    gneed = fq(ctypes.byref(d), 65)
    assert g(ctypes.byref(d), 16, 65, 16, 1, 16, 16, 16, 16, 16, 16, 16, gneed, None) == \
        SW_ERR_UNSUPPORTED
    assert g(ctypes.byref(d), 16, 0, 16, 1, 16, 16, 16, 16, 16, 16, 16, gneed, None) == \
        SW_ERR_UNSUPPORTED
    assert g(ctypes.byref(d), 16, 64, 16, 1, None, 16, 16, 16, 16, 16, 16, gneed, None) == \
        SW_ERR_NULL


def test_forward_no_alloc_validation(lib):
    # every rejection happens before the device is touched (no GPU here)
    P = ctypes.c_void_p
    f = lib.sw_moe_forward_no_alloc
    f.argtypes = [ctypes.POINTER(Dims), P, ctypes.c_int32, P, P, ctypes.c_int32, P, P, P, P, P, P,
                  P, P]
    q = lib.sw_moe_forward_workspace_bytes
    q.argtypes = [ctypes.POINTER(Dims), ctypes.c_int32]
    q.restype = ctypes.c_size_t
    limit = 32 << 20
    d = Dims(2048, 768, 128, 8)
    args = dict(x=16, w13=16, w2=16, lay=0, tw=16, c=16, o=16, p=16, a=16, na=16, out=16)

    def call(T, **kw):
        a = dict(args, **kw)
        return f(ctypes.byref(d), a["x"], T, a["w13"], a["w2"], a["lay"], a["tw"], a["c"], a["o"],
                 a["p"], a["a"], a["na"], a["out"], None)

    # the scratch holds (4I + 4H) bytes a pair: 2978 pairs at H 2048, I 768
    assert q(ctypes.byref(d), 372) <= limit < q(ctypes.byref(d), 373)
    assert call(373) == SW_ERR_WORKSPACE
    assert call(4096) == SW_ERR_WORKSPACE
    assert call(0) == SW_OK                      # nothing to do, nothing launched
    assert call(-1) == SW_ERR_SHAPE
    assert call(64, na=None) == SW_ERR_NULL
    assert call(64, x=None) == SW_ERR_NULL
    assert call(64, p=18) == SW_ERR_ALIGN
    assert call(64, out=20) == SW_ERR_ALIGN
    assert call(64, lay=2) == SW_ERR_SHAPE
    d.top_k = 200
    assert call(4) == SW_ERR_SHAPE               # k > m


def _families(lib, d, T, layout=1):
    gu, dn = ctypes.c_int32(-1), ctypes.c_int32(-1)
    st = lib.sw_moe_forward_kernels(ctypes.byref(d), T, layout, ctypes.byref(gu), ctypes.byref(dn))
    return st, gu.value, dn.value


def test_forward_kernel_families(lib):
    # sw_kernel_family: none 0, prefill 1, split-K 2, wave 3, generic 4 (host logic only)
    NONE, PREFILL, SPLIT_K, WAVE, GENERIC = range(5)
    dec = Dims(2048, 768, 64, 8)      # the pruned batch-64 decode layer
    assert _families(lib, dec, 64) == (SW_OK, WAVE, WAVE)
    assert _families(lib, dec, 1) == (SW_OK, SPLIT_K, SPLIT_K)
    assert _families(lib, dec, 0) == (SW_OK, NONE, NONE)
    pre = Dims(2048, 512, 256, 8)     # the 4096-token prefill layer
    assert _families(lib, pre, 4096) == (SW_OK, PREFILL, PREFILL)
    assert _families(lib, pre, 4096, layout=0) == (SW_OK, PREFILL, PREFILL)
    # from 16 pairs per expert on, the prefill kernels; under it, or on a
    # pool under 16, the decode kernels
    assert _families(lib, pre, 512)[1:] == (PREFILL, PREFILL)
    assert _families(lib, pre, 511)[1:] == (WAVE, WAVE)
    assert _families(lib, pre, 256)[1:] == (WAVE, WAVE)
    assert _families(lib, Dims(256, 128, 8, 2), 400)[1:] == (WAVE, WAVE)
    # the prefill test shapes (hidden 256 and 384, I 128) do take the prefill kernels
    assert _families(lib, Dims(256, 128, 16, 4), 512)[1:] == (PREFILL, PREFILL)
    assert _families(lib, Dims(384, 128, 16, 4), 512)[1:] == (PREFILL, PREFILL)
    assert _families(lib, Dims(256, 128, 16, 2), 400)[1:] == (PREFILL, PREFILL)
    # K not in whole pipeline rounds: not the prefill kernels
    assert _families(lib, Dims(2048, 192, 256, 8), 4096)[2] != PREFILL
    # a row-major shape outside the streaming kernels' limits
    assert _families(lib, Dims(40, 40, 16, 2), 8, layout=0)[1:] == (GENERIC, GENERIC)
    # errors as sw_moe_forward reports them
    gu = ctypes.c_int32()
    assert lib.sw_moe_forward_kernels(None, 1, 1, ctypes.byref(gu), ctypes.byref(gu)) == SW_ERR_NULL
    assert lib.sw_moe_forward_kernels(ctypes.byref(dec), 1, 1, None, ctypes.byref(gu)) == SW_ERR_NULL
    assert _families(lib, dec, -1)[0] == SW_ERR_SHAPE
    assert _families(lib, dec, 4, layout=7)[0] == SW_ERR_SHAPE
    assert _families(lib, Dims(40, 40, 16, 2), 8, layout=1)[0] == SW_ERR_UNSUPPORTED


def test_pack_validation(lib):
    P = ctypes.c_void_p
    f = lib.sw_moe_pack_experts
    f.argtypes = [ctypes.POINTER(Dims), P, P, P, P, P]
    assert f(ctypes.byref(Dims(72, 32, 4, 2)), 16, 16, 16, 16, None) == SW_ERR_UNSUPPORTED
    assert f(ctypes.byref(Dims(4096, 32, 4, 2)), 16, 16, 16, 16, None) == SW_ERR_UNSUPPORTED
    assert f(ctypes.byref(Dims(64, 32, 4, 2)), 16, None, None, None, None) == SW_ERR_NULL
    assert f(ctypes.byref(Dims(64, 32, 4, 2)), 16, None, 24, None, None) == SW_ERR_ALIGN


def _prototypes(header=HEADER, prefix="sw_"):
    """name -> list of parameter declarations, parsed from the header."""
    text = re.sub(r"/\*.*?\*/", "", open(header).read(), flags=re.S)
    protos = {}
    for m in re.finditer(r"\b(" + prefix + r"\w+)\s*\(([^;{]*?)\)\s*;", text, flags=re.S):
        params = [p.strip() for p in m.group(2).split(",") if p.strip() and p.strip() != "void"]
        protos[m.group(1)] = params
    return protos


def test_binding_signatures_match_the_header():
    # A ctypes argtypes list shorter than the C prototype silently passes the
    # trailing arguments as default-converted C ints (a 64-bit stream handle
    # would arrive with garbage in its upper half), so check every binding.
    from paper_2609_34117_amd import slimwise

    protos = _prototypes()
    assert set(slimwise.LIB.signatures) == set(protos)
    for name, (args, _res) in slimwise.LIB.signatures.items():
        params = protos[name]
        assert len(args) == len(params), (name, len(args), len(params))
        for a, decl in zip(args, params):
            if "*" in decl:
                assert a is ctypes.c_void_p or issubclass(a, ctypes._Pointer), (name, decl, a)
            elif decl.startswith("size_t"):
                assert a is ctypes.c_size_t, (name, decl, a)
            elif decl.startswith("int32_t"):
                assert a is ctypes.c_int32, (name, decl, a)
            elif decl.startswith("int "):
                assert a is ctypes.c_int, (name, decl, a)
            else:
                raise AssertionError(f"unhandled parameter {decl} of {name}")


GEN_HEADER = os.path.join(ROOT, "include", "swgen.h")
GEN_LIB_PATH = os.path.join(ROOT, "paper_2609_34117_amd", "libswgen.so")


def test_input_draw_library_exports_and_binding_match_its_header():
    from paper_2609_34117_amd import gen

    protos = _prototypes(GEN_HEADER, "swg_")
    assert protos, "no declarations parsed"
    out = subprocess.run(["nm", "-D", "--defined-only", GEN_LIB_PATH], capture_output=True,
                         text=True, check=True).stdout
    exported = set(line.split()[-1] for line in out.splitlines() if line.strip())
    assert set(protos) <= exported
    assert set(gen.LIB.signatures) == set(protos)
    for name, (args, _res) in gen.LIB.signatures.items():
        params = protos[name]
        assert len(args) == len(params), (name, len(args), len(params))
        for a, decl in zip(args, params):
            if "*" in decl:
                assert a is ctypes.c_void_p, (name, decl, a)
            elif decl.startswith("uint64_t"):
                assert a is ctypes.c_uint64, (name, decl, a)
            elif decl.startswith("float"):
                assert a is ctypes.c_float, (name, decl, a)
            else:
                raise AssertionError(f"unhandled parameter {decl} of {name}")
    # no work and a NULL destination: validated without a launch
    assert gen.LIB.swg_philox_normal_bf16(None, 0, 1, 2, 0, 0.02, None) == 0
    assert gen.LIB.swg_philox_normal_bf16(None, 5, 1, 2, 0, 0.02, None) == 1

