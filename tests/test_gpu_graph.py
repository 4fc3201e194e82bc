"""A decode step (route + dispatch, expert FFNs, combine, shared expert)
captured in a HIP graph: every replay, with eager work and synchronisations
between the replays, equals the eager step bit for bit and matches the
oracle.  The library enqueues only kernels on the caller's stream (no
allocation, copy or memset), which is what makes the step capturable."""
import numpy as np
import pytest

import oracle
from paper_2609_34117_amd import inputs as I
from parity import compare_out

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module")
def sw():
    assert torch.cuda.is_available(), "GPU tests need a device"
    from paper_2609_34117_amd import slimwise

    return slimwise


def dev(a):
    a = np.ascontiguousarray(a)
    return torch.from_numpy(a.view(np.int16) if a.dtype == np.uint16 else a).cuda()


def host(t):
    a = t.cpu().numpy()
    return a.view(np.uint16) if a.dtype == np.int16 else a


# batch 2 runs the split-K kernels, batch 64 the wave-streaming kernels
@pytest.mark.parametrize("batch", [2, 64])
def test_graph_replays_equal_the_eager_step(sw, batch):
    cfg = I.CONFIGS["decode_sweep"]
    L = I.make_layer(cfg)
    H, Iw, m, k = cfg.hidden, cfg.inter, cfg.n_experts, cfg.top_k
    g = np.random.default_rng([411, batch])
    i_s = 2 * Iw
    w13s = I.to_bf16_bits(0.02 * g.standard_normal((2 * i_s, H), dtype=np.float32))
    w2s = I.to_bf16_bits(0.02 * g.standard_normal((H, i_s), dtype=np.float32))
    gate = (0.05 * g.standard_normal(H)).astype(np.float32)
    xs = [I.make_x(cfg, tokens=batch, rep=500 + j) for j in range(3)]
    dx = [dev(x) for x in xs]
    wr, w13, w2 = dev(L["wr"]), dev(L["w13"]), dev(L["w2"])
    d13s, d2s, dgate = dev(w13s[None]), dev(w2s[None]), dev(gate)

    d = sw.dims(H, Iw, m, k)
    ids = torch.empty((batch, k), dtype=torch.int32, device="cuda")
    w = torch.empty((batch, k), dtype=torch.float32, device="cuda")
    gap = torch.empty(batch, dtype=torch.float32, device="cuda")
    plan = sw.alloc_plan(batch, m, k, "cuda")
    out = torch.empty((batch, H), dtype=torch.float32, device="cuda")
    rws = sw.workspace(sw.sw_moe_route_workspace_bytes(d, batch), "cuda")
    fws = sw.workspace(sw.sw_moe_forward_workspace_bytes(d, batch), "cuda")
    sws = sw.workspace(sw.sw_moe_shared_workspace_bytes(sw.dims(H, i_s, 1, 1), batch), "cuda")

    def step(x):
        sw.sw_moe_route_dispatch(x, wr, k, out=(ids, w, gap), plan=plan, ws=rws)
        sw.sw_moe_forward(x, w13, w2, w, plan, out=out, ws=fws)
        sw.sw_moe_shared_expert(x, d13s, d2s, dgate, out, ws=sws)

    eager = []
    for x in dx:
        step(x)
        torch.cuda.synchronize()
        eager.append((out.clone(), ids.clone()))

    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        step(dx[2])
    torch.cuda.synchronize()
    for rep in range(4):
        # eager work on the same buffers between the replays
        step(dx[rep % 2])
        torch.cuda.synchronize()
        assert torch.equal(out, eager[rep % 2][0])
        out.fill_(float("nan"))
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(out, eager[2][0]), f"replay {rep}"
        assert torch.equal(ids, eager[2][1]), f"replay {rep}"

    # and the step itself against the oracle (layer + shared expert)
    o_ids = host(eager[2][1])
    o_w = host(w)
    want = oracle.forward(xs[2], L["w13"], L["w2"], o_ids, o_w)
    want = oracle.shared_expert(xs[2], w13s, w2s, gate, out=want)
    compare_out(host(out), want)


# the one-call layer at batch 64, whose gate/up launch builds the plan: over
# the full pool (idle experts expected, no guess), over the 75% pool (the
# fully-active guess), and at 50% with the shared expert folded in 4 token
# groups
@pytest.mark.parametrize("pruning,n_shared", [(0.0, 0), (0.75, 0), (0.5, 2)])
def test_graph_replays_of_the_layer_call(sw, pruning, n_shared):
    cfg = I.CONFIGS["decode_sweep"]
    L = I.make_layer(cfg)
    H, Iw, k, T = cfg.hidden, cfg.inter, cfg.top_k, 64
    w13, w2, wr = L["w13"], L["w2"], L["wr"]
    if pruning:
        kept, _, _, w13, w2, wr, _ = oracle.prune_compact(L["importance"], cfg.n_keep(pruning), k,
                                                          w13=w13, w2=w2, wr=wr)
    m = w13.shape[0]
    groups = 4 if n_shared else 1
    if n_shared:
        g = np.random.default_rng(421)
        p13 = I.to_bf16_bits(0.02 * g.standard_normal((n_shared, 2 * Iw, H), dtype=np.float32))
        p2 = I.to_bf16_bits(0.02 * g.standard_normal((n_shared, H, Iw), dtype=np.float32))
        w13 = np.concatenate([w13] + [p13] * groups)
        w2 = np.concatenate([w2] + [p2] * groups)
        wr = np.concatenate([wr, (0.05 * g.standard_normal((1, H))).astype(np.float32)])
    dw13, dw2 = sw.sw_moe_pack_experts(dev(w13), dev(w2))
    dwr = dev(wr)
    xs = [dev(I.make_x(cfg, tokens=T, rep=600 + j)) for j in range(3)]
    kout, mp = k + n_shared, m + groups * n_shared
    ids = torch.empty((T, kout), dtype=torch.int32, device="cuda")
    w = torch.empty((T, kout), dtype=torch.float32, device="cuda")
    gap = torch.empty(T, dtype=torch.float32, device="cuda")
    plan = sw.alloc_plan(T, mp, kout, "cuda")
    out = torch.empty((T, H), dtype=torch.float32, device="cuda")
    ws = sw.workspace(sw.sw_moe_layer_workspace_bytes(sw.dims(H, Iw, m, k), T, n_shared, groups),
                      "cuda")
    d = sw.dims(H, Iw, mp, kout)
    assert sw.sw_moe_gate_up_builds_plan(d, T, sw.TILED)

    def step(x):
        sw.sw_moe_layer(x, dwr, k, dw13, dw2, layout=sw.TILED, n_shared=n_shared,
                        n_groups=groups, route_out=(ids, w, gap), plan=plan, out=out, ws=ws)

    eager = []
    for x in xs:
        step(x)
        torch.cuda.synchronize()
        eager.append((out.clone(), ids.clone(), plan.perm.clone(), plan.offsets.clone()))
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        step(xs[2])
    torch.cuda.synchronize()
    for rep in range(4):
        step(xs[rep % 2])
        torch.cuda.synchronize()
        assert torch.equal(out, eager[rep % 2][0])
        out.fill_(float("nan"))
        plan.perm.fill_(-7)
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(out, eager[2][0]), f"replay {rep}"
        assert torch.equal(ids, eager[2][1]), f"replay {rep}"
        assert torch.equal(plan.perm, eager[2][2]), f"replay {rep}"
        assert torch.equal(plan.offsets, eager[2][3]), f"replay {rep}"
