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
