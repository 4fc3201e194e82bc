"""The allocation-free forward (sw_moe_forward_no_alloc, the library's static
device scratch) against sw_moe_forward with a caller workspace: bit for bit
on two calls in a row, the second smaller, and rejected beyond its scratch."""
import numpy as np
import pytest

import oracle
from paper_2609_34117_amd import inputs as I
from parity import compare_out, oracle_forward_rows

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


def _dev(a):
    a = np.ascontiguousarray(a)
    return torch.from_numpy(a.view(np.int16) if a.dtype == np.uint16 else a).cuda()


@pytest.fixture(scope="module")
def sw():
    assert torch.cuda.is_available(), "GPU tests need a device"
    from paper_2609_34117_amd import slimwise

    return slimwise


@pytest.mark.parametrize("tiled", [False, True])
def test_no_alloc_forward_equals_the_workspace_forward(sw, tiled):
    cfg = I.CONFIGS["decode_b64"]
    L = I.make_layer(cfg)
    w13, w2, wr = _dev(L["w13"]), _dev(L["w2"]), _dev(L["wr"])
    layout = sw.ROW_MAJOR
    if tiled:
        w13, w2 = sw.sw_moe_pack_experts(w13, w2)
        layout = sw.TILED
    # two calls in a row on the same scratch, the second with fewer tokens
    # (batch 64 on the wave kernels, then 5 tokens on the split-K kernels),
    # then the first again
    for tokens, rep in ((64, 0), (5, 1), (64, 0)):
        x_np = I.make_x(cfg, tokens=tokens, rep=rep)
        x = _dev(x_np)
        ids, w, gap, plan = sw.sw_moe_route_dispatch(x, wr, cfg.top_k)
        want = sw.sw_moe_forward(x, w13, w2, w, plan, layout=layout)
        out = torch.full((tokens, cfg.hidden), float("nan"), device="cuda")
        got = sw.sw_moe_forward_no_alloc(x, w13, w2, w, plan, layout=layout, out=out)
        torch.cuda.synchronize()
        assert got.data_ptr() == out.data_ptr()
        assert torch.equal(got, want), (tokens, tiled)
        o_out = oracle_forward_rows(oracle.forward, x_np, L["w13"], L["w2"], ids.cpu().numpy(),
                                    w.cpu().numpy())
        compare_out(got.cpu().numpy(), o_out)


def test_no_alloc_forward_rejects_calls_beyond_its_scratch(sw):
    cfg = I.CONFIGS["decode_sweep"]
    d = sw.dims(cfg.hidden, cfg.inter, cfg.n_experts, cfg.top_k)
    # (4I + 4H) bytes a pair: 409 tokens at top-8 fit, 410 do not
    assert sw.sw_moe_forward_workspace_bytes(d, 409) <= sw.NO_ALLOC_SCRATCH_BYTES
    assert sw.sw_moe_forward_workspace_bytes(d, 410) > sw.NO_ALLOC_SCRATCH_BYTES
    T = 410
    x = torch.zeros((T, cfg.hidden), dtype=torch.int16, device="cuda")
    w13 = torch.zeros((cfg.n_experts, 2 * cfg.inter, cfg.hidden), dtype=torch.int16, device="cuda")
    w2 = torch.zeros((cfg.n_experts, cfg.hidden, cfg.inter), dtype=torch.int16, device="cuda")
    w = torch.zeros((T, cfg.top_k), device="cuda")
    plan = sw.alloc_plan(T, cfg.n_experts, cfg.top_k, "cuda")
    with pytest.raises(sw.SlimwiseError, match="SW_ERR_WORKSPACE"):
        sw.sw_moe_forward_no_alloc(x, w13, w2, w, plan)
