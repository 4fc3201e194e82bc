"""GPU checks of the device-drawn expert pools and of the skewed 40-layer
stack: the device stream equals the host stream bit for bit, and checked
layers of the stack match the oracle (routing and the forward over all
tokens, every active expert redrawn on the host)."""
from concurrent.futures import ThreadPoolExecutor

import numpy as np
import pytest

import oracle
from paper_2609_34117_amd import inputs as I
from parity import compare_out, compare_routing, oracle_forward_rows, oracle_threads

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module")
def libs():
    assert torch.cuda.is_available(), "GPU tests need a device"
    from paper_2609_34117_amd import gen, slimwise

    return slimwise, gen


def host(t):
    a = t.cpu().numpy()
    return a.view(np.uint16) if a.dtype == np.int16 else a


def dev(a):
    a = np.ascontiguousarray(a)
    return torch.from_numpy(a.view(np.int16) if a.dtype == np.uint16 else a).cuda()


@pytest.mark.parametrize("n,start,std,key", [
    (1000, 0, 0.02, (4, 0, 2)),
    (12345, 2 ** 33 + 7, 0.02, (4, 39, 3)),
    (4096 + 5, 77, 1.0, (100, 1, 2)),
])
def test_device_draws_equal_host_draws(libs, n, start, std, key):
    _, gen = libs
    k = I.philox_key(*key)
    want = I.philox_normal_bf16(k, start, n, std)
    buf = torch.empty(n + 1, dtype=torch.int16, device="cuda")
    # aligned destination (16-byte stores) and one shifted by an element (tail path)
    for off in (0, 1):
        d = buf[off:off + n]
        gen.philox_normal_bf16(d, k, start, std)
        torch.cuda.synchronize()
        np.testing.assert_array_equal(host(d), want)


def _draw_experts(cfg, layer, experts, cache):
    """Host draws of the experts' W13 and W2 (the same bits the device drew),
    in threads, cached per layer."""
    todo = [int(e) for e in experts if int(e) not in cache]

    def one(e):
        return e, (I.philox_expert_slice(cfg, layer, "w13", [e])[0],
                   I.philox_expert_slice(cfg, layer, "w2", [e])[0])

    with ThreadPoolExecutor(oracle_threads()) as ex:
        for e, w in ex.map(one, todo):
            cache[e] = w


@pytest.mark.parametrize("layer", [0, 19, 39])
def test_skewed_stack_layer_parity(libs, layer):
    sw, gen = libs
    cfg = I.CONFIGS["skewed_stack"]
    H, Iw, m, k, T = cfg.hidden, cfg.inter, cfg.n_experts, cfg.top_k, cfg.tokens
    w13 = torch.empty((m, 2 * Iw, H), dtype=torch.int16, device="cuda")
    w2 = torch.empty((m, H, Iw), dtype=torch.int16, device="cuda")
    gen.philox_normal_bf16(w13, I.philox_key(cfg.config_id, layer, I.W13), 0, cfg.w_std)
    gen.philox_normal_bf16(w2, I.philox_key(cfg.config_id, layer, I.W2), 0, cfg.w_std)
    L = I.make_layer(cfg, layer=layer, experts=False)
    n_keep = cfg.n_keep(0.5)
    _, _, mask, *_ = oracle.prune_compact(L["importance"], n_keep, k)
    cache = {}
    for keep in (None, mask):
        g = sw.moe_layer(dev(L["x"]), dev(L["wr"]), w13, w2, k,
                         keep_mask=None if keep is None else dev(keep), bias=dev(L["bias"]))
        g_ids, g_w = host(g["topk_ids"]), host(g["topk_w"])
        o_ids, o_w, o_gap, o_z = oracle.route(L["x"], L["wr"], k, keep_mask=keep, bias=L["bias"],
                                              want_logits=True)
        r = compare_routing(g_ids, g_w, o_ids, o_w, o_z, keep, k, g_gap=host(g["gap"]), o_gap=o_gap,
                            what=f"stack layer {layer} {'masked' if keep is not None else 'full'}")
        counts, offsets, perm, active, n_active = oracle.dispatch(g_ids, m)
        np.testing.assert_array_equal(host(g["plan"].counts), counts)
        np.testing.assert_array_equal(host(g["plan"].offsets), offsets)
        np.testing.assert_array_equal(host(g["plan"].perm)[: g_ids.size], perm)
        assert int(g["plan"].n_active.item()) == n_active
        # forward of every token, its experts drawn on the host
        _draw_experts(cfg, layer, active, cache)
        ow13 = np.stack([cache[int(e)][0] for e in active])
        ow2 = np.stack([cache[int(e)][1] for e in active])
        local = np.searchsorted(active, g_ids).astype(np.int32)
        o_out = oracle_forward_rows(oracle.forward, L["x"], ow13, ow2, local, g_w)
        err, rel = compare_out(host(g["out"]), o_out)
        frac = n_active / (m if keep is None else n_keep)
        print(f"layer {layer} {'masked' if keep is not None else 'full'}: n_active={n_active} "
              f"({frac:.2%} of the pool) multi-pass experts={(counts > 32).sum()} "
              f"max pairs/expert={counts.max()} near_ties={r['near_ties']} "
              f"max|err|={err:.3g} rel={rel:.3g}")
