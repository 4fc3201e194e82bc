"""The benchmark's host-side legs on the CPU: the oracle baseline with its
host details and the routing check of the bench batches (no GPU needed)."""
import os
import sys

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import bench  # noqa: E402
import oracle  # noqa: E402
from paper_2609_34117_amd import inputs as I  # noqa: E402


def test_cpu_baseline_reports_host_details_and_checks_routing():
    cfg = I.CONFIGS["tiny"]
    L = I.make_layer(cfg)
    _, _, _, _, _, wr, _ = oracle.prune_compact(L["importance"], cfg.n_keep(0.5), cfg.top_k,
                                                w13=L["w13"], w2=L["w2"], wr=L["wr"])
    ids = [oracle.route(I.make_x(cfg, tokens=8, rep=r), wr, cfg.top_k)[0] for r in range(3)]
    out = bench.cpu_baseline(cfg, L, 0.5, 0.5, 8, gpu_ids=ids)
    assert out["kind"] == "oracle" and out["cores"] == 1 and out["value"] > 0
    for key in ("nproc", "cpu_model", "compiler", "cflags"):
        assert out[key]
    r = out["bench_batches_routing"]
    assert r["tokens"] == 24 and r["topk_sets_differing_without_a_tie"] == 0
    # a planted routing difference is counted
    bad = [i.copy() for i in ids]
    bad[0][0] = np.roll(bad[0][0], 1) if cfg.top_k > 1 else bad[0][0]
    bad[1][2, 0] = (bad[1][2, 0] + 1) % cfg.n_keep(0.5)
    bad[1][2, 1] = (bad[1][2, 1] + 1) % cfg.n_keep(0.5)
    r2 = bench.routing_check(cfg, wr, [I.make_x(cfg, tokens=8, rep=k) for k in range(3)], bad)
    assert r2["topk_sets_differing_without_a_tie"] >= 1


def test_paper_context_is_quoted():
    assert bench.PAPER_CONTEXT["decode_gain_50pct_pd_disaggregated"] == "1.40-1.81x"
