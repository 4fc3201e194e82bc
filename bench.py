"""Benchmark of the batched-decode MoE layer (route -> dispatch -> expert FFNs
-> combine) on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME]

One step = one pass of the whole layer (route + dispatch in one call, then
gate_up, down, combine) over one batch of synthetic tokens, with every input
already resident in HBM.  Batches rotate over pre-generated token sets and
each pool over 4 copies at distinct addresses, so the 256 MB Infinity Cache
cannot serve expert bytes from one step to the next.

Workloads (the default line is decode_b64):
  decode_b64    H 2048, 128 experts, top-8, I 768, batch 64: the 50% pruned
                decoder (64 kept experts, compacted pool) and the unpruned
                pool, for the speedup.
  decode_sweep  H 2048, 256 experts, top-8, I 512: batches 1..256 at 0, 25,
                50 and 75% pruning (unique expert bytes per step next to
                Eq. 1's expectation); `value` is batch 64 at 50%.
  prefill       the same layer shape, 4096 tokens through the full pool.
  decode_shared the decode sweep's layer at batch 64 with the shared expert of
                the distilled pruned decoder (width 2 I, sigmoid gate), 0 and
                50% pruning, each with and without the shared expert.
  colocated     one resident full pool (the decode sweep's layer): an
                unmasked 4096-token prefill forward, and batch-64 decode with
                the 50% router mask, next to decode on the compacted pool
                (the mask's cost).
  skewed_stack  40 such layers at batch 256 with a Zipf(1.1) router bias per
                layer (60 GiB of experts, drawn on the device), the full
                stack and the 50% pruned one (top 128 experts by
                popularity); one step = the 40 layers back to back.

Prints one JSON line.  `roofline` describes the dominant kernel (gate_up,
which streams 2/3 of each active expert's bytes): algorithmic bytes per
launch (the unique expert bytes n_active * 2 * I * H * 2) over its mean
launch duration, measured with HIP events around back-to-back launches on the
launch stream (for prefill, also its flops against the bf16 MFMA peak).
`traffic` is the HBM byte count of one such launch from the FETCH_SIZE /
WRITE_SIZE hardware counters, scaled by what those counters read for plain
device copies of known size; it is reported only for the workload and kernel
sources the counters were taken on.  `cpu_baseline` is the single-threaded C
oracle timed on a bounded sample of the same workload.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

from paper_2609_34117_amd import inputs as I  # noqa: E402

METRIC = "MoE decode-layer tokens/s + achieved HBM GB/s, batch 64, 0% vs 50% pruned"
HBM_PEAK_GBS = 8000.0
MFMA_BF16_PEAK_TFLOPS = 2500.0
N_X = 16
N_COPIES = 4
# The paper's own decode-throughput gains of the pruned decoder (Section 4.3,
# Fig. 4): end-to-end serving ratios on two A100-80GB GPUs under vLLM, at a
# fixed per-user latency target, including larger batches from the freed
# expert memory.  Context for the layer-level speedup measured here, not a
# target.
PAPER_CONTEXT = {
    "decode_gain_50pct_pd_disaggregated": "1.40-1.81x",
    "decode_gain_75pct_pd_disaggregated": "1.65-2.39x",
    "decode_gain_50pct_pd_colocated": "1.36-1.72x",
    "hardware": "2x A100-80GB, vLLM, end to end, 256-expert top-8 40-layer model",
    "where": "Section 4.3, Fig. 4",
}

# HBM traffic of one gate_up launch on the default workload (batch 64, 50%
# pruned, tiled pool), from two rocprofv3 --pmc passes of
# `bench.py --no-cpu-baseline --steps 20 --warmup 5` (summary in
# profiles/gate_up_wave_decode_b64_hbm_traffic.md): FETCH_SIZE 197812.39 KiB x
# 1.99982 (the ratio of bytes copied to FETCH_SIZE over 12 plain device copies
# of 192-768 MiB) + WRITE_SIZE 1570.74 KiB x 1.0 (WRITE_SIZE of the copies is
# exact).  The figure holds while the gate/up kernel's sources hash as below.
KERNEL_SOURCES = ("paper_2609_34117_amd/csrc/expert_stream.hip",
                  "paper_2609_34117_amd/csrc/sw_device.h",
                  "paper_2609_34117_amd/csrc/dispatch_block.h")
GATE_UP_TRAFFIC = dict(sources_sha256="fde0ac45004e4df8a0f3889d303304bd170f73ac8af53e0be8cb7b9e4dc5deac",
                       workload=("decode_b64", 64, 0.5, "tiled"),
                       bytes_per_launch=int(round((197812.39 * 1.99982 + 1570.74) * 1024)))


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", default="decode_b64",
                    choices=["decode_b64", "decode_sweep", "prefill", "skewed_stack",
                             "decode_shared", "colocated"])
    ap.add_argument("--sweep-steps", type=int, default=50,
                    help="timed steps per (batch, pruning) point of decode_sweep")
    ap.add_argument("--batch", type=int, default=None)
    ap.add_argument("--pruning", type=float, default=0.5)
    ap.add_argument("--layout", default="tiled", choices=["tiled", "row_major"])
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=10.0)
    return ap.parse_args()


class Pool:
    """One expert pool (full or compacted) resident on the device, N_COPIES times."""

    def __init__(self, w13, w2, wr, layout, bias=None, shared=None, n_shared=0, n_groups=1):
        self.w13 = [w13] + [w13.clone() for _ in range(N_COPIES - 1)]
        self.w2 = [w2] + [w2.clone() for _ in range(N_COPIES - 1)]
        self.wr = wr
        self.bias = bias
        self.layout = layout
        # n_shared > 0: the shared expert folded into the plan -- n_groups
        # copies of its parts follow the routed experts in w13 / w2 and its
        # gate row follows the router rows in wr
        self.n_shared = n_shared
        self.n_groups = n_groups
        self.m = wr.shape[0] - (1 if n_shared else 0)  # routed experts
        self.shared = shared  # (w13_s, w2_s, gate_w) run by the separate call, or None
        self.keep_mask = None  # router mask over this pool (colocated decode), or None


class Runner:
    """Preallocated buffers for one (pool, batch) configuration."""

    def __init__(self, sw, torch, pool: Pool, cfg, T, dev):
        self.sw, self.torch, self.pool, self.cfg, self.T = sw, torch, pool, cfg, T
        k, H, Iw = cfg.top_k, cfg.hidden, cfg.inter
        S = pool.n_shared
        # slots a token, experts of the plan
        self.kout, self.m_plan = k + S, pool.m + pool.n_groups * S
        self.ids = torch.empty((T, self.kout), dtype=torch.int32, device=dev)
        self.w = torch.empty((T, self.kout), dtype=torch.float32, device=dev)
        self.gap = torch.empty(T, dtype=torch.float32, device=dev)
        self.plan = sw.alloc_plan(T, self.m_plan, self.kout, dev)
        self.out = torch.empty((T, H), dtype=torch.float32, device=dev)
        d = sw.dims(H, Iw, pool.m, k)
        rbytes = (sw.sw_moe_route_shared_workspace_bytes(d, T, S, pool.n_groups) if S else
                  sw.sw_moe_route_workspace_bytes(d, T))
        self.rws = sw.workspace(rbytes, dev)
        fd = sw.dims(H, Iw, self.m_plan, self.kout)
        self.fws = sw.workspace(sw.sw_moe_forward_workspace_bytes(fd, T), dev)
        self.lws = sw.workspace(sw.sw_moe_layer_workspace_bytes(d, T, S, pool.n_groups), dev)
        self.sws = None
        if pool.shared is not None:
            ds = sw.dims(H, pool.shared[1].shape[-1], 1, 1)
            self.sws = sw.workspace(sw.sw_moe_shared_workspace_bytes(ds, T), dev)

    def route(self, x, plan):
        sw, p = self.sw, self.pool
        if p.n_shared:
            sw.sw_moe_route_dispatch_shared(x, p.wr, self.cfg.top_k, p.n_shared,
                                            n_groups=p.n_groups, bias=p.bias,
                                            keep_mask=p.keep_mask,
                                            out=(self.ids, self.w, self.gap), plan=plan,
                                            ws=self.rws)
        else:
            sw.sw_moe_route_dispatch(x, p.wr, self.cfg.top_k, bias=p.bias, keep_mask=p.keep_mask,
                                     out=(self.ids, self.w, self.gap), plan=plan, ws=self.rws)

    def layer(self, x, c, phase=None, bufs=None):
        """sw_moe_layer on batch `x` and pool copy `c` (one phase of it
        with `phase`), into this runner's buffers or `bufs` (a tuple of
        ids, w, gap, plan, out, workspace)."""
        sw, p = self.sw, self.pool
        ids, w, gap, plan, out, ws = bufs or (self.ids, self.w, self.gap, self.plan, self.out,
                                             self.lws)
        sw.sw_moe_layer(x, p.wr, self.cfg.top_k, p.w13[c], p.w2[c], layout=p.layout,
                        n_shared=p.n_shared, n_groups=p.n_groups, bias=p.bias,
                        keep_mask=p.keep_mask, route_out=(ids, w, gap), plan=plan, out=out,
                        ws=ws, phase=phase)

    def buffers(self):
        """A set of layer buffers of its own (ids, w, gap, plan, out, workspace)."""
        t, dev = self.torch, self.out.device
        return (t.empty_like(self.ids), t.empty_like(self.w), t.empty_like(self.gap),
                self.sw.alloc_plan(self.T, self.m_plan, self.kout, dev), t.empty_like(self.out),
                t.empty_like(self.lws))

    def step(self, x, c, ev=None):
        """One layer step: one sw_moe_layer call (with a separate shared
        expert, route + dispatch, the forward and the shared expert's call).
        With ev, the layer's four phases with events between them: the
        routing, then gate/up, down and combine."""
        sw, p = self.sw, self.pool
        if p.shared is None:
            if ev is None:
                self.layer(x, c)
                return
            self.layer(x, c, phase=0)
            for i in range(3):
                ev[i].record()
                self.layer(x, c, phase=i + 1)
            ev[3].record()
            return
        if ev is None:
            self.route(x, self.plan)
            sw.sw_moe_forward(x, p.w13[c], p.w2[c], self.w, self.plan, layout=p.layout,
                              out=self.out, ws=self.fws)
            sw.sw_moe_shared_expert(x, *p.shared, self.out, layout=p.layout, ws=self.sws)
            return
        self.route(x, self.plan)
        ev[0].record()
        sw.sw_moe_forward_gate_up(x, p.w13[c], self.kout, self.plan, self.fws, layout=p.layout)
        ev[1].record()
        sw.sw_moe_forward_down(self.T, p.w2[c], self.kout, self.plan, self.fws, layout=p.layout)
        ev[2].record()
        sw.sw_moe_forward_combine(self.w, self.cfg.hidden, self.cfg.inter, self.m_plan, self.plan,
                                  self.out, self.fws)
        ev[3].record()


def time_runner(torch, r: Runner, xs, steps, warmup):
    for s in range(warmup):
        r.step(xs[s % len(xs)], s % N_COPIES)
    torch.cuda.synchronize()
    # (a) whole steps, nothing recorded between kernels
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for s in range(steps):
        r.step(xs[s % len(xs)], s % N_COPIES)
    e1.record()
    torch.cuda.synchronize()
    t_step = e0.elapsed_time(e1) / 1e3 / steps
    # (b) the same steps with events around each forward phase
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(steps)]
    for s in range(steps):
        r.step(xs[s % len(xs)], s % N_COPIES, ev=evs[s])
    torch.cuda.synchronize()
    phase = np.array([[ev[i].elapsed_time(ev[i + 1]) / 1e3 for i in range(3)] for ev in evs])
    # n_active of every rotated batch (deterministic given the batch)
    n_act = []
    for j in range(len(xs)):
        r.step(xs[j], 0)
        n_act.append(int(r.plan.n_active.item()))
    n_act_steps = np.array([n_act[s % len(xs)] for s in range(steps)], float)
    kern = time_kernels(torch, r, xs, steps)
    kern["graph_step"], kern["graph_same"] = time_graph(torch, r, xs, max(4, steps // len(xs)))
    return t_step, phase, n_act_steps, n_act, kern


def time_graph(torch, r: Runner, xs, reps):
    """Mean step time with the host out of the loop: len(xs) steps (rotating
    the batches and the pool copies) captured once in a HIP graph and
    replayed `reps` times.  Returns (seconds per step, whether the graph's
    last output equals the eager step's bit for bit)."""
    G = len(xs)
    r.step(xs[G - 1], (G - 1) % N_COPIES)
    torch.cuda.synchronize()
    ref = r.out.clone()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        for j in range(G):
            r.step(xs[j], j % N_COPIES)
    torch.cuda.synchronize()
    same = True
    for _ in range(2):
        r.out.zero_()
        g.replay()
        torch.cuda.synchronize()
        same = same and bool(torch.equal(r.out, ref))
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        g.replay()
    e1.record()
    torch.cuda.synchronize()
    del g
    return e0.elapsed_time(e1) / 1e3 / (reps * G), same


def time_kernels(torch, r: Runner, xs, steps):
    """Mean launch duration of gate_up and of down: `steps` launches of one
    kernel back to back between two HIP events on the launch stream, rotating
    the batches (each with layer buffers of its own, routed once) and the
    pool copies.  Each is the step's own launch: phase 1 and phase 2 of
    sw_moe_layer (on decode batches the gate/up launch selects the experts
    and builds the plan on the way).  (The small kernels are shorter than a
    host call, so their durations come from the kernel trace instead.)"""
    sw, p, k = r.sw, r.pool, r.kout
    if p.shared is None:
        bufs = [r.buffers() for _ in xs]
        for j, x in enumerate(xs):
            r.layer(x, 0, phase=0, bufs=bufs[j])
            r.layer(x, 0, phase=1, bufs=bufs[j])
    else:
        plans = []
        for x in xs:
            plan = sw.alloc_plan(r.T, r.m_plan, r.kout, x.device)
            r.route(x, plan)
            plans.append(plan)
    torch.cuda.synchronize()
    out = {}

    def launch(name, s):
        j, c = s % len(xs), s % N_COPIES
        if p.shared is None:
            r.layer(xs[j], c, phase=1 if name == "gate_up" else 2, bufs=bufs[j])
        elif name == "down":
            sw.sw_moe_forward_down(r.T, p.w2[c], k, plans[j], r.fws, layout=p.layout)
        else:
            sw.sw_moe_forward_gate_up(xs[j], p.w13[c], k, plans[j], r.fws, layout=p.layout)

    for name in ("gate_up", "down"):
        for s in range(4):
            launch(name, s)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for s in range(steps):
            launch(name, s)
        e1.record()
        torch.cuda.synchronize()
        out[name] = e0.elapsed_time(e1) / 1e3 / steps
    return out


def sources_sha256():
    h = hashlib.sha256()
    for rel in KERNEL_SOURCES:
        with open(os.path.join(ROOT, rel), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def host_details():
    """The GPU machine's host as the oracle ran on it: logical CPUs, CPU model,
    and how the oracle was compiled."""
    import subprocess

    import oracle

    model = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    try:
        cc = subprocess.run(["gcc", "--version"], capture_output=True, text=True).stdout.splitlines()[0]
    except (OSError, IndexError):
        cc = "gcc"
    try:
        usable = len(os.sched_getaffinity(0))
    except AttributeError:
        usable = os.cpu_count()
    return dict(nproc=os.cpu_count(), usable_cpus=usable, cpu_model=model, compiler=cc,
                cflags=" ".join(oracle.CFLAGS))


def routing_check(cfg, wr, xs_np, gpu_ids, keep_mask=None, bias=None):
    """Near ties of the benchmark's own batches (tokens whose oracle gap
    z_(k) - z_(k+1) is below 1e-5) and the tokens whose GPU top-k set differs
    from the oracle's without such a tie (expected 0)."""
    import oracle

    near = differ = tokens = 0
    for x, g in zip(xs_np, gpu_ids):
        o_ids, _, o_gap = oracle.route(x, wr, cfg.top_k, keep_mask=keep_mask, bias=bias)
        tie = o_gap < 1e-5
        same = np.all(np.sort(o_ids, axis=1) == np.sort(g, axis=1), axis=1)
        near += int(tie.sum())
        differ += int((~same & ~tie).sum())
        tokens += x.shape[0]
    return dict(tokens=tokens, near_ties=near, topk_sets_differing_without_a_tie=differ)


def cpu_baseline(cfg, L, pruning, seconds, tokens, gpu_ids=None):
    """The C oracle (single-threaded) on the same layer: whole batches of
    `tokens` tokens through route + dispatch + forward until `seconds` have
    passed.  With `gpu_ids` (the GPU's top-k ids of the benchmark's batches on
    the pruned pool), also the routing check of those batches."""
    import oracle

    k = cfg.top_k
    if pruning > 0:
        n_keep = cfg.n_keep(pruning)
        _, _, _, w13, w2, wr, _ = oracle.prune_compact(L["importance"], n_keep, k, w13=L["w13"],
                                                       w2=L["w2"], wr=L["wr"])
    else:
        w13, w2, wr = L["w13"], L["w2"], L["wr"]
    done, elapsed, batches = 0, 0.0, 0
    while elapsed < seconds and batches < N_X:
        x = I.make_x(cfg, tokens=tokens, rep=batches)
        t0 = time.perf_counter()
        oracle.layer(x, wr, w13, w2, k)
        elapsed += time.perf_counter() - t0
        done += x.shape[0]
        batches += 1
    out = dict(value=round(done / elapsed, 2), unit="tokens/s", cores=1, kind="oracle",
               sample=f"{batches} batch(es) of {tokens} tokens through the {int(pruning * 100)}% "
                      f"pruned {cfg.name} layer (route+dispatch+forward), {elapsed:.1f} s, 1 thread")
    out.update(host_details())
    if gpu_ids is not None:
        xs_np = [I.make_x(cfg, tokens=tokens, rep=r) for r in range(len(gpu_ids))]
        out["bench_batches_routing"] = routing_check(cfg, wr, xs_np, gpu_ids)
    return out


def up(torch, dev, a):
    a = np.ascontiguousarray(a)
    return torch.from_numpy(a.view(np.int16) if a.dtype == np.uint16 else a).to(dev)


def build_pools(sw, torch, cfg, L, prunings, layout, dev):
    """pruning -> Pool: the full pool for 0, compacted pools otherwise (the
    tiled layout is packed once, then the tiled pool is compacted)."""
    w13, w2, wr, imp = (up(torch, dev, L[k]) for k in ("w13", "w2", "wr", "importance"))
    if layout == sw.TILED:
        w13, w2 = sw.sw_moe_pack_experts(w13, w2)
    pools = {}
    for p in prunings:
        if p == 0:
            pools[p] = Pool(w13, w2, wr, layout)
        else:
            c = sw.sw_moe_prune_compact(imp, cfg.n_keep(p), cfg.top_k, w13=w13, w2=w2, wr=wr)
            pools[p] = Pool(c["w13"], c["w2"], c["wr"], layout)
    torch.cuda.synchronize()
    return pools


def measure(sw, torch, pool, cfg, T, xs, steps, warmup, dev):
    """Times one pool at batch T; returns the summary of its steps."""
    r = Runner(sw, torch, pool, cfg, T, dev)
    t_step, phase, nact_steps, _, kern = time_runner(torch, r, xs, steps, warmup)
    H, Iw, k, m = cfg.hidden, cfg.inter, cfg.top_k, pool.m
    t_gu, t_dn, t_cb = phase.mean(axis=0)
    fwd = phase.sum(axis=1)
    U = nact_steps * 3 * H * Iw * 2
    n_mean = float(nact_steps.mean())
    if not kern["graph_same"]:
        raise RuntimeError("graph replay differs from the eager step")
    return dict(t_step_us=t_step * 1e6, tokens_per_s=T / t_step,
                t_step_graph_us=kern["graph_step"] * 1e6, tokens_per_s_graph=T / kern["graph_step"],
                t_gate_up_us=t_gu * 1e6, t_down_us=t_dn * 1e6, t_combine_us=t_cb * 1e6,
                n_active_mean=n_mean,
                eq1_expected=float(m * (1 - (1 - k / m) ** T)) + pool.n_shared * pool.n_groups,
                unique_MiB_per_step=float(U.mean() / 2 ** 20),
                gate_up_launch_us=kern["gate_up"] * 1e6, down_launch_us=kern["down"] * 1e6,
                gate_up_GBps=n_mean * 2 * H * Iw * 2 / kern["gate_up"] / 1e9,
                down_GBps=n_mean * H * Iw * 2 / kern["down"] / 1e9,
                fwd_GBps=float(U.sum() / fwd.sum() / 1e9),
                layer_GBps=float(U.mean() / t_step / 1e9))


def rounded(d):
    return {k: round(v, 3) if isinstance(v, float) else v for k, v in d.items()}


def base_line(args, cfg, T, value, t_step_us, steps):
    return {
        "metric": METRIC,
        "value": round(value, 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": steps,
        "warmup": args.warmup,
        "ms_per_step": round(t_step_us / 1e3, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded N(0,0.02) bf16 experts, N(0,1) tokens, uniform importance)",
    }


def hbm_roofline(cfg, T, pruning, layout, s, kernel="gate_up_wave_kernel"):
    """The gate_up roofline object of one measured point."""
    achieved = s["gate_up_GBps"]
    traffic = None
    if (GATE_UP_TRAFFIC["sources_sha256"] == sources_sha256()
            and GATE_UP_TRAFFIC["workload"] == (cfg.name, T, pruning, layout)):
        traffic = GATE_UP_TRAFFIC["bytes_per_launch"]
    return {
        "bound": "hbm", "kernel": kernel,
        "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
        "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": traffic,
        "traffic_unit": "bytes/launch",
        "algorithmic_bytes_per_launch": int(round(s["n_active_mean"] * 2 * cfg.hidden * cfg.inter * 2)),
        "launch_us": round(s["gate_up_launch_us"], 3),
    }


def run_decode_b64(args, sw, torch, dev):
    cfg = I.CONFIGS["decode_b64"]
    T = args.batch or cfg.tokens
    L = I.make_layer(cfg)
    layout = sw.TILED if args.layout == "tiled" else sw.ROW_MAJOR
    pools = build_pools(sw, torch, cfg, L, (args.pruning, 0.0), layout, dev)
    xs = [up(torch, dev, I.make_x(cfg, tokens=T, rep=r)) for r in range(N_X)]
    sp = measure(sw, torch, pools[args.pruning], cfg, T, xs, args.steps, args.warmup, dev)
    sf = measure(sw, torch, pools[0.0], cfg, T, xs, args.steps, args.warmup, dev)
    n_keep = cfg.n_keep(args.pruning)
    line = base_line(args, cfg, T, sp["tokens_per_s"], sp["t_step_us"], args.steps)
    line["config"] = {
        "workload": f"{cfg.name}: decode MoE layer H {cfg.hidden}, {cfg.n_experts} experts, "
                    f"top-{cfg.top_k}, I {cfg.inter}, batch {T}, {int(args.pruning * 100)}% pruned "
                    f"({n_keep} kept, compacted)",
        "hidden": cfg.hidden, "n_experts": cfg.n_experts, "n_kept": n_keep, "top_k": cfg.top_k,
        "inter": cfg.inter, "batch": T, "pruning": args.pruning, "weight_layout": args.layout,
        "parallelism": "none (1 GPU)",
    }
    line["roofline"] = hbm_roofline(cfg, T, args.pruning, args.layout, sp)
    line["detail"] = {
        "pruned": rounded(sp), "full": rounded(sf),
        "speedup_pruned_vs_full": round(sf["t_step_us"] / sp["t_step_us"], 3),
        "ideal_byte_ratio": round(sf["n_active_mean"] / sp["n_active_mean"], 3),
        "paper_context": PAPER_CONTEXT,
    }
    if not args.no_cpu_baseline:
        gpu_ids = [sw.sw_moe_route(x, pools[args.pruning].wr, cfg.top_k)[0].cpu().numpy()
                   for x in xs]
        line["cpu_baseline"] = cpu_baseline(cfg, L, args.pruning, args.cpu_seconds, T,
                                            gpu_ids=gpu_ids)
        line["detail"]["near_ties"] = line["cpu_baseline"]["bench_batches_routing"]["near_ties"]
    return line


def run_decode_sweep(args, sw, torch, dev):
    cfg = I.CONFIGS["decode_sweep"]
    L = I.make_layer(cfg)
    layout = sw.TILED if args.layout == "tiled" else sw.ROW_MAJOR
    prunings = (0.0, 0.25, 0.5, 0.75)
    batches = I.SWEEP_BATCHES
    head_at = (64, 0.5)
    if args.batch is not None:  # one batch size, at 0% and at --pruning only
        batches, head_at = (args.batch,), (args.batch, args.pruning)
        prunings = (0.0,) if args.pruning == 0.0 else (0.0, args.pruning)
    pools = build_pools(sw, torch, cfg, L, prunings, layout, dev)
    rows, at = [], {}
    for T in batches:
        xs = [up(torch, dev, I.make_x(cfg, tokens=T, rep=r)) for r in range(N_X)]
        for p in prunings:
            s = measure(sw, torch, pools[p], cfg, T, xs, args.sweep_steps, args.warmup, dev)
            at[(T, p)] = s
            rows.append(dict(batch=T, pruning=p, m_pool=pools[p].m, **rounded(s)))
            print(f"# batch {T:3d} pruning {p:.2f}: {s['tokens_per_s']:.0f} tokens/s, "
                  f"step {s['t_step_us']:.1f} us (graph {s['t_step_graph_us']:.1f} us), n_active {s['n_active_mean']:.1f} "
                  f"(Eq. 1 {s['eq1_expected']:.1f}), fwd {s['fwd_GBps']:.0f} GB/s",
                  file=sys.stderr, flush=True)
    head = at[head_at]
    line = base_line(args, cfg, head_at[0], head["tokens_per_s"], head["t_step_us"],
                     args.sweep_steps)
    line["config"] = {
        "workload": f"{cfg.name}: decode MoE layer H {cfg.hidden}, {cfg.n_experts} experts, "
                    f"top-{cfg.top_k}, I {cfg.inter}; value at batch {head_at[0]}, "
                    f"{int(head_at[1] * 100)}% pruned ({cfg.n_keep(head_at[1])} kept, compacted); "
                    f"batches {list(batches)} x pruning {list(prunings)} in detail",
        "hidden": cfg.hidden, "n_experts": cfg.n_experts, "top_k": cfg.top_k, "inter": cfg.inter,
        "batch": head_at[0], "pruning": head_at[1], "weight_layout": args.layout,
        "parallelism": "none (1 GPU)",
    }
    line["roofline"] = hbm_roofline(cfg, head_at[0], head_at[1], args.layout, head)
    b = head_at[0]
    line["detail"] = {
        "sweep": rows,
        f"speedup_vs_full_at_b{b}": {
            str(p): round(at[(b, 0.0)]["t_step_us"] / at[(b, p)]["t_step_us"], 3) for p in prunings},
    }
    if not args.no_cpu_baseline:
        line["cpu_baseline"] = cpu_baseline(cfg, L, head_at[1], args.cpu_seconds, head_at[0])
    return line


def run_prefill(args, sw, torch, dev):
    cfg = I.CONFIGS["prefill"]
    T = args.batch or cfg.tokens
    L = I.make_layer(cfg)
    layout = sw.TILED if args.layout == "tiled" else sw.ROW_MAJOR
    pools = build_pools(sw, torch, cfg, L, (0.0,), layout, dev)
    xs = [up(torch, dev, I.make_x(cfg, tokens=T, rep=r)) for r in range(4)]
    steps = min(args.steps, 20)
    s = measure(sw, torch, pools[0.0], cfg, T, xs, steps, min(args.warmup, 5), dev)
    H, Iw, k, m = cfg.hidden, cfg.inter, cfg.top_k, cfg.n_experts
    flops_gate_up = 2.0 * T * k * 2 * Iw * H
    flops = flops_gate_up + 2.0 * T * k * H * Iw + 2.0 * T * m * H
    gu_tflops = flops_gate_up / (s["gate_up_launch_us"] * 1e-6) / 1e12
    line = base_line(args, cfg, T, s["tokens_per_s"], s["t_step_us"], steps)
    line["config"] = {
        "workload": f"{cfg.name}: MoE layer H {H}, {m} experts, top-{k}, I {Iw}, {T} tokens, "
                    f"full pool (prefill shape)",
        "hidden": H, "n_experts": m, "top_k": k, "inter": Iw, "batch": T, "pruning": 0.0,
        "weight_layout": args.layout, "parallelism": "none (1 GPU)",
    }
    # ~128 tokens per expert give 128 FLOP per weight byte, below the chip's
    # 2500 / 8 = 312 FLOP/B balance point: the launch is bound by the weight
    # stream, and the MFMA rate is reported beside it
    line["roofline"] = hbm_roofline(cfg, T, 0.0, args.layout, s, kernel="gate_up_prefill_kernel")
    line["roofline"]["mfma"] = {
        "bound": "mfma", "kernel": "gate_up_prefill_kernel",
        "achieved": round(gu_tflops, 2), "peak": MFMA_BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
        "frac": round(gu_tflops / MFMA_BF16_PEAK_TFLOPS, 4),
        "algorithmic_flops_per_launch": flops_gate_up,
    }
    line["detail"] = {"full": rounded(s), "layer_flops": flops,
                      "layer_TFLOPs": round(flops / (s["t_step_us"] * 1e-6) / 1e12, 2)}
    if not args.no_cpu_baseline:
        line["cpu_baseline"] = cpu_baseline(cfg, L, 0.0, args.cpu_seconds, 64)
    return line


def run_decode_shared(args, sw, torch, dev):
    import copy

    cfg = I.CONFIGS["decode_sweep"]
    T, H, Iw = 64, cfg.hidden, cfg.inter
    S = 2
    Is = S * Iw  # the distilled decoder's shared expert: twice the original width
    # token groups of the folded parts: at most 16 tokens a copy, so that each
    # part is a one-pass, one-column-block expert of the decode kernels (every
    # further copy streams the shared weights once more; at batch 64 the
    # step measured 83 / 16.7 / 13.9 / 20.3 us above the routed layer with
    # 1 / 2 / 4 / 8 copies)
    groups = (T + 15) // 16
    L = I.make_layer(cfg)
    layout = sw.TILED if args.layout == "tiled" else sw.ROW_MAJOR
    pools = build_pools(sw, torch, cfg, L, (0.5, 0.0), layout, dev)
    g = np.random.default_rng([cfg.config_id, 0, 6])
    w13s = I.to_bf16_bits(np.float32(cfg.w_std) * g.standard_normal((2 * Is, H), dtype=np.float32))
    w2s = I.to_bf16_bits(np.float32(cfg.w_std) * g.standard_normal((H, Is), dtype=np.float32))
    gate_w = (cfg.wr_std * g.standard_normal(H)).astype(np.float32)
    # the separate call's operands: one expert of width Is
    w13s_d, w2s_d = up(torch, dev, w13s[None]), up(torch, dev, w2s[None])
    # the folded form: S parts of width I appended to the pool, the gate row
    # to the router (part s = intermediate units s*I .. (s+1)*I - 1)
    p13 = np.stack([np.concatenate([w13s[s * Iw:(s + 1) * Iw], w13s[Is + s * Iw:Is + (s + 1) * Iw]])
                    for s in range(S)])
    p2 = np.stack([np.ascontiguousarray(w2s[:, s * Iw:(s + 1) * Iw]) for s in range(S)])
    p13_d, p2_d = up(torch, dev, p13), up(torch, dev, p2)
    if layout == sw.TILED:
        w13s_d, w2s_d = sw.sw_moe_pack_experts(w13s_d, w2s_d)
        p13_d, p2_d = sw.sw_moe_pack_experts(p13_d, p2_d)
    gate_d = up(torch, dev, gate_w)
    xs = [up(torch, dev, I.make_x(cfg, tokens=T, rep=r)) for r in range(N_X)]
    res = {}
    for p in (0.5, 0.0):
        base = pools[p]
        res[(p, "none")] = measure(sw, torch, base, cfg, T, xs, args.steps, args.warmup, dev)
        for how, G in (("folded", groups), ("folded, one copy", 1)):
            folded = Pool(torch.cat([base.w13[0]] + [p13_d] * G),
                          torch.cat([base.w2[0]] + [p2_d] * G),
                          torch.cat([base.wr, gate_d[None]]), layout, n_shared=S, n_groups=G)
            res[(p, how)] = measure(sw, torch, folded, cfg, T, xs, args.steps, args.warmup, dev)
            del folded
        separate = copy.copy(base)
        separate.shared = (w13s_d, w2s_d, gate_d)
        res[(p, "separate")] = measure(sw, torch, separate, cfg, T, xs, args.steps, args.warmup, dev)
    head = res[(0.5, "folded")]
    line = base_line(args, cfg, T, head["tokens_per_s"], head["t_step_us"], args.steps)
    line["config"] = {
        "workload": f"decode_shared: decode MoE layer H {H}, {cfg.n_experts} experts, top-{cfg.top_k}, "
                    f"I {Iw}, batch {T}, 50% pruned ({cfg.n_keep(0.5)} kept, compacted) plus a shared "
                    f"expert of width {Is} behind a sigmoid gate, folded into the plan as {S} parts "
                    f"in {groups} token groups",
        "hidden": H, "n_experts": cfg.n_experts, "n_kept": cfg.n_keep(0.5), "top_k": cfg.top_k,
        "inter": Iw, "shared_inter": Is, "shared_parts": S, "shared_groups": groups, "batch": T,
        "pruning": 0.5,
        "weight_layout": args.layout, "parallelism": "none (1 GPU)",
    }
    line["roofline"] = hbm_roofline(cfg, T, 0.5, args.layout, head)
    line["detail"] = {f"{int(p * 100)}% {how}": rounded(v) for (p, how), v in res.items()}
    line["detail"]["shared_expert_us"] = {
        f"{int(p * 100)}% {how}": round(res[(p, how)]["t_step_us"] - res[(p, "none")]["t_step_us"], 3)
        for p in (0.5, 0.0) for how in ("folded", "folded, one copy", "separate")}
    line["detail"]["shared_expert_us_graph"] = {
        f"{int(p * 100)}% {how}": round(res[(p, how)]["t_step_graph_us"]
                                       - res[(p, "none")]["t_step_graph_us"], 3)
        for p in (0.5, 0.0) for how in ("folded", "folded, one copy", "separate")}
    line["detail"]["shared_expert_MiB"] = 3 * H * Is * 2 / 2 ** 20
    line["detail"]["speedup_pruned_vs_full_with_shared"] = round(
        res[(0.0, "folded")]["t_step_us"] / res[(0.5, "folded")]["t_step_us"], 3)
    if not args.no_cpu_baseline:
        line["cpu_baseline"] = cpu_baseline(cfg, L, 0.5, args.cpu_seconds, T)
    return line


def route_phase(s):
    """Routing time of a measured point (with the dispatch where the gate/up
    launch does not build the plan): the eager step minus its forward phases
    (each timed between events on the launch stream)."""
    return s["t_step_us"] - s["t_gate_up_us"] - s["t_down_us"] - s["t_combine_us"]


def run_colocated(args, sw, torch, dev):
    import copy

    cfg = I.CONFIGS["decode_sweep"]
    T, H, Iw, m, k = 64, cfg.hidden, cfg.inter, cfg.n_experts, cfg.top_k
    L = I.make_layer(cfg)
    layout = sw.TILED if args.layout == "tiled" else sw.ROW_MAJOR
    pools = build_pools(sw, torch, cfg, L, (0.5, 0.0), layout, dev)
    n_keep = cfg.n_keep(0.5)
    mask = sw.sw_moe_prune_compact(up(torch, dev, L["importance"]), n_keep, k, hidden=H,
                                   compact=False)["keep_mask"]
    masked = copy.copy(pools[0.0])
    masked.keep_mask = mask
    xs = [up(torch, dev, I.make_x(cfg, tokens=T, rep=r)) for r in range(N_X)]
    sm = measure(sw, torch, masked, cfg, T, xs, args.steps, args.warmup, dev)
    sc = measure(sw, torch, pools[0.5], cfg, T, xs, args.steps, args.warmup, dev)
    sf = measure(sw, torch, pools[0.0], cfg, T, xs, args.steps, args.warmup, dev)
    # the prefill phase on the same resident pool, no mask
    xp = [up(torch, dev, I.make_x(I.CONFIGS["prefill"], rep=r)) for r in range(2)]
    sp = measure(sw, torch, pools[0.0], cfg, 4096, xp, 10, 2, dev)
    line = base_line(args, cfg, T, sm["tokens_per_s"], sm["t_step_us"], args.steps)
    line["config"] = {
        "workload": f"colocated: one resident pool of {m} experts (H {H}, top-{k}, I {Iw}); decode "
                    f"batch {T} with the 50% router mask ({n_keep} eligible), prefill 4096 tokens "
                    f"unmasked",
        "hidden": H, "n_experts": m, "n_kept": n_keep, "top_k": k, "inter": Iw, "batch": T,
        "pruning": 0.5, "weight_layout": args.layout, "parallelism": "none (1 GPU)",
    }
    line["roofline"] = hbm_roofline(cfg, T, 0.5, args.layout, sm)
    line["detail"] = {
        "masked_full_pool": rounded(sm), "compacted_pool": rounded(sc), "unmasked_full_pool": rounded(sf),
        "prefill_unmasked_4096": rounded(sp),
        # the mask's cost per layer: masked full pool minus compacted pool, from
        # graph replay (no host calls in the difference) and per phase; the
        # eager difference includes host-side noise and is kept for reference
        "mask_overhead_us_per_layer": round(sm["t_step_graph_us"] - sc["t_step_graph_us"], 3),
        "mask_overhead_us_per_layer_eager": round(sm["t_step_us"] - sc["t_step_us"], 3),
        "mask_overhead_us_by_phase": {
            "route_dispatch": round(route_phase(sm) - route_phase(sc), 3),
            "gate_up": round(sm["gate_up_launch_us"] - sc["gate_up_launch_us"], 3),
            "down": round(sm["down_launch_us"] - sc["down_launch_us"], 3),
            "combine": round(sm["t_combine_us"] - sc["t_combine_us"], 3),
        },
        "speedup_masked_vs_full": round(sf["t_step_us"] / sm["t_step_us"], 3),
    }
    if not args.no_cpu_baseline:
        line["cpu_baseline"] = cpu_baseline(cfg, L, 0.5, args.cpu_seconds, T)
    return line


def run_skewed_stack(args, sw, torch, dev):
    import oracle
    from paper_2609_34117_amd import gen

    cfg = I.CONFIGS["skewed_stack"]
    T, H, Iw, m, k = cfg.tokens, cfg.hidden, cfg.inter, cfg.n_experts, cfg.top_k
    n_keep = cfg.n_keep(0.5)
    layout = sw.TILED if args.layout == "tiled" else sw.ROW_MAJOR
    layers = []
    for li in range(cfg.n_layers):
        w13 = torch.empty((m, 2 * Iw, H), dtype=torch.int16, device=dev)
        w2 = torch.empty((m, H, Iw), dtype=torch.int16, device=dev)
        gen.philox_normal_bf16(w13, I.philox_key(cfg.config_id, li, I.W13), 0, cfg.w_std)
        gen.philox_normal_bf16(w2, I.philox_key(cfg.config_id, li, I.W2), 0, cfg.w_std)
        if layout == sw.TILED:
            w13, w2 = sw.sw_moe_pack_experts(w13, w2)
        L = I.make_layer(cfg, layer=li, experts=False)
        wr, bias, imp = (up(torch, dev, L[n]) for n in ("wr", "bias", "importance"))
        c = sw.sw_moe_prune_compact(imp, n_keep, k, w13=w13, w2=w2, wr=wr, bias=bias)
        xs = [up(torch, dev, I.make_x(cfg, layer=li, rep=r)) for r in range(2)]
        x64 = up(torch, dev, I.make_x(cfg, tokens=64, layer=li, rep=7))
        layers.append(dict(full=(w13, w2, wr, bias, m), pruned=(c["w13"], c["w2"], c["wr"], c["bias"], n_keep),
                           xs=xs, x64=x64))
        torch.cuda.synchronize()
        print(f"# layer {li} drawn and packed", file=sys.stderr, flush=True)

    d_full, d_pr = sw.dims(H, Iw, m, k), sw.dims(H, Iw, n_keep, k)
    rws = sw.workspace(max(sw.sw_moe_route_workspace_bytes(d_full, T),
                           sw.sw_moe_route_workspace_bytes(d_pr, T)), dev)
    fws = sw.workspace(sw.sw_moe_forward_workspace_bytes(d_full, T), dev)
    ids = torch.empty((T, k), dtype=torch.int32, device=dev)
    w = torch.empty((T, k), dtype=torch.float32, device=dev)
    gap = torch.empty(T, dtype=torch.float32, device=dev)
    out = torch.empty((T, H), dtype=torch.float32, device=dev)
    plans = {"full": [sw.alloc_plan(T, m, k, dev) for _ in layers],
             "pruned": [sw.alloc_plan(T, n_keep, k, dev) for _ in layers]}

    def step(which, r):
        for li, Lr in enumerate(layers):
            w13, w2, wr, bias, mp = Lr[which]
            x = Lr["xs"][r % 2]
            sw.sw_moe_route_dispatch(x, wr, k, bias=bias, out=(ids, w, gap), plan=plans[which][li],
                                     ws=rws)
            sw.sw_moe_forward(x, w13, w2, w, plans[which][li], layout=layout, out=out, ws=fws)

    steps = max(2, min(args.steps, 10))
    res = {}
    for which in ("pruned", "full"):
        for r in range(2):
            step(which, r)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for r in range(steps):
            step(which, r)
        e1.record()
        torch.cuda.synchronize()
        t = e0.elapsed_time(e1) / 1e3 / steps
        n_act = np.array([int(p.n_active.item()) for p in plans[which]])  # of the last step
        vol = []
        for Lr in layers:  # pool fraction a batch of 64 touches
            w13, w2, wr, bias, mp = Lr[which]
            _, _, _, pl = sw.sw_moe_route_dispatch(Lr["x64"], wr, k, bias=bias)
            vol.append(int(pl.n_active.item()) / mp)
        U = n_act.sum() * 3 * H * Iw * 2
        res[which] = dict(t_step_us=t * 1e6, tokens_per_s=T / t, n_active_mean=float(n_act.mean()),
                          pool_fraction_b256=float(n_act.mean() / (m if which == "full" else n_keep)),
                          pool_fraction_b64=float(np.mean(vol)),
                          unique_GiB_per_step=float(U / 2 ** 30), fwd_layer_GBps=float(U / t / 1e9))
        print(f"# {which}: {res[which]}", file=sys.stderr, flush=True)
    sp, sf = res["pruned"], res["full"]
    line = base_line(args, cfg, T, sp["tokens_per_s"], sp["t_step_us"], steps)
    line["config"] = {
        "workload": f"{cfg.name}: {cfg.n_layers} MoE layers H {H}, {m} experts, top-{k}, I {Iw}, "
                    f"batch {T}, Zipf({cfg.zipf_s}) router bias (beta {cfg.zipf_beta}), 50% pruned "
                    f"({n_keep} kept by popularity, compacted); step = all {cfg.n_layers} layers",
        "hidden": H, "n_experts": m, "n_kept": n_keep, "top_k": k, "inter": Iw, "batch": T,
        "layers": cfg.n_layers, "pruning": 0.5, "weight_layout": args.layout,
        "parallelism": "none (1 GPU)",
    }
    line["data"] = ("synthetic: experts drawn on the device from a counter-based stream "
                    "(Philox4x64-10, ~N(0,0.02) bf16), routers and tokens seeded on the host")
    # roofline: the stack's unique expert bytes over its step time
    ach = sp["fwd_layer_GBps"]
    line["roofline"] = {"bound": "hbm", "kernel": "whole step (40 layers)", "achieved": round(ach, 1),
                        "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": round(ach / HBM_PEAK_GBS, 4),
                        "traffic": None}
    line["detail"] = {"pruned": rounded(sp), "full": rounded(sf),
                      "speedup_pruned_vs_full": round(sf["t_step_us"] / sp["t_step_us"], 3)}
    if not args.no_cpu_baseline:
        line["cpu_baseline"] = stack_cpu_baseline(cfg, n_keep, args.cpu_seconds)
    return line


def stack_cpu_baseline(cfg, n_keep, seconds):
    """The C oracle on layer 0 of the pruned stack (route + dispatch +
    forward) for batches of 8 tokens, extrapolated to the 40 layers; only the
    experts the batch selects are drawn on the host."""
    import oracle

    L = I.make_layer(cfg, layer=0, experts=False)
    kept, remap, mask, *_ = oracle.prune_compact(L["importance"], n_keep, cfg.top_k)
    done, elapsed, batches = 0, 0.0, 0
    while elapsed < seconds and batches < 8:
        x = I.make_x(cfg, tokens=8, layer=0, rep=100 + batches)
        ids, w, _ = oracle.route(x, L["wr"], cfg.top_k, keep_mask=mask, bias=L["bias"])
        used = np.unique(ids)
        w13 = I.philox_expert_slice(cfg, 0, "w13", used)
        w2 = I.philox_expert_slice(cfg, 0, "w2", used)
        local = np.searchsorted(used, ids).astype(np.int32)
        t0 = time.perf_counter()
        oracle.route(x, L["wr"], cfg.top_k, keep_mask=mask, bias=L["bias"])
        oracle.dispatch(ids, cfg.n_experts)
        oracle.forward(x, w13, w2, local, w)
        elapsed += time.perf_counter() - t0
        done += x.shape[0]
        batches += 1
    per_layer = done / elapsed
    return dict(value=round(per_layer / cfg.n_layers, 3), unit="tokens/s", cores=1, kind="oracle",
                sample=f"{batches} batch(es) of 8 tokens through layer 0 of the pruned stack "
                       f"(route+dispatch+forward, {elapsed:.1f} s, 1 thread), extrapolated to "
                       f"{cfg.n_layers} layers")


def main():
    args = parse()
    if args.gpus != 1:
        print(json.dumps({"error": "this build runs on one GPU: the layer is not sharded; "
                                   "run with --gpus 1"}))
        sys.exit(2)
    import torch

    from paper_2609_34117_amd import slimwise as sw

    dev = torch.device("cuda:0")
    run = {"decode_b64": run_decode_b64, "decode_sweep": run_decode_sweep,
           "prefill": run_prefill, "skewed_stack": run_skewed_stack,
           "decode_shared": run_decode_shared, "colocated": run_colocated}[args.workload]
    print(json.dumps(run(args, sw, torch, dev)), flush=True)


if __name__ == "__main__":
    main()
