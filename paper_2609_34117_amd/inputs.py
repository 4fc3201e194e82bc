"""Seeded synthetic inputs for the batched-decode MoE layer.

This module only draws data: shapes, distributions and seeds.  It holds no
step of the layer's arithmetic, so the HIP library's tests and the CPU oracle
can both consume exactly the same bytes from it.

Workloads stand in for a Qwen3.6-35B-A3B-like MoE layer (256 routed experts,
top-8, 40 layers, a 60 GiB bf16 expert pool; Section 2.1 and Fig. 2 of the
paper) and for its REAP-selected kept sets, neither of which is available:
weights are i.i.d. normal, importance scores are uniform, so the kept set is a
seeded random subset.

Seeding: ``numpy.random.default_rng([config_id, layer, tensor_id, rep])`` with
tensor ids x=0, router=1, W13=2, W2=3, importance=4, popularity=5.

Expert pools too large to draw on the host (the 40-layer, 60 GiB stack) use a
counter-based stream instead, so any element range can be drawn anywhere:
element i of a tensor is a function of (key, i) alone.  The stream is
Philox4x64-10 (Salmon, Moraes, Dror and Shaw, "Parallel random numbers: as
easy as 1, 2, 3", SC 2011); here numpy's implementation of it draws the host
side, and the HIP library of synthetic inputs implements it independently
for the device.  See ``philox_normal_bf16``.
"""
from __future__ import annotations

import dataclasses
from typing import Optional

import numpy as np

X, WR, W13, W2, IMPORTANCE, POPULARITY = range(6)


@dataclasses.dataclass(frozen=True)
class MoEConfig:
    name: str
    config_id: int
    hidden: int
    n_experts: int
    top_k: int
    inter: int
    tokens: int
    w_std: float = 0.02
    wr_std: float = 0.02
    zipf_s: Optional[float] = None      # per-expert logit bias from a Zipf popularity
    zipf_beta: float = 0.25             # bias = beta * ln(p_e)
    n_layers: int = 1

    def expert_bytes(self) -> int:
        """bf16 bytes of one expert: W13 (2I x H) plus W2 (H x I)."""
        return 3 * self.hidden * self.inter * 2

    def n_keep(self, pruning: float) -> int:
        keep = self.n_experts * (1.0 - pruning)
        n = int(round(keep))
        if abs(keep - n) > 1e-9:
            raise ValueError(f"pruning {pruning} of {self.n_experts} experts is not an integer count")
        return n


# The five workloads (tiny parity case, the batch-64 decode layer, the decode
# sweep shape, the prefill-shaped contrast and the skewed 40-layer stack).
CONFIGS = {
    "tiny": MoEConfig("tiny", 0, hidden=256, n_experts=16, top_k=2, inter=128, tokens=8),
    "decode_b64": MoEConfig("decode_b64", 1, hidden=2048, n_experts=128, top_k=8, inter=768, tokens=64),
    "decode_sweep": MoEConfig("decode_sweep", 2, hidden=2048, n_experts=256, top_k=8, inter=512, tokens=64),
    "prefill": MoEConfig("prefill", 3, hidden=2048, n_experts=256, top_k=8, inter=512, tokens=4096),
    "skewed_stack": MoEConfig("skewed_stack", 4, hidden=2048, n_experts=256, top_k=8, inter=512,
                              tokens=256, zipf_s=1.1, zipf_beta=0.25, n_layers=40),
}

SWEEP_BATCHES = (1, 8, 32, 64, 128, 256)
SWEEP_PRUNING = (0.0, 0.25, 0.5, 0.75)


def rng(config_id: int, layer: int, tensor_id: int, rep: int = 0) -> np.random.Generator:
    return np.random.default_rng([config_id, layer, tensor_id, rep])


def to_bf16_bits(a: np.ndarray) -> np.ndarray:
    """Round fp32 values to the nearest bf16 (ties to even); return uint16 bits.

    Inputs are finite normal draws, so no NaN/Inf handling is needed."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    u = a.view(np.uint32)
    lsb = (u >> np.uint32(16)) & np.uint32(1)
    r = (u + np.uint32(0x7FFF) + lsb) >> np.uint32(16)
    return r.astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    """Exact widening of bf16 bit patterns (for building test expectations)."""
    return (np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def normal_bf16(g: np.random.Generator, shape, std: float, chunk: int = 1 << 24) -> np.ndarray:
    """N(0, std) draws in fp32, rounded to bf16 bits, generated in chunks."""
    n = int(np.prod(shape))
    out = np.empty(n, np.uint16)
    for s in range(0, n, chunk):
        e = min(n, s + chunk)
        v = g.standard_normal(e - s, dtype=np.float32)
        v *= np.float32(std)
        out[s:e] = to_bf16_bits(v)
    return out.reshape(shape)


def make_x(cfg: MoEConfig, tokens: Optional[int] = None, layer: int = 0, rep: int = 0) -> np.ndarray:
    """Token activations ~N(0, 1), bf16 bits [T, H]."""
    t = cfg.tokens if tokens is None else tokens
    return normal_bf16(rng(cfg.config_id, layer, X, rep), (t, cfg.hidden), 1.0)


def make_router(cfg: MoEConfig, layer: int = 0) -> np.ndarray:
    g = rng(cfg.config_id, layer, WR)
    v = g.standard_normal((cfg.n_experts, cfg.hidden), dtype=np.float32)
    v *= np.float32(cfg.wr_std)
    return v


def make_experts(cfg: MoEConfig, layer: int = 0):
    """W13 [m, 2I, H] (gate rows then up rows) and W2 [m, H, I], bf16 bits."""
    w13 = normal_bf16(rng(cfg.config_id, layer, W13), (cfg.n_experts, 2 * cfg.inter, cfg.hidden), cfg.w_std)
    w2 = normal_bf16(rng(cfg.config_id, layer, W2), (cfg.n_experts, cfg.hidden, cfg.inter), cfg.w_std)
    return w13, w2


def make_importance(cfg: MoEConfig, layer: int = 0) -> np.ndarray:
    """Per-expert importance scores ~U(0, 1) (stand-in for calibration
    statistics).  For the skewed stack the score is the popularity itself, so
    the kept set is the most popular experts."""
    if cfg.zipf_s is not None:
        return zipf_popularity(cfg, layer).astype(np.float32)
    return rng(cfg.config_id, layer, IMPORTANCE).random(cfg.n_experts, dtype=np.float32)


def zipf_popularity(cfg: MoEConfig, layer: int = 0) -> np.ndarray:
    """Zipf(s) popularity p_e over a seeded random ranking of the experts
    (rank r_e in 1..m, p_e proportional to r_e^-s)."""
    g = rng(cfg.config_id, layer, POPULARITY)
    ranks = g.permutation(cfg.n_experts) + 1
    p = ranks.astype(np.float64) ** (-float(cfg.zipf_s))
    return p / p.sum()


def make_bias(cfg: MoEConfig, layer: int = 0) -> Optional[np.ndarray]:
    """Router logit bias beta * ln(p_e) for the skewed stack, else None."""
    if cfg.zipf_s is None:
        return None
    return (cfg.zipf_beta * np.log(zipf_popularity(cfg, layer))).astype(np.float32)


def make_layer(cfg: MoEConfig, layer: int = 0, tokens: Optional[int] = None, rep: int = 0,
               experts: bool = True) -> dict:
    """All inputs of one layer as numpy arrays."""
    d = dict(cfg=cfg, x=make_x(cfg, tokens, layer, rep), wr=make_router(cfg, layer),
             importance=make_importance(cfg, layer), bias=make_bias(cfg, layer))
    if experts:
        d["w13"], d["w2"] = make_experts(cfg, layer)
    return d


def small_config(hidden=64, n_experts=8, top_k=2, inter=32, tokens=5, name="custom") -> MoEConfig:
    """An ad-hoc shape for edge-case tests (config id 100)."""
    return MoEConfig(name, 100, hidden=hidden, n_experts=n_experts, top_k=top_k, inter=inter, tokens=tokens)


# ---------------------------------------------------------------------------
# counter-based normal draws (Philox4x64-10 + Irwin-Hall)

IRWIN_HALL_MEAN = 12 * 65535 // 2  # 393210: mean of a sum of 12 uniform 16-bit integers


def philox_key(config_id: int, layer: int, tensor_id: int) -> np.ndarray:
    """Philox key of one tensor: (config_id << 32 | layer, tensor_id)."""
    return np.array([(config_id << 32) | layer, tensor_id], dtype=np.uint64)


def philox_normal_bf16(key: np.ndarray, start: int, n: int, std: float) -> np.ndarray:
    """Elements start .. start + n - 1 of a tensor ~N(0, std), as bf16 bits.

    Element i takes the Philox4x64-10 block of counter (i + 1, 0, 0, 0) under
    `key`; the twelve 16-bit halves of the block's first three 64-bit words
    (low half first) are summed, S, and the value is
    float32(S - 393210) * float32(std / 65536), rounded to bf16 (ties to
    even).  The sum of 12 uniform integers on [0, 65535] has mean 393210 and
    standard deviation ~65536 (Irwin-Hall), so the value is ~N(0, std)
    truncated at +-6 std.  Both products are exact or correctly rounded fp32
    operations, so any IEEE implementation gives the same bits."""
    out = np.empty(n, np.uint16)
    scale = np.float32(np.float32(std) / np.float32(65536.0))
    chunk = 1 << 22
    for s0 in range(0, n, chunk):
        m = min(chunk, n - s0)
        # numpy's Philox advances the counter before each block: starting
        # from counter start + s0, the first block uses start + s0 + 1
        bg = np.random.Philox(key=key, counter=np.array([start + s0, 0, 0, 0], dtype=np.uint64))
        words = np.ascontiguousarray(bg.random_raw(4 * m).reshape(m, 4)[:, :3])
        sums = words.view("<u2").reshape(m, 12).sum(axis=1, dtype=np.int64)
        v = (sums - IRWIN_HALL_MEAN).astype(np.float32) * scale
        out[s0:s0 + m] = to_bf16_bits(v)
    return out


def philox_expert_slice(cfg: MoEConfig, layer: int, which: str, experts) -> np.ndarray:
    """Host copy of the counter-drawn W13 or W2 rows of the given experts
    (the same bits the device draws for the whole pool)."""
    if which == "w13":
        tid, per, shape = W13, 2 * cfg.inter * cfg.hidden, (2 * cfg.inter, cfg.hidden)
    else:
        tid, per, shape = W2, cfg.hidden * cfg.inter, (cfg.hidden, cfg.inter)
    key = philox_key(cfg.config_id, layer, tid)
    return np.stack([philox_normal_bf16(key, int(e) * per, per, cfg.w_std).reshape(shape)
                     for e in experts])

