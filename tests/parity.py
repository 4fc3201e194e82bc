"""Comparison helpers for the GPU parity tests (HIP library vs CPU oracle).

Routing (Section 3.1, Eq. 2 and the renormalisation over the k selected):

  - Near tie.  A token is a near tie when the oracle's gap z_(k) - z_(k+1)
    between its k-th and (k+1)-th largest eligible logits is below NEAR_TIE.
    This is the only exemption from bit-exact ids: for such a token the
    experts tied with z_(k) (the oracle's ranks linked to rank k by adjacent
    gaps below NEAR_TIE) may be exchanged for one another, so a different
    k-th choice is accepted when its oracle logit is within NEAR_TIE of
    z_(k).  Every other selected id must still be the oracle's.
  - Ties inside the top k.  Where two adjacent logits among the first k
    differ by less than NEAR_TIE the order of those experts may differ (the
    GPU sums each dot product in another order, ~1e-6 apart at these
    magnitudes), but the set of ids must be the oracle's exactly.
  - Every other rank: the GPU id equals the oracle id at that rank.
  - Gates: |dw| <= GATE_TOL at every slot, and per id for every id both
    sides selected.  Gates are a continuous function of the sorted selected
    logits, so both hold for near-tie tokens as well.
  - Gap: |dgap| <= GAP_TOL * max(1, |z_(k)|, |z_(k+1)|) for every token
    (order statistics move by at most the largest logit error, so the gap is
    continuous in the logits even where the ids differ; the error of an fp32
    logit grows with its magnitude, ~4e-6 at |z| = 50 where a bias forces an
    expert); +inf (exactly k eligible experts) and NaN (fewer than k) must
    agree exactly.

Outputs: max |err| <= 2e-2 and normwise relative error
sum|err| / sum|ref| <= 5e-3 against the fp32-accumulated oracle.
"""
from __future__ import annotations

import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np

NEAR_TIE = 1e-5
GATE_TOL = 1e-5
GAP_TOL = 1e-5
OUT_MAX_ABS = 2e-2
OUT_REL = 5e-3

# near-tie counts of every routing comparison of the session, printed in the
# terminal summary (conftest.py); CURRENT_CASE names the running test
RECORDS: list = []
CURRENT_CASE = ""


def _eligible_logits(logits, keep_mask):
    z = logits.astype(np.float64).copy()
    if keep_mask is not None:
        z[:, np.asarray(keep_mask) == 0] = -np.inf
    return z


def near_tie_tokens(logits, keep_mask, k):
    """Tokens whose oracle gap z_(k) - z_(k+1) over the eligible experts is
    below NEAR_TIE (the only exemption from bit-exact ids)."""
    z = _eligible_logits(logits, keep_mask)
    if z.shape[1] <= k:
        return np.zeros(len(z), bool)
    top = -np.sort(-z, axis=1)[:, : k + 1]
    gap = top[:, k - 1] - top[:, k]
    gap = np.where(np.isnan(gap), np.inf, gap)
    return gap < NEAR_TIE


def compare_routing(g_ids, g_w, o_ids, o_w, o_logits, keep_mask, k, g_gap=None, o_gap=None,
                    what="route"):
    """Asserts routing parity under the rule in this module's docstring.

    Returns a dict: near_ties (tokens with z_(k) - z_(k+1) < NEAR_TIE),
    near_tie_swaps (of those, tokens whose GPU k-th choice differs),
    inner_ties (tokens with an adjacent gap < NEAR_TIE inside the top k),
    inner_reorders (of those, tokens whose GPU order differs), and the
    largest gate and gap differences."""
    g_ids = np.asarray(g_ids)
    o_ids = np.asarray(o_ids)
    g_w = np.asarray(g_w, np.float64)
    o_w = np.asarray(o_w, np.float64)
    t = o_ids.shape[0]
    z = _eligible_logits(o_logits, keep_mask)
    m = z.shape[1]
    order = np.argsort(-z, axis=1, kind="stable")
    zs = np.take_along_axis(z, order, axis=1)
    stats = dict(case=CURRENT_CASE, what=what, tokens=t, near_ties=0, near_tie_swaps=0, inner_ties=0,
                 inner_reorders=0, max_dw=0.0, max_dgap=0.0)
    for i in range(t):
        n_elig = int(np.isfinite(zs[i]).sum())
        kk = min(k, n_elig)
        assert np.array_equal(order[i, :kk], o_ids[i, :kk]), (what, i, "oracle ids vs its logits")
        # tie groups: oracle ranks linked by adjacent gaps below NEAR_TIE
        tie_next = np.zeros(m, bool)
        tie_next[: n_elig - 1] = (zs[i, : n_elig - 1] - zs[i, 1:n_elig]) < NEAR_TIE
        group = np.concatenate([[0], np.cumsum(~tie_next[:-1])])
        rank_of = np.empty(m, np.int64)
        rank_of[order[i]] = np.arange(m)
        near = kk == k and n_elig > k and tie_next[k - 1]
        # the boundary group (ranks tied with rank k) may trade members across
        # the k-th place; every other group stays inside or outside the top k
        boundary = set(order[i, group == group[k - 1]].tolist()) if near else set()
        gi = g_ids[i, :kk].tolist()
        oi = o_ids[i, :kk].tolist()
        assert np.all(g_ids[i, kk:] == -1), (what, i, "slots past the eligible count")
        assert len(set(gi)) == kk, (what, i, "repeated id", gi)
        assert all(0 <= e < m for e in gi), (what, i, "id out of range", gi)
        if keep_mask is not None:
            assert all(keep_mask[e] == 1 for e in gi), (what, i, "pruned expert selected", gi)
        assert set(gi) - boundary == set(oi) - boundary, (what, i, gi, oi)
        for r in range(kk):
            # the GPU's expert at rank r is one the oracle ranks in rank r's
            # tie group; an untied rank is a group of one, so its id is exact
            assert group[rank_of[gi[r]]] == group[r], (what, i, r, gi, oi)
        if near:
            stats["near_ties"] += 1
            stats["near_tie_swaps"] += int(set(gi) != set(oi))
        inner = bool(np.any(tie_next[: max(kk - 1, 0)]))
        stats["inner_ties"] += int(inner)
        if inner and gi != oi and set(gi) == set(oi):
            stats["inner_reorders"] += 1
        # gates: per slot, and per id over the ids both sides selected
        dw = float(np.abs(g_w[i] - o_w[i]).max()) if k else 0.0
        for e in set(gi) & set(oi):
            dw = max(dw, abs(g_w[i, gi.index(e)] - o_w[i, oi.index(e)]))
        assert dw <= GATE_TOL, (what, i, "gate error", dw)
        stats["max_dw"] = max(stats["max_dw"], dw)
    if g_gap is not None and o_gap is not None:
        g_gap = np.asarray(g_gap, np.float64)
        o_gap = np.asarray(o_gap, np.float64)
        assert np.array_equal(np.isnan(g_gap), np.isnan(o_gap)), (what, "NaN gaps differ")
        assert np.array_equal(np.isposinf(g_gap), np.isposinf(o_gap)), (what, "+inf gaps differ")
        fin = np.isfinite(o_gap)
        assert np.all(np.isfinite(g_gap[fin])), (what, "non-finite GPU gap")
        if fin.any() and m > k:
            scale = np.maximum(1.0, np.maximum(np.abs(zs[:, k - 1]), np.abs(zs[:, k])))
            dg = np.abs(g_gap - o_gap)[fin]
            assert np.all(dg <= GAP_TOL * scale[fin]), (what, "gap error", float(dg.max()))
            stats["max_dgap"] = float(dg.max())
    RECORDS.append(stats)
    return stats


def compare_out(g_out, o_out, what="out"):
    err = np.abs(g_out.astype(np.float64) - o_out.astype(np.float64))
    denom = np.abs(o_out.astype(np.float64)).sum()
    rel = err.sum() / denom if denom > 0 else err.sum()
    assert np.isfinite(g_out).all(), f"{what}: non-finite values"
    if err.size:
        assert err.max() <= OUT_MAX_ABS, f"{what}: max|err| {err.max():.3g}"
    assert rel <= OUT_REL, f"{what}: normwise rel err {rel:.3g}"
    return (float(err.max()) if err.size else 0.0), float(rel)


def oracle_threads() -> int:
    """Worker threads for oracle calls over many tokens (the oracle itself is
    single-threaded; ctypes releases the GIL during each call)."""
    return max(1, min(16, os.cpu_count() or 1))


def oracle_forward_rows(fwd, x, w13, w2, ids, w, rows=None, chunk=64):
    """The oracle's forward of the given token rows (all rows by default),
    split over threads in chunks of tokens.  Each token's output depends only
    on its own row, so the result is the same as one call."""
    rows = np.arange(ids.shape[0]) if rows is None else np.asarray(rows)
    parts = [rows[s:s + chunk] for s in range(0, len(rows), chunk)]

    def one(r):
        return fwd(np.ascontiguousarray(x[r]), w13, w2, np.ascontiguousarray(ids[r]),
                   np.ascontiguousarray(w[r]))

    if not parts:
        return np.zeros((0, x.shape[1]), np.float32)
    with ThreadPoolExecutor(oracle_threads()) as ex:
        outs = list(ex.map(one, parts))
    return np.concatenate(outs)


def plan_rows(counts, offsets, perm, top_k, pass_tokens=(16, 32, 160)):
    """Token rows that reach the edges of every active expert's work: its
    first and last pair, and the first and last pair of every block of
    `pass_tokens` pairs (the decode kernels' 16-token column blocks and
    32-token passes, the prefill kernels' 160-token passes), so a sample
    covers each expert's last pass and its last (ragged) column block."""
    counts = np.asarray(counts)
    offsets = np.asarray(offsets)
    perm = np.asarray(perm)
    pairs = set()
    for e in np.flatnonzero(counts > 0):
        s, n = int(offsets[e]), int(counts[e])
        pairs.update((s, s + n - 1))
        for p in pass_tokens:
            for b in range(0, n, p):
                pairs.update((s + b, s + min(b + p, n) - 1))
    return np.unique(perm[sorted(pairs)] // top_k)
