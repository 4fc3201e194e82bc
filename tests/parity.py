"""Comparison helpers for the GPU parity tests (HIP library vs CPU oracle).

Tolerances:
  - top-k ids and dispatch plans: bit-exact, except near ties.  A token is a
    near tie when two adjacent logits among the oracle's top k+1 differ by
    less than NEAR_TIE (fp32 dot products summed in different orders differ
    by ~1e-6 at these magnitudes, so such tokens may legitimately select or
    order differently).  Near ties are counted and reported, and for them
    the selected logits must agree with the oracle's to NEAR_TIE.
  - gates: |dw| <= 1e-5 on tokens that are not near ties.
  - layer outputs: max |err| <= 2e-2 and normwise relative error
    sum|err| / sum|ref| <= 5e-3 against the fp32-accumulated oracle.
"""
import numpy as np

NEAR_TIE = 1e-5
GATE_TOL = 1e-5
OUT_MAX_ABS = 2e-2
OUT_REL = 5e-3


def near_tie_tokens(logits, keep_mask, k):
    """Tokens whose oracle top-(k+1) logits contain an adjacent gap < NEAR_TIE."""
    z = logits.astype(np.float64).copy()
    if keep_mask is not None:
        z[:, keep_mask == 0] = -np.inf
    top = -np.sort(-z, axis=1)[:, : k + 1]
    gaps = top[:, :-1] - top[:, 1:]
    gaps = np.where(np.isnan(gaps), np.inf, gaps)
    return np.min(gaps, axis=1) < NEAR_TIE if top.shape[1] > 1 else np.zeros(len(z), bool)


def compare_routing(g_ids, g_w, o_ids, o_w, o_logits, keep_mask, k):
    """Asserts routing parity; returns the number of near-tie tokens."""
    near = near_tie_tokens(o_logits, keep_mask, k)
    far = ~near
    np.testing.assert_array_equal(g_ids[far], o_ids[far])
    if far.any():
        dw = np.abs(g_w[far] - o_w[far]).max()
        assert dw <= GATE_TOL, f"gate error {dw}"
    for t in np.flatnonzero(near):
        # every selected expert is eligible and its logit is within NEAR_TIE of
        # the oracle's logit at the same rank
        zg = o_logits[t, g_ids[t]].astype(np.float64)
        zo = o_logits[t, o_ids[t]].astype(np.float64)
        assert len(set(g_ids[t].tolist())) == k
        if keep_mask is not None:
            assert np.all(keep_mask[g_ids[t]] == 1)
        assert np.all(np.abs(np.sort(zg)[::-1] - zo) < NEAR_TIE), (t, zg, zo)
        np.testing.assert_allclose(g_w[t].sum(), 1.0, atol=1e-5)
    return int(near.sum())


def compare_out(g_out, o_out, what="out"):
    err = np.abs(g_out.astype(np.float64) - o_out.astype(np.float64))
    denom = np.abs(o_out.astype(np.float64)).sum()
    rel = err.sum() / denom if denom > 0 else err.sum()
    assert np.isfinite(g_out).all(), f"{what}: non-finite values"
    assert err.max() <= OUT_MAX_ABS, f"{what}: max|err| {err.max():.3g}"
    assert rel <= OUT_REL, f"{what}: normwise rel err {rel:.3g}"
    return float(err.max()), float(rel)
