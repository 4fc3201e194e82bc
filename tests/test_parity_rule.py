"""The routing comparison rule of the GPU parity tests, checked on the CPU
with hand-made logits: what it accepts and what it rejects."""
import numpy as np
import pytest

import oracle
from paper_2609_34117_amd import inputs as I
from parity import NEAR_TIE, compare_routing, near_tie_tokens, plan_rows


def _gates(z, ids):
    s = z[ids] - z[ids].max()
    e = np.exp(s.astype(np.float64))
    return (e / e.sum()).astype(np.float32)


def _route(z, k):
    ids = np.argsort(-z.astype(np.float64), kind="stable")[:k]
    srt = np.sort(z.astype(np.float64))[::-1]
    gap = srt[k - 1] - srt[k] if len(z) > k else np.inf
    return ids.astype(np.int32), _gates(z, ids), np.float32(gap)


def _case(rows, k):
    z = np.array(rows, np.float32)
    o = [_route(r, k) for r in z]
    return z, np.stack([a for a, _, _ in o]), np.stack([b for _, b, _ in o]), np.array([c for _, _, c in o])


def test_identical_routing_passes_and_counts_nothing():
    z, ids, w, gap = _case([[0.5, 0.1, 0.9, -0.3, 0.2]], 2)
    s = compare_routing(ids, w, ids, w, z, None, 2, g_gap=gap, o_gap=gap)
    assert s["near_ties"] == 0 and s["inner_ties"] == 0


def test_near_tie_at_k_allows_the_kth_choice_to_change():
    d = 0.3 * NEAR_TIE
    z, ids, w, gap = _case([[0.9, 0.5, 0.2, 0.2 - d, -1.0]], 3)
    g_ids = ids.copy()
    g_ids[0, 2] = 3                      # the tied (k+1)-th expert instead of the k-th
    g_w = _gates(z[0], g_ids[0])[None]
    s = compare_routing(g_ids, g_w, ids, w, z, None, 3, g_gap=gap, o_gap=gap)
    assert s["near_ties"] == 1 and s["near_tie_swaps"] == 1


def test_near_tie_at_k_does_not_exempt_the_other_slots():
    d = 0.3 * NEAR_TIE
    z, ids, w, gap = _case([[0.9, 0.5, 0.2, 0.2 - d, -1.0]], 3)
    g_ids = ids.copy()
    g_ids[0, 0] = 4                      # a wrong first choice
    with pytest.raises(AssertionError):
        compare_routing(g_ids, w, ids, w, z, None, 3)


def test_a_swap_without_a_tie_fails():
    z, ids, w, gap = _case([[0.9, 0.5, 0.2, 0.1, -1.0]], 3)
    g_ids = ids.copy()
    g_ids[0, 2] = 3
    with pytest.raises(AssertionError):
        compare_routing(g_ids, w, ids, w, z, None, 3)


def test_tie_inside_top_k_allows_reorder_but_not_another_set():
    d = 0.3 * NEAR_TIE
    z, ids, w, gap = _case([[0.9, 0.5, 0.5 - d, 0.1, -1.0]], 3)
    g_ids = ids.copy()
    g_ids[0, [1, 2]] = g_ids[0, [2, 1]]   # the tied pair reordered
    g_w = w.copy()
    g_w[0, [1, 2]] = g_w[0, [2, 1]]
    s = compare_routing(g_ids, g_w, ids, w, z, None, 3, g_gap=gap, o_gap=gap)
    assert s["inner_ties"] == 1 and s["inner_reorders"] == 1 and s["near_ties"] == 0
    bad = ids.copy()
    bad[0, 2] = 3                         # the set changes: no near tie at k
    with pytest.raises(AssertionError):
        compare_routing(bad, w, ids, w, z, None, 3)


def test_gate_and_gap_errors_fail():
    z, ids, w, gap = _case([[0.9, 0.5, 0.2, 0.1, -1.0]], 2)
    with pytest.raises(AssertionError):
        compare_routing(ids, w + 3e-5, ids, w, z, None, 2)
    with pytest.raises(AssertionError):
        compare_routing(ids, w, ids, w, z, None, 2, g_gap=gap + 3e-5, o_gap=gap)
    with pytest.raises(AssertionError):
        compare_routing(ids, w, ids, w, z, None, 2, g_gap=np.array([np.inf], np.float32), o_gap=gap)


def test_masked_expert_selected_fails_and_exactly_k_eligible_is_inf():
    z, ids, w, gap = _case([[0.9, 0.5, 0.2, 0.1, -1.0]], 2)
    mask = np.array([1, 0, 1, 0, 0], np.uint8)
    o_ids, o_w, o_gap, o_z = oracle.route(I.to_bf16_bits(np.eye(5, dtype=np.float32)[:1] * 0 + 1),
                                          np.eye(5, dtype=np.float32) * z[0][:, None], 2,
                                          keep_mask=mask, want_logits=True)
    assert np.isposinf(o_gap[0])
    compare_routing(o_ids, o_w, o_ids, o_w, o_z, mask, 2, g_gap=o_gap, o_gap=o_gap)
    with pytest.raises(AssertionError):
        compare_routing(ids, w, o_ids, o_w, o_z, mask, 2)   # expert 1 is pruned


def test_near_tie_tokens_uses_only_the_kth_gap():
    d = 0.3 * NEAR_TIE
    z = np.array([[0.9, 0.9 - d, 0.2, 0.1], [0.9, 0.5, 0.2, 0.2 - d]], np.float32)
    assert near_tie_tokens(z, None, 2).tolist() == [False, False]
    assert near_tie_tokens(z, None, 3).tolist() == [False, True]


def test_plan_rows_reach_every_pass_edge():
    # one expert with 70 pairs (passes 0-31, 32-63, 64-69), one with 1 pair
    ids = np.array([[0, 1] if t == 5 else [0, 2] for t in range(70)], np.int32)
    counts, offsets, perm, active, n = oracle.dispatch(ids, 3)
    rows = set(plan_rows(counts, offsets, perm, 2).tolist())
    assert {0, 31, 32, 63, 64, 69, 5} <= rows
