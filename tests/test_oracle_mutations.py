"""Plant plausible mistakes in the CPU oracle and check that the pins catch them.

Each case swaps one oracle function for a subtly wrong copy (on the CPU, inside
this process only) and asserts that at least one pin of
tests/test_oracle_pins.py then fails.  Nothing here touches the GPU path.
"""
import functools

import numpy as np
import pytest

from oracle import moe_oracle as O
import tests.test_oracle_pins as P


def _tie_high_index_wins(Z, k):
    Z = np.asarray(Z, np.float32)
    T, E = Z.shape
    experts = np.broadcast_to(-np.arange(E), (T, E))
    order = np.lexsort((experts, -Z.astype(np.float64)), axis=-1)
    return np.sort(order[:, :k], axis=1).astype(np.int32)


def _weights_not_renormalised(Z, idx):
    z = np.asarray(Z, np.float64)
    p = np.exp(z - z.max(axis=1, keepdims=True))
    p = p / p.sum(axis=1, keepdims=True)
    return np.take_along_axis(p, np.asarray(idx, np.int64), axis=1)


def _silu_dropped_x(x):
    return 1.0 / (1.0 + np.exp(-x))


def _ffn_gate_up_swapped(x, Wg, Wu, Wd):
    return O.silu(np.asarray(x, np.float64) @ np.asarray(Wu, np.float64)) \
        * (np.asarray(x, np.float64) @ np.asarray(Wg, np.float64)) @ np.asarray(Wd, np.float64)


def _dsilu_dropped_term(a):
    return 1.0 / (1.0 + np.exp(-a))


def _softmax_bwd_sign(w, dg):
    return w * (dg + (w * dg).sum(axis=1, keepdims=True))


def _schedule_swapped_rows(A, L, c=0):
    Phi = _orig_sort_key(A, L, c)
    if len(Phi) > 1:
        Phi = Phi.copy()
        Phi[[0, 1]] = Phi[[1, 0]]
    return Phi


def _schedule_rank_major(A, L, c=0):
    """Orders a region by source rank before ordinal (no interleave)."""
    A = np.asarray(A, np.int64)
    rows = []
    for r in range(A.shape[0]):
        for j in range(A.shape[1]):
            if c * L <= A[r, j] < (c + 1) * L:
                rows.append((A[r, j] - c * L, r, j))
    rows.sort()
    return np.array([(r, j) for (_, r, j) in rows], np.int64).reshape(-1, 2)


_orig_sort_key = O.schedule_sort_key
_orig_backward = O.moe_backward


def _backward_unweighted_down(X, W_r, W, idx, w, dY):
    out = _orig_backward(X, W_r, W, idx, w, dY)
    # recompute dW_down without the router weight
    X64 = np.asarray(X, np.float64)
    for e in range(W["W_gate"].shape[0]):
        ts, _ = np.nonzero(np.asarray(idx) == e)
        if ts.size:
            h = O.silu(X64[ts] @ W["W_gate"][e]) * (X64[ts] @ W["W_up"][e])
            out["dW_down"][e] = h.T @ np.asarray(dY, np.float64)[ts]
    return out


def _backward_transposed_router(X, W_r, W, idx, w, dY):
    out = _orig_backward(X, W_r, W, idx, w, dY)
    out["dX"] = out["dX"] - out["dZ"] @ np.asarray(W_r, np.float64).T
    return out


PINS = [P.test_topk_exact_ties_golden, P.test_gate_weights_closed_forms,
        P.test_single_expert_is_plain_swiglu_ffn, P.test_k_equal_E_is_dense_softmax_mixture,
        P.test_identical_experts_ignore_routing, P.test_forward_matches_torch_layer_with_library_topk,
        P.test_backward_central_finite_differences, P.test_backward_matches_torch_autograd,
        P.test_algorithm1_hand_worked_two_ranks, P.test_plan_invariants_and_stable_sort,
        functools.partial(P.test_schedule_positions_follow_algorithm1_formula, 3, 4, 20, 3, 1),
        P.test_router_gradient_identity]


@pytest.mark.parametrize("name,replacement", [
    ("topk_select", _tie_high_index_wins),
    ("gate_weights", _weights_not_renormalised),
    ("silu", _silu_dropped_x),
    ("expert_ffn", _ffn_gate_up_swapped),
    ("_dsilu", _dsilu_dropped_term),
    ("softmax_restricted_backward", _softmax_bwd_sign),
    ("schedule_sort_key", _schedule_swapped_rows),
    ("schedule_sort_key", _schedule_rank_major),
    ("moe_backward", _backward_unweighted_down),
    ("moe_backward", _backward_transposed_router),
])
def test_planted_mistake_is_caught(monkeypatch, name, replacement):
    monkeypatch.setattr(O, name, replacement)
    failures = 0
    for pin in PINS:
        try:
            pin()
        except AssertionError:
            failures += 1
    assert failures >= 1, f"no pin caught the planted mistake in {name}"
