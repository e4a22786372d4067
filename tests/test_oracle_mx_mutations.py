"""Plant plausible mistakes in the MXFP8 oracle and check that its pins catch them.

Each case swaps one piece of oracle/mx_oracle.py for a subtly wrong copy (on
the CPU, in this process only) and asserts that at least one pin of
tests/test_oracle_mx_pins.py then fails.
"""
import functools

import numpy as np
import pytest

from oracle import moe_oracle as O
from oracle import mx_oracle as M
import tests.test_oracle_mx_pins as P

_orig_round = M.e4m3_round


def _round_truncating(x):
    x = np.asarray(x, np.float64)
    a = np.abs(x)
    _, ex = np.frexp(np.where(a > 0, a, 1.0))
    e = np.maximum(ex - 1, M.E4M3_EMIN)
    m = np.floor(a / np.exp2(e - 3.0))
    return _orig_round(np.sign(x) * m * np.exp2(e - 3.0))


def _round_ties_away(x):
    x = np.asarray(x, np.float64)
    a = np.abs(x)
    _, ex = np.frexp(np.where(a > 0, a, 1.0))
    e = np.maximum(ex - 1, M.E4M3_EMIN)
    m = np.floor(a / np.exp2(e - 3.0) + 0.5)
    return _orig_round(np.where(x < 0, -1.0, 1.0) * m * np.exp2(e - 3.0))


def _round_not_saturating(x):
    codes = _orig_round(x)
    big = np.abs(np.asarray(x, np.float64)) > 448
    return np.where(big, codes | 0x7F, codes).astype(np.uint8)     # NaN pattern


def _scale_rounded_up(amax):
    amax = np.asarray(amax, np.float64)
    se = np.ceil(np.log2(np.where(amax > 0, amax, 1.0) / 448.0))
    return np.clip(np.where(amax > 0, se, -127), -127, 127).astype(np.int64)


def _forward_variant(X, W, idx, w, x_axis=1, wg_axis=1, wd_axis=1, h_axis=1, quant_x=True,
                     quant_wd=True):
    X = np.asarray(X, np.float64)
    T, d = X.shape
    E = W["W_gate"].shape[0]
    k = idx.shape[1]
    counts, offsets, perm, route_pos = O.plan(idx, E)
    tok = perm // k
    Xh = M.mx_qdq(X, axis=x_axis) if quant_x else X
    Wg = M.mx_qdq(W["W_gate"], axis=wg_axis)
    Wu = M.mx_qdq(W["W_up"], axis=1)
    Wd = M.mx_qdq(W["W_down"], axis=wd_axis) if quant_wd else np.asarray(W["W_down"], np.float64)
    f = W["W_gate"].shape[2]
    H = np.zeros((T * k, f))
    for e in range(E):
        rows = slice(offsets[e], offsets[e + 1])
        H[rows] = O.silu(Xh[tok[rows]] @ Wg[e]) * (Xh[tok[rows]] @ Wu[e])
    Hq = M.mx_qdq(H, axis=h_axis)
    Yexp = np.zeros((T * k, d))
    for e in range(E):
        rows = slice(offsets[e], offsets[e + 1])
        Yexp[rows] = Hq[rows] @ Wd[e]
    Y = np.zeros((T, d))
    if W.get("Wg_s") is not None:
        Y += O.expert_ffn(X, W["Wg_s"], W["Wu_s"], W["Wd_s"])
    for s in range(k):
        Y += w[:, s:s + 1] * Yexp[route_pos[np.arange(T) * k + s]]
    return dict(Y=Y)


PINS = [P.test_e4m3_decode_closed_forms, P.test_e4m3_round_matches_exhaustive_search,
        lambda: [P.test_shared_exponent_closed_form(a, e) for a, e in
                 [(1.0, -8), (1.999, -8), (448.0, 0), (511.0, 0), (512.0, 1), (0.0, -127)]],
        P.test_round_trip_is_exact_on_the_grid, P.test_error_bound_of_the_definition,
        P.test_blocks_run_along_the_given_axis,
        P.test_layer_close_to_fp64_under_wide_row_and_column_scales,
        P.test_every_routed_operand_is_quantized_along_its_axis,
        P.test_layer_output_is_power_of_two_equivariant_in_w_down]


@pytest.mark.parametrize("name,replacement", [
    ("E4M3_EMAX", 7),
    ("e4m3_round", _round_truncating),
    ("e4m3_round", _round_ties_away),
    ("e4m3_round", _round_not_saturating),
    ("shared_exponent", _scale_rounded_up),
    ("moe_forward_mx", functools.partial(_forward_variant, wg_axis=2)),
    ("moe_forward_mx", functools.partial(_forward_variant, wd_axis=2)),
    ("moe_forward_mx", functools.partial(_forward_variant, h_axis=0)),
    ("moe_forward_mx", functools.partial(_forward_variant, quant_x=False)),
    ("moe_forward_mx", functools.partial(_forward_variant, quant_wd=False)),
], ids=["emax7", "truncate", "ties_away", "no_saturation", "scale_ceil", "w_gate_axis",
        "w_down_axis", "h_axis", "x_unquantised", "w_down_unquantised"])
def test_planted_mistake_is_caught(monkeypatch, name, replacement):
    monkeypatch.setattr(M, name, replacement)
    failures = 0
    for pin in PINS:
        try:
            with np.errstate(all="ignore"):
                pin()
        except AssertionError:
            failures += 1
    assert failures >= 1, f"no pin caught the planted mistake in {name}"


def test_unmutated_oracle_passes_every_pin():
    with np.errstate(all="ignore"):
        for pin in PINS:
            pin()
