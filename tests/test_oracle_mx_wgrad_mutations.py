"""Plant plausible mistakes in the opt-in MXFP8 weight gradients of the
MXFP8 backward oracle and check that its pins catch each one (CPU only; the
mutated copy lives in this process).  The mutants change only the weight
gradients; everything else comes from the unmutated oracle."""
import functools

import numpy as np
import pytest

from oracle import moe_oracle as O
from oracle import mx_oracle as M
import tests.test_oracle_mx_wgrad_pins as P

F64 = np.float64


def _along(v, axis):
    """Round trip in blocks of 32 along `axis`, zero-padded."""
    v = np.asarray(v, F64)
    n = v.shape[axis]
    pad = (-n) % 32
    if pad:
        widths = [(0, 0)] * v.ndim
        widths[axis] = (0, pad)
        v = np.pad(v, widths)
    return np.take(M.mx_qdq(v, axis), np.arange(n), axis=axis)


def _variant(X, W_r, W, idx, w, dY, quant=True, wgrad_mx=False, grid="expert", x_axis=0, dy_axis=0,
             quant_x=True, quant_dy=True, quant_da=True, quant_wh=True):
    orig = M.__dict__["_original_backward"]
    out = orig(X, W_r, W, idx, w, dY, quant=quant, wgrad_mx=False)
    if not (quant and wgrad_mx):
        return out
    X = np.asarray(X, F64)
    dY = np.asarray(dY, F64)
    E = W["W_gate"].shape[0]
    Xh, dYh = M.mx_qdq(X, 1), M.mx_qdq(dY, 1)
    parts = []
    for e in range(E):
        ts, ss = np.nonzero(np.asarray(idx) == e)
        Wg, Wu, Wd = (np.asarray(W[key][e], F64) for key in ("W_gate", "W_up", "W_down"))
        a = Xh[ts] @ M.mx_qdq(Wg, 0)
        b = Xh[ts] @ M.mx_qdq(Wu, 0)
        h = O.silu(a) * b
        we = np.asarray(w, F64)[ts, ss][:, None]
        dh = we * (dYh[ts] @ M.mx_qdq(Wd, 1).T)
        dA = dh * b * O._dsilu(a)
        dB = dh * O.silu(a)
        parts.append(dict(x=X[ts], dy=dY[ts], da=dA, db=dB, wh=we * h))

    def tq(name, axis=0, on=True):
        """The operand `name` of every expert after its weight-gradient quantiser."""
        if not on:
            return [pt[name] for pt in parts]
        if axis == 1:
            return [_along(pt[name], 1) if len(pt[name]) else pt[name] for pt in parts]
        if grid == "global":     # one 32-row grid over all plan positions
            allv = np.concatenate([pt[name] for pt in parts], axis=0)
            q = _along(allv, 0)
            cut = np.cumsum([0] + [len(pt[name]) for pt in parts])
            return [q[cut[i]:cut[i + 1]] for i in range(E)]
        return [M.mx_qdq_token_blocks(pt[name]) for pt in parts]

    xs, dys = tq("x", x_axis, quant_x), tq("dy", dy_axis, quant_dy)
    das, dbs, whs = tq("da", 0, quant_da), tq("db", 0, quant_da), tq("wh", 0, quant_wh)
    for e in range(E):
        out["dW_gate"][e] = xs[e].T @ das[e]
        out["dW_up"][e] = xs[e].T @ dbs[e]
        out["dW_down"][e] = whs[e].T @ dys[e]
    return out


PINS = [P.test_without_quantisation_it_is_the_bf16_backward, P.test_power_of_two_equivariance_in_dY,
        P.test_blocks_restart_at_each_expert, P.test_dY_enters_dW_down_along_tokens,
        P.test_tiny_dY_rows_flush_out_of_dW_down, P.test_tiny_gate_weights_flush_dA_dB_and_wh,
        P.test_only_the_quantised_X_enters_the_products, P.test_accuracy_under_wide_column_scales,
        P.test_close_to_the_bf16_backward]

MUTANTS = {
    "blocks_across_experts": dict(grid="global"),
    "X_along_d": dict(x_axis=1),
    "dY_along_d": dict(dy_axis=1),
    "X_unquantised": dict(quant_x=False),
    "dY_unquantised": dict(quant_dy=False),
    "dA_dB_unquantised": dict(quant_da=False),
    "wh_unquantised": dict(quant_wh=False),
}


@pytest.fixture(autouse=True)
def _keep_original(monkeypatch):
    monkeypatch.setitem(M.__dict__, "_original_backward", M.moe_backward_mx)


def test_unmutated_variant_is_the_oracle():
    X, W_r, W, idx, wts, dY = P.layer(fs=64, seed=10)
    a = _variant(X, W_r, W, idx, wts, dY, wgrad_mx=True)
    b = M.moe_backward_mx(X, W_r, W, idx, wts, dY, wgrad_mx=True)
    for key in P.WG + ("dX", "dZ", "dWg_s"):
        assert np.allclose(a[key], b[key], rtol=0, atol=1e-12 * np.abs(b[key]).max()), key


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_planted_mistake_is_caught(monkeypatch, name):
    monkeypatch.setattr(M, "moe_backward_mx", functools.partial(_variant, **MUTANTS[name]))
    failures = 0
    for pin in PINS:
        try:
            with np.errstate(all="ignore"):
                pin()
        except AssertionError:
            failures += 1
    assert failures >= 1, f"no pin caught {name}"
