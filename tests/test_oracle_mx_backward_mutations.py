"""Plant plausible mistakes in the MXFP8 backward oracle and check that its
pins catch each one (CPU only; the mutated copy lives in this process)."""
import functools

import numpy as np
import pytest

from oracle import moe_oracle as O
from oracle import mx_oracle as M
import tests.test_oracle_mx_backward_pins as P

F64 = np.float64


def _qdq_padded(v, axis):
    """Quantise-dequantise along `axis`, zero-padding it to a multiple of 32
    (what blocks along a ragged token axis would need)."""
    v = np.asarray(v, F64)
    n = v.shape[axis]
    pad = (-n) % 32
    if pad:
        widths = [(0, 0)] * v.ndim
        widths[axis] = (0, pad)
        v = np.pad(v, widths)
    return np.take(M.mx_qdq(v, axis), np.arange(n), axis=axis)


def _variant(X, W_r, W, idx, w, dY, quant=True, dy_axis=1, wd_axis=1, da_axis=1, wg_axis=1,
             wgrad_x_quantised=False, wgrad_dy_quantised=False, quantise_dB=True, forward_quantised=True):
    """moe_backward_mx with one of its choices switchable."""
    qdq = _qdq_padded if quant else (lambda v, axis: np.asarray(v, F64))
    X = np.asarray(X, F64)
    dY = np.asarray(dY, F64)
    T, d = X.shape
    E, _, f = W["W_gate"].shape
    k = idx.shape[1]
    Xh = qdq(X, 1) if forward_quantised else X
    dYh = qdq(dY, dy_axis)
    dX = np.zeros((T, d))
    dWg = np.zeros((E, d, f))
    dWu = np.zeros((E, d, f))
    dWd = np.zeros((E, f, d))
    dg = np.zeros((T, k))
    for e in range(E):
        ts, ss = np.nonzero(np.asarray(idx) == e)
        if ts.size == 0:
            continue
        Wg, Wu, Wd = (np.asarray(W[key][e], F64) for key in ("W_gate", "W_up", "W_down"))
        fq = qdq if forward_quantised else (lambda v, axis: v)
        a = Xh[ts] @ fq(Wg, 0)
        b = Xh[ts] @ fq(Wu, 0)
        h = O.silu(a) * b
        we = np.asarray(w, F64)[ts, ss][:, None]
        dhp = dYh[ts] @ qdq(Wd, wd_axis).T
        dg[ts, ss] = (dhp * h).sum(axis=1)
        dh = we * dhp
        dA = dh * b * O._dsilu(a)
        dB = dh * O.silu(a)
        xw = Xh[ts] if wgrad_x_quantised else X[ts]
        dWg[e] = xw.T @ dA
        dWu[e] = xw.T @ dB
        dWd[e] = (we * h).T @ (dYh[ts] if wgrad_dy_quantised else dY[ts])
        dBq = qdq(dB, da_axis) if quantise_dB else dB
        np.add.at(dX, ts, qdq(dA, da_axis) @ qdq(Wg, wg_axis).T + dBq @ qdq(Wu, wg_axis).T)
    dz_sel = O.softmax_restricted_backward(np.asarray(w, F64), dg)
    dZ = np.zeros((T, W_r.shape[1]))
    np.put_along_axis(dZ, np.asarray(idx, np.int64), dz_sel, axis=1)
    dX += dZ @ np.asarray(W_r, F64).T
    out = dict(dX=dX, dW_gate=dWg, dW_up=dWu, dW_down=dWd, dW_r=X.T @ dZ, dZ=dZ, dg=dg,
               dWg_s=None, dWu_s=None, dWd_s=None)
    if W.get("Wg_s") is not None:
        ref = M.__dict__["_original_backward"](X, W_r, W, idx, w, dY, quant=quant)
        for key in ("dWg_s", "dWu_s", "dWd_s"):
            out[key] = ref[key]
        out["dX"] = out["dX"] + (ref["dX"] - _routed_only(X, W_r, W, idx, w, dY, quant))
    return out


def _routed_only(X, W_r, W, idx, w, dY, quant):
    W0 = dict(W, Wg_s=None, Wu_s=None, Wd_s=None)
    return M.__dict__["_original_backward"](X, W_r, W0, idx, w, dY, quant=quant)["dX"]


PINS = [P.test_without_quantisation_it_is_the_bf16_backward, P.test_power_of_two_equivariance_in_dY,
        P.test_dY_is_quantised_per_token_along_d, P.test_W_down_is_quantised_along_d,
        P.test_accuracy_under_wide_token_scales, P.test_accuracy_under_wide_weight_scales,
        P.test_close_to_the_bf16_backward, P.test_quantised_products_ignore_tiny_changes_of_their_inputs,
        P.test_weight_gradients_read_the_unquantised_X]

MUTANTS = {
    "dY_along_tokens": dict(dy_axis=0),
    "W_down_along_f": dict(wd_axis=0),
    "dA_dB_along_tokens": dict(da_axis=0),
    "W_gate_W_up_along_d": dict(wg_axis=0),
    "wgrad_on_quantised_X": dict(wgrad_x_quantised=True),
    "wgrad_on_quantised_dY": dict(wgrad_dy_quantised=True),
    "dB_unquantised": dict(quantise_dB=False),
    "forward_unquantised": dict(forward_quantised=False),
}


@pytest.fixture(autouse=True)
def _keep_original(monkeypatch):
    monkeypatch.setitem(M.__dict__, "_original_backward", M.moe_backward_mx)


def test_unmutated_variant_is_the_oracle():
    X, W_r, W, idx, wts, dY = P.layer(fs=64, seed=9)
    a = _variant(X, W_r, W, idx, wts, dY)
    b = M.moe_backward_mx(X, W_r, W, idx, wts, dY)
    for key in P.KEYS + ("dWg_s", "dWu_s", "dWd_s"):
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
