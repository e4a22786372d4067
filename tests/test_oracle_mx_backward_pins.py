"""Pins of the MXFP8 backward oracle (CPU only).

The MXFP8 backward is the BF16 backward with some operands passed through
the microscaling quantiser.  It is pinned against:

* the BF16 backward itself, reached by switching the quantiser off;
* power-of-two equivariance in dY: scaling dY by 2**s scales every gradient
  by exactly 2**s;
* sensitivity to the quantisation axes: moving dY or W_down by less than a
  quarter of their own MX grid spacing (block maxima kept) leaves the outputs
  computed from their quantised values bit-identical, and the weight
  gradients computed from the raw dY change;
* accuracy under wide scales: token rows of dY, or rows of W_gate / W_up
  (the d index), spread over 2**24 keep every row or column of dX within
  tens of per cent of the fp64 BF16 backward.  A block that ran across the
  scales would flush the small ones to zero.
"""
import numpy as np

from oracle import moe_oracle as O
from oracle import mx_oracle as M
from paper_2609_36070_amd.workloads import Workload, make_inputs

KEYS = ("dX", "dW_gate", "dW_up", "dW_down", "dW_r", "dZ", "dg")


def layer(T=64, d=128, E=4, k=2, f=96, fs=0, seed=0):
    w = Workload("mxb", T=T, d=d, E=E, k=k, f=f, f_s=fs, bias_std=0.5, backward=True)
    inp = make_inputs(w, seed)
    Z = O.router_logits(inp["X"], inp["W_r"], inp["bias"])
    idx = O.topk_select(Z, k)
    wts = O.gate_weights(Z, idx)
    W = {key: inp[key] for key in ("W_gate", "W_up", "W_down", "Wg_s", "Wu_s", "Wd_s")}
    return inp["X"].astype(np.float64), inp["W_r"], W, idx, wts, inp["dY"].astype(np.float64)


def test_without_quantisation_it_is_the_bf16_backward():
    X, W_r, W, idx, wts, dY = layer(fs=64, seed=1)
    a = M.moe_backward_mx(X, W_r, W, idx, wts, dY, quant=False)
    b = O.moe_backward(X, W_r, W, idx, wts, dY)
    for key in KEYS + ("dWg_s", "dWu_s", "dWd_s"):
        assert np.allclose(a[key], b[key], rtol=0, atol=1e-12 * np.abs(b[key]).max()), key


def test_power_of_two_equivariance_in_dY():
    X, W_r, W, idx, wts, dY = layer(fs=64, seed=2)
    base = M.moe_backward_mx(X, W_r, W, idx, wts, dY)
    scaled = M.moe_backward_mx(X, W_r, W, idx, wts, dY * 2.0 ** 5)
    for key in KEYS + ("dWg_s", "dWu_s", "dWd_s"):
        assert np.array_equal(scaled[key], base[key] * 2.0 ** 5), key


def _sub_ulp(v, axis, rng):
    """v on its MX grid, and v moved by at most a quarter of its own grid
    spacing with every block maximum kept (so neither codes nor scales move)."""
    q, sc = M.mx_quantize(v, axis)
    r = M.mx_dequantize(q, sc, axis)
    blocks = np.moveaxis(r, axis, -1)
    scale = np.repeat(np.exp2(np.moveaxis(sc.astype(float), axis, -1) - 127), 32, axis=-1)
    s = np.abs(blocks) / scale
    ulp = np.where(s >= 2.0 ** -6, np.exp2(np.floor(np.log2(np.maximum(s, 1e-300))) - 3), 2.0 ** -9) * scale
    moved = blocks + rng.uniform(-0.25, 0.25, blocks.shape) * ulp
    bmax = np.abs(blocks).reshape(blocks.shape[:-1] + (-1, 32)).max(axis=-1)
    keep = np.abs(blocks) == np.repeat(bmax, 32, axis=-1)
    moved = np.where(keep, blocks, moved)
    return np.moveaxis(blocks, -1, axis), np.moveaxis(moved, -1, axis)


def test_dY_is_quantised_per_token_along_d():
    rng = np.random.default_rng(3)
    X, W_r, W, idx, wts, dY = layer(seed=3)
    dYg, dYp = _sub_ulp(dY, 1, rng)
    a = M.moe_backward_mx(X, W_r, W, idx, wts, dYg)
    b = M.moe_backward_mx(X, W_r, W, idx, wts, dYp)
    for key in ("dX", "dW_gate", "dW_up", "dW_r", "dZ", "dg"):
        assert np.array_equal(a[key], b[key]), key          # all through Q(dY)
    assert not np.array_equal(a["dW_down"], b["dW_down"])   # the raw dY


def test_W_down_is_quantised_along_d():
    rng = np.random.default_rng(4)
    X, W_r, W, idx, wts, dY = layer(seed=4)
    Wg, Wp = dict(W), dict(W)
    Wg["W_down"], Wp["W_down"] = _sub_ulp(np.asarray(W["W_down"], np.float64), 2, rng)
    a = M.moe_backward_mx(X, W_r, Wg, idx, wts, dY)
    b = M.moe_backward_mx(X, W_r, Wp, idx, wts, dY)
    for key in KEYS:
        assert np.array_equal(a[key], b[key]), key


def test_quantised_products_ignore_tiny_changes_of_their_inputs():
    """A 2**-30 relative change of the gate weights moves dA and dB by far less
    than their MX grid spacing: the routed dX (computed from Q(dA), Q(dB))
    stays bit-identical, while the weight gradients (raw dA, dB) move.  W_r is
    zeroed after routing, so dX holds the routed terms alone."""
    X, W_r, W, idx, wts, dY = layer(seed=10)
    W_r0 = np.zeros_like(np.asarray(W_r, np.float64))
    a = M.moe_backward_mx(X, W_r0, W, idx, wts, dY)
    b = M.moe_backward_mx(X, W_r0, W, idx, wts * (1 + 2.0 ** -30), dY)
    assert np.array_equal(a["dX"], b["dX"])
    for key in ("dW_gate", "dW_up", "dW_down"):
        assert not np.array_equal(a[key], b[key]), key


def test_weight_gradients_read_the_unquantised_X():
    """Moving X by less than a quarter of its MX grid spacing changes nothing
    computed from Q(X) (the forward pre-activations, hence dg, dZ, dW_down and
    the routed dX), but changes dW_gate, dW_up and dW_r, which read X itself."""
    rng = np.random.default_rng(11)
    X, W_r, W, idx, wts, dY = layer(seed=11)
    W_r0 = np.zeros_like(np.asarray(W_r, np.float64))
    Xg, Xp = _sub_ulp(X, 1, rng)
    a = M.moe_backward_mx(Xg, W_r0, W, idx, wts, dY)
    b = M.moe_backward_mx(Xp, W_r0, W, idx, wts, dY)
    for key in ("dg", "dZ", "dW_down", "dX"):
        assert np.array_equal(a[key], b[key]), key
    for key in ("dW_gate", "dW_up", "dW_r"):
        assert not np.array_equal(a[key], b[key]), key


def _rel_rows(got, ref, axis):
    err = np.abs(got - ref).max(axis=axis)
    return err / np.maximum(np.abs(ref).max(axis=axis), 1e-300)


def test_accuracy_under_wide_token_scales():
    X, W_r, W, idx, wts, dY = layer(seed=5)
    dY = dY * np.exp2(4.0 * (np.arange(dY.shape[0]) % 7))[:, None]
    ref = O.moe_backward(X, W_r, W, idx, wts, dY)
    mx = M.moe_backward_mx(X, W_r, W, idx, wts, dY)
    assert _rel_rows(mx["dX"], ref["dX"], 1).max() < 0.35          # every token row


def test_accuracy_under_wide_weight_scales():
    """Rows of W_gate and W_up (the d index) spread over 2**24: every column of
    dX keeps its own relative accuracy, since dX reads each weight row as its
    own blocks (along f).  Blocks across rows would flush the small rows."""
    X, W_r, W, idx, wts, dY = layer(seed=6)
    W = dict(W)
    d = W["W_gate"].shape[1]
    row_scale = np.exp2(4.0 * (np.arange(d) % 7) - 24.0)[None, :, None]
    W["W_gate"] = W["W_gate"] * row_scale
    W["W_up"] = W["W_up"] * row_scale
    ref = O.moe_backward(X, W_r, W, idx, wts, dY)
    mx = M.moe_backward_mx(X, W_r, W, idx, wts, dY)
    routed = mx["dX"] - mx["dZ"] @ np.asarray(W_r, np.float64).T
    routed_ref = ref["dX"] - ref["dZ"] @ np.asarray(W_r, np.float64).T
    assert _rel_rows(routed, routed_ref, 0).max() < 0.35


def test_close_to_the_bf16_backward():
    X, W_r, W, idx, wts, dY = layer(fs=64, seed=7)
    ref = O.moe_backward(X, W_r, W, idx, wts, dY)
    mx = M.moe_backward_mx(X, W_r, W, idx, wts, dY)
    for key in ("dX", "dW_gate", "dW_up", "dW_down"):
        rel = np.abs(mx[key] - ref[key]).max() / np.abs(ref[key]).max()
        assert 1e-4 < rel < 0.15, (key, rel)            # quantised, but close
    for key in ("dWg_s", "dWu_s", "dWd_s"):
        assert np.array_equal(mx[key], ref[key]), key   # the shared expert stays BF16


def test_sampled_evaluation_matches_the_full_backward():
    """The per-token and per-column evaluations used at full size give the
    full MXFP8 backward's rows and columns."""
    X, W_r, W, idx, wts, dY = layer(fs=64, seed=12)
    full = M.moe_backward_mx(X, W_r, W, idx, wts, dY)
    toks = np.array([0, 5, 17, 63])
    dX, dZ, dg = M.mx_token_backward(X, W_r, W, idx, wts, dY, toks)
    for name, got, ref in (("dX", dX, full["dX"][toks]), ("dZ", dZ, full["dZ"][toks]),
                           ("dg", dg, full["dg"][toks])):
        assert np.allclose(got, ref, rtol=0, atol=1e-12 * np.abs(ref).max()), name
    cols = np.array([0, 33, 95])
    for e in range(W["W_gate"].shape[0]):
        a, b, c = M.mx_expert_weight_grad_columns(X, W, idx, wts, dY, e, cols)
        for got, ref in ((a, full["dW_gate"][e][:, cols]), (b, full["dW_up"][e][:, cols]),
                         (c, full["dW_down"][e][cols, :])):
            assert np.allclose(got, ref, rtol=0, atol=1e-12 * max(np.abs(ref).max(), 1e-30))
