"""Pins of the opt-in MXFP8 weight gradients of the MXFP8 backward oracle
(CPU only).

With wgrad_mx the weight-gradient products read their operands quantised
along the token axis, in blocks of 32 consecutive plan positions that start
at each expert's first row.  The routing is an input of the oracle, so these
tests choose it.  They pin:

* the reduction to the BF16 backward with the quantiser switched off, and
  exact power-of-two equivariance in dY;
* blocks local to an expert: the rows of one expert, scaled by 2**6, leave
  another expert's gradients bit-identical although its last block is partial;
* the token axis for dY: a move below a quarter of its token-axis grid
  spacing leaves dW_down bit-identical, a move on the d-axis grid does not;
* flushing along tokens: in a block with one large row, rows far smaller
  contribute nothing (dY to dW_down; dA, dB and w h via tiny gate weights);
* X: only its quantised value enters the products (moves below a quarter of
  both grid spacings change nothing), and columns spread over 2**28 keep
  their rows' relative accuracy (blocks along tokens, not along d);
* closeness to the BF16 backward, and the sampled per-column evaluation.
"""
import numpy as np

from oracle import moe_oracle as O
from oracle import mx_oracle as M
from paper_2609_36070_amd.workloads import Workload, make_inputs

WG = ("dW_gate", "dW_up", "dW_down")


def layer(T=64, d=128, E=4, k=2, f=96, fs=0, seed=0):
    w = Workload("mxw", T=T, d=d, E=E, k=k, f=f, f_s=fs, bias_std=0.5, backward=True)
    inp = make_inputs(w, seed)
    Z = O.router_logits(inp["X"], inp["W_r"], inp["bias"])
    idx = O.topk_select(Z, k)
    wts = O.gate_weights(Z, idx)
    W = {key: inp[key] for key in ("W_gate", "W_up", "W_down", "Wg_s", "Wu_s", "Wd_s")}
    return inp["X"].astype(np.float64), inp["W_r"], W, idx, wts, inp["dY"].astype(np.float64)


def forced(T, n0, seed, d=64, f=64):
    """Two experts, k = 1: tokens 0 .. n0-1 on expert 0, the rest on expert 1,
    every gate weight 1."""
    X, W_r, W, _, _, dY = layer(T=T, d=d, E=2, k=1, f=f, seed=seed)
    idx = np.where(np.arange(T) < n0, 0, 1).astype(np.int32)[:, None]
    return X, W_r, W, idx, np.ones((T, 1)), dY


def bwd(X, W_r, W, idx, w, dY, **kw):
    return M.moe_backward_mx(X, W_r, W, idx, w, dY, wgrad_mx=True, **kw)


def test_token_block_quantiser_pads_with_zeros_and_keeps_columns_apart():
    rng = np.random.default_rng(0)
    v = rng.standard_normal((45, 64)) * np.exp2(rng.integers(-6, 6, (1, 64)))
    q = M.mx_qdq_token_blocks(v)
    # rows 32..44 form a block of their own, completed with zeros
    assert np.array_equal(q[32:], M.mx_qdq(np.vstack([v[32:], np.zeros((19, 64))]), 0)[:13])
    # a column does not see its neighbours
    v2 = v.copy()
    v2[:, 7] *= 2.0 ** 20
    q2 = M.mx_qdq_token_blocks(v2)
    assert np.array_equal(np.delete(q2, 7, axis=1), np.delete(q, 7, axis=1))
    assert M.mx_qdq_token_blocks(v[:0]).shape == (0, 64)


def test_without_quantisation_it_is_the_bf16_backward():
    X, W_r, W, idx, wts, dY = layer(fs=64, seed=1)
    a = bwd(X, W_r, W, idx, wts, dY, quant=False)
    b = O.moe_backward(X, W_r, W, idx, wts, dY)
    for key in WG:
        assert np.allclose(a[key], b[key], rtol=0, atol=1e-12 * np.abs(b[key]).max()), key


def test_power_of_two_equivariance_in_dY():
    X, W_r, W, idx, wts, dY = layer(fs=64, seed=2)
    base = bwd(X, W_r, W, idx, wts, dY)
    scaled = bwd(X, W_r, W, idx, wts, dY * 2.0 ** 5)
    for key in WG + ("dX", "dZ", "dW_r"):
        assert np.array_equal(scaled[key], base[key] * 2.0 ** 5), key


def test_blocks_restart_at_each_expert():
    """Expert 0 holds 33 tokens: its second block has one row.  Scaling the
    rows of expert 1 (its X and dY) by 2**6 leaves expert 0's weight
    gradients bit-identical; a block grid running across the expert boundary
    would flush expert 0's last row."""
    X, W_r, W, idx, wts, dY = forced(T=70, n0=33, seed=3)
    a = bwd(X, W_r, W, idx, wts, dY)
    X2, dY2 = X.copy(), dY.copy()
    X2[33:] *= 2.0 ** 6
    dY2[33:] *= 2.0 ** 6
    b = bwd(X2, W_r, W, idx, wts, dY2)
    for key in WG:
        assert np.array_equal(a[key][0], b[key][0]), key
        assert not np.array_equal(a[key][1], b[key][1]), key


def _grid_move(v, axis, rng):
    """v moved by under a quarter of its MX grid spacing along `axis`
    (blocks of 32 from index 0), block maxima kept; v itself is first put on
    that grid."""
    q, sc = M.mx_quantize(v, axis)
    r = M.mx_dequantize(q, sc, axis)
    blocks = np.moveaxis(r, axis, -1)
    scale = np.repeat(np.exp2(np.moveaxis(sc.astype(float), axis, -1) - 127), 32, axis=-1)
    s = np.abs(blocks) / scale
    ulp = np.where(s >= 2.0 ** -6, np.exp2(np.floor(np.log2(np.maximum(s, 1e-300))) - 3), 2.0 ** -9) * scale
    moved = blocks + rng.uniform(-0.25, 0.25, blocks.shape) * ulp
    bmax = np.abs(blocks).reshape(blocks.shape[:-1] + (-1, 32)).max(axis=-1)
    moved = np.where(np.abs(blocks) == np.repeat(bmax, 32, axis=-1), blocks, moved)
    return np.moveaxis(blocks, -1, axis), np.moveaxis(moved, -1, axis)


def test_dY_enters_dW_down_along_tokens():
    """One expert of 64 tokens (two token blocks).  On dY's token-axis grid,
    sub-ulp moves leave dW_down bit-identical; on its d-axis grid they leave
    everything read through Q_d(dY) bit-identical and move dW_down."""
    rng = np.random.default_rng(4)
    X, W_r, W, idx, wts, dY = forced(T=64, n0=64, seed=4)
    on_t, moved_t = _grid_move(dY, 0, rng)
    a, b = bwd(X, W_r, W, idx, wts, on_t), bwd(X, W_r, W, idx, wts, moved_t)
    assert np.array_equal(a["dW_down"], b["dW_down"])
    on_d, moved_d = _grid_move(dY, 1, rng)
    a, b = bwd(X, W_r, W, idx, wts, on_d), bwd(X, W_r, W, idx, wts, moved_d)
    for key in ("dX", "dZ", "dW_gate", "dW_up"):
        assert np.array_equal(a[key], b[key]), key
    assert not np.array_equal(a["dW_down"], b["dW_down"])


def test_tiny_dY_rows_flush_out_of_dW_down():
    """dY rows 1..31 of a block at least 2**20 below row 0 in every column
    (row 0 at 2**12 throughout) quantise to zero along the token axis: dW_down
    equals the one with those rows zeroed (w h does not depend on dY)."""
    X, W_r, W, idx, wts, dY = forced(T=32, n0=32, seed=5)
    dY = dY.copy()
    dY[0] = np.where(dY[0] < 0, -1.0, 1.0) * 2.0 ** 12
    dY[1:] *= 2.0 ** -12
    zeroed = dY.copy()
    zeroed[1:] = 0.0
    a, b = bwd(X, W_r, W, idx, wts, dY), bwd(X, W_r, W, idx, wts, zeroed)
    assert np.array_equal(a["dW_down"], b["dW_down"])
    assert np.abs(a["dW_down"]).max() > 0


def test_tiny_gate_weights_flush_dA_dB_and_wh():
    """Gate weights 2**-40 on tokens 1..31 scale their dA, dB and w h rows
    down by 2**40 against token 0's: along the token axis they quantise to
    zero, so the weight gradients equal those with these gate weights 0."""
    X, W_r, W, idx, _, dY = forced(T=32, n0=32, seed=6)
    w_tiny = np.full((32, 1), 2.0 ** -40)
    w_tiny[0] = 1.0
    w_zero = np.where(np.arange(32)[:, None] == 0, 1.0, 0.0)
    a, b = bwd(X, W_r, W, idx, w_tiny, dY), bwd(X, W_r, W, idx, w_zero, dY)
    for key in WG:
        assert np.array_equal(a[key], b[key]), key
        assert np.abs(a[key]).max() > 0, key


def test_only_the_quantised_X_enters_the_products():
    """X of powers of two in [2**-4, 2**4], with a 2**4 in every 32-block of
    either axis (column t mod 32 of token t), lies on both of its MX grids,
    and moving every other entry by 2**-6 of itself stays below a quarter of
    the grid spacing on both.  The forward and every weight gradient stay
    bit-identical, while weight gradients on the raw X move."""
    rng = np.random.default_rng(9)
    X, W_r, W, idx, wts, dY = forced(T=32, n0=32, seed=9)
    T, d = X.shape
    X = np.exp2(rng.integers(-4, 4, (T, d))) * np.where(rng.random((T, d)) < 0.5, -1.0, 1.0)
    peak = (np.arange(d)[None, :] % 32) == (np.arange(T)[:, None] % 32)
    X = np.where(peak, 2.0 ** 4, X)
    X2 = np.where(peak, X, X * (1 + 2.0 ** -6))
    a, b = bwd(X, W_r, W, idx, wts, dY), bwd(X2, W_r, W, idx, wts, dY)
    for key in WG + ("dX", "dZ", "dg"):
        assert np.array_equal(a[key], b[key]), key
    # the move is real: weight gradients on the raw X (the default) see it
    a0 = M.moe_backward_mx(X, W_r, W, idx, wts, dY)
    b0 = M.moe_backward_mx(X2, W_r, W, idx, wts, dY)
    assert not np.array_equal(a0["dW_gate"], b0["dW_gate"])


def test_accuracy_under_wide_column_scales():
    """Columns of X (the d index) spread over 2**28 (the largest of order 1, so
    the forward stays in range): every row of dW_gate and
    dW_up keeps its own relative accuracy against the fp64 BF16 backward, since
    the weight gradients read X in blocks along tokens.  Blocks along d would
    flush the small columns' rows."""
    X, W_r, W, idx, wts, dY = layer(T=128, seed=11)
    d = X.shape[1]
    X = X * np.exp2(4.0 * (np.arange(d) % 8) - 28.0)[None, :]
    ref = O.moe_backward(X, W_r, W, idx, wts, dY)
    mx = bwd(X, W_r, W, idx, wts, dY)
    for key in ("dW_gate", "dW_up"):
        for e in range(W["W_gate"].shape[0]):
            err = np.abs(mx[key][e] - ref[key][e]).max(axis=1)
            scale = np.abs(ref[key][e]).max(axis=1)
            ok = scale > 0
            assert (err[ok] / scale[ok]).max() < 0.35, (key, e)


def test_close_to_the_bf16_backward():
    X, W_r, W, idx, wts, dY = layer(T=256, fs=64, seed=7)
    ref = O.moe_backward(X, W_r, W, idx, wts, dY)
    mx = bwd(X, W_r, W, idx, wts, dY)
    for key in WG:
        rel = np.abs(mx[key] - ref[key]).max() / np.abs(ref[key]).max()
        assert 1e-4 < rel < 0.2, (key, rel)            # quantised, but close
    base = M.moe_backward_mx(X, W_r, W, idx, wts, dY)
    for key in ("dX", "dZ", "dg", "dW_r", "dWg_s", "dWu_s", "dWd_s"):
        assert np.array_equal(mx[key], base[key]), key  # only the weight gradients change


def test_sampled_columns_match_the_full_backward():
    X, W_r, W, idx, wts, dY = layer(fs=64, seed=8)
    full = bwd(X, W_r, W, idx, wts, dY)
    cols = np.array([0, 33, 95])
    for e in range(W["W_gate"].shape[0]):
        a, b, c = M.mx_expert_weight_grad_columns(X, W, idx, wts, dY, e, cols, wgrad_mx=True)
        for got, ref in ((a, full["dW_gate"][e][:, cols]), (b, full["dW_up"][e][:, cols]),
                         (c, full["dW_down"][e][cols, :])):
            assert np.allclose(got, ref, rtol=0, atol=1e-12 * max(np.abs(ref).max(), 1e-30))
