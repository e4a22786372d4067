"""Pins of the MXFP8 oracle against facts that do not come from it (CPU only).

The E4M3 grid and the microscaling rule are fixed by their definitions; the
oracle's arithmetic rounding is checked against a nearest-value search over
the decode table, its scales against closed forms, and the layer against the
fp64 layer and against perturbations that must not change any code.
"""
import math

import numpy as np
import pytest

from oracle import moe_oracle as O
from oracle import mx_oracle as M
from paper_2609_36070_amd.workloads import Workload, make_inputs


def table():
    codes = np.arange(256)
    return codes, M.e4m3_value(codes)


def brute_round(v):
    """Nearest finite E4M3 value by exhaustive search; ties to the even code;
    magnitudes above 448 saturate."""
    codes, vals = table()
    finite = ~np.isnan(vals)
    out = np.empty(len(v), np.uint8)
    for i, x in enumerate(v):
        if abs(x) > 448:
            out[i] = 0x7E | (0x80 if x < 0 else 0)
            continue
        # codes of x's own sign (a negative value that rounds to zero is -0)
        cand = codes[finite & ((codes >> 7) == (1 if np.signbit(x) else 0))]
        cv = M.e4m3_value(cand)
        dist = np.abs(cv - x)
        best = dist.min()
        tied = cand[dist == best]
        # among equal distances: the code with an even mantissa (ties to even)
        even = [c for c in tied if c % 2 == 0]
        out[i] = min(even) if even else min(tied)
    return out


def test_e4m3_decode_closed_forms():
    assert M.e4m3_value(0x00) == 0.0
    assert M.e4m3_value(0x01) == 2.0 ** -9          # smallest subnormal
    assert M.e4m3_value(0x07) == 7 * 2.0 ** -9      # largest subnormal
    assert M.e4m3_value(0x08) == 2.0 ** -6          # smallest normal
    assert M.e4m3_value(0x38) == 1.0
    assert M.e4m3_value(0x3F) == 1.875
    assert M.e4m3_value(0x7E) == 448.0              # largest finite
    assert np.isnan(M.e4m3_value(0x7F)) and np.isnan(M.e4m3_value(0xFF))
    assert M.e4m3_value(0xB8) == -1.0
    pos = M.e4m3_value(np.arange(0x01, 0x7F))
    assert len(pos) == 126 and np.all(np.diff(pos) > 0)            # strictly increasing
    assert np.array_equal(M.e4m3_value(np.arange(0x80, 0xFF)), -M.e4m3_value(np.arange(0, 0x7F)))


def test_e4m3_round_matches_exhaustive_search():
    rng = np.random.default_rng(0)
    mags = np.exp2(rng.uniform(-12, 9.5, 3000))
    v = mags * rng.choice([-1, 1], mags.size)
    _, vals = table()
    pos = np.sort(vals[(vals > 0) & ~np.isnan(vals)])
    mids = (pos[1:] + pos[:-1]) / 2                    # exact ties between neighbours
    extra = np.concatenate([mids, -mids, [pos[0] / 2, 0.0, 448.0, 464.0, 470.0, 479.9, 480.0,
                                          500.0, 1e4, -1e4, 2.0 ** -10, 3 * 2.0 ** -11]])
    v = np.concatenate([v, extra])
    assert np.array_equal(M.e4m3_round(v), brute_round(v))


@pytest.mark.parametrize("amax,expect", [
    (1.0, -8), (1.5, -8), (1.999, -8), (2.0, -7), (448.0, 0), (511.0, 0), (512.0, 1),
    (2.0 ** -6, -14), (3.0 * 2.0 ** 20, 13), (2.0 ** -200, -127), (2.0 ** 200, 127), (0.0, -127),
])
def test_shared_exponent_closed_form(amax, expect):
    assert int(M.shared_exponent(amax)) == expect
    if 0 < amax < 2.0 ** 100 and amax > 2.0 ** -100:
        assert math.floor(math.log2(amax)) - 8 == expect


def test_round_trip_is_exact_on_the_grid():
    """Blocks of E4M3 values times 2**s whose maximum lies in [256, 448] * 2**s:
    the scale is exactly 2**s and the round trip is the identity."""
    rng = np.random.default_rng(1)
    blocks, exps = [], []
    for _ in range(200):
        s = int(rng.integers(-30, 30))
        codes = rng.integers(0, 0x7F, 32)
        codes[0] = rng.integers(0x78, 0x7F)
        signs = rng.choice([-1.0, 1.0], 32)
        blocks.append(signs * M.e4m3_value(codes) * 2.0 ** s)
        exps.append(s)
    v = np.stack(blocks)
    q, sc = M.mx_quantize(v, axis=1)
    assert np.array_equal(sc[:, 0].astype(int) - 127, np.array(exps))
    assert np.array_equal(M.mx_dequantize(q, sc, axis=1), v)


def test_error_bound_of_the_definition():
    rng = np.random.default_rng(2)
    v = rng.standard_normal((64, 256)) * np.exp2(rng.integers(-20, 20, (64, 1)))
    q, sc = M.mx_quantize(v, axis=1)
    r = M.mx_dequantize(q, sc, axis=1)
    X = np.repeat(np.exp2(sc.astype(float) - 127), 32, axis=1)       # block scale per element
    s = np.abs(v) / X                                                  # scaled magnitude
    clamped = s > 448
    half_ulp = np.where(s >= 2.0 ** -6, np.exp2(np.floor(np.log2(np.maximum(s, 1e-300))) - 4),
                        2.0 ** -10) * X
    err = np.abs(r - v)
    assert np.all(err[~clamped] <= half_ulp[~clamped])
    assert np.all(err[clamped] <= 64 * X[clamped])
    assert np.all(np.abs(v).reshape(64, 8, 32).max(axis=2) / np.exp2(sc.astype(float) - 127) >= 256)


def test_blocks_run_along_the_given_axis():
    """Columns whose scales differ by 2**4 apart: blocks along axis 0 keep every
    element to 1/16 relative; blocks across columns would flush small ones."""
    rng = np.random.default_rng(3)
    W = rng.uniform(1.0, 1.75, (64, 16)) * np.exp2(4.0 * np.arange(16))
    r = M.mx_qdq(W, axis=0)
    assert np.all(np.abs(r - W) <= W / 16)
    assert np.max(np.abs(M.mx_qdq(W.T, axis=1).T - W) / W) <= 1 / 16


def _layer(T=64, d=128, E=4, k=2, f=96, seed=0, fs=0):
    w = Workload("mx", T=T, d=d, E=E, k=k, f=f, f_s=fs, bias_std=0.5)
    inp = make_inputs(w, seed)
    Z = O.router_logits(inp["X"], inp["W_r"], inp["bias"])
    idx = O.topk_select(Z, k)
    wts = O.gate_weights(Z, idx)
    W = {key: inp[key] for key in ("W_gate", "W_up", "W_down", "Wg_s", "Wu_s", "Wd_s")}
    return inp["X"].astype(np.float64), W, idx, wts


def test_layer_close_to_fp64_under_wide_row_and_column_scales():
    """Token rows and weight columns spread over 2**24: with every tensor
    blocked along its own contraction axis, each output row stays within a
    few tens of per cent of its own magnitude (a saturated block maximum
    alone loses 1/8).  A block running across rows or columns would flush
    whole rows or columns to zero instead."""
    X, W, idx, wts = _layer(d=128, f=96)
    T = X.shape[0]
    X = X * np.exp2(4.0 * (np.arange(T) % 7))[:, None]
    W = dict(W)
    W["W_gate"] = W["W_gate"] * np.exp2(3.0 * (np.arange(96) % 5))[None, None, :]
    W["W_down"] = W["W_down"] * np.exp2(3.0 * (np.arange(128) % 5))[None, None, :]
    ref = O.moe_forward(X, W, idx, wts)["Y"]
    mx = M.moe_forward_mx(X, W, idx, wts)["Y"]
    rel = np.abs(mx - ref).max(axis=1) / np.abs(ref).max(axis=1)
    assert rel.max() < 0.35, rel.max()


def _sub_ulp(v, axis, rng):
    """v moved by at most a quarter of its own grid spacing (its codes stay)."""
    q, sc = M.mx_quantize(v, axis)
    r = M.mx_dequantize(q, sc, axis)
    Xs = np.repeat(np.exp2(np.moveaxis(sc.astype(float), axis, -1) - 127), 32, axis=-1)
    Xs = np.moveaxis(Xs, -1, axis)
    s = np.abs(r) / Xs
    ulp = np.where(s >= 2.0 ** -6, np.exp2(np.floor(np.log2(np.maximum(s, 1e-300))) - 3), 2.0 ** -9) * Xs
    # keep each block's maximum (it fixes the scale) and stay off rounding ties
    out = r + rng.uniform(-0.25, 0.25, r.shape) * ulp
    blocks = np.moveaxis(r, axis, -1)
    bmax = np.abs(blocks).reshape(blocks.shape[:-1] + (-1, 32)).max(axis=-1)
    keep = np.abs(blocks) == np.repeat(bmax, 32, axis=-1)
    out = np.moveaxis(np.where(keep, blocks, np.moveaxis(out, axis, -1)), -1, axis)
    return r, out


def test_every_routed_operand_is_quantized_along_its_axis():
    """Moving X or a routed weight by less than half of its own MX grid
    spacing (block maxima fixed) must leave the MXFP8 layer bit-identical;
    moving the shared-expert weights must not (they stay BF16)."""
    rng = np.random.default_rng(4)
    X, W, idx, wts = _layer(seed=1)
    Xg, Xp = _sub_ulp(X, 1, rng)
    Wg = {key: W[key] for key in ("W_gate", "W_up", "W_down")}
    for key in Wg:
        Wg[key] = _sub_ulp(W[key], 1, rng)[0]
    base = M.moe_forward_mx(Xg, dict(W, **Wg), idx, wts)["Y"]
    assert np.array_equal(M.moe_forward_mx(Xp, dict(W, **Wg), idx, wts)["Y"], base)
    for key in ("W_gate", "W_up", "W_down"):
        moved = dict(W, **Wg)
        moved[key] = _sub_ulp(Wg[key], 1, rng)[1]
        assert np.array_equal(M.moe_forward_mx(Xg, moved, idx, wts)["Y"], base), key
    X2, W2, idx2, wts2 = _layer(seed=2, fs=128)
    b2 = M.moe_forward_mx(X2, W2, idx2, wts2)["Y"]
    W3 = dict(W2)
    W3["Wd_s"] = W2["Wd_s"] * (1 + 2.0 ** -20)
    assert not np.array_equal(M.moe_forward_mx(X2, W3, idx2, wts2)["Y"], b2)


def test_layer_output_is_power_of_two_equivariant_in_w_down():
    X, W, idx, wts = _layer(seed=3)
    base = M.moe_forward_mx(X, W, idx, wts)["Y"]
    W2 = dict(W)
    W2["W_down"] = W["W_down"] * 2.0 ** 5
    assert np.array_equal(M.moe_forward_mx(X, W2, idx, wts)["Y"], base * 2.0 ** 5)
