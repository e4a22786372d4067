"""Plain CPU oracle of the MXFP8 routed-expert forward (float64 numpy).

TEST INFRASTRUCTURE ONLY.  Only the test-suite, the package smoke check and the
benchmark's CPU-baseline leg may import this module.  The GPU library never
calls it and shares no code with it.

The paper runs its routed experts in MXFP8 and keeps the shared expert in BF16
(§3.4 "MXFP8 Support"): weights are quantised ahead of time by their own
kernel, activations are quantised where they are produced (dispatch, the
grouped GEMMs, the gated activation).  MXFP8 is the OCP microscaling format
the paper cites: blocks of elements share one power-of-two scale.

Readings of what the paper leaves open:

* elements are OCP FP8 E4M3 (exponent bias 7, no infinities, largest finite
  magnitude 448, S.1111.111 is NaN);
* a block is 32 consecutive elements along the contraction (K) dimension of
  the GEMM that consumes the tensor, with one E8M0 scale (a biased exponent,
  bias 127) per block;
* scale: the microscaling definition, shared_exp = floor(log2(amax)) - emax
  with emax = 8 (the largest E4M3 exponent), clamped to [-127, 127]; an
  all-zero block takes -127;
* elements: v / 2**shared_exp rounded to the nearest E4M3 value (ties to the
  even code), saturating at +-448 (the block maximum can exceed 448 after
  scaling, since amax / 2**shared_exp lies in [256, 512));
* quantised tensors: X per token along d (once per token, before the gather),
  W_gate and W_up along d, W_down along f, and the gated activation H along f
  (straight from its fp32 value); products are exact and accumulate in fp32 on
  the GPU (here in float64); the expert output Yexp is rounded to bf16 as in
  the BF16 path, and the shared expert and the combine are the BF16 path's.
"""
from __future__ import annotations

import numpy as np

from oracle import moe_oracle as O

F64 = np.float64
E4M3_EMAX = 8          # largest unbiased exponent of an E4M3 normal
E4M3_MAX = 448.0       # 1.75 * 2**8
E4M3_EMIN = -6         # exponent of the smallest normal; subnormals are k * 2**-9
BLOCK = 32
SCALE_BIAS = 127


# ---------------------------------------------------------------------------
# E4M3 elements
# ---------------------------------------------------------------------------

def e4m3_value(code):
    """Value of E4M3 codes (float64; NaN for S.1111.111)."""
    c = np.asarray(code, np.int64)
    s = (c >> 7) & 1
    e = (c >> 3) & 15
    m = c & 7
    mag = np.where(e == 0, m * 2.0 ** (E4M3_EMIN - 3), (8 + m) * np.exp2(e - 7 - 3.0))
    mag = np.where((e == 15) & (m == 7), np.nan, mag)
    return np.where(s == 1, -mag, mag)


def e4m3_round(x):
    """Nearest E4M3 code of each value (ties to the even code), saturating at
    +-448.  Values must be finite."""
    x = np.asarray(x, F64)
    sign = (np.signbit(x)).astype(np.int64)
    a = np.abs(x)
    # binade exponent of |x| (the subnormal range shares the quantum of 2**-6)
    _, ex = np.frexp(np.where(a > 0, a, 1.0))
    e = np.maximum(ex - 1, E4M3_EMIN)
    q = np.exp2(e - 3.0)                       # spacing of the grid in that binade
    m = np.rint(a / q).astype(np.int64)        # round half to even
    # rounding up to the next binade: m == 16 means (1.0) * 2**(e+1)
    up = m == 16
    e = np.where(up, e + 1, e)
    m = np.where(up, 8, m)
    normal = m >= 8
    code = np.where(normal, ((e + 7) << 3) | (m - 8), m)
    code = np.where(m * np.exp2(e - 3.0) > E4M3_MAX, 0x7E, code)   # saturate
    code = np.where(a == 0, 0, code)
    return ((sign << 7) | code).astype(np.uint8)


# ---------------------------------------------------------------------------
# Microscaling blocks
# ---------------------------------------------------------------------------

def _blocks(v, axis):
    v = np.moveaxis(np.asarray(v, F64), axis, -1)
    n = v.shape[-1]
    if n % BLOCK:
        raise ValueError(f"length {n} along the block axis is not a multiple of {BLOCK}")
    return v.reshape(v.shape[:-1] + (n // BLOCK, BLOCK))


def shared_exponent(amax):
    """floor(log2(amax)) - 8, clamped to the E8M0 range; -127 for amax = 0."""
    amax = np.asarray(amax, F64)
    _, ex = np.frexp(np.where(amax > 0, amax, 1.0))
    se = (ex - 1) - E4M3_EMAX
    se = np.where(amax > 0, se, -SCALE_BIAS)
    return np.clip(se, -SCALE_BIAS, SCALE_BIAS).astype(np.int64)


def mx_quantize(v, axis):
    """MXFP8 quantisation along `axis` (a multiple of 32 long).

    Returns (codes uint8 with v's shape, scales uint8 = shared_exp + 127 with
    the block axis shortened 32-fold)."""
    b = _blocks(v, axis)
    se = shared_exponent(np.max(np.abs(b), axis=-1))
    codes = e4m3_round(np.ldexp(b, -se[..., None]))
    codes = np.moveaxis(codes.reshape(codes.shape[:-2] + (-1,)), -1, axis)
    scales = np.moveaxis((se + SCALE_BIAS).astype(np.uint8), -1, axis)
    return codes, scales


def mx_dequantize(codes, scales, axis):
    b = _blocks(e4m3_value(codes), axis)
    se = np.moveaxis(np.asarray(scales, np.int64), axis, -1) - SCALE_BIAS
    out = np.ldexp(b, se[..., None])
    return np.moveaxis(out.reshape(out.shape[:-2] + (-1,)), -1, axis)


def mx_qdq(v, axis):
    """Value after an MXFP8 round trip."""
    return mx_dequantize(*mx_quantize(v, axis), axis)


# ---------------------------------------------------------------------------
# The routed-expert forward in MXFP8 (§3.4 "MXFP8 Support"), shared expert and
# combine as in BF16 (§2.1 equation)
# ---------------------------------------------------------------------------

def quantize_weights(W):
    """Pre-quantised routed weights: W_gate, W_up along d; W_down along f.
    Returns dict of (codes, scales) keyed like W, each in W's own layout."""
    return {
        "W_gate": mx_quantize(W["W_gate"], axis=1),
        "W_up": mx_quantize(W["W_up"], axis=1),
        "W_down": mx_quantize(W["W_down"], axis=1),
    }


def moe_forward_mx(X, W, idx, w):
    """Forward of the layer with MXFP8 routed experts.

    Returns dict(Y [T,d], H [T*k, f] (fp64, before its quantisation),
    Hq (dequantised H), Yexp [T*k, d] (fp64, before bf16 rounding), Ysh,
    Xq (codes, scales), plan arrays) in plan-position order."""
    X = np.asarray(X, F64)
    T, d = X.shape
    E = W["W_gate"].shape[0]
    k = idx.shape[1]
    counts, offsets, perm, route_pos = O.plan(idx, E)
    tok = perm // k
    Xq = mx_quantize(X, axis=1)
    Xh = mx_dequantize(*Xq, axis=1)
    Wg = mx_qdq(W["W_gate"], axis=1)
    Wu = mx_qdq(W["W_up"], axis=1)
    Wd = mx_qdq(W["W_down"], axis=1)
    f = W["W_gate"].shape[2]
    H = np.zeros((T * k, f), F64)
    for e in range(E):
        rows = slice(offsets[e], offsets[e + 1])
        xe = Xh[tok[rows]]
        H[rows] = O.silu(xe @ Wg[e]) * (xe @ Wu[e])
    Hq = mx_qdq(H, axis=1)
    Yexp = np.zeros((T * k, d), F64)
    for e in range(E):
        rows = slice(offsets[e], offsets[e + 1])
        Yexp[rows] = Hq[rows] @ Wd[e]
    Ysh = None
    Y = np.zeros((T, d), F64)
    if W.get("Wg_s") is not None:
        Ysh = O.expert_ffn(X, W["Wg_s"], W["Wu_s"], W["Wd_s"])
        Y += Ysh
    for s in range(k):
        Y += w[:, s:s + 1] * Yexp[route_pos[np.arange(T) * k + s]]
    return dict(Y=Y, H=H, Hq=Hq, Yexp=Yexp, Ysh=Ysh, Xq=Xq, counts=counts,
                offsets=offsets, perm=perm, route_pos=route_pos)



def mx_qdq_token_blocks(v):
    """One expert's rows (in its plan order) after an MXFP8 round trip along
    the token axis: blocks of 32 consecutive rows from the expert's first row,
    one scale per column of a block; the last block is completed with zero
    rows (which leave its maximum unchanged) that are dropped again."""
    v = np.asarray(v, F64)
    n = v.shape[0]
    if n == 0:
        return v
    pad = (-n) % BLOCK
    vp = np.concatenate([v, np.zeros((pad,) + v.shape[1:], F64)], axis=0)
    return mx_qdq(vp, 0)[:n]


def moe_backward_mx(X, W_r, W, idx, w, dY, quant=True, wgrad_mx=False, keep=False):
    """Backward of the layer with MXFP8 routed experts (teacher-forced on idx, w).

    Readings (§3.4 "MXFP8 Support" names MXFP8 training and fused activation
    quantisation; it does not say which backward products run in MXFP8):

    * the pre-activations a, b and the activation h come from the MXFP8
      forward (X quantised along d, W_gate / W_up along d) and enter the
      backward at full precision, exactly as in the BF16 oracle: the method
      quantises only GEMM operands, and it fuses each quantisation into the
      kernel that produces the values, so a quantiser reads the producer's
      own result, never a rounded copy of it (§3.4 "MXFP8 Support");
    * the two products that contract over a model dimension run in MXFP8:
      dh' = Q_d(dY) Q_d(W_down[e])^T (dY per token and W_down per row, blocks
      along d), and dX_e = Q_f(dA) Q_f(W_gate[e])^T + Q_f(dB) Q_f(W_up[e])^T
      (dA, dB quantised along f from their fp32 values, W_gate / W_up per row
      of [d, f], blocks along f);
    * the weight-gradient products contract over each expert's ragged token
      set and stay BF16: dW_gate = X_e^T dA, dW_up = X_e^T dB,
      dW_down = (w h)^T dY_e, with the unquantised X, dY and the
      full-precision dA, dB (the gradient passes straight through the
      quantiser);
    * the router-weight gradient, the softmax backward, dW_r, the shared expert
      (BF16) and dX's router term are those of the BF16 backward.

    With wgrad_mx (the opt-in MXFP8 weight gradients), the weight-gradient
    products run in MXFP8 too.  They contract over the expert's tokens, so
    each operand is quantised along the token axis, per expert
    (mx_qdq_token_blocks): X and dY as given, and dA, dB, w h as the
    gated-activation backward produces them (full precision, the same
    reading as for a and b above):
      dW_gate = Q_t(X_e)^T Q_t(dA_e), dW_up = Q_t(X_e)^T Q_t(dB_e),
      dW_down = Q_t(w h)^T Q_t(dY_e).

    quant=False replaces every quantise-dequantise by the identity, which must
    reproduce moe_oracle.moe_backward.

    keep=True also returns, under "routes", each expert's pre-activations a,
    b, the gradients dA, dB and the weighted activation w h, one row per
    route of the expert in ascending route id (the plan order).
    """
    qdq = mx_qdq if quant else (lambda v, axis: np.asarray(v, F64))
    X = np.asarray(X, F64)
    dY = np.asarray(dY, F64)
    T, d = X.shape
    E, _, f = W["W_gate"].shape
    k = idx.shape[1]
    Xh = qdq(X, 1)
    dYh = qdq(dY, 1)
    dX = np.zeros((T, d), F64)
    dWg = np.zeros((E, d, f), F64)
    dWu = np.zeros((E, d, f), F64)
    dWd = np.zeros((E, f, d), F64)
    dg = np.zeros((T, k), F64)
    routes = []
    for e in range(E):
        ts, ss = np.nonzero(np.asarray(idx) == e)
        if ts.size == 0:
            routes.append(None)
            continue
        Wg = np.asarray(W["W_gate"][e], F64)
        Wu = np.asarray(W["W_up"][e], F64)
        Wd = np.asarray(W["W_down"][e], F64)
        a = Xh[ts] @ qdq(Wg, 0)                # forward: blocks of W_gate[e] [d, f] along d
        b = Xh[ts] @ qdq(Wu, 0)
        h = O.silu(a) * b
        we = np.asarray(w, F64)[ts, ss][:, None]
        dhp = dYh[ts] @ qdq(Wd, 1).T           # W_down[e] [f, d], blocks along d
        dg[ts, ss] = (dhp * h).sum(axis=1)
        dh = we * dhp
        dA = dh * b * O._dsilu(a)
        dB = dh * O.silu(a)
        if keep:
            routes.append(dict(a=a, b=b, dA=dA, dB=dB, wh=we * h))
        if quant and wgrad_mx:
            xt = mx_qdq_token_blocks(X[ts])
            dWg[e] = xt.T @ mx_qdq_token_blocks(dA)
            dWu[e] = xt.T @ mx_qdq_token_blocks(dB)
            dWd[e] = mx_qdq_token_blocks(we * h).T @ mx_qdq_token_blocks(dY[ts])
        else:
            dWg[e] = X[ts].T @ dA
            dWu[e] = X[ts].T @ dB
            dWd[e] = (we * h).T @ dY[ts]
        np.add.at(dX, ts, qdq(dA, 1) @ qdq(Wg, 1).T + qdq(dB, 1) @ qdq(Wu, 1).T)
    dz_sel = O.softmax_restricted_backward(np.asarray(w, F64), dg)
    dZ = np.zeros((T, W_r.shape[1]), F64)
    np.put_along_axis(dZ, np.asarray(idx, np.int64), dz_sel, axis=1)
    dW_r = X.T @ dZ
    dX += dZ @ np.asarray(W_r, F64).T
    out = dict(dX=dX, dW_gate=dWg, dW_up=dWu, dW_down=dWd, dW_r=dW_r, dZ=dZ, dg=dg,
               dWg_s=None, dWu_s=None, dWd_s=None)
    if keep:
        out["routes"] = routes
    if W.get("Wg_s") is not None:             # the shared expert stays BF16
        Wg = np.asarray(W["Wg_s"], F64)
        Wu = np.asarray(W["Wu_s"], F64)
        Wd = np.asarray(W["Wd_s"], F64)
        a = X @ Wg
        b = X @ Wu
        dhs = dY @ Wd.T
        dA = dhs * b * O._dsilu(a)
        dB = dhs * O.silu(a)
        out["dWg_s"] = X.T @ dA
        out["dWu_s"] = X.T @ dB
        out["dWd_s"] = (O.silu(a) * b).T @ dY
        out["dX"] = out["dX"] + dA @ Wg.T + dB @ Wu.T
    return out


# ---------------------------------------------------------------------------
# Sampled evaluation of the MXFP8 backward for full-size workloads: each
# sampled output follows the same definition as moe_backward_mx, restricted
# to what it depends on.
# ---------------------------------------------------------------------------

def _mx_expert_weights(W, e):
    """The routed weights of expert e as the MXFP8 passes see them."""
    Wg = np.asarray(W["W_gate"][e], F64)
    Wu = np.asarray(W["W_up"][e], F64)
    Wd = np.asarray(W["W_down"][e], F64)
    return dict(g_fwd=mx_qdq(Wg, 0), u_fwd=mx_qdq(Wu, 0), d_bwd=mx_qdq(Wd, 1),
                g_bwd=mx_qdq(Wg, 1), u_bwd=mx_qdq(Wu, 1))


def mx_token_backward(X, W_r, W, idx, w, dY, tokens):
    """dX, dZ and dg of moe_backward_mx for the given tokens only."""
    X = np.asarray(X, F64)
    dY = np.asarray(dY, F64)
    E = W["W_gate"].shape[0]
    tokens = np.asarray(tokens)
    k = idx.shape[1]
    cache = {}
    dX = np.zeros((len(tokens), X.shape[1]))
    dg = np.zeros((len(tokens), k))
    for n, t in enumerate(tokens):
        xq = mx_qdq(X[t:t + 1], 1)[0]
        dyq = mx_qdq(dY[t:t + 1], 1)[0]
        for s in range(k):
            e = int(idx[t, s])
            if e not in cache:
                cache[e] = _mx_expert_weights(W, e)
            q = cache[e]
            a = xq @ q["g_fwd"]
            b = xq @ q["u_fwd"]
            dhp = q["d_bwd"] @ dyq
            dg[n, s] = dhp @ (O.silu(a) * b)
            dh = w[t, s] * dhp
            dA = dh * b * O._dsilu(a)
            dB = dh * O.silu(a)
            dX[n] += q["g_bwd"] @ mx_qdq(dA[None, :], 1)[0] + q["u_bwd"] @ mx_qdq(dB[None, :], 1)[0]
    dz_sel = O.softmax_restricted_backward(np.asarray(w, F64)[tokens], dg)
    dZ = np.zeros((len(tokens), W_r.shape[1]))
    np.put_along_axis(dZ, np.asarray(idx, np.int64)[tokens], dz_sel, axis=1)
    dX += dZ @ np.asarray(W_r, F64).T
    if W.get("Wg_s") is not None:
        Wg, Wu, Wd = (np.asarray(W[key], F64) for key in ("Wg_s", "Wu_s", "Wd_s"))
        x = X[tokens]
        a, b = x @ Wg, x @ Wu
        dhs = dY[tokens] @ Wd.T
        dX += (dhs * b * O._dsilu(a)) @ Wg.T + (dhs * O.silu(a)) @ Wu.T
    return dX, dZ, dg


def mx_expert_weight_grad_columns(X, W, idx, w, dY, e, cols, wgrad_mx=False, keep=False):
    """dW_gate[e][:, cols], dW_up[e][:, cols] and dW_down[e][cols, :] of
    moe_backward_mx (token-axis blocks are per column, so the selected
    columns need only their own operand columns).  keep=True also returns the
    expert's operand columns dA[:, cols], dB[:, cols], (w h)[:, cols] in plan
    order, as a fourth element (a dict)."""
    X = np.asarray(X, F64)
    dY = np.asarray(dY, F64)
    ts, ss = np.nonzero(np.asarray(idx) == e)
    Wg = np.asarray(W["W_gate"][e], F64)
    Wu = np.asarray(W["W_up"][e], F64)
    Wd = np.asarray(W["W_down"][e], F64)
    xq = mx_qdq(X[ts], 1)
    a = xq @ mx_qdq(Wg, 0)[:, cols]
    b = xq @ mx_qdq(Wu, 0)[:, cols]
    dhp = mx_qdq(dY[ts], 1) @ mx_qdq(Wd, 1)[cols, :].T
    we = np.asarray(w, F64)[ts, ss][:, None]
    dh = we * dhp
    dA = dh * b * O._dsilu(a)
    dB = dh * O.silu(a)
    h = O.silu(a) * b
    if wgrad_mx:
        qt = mx_qdq_token_blocks
        xt = qt(X[ts])
        out = (xt.T @ qt(dA), xt.T @ qt(dB), qt(we * h).T @ qt(dY[ts]))
    else:
        out = (X[ts].T @ dA, X[ts].T @ dB, (we * h).T @ dY[ts])
    if keep:
        return out + (dict(dA=dA, dB=dB, wh=we * h),)
    return out
