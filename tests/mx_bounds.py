"""Allowances for products of MXFP8-quantised operands whose quantiser input
the GPU computes itself (test infrastructure; built from the oracle's values
only).

E4M3 rounding is a step function.  When the GPU's fp32 value of an element
and the oracle's fp64 value differ by at most w, both are correct inputs, and
the two round trips may land one grid step apart wherever the oracle's value
lies within w of a rounding boundary (or the block maximum within w of a
power of two, which moves the block's scale).  token_qdq_spread bounds that
difference per element from the oracle's values; product_allowance carries it
through a contraction over tokens.  The premise (inputs within w) is itself
checked element-wise on the GPU's stored values.
"""
import numpy as np

from oracle import mx_oracle as M

W_REL = 1e-4       # quantiser-input window, relative to the operand's max |value|


def token_qdq_spread(V, w):
    """Largest |q' - q| per element of one expert's operand V ([n, C], rows in
    plan order, 32-row blocks from the first row), where q is the oracle's
    token-axis round trip and q' the round trip of any input within w of V
    elementwise (each block's scale free to follow its block maximum)."""
    V = np.asarray(V, np.float64)
    n, C = V.shape
    if n == 0:
        return V
    pad = (-n) % M.BLOCK
    b = np.concatenate([V, np.zeros((pad, C))]).reshape(-1, M.BLOCK, C)
    amax = np.abs(b).max(axis=1, keepdims=True)
    s0 = M.shared_exponent(amax)

    def rt(x, s):
        return M.e4m3_value(M.e4m3_round(np.ldexp(x, -s))) * np.exp2(s.astype(np.float64))
    q0 = rt(b, s0)
    spread = np.zeros_like(b)
    for s in (M.shared_exponent(np.maximum(amax - w, 0.0)), M.shared_exponent(amax + w)):
        for dv in (-w, w):
            spread = np.maximum(spread, np.abs(rt(b + dv, s) - q0))
    return spread.reshape(-1, C)[:n]


def product_allowance(P, Q, spread_P=None, spread_Q=None):
    """Bound on |P'^T Q' - P^T Q| elementwise for |P' - P| <= spread_P and
    |Q' - Q| <= spread_Q (either may be None = exact): |P|^T sQ + sP^T |Q| +
    sP^T sQ."""
    P, Q = np.abs(np.asarray(P, np.float64)), np.abs(np.asarray(Q, np.float64))
    out = np.zeros((P.shape[1], Q.shape[1]))
    if spread_Q is not None:
        out += P.T @ spread_Q
    if spread_P is not None:
        out += spread_P.T @ Q
        if spread_Q is not None:
            out += spread_P.T @ spread_Q
    return out
