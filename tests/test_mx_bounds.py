"""CPU checks of the quantisation-flip allowance used by the MXFP8 weight-
gradient parity tests: every input within the window must round-trip to a
value within the computed spread of the oracle's, and the product allowance
must cover every product of such operands."""
import numpy as np

from oracle import mx_oracle as M
from tests.mx_bounds import product_allowance, token_qdq_spread


def _operand(rng, n, C):
    V = rng.standard_normal((n, C)) * np.exp2(rng.integers(-3, 4, size=(1, C)))
    # plant values on E4M3 rounding midpoints and block maxima on powers of two
    V[0, :] = 2.0 ** rng.integers(-2, 3, size=C)
    V[1, :] = V[0, :] * (1 + 1.0 / 16)           # halfway between two E4M3 values
    return V


def test_zero_window_has_zero_spread():
    V = _operand(np.random.default_rng(0), 70, 9)
    assert np.all(token_qdq_spread(V, 0.0) == 0.0)


def test_spread_covers_every_input_within_the_window():
    rng = np.random.default_rng(1)
    for n in (1, 31, 32, 70):
        V = _operand(rng, max(n, 2), 12)[:n]
        w = 1e-3 * np.abs(V).max()
        sp = token_qdq_spread(V, w)
        q0 = M.mx_qdq_token_blocks(V)
        for trial in range(200):
            if trial % 3 == 0:
                d = w * rng.choice([-1.0, 1.0], size=V.shape)       # window corners
            else:
                d = w * rng.uniform(-1, 1, size=V.shape)
            dq = np.abs(M.mx_qdq_token_blocks(V + d) - q0)
            assert np.all(dq <= sp + 1e-300), (n, trial)
        assert np.any(sp > 0)                                      # the planted ties do flip


def test_product_allowance_covers_perturbed_products():
    rng = np.random.default_rng(2)
    P, Q = rng.standard_normal((40, 5)), rng.standard_normal((40, 7))
    sP, sQ = 0.01 * rng.random((40, 5)), 0.02 * rng.random((40, 7))
    A = product_allowance(P, Q, sP, sQ)
    for _ in range(300):
        Pp = P + sP * rng.uniform(-1, 1, P.shape)
        Qp = Q + sQ * rng.uniform(-1, 1, Q.shape)
        assert np.all(np.abs(Pp.T @ Qp - P.T @ Q) <= A + 1e-12)
    assert np.array_equal(product_allowance(P, Q, None, None), np.zeros((5, 7)))
