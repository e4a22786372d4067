"""GPU parity at the full workload sizes, in the launch configuration the
benchmark times.

Integer outputs (top-k, plan) are compared in full.  Floating-point outputs
are compared on seeded samples the oracle computes one by one (token rows of Y
and dX, columns of every expert's weight gradients); dZ of every token comes
from the oracle's own expert outputs, and dW_r = X^T dZ from that dZ.
"""
import numpy as np
import pytest
import torch

from oracle import moe_oracle as O
from paper_2609_36070_amd.workloads import WORKLOADS
from tests.parity import (assert_close, check_route_and_plan, run_layer, say, to_np,
                          weights_dict)

pytestmark = pytest.mark.gpu

N_TOKENS_FWD = 40
N_TOKENS_BWD = 10


def sample_tokens(T, n, seed):
    rng = np.random.default_rng(seed)
    return np.unique(np.concatenate([[0, T - 1], rng.choice(T, n, replace=False)]))


@pytest.mark.parametrize("name", ["many_experts", "hot_expert", "large_shared"])
def test_full_size_forward(name):
    w = WORKLOADS[name]
    L, inp = run_layer(w, seed=0)
    Zo, idx_g = check_route_and_plan(L, inp, w)
    counts = to_np(L.counts)
    say(f"  expert load: min {counts.min()} mean {counts.mean():.1f} max {counts.max()}")
    if name == "hot_expert":
        assert counts[0] >= int(0.1 * w.T)       # the hot tokens all reach expert 0
    w_orc = O.gate_weights(Zo, idx_g)
    toks = sample_tokens(w.T, N_TOKENS_FWD, 1)
    ref = O.moe_forward_dense(inp["X"], weights_dict(inp, as_f64=True), idx_g, w_orc, toks)
    assert_close("Y[sampled tokens]", to_np(L.Y)[toks], ref)


@pytest.mark.timeout(600)
def test_full_size_training_step_and_determinism():
    w = WORKLOADS["large_shared_train"]
    L, inp = run_layer(w, seed=0)
    Zo, idx_g = check_route_and_plan(L, inp, w)
    w_orc = O.gate_weights(Zo, idx_g)
    W64 = weights_dict(inp, as_f64=True)

    # forward rows
    toks = sample_tokens(w.T, N_TOKENS_BWD, 2)
    ref = O.moe_forward_dense(inp["X"], W64, idx_g, w_orc, toks)
    assert_close("Y[sampled tokens]", to_np(L.Y)[toks], ref)

    # dX and dZ rows
    dX_ref, dZ_ref, _ = O.token_backward(inp["X"], inp["W_r"], W64, idx_g, w_orc, inp["dY"], toks)
    assert_close("dX[sampled tokens]", to_np(L.dX)[toks], dX_ref)
    assert_close("dZ[sampled tokens]", to_np(L.dZ)[toks], dZ_ref)

    # dZ of every token from the oracle's own expert outputs (about 11.5
    # TFLOP of fp64 on the host), and dW_r = X^T dZ from it
    say("  oracle router gradient over all tokens ...")
    dZ_orc, _ = O.router_gradient(inp["X"], W64, idx_g, w_orc, inp["dY"])
    assert_close("dZ[all tokens]", to_np(L.dZ), dZ_orc)
    dWr_ref = inp["X"].astype(np.float64).T @ dZ_orc
    assert_close("dW_r", to_np(L.dW_r), dWr_ref)

    # weight-gradient columns of every expert (seeded, different per expert)
    # and of the shared expert
    rng = np.random.default_rng(3)
    for e in list(range(w.E)) + ["shared"]:
        cols = np.unique(np.concatenate([[0, w.f - 1], rng.choice(w.f, 2, replace=False)]))
        a, b, c = O.expert_weight_grad_columns(inp["X"], W64, idx_g, w_orc, inp["dY"], e, cols)
        if e == "shared":
            g_gate, g_up, g_down = to_np(L.dWg_s), to_np(L.dWu_s), to_np(L.dWd_s)
        else:
            g_gate, g_up, g_down = to_np(L.dW_gate[e]), to_np(L.dW_up[e]), to_np(L.dW_down[e])
        assert_close(f"dW_gate[{e}][:, cols]", g_gate[:, cols], a)
        assert_close(f"dW_up[{e}][:, cols]", g_up[:, cols], b)
        assert_close(f"dW_down[{e}][cols, :]", g_down[cols, :], c)

    # bitwise determinism over 5 runs
    names = ("logits", "topk_idx", "topk_w", "perm", "route_pos", "Y", "dX", "dW_gate", "dW_up",
             "dW_down", "dW_r", "dZ", "dWg_s", "dWu_s", "dWd_s")
    first = {n: getattr(L, n).clone() for n in names}
    for rep in range(4):
        L.step()
        torch.cuda.synchronize()
        for n in names:
            assert torch.equal(getattr(L, n), first[n]), (rep, n)
    say("  5 runs bitwise identical")
