"""GPU parity of the MXFP8 training step: moe_forward_mx with the
pre-activations kept, then moe_backward_mx (§3.4 "MXFP8 Support").

Byte work is bit-exact against the oracle wherever both sides quantise the
same values: dY (per token along d) and the backward weight layouts (W_gate,
W_up along f; W_down along d).  dA and dB are quantised from the GPU's own
fp32 values, so they and everything downstream are floats checked against
the oracle's MXFP8 backward to the usual per-tensor bar.
"""
import numpy as np
import pytest
import torch

from oracle import moe_oracle as O
from oracle import mx_oracle as M
from paper_2609_36070_amd import binding as B
from paper_2609_36070_amd.layer import DeviceLayer
from paper_2609_36070_amd.workloads import WORKLOADS, Workload, make_inputs
from tests.parity import assert_close, check_route_and_plan, say, to_np, weights_dict

pytestmark = pytest.mark.gpu


def mx_train_layer(w, seed):
    inp = make_inputs(w, seed)
    say(f"[gpu] mx train {w.name} T={w.T} d={w.d} E={w.E} k={w.k} f={w.f} f_s={w.f_s} seed={seed}")
    L = DeviceLayer(w, inp, mx=True)
    assert L.with_backward
    L.step_mx()
    torch.cuda.synchronize()
    return L, inp


def check_bwd_weight_codes(L, inp, experts):
    for key, q, sc in (("W_gate", L.Wg_qb, L.Wg_scb), ("W_up", L.Wu_qb, L.Wu_scb),
                       ("W_down", L.Wd_qb, L.Wd_scb)):
        for e in experts:
            codes, scales = M.mx_quantize(inp[key][e], axis=1)    # rows along their own axis
            assert np.array_equal(to_np(q[e]), codes), f"{key}[{e}] codes"
            assert np.array_equal(to_np(sc[e]), scales), f"{key}[{e}] scales"


def mx_backward_parity(w, seed):
    L, inp = mx_train_layer(w, seed)
    Zo, idx_g = check_route_and_plan(L, inp, w)
    w_orc = O.gate_weights(Zo, idx_g)
    check_bwd_weight_codes(L, inp, range(w.E))
    dyq, dys = M.mx_quantize(inp["dY"], axis=1)
    assert np.array_equal(to_np(L.mx_ws_tensor(B.WS_DYQ, torch.uint8, (w.T, w.d))), dyq)
    assert np.array_equal(to_np(L.mx_ws_tensor(B.WS_DYS, torch.uint8, (w.T, w.d // 32))), dys)
    g = M.moe_backward_mx(inp["X"], inp["W_r"], weights_dict(inp), idx_g, w_orc, inp["dY"])
    for n in ("dX", "dW_gate", "dW_up", "dW_down", "dZ", "dW_r"):
        assert_close(n, to_np(getattr(L, n)), g[n])
    R = w.T * w.k
    dg_pos = to_np(L.mx_ws_tensor(B.WS_DG, torch.float32, (R,)))
    rp = to_np(L.route_pos)[:R]
    assert_close("dg", dg_pos[rp].reshape(w.T, w.k), g["dg"])
    if w.f_s:
        for n in ("dWg_s", "dWu_s", "dWd_s"):
            assert_close(n, to_np(getattr(L, n)), g[n])
    assert L.error_word() == 0
    return L, inp


def test_mx_backward_ragged():
    mx_backward_parity(Workload("mx_ragged_train", T=1000, d=512, E=6, k=2, f=512, f_s=256,
                                bias_std=0.5, backward=True), seed=31)


@pytest.mark.parametrize("w", [
    Workload("mx_one_token", T=1, d=256, E=8, k=3, f=256, f_s=256, backward=True),
    Workload("mx_k_equals_E", T=300, d=256, E=4, k=4, f=512, bias_std=0.5, backward=True),
    Workload("mx_empty_experts", T=40, d=256, E=64, k=1, f=256, bias_std=3.0, backward=True),
    Workload("mx_many_tiles", T=700, d=768, E=3, k=2, f=768, backward=True),
], ids=lambda w: w.name)
def test_mx_backward_edge_shapes(w):
    mx_backward_parity(w, seed=32)


def test_mx_backward_no_tokens():
    w = Workload("mx_none_train", T=0, d=256, E=4, k=2, f=256, f_s=256, backward=True)
    L = DeviceLayer(w, make_inputs(w, 0), mx=True)
    for n in ("dW_gate", "dW_up", "dW_down", "dW_r", "dWg_s", "dWu_s", "dWd_s"):
        getattr(L, n).fill_(3.0)
    L.step_mx()
    torch.cuda.synchronize()
    for n in ("dW_gate", "dW_up", "dW_down", "dW_r", "dWg_s", "dWu_s", "dWd_s"):
        assert torch.count_nonzero(getattr(L, n)) == 0, n


def test_mx_backward_determinism():
    w = Workload("mx_det_train", T=1000, d=512, E=6, k=2, f=512, f_s=256, bias_std=0.5,
                 backward=True)
    L, _ = mx_train_layer(w, 33)
    names = ("Y", "dX", "dW_gate", "dW_up", "dW_down", "dW_r", "dZ", "dWg_s", "dWu_s", "dWd_s")
    first = {n: getattr(L, n).clone() for n in names}
    for _ in range(3):
        L.step_mx()
        torch.cuda.synchronize()
        for n in names:
            assert torch.equal(getattr(L, n), first[n]), n


def test_mx_training_step_full_size_sampled():
    """The training workload in MXFP8: the backward weight codes of two
    experts bit-exact; sampled token rows of dX, dZ and dg, and weight-gradient
    columns of two experts, against the oracle's per-token / per-column MXFP8
    backward."""
    w = WORKLOADS["large_shared_train"]
    L, inp = mx_train_layer(w, 0)
    check_bwd_weight_codes(L, inp, [0, w.E - 1])
    Zo, idx_g = check_route_and_plan(L, inp, w)
    w_orc = O.gate_weights(Zo, idx_g)
    W = weights_dict(inp, as_f64=True)
    rng = np.random.default_rng(6)
    toks = np.unique(np.concatenate([[0, w.T - 1], rng.choice(w.T, 6, replace=False)]))
    dX, dZ, dg = M.mx_token_backward(inp["X"], inp["W_r"], W, idx_g, w_orc, inp["dY"], toks)
    assert_close("dX[sampled tokens]", to_np(L.dX)[toks], dX)
    assert_close("dZ[sampled tokens]", to_np(L.dZ)[toks], dZ)
    R = w.T * w.k
    dg_pos = to_np(L.mx_ws_tensor(B.WS_DG, torch.float32, (R,)))
    rp = to_np(L.route_pos)[:R].reshape(w.T, w.k)
    assert_close("dg[sampled tokens]", dg_pos[rp[toks]], dg)
    cols = np.array([0, 777, w.f - 1])
    for e in (0, w.E - 1):
        a, b, c = M.mx_expert_weight_grad_columns(inp["X"], W, idx_g, w_orc, inp["dY"], e, cols)
        assert_close(f"dW_gate[{e}][:, cols]", to_np(L.dW_gate[e])[:, cols], a)
        assert_close(f"dW_up[{e}][:, cols]", to_np(L.dW_up[e])[:, cols], b)
        assert_close(f"dW_down[{e}][cols, :]", to_np(L.dW_down[e])[cols, :], c)
    assert L.error_word() == 0
