"""GPU parity of the fused persistent forward (moe_forward_fused).

The fused launch runs the same tile code as the separate launches and adds
the combine in the same order, so every output must equal moe_forward's
bitwise; it is also checked against the oracle.  The error word must stay 0
(bit 1 would mean a dependency wait gave up).
"""
import numpy as np
import pytest
import torch

from oracle import moe_oracle as O
from paper_2609_36070_amd import binding as B
from paper_2609_36070_amd.layer import DeviceLayer
from paper_2609_36070_amd.workloads import WORKLOADS, Workload, make_inputs
from tests.parity import assert_close, check_route_and_plan, say, to_np, weights_dict

pytestmark = pytest.mark.gpu

RAGGED_TRAIN = Workload("ragged_train", T=1000, d=512, E=6, k=2, f=512, f_s=256, bias_std=0.5,
                        backward=True)


def regions(L, w):
    """The forward's outputs; with dense routing (k == E) the combine is folded
    into the down product, so Yexp and Ysh are not written."""
    R = w.T * w.k
    out = {"Y": L.Y.clone(),
           "H": L.ws_tensor(B.WS_H, torch.bfloat16, (R, w.f)).clone()}
    if w.k != w.E:
        out["Yexp"] = L.ws_tensor(B.WS_YEXP, torch.bfloat16, (R, w.d)).clone()
        if w.f_s:
            out["Ysh"] = L.ws_tensor(B.WS_YSH, torch.bfloat16, (w.T, w.d)).clone()
    if L.with_backward:
        out["A"] = L.ws_tensor(B.WS_A, torch.bfloat16, (R, w.f)).clone()
        out["B"] = L.ws_tensor(B.WS_B, torch.bfloat16, (R, w.f)).clone()
    return out


def run_both(w, seed):
    """Route + plan once, then the separate-launch forward and the fused one
    on the same buffers; returns both sets of outputs."""
    inp = make_inputs(w, seed)
    say(f"[gpu] fused {w.name} T={w.T} d={w.d} E={w.E} k={w.k} f={w.f} f_s={w.f_s} seed={seed}")
    L = DeviceLayer(w, inp)
    L.route()
    L.plan()
    L.forward()
    torch.cuda.synchronize()
    ref = regions(L, w)
    L.Y.fill_(7.0)                  # clobber, so stale values cannot pass
    L.ws_tensor(B.WS_YEXP, torch.bfloat16, (w.T * w.k, w.d)).fill_(7.0)
    L.forward_fused()
    torch.cuda.synchronize()
    assert L.error_word() == 0, f"error word {L.error_word()}"
    return L, inp, ref, regions(L, w)


def assert_bitwise(ref, got):
    for n in ref:
        assert torch.equal(ref[n], got[n]), f"{n} differs from the separate-launch forward"
    say("  bitwise equal to moe_forward: " + ", ".join(ref))


@pytest.mark.parametrize("w", [RAGGED_TRAIN,
                               Workload("dense_shared_train", T=700, d=512, E=4, k=4, f=512,
                                        f_s=256, bias_std=0.5, backward=True)],
                         ids=lambda w: w.name)
def test_fused_training_layer(w):
    L, inp, ref, got = run_both(w, 21)
    assert_bitwise(ref, got)
    Zo, idx_g = check_route_and_plan(L, inp, w)
    w_orc = O.gate_weights(Zo, idx_g)
    fw = O.moe_forward(inp["X"], weights_dict(inp), idx_g, w_orc)
    assert_close("Y", to_np(got["Y"]), fw["Y"])
    # the backward runs on what the fused forward saved
    L.backward()
    torch.cuda.synchronize()
    g = O.moe_backward(inp["X"], inp["W_r"], weights_dict(inp), idx_g, w_orc, inp["dY"])
    for n in ("dX", "dW_gate", "dW_up", "dW_down", "dZ", "dW_r", "dWg_s", "dWu_s", "dWd_s"):
        assert_close(n, to_np(getattr(L, n)), g[n])


@pytest.mark.parametrize("w", [
    Workload("one_token", T=1, d=256, E=8, k=3, f=256, f_s=256),
    Workload("k_equals_E", T=300, d=256, E=4, k=4, f=512, bias_std=0.5),
    Workload("empty_experts", T=40, d=256, E=64, k=1, f=256, bias_std=3.0),
    Workload("many_tiles", T=700, d=768, E=3, k=2, f=768),
    Workload("no_shared_k16", T=600, d=256, E=32, k=16, f=256, bias_std=0.5),
    Workload("max_experts", T=2000, d=256, E=256, k=4, f=256, f_s=512, bias_std=1.0),
    Workload("dense_shared", T=555, d=768, E=6, k=6, f=256, f_s=512, bias_std=0.5),
], ids=lambda w: w.name)
def test_fused_edge_shapes(w):
    L, inp, ref, got = run_both(w, 22)
    assert_bitwise(ref, got)
    Zo, idx_g = check_route_and_plan(L, inp, w)
    fw = O.moe_forward(inp["X"], weights_dict(inp), idx_g, O.gate_weights(Zo, idx_g))
    assert_close("Y", to_np(got["Y"]), fw["Y"])


def test_fused_no_tokens():
    w = Workload("no_tokens", T=0, d=256, E=8, k=2, f=256, f_s=256)
    L = DeviceLayer(w, make_inputs(w, 0))
    L.route()
    L.plan()
    L.forward_fused()
    torch.cuda.synchronize()
    assert L.error_word() == 0


def test_fused_repeat_and_graph_replay():
    w = RAGGED_TRAIN
    L, _, ref, got = run_both(w, 23)
    assert_bitwise(ref, got)
    for _ in range(3):
        L.forward_fused()
        torch.cuda.synchronize()
        assert_bitwise(ref, regions(L, w))
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        L.forward_fused()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        L.forward_fused()
    torch.cuda.synchronize()
    for _ in range(3):
        L.Y.fill_(3.0)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        assert L.error_word() == 0
        assert_bitwise(ref, regions(L, w))


@pytest.mark.parametrize("name", ["large_shared", "many_experts", "hot_expert"])
def test_fused_full_size(name):
    """The benchmark workloads: bitwise against the separate launches (which
    the full-size parity tests check against the oracle), plus sampled
    token rows of Y against the oracle."""
    w = WORKLOADS[name]
    L, inp, ref, got = run_both(w, 0)
    assert_bitwise(ref, got)
    Zo, idx_g = check_route_and_plan(L, inp, w)
    rng = np.random.default_rng(4)
    toks = np.unique(np.concatenate([[0, w.T - 1], rng.choice(w.T, 8, replace=False)]))
    ref_rows = O.moe_forward_dense(inp["X"], weights_dict(inp, as_f64=True), idx_g,
                                   O.gate_weights(Zo, idx_g), toks)
    assert_close("Y[sampled tokens]", to_np(got["Y"])[toks], ref_rows)
