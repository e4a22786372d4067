"""GPU parity at sizes the oracle evaluates in full (every output element).

Shapes span several MFMA tiles in M, N and K with ragged expert regions, plus
the degenerate cases: one token, k = E, empty experts, no tokens.
"""
import numpy as np
import pytest
import torch

from oracle import moe_oracle as O
from paper_2609_36070_amd import binding as B
from paper_2609_36070_amd.workloads import WORKLOADS, Workload
from tests.parity import (assert_close, check_route_and_plan, run_layer, say, to_np,
                          weights_dict)

pytestmark = pytest.mark.gpu

RAGGED_TRAIN = Workload("ragged_train", T=1000, d=512, E=6, k=2, f=512, f_s=256, bias_std=0.5,
                        backward=True)


def forward_parity(w, seed=0):
    L, inp = run_layer(w, seed)
    Zo, idx_g = check_route_and_plan(L, inp, w)
    w_orc = O.gate_weights(Zo, idx_g)
    fw = O.moe_forward(inp["X"], weights_dict(inp), idx_g, w_orc)
    R = w.T * w.k
    assert_close("Y", to_np(L.Y), fw["Y"])
    H = to_np(L.ws_tensor(B.WS_H, torch.bfloat16, (R, w.f)))
    if w.k == w.E:
        # dense routing: H holds w h (the combine is folded into the down
        # product, so there is no Yexp and no Ysh)
        perm = O.plan(idx_g, w.E)[2]
        w_pos = w_orc.reshape(-1)[perm][:, None]
        assert_close("w H", H, w_pos * fw["H"])
    else:
        assert_close("H", H, fw["H"])
        assert_close("Yexp", to_np(L.ws_tensor(B.WS_YEXP, torch.bfloat16, (R, w.d))), fw["Yexp"])
        if w.f_s:
            assert_close("Ysh", to_np(L.ws_tensor(B.WS_YSH, torch.bfloat16, (w.T, w.d))), fw["Ysh"])
    if w.backward:
        assert_close("A", to_np(L.ws_tensor(B.WS_A, torch.bfloat16, (R, w.f))), fw["A"])
        assert_close("B", to_np(L.ws_tensor(B.WS_B, torch.bfloat16, (R, w.f))), fw["B"])
    return L, inp, Zo, idx_g, w_orc


def backward_parity(L, inp, w, idx_g, w_orc):
    g = O.moe_backward(inp["X"], inp["W_r"], weights_dict(inp), idx_g, w_orc, inp["dY"])
    assert_close("dX", to_np(L.dX), g["dX"])
    assert_close("dW_gate", to_np(L.dW_gate), g["dW_gate"])
    assert_close("dW_up", to_np(L.dW_up), g["dW_up"])
    assert_close("dW_down", to_np(L.dW_down), g["dW_down"])
    assert_close("dZ", to_np(L.dZ), g["dZ"])
    assert_close("dW_r", to_np(L.dW_r), g["dW_r"])
    R = w.T * w.k
    dg_pos = to_np(L.ws_tensor(B.WS_DG, torch.float32, (R,)))
    rp = to_np(L.route_pos)[:R]
    assert_close("dg", dg_pos[rp].reshape(w.T, w.k), g["dg"])
    if w.f_s:
        assert_close("dWg_s", to_np(L.dWg_s), g["dWg_s"])
        assert_close("dWu_s", to_np(L.dWu_s), g["dWu_s"])
        assert_close("dWd_s", to_np(L.dWd_s), g["dWd_s"])


def test_tiny_forward():
    forward_parity(WORKLOADS["tiny"])


def test_ragged_forward_backward():
    L, inp, Zo, idx_g, w_orc = forward_parity(RAGGED_TRAIN, seed=1)
    backward_parity(L, inp, RAGGED_TRAIN, idx_g, w_orc)


@pytest.mark.parametrize("w", [
    Workload("one_token", T=1, d=256, E=8, k=3, f=256, f_s=256, backward=True),
    Workload("k_equals_E", T=300, d=256, E=4, k=4, f=512, bias_std=0.5, backward=True),
    Workload("empty_experts", T=40, d=256, E=64, k=1, f=256, bias_std=3.0, backward=True),
    Workload("many_tiles", T=700, d=768, E=3, k=2, f=768, backward=True),
    # the small-expert-count reverse combine: 16 experts with a token count
    # that leaves a partial token group and a partial 128-chunk column block;
    # 8 experts over two column blocks, the second partial
    Workload("sixteen_experts", T=333, d=768, E=16, k=5, f=256, f_s=256, bias_std=0.5,
             backward=True),
    Workload("eight_experts_wide", T=77, d=1280, E=8, k=2, f=256, bias_std=0.5, backward=True),
    # dense routing (k == E) with a shared expert: the combines fold into the
    # down and dX products; a partial token tile, several column tiles, a
    # shared width that differs from the routed one, and one expert
    Workload("dense_shared", T=555, d=768, E=6, k=6, f=256, f_s=512, bias_std=0.5, backward=True),
    Workload("dense_one_expert", T=260, d=512, E=1, k=1, f=512, f_s=256, backward=True),
    Workload("dense_sixteen", T=130, d=256, E=16, k=16, f=256, backward=True),
    # the router for 128 or more experts (d sliced across blocks, partial
    # logits added in a reduce kernel) through a whole training step, with a
    # padded expert count, empty experts and k = 16
    Workload("experts_128_train", T=600, d=512, E=128, k=8, f=256, f_s=256, bias_std=0.5,
             backward=True),
    Workload("experts_200_train", T=257, d=768, E=200, k=16, f=256, bias_std=1.0, backward=True),
], ids=lambda w: w.name)
def test_edge_shapes(w):
    L, inp, Zo, idx_g, w_orc = forward_parity(w, seed=2)
    counts = to_np(L.counts)
    if w.name == "empty_experts":
        assert (counts == 0).any()
    backward_parity(L, inp, w, idx_g, w_orc)


def test_no_tokens():
    w = Workload("no_tokens", T=0, d=256, E=8, k=2, f=256, f_s=256, backward=True)
    inp = {"X": np.zeros((0, 256), np.float32), "W_r": np.ones((256, 8), np.float32),
           "bias": None,
           "W_gate": np.ones((8, 256, 256), np.float32), "W_up": np.ones((8, 256, 256), np.float32),
           "W_down": np.ones((8, 256, 256), np.float32),
           "Wg_s": np.ones((256, 256), np.float32), "Wu_s": np.ones((256, 256), np.float32),
           "Wd_s": np.ones((256, 256), np.float32), "dY": np.zeros((0, 256), np.float32)}
    L, _ = run_layer(w, inputs=inp)
    assert np.all(to_np(L.counts) == 0) and np.all(to_np(L.offsets) == 0)
    for name in ("dW_gate", "dW_up", "dW_down", "dW_r", "dWg_s", "dWu_s", "dWd_s"):
        assert np.all(to_np(getattr(L, name)) == 0), name


def test_identical_experts_router_gradient_vanishes():
    w = Workload("identical", T=200, d=256, E=8, k=2, f=256, backward=True)
    from paper_2609_36070_amd.workloads import make_inputs
    inp = make_inputs(w, 3)
    for key in ("W_gate", "W_up", "W_down"):
        inp[key] = np.repeat(inp[key][:1], w.E, axis=0)
    L, _ = run_layer(w, inputs=inp)
    dZ = to_np(L.dZ)
    Y = to_np(L.Y).astype(np.float64)
    ref = O.expert_ffn(inp["X"], inp["W_gate"][0], inp["W_up"][0], inp["W_down"][0])
    assert_close("Y(identical)", Y, ref)
    # dg is equal across a token's slots up to bf16 rounding, so dZ is tiny
    assert np.abs(dZ).max() <= 2e-2 * np.abs(to_np(L.ws_tensor(B.WS_DG, torch.float32,
                                                               (w.T * w.k,)))).max()


def test_saturated_gated_activation():
    """Gate weights scaled by 64 (a power of two, so still bf16-exact): the
    gate pre-activations reach a few hundred in magnitude, so the logistic
    function saturates at 0 and 1 and its exponential overflows for the most
    negative ones.  Forward and backward against the oracle, every element."""
    w = Workload("saturated", T=300, d=256, E=4, k=2, f=256, f_s=256, bias_std=0.5, backward=True)
    from paper_2609_36070_amd.workloads import make_inputs
    inp = make_inputs(w, 7)
    for key in ("W_gate", "Wg_s"):
        inp[key] = inp[key] * np.float32(64.0)
    L, _ = run_layer(w, inputs=inp)
    Zo, idx_g = check_route_and_plan(L, inp, w)
    w_orc = O.gate_weights(Zo, idx_g)
    fw = O.moe_forward(inp["X"], weights_dict(inp), idx_g, w_orc)
    amax = float(np.abs(fw["A"]).max())
    say(f"  max |a| = {amax:.1f}")
    assert amax > 100.0, "the fixture must reach the saturated range"
    assert_close("Y", to_np(L.Y), fw["Y"])
    R = w.T * w.k
    assert_close("H", to_np(L.ws_tensor(B.WS_H, torch.bfloat16, (R, w.f))), fw["H"])
    backward_parity(L, inp, w, idx_g, w_orc)


def test_bad_expert_index_sets_error_word():
    w = Workload("bad_idx", T=64, d=256, E=8, k=2, f=256)
    from paper_2609_36070_amd.workloads import make_inputs
    L, inp = run_layer(w, inputs=make_inputs(w, 4))
    idx = L.topk_idx.clone()
    idx[5, 1] = 9          # out of range
    idx[7, 0] = -1
    L.topk_idx.copy_(idx)
    L.plan()
    torch.cuda.synchronize()
    assert L.error_word() == 1
    assert int(to_np(L.offsets)[-1]) == w.T * w.k - 2
    rp = to_np(L.route_pos)
    assert rp[5 * 2 + 1] == -1 and rp[7 * 2] == -1
    L.forward()   # must stay in bounds with unplaced routes
    torch.cuda.synchronize()
    L.topk_idx.copy_(torch.clamp(idx, 0, w.E - 1))
    L.plan()
    torch.cuda.synchronize()
    assert L.error_word() == 0


def test_dispatch_matches_gather():
    w = Workload("dispatch", T=333, d=512, E=5, k=2, f=256, bias_std=0.5)
    from paper_2609_36070_amd.workloads import make_inputs
    inp = make_inputs(w, 5)
    L, _ = run_layer(w, inputs=inp)
    R = w.T * w.k
    Xperm = torch.empty((R, w.d), dtype=torch.bfloat16, device="cuda")
    B.moe_dispatch(L.shape, L.X, L.plan_bufs, Xperm)
    torch.cuda.synchronize()
    perm = to_np(L.perm)[:R]
    assert np.array_equal(to_np(Xperm), inp["X"][perm // w.k])


def test_determinism_bitwise_repeat():
    w = RAGGED_TRAIN
    from paper_2609_36070_amd.workloads import make_inputs
    L, _ = run_layer(w, inputs=make_inputs(w, 6))
    names = ("logits", "topk_idx", "topk_w", "perm", "route_pos", "Y", "dX", "dW_gate", "dW_up",
             "dW_down", "dW_r", "dZ", "dWg_s", "dWu_s", "dWd_s")
    first = {n: getattr(L, n).clone() for n in names}
    for rep in range(3):
        L.step()
        torch.cuda.synchronize()
        for n in names:
            assert torch.equal(getattr(L, n), first[n]), (rep, n)


def test_graph_capture_replays_match_eager():
    """The whole step captured in a HIP graph; every replay equals the eager run bitwise."""
    from paper_2609_36070_amd.workloads import make_inputs
    w = RAGGED_TRAIN
    L, _ = run_layer(w, inputs=make_inputs(w, 7))
    names = ("logits", "topk_idx", "topk_w", "counts", "offsets", "perm", "route_pos", "Y", "dX",
             "dW_gate", "dW_up", "dW_down", "dW_r", "dZ", "dWg_s", "dWu_s", "dWd_s")
    eager = {n: getattr(L, n).clone() for n in names}
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        L.step()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        L.step()
    torch.cuda.synchronize()
    for rep in range(3):
        for n in names:                     # eager work between replays: clobber every output
            getattr(L, n).fill_(-7 if getattr(L, n).dtype == torch.int32 else 3.0)
        L.ws.fill_(0xA5)                    # and the workspace: nothing carries over between steps
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        for n in names:
            assert torch.equal(getattr(L, n), eager[n]), (rep, n)
    say("  graph replays bitwise equal to eager")


def test_two_layers_on_two_streams():
    """Two layers with their own workspaces, one stepping in BF16 and one in
    MXFP8 (MXFP8 weight gradients), issued alternately on two streams so that
    their kernels overlap, give the same bits as their stand-alone steps: the
    library keeps no state outside the buffers it is given."""
    from paper_2609_36070_amd.layer import DeviceLayer
    from paper_2609_36070_amd.workloads import make_inputs
    w = RAGGED_TRAIN
    say(f"[gpu] two streams: {w.name} BF16 seed 41 and MXFP8 seed 42")
    a = DeviceLayer(w, make_inputs(w, 41))
    b = DeviceLayer(w, make_inputs(w, 42), mx=True, mx_wgrad=True)
    names = ("Y", "dX", "dW_gate", "dW_up", "dW_down", "dW_r", "dZ", "dWg_s", "dWu_s", "dWd_s")
    a.step()
    b.step_mx()
    torch.cuda.synchronize()
    ref_a = {n: getattr(a, n).clone() for n in names}
    ref_b = {n: getattr(b, n).clone() for n in names}
    sa, sb = torch.cuda.Stream(), torch.cuda.Stream()
    sa.wait_stream(torch.cuda.current_stream())
    sb.wait_stream(torch.cuda.current_stream())
    for _ in range(3):
        with torch.cuda.stream(sa):
            a.step()
        with torch.cuda.stream(sb):
            b.step_mx()
    torch.cuda.synchronize()
    for n in names:
        assert torch.equal(getattr(a, n), ref_a[n]), ("bf16", n)
        assert torch.equal(getattr(b, n), ref_b[n]), ("mxfp8", n)
    assert a.error_word() == 0 and b.error_word() == 0
