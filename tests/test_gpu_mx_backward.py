"""GPU parity of the MXFP8 training step: moe_forward_mx with the
pre-activations kept, then moe_backward_mx (§3.4 "MXFP8 Support").

Byte work is bit-exact against the oracle wherever both sides quantise the
same values: dY (per token along d) and the backward weight layouts (W_gate,
W_up along f; W_down along d), and, with the MXFP8 weight gradients, X and dY
along each expert's tokens.  dA, dB and w h are quantised from the GPU's own
fp32 values (and the oracle's fp64 ones), so they, the values the GPU stores
between its passes and everything downstream are floats checked element-wise
against the oracle's own MXFP8 backward to the usual per-tensor bar; no
comparison feeds the oracle a value taken from the GPU.
"""
import numpy as np
import pytest
import torch

from oracle import moe_oracle as O
from oracle import mx_oracle as M
from paper_2609_36070_amd import binding as B
from paper_2609_36070_amd.layer import DeviceLayer
from paper_2609_36070_amd.workloads import WORKLOADS, Workload, make_inputs
from tests.mx_bounds import W_REL, product_allowance, token_qdq_spread
from tests.parity import REL_TOL, assert_close, check_route_and_plan, say, to_np, weights_dict

pytestmark = pytest.mark.gpu


def mx_train_layer(w, seed, wgrad=False):
    inp = make_inputs(w, seed)
    say(f"[gpu] mx train {w.name} T={w.T} d={w.d} E={w.E} k={w.k} f={w.f} f_s={w.f_s} seed={seed}"
        f" mxfp8 wgrad={wgrad}")
    L = DeviceLayer(w, inp, mx=True, mx_wgrad=wgrad)
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


def padded_offsets(L, w):
    """The padded expert offsets: each count rounded up to 128 positions."""
    counts = to_np(L.counts).astype(np.int64)
    poff = np.zeros(w.E + 1, np.int64)
    poff[1:] = np.cumsum((counts + 127) // 128 * 128)
    assert np.array_equal(to_np(L.mx_ws_tensor(B.WS_POFF, torch.int32, (w.E + 1,))), poff)
    return poff


def check_token_codes(L, inp, w, idx_g, experts, cols=None):
    """X^T and dY^T quantised along each expert's tokens (32-position blocks
    from the expert's first row, zeros past its rows), bit-exact against the
    oracle's quantiser on the same values; cols: a sample of the d columns."""
    poff = padded_offsets(L, w)
    if w.k == w.E:
        # dense routing: every expert's rows are the same tokens in the same
        # order, so the library quantises expert 0's range once and every
        # expert's product reads it
        experts = [0]
    _, nbytes = B.moe_mx_workspace_region(L.shape, B.WS_XTQ)
    P = nbytes // w.d
    assert P % 128 == 0 and P >= poff[-1]
    cols = np.arange(w.d) if cols is None else np.asarray(cols)
    sel = torch.as_tensor(cols, device=L.ws.device)
    for key, qw, sw in (("X", B.WS_XTQ, B.WS_XTS), ("dY", B.WS_DYTQ, B.WS_DYTS)):
        q = to_np(L.mx_ws_tensor(qw, torch.uint8, (w.d, P))[sel])
        sc = to_np(L.mx_ws_tensor(sw, torch.uint8, (w.d, P // 32))[sel])
        for e in experts:
            ts = np.nonzero(idx_g == e)[0]              # the expert's rows in plan order
            n = int(poff[e + 1] - poff[e])
            v = np.zeros((n, cols.size))
            v[:ts.size] = inp[key][np.ix_(ts, cols)]
            codes, scales = M.mx_quantize(v, axis=0)
            assert np.array_equal(q[:, poff[e]:poff[e + 1]], codes.T), f"{key}^T[{e}] codes"
            assert np.array_equal(sc[:, poff[e] // 32:poff[e + 1] // 32], scales.T), \
                f"{key}^T[{e}] scales"


def check_route_intermediates(L, w, g, wgrad):
    """What the GPU stored between its passes, element-wise against the
    oracle's own values: the fp32 pre-activations A, B of the forward, and
    dA, dB, w h of the gated-activation backward.  With the MXFP8 weight
    gradients these are the token-axis quantisers' fp32 inputs, and they must
    lie within the quantiser-input window W_REL * max|value| of the oracle's
    (the premise of the weight-gradient allowance); in bf16 they take the
    usual bar."""
    R = w.T * w.k
    offs = to_np(L.offsets)
    keys = [("a", B.WS_AF, torch.float32, REL_TOL), ("b", B.WS_BF, torch.float32, REL_TOL)]
    if wgrad:
        keys += [("dA", B.WS_DAF, torch.float32, W_REL), ("dB", B.WS_DBF, torch.float32, W_REL),
                 ("wh", B.WS_HWF, torch.float32, W_REL)]
    else:
        keys += [("dA", B.WS_DA, torch.bfloat16, REL_TOL), ("dB", B.WS_DB, torch.bfloat16, REL_TOL),
                 ("wh", B.WS_HW, torch.bfloat16, REL_TOL)]
    for key, region, dt, rel in keys:
        got = to_np(L.mx_ws_tensor(region, dt, (R, w.f)))
        ref = np.zeros((R, w.f))
        for e, r in enumerate(g["routes"]):
            if r is not None:
                ref[offs[e]:offs[e + 1]] = r[key]
        assert_close(f"stored {key} ({dt})", got, ref, rel=rel)


def assert_close_allow(name, gpu, ref, allow):
    """max|gpu - ref| <= REL_TOL max|ref| + allow, element by element: the
    per-tensor bar plus the largest change that E4M3 rounding decisions taken
    on quantiser inputs within the window can make (tests/mx_bounds.py)."""
    gpu = np.asarray(gpu, np.float64)
    ref = np.asarray(ref, np.float64)
    err = np.abs(gpu - ref)
    bar = REL_TOL * np.abs(ref).max()
    excess = float((err - allow).max()) if err.size else 0.0
    say(f"  {name}: max|err|={err.max() if err.size else 0:.3e} max|ref|={np.abs(ref).max() if ref.size else 0:.3e}"
        f" max allowance={allow.max() if allow.size else 0:.3e} max(err - allowance)={excess:.3e}"
        f" (bar {bar:.3e})")
    assert np.all(err <= bar + allow), name


def wgrad_allowances(inp, g, idx, E):
    """Per expert, the flip allowances of dW_gate, dW_up (X exact, dA / dB
    ambiguous) and dW_down (w h ambiguous, dY exact), from the oracle's
    operands only (g["routes"][e] holds the expert's dA, dB, w h)."""
    qt = M.mx_qdq_token_blocks
    routes = [r for r in g["routes"] if r is not None]
    win = {key: W_REL * max(float(np.abs(r[key]).max()) for r in routes) for key in ("dA", "dB", "wh")}
    out = []
    for e in range(E):
        r = g["routes"][e]
        if r is None:
            out.append(None)
            continue
        ts = np.nonzero(idx == e)[0]
        xq = qt(inp["X"][ts].astype(np.float64))
        dyq = qt(inp["dY"][ts].astype(np.float64))
        a_g = product_allowance(xq, qt(r["dA"]), None, token_qdq_spread(r["dA"], win["dA"]))
        a_u = product_allowance(xq, qt(r["dB"]), None, token_qdq_spread(r["dB"], win["dB"]))
        a_d = product_allowance(qt(r["wh"]), dyq, token_qdq_spread(r["wh"], win["wh"]), None)
        out.append((a_g, a_u, a_d))
    return out


def check_weight_grads(L, inp, w, g, idx, wgrad):
    names = ("dW_gate", "dW_up", "dW_down")
    if not wgrad:
        for n in names:
            assert_close(n, to_np(getattr(L, n)), g[n])
        return
    allow = wgrad_allowances(inp, g, idx, w.E)
    for i, n in enumerate(names):
        A = np.zeros(getattr(L, n).shape)
        for e, al in enumerate(allow):
            if al is not None:
                A[e] = al[i]
        assert_close_allow(n, to_np(getattr(L, n)), g[n], A)


def mx_backward_parity(w, seed, wgrad=False):
    L, inp = mx_train_layer(w, seed, wgrad)
    Zo, idx_g = check_route_and_plan(L, inp, w)
    w_orc = O.gate_weights(Zo, idx_g)
    check_bwd_weight_codes(L, inp, range(w.E))
    dyq, dys = M.mx_quantize(inp["dY"], axis=1)
    assert np.array_equal(to_np(L.mx_ws_tensor(B.WS_DYQ, torch.uint8, (w.T, w.d))), dyq)
    assert np.array_equal(to_np(L.mx_ws_tensor(B.WS_DYS, torch.uint8, (w.T, w.d // 32))), dys)
    if wgrad:
        check_token_codes(L, inp, w, idx_g, range(w.E))
    g = M.moe_backward_mx(inp["X"], inp["W_r"], weights_dict(inp), idx_g, w_orc, inp["dY"],
                          wgrad_mx=wgrad, keep=True)
    check_route_intermediates(L, w, g, wgrad)
    for n in ("dX", "dZ", "dW_r"):
        assert_close(n, to_np(getattr(L, n)), g[n])
    check_weight_grads(L, inp, w, g, idx_g, wgrad)
    R = w.T * w.k
    dg_pos = to_np(L.mx_ws_tensor(B.WS_DG, torch.float32, (R,)))
    rp = to_np(L.route_pos)[:R]
    assert_close("dg", dg_pos[rp].reshape(w.T, w.k), g["dg"])
    if w.f_s:
        for n in ("dWg_s", "dWu_s", "dWd_s"):
            assert_close(n, to_np(getattr(L, n)), g[n])
    assert L.error_word() == 0
    return L, inp


@pytest.mark.parametrize("wgrad", [False, True], ids=["bf16_wgrad", "mxfp8_wgrad"])
def test_mx_backward_ragged(wgrad):
    mx_backward_parity(Workload("mx_ragged_train", T=1000, d=512, E=6, k=2, f=512, f_s=256,
                                bias_std=0.5, backward=True), seed=31, wgrad=wgrad)


EDGE = [
    Workload("mx_one_token", T=1, d=256, E=8, k=3, f=256, f_s=256, backward=True),
    Workload("mx_k_equals_E", T=300, d=256, E=4, k=4, f=512, bias_std=0.5, backward=True),
    Workload("mx_empty_experts", T=40, d=256, E=64, k=1, f=256, bias_std=3.0, backward=True),
    Workload("mx_many_tiles", T=700, d=768, E=3, k=2, f=768, backward=True),
]


@pytest.mark.parametrize("w", EDGE, ids=lambda w: w.name)
def test_mx_backward_edge_shapes(w):
    mx_backward_parity(w, seed=32)


MANY = [
    Workload("mx_128_experts_train", T=600, d=512, E=128, k=8, f=256, f_s=256, bias_std=0.5,
             backward=True),
    Workload("mx_200_experts_train", T=257, d=768, E=200, k=16, f=256, bias_std=1.0, backward=True),
]


@pytest.mark.parametrize("wgrad", [False, True], ids=["bf16_wgrad", "mxfp8_wgrad"])
@pytest.mark.parametrize("w", MANY, ids=lambda w: w.name)
def test_mx_backward_many_experts(w, wgrad):
    """More than 64 experts (several 64-expert groups in every GEMM's expert
    lookup and in the weight gradients' tile map), many of them with a few
    rows, with both weight-gradient variants."""
    mx_backward_parity(w, seed=33, wgrad=wgrad)


@pytest.mark.parametrize("w", EDGE + [
    Workload("mx_wgrad_block_edges", T=160, d=512, E=5, k=3, f=256, f_s=256, bias_std=1.0,
             backward=True),
    Workload("mx_sixteen_experts", T=333, d=768, E=16, k=5, f=256, f_s=256, backward=True),
], ids=lambda w: w.name)
def test_mx_wgrad_edge_shapes(w):
    """MXFP8 weight gradients: one token per expert, every expert holding
    every token, empty experts, several tiles each way, ragged counts."""
    mx_backward_parity(w, seed=34, wgrad=True)


def test_mx_wgrad_block_aligned_counts():
    """Routes forced so that the experts hold exactly 128, 32, 96, 0 and 256
    rows: regions with no padding, a single 32-block, a partial 128-span, an
    empty expert and two full spans.  The weights are the restricted softmax
    of the GPU's logits over the forced sets."""
    w = Workload("mx_aligned_train", T=256, d=256, E=5, k=2, f=256, f_s=256, backward=True)
    inp = make_inputs(w, 36)
    say(f"[gpu] mx train {w.name} forced counts 128/32/96/0/256, mxfp8 wgrad")
    L = DeviceLayer(w, inp, mx=True, mx_wgrad=True)
    idx = np.empty((w.T, w.k), np.int32)
    idx[:, 1] = 4
    idx[:128, 0], idx[128:160, 0], idx[160:, 0] = 0, 1, 2
    L.route()
    torch.cuda.synchronize()
    wts = O.gate_weights(O.router_logits(inp["X"], inp["W_r"], inp.get("bias")), idx).astype(np.float32)
    L.topk_idx.copy_(torch.from_numpy(idx))
    L.topk_w.copy_(torch.from_numpy(wts))
    L.plan()
    L.forward_mx()
    L.backward_mx()
    torch.cuda.synchronize()
    assert np.array_equal(to_np(L.counts), [128, 32, 96, 0, 256])
    check_token_codes(L, inp, w, idx, range(w.E))
    g = M.moe_backward_mx(inp["X"], inp["W_r"], weights_dict(inp), idx, wts.astype(np.float64),
                          inp["dY"], wgrad_mx=True, keep=True)
    check_route_intermediates(L, w, g, True)
    for n in ("dX", "dZ", "dW_r", "dWg_s", "dWu_s", "dWd_s"):
        assert_close(n, to_np(getattr(L, n)), g[n])
    check_weight_grads(L, inp, w, g, idx, True)
    assert torch.count_nonzero(L.dW_gate[3]) == 0 and torch.count_nonzero(L.dW_down[3]) == 0
    assert L.error_word() == 0


def test_mx_wgrad_changes_only_weight_gradients():
    """The switch changes the three routed weight gradients and nothing else
    (bit-exact), and they stay close to the BF16 ones."""
    w = Workload("mx_switch_train", T=600, d=512, E=4, k=2, f=512, f_s=256, bias_std=0.5,
                 backward=True)
    L, _ = mx_train_layer(w, 35, wgrad=True)
    names = ("Y", "dX", "dW_r", "dZ", "dWg_s", "dWu_s", "dWd_s")
    on = {n: getattr(L, n).clone() for n in names + ("dW_gate", "dW_up", "dW_down")}
    L.mx_wgrad = False
    L.step_mx()
    torch.cuda.synchronize()
    for n in names:
        assert torch.equal(getattr(L, n), on[n]), n
    for n in ("dW_gate", "dW_up", "dW_down"):
        assert not torch.equal(getattr(L, n), on[n]), n
        assert_close(f"{n} mxfp8 vs bf16", to_np(on[n]), to_np(getattr(L, n)), rel=0.2)


@pytest.mark.parametrize("wgrad", [False, True], ids=["bf16_wgrad", "mxfp8_wgrad"])
def test_mx_backward_no_tokens(wgrad):
    w = Workload("mx_none_train", T=0, d=256, E=4, k=2, f=256, f_s=256, backward=True)
    L = DeviceLayer(w, make_inputs(w, 0), mx=True, mx_wgrad=wgrad)
    for n in ("dW_gate", "dW_up", "dW_down", "dW_r", "dWg_s", "dWu_s", "dWd_s"):
        getattr(L, n).fill_(3.0)
    L.step_mx()
    torch.cuda.synchronize()
    for n in ("dW_gate", "dW_up", "dW_down", "dW_r", "dWg_s", "dWu_s", "dWd_s"):
        assert torch.count_nonzero(getattr(L, n)) == 0, n


@pytest.mark.parametrize("wgrad", [False, True], ids=["bf16_wgrad", "mxfp8_wgrad"])
def test_mx_backward_determinism(wgrad):
    w = Workload("mx_det_train", T=1000, d=512, E=6, k=2, f=512, f_s=256, bias_std=0.5,
                 backward=True)
    L, _ = mx_train_layer(w, 33, wgrad)
    names = ("Y", "dX", "dW_gate", "dW_up", "dW_down", "dW_r", "dZ", "dWg_s", "dWu_s", "dWd_s")
    first = {n: getattr(L, n).clone() for n in names}
    for _ in range(3):
        L.step_mx()
        torch.cuda.synchronize()
        for n in names:
            assert torch.equal(getattr(L, n), first[n]), n


@pytest.mark.parametrize("wgrad", [False, True], ids=["bf16_wgrad", "mxfp8_wgrad"])
def test_mx_training_graph_replay(wgrad):
    """route + plan + the MXFP8 forward and backward captured in one HIP
    graph.  Before each replay every output and the whole workspace are
    overwritten by eager fills; every replay equals the eager step bitwise."""
    w = Workload("mx_graph_train", T=500, d=512, E=6, k=2, f=512, f_s=256, bias_std=0.5,
                 backward=True)
    L, _ = mx_train_layer(w, 37, wgrad)
    names = ("logits", "topk_idx", "topk_w", "counts", "offsets", "perm", "route_pos", "Y", "dX",
             "dW_gate", "dW_up", "dW_down", "dW_r", "dZ", "dWg_s", "dWu_s", "dWd_s")
    eager = {n: getattr(L, n).clone() for n in names}
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        L.step_mx()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        L.step_mx()
    torch.cuda.synchronize()
    for rep in range(3):
        for n in names:
            getattr(L, n).fill_(-7 if getattr(L, n).dtype == torch.int32 else 3.0)
        L.ws.fill_(0xA5)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        for n in names:
            assert torch.equal(getattr(L, n), eager[n]), (rep, n)
    assert L.error_word() == 0
    say("  graph replays bitwise equal to eager")


@pytest.mark.parametrize("wgrad", [False, True], ids=["bf16_wgrad", "mxfp8_wgrad"])
def test_mx_training_step_full_size_sampled(wgrad):
    """The training workload in MXFP8: the backward weight codes of two
    experts bit-exact (with the MXFP8 weight gradients also X^T and dY^T of
    two experts on sampled columns); sampled token rows of dX, dZ and dg, and
    weight-gradient columns of two experts, against the oracle's per-token /
    per-column MXFP8 backward."""
    w = WORKLOADS["large_shared_train"]
    L, inp = mx_train_layer(w, 0, wgrad)
    check_bwd_weight_codes(L, inp, [0, w.E - 1])
    Zo, idx_g = check_route_and_plan(L, inp, w)
    if wgrad:
        check_token_codes(L, inp, w, idx_g, [0, w.E - 1],
                          cols=np.r_[0:32, 3000:3008, w.d - 32:w.d])
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
    offs = to_np(L.offsets)
    qt = M.mx_qdq_token_blocks
    for e in (0, w.E - 1):
        a, b, c, ops = M.mx_expert_weight_grad_columns(inp["X"], W, idx_g, w_orc, inp["dY"], e,
                                                       cols, wgrad_mx=wgrad, keep=True)
        got = (to_np(L.dW_gate[e])[:, cols], to_np(L.dW_up[e])[:, cols],
               to_np(L.dW_down[e])[cols, :])
        names = (f"dW_gate[{e}][:, cols]", f"dW_up[{e}][:, cols]", f"dW_down[{e}][cols, :]")
        if not wgrad:
            for n, gv, ref in zip(names, got, (a, b, c)):
                assert_close(n, gv, ref)
            continue
        # the quantiser inputs the GPU stored, on the sampled columns, within
        # the window of the oracle's (windows from these columns' maxima)
        sel = torch.as_tensor(cols, device=L.ws.device)
        win = {}
        for key, region in (("dA", B.WS_DAF), ("dB", B.WS_DBF), ("wh", B.WS_HWF)):
            got_op = to_np(L.mx_ws_tensor(region, torch.float32, (R, w.f))[offs[e]:offs[e + 1]][:, sel])
            win[key] = W_REL * float(np.abs(ops[key]).max())
            assert_close(f"stored {key}[{e}][:, cols]", got_op, ops[key], rel=W_REL)
        ts = np.nonzero(idx_g == e)[0]
        xq = qt(inp["X"][ts].astype(np.float64))
        dyq = qt(inp["dY"][ts].astype(np.float64))
        allow = (product_allowance(xq, qt(ops["dA"]), None, token_qdq_spread(ops["dA"], win["dA"])),
                 product_allowance(xq, qt(ops["dB"]), None, token_qdq_spread(ops["dB"], win["dB"])),
                 product_allowance(qt(ops["wh"]), dyq, token_qdq_spread(ops["wh"], win["wh"]), None))
        for n, gv, ref, al in zip(names, got, (a, b, c), allow):
            assert_close_allow(n, gv, ref, al)
    assert L.error_word() == 0
