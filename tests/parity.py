"""Shared helpers of the GPU parity tests: run the HIP path, run the oracle
teacher-forced on the GPU's selection, compare."""
from __future__ import annotations

import sys

import numpy as np
import torch

from oracle import moe_oracle as O
from paper_2609_36070_amd.layer import DeviceLayer
from paper_2609_36070_amd.workloads import Workload, make_inputs

REL_TOL = 2e-2           # max|gpu - oracle| <= REL_TOL * max|oracle|, per tensor
LOGIT_ABS_TOL = 1e-4     # router logits: absolute bound (logits are O(1))


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def to_np(t):
    if t.dtype == torch.bfloat16:
        t = t.float()
    return t.detach().cpu().numpy()


def rel_err(gpu, ref):
    gpu = np.asarray(gpu, np.float64)
    ref = np.asarray(ref, np.float64)
    scale = np.abs(ref).max() if ref.size else 0.0
    err = np.abs(gpu - ref).max() if ref.size else 0.0
    return err, scale


def assert_close(name, gpu, ref, rel=REL_TOL):
    err, scale = rel_err(gpu, ref)
    say(f"  {name}: max|err|={err:.3e} max|ref|={scale:.3e}")
    if scale == 0.0:
        assert err <= 1e-6, name
    else:
        assert err <= rel * scale, f"{name}: {err} > {rel} * {scale}"


def weights_dict(inp, as_f64=False):
    keys = ("W_gate", "W_up", "W_down", "Wg_s", "Wu_s", "Wd_s")
    W = {k: inp.get(k) for k in keys}
    if as_f64:
        W = {k: (None if v is None else v.astype(np.float64)) for k, v in W.items()}
    return W


def run_layer(w: Workload, seed=0, inputs=None):
    inp = make_inputs(w, seed) if inputs is None else inputs
    say(f"[gpu] {w.name} T={w.T} d={w.d} E={w.E} k={w.k} f={w.f} f_s={w.f_s} seed={seed}")
    L = DeviceLayer(w, inp)
    L.step()
    torch.cuda.synchronize()
    return L, inp


def check_route_and_plan(L: DeviceLayer, inp, w: Workload):
    """Router (P1, P2a, P2b), weights and plan (P3) against the oracle."""
    Zg = to_np(L.logits)
    Zo = O.router_logits(inp["X"], inp["W_r"], inp.get("bias"))
    delta = float(np.abs(Zg.astype(np.float64) - Zo).max()) if Zo.size else 0.0
    say(f"  logits: delta={delta:.3e}")
    assert delta <= LOGIT_ABS_TOL
    idx_g = to_np(L.topk_idx).astype(np.int32)
    # P2a: selection on the GPU's own logits is exact
    assert np.array_equal(O.topk_select(Zg, w.k), idx_g)
    # P2b: tokens with a margin above 2*delta pick the oracle's experts
    idx_o = O.topk_select(Zo, w.k)
    safe = O.topk_margin(Zo, w.k) > 2 * delta
    assert np.array_equal(idx_o[safe], idx_g[safe])
    n_close = int((~safe).sum())
    n_diff = int((idx_o != idx_g).any(axis=1).sum())
    say(f"  top-k: {n_close} near-tie tokens, {n_diff} differ from the oracle's own selection")
    assert n_close <= max(1, w.T // 1000)
    # weights: the GPU's fp32 softmax on its own logits
    wg = to_np(L.topk_w)
    w_own = O.gate_weights(Zg, idx_g)
    assert np.abs(wg - w_own).max() <= 1e-5
    # P3: plan, bit-exact
    counts, offsets, perm, route_pos = O.plan(idx_g, w.E)
    assert np.array_equal(to_np(L.counts), counts)
    assert np.array_equal(to_np(L.offsets), offsets)
    R = w.T * w.k
    assert np.array_equal(to_np(L.perm)[:R], perm)
    assert np.array_equal(to_np(L.route_pos)[:R], route_pos)
    assert L.error_word() == 0
    return Zo, idx_g
