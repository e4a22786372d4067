"""Pins of the CPU oracle against facts that do not come from the oracle itself.

Every test here runs on the CPU.  Each pins one part of the oracle to brute
force, a hand-worked example, a closed form, a special case that reduces to a
library routine, or finite differences, so that a dropped term, a wrong sign,
a wrong index or a transposed operand in the oracle fails at least one of them
(tests/test_oracle_mutations.py plants such mistakes and checks that).
"""
import itertools
import os

import numpy as np
import pytest
import torch

from oracle import moe_oracle as O

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _rng(seed=0):
    return np.random.default_rng(seed)


def _bf16(a):
    from paper_2609_36070_amd.workloads import to_bf16
    return to_bf16(np.asarray(a, np.float32))


def small_layer(T=12, d=16, E=6, k=2, f=8, f_s=0, seed=0, identical=False):
    rng = _rng(seed)
    X = _bf16(rng.standard_normal((T, d)))
    W_r = _bf16(rng.standard_normal((d, E)) / np.sqrt(d))
    W = dict(
        W_gate=_bf16(rng.standard_normal((E, d, f)) / np.sqrt(d)),
        W_up=_bf16(rng.standard_normal((E, d, f)) / np.sqrt(d)),
        W_down=_bf16(rng.standard_normal((E, f, d)) / np.sqrt(f)),
    )
    if identical:
        for key in ("W_gate", "W_up", "W_down"):
            W[key] = np.repeat(W[key][:1], E, axis=0)
    if f_s:
        W["Wg_s"] = _bf16(rng.standard_normal((d, f_s)) / np.sqrt(d))
        W["Wu_s"] = _bf16(rng.standard_normal((d, f_s)) / np.sqrt(d))
        W["Wd_s"] = _bf16(rng.standard_normal((f_s, d)) / np.sqrt(f_s))
    dY = _bf16(rng.standard_normal((T, d)))
    return X, W_r, W, dY


# ---------------------------------------------------------------------------
# top-k
# ---------------------------------------------------------------------------

def brute_force_topk(z, k):
    """The unique k-subset whose every key (-z_e, e) precedes every unselected key."""
    E = len(z)
    found = []
    for sub in itertools.combinations(range(E), k):
        rest = [e for e in range(E) if e not in sub]
        if all((-z[a], a) < (-z[b], b) for a in sub for b in rest):
            found.append(list(sub))
    assert len(found) == 1
    return found[0]


@pytest.mark.parametrize("k", [1, 2, 3, 8])
def test_topk_brute_force_random_and_tied(k):
    rng = _rng(k)
    E = 8
    rows = [rng.standard_normal(E).astype(np.float32) for _ in range(40)]
    # heavy ties: small integers
    rows += [rng.integers(-2, 3, E).astype(np.float32) for _ in range(60)]
    Z = np.stack(rows)
    got = O.topk_select(Z, k)
    for t in range(Z.shape[0]):
        assert list(got[t]) == brute_force_topk([float(v) for v in Z[t]], k)


def _read_golden_topk():
    cases = []
    with open(os.path.join(GOLDEN, "topk_ties.txt")) as fh:
        for line in fh:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            k, logits, bias, exp = [p.strip() for p in line.split("|")]
            cases.append((int(k), [int(v) for v in logits.split()],
                          [int(v) for v in bias.split()], [int(v) for v in exp.split()]))
    return cases


def test_topk_exact_ties_golden():
    for k, logits, bias, expected in _read_golden_topk():
        E = len(logits)
        d = 4
        X = np.zeros((1, d), np.float32)
        X[0, 1] = 1.0                     # one-hot token
        W_r = np.zeros((d, E), np.float32)
        W_r[1] = logits
        Z = O.router_logits(X, W_r, np.array(bias, np.float32))
        assert list(O.topk_select(Z, k)[0]) == expected


def test_gate_weights_closed_forms():
    rng = _rng(3)
    Z = rng.standard_normal((50, 16)).astype(np.float32)
    for k in (1, 2, 5, 16):
        idx = O.topk_select(Z, k)
        w = O.gate_weights(Z, idx)
        assert np.allclose(w.sum(axis=1), 1.0, atol=1e-12, rtol=0)
        # restricted softmax exp(z_s) / sum_{selected} exp(z): a second formulation
        zs = np.take_along_axis(Z.astype(np.float64), idx.astype(np.int64), axis=1)
        ref = np.exp(zs) / np.exp(zs).sum(axis=1, keepdims=True)
        assert np.allclose(w, ref, atol=1e-13, rtol=0)
        # larger logit -> larger weight
        assert np.all((np.diff(zs, axis=1) > 0) == (np.diff(w, axis=1) > 0))
    # equal logits -> 1/k
    for k in (2, 8):
        Z = np.zeros((3, 8), np.float32)
        w = O.gate_weights(Z, O.topk_select(Z, k))
        assert np.allclose(w, 1.0 / k, atol=1e-15, rtol=0)
    # k = 1 -> weight exactly 1
    Z = rng.standard_normal((10, 8)).astype(np.float32)
    assert np.all(O.gate_weights(Z, O.topk_select(Z, 1)) == 1.0)


def test_gate_weights_match_torch_softmax_for_k_equal_E():
    rng = _rng(4)
    Z = rng.standard_normal((20, 8)).astype(np.float32)
    idx = O.topk_select(Z, 8)
    assert np.all(idx == np.arange(8))
    ref = torch.softmax(torch.from_numpy(Z).double(), dim=1).numpy()
    assert np.allclose(O.gate_weights(Z, idx), ref, atol=1e-14, rtol=0)


def test_topk_margin():
    Z = np.array([[3, 1, 2, 0.5], [1, 1, 1, 1]], np.float32)
    assert np.allclose(O.topk_margin(Z, 2), [1.0, 0.0])
    assert np.all(np.isinf(O.topk_margin(Z, 4)))


# ---------------------------------------------------------------------------
# dispatch schedule
# ---------------------------------------------------------------------------

def _read_golden_alg1():
    cases = []
    with open(os.path.join(GOLDEN, "alg1_two_ranks.txt")) as fh:
        for line in fh:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            c, M, S, Phi = [p.strip() for p in line.split("|")]
            M = np.array([[int(v) for v in row.split()] for row in M.split(";")])
            S = np.array([int(v) for v in S.split()])
            Phi = np.array([[int(x) for x in pair.split(",")] for pair in Phi.split()])
            cases.append((int(c), M, S, Phi))
    return cases


def test_algorithm1_hand_worked_two_ranks():
    A = np.array([[0, 1, 1, 2, 0, 3], [1, 0, 3, 0, 0, 1]])
    for c, M, S, Phi in _read_golden_alg1():
        gM, gS, gPhi = O.schedule(A, 2, c)
        assert np.array_equal(gM, M) and np.array_equal(gS, S)
        assert np.array_equal(gPhi, Phi)


@pytest.mark.parametrize("R,L,N,K,c", [(1, 8, 50, 2, 0), (3, 4, 20, 3, 1), (4, 2, 16, 2, 3),
                                       (2, 5, 30, 4, 0), (1, 1, 7, 1, 0), (5, 3, 12, 2, 4)])
def test_schedule_positions_follow_algorithm1_formula(R, L, N, K, c):
    """Every scheduled route sits where Algorithm 1's position formula puts it:
    p = S[l] + sum_r' min(M[r', l], o) + #{r' < r : M[r', l] > o}, with o the
    number of earlier routes of rank r to the same expert.  Also: Phi lists
    every local route exactly once, each expert's rows form one contiguous
    region starting at S[l], a rank's routes keep their order inside it, and
    the ranks take turns (the i-th routes of all ranks precede the
    (i+1)-th)."""
    rng = _rng(R * 100 + L)
    # distinct experts per token, as top-K selection produces
    A = np.stack([np.concatenate([rng.choice(R * L, K, replace=False) for _ in range(N)])
                  for _ in range(R)])
    M, S, Phi = O.schedule(A, L, c)
    # counts and region starts from their definitions
    for r in range(R):
        for l in range(L):
            assert M[r, l] == int(np.sum(A[r] == c * L + l))
    assert np.array_equal(S, np.concatenate([[0], np.cumsum(M.sum(0))[:-1]]))
    local = [(r, j) for r in range(R) for j in range(A.shape[1]) if c * L <= A[r, j] < (c + 1) * L]
    assert sorted(map(tuple, Phi.tolist())) == sorted(local)      # each local route once
    for p, (r, j) in enumerate(Phi):
        l = A[r, j] - c * L
        o = int(np.sum(A[r, :j] == A[r, j]))
        want = S[l] + sum(min(int(M[q, l]), o) for q in range(R)) \
            + sum(1 for q in range(r) if M[q, l] > o)
        assert p == want, (p, r, j)
    for l in range(L):
        reg = Phi[S[l]:S[l] + M[:, l].sum()]
        assert np.all(A[reg[:, 0], reg[:, 1]] == c * L + l)          # contiguous region
        for r in range(R):
            js = reg[reg[:, 0] == r, 1]
            assert np.all(np.diff(js) > 0)                          # rank order kept
        # round robin: position of each rank's i-th route grows with i, and
        # all i-th routes come before any (i+1)-th one
        ords = [int(np.sum(A[r, :j] == A[r, j])) for r, j in reg]
        assert ords == sorted(ords)


def test_plan_invariants_and_stable_sort():
    rng = _rng(7)
    for T, E, k in [(37, 8, 2), (64, 16, 4), (10, 3, 3), (1, 4, 1), (200, 64, 8)]:
        Z = rng.standard_normal((T, E)).astype(np.float32)
        Z[:, 0] += 1.5  # skew toward expert 0
        idx = O.topk_select(Z, k)
        counts, offsets, perm, route_pos = O.plan(idx, E)
        flat = idx.reshape(-1)
        R = T * k
        assert counts.sum() == R and offsets[E] == R            # nothing dropped
        assert np.array_equal(counts, np.bincount(flat, minlength=E))
        assert np.array_equal(offsets[:E], np.concatenate([[0], np.cumsum(counts)[:-1]]))
        assert np.array_equal(np.sort(perm), np.arange(R))      # a permutation
        assert np.array_equal(route_pos[perm], np.arange(R))    # inverse
        assert np.array_equal(perm, np.argsort(flat, kind="stable"))
        for e in range(E):
            seg = perm[offsets[e]:offsets[e + 1]]
            assert np.all(flat[seg] == e) and np.all(np.diff(seg) > 0)


def test_plan_empty_experts():
    idx = np.array([[0, 3], [0, 3], [3, 5]], np.int32)
    counts, offsets, perm, route_pos = O.plan(idx, 6)
    assert list(counts) == [2, 0, 0, 3, 0, 1]
    assert list(offsets) == [0, 2, 2, 2, 5, 5, 6]
    assert list(perm) == [0, 2, 1, 3, 4, 5]


# ---------------------------------------------------------------------------
# forward
# ---------------------------------------------------------------------------

def _torch_swiglu(x, Wg, Wu, Wd):
    x = torch.from_numpy(np.asarray(x, np.float64))
    g = x @ torch.from_numpy(np.asarray(Wg, np.float64))
    u = x @ torch.from_numpy(np.asarray(Wu, np.float64))
    return (torch.nn.functional.silu(g) * u) @ torch.from_numpy(np.asarray(Wd, np.float64))


def test_single_expert_is_plain_swiglu_ffn():
    X, W_r, W, _ = small_layer(T=9, d=16, E=1, k=1, f=24)
    Z = O.router_logits(X, W_r)
    idx = O.topk_select(Z, 1)
    w = O.gate_weights(Z, idx)
    ref = _torch_swiglu(X, W["W_gate"][0], W["W_up"][0], W["W_down"][0]).numpy()
    assert np.allclose(O.moe_forward(X, W, idx, w)["Y"], ref, atol=1e-12, rtol=0)
    assert np.allclose(O.moe_forward_dense(X, W, idx, w), ref, atol=1e-12, rtol=0)


def test_k_equal_E_is_dense_softmax_mixture():
    X, W_r, W, _ = small_layer(T=10, d=16, E=4, k=4, f=8, f_s=12)
    Z = O.router_logits(X, W_r)
    idx = O.topk_select(Z, 4)
    w = O.gate_weights(Z, idx)
    p = torch.softmax(torch.from_numpy(Z).double(), dim=1)
    ref = _torch_swiglu(X, W["Wg_s"], W["Wu_s"], W["Wd_s"])
    for e in range(4):
        ref = ref + p[:, e:e + 1] * _torch_swiglu(X, W["W_gate"][e], W["W_up"][e], W["W_down"][e])
    assert np.allclose(O.moe_forward(X, W, idx, w)["Y"], ref.numpy(), atol=1e-12, rtol=0)


def test_identical_experts_ignore_routing():
    X, W_r, W, _ = small_layer(T=15, d=16, E=6, k=3, f=8, f_s=8, identical=True)
    Z = O.router_logits(X, W_r)
    idx = O.topk_select(Z, 3)
    w = O.gate_weights(Z, idx)
    ref = _torch_swiglu(X, W["W_gate"][0], W["W_up"][0], W["W_down"][0]) \
        + _torch_swiglu(X, W["Wg_s"], W["Wu_s"], W["Wd_s"])
    assert np.allclose(O.moe_forward(X, W, idx, w)["Y"], ref.numpy(), atol=1e-12, rtol=0)


def test_dense_and_permuted_forward_agree():
    X, W_r, W, _ = small_layer(T=33, d=16, E=7, k=3, f=8, f_s=4, seed=5)
    Z = O.router_logits(X, W_r)
    idx = O.topk_select(Z, 3)
    w = O.gate_weights(Z, idx)
    fw = O.moe_forward(X, W, idx, w)
    assert np.allclose(fw["Y"], O.moe_forward_dense(X, W, idx, w), atol=1e-12, rtol=0)
    # the kept intermediates follow their definitions in plan order
    tok = fw["perm"] // 3
    for p in (0, 17, 98):
        e = int(np.searchsorted(fw["offsets"], p, side="right") - 1)
        ref = _torch_swiglu(X[tok[p]:tok[p] + 1], W["W_gate"][e], W["W_up"][e], W["W_down"][e])
        assert np.allclose(fw["Yexp"][p], ref.numpy()[0], atol=1e-12)


def test_forward_matches_torch_layer_with_library_topk():
    """The whole layer against torch.topk / torch.softmax on tie-free logits."""
    X, W_r, W, _ = small_layer(T=25, d=16, E=8, k=3, f=8, f_s=8, seed=11)
    bias = np.array([0.3, -0.2, 0, 0.1, 0.5, -0.4, 0.2, 0], np.float32)
    Z = O.router_logits(X, W_r, bias)
    zt = torch.from_numpy(Z).double()
    vals, ind = torch.topk(zt, 3, dim=1)
    ind_sorted, order = torch.sort(ind, dim=1)
    assert np.array_equal(O.topk_select(Z, 3), ind_sorted.numpy())
    s = torch.softmax(zt, dim=1).gather(1, ind_sorted)
    s = s / s.sum(1, keepdim=True)
    ref = _torch_swiglu(X, W["Wg_s"], W["Wu_s"], W["Wd_s"])
    for t in range(25):
        for slot in range(3):
            e = int(ind_sorted[t, slot])
            ref[t] += s[t, slot] * _torch_swiglu(X[t:t + 1], W["W_gate"][e], W["W_up"][e],
                                                W["W_down"][e])[0]
    idx = O.topk_select(Z, 3)
    out = O.moe_forward(X, W, idx, O.gate_weights(Z, idx))["Y"]
    assert np.allclose(out, ref.numpy(), atol=1e-12, rtol=0)


# ---------------------------------------------------------------------------
# backward
# ---------------------------------------------------------------------------

def _loss(X, W_r, bias, W, idx, dY):
    """<dY, Y> with the selection held fixed and fp64 logits."""
    Z = O.router_logits(X, W_r, bias, out_dtype=np.float64)
    w = O.gate_weights(Z, idx)
    return float((O.moe_forward_dense(X, W, idx, w) * dY).sum())


def test_backward_central_finite_differences():
    T, d, E, k, f, fs = 4, 8, 4, 2, 8, 8
    X, W_r, W, dY = small_layer(T=T, d=d, E=E, k=k, f=f, f_s=fs, seed=21)
    X = X.astype(np.float64)
    W_r = W_r.astype(np.float64)
    W = {key: v.astype(np.float64) for key, v in W.items()}
    bias = np.array([0.1, -0.3, 0.2, 0.0])
    idx = O.topk_select(O.router_logits(X, W_r, bias), k)
    w = O.gate_weights(O.router_logits(X, W_r, bias, out_dtype=np.float64), idx)
    g = O.moe_backward(X, W_r, W, idx, w, dY)
    h = 1e-6
    rng = _rng(1)

    def check(name, arr, grad, n=12):
        flat = arr.reshape(-1)
        for i in rng.choice(flat.size, size=min(n, flat.size), replace=False):
            old = flat[i]
            flat[i] = old + h
            lp = _loss(X, W_r, bias, W, idx, dY)
            flat[i] = old - h
            lm = _loss(X, W_r, bias, W, idx, dY)
            flat[i] = old
            fd = (lp - lm) / (2 * h)
            assert abs(fd - grad.reshape(-1)[i]) <= 1e-6 * max(1.0, abs(fd)), (name, i, fd)

    check("X", X, g["dX"], n=32)
    check("W_r", W_r, g["dW_r"], n=32)
    check("W_gate", W["W_gate"], g["dW_gate"])
    check("W_up", W["W_up"], g["dW_up"])
    check("W_down", W["W_down"], g["dW_down"])
    check("Wg_s", W["Wg_s"], g["dWg_s"])
    check("Wu_s", W["Wu_s"], g["dWu_s"])
    check("Wd_s", W["Wd_s"], g["dWd_s"])


def test_backward_matches_torch_autograd():
    T, d, E, k, f, fs = 9, 16, 5, 2, 8, 6
    X, W_r, W, dY = small_layer(T=T, d=d, E=E, k=k, f=f, f_s=fs, seed=31)
    Z = O.router_logits(X, W_r)
    idx = O.topk_select(Z, k)
    w = O.gate_weights(O.router_logits(X, W_r, out_dtype=np.float64), idx)
    g = O.moe_backward(X, W_r, W, idx, w, dY)

    tt = {n: torch.tensor(np.asarray(v, np.float64), requires_grad=True)
          for n, v in dict(X=X, W_r=W_r, **W).items()}
    zt = tt["X"] @ tt["W_r"]
    it = torch.from_numpy(idx.astype(np.int64))
    s = torch.softmax(zt.gather(1, it), dim=1)
    act = torch.nn.functional.silu
    Y = (act(tt["X"] @ tt["Wg_s"]) * (tt["X"] @ tt["Wu_s"])) @ tt["Wd_s"]
    for slot in range(k):
        e = it[:, slot]
        a = torch.einsum("td,tdf->tf", tt["X"], tt["W_gate"][e])
        b = torch.einsum("td,tdf->tf", tt["X"], tt["W_up"][e])
        o = torch.einsum("tf,tfd->td", act(a) * b, tt["W_down"][e])
        Y = Y + s[:, slot:slot + 1] * o
    (Y * torch.from_numpy(dY.astype(np.float64))).sum().backward()
    pairs = dict(dX="X", dW_r="W_r", dW_gate="W_gate", dW_up="W_up", dW_down="W_down",
                 dWg_s="Wg_s", dWu_s="Wu_s", dWd_s="Wd_s")
    for ours, theirs in pairs.items():
        assert np.allclose(g[ours], tt[theirs].grad.numpy(), atol=1e-11, rtol=1e-9), ours


def test_router_gradient_identity():
    """dg = <dY W_down^T, h> equals <dY, f_e(x)> computed from the forward outputs."""
    X, W_r, W, dY = small_layer(T=20, d=16, E=6, k=3, f=8, seed=41)
    Z = O.router_logits(X, W_r)
    idx = O.topk_select(Z, 3)
    w = O.gate_weights(Z, idx)
    fw = O.moe_forward(X, W, idx, w)
    g = O.moe_backward(X, W_r, W, idx, w, dY)
    j = np.arange(20)[:, None] * 3 + np.arange(3)[None, :]
    direct = (fw["Yexp"][fw["route_pos"][j]] * dY.astype(np.float64)[:, None, :]).sum(-1)
    assert np.allclose(g["dg"], direct, atol=1e-12, rtol=0)


def test_identical_experts_give_zero_router_gradient():
    X, W_r, W, dY = small_layer(T=14, d=16, E=5, k=2, f=8, identical=True, seed=51)
    Z = O.router_logits(X, W_r)
    idx = O.topk_select(Z, 2)
    g = O.moe_backward(X, W_r, W, idx, O.gate_weights(Z, idx), dY)
    assert np.abs(g["dZ"]).max() < 1e-12 and np.abs(g["dW_r"]).max() < 1e-12


def test_sampled_backward_helpers_match_full_backward():
    X, W_r, W, dY = small_layer(T=30, d=16, E=4, k=2, f=8, f_s=8, seed=61)
    Z = O.router_logits(X, W_r)
    idx = O.topk_select(Z, 2)
    w = O.gate_weights(Z, idx)
    g = O.moe_backward(X, W_r, W, idx, w, dY)
    toks = [0, 7, 29]
    dX, dZ, dg = O.token_backward(X, W_r, W, idx, w, dY, toks)
    assert np.allclose(dX, g["dX"][toks], atol=1e-12)
    assert np.allclose(dZ, g["dZ"][toks], atol=1e-12)
    cols = [1, 5]
    for e in (0, 3, "shared"):
        a, b, c = O.expert_weight_grad_columns(X, W, idx, w, dY, e, cols)
        ref = ("dWg_s", "dWu_s", "dWd_s") if e == "shared" else ("dW_gate", "dW_up", "dW_down")
        G = [g[r] if e == "shared" else g[r][e] for r in ref]
        assert np.allclose(a, G[0][:, cols], atol=1e-12)
        assert np.allclose(b, G[1][:, cols], atol=1e-12)
        assert np.allclose(c, G[2][cols, :], atol=1e-12)


def test_router_gradient_from_expert_outputs_matches_backward():
    """router_gradient forms <dY, f_e(x)> from the expert outputs themselves;
    moe_backward takes the §3.4 identity.  Both must give the same dZ and dg
    (chunk sizes below an expert's route count exercise the chunking)."""
    X, W_r, W, dY = small_layer(T=40, d=16, E=5, k=3, f=8, f_s=8, seed=71)
    Z = O.router_logits(X, W_r)
    idx = O.topk_select(Z, 3)
    w = O.gate_weights(Z, idx)
    g = O.moe_backward(X, W_r, W, idx, w, dY)
    for chunk in (3, 4096):
        dZ, dg = O.router_gradient(X, W, idx, w, dY, chunk=chunk)
        assert np.allclose(dZ, g["dZ"], rtol=0, atol=1e-12 * np.abs(g["dZ"]).max())
        assert np.allclose(dg, g["dg"], rtol=0, atol=1e-12 * np.abs(g["dg"]).max())
