"""Plain CPU oracle of one GPU's share of the MoE layer (forward and backward).

TEST INFRASTRUCTURE ONLY.  Only the test-suite, the package smoke check and the
benchmark's CPU-baseline leg may import this module.  The GPU library never
calls it, shares no code with it, and must fail loudly when its HIP build is
missing instead of falling back here.

Everything is written for a reader holding the paper ("Mixture-of-Kittens: MoE
Megakernel for NVL72s"); each function names the passage it follows.  The
arithmetic is float64 numpy; the only fp32 quantity is the router logit tensor
Z, because top-k selection is an integer decision taken on fp32 logits on both
sides (the GPU computes them in fp32).

Readings of points the paper leaves open (numbered as in the design notes):

* score function: softmax over the local logits, renormalised over the selected
  set, i.e. a softmax restricted to the selected experts (§2.1 equation);
* ranking key: fp32 logits, larger first, ties won by the lower expert index;
* slot order: a token's selected experts are emitted in ascending expert id,
  so the route id j = t*k + slot depends only on the selected *set*;
* route flattening: j = t*k + slot (token-major), the "route j" of
  Algorithm 1's input matrix A;
* router bias: added to the logits, so it changes both selection and weights;
* activation: phi = SiLU applied to the gate branch (SwiGLU);
* weight orientation: row vectors, x @ W_gate[e] with W_gate[e] of shape [d, f]
  (the transpose of the paper's column-vector W_gate in R^{I x D});
* combine order: start from the shared expert output (0 without one) and add
  the routed terms w * f_e(x) in ascending expert id.
"""
from __future__ import annotations

import numpy as np

F64 = np.float64


# ---------------------------------------------------------------------------
# Router (§2.1: the router's projection picks a token's top-k routed experts
# and gives each of them a weight)
# ---------------------------------------------------------------------------

def router_logits(X, W_r, bias=None, out_dtype=np.float32):
    """Z = X @ W_r + bias, accumulated in float64 and rounded once to fp32.

    out_dtype=float64 keeps the exact value (used for finite differences,
    where the selection is held fixed and no integer decision is taken).
    """
    Z = np.asarray(X, F64) @ np.asarray(W_r, F64)
    if bias is not None:
        Z = Z + np.asarray(bias, F64)[None, :]
    return Z.astype(out_dtype)


def topk_select(Z, k):
    """The k largest logits of each row, ties to the lower expert index.

    Orders the experts of every token by the key (-z, e) and keeps the first k,
    then emits the kept expert ids in ascending order.  Z must be the fp32
    logit tensor; returns int32 [T, k].
    """
    Z = np.asarray(Z, np.float32)
    T, E = Z.shape
    if not 1 <= k <= E:
        raise ValueError("need 1 <= k <= E")
    experts = np.broadcast_to(np.arange(E), (T, E))
    # np.lexsort sorts by the last key first: primary -z, secondary e.
    order = np.lexsort((experts, -Z.astype(F64)), axis=-1)
    return np.sort(order[:, :k], axis=1).astype(np.int32)


def topk_margin(Z, k):
    """Gap between the k-th and (k+1)-th largest logit of each token (inf if k == E)."""
    Z = np.asarray(Z, F64)
    if k == Z.shape[1]:
        return np.full(Z.shape[0], np.inf)
    s = -np.sort(-Z, axis=1)
    return s[:, k - 1] - s[:, k]


def gate_weights(Z, idx):
    """Router weights s_i / sum_{j in E} s_j of §2.1 with s = softmax(Z).

    Full softmax over all local experts, then renormalised over the selected
    set; returns float64 [T, k] in the slot order of idx.
    """
    z = np.asarray(Z, F64)
    p = np.exp(z - z.max(axis=1, keepdims=True))
    p = p / p.sum(axis=1, keepdims=True)
    s = np.take_along_axis(p, np.asarray(idx, np.int64), axis=1)
    return s / s.sum(axis=1, keepdims=True)


# ---------------------------------------------------------------------------
# Dispatch schedule (§3.1, Algorithm 1 through its sort-key statement)
# ---------------------------------------------------------------------------

def schedule_counts(A, L, c=0):
    """Route counts per (source rank, local expert) and region starts (§3.1).

    A: int [R, N*K] global expert id of route j on source rank r.
    L: local experts per rank; c: current rank (local expert l is global
    c*L + l).  Returns (M [R, L], S [L]): M[r, l] counts the routes of rank r
    to local expert l, and S[l] is the sum of M over all ranks and over the
    experts before l (where l's region of the receive buffer starts).
    """
    A = np.asarray(A, np.int64)
    R = A.shape[0]
    M = np.zeros((R, L), np.int64)
    for r in range(R):
        loc = A[r][(A[r] >= c * L) & (A[r] < (c + 1) * L)] - c * L
        M[r] = np.bincount(loc, minlength=L)
    S = np.concatenate([[0], np.cumsum(M.sum(axis=0))[:-1]]).astype(np.int64)
    return M, S


def schedule_sort_key(A, L, c=0):
    """The pull-based dispatch schedule of §3.1 from its sort-key statement.

    Sorts the local routes by (local expert l, per-source-rank ordinal o,
    source rank r), where o counts earlier routes of rank r to the same expert.
    Returns Phi [P, 2] of (r, j): buffer position p receives route j of rank r.
    """
    A = np.asarray(A, np.int64)
    R, NK = A.shape
    rows = []
    for r in range(R):
        # ordinal = rank of j among equal expert ids of row r (stable order)
        order = np.argsort(A[r], kind="stable")
        ordinal = np.empty(NK, np.int64)
        sorted_ids = A[r][order]
        starts = np.searchsorted(sorted_ids, sorted_ids, side="left")
        ordinal[order] = np.arange(NK) - starts
        for j in range(NK):
            if c * L <= A[r, j] < (c + 1) * L:
                rows.append((A[r, j] - c * L, ordinal[j], r, j))
    rows.sort()
    return np.array([(r, j) for (_, _, r, j) in rows], np.int64).reshape(-1, 2)


def schedule(A, L, c=0):
    """Algorithm 1's outputs (§3.1): (M, S, Phi), as schedule_counts and
    schedule_sort_key define them."""
    M, S = schedule_counts(A, L, c)
    return M, S, schedule_sort_key(A, L, c)


def plan(idx, E):
    """Single-GPU dispatch plan: Algorithm 1 with one source rank (R = 1, c = 0).

    idx: int [T, k] selected experts.  Routes are flattened as j = t*k + slot.
    Returns int32 arrays counts[E], offsets[E+1], perm[T*k] (position -> route
    j) and route_pos[T*k] (route j -> position).  With one rank the position
    formula reduces to p = o, so each expert's region lists its routes in
    ascending j: a stable counting sort by expert.
    """
    idx = np.asarray(idx, np.int64)
    A = idx.reshape(1, -1)
    M, S, Phi = schedule(A, E, 0)
    counts = M[0].astype(np.int32)
    offsets = np.zeros(E + 1, np.int32)
    offsets[:E] = S
    offsets[E] = counts.sum()
    perm = Phi[:, 1].astype(np.int32)
    route_pos = np.full(A.shape[1], -1, np.int32)
    route_pos[perm] = np.arange(perm.size, dtype=np.int32)
    return counts, offsets, perm, route_pos


# ---------------------------------------------------------------------------
# Expert FFNs and the layer (§2.1 equation)
# ---------------------------------------------------------------------------

def silu(x):
    return x / (1.0 + np.exp(-x))


def expert_ffn(x, Wg, Wu, Wd):
    """f_i(x) = W_down (phi(W_gate x) * W_up x) in row-vector form, phi = SiLU."""
    x = np.asarray(x, F64)
    a = x @ np.asarray(Wg, F64)
    b = x @ np.asarray(Wu, F64)
    return (silu(a) * b) @ np.asarray(Wd, F64)


def moe_forward_dense(X, W, idx, w, tokens=None):
    """The §2.1 layer written out per token: shared(x) + sum_i w_i f_i(x).

    W: dict with W_gate [E,d,f], W_up, W_down [E,f,d] and optional Wg_s, Wu_s,
    Wd_s.  idx/w: [T, k] selected experts and their (renormalised) weights.
    tokens: optional token subset.  No permutation, no plan.  float64 [n, d].
    """
    X = np.asarray(X, F64)
    toks = np.arange(X.shape[0]) if tokens is None else np.asarray(tokens)
    Y = np.zeros((toks.size, X.shape[1]), F64)
    for n, t in enumerate(toks):
        x = X[t:t + 1]
        y = np.zeros((1, X.shape[1]), F64)
        if W.get("Wg_s") is not None:
            y = y + expert_ffn(x, W["Wg_s"], W["Wu_s"], W["Wd_s"])
        for s in range(idx.shape[1]):
            e = int(idx[t, s])
            y = y + w[t, s] * expert_ffn(x, W["W_gate"][e], W["W_up"][e], W["W_down"][e])
        Y[n] = y[0]
    return Y


def moe_forward(X, W, idx, w):
    """The same layer evaluated expert by expert through the dispatch plan.

    Mirrors the permuted formulation (gather rows into expert-contiguous
    regions, run each expert's FFN on its region, combine in ascending expert
    order) and returns the intermediates the GPU path keeps:
    dict(Y [T,d], A, B, H [T*k, f] in plan-position order, Yexp [T*k, d],
    Ysh [T,d] or None, plan arrays).
    """
    X = np.asarray(X, F64)
    T, d = X.shape
    E = W["W_gate"].shape[0]
    k = idx.shape[1]
    counts, offsets, perm, route_pos = plan(idx, E)
    tok = perm // k
    f = W["W_gate"].shape[2]
    A = np.zeros((T * k, f), F64)
    B = np.zeros((T * k, f), F64)
    Yexp = np.zeros((T * k, d), F64)
    for e in range(E):
        rows = slice(offsets[e], offsets[e + 1])
        xe = X[tok[rows]]
        A[rows] = xe @ np.asarray(W["W_gate"][e], F64)
        B[rows] = xe @ np.asarray(W["W_up"][e], F64)
        Yexp[rows] = (silu(A[rows]) * B[rows]) @ np.asarray(W["W_down"][e], F64)
    H = silu(A) * B
    Ysh = None
    Y = np.zeros((T, d), F64)
    if W.get("Wg_s") is not None:
        Ysh = expert_ffn(X, W["Wg_s"], W["Wu_s"], W["Wd_s"])
        Y += Ysh
    # combine: a token's selected experts are in ascending order in idx
    for s in range(k):
        Y += w[:, s:s + 1] * Yexp[route_pos[np.arange(T) * k + s]]
    return dict(Y=Y, A=A, B=B, H=H, Yexp=Yexp, Ysh=Ysh, counts=counts,
                offsets=offsets, perm=perm, route_pos=route_pos)


# ---------------------------------------------------------------------------
# Backward.  The gradient of the §2.1 layer by the chain rule; the router
# weight gradient uses the identity of §3.4 ("Router Weight Gradient
# Computation"): <dY, f_e(x)> = <dY W_down^T, h> with h the gated activation.
# ---------------------------------------------------------------------------

def _dsilu(a):
    s = 1.0 / (1.0 + np.exp(-a))
    return s * (1.0 + a * (1.0 - s))


def softmax_restricted_backward(w, dg):
    """dL/dz_u for u in the selected set, given w = softmax restricted to it.

    dw_s/dz_u = w_s (delta_su - w_u), so dz_u = w_u (dg_u - sum_s w_s dg_s).
    Unselected logits get exactly zero (the renormalised weights do not
    depend on them).  w, dg: [T, k] -> [T, k].
    """
    return w * (dg - (w * dg).sum(axis=1, keepdims=True))


def moe_backward(X, W_r, W, idx, w, dY):
    """All gradients of the layer for upstream gradient dY, selection held fixed.

    Returns dict dX [T,d], dW_gate/dW_up [E,d,f], dW_down [E,f,d], dW_r [d,E],
    dZ [T,E] (gradient wrt the logits), dg [T,k] (<dY, f_e(x)>), and the
    shared-expert gradients dWg_s, dWu_s, dWd_s (None without one).
    """
    X = np.asarray(X, F64)
    dY = np.asarray(dY, F64)
    T, d = X.shape
    E, _, f = W["W_gate"].shape
    k = idx.shape[1]
    dX = np.zeros((T, d), F64)
    dWg = np.zeros((E, d, f), F64)
    dWu = np.zeros((E, d, f), F64)
    dWd = np.zeros((E, f, d), F64)
    dg = np.zeros((T, k), F64)
    for e in range(E):
        ts, ss = np.nonzero(np.asarray(idx) == e)
        if ts.size == 0:
            continue
        Wg = np.asarray(W["W_gate"][e], F64)
        Wu = np.asarray(W["W_up"][e], F64)
        Wd = np.asarray(W["W_down"][e], F64)
        x = X[ts]
        a = x @ Wg
        b = x @ Wu
        h = silu(a) * b
        dy = dY[ts]
        we = np.asarray(w, F64)[ts, ss][:, None]
        dhp = dy @ Wd.T                        # gradient wrt h of the unweighted output
        dg[ts, ss] = (dhp * h).sum(axis=1)     # = <dY, f_e(x)>, the §3.4 identity
        dh = we * dhp
        dA = dh * b * _dsilu(a)
        dB = dh * silu(a)
        dWg[e] = x.T @ dA
        dWu[e] = x.T @ dB
        dWd[e] = (we * h).T @ dy
        np.add.at(dX, ts, dA @ Wg.T + dB @ Wu.T)
    dz_sel = softmax_restricted_backward(np.asarray(w, F64), dg)
    dZ = np.zeros((T, W_r.shape[1]), F64)
    np.put_along_axis(dZ, np.asarray(idx, np.int64), dz_sel, axis=1)
    W_r64 = np.asarray(W_r, F64)
    dW_r = X.T @ dZ
    dX += dZ @ W_r64.T
    out = dict(dX=dX, dW_gate=dWg, dW_up=dWu, dW_down=dWd, dW_r=dW_r, dZ=dZ,
               dg=dg, dWg_s=None, dWu_s=None, dWd_s=None)
    if W.get("Wg_s") is not None:
        Wg = np.asarray(W["Wg_s"], F64)
        Wu = np.asarray(W["Wu_s"], F64)
        Wd = np.asarray(W["Wd_s"], F64)
        a = X @ Wg
        b = X @ Wu
        h = silu(a) * b
        dh = dY @ Wd.T
        dA = dh * b * _dsilu(a)
        dB = dh * silu(a)
        out["dWg_s"] = X.T @ dA
        out["dWu_s"] = X.T @ dB
        out["dWd_s"] = h.T @ dY
        dX += dA @ Wg.T + dB @ Wu.T
    return out


# ---------------------------------------------------------------------------
# Sampled evaluation for full-size workloads, where the whole backward is far
# too slow on a CPU.  Each sampled output is computed from its own definition.
# ---------------------------------------------------------------------------

def token_backward(X, W_r, W, idx, w, dY, tokens):
    """dX rows and dZ rows of the given tokens (per token, no plan).

    Each token's dX needs only its own routes: its experts' FFN backward, the
    restricted-softmax backward of its own logits, and the router term.
    Returns (dX [n, d], dZ [n, E], dg [n, k]) in float64.
    """
    X = np.asarray(X, F64)
    E = W["W_gate"].shape[0]
    k = idx.shape[1]
    W_r64 = np.asarray(W_r, F64)
    dXs = np.zeros((len(tokens), X.shape[1]), F64)
    dZs = np.zeros((len(tokens), E), F64)
    dgs = np.zeros((len(tokens), k), F64)
    for n, t in enumerate(tokens):
        x = X[t:t + 1]
        dy = np.asarray(dY[t:t + 1], F64)
        dx = np.zeros_like(x)
        for s in range(k):
            e = int(idx[t, s])
            Wg = np.asarray(W["W_gate"][e], F64)
            Wu = np.asarray(W["W_up"][e], F64)
            Wd = np.asarray(W["W_down"][e], F64)
            a = x @ Wg
            b = x @ Wu
            h = silu(a) * b
            dhp = dy @ Wd.T
            dgs[n, s] = float((dhp * h).sum())
            dh = w[t, s] * dhp
            dx += (dh * b * _dsilu(a)) @ Wg.T + (dh * silu(a)) @ Wu.T
        dz = softmax_restricted_backward(np.asarray(w[t:t + 1], F64), dgs[n:n + 1])[0]
        dZs[n, np.asarray(idx[t], np.int64)] = dz
        dx += dZs[n:n + 1] @ W_r64.T
        if W.get("Wg_s") is not None:
            Wg = np.asarray(W["Wg_s"], F64)
            Wu = np.asarray(W["Wu_s"], F64)
            Wd = np.asarray(W["Wd_s"], F64)
            a = x @ Wg
            b = x @ Wu
            dh = dy @ Wd.T
            dx += (dh * b * _dsilu(a)) @ Wg.T + (dh * silu(a)) @ Wu.T
        dXs[n] = dx[0]
    return dXs, dZs, dgs


def router_gradient(X, W, idx, w, dY, chunk=4096):
    """dZ [T, E] and dg [T, k] of every token, from the definition of the
    router weights' role in the §2.1 layer: Y depends on w[t, e] only through
    the term w[t, e] f_e(x_t), so dL/dw[t, e] = <dY[t], f_e(x_t)>; dZ then
    follows from the restricted-softmax Jacobian.  Unlike moe_backward (which
    takes the §3.4 identity <dY W_down^T, h>), this forms each expert output
    f_e(x) in full.  Tokens go through each expert in chunks to bound memory.
    """
    X = np.asarray(X, F64)
    T = X.shape[0]
    E = W["W_gate"].shape[0]
    k = idx.shape[1]
    dg = np.zeros((T, k), F64)
    for e in range(E):
        ts, ss = np.nonzero(np.asarray(idx) == e)
        if ts.size == 0:
            continue
        Wg = np.asarray(W["W_gate"][e], F64)
        Wu = np.asarray(W["W_up"][e], F64)
        Wd = np.asarray(W["W_down"][e], F64)
        for c0 in range(0, ts.size, chunk):
            t, s = ts[c0:c0 + chunk], ss[c0:c0 + chunk]
            fe = expert_ffn(X[t], Wg, Wu, Wd)
            dg[t, s] = (np.asarray(dY[t], F64) * fe).sum(axis=1)
    dz_sel = softmax_restricted_backward(np.asarray(w, F64), dg)
    dZ = np.zeros((T, E), F64)
    np.put_along_axis(dZ, np.asarray(idx, np.int64), dz_sel, axis=1)
    return dZ, dg


def expert_weight_grad_columns(X, W, idx, w, dY, e, cols):
    """Columns `cols` of dW_gate[e], dW_up[e] and rows `cols` of dW_down[e].

    Each needs only the matching intermediate columns over every route of
    expert e.  Returns (dWg[:, cols], dWu[:, cols], dWd[cols, :]) in float64.
    For the shared expert pass e = "shared" (weight 1 for every token).
    """
    X = np.asarray(X, F64)
    cols = np.asarray(cols)
    if e == "shared":
        ts = np.arange(X.shape[0])
        we = np.ones((ts.size, 1), F64)
        Wg, Wu, Wd = W["Wg_s"], W["Wu_s"], W["Wd_s"]
    else:
        ts, ss = np.nonzero(np.asarray(idx) == e)
        we = np.asarray(w, F64)[ts, ss][:, None]
        Wg, Wu, Wd = W["W_gate"][e], W["W_up"][e], W["W_down"][e]
    x = X[ts]
    dy = np.asarray(dY, F64)[ts]
    a = x @ np.asarray(Wg, F64)[:, cols]
    b = x @ np.asarray(Wu, F64)[:, cols]
    dhp = dy @ np.asarray(Wd, F64)[cols, :].T
    dh = we * dhp
    dA = dh * b * _dsilu(a)
    dB = dh * silu(a)
    h = silu(a) * b
    return x.T @ dA, x.T @ dB, (we * h).T @ dy
