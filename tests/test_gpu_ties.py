"""GPU router selection on exact ties (the §2.1 router with the tie reading
used throughout: among equal logits the lower expert id wins, and the kept
ids are listed in ascending order).

Every logit here is an exact integer in fp32 whatever order the summation
takes: X and W_r hold small integers (exact in bf16), the bias holds
integers, and no partial sum leaves the range fp32 represents exactly.  So
the GPU's logits must equal the oracle's bit for bit, and the selection,
weights and plan are compared bit-exactly against the oracle on every token,
with no margin exemption.
"""
import os

import numpy as np
import pytest
import torch

from oracle import moe_oracle as O
from paper_2609_36070_amd import binding as B
from tests.parity import say, to_np

pytestmark = pytest.mark.gpu

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def read_golden_topk():
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


def route_and_plan(X, W_r, bias, k):
    """moe_route + moe_plan through the C ABI on host arrays (X [T, d] and W_r
    [d, E] small integers, bias [E] integers or None)."""
    T, d = X.shape
    E = W_r.shape[1]
    dev = torch.device("cuda")
    sh = B.make_shape(T, d, E, k, 256, 0)
    ws = torch.zeros(B.moe_workspace_bytes(sh, False), dtype=torch.uint8, device=dev)
    Xd = torch.from_numpy(X.astype(np.float32)).to(torch.bfloat16).to(dev)
    Wd = torch.from_numpy(W_r.astype(np.float32)).to(torch.bfloat16).to(dev)
    # the bf16 copies must hold the integers exactly
    assert np.array_equal(Xd.float().cpu().numpy(), X) and np.array_equal(Wd.float().cpu().numpy(), W_r)
    bd = None if bias is None else torch.from_numpy(np.asarray(bias, np.float32)).to(dev)
    logits = torch.empty((T, E), dtype=torch.float32, device=dev)
    idx = torch.empty((T, k), dtype=torch.int32, device=dev)
    wts = torch.empty((T, k), dtype=torch.float32, device=dev)
    R = T * k
    counts = torch.empty((E,), dtype=torch.int32, device=dev)
    offsets = torch.empty((E + 1,), dtype=torch.int32, device=dev)
    perm = torch.empty((max(R, 1),), dtype=torch.int32, device=dev)
    route_pos = torch.empty((max(R, 1),), dtype=torch.int32, device=dev)
    B.moe_route(sh, Xd, Wd, bd, logits, idx, wts, ws)
    B.moe_plan(sh, idx, B.plan_bufs(counts, offsets, perm, route_pos), ws)
    torch.cuda.synchronize()
    off, _ = B.moe_workspace_region(sh, False, B.WS_ERROR)
    err = int(ws[off:off + 4].view(torch.int32).item())
    return (to_np(logits), to_np(idx), to_np(wts),
            (to_np(counts), to_np(offsets), to_np(perm)[:R], to_np(route_pos)[:R]), err)


def check_exact(X, W_r, bias, k):
    Zg, idx, wts, plan, err = route_and_plan(X, W_r, bias, k)
    Zo = O.router_logits(X, W_r, None if bias is None else np.asarray(bias, np.float32))
    assert np.array_equal(Zg.astype(np.float64), Zo), "integer logits must be exact"
    idx_o = O.topk_select(Zo, k)
    assert np.array_equal(idx, idx_o), "selection"
    # the weights are an fp32 softmax over the k kept logits: one exp each
    # (within 2 ulp), k - 1 additions, a reciprocal and a product, so their
    # relative error is within (3.5 + (k - 1) / 2) units of 2^-23
    w_o = O.gate_weights(Zo, idx_o)
    werr = float((np.abs(wts - w_o) / w_o).max()) if wts.size else 0.0
    assert werr <= (3.5 + (k - 1) / 2) * 2.0 ** -23, f"weights off by {werr} (relative)"
    for got, ref, name in zip(plan, O.plan(idx_o, W_r.shape[1]),
                              ("counts", "offsets", "perm", "route_pos")):
        assert np.array_equal(got, ref), name
    assert err == 0
    return Zo, idx, wts


@pytest.mark.parametrize("case", range(len(read_golden_topk())))
def test_golden_ties_on_gpu(case):
    """Each hand-written row of the tie fixture as a one-token layer:
    X = one-hot, W_r's row = the fixture's logits, the fixture's bias."""
    k, logits, bias, expected = read_golden_topk()[case]
    E, d = len(logits), 256
    X = np.zeros((1, d), np.float32)
    X[0, 5] = 1.0
    W_r = np.zeros((d, E), np.float32)
    W_r[5] = logits
    say(f"[gpu] golden tie row {case}: k={k} logits={logits} bias={bias}")
    _, idx, wts = check_exact(X, W_r, np.array(bias, np.float32), k)
    assert list(idx[0]) == expected
    Zs = np.array(logits, np.float64) + np.array(bias, np.float64)
    if np.all(Zs[expected] == Zs[expected[0]]) and k in (1, 2, 4, 8):
        assert np.all(wts[0] == np.float32(1.0 / k)), "equal logits give exactly 1/k"


def test_all_zero_tokens_pick_the_first_k():
    """Zero X rows and no bias: every logit is 0, so every token must pick
    experts 0 .. k-1 with weight exactly 1/k, and the plan fills each of those
    experts with all tokens in order."""
    T, d, E, k = 300, 512, 64, 8
    X = np.zeros((T, d), np.float32)
    W_r = np.random.default_rng(0).integers(-3, 4, size=(d, E)).astype(np.float32)
    say(f"[gpu] all-zero tokens T={T} E={E} k={k}")
    _, idx, wts = check_exact(X, W_r, None, k)
    assert np.all(idx == np.arange(k)[None, :])
    assert np.all(wts == np.float32(1.0 / k))


def planted_ties(T, d, E, k, seed):
    """Sparse 0/1 X and W_r: logits are small non-negative integers, so most
    tokens have several experts tied at the k-th largest value."""
    rng = np.random.default_rng(seed)
    X = (rng.random((T, d)) < 0.02).astype(np.float32)
    W_r = (rng.random((d, E)) < 0.05).astype(np.float32)
    bias = rng.integers(0, 2, size=E).astype(np.float32)
    return X, W_r, bias


@pytest.mark.parametrize("T,d,E,k", [(2048, 512, 128, 8), (1024, 768, 256, 16), (777, 256, 32, 8)])
def test_planted_ties_at_the_kth_slot(T, d, E, k):
    X, W_r, bias = planted_ties(T, d, E, k, seed=E + k)
    say(f"[gpu] planted ties T={T} d={d} E={E} k={k}")
    Zo, idx, _ = check_exact(X, W_r, bias, k)
    srt = -np.sort(-Zo, axis=1)
    tied = int((srt[:, k - 1] == srt[:, k]).sum())
    say(f"  {tied} of {T} tokens have a tie across the k-th slot")
    assert tied >= T // 2, "the fixture must actually tie at the k-th slot"


@pytest.mark.parametrize("T,d,E,k", [(16461, 256, 32, 8), (8197, 256, 128, 8), (16400, 256, 64, 6)])
def test_planted_ties_large_batches(T, d, E, k):
    """Batches large enough that each wave of the router serves two or four
    16-token tiles per W_r fragment, with a ragged last block."""
    X, W_r, bias = planted_ties(T, d, E, k, seed=T)
    say(f"[gpu] planted ties, large batch T={T} d={d} E={E} k={k}")
    Zo, _, _ = check_exact(X, W_r, bias, k)
    srt = -np.sort(-Zo, axis=1)
    assert int((srt[:, k - 1] == srt[:, k]).sum()) >= T // 2


def test_every_expert_kept_large_batch():
    """k == E on a large ragged batch: every token keeps every expert, in id
    order, with the softmax weights of all its logits."""
    T, d, E = 16390, 256, 8
    X, W_r, bias = planted_ties(T, d, E, E, seed=5)
    say(f"[gpu] k == E, large batch T={T} E={E}")
    _, idx, _ = check_exact(X, W_r, bias, E)
    assert np.all(idx == np.arange(E)[None, :])


@pytest.mark.parametrize("T,d,E,k", [(32800, 256, 128, 8), (33000, 256, 256, 16), (300, 512, 128, 8),
                                     (5000, 1024, 200, 10)])
def test_split_router_slice_counts(T, d, E, k):
    """The router for 128 or more experts at one slice of d (256 or more
    128-token tiles: the tile kernel selects itself), at eight slices (few
    tokens), and with a padded expert count and k = 10; exact ties at the
    k-th slot throughout."""
    X, W_r, bias = planted_ties(T, d, E, k, seed=T + E)
    say(f"[gpu] split router T={T} d={d} E={E} k={k}")
    Zo, _, _ = check_exact(X, W_r, bias, k)
    srt = -np.sort(-Zo, axis=1)
    assert int((srt[:, k - 1] == srt[:, k]).sum()) >= T // 2


@pytest.mark.parametrize("T,d,E,k", [(8192, 2048, 128, 8), (3000, 1024, 256, 16)])
def test_split_router_repeats_bitwise(T, d, E, k):
    """Random fp32-valued logits through the router for 128 or more experts
    (partial logits of several d slices added in a fixed order): three calls
    give the same logits, ids and weights bit for bit."""
    rng = np.random.default_rng(T + d)
    X = rng.standard_normal((T, d), dtype=np.float32)
    W_r = rng.standard_normal((d, E), dtype=np.float32) / np.float32(np.sqrt(d))
    sh = B.make_shape(T, d, E, k, 256, 0)
    dev = torch.device("cuda")
    ws = torch.empty(B.moe_workspace_bytes(sh, False), dtype=torch.uint8, device=dev)
    Xd = torch.from_numpy(X).to(torch.bfloat16).to(dev)
    Wd = torch.from_numpy(W_r).to(torch.bfloat16).to(dev)
    bias = torch.from_numpy(rng.standard_normal(E, dtype=np.float32) * np.float32(0.5)).to(dev)
    say(f"[gpu] split router repeats T={T} d={d} E={E} k={k}")
    runs = []
    for _ in range(3):
        logits = torch.empty((T, E), dtype=torch.float32, device=dev)
        idx = torch.empty((T, k), dtype=torch.int32, device=dev)
        wts = torch.empty((T, k), dtype=torch.float32, device=dev)
        ws.fill_(0x5A)   # stale partials from an earlier call must not matter
        B.moe_route(sh, Xd, Wd, bias, logits, idx, wts, ws)
        torch.cuda.synchronize()
        runs.append((logits, idx, wts))
    for r in runs[1:]:
        for a, b in zip(runs[0], r):
            assert torch.equal(a, b)
    # and the selection is the oracle's on the GPU's own logits
    Zg = to_np(runs[0][0])
    assert np.array_equal(O.topk_select(Zg, k), to_np(runs[0][1]))
