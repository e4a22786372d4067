"""moe_plan_noalloc (the plan with library-held scratch, for callers that
cannot allocate) against moe_plan with a caller workspace and against the
oracle's plan: two calls in a row, the second on a smaller input, then an
input with an out-of-range expert id."""
import numpy as np
import pytest
import torch

from oracle import moe_oracle as O
from paper_2609_36070_amd import binding as B
from tests.parity import say, to_np

pytestmark = pytest.mark.gpu


def _idx(T, E, k, seed):
    Z = np.random.default_rng(seed).standard_normal((T, E)).astype(np.float32)
    Z[:, 0] += 1.0                          # a hot expert
    Z[:, E - 1] -= 4.0                      # an expert that is almost always empty
    return O.topk_select(Z, k).astype(np.int32)


def _bufs(E, R, dev):
    i32 = torch.int32
    return (torch.full((E,), -9, dtype=i32, device=dev), torch.full((E + 1,), -9, dtype=i32, device=dev),
            torch.full((max(R, 1),), -9, dtype=i32, device=dev),
            torch.full((max(R, 1),), -9, dtype=i32, device=dev))


def _run_both(idx, E):
    T, k = idx.shape
    R = T * k
    dev = torch.device("cuda")
    sh = B.make_shape(T, 256, E, k, 256, 0)
    idx_d = torch.from_numpy(idx).to(dev)
    ref = _bufs(E, R, dev)
    ws = torch.zeros(B.moe_workspace_bytes(sh, False), dtype=torch.uint8, device=dev)
    B.moe_plan(sh, idx_d, B.plan_bufs(*ref), ws)
    got = _bufs(E, R, dev)
    err = torch.full((4,), -9, dtype=torch.int32, device=dev)
    B.moe_plan_noalloc(sh, idx_d, B.plan_bufs(*got), err)
    torch.cuda.synchronize()
    off, _ = B.moe_workspace_region(sh, False, B.WS_ERROR)
    ref_err = int(ws[off:off + 4].view(torch.int32).item())
    return [to_np(t) for t in ref], [to_np(t) for t in got], ref_err, int(err[0].item())


def _check_equal(idx, E, expect_err):
    ref, got, ref_err, err = _run_both(idx, E)
    R = idx.size
    placed = int(ref[1][E])
    assert err == ref_err == expect_err
    assert np.array_equal(got[0], ref[0]), "counts"
    assert np.array_equal(got[1], ref[1]), "offsets"
    assert np.array_equal(got[2][:placed], ref[2][:placed]), "perm"
    assert np.array_equal(got[3][:R], ref[3][:R]), "route_pos"
    return got


def test_plan_noalloc_matches_plan_on_two_calls_then_a_smaller_one():
    E, k = 64, 6
    for T, seed in ((5000, 1), (700, 2)):
        idx = _idx(T, E, k, seed)
        say(f"[gpu] moe_plan_noalloc T={T} E={E} k={k}")
        got = _check_equal(idx, E, 0)
        counts, offsets, perm, route_pos = O.plan(idx, E)
        assert np.array_equal(got[0], counts) and np.array_equal(got[1], offsets)
        assert np.array_equal(got[2][:T * k], perm) and np.array_equal(got[3][:T * k], route_pos)


def test_plan_noalloc_reports_bad_ids_like_plan():
    E, k = 16, 2
    idx = _idx(300, E, k, 3)
    idx[17, 1] = E + 3                     # out of range: left unplaced, error word 1
    say(f"[gpu] moe_plan_noalloc with an invalid id, T=300 E={E} k={k}")
    got = _check_equal(idx, E, 1)
    assert got[3][17 * k + 1] == -1
    # a valid call afterwards clears the word again
    _check_equal(_idx(300, E, k, 4), E, 0)


def test_plan_noalloc_rejects_too_large_shapes_before_launching():
    sh = B.make_shape(300000, 256, 256, 8, 256, 0)      # needs ~4.8 MB of plan scratch
    assert B.moe_plan_noalloc(sh, None, B.plan_bufs(None, None, None, None), None,
                              raise_on_error=False) == B.MOE_EINVAL
    dev = torch.device("cuda")
    t = torch.zeros(16, dtype=torch.int32, device=dev)
    pb = B.plan_bufs(t, t, t, t)
    assert B.moe_plan_noalloc(sh, t, pb, t, raise_on_error=False) == B.MOE_EUNSUPPORTED
