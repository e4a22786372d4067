"""Host-side checks of the C ABI (CPU only: no kernel is ever launched here).

The library must load, export every function include/moe.h declares, size
its workspace from the shape alone, and reject bad arguments before touching
the GPU.
"""
import ctypes
import os
import re

import pytest

from paper_2609_36070_amd import binding as B
from paper_2609_36070_amd.workloads import WORKLOADS

HEADER = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))),
                      "include", "moe.h")

FAKE = 0x10000          # 16-byte aligned non-null address; never dereferenced on these paths
MISALIGNED = 0x10008


def declared_functions():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"\b(moe_[a-z_]+)\s*\(", text)))


def test_library_exports_every_declared_function():
    L = B.lib()
    names = declared_functions()
    assert names, "no declarations parsed"
    for n in names:
        assert hasattr(L, n), n
    assert set(names) == set(B.EXPORTS)
    assert "gfx950" in B.version()


def test_library_resolves_every_symbol():
    """Every symbol the library references must be defined (a kernel whose
    host launch stub went missing would otherwise fail only at its launch)."""
    ctypes.CDLL(B.LIB_PATH, mode=os.RTLD_NOW | os.RTLD_LOCAL)


def test_status_strings():
    for s in range(5):
        assert B.status_string(s)
    assert B.status_string(99) == "unknown status"


@pytest.mark.parametrize("name", sorted(WORKLOADS))
def test_workspace_sizes(name):
    w = WORKLOADS[name]
    sh = B.make_shape(w.T, w.d, w.E, w.k, w.f, w.f_s)
    fwd = B.moe_workspace_bytes(sh, False)
    bwd = B.moe_workspace_bytes(sh, True)
    R = w.T * w.k
    assert fwd >= R * w.f * 2 * 3 + R * w.d * 2           # A, B, H, Yexp at least
    assert bwd >= fwd + R * w.d * 2                       # plus dXperm
    for which in list(range(B.WS_DXPERM + 1)) + [B.WS_HW]:
        off, nb = B.moe_workspace_region(sh, True, which)
        assert off % 256 == 0 and off + nb <= bwd
    off, nb = B.moe_workspace_region(sh, True, B.WS_HW)
    assert nb == R * w.f * 2 and off >= fwd                  # backward only
    with pytest.raises(B.MoeError):
        B.moe_workspace_region(sh, False, B.WS_HW)


def test_workspace_zero_for_bad_shapes():
    assert B.moe_workspace_bytes(B.make_shape(16, 100, 8, 2, 256), False) == 0   # d % 256
    assert B.moe_workspace_bytes(B.make_shape(16, 256, 4, 5, 256), False) == 0   # k > E
    assert B.moe_workspace_bytes(B.make_shape(16, 256, 300, 2, 256), False) == 0  # E > 256


def _route(shape, **kw):
    args = dict(X=FAKE, W_r=FAKE, bias=None, logits=FAKE, topk_idx=FAKE, topk_w=FAKE, ws=FAKE,
                ws_bytes=1 << 40)
    args.update(kw)
    return B.lib().moe_route(ctypes.byref(shape), args["X"], args["W_r"], args["bias"],
                             args["logits"], args["topk_idx"], args["topk_w"], args["ws"],
                             args["ws_bytes"], None)


def test_route_validation():
    ok = B.make_shape(64, 256, 8, 2, 256)
    assert _route(ok, X=None) == B.MOE_EINVAL
    assert _route(ok, logits=MISALIGNED) == B.MOE_EINVAL
    assert _route(ok, bias=MISALIGNED) == B.MOE_EINVAL
    assert _route(ok, ws=None) == B.MOE_EINVAL
    assert _route(ok, ws_bytes=16) == B.MOE_ENOSPACE
    assert _route(B.make_shape(64, 256, 4, 5, 256)) == B.MOE_EINVAL          # k > E
    assert _route(B.make_shape(64, 0, 8, 2, 256)) == B.MOE_EINVAL            # d <= 0
    assert _route(B.make_shape(-1, 256, 8, 2, 256)) == B.MOE_EINVAL          # T < 0
    assert _route(B.make_shape(64, 192, 8, 2, 256)) == B.MOE_EUNSUPPORTED    # d % 256
    assert _route(B.make_shape(64, 256, 32, 17, 256)) == B.MOE_EUNSUPPORTED  # k > 16
    assert _route(B.make_shape(64, 256, 8, 2, 320)) == B.MOE_EUNSUPPORTED    # f % 256
    assert _route(B.make_shape(1 << 28, 256, 64, 16, 256)) == B.MOE_EUNSUPPORTED  # T*k >= 2^31
    assert B.lib().moe_route(None, FAKE, FAKE, None, FAKE, FAKE, FAKE, FAKE, 1 << 40, None) \
        == B.MOE_EINVAL


def test_plan_forward_backward_validation():
    L = B.lib()
    sh = B.make_shape(64, 256, 8, 2, 256)
    plan = B.MoePlanBufs(FAKE, FAKE, FAKE, FAKE)
    bad_plan = B.MoePlanBufs(FAKE, None, FAKE, FAKE)
    big = 1 << 40
    assert L.moe_plan(ctypes.byref(sh), FAKE, ctypes.byref(bad_plan), FAKE, big, None) == B.MOE_EINVAL
    assert L.moe_plan(ctypes.byref(sh), FAKE, ctypes.byref(plan), FAKE, 8, None) == B.MOE_ENOSPACE
    assert L.moe_plan(ctypes.byref(sh), None, ctypes.byref(plan), FAKE, big, None) == B.MOE_EINVAL
    assert L.moe_dispatch(ctypes.byref(sh), FAKE, ctypes.byref(plan), None, None) == B.MOE_EINVAL

    w = B.MoeWeights(FAKE, FAKE, FAKE, None, None, None)
    w_shared_extra = B.MoeWeights(FAKE, FAKE, FAKE, FAKE, FAKE, FAKE)
    assert L.moe_forward(ctypes.byref(sh), FAKE, ctypes.byref(w_shared_extra), FAKE, FAKE,
                         ctypes.byref(plan), FAKE, 1, FAKE, big, None, None) == B.MOE_EINVAL
    sh_s = B.make_shape(64, 256, 8, 2, 256, 256)
    assert L.moe_forward(ctypes.byref(sh_s), FAKE, ctypes.byref(w), FAKE, FAKE,
                         ctypes.byref(plan), FAKE, 1, FAKE, big, None, None) == B.MOE_EINVAL
    assert L.moe_forward(ctypes.byref(sh), FAKE, ctypes.byref(w), FAKE, FAKE,
                         ctypes.byref(plan), FAKE, 1, FAKE, 64, None, None) == B.MOE_ENOSPACE
    fwd_bytes = B.moe_workspace_bytes(sh, False)
    g = B.MoeGrads(FAKE, FAKE, FAKE, FAKE, None, None, None, None)
    # backward needs the larger workspace
    assert L.moe_backward(ctypes.byref(sh), FAKE, FAKE, FAKE, ctypes.byref(w), FAKE, FAKE,
                          ctypes.byref(plan), FAKE, ctypes.byref(g), FAKE, fwd_bytes,
                          None, None) == B.MOE_ENOSPACE
    g_bad = B.MoeGrads(FAKE, FAKE, None, FAKE, None, None, None, None)
    assert L.moe_backward(ctypes.byref(sh), FAKE, FAKE, FAKE, ctypes.byref(w), FAKE, FAKE,
                          ctypes.byref(plan), FAKE, ctypes.byref(g_bad), FAKE, big,
                          None, None) == B.MOE_EINVAL
    assert L.moe_backward(ctypes.byref(sh), FAKE, FAKE, FAKE, ctypes.byref(w), FAKE, FAKE,
                          ctypes.byref(plan), MISALIGNED, ctypes.byref(g), FAKE, big,
                          None, None) == B.MOE_EINVAL


@pytest.mark.parametrize("name", sorted(WORKLOADS))
def test_ring_workspace_sizes(name):
    """The ring workspace shrinks with the ring and never exceeds the one-pass
    one; a ring holding every route needs exactly the one-pass activations."""
    w = WORKLOADS[name]
    sh = B.make_shape(w.T, w.d, w.E, w.k, w.f, w.f_s)
    R = w.T * w.k
    for bwd in (False, True):
        full = B.moe_workspace_bytes(sh, bwd)
        sizes = [B.moe_ring_workspace_bytes(sh, c, bwd) for c in (256, max(R // 2, 1), R, 4 * R)]
        assert all(0 < b for b in sizes)
        assert sizes[0] <= sizes[1] <= sizes[2] == sizes[3]
        # the ring adds an fp32 per-token accumulator and two clipped-offset arrays
        extra = w.T * w.d * 4 + 8 * (w.E + 1) + 2 * 256
        assert sizes[2] <= full + extra
        per_row = (3 * w.f + w.d + (3 * w.f + w.d if bwd else 0)) * 2
        assert sizes[2] - sizes[1] >= (R - R // 2) * per_row - 16 * 256


def test_ring_validation():
    L = B.lib()
    sh = B.make_shape(64, 256, 8, 2, 256)
    plan = B.MoePlanBufs(FAKE, FAKE, FAKE, FAKE)
    w = B.MoeWeights(FAKE, FAKE, FAKE, None, None, None)
    g = B.MoeGrads(FAKE, FAKE, FAKE, FAKE, None, None, None, None)
    big = 1 << 40
    assert B.moe_ring_workspace_bytes(sh, 0, True) == 0
    assert B.moe_ring_workspace_bytes(sh, 1 << 31, True) == 0
    assert B.moe_ring_workspace_bytes(B.make_shape(16, 100, 8, 2, 256), 256, False) == 0

    def fwd(ring, ws_bytes=big, weights=w, Y=FAKE):
        return L.moe_forward_ring(ctypes.byref(sh), FAKE, ctypes.byref(weights), FAKE, FAKE,
                                  ctypes.byref(plan), Y, ring, 1, FAKE, ws_bytes, None)

    def bwd(ring, ws_bytes=big, grads=g):
        return L.moe_backward_ring(ctypes.byref(sh), FAKE, FAKE, FAKE, ctypes.byref(w), FAKE,
                                   FAKE, ctypes.byref(plan), FAKE, ctypes.byref(grads), ring, FAKE,
                                   ws_bytes, None)

    assert fwd(0) == B.MOE_EINVAL and bwd(-5) == B.MOE_EINVAL
    assert fwd(1 << 31) == B.MOE_EUNSUPPORTED
    assert fwd(64, Y=MISALIGNED) == B.MOE_EINVAL
    assert fwd(64, weights=B.MoeWeights(FAKE, FAKE, FAKE, FAKE, FAKE, FAKE)) == B.MOE_EINVAL
    need_f = B.moe_ring_workspace_bytes(sh, 64, False)
    need_b = B.moe_ring_workspace_bytes(sh, 64, True)
    assert fwd(64, ws_bytes=need_f - 1) == B.MOE_ENOSPACE
    assert bwd(64, ws_bytes=need_f) == B.MOE_ENOSPACE       # backward needs the larger one
    assert bwd(64, ws_bytes=need_b - 1) == B.MOE_ENOSPACE
    assert bwd(64, grads=B.MoeGrads(FAKE, FAKE, None, FAKE, None, None, None, None)) == B.MOE_EINVAL


def test_fused_forward_validation():
    L = B.lib()
    sh = B.make_shape(64, 256, 8, 2, 256)
    plan = B.MoePlanBufs(FAKE, FAKE, FAKE, FAKE)
    w = B.MoeWeights(FAKE, FAKE, FAKE, None, None, None)
    big = 1 << 40

    def fwd(shape=sh, weights=w, Y=FAKE, ws_bytes=big, X=FAKE):
        return L.moe_forward_fused(ctypes.byref(shape), X, ctypes.byref(weights), FAKE, FAKE,
                                   ctypes.byref(plan), Y, 1, FAKE, ws_bytes, None)

    assert fwd(X=None) == B.MOE_EINVAL
    assert fwd(Y=MISALIGNED) == B.MOE_EINVAL
    assert fwd(weights=B.MoeWeights(FAKE, FAKE, FAKE, FAKE, FAKE, FAKE)) == B.MOE_EINVAL
    assert fwd(ws_bytes=B.moe_workspace_bytes(sh, False) - 1) == B.MOE_ENOSPACE
    assert fwd(shape=B.make_shape(64, 192, 8, 2, 256)) == B.MOE_EUNSUPPORTED


def test_schedule_workspace_and_validation():
    L = B.lib()
    # error word + per-(rank, chunk) flags + per-(rank, chunk, expert) counts
    ws = B.moe_schedule_workspace_bytes(64, 16384, 4)
    assert ws >= 4 + 64 * 4 + 64 * 4 * 4
    assert B.moe_schedule_workspace_bytes(64, 2 * 16384, 4) > ws    # grows with the row length
    assert B.moe_schedule_workspace_bytes(4, 0, 32) > 0          # no routes is valid
    assert B.moe_schedule_workspace_bytes(0, 16, 4) == 0         # R < 1
    assert B.moe_schedule_workspace_bytes(2048, 16, 4) == 0      # R > 1024
    assert B.moe_schedule_workspace_bytes(4, 16, 300) == 0       # L > 256
    assert B.moe_schedule_workspace_bytes(1024, 1 << 21, 4) == 0  # R*NK >= 2^31
    assert B.moe_schedule_workspace_bytes(1024, 16, 8) > 0       # count table of 8192
    assert B.moe_schedule_workspace_bytes(1024, 16, 9) == 0      # count table above 8192
    assert B.moe_schedule_workspace_bytes(1021, 16, 8) > 0       # R rounds up to 1024

    def call(R=4, NK=64, Lx=8, c=1, A=FAKE, M=FAKE, S=FAKE, phi=FAKE, rows=256, w=FAKE,
             nb=1 << 40):
        return L.moe_schedule(R, NK, Lx, c, A, M, S, phi, rows, w, nb, None)

    assert call(c=4) == B.MOE_EINVAL          # c >= R
    assert call(c=-1) == B.MOE_EINVAL
    assert call(NK=-1) == B.MOE_EINVAL
    assert call(Lx=0) == B.MOE_EINVAL
    assert call(A=None) == B.MOE_EINVAL
    assert call(phi=MISALIGNED) == B.MOE_EINVAL
    assert call(rows=-1) == B.MOE_EINVAL
    assert call(w=None) == B.MOE_EINVAL
    assert call(nb=8) == B.MOE_ENOSPACE
    assert call(R=2000, c=0) == B.MOE_EUNSUPPORTED
    assert call(Lx=512) == B.MOE_EUNSUPPORTED


def test_mx_workspace_and_validation():
    L = B.lib()
    sh = B.make_shape(64, 256, 8, 2, 256, 256)
    mx_bytes = B.moe_mx_workspace_bytes(sh)
    assert mx_bytes >= B.moe_workspace_bytes(sh, False) + 64 * 256 + 128 * 256
    for which in (B.WS_ERROR, B.WS_YEXP, B.WS_YSH, B.WS_XQ, B.WS_XS, B.WS_HQ, B.WS_HS):
        off, nb = B.moe_mx_workspace_region(sh, which)
        assert off % 256 == 0 and off + nb <= mx_bytes
    off, nb = B.moe_mx_workspace_region(sh, B.WS_A)               # the shared layout's regions
    assert (off, nb) == B.moe_workspace_region(sh, True, B.WS_A)
    mxb = B.moe_mx_workspace_bytes(sh, True)
    assert mxb >= B.moe_workspace_bytes(sh, True) + 64 * 256 + 2 * 128 * 256
    for which in (B.WS_DYQ, B.WS_DYS, B.WS_DAQ, B.WS_DAS, B.WS_DBQ, B.WS_DBS):
        off, nb = B.moe_mx_workspace_region(sh, which)
        assert off % 256 == 0 and off + nb <= mxb
        assert off >= B.moe_workspace_bytes(sh, True)           # past every BF16 region
    assert B.moe_mx_workspace_bytes(B.make_shape(1 << 20, 4096, 8, 2, 256)) == 0   # T*d >= 2^32
    # MXFP8 weight gradients: the token-axis operands after everything else
    mxw = B.moe_mx_workspace_bytes(sh, 2)
    P = (sh.T * sh.k + 128 * sh.E + 127) // 128 * 128
    assert mxw >= mxb + (2 * sh.d + 3 * sh.f) * P
    for which, size in ((B.WS_POFF, (sh.E + 1) * 4), (B.WS_XTQ, sh.d * P), (B.WS_XTS, sh.d * P // 32),
                        (B.WS_DYTQ, sh.d * P), (B.WS_DYTS, sh.d * P // 32)):
        off, nb = B.moe_mx_workspace_region(sh, which)
        assert nb == size and off % 256 == 0 and off >= mxb and off + nb <= mxw, which
    assert B.moe_mx_workspace_bytes(sh, 3) == 0 and B.moe_mx_workspace_bytes(sh, -1) == 0
    # d * P >= 2^32 while T*d, T*k*f and E*f*d stay below it
    big_t = B.make_shape(1 << 18, 4096, 8, 8, 256, 256)
    assert B.moe_mx_workspace_bytes(big_t, 1) > 0 and B.moe_mx_workspace_bytes(big_t, 2) == 0
    w = B.MoeWeights(None, None, None, FAKE, FAKE, FAKE)          # routed bf16 weights unused
    mx = B.MoeMxWeights(FAKE, FAKE, FAKE, FAKE, FAKE, FAKE)
    plan = B.MoePlanBufs(FAKE, FAKE, FAKE, FAKE)
    big = 1 << 40

    def fwd(shape=sh, X=FAKE, weights=w, q=mx, Y=FAKE, nb=big):
        return L.moe_forward_mx(ctypes.byref(shape), X, ctypes.byref(weights), ctypes.byref(q),
                                FAKE, FAKE, ctypes.byref(plan), Y, 0, FAKE, nb, None, None)

    assert fwd(nb=mx_bytes - 1) == B.MOE_ENOSPACE
    assert fwd(X=None) == B.MOE_EINVAL
    assert fwd(Y=MISALIGNED) == B.MOE_EINVAL
    assert fwd(q=B.MoeMxWeights(FAKE, None, FAKE, FAKE, FAKE, FAKE)) == B.MOE_EINVAL
    assert fwd(weights=B.MoeWeights(None, None, None, None, None, None)) == B.MOE_EINVAL  # shared
    sh_ns = B.make_shape(64, 256, 8, 2, 256)
    assert fwd(shape=sh_ns) == B.MOE_EINVAL                       # shared weights without f_shared
    assert fwd(shape=B.make_shape(1 << 20, 4096, 8, 2, 256)) == B.MOE_EUNSUPPORTED
    wq = B.MoeWeights(FAKE, FAKE, FAKE, None, None, None)
    assert L.moe_mx_quantize_weights(ctypes.byref(sh), ctypes.byref(B.MoeWeights()),
                                     ctypes.byref(mx), None) == B.MOE_EINVAL
    assert L.moe_mx_quantize_weights(ctypes.byref(sh), ctypes.byref(wq),
                                     ctypes.byref(B.MoeMxWeights()), None) == B.MOE_EINVAL
    assert L.moe_mx_quantize_weights_bwd(ctypes.byref(sh), ctypes.byref(wq),
                                         ctypes.byref(B.MoeMxBwdWeights()), None) == B.MOE_EINVAL
    # backward: workspace, weights and gradient checks
    wb = B.MoeWeights(FAKE, FAKE, FAKE, FAKE, FAKE, FAKE)
    qb = B.MoeMxBwdWeights(FAKE, FAKE, FAKE, FAKE, FAKE, FAKE)
    g = B.MoeGrads(FAKE, FAKE, FAKE, FAKE, None, FAKE, FAKE, FAKE)

    def bwd(q=qb, grads=g, nb=big, dX=FAKE, wgrad=0, shape=sh):
        return L.moe_backward_mx(ctypes.byref(shape), FAKE, FAKE, FAKE, ctypes.byref(wb),
                                 ctypes.byref(q), FAKE, FAKE, ctypes.byref(plan), dX,
                                 ctypes.byref(grads), wgrad, FAKE, nb, None)

    assert bwd(nb=mxb - 1) == B.MOE_ENOSPACE
    assert bwd(nb=mxw - 1, wgrad=1) == B.MOE_ENOSPACE             # room for the token-axis operands
    assert bwd(wgrad=2) == B.MOE_EINVAL
    assert bwd(wgrad=1, shape=big_t) == B.MOE_EUNSUPPORTED
    assert bwd(q=B.MoeMxBwdWeights(FAKE, FAKE, None, FAKE, FAKE, FAKE)) == B.MOE_EINVAL
    assert bwd(grads=B.MoeGrads(FAKE, None, FAKE, FAKE, None, FAKE, FAKE, FAKE)) == B.MOE_EINVAL
    assert bwd(dX=MISALIGNED) == B.MOE_EINVAL


def test_oracle_is_not_imported_by_the_package():
    import sys
    import importlib
    for mod in ("paper_2609_36070_amd", "paper_2609_36070_amd.binding",
                "paper_2609_36070_amd.layer", "paper_2609_36070_amd.workloads"):
        importlib.import_module(mod)
    pkg_dir = os.path.dirname(B.__file__)
    for fn in os.listdir(pkg_dir):
        if fn.endswith(".py"):
            src = open(os.path.join(pkg_dir, fn)).read()
            assert "import oracle" not in src and "from oracle" not in src, fn


def test_plan_noalloc_validation():
    """Rejected on the host before any HIP call: bad pointers, and shapes whose
    plan scratch exceeds the library-held array."""
    sh = B.make_shape(1000, 256, 8, 2, 256, 0)
    pb = B.MoePlanBufs(FAKE, FAKE, FAKE, FAKE)
    L = B.lib()
    assert L.moe_plan_noalloc(ctypes.byref(sh), None, ctypes.byref(pb), FAKE, None) == B.MOE_EINVAL
    assert L.moe_plan_noalloc(ctypes.byref(sh), FAKE, ctypes.byref(pb), None, None) == B.MOE_EINVAL
    assert L.moe_plan_noalloc(ctypes.byref(sh), FAKE, ctypes.byref(pb), MISALIGNED, None) == B.MOE_EINVAL
    bad = B.MoePlanBufs(FAKE, None, FAKE, FAKE)
    assert L.moe_plan_noalloc(ctypes.byref(sh), FAKE, ctypes.byref(bad), FAKE, None) == B.MOE_EINVAL
    big = B.make_shape(300000, 256, 256, 8, 256, 0)     # ~4.8 MB of scratch needed
    assert L.moe_plan_noalloc(ctypes.byref(big), FAKE, ctypes.byref(pb), FAKE, None) == B.MOE_EUNSUPPORTED
    ok = B.make_shape(200000, 256, 256, 8, 256, 0)      # ~3.2 MB: admitted (not run here)
    assert 8 * -(-200000 * 8 // 1024) * 256 + 4 * -(-200000 * 8 // 1024) <= B.PLAN_NOALLOC_SCRATCH_BYTES
    del ok

