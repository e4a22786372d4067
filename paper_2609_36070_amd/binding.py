"""ctypes binding of libmoe.so: one Python function per C entry point.

Argument marshalling only.  Tensors are torch tensors on the GPU (passed by
data pointer); every step of the layer runs in the HIP library.  The library
must be built in-tree first (``python -m paper_2609_36070_amd.build``); if it
is missing, loading raises instead of falling back to anything else.
"""
from __future__ import annotations

import ctypes
import os

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libmoe.so")

c_void_p = ctypes.c_void_p
c_int64 = ctypes.c_int64
c_size_t = ctypes.c_size_t
c_int = ctypes.c_int

MOE_OK, MOE_EINVAL, MOE_EUNSUPPORTED, MOE_ENOSPACE, MOE_EHIP = range(5)
WS_ERROR, WS_A, WS_B, WS_H, WS_YEXP, WS_YSH, WS_DG, WS_DA, WS_DB, WS_DXPERM = range(10)
WS_XQ, WS_XS, WS_HQ, WS_HS = range(10, 14)
WS_DYQ, WS_DYS, WS_DAQ, WS_DAS, WS_DBQ, WS_DBS = range(14, 20)
WS_POFF, WS_XTQ, WS_XTS, WS_DYTQ, WS_DYTS = range(20, 25)
WS_HW = 25
WS_AF, WS_BF, WS_DAF, WS_DBF, WS_HWF = range(26, 31)

EXPORTS = ("moe_workspace_bytes", "moe_workspace_region", "moe_route", "moe_plan",
           "moe_schedule_workspace_bytes", "moe_schedule", "moe_dispatch", "moe_forward",
           "moe_backward", "moe_mx_quantize_weights", "moe_mx_workspace_bytes",
           "moe_mx_workspace_region", "moe_forward_mx", "moe_ring_workspace_bytes",
           "moe_forward_ring", "moe_backward_ring", "moe_forward_fused",
           "moe_mx_quantize_weights_bwd", "moe_backward_mx", "moe_plan_noalloc", "moe_status_string",
           "moe_version")
PLAN_NOALLOC_SCRATCH_BYTES = 4 << 20


class MoeShape(ctypes.Structure):
    _fields_ = [("T", c_int64), ("d", c_int64), ("E", c_int64), ("k", c_int64),
                ("f", c_int64), ("f_shared", c_int64)]


class MoeWeights(ctypes.Structure):
    _fields_ = [(n, c_void_p) for n in ("W_gate", "W_up", "W_down", "Wg_s", "Wu_s", "Wd_s")]


class MoeMxWeights(ctypes.Structure):
    _fields_ = [(n, c_void_p) for n in ("Wg_q", "Wu_q", "Wd_q", "Wg_s", "Wu_s", "Wd_s")]


class MoeMxBwdWeights(ctypes.Structure):
    _fields_ = [(n, c_void_p) for n in ("Wg_q", "Wu_q", "Wd_q", "Wg_s", "Wu_s", "Wd_s")]


class MoePlanBufs(ctypes.Structure):
    _fields_ = [(n, c_void_p) for n in ("counts", "offsets", "perm", "route_pos")]


class MoeGrads(ctypes.Structure):
    _fields_ = [(n, c_void_p) for n in ("dW_gate", "dW_up", "dW_down", "dW_r", "dZ",
                                        "dWg_s", "dWu_s", "dWd_s")]


MAX_STAGE_EVENTS = 16
FWD_STAGES = ("prologue", "up_routed", "up_shared", "down_routed", "down_shared", "combine")
BWD_STAGES = ("prologue", "dgrad_routed", "softmax_bwd", "dx_routed", "wgrad_gate_up",
              "wgrad_down", "dgrad_shared", "dx_shared", "wgrad_shared", "dw_router",
              "reverse_combine")


class MoeStageEvents(ctypes.Structure):
    _fields_ = [("ev", c_void_p * MAX_STAGE_EVENTS)]


class MoeError(RuntimeError):
    def __init__(self, fn, status):
        super().__init__(f"{fn} failed: {status_string(status)} ({status})")
        self.status = status


_lib = None


def lib():
    """Load libmoe.so (raises FileNotFoundError if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise FileNotFoundError(
                f"{LIB_PATH} not found: build it with python -m paper_2609_36070_amd.build")
        # bind every symbol now: a missing kernel stub fails here, not at a launch
        L = ctypes.CDLL(LIB_PATH, mode=os.RTLD_NOW | os.RTLD_LOCAL)
        P = ctypes.POINTER
        L.moe_workspace_bytes.argtypes = [P(MoeShape), c_int]
        L.moe_workspace_bytes.restype = c_size_t
        L.moe_workspace_region.argtypes = [P(MoeShape), c_int, c_int, P(c_size_t), P(c_size_t)]
        L.moe_route.argtypes = [P(MoeShape)] + [c_void_p] * 7 + [c_size_t, c_void_p]
        L.moe_plan.argtypes = [P(MoeShape), c_void_p, P(MoePlanBufs), c_void_p, c_size_t, c_void_p]
        L.moe_plan_noalloc.argtypes = [P(MoeShape), c_void_p, P(MoePlanBufs), c_void_p, c_void_p]
        L.moe_dispatch.argtypes = [P(MoeShape), c_void_p, P(MoePlanBufs), c_void_p, c_void_p]
        L.moe_schedule_workspace_bytes.argtypes = [ctypes.c_int64] * 3
        L.moe_schedule_workspace_bytes.restype = c_size_t
        L.moe_schedule.argtypes = ([ctypes.c_int64] * 4 + [c_void_p] * 4
                                   + [ctypes.c_int64, c_void_p, c_size_t, c_void_p])
        L.moe_forward.argtypes = [P(MoeShape), c_void_p, P(MoeWeights), c_void_p, c_void_p,
                                  P(MoePlanBufs), c_void_p, c_int, c_void_p, c_size_t, c_void_p,
                                  P(MoeStageEvents)]
        L.moe_backward.argtypes = [P(MoeShape), c_void_p, c_void_p, c_void_p, P(MoeWeights),
                                   c_void_p, c_void_p, P(MoePlanBufs), c_void_p, P(MoeGrads),
                                   c_void_p, c_size_t, c_void_p, P(MoeStageEvents)]
        L.moe_mx_quantize_weights.argtypes = [P(MoeShape), P(MoeWeights), P(MoeMxWeights),
                                              c_void_p]
        L.moe_mx_workspace_bytes.argtypes = [P(MoeShape), c_int]
        L.moe_mx_workspace_bytes.restype = c_size_t
        L.moe_mx_workspace_region.argtypes = [P(MoeShape), c_int, P(c_size_t), P(c_size_t)]
        L.moe_forward_mx.argtypes = [P(MoeShape), c_void_p, P(MoeWeights), P(MoeMxWeights),
                                     c_void_p, c_void_p, P(MoePlanBufs), c_void_p, c_int,
                                     c_void_p, c_size_t, c_void_p, P(MoeStageEvents)]
        L.moe_mx_quantize_weights_bwd.argtypes = [P(MoeShape), P(MoeWeights), P(MoeMxBwdWeights),
                                                  c_void_p]
        L.moe_backward_mx.argtypes = [P(MoeShape), c_void_p, c_void_p, c_void_p, P(MoeWeights),
                                      P(MoeMxBwdWeights), c_void_p, c_void_p, P(MoePlanBufs),
                                      c_void_p, P(MoeGrads), c_int, c_void_p, c_size_t, c_void_p]
        L.moe_forward_fused.argtypes = [P(MoeShape), c_void_p, P(MoeWeights), c_void_p, c_void_p,
                                        P(MoePlanBufs), c_void_p, c_int, c_void_p, c_size_t,
                                        c_void_p]
        L.moe_ring_workspace_bytes.argtypes = [P(MoeShape), ctypes.c_int64, c_int]
        L.moe_ring_workspace_bytes.restype = c_size_t
        L.moe_forward_ring.argtypes = [P(MoeShape), c_void_p, P(MoeWeights), c_void_p, c_void_p,
                                       P(MoePlanBufs), c_void_p, ctypes.c_int64, c_int, c_void_p,
                                       c_size_t, c_void_p]
        L.moe_backward_ring.argtypes = [P(MoeShape), c_void_p, c_void_p, c_void_p, P(MoeWeights),
                                        c_void_p, c_void_p, P(MoePlanBufs), c_void_p, P(MoeGrads),
                                        ctypes.c_int64, c_void_p, c_size_t, c_void_p]
        for fn in ("moe_route", "moe_plan", "moe_schedule", "moe_dispatch", "moe_forward",
                   "moe_backward", "moe_workspace_region", "moe_mx_quantize_weights",
                   "moe_mx_workspace_region", "moe_forward_mx", "moe_forward_ring",
                   "moe_backward_ring", "moe_forward_fused", "moe_mx_quantize_weights_bwd",
                   "moe_backward_mx"):
            getattr(L, fn).restype = c_int
        L.moe_status_string.argtypes = [c_int]
        L.moe_status_string.restype = ctypes.c_char_p
        L.moe_version.argtypes = []
        L.moe_version.restype = ctypes.c_char_p
        _lib = L
    return _lib


def status_string(status: int) -> str:
    return lib().moe_status_string(status).decode()


def version() -> str:
    return lib().moe_version().decode()


def _p(t):
    """Device pointer of a tensor (None -> NULL); plain ints pass through."""
    if t is None:
        return None
    if isinstance(t, int):
        return t
    if t.numel() == 0:
        # torch reports NULL for empty tensors; pass the (non-empty) storage instead
        return t.untyped_storage().data_ptr()
    return t.data_ptr()


def _stream(stream):
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    return stream if isinstance(stream, int) else stream.cuda_stream


def _check(fn, status, raise_on_error):
    if raise_on_error and status != MOE_OK:
        raise MoeError(fn, status)
    return status


def make_shape(T, d, E, k, f, f_shared=0) -> MoeShape:
    return MoeShape(T, d, E, k, f, f_shared)


def moe_workspace_bytes(shape: MoeShape, with_backward: bool) -> int:
    return int(lib().moe_workspace_bytes(ctypes.byref(shape), int(bool(with_backward))))


def moe_workspace_region(shape: MoeShape, with_backward: bool, which: int):
    off, nb = c_size_t(0), c_size_t(0)
    st = lib().moe_workspace_region(ctypes.byref(shape), int(bool(with_backward)), which,
                                    ctypes.byref(off), ctypes.byref(nb))
    _check("moe_workspace_region", st, True)
    return off.value, nb.value


def moe_route(shape, X, W_r, bias, logits, topk_idx, topk_w, ws, ws_bytes=None, stream=None,
              raise_on_error=True):
    nbytes = ws.numel() * ws.element_size() if ws_bytes is None else ws_bytes
    st = lib().moe_route(ctypes.byref(shape), _p(X), _p(W_r), _p(bias), _p(logits), _p(topk_idx),
                         _p(topk_w), _p(ws), nbytes, _stream(stream))
    return _check("moe_route", st, raise_on_error)


def plan_bufs(counts, offsets, perm, route_pos) -> MoePlanBufs:
    return MoePlanBufs(_p(counts), _p(offsets), _p(perm), _p(route_pos))


def weights_struct(W_gate, W_up, W_down, Wg_s=None, Wu_s=None, Wd_s=None) -> MoeWeights:
    return MoeWeights(_p(W_gate), _p(W_up), _p(W_down), _p(Wg_s), _p(Wu_s), _p(Wd_s))


def grads_struct(dW_gate, dW_up, dW_down, dW_r, dZ=None, dWg_s=None, dWu_s=None,
                 dWd_s=None) -> MoeGrads:
    return MoeGrads(_p(dW_gate), _p(dW_up), _p(dW_down), _p(dW_r), _p(dZ), _p(dWg_s), _p(dWu_s),
                    _p(dWd_s))


def moe_plan(shape, topk_idx, plan: MoePlanBufs, ws, ws_bytes=None, stream=None,
             raise_on_error=True):
    nbytes = ws.numel() * ws.element_size() if ws_bytes is None else ws_bytes
    st = lib().moe_plan(ctypes.byref(shape), _p(topk_idx), ctypes.byref(plan), _p(ws), nbytes,
                        _stream(stream))
    return _check("moe_plan", st, raise_on_error)


def moe_plan_noalloc(shape, topk_idx, plan: MoePlanBufs, error_word, stream=None,
                     raise_on_error=True):
    st = lib().moe_plan_noalloc(ctypes.byref(shape), _p(topk_idx), ctypes.byref(plan),
                                _p(error_word), _stream(stream))
    return _check("moe_plan_noalloc", st, raise_on_error)


def moe_schedule_workspace_bytes(R: int, NK: int, L: int) -> int:
    return int(lib().moe_schedule_workspace_bytes(R, NK, L))


def moe_schedule(R, NK, L, c, A, M, S, phi, phi_rows, ws, ws_bytes=None, stream=None,
                 raise_on_error=True):
    nbytes = ws.numel() * ws.element_size() if ws_bytes is None else ws_bytes
    st = lib().moe_schedule(R, NK, L, c, _p(A), _p(M), _p(S), _p(phi), phi_rows, _p(ws), nbytes,
                            _stream(stream))
    return _check("moe_schedule", st, raise_on_error)


def mx_weights_struct(Wg_q, Wu_q, Wd_q, Wg_s, Wu_s, Wd_s) -> MoeMxWeights:
    return MoeMxWeights(_p(Wg_q), _p(Wu_q), _p(Wd_q), _p(Wg_s), _p(Wu_s), _p(Wd_s))


def moe_mx_workspace_bytes(shape: MoeShape, with_backward: int = 0) -> int:
    """with_backward: 0 forward, 1 with the MXFP8 backward, 2 with its MXFP8
    weight gradients too."""
    return int(lib().moe_mx_workspace_bytes(ctypes.byref(shape), int(with_backward)))


def mx_bwd_weights_struct(Wg_q, Wu_q, Wd_q, Wg_s, Wu_s, Wd_s) -> MoeMxBwdWeights:
    return MoeMxBwdWeights(_p(Wg_q), _p(Wu_q), _p(Wd_q), _p(Wg_s), _p(Wu_s), _p(Wd_s))


def moe_mx_quantize_weights_bwd(shape, weights: MoeWeights, mx: MoeMxBwdWeights, stream=None,
                                raise_on_error=True):
    st = lib().moe_mx_quantize_weights_bwd(ctypes.byref(shape), ctypes.byref(weights),
                                           ctypes.byref(mx), _stream(stream))
    return _check("moe_mx_quantize_weights_bwd", st, raise_on_error)


def moe_backward_mx(shape, dY, X, W_r, weights: MoeWeights, mx: MoeMxBwdWeights, topk_idx, topk_w,
                    plan: MoePlanBufs, dX, grads: MoeGrads, ws, ws_bytes=None, stream=None,
                    raise_on_error=True, wgrad_mxfp8=False):
    nbytes = ws.numel() * ws.element_size() if ws_bytes is None else ws_bytes
    st = lib().moe_backward_mx(ctypes.byref(shape), _p(dY), _p(X), _p(W_r), ctypes.byref(weights),
                               ctypes.byref(mx), _p(topk_idx), _p(topk_w), ctypes.byref(plan),
                               _p(dX), ctypes.byref(grads), int(wgrad_mxfp8), _p(ws), nbytes,
                               _stream(stream))
    return _check("moe_backward_mx", st, raise_on_error)


def moe_mx_workspace_region(shape: MoeShape, which: int):
    off, nb = c_size_t(0), c_size_t(0)
    st = lib().moe_mx_workspace_region(ctypes.byref(shape), which, ctypes.byref(off),
                                       ctypes.byref(nb))
    _check("moe_mx_workspace_region", st, True)
    return off.value, nb.value


def moe_mx_quantize_weights(shape, weights: MoeWeights, mx: MoeMxWeights, stream=None,
                            raise_on_error=True):
    st = lib().moe_mx_quantize_weights(ctypes.byref(shape), ctypes.byref(weights),
                                       ctypes.byref(mx), _stream(stream))
    return _check("moe_mx_quantize_weights", st, raise_on_error)


def moe_forward_mx(shape, X, weights: MoeWeights, mx: MoeMxWeights, topk_idx, topk_w,
                   plan: MoePlanBufs, Y, ws, ws_bytes=None, stream=None, raise_on_error=True,
                   events: MoeStageEvents = None, save_for_backward=False):
    nbytes = ws.numel() * ws.element_size() if ws_bytes is None else ws_bytes
    st = lib().moe_forward_mx(ctypes.byref(shape), _p(X), ctypes.byref(weights), ctypes.byref(mx),
                              _p(topk_idx), _p(topk_w), ctypes.byref(plan), _p(Y),
                              int(bool(save_for_backward)), _p(ws), nbytes, _stream(stream),
                              None if events is None else ctypes.byref(events))
    return _check("moe_forward_mx", st, raise_on_error)


def moe_dispatch(shape, X, plan: MoePlanBufs, Xperm, stream=None, raise_on_error=True):
    st = lib().moe_dispatch(ctypes.byref(shape), _p(X), ctypes.byref(plan), _p(Xperm),
                            _stream(stream))
    return _check("moe_dispatch", st, raise_on_error)


def moe_forward(shape, X, weights: MoeWeights, topk_idx, topk_w, plan: MoePlanBufs, Y,
                save_for_backward, ws, ws_bytes=None, stream=None, raise_on_error=True,
                events: MoeStageEvents = None):
    nbytes = ws.numel() * ws.element_size() if ws_bytes is None else ws_bytes
    st = lib().moe_forward(ctypes.byref(shape), _p(X), ctypes.byref(weights), _p(topk_idx),
                           _p(topk_w), ctypes.byref(plan), _p(Y), int(bool(save_for_backward)),
                           _p(ws), nbytes, _stream(stream),
                           None if events is None else ctypes.byref(events))
    return _check("moe_forward", st, raise_on_error)


def moe_backward(shape, dY, X, W_r, weights: MoeWeights, topk_idx, topk_w, plan: MoePlanBufs, dX,
                 grads: MoeGrads, ws, ws_bytes=None, stream=None, raise_on_error=True,
                 events: MoeStageEvents = None):
    nbytes = ws.numel() * ws.element_size() if ws_bytes is None else ws_bytes
    st = lib().moe_backward(ctypes.byref(shape), _p(dY), _p(X), _p(W_r), ctypes.byref(weights),
                            _p(topk_idx), _p(topk_w), ctypes.byref(plan), _p(dX),
                            ctypes.byref(grads), _p(ws), nbytes, _stream(stream),
                            None if events is None else ctypes.byref(events))
    return _check("moe_backward", st, raise_on_error)


def moe_ring_workspace_bytes(shape: MoeShape, ring_rows: int, with_backward: bool) -> int:
    return int(lib().moe_ring_workspace_bytes(ctypes.byref(shape), int(ring_rows),
                                              int(bool(with_backward))))


def moe_forward_ring(shape, X, weights: MoeWeights, topk_idx, topk_w, plan: MoePlanBufs, Y,
                     ring_rows, save_for_backward, ws, ws_bytes=None, stream=None,
                     raise_on_error=True):
    nbytes = ws.numel() * ws.element_size() if ws_bytes is None else ws_bytes
    st = lib().moe_forward_ring(ctypes.byref(shape), _p(X), ctypes.byref(weights), _p(topk_idx),
                                _p(topk_w), ctypes.byref(plan), _p(Y), int(ring_rows),
                                int(bool(save_for_backward)), _p(ws), nbytes, _stream(stream))
    return _check("moe_forward_ring", st, raise_on_error)


def moe_backward_ring(shape, dY, X, W_r, weights: MoeWeights, topk_idx, topk_w,
                      plan: MoePlanBufs, dX, grads: MoeGrads, ring_rows, ws, ws_bytes=None,
                      stream=None, raise_on_error=True):
    nbytes = ws.numel() * ws.element_size() if ws_bytes is None else ws_bytes
    st = lib().moe_backward_ring(ctypes.byref(shape), _p(dY), _p(X), _p(W_r),
                                 ctypes.byref(weights), _p(topk_idx), _p(topk_w),
                                 ctypes.byref(plan), _p(dX), ctypes.byref(grads), int(ring_rows),
                                 _p(ws), nbytes, _stream(stream))
    return _check("moe_backward_ring", st, raise_on_error)


def moe_forward_fused(shape, X, weights: MoeWeights, topk_idx, topk_w, plan: MoePlanBufs, Y,
                      save_for_backward, ws, ws_bytes=None, stream=None, raise_on_error=True):
    nbytes = ws.numel() * ws.element_size() if ws_bytes is None else ws_bytes
    st = lib().moe_forward_fused(ctypes.byref(shape), _p(X), ctypes.byref(weights), _p(topk_idx),
                                 _p(topk_w), ctypes.byref(plan), _p(Y),
                                 int(bool(save_for_backward)), _p(ws), nbytes, _stream(stream))
    return _check("moe_forward_fused", st, raise_on_error)
