"""Device buffers for one MoE layer and the call sequence of one step.

Torch provides device memory and the stream; every computation is a call
into libmoe.so through :mod:`paper_2609_36070_amd.binding`.
"""
from __future__ import annotations

import numpy as np
import torch

from . import binding as B
from .workloads import Workload


def _empty(shape, dtype, device):
    """Uninitialised tensor whose data pointer is valid even when it has no elements."""
    n = int(np.prod(shape))
    return torch.empty((max(n, 1),), dtype=dtype, device=device)[:n].view(*shape)


def _dev_bf16(a, device):
    if a is None:
        return None
    a = np.ascontiguousarray(a, np.float32)
    out = _empty(a.shape, torch.bfloat16, device)
    if a.size:
        out.copy_(torch.from_numpy(a).to(torch.bfloat16))
    return out


class DeviceLayer:
    """All tensors of one layer instance on the GPU, laid out as the C ABI expects."""

    def __init__(self, w: Workload, inputs: dict, device="cuda", with_backward=None, mx=False,
                 ring_rows=None, mx_wgrad=False):
        """ring_rows: run forward/backward in bounded memory, with the per-route
        activations in a ring of that many rows (None: room for all T*k routes).
        mx_wgrad: the MXFP8 backward computes its weight gradients in MXFP8."""
        self.w = w
        self.mx = mx
        self.mx_wgrad = bool(mx_wgrad)
        self.ring_rows = ring_rows
        self.device = torch.device(device)
        self.with_backward = w.backward if with_backward is None else with_backward
        T, d, E, k, f, fs = w.T, w.d, w.E, w.k, w.f, w.f_s
        dev = self.device
        self.shape = B.make_shape(T, d, E, k, f, fs)
        self.X = _dev_bf16(inputs["X"], dev)
        self.W_r = _dev_bf16(inputs["W_r"], dev)
        self.bias = None if inputs.get("bias") is None else \
            torch.from_numpy(np.asarray(inputs["bias"], np.float32)).to(dev)
        self.W_gate = _dev_bf16(inputs["W_gate"], dev)
        self.W_up = _dev_bf16(inputs["W_up"], dev)
        self.W_down = _dev_bf16(inputs["W_down"], dev)
        self.Wg_s = _dev_bf16(inputs.get("Wg_s"), dev)
        self.Wu_s = _dev_bf16(inputs.get("Wu_s"), dev)
        self.Wd_s = _dev_bf16(inputs.get("Wd_s"), dev)
        self.dY = _dev_bf16(inputs.get("dY"), dev) if self.with_backward else None

        i32, f32, bf = torch.int32, torch.float32, torch.bfloat16
        R = T * k
        self.logits = _empty((T, E), f32, dev)
        self.topk_idx = _empty((T, k), i32, dev)
        self.topk_w = _empty((T, k), f32, dev)
        self.counts = _empty((E,), i32, dev)
        self.offsets = _empty((E + 1,), i32, dev)
        self.perm = _empty((R,), i32, dev)
        self.route_pos = _empty((R,), i32, dev)
        self.Y = _empty((T, d), bf, dev)
        if ring_rows is None:
            nbytes = B.moe_workspace_bytes(self.shape, self.with_backward)
        else:
            if mx:
                raise ValueError("the MXFP8 forward has no bounded-memory variant")
            nbytes = B.moe_ring_workspace_bytes(self.shape, ring_rows, self.with_backward)
        if nbytes == 0:
            raise ValueError(f"unsupported shape {w}")
        if mx:
            mx_bytes = B.moe_mx_workspace_bytes(
                self.shape, (2 if self.mx_wgrad else 1) if self.with_backward else 0)
            if mx_bytes == 0:
                raise ValueError(f"shape unsupported in MXFP8 {w}")
            nbytes = max(nbytes, mx_bytes)
        self.ws = torch.empty((nbytes,), dtype=torch.uint8, device=dev)
        self.weights = B.weights_struct(self.W_gate, self.W_up, self.W_down,
                                        self.Wg_s, self.Wu_s, self.Wd_s)
        self.plan_bufs = B.plan_bufs(self.counts, self.offsets, self.perm, self.route_pos)
        if self.with_backward:
            self.dX = _empty((T, d), bf, dev)
            self.dW_gate = torch.empty((E, d, f), dtype=f32, device=dev)
            self.dW_up = torch.empty((E, d, f), dtype=f32, device=dev)
            self.dW_down = torch.empty((E, f, d), dtype=f32, device=dev)
            self.dW_r = torch.empty((d, E), dtype=f32, device=dev)
            self.dZ = _empty((T, E), f32, dev)
            if fs:
                self.dWg_s = torch.empty((d, fs), dtype=f32, device=dev)
                self.dWu_s = torch.empty((d, fs), dtype=f32, device=dev)
                self.dWd_s = torch.empty((fs, d), dtype=f32, device=dev)
            else:
                self.dWg_s = self.dWu_s = self.dWd_s = None
            self.grads = B.grads_struct(self.dW_gate, self.dW_up, self.dW_down, self.dW_r, self.dZ,
                                        self.dWg_s, self.dWu_s, self.dWd_s)

        if mx:
            u8 = torch.uint8
            self.Wg_q = torch.empty((E, f, d), dtype=u8, device=dev)
            self.Wu_q = torch.empty((E, f, d), dtype=u8, device=dev)
            self.Wd_q = torch.empty((E, d, f), dtype=u8, device=dev)
            self.Wg_sc = torch.empty((E, f, d // 32), dtype=u8, device=dev)
            self.Wu_sc = torch.empty((E, f, d // 32), dtype=u8, device=dev)
            self.Wd_sc = torch.empty((E, d, f // 32), dtype=u8, device=dev)
            self.mx_weights = B.mx_weights_struct(self.Wg_q, self.Wu_q, self.Wd_q, self.Wg_sc,
                                                  self.Wu_sc, self.Wd_sc)
            if self.with_backward:
                # backward layouts: each weight row quantised along its own axis
                self.Wg_qb = torch.empty((E, d, f), dtype=u8, device=dev)
                self.Wu_qb = torch.empty((E, d, f), dtype=u8, device=dev)
                self.Wd_qb = torch.empty((E, f, d), dtype=u8, device=dev)
                self.Wg_scb = torch.empty((E, d, f // 32), dtype=u8, device=dev)
                self.Wu_scb = torch.empty((E, d, f // 32), dtype=u8, device=dev)
                self.Wd_scb = torch.empty((E, f, d // 32), dtype=u8, device=dev)
                self.mx_bwd_weights = B.mx_bwd_weights_struct(self.Wg_qb, self.Wu_qb, self.Wd_qb,
                                                              self.Wg_scb, self.Wu_scb, self.Wd_scb)
            self.quantize_mx()

    # -- the four calls of the path --------------------------------------
    def route(self, stream=None):
        B.moe_route(self.shape, self.X, self.W_r, self.bias, self.logits, self.topk_idx,
                    self.topk_w, self.ws, stream=stream)

    def plan(self, stream=None):
        B.moe_plan(self.shape, self.topk_idx, self.plan_bufs, self.ws, stream=stream)

    def forward(self, save_for_backward=None, stream=None, events=None):
        save = self.with_backward if save_for_backward is None else save_for_backward
        if self.ring_rows is not None:
            if events is not None:
                raise ValueError("stage events are not recorded in bounded-memory execution")
            B.moe_forward_ring(self.shape, self.X, self.weights, self.topk_idx, self.topk_w,
                               self.plan_bufs, self.Y, self.ring_rows, save, self.ws,
                               stream=stream)
            return
        B.moe_forward(self.shape, self.X, self.weights, self.topk_idx, self.topk_w,
                      self.plan_bufs, self.Y, save, self.ws, stream=stream, events=events)

    def forward_fused(self, save_for_backward=None, stream=None):
        """The forward as one persistent launch (same results as forward())."""
        if self.ring_rows is not None:
            raise ValueError("the fused forward has no bounded-memory variant")
        save = self.with_backward if save_for_backward is None else save_for_backward
        B.moe_forward_fused(self.shape, self.X, self.weights, self.topk_idx, self.topk_w,
                            self.plan_bufs, self.Y, save, self.ws, stream=stream)

    def backward(self, stream=None, events=None):
        if self.ring_rows is not None:
            if events is not None:
                raise ValueError("stage events are not recorded in bounded-memory execution")
            B.moe_backward_ring(self.shape, self.dY, self.X, self.W_r, self.weights,
                                self.topk_idx, self.topk_w, self.plan_bufs, self.dX, self.grads,
                                self.ring_rows, self.ws, stream=stream)
            return
        B.moe_backward(self.shape, self.dY, self.X, self.W_r, self.weights, self.topk_idx,
                       self.topk_w, self.plan_bufs, self.dX, self.grads, self.ws, stream=stream,
                       events=events)

    def quantize_mx(self, stream=None):
        """Pre-quantise the routed weights to MXFP8 (once per weight update)."""
        B.moe_mx_quantize_weights(self.shape, self.weights, self.mx_weights, stream=stream)
        if self.with_backward:
            B.moe_mx_quantize_weights_bwd(self.shape, self.weights, self.mx_bwd_weights,
                                          stream=stream)

    def forward_mx(self, stream=None, events=None, save_for_backward=None):
        save = self.with_backward if save_for_backward is None else save_for_backward
        B.moe_forward_mx(self.shape, self.X, self.weights, self.mx_weights, self.topk_idx,
                         self.topk_w, self.plan_bufs, self.Y, self.ws, stream=stream,
                         events=events, save_for_backward=save)

    def backward_mx(self, stream=None):
        B.moe_backward_mx(self.shape, self.dY, self.X, self.W_r, self.weights, self.mx_bwd_weights,
                          self.topk_idx, self.topk_w, self.plan_bufs, self.dX, self.grads, self.ws,
                          stream=stream, wgrad_mxfp8=self.mx_wgrad)

    def step_mx(self, stream=None, fwd_events=None):
        """Route, plan, the MXFP8 forward (and the MXFP8 backward)."""
        self.route(stream)
        self.plan(stream)
        self.forward_mx(stream=stream, events=fwd_events)
        if self.with_backward:
            self.backward_mx(stream)

    def step(self, stream=None, fwd_events=None, bwd_events=None):
        """One pass of the whole path: route, plan, forward (and backward)."""
        self.route(stream)
        self.plan(stream)
        self.forward(stream=stream, events=fwd_events)
        if self.with_backward:
            self.backward(stream, events=bwd_events)

    # -- inspection -------------------------------------------------------
    def ws_tensor(self, which, dtype, shape):
        if self.ring_rows is not None and which != B.WS_ERROR:
            raise ValueError("named regions describe the one-pass layout only")
        off, nbytes = B.moe_workspace_region(self.shape, self.with_backward, which)
        return self.ws[off:off + nbytes].view(dtype).view(*shape)

    def mx_ws_tensor(self, which, dtype, shape):
        off, nbytes = B.moe_mx_workspace_region(self.shape, which)
        return self.ws[off:off + nbytes].view(dtype).view(*shape)

    def error_word(self) -> int:
        return int(self.ws_tensor(B.WS_ERROR, torch.int32, (1,)).item())
