"""Seeded synthetic MoE-layer workloads.

This module only *makes inputs*: it draws tensors from a seeded generator and
rounds them to bf16.  It holds none of the layer's arithmetic, so both the CPU
oracle side of the tests and the GPU path can consume the same arrays.

Input recipe (the paper generates router logits and model inputs from a
standard normal distribution and hands every implementation bitwise-identical
copies, §4.1 "MoE Layer Benchmarks"):

* ``rng = numpy.random.default_rng(seed)`` (PCG64), draws in this order:
  X[T,d]; W_r[d,E]; bias[E] (if the workload has one); W_gate[E,d,f];
  W_up[E,d,f]; W_down[E,f,d]; then Wg_s[d,f_s], Wu_s[d,f_s], Wd_s[f_s,d]
  (if there is a shared expert); then the hot-token subset (if any); then
  dY[T,d] (training workloads).
* every value is ``standard_normal(float32) * std`` with std = 1 for X and dY,
  1/sqrt(fan_in) for every weight (so logits are about N(0,1)), 0.5 for the
  per-expert router bias.
* hot-expert workloads: a seeded choice of floor(0.1*T) tokens gets
  ``x += 8 * w0 / |w0|^2`` (w0 = router column 0 before rounding), which lifts
  their expert-0 logit by about 8 standard deviations.
* X, W_r, all expert weights and dY are rounded to bf16 (round to nearest
  even); the bias stays fp32.

Arrays are returned as float32 numpy arrays whose values are exactly
representable in bf16.
"""
from __future__ import annotations

import dataclasses
import numpy as np


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    T: int          # tokens on this GPU
    d: int          # hidden size (the paper's D)
    E: int          # local routed experts
    k: int          # routes per token (top-k)
    f: int          # routed-expert intermediate size (the paper's I)
    f_s: int = 0    # shared-expert intermediate size, 0 = no shared expert
    bias_std: float = 0.0   # per-expert router-logit bias std, 0 = no bias
    hot_frac: float = 0.0   # fraction of tokens pushed onto expert 0
    backward: bool = False  # training workload (needs dY)
    note: str = ""

    @property
    def routes(self) -> int:
        return self.T * self.k

    def fwd_flops(self) -> float:
        """Expert-FFN FLOPs of one forward pass, 6*T*(k*f + f_s)*d (§4.1)."""
        return 6.0 * self.T * (self.k * self.f + self.f_s) * self.d

    def bwd_flops(self) -> float:
        """The backward pass counts twice the forward FLOPs (§4.1)."""
        return 2.0 * self.fwd_flops()

    def scaled(self, **kw) -> "Workload":
        return dataclasses.replace(self, **kw)


WORKLOADS = {
    "tiny": Workload(
        "tiny", T=256, d=256, E=8, k=2, f=512,
        note="tiny layer, top-2 of 8, no shared expert"),
    "many_experts": Workload(
        "many_experts", T=8192, d=2048, E=128, k=8, f=768, bias_std=0.5,
        note="128 small experts, top-8, per-expert bias skews the load"),
    "hot_expert": Workload(
        "hot_expert", T=16384, d=4096, E=32, k=8, f=1536, hot_frac=0.1,
        note="32 local experts (share of 128), 10% of tokens forced to expert 0"),
    "large_shared": Workload(
        "large_shared", T=16384, d=7168, E=8, k=8, f=2048, f_s=2048, bias_std=0.5,
        note="8 local experts (share of 256), top-8 over the local set, shared expert"),
    "large_shared_train": Workload(
        "large_shared_train", T=16384, d=7168, E=8, k=8, f=2048, f_s=2048,
        bias_std=0.5, backward=True,
        note="forward + backward of the large_shared layer"),
}


def to_bf16(a: np.ndarray) -> np.ndarray:
    """Round float32 values to the nearest bf16 (ties to even); returns float32."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    u = a.view(np.uint32).astype(np.uint64)
    u = (u + 0x7FFF + ((u >> 16) & 1)) >> 16
    return (u.astype(np.uint32) << 16).view(np.float32)


def bf16_bits(a: np.ndarray) -> np.ndarray:
    """The bf16 bit patterns (uint16) of a float32 array of bf16-exact values."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    return (a.view(np.uint32) >> 16).astype(np.uint16)


def make_inputs(w: Workload, seed: int = 0) -> dict:
    """Draw the workload's tensors (see the module docstring for the recipe)."""
    rng = np.random.default_rng(seed)
    T, d, E, f, fs = w.T, w.d, w.E, w.f, w.f_s

    def normal(shape, std):
        return rng.standard_normal(shape, dtype=np.float32) * np.float32(std)

    X = normal((T, d), 1.0)
    W_r = normal((d, E), 1.0 / np.sqrt(d))
    bias = normal((E,), w.bias_std) if w.bias_std > 0 else None
    W_gate = normal((E, d, f), 1.0 / np.sqrt(d))
    W_up = normal((E, d, f), 1.0 / np.sqrt(d))
    W_down = normal((E, f, d), 1.0 / np.sqrt(f))
    if fs > 0:
        Wg_s = normal((d, fs), 1.0 / np.sqrt(d))
        Wu_s = normal((d, fs), 1.0 / np.sqrt(d))
        Wd_s = normal((fs, d), 1.0 / np.sqrt(fs))
    else:
        Wg_s = Wu_s = Wd_s = None
    hot = None
    if w.hot_frac > 0:
        n_hot = int(np.floor(w.hot_frac * T))
        hot = np.sort(rng.choice(T, size=n_hot, replace=False)).astype(np.int64)
        w0 = W_r[:, 0].astype(np.float64)
        X[hot] += (8.0 * w0 / np.dot(w0, w0)).astype(np.float32)
    dY = normal((T, d), 1.0) if w.backward else None

    out = dict(
        X=to_bf16(X), W_r=to_bf16(W_r), bias=bias,
        W_gate=to_bf16(W_gate), W_up=to_bf16(W_up), W_down=to_bf16(W_down),
        Wg_s=None if Wg_s is None else to_bf16(Wg_s),
        Wu_s=None if Wu_s is None else to_bf16(Wu_s),
        Wd_s=None if Wd_s is None else to_bf16(Wd_s),
        dY=None if dY is None else to_bf16(dY),
        hot_tokens=hot,
    )
    return out


# ---------------------------------------------------------------------------
# All-gathered route tables for the multi-rank dispatch schedule
# ---------------------------------------------------------------------------

@dataclasses.dataclass(frozen=True)
class RouteTable:
    name: str
    R: int          # source ranks (expert-parallel degree)
    N: int          # tokens per rank
    K: int          # routes per token
    L: int          # experts per rank (R*L experts in all)
    bias_std: float = 0.5   # per-expert popularity skew: weight exp(bias), bias ~ N(0, std)
    hot_frac: float = 0.0   # fraction of tokens that always take global expert 0
    note: str = ""

    @property
    def NK(self) -> int:
        return self.N * self.K


ROUTE_TABLES = {
    "ep4": RouteTable("ep4", R=4, N=16384, K=8, L=32, hot_frac=0.1,
                      note="128 experts over 4 ranks (the hot-expert layer's global view)"),
    "ep16": RouteTable("ep16", R=16, N=4096, K=8, L=16,
                       note="256 experts over 16 ranks"),
    "ep64": RouteTable("ep64", R=64, N=2048, K=8, L=4,
                       note="256 experts over 64 ranks, 2048 tokens per rank"),
}


def make_route_table(t: RouteTable, seed: int = 0) -> np.ndarray:
    """A[R, N*K] int32, token-major (route j = token*K + slot).

    Each token draws K distinct experts out of R*L without replacement with
    probabilities proportional to exp(bias) (Gumbel top-K sampling), lists
    them in ascending id, and a seeded ``hot_frac`` of the tokens always
    includes expert 0.  Draw order: bias[R*L], the hot-token subset, then
    the Gumbel noise in blocks of 4096 tokens.
    """
    rng = np.random.default_rng(seed)
    E, T = t.R * t.L, t.R * t.N
    bias = rng.standard_normal(E) * t.bias_std
    hot = np.zeros(T, bool)
    if t.hot_frac > 0:
        hot[rng.choice(T, size=int(np.floor(t.hot_frac * T)), replace=False)] = True
    out = np.empty((T, t.K), np.int32)
    for s in range(0, T, 4096):
        e = min(T, s + 4096)
        g = rng.gumbel(size=(e - s, E)) + bias
        g[hot[s:e], 0] = np.inf
        pick = np.argpartition(-g, t.K - 1, axis=1)[:, :t.K]
        out[s:e] = np.sort(pick, axis=1)
    return out.reshape(t.R, t.N * t.K)
