"""Seeded synthetic workloads for the MoCE forward pass.

This module only draws random tensors with the shapes and value distributions of
the layers the paper replaces (ResNet bottleneck entrance projections, a
token-wise ViT projection).  It performs none of the layer's arithmetic: no
pooling, gating, softmax, mixing, support sorting or coverage computation.  The
supports it returns are in the order they were sampled, not the canonical
descending-logit order; putting them in that order is part of the method and is
done by whoever consumes them (the HIP library or the CPU reference).

Both the HIP path and the CPU reference consume these arrays, so the module is
deliberately free of anything either of them computes.

Recipe (all draws from numpy ``Generator(PCG64)``, one child stream per tensor):

* ``x``: standard normal float32, passed through ``max(v, 0)`` for the
  post-ReLU convolutional activations (left signed for the pre-activation ViT
  tokens), then rounded to bfloat16 (round to nearest, ties to even) unless the
  workload is float32.  bf16 values are returned as their uint16 bit patterns.
* supports ``s[o, :]``: ``k`` distinct channels drawn uniformly without
  replacement, independently per routed expert (the random fixed assignment of
  the paper's support-design ablation).  When ``exclude > 0`` that many channels
  are first set aside and every support is drawn from the rest, redrawing until
  the rest is fully covered, so that exactly ``exclude`` channels are left to
  the residual expert.
* selected logits ``w ~ N(0, 1)``; gate slopes ``a ~ N(0, 1/k)``; gate offsets
  ``c = 0``.
* parameters of the paper's two-layer temperature gate (hidden width ``k``,
  ReLU, biases, scalar output): ``W1 ~ N(0, 1/k)``, ``b1 ~ N(0, 0.1^2)``,
  ``w2 ~ N(0, 1/k)``, ``b2 = 0``, ``tau`` range ``[0.2, 6.0]``.
"""
from __future__ import annotations

import dataclasses
from typing import Dict, Optional

import numpy as np

F32 = "f32"
BF16 = "bf16"
NCHW = "nchw"
NHWC = "nhwc"


@dataclasses.dataclass(frozen=True)
class Workload:
    """Shape and distribution of one MoCE layer instance.

    ``E`` counts all outputs: ``E - 1`` routed experts plus the residual one.
    Token inputs ``[B, N, C]`` are channels-last with ``H = N`` and ``W = 1``.
    """

    name: str
    B: int
    C: int
    E: int
    k: int
    H: int
    W: int
    dtype: str
    layouts: tuple
    signed: bool = False
    exclude: int = 0
    seed: int = 0

    @property
    def HW(self) -> int:
        return self.H * self.W

    @property
    def n_routed(self) -> int:
        return self.E - 1

    @property
    def elem_bytes(self) -> int:
        return 4 if self.dtype == F32 else 2

    def x_bytes(self) -> int:
        return self.B * self.C * self.HW * self.elem_bytes

    def y_bytes(self) -> int:
        return self.B * self.E * self.HW * self.elem_bytes

    def param_bytes(self) -> int:
        # int32 support + float32 logits + float32 gate slopes + float32 offsets
        r = self.n_routed
        return r * self.k * 4 * 3 + r * 4

    def describe(self) -> Dict[str, object]:
        return {
            "workload": self.name,
            "B": self.B, "C_in": self.C, "C_out": self.E, "k": self.k,
            "H": self.H, "W": self.W, "dtype": self.dtype,
        }


WORKLOADS: Dict[str, Workload] = {
    w.name: w
    for w in (
        Workload("tiny", B=2, C=64, E=16, k=8, H=8, W=8, dtype=F32,
                 layouts=(NCHW,), seed=0),
        Workload("resnet50_stage1", B=64, C=256, E=64, k=32, H=56, W=56,
                 dtype=BF16, layouts=(NCHW,), seed=1),
        Workload("resnet50_stage3", B=64, C=1024, E=256, k=64, H=14, W=14,
                 dtype=BF16, layouts=(NCHW, NHWC), exclude=51, seed=2),
        Workload("resnet50_stage4", B=128, C=2048, E=512, k=128, H=7, W=7,
                 dtype=BF16, layouts=(NHWC,), seed=3),
        Workload("vit_tokens", B=256, C=768, E=192, k=48, H=197, W=1,
                 dtype=BF16, layouts=(NHWC,), signed=True, seed=4),
    )
}


def f32_to_bf16_bits(v: np.ndarray) -> np.ndarray:
    """Round float32 values to bfloat16, nearest with ties to even.

    Returns the uint16 bit patterns.  Inputs must be finite (they are here).
    """
    u = np.ascontiguousarray(v, dtype=np.float32).view(np.uint32)
    rounded = u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))
    return (rounded >> np.uint32(16)).astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    """Widen bfloat16 bit patterns to float32 (exact)."""
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def _streams(seed: int):
    ss = np.random.SeedSequence(seed)
    return [np.random.Generator(np.random.PCG64(c)) for c in ss.spawn(5)]


def draw_supports(rng: np.random.Generator, C: int, n_routed: int, k: int,
                  exclude: int = 0) -> np.ndarray:
    """``n_routed`` rows of ``k`` distinct channels in sampling order (int32)."""
    if exclude == 0:
        rows = [rng.choice(C, size=k, replace=False) for _ in range(n_routed)]
        return np.asarray(rows, dtype=np.int32).reshape(n_routed, k)
    excluded = rng.choice(C, size=exclude, replace=False)
    keep = np.setdiff1d(np.arange(C), excluded)
    if k > keep.size:
        raise ValueError("support size exceeds the channels left after exclusion")
    for _ in range(1000):
        rows = [keep[rng.choice(keep.size, size=k, replace=False)] for _ in range(n_routed)]
        s = np.asarray(rows, dtype=np.int32).reshape(n_routed, k)
        if np.unique(s).size == keep.size:
            return s
    raise RuntimeError("could not draw supports covering every kept channel")


def generate(wl: Workload, layout: Optional[str] = None, with_x: bool = True,
             batch: Optional[int] = None) -> Dict[str, np.ndarray]:
    """Draw one seeded instance of ``wl``.

    ``layout`` picks NCHW (``x[B, C, H, W]``) or channels-last
    (``x[B, H, W, C]``); both layouts of one workload hold the same logical
    tensor.  ``batch`` draws only the first ``batch`` images (the same values
    as the full draw's first images).  Returned keys: ``x`` (float32, or uint16
    bf16 bits), ``s``, ``w``, ``a``, ``c``, ``W1``, ``b1``, ``w2``, ``b2``,
    ``tau_min``, ``tau_max``.
    """
    layout = layout or wl.layouts[0]
    if layout not in (NCHW, NHWC):
        raise ValueError(layout)
    rx, rs, rw, ra, rg = _streams(wl.seed)
    out: Dict[str, np.ndarray] = {}
    B = wl.B if batch is None else batch
    if with_x:
        # values are drawn in the workload's first listed layout, image by image
        native = wl.layouts[0]
        shape_native = (wl.C, wl.HW) if native == NCHW else (wl.HW, wl.C)
        per_image = wl.C * wl.HW
        x = rx.standard_normal(B * per_image, dtype=np.float32).reshape((B,) + shape_native)
        if not wl.signed:
            np.maximum(x, 0.0, out=x)
        if native != layout:
            x = np.ascontiguousarray(np.swapaxes(x, 1, 2))
        if layout == NCHW:
            x = x.reshape(B, wl.C, wl.H, wl.W)
        else:
            x = x.reshape(B, wl.H, wl.W, wl.C)
        out["x"] = f32_to_bf16_bits(x) if wl.dtype == BF16 else np.ascontiguousarray(x)
    r, k = wl.n_routed, wl.k
    out["s"] = draw_supports(rs, wl.C, r, k, wl.exclude)
    out["w"] = rw.standard_normal((r, k), dtype=np.float32)
    out["a"] = (ra.standard_normal((r, k), dtype=np.float32) * np.float32(k ** -0.5)).astype(np.float32)
    out["c"] = np.zeros(r, dtype=np.float32)
    out["W1"] = (rg.standard_normal((k, k), dtype=np.float32) * np.float32(k ** -0.5)).astype(np.float32)
    out["b1"] = (rg.standard_normal(k, dtype=np.float32) * np.float32(0.1)).astype(np.float32)
    out["w2"] = (rg.standard_normal(k, dtype=np.float32) * np.float32(k ** -0.5)).astype(np.float32)
    out["b2"] = np.float32(0.0)
    out["tau_min"] = np.float32(0.2)
    out["tau_max"] = np.float32(6.0)
    return out


def router_params(wl: Workload, d: int = 32) -> Dict[str, np.ndarray]:
    """Synthetic parameters of the input-conditioned variant (Sec. 4.5 Eq. 11)
    for ``wl``: the full static routing logits ``L[E-1, C] ~ N(0, 1)`` and the
    router ``Wh[d, C] ~ N(0, 4/C)``, ``bh[d] ~ N(0, 0.1^2)``, channel
    embeddings ``v[C, d] ~ N(0, 1)`` and expert embeddings
    ``q[E-1, d] ~ N(0, 1/d)`` (float32), scaled so that the per-example
    offset is of the order of the logits' spread and the examples' supports
    differ."""
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([wl.seed, 11])))
    R, C = wl.n_routed, wl.C
    return {
        "L": rng.standard_normal((R, C), dtype=np.float32),
        "Wh": (rng.standard_normal((d, C), dtype=np.float32) * np.float32(2.0 / np.sqrt(C))).astype(np.float32),
        "bh": (rng.standard_normal(d, dtype=np.float32) * np.float32(0.1)).astype(np.float32),
        "v": rng.standard_normal((C, d), dtype=np.float32),
        "q": (rng.standard_normal((R, d), dtype=np.float32) * np.float32(1.0 / np.sqrt(d))).astype(np.float32),
    }


def random_descriptor(B: int, C: int, seed: int, signed: bool = False) -> np.ndarray:
    """A synthetic per-(image, channel) descriptor for testing the gate alone."""
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, 7])))
    d = rng.standard_normal((B, C), dtype=np.float32) * np.float32(0.5)
    if not signed:
        d = np.abs(d)
    return d.astype(np.float32)
