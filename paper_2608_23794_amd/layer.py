"""A MoCE layer held on the GPU, driven through the C ABI.

``MoceLayer`` owns the device copies of a layer's parameters (support rows,
selected logits, gate parameters), prepares the supports once with
``moce_support_prepare`` and then forwards batches with ``moce_forward`` or
the individual ``moce_pool`` / ``moce_gate`` / ``moce_mix`` calls.  Torch
provides device memory and the current stream; every step of the layer runs in
libmoce's HIP kernels.
"""
from __future__ import annotations

from typing import Optional

import numpy as np
import torch

from . import binding as mb

_DT = {"f32": mb.MOCE_F32, "bf16": mb.MOCE_BF16}
_LAYOUT = {"nchw": mb.MOCE_NCHW, "nhwc": mb.MOCE_NHWC}
_TORCH_DT = {"f32": torch.float32, "bf16": torch.bfloat16}


def _dev(a, dtype, device) -> torch.Tensor:
    return torch.as_tensor(np.ascontiguousarray(a), dtype=dtype).to(device)


class MoceLayer:
    def __init__(self, C: int, E: int, k: int, H: int, W: int, dtype: str, layout: str,
                 s: np.ndarray, w: np.ndarray, gate: str = "softplus", a=None, c=None,
                 W1=None, b1=None, w2=None, b2: float = 0.0, tau_min: float = 0.2, tau_max: float = 6.0,
                 device: str = "cuda", allow_invalid: bool = False):
        self.C, self.E, self.k, self.H, self.W = C, E, k, H, W
        self.R = E - 1
        self.dtype, self.layout, self.device = dtype, layout, device
        i32, f32 = torch.int32, torch.float32
        R = self.R
        self.s = _dev(np.asarray(s, np.int32).reshape(R, k), i32, device)
        self.w = _dev(np.asarray(w, np.float32).reshape(R, k), f32, device)
        self.s_c = torch.empty((R, k), dtype=i32, device=device)
        self.w_c = torch.empty((R, k), dtype=f32, device=device)
        self.covered = torch.empty(C, dtype=torch.uint8, device=device)
        self.U = torch.empty(C, dtype=i32, device=device)
        self.info = torch.empty(2, dtype=i32, device=device)
        self._keep = []
        if gate == "softplus":
            self.a = _dev(np.asarray(a, np.float32).reshape(R, k), f32, device)
            self.c = _dev(np.asarray(c, np.float32).reshape(R), f32, device)
            self.gate = mb.make_gate(mb.MOCE_GATE_SOFTPLUS_LINEAR, a=self.a, c=self.c)
        elif gate == "mlp":
            self.W1 = _dev(np.asarray(W1, np.float32).reshape(k, k), f32, device)
            self.b1 = _dev(np.asarray(b1, np.float32).reshape(k), f32, device)
            self.w2 = _dev(np.asarray(w2, np.float32).reshape(k), f32, device)
            self.gate = mb.make_gate(mb.MOCE_GATE_MLP_SIGMOID, W1=self.W1, b1=self.b1, w2=self.w2,
                                     b2=float(b2), tau_min=float(tau_min), tau_max=float(tau_max))
        else:
            raise ValueError(gate)
        self.status, self.nU, self.bad_expert = self.prepare(check=False)
        # A failed preparation leaves s_c and U unspecified (channels may lie
        # outside [0, C)), and the kernels do not validate indices.  Such a
        # layer is only kept for inspecting the status (allow_invalid=True),
        # and every entry method below refuses to run on it.
        if self.status != 0 and not allow_invalid:
            raise mb.MoceError("moce_support_prepare", self.status, f"(first bad expert {self.bad_expert})")

    # -- construction helpers ------------------------------------------------
    @classmethod
    def from_workload(cls, wl, params: dict, layout: Optional[str] = None, gate: str = "softplus",
                      device: str = "cuda") -> "MoceLayer":
        return cls(wl.C, wl.E, wl.k, wl.H, wl.W, wl.dtype, layout or wl.layouts[0], params["s"], params["w"],
                   gate=gate, a=params.get("a"), c=params.get("c"), W1=params.get("W1"),
                   b1=params.get("b1"), w2=params.get("w2"), b2=float(params.get("b2", 0.0)),
                   tau_min=float(params.get("tau_min", 0.2)), tau_max=float(params.get("tau_max", 6.0)),
                   device=device)

    def desc(self, B: int) -> mb.moce_desc:
        return mb.make_desc(B, self.C, self.H, self.W, self.E, self.k, _DT[self.dtype], _LAYOUT[self.layout])

    @property
    def torch_dtype(self):
        return _TORCH_DT[self.dtype]

    def y_shape(self, B: int):
        return (B, self.E, self.H, self.W) if self.layout == "nchw" else (B, self.H, self.W, self.E)

    def _stream(self):
        return torch.cuda.current_stream(self.device)

    def _ready(self):
        if self.status != 0:
            raise mb.MoceError("MoceLayer", self.status, "(support preparation failed; the layer cannot run)")

    # -- the C ABI -------------------------------------------------------------
    def prepare(self, check: bool = True):
        return mb.moce_support_prepare(self.desc(1), self.s, self.w, self.s_c, self.w_c, self.covered, self.U,
                                       self.info, self._stream(), check=check)

    def pool(self, x: torch.Tensor, d: Optional[torch.Tensor] = None) -> torch.Tensor:
        self._ready()
        B = x.shape[0]
        if d is None:
            d = torch.empty((B, self.C), dtype=torch.float32, device=self.device)
        mb.moce_pool(self.desc(B), x, d, self._stream())
        return d

    def gate_tau(self, d: torch.Tensor, with_alpha: bool = True):
        self._ready()
        B = d.shape[0]
        tau = torch.empty((B, self.R), dtype=torch.float32, device=self.device)
        alpha = torch.empty((B, self.R, self.k), dtype=torch.float32, device=self.device) if with_alpha else None
        mb.moce_gate(self.desc(B), d, self.s_c, self.w_c, self.gate, tau, alpha, self._stream())
        return tau, alpha

    def gate_mix(self, x: torch.Tensor, d: torch.Tensor, y: Optional[torch.Tensor] = None) -> torch.Tensor:
        """moce_gate_mix: temperatures, coefficients and mixing in one kernel from the pooled d."""
        self._ready()
        B = x.shape[0]
        if y is None:
            y = torch.empty(self.y_shape(B), dtype=x.dtype, device=self.device)
        mb.moce_gate_mix(self.desc(B), x, d, self.s_c, self.w_c, self.gate, self.U if self.nU else None, self.nU,
                         y, self._stream())
        return y

    def mix(self, x: torch.Tensor, alpha: torch.Tensor, y: Optional[torch.Tensor] = None) -> torch.Tensor:
        self._ready()
        B = x.shape[0]
        if y is None:
            y = torch.empty(self.y_shape(B), dtype=x.dtype, device=self.device)
        mb.moce_mix(self.desc(B), x, self.s_c, alpha, self.U if self.nU else None, self.nU, y, self._stream())
        return y

    def workspace_bytes(self, B: int) -> int:
        return mb.moce_forward_workspace_bytes(self.desc(B))

    def new_workspace(self, B: int) -> torch.Tensor:
        return torch.empty(max(self.workspace_bytes(B), 1), dtype=torch.uint8, device=self.device)

    def forward(self, x: torch.Tensor, y: Optional[torch.Tensor] = None,
                ws: Optional[torch.Tensor] = None, epilogue=None) -> torch.Tensor:
        """moce_forward, or with epilogue = (scale, shift, relu) moce_forward_ex (scale and shift: device
        float32 [E] or both None)."""
        self._ready()
        B = x.shape[0]
        if y is None:
            y = torch.empty(self.y_shape(B), dtype=x.dtype, device=self.device)
        if ws is None:
            ws = self.new_workspace(B)
        if epilogue is None:
            mb.moce_forward(self.desc(B), x, self.s_c, self.w_c, self.gate, self.U if self.nU else None, self.nU,
                            y, ws, ws.numel(), self._stream())
        else:
            scale, shift, relu = epilogue
            ep = mb.make_epilogue(scale, shift, relu)
            mb.moce_forward_ex(self.desc(B), x, self.s_c, self.w_c, self.gate, self.U if self.nU else None,
                               self.nU, ep, y, ws, ws.numel(), self._stream())
        return y

    # -- backward --------------------------------------------------------------
    def backward_workspace_bytes(self, B: int) -> int:
        return mb.moce_backward_workspace_bytes(self.desc(B), self.gate.kind)

    def new_backward_workspace(self, B: int) -> torch.Tensor:
        n = self.backward_workspace_bytes(B)
        if n == 0:
            raise mb.MoceError("moce_backward_workspace_bytes", -10, "(shape beyond the backward's limits)")
        return torch.empty(n, dtype=torch.uint8, device=self.device)

    def backward(self, x: torch.Tensor, dy: torch.Tensor, dx: Optional[torch.Tensor] = None,
                 ws: Optional[torch.Tensor] = None) -> dict:
        """moce_backward: dx, dw [E-1][k] (prepared rows) and the gate's parameter gradients."""
        self._ready()
        B = x.shape[0]
        f32, dev = torch.float32, self.device
        if dx is None:
            dx = torch.empty_like(x)
        if ws is None:
            ws = self.new_backward_workspace(B)
        R, k = self.R, self.k
        out = {"dx": dx, "dw": torch.empty((R, k), dtype=f32, device=dev)}
        if self.gate.kind == mb.MOCE_GATE_SOFTPLUS_LINEAR:
            out["da"] = torch.empty((R, k), dtype=f32, device=dev)
            out["dc"] = torch.empty(max(R, 1), dtype=f32, device=dev)
            grads = mb.make_gate_grads(da=out["da"], dc=out["dc"])
        else:
            out["dW1"] = torch.empty((k, k), dtype=f32, device=dev)
            out["db1"] = torch.empty(k, dtype=f32, device=dev)
            out["dw2"] = torch.empty(k, dtype=f32, device=dev)
            out["db2"] = torch.empty(1, dtype=f32, device=dev)
            grads = mb.make_gate_grads(dW1=out["dW1"], db1=out["db1"], dw2=out["dw2"], db2=out["db2"])
        mb.moce_backward(self.desc(B), x, dy, self.s_c, self.w_c, self.gate, dx, out["dw"], grads, ws, ws.numel(),
                         self._stream())
        return out

    def logit_backward(self, L: torch.Tensor, dw: Optional[torch.Tensor], eps: float, lam: float):
        """moce_logit_backward over the full logits L [E-1][C]: (loss, dL)."""
        R, C = self.R, self.C
        n = mb.moce_logit_backward_workspace_bytes(R, C)
        ws = torch.empty(max(n, 1), dtype=torch.uint8, device=self.device)
        loss = torch.empty(1, dtype=torch.float32, device=self.device)
        dL = torch.empty((R, C), dtype=torch.float32, device=self.device)
        mb.moce_logit_backward(R, C, self.k, L, self.s_c if dw is not None else None, dw, eps, lam, loss, dL, ws, n,
                               self._stream())
        return loss, dL


class DynamicMoceLayer:
    """The layer with input-conditioned supports (Sec. 4.5 Eq. 11): device
    copies of the full routing logits, the router and the gate, and the
    library's dynamic forward over them."""

    def __init__(self, C: int, E: int, k: int, H: int, W: int, dtype: str, layout: str, L, Wh, bh, v, q,
                 gate: str = "softplus", a=None, c=None, W1=None, b1=None, w2=None, b2: float = 0.0,
                 tau_min: float = 0.2, tau_max: float = 6.0, device: str = "cuda"):
        self.C, self.E, self.k, self.H, self.W = C, E, k, H, W
        self.R = R = E - 1
        self.dtype, self.layout, self.device = dtype, layout, device
        f32 = torch.float32
        self.dd = int(np.asarray(Wh).shape[0])
        self.L = _dev(np.asarray(L, np.float32).reshape(R, C), f32, device)
        self.Wh = _dev(np.asarray(Wh, np.float32).reshape(self.dd, C), f32, device)
        self.bh = _dev(np.asarray(bh, np.float32).reshape(self.dd), f32, device)
        self.v = _dev(np.asarray(v, np.float32).reshape(C, self.dd), f32, device)
        self.q = _dev(np.asarray(q, np.float32).reshape(R, self.dd), f32, device)
        self.router = mb.make_router(self.dd, self.Wh, self.bh, self.v, self.q)
        if gate == "softplus":
            self.a = _dev(np.asarray(a, np.float32).reshape(R, k), f32, device)
            self.c = _dev(np.asarray(c, np.float32).reshape(R), f32, device)
            self.gate = mb.make_gate(mb.MOCE_GATE_SOFTPLUS_LINEAR, a=self.a, c=self.c)
        elif gate == "mlp":
            self.W1 = _dev(np.asarray(W1, np.float32).reshape(k, k), f32, device)
            self.b1 = _dev(np.asarray(b1, np.float32).reshape(k), f32, device)
            self.w2 = _dev(np.asarray(w2, np.float32).reshape(k), f32, device)
            self.gate = mb.make_gate(mb.MOCE_GATE_MLP_SIGMOID, W1=self.W1, b1=self.b1, w2=self.w2,
                                     b2=float(b2), tau_min=float(tau_min), tau_max=float(tau_max))
        else:
            raise ValueError(gate)

    @classmethod
    def from_workload(cls, wl, params: dict, router: dict, layout: Optional[str] = None, gate: str = "softplus",
                      device: str = "cuda") -> "DynamicMoceLayer":
        return cls(wl.C, wl.E, wl.k, wl.H, wl.W, wl.dtype, layout or wl.layouts[0], router["L"], router["Wh"],
                   router["bh"], router["v"], router["q"], gate=gate, a=params.get("a"), c=params.get("c"),
                   W1=params.get("W1"), b1=params.get("b1"), w2=params.get("w2"), b2=float(params.get("b2", 0.0)),
                   tau_min=float(params.get("tau_min", 0.2)), tau_max=float(params.get("tau_max", 6.0)),
                   device=device)

    def desc(self, B: int) -> mb.moce_desc:
        return mb.make_desc(B, self.C, self.H, self.W, self.E, self.k, _DT[self.dtype], _LAYOUT[self.layout])

    def y_shape(self, B: int):
        return (B, self.E, self.H, self.W) if self.layout == "nchw" else (B, self.H, self.W, self.E)

    def workspace_bytes(self, B: int) -> int:
        return mb.moce_forward_dynamic_workspace_bytes(self.desc(B), self.dd)

    def new_workspace(self, B: int) -> torch.Tensor:
        return torch.empty(max(self.workspace_bytes(B), 1), dtype=torch.uint8, device=self.device)

    def forward(self, x: torch.Tensor, y: Optional[torch.Tensor] = None, ws: Optional[torch.Tensor] = None,
                S_out: Optional[torch.Tensor] = None) -> torch.Tensor:
        B = x.shape[0]
        if y is None:
            y = torch.empty(self.y_shape(B), dtype=x.dtype, device=self.device)
        if ws is None:
            ws = self.new_workspace(B)
        mb.moce_forward_dynamic(self.desc(B), x, self.L, self.router, self.gate, y, S_out, ws, ws.numel(),
                                torch.cuda.current_stream())
        return y


def to_device_x(x: np.ndarray, dtype: str, device: str = "cuda") -> torch.Tensor:
    """Uploads f32 values or bf16 bit patterns (uint16) as a float32/bfloat16 tensor."""
    if dtype == "f32":
        return torch.from_numpy(np.ascontiguousarray(x, np.float32)).to(device)
    bits = np.ascontiguousarray(x, np.uint16).view(np.int16)
    return torch.from_numpy(bits).to(device).view(torch.bfloat16)


def to_host_f64(y: torch.Tensor) -> np.ndarray:
    """Exact float64 copy of a float32 or bfloat16 device tensor."""
    return y.float().cpu().numpy().astype(np.float64)
