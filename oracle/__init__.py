"""CPU reference ("oracle") for the MoCE forward pass.

TEST INFRASTRUCTURE ONLY.  Only the test suite, ``__graft_entry__.smoke()`` and
the benchmark's CPU-baseline leg may import this package.  The HIP library and
its Python binding never import it, and it never imports them.

The forward arithmetic lives in ``moce_oracle.c`` (plain double-precision loops);
this module only compiles that file and marshals numpy arrays through ctypes.
The gradients (``backward.py``) are plain float64 numpy, pinned by finite
differences through the C forward.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from typing import Dict, Optional

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "moce_oracle.c")
_LIB_PATH = os.path.join(_HERE, "libmoce_oracle.so")
_lib = None

NCHW, NHWC = 0, 1
F32, BF16 = 0, 1


class SupportError(ValueError):
    def __init__(self, expert: int):
        super().__init__(f"invalid support row for routed expert {expert}")
        self.expert = expert


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (-O2, OpenMP over images, no intrinsics)."""
    if force or not os.path.exists(_LIB_PATH):
        tmp = _LIB_PATH + ".tmp"
        subprocess.check_call(["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-std=c99",
                               "-Wall", "-o", tmp, _SRC, "-lm"])
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            build(force=True)
        lib = ctypes.CDLL(_LIB_PATH)
        P = ctypes.c_void_p
        I = ctypes.c_int
        lib.moce_oracle_prepare.argtypes = [I, I, I, P, P, P, P, P, P, P]
        lib.moce_oracle_prepare.restype = I
        lib.moce_oracle_pool.argtypes = [I, I, I, I, I, P, P]
        lib.moce_oracle_gate_softplus.argtypes = [I, I, I, I, P, P, P, P, P]
        lib.moce_oracle_gate_mlp.argtypes = [I, I, I, I, P, P, P, P, P, ctypes.c_float,
                                             ctypes.c_float, ctypes.c_float, P]
        lib.moce_oracle_softmax.argtypes = [I, I, I, P, P, P]
        lib.moce_oracle_mix.argtypes = [I, I, I, I, I, I, I, P, P, P, P, I, P, P]
        lib.moce_oracle_router.argtypes = [I, I, I, P, P, P, P]
        lib.moce_oracle_dynamic_logits.argtypes = [I, I, I, I, P, P, P, P, P]
        lib.moce_oracle_topk.argtypes = [I, I, I, P, P, P]
        lib.moce_oracle_dynamic_uncovered.argtypes = [I, I, I, I, P, P, P]
        lib.moce_oracle_threads.restype = I
        lib.moce_oracle_set_threads.argtypes = [I]
        _lib = lib
    return _lib


def _ptr(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p)


def _c(a, dtype) -> np.ndarray:
    return np.ascontiguousarray(a, dtype=dtype)


def threads() -> int:
    return _load().moce_oracle_threads()


def set_threads(n: int) -> None:
    """Sets the OpenMP thread count of the oracle's loops (results do not depend on it)."""
    _load().moce_oracle_set_threads(int(n))


def prepare(C: int, E: int, s: np.ndarray, w: np.ndarray):
    """Canonical supports, coverage mask and uncovered set.

    Returns ``(s_canon, w_canon, covered, U, nU)``.  Raises ``SupportError``
    naming the first invalid routed expert, ``ValueError`` for a bad shape.
    """
    s = _c(s, np.int32)
    w = _c(w, np.float32)
    if s.ndim != 2 or s.shape != w.shape or s.shape[0] != max(E - 1, 0):
        raise ValueError(f"s and w must both be [E-1, k]; got {s.shape}, {w.shape}, E={E}")
    k = s.shape[1]
    s_out = np.zeros_like(s)
    w_out = np.zeros_like(w)
    covered = np.zeros(max(C, 1), np.uint8)
    U = np.zeros(max(C, 1), np.int32)
    nU = np.zeros(1, np.int32)
    r = _load().moce_oracle_prepare(C, E, k, _ptr(s), _ptr(w), _ptr(s_out), _ptr(w_out),
                                    _ptr(covered), _ptr(U), _ptr(nU))
    if r == -2:
        raise ValueError(f"invalid shape C={C} E={E} k={k}")
    if r >= 0:
        raise SupportError(r)
    n = int(nU[0])
    return s_out, w_out, covered[:C], U[:n].copy(), n


def _layout_dims(x: np.ndarray, layout: int):
    if layout == NCHW:
        B, C = x.shape[0], x.shape[1]
        HW = int(np.prod(x.shape[2:]))
    else:
        B, C = x.shape[0], x.shape[-1]
        HW = int(np.prod(x.shape[1:-1]))
    return B, C, HW


def _elem(x: np.ndarray) -> int:
    if x.dtype == np.float32:
        return F32
    if x.dtype == np.uint16:
        return BF16
    raise TypeError(f"x must be float32 or uint16 bf16 bits, got {x.dtype}")


def pool(x: np.ndarray, layout: int = NCHW) -> np.ndarray:
    """Descriptor ``d[B, C]`` (float64)."""
    x = np.ascontiguousarray(x)
    B, C, HW = _layout_dims(x, layout)
    d = np.zeros((B, C), np.float64)
    _load().moce_oracle_pool(B, C, HW, layout, _elem(x), _ptr(x), _ptr(d))
    return d


def gate_softplus(d: np.ndarray, s_canon: np.ndarray, a: np.ndarray, c: np.ndarray) -> np.ndarray:
    d = _c(d, np.float64)
    s_canon = _c(s_canon, np.int32)
    a = _c(a, np.float32)
    c = _c(c, np.float32)
    B, C = d.shape
    R, k = s_canon.shape
    tau = np.zeros((B, R), np.float64)
    _load().moce_oracle_gate_softplus(B, C, R + 1, k, _ptr(d), _ptr(s_canon), _ptr(a), _ptr(c), _ptr(tau))
    return tau


def gate_mlp(d: np.ndarray, s_canon: np.ndarray, W1, b1, w2, b2, tau_min, tau_max) -> np.ndarray:
    d = _c(d, np.float64)
    s_canon = _c(s_canon, np.int32)
    W1 = _c(W1, np.float32)
    b1 = _c(b1, np.float32)
    w2 = _c(w2, np.float32)
    B, C = d.shape
    R, k = s_canon.shape
    tau = np.zeros((B, R), np.float64)
    _load().moce_oracle_gate_mlp(B, C, R + 1, k, _ptr(d), _ptr(s_canon), _ptr(W1), _ptr(b1), _ptr(w2),
                                 float(b2), float(tau_min), float(tau_max), _ptr(tau))
    return tau


def softmax(w_canon: np.ndarray, tau: np.ndarray) -> np.ndarray:
    w_canon = _c(w_canon, np.float32)
    tau = _c(tau, np.float64)
    R, k = w_canon.shape
    B = tau.shape[0]
    alpha = np.zeros((B, R, k), np.float64)
    _load().moce_oracle_softmax(B, R + 1, k, _ptr(w_canon), _ptr(tau), _ptr(alpha))
    return alpha


def mix(x: np.ndarray, s_canon: np.ndarray, alpha: np.ndarray, U: np.ndarray, E: int,
        layout: int = NCHW):
    """Returns ``(y, mag)`` in the layout of ``x`` with ``E`` channels (float64)."""
    x = np.ascontiguousarray(x)
    s_canon = _c(s_canon, np.int32)
    alpha = _c(alpha, np.float64)
    nU = int(len(U))
    U = _c(U, np.int32) if nU else np.zeros(1, np.int32)
    B, C, HW = _layout_dims(x, layout)
    k = s_canon.shape[1] if s_canon.ndim == 2 else 1
    if layout == NCHW:
        yshape = (B, E) + x.shape[2:]
    else:
        yshape = x.shape[:-1] + (E,)
    y = np.zeros(yshape, np.float64)
    mag = np.zeros(yshape, np.float64)
    _load().moce_oracle_mix(B, C, E, k, HW, layout, _elem(x), _ptr(x), _ptr(s_canon), _ptr(alpha),
                            _ptr(U), nU, _ptr(y), _ptr(mag))
    return y, mag


def forward(x: np.ndarray, s: np.ndarray, w: np.ndarray, E: int, layout: int = NCHW,
            gate: str = "softplus", a=None, c=None, W1=None, b1=None, w2=None, b2=0.0,
            tau_min=0.2, tau_max=6.0) -> Dict[str, np.ndarray]:
    """The whole layer: prepare, pool, temperature, softmax, mix and residual."""
    x = np.ascontiguousarray(x)
    _, C, _ = _layout_dims(x, layout)
    s_c, w_c, covered, U, nU = prepare(C, E, s, w)
    d = pool(x, layout)
    if gate == "softplus":
        tau = gate_softplus(d, s_c, a, c)
    elif gate == "mlp":
        tau = gate_mlp(d, s_c, W1, b1, w2, b2, tau_min, tau_max)
    else:
        raise ValueError(gate)
    alpha = softmax(w_c, tau)
    y, mag = mix(x, s_c, alpha, U, E, layout)
    return {"s": s_c, "w": w_c, "covered": covered, "U": U, "nU": nU, "d": d, "tau": tau,
            "alpha": alpha, "y": y, "mag": mag}


def epilogue(y: np.ndarray, scale, shift, relu: bool, layout: int = NCHW) -> np.ndarray:
    """The output epilogue of the replaced projection's block (Sec. 4.1: batch normalisation and the
    block's nonlinearity follow the layer): per output channel o, act(scale[o] y + shift[o]) with act
    = ReLU when ``relu``, in float64 on top of ``y`` (the layer's output, channel axis 1 for NCHW and
    last for channels-last).  ``scale`` None means no affine map."""
    y = np.asarray(y, np.float64)
    if scale is not None:
        sh = [1] * y.ndim
        ax = 1 if layout == NCHW else y.ndim - 1
        sh[ax] = -1
        y = y * np.asarray(scale, np.float64).reshape(sh) + np.asarray(shift, np.float64).reshape(sh)
    if relu:
        y = np.maximum(y, 0.0)
    return y


# ---------------------------------------------------------------------------
# Input-conditioned (dynamic) support, Sec. 4.5 Eq. 11

def router(d: np.ndarray, Wh, bh) -> np.ndarray:
    """The router's bottleneck h = ReLU(Wh d + bh) per example, [B, dd] (float64)."""
    d = _c(d, np.float64)
    Wh = _c(Wh, np.float32)
    bh = _c(bh, np.float32)
    B, C = d.shape
    dd = Wh.shape[0]
    h = np.zeros((B, dd), np.float64)
    _load().moce_oracle_router(B, C, dd, _ptr(d), _ptr(Wh), _ptr(bh), _ptr(h))
    return h


def dynamic_logits(h: np.ndarray, L, q, v) -> np.ndarray:
    """Per-example routing logits L(X)[b, e, c] = L[e, c] + <q_e * h_b, v_c>, [B, E-1, C]."""
    h = _c(h, np.float64)
    L = _c(L, np.float32)
    q = _c(q, np.float32)
    v = _c(v, np.float32)
    B, dd = h.shape
    R, C = L.shape
    Lx = np.zeros((B, R, C), np.float64)
    _load().moce_oracle_dynamic_logits(B, C, R, dd, _ptr(h), _ptr(L), _ptr(q), _ptr(v), _ptr(Lx))
    return Lx


def topk(Lx: np.ndarray, k: int):
    """The k largest entries of each row of the last axis, ties to the lower
    channel, in canonical order: ``(S, W)`` with S the channels (int32) and W
    their values."""
    Lx = _c(Lx, np.float64)
    C = Lx.shape[-1]
    rows = int(np.prod(Lx.shape[:-1]))
    S = np.zeros(Lx.shape[:-1] + (k,), np.int32)
    W = np.zeros(Lx.shape[:-1] + (k,), np.float64)
    _load().moce_oracle_topk(rows, C, k, _ptr(Lx), _ptr(S), _ptr(W))
    return S, W


def dynamic_uncovered(S: np.ndarray, C: int):
    """Per example the channels in none of its supports: a list of B ascending arrays."""
    S = _c(S, np.int32)
    B, R, k = S.shape
    U = np.zeros((B, max(C, 1)), np.int32)
    nU = np.zeros(B, np.int32)
    _load().moce_oracle_dynamic_uncovered(B, C, R, k, _ptr(S), _ptr(U), _ptr(nU))
    return [U[b, :nU[b]].copy() for b in range(B)]


def dynamic_forward(x: np.ndarray, L, Wh, bh, v, q, k: int, E: int, layout: int = NCHW,
                    gate: str = "softplus", a=None, c=None, W1=None, b1=None, w2=None, b2=0.0,
                    tau_min=0.2, tau_max=6.0, S=None, W=None) -> Dict[str, np.ndarray]:
    """The layer with input-conditioned supports: GAP, router, per-example
    logits, per-example TopK, and then per example the static layer's
    temperature (from z at that example's support), softmax over the
    example's logits at its support, mix and residual over U(X).

    ``S``/``W`` (optional, [B, E-1, k]) replace the selection by a given one,
    in canonical order, for checking a device selection that differs from this
    one only on ties and near-ties."""
    x = np.ascontiguousarray(x)
    B, C, _ = _layout_dims(x, layout)
    d = pool(x, layout)
    h = router(d, Wh, bh)
    Lx = dynamic_logits(h, L, q, v)
    S_ref, W_ref = topk(Lx, k)
    if S is None:
        S, W = S_ref, W_ref
    Ulist = dynamic_uncovered(S, C)
    R = E - 1
    yshape = (B, E) + x.shape[2:] if layout == NCHW else x.shape[:-1] + (E,)
    y = np.zeros(yshape, np.float64)
    mag = np.zeros(yshape, np.float64)
    tau = np.zeros((B, R), np.float64)
    alpha = np.zeros((B, R, k), np.float64)
    for b in range(B):
        db = d[b:b + 1]
        if gate == "softplus":
            tb = gate_softplus(db, S[b], a, c)
        elif gate == "mlp":
            tb = gate_mlp(db, S[b], W1, b1, w2, b2, tau_min, tau_max)
        else:
            raise ValueError(gate)
        ab = softmax(W[b].astype(np.float32), tb)
        yb, mb = mix(x[b:b + 1], S[b], ab, Ulist[b], E, layout)
        y[b], mag[b], tau[b], alpha[b] = yb[0], mb[0], tb[0], ab[0]
    return {"d": d, "h": h, "Lx": Lx, "S": S, "W": W, "S_ref": S_ref, "W_ref": W_ref, "U": Ulist,
            "tau": tau, "alpha": alpha, "y": y, "mag": mag}
