"""ctypes binding of libmoce.so, the C ABI declared in include/moce.h.

Argument marshalling only: every function forwards to the C entry point of
the same name.  Array arguments are device pointers given as ints or as
objects with a ``data_ptr()`` method (torch tensors); ``stream`` is a
``hipStream_t`` as an int (0 = the null stream) or a torch stream.  A non-OK
status raises ``MoceError``.  There is no CPU fallback: if the library is not
built, loading fails with an error naming the build step.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Tuple

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libmoce.so")

MOCE_F32, MOCE_BF16 = 0, 1
MOCE_NCHW, MOCE_NHWC = 0, 1
MOCE_GATE_SOFTPLUS_LINEAR, MOCE_GATE_MLP_SIGMOID = 0, 1

STATUS = {
    0: "MOCE_OK", -1: "MOCE_ERR_NULL", -2: "MOCE_ERR_SHAPE", -3: "MOCE_ERR_DTYPE",
    -4: "MOCE_ERR_LAYOUT", -5: "MOCE_ERR_SUPPORT", -6: "MOCE_ERR_GATE", -7: "MOCE_ERR_WORKSPACE",
    -8: "MOCE_ERR_ALIGN", -9: "MOCE_ERR_DEVICE", -10: "MOCE_ERR_UNSUPPORTED",
}

# Every function include/moce.h declares, in declaration order.
ENTRY_POINTS = (
    "moce_support_prepare", "moce_support_prepare16", "moce_pool", "moce_gate", "moce_gate_mix", "moce_mix",
    "moce_forward_workspace_bytes", "moce_forward_path", "moce_forward", "moce_forward_ex", "moce_forward_static",
    "moce_forward_dynamic_workspace_bytes", "moce_forward_dynamic", "moce_backward_workspace_bytes",
    "moce_backward", "moce_logit_backward_workspace_bytes", "moce_logit_backward", "moce_status_str",
    "moce_abi_version",
)

MOCE_STATIC_SCRATCH_BYTES = 16 << 20


class MoceError(RuntimeError):
    def __init__(self, fn: str, status: int, detail: str = ""):
        self.status = status
        name = STATUS.get(status, str(status))
        super().__init__(f"{fn} failed: {name}{(' ' + detail) if detail else ''}")


class moce_desc(ctypes.Structure):
    _fields_ = [("B", ctypes.c_int64), ("C", ctypes.c_int64), ("H", ctypes.c_int64), ("W", ctypes.c_int64),
                ("E", ctypes.c_int32), ("k", ctypes.c_int32), ("x_dtype", ctypes.c_int32),
                ("y_dtype", ctypes.c_int32), ("layout", ctypes.c_int32), ("reserved", ctypes.c_int32)]


class moce_router(ctypes.Structure):
    _fields_ = [("d", ctypes.c_int32), ("reserved", ctypes.c_int32), ("Wh", ctypes.c_void_p),
                ("bh", ctypes.c_void_p), ("v", ctypes.c_void_p), ("q", ctypes.c_void_p)]


class moce_gate_params(ctypes.Structure):
    _fields_ = [("kind", ctypes.c_int32), ("reserved", ctypes.c_int32),
                ("a", ctypes.c_void_p), ("c", ctypes.c_void_p), ("W1", ctypes.c_void_p),
                ("b1", ctypes.c_void_p), ("w2", ctypes.c_void_p),
                ("b2", ctypes.c_float), ("tau_min", ctypes.c_float), ("tau_max", ctypes.c_float)]


class moce_epilogue(ctypes.Structure):
    _fields_ = [("scale", ctypes.c_void_p), ("shift", ctypes.c_void_p), ("relu", ctypes.c_int32),
                ("reserved", ctypes.c_int32)]


class moce_gate_grads(ctypes.Structure):
    _fields_ = [("da", ctypes.c_void_p), ("dc", ctypes.c_void_p), ("dW1", ctypes.c_void_p),
                ("db1", ctypes.c_void_p), ("dw2", ctypes.c_void_p), ("db2", ctypes.c_void_p)]


_lib = None


def load(path: Optional[str] = None) -> ctypes.CDLL:
    """Loads libmoce.so (raises if it has not been built)."""
    global _lib
    if _lib is not None and path is None:
        return _lib
    p = path or LIB_PATH
    if not os.path.exists(p):
        raise RuntimeError(f"{p} is missing: build it with `python -m paper_2608_23794_amd.build` "
                           "(or __graft_entry__.build()); there is no fallback path")
    lib = ctypes.CDLL(p)
    P, I32, SZ = ctypes.c_void_p, ctypes.c_int32, ctypes.c_size_t
    D = ctypes.POINTER(moce_desc)
    G = ctypes.POINTER(moce_gate_params)
    IP = ctypes.POINTER(ctypes.c_int32)
    lib.moce_support_prepare.argtypes = [D, P, P, P, P, P, P, P, IP, IP, P]
    lib.moce_support_prepare16.argtypes = [D, P, P, P, P, P, P, P, IP, IP, P]
    lib.moce_pool.argtypes = [D, P, P, P]
    lib.moce_gate.argtypes = [D, P, P, P, G, P, P, P]
    lib.moce_gate_mix.argtypes = [D, P, P, P, P, G, P, I32, P, P]
    lib.moce_mix.argtypes = [D, P, P, P, P, I32, P, P]
    lib.moce_forward_workspace_bytes.argtypes = [D]
    lib.moce_forward_workspace_bytes.restype = SZ
    lib.moce_forward_path.argtypes = [D, ctypes.c_int]
    lib.moce_forward.argtypes = [D, P, P, P, G, P, I32, P, P, SZ, P]
    lib.moce_forward_ex.argtypes = [D, P, P, P, G, P, I32, ctypes.POINTER(moce_epilogue), P, P, SZ, P]
    lib.moce_forward_static.argtypes = [D, P, P, P, G, P, I32, P, P]
    lib.moce_forward_dynamic_workspace_bytes.argtypes = [D, I32]
    lib.moce_forward_dynamic_workspace_bytes.restype = SZ
    lib.moce_forward_dynamic.argtypes = [D, P, P, ctypes.POINTER(moce_router), G, P, P, P, SZ, P]
    lib.moce_backward_workspace_bytes.argtypes = [D, ctypes.c_int]
    lib.moce_backward_workspace_bytes.restype = SZ
    lib.moce_backward.argtypes = [D, P, P, P, P, G, P, P, ctypes.POINTER(moce_gate_grads), P, SZ, P]
    lib.moce_logit_backward_workspace_bytes.argtypes = [I32, ctypes.c_int64]
    lib.moce_logit_backward_workspace_bytes.restype = SZ
    lib.moce_logit_backward.argtypes = [I32, ctypes.c_int64, I32, P, P, P, ctypes.c_float, ctypes.c_float, P, P,
                                        P, SZ, P]
    lib.moce_status_str.argtypes = [ctypes.c_int]
    lib.moce_status_str.restype = ctypes.c_char_p
    lib.moce_abi_version.restype = ctypes.c_int
    for name in ("moce_support_prepare", "moce_support_prepare16", "moce_pool", "moce_gate", "moce_gate_mix", "moce_mix", "moce_forward", "moce_forward_ex",
                 "moce_forward_static", "moce_forward_dynamic", "moce_backward", "moce_logit_backward"):
        getattr(lib, name).restype = ctypes.c_int
    if path is None:
        _lib = lib
    return lib


def _ptr(a) -> Optional[int]:
    if a is None:
        return None
    if isinstance(a, int):
        return a
    return a.data_ptr()


def _stream(st) -> Optional[int]:
    if st is None or isinstance(st, int):
        return st or None
    return st.cuda_stream


def _check(fn: str, status: int):
    if status != 0:
        raise MoceError(fn, status)


def make_desc(B: int, C: int, H: int, W: int, E: int, k: int, dtype: int, layout: int) -> moce_desc:
    return moce_desc(B, C, H, W, E, k, dtype, dtype, layout, 0)


def make_gate(kind: int = MOCE_GATE_SOFTPLUS_LINEAR, a=None, c=None, W1=None, b1=None, w2=None,
              b2: float = 0.0, tau_min: float = 0.2, tau_max: float = 6.0) -> moce_gate_params:
    return moce_gate_params(kind, 0, _ptr(a), _ptr(c), _ptr(W1), _ptr(b1), _ptr(w2), b2, tau_min, tau_max)


def moce_abi_version() -> int:
    return load().moce_abi_version()


def moce_status_str(status: int) -> str:
    return load().moce_status_str(status).decode()


def moce_support_prepare(desc: moce_desc, s, w, s_out, w_out, covered, U, info, stream=None,
                         check: bool = True) -> Tuple[int, int, int]:
    """Returns (status, nU, bad_expert); raises on error unless check=False."""
    nU = ctypes.c_int32(-1)
    bad = ctypes.c_int32(-1)
    st = load().moce_support_prepare(ctypes.byref(desc), _ptr(s), _ptr(w), _ptr(s_out), _ptr(w_out),
                                     _ptr(covered), _ptr(U), _ptr(info), ctypes.byref(nU),
                                     ctypes.byref(bad), _stream(stream))
    if check and st != 0:
        raise MoceError("moce_support_prepare", st, f"(first bad expert {bad.value})")
    return st, nU.value, bad.value


def moce_support_prepare16(desc: moce_desc, s16, w, s_out, w_out, covered, U, info, stream=None,
                           check: bool = True) -> Tuple[int, int, int]:
    """moce_support_prepare from 16-bit supports; returns (status, nU, bad_expert)."""
    nU = ctypes.c_int32(-1)
    bad = ctypes.c_int32(-1)
    st = load().moce_support_prepare16(ctypes.byref(desc), _ptr(s16), _ptr(w), _ptr(s_out), _ptr(w_out),
                                       _ptr(covered), _ptr(U), _ptr(info), ctypes.byref(nU),
                                       ctypes.byref(bad), _stream(stream))
    if check and st != 0:
        raise MoceError("moce_support_prepare16", st, f"(first bad expert {bad.value})")
    return st, nU.value, bad.value


def moce_pool(desc: moce_desc, x, d, stream=None) -> None:
    _check("moce_pool", load().moce_pool(ctypes.byref(desc), _ptr(x), _ptr(d), _stream(stream)))


def moce_gate(desc: moce_desc, d, s, w, gate: moce_gate_params, tau, alpha=None, stream=None) -> None:
    _check("moce_gate", load().moce_gate(ctypes.byref(desc), _ptr(d), _ptr(s), _ptr(w), ctypes.byref(gate),
                                         _ptr(tau), _ptr(alpha), _stream(stream)))


def moce_gate_mix(desc: moce_desc, x, d, s, w, gate: moce_gate_params, U, nU: int, y, stream=None) -> None:
    _check("moce_gate_mix", load().moce_gate_mix(ctypes.byref(desc), _ptr(x), _ptr(d), _ptr(s), _ptr(w),
                                                 ctypes.byref(gate), _ptr(U), nU, _ptr(y), _stream(stream)))


def moce_mix(desc: moce_desc, x, s, alpha, U, nU: int, y, stream=None) -> None:
    _check("moce_mix", load().moce_mix(ctypes.byref(desc), _ptr(x), _ptr(s), _ptr(alpha), _ptr(U), nU,
                                       _ptr(y), _stream(stream)))


def moce_forward_workspace_bytes(desc: moce_desc) -> int:
    return int(load().moce_forward_workspace_bytes(ctypes.byref(desc)))


PATH_GENERIC, PATH_TILE, PATH_MFMA, PATH_MFMA_GATE, PATH_SCHEDULED, PATH_GATHER = 0, 1, 2, 3, 4, 5


def moce_forward_path(desc: moce_desc, gate_kind: int) -> int:
    """PATH_GATHER, PATH_SCHEDULED, PATH_MFMA_GATE, PATH_MFMA, PATH_TILE or PATH_GENERIC: the kernels
    moce_forward uses for desc
    (moce_mix: the same, PATH_MFMA for PATH_MFMA_GATE)."""
    r = int(load().moce_forward_path(ctypes.byref(desc), gate_kind))
    if r < 0:
        raise MoceError("moce_forward_path", r)
    return r


def moce_forward(desc: moce_desc, x, s, w, gate: moce_gate_params, U, nU: int, y, ws, ws_bytes: int,
                 stream=None) -> None:
    _check("moce_forward", load().moce_forward(ctypes.byref(desc), _ptr(x), _ptr(s), _ptr(w),
                                               ctypes.byref(gate), _ptr(U), nU, _ptr(y), _ptr(ws),
                                               ws_bytes, _stream(stream)))


def make_epilogue(scale=None, shift=None, relu: bool = False) -> moce_epilogue:
    """An epilogue struct over device arrays (they must outlive its use)."""
    return moce_epilogue(_ptr(scale), _ptr(shift), 1 if relu else 0, 0)


def moce_forward_ex(desc: moce_desc, x, s, w, gate: moce_gate_params, U, nU: int, ep: Optional[moce_epilogue], y, ws,
                    ws_bytes: int, stream=None) -> None:
    _check("moce_forward_ex", load().moce_forward_ex(ctypes.byref(desc), _ptr(x), _ptr(s), _ptr(w),
                                                     ctypes.byref(gate), _ptr(U), nU,
                                                     ctypes.byref(ep) if ep is not None else None, _ptr(y),
                                                     _ptr(ws), ws_bytes, _stream(stream)))


def moce_forward_static(desc: moce_desc, x, s, w, gate: moce_gate_params, U, nU: int, y, stream=None) -> None:
    _check("moce_forward_static", load().moce_forward_static(ctypes.byref(desc), _ptr(x), _ptr(s), _ptr(w),
                                                             ctypes.byref(gate), _ptr(U), nU, _ptr(y),
                                                             _stream(stream)))


def make_router(d: int, Wh, bh, v, q) -> moce_router:
    """A router struct over device arrays (they must outlive its use)."""
    return moce_router(int(d), 0, _ptr(Wh), _ptr(bh), _ptr(v), _ptr(q))


def moce_forward_dynamic_workspace_bytes(desc: moce_desc, d: int) -> int:
    return int(load().moce_forward_dynamic_workspace_bytes(ctypes.byref(desc), int(d)))


def moce_forward_dynamic(desc: moce_desc, x, L, router: moce_router, gate: moce_gate_params, y, S_out, ws,
                         ws_bytes: int, stream=None) -> None:
    _check("moce_forward_dynamic", load().moce_forward_dynamic(ctypes.byref(desc), _ptr(x), _ptr(L),
                                                               ctypes.byref(router), ctypes.byref(gate), _ptr(y),
                                                               _ptr(S_out), _ptr(ws), ws_bytes, _stream(stream)))


def make_gate_grads(da=None, dc=None, dW1=None, db1=None, dw2=None, db2=None) -> moce_gate_grads:
    """A gate-gradient struct over device arrays (they must outlive its use)."""
    return moce_gate_grads(_ptr(da), _ptr(dc), _ptr(dW1), _ptr(db1), _ptr(dw2), _ptr(db2))


def moce_backward_workspace_bytes(desc: moce_desc, gate_kind: int) -> int:
    return int(load().moce_backward_workspace_bytes(ctypes.byref(desc), int(gate_kind)))


def moce_backward(desc: moce_desc, x, dy, s, w, gate: moce_gate_params, dx, dw, grads: moce_gate_grads, ws,
                  ws_bytes: int, stream=None) -> None:
    _check("moce_backward", load().moce_backward(ctypes.byref(desc), _ptr(x), _ptr(dy), _ptr(s), _ptr(w),
                                                 ctypes.byref(gate), _ptr(dx), _ptr(dw), ctypes.byref(grads),
                                                 _ptr(ws), ws_bytes, _stream(stream)))


def moce_logit_backward_workspace_bytes(R: int, C: int) -> int:
    return int(load().moce_logit_backward_workspace_bytes(int(R), int(C)))


def moce_logit_backward(R: int, C: int, k: int, L, s, dw, eps: float, lam: float, loss, dL, ws, ws_bytes: int,
                        stream=None) -> None:
    _check("moce_logit_backward", load().moce_logit_backward(int(R), int(C), int(k), _ptr(L), _ptr(s), _ptr(dw),
                                                             float(eps), float(lam), _ptr(loss), _ptr(dL),
                                                             _ptr(ws), ws_bytes, _stream(stream)))


def raw_status(fn: str, *args) -> int:
    """Calls an entry point with raw ctypes arguments and returns its status
    (used to exercise host-side error paths)."""
    return getattr(load(), fn)(*args)
