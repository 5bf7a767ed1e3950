"""The C ABI library: it loads, exports every entry point include/moce.h
declares, and rejects invalid arguments on the host before any GPU work.

Every call here fails host-side validation, so nothing reaches the GPU; the
pointers are placeholders that are never dereferenced.
"""
import ctypes
import os
import re
import subprocess

import pytest

from paper_2608_23794_amd import binding as mb

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "moce.h")

FAKE = 0x10000  # 64 KiB-aligned placeholder address, never dereferenced
FAKE_UNALIGNED = 0x10008


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return re.findall(r"^[A-Za-z_][\w \*]*?\b(moce_\w+)\s*\(", text, flags=re.M)


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(mb.LIB_PATH):
        from paper_2608_23794_amd import build
        build.build()
    return mb.load()


def test_header_declares_the_binding_entry_points():
    assert sorted(declared_functions()) == sorted(mb.ENTRY_POINTS)


def test_library_exports_every_declared_symbol(lib):
    out = subprocess.run(["nm", "-D", "--defined-only", mb.LIB_PATH], capture_output=True, text=True,
                         check=True).stdout
    exported = set(re.findall(r"\b(moce_\w+)\b", out))
    for name in declared_functions():
        assert name in exported, name
        assert getattr(lib, name) is not None


def test_abi_version_and_status_strings(lib):
    assert mb.moce_abi_version() == 1
    for code, name in mb.STATUS.items():
        assert mb.moce_status_str(code).startswith(name)
    assert mb.moce_status_str(12345) == "unknown moce_status"


def good_desc(**kw):
    d = dict(B=2, C=64, H=8, W=8, E=16, k=8, dtype=mb.MOCE_BF16, layout=mb.MOCE_NCHW)
    d.update(kw)
    return mb.make_desc(d["B"], d["C"], d["H"], d["W"], d["E"], d["k"], d["dtype"], d["layout"])


BAD_DESCS = [
    (dict(B=0), -2),
    (dict(C=0), -2), (dict(H=0), -2), (dict(W=-1), -2),
    (dict(E=0), -2), (dict(E=65), -2), (dict(k=0), -2), (dict(k=65), -2),
    (dict(dtype=7), -3), (dict(layout=2), -4),
    (dict(H=1 << 31), -10), (dict(C=1 << 20, H=1 << 11, W=1 << 11), -10),
]


def _call_pool(desc, x=FAKE, d=FAKE):
    return mb.raw_status("moce_pool", ctypes.byref(desc), x, d, None)


def _call_mix(desc, x=FAKE, s=FAKE, alpha=FAKE, U=FAKE, nU=0, y=FAKE):
    return mb.raw_status("moce_mix", ctypes.byref(desc), x, s, alpha, U, nU, y, None)


def _call_gate(desc, gate, d=FAKE, s=FAKE, w=FAKE, tau=FAKE, alpha=FAKE):
    g = ctypes.byref(gate) if gate is not None else None
    return mb.raw_status("moce_gate", ctypes.byref(desc), d, s, w, g, tau, alpha, None)


def _call_forward(desc, gate, x=FAKE, s=FAKE, w=FAKE, U=FAKE, nU=0, y=FAKE, ws=FAKE, ws_bytes=1 << 30):
    g = ctypes.byref(gate) if gate is not None else None
    return mb.raw_status("moce_forward", ctypes.byref(desc), x, s, w, g, U, nU, y, ws, ws_bytes, None)


def _call_gate_mix(desc, gate, x=FAKE, d=FAKE, s=FAKE, w=FAKE, U=FAKE, nU=0, y=FAKE):
    g = ctypes.byref(gate) if gate is not None else None
    return mb.raw_status("moce_gate_mix", ctypes.byref(desc), x, d, s, w, g, U, nU, y, None)


def _call_prepare(desc, s=FAKE, w=FAKE, s_out=FAKE + 256, w_out=FAKE + 512, covered=FAKE, U=FAKE, info=FAKE,
                  nU=True, bad=True):
    n = ctypes.c_int32(0)
    b = ctypes.c_int32(0)
    return mb.raw_status("moce_support_prepare", ctypes.byref(desc), s, w, s_out, w_out, covered, U, info,
                         ctypes.byref(n) if nU else None, ctypes.byref(b) if bad else None, None)


@pytest.mark.parametrize("change,code", [(c, s) for c, s in BAD_DESCS])
def test_descriptor_errors_every_entry_point(lib, change, code):
    desc = good_desc(**change)
    gate = mb.make_gate(a=FAKE, c=FAKE)
    assert _call_pool(desc) == code
    assert _call_mix(desc) == code
    assert _call_gate(desc, gate) == code
    assert _call_forward(desc, gate) == code
    assert _call_prepare(desc) == code
    assert lib.moce_forward_workspace_bytes(ctypes.byref(desc)) == 0


def test_mismatched_x_and_y_types(lib):
    desc = good_desc()
    desc.y_dtype = mb.MOCE_F32
    assert _call_pool(desc) == -3


def test_null_descriptor(lib):
    assert mb.raw_status("moce_pool", None, FAKE, FAKE, None) == -1
    assert lib.moce_forward_workspace_bytes(None) == 0


def test_null_pointers(lib):
    desc = good_desc()
    gate = mb.make_gate(a=FAKE, c=FAKE)
    assert _call_pool(desc, x=None) == -1
    assert _call_pool(desc, d=None) == -1
    assert _call_mix(desc, x=None) == -1
    assert _call_mix(desc, s=None) == -1
    assert _call_mix(desc, alpha=None) == -1
    assert _call_mix(desc, y=None) == -1
    assert _call_mix(desc, U=None, nU=3) == -1
    assert _call_gate(desc, gate, d=None) == -1
    assert _call_gate(desc, gate, tau=None) == -1
    assert _call_gate(desc, None) == -1
    assert _call_gate(desc, mb.make_gate(a=None, c=FAKE)) == -1
    assert _call_gate(desc, mb.make_gate(mb.MOCE_GATE_MLP_SIGMOID, W1=None, b1=FAKE, w2=FAKE)) == -1
    assert _call_forward(desc, gate, x=None) == -1
    assert _call_forward(desc, gate, w=None) == -1
    assert _call_forward(desc, gate, U=None, nU=2) == -1
    assert _call_forward(desc, None) == -1
    assert _call_prepare(desc, covered=None) == -1
    assert _call_prepare(desc, info=None) == -1
    assert _call_prepare(desc, nU=False) == -1
    assert _call_prepare(desc, bad=False) == -1
    assert _call_prepare(desc, s_out=FAKE) == -1  # s_out aliases s


def test_alignment_and_residual_count(lib):
    desc = good_desc()
    gate = mb.make_gate(a=FAKE, c=FAKE)
    assert _call_pool(desc, x=FAKE_UNALIGNED) == -8
    assert _call_mix(desc, y=FAKE_UNALIGNED) == -8
    assert _call_forward(desc, gate, x=FAKE_UNALIGNED) == -8
    assert _call_forward(desc, gate, ws=FAKE + 64) == -8
    assert _call_mix(desc, nU=-1) == -2
    assert _call_mix(desc, nU=65) == -2
    assert _call_forward(desc, gate, nU=65) == -2


def test_gate_mix_errors(lib):
    """The one-kernel gate and mix: host-side checks, and only where the forward takes that path."""
    fused = good_desc(k=32)
    gate = mb.make_gate(a=FAKE, c=FAKE)
    assert lib.moce_forward_path(ctypes.byref(fused), mb.MOCE_GATE_SOFTPLUS_LINEAR) == mb.PATH_MFMA_GATE
    for change, code in BAD_DESCS:
        assert _call_gate_mix(good_desc(**{"k": 32, **change}), gate) == code
    assert _call_gate_mix(fused, None) == -1
    assert _call_gate_mix(fused, mb.make_gate(a=None, c=FAKE)) == -1
    assert _call_gate_mix(fused, mb.make_gate(kind=9, a=FAKE, c=FAKE)) == -6
    mlp = mb.make_gate(mb.MOCE_GATE_MLP_SIGMOID, W1=FAKE, b1=FAKE, w2=FAKE)
    assert lib.moce_forward_path(ctypes.byref(fused), mb.MOCE_GATE_MLP_SIGMOID) == mb.PATH_MFMA
    for desc, g in [(good_desc(k=8), gate), (fused, mlp), (good_desc(k=32, dtype=mb.MOCE_F32), gate),
                    (good_desc(k=32, layout=mb.MOCE_NHWC), gate), (good_desc(C=48, k=32), gate),
                    (good_desc(k=32, E=1), gate)]:
        assert _call_gate_mix(desc, g) == -10
        assert lib.moce_forward_path(ctypes.byref(desc), g.kind) != mb.PATH_MFMA_GATE
    for name in ("x", "d", "s", "w", "y"):
        assert _call_gate_mix(fused, gate, **{name: None}) == -1
    assert _call_gate_mix(fused, gate, U=None, nU=2) == -1
    assert _call_gate_mix(fused, gate, nU=65) == -2
    assert _call_gate_mix(fused, gate, nU=-1) == -2
    assert _call_gate_mix(fused, gate, x=FAKE_UNALIGNED) == -8
    assert _call_gate_mix(fused, gate, y=FAKE_UNALIGNED) == -8


def test_gate_parameter_errors(lib):
    desc = good_desc()
    assert _call_gate(desc, mb.make_gate(kind=9, a=FAKE, c=FAKE)) == -6
    mlp = dict(kind=mb.MOCE_GATE_MLP_SIGMOID, W1=FAKE, b1=FAKE, w2=FAKE)
    assert _call_gate(desc, mb.make_gate(**mlp, tau_min=0.0)) == -6
    assert _call_gate(desc, mb.make_gate(**mlp, tau_min=2.0, tau_max=1.0)) == -6
    assert _call_gate(desc, mb.make_gate(**mlp, tau_max=float("inf"))) == -6
    assert _call_gate(desc, mb.make_gate(**mlp, b2=float("nan"))) == -6
    big = good_desc(C=512, k=300)
    assert _call_gate(big, mb.make_gate(**mlp)) == -10


def test_workspace_size_and_errors(lib):
    desc = good_desc()
    need = lib.moce_forward_workspace_bytes(ctypes.byref(desc))
    # d [2][64] + tau [2][15] + softmax statistics [3][2][15] + alpha [2][15][8], each rounded up to 256 bytes
    assert need == 512 + 256 + 512 + 1024
    gate = mb.make_gate(a=FAKE, c=FAKE)
    assert _call_forward(desc, gate, ws=None) == -7
    assert _call_forward(desc, gate, ws_bytes=need - 1) == -7
    nhwc = good_desc(layout=mb.MOCE_NHWC)
    # bf16 channels-last with k <= 16 takes the gather: the coefficients as in the channels-first layout
    assert mb.moce_forward_path(nhwc, mb.MOCE_GATE_SOFTPLUS_LINEAR) == mb.PATH_GATHER
    assert lib.moce_forward_workspace_bytes(ctypes.byref(nhwc)) == 512 + 256 + 512 + 1024
    # with larger supports and C a multiple of 64 it takes the scheduled mix: no coefficients, but the support
    # schedule of one expert range with eight builder buckets (offsets [8][1 step + 1] in 256 bytes, entries
    # [8][2 * 16 k + C] of 8 bytes)
    nhwc = good_desc(layout=mb.MOCE_NHWC, k=24)
    assert mb.moce_forward_path(nhwc, mb.MOCE_GATE_SOFTPLUS_LINEAR) == mb.PATH_SCHEDULED
    assert lib.moce_forward_workspace_bytes(ctypes.byref(nhwc)) == 512 + 256 + 512 + 256 + 8 * (32 * 24 + 64) * 8
    f32 = good_desc(layout=mb.MOCE_NHWC, dtype=mb.MOCE_F32)
    assert lib.moce_forward_workspace_bytes(ctypes.byref(f32)) == 512 + 256 + 512


def test_prepare_limits(lib):
    assert _call_prepare(good_desc(C=1 << 25, H=1, W=1, E=2, k=4097)) == -10


def _call_static(desc, gate, x=FAKE, s=FAKE, w=FAKE, U=FAKE, nU=0, y=FAKE):
    g = ctypes.byref(gate) if gate is not None else None
    return mb.raw_status("moce_forward_static", ctypes.byref(desc), x, s, w, g, U, nU, y, None)


def test_forward_static_host_errors(lib):
    """The forward without a workspace argument: every host-side check runs before the library looks up
    its device array, including the size limit of that array."""
    gate = mb.make_gate(a=FAKE, c=FAKE)
    for change, code in BAD_DESCS:
        assert _call_static(good_desc(**change), gate) == code
    desc = good_desc()
    assert _call_static(desc, None) == -1
    assert _call_static(desc, gate, x=None) == -1
    assert _call_static(desc, gate, w=None) == -1
    assert _call_static(desc, gate, U=None, nU=2) == -1
    assert _call_static(desc, gate, nU=65) == -2
    assert _call_static(desc, gate, y=FAKE_UNALIGNED) == -8
    # a workspace beyond the array: B * R * k coefficients of 4 bytes alone exceed 16 MiB (H W = 2 keeps
    # the shape off the scheduled mix, which holds no coefficients)
    big = good_desc(B=64, C=4096, E=4096, k=64, H=1, W=2)
    assert lib.moce_forward_workspace_bytes(ctypes.byref(big)) > mb.MOCE_STATIC_SCRATCH_BYTES
    assert _call_static(big, gate) == -7


def _call_dynamic(desc, gate, router, x=FAKE, L=FAKE, y=FAKE, S_out=None, ws=FAKE, ws_bytes=1 << 30):
    r = ctypes.byref(router) if router is not None else None
    return mb.raw_status("moce_forward_dynamic", ctypes.byref(desc), x, L, r, ctypes.byref(gate), y, S_out, ws,
                         ws_bytes, None)


def test_forward_dynamic_host_errors(lib):
    """Every host-side check of the input-conditioned forward returns before any launch (all the
    addresses here are placeholders that are never dereferenced)."""
    desc = good_desc()
    gate = mb.make_gate(a=FAKE, c=FAKE)
    router = mb.moce_router(8, 0, FAKE, FAKE, FAKE, FAKE)
    assert _call_dynamic(desc, gate, None) == -1
    assert _call_dynamic(desc, gate, router, L=None) == -1
    assert _call_dynamic(desc, gate, mb.moce_router(8, 0, FAKE, None, FAKE, FAKE)) == -1
    assert _call_dynamic(desc, gate, mb.moce_router(0, 0, FAKE, FAKE, FAKE, FAKE)) == -2
    assert _call_dynamic(desc, gate, mb.moce_router(65, 0, FAKE, FAKE, FAKE, FAKE)) == -10
    assert _call_dynamic(good_desc(C=5000, k=8), gate, router) == -10
    assert _call_dynamic(good_desc(C=1024, k=600), gate, router) == -10
    assert _call_dynamic(desc, gate, router, x=FAKE_UNALIGNED) == -8
    assert _call_dynamic(desc, gate, router, ws=None) == -7
    need = lib.moce_forward_dynamic_workspace_bytes(ctypes.byref(desc), 8)
    assert need > 0
    assert _call_dynamic(desc, gate, router, ws_bytes=need - 1) == -7
    assert _call_dynamic(desc, gate, router, ws=FAKE_UNALIGNED, ws_bytes=need) == -8
    assert lib.moce_forward_dynamic_workspace_bytes(ctypes.byref(desc), 65) == 0


def test_forward_dynamic_workspace_layout(lib):
    """d [B][C], h [B][d], the transposed channel embeddings [d][C], supports and their logits
    [B][E-1][k], U [B][C], nU [B], tau [B][E-1] and the coefficients [B][E-1][k], each rounded up to
    256 bytes."""
    desc = good_desc()
    B, C, R, k, d = desc.B, desc.C, desc.E - 1, desc.k, 8
    r = lambda n: (n + 255) // 256 * 256
    expect = (r(B * C * 4) + r(B * d * 4) + r(d * C * 4) + 2 * r(B * R * k * 4) + r(B * C * 4) + r(B * 4)
              + r(B * R * 4) + r(B * R * k * 4))
    assert lib.moce_forward_dynamic_workspace_bytes(ctypes.byref(desc), d) == expect


def _call_backward(desc, gate, grads, x=FAKE, dy=FAKE, s=FAKE, w=FAKE, dx=FAKE, dw=FAKE, ws=FAKE,
                   ws_bytes=1 << 30):
    g = ctypes.byref(grads) if grads is not None else None
    return mb.raw_status("moce_backward", ctypes.byref(desc), x, dy, s, w, ctypes.byref(gate), dx, dw, g, ws,
                         ws_bytes, None)


def test_backward_host_errors(lib):
    """Every host-side check of the backward returns before any launch."""
    desc = good_desc()
    gate = mb.make_gate(a=FAKE, c=FAKE)
    grads = mb.moce_gate_grads(FAKE, FAKE, None, None, None, None)
    for kw, code in BAD_DESCS:
        assert _call_backward(good_desc(**kw), gate, grads) == code, kw
    assert _call_backward(desc, gate, None) == -1
    assert _call_backward(desc, gate, grads, dy=None) == -1
    assert _call_backward(desc, gate, grads, dx=None) == -1
    assert _call_backward(desc, gate, grads, dw=None) == -1
    assert _call_backward(desc, gate, mb.moce_gate_grads(FAKE, None, None, None, None, None)) == -1
    mlp = mb.make_gate(mb.MOCE_GATE_MLP_SIGMOID, W1=FAKE, b1=FAKE, w2=FAKE)
    assert _call_backward(desc, mlp, grads) == -1          # the MLP's gradient arrays are missing
    assert _call_backward(desc, mb.make_gate(7), grads) == -6
    assert _call_backward(good_desc(C=1200, k=1025, E=16), gate, grads) == -10
    mlp_all = mb.moce_gate_grads(None, None, FAKE, FAKE, FAKE, FAKE)
    assert _call_backward(good_desc(C=256, k=129), mlp, mlp_all) == -10
    assert _call_backward(desc, gate, grads, dy=FAKE_UNALIGNED) == -8
    assert _call_backward(desc, gate, grads, ws=None) == -7
    need = lib.moce_backward_workspace_bytes(ctypes.byref(desc), mb.MOCE_GATE_SOFTPLUS_LINEAR)
    assert need > 0
    assert _call_backward(desc, gate, grads, ws_bytes=need - 1) == -7
    assert _call_backward(desc, gate, grads, ws=FAKE_UNALIGNED, ws_bytes=need) == -8
    assert lib.moce_backward_workspace_bytes(ctypes.byref(desc), 7) == 0
    assert lib.moce_backward_workspace_bytes(ctypes.byref(good_desc(C=256, k=129)), mb.MOCE_GATE_MLP_SIGMOID) == 0


def test_backward_workspace_grows_with_the_mlp_gate(lib):
    desc = good_desc()
    sp = lib.moce_backward_workspace_bytes(ctypes.byref(desc), mb.MOCE_GATE_SOFTPLUS_LINEAR)
    ml = lib.moce_backward_workspace_bytes(ctypes.byref(desc), mb.MOCE_GATE_MLP_SIGMOID)
    B, R, k = desc.B, desc.E - 1, desc.k
    assert ml >= sp + B * R * k * 4 and sp % 256 == 0 and ml % 256 == 0


def test_logit_backward_host_errors(lib):
    def call(R=4, C=64, k=8, L=FAKE, s=FAKE, dw=FAKE, eps=1e-8, lam=1.0, dL=FAKE, ws=FAKE, ws_bytes=1 << 20):
        return mb.raw_status("moce_logit_backward", R, C, k, L, s, dw, ctypes.c_float(eps), ctypes.c_float(lam),
                             None, dL, ws, ws_bytes, None)
    assert call(L=None) == -1 and call(dL=None) == -1 and call(ws=None) == -1
    assert call(s=None) == -1 and call(dw=None) == -1
    assert call(R=0) == -2 and call(C=0) == -2 and call(k=0) == -2 and call(k=65) == -2
    assert call(eps=-1.0) == -2 and call(eps=float("nan")) == -2
    assert call(C=32769) == -10
    need = lib.moce_logit_backward_workspace_bytes(4, 64)
    assert need == (2 * 4 + 64 + 3) * 4 + 256 - (2 * 4 + 64 + 3) * 4 % 256
    assert call(ws_bytes=need - 1) == -7
    assert call(ws=FAKE_UNALIGNED) == -8
    assert lib.moce_logit_backward_workspace_bytes(0, 64) == 0
    assert lib.moce_logit_backward_workspace_bytes(4, 40000) == 0


def test_forward_ex_host_errors(lib):
    desc = good_desc()
    gate = mb.make_gate(a=FAKE, c=FAKE)

    def call(ep, ws=FAKE, ws_bytes=1 << 30):
        e = ctypes.byref(ep) if ep is not None else None
        return mb.raw_status("moce_forward_ex", ctypes.byref(desc), FAKE, FAKE, FAKE, ctypes.byref(gate), FAKE, 4, e,
                             FAKE, ws, ws_bytes, None)
    assert call(mb.moce_epilogue(FAKE, None, 0, 0)) == -1
    assert call(mb.moce_epilogue(None, FAKE, 1, 0)) == -1
    assert call(mb.moce_epilogue(FAKE, FAKE, 1, 0), ws=None) == -7
    assert call(None, ws=None) == -7
    for kw, code in BAD_DESCS:
        d = good_desc(**kw)
        assert mb.raw_status("moce_forward_ex", ctypes.byref(d), FAKE, FAKE, FAKE, ctypes.byref(gate), FAKE, 4, None,
                             FAKE, FAKE, 1 << 30, None) == code, kw


def test_support_prepare16_host_errors(lib):
    nU = ctypes.c_int32(0)
    bad = ctypes.c_int32(0)

    def call(desc, s=FAKE, info=FAKE):
        return mb.raw_status("moce_support_prepare16", ctypes.byref(desc), s, FAKE, FAKE + 4096, FAKE + 8192, FAKE,
                             FAKE, info, ctypes.byref(nU), ctypes.byref(bad), None)
    assert call(good_desc(), s=None) == -1
    assert call(good_desc(), info=None) == -1
    assert call(good_desc(C=70000, k=8, E=16)) == -10    # 16-bit indices reach 65535
    for kw, code in BAD_DESCS:
        assert call(good_desc(**kw)) == code, kw
