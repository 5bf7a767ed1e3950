"""GPU parity of the input-conditioned (dynamic) support path (Sec. 4.5 Eq. 11) against the oracle.

The selection is an integer decision taken from floating-point logits: the device forms the
example's logits in float32 from its own pooled descriptor, the oracle in float64 from the exact one.
The test therefore checks that the device's supports are a valid top k of the oracle's logits up to
a margin (every selected logit at least, every other logit at most, the oracle's k-th largest within
``EPS``; the order canonical within ``EPS``), and that they agree with the oracle's own selection
wherever the k-th and (k+1)-th largest logits are further apart than ``2 EPS``.  The outputs are then
compared with the oracle's layer evaluated at the device's supports (the oracle's logits there), to the
static layer's tolerances.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2608_23794_amd import inputs
from paper_2608_23794_amd.layer import DynamicMoceLayer, to_device_x, to_host_f64

pytestmark = [pytest.mark.gpu, pytest.mark.usefixtures("oracle_lib")]

OL = {"nchw": oracle.NCHW, "nhwc": oracle.NHWC}
EPS = 1e-4

CASES = [("tiny", "nchw"), ("tiny", "nhwc"), ("resnet50_stage1", "nchw"), ("resnet50_stage3", "nchw"),
         ("resnet50_stage3", "nhwc"), ("resnet50_stage4", "nhwc"), ("vit_tokens", "nhwc")]


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need a visible MI355X"
    yield
    torch.cuda.synchronize()


def check_y(y, y_ref, mag, dtype):
    err = np.abs(y - y_ref)
    rtol = 1e-5 if dtype == "f32" else 1e-2
    e = (err / np.maximum(mag, 1e-30)).max()
    assert e <= rtol, f"y: max |y - y_ref| / M = {e:.3e}"
    if dtype == "bf16":
        assert np.all(err <= 2.0 ** -8 * np.abs(y_ref) + 1e-5 * mag), "y: beyond one bf16 rounding"


def check_selection(S, Lx, k):
    """S [n, R, k] device supports, Lx [n, R, C] oracle logits (float64)."""
    n, R, C = Lx.shape
    agree = 0
    for b in range(n):
        for e in range(R):
            vals, sel = Lx[b, e], S[b, e]
            assert np.unique(sel).size == k and sel.min() >= 0 and sel.max() < C
            srt = np.sort(vals)[::-1]
            kth = srt[k - 1]
            mask = np.zeros(C, bool)
            mask[sel] = True
            assert vals[mask].min() >= kth - EPS, (b, e)
            if k < C:
                assert vals[~mask].max() <= kth + EPS, (b, e)
            assert np.all(vals[sel][:-1] >= vals[sel][1:] - EPS), (b, e)
            if k == C or srt[k - 1] - srt[k] > 2 * EPS:
                ref = np.lexsort((np.arange(C), -vals))[:k]
                np.testing.assert_array_equal(np.sort(sel), np.sort(ref))
                agree += 1
    return agree


def run_case(wl, layout, B=None, images=None, gate="softplus"):
    g = inputs.generate(wl, layout, batch=B)
    rt = inputs.router_params(wl)
    layer = DynamicMoceLayer.from_workload(wl, g, rt, layout, gate=gate)
    x = to_device_x(g["x"], wl.dtype)
    Bn = x.shape[0]
    S = torch.empty((Bn, wl.E - 1, wl.k), dtype=torch.int32, device="cuda")
    y = to_host_f64(layer.forward(x, S_out=S))
    S = S.cpu().numpy()
    imgs = list(range(Bn)) if images is None else images
    xs = g["x"][imgs]
    d = oracle.pool(xs, OL[layout])
    Lx = oracle.dynamic_logits(oracle.router(d, rt["Wh"], rt["bh"]), rt["L"], rt["q"], rt["v"])
    agree = check_selection(S[imgs], Lx, wl.k)
    W = np.take_along_axis(Lx, S[imgs].astype(np.int64), axis=2)
    kw = dict(a=g["a"], c=g["c"]) if gate == "softplus" else dict(
        W1=g["W1"], b1=g["b1"], w2=g["w2"], b2=g["b2"], tau_min=g["tau_min"], tau_max=g["tau_max"])
    ref = oracle.dynamic_forward(xs, rt["L"], rt["Wh"], rt["bh"], rt["v"], rt["q"], wl.k, wl.E, OL[layout],
                                 gate=gate, S=S[imgs], W=W, **kw)
    check_y(y[imgs], ref["y"], ref["mag"], wl.dtype)
    return S, agree


@pytest.mark.parametrize("name,layout", CASES)
def test_dynamic_forward(name, layout):
    """The full batch runs on the device; the oracle checks the first two images and the last."""
    wl = inputs.WORKLOADS[name]
    imgs = sorted({0, 1, wl.B - 1}) if wl.B > 3 else None
    S, agree = run_case(wl, layout, images=imgs)
    assert agree > 0
    # the supports do depend on the example
    assert any(not np.array_equal(S[0], S[b]) for b in range(1, S.shape[0])) or wl.B == 1


@pytest.mark.parametrize("name,layout", [("tiny", "nchw"), ("resnet50_stage3", "nhwc")])
def test_dynamic_forward_mlp_gate(name, layout):
    wl = inputs.WORKLOADS[name]
    run_case(wl, layout, B=4, gate="mlp")


@pytest.mark.parametrize("B,C,E,k,d,H,W,dtype,layout", [
    (3, 40, 5, 40, 3, 2, 3, "f32", "nchw"),      # k = C: every channel in every support, U(X) empty
    (2, 96, 33, 1, 1, 3, 3, "bf16", "nhwc"),     # k = 1, d = 1
    (2, 300, 20, 200, 64, 1, 5, "f32", "nhwc"),  # k past a power of two, the widest router
    (1, 70, 2, 9, 5, 1, 1, "bf16", "nchw"),      # one routed expert, one position
    (2, 4096, 9, 512, 16, 1, 2, "f32", "nhwc"),  # the size limits: C = 4096, k = 512
    # bfloat16 NCHW with C <= 256 and H W a multiple of 8 takes the tile mix, which reloads the
    # supports when the image changes: one tile per image, a ragged last tile, and a coefficient
    # table too large to prefetch in registers
    (6, 64, 17, 8, 4, 4, 6, "bf16", "nchw"),
    (3, 256, 64, 16, 8, 12, 12, "bf16", "nchw"),
    (2, 200, 200, 12, 8, 8, 8, "bf16", "nchw"),
])
def test_dynamic_forward_edges(B, C, E, k, d, H, W, dtype, layout):
    rng = np.random.default_rng(B * 7919 + C)
    R = E - 1
    shape = (B, C, H, W) if layout == "nchw" else (B, H, W, C)
    x = np.maximum(rng.standard_normal(shape), 0).astype(np.float32)
    if dtype == "bf16":
        x = inputs.f32_to_bf16_bits(x)
    L = rng.standard_normal((R, C)).astype(np.float32)
    L[0, :8] = 0.5                                   # exact ties in the static logits
    Wh = (rng.standard_normal((d, C)) * 2 / np.sqrt(C)).astype(np.float32)
    bh = (rng.standard_normal(d) * 0.1).astype(np.float32)
    v = rng.standard_normal((C, d)).astype(np.float32)
    q = (rng.standard_normal((R, d)) / np.sqrt(d)).astype(np.float32)
    a = (rng.standard_normal((R, k)) / np.sqrt(k)).astype(np.float32)
    c = np.zeros(R, np.float32)
    layer = DynamicMoceLayer(C, E, k, H, W, dtype, layout, L, Wh, bh, v, q, a=a, c=c)
    xd = to_device_x(x, dtype)
    S = torch.empty((B, R, k), dtype=torch.int32, device="cuda")
    y = to_host_f64(layer.forward(xd, S_out=S))
    S = S.cpu().numpy()
    d_ref = oracle.pool(x, OL[layout])
    Lx = oracle.dynamic_logits(oracle.router(d_ref, Wh, bh), L, q, v)
    check_selection(S, Lx, k)
    Wsel = np.take_along_axis(Lx, S.astype(np.int64), axis=2)
    ref = oracle.dynamic_forward(x, L, Wh, bh, v, q, k, E, OL[layout], a=a, c=c, S=S, W=Wsel)
    check_y(y, ref["y"], ref["mag"], dtype)


def test_dynamic_forward_without_offset_matches_static_supports():
    """q = 0: the device's supports are the top k of the static logits for every example, ties to the
    lower channel, bit for bit (the logits are then the given float32 values on both sides)."""
    wl = inputs.WORKLOADS["resnet50_stage3"]
    g = inputs.generate(wl, "nhwc", batch=3)
    rt = dict(inputs.router_params(wl))
    rt["q"] = np.zeros_like(rt["q"])
    rt["L"] = np.round(rt["L"] * 4) / 4          # many exact ties
    layer = DynamicMoceLayer.from_workload(wl, g, rt, "nhwc")
    S = torch.empty((3, wl.E - 1, wl.k), dtype=torch.int32, device="cuda")
    layer.forward(to_device_x(g["x"], wl.dtype), S_out=S)
    S = S.cpu().numpy()
    ref = np.stack([np.lexsort((np.arange(wl.C), -row))[:wl.k] for row in rt["L"].astype(np.float64)])
    for b in range(3):
        np.testing.assert_array_equal(S[b], ref)
