"""GPU parity of the layer's backward (moce_backward) and of the routing-logit gradient with the coverage
loss (moce_logit_backward) against the oracle's float64 gradients, on the same seeded inputs.

Tolerances, from the arithmetic: every gradient is a float32 sum (over positions, support entries and
images) of products of float32 or bfloat16 values, so its error is a few float32 roundings of the
largest partial sums, well below 2e-5 of the tensor's largest entry at these sizes.  dx in bfloat16 is
rounded once more on its way out (half an ulp, 2^-9 of the value), so it may differ by 2^-8 of the
value on top.  The comparison scale of a parameter gradient is its largest entry over the tensor,
since single entries can cancel to near zero.
"""
import numpy as np
import pytest
import torch

import oracle
from oracle import backward as ob
from paper_2608_23794_amd import inputs
from paper_2608_23794_amd import binding as mb
from paper_2608_23794_amd.layer import MoceLayer, to_device_x, to_host_f64

pytestmark = [pytest.mark.gpu, pytest.mark.usefixtures("oracle_lib")]

OL = {"nchw": oracle.NCHW, "nhwc": oracle.NHWC}
RTOL_F32 = 2e-5


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need a visible MI355X"
    yield
    torch.cuda.synchronize()


def close(name, dev, ref, bf16=False, rtol=RTOL_F32):
    dev = np.asarray(dev, np.float64)
    ref = np.asarray(ref, np.float64)
    assert dev.shape == ref.shape, (name, dev.shape, ref.shape)
    scale = max(np.abs(ref).max(), 1e-30)
    bound = rtol * scale + (2.0 ** -8 * np.abs(ref) if bf16 else 0.0)
    err = np.abs(dev - ref)
    worst = np.unravel_index(np.argmax(err - bound), err.shape)
    assert np.all(err <= bound), f"{name}: |dev - ref| = {err[worst]:.3e} at {worst}, bound {np.asarray(bound).max():.3e}"


def make_dy(shape, dtype, seed):
    g = np.random.default_rng(seed).standard_normal(shape).astype(np.float32)
    if dtype == "bf16":
        bits = inputs.f32_to_bf16_bits(g)
        return bits, inputs.bf16_bits_to_f32(bits).astype(np.float64)
    return g, g.astype(np.float64)


def oracle_grads(layer, x, dy64, gate, params, images=None):
    """Oracle gradients over the canonical rows (so dw comes in the device's order), summed over chunks
    of images; dx only for `images` (all when None)."""
    s_c = layer.s_c.cpu().numpy()
    w_c = layer.w_c.cpu().numpy()
    kw = dict(a=params["a"], c=params["c"]) if gate == "softplus" else dict(
        W1=params["W1"], b1=params["b1"], w2=params["w2"], b2=params["b2"], tau_min=params["tau_min"],
        tau_max=params["tau_max"])
    B = x.shape[0]
    acc = {}
    dx = {}
    step = max(1, int(4e6 // max(1, layer.R * layer.k * layer.H * layer.W)))
    for b0 in range(0, B, step):
        sl = slice(b0, min(B, b0 + step))
        g = ob.layer_backward(x[sl], s_c, w_c, layer.E, dy64[sl], layout=OL[layer.layout], gate=gate, **kw)
        for n in ("dw", "da", "dc", "dW1", "db1", "dw2", "db2"):
            if n in g:
                acc[n] = acc.get(n, 0.0) + np.asarray(g[n])
        for j, b in enumerate(range(sl.start, sl.stop)):
            if images is None or b in images:
                dx[b] = g["dx"][j]
    return acc, dx


def run(layer, x_host, dtype, gate, params, seed=0, images=None):
    B = x_host.shape[0]
    x = to_device_x(x_host, dtype)
    dyh, dy64 = make_dy(layer.y_shape(B), dtype, seed)
    dy = to_device_x(dyh, dtype)
    out = layer.backward(x, dy)
    torch.cuda.synchronize()
    ref, rdx = oracle_grads(layer, x_host, dy64, gate, params, images)
    dx = to_host_f64(out["dx"])
    for b, v in rdx.items():
        close(f"dx[{b}]", dx[b], v, bf16=dtype == "bf16")
    if layer.R > 0:
        close("dw", out["dw"].cpu().numpy(), ref["dw"])
        if gate == "softplus":
            close("da", out["da"].cpu().numpy(), ref["da"])
            close("dc", out["dc"].cpu().numpy()[:layer.R], ref["dc"])
        else:
            close("dW1", out["dW1"].cpu().numpy(), ref["dW1"])
            close("db1", out["db1"].cpu().numpy(), ref["db1"])
            close("dw2", out["dw2"].cpu().numpy(), ref["dw2"])
            close("db2", out["db2"].cpu().numpy()[0], ref["db2"])
    return out


CASES = [("tiny", "nchw", None), ("resnet50_stage1", "nchw", 2), ("resnet50_stage3", "nchw", 3),
         ("resnet50_stage3", "nhwc", 3), ("resnet50_stage4", "nhwc", 2), ("vit_tokens", "nhwc", 2)]


@pytest.mark.parametrize("name,layout,B", CASES)
def test_backward_matches_oracle(name, layout, B):
    wl = inputs.WORKLOADS[name]
    g = inputs.generate(wl, layout, batch=B)
    layer = MoceLayer.from_workload(wl, g, layout)
    run(layer, g["x"], wl.dtype, "softplus", g, seed=wl.seed)


@pytest.mark.parametrize("name,layout,B", [("tiny", "nchw", None), ("resnet50_stage3", "nhwc", 2),
                                           ("resnet50_stage1", "nchw", 2)])
def test_backward_mlp_gate_matches_oracle(name, layout, B):
    wl = inputs.WORKLOADS[name]
    g = inputs.generate(wl, layout, batch=B)
    layer = MoceLayer.from_workload(wl, g, layout, gate="mlp")
    run(layer, g["x"], wl.dtype, "mlp", g, seed=wl.seed + 1)


def test_backward_full_batch_stage3_nhwc():
    """The whole batch of 64 images on the device; the parameter gradients against the oracle summed
    over every image, dx on the first, a middle and the last image."""
    wl = inputs.WORKLOADS["resnet50_stage3"]
    g = inputs.generate(wl, "nhwc")
    layer = MoceLayer.from_workload(wl, g, "nhwc")
    run(layer, g["x"], wl.dtype, "softplus", g, seed=5, images={0, 31, wl.B - 1})


def rand_layer(seed, B, C, E, k, H, W, dtype, layout, gate="softplus"):
    rng = np.random.default_rng(seed)
    R = E - 1
    s = np.array([rng.choice(C, size=k, replace=False) for _ in range(R)], np.int32).reshape(R, k)
    w = (rng.standard_normal((R, k)) * 1.5).astype(np.float32)
    shape = (B, C, H, W) if layout == "nchw" else (B, H, W, C)
    x = (rng.standard_normal(shape) + 0.3).astype(np.float32)
    if dtype == "bf16":
        x = inputs.f32_to_bf16_bits(x)
    p = dict(a=(rng.standard_normal((R, k)) * 0.7).astype(np.float32),
             c=(rng.standard_normal(R) * 0.5).astype(np.float32),
             W1=(rng.standard_normal((k, k)) / np.sqrt(k)).astype(np.float32),
             b1=(rng.standard_normal(k) * 0.2).astype(np.float32),
             w2=(rng.standard_normal(k) / np.sqrt(k)).astype(np.float32), b2=np.float32(0.1), tau_min=0.2,
             tau_max=6.0)
    layer = MoceLayer(C, E, k, H, W, dtype, layout, s, w, gate=gate, **p)
    return layer, x, p


@pytest.mark.parametrize("B,C,E,k,H,W,dtype,layout", [
    (2, 40, 1, 5, 3, 3, "f32", "nchw"),        # no routed expert: every channel is in U
    (2, 40, 6, 1, 2, 3, "bf16", "nhwc"),       # k = 1: alpha = 1, no gradient reaches the gate
    (2, 24, 4, 24, 2, 2, "f32", "nhwc"),       # k = C: U empty
    (3, 37, 9, 7, 3, 5, "bf16", "nchw"),       # C not a multiple of 8, odd plane
    (2, 130, 17, 70, 1, 1, "bf16", "nhwc"),    # one position, k past 64
    (1, 300, 33, 200, 2, 7, "f32", "nhwc"),    # k past 128
    (2, 264, 72, 9, 5, 8, "bf16", "nhwc"),     # matrix-core dalpha: ragged channel and expert blocks, 2 steps
    (2, 72, 16, 7, 9, 8, "bf16", "nchw"),      # matrix-core dalpha, NCHW: 72 positions, a ragged last step
    (1, 48, 24, 6, 5, 4, "bf16", "nchw"),      # NCHW with 4-position loads
    (2, 512, 9, 255, 2, 3, "bf16", "nhwc"),    # the byte table's limit k = 255
    (2, 512, 9, 256, 2, 3, "bf16", "nhwc"),    # k = 256: the generic kernel
    (1, 264, 136, 9, 7, 10, "bf16", "nhwc"),   # matrix-core dx: 2 channel blocks, 3 expert chunks, 2 position tiles
    (1, 300, 136, 5, 6, 6, "bf16", "nchw"),    # the same, NCHW with 4-position loads
])
def test_backward_edge_shapes(B, C, E, k, H, W, dtype, layout):
    layer, x, p = rand_layer(B * 1000 + C, B, C, E, k, H, W, dtype, layout)
    run(layer, x, dtype, "softplus", p, seed=C)


@pytest.mark.parametrize("B,C,E,k,H,W,dtype,layout", [
    (2, 37, 9, 7, 3, 5, "bf16", "nchw"),
    (2, 300, 33, 128, 1, 3, "f32", "nhwc"),    # the MLP backward's limit k = 128
])
def test_backward_mlp_edge_shapes(B, C, E, k, H, W, dtype, layout):
    layer, x, p = rand_layer(B * 77 + C, B, C, E, k, H, W, dtype, layout, gate="mlp")
    run(layer, x, dtype, "mlp", p, seed=C + 1)


def test_backward_residual_only_upstream_is_exact_mean():
    """dy zero on the routed outputs: dx is dy_res / |U| on U and 0 elsewhere, and nothing reaches w or
    the gate (exact zeros on both sides)."""
    layer, x, p = rand_layer(3, 2, 48, 5, 4, 3, 3, "f32", "nchw")
    xd = to_device_x(x, "f32")
    dy = torch.zeros(layer.y_shape(2), dtype=torch.float32, device="cuda")
    dy[:, 4] = torch.randn(2, 3, 3, device="cuda")
    out = layer.backward(xd, dy)
    torch.cuda.synchronize()
    U = layer.U.cpu().numpy()[:layer.nU]
    ref = np.zeros(x.shape)
    ref[:, U] = (dy[:, 4:5].cpu().numpy() / np.float32(layer.nU)).astype(np.float32)
    np.testing.assert_array_equal(out["dx"].cpu().numpy(), ref.astype(np.float32))
    assert torch.all(out["dw"] == 0) and torch.all(out["da"] == 0) and torch.all(out["dc"][:4] == 0)


@pytest.mark.parametrize("R,C,k,eps,lam", [(63, 256, 32, 1e-8, 5e-4), (255, 1024, 64, 1e-8, 0.05),
                                           (7, 100, 9, 0.3, 1.0), (3, 32768, 5, 1e-8, 2.0)])
def test_logit_backward_matches_oracle(R, C, k, eps, lam):
    rng = np.random.default_rng(R + C)
    L = (rng.standard_normal((R, C)) * 0.5).astype(np.float32)
    s = np.argsort(-L, axis=1, kind="stable")[:, :k].astype(np.int32)
    w = np.take_along_axis(L, s, axis=1)
    layer = MoceLayer(C, R + 1, k, 1, 1, "f32", "nchw", s, w, a=np.zeros((R, k), np.float32),
                      c=np.zeros(R, np.float32))
    s_c = layer.s_c.cpu().numpy()
    dw = rng.standard_normal((R, k)).astype(np.float32)
    Ld = torch.from_numpy(L).cuda()
    loss, dL = layer.logit_backward(Ld, torch.from_numpy(dw).cuda(), eps, lam)
    loss0, dL0 = layer.logit_backward(Ld, None, eps, lam)
    torch.cuda.synchronize()
    ref_loss = ob.coverage_loss(L, eps)
    G = lam * ob.coverage_grad(L, eps)
    assert float(loss.cpu()[0]) == pytest.approx(ref_loss, rel=1e-4, abs=1e-7)
    assert float(loss0.cpu()[0]) == float(loss.cpu()[0])
    close("dL (coverage only)", dL0.cpu().numpy(), G, rtol=1e-4)
    full = G.copy()
    np.put_along_axis(full, s_c.astype(np.int64), np.take_along_axis(full, s_c.astype(np.int64), 1) + dw, 1)
    close("dL", dL.cpu().numpy(), full, rtol=1e-4)
