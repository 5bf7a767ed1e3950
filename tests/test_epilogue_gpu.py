"""GPU parity of the forward with the output epilogue (moce_forward_ex): per output channel
act(scale[o] y + shift[o]), the batch normalisation and nonlinearity that follow the replaced
projection (Sec. 4.1), against the oracle's layer followed by oracle.epilogue.

Tolerance, from the arithmetic: with M the oracle's magnitude of y (reading 10), the epilogue's value
has magnitude M' = |scale| M + |shift|, and float32 rounding keeps the error below 1e-5 M'.  A bf16
output is rounded once after the epilogue on the matrix-core paths and twice (before and after it) on
the paths that apply it in a second pass, so bf16 values may differ by 2^-8 (|scale y| + |y'|) on top.
With scale = 1, shift = 0 and no ReLU the result equals moce_forward bit for bit on every path.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2608_23794_amd import binding as mb
from paper_2608_23794_amd import inputs
from paper_2608_23794_amd.layer import MoceLayer, to_device_x, to_host_f64

pytestmark = [pytest.mark.gpu, pytest.mark.usefixtures("oracle_lib")]

OL = {"nchw": oracle.NCHW, "nhwc": oracle.NHWC}


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need a visible MI355X"
    yield
    torch.cuda.synchronize()


def check(y, y_ref, yhat_ref, mag, scale, shift, dtype, layout):
    ax = 1 if layout == "nchw" else -1
    shp = [1] * y.ndim
    shp[ax] = -1
    sc = np.abs(scale).reshape(shp) if scale is not None else 1.0
    sf = np.abs(shift).reshape(shp) if shift is not None else 0.0
    magp = sc * mag + sf
    err = np.abs(y - yhat_ref)
    bound = 1e-5 * magp + 1e-30
    if dtype == "bf16":
        pre = np.abs(y_ref) * sc
        bound = bound + 2.0 ** -8 * (pre + np.abs(yhat_ref))
    worst = np.unravel_index(np.argmax(err - bound), err.shape)
    assert np.all(err <= bound), f"|y - ref| = {err[worst]:.3e} at {worst}, bound {bound[worst]:.3e}"


def run(layer, x_host, dtype, layout, ref, scale, shift, relu):
    E = layer.E
    xd = to_device_x(x_host, dtype)
    sd = torch.from_numpy(scale).cuda() if scale is not None else None
    fd = torch.from_numpy(shift).cuda() if shift is not None else None
    y = to_host_f64(layer.forward(xd, epilogue=(sd, fd, relu)))
    yhat = oracle.epilogue(ref["y"], scale, shift, relu, OL[layout])
    check(y, ref["y"], yhat, ref["mag"], scale, shift, dtype, layout)
    return xd


def params(E, seed):
    rng = np.random.default_rng(seed)
    scale = (rng.standard_normal(E) * 0.8 + 1.0).astype(np.float32)
    shift = (rng.standard_normal(E) * 0.3).astype(np.float32)
    return scale, shift


# (workload, layout, batch): the matrix-core paths (stage 1 with the gate inside the mix; the
# scheduled channels-last mix) apply the epilogue to the accumulators, the others in a second pass
CASES = [("tiny", "nchw", None), ("resnet50_stage1", "nchw", 3), ("resnet50_stage3", "nchw", 3),
         ("resnet50_stage3", "nhwc", 4), ("resnet50_stage4", "nhwc", 3), ("vit_tokens", "nhwc", 3)]


@pytest.mark.parametrize("name,layout,B", CASES)
@pytest.mark.parametrize("relu", [False, True])
def test_forward_epilogue(name, layout, B, relu):
    wl = inputs.WORKLOADS[name]
    g = inputs.generate(wl, layout, batch=B)
    ref = oracle.forward(g["x"], g["s"], g["w"], wl.E, OL[layout], a=g["a"], c=g["c"])
    layer = MoceLayer.from_workload(wl, g, layout)
    scale, shift = params(wl.E, wl.seed)
    run(layer, g["x"], wl.dtype, layout, ref, scale, shift, relu)


@pytest.mark.parametrize("name,layout,B", CASES)
def test_relu_only_epilogue(name, layout, B):
    wl = inputs.WORKLOADS[name]
    g = inputs.generate(wl, layout, batch=B)
    ref = oracle.forward(g["x"], g["s"], g["w"], wl.E, OL[layout], a=g["a"], c=g["c"])
    layer = MoceLayer.from_workload(wl, g, layout)
    run(layer, g["x"], wl.dtype, layout, ref, None, None, True)


def test_epilogue_on_mfma_path_with_gate_kernel_and_tile_path():
    """The MLP gate on the stage-1 shape (gate kernel, then the matrix-core mix), and an NCHW bf16 shape
    outside the matrix-core limits (the tile kernel, then the second pass)."""
    wl = inputs.WORKLOADS["resnet50_stage1"]
    g = inputs.generate(wl, batch=2)
    ref = oracle.forward(g["x"], g["s"], g["w"], wl.E, oracle.NCHW, gate="mlp", W1=g["W1"], b1=g["b1"],
                         w2=g["w2"], b2=g["b2"], tau_min=g["tau_min"], tau_max=g["tau_max"])
    layer = MoceLayer.from_workload(wl, g, "nchw", gate="mlp")
    assert mb.moce_forward_path(layer.desc(2), mb.MOCE_GATE_MLP_SIGMOID) == mb.PATH_MFMA
    scale, shift = params(wl.E, 5)
    run(layer, g["x"], wl.dtype, "nchw", ref, scale, shift, True)

    rng = np.random.default_rng(3)
    B, C, E, k, H, W = 2, 200, 40, 12, 4, 6
    s = np.array([rng.choice(C, size=k, replace=False) for _ in range(E - 1)], np.int32)
    w = rng.standard_normal((E - 1, k)).astype(np.float32)
    a = (rng.standard_normal((E - 1, k)) / np.sqrt(k)).astype(np.float32)
    c = np.zeros(E - 1, np.float32)
    x = inputs.f32_to_bf16_bits(np.maximum(rng.standard_normal((B, C, H, W)), 0).astype(np.float32))
    layer = MoceLayer(C, E, k, H, W, "bf16", "nchw", s, w, a=a, c=c)
    assert mb.moce_forward_path(layer.desc(B), mb.MOCE_GATE_SOFTPLUS_LINEAR) == mb.PATH_TILE
    ref = oracle.forward(x, s, w, E, oracle.NCHW, a=a, c=c)
    scale, shift = params(E, 6)
    run(layer, x, "bf16", "nchw", ref, scale, shift, True)


@pytest.mark.parametrize("name,layout,B", CASES)
def test_identity_epilogue_is_the_plain_forward(name, layout, B):
    wl = inputs.WORKLOADS[name]
    g = inputs.generate(wl, layout, batch=B)
    layer = MoceLayer.from_workload(wl, g, layout)
    xd = to_device_x(g["x"], wl.dtype)
    y0 = layer.forward(xd).clone()
    one = torch.ones(wl.E, dtype=torch.float32, device="cuda")
    zero = torch.zeros(wl.E, dtype=torch.float32, device="cuda")
    y1 = layer.forward(xd, epilogue=(one, zero, False))
    assert torch.equal(y0.view(torch.int16) if y0.dtype == torch.bfloat16 else y0.view(torch.int32),
                       y1.view(torch.int16) if y1.dtype == torch.bfloat16 else y1.view(torch.int32))
