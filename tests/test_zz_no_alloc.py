"""moce_forward_static, the forward without a workspace argument (for callers
that cannot allocate), against moce_forward on the same inputs: the same
kernels with the workspace in the library's per-device array, so the outputs
must be identical bit for bit.  Two calls in a row, the second on a smaller
batch, so that the second call runs over what the first left in the array."""
import numpy as np
import pytest
import torch

from paper_2608_23794_amd import binding as mb
from paper_2608_23794_amd import inputs
from paper_2608_23794_amd.layer import MoceLayer, to_device_x

pytestmark = pytest.mark.gpu

CASES = [
    # workload, layout, batch of the first call, batch of the second (smaller) call
    ("resnet50_stage1", "nchw", 24, 7),     # pooling, then gate and mix in one kernel
    ("resnet50_stage3", "nhwc", 16, 5),     # pooling, gate (statistics), scheduled mix
    ("resnet50_stage3", "nchw", 12, 3),     # pooling, gate (coefficients), mix
    ("tiny", "nchw", 2, 1),
]


@pytest.mark.parametrize("name,layout,b1,b2", CASES)
def test_static_forward_equals_forward(name, layout, b1, b2):
    assert torch.cuda.is_available()
    wl = inputs.WORKLOADS[name]
    g = inputs.generate(wl, layout, batch=b1)
    layer = MoceLayer.from_workload(wl, g, layout)
    x1 = to_device_x(g["x"], wl.dtype)
    # the second input: other values and fewer images
    x2 = (x1[:b2].float() * -1.5 + 0.25).to(x1.dtype).contiguous()
    iv = torch.int16 if wl.dtype == "bf16" else torch.int32
    U = layer.U if layer.nU else None
    for x in (x1, x2):
        B = x.shape[0]
        desc = layer.desc(B)
        assert mb.moce_forward_workspace_bytes(desc) <= mb.MOCE_STATIC_SCRATCH_BYTES
        y_ref = layer.forward(x)
        y = torch.full_like(y_ref, float("nan"))
        mb.moce_forward_static(desc, x, layer.s_c, layer.w_c, layer.gate, U, layer.nU, y,
                               torch.cuda.current_stream())
        torch.cuda.synchronize()
        assert torch.equal(y.view(iv), y_ref.view(iv)), f"{name}/{layout} B={B}"


def test_static_forward_full_stage1_batch():
    """The benchmark's stage-1 layer at its full batch fits the array and matches moce_forward."""
    wl = inputs.WORKLOADS["resnet50_stage1"]
    g = inputs.generate(wl)
    layer = MoceLayer.from_workload(wl, g)
    x = to_device_x(g["x"], wl.dtype)
    y_ref = layer.forward(x)
    y = torch.empty_like(y_ref)
    mb.moce_forward_static(layer.desc(wl.B), x, layer.s_c, layer.w_c, layer.gate, None, layer.nU, y)
    torch.cuda.synchronize()
    assert torch.equal(y.view(torch.int16), y_ref.view(torch.int16))


def test_static_forward_on_the_gather_path():
    """A channels-last layer with small supports (the gather path: coefficients in the array), two
    calls in a row, the second on fewer images with other values."""
    rng = np.random.default_rng(91)
    B, C, E, k, H, W = 6, 256, 72, 8, 9, 9
    R = E - 1
    s = np.array([rng.choice(C, k, replace=False) for _ in range(R)], np.int32)
    w = rng.standard_normal((R, k)).astype(np.float32)
    a = (rng.standard_normal((R, k)) * k ** -0.5).astype(np.float32)
    c = np.zeros(R, np.float32)
    x = inputs.f32_to_bf16_bits(np.maximum(rng.standard_normal((B, H, W, C)), 0).astype(np.float32))
    layer = MoceLayer(C, E, k, H, W, "bf16", "nhwc", s, w, a=a, c=c)
    assert mb.moce_forward_path(layer.desc(B), mb.MOCE_GATE_SOFTPLUS_LINEAR) == mb.PATH_GATHER
    x1 = to_device_x(x, "bf16")
    x2 = (x1[:2].float() * -1.5 + 0.25).to(x1.dtype).contiguous()
    U = layer.U if layer.nU else None
    for xx in (x1, x2):
        desc = layer.desc(xx.shape[0])
        y_ref = layer.forward(xx)
        y = torch.full_like(y_ref, float("nan"))
        mb.moce_forward_static(desc, xx, layer.s_c, layer.w_c, layer.gate, U, layer.nU, y,
                               torch.cuda.current_stream())
        torch.cuda.synchronize()
        assert torch.equal(y.view(torch.int16), y_ref.view(torch.int16))
