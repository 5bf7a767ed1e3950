"""GPU parity of the channels-last gather mix (MOCE_PATH_GATHER: bfloat16 NHWC with k <= 16, the
paper's ResNet-50 setting of Sec. 4.1 with k = 8) against the oracle, through the C ABI.

Bar, as for every forward: |y - y_ref| <= 1e-2 M (M the oracle's magnitude sum_i alpha_i |x_i|) and
within one bf16 rounding of the float32 result, |y - y_ref| <= 2^-8 |y_ref| + 1e-5 M.  Single-channel
supports (k = 1) and the one-hot limit are exact copies.  Shapes span several step buffers and work
ranges, ragged position octets (H W not a multiple of 8), one to four routed experts per thread,
both support-register widths (k <= 8, k <= 16), empty and non-empty residual sets, the size limits
(C = 4096, E - 1 = 1024), and one ResNet-50 entrance at the benchmark's batch of 512 on sampled images.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2608_23794_amd import binding as mb
from paper_2608_23794_amd import inputs
from paper_2608_23794_amd.layer import MoceLayer, to_device_x, to_host_f64

pytestmark = [pytest.mark.gpu, pytest.mark.usefixtures("oracle_lib")]


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need a visible MI355X"
    mb.load()
    yield
    torch.cuda.synchronize()


def custom(B, C, E, k, H, W, seed, signed=False, cyclic=False):
    rng = np.random.default_rng(seed)
    R = E - 1
    if cyclic:
        s = np.array([[(e * k + j) % C for j in range(k)] for e in range(R)], np.int32).reshape(R, k)
    else:
        s = np.array([rng.choice(C, k, replace=False) for _ in range(R)], np.int32).reshape(R, k)
    w = rng.standard_normal((R, k)).astype(np.float32)
    a = (rng.standard_normal((R, k)) * k ** -0.5).astype(np.float32)
    c = rng.standard_normal(R).astype(np.float32) * np.float32(0.5)
    x = rng.standard_normal((B, H, W, C)).astype(np.float32)
    if not signed:
        x = np.maximum(x, 0)
    return inputs.f32_to_bf16_bits(x), s, w, a, c


def check_y(y, y_ref, mag):
    err = np.abs(y - y_ref)
    norm = err / np.maximum(mag, 1e-30)
    worst = np.unravel_index(np.argmax(norm), norm.shape)
    assert norm.max() <= 1e-2, f"y: max error/M {norm.max():.3e} at {worst}"
    bound = 2.0 ** -8 * np.abs(y_ref) + 1e-5 * mag + 1e-30
    assert np.all(err <= bound), f"y: {int((err > bound).sum())} outputs beyond one bf16 rounding"


GATHER = [
    # B, C, E, k, H, W, extra
    (3, 16, 9, 8, 13, 13, {}),                  # 18-row octets: many octets per step, ragged 169 positions
    (3, 64, 64, 8, 56, 56, {}),                 # ResNet-50 stage-1 entrance: 14 steps per image range
    (2, 512, 300, 8, 5, 7, {}),                 # two routed experts per thread, 35 positions
    (2, 2048, 1025, 4, 7, 7, {}),               # E - 1 = 1024: four experts per thread
    (2, 1024, 40, 16, 7, 7, {}),                # 16 support registers, one octet per step, |U| large
    (2, 2048, 513, 12, 3, 5, {}),               # two experts per thread with 16 support registers
    (2, 4096, 700, 8, 3, 3, {}),                # C = 4096 with three experts per thread
    (1, 24, 20, 3, 3, 3, {}),                   # k below the register width; fewer than 8 positions
    (2, 4096, 24, 8, 2, 3, {}),                 # C = 4096: 144 KB of step buffers
    (2, 2048, 512, 8, 7, 7, dict(signed=True)),  # ResNet-50 stage-4 entrance, signed inputs
    (2, 64, 8, 4, 5, 5, {}),
    (2, 128, 40, 7, 3, 11, dict(signed=True)),
    (2, 256, 16, 8, 4, 4, dict(cyclic=True)),   # cyclic supports: U = channels 120..255
    (2, 256, 64, 4, 4, 4, dict(cyclic=True)),   # cyclic supports covering C exactly: U empty
    (4, 512, 40, 1, 6, 6, {}),                  # k = 1: exact copies
    (2, 64, 2, 8, 3, 5, {}),                    # one routed expert
    (1, 8, 2, 1, 1, 1, {}),                     # the smallest shape
    (2, 96, 20, 16, 7, 7, {}),                  # C a multiple of 8 but not of 64, E not a multiple of 8
]


@pytest.mark.parametrize("B,C,E,k,H,W,extra", GATHER)
def test_gather_forward_shapes(B, C, E, k, H, W, extra):
    x, s, w, a, c = custom(B, C, E, k, H, W, seed=B * 131 + C + E + k, **extra)
    ref = oracle.forward(x, s, w, E, oracle.NHWC, a=a, c=c)
    layer = MoceLayer(C, E, k, H, W, "bf16", "nhwc", s, w, a=a, c=c)
    assert mb.moce_forward_path(layer.desc(B), mb.MOCE_GATE_SOFTPLUS_LINEAR) == mb.PATH_GATHER
    assert layer.nU == ref["nU"]
    y = to_host_f64(layer.forward(to_device_x(x, "bf16")))
    check_y(y, ref["y"], ref["mag"])
    if ref["nU"] == 0:
        assert np.all(y[..., E - 1] == 0.0)
    if k == 1:
        assert np.array_equal(y[..., :E - 1], ref["y"][..., :E - 1])


@pytest.mark.parametrize("B,C,E,k,H,W", [(2, 512, 300, 8, 5, 7), (2, 1024, 40, 16, 7, 7)])
def test_gather_mix_with_given_coefficients(B, C, E, k, H, W):
    """moce_mix on the gather path, with the oracle's coefficients as input."""
    x, s, w, a, c = custom(B, C, E, k, H, W, seed=7 + k)
    ref = oracle.forward(x, s, w, E, oracle.NHWC, a=a, c=c)
    layer = MoceLayer(C, E, k, H, W, "bf16", "nhwc", s, w, a=a, c=c)
    alpha = torch.from_numpy(ref["alpha"].astype(np.float32)).cuda()
    y = to_host_f64(layer.mix(to_device_x(x, "bf16"), alpha))
    check_y(y, ref["y"], ref["mag"])


def test_gather_forward_equals_stages():
    """The forward's coefficients are those moce_gate writes, so forward and pool + gate + mix agree bit
    for bit on the gather path."""
    B, C, E, k, H, W = 3, 256, 120, 12, 9, 9
    x, s, w, a, c = custom(B, C, E, k, H, W, seed=11, signed=True)
    layer = MoceLayer(C, E, k, H, W, "bf16", "nhwc", s, w, a=a, c=c)
    xd = to_device_x(x, "bf16")
    y = layer.forward(xd)
    _, alpha = layer.gate_tau(layer.pool(xd))
    y_st = layer.mix(xd, alpha)
    torch.cuda.synchronize()
    assert torch.equal(y.view(torch.int16), y_st.view(torch.int16))


def test_gather_mlp_gate_and_one_hot():
    """The paper's MLP gate on the gather path, and the one-hot limit as exact copies."""
    B, C, E, k, H, W = 2, 512, 64, 8, 6, 6
    x, s, w, a, c = custom(B, C, E, k, H, W, seed=17, signed=True)
    rng = np.random.default_rng(18)
    W1 = (rng.standard_normal((k, k)) * k ** -0.5).astype(np.float32)
    b1 = (rng.standard_normal(k) * 0.1).astype(np.float32)
    w2 = (rng.standard_normal(k) * k ** -0.5).astype(np.float32)
    ref = oracle.forward(x, s, w, E, oracle.NHWC, gate="mlp", W1=W1, b1=b1, w2=w2, b2=0.0)
    layer = MoceLayer(C, E, k, H, W, "bf16", "nhwc", s, w, gate="mlp", W1=W1, b1=b1, w2=w2, b2=0.0)
    assert mb.moce_forward_path(layer.desc(B), mb.MOCE_GATE_MLP_SIGMOID) == mb.PATH_GATHER
    check_y(to_host_f64(layer.forward(to_device_x(x, "bf16"))), ref["y"], ref["mag"])
    w[:, 0] = w.max(axis=1) + 1.0
    a[:] = 0.0
    c[:] = -1e4
    ref = oracle.forward(x, s, w, E, oracle.NHWC, a=a, c=c)
    layer = MoceLayer(C, E, k, H, W, "bf16", "nhwc", s, w, a=a, c=c)
    y = to_host_f64(layer.forward(to_device_x(x, "bf16")))
    assert np.array_equal(y[..., :E - 1], ref["y"][..., :E - 1])


@pytest.mark.parametrize("relu", [False, True])
def test_gather_epilogue(relu):
    """The per-channel affine map and ReLU applied to the float32 accumulators before the one rounding."""
    B, C, E, k, H, W = 2, 256, 72, 8, 7, 7
    x, s, w, a, c = custom(B, C, E, k, H, W, seed=23, signed=True)
    ref = oracle.forward(x, s, w, E, oracle.NHWC, a=a, c=c)
    layer = MoceLayer(C, E, k, H, W, "bf16", "nhwc", s, w, a=a, c=c)
    rng = np.random.default_rng(24)
    scale = (rng.standard_normal(E) * 0.8 + 1.0).astype(np.float32)
    shift = (rng.standard_normal(E) * 0.3).astype(np.float32)
    y = to_host_f64(layer.forward(to_device_x(x, "bf16"),
                                  epilogue=(torch.from_numpy(scale).cuda(), torch.from_numpy(shift).cuda(), relu)))
    yhat = oracle.epilogue(ref["y"], scale, shift, relu, oracle.NHWC)
    magp = np.abs(scale) * ref["mag"] + np.abs(shift)
    bound = 1e-5 * magp + 2.0 ** -8 * np.abs(yhat) + 1e-30
    err = np.abs(y - yhat)
    assert np.all(err <= bound), f"{int((err > bound).sum())} outputs beyond the bound, worst {err.max():.3e}"


def test_gather_resnet50_entrance_full_batch_sampled():
    """The stage-4 entrance projection (C = 2048, E = 512, 7 x 7) at batch 512 with k = 8, as the
    replaced-operator timing runs it: every image is independent, so the oracle's forward of a few
    sampled images is the reference for those images' outputs."""
    B, C, E, k, H, W = 512, 2048, 512, 8, 7, 7
    x, s, w, a, c = custom(B, C, E, k, H, W, seed=2048)
    layer = MoceLayer(C, E, k, H, W, "bf16", "nhwc", s, w, a=a, c=c)
    assert mb.moce_forward_path(layer.desc(B), mb.MOCE_GATE_SOFTPLUS_LINEAR) == mb.PATH_GATHER
    y = layer.forward(to_device_x(x, "bf16"))
    torch.cuda.synchronize()
    for b in (0, 1, 255, 510, 511):
        ref = oracle.forward(x[b:b + 1], s, w, E, oracle.NHWC, a=a, c=c)
        check_y(to_host_f64(y[b:b + 1]), ref["y"], ref["mag"])
