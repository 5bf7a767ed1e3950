"""The seeded workload generator: determinism, rounding and structure."""
import numpy as np
import pytest
import torch

from paper_2608_23794_amd import inputs


def test_bf16_rounding_matches_torch():
    rng = np.random.default_rng(0)
    v = np.concatenate([rng.standard_normal(100000).astype(np.float32) * 10,
                        np.array([0.0, -0.0, 1.0, 1.00390625, 1.01171875, 3.4e38, -1e-40], np.float32)])
    # exact ties: 1 + 2^-8 rounds to even (down), 1 + 3*2^-8 rounds up
    ours = inputs.f32_to_bf16_bits(v)
    ref = torch.from_numpy(v).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(ours, ref)
    back = inputs.bf16_bits_to_f32(ours)
    assert np.array_equal(back, torch.from_numpy(v).to(torch.bfloat16).float().numpy())


def test_generation_is_deterministic_and_batch_prefix_stable():
    wl = inputs.WORKLOADS["tiny"]
    g1 = inputs.generate(wl)
    g2 = inputs.generate(wl)
    for key in ("x", "s", "w", "a", "c", "W1"):
        assert np.array_equal(g1[key], g2[key])
    wl3 = inputs.WORKLOADS["resnet50_stage3"]
    part = inputs.generate(wl3, batch=2)
    full = inputs.generate(wl3, batch=5)
    assert np.array_equal(part["x"], full["x"][:2])
    assert np.array_equal(part["s"], full["s"])


def test_layouts_hold_the_same_tensor():
    wl = inputs.WORKLOADS["resnet50_stage3"]
    a = inputs.generate(wl, "nchw", batch=2)["x"]
    b = inputs.generate(wl, "nhwc", batch=2)["x"]
    assert np.array_equal(a.transpose(0, 2, 3, 1), b)


@pytest.mark.parametrize("name", list(inputs.WORKLOADS))
def test_workload_structure(name):
    wl = inputs.WORKLOADS[name]
    g = inputs.generate(wl, batch=1)
    R, k = wl.E - 1, wl.k
    assert g["s"].shape == (R, k) and g["s"].dtype == np.int32
    assert g["w"].shape == (R, k) and g["a"].shape == (R, k) and g["c"].shape == (R,)
    for row in g["s"]:
        assert len(set(row.tolist())) == k and row.min() >= 0 and row.max() < wl.C
    x = g["x"]
    xf = inputs.bf16_bits_to_f32(x) if wl.dtype == inputs.BF16 else x
    if wl.signed:
        assert (xf < 0).mean() > 0.4
    else:
        assert xf.min() == 0.0 and (xf == 0).mean() > 0.45
    union = np.unique(g["s"]).size
    if wl.exclude:
        assert union == wl.C - wl.exclude
    assert abs(float(g["a"].std()) - k ** -0.5) < 0.2 * k ** -0.5
