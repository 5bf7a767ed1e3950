"""The cost model of Sec. 3.5 reproduces the figures the paper prints."""
import json
import os

import pytest

from paper_2608_23794_amd import cost

GOLD = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "paper_cost_figures.json")))


def _round(v, nd):
    return round(v + 0.0, nd)


@pytest.mark.parametrize("depth", ["50", "101", "152"])
def test_table1_macs_and_params(depth):
    g = GOLD["resnet"][depth]
    s = cost.resnet_replacement_summary(int(depth), k=8)
    assert s["layers"] == g["layers"]
    net = g["dense_gmacs"] * 1e9 - s["dense_macs"] + s["moce_macs"]
    assert _round(net / 1e9, 3) == g["moce_gmacs"]
    dense_params = cost.resnet_param_count(int(depth))
    assert _round(dense_params / 1e6, 2) == g["dense_params_m"]
    base = dense_params - s["replaced_weights"] + s["gate_params"]
    assert _round((base + s["deployed_logits"]) / 1e6, 2) == g["deploy_params_m"]
    assert _round((base + s["training_logits"]) / 1e6, 2) == g["train_params_m"]


def test_resnet50_replaced_operator_figures():
    g = GOLD["resnet50_replaced"]
    s = cost.resnet_replacement_summary(50, k=8)
    assert _round(s["dense_macs"] / 1e6, 1) == g["dense_mmacs"]
    assert _round(s["moce_macs"] / 1e6, 1) == g["moce_mmacs"]
    assert round(s["dense_macs"] / s["moce_macs"]) == g["reduction_x"]
    assert _round(100 * s["dense_macs"] / 4.112e9, 1) == g["share_pct"]
    net = 4.112e9 - s["dense_macs"] + s["moce_macs"]
    assert _round(100 * (1 - net / 4.112e9), 1) == g["network_reduction_pct"]
    p50 = cost.resnet_param_count(50)
    dep = p50 - s["replaced_weights"] + s["deployed_logits"] + s["gate_params"]
    assert _round(100 * (1 - dep / p50), 1) == g["deploy_param_reduction_pct"]
    assert _round(s["replaced_weights"] / 1e6, 2) == g["replaced_weights_m"]
    assert _round(s["deployed_logits"] / 1e3, 1) == g["deployed_logits_k"]
    assert round(s["index_bytes_16bit"] / 1e3) == g["index_kb_16bit"]
    assert _round(s["gate_macs"] / 1e9, 5) == g["gate_gmacs"]


def test_deeper_backbone_reductions():
    g = GOLD["reductions_pct"]
    for depth, dense in ((101, 7.834e9), (152, 11.559e9)):
        params = cost.resnet_param_count(depth)
        s = cost.resnet_replacement_summary(depth, k=8)
        net = dense - s["dense_macs"] + s["moce_macs"]
        dep = params - s["replaced_weights"] + s["deployed_logits"] + s["gate_params"]
        assert _round(100 * (1 - net / dense), 1) == g[f"{depth}_macs"]
        assert _round(100 * (1 - dep / params), 1) == g[f"{depth}_deploy_params"]


def test_break_even():
    g = GOLD["k_star"]
    assert round(cost.k_star(256, 64)) == g["C256_E64"]
    assert round(cost.k_star(2048, 512)) == g["C2048_E512"]
    assert round(cost.k_star(64, 64)) == g["C64_E64"]
    # at k*, Eq. 8 under |U| = C equals the dense cost exactly when k* is integral
    C, E = 63 * 4, 64
    k = cost.k_star(C, E)
    assert k == int(k) and cost.moce_macs(C, E, int(k), 1) == cost.dense_macs(C, E, 1)


def test_intensity_and_ratio():
    g = GOLD["intensity_2048_512_fp32"]
    dense, moce = cost.intensity_fp32(2048, 512, 8)
    assert round(dense) == g["dense_flop_per_byte"]
    assert round(moce, 1) == g["moce_flop_per_byte"]
    assert round(cost.dense_macs(2048, 512, 1) / cost.moce_macs(2048, 512, 8, 1)) == g["mac_reduction_x"]
    for C, E, k in ((256, 64, 8), (2048, 512, 8), (768, 192, 48)):
        assert cost.moce_macs(C, E, k, 1) / cost.dense_macs(C, E, 1) <= cost.ratio_bound(C, E, k)


def test_layer_traffic_stage1():
    t = cost.layer_traffic(64, 256, 64, 32, 56 * 56, 2)
    assert t["x"] == 102_760_448 and t["y"] == 25_690_112
    assert t["metric"] == 231_235_452
    assert t["compulsory"] == t["metric"] - t["x"]
