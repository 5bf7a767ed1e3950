"""Cost model of a MoCE layer (Sec. 3.5, Eqs. 8-10) and traffic accounting.

Host-side arithmetic only: MAC counts, the break-even support size, the
parameter counts of a deployed ResNet, and the byte counts used to price a
forward pass against the HBM roofline.
"""
from __future__ import annotations

from typing import Dict, List, Optional, Tuple


def dense_macs(C: int, E: int, HW: int) -> int:
    """Pointwise projection, Eq. 1: C*E MACs per position."""
    return C * E * HW


def moce_macs(C: int, E: int, k: int, HW: int, n_uncovered: Optional[int] = None,
              gate_macs: int = 0) -> int:
    """Eq. 8: routed mixing + pooling + residual + gate.

    ``n_uncovered=None`` takes the conservative bound |U| = C used by the
    paper's reported totals.
    """
    u = C if n_uncovered is None else n_uncovered
    return ((E - 1) * k + C + u) * HW + gate_macs


def ratio_bound(C: int, E: int, k: int) -> float:
    """Eq. 9: M_MoCE / M_dense <~ k/C + 2/E."""
    return k / C + 2.0 / E


def k_star(C: int, E: int) -> float:
    """Eq. 10: the support size at which MoCE costs as much as the dense map."""
    return C * (E - 2) / (E - 1)


def gate_mlp_macs(E: int, k: int) -> int:
    """The shared two-layer gate (hidden width k, scalar output) per example."""
    return (E - 1) * (k * k + k)


_BLOCKS = {50: (3, 4, 6, 3), 101: (3, 4, 23, 3), 152: (3, 8, 36, 3)}
_WIDTH = (64, 128, 256, 512)
_RES = (56, 28, 14, 7)


def resnet_entrance_projections(depth: int) -> List[Tuple[int, int, int]]:
    """(C_in, C_out, H*W) of every bottleneck entrance 1x1 projection.

    Each stage's first projection is counted at the stage's output
    resolution, the accounting under which the paper's Table 1 totals
    reproduce.
    """
    out = []
    c_in = 64
    for stage, n in enumerate(_BLOCKS[depth]):
        width = _WIDTH[stage]
        hw = _RES[stage] ** 2
        for blk in range(n):
            out.append((c_in, width, hw))
            c_in = width * 4
    return out


def resnet_param_count(depth: int, classes: int = 1000) -> int:
    """Learned values of a bottleneck ResNet (convolutions, BatchNorm affine, fc)."""
    n = 7 * 7 * 3 * 64 + 2 * 64
    c_in = 64
    for stage, blocks in enumerate(_BLOCKS[depth]):
        w = _WIDTH[stage]
        for blk in range(blocks):
            n += c_in * w + 2 * w + 9 * w * w + 2 * w + w * 4 * w + 2 * 4 * w
            if blk == 0:
                n += c_in * 4 * w + 2 * 4 * w
            c_in = 4 * w
    return n + c_in * classes + classes


def resnet_replacement_summary(depth: int, k: int = 8) -> Dict[str, float]:
    layers = resnet_entrance_projections(depth)
    dense = sum(dense_macs(C, E, hw) for C, E, hw in layers)
    moce = sum(moce_macs(C, E, k, hw) for C, E, hw in layers)
    gate = sum(gate_mlp_macs(E, k) for C, E, _ in layers)
    weights = sum(C * E for C, E, _ in layers)
    logits_deployed = sum((E - 1) * k for C, E, _ in layers)
    logits_training = sum((E - 1) * C for C, E, _ in layers)
    gate_params = len(layers) * (k * k + 2 * k + 1)
    return {
        "layers": len(layers),
        "dense_macs": dense,
        "moce_macs": moce,
        "gate_macs": gate,
        "replaced_weights": weights,
        "deployed_logits": logits_deployed,
        "index_bytes_16bit": 2 * logits_deployed,
        "training_logits": logits_training,
        "gate_params": gate_params,
    }


def intensity_fp32(C: int, E: int, k: int) -> Tuple[float, float]:
    """FLOP per byte of activation traffic (C+E)*HW*4 for dense and MoCE (Sec. 3.5)."""
    bytes_per_pos = (C + E) * 4
    dense = 2.0 * C * E / bytes_per_pos
    moce = 2.0 * ((E - 1) * k + 2 * C) / bytes_per_pos
    return dense, moce


def layer_traffic(B: int, C: int, E: int, k: int, HW: int, elem_bytes: int) -> Dict[str, int]:
    """Byte counts of one forward pass over a batch.

    ``metric`` counts two reads of x (pooling, then the gather), the write of
    y and the parameters (int32 support, float32 logits, slopes, offsets).
    ``compulsory`` counts x once: the least any implementation must move.
    """
    x = B * C * HW * elem_bytes
    y = B * E * HW * elem_bytes
    params = (E - 1) * k * 12 + (E - 1) * 4
    return {"x": x, "y": y, "params": params, "metric": 2 * x + y + params,
            "compulsory": x + y + params}


def layer_flops(B: int, E: int, k: int, HW: int, n_uncovered: int, C: int) -> Dict[str, int]:
    fma = B * HW * (E - 1) * k
    return {"mix_fma": fma, "pool_add": B * C * HW, "residual_add": B * HW * n_uncovered}
