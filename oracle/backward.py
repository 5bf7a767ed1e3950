"""CPU reference gradients of the static layer and of the coverage loss.

TEST INFRASTRUCTURE ONLY (see the package docstring).  Plain numpy in float64, the chain rule written
out step by step over the forward of Sec. 3 (GAP descriptor, gate, softmax of Eq. 4 over the selected
logits, routed sum of Eq. 5, residual mean of Eq. 6) and over the coverage loss of Eq. 7.  The
selection itself (the static top-k supports of Eq. 2) is fixed: gradients reach the selected logits
w = L[e, s_e], and the full logits L only through the coverage loss.
"""
from __future__ import annotations

from typing import Dict

import numpy as np

from . import NCHW, prepare


def _x64(x: np.ndarray) -> np.ndarray:
    if x.dtype == np.uint16:
        return (x.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    return x.astype(np.float64)


def _planes(a: np.ndarray, layout: int) -> np.ndarray:
    """[B, C, HW] view of an NCHW or channels-last tensor."""
    B = a.shape[0]
    if layout == NCHW:
        return a.reshape(B, a.shape[1], -1)
    return np.moveaxis(a.reshape(B, -1, a.shape[-1]), 2, 1)


def _unplanes(p: np.ndarray, shape, layout: int) -> np.ndarray:
    if layout == NCHW:
        return p.reshape(shape)
    return np.moveaxis(p, 1, 2).reshape(shape)


def _sigmoid(t):
    return 1.0 / (1.0 + np.exp(-t))


def layer_backward(x: np.ndarray, s: np.ndarray, w: np.ndarray, E: int, dy: np.ndarray, layout: int = NCHW,
                   gate: str = "softplus", a=None, c=None, W1=None, b1=None, w2=None, b2=0.0, tau_min=0.2,
                   tau_max=6.0) -> Dict[str, np.ndarray]:
    """Gradients of l = sum(dy * y) for the static layer y = MoCE(x).

    Returns dx (the layout of x), dw [E-1, k] for the rows as given (any order), and the gate's:
    da [E-1, k], dc [E-1] (softplus-linear) or dW1 [k, k], db1 [k], dw2 [k], db2 (MLP)."""
    X = _planes(_x64(x), layout)                      # [B, C, HW]
    B, C, HW = X.shape
    R = E - 1
    s_c, w_c, covered, U, nU = prepare(C, E, s, w)    # canonical rows (gate positions)
    k = s_c.shape[1] if R > 0 else 0
    DY = _planes(dy.astype(np.float64), layout)       # [B, E, HW]
    dX = np.zeros_like(X)
    out = {}
    if R > 0:
        wc = w_c.astype(np.float64)
        d = X.mean(axis=2)                            # GAP descriptor [B, C]
        z = d[:, s_c]                                 # [B, R, k] gate inputs
        tmin, tmax = float(np.float32(tau_min)), float(np.float32(tau_max))   # float32 parameters
        if gate == "softplus":
            g = c.astype(np.float64)[None, :] + np.einsum("ei,bei->be", a.astype(np.float64), z)
            tau = np.logaddexp(0.0, g) + 1e-3
        else:
            hpre = np.einsum("ji,bei->bej", W1.astype(np.float64), z) + b1.astype(np.float64)
            hr = np.maximum(hpre, 0.0)
            g = np.einsum("j,bej->be", w2.astype(np.float64), hr) + float(np.float32(b2))
            sg = _sigmoid(g)
            tau = tmin + (tmax - tmin) * sg
        zz = wc[None] / tau[:, :, None]               # softmax argument
        zz = zz - zz.max(axis=2, keepdims=True)
        alpha = np.exp(zz)
        alpha /= alpha.sum(axis=2, keepdims=True)     # [B, R, k]
        # routed outputs y[b, e, p] = sum_i alpha[b, e, i] X[b, s[e, i], p]
        Xs = X[:, s_c, :]                             # [B, R, k, HW]
        dalpha = np.einsum("bep,beip->bei", DY[:, :R, :], Xs)
        # softmax: alpha = softmax(w / tau)
        dzz = alpha * (dalpha - (alpha * dalpha).sum(axis=2, keepdims=True))
        dw_c = (dzz / tau[:, :, None]).sum(axis=0)    # [R, k]
        dtau = -(dzz * wc[None]).sum(axis=2) / tau ** 2
        if gate == "softplus":
            dg = dtau * _sigmoid(g)
            out["da"] = np.einsum("be,bei->ei", dg, z)
            out["dc"] = dg.sum(axis=0)
            dz = dg[:, :, None] * a.astype(np.float64)[None]
        else:
            dg = dtau * (tmax - tmin) * sg * (1.0 - sg)
            out["dw2"] = np.einsum("be,bej->j", dg, hr)
            out["db2"] = float(dg.sum())
            dh = dg[:, :, None] * w2.astype(np.float64)[None, None, :] * (hpre > 0)
            out["dW1"] = np.einsum("bej,bei->ji", dh, z)
            out["db1"] = dh.sum(axis=(0, 1))
            dz = np.einsum("bej,ji->bei", dh, W1.astype(np.float64))
        # the gate inputs back to the descriptor, the descriptor back to x
        dd = np.zeros((B, C))
        for e in range(R):
            np.add.at(dd, (slice(None), s_c[e]), dz[:, e, :])
        dX += dd[:, :, None] / HW
        # the routed sums back to x
        for e in range(R):
            np.add.at(dX, (slice(None), s_c[e], slice(None)), alpha[:, e, :, None] * DY[:, e, None, :])
        # dw for the rows in the caller's order
        dw = np.zeros((R, k))
        for e in range(R):
            pos = {int(ch): i for i, ch in enumerate(s_c[e])}
            for j in range(k):
                dw[e, j] = dw_c[e, pos[int(s[e, j])]]
        out["dw"] = dw
        out["tau"], out["alpha"], out["s_canon"] = tau, alpha, s_c
    if nU > 0:
        dX[:, U, :] += DY[:, R, None, :] / nU
    out["dx"] = _unplanes(dX, x.shape, layout)
    return out


def coverage_loss(L: np.ndarray, eps: float) -> float:
    """Eq. 7: p[e, c] = softmax_c(L[e]), u[c] = mean_e p[e, c], mean u over c, squared deviations
    over (mean u)^2 + eps."""
    L = L.astype(np.float64)
    p = np.exp(L - L.max(axis=1, keepdims=True))
    p /= p.sum(axis=1, keepdims=True)
    u = p.mean(axis=0)
    ub = u.mean()
    return float(((u - ub) ** 2).sum() / (ub ** 2 + eps))


def coverage_grad(L: np.ndarray, eps: float) -> np.ndarray:
    """dL_cov / dL [E-1, C]: the loss through u (ub a function of u too), u through each row's
    softmax (u_c = mean over rows of p[e, c])."""
    L = L.astype(np.float64)
    R, C = L.shape
    p = np.exp(L - L.max(axis=1, keepdims=True))
    p /= p.sum(axis=1, keepdims=True)
    u = p.mean(axis=0)
    ub = u.mean()
    den = ub ** 2 + eps
    num = ((u - ub) ** 2).sum()
    # num = sum_c (u_c - ub)^2 with ub = mean u: d num / d u_c = 2 (u_c - ub), since the deviations
    # sum to zero; den = ub^2 + eps: d den / d u_c = 2 ub / C
    du = 2.0 * (u - ub) / den - num * (2.0 * ub / C) / den ** 2
    dp = np.broadcast_to(du / R, (R, C))
    return p * (dp - (p * dp).sum(axis=1, keepdims=True))
