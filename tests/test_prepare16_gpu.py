"""The 16-bit support storage (Sec. 3.5, Storage): moce_support_prepare16 on uint16 channel indices
gives the same prepared rows, covered flags, uncovered set and error reports as moce_support_prepare on
the same indices in int32, bit for bit."""
import numpy as np
import pytest
import torch

from paper_2608_23794_amd import binding as mb
from paper_2608_23794_amd import inputs

pytestmark = pytest.mark.gpu


def prep(fn, desc, s, w, C, R, k):
    dev = "cuda"
    s_out = torch.empty((R, k), dtype=torch.int32, device=dev)
    w_out = torch.empty((R, k), dtype=torch.float32, device=dev)
    covered = torch.empty(C, dtype=torch.uint8, device=dev)
    U = torch.zeros(C, dtype=torch.int32, device=dev)
    info = torch.empty(2, dtype=torch.int32, device=dev)
    st, nU, bad = fn(desc, s, w, s_out, w_out, covered, U, info, check=False)
    torch.cuda.synchronize()
    return st, nU, bad, s_out.cpu().numpy(), w_out.cpu().numpy(), covered.cpu().numpy(), U.cpu().numpy()[:max(nU, 0)]


@pytest.mark.parametrize("name", ["tiny", "resnet50_stage3", "resnet50_stage4", "vit_tokens"])
def test_prepare16_equals_prepare32(name):
    wl = inputs.WORKLOADS[name]
    g = inputs.generate(wl, wl.layouts[0], batch=1)
    R, k, C = wl.E - 1, wl.k, wl.C
    desc = mb.make_desc(1, C, wl.H, wl.W, wl.E, k, mb.MOCE_BF16, mb.MOCE_NHWC)
    s32 = torch.from_numpy(np.ascontiguousarray(g["s"], np.int32)).cuda()
    s16 = torch.from_numpy(np.ascontiguousarray(g["s"]).astype(np.uint16).view(np.int16)).cuda()
    w = torch.from_numpy(np.ascontiguousarray(g["w"], np.float32)).cuda()
    a = prep(mb.moce_support_prepare, desc, s32, w, C, R, k)
    b = prep(mb.moce_support_prepare16, desc, s16, w, C, R, k)
    assert a[0] == 0 and b[0] == 0
    assert a[1:3] == b[1:3]
    for u, v in zip(a[3:], b[3:]):
        np.testing.assert_array_equal(u, v)


def test_prepare16_reports_the_same_bad_row():
    C, E, k = 300, 9, 6
    rng = np.random.default_rng(0)
    s = np.array([rng.choice(C, k, replace=False) for _ in range(E - 1)], np.int64)
    s[5, 2] = s[5, 4]      # a repeated channel in row 5
    s[7, 0] = C + 3        # out of range in row 7
    w = rng.standard_normal((E - 1, k)).astype(np.float32)
    desc = mb.make_desc(1, C, 1, 1, E, k, mb.MOCE_F32, mb.MOCE_NCHW)
    wd = torch.from_numpy(w).cuda()
    a = prep(mb.moce_support_prepare, desc, torch.from_numpy(s.astype(np.int32)).cuda(), wd, C, E - 1, k)
    b = prep(mb.moce_support_prepare16, desc, torch.from_numpy(s.astype(np.uint16).view(np.int16)).cuda(), wd, C,
             E - 1, k)
    assert a[0] == b[0] == -5 and a[2] == b[2] == 5
