"""The fragment-packed weight layout: the pack kernel is a pure relayout.

Block (rb, kb) of 16 rows x 32 columns of a row-major [rows][cols] matrix becomes 64 lanes x
8 elements at block index rb * (cols / 32) + kb, lane l holding row 16 rb + l % 16 and columns
32 kb + 8 (l / 16) .. + 7: numpy's reshape / transpose of the host weights must give the
device result bit for bit.
"""
import numpy as np
import pytest

from paper_2607_23099_amd import damoe, synth
from tests.gpu_common import torch_cuda

pytestmark = pytest.mark.gpu


def pack_reference(m: np.ndarray) -> np.ndarray:
    rows, cols = m.shape
    # [rb][r][kb][g][8] -> [rb][kb][g][r][8]; lane = g * 16 + r
    return m.reshape(rows // 16, 16, cols // 32, 4, 8).transpose(0, 2, 3, 1, 4).reshape(-1)


@pytest.mark.parametrize("shape", [synth.TINY, synth.Shape("pack-fp8", E=3, k=2, H=512, I=1024, shape_id=7,
                                                           wdtype="fp8")], ids=["bf16", "fp8"])
def test_pack_matches_reshape(shape):
    torch = torch_cuda()
    from paper_2607_23099_amd.moe import DeviceLayer
    rm = DeviceLayer(shape, packed=False)
    pk = DeviceLayer(shape, packed=True)
    torch.cuda.synchronize()
    for name in ("w1", "w3", "w2"):
        a = rm.w[name].view(torch.uint8).cpu().numpy()
        b = pk.w[name].view(torch.uint8).cpu().numpy()
        eb = 1 if shape.wdtype == "fp8" else 2
        _, r, c = synth.weight_dims(shape, name)
        for e in range(shape.E):
            src = a[e].reshape(r, c * eb)
            if eb == 2:
                src = src.view(np.uint16)
            want = pack_reference(src).view(np.uint8)
            np.testing.assert_array_equal(b[e].reshape(-1), want)
        if shape.wdtype == "fp8":
            np.testing.assert_array_equal(rm.s[name].cpu().numpy(), pk.s[name].cpu().numpy())
