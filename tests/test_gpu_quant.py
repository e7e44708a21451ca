"""GPU check of the fp8-MFMA variants' h quantisation: their GEMM1 (the big-tile kernel for
big8_bm256, the deep-ring kernel for deep8_bm64) writes h rounded to bf16, then as e4m3 codes with
one E8M0 scale per 32 features of a row (stage-major, in 4-byte words per 64 features).  The same
kernel with the bf16-h variant (big_bm256: h stage-major; deep_bm64: h row-major) stores the bf16 h
itself, from the same accumulation, so the codes and scales must equal those of the test-side MX
quantiser (tests/mx_ref.py, written from the OCP formats) applied to that bf16 h, bit for bit."""
import numpy as np
import pytest

from paper_2607_23099_amd import damoe, synth
from tests.gpu_common import log, torch_cuda
from tests.mx_ref import mx_quantise

pytestmark = pytest.mark.gpu

SMALL_FP8 = synth.Shape("small-fp8", E=8, k=2, H=512, I=1024, shape_id=5, wdtype="fp8")


@pytest.fixture(scope="module", params=[False, True], ids=["rowmajor", "packed"])
def small_fp8(request):
    torch = torch_cuda()
    from paper_2607_23099_amd.moe import DeviceLayer, Path
    dl = DeviceLayer(SMALL_FP8, packed=request.param)
    yield dl, Path(dl, 600)
    torch.cuda.empty_cache()


@pytest.mark.parametrize("pair", [("big_bm256", "big8_bm256"), ("deep_bm64", "deep8_bm64")], ids=["big", "deep"])
@pytest.mark.parametrize("T,alpha,seed", [(3, 1.0, 41), (100, 1.0, 42), (600, 0.05, 43)])
def test_h_quantised_bit_exact(small_fp8, pair, T, alpha, seed):
    torch = torch_cuda()
    dl, path = small_fp8
    sh = dl.shape
    names = [damoe.variant_name(v) for v in range(damoe.num_variants())]
    big, big8 = names.index(pair[0]), names.index(pair[1])
    r = synth.routing(sh.E, sh.k, T, alpha, [seed])
    path.set_routing(r)
    path.fill_x(T, seed)
    if T > 1:
        path.x[1] *= 1e6  # a row of large activations (h ~ 1e12): large scale exponents
    path.route(T)
    A = T * sh.k
    lo = damoe.workspace_layout(sh.E, sh.k, sh.H, sh.I, T)
    log(f"h quantisation T={T}: GEMM1 of {names[big]} then of {names[big8]}")
    path.fused_stage(0, T, big)
    torch.cuda.synchronize()
    # The big-tile kernel's h is stage-major in its GEMM2's stages, 64 columns with fp8
    # weights: [I / 64][A][64] bf16; the deep-ring kernel's is row-major [A][I].
    h = path.ws[lo["h"]: lo["h"] + A * sh.I * 2].view(torch.bfloat16).float().cpu().numpy()
    if pair[0] == "big_bm256":
        h = h.astype(np.float64).reshape(sh.I // 64, A, 64).transpose(1, 0, 2).reshape(A, sh.I)
    else:
        h = h.astype(np.float64).reshape(A, sh.I)
    path.fused_stage(0, T, big8)
    torch.cuda.synchronize()
    # Stage-major: codes [I / 64][A][64], scale words [I / 64][A][4] whose bytes 0 and 1 are the
    # scales of the two 32-feature blocks of the 64.
    q = path.ws[lo["h"]: lo["h"] + A * sh.I].cpu().numpy().reshape(sh.I // 64, A, 64)
    q = q.transpose(1, 0, 2).reshape(A, sh.I)
    s = path.ws[lo["h"] + A * sh.I: lo["h"] + A * sh.I + A * sh.I // 16].cpu().numpy().reshape(sh.I // 64, A, 4)
    s = s[:, :, :2].transpose(1, 0, 2).reshape(A, sh.I // 32)
    assert np.all(np.isfinite(h))
    q_ref, s_ref = mx_quantise(h)
    np.testing.assert_array_equal(s, s_ref)
    zero = (q_ref & 0x7F) == 0  # +0 and -0 both decode to zero
    np.testing.assert_array_equal(q[~zero], q_ref[~zero])
    assert np.all((q[zero] & 0x7F) == 0)
    assert damoe.read_device_error(path.ws) == 0
