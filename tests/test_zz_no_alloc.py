"""The allocation-free layer call against the two calls it stands for.

damoe_moe_layer_noalloc runs damoe_route_dispatch and then damoe_fused_moe with the
library's own fixed device array as their workspace.  On the same inputs it must give the same
routing outputs and the same y, bit for bit, as those two calls on a caller workspace; two calls
in a row, the second with fewer tokens, show that nothing of the first call's contents in the
shared array leaks into the second.
"""
import numpy as np
import pytest

from paper_2607_23099_amd import damoe, synth
from tests.gpu_common import log, torch_cuda

pytestmark = pytest.mark.gpu

SMALL_FP8 = synth.Shape("small-fp8", E=8, k=2, H=512, I=1024, shape_id=5, wdtype="fp8")


def _table(sh, kids, noda):
    rng = np.random.default_rng(17)
    q = -np.sort(-rng.integers(0, 1 << 15, (len(kids), sh.E)), axis=1).astype(np.int32)
    q[0] = 0
    q[0, 0] = 1 << 15  # a one-hot exemplar, so skewed routings pick kids[0]
    return damoe.Table.create(damoe.TableData(
        E=sh.E, k=sh.k, H=sh.H, I=sh.I, wdtype=0, bucket_T=np.array([1 << 20]), n_ex=np.array([len(kids)]),
        Q=q, kid=np.asarray(kids), noda=np.array([noda])))


def _outputs(path, T):
    return {n: getattr(path, n).clone() for n in ("counts", "offsets", "numden", "bucket", "variant")} | \
        {"perm": path.perm[:T * path.dl.shape.k].clone(), "inv_perm": path.inv_perm[:T * path.dl.shape.k].clone(),
         "y": path.y[:T].clone()}


@pytest.mark.parametrize("shape,kids,calls", [
    (synth.TINY, [7, 0, 3, 6], [(250, 0.05, 1), (37, 1.0, 2)]),
    (SMALL_FP8, [6, 1, 7], [(300, 0.05, 3), (64, 10.0, 4)]),
    (synth.TINY, [2, 4], [(2048, 0.3, 5), (1, 1.0, 6)]),  # the multi-block routing, then one token
], ids=["tiny", "small-fp8", "tiny-multiblock"])
def test_noalloc_equals_route_dispatch_then_fused(shape, kids, calls):
    torch = torch_cuda()
    from paper_2607_23099_amd.moe import DeviceLayer, Path
    dl = DeviceLayer(shape)
    sh = dl.shape
    table = _table(sh, kids, kids[-1])
    t_max = max(c[0] for c in calls)
    ref_path, path = Path(dl, t_max), Path(dl, t_max)
    for T, alpha, seed in calls:
        log(f"noalloc {shape.name} T={T} alpha={alpha}")
        r = synth.routing(sh.E, sh.k, T, alpha, [seed])
        for p in (ref_path, path):
            p.set_routing(r)
            p.fill_x(T, seed)
            p.y.fill_(float("nan"))
            p.perm.fill_(-5)
            p.inv_perm.fill_(-5)
            p.variant.fill_(-5)
        ref_path.route_dispatch(table, T)
        ref_path.fused(T, -1)
        damoe.moe_layer_noalloc(table, dl.layer, path.x, path.ids, path.w, T, path.counts, path.offsets, path.perm,
                                path.inv_perm, path.numden, path.bucket, path.variant, path.y)
        torch.cuda.synchronize()
        want, got = _outputs(ref_path, T), _outputs(path, T)
        for name in want:
            assert torch.equal(got[name].view(torch.int16) if name == "y" else got[name],
                               want[name].view(torch.int16) if name == "y" else want[name]), (name, T)
        assert int(got["variant"].item()) in kids
        assert bool(torch.isfinite(got["y"].float()).all())
        assert damoe.read_device_error(ref_path.ws) == 0


def test_noalloc_rejects_calls_beyond_its_array():
    # DeepSeek-V3 shape: T = 128 needs about 19 MB of workspace and fits; T = 512 needs about
    # 76 MB and is refused on the host before any launch, as is an invalid layer.
    torch = torch_cuda()
    sh = synth.DS
    lim = damoe.noalloc_scratch_bytes()
    lo_ok = damoe.workspace_layout(sh.E, sh.k, sh.H, sh.I, 128)
    lo_big = damoe.workspace_layout(sh.E, sh.k, sh.H, sh.I, 512)
    assert lo_ok["total"] <= lim < lo_big["total"]
    dummy = torch.zeros(16, dtype=torch.int32, device="cuda")
    layer = damoe.make_layer(sh.E, sh.k, sh.H, sh.I, damoe.W_BF16, dummy, dummy, dummy)
    table = damoe.Table.create(damoe.TableData(
        E=sh.E, k=sh.k, H=sh.H, I=sh.I, wdtype=0, bucket_T=np.array([1 << 20]), n_ex=np.array([1]),
        Q=np.full((1, sh.E), 2048, np.int32), kid=np.array([0]), noda=np.array([0])))
    with pytest.raises(damoe.DamoeError) as ei:
        damoe.moe_layer_noalloc(table, layer, dummy, dummy, dummy, 512, dummy, dummy, dummy, dummy, dummy, dummy,
                                dummy, dummy)
    assert ei.value.code == -3
    bad = damoe.make_layer(sh.E, sh.k + 1, sh.H, sh.I, damoe.W_BF16, dummy, dummy, dummy)
    with pytest.raises(damoe.DamoeError) as ei:
        damoe.moe_layer_noalloc(table, bad, dummy, dummy, dummy, 4, dummy, dummy, dummy, dummy, dummy, dummy,
                                dummy, dummy)
    assert ei.value.code == -4  # the table was built for another k
    torch.cuda.synchronize()
