"""The whole a2-a8 path captured in one HIP graph per token count (Sec. IV-C: the choice
stays on the device, so the kernel sequence is fixed and capturable).

Every replay is checked against an eager call of the same routing; the routing and the
activations change between replays (eager work in between), and replays repeat."""
import numpy as np
import pytest

from paper_2607_23099_amd import damoe, synth
from tests.gpu_common import TOL, bf16_rows, log, one_bucket_table, oracle_rows, row_err, torch_cuda

pytestmark = pytest.mark.gpu


# T = 4100 routes its 8200 assignments in blocks of 2048 (three launches in the graph, the last
# block ragged).
@pytest.mark.parametrize("kids,noda,T", [([0, 1, 3], 0, 96), ([6, 7, 6], 7, 96), ([2], 2, 96),
                                         ([0, 1, 3], 0, 4100), ([6, 7, 6], 7, 4100)],
                         ids=["stream-variants", "tiled-and-big", "single-variant",
                              "stream-variants-blocks", "tiled-and-big-blocks"])
def test_graph_replays_match_eager(kids, noda, T):
    torch = torch_cuda()
    from paper_2607_23099_amd.moe import DeviceLayer, Path
    sh = synth.TINY
    dl = DeviceLayer(sh, packed=True)
    path = Path(dl, max(T, 256))
    table = one_bucket_table(sh, kids, noda)
    routings = [synth.routing(sh.E, sh.k, T, a, [40 + i]) for i, a in enumerate((1.0, 0.05, 10.0, 0.3))]

    # Eager reference of every routing.
    eager, chosen = [], []
    for i, r in enumerate(routings):
        path.set_routing(r)
        path.fill_x(T, 40 + i)
        path.route_dispatch(table, T)
        path.fused(T, -1)
        torch.cuda.synchronize()
        eager.append(path.y[:T].clone())
        chosen.append(int(path.variant.item()))
    log(f"graph test kids={kids} T={T}: eager variants {chosen}")

    # Capture once on a side stream (the calls run on torch's current stream).
    path.set_routing(routings[0])
    path.fill_x(T, 40)
    g = torch.cuda.CUDAGraph()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        path.route_dispatch(table, T)  # warm-up outside the capture
        path.fused(T, -1)
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    with torch.cuda.graph(g, stream=s):
        path.route_dispatch(table, T)
        path.fused(T, -1)
    torch.cuda.synchronize()

    for rep in range(3):
        for i, r in enumerate(routings):
            path.set_routing(r)        # eager work between replays
            path.fill_x(T, 40 + i)
            path.y.fill_(float("nan"))
            torch.cuda.synchronize()
            g.replay()
            torch.cuda.synchronize()
            assert int(path.variant.item()) == chosen[i], (rep, i)
            assert torch.equal(path.y[:T], eager[i]), (rep, i)
    assert damoe.read_device_error(path.ws) == 0

    # And the eager result is the layer itself.
    ref = oracle_rows(sh, routings[1], 41, np.arange(T))
    assert row_err(bf16_rows(eager[1], np.arange(T)), ref) <= TOL["bf16"]
