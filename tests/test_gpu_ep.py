"""GPU parity of expert-parallel rank layers: one rank's experts as views into the full layer,
its share of a global routing with masked slots (the experts of other ranks), every variant
against the CPU oracle on the rank's partial sums (Sec. V-F runs the fused layer per rank)."""
import numpy as np
import pytest

from paper_2607_23099_amd import damoe, synth
from tests.gpu_common import TOL, bf16_rows, log, oracle_rows, row_err, torch_cuda

pytestmark = pytest.mark.gpu

SMALL = synth.Shape("small16", E=16, k=4, H=256, I=512, shape_id=7)


def _rank_case(full_shape, dl, ep, rank, T, alpha, seed, rows=None, extra_masked=()):
    """Runs every variant on one rank's share; returns the worst row error against the oracle."""
    torch = torch_cuda()
    from paper_2607_23099_amd.moe import Path, RankLayer
    el = full_shape.E // ep
    local_shape = synth.Shape(f"{full_shape.name}-ep{ep}", E=el, k=full_shape.k, H=full_shape.H,
                              I=full_shape.I, shape_id=full_shape.shape_id, wdtype=full_shape.wdtype)
    rl = RankLayer(dl, ep, rank, local_shape)
    r = synth.routing(full_shape.E, full_shape.k, T, alpha, seed)
    keep, ids, w = synth.ep_local(r, ep, rank)
    for t in extra_masked:  # whole tokens whose every slot is remote
        ids[t] = -1
    tl = len(keep)
    rl_routing = synth.Routing(ids, w, None, el, full_shape.k, alpha)
    path = Path(rl, max(tl, 1))
    src = synth.ExpertWeightSource(full_shape)
    rows = np.arange(tl) if rows is None else np.asarray(rows)
    ref = oracle_rows(local_shape, rl_routing, 70 + rank, rows, lambda e: src(rl.global_expert(e)))
    worst = 0.0
    for v in range(damoe.num_variants()):
        if not damoe.variant_supports(v, rl.wdtype):
            continue
        path.set_routing(rl_routing)
        path.fill_x(tl, 70 + rank)
        path.y.fill_(float("nan"))
        path.route(tl)
        path.fused(tl, v)
        torch.cuda.synchronize()
        y = bf16_rows(path.y, rows)
        for t in extra_masked:
            if t in rows:
                assert np.all(y[list(rows).index(t)] == 0.0)
        worst = max(worst, row_err(y, ref))
    assert damoe.read_device_error(path.ws) == 0  # masked slots are not errors
    return worst, tl


@pytest.mark.parametrize("ep", [2, 4])
def test_small_rank_layers_every_variant(ep):
    torch = torch_cuda()
    from paper_2607_23099_amd.moe import DeviceLayer
    dl = DeviceLayer(SMALL)
    for rank in range(ep):
        err, tl = _rank_case(SMALL, dl, ep, rank, 60, 0.5, [31, ep, rank], extra_masked=(1,))
        log(f"small16 ep={ep} rank={rank}: {tl} local tokens, worst row error {err:.2e}")
        assert err <= TOL["bf16"]
    del dl
    torch.cuda.empty_cache()


def test_dsv3_rank_layer_ep4():
    torch = torch_cuda()
    from paper_2607_23099_amd.moe import DeviceLayer
    log("filling DeepSeek-V3-shaped bf16 layer (22.5 GB) for its EP=4 ranks")
    dl = DeviceLayer(synth.DS)
    err, tl = _rank_case(synth.DS, dl, 4, 2, 128, 1.0, synth.seed_ep(128, 0), rows=[0, 7, 19])
    log(f"dsv3 ep=4 rank=2: {tl} local tokens, worst row error {err:.2e}")
    assert err <= TOL["bf16"]
    del dl
    torch.cuda.empty_cache()
