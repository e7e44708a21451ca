"""damoe_tune on the GPU: the table it builds is well formed and drives dispatch.

The kernel choices depend on timings (parity unpinned); the exemplars are
checked for the properties the construction fixes (sorted, unit L2 norm up to
quantisation, skew ordered by the ddist:X grid).
"""
import numpy as np
import pytest

import oracle
from paper_2607_23099_amd import damoe, synth
from tests.gpu_common import TOL, bf16_rows, log, oracle_rows, row_err, torch_cuda

pytestmark = pytest.mark.gpu


def test_tune_tiny_table(tmp_path):
    torch = torch_cuda()
    from paper_2607_23099_amd.moe import DeviceLayer, Path
    from paper_2607_23099_amd.tune_tables import EXTENDED_SKEWS, REPEAT_F, tune_shape
    log("tuning the tiny layer")
    table, secs, buckets, dl = tune_shape("tiny", 64, samples=2, reps=2, seed=5, verbose=False)
    sh = dl.shape
    td = table.data(sh.E)
    nsk = len(EXTENDED_SKEWS)
    assert list(td.bucket_T) == buckets == [1, 2, 4, 8, 16, 32, 64]
    assert list(td.n_ex) == [nsk + len(REPEAT_F)] * len(buckets)
    # Repeated-row exemplars follow the skews'.  At f = 100 every token of a sample takes one
    # row, so each sample's sorted histogram is k equal counts: the exemplar is k entries of
    # 2^15 / sqrt(k), then zeros, in every bucket.
    assert REPEAT_F[-1] == 100
    step = np.zeros(sh.E, np.int64)
    step[:sh.k] = int(np.rint(2 ** 15 / np.sqrt(sh.k)))
    for b in range(len(buckets)):
        np.testing.assert_array_equal(td.Q[td.bucket_rows(b)][nsk + len(REPEAT_F) - 1], step)
    nv = damoe.num_variants()
    assert td.kid.min() >= 0 and td.kid.max() < nv and td.noda.min() >= 0 and td.noda.max() < nv
    for q in td.Q:
        assert np.all(np.diff(q) <= 0)                          # sorted, descending
        assert abs(np.linalg.norm(q / 2 ** 15) - 1) < sh.E * 0.5 / 2 ** 15 + 1e-9
    # With enough tokens (T = 64 over 8 experts), a larger skew multiplier X concentrates the
    # exemplar: the most skewed grid point's top entry exceeds the least skewed one's.
    rows = td.bucket_rows(len(buckets) - 1)
    assert td.Q[rows][nsk - 1][0] > td.Q[rows][0][0]
    # Save / load round trip, then adaptive dispatch with the tuned table.
    p = str(tmp_path / "tiny.damoe")
    table.save(p)
    t2 = damoe.Table.load(p)
    np.testing.assert_array_equal(t2.data(sh.E).Q, td.Q)
    path = Path(dl, 64)
    r = synth.routing(sh.E, sh.k, 50, 0.2, [31])
    path.set_routing(r)
    path.fill_x(50, 31)
    path.route_dispatch(t2, 50)
    path.fused(50, -1)
    torch.cuda.synchronize()
    c = oracle.histogram(r.ids, sh.E)
    i, _ = oracle.match(c, td.Q[td.bucket_rows(oracle.select_bucket(td.bucket_T, 50))])
    assert int(path.variant.item()) == int(td.kid[td.bucket_rows(6)][i])
    ref = oracle_rows(sh, r, 31, np.arange(50))
    assert row_err(bf16_rows(path.y, np.arange(50)), ref) <= TOL["bf16"]
    # A batch of one repeated row scores the f = 100 exemplar at its maximum (cosine 1); the
    # device picks what the oracle's match picks.  (With E = 8 and k = 2 the most skewed
    # Dirichlet exemplars are step-shaped as well, so the winner may be one of them.)
    rr = synth.routing_repeated(sh.E, sh.k, 50, 100, 1.0, [32])
    path.set_routing(rr)
    path.route_dispatch(t2, 50)
    torch.cuda.synchronize()
    ch = oracle.histogram(rr.ids, sh.E)
    i, scores = oracle.match(ch, td.Q[td.bucket_rows(6)])
    assert scores[i] == scores.max() >= int(np.dot(np.sort(ch)[::-1].astype(np.int64), step))
    assert int(path.variant.item()) == int(td.kid[td.bucket_rows(6)][i])


def test_tune_expert_parallel_rank():
    # ep > 1: samples are one rank's share of routings over E * ep experts (remote slots
    # masked); the table is well formed and its exemplars come from the rank's histograms.
    torch = torch_cuda()
    from paper_2607_23099_amd.moe import DeviceLayer
    sh = synth.Shape("small-rank", E=4, k=4, H=256, I=512, shape_id=7)
    dl = DeviceLayer(sh)
    x = torch.empty((16, sh.H), dtype=torch.bfloat16, device="cuda")
    synth.fill_bf16_device(x.data_ptr(), x.numel(), seed=synth.x_seed(3), tensor=synth.T_X, slab_elems=x.numel(),
                           sigma=1.0, stream=torch.cuda.current_stream().cuda_stream)
    table = damoe.tune(dl.layer, [1, 4, 16], [1.1, 4.0], x, samples=2, reps=1, seed=9, ep=4)
    td = table.data(sh.E)
    nv = damoe.num_variants()
    assert list(td.bucket_T) == [1, 4, 16] and list(td.n_ex) == [2, 2, 2]
    assert td.kid.min() >= 0 and td.kid.max() < nv and td.noda.max() < nv
    for q in td.Q:
        assert np.all(np.diff(q) <= 0) and q[0] > 0
    with pytest.raises(damoe.DamoeError):
        damoe.tune(dl.layer, [1], [1.1], x, samples=1, reps=1, ep=-1)
    with pytest.raises(damoe.DamoeError):  # repeated rows are not combined with expert parallelism
        damoe.tune(dl.layer, [1], [1.1], x, samples=1, reps=1, ep=4, repeat_f=[50])
    del dl
    torch.cuda.empty_cache()
