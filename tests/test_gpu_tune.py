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
    from paper_2607_23099_amd.tune_tables import EXTENDED_SKEWS, tune_shape
    log("tuning the tiny layer")
    table, secs, buckets, dl = tune_shape("tiny", 64, samples=2, reps=2, seed=5, verbose=False)
    sh = dl.shape
    td = table.data(sh.E)
    assert list(td.bucket_T) == buckets == [1, 2, 4, 8, 16, 32, 64]
    assert list(td.n_ex) == [len(EXTENDED_SKEWS)] * len(buckets)
    nv = damoe.num_variants()
    assert td.kid.min() >= 0 and td.kid.max() < nv and td.noda.min() >= 0 and td.noda.max() < nv
    for q in td.Q:
        assert np.all(np.diff(q) <= 0)                          # sorted, descending
        assert abs(np.linalg.norm(q / 2 ** 15) - 1) < sh.E * 0.5 / 2 ** 15 + 1e-9
    # With enough tokens (T = 64 over 8 experts), a larger skew multiplier X concentrates the
    # exemplar: the most skewed grid point's top entry exceeds the least skewed one's.
    rows = td.bucket_rows(len(buckets) - 1)
    assert td.Q[rows][-1][0] > td.Q[rows][0][0]
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
