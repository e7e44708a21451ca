"""The parity tests' choice of token rows (CPU): rows from the oracle's own tile lists that
reach every tile-position class of the large-size cases."""
import numpy as np

import oracle
from paper_2607_23099_amd import synth
from tests.gpu_common import tile_rows


def test_tile_rows_cover_the_tile_classes():
    # The row choice itself: on a prefill-sized routing every listed class is present.
    sh = synth.DS
    r = synth.routing(sh.E, sh.k, 4096, 0.05, synth.seed_prefill(4096, 0.05, 0))
    rows = tile_rows(r, sh.E, seed=1)
    assert len(rows) >= 64 and len(np.unique(rows)) == len(rows)
    counts = oracle.histogram(r.ids, sh.E)
    offsets, perm, _ = oracle.permute(r.ids, sh.E)
    tok = set(rows.tolist())
    t256 = oracle.tiles(counts, 256)
    full = t256[t256[:, 2] == 256]
    s_ = int(full[len(full) // 2][0])
    assert int(perm[s_ + 128]) // sh.k in tok and int(perm[s_ + 255]) // sh.k in tok
    last = oracle.tiles(counts, 16)[-1]
    assert int(perm[last[0] + last[2] - 1]) // sh.k in tok
