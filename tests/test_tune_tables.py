"""Host-side helpers of the offline tuner: the token-bucket grids and the merge of tables tuned
over disjoint token ranges (no GPU)."""
import os

import pytest

from paper_2607_23099_amd import damoe
from paper_2607_23099_amd.tune_tables import bucket_grid, merge_tables

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
KIMI = os.path.join(ROOT, "paper_2607_23099_amd", "tables", "kimi-k2.damoe")


def test_bucket_grids():
    assert bucket_grid(128) == [1, 2, 4, 8, 16, 32, 64, 128]
    half = bucket_grid(8192, "half")
    assert half[:10] == [1, 2, 3, 4, 6, 8, 12, 16, 24, 32] and half[-3:] == [4096, 6144, 8192]
    # Every T in [1, 8192] lies within 1.5x below the smallest bucket >= T.
    for T in range(1, 8193):
        b = next(x for x in half if x >= T)
        assert b < 1.5 * T + 1
    assert bucket_grid(3, "half") == [1, 2, 3]
    with pytest.raises(ValueError):
        bucket_grid(8, "third")


def _split(path, at, tmp_path):
    lines = open(path).read().splitlines()
    head, shape = lines[0], lines[1].split()
    blocks, i = [], 2
    while i < len(lines):
        n = int(lines[i].split()[2])
        blocks.append(lines[i:i + 1 + n])
        i += 1 + n
    out = []
    for name, part in (("lo", blocks[:at]), ("hi", blocks[at:])):
        p = tmp_path / f"{name}.damoe"
        p.write_text(head + "\n" + " ".join(shape[:5] + [str(len(part))]) + "\n" +
                     "\n".join(sum(part, [])) + "\n")
        out.append(str(p))
    return out


def test_merge_reassembles_a_split_table(tmp_path):
    lo, hi = _split(KIMI, 6, tmp_path)
    merged = tmp_path / "merged.damoe"
    merge_tables([lo, hi], str(merged))
    assert merged.read_text() == open(KIMI).read()
    damoe.Table.load(str(merged))


def test_merge_rejects_overlap_and_other_shapes(tmp_path):
    lo, hi = _split(KIMI, 6, tmp_path)
    with pytest.raises(ValueError):
        merge_tables([hi, lo], str(tmp_path / "x.damoe"))  # buckets out of order
    other = os.path.join(ROOT, "paper_2607_23099_amd", "tables", "dsv3.damoe")
    with pytest.raises(ValueError):
        merge_tables([lo, other], str(tmp_path / "y.damoe"))  # E = 384 vs 256
