"""Shared helpers of the GPU parity tests (the HIP path vs the CPU oracle)."""
import numpy as np

import oracle
from paper_2607_23099_amd import damoe, synth

# Tolerances on y, row-normalised max error (bf16 / fp8 weights, fp32 accumulation).
TOL = {"bf16": 2e-2, "fp8": 6e-2}


def torch_cuda():
    import torch
    if not torch.cuda.is_available():
        raise RuntimeError("GPU tests need a ROCm GPU")
    return torch


def log(msg):
    print(msg, flush=True)


def row_err(y_gpu: np.ndarray, y_ref: np.ndarray) -> float:
    """max over rows of max|y - y_ref| / max|y_ref| (rows with y_ref == 0 must be exactly 0)."""
    worst = 0.0
    for g, r in zip(y_gpu, y_ref):
        m = np.max(np.abs(r))
        d = np.max(np.abs(g - r))
        worst = max(worst, d / m if m > 0 else (0.0 if d == 0 else np.inf))
    return worst


def oracle_rows(shape: synth.Shape, r: synth.Routing, x_tag: int, rows, src=None) -> np.ndarray:
    rows = np.asarray(rows, np.int64)
    x_rows = synth.activations_host(r.T, shape.H, x_tag, rows)
    ids_sub = r.ids[rows]
    experts = np.unique(ids_sub[(ids_sub >= 0) & (ids_sub < shape.E)])
    # moe_rows takes the full ids/w and row indices; pass local copies restricted to the rows.
    return oracle.moe_rows(ids_sub, r.w[rows], shape.k, np.arange(len(rows)), x_rows, shape.H, shape.I,
                           experts, src or synth.ExpertWeightSource(shape))


def bf16_rows(y_tensor, rows) -> np.ndarray:
    import torch
    idx = torch.as_tensor(np.asarray(rows, np.int64), device=y_tensor.device)
    return y_tensor.index_select(0, idx).float().cpu().numpy().astype(np.float64)


def tiles_expected(counts, bm):
    t = oracle.tiles(counts, bm)
    return np.stack([t[:, 0], t[:, 1] | (t[:, 2] << 16)], axis=1).astype(np.int64) if len(t) else \
        np.zeros((0, 2), np.int64)


def one_bucket_table(sh, kids, noda):
    """A one-bucket dispatch table whose exemplars map to `kids` (scored on every call)."""
    rng = np.random.default_rng(7)
    q = -np.sort(-rng.integers(0, 1 << 15, (len(kids), sh.E)), axis=1).astype(np.int32)
    return damoe.Table.create(damoe.TableData(E=sh.E, k=sh.k, H=sh.H, I=sh.I, wdtype=0,
                                              bucket_T=np.array([1 << 20]), n_ex=np.array([len(kids)]),
                                              Q=q, kid=np.asarray(kids), noda=np.array([noda])))


def tile_rows(r: synth.Routing, E: int, n_min: int = 64, seed: int = 0) -> np.ndarray:
    """Token rows whose outputs cover the tile-position classes of every tile size.

    The tiles are the oracle's (``oracle.tiles`` over its histogram, positions through its
    permutation), not the GPU's.  For each tile size BM in {16, 32, 64, 128, 256}:
      * the first and last row of the first tile, of the last tile (the last work-queue chunk
        of the large-tile kernels) and of the first full tile;
      * the rows of the hottest expert's last (ragged) tile: all of them up to 16, else 16
        spread over it, both ends included;
      * for BM = 256, the first and last row of token blocks 4..7 (rows 128..255) of a full
        256-row tile;
    then the position of a one-token expert, if any, and random rows up to n_min.  The tokens
    of these positions (position p holds assignment perm[p], token perm[p] // k) are returned,
    sorted and unique; every row when T <= n_min."""
    T, k = r.T, r.k
    if T <= n_min:
        return np.arange(T)
    counts = oracle.histogram(r.ids, E)
    offsets, perm, _ = oracle.permute(r.ids, E)
    pos = set()
    hot = int(np.argmax(counts))
    for cls in range(5):
        bm = 16 << cls
        t = oracle.tiles(counts, bm)  # rows of (start, expert, rows)
        if not len(t):
            continue
        full = t[t[:, 2] == bm]
        for s_, _, n_ in [t[0], t[-1]] + ([full[0]] if len(full) else []):
            pos.update((int(s_), int(s_ + n_ - 1)))
        last_hot = t[t[:, 1] == hot][-1]
        n_ = int(last_hot[2])
        pos.update(int(last_hot[0]) + np.unique(np.linspace(0, n_ - 1, min(n_, 16)).round().astype(int)))
        if bm == 256 and len(full):
            s_ = int(full[len(full) // 2][0])
            for blk in range(4, 8):
                pos.update((s_ + 32 * blk, s_ + 32 * blk + 31))
    ones = np.flatnonzero(counts == 1)
    if len(ones):
        pos.add(int(offsets[ones[0]]))
    rows = set(int(perm[p]) // k for p in pos)
    rng = np.random.default_rng([int(seed), T])
    extra = rng.permutation(T)
    i = 0
    while len(rows) < n_min:
        rows.add(int(extra[i]))
        i += 1
    return np.array(sorted(rows), np.int64)


class Reference:
    """Oracle outputs of several cases of one layer shape, from one expert-major pass.

    Each case is (routing, x rows, row indices); the rows of all cases become the token rows
    of one call of ``oracle.moe_rows``, so each expert's weights are regenerated once for all
    of them.  ``y[name]`` holds a case's reference rows (fp64)."""

    def __init__(self, shape: synth.Shape, cases: dict, src=None):
        names = list(cases)
        ids, w, x, sizes = [], [], [], []
        for n in names:
            r, x_rows, rows = cases[n]
            ids.append(r.ids[rows])
            w.append(r.w[rows])
            x.append(x_rows)
            sizes.append(len(rows))
        ids = np.concatenate(ids)
        w = np.concatenate(w)
        x = np.concatenate(x)
        experts = np.unique(ids[(ids >= 0) & (ids < shape.E)])
        src = src or synth.ExpertWeightSource(shape)
        seen = [0]

        def weights(e):
            seen[0] += 1
            if seen[0] % 64 == 0:
                log(f"  oracle {shape.name}: expert {seen[0]} of {len(experts)}")
            return src(e)

        log(f"oracle {shape.name}: {len(names)} cases, {len(ids)} token rows, {len(experts)} experts")
        y = oracle.moe_rows(ids, w, shape.k, np.arange(len(ids)), x, shape.H, shape.I, experts, weights)
        self.rows = {n: cases[n][2] for n in names}
        self.y = {}
        o = 0
        for n, m in zip(names, sizes):
            self.y[n] = y[o:o + m]
            o += m


def variants_agree(y_a, y_b, T: int) -> float:
    """Row-normalised max difference of two GPU outputs over all T rows (on the device)."""
    a = y_a[:T].float()
    b = y_b[:T].float()
    d = (a - b).abs().amax(dim=1)
    m = b.abs().amax(dim=1)
    bad = (m == 0) & (d > 0)
    if bool(bad.any()):
        return float("inf")
    return float((d / m.clamp_min(1e-30)).max().item())
