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
