"""CPU oracle of the distribution-aware fused-MoE path (test infrastructure).

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package.  It is a thin ctypes wrapper over
``oracle.c`` (plain C, fp64) and imports nothing from the HIP path.
"""
from __future__ import annotations

import ctypes
import os
import shutil
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB = os.path.join(_HERE, "liboracle.so")
SRC = os.path.join(_HERE, "oracle.c")

# Skew multipliers X of the Effective Experts buckets (exact fractions).
EFFEXP_X = [(11, 10), (13, 10), (3, 2), (17, 10), (2, 1), (5, 2), (4, 1), (6, 1), (8, 1),
            (12, 1), (16, 1), (24, 1), (32, 1)]


def build(verbose: bool = False) -> str:
    cc = shutil.which("gcc") or "cc"
    cmd = [cc, "-O2", "-std=c11", "-fopenmp", "-fPIC", "-shared", SRC, "-o", LIB + ".tmp", "-lm"]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"oracle build failed:\n{r.stdout}")
    os.replace(LIB + ".tmp", LIB)
    return LIB


_lib = None


def lib() -> ctypes.CDLL:
    global _lib
    if _lib is None:
        if not os.path.exists(LIB):
            build()
        L = ctypes.CDLL(LIB)
        vp, i32, i64, u64, f64 = (ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_uint64,
                                  ctypes.c_double)
        sig = {
            "oracle_histogram": ([vp, i64, i32, vp], i64),
            "oracle_effexp": ([vp, i32, vp, vp, vp], None),
            "oracle_effexp_bucket": ([u64, u64, i32], i32),
            "oracle_permute": ([vp, i64, i32, vp, vp, vp], None),
            "oracle_select_bucket": ([vp, i32, i32], i32),
            "oracle_match": ([vp, i32, vp, i32, vp], i32),
            "oracle_tiles": ([vp, i32, i32, vp], i64),
            "oracle_moe_expert_bf16": ([i32, vp, vp, i32, vp, i32, vp, i32, i32, vp, vp, vp, vp], i64),
            "oracle_moe_expert_fp8": ([i32, vp, vp, i32, vp, i32, vp, i32, i32, vp, vp, vp, vp, vp, vp,
                                       vp], i64),
            "oracle_alpha_search": ([i32, f64, i32, i32, u64], f64),
            "oracle_mean_effexp": ([i32, f64, i32, u64], f64),
            "oracle_exemplar": ([vp, i32, i32, vp], None),
            "oracle_fastest_mean": ([vp, i32, i32], i32),
            "oracle_dirichlet_logp": ([i32, f64, ctypes.c_uint32, u64, vp], None),
            "oracle_router": ([vp, vp, vp, i32, i32, i32, i32, vp, vp, vp], None),
            "oracle_topk_softmax": ([vp, i32, i32, i32, vp, vp], None),
            "oracle_effexp_map": ([vp, vp, i32, i32, i32, vp], None),
            "oracle_moe_expert_mxfp4": ([i32, vp, vp, i32, vp, i32, vp, i32, i32, vp, vp, vp, vp, vp, vp, vp],
                                        ctypes.c_int64),
            "oracle_mxfp4_value": ([ctypes.c_uint8, ctypes.c_uint8], f64),
        }
        for name, (args, res) in sig.items():
            fn = getattr(L, name)
            fn.argtypes = args
            fn.restype = res
        _lib = L
    return _lib


def _c(a, dtype):
    return np.ascontiguousarray(np.asarray(a, dtype=dtype))


def histogram(ids, E: int) -> np.ndarray:
    ids = _c(ids, np.int32).ravel()
    counts = np.zeros(E, np.int64)
    lib().oracle_histogram(ids.ctypes.data, ids.size, E, counts.ctypes.data)
    return counts


def effexp(counts):
    counts = _c(counts, np.int64)
    num, den, eff = ctypes.c_uint64(), ctypes.c_uint64(), ctypes.c_double()
    lib().oracle_effexp(counts.ctypes.data, counts.size, ctypes.byref(num), ctypes.byref(den),
                        ctypes.byref(eff))
    return int(num.value), int(den.value), float(eff.value)


def effexp_bucket(num: int, den: int, E: int) -> int:
    return int(lib().oracle_effexp_bucket(num, den, E))


def permute(ids, E: int):
    ids = _c(ids, np.int32).ravel()
    A = ids.size
    offsets = np.zeros(E + 1, np.int64)
    perm = np.zeros(max(A, 1), np.int64)
    inv = np.zeros(max(A, 1), np.int64)
    lib().oracle_permute(ids.ctypes.data, A, E, offsets.ctypes.data, perm.ctypes.data, inv.ctypes.data)
    n = int(offsets[E])
    return offsets, perm[:n], inv[:A]


def select_bucket(bucket_T, T: int) -> int:
    b = _c(bucket_T, np.int32)
    return int(lib().oracle_select_bucket(b.ctypes.data, b.size, int(T)))


def match(counts, Q):
    counts = _c(counts, np.int64)
    Q = _c(Q, np.int32)
    n_ex = Q.shape[0]
    scores = np.zeros(max(n_ex, 1), np.int64)
    i = lib().oracle_match(counts.ctypes.data, counts.size, Q.ctypes.data, n_ex, scores.ctypes.data)
    return int(i), scores[:n_ex]


def tiles(counts, BM: int) -> np.ndarray:
    counts = _c(counts, np.int64)
    max_tiles = int(sum((int(c) + BM - 1) // BM for c in counts))
    out = np.zeros((max(max_tiles, 1), 3), np.int64)
    n = lib().oracle_tiles(counts.ctypes.data, counts.size, BM, out.ctypes.data)
    return out[:n]


def moe_rows(ids, w, k: int, rows, x_rows, H: int, I: int, experts, weights_of) -> np.ndarray:
    """Layer output y[len(rows)][H] in fp64 for the listed token rows.

    ``weights_of(e)`` returns expert e's weights, either bf16 bit patterns
    ``(W1 [I][H], W3 [I][H], W2 [H][I])`` (uint16), fp8 pairs ``((q1, s1), (q3, s3), (q2, s2))``
    with float32 block scales, or MXFP4 pairs of the same form with packed e2m1 codes
    (uint8 [rows][cols / 2]) and E8M0 scales (uint8 [rows][cols / 32]); experts are visited one at a time
    (expert-major), so only one expert's weights are held at once.  Slots whose id is not
    among ``experts`` (masked slots, id < 0) contribute nothing.
    """
    ids = _c(ids, np.int32)
    w = _c(w, np.float32)
    rows = _c(rows, np.int32)
    x_rows = _c(x_rows, np.uint16)
    y = np.zeros((rows.size, H), np.float64)
    L = lib()
    for e in experts:
        if int(e) < 0:
            raise ValueError("expert ids are >= 0: a negative id is a masked slot, never an expert")
        wt = weights_of(int(e))
        if isinstance(wt[0], tuple) and np.asarray(wt[0][1]).dtype == np.uint8:
            (q1, s1), (q3, s3), (q2, s2) = [(_c(q, np.uint8), _c(s, np.uint8)) for q, s in wt]
            L.oracle_moe_expert_mxfp4(int(e), ids.ctypes.data, w.ctypes.data, k, rows.ctypes.data,
                                      rows.size, x_rows.ctypes.data, H, I, q1.ctypes.data,
                                      s1.ctypes.data, q3.ctypes.data, s3.ctypes.data, q2.ctypes.data,
                                      s2.ctypes.data, y.ctypes.data)
        elif isinstance(wt[0], tuple):
            (q1, s1), (q3, s3), (q2, s2) = [(_c(q, np.uint8), _c(s, np.float32)) for q, s in wt]
            L.oracle_moe_expert_fp8(int(e), ids.ctypes.data, w.ctypes.data, k, rows.ctypes.data,
                                    rows.size, x_rows.ctypes.data, H, I, q1.ctypes.data,
                                    s1.ctypes.data, q3.ctypes.data, s3.ctypes.data, q2.ctypes.data,
                                    s2.ctypes.data, y.ctypes.data)
        else:
            w1, w3, w2 = [_c(m, np.uint16) for m in wt]
            L.oracle_moe_expert_bf16(int(e), ids.ctypes.data, w.ctypes.data, k, rows.ctypes.data,
                                     rows.size, x_rows.ctypes.data, H, I, w1.ctypes.data,
                                     w3.ctypes.data, w2.ctypes.data, y.ctypes.data)
    return y


def alpha_search(E: int, target: float, S: int = 64, iters: int = 60, seed: int = 0) -> float:
    return float(lib().oracle_alpha_search(E, float(target), S, iters, seed))


def mean_effexp(E: int, alpha: float, S: int = 64, seed: int = 0) -> float:
    return float(lib().oracle_mean_effexp(E, float(alpha), S, seed))


def exemplar(counts) -> np.ndarray:
    counts = _c(counts, np.int64)
    S, E = counts.shape
    Q = np.zeros(E, np.int32)
    lib().oracle_exemplar(counts.ctypes.data, S, E, Q.ctypes.data)
    return Q


def fastest_mean(lat) -> int:
    lat = _c(lat, np.float64)
    S, V = lat.shape
    return int(lib().oracle_fastest_mean(lat.ctypes.data, S, V))


def dirichlet_logp(E: int, alpha: float, s: int, seed: int = 0) -> np.ndarray:
    out = np.zeros(E, np.float64)
    lib().oracle_dirichlet_logp(E, float(alpha), int(s), int(seed), out.ctypes.data)
    return out


def router(x_bf16, wg_bf16, k: int, bias=None):
    """Gating logits (fp64), top-k ids (descending, ties to the lower id) and softmax gates over
    the k chosen logits.  x_bf16 [T][H] and wg_bf16 [E][H] are uint16 bf16 bit patterns."""
    x = _c(x_bf16, np.uint16)
    wg = _c(wg_bf16, np.uint16)
    T, H = x.shape
    E = wg.shape[0]
    b = None if bias is None else _c(bias, np.float32)
    logits = np.zeros((T, E), np.float64)
    ids = np.zeros((T, k), np.int32)
    w = np.zeros((T, k), np.float64)
    lib().oracle_router(x.ctypes.data, wg.ctypes.data, None if b is None else b.ctypes.data, T, H, E, k,
                        logits.ctypes.data, ids.ctypes.data, w.ctypes.data)
    return logits, ids, w


def topk_softmax(logits, k: int):
    """Top-k ids (descending, ties to the lower id) and softmax gates over the chosen slots of
    the given logits [T][E] (taken as fp64)."""
    l = _c(logits, np.float64)
    T, E = l.shape
    ids = np.zeros((T, k), np.int32)
    w = np.zeros((T, k), np.float64)
    lib().oracle_topk_softmax(l.ctypes.data, T, E, k, ids.ctypes.data, w.ctypes.data)
    return ids, w


def effexp_map(Q, kid, noda: int):
    """Variant per Effective Experts bucket -1..13 (15 entries) of one token bucket's exemplars."""
    q = _c(Q, np.int32)
    k = _c(kid, np.int32)
    n_ex, E = q.shape
    out = np.zeros(15, np.int32)
    lib().oracle_effexp_map(q.ctypes.data, k.ctypes.data, n_ex, E, int(noda), out.ctypes.data)
    return out


def mxfp4_value(code: int, scale: int) -> float:
    """Decoded MXFP4 element: e2m1(code) * 2^(scale - 127)."""
    return float(lib().oracle_mxfp4_value(code, scale))
