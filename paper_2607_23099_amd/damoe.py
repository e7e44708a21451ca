"""ctypes binding of ``libdamoe.so`` (the C-ABI declared in ``include/damoe.h``).

Argument marshalling only: every step of the path runs in the library's HIP
kernels.  Tensors are passed as device pointers (``tensor.data_ptr()``) and
streams as raw ``hipStream_t`` handles; PyTorch is only used by callers to own
device memory.  Loading fails loudly if the library has not been built.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libdamoe.so")

N_TILE_SIZES = 5
W_BF16, W_FP8_B128, W_MXFP4 = 0, 1, 2
DEVERR_EXPERT_ID, DEVERR_TILES, DEVERR_VARIANT, DEVERR_COUNTS = 1, 2, 4, 8
LAYOUT_ROWMAJOR, LAYOUT_FRAG16 = 0, 1

STATUS = {0: "ok", -1: "invalid argument", -2: "unsupported", -3: "workspace too small",
          -4: "table mismatch", -5: "hip error", -6: "out of memory", -7: "io error"}

EXPORTED = [
    "damoe_status_string", "damoe_workspace_layout", "damoe_workspace_size", "damoe_route_histogram",
    "damoe_table_create", "damoe_table_destroy", "damoe_table_info", "damoe_table_save",
    "damoe_table_load", "damoe_dispatch", "damoe_fused_moe", "damoe_num_variants", "damoe_variant_name",
    "damoe_variant_tile_m", "damoe_variant_supports", "damoe_tune", "damoe_alpha_search",
    "damoe_read_device_error", "damoe_fused_moe_stage", "damoe_route_dispatch", "damoe_pack_weights",
    "damoe_table_candidates", "damoe_router", "damoe_router_workspace_size", "damoe_route_dispatch_effexp",
    "damoe_table_effexp_map", "damoe_table_effexp_candidates", "damoe_noalloc_scratch_bytes",
    "damoe_moe_layer_noalloc",
]


class DamoeError(RuntimeError):
    def __init__(self, fn: str, code: int):
        super().__init__(f"{fn} failed: {code} ({STATUS.get(code, 'unknown')})")
        self.code = code


class Layer(ctypes.Structure):
    _fields_ = [("E", ctypes.c_int32), ("k", ctypes.c_int32), ("H", ctypes.c_int32),
                ("I", ctypes.c_int32), ("wdtype", ctypes.c_int32), ("layout", ctypes.c_int32),
                ("w1", ctypes.c_void_p),
                ("w3", ctypes.c_void_p), ("w2", ctypes.c_void_p), ("s1", ctypes.c_void_p),
                ("s3", ctypes.c_void_p), ("s2", ctypes.c_void_p)]


class WsLayout(ctypes.Structure):
    _fields_ = [("total", ctypes.c_size_t), ("ctrl", ctypes.c_size_t),
                ("tiles", ctypes.c_size_t * N_TILE_SIZES), ("tiles_cap", ctypes.c_size_t),
                ("h", ctypes.c_size_t), ("out", ctypes.c_size_t), ("route", ctypes.c_size_t)]


class TableDesc(ctypes.Structure):
    _fields_ = [("E", ctypes.c_int32), ("k", ctypes.c_int32), ("H", ctypes.c_int32),
                ("I", ctypes.c_int32), ("wdtype", ctypes.c_int32), ("n_buckets", ctypes.c_int32),
                ("bucket_T", ctypes.c_void_p), ("n_ex", ctypes.c_void_p), ("Q", ctypes.c_void_p),
                ("kid", ctypes.c_void_p), ("noda", ctypes.c_void_p)]


class TuneConfig(ctypes.Structure):
    _fields_ = [("n_buckets", ctypes.c_int32), ("bucket_T", ctypes.c_void_p),
                ("n_skews", ctypes.c_int32), ("skew_X", ctypes.c_void_p), ("samples", ctypes.c_int32),
                ("reps", ctypes.c_int32), ("alpha_samples", ctypes.c_int32),
                ("alpha_iters", ctypes.c_int32), ("seed", ctypes.c_uint64), ("x", ctypes.c_void_p),
                ("verbose", ctypes.c_int32), ("ep", ctypes.c_int32), ("n_repeat", ctypes.c_int32),
                ("repeat_f", ctypes.c_void_p), ("flush_mib", ctypes.c_int32)]


_lib = None


def lib() -> ctypes.CDLL:
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is not built: run __graft_entry__.build() "
                               "(the fused-MoE path has no fallback)")
        L = ctypes.CDLL(LIB_PATH)
        vp, i32, u32, u64, sz, f64 = (ctypes.c_void_p, ctypes.c_int32, ctypes.c_uint32, ctypes.c_uint64,
                                      ctypes.c_size_t, ctypes.c_double)
        sigs = {
            "damoe_status_string": ([i32], ctypes.c_char_p),
            "damoe_workspace_layout": ([i32, i32, i32, i32, i32, vp], i32),
            "damoe_workspace_size": ([vp, i32], sz),
            "damoe_route_histogram": ([vp, i32, i32, i32, vp, vp, vp, vp, vp, vp, vp, sz, vp], i32),
            "damoe_table_create": ([vp, vp], i32),
            "damoe_table_destroy": ([vp], None),
            "damoe_table_info": ([vp, vp, vp, vp, vp, vp, vp, vp], i32),
            "damoe_table_save": ([vp, ctypes.c_char_p], i32),
            "damoe_table_load": ([ctypes.c_char_p, vp], i32),
            "damoe_dispatch": ([vp, vp, i32, vp, vp, sz, vp], i32),
            "damoe_route_dispatch": ([vp, vp, i32, i32, i32, vp, vp, vp, vp, vp, vp, vp, vp, sz, vp], i32),
            "damoe_fused_moe": ([vp, vp, vp, i32, vp, vp, vp, i32, u32, vp, vp, sz, vp], i32),
            "damoe_fused_moe_stage": ([vp, i32, vp, vp, i32, vp, vp, vp, i32, u32, vp, vp, sz, vp], i32),
            "damoe_table_candidates": ([vp, i32], u32),
            "damoe_num_variants": ([], i32),
            "damoe_variant_name": ([i32], ctypes.c_char_p),
            "damoe_variant_tile_m": ([i32], i32),
            "damoe_variant_supports": ([i32, i32], i32),
            "damoe_tune": ([vp, vp, vp, vp], i32),
            "damoe_alpha_search": ([i32, f64, i32, i32, u64], f64),
            "damoe_read_device_error": ([vp, vp, vp], i32),
            "damoe_pack_weights": ([vp, vp, vp, vp, vp], i32),
            "damoe_router": ([vp, vp, vp, i32, i32, i32, i32, vp, vp, vp, vp, sz, vp], i32),
            "damoe_router_workspace_size": ([i32, i32, i32], sz),
            "damoe_route_dispatch_effexp": ([vp, vp, i32, i32, i32, vp, vp, vp, vp, vp, vp, vp, vp, sz, vp], i32),
            "damoe_table_effexp_map": ([vp, i32, vp], i32),
            "damoe_table_effexp_candidates": ([vp, i32], u32),
            "damoe_noalloc_scratch_bytes": ([], sz),
            "damoe_moe_layer_noalloc": ([vp, vp, vp, vp, vp, i32, vp, vp, vp, vp, vp, vp, vp, vp, vp], i32),
        }
        for name, (args, res) in sigs.items():
            fn = getattr(L, name)
            fn.argtypes = args
            fn.restype = res
        _lib = L
    return _lib


def _check(fn: str, rc: int):
    if rc != 0:
        raise DamoeError(fn, rc)


def _p(t) -> int:
    """Device (or host numpy) pointer of a tensor, or 0 for None."""
    if t is None:
        return 0
    if isinstance(t, np.ndarray):
        return t.ctypes.data
    return t.data_ptr()


def _stream(stream) -> int:
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


# ---------------------------------------------------------------- registry / layout

def num_variants() -> int:
    return int(lib().damoe_num_variants())


def variant_name(v: int) -> str:
    n = lib().damoe_variant_name(v)
    return n.decode() if n else ""


def variant_tile_m(v: int) -> int:
    return int(lib().damoe_variant_tile_m(v))


def variant_supports(v: int, wdtype: int) -> bool:
    return bool(lib().damoe_variant_supports(v, wdtype))


def workspace_layout(E: int, k: int, H: int, I: int, T: int) -> dict:
    lo = WsLayout()
    _check("damoe_workspace_layout", lib().damoe_workspace_layout(E, k, H, I, T, ctypes.byref(lo)))
    return {"total": lo.total, "ctrl": lo.ctrl, "tiles": list(lo.tiles), "tiles_cap": lo.tiles_cap,
            "h": lo.h, "out": lo.out, "route": lo.route}


def make_layer(E, k, H, I, wdtype, w1, w3, w2, s1=None, s3=None, s2=None, layout=LAYOUT_ROWMAJOR) -> Layer:
    return Layer(E, k, H, I, wdtype, layout, _p(w1), _p(w3), _p(w2), _p(s1), _p(s3), _p(s2))


def pack_weights(layer: Layer, w1, w3, w2, stream=None):
    _check("damoe_pack_weights", lib().damoe_pack_weights(ctypes.byref(layer), _p(w1), _p(w3), _p(w2),
                                                          _stream(stream)))


def workspace_size(layer: Layer, T_max: int) -> int:
    return int(lib().damoe_workspace_size(ctypes.byref(layer), T_max))


def alpha_search(E: int, target: float, samples: int = 64, iters: int = 60, seed: int = 0) -> float:
    return float(lib().damoe_alpha_search(E, float(target), samples, iters, seed))


# ---------------------------------------------------------------- stream-ordered calls

def route_histogram(ids, T, k, E, counts, offsets, perm, inv_perm, numden, bucket, ws, stream=None):
    _check("damoe_route_histogram", lib().damoe_route_histogram(
        _p(ids), T, k, E, _p(counts), _p(offsets), _p(perm), _p(inv_perm), _p(numden), _p(bucket),
        _p(ws), ws.numel() * ws.element_size(), _stream(stream)))


def route_dispatch(table: "Table", ids, T, k, E, counts, offsets, perm, inv_perm, numden, bucket,
                   variant_id, ws, stream=None):
    _check("damoe_route_dispatch", lib().damoe_route_dispatch(
        table.handle, _p(ids), T, k, E, _p(counts), _p(offsets), _p(perm), _p(inv_perm), _p(numden),
        _p(bucket), _p(variant_id), _p(ws), ws.numel() * ws.element_size(), _stream(stream)))


def route_dispatch_effexp(table: "Table", ids, T, k, E, counts, offsets, perm, inv_perm, numden, bucket,
                          variant_id, ws, stream=None):
    _check("damoe_route_dispatch_effexp", lib().damoe_route_dispatch_effexp(
        table.handle, _p(ids), T, k, E, _p(counts), _p(offsets), _p(perm), _p(inv_perm), _p(numden),
        _p(bucket), _p(variant_id), _p(ws), ws.numel() * ws.element_size(), _stream(stream)))


def dispatch(table: "Table", counts, T, variant_id, ws, stream=None):
    _check("damoe_dispatch", lib().damoe_dispatch(table.handle, _p(counts), T, _p(variant_id), _p(ws),
                                                  ws.numel() * ws.element_size(), _stream(stream)))


def fused_moe(layer: Layer, x, w, T, perm, inv_perm, variant_id, force_variant, y, ws, stream=None,
              candidates: int = 0):
    """candidates: bit mask of the variant ids *variant_id may hold (Table.candidates(T)); 0 = all."""
    _check("damoe_fused_moe", lib().damoe_fused_moe(
        ctypes.byref(layer), _p(x), _p(w), T, _p(perm), _p(inv_perm), _p(variant_id), int(force_variant),
        int(candidates), _p(y), _p(ws), ws.numel() * ws.element_size(), _stream(stream)))


def fused_moe_stage(layer: Layer, stage, x, w, T, perm, inv_perm, variant_id, force_variant, y, ws,
                    stream=None, candidates: int = 0):
    _check("damoe_fused_moe_stage", lib().damoe_fused_moe_stage(
        ctypes.byref(layer), int(stage), _p(x), _p(w), T, _p(perm), _p(inv_perm), _p(variant_id),
        int(force_variant), int(candidates), _p(y), _p(ws), ws.numel() * ws.element_size(),
        _stream(stream)))


def noalloc_scratch_bytes() -> int:
    return int(lib().damoe_noalloc_scratch_bytes())


def moe_layer_noalloc(table: "Table", layer: Layer, x, ids, w, T, counts, offsets, perm, inv_perm, numden, bucket,
                      variant_id, y, stream=None):
    """route_dispatch + fused_moe with the library's own fixed workspace (no workspace argument)."""
    _check("damoe_moe_layer_noalloc", lib().damoe_moe_layer_noalloc(
        table.handle, ctypes.byref(layer), _p(x), _p(ids), _p(w), T, _p(counts), _p(offsets), _p(perm),
        _p(inv_perm), _p(numden), _p(bucket), _p(variant_id), _p(y), _stream(stream)))


def router_workspace_size(E: int, H: int, T_max: int) -> int:
    return int(lib().damoe_router_workspace_size(E, H, T_max))


def router(x, wg, bias, T, H, E, k, logits, ids, w, ws, stream=None):
    _check("damoe_router", lib().damoe_router(_p(x), _p(wg), _p(bias), T, H, E, k, _p(logits), _p(ids), _p(w),
                                              _p(ws), ws.numel() * ws.element_size(), _stream(stream)))


def read_device_error(ws, stream=None) -> int:
    code = ctypes.c_int32()
    _check("damoe_read_device_error", lib().damoe_read_device_error(_p(ws), ctypes.byref(code),
                                                                   _stream(stream)))
    return int(code.value)


# ---------------------------------------------------------------- tables

@dataclass
class TableData:
    E: int
    k: int
    H: int
    I: int
    wdtype: int
    bucket_T: np.ndarray
    n_ex: np.ndarray
    Q: np.ndarray       # [sum n_ex][E]
    kid: np.ndarray
    noda: np.ndarray

    def bucket_rows(self, b: int):
        s = int(self.n_ex[:b].sum())
        return slice(s, s + int(self.n_ex[b]))


class Table:
    def __init__(self, handle: int):
        self.handle = ctypes.c_void_p(handle)
        self._candidates = {}  # T -> mask; tables are immutable, so the lookup is cached
        self._eff_candidates = {}

    @classmethod
    def create(cls, td: TableData) -> "Table":
        arrs = [np.ascontiguousarray(np.asarray(a, np.int32)) for a in
                (td.bucket_T, td.n_ex, td.Q, td.kid, td.noda)]
        d = TableDesc(td.E, td.k, td.H, td.I, td.wdtype, len(arrs[0]), *[a.ctypes.data for a in arrs])
        h = ctypes.c_void_p()
        _check("damoe_table_create", lib().damoe_table_create(ctypes.byref(d), ctypes.byref(h)))
        return cls(h.value)

    @classmethod
    def load(cls, path: str) -> "Table":
        h = ctypes.c_void_p()
        _check("damoe_table_load", lib().damoe_table_load(path.encode(), ctypes.byref(h)))
        return cls(h.value)

    def candidates(self, T: int) -> int:
        """Bit mask of the variants dispatch may choose for T tokens (see damoe_table_candidates)."""
        m = self._candidates.get(T)
        if m is None:
            m = self._candidates[T] = int(lib().damoe_table_candidates(self.handle, int(T)))
        return m

    def effexp_map(self, T: int) -> np.ndarray:
        """Variant per Effective Experts bucket -1..13 for T's token bucket."""
        m = np.zeros(15, np.int32)
        _check("damoe_table_effexp_map", lib().damoe_table_effexp_map(self.handle, T, m.ctypes.data))
        return m

    def effexp_candidates(self, T: int) -> int:
        """Bit mask of the variants the Effective-Experts dispatch may write for T tokens."""
        m = self._eff_candidates.get(T)
        if m is None:
            m = self._eff_candidates[T] = int(lib().damoe_table_effexp_candidates(self.handle, int(T)))
        return m

    def save(self, path: str):
        _check("damoe_table_save", lib().damoe_table_save(self.handle, path.encode()))

    def data(self, E: int) -> TableData:
        nb, nt = ctypes.c_int32(), ctypes.c_int32()
        _check("damoe_table_info", lib().damoe_table_info(self.handle, ctypes.byref(nb), ctypes.byref(nt),
                                                          None, None, None, None, None))
        bT, nex, noda = (np.zeros(nb.value, np.int32) for _ in range(3))
        kid = np.zeros(nt.value, np.int32)
        Q = np.zeros((nt.value, E), np.int32)
        _check("damoe_table_info", lib().damoe_table_info(self.handle, None, None, bT.ctypes.data,
                                                          nex.ctypes.data, Q.ctypes.data,
                                                          kid.ctypes.data, noda.ctypes.data))
        return TableData(E, 0, 0, 0, 0, bT, nex, Q, kid, noda)

    def close(self):
        if self.handle:
            lib().damoe_table_destroy(self.handle)
            self.handle = ctypes.c_void_p()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def tune(layer: Layer, bucket_T, skew_X, x, *, samples=10, reps=5, alpha_samples=64, alpha_iters=60,
         seed=0, verbose=False, ep=1, repeat_f=(), flush_mib=0, stream=None) -> Table:
    bT = np.ascontiguousarray(np.asarray(bucket_T, np.int32))
    sx = np.ascontiguousarray(np.asarray(skew_X, np.float64))
    rf = np.ascontiguousarray(np.asarray(repeat_f, np.int32))
    cfg = TuneConfig(len(bT), bT.ctypes.data, len(sx), sx.ctypes.data, samples, reps, alpha_samples,
                     alpha_iters, seed, _p(x), int(verbose), int(ep), len(rf), rf.ctypes.data if len(rf) else None,
                     int(flush_mib))
    h = ctypes.c_void_p()
    _check("damoe_tune", lib().damoe_tune(ctypes.byref(layer), ctypes.byref(cfg), ctypes.byref(h),
                                          _stream(stream)))
    return Table(h.value)
