"""Seeded synthetic inputs for the fused-MoE path: routing and bulk tensors.

This module is the one piece shared by the product side (benchmark, tuner
driver) and the test side (oracle checks).  It contains no arithmetic of the
method itself (no histogram, no Effective Experts, no permutation, no FFN):
it only draws inputs.

Routing (small, host side, numpy ``default_rng``) follows the symmetric
Dirichlet routing model of the paper (Sec. II-D, Eq. (1)):

1. ``log p``: E draws of Gamma(alpha+1) and E uniforms, combined in log space
   as ``log G = log Gamma(alpha+1) + log(U)/alpha`` (the standard boost for
   alpha < 1) and normalised with logsumexp, so that no entry underflows to
   -inf even at alpha = 0.03.
2. optional hot experts (``choice(E, n_hot, replace=False)``): a fraction
   ``hot_mass`` of the probability is moved onto them,
   ``p' = (1 - hot_mass) p + hot_mass / n_hot * [e in hot]``.
3. Gumbel-top-k: ``key = log p - log(-log U)`` per (token, expert), the k
   largest keys are the token's experts, in descending key order (ties, of
   probability zero, to the lower expert id).
4. gates: softmax over the k chosen slots of N(0,1) logits, in float64, then
   stored as float32.

Bulk tensors (activations and expert weights) come from a counter-based
generator (Philox4x32-10 + Irwin-Hall(8), see ``synth_fill.hip``) that exists
both as a device fill and as a host fill with identical bits, so the oracle
can regenerate any single expert slab that the GPU holds.
"""
from __future__ import annotations

import ctypes
import math
import os
from dataclasses import dataclass

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libdamoe_synth.so")

# Standard deviation of the centred Irwin-Hall sum of 8 uniforms on 0..65535.
IH8_STD = math.sqrt(8.0 * (65536.0 ** 2 - 1.0) / 12.0)

# Tensor ids of the counter-based generator.
T_X, T_W1, T_W2, T_W3, T_WG = 0, 1, 2, 3, 4


def ih_scale(sigma: float) -> float:
    """fp32 multiplier that turns the centred Irwin-Hall sum into N(0, sigma^2)."""
    return float(np.float32(sigma / IH8_STD))


_lib = None


def lib() -> ctypes.CDLL:
    """Load the generator library (built by the package build step)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(
                f"{LIB_PATH} is not built; run __graft_entry__.build() first")
        L = ctypes.CDLL(LIB_PATH)
        u64, u32, f32, vp = ctypes.c_uint64, ctypes.c_uint32, ctypes.c_float, ctypes.c_void_p
        L.synth_philox4x32_10.argtypes = [vp, vp, vp]
        L.synth_philox4x32_10.restype = None
        L.synth_fill_bf16_host.argtypes = [vp, u64, u64, u64, u32, u64, u32, f32]
        L.synth_fill_bf16_host.restype = None
        L.synth_fill_bf16_device.argtypes = [vp, u64, u64, u64, u32, u64, u32, f32, vp]
        L.synth_fill_bf16_device.restype = ctypes.c_int
        L.synth_fill_fp8_b128_host.argtypes = [vp, vp, u32, u32, u32, u32, u64, u32, f32]
        L.synth_fill_fp8_b128_host.restype = ctypes.c_int
        L.synth_fill_fp8_b128_device.argtypes = [vp, vp, u32, u32, u32, u32, u64, u32, f32, vp]
        L.synth_fill_fp8_b128_device.restype = ctypes.c_int
        L.synth_fill_mxfp4_host.argtypes = [vp, vp, u32, u32, u32, u32, u64, u32, f32]
        L.synth_fill_mxfp4_host.restype = ctypes.c_int
        L.synth_fill_mxfp4_device.argtypes = [vp, vp, u32, u32, u32, u32, u64, u32, f32, vp]
        L.synth_fill_mxfp4_device.restype = ctypes.c_int
        L.synth_mxfp4_quantize_host.argtypes = [vp, u64, vp, vp]
        L.synth_mxfp4_quantize_host.restype = None
        _lib = L
    return _lib


def philox4x32_10(ctr, key) -> np.ndarray:
    c = np.ascontiguousarray(np.asarray(ctr, dtype=np.uint32))
    k = np.ascontiguousarray(np.asarray(key, dtype=np.uint32))
    out = np.zeros(4, dtype=np.uint32)
    lib().synth_philox4x32_10(c.ctypes.data, k.ctypes.data, out.ctypes.data)
    return out


def fill_bf16_host(n: int, *, seed: int, tensor: int, slab0: int = 0, slab_elems: int | None = None,
                   start: int = 0, sigma: float = 1.0, out: np.ndarray | None = None) -> np.ndarray:
    """Host bf16 values (as uint16 bit patterns) of elements start..start+n-1."""
    if out is None:
        out = np.empty(int(n), dtype=np.uint16)
    elif out.dtype != np.uint16 or out.size != int(n) or not out.flags.c_contiguous:
        raise ValueError("out must be a contiguous uint16 array of n elements")
    se = int(slab_elems) if slab_elems else max(int(start) + int(n), 1)
    lib().synth_fill_bf16_host(out.ctypes.data, int(n), int(start), se, int(slab0), int(seed),
                               int(tensor), ih_scale(sigma))
    return out


def fill_bf16_device(ptr: int, n: int, *, seed: int, tensor: int, slab0: int = 0,
                     slab_elems: int | None = None, start: int = 0, sigma: float = 1.0,
                     stream: int = 0) -> None:
    se = int(slab_elems) if slab_elems else max(int(start) + int(n), 1)
    rc = lib().synth_fill_bf16_device(ctypes.c_void_p(ptr), int(n), int(start), se, int(slab0),
                                      int(seed), int(tensor), ih_scale(sigma), ctypes.c_void_p(stream))
    if rc != 0:
        raise RuntimeError(f"synth_fill_bf16_device failed with hip error {rc}")


def fill_fp8_host(rows: int, cols: int, n_slabs: int, *, seed: int, tensor: int, slab0: int = 0,
                  sigma: float = 0.02):
    q = np.empty((n_slabs, rows, cols), dtype=np.uint8)
    s = np.empty((n_slabs, rows // 128, cols // 128), dtype=np.float32)
    rc = lib().synth_fill_fp8_b128_host(q.ctypes.data, s.ctypes.data, rows, cols, slab0, n_slabs,
                                        int(seed), int(tensor), ih_scale(sigma))
    if rc != 0:
        raise ValueError("fp8 fill needs rows and cols divisible by 128")
    return q, s


def fill_fp8_device(q_ptr: int, s_ptr: int, rows: int, cols: int, n_slabs: int, *, seed: int,
                    tensor: int, slab0: int = 0, sigma: float = 0.02, stream: int = 0) -> None:
    rc = lib().synth_fill_fp8_b128_device(ctypes.c_void_p(q_ptr), ctypes.c_void_p(s_ptr), rows, cols,
                                          slab0, n_slabs, int(seed), int(tensor), ih_scale(sigma),
                                          ctypes.c_void_p(stream))
    if rc != 0:
        raise RuntimeError(f"synth_fill_fp8_b128_device failed with code {rc}")


def fill_mxfp4_host(rows: int, cols: int, n_slabs: int, *, seed: int, tensor: int, slab0: int = 0,
                    sigma: float = 0.02):
    """MXFP4 quantisation of the generator's bf16 values: packed e2m1 codes
    [n_slabs][rows][cols / 2] and E8M0 scales [n_slabs][rows][cols / 32] (uint8)."""
    q = np.empty((n_slabs, rows, cols // 2), dtype=np.uint8)
    s = np.empty((n_slabs, rows, cols // 32), dtype=np.uint8)
    rc = lib().synth_fill_mxfp4_host(q.ctypes.data, s.ctypes.data, rows, cols, slab0, n_slabs, int(seed),
                                     int(tensor), ih_scale(sigma))
    if rc != 0:
        raise ValueError("MXFP4 fill needs cols divisible by 32")
    return q, s


def mxfp4_quantize(w) -> tuple:
    """MXFP4 quantisation of float32 values in blocks of 32: (packed codes [n/2], E8M0 [n/32])."""
    w = np.ascontiguousarray(np.asarray(w, np.float32).ravel())
    if w.size % 32:
        raise ValueError("blocks of 32")
    q = np.empty(w.size // 2, np.uint8)
    s = np.empty(w.size // 32, np.uint8)
    lib().synth_mxfp4_quantize_host(w.ctypes.data, w.size // 32, q.ctypes.data, s.ctypes.data)
    return q, s


def fill_mxfp4_device(q_ptr: int, s_ptr: int, rows: int, cols: int, n_slabs: int, *, seed: int, tensor: int,
                      slab0: int = 0, sigma: float = 0.02, stream: int = 0) -> None:
    rc = lib().synth_fill_mxfp4_device(ctypes.c_void_p(q_ptr), ctypes.c_void_p(s_ptr), rows, cols, slab0, n_slabs,
                                       int(seed), int(tensor), ih_scale(sigma), ctypes.c_void_p(stream))
    if rc != 0:
        raise RuntimeError(f"synth_fill_mxfp4_device failed with code {rc}")


# ----------------------------------------------------------------------------------------------
# Routing
# ----------------------------------------------------------------------------------------------

def _logsumexp(v: np.ndarray) -> float:
    m = float(np.max(v))
    return m + math.log(float(np.sum(np.exp(v - m))))


def _open_uniform(rng: np.random.Generator, size) -> np.ndarray:
    # random() is a multiple of 2^-53 in [0, 1); the half-step offset keeps it in (0, 1).
    return rng.random(size) + 2.0 ** -54


def dirichlet_logp(rng: np.random.Generator, E: int, alpha: float) -> np.ndarray:
    """log of one draw p ~ Dir(alpha * ones(E)), computed in log space."""
    g = rng.standard_gamma(alpha + 1.0, size=E)
    u = _open_uniform(rng, E)
    logg = np.log(g) + np.log(u) / alpha
    return logg - _logsumexp(logg)


@dataclass
class Routing:
    ids: np.ndarray      # int32 [T, k], row-distinct expert ids in [0, E)
    w: np.ndarray        # float32 [T, k], each row sums to 1 (up to fp32 rounding)
    logp: np.ndarray     # float64 [E], log of the routing probability vector
    E: int
    k: int
    alpha: float | None

    @property
    def T(self) -> int:
        return int(self.ids.shape[0])


def routing(E: int, k: int, T: int, alpha: float | None, seed, *, n_hot: int = 0,
            hot_mass: float = 0.4) -> Routing:
    """Dirichlet (alpha) or uniform (alpha=None) routing of T tokens to top-k of E experts."""
    if not (1 <= k <= E):
        raise ValueError("need 1 <= k <= E")
    rng = np.random.default_rng(seed)
    if alpha is None:
        logp = np.full(E, -math.log(E))
    else:
        logp = dirichlet_logp(rng, E, float(alpha))
    if n_hot:
        hot = rng.choice(E, n_hot, replace=False)
        add = np.full(E, -np.inf)
        add[hot] = math.log(hot_mass / n_hot)
        logp = np.logaddexp(math.log1p(-hot_mass) + logp, add)
    if T == 0:
        return Routing(np.zeros((0, k), np.int32), np.zeros((0, k), np.float32), logp, E, k, alpha)
    u = _open_uniform(rng, (T, E))
    keys = logp[None, :] - np.log(-np.log(u))
    order = np.argsort(-keys, axis=1, kind="stable")[:, :k]
    logits = rng.standard_normal((T, k))
    z = np.exp(logits - logits.max(axis=1, keepdims=True))
    w = z / z.sum(axis=1, keepdims=True)
    return Routing(order.astype(np.int32), w.astype(np.float32), logp, E, k, alpha)


def routing_repeated(E: int, k: int, T: int, f: int, alpha: float, seed) -> Routing:
    """Routing of T tokens in groups that repeat one row each: the token analog of the paper's
    imbalance factor f (Sec. V-E), where groups of about f% of a batch's prompts share one
    prompt.  f = 0: every token draws its own row; f > 0: groups of max(1, round(f T / 100))
    consecutive tokens take one row (ids and gates), drawn like `routing` for one token per
    group from a common Dirichlet(alpha) p; f = 100: one row for the whole batch."""
    if not 0 <= f <= 100:
        raise ValueError("f is a percentage")
    g = 1 if f == 0 else max(1, int(round(f * T / 100.0)))
    n = -(-T // g) if T else 0
    base = routing(E, k, n, alpha, seed)
    if T == 0:
        return base
    rows = np.repeat(np.arange(n), g)[:T]
    return Routing(base.ids[rows].copy(), base.w[rows].copy(), base.logp, E, k, alpha)


def ep_local(r: Routing, ep: int, rank: int):
    """One expert-parallel rank's share of a routing over E experts: experts
    [rank E / ep, (rank + 1) E / ep) are local.  Returns (token indices of the tokens with at
    least one local slot, their local ids [T_l][k] = id - rank E / ep, or -1 for a slot whose
    expert is on another rank, and their gates, unchanged: the rank computes its partial sum)."""
    if r.E % ep:
        raise ValueError("E must split evenly over the ranks")
    el = r.E // ep
    lo = rank * el
    local = (r.ids >= lo) & (r.ids < lo + el)
    keep = np.nonzero(local.any(axis=1))[0]
    ids = np.where(local, r.ids - lo, -1)[keep].astype(np.int32)
    return keep, ids, r.w[keep].copy()


# ----------------------------------------------------------------------------------------------
# Named workloads (shapes and seeds)
# ----------------------------------------------------------------------------------------------

@dataclass(frozen=True)
class Shape:
    name: str
    E: int
    k: int
    H: int
    I: int
    shape_id: int          # seeds the weights
    wdtype: str = "bf16"   # "bf16", "fp8" or "mxfp4"
    w_sigma: float = 0.02

    @property
    def weight_seed(self) -> int:
        return 0x5EED0000 + self.shape_id


TINY = Shape("tiny", E=8, k=2, H=256, I=512, shape_id=0)
DS = Shape("dsv3", E=256, k=8, H=7168, I=2048, shape_id=1)
DS_FP8 = Shape("dsv3-fp8", E=256, k=8, H=7168, I=2048, shape_id=1, wdtype="fp8")
DS_MXFP4 = Shape("dsv3-mxfp4", E=256, k=8, H=7168, I=2048, shape_id=1, wdtype="mxfp4")
KIMI = Shape("kimi-k2", E=384, k=8, H=7168, I=2048, shape_id=3)
# One expert-parallel rank's layer of DeepSeek-V3 at EP = 2, 4, 8 (weights of its own experts).
DS_EP = {ep: Shape(f"dsv3-ep{ep}", E=256 // ep, k=8, H=7168, I=2048, shape_id=1) for ep in (2, 4, 8)}

# Weight matrices of expert e (row-major): W1, W3: [I][H]; W2: [H][I].
WEIGHT_TENSORS = {"w1": (T_W1, "I", "H"), "w3": (T_W3, "I", "H"), "w2": (T_W2, "H", "I")}


def weight_dims(shape: Shape, name: str):
    tid, r, c = WEIGHT_TENSORS[name]
    return tid, getattr(shape, r), getattr(shape, c)


def expert_weights_host(shape: Shape, e: int, out=None):
    """bf16 bit patterns (uint16) of expert e: (W1 [I][H], W3 [I][H], W2 [H][I]).

    ``out`` may be a previous result to refill in place (avoids first-touch cost)."""
    res = []
    for i, name in enumerate(("w1", "w3", "w2")):
        tid, r, c = weight_dims(shape, name)
        buf = None if out is None else out[i].reshape(-1)
        res.append(fill_bf16_host(r * c, seed=shape.weight_seed, tensor=tid, slab0=e,
                                  slab_elems=r * c, sigma=shape.w_sigma, out=buf).reshape(r, c))
    return tuple(res)


def expert_weights_mxfp4_host(shape: Shape, e: int):
    """MXFP4 weights of expert e: ((q1, s1), (q3, s3), (q2, s2)), codes and E8M0 scales."""
    out = []
    for name in ("w1", "w3", "w2"):
        tid, r, c = weight_dims(shape, name)
        q, s = fill_mxfp4_host(r, c, 1, seed=shape.weight_seed, tensor=tid, slab0=e, sigma=shape.w_sigma)
        out.append((q[0], s[0]))
    return tuple(out)


class ExpertWeightSource:
    """Callable e -> expert e's host weights, refilling one set of buffers."""

    def __init__(self, shape: Shape):
        self.shape = shape
        self.buf = None

    def __call__(self, e: int):
        if self.shape.wdtype == "fp8":
            return expert_weights_fp8_host(self.shape, e)
        if self.shape.wdtype == "mxfp4":
            return expert_weights_mxfp4_host(self.shape, e)
        self.buf = expert_weights_host(self.shape, e, self.buf)
        return self.buf


def expert_weights_fp8_host(shape: Shape, e: int):
    """fp8 block-128 weights of expert e: ((q1, s1), (q3, s3), (q2, s2))."""
    out = []
    for name in ("w1", "w3", "w2"):
        tid, r, c = weight_dims(shape, name)
        q, s = fill_fp8_host(r, c, 1, seed=shape.weight_seed, tensor=tid, slab0=e, sigma=shape.w_sigma)
        out.append((q[0], s[0]))
    return tuple(out)


def gate_sigma(H: int) -> float:
    """Gate weights N(0, 1/H): the logits of N(0, 1) tokens then have unit variance."""
    return 1.0 / math.sqrt(H)


def gate_weights_host(shape: Shape) -> np.ndarray:
    """bf16 gate weights Wg [E][H] (uint16) of the shape's router."""
    n = shape.E * shape.H
    return fill_bf16_host(n, seed=shape.weight_seed, tensor=T_WG, slab_elems=n,
                          sigma=gate_sigma(shape.H)).reshape(shape.E, shape.H)


def gate_bias(E: int, alpha: float | None, seed) -> np.ndarray:
    """Per-expert gate bias: log p of one Dirichlet(alpha) draw (float32), or zeros for None.

    Added to unit-variance logits it skews the router's choices towards the high-p experts,
    the more the smaller alpha, like the routing model above."""
    if alpha is None:
        return np.zeros(E, np.float32)
    return dirichlet_logp(np.random.default_rng(seed), E, float(alpha)).astype(np.float32)


def x_seed(tag: int) -> int:
    return 0xA11CE000 + int(tag)


def activations_host(T: int, H: int, tag: int, rows=None) -> np.ndarray:
    """bf16 activations [T][H] (uint16); ``rows`` selects a subset of token rows."""
    if rows is None:
        return fill_bf16_host(T * H, seed=x_seed(tag), tensor=T_X, slab_elems=max(T * H, 1),
                              sigma=1.0).reshape(T, H)
    rows = np.asarray(rows, dtype=np.int64)
    out = np.empty((len(rows), H), dtype=np.uint16)
    for i, t in enumerate(rows):
        out[i] = fill_bf16_host(H, seed=x_seed(tag), tensor=T_X, start=int(t) * H,
                                slab_elems=max(T * H, 1), sigma=1.0)
    return out


def bf16_to_f64(u16: np.ndarray) -> np.ndarray:
    return (np.asarray(u16, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def f32_to_bf16_bits(f: np.ndarray) -> np.ndarray:
    u = np.ascontiguousarray(np.asarray(f, dtype=np.float32)).view(np.uint32).astype(np.uint64)
    u = (u + 0x7FFF + ((u >> 16) & 1)) >> 16
    return u.astype(np.uint16)


# Seeds of the named sweeps.
def seed_decode(T: int, alpha: float, rep: int):
    return [1, int(T), int(round(1000 * alpha)), int(rep)]


def seed_prefill(T: int, alpha: float, rep: int):
    return [2, int(T), int(round(1000 * alpha)), int(rep)]


def seed_kimi(T: int, rep: int):
    return [3, int(T), int(rep)]


def seed_imbalance(T: int, f: int, rep: int):
    return [5, int(T), int(f), int(rep)]


def seed_ep(T: int, rep: int):
    return [6, int(T), int(rep)]


def seed_trace_step(step: int):
    return [4, 0, int(step)]


def seed_trace_tune(*rest):
    return [4, 1, *[int(r) for r in rest]]


def trace_step_params(step: int, t_max: int = 8192, a_lo: float = 0.03, a_hi: float = 10.0):
    """(T, alpha) of one dispatch-trace step: T log-uniform in [1, t_max], alpha log-uniform."""
    rng = np.random.default_rng([4, 2, int(step)])
    T = int(math.floor(math.exp(rng.uniform(0.0, math.log(t_max)))))
    T = min(max(T, 1), t_max)
    alpha = math.exp(rng.uniform(math.log(a_lo), math.log(a_hi)))
    return T, alpha
