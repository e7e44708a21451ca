"""Device-side layer and buffers for driving the C-ABI from Python.

``DeviceLayer`` holds one MoE layer's expert weights in HBM (filled on the
device by the seeded generator), ``Path`` owns every buffer one call sequence
needs (router output, routing, histogram, permutation, variant id, activations,
output, workspaces).  Both only allocate at construction; the per-step methods call
the library and nothing else.
"""
from __future__ import annotations

import torch

from . import damoe, synth


class DeviceLayer:
    """One layer's weights in HBM.  ``packed`` converts them to the fragment-packed layout
    (the fast path) after the row-major fill; the row-major copy is released."""

    def __init__(self, shape: synth.Shape, device: str = "cuda", packed: bool = True):
        self.shape = shape
        E, H, I = shape.E, shape.H, shape.I
        self.wdtype = {"fp8": damoe.W_FP8_B128, "mxfp4": damoe.W_MXFP4}.get(shape.wdtype, damoe.W_BF16)
        stream = torch.cuda.current_stream(device).cuda_stream
        self.w, self.s = {}, {}
        for name in ("w1", "w3", "w2"):
            tid, r, c = synth.weight_dims(shape, name)
            if self.wdtype == damoe.W_BF16:
                t = torch.empty((E, r, c), dtype=torch.bfloat16, device=device)
                synth.fill_bf16_device(t.data_ptr(), t.numel(), seed=shape.weight_seed, tensor=tid,
                                       slab_elems=r * c, sigma=shape.w_sigma, stream=stream)
                self.w[name] = t
            elif self.wdtype == damoe.W_MXFP4:
                q = torch.empty((E, r, c // 2), dtype=torch.uint8, device=device)
                s = torch.empty((E, r, c // 32), dtype=torch.uint8, device=device)
                synth.fill_mxfp4_device(q.data_ptr(), s.data_ptr(), r, c, E, seed=shape.weight_seed, tensor=tid,
                                        sigma=shape.w_sigma, stream=stream)
                self.w[name], self.s[name] = q, s
            else:
                q = torch.empty((E, r, c), dtype=torch.uint8, device=device)
                s = torch.empty((E, r // 128, c // 128), dtype=torch.float32, device=device)
                synth.fill_fp8_device(q.data_ptr(), s.data_ptr(), r, c, E, seed=shape.weight_seed,
                                      tensor=tid, sigma=shape.w_sigma, stream=stream)
                self.w[name], self.s[name] = q, s
        self.layer = damoe.make_layer(E, shape.k, H, I, self.wdtype, self.w["w1"], self.w["w3"],
                                      self.w["w2"], self.s.get("w1"), self.s.get("w3"), self.s.get("w2"))
        self.packed = packed
        if packed:
            if self.wdtype == damoe.W_MXFP4:  # codes and scales into one array of quad fragments
                dst = {n: torch.empty((E, t.shape[1] * t.shape[2] * 17 // 16), dtype=torch.uint8, device=device)
                       for n, t in self.w.items()}
            else:
                dst = {n: torch.empty_like(t) for n, t in self.w.items()}
            damoe.pack_weights(self.layer, dst["w1"], dst["w3"], dst["w2"])
            torch.cuda.synchronize()
            self.w = dst
            if self.wdtype == damoe.W_MXFP4:
                self.s = {}
            self.layer = damoe.make_layer(E, shape.k, H, I, self.wdtype, dst["w1"], dst["w3"], dst["w2"],
                                          self.s.get("w1"), self.s.get("w3"), self.s.get("w2"),
                                          layout=damoe.LAYOUT_FRAG16)

    @property
    def weight_bytes_per_expert(self) -> int:
        sh = self.shape
        if self.wdtype == damoe.W_BF16:
            return 3 * sh.H * sh.I * 2
        if self.wdtype == damoe.W_MXFP4:
            return 3 * sh.H * sh.I // 2 + 3 * sh.H * sh.I // 32
        return 3 * sh.H * sh.I + 3 * (sh.H // 128) * (sh.I // 128) * 4


class RankLayer:
    """Expert-parallel rank `rank` of `ep`: a layer over the full layer's experts
    [rank E / ep, (rank + 1) E / ep), as views into its weight tensors (no copy)."""

    def __init__(self, full: DeviceLayer, ep: int, rank: int, shape: synth.Shape):
        sh = full.shape
        if sh.E % ep or shape.E != sh.E // ep:
            raise ValueError("rank shape does not split the layer")
        self.shape, self.full, self.ep, self.rank = shape, full, ep, rank
        lo = rank * shape.E
        self.w = {n: t[lo: lo + shape.E] for n, t in full.w.items()}
        self.s = {n: t[lo: lo + shape.E] for n, t in full.s.items()}
        self.wdtype, self.packed = full.wdtype, full.packed
        self.layer = damoe.make_layer(shape.E, shape.k, shape.H, shape.I, self.wdtype, self.w["w1"], self.w["w3"],
                                      self.w["w2"], self.s.get("w1"), self.s.get("w3"), self.s.get("w2"),
                                      layout=damoe.LAYOUT_FRAG16 if full.packed else damoe.LAYOUT_ROWMAJOR)

    def global_expert(self, e: int) -> int:
        return self.rank * self.shape.E + e


class Gate:
    """The router's weights in HBM: Wg [E][H] bf16 from the seeded generator and a per-expert
    fp32 bias (zeros unless set)."""

    def __init__(self, shape: synth.Shape, device: str = "cuda"):
        self.shape = shape
        n = shape.E * shape.H
        self.wg = torch.empty((shape.E, shape.H), dtype=torch.bfloat16, device=device)
        synth.fill_bf16_device(self.wg.data_ptr(), n, seed=shape.weight_seed, tensor=synth.T_WG, slab_elems=n,
                               sigma=synth.gate_sigma(shape.H), stream=torch.cuda.current_stream(device).cuda_stream)
        self.bias = torch.zeros(shape.E, dtype=torch.float32, device=device)

    def set_bias(self, bias):
        self.bias.copy_(torch.as_tensor(bias, dtype=torch.float32))


class Path:
    """Buffers for calls with up to T_max tokens on one layer."""

    def __init__(self, dl: DeviceLayer, T_max: int, device: str = "cuda"):
        sh = dl.shape
        self.dl, self.T_max = dl, T_max
        A = max(T_max * sh.k, 1)
        i32 = dict(dtype=torch.int32, device=device)
        self.ids = torch.zeros(A, **i32)
        self.w = torch.zeros(A, dtype=torch.float32, device=device)
        self.counts = torch.zeros(sh.E, **i32)
        self.offsets = torch.zeros(sh.E + 1, **i32)
        self.perm = torch.zeros(A, **i32)
        self.inv_perm = torch.zeros(A, **i32)
        self.numden = torch.zeros(2, dtype=torch.int64, device=device)
        self.bucket = torch.zeros(1, **i32)
        self.variant = torch.zeros(1, **i32)
        self.x = torch.zeros((max(T_max, 1), sh.H), dtype=torch.bfloat16, device=device)
        self.y = torch.zeros((max(T_max, 1), sh.H), dtype=torch.bfloat16, device=device)
        self.ws = torch.zeros(damoe.workspace_size(dl.layer, T_max), dtype=torch.uint8, device=device)
        self.candidates = 0  # variants the last dispatch could choose (0 = all)
        self.logits = torch.zeros((max(T_max, 1), sh.E), dtype=torch.float32, device=device)
        self.router_ws = torch.zeros(damoe.router_workspace_size(sh.E, sh.H, T_max), dtype=torch.uint8,
                                     device=device)

    def set_routing(self, r: synth.Routing):
        T = r.T
        if T > self.T_max:
            raise ValueError("routing larger than T_max")
        if T:
            self.ids[: T * r.k].copy_(torch.from_numpy(r.ids.ravel()))
            self.w[: T * r.k].copy_(torch.from_numpy(r.w.ravel()))

    def fill_x(self, T: int, tag: int):
        if T:
            synth.fill_bf16_device(self.x.data_ptr(), T * self.dl.shape.H, seed=synth.x_seed(tag),
                                   tensor=synth.T_X, slab_elems=T * self.dl.shape.H, sigma=1.0,
                                   stream=torch.cuda.current_stream().cuda_stream)

    def router(self, gate: Gate, T: int, logits: bool = True, stream=None):
        """Gating logits, top-k ids and gates of the first T tokens of x into ids / w."""
        sh = self.dl.shape
        damoe.router(self.x, gate.wg, gate.bias, T, sh.H, sh.E, sh.k, self.logits if logits else None, self.ids,
                     self.w, self.router_ws, stream)

    def route(self, T: int, ids=None, stream=None):
        sh = self.dl.shape
        damoe.route_histogram(self.ids if ids is None else ids, T, sh.k, sh.E, self.counts, self.offsets,
                              self.perm, self.inv_perm, self.numden, self.bucket, self.ws, stream)

    def route_dispatch(self, table: damoe.Table, T: int, ids=None, stream=None):
        sh = self.dl.shape
        self.candidates = table.candidates(T)
        damoe.route_dispatch(table, self.ids if ids is None else ids, T, sh.k, sh.E, self.counts, self.offsets,
                             self.perm, self.inv_perm, self.numden, self.bucket, self.variant, self.ws, stream)

    def route_dispatch_effexp(self, table: damoe.Table, T: int, ids=None, stream=None):
        sh = self.dl.shape
        self.candidates = table.effexp_candidates(T)
        damoe.route_dispatch_effexp(table, self.ids if ids is None else ids, T, sh.k, sh.E, self.counts,
                                    self.offsets, self.perm, self.inv_perm, self.numden, self.bucket, self.variant,
                                    self.ws, stream)

    def dispatch(self, table: damoe.Table, T: int, stream=None):
        self.candidates = table.candidates(T)
        damoe.dispatch(table, self.counts, T, self.variant, self.ws, stream)

    def fused(self, T: int, force_variant: int = -1, w=None, stream=None):
        damoe.fused_moe(self.dl.layer, self.x, self.w if w is None else w, T, self.perm, self.inv_perm,
                        self.variant, force_variant, self.y, self.ws, stream, candidates=self.candidates)

    def fused_stage(self, stage: int, T: int, force_variant: int = -1, w=None, stream=None):
        damoe.fused_moe_stage(self.dl.layer, stage, self.x, self.w if w is None else w, T, self.perm,
                              self.inv_perm, self.variant, force_variant, self.y, self.ws, stream,
                              candidates=self.candidates)

    def ctrl(self):
        lo = damoe.workspace_layout(self.dl.shape.E, self.dl.shape.k, self.dl.shape.H, self.dl.shape.I,
                                    self.T_max)
        return self.ws[lo["ctrl"]: lo["ctrl"] + 256].view(torch.int32).cpu().numpy()

    def tiles(self, T: int, cls: int):
        sh = self.dl.shape
        lo = damoe.workspace_layout(sh.E, sh.k, sh.H, sh.I, T)
        off = lo["tiles"][cls]
        n = int(self.ws[off: off + 4].view(torch.int32).item())
        ent = self.ws[off + 8: off + 8 + 8 * n].view(torch.int32).cpu().numpy().reshape(n, 2)
        return ent
