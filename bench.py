#!/usr/bin/env python3
"""Benchmark of the distribution-aware fused-MoE path on one MI355X.

Workload (default): the DeepSeek-V3-shaped decode sweep, E=256, top-8,
H=7168, I=2048, bf16 weights, T in {1, 8, 32, 128} x Dirichlet alpha in
{0.05, 0.3, 1, 10}.  One step is one pass of the whole hot path -- routing
histogram + Effective Experts + permutation (a2-a4), exemplar dispatch (a5)
and the fused expert computation (a6-a8) with the variant chosen on the
device -- over each of the 16 sweep points, every point on its own routing
(4 routings per point, rotated between steps so the 256 MB Infinity Cache
cannot serve repeated weights).  All inputs are resident in HBM before the
timed region.

value = geomean over the 16 points of the median path latency over the timed
steps (us per layer; each point's mean is reported beside it), the call made
as a caller makes it: route + dispatch, then one fused call, between two
events.  Each step is queued behind a ~1 ms GPU spin, so the events time the
GPU, not the host.  Timed steps alternate between that clean form and an
instrumented one with an event between every two kernels (per-kernel times).
roofline = the dominant kernel (grouped GEMM1 + SwiGLU): algorithmic bytes
(W1 and W3 of every touched expert + the token rows) / its mean duration,
timed with HIP events on its own stream in the instrumented steps.
per_point = each point's path latency with its own roofline: the touched
experts' three matrices + x + y + ids and gates over 8 TB/s (roofline_us) and
roofline_us / path_us (roofline_frac).
cpu_baseline = the fp64 CPU oracle on every sweep point in full, geomean of its
per-point layer times (us, like value).
dispatch_trace = the other half of the metric, after the timed region: a
paired 100-step Kimi-K2 trace (adaptive dispatch against the best static token
bucket, NoDA and the per-step best variant, with bootstrap 95% intervals and the
protocol's A/A noise floor), with its own oracle leg.
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

DECODE_T = (1, 8, 32, 128)
DECODE_ALPHA = (0.05, 0.3, 1.0, 10.0)
REPS = 4
HBM_PEAK_GBS = 8000.0
TABLE_DIR = os.path.join(ROOT, "paper_2607_23099_amd", "tables")
PAPER_SKEWS = [1.1, 1.3, 1.5, 1.7, 2.0, 2.5, 4.0]
EXTENDED_SKEWS = PAPER_SKEWS + [6.0, 8.0, 12.0, 16.0, 24.0, 32.0]


def log(msg):
    print(msg, file=sys.stderr, flush=True)


# HBM traffic summaries of the decode roofline stage (GEMM1 + SwiGLU), per weight format: file,
# rocprof kernel name prefixes of the stage's kernels (the first is launched by every call; a
# call whose device-side choice is another class's variant runs that class's kernel, and the
# others return at once), and the bench flag that selects the format.
TRAFFIC = {
    "bf16": (os.path.join(ROOT, "profiles", "k_gemm_glu_decode_sweep_traffic.txt"),
             ("k_gemm<true", "k_gemm_deep<true", "k_gemm_big<true"), ""),
    "mxfp4": (os.path.join(ROOT, "profiles", "k_gemm_fp4_glu_decode_sweep_traffic.txt"), ("k_gemm_fp4<true",),
              " --wdtype mxfp4"),
}
GEMM_SOURCES = ("csrc/gemm.hip", "csrc/device.h", "csrc/common.h", "csrc/queue.h")


def gemm_source_digest() -> str:
    import hashlib
    h = hashlib.sha256()
    for f in GEMM_SOURCES:
        with open(os.path.join(ROOT, "paper_2607_23099_amd", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def measured_traffic(wdtype: str = "bf16"):
    """HBM bytes per GEMM1 launch from the committed counter summary, or None when it is missing
    or was taken on other kernel sources."""
    try:
        kv = dict(l.split(":", 1) for l in open(TRAFFIC[wdtype][0]).read().splitlines() if ":" in l)
    except OSError:
        return None
    kv = {k.strip(): v.strip() for k, v in kv.items()}
    if kv.get("source_digest") != gemm_source_digest():
        return None
    return int(float(kv["hbm_bytes_per_launch"]))


def summarize_traffic(pmc_dir: str, wdtype: str = "bf16"):
    """Write the traffic summary of the GEMM1 kernel of `wdtype` from four rocprofv3 --pmc runs
    under pmc_dir (subfolders fetch/, write/: the decode sweep; copy_fetch/, copy_write/:
    `--workload copy`).  Counters are in KiB per dispatch; each is scaled by what it reads for
    the plain copy of known size."""
    import csv
    import glob

    def values(sub, counter, match):
        f = glob.glob(os.path.join(pmc_dir, sub, "**", "*counter_collection.csv"), recursive=True)[0]
        return [float(r["Counter_Value"]) * 1024 for r in csv.DictReader(open(f))
                if r["Counter_Name"] == counter and match(r["Kernel_Name"])]

    path, prefixes, flag = TRAFFIC[wdtype]
    is_glu = lambda n: any(p_ in n for p_ in prefixes)
    is_copy = lambda n: "copy" in n.lower() or "elementwise" in n.lower()
    n_copy = 4 << 30
    fcal = max(values("copy_fetch", "FETCH_SIZE", is_copy)) / n_copy
    wcal = max(values("copy_write", "WRITE_SIZE", is_copy)) / n_copy
    # Per GEMM1 call: the bytes of all of the stage's kernels over the calls (launches of the
    # kernel that every call launches).
    calls = len(values("fetch", "FETCH_SIZE", lambda n: prefixes[0] in n))
    fetch = sum(values("fetch", "FETCH_SIZE", is_glu)) / calls
    write = sum(values("write", "WRITE_SIZE", is_glu)) / calls
    per_launch = fetch / fcal + write / wcal
    with open(path, "w") as f:
        f.write(f"# HBM traffic of the GEMM1 + SwiGLU stage ({', '.join(p_ + '...>' for p_ in prefixes)}) over "
                f"the DeepSeek-V3 decode sweep{flag}, per call\n")
        f.write("# rocprofv3 --pmc FETCH_SIZE (then WRITE_SIZE) --output-format csv -d <dir>/fetch -- "
                f"python3 -u bench.py --steps 2 --warmup 1 --no-cpu-baseline --bench-trace-steps 0{flag}\n")
        f.write("# calibration: the same counters on python3 -u bench.py --workload copy --steps 3 "
                "(4 GiB read + 4 GiB written per call)\n")
        f.write(f"source_digest: {gemm_source_digest()}\n")
        f.write(f"launches: {calls}\n")
        f.write(f"fetch_calibration: {fcal:.4f}\n")
        f.write(f"write_calibration: {wcal:.4f}\n")
        f.write(f"fetch_bytes_per_launch: {fetch / fcal:.0f}\n")
        f.write(f"write_bytes_per_launch: {write / wcal:.0f}\n")
        f.write(f"hbm_bytes_per_launch: {per_launch:.0f}\n")
    print(open(path).read())


def summarize_trace(db_glob: str):
    """Print the per-kernel table (calls, total / average / min / max duration, share of the
    traced kernel time) of a rocprofv3 --kernel-trace run from its SQLite output
    (`<dir>/**/*_results.db`)."""
    import glob
    import sqlite3

    rows = {}
    for db in sorted(glob.glob(db_glob, recursive=True)):
        con = sqlite3.connect(db)
        for name, dur in con.execute("select name, duration from kernels"):
            rows.setdefault(name, []).append(dur / 1e3)
        con.close()
    total = sum(sum(v) for v in rows.values()) or 1.0
    print("| kernel | calls | total us | avg us | min us | max us | % GPU time |")
    print("|---|---|---|---|---|---|---|")
    for name, v in sorted(rows.items(), key=lambda kv: -sum(kv[1])):
        print(f"| `{name[:90]}` | {len(v)} | {sum(v):.0f} | {sum(v) / len(v):.2f} | {min(v):.2f} | "
              f"{max(v):.2f} | {100 * sum(v) / total:.2f} |")


def geomean(v):
    v = [x for x in v if x > 0]
    return math.exp(sum(math.log(x) for x in v) / len(v)) if v else 0.0


def touched_experts(ids) -> int:
    return int(len(np.unique(ids)))


def oracle_cores() -> int:
    """Host threads the oracle's OpenMP loops use."""
    return int(os.environ.get("OMP_NUM_THREADS", os.cpu_count() or 1))


def oracle_leg(shape, cases: dict) -> dict:
    """The fp64 CPU oracle timed on the host cores, beside a GPU figure.

    cases: name -> (routing, x tag, token rows or None for every row).  The oracle runs expert
    by expert over the union of the cases, as it does on one call: each expert's weights are
    generated once (not timed), then its share of every case is timed.  Per case: `us` (the
    measured oracle time of the rows taken), `assignments` (their slots), `A` (the call's), and
    `us_call` = us A / assignments: the layer call's oracle time, measured when every row is
    taken and extrapolated per assignment otherwise (`extrapolated`)."""
    import oracle
    from paper_2607_23099_amd import synth
    oracle.build()
    src = synth.ExpertWeightSource(shape)
    prep = {}
    for n, (r, x_tag, rows) in cases.items():
        rows = np.arange(r.T) if rows is None else np.asarray(rows, np.int64)
        ids = r.ids[rows]
        prep[n] = (ids, r.w[rows], synth.activations_host(r.T, shape.H, x_tag, rows),
                   int(np.sum((r.ids >= 0) & (r.ids < shape.E))), int(np.sum((ids >= 0) & (ids < shape.E))),
                   len(rows) < r.T)
    experts = sorted({int(e) for p in prep.values() for e in np.unique(p[0]) if 0 <= e < shape.E})
    spent = {n: 0.0 for n in prep}
    t_start = time.perf_counter()
    for i, e in enumerate(experts):
        wts = src(e)
        for n, (ids, w, x, _, _, _) in prep.items():
            if not np.any(ids == e):
                continue
            t0 = time.perf_counter()
            oracle.moe_rows(ids, w, shape.k, np.arange(len(ids)), x, shape.H, shape.I, [e], lambda _e: wts)
            spent[n] += time.perf_counter() - t0
        if (i + 1) % 64 == 0:
            log(f"oracle {shape.name}: expert {i + 1}/{len(experts)} ({time.perf_counter() - t_start:.0f} s)")
    out = {}
    for n, (_, _, _, A, a, sampled) in prep.items():
        us = spent[n] * 1e6
        out[n] = {"us": round(us, 1), "assignments": a, "A": A, "us_call": round(us * A / max(a, 1), 1),
                  "extrapolated": sampled}
    return out


def load_or_tune_table(dl, x, quick, buckets=DECODE_T):
    from paper_2607_23099_amd import damoe
    path = os.path.join(TABLE_DIR, f"{dl.shape.name}.damoe")
    if os.path.exists(path) and not quick:
        try:
            return damoe.Table.load(path), f"loaded {os.path.relpath(path, ROOT)}"
        except damoe.DamoeError as e:
            log(f"table {path} unusable ({e}); tuning a quick one")
    t0 = time.perf_counter()
    table = damoe.tune(dl.layer, list(buckets), EXTENDED_SKEWS, x, samples=3, reps=3, alpha_samples=32,
                       alpha_iters=50, seed=0x7AB1E)
    return table, f"quick-tuned at start-up in {time.perf_counter() - t0:.1f} s (S=3, reps=3)"


def bootstrap_ci(ratios: np.ndarray, n: int = 2000, seed: int = 0) -> list:
    """95% interval of the geomean of per-step ratios, resampling the steps."""
    rng = np.random.default_rng(seed)
    lr = np.log(ratios)
    g = np.exp(lr[rng.integers(0, len(lr), (n, len(lr)))].mean(axis=1))
    return [round(float(np.quantile(g, 0.025)), 4), round(float(np.quantile(g, 0.975)), 4)]


def trace_measure(torch, dl, path, table, n_steps: int, reps: int, t_max: int = 8192, log_every: int = 50) -> dict:
    """Paired dispatch trace on one layer (Kimi-K2 shape): steps with T log-uniform in
    [1, t_max] and Dirichlet alpha log-uniform in [0.03, 10], a fresh routing per step.

    Per step, every configuration runs reps + 1 times (the first untimed), in an order shuffled
    anew for every pass, each behind a 1 GiB write that evicts the weights from the L2 caches
    and the 256 MB Infinity Cache:
      * variant v: routing without the match, then the fused call with the one-bit candidate
        mask of v -- the same launch path adaptive dispatch takes for a one-kernel bucket;
      * adaptive, twice (A and A'): routing with the exemplar match, then the fused call with
        the bucket's candidates, the kernels reading the device-side choice.
    Latencies are path times (a2-a8), medians over the timed passes.  A' against A is the
    noise floor of the protocol; the per-step best is the minimum over the variants."""
    from paper_2607_23099_amd import damoe, synth
    shape = dl.shape
    td = table.data(shape.E)
    V = [v for v in range(damoe.num_variants()) if damoe.variant_supports(v, dl.wdtype)]
    configs = [("v", v) for v in V] + [("adaptive", 0), ("adaptive", 1)]
    flush = torch.empty(1 << 30, dtype=torch.uint8, device="cuda")
    stream = torch.cuda.current_stream()
    ev = lambda: torch.cuda.Event(enable_timing=True)
    steps = []
    t_start = time.perf_counter()
    for s in range(n_steps):
        T, alpha = synth.trace_step_params(s, t_max)
        r = synth.routing(shape.E, shape.k, T, alpha, synth.seed_trace_step(s))
        path.set_routing(r)
        rng = np.random.default_rng([9, s])
        runs = {c: [] for c in configs}
        for rep in range(reps + 1):
            for ci in rng.permutation(len(configs)):
                kind, v = configs[ci]
                flush.fill_(rep & 0xFF)
                e0, e1 = ev(), ev()
                e0.record(stream)
                if kind == "adaptive":
                    path.route_dispatch(table, T)
                else:
                    path.route(T)
                    path.candidates = 1 << v
                path.fused(T, -1)
                e1.record(stream)
                if rep:
                    runs[configs[ci]].append((e0, e1))
        torch.cuda.synchronize()
        lat = {c: float(np.median([a.elapsed_time(b) for a, b in runs[c]])) * 1e3 for c in configs}
        b = next((i for i, bt in enumerate(td.bucket_T) if T <= bt), len(td.bucket_T) - 1)
        steps.append({"step": s, "T": T, "alpha": alpha, "bucket": b, "chosen": int(path.variant.item()),
                      "adaptive": lat[("adaptive", 0)], "adaptive_b": lat[("adaptive", 1)],
                      "lat": [lat[("v", v)] for v in V]})
        if (s + 1) % log_every == 0:
            log(f"trace step {s + 1}/{n_steps} ({time.perf_counter() - t_start:.0f} s)")
    del flush
    L = np.array([st["lat"] for st in steps])
    A = np.array([st["adaptive"] for st in steps])
    A2 = np.array([st["adaptive_b"] for st in steps])
    B = np.array([st["bucket"] for st in steps])
    step_best = L.min(axis=1)
    noda = np.array([L[i, V.index(int(td.noda[B[i]]))] for i in range(len(steps))])
    chosen = np.array([L[i, V.index(st["chosen"])] if st["chosen"] in V else np.nan for i, st in enumerate(steps)])
    static = np.zeros(len(steps))
    static_choice = {}
    for b in sorted(set(B.tolist())):
        idx = np.where(B == b)[0]
        gm = [np.exp(np.mean(np.log(L[idx, j]))) for j in range(len(V))]
        j = int(np.argmin(gm))
        static_choice[int(td.bucket_T[b])] = damoe.variant_name(V[j])
        static[idx] = L[idx, j]
    g = lambda x: float(np.exp(np.mean(np.log(x))))
    per_bucket = {}
    for b in sorted(set(B.tolist())):
        idx = np.where(B == b)[0]
        per_bucket[int(td.bucket_T[b])] = {
            "steps": int(len(idx)),
            "adaptive_pct_of_step_best": round(100 * g(A[idx] / step_best[idx]), 1),
            "best_static_pct_of_step_best": round(100 * g(static[idx] / step_best[idx]), 1),
            "noda_pct_of_step_best": round(100 * g(noda[idx] / step_best[idx]), 1),
        }
    ok = ~np.isnan(chosen)
    res = {
        "steps": len(steps),
        "reps": reps,
        "speedup_vs_best_static": round(g(static / A), 4),
        "speedup_vs_best_static_ci95": bootstrap_ci(static / A),
        "speedup_vs_noda": round(g(noda / A), 4),
        "speedup_vs_noda_ci95": bootstrap_ci(noda / A, seed=1),
        "adaptive_over_step_best": round(g(A / step_best), 4),
        "adaptive_over_step_best_ci95": bootstrap_ci(A / step_best, seed=2),
        "best_static_over_step_best": round(g(static / step_best), 4),
        # A' over A: the same configuration timed twice, the protocol's noise floor.
        "aa_noise": round(g(A2 / A), 4),
        "aa_noise_ci95": bootstrap_ci(A2 / A, seed=3),
        # Adaptive over its own choice forced: the cost of the match and the device-side read.
        "adaptive_over_chosen_forced": round(g(A[ok] / chosen[ok]), 4),
        "chose_step_best_fraction": round(float(np.mean([V[int(np.argmin(st["lat"]))] == st["chosen"]
                                                         for st in steps])), 3),
        "best_static_choice": static_choice,
        "per_bucket": per_bucket,
    }
    lo = res["speedup_vs_best_static_ci95"][0]
    res["faster_than_best_static"] = bool(lo > 1.0 and lo > res["aa_noise_ci95"][1])
    res["within_5pct_of_step_best"] = bool(res["adaptive_over_step_best_ci95"][1] <= 1.05)
    res["_steps"] = steps
    res["_adaptive_us"] = A
    return res


def trace_oracle(shape, steps, rows_per_step: int = 4) -> dict:
    """The oracle beside the trace: per step, its time on min(T, rows_per_step) token rows of the
    step's routing, extrapolated per assignment to the step's T k; geomean over the steps."""
    from paper_2607_23099_amd import synth
    cases = {}
    for st in steps:
        r = synth.routing(shape.E, shape.k, st["T"], st["alpha"], synth.seed_trace_step(st["step"]))
        rng = np.random.default_rng([10, st["step"]])
        rows = np.sort(rng.choice(r.T, min(r.T, rows_per_step), replace=False))
        cases[st["step"]] = (r, 4, rows)
    leg = oracle_leg(shape, cases)
    us = [leg[n]["us_call"] for n in cases]
    return {"value": round(geomean(us), 1), "unit": "us", "cores": oracle_cores(), "kind": "oracle",
            "sample": f"every trace step on min(T, {rows_per_step}) token rows, fp64, expert-major, weight "
                      "generation excluded; extrapolated per assignment to each step's T k; geomean over steps"}


def run_trace(args):
    """Dispatch trace on the Kimi-K2 shape: adaptive vs per-step best vs static buckets."""
    import torch
    from paper_2607_23099_amd import synth
    from paper_2607_23099_amd.moe import DeviceLayer, Path

    shape = synth.KIMI
    T_MAX = 8192
    log(f"filling {shape.name} weights on the device ({shape.E} experts, bf16)")
    dl = DeviceLayer(shape)
    path = Path(dl, T_MAX)
    path.fill_x(T_MAX, 4)
    torch.cuda.synchronize()
    table, note = load_or_tune_table(dl, path.x, args.quick_tune, [2 ** i for i in range(14)])
    log(f"dispatch table: {note}")
    res = trace_measure(torch, dl, path, table, args.trace_steps, args.trace_reps, T_MAX)
    steps, A = res.pop("_steps"), res.pop("_adaptive_us")
    out = {
        "metric": "geomean dispatch speedup over the best static token-count bucket (Kimi-K2 trace)",
        "value": res["speedup_vs_best_static"],
        "unit": "x",
        "n_gpus": 1,
        "steps": len(steps),
        "warmup": 1,
        "ms_per_step": round(float(np.mean(A)) / 1e3, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": f"kimi-k2 dispatch trace: E=384 top-8 H=7168 I=2048 bf16, {len(steps)} steps, "
                               "T log-uniform in [1,8192], Dirichlet alpha log-uniform in [0.03,10]",
                   "table": note},
        **res,
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = trace_oracle(shape, steps)
    gdir = os.path.join(ROOT, "gpurun_out")
    if os.path.isdir(gdir):
        with open(os.path.join(gdir, "trace_steps.json"), "w") as f:
            json.dump(steps, f)
    print(json.dumps(out), flush=True)


def run_dispatch(args):
    """Dispatch mechanisms on the DeepSeek-V3 decode shape (the analog of the paper's table of
    conditional-graph costs, Sec. V-C): the whole a2-a8 call, host wall clock from an idle
    stream to the end of the call, for
      host      route + match, the variant id copied to the host, then the forced variant
      device    route + match, the kernels read the id in device memory (this build)
      single    route with a one-variant table (no match) + device id
      fixed     route without any dispatch + the forced variant
      graph-*   the device and fixed sequences captured once in a HIP graph and replayed."""
    import torch
    from paper_2607_23099_amd import damoe, synth
    from paper_2607_23099_amd.moe import DeviceLayer, Path

    shape = synth.DS
    log(f"filling {shape.name} weights on the device ({shape.E} experts, bf16)")
    dl = DeviceLayer(shape)
    path = Path(dl, max(DECODE_T))
    path.fill_x(max(DECODE_T), 1)
    torch.cuda.synchronize()
    tuned, note = load_or_tune_table(dl, path.x, args.quick_tune)
    td = tuned.data(shape.E)
    alpha, n = 0.3, args.dispatch_reps
    rows = {}
    for T in DECODE_T:
        b = next((i for i, bt in enumerate(td.bucket_T) if T <= bt), len(td.bucket_T) - 1)
        sl = td.bucket_rows(b)
        q = td.Q[sl]
        best = int(np.bincount(td.kid[sl]).argmax())
        other = 1 if best != 1 else 0
        kid = np.full(len(q), best)
        kid[-1] = other  # two kernels in the row: every call scores the exemplars
        mk = lambda k_: damoe.Table.create(damoe.TableData(E=shape.E, k=shape.k, H=shape.H, I=shape.I, wdtype=0,
                                                           bucket_T=np.array([T]), n_ex=np.array([len(q)]), Q=q,
                                                           kid=k_, noda=np.array([best])))
        match_t, single_t = mk(kid), mk(np.full(len(q), best))
        r = synth.routing(shape.E, shape.k, T, alpha, synth.seed_decode(T, alpha, 0))
        path.set_routing(r)
        path.route_dispatch(match_t, T)
        torch.cuda.synchronize()
        v = int(path.variant.item())

        def host():
            path.route_dispatch(match_t, T)
            path.fused(T, int(path.variant.item()))

        def device():
            path.route_dispatch(match_t, T)
            path.fused(T, -1)

        def single():
            path.route_dispatch(single_t, T)
            path.fused(T, -1)

        def fixed():
            path.route(T)
            path.fused(T, v)

        graphs = {}
        for name, fn in (("graph-device", device), ("graph-fixed", fixed)):
            s_ = torch.cuda.Stream()
            s_.wait_stream(torch.cuda.current_stream())
            with torch.cuda.stream(s_):
                fn()
            torch.cuda.current_stream().wait_stream(s_)
            torch.cuda.synchronize()
            g_ = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g_, stream=s_):
                fn()
            torch.cuda.synchronize()
            graphs[name] = g_
        mech = {"host": host, "device": device, "single": single, "fixed": fixed,
                "graph-device": graphs["graph-device"].replay, "graph-fixed": graphs["graph-fixed"].replay}
        res = {}
        for name, fn in mech.items():
            for _ in range(5):
                fn()
            torch.cuda.synchronize()
            ts = []
            for _ in range(n):
                t0 = time.perf_counter()
                fn()
                torch.cuda.synchronize()
                ts.append((time.perf_counter() - t0) * 1e6)
            res[name] = round(float(np.median(ts)), 1)
        res["variant"] = damoe.variant_name(v)
        rows[f"T{T}"] = res
        log(f"dispatch T={T}: {res}")
    over = lambda name: [rows[k][name] - rows[k]["fixed"] for k in rows]
    out = {
        "metric": "device-side dispatch overhead over a fixed kernel (DeepSeek-V3 decode, median over T)",
        "value": round(float(np.median(over("device"))), 1),
        "unit": "us",
        "n_gpus": 1,
        "steps": n,
        "warmup": 5,
        "ms_per_step": round(float(np.mean([rows[k]["device"] for k in rows])) / 1e3, 4),
        "higher_is_better": False,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": "dsv3 dispatch mechanisms: E=256 top-8 H=7168 I=2048 bf16, T in {1,8,32,128}, "
                               "alpha=0.3, host wall clock per layer call (idle stream to completion)",
                   "table": note},
        "host_copyback_overhead_us": round(float(np.median(over("host"))), 1),
        "single_variant_overhead_us": round(float(np.median(over("single"))), 1),
        "graph_device_over_graph_fixed_us": round(float(np.median(
            [rows[k]["graph-device"] - rows[k]["graph-fixed"] for k in rows])), 1),
        "per_T_us": rows,
    }
    print(json.dumps(out), flush=True)


def bucket_of(td, T: int) -> int:
    return next((i for i, bt in enumerate(td.bucket_T) if T <= bt), len(td.bucket_T) - 1)


def router_bytes(shape, T: int) -> int:
    """Algorithmic HBM bytes of one router call: gate weights and token rows read once, ids and
    gates written (no logits output)."""
    return shape.E * shape.H * 2 + T * shape.H * 2 + T * shape.k * 8


def run_e2e(args):
    """End-to-end MoE layer on the DeepSeek-V3 decode shape (the analog of the paper's
    end-to-end latency figure, Sec. V-C): router (gating logits, top-k, softmax gates), routing
    metadata, dispatch and the fused experts, captured in one HIP graph per token count and
    replayed.  DA-MoE (exemplar match, device-side id) against NoDA (route without a match, the
    bucket's static variant).  The skew comes from the router: a per-expert bias log p,
    p ~ Dirichlet(alpha), over unit-variance logits; REPS token sets and bias draws per point
    are rotated between replays."""
    import torch
    from paper_2607_23099_amd import damoe, synth
    from paper_2607_23099_amd.moe import DeviceLayer, Gate, Path

    shape = synth.DS
    log(f"filling {shape.name} weights and gate on the device")
    dl = DeviceLayer(shape)
    gate = Gate(shape)
    Tm = max(DECODE_T)
    path = Path(dl, Tm)
    stream = torch.cuda.current_stream()
    xs = []
    for rep in range(REPS):
        t = torch.empty((Tm, shape.H), dtype=torch.bfloat16, device="cuda")
        synth.fill_bf16_device(t.data_ptr(), Tm * shape.H, seed=synth.x_seed(700 + rep), tensor=synth.T_X,
                               slab_elems=Tm * shape.H, sigma=1.0, stream=stream.cuda_stream)
        xs.append(t)
    biases = {(a, rep): torch.from_numpy(synth.gate_bias(shape.E, a, [8, int(round(1000 * a)), rep])).cuda()
              for a in DECODE_ALPHA for rep in range(REPS)}
    path.x.copy_(xs[0])
    torch.cuda.synchronize()
    table, note = load_or_tune_table(dl, path.x, args.quick_tune)
    td = table.data(shape.E)

    def capture(fn):
        s_ = torch.cuda.Stream()
        s_.wait_stream(stream)
        with torch.cuda.stream(s_):
            fn()
        stream.wait_stream(s_)
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=s_):
            fn()
        torch.cuda.synchronize()
        return g

    graphs, noda_v = {}, {}
    for T in DECODE_T:
        noda_v[T] = int(td.noda[bucket_of(td, T)])

        def da(T=T):
            path.router(gate, T, logits=False)
            path.route_dispatch(table, T)
            path.fused(T, -1)

        def nd(T=T):
            path.router(gate, T, logits=False)
            path.route(T)
            path.candidates = 0
            path.fused(T, noda_v[T])

        graphs[T] = {"da": capture(da), "noda": capture(nd),
                     "router": capture(lambda T=T: path.router(gate, T, logits=False))}

    ev = lambda: torch.cuda.Event(enable_timing=True)
    # A replay of a short graph is host-bound when the stream is idle: the events would time
    # the host's launch.  Each timed replay is therefore queued behind a GPU spin of ~300 us,
    # so the graph's work is already in the queue when the first event fires.
    spin = gpu_spin(torch, stream)
    rows, t_wall = {}, time.perf_counter()
    for T in DECODE_T:
        for a in DECODE_ALPHA:
            row = {}
            chosen, effs = [], []
            for rep in range(REPS):  # untimed: the variant and skew each rotation leads to
                path.x[:T].copy_(xs[rep][:T])
                gate.bias.copy_(biases[a, rep])
                graphs[T]["da"].replay()
                torch.cuda.synchronize()
                chosen.append(damoe.variant_name(int(path.variant.item())))
                nd_ = path.numden.cpu().numpy()
                effs.append(float(nd_[0]) / max(float(nd_[1]), 1.0))
            row["variants"] = chosen
            row["eff_experts"] = round(float(np.mean(effs)), 1)
            for mode in ("da", "noda", "router"):
                g = graphs[T][mode]
                pairs = []
                for s in range(args.warmup + args.steps):
                    rep = s % REPS
                    path.x[:T].copy_(xs[rep][:T])
                    gate.bias.copy_(biases[a, rep])
                    torch.cuda._sleep(spin)
                    e0, e1 = ev(), ev()
                    e0.record(stream)
                    g.replay()
                    e1.record(stream)
                    if s >= args.warmup:
                        pairs.append((e0, e1))
                torch.cuda.synchronize()
                row[f"{mode}_us"] = round(float(np.mean([p[0].elapsed_time(p[1]) for p in pairs])) * 1e3, 2)
            row["noda_variant"] = damoe.variant_name(noda_v[T])
            row["router_GBs"] = round(router_bytes(shape, T) / (row["router_us"] * 1e-6) / 1e9, 1)
            rows[f"T{T}_a{a}"] = row
            log(f"e2e T={T} alpha={a}: {row}")
    wall = time.perf_counter() - t_wall
    da_g = geomean([r["da_us"] for r in rows.values()])
    nd_g = geomean([r["noda_us"] for r in rows.values()])
    out = {
        "metric": "end-to-end MoE layer latency in one graph (router + metadata + dispatch + fused experts), "
                  "geomean over the DeepSeek-V3 decode skew sweep",
        "value": round(da_g, 2),
        "unit": "us",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(wall / max(args.steps, 1) * 1e3, 3),
        "higher_is_better": False,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": "dsv3-e2e: E=256 top-8 H=7168 I=2048 bf16, T in {1,8,32,128} x router bias "
                               "log Dirichlet(alpha), alpha in {0.05,0.3,1,10}, graph replay",
                   "table": note},
        "noda_us": round(nd_g, 2),
        "speedup_vs_noda": round(nd_g / da_g, 4),
        "router_us_geomean": round(geomean([r["router_us"] for r in rows.values()]), 2),
        "per_point": rows,
    }
    print(json.dumps(out), flush=True)


ROUTER_T = (1, 8, 32, 128, 1024, 4096, 8192)
MFMA_BF16_PEAK_TFS = 2500.0


def gpu_spin(torch, stream, us: float = 300.0):
    """Cycles of torch's GPU spin that take ~us microseconds: queued before a short timed call,
    the spin keeps the GPU busy while the host enqueues the call, so events time the GPU."""
    ev = lambda: torch.cuda.Event(enable_timing=True)
    torch.cuda._sleep(1 << 16)  # the first call pays its own start-up
    torch.cuda.synchronize()
    e0, e1 = ev(), ev()
    torch.cuda._sleep(1 << 16)  # busy while the events and the measured spin are queued
    e0.record(stream)
    torch.cuda._sleep(1 << 22)
    e1.record(stream)
    torch.cuda.synchronize()
    return max(1, int((1 << 22) * us * 1e-3 / max(e0.elapsed_time(e1), 1e-3)))


def run_router(args):
    """The router alone (gating logits, top-k, softmax gates) on the DeepSeek-V3 and Kimi-K2
    gate shapes over decode and prefill token counts: GPU time per call (HIP events behind a
    spin), algorithmic bytes (gate weights + token rows + ids and gates) and FLOPs, and the
    fraction of the bounding roofline t_roof = max(bytes / 8 TB/s, flops / 2.5 PFLOP/s)."""
    import torch
    from paper_2607_23099_amd import damoe, synth
    from paper_2607_23099_amd.moe import Gate

    stream = torch.cuda.current_stream()
    spin = gpu_spin(torch, stream)
    ev = lambda: torch.cuda.Event(enable_timing=True)
    rows = {}
    for sh in (synth.DS, synth.KIMI):
        gate = Gate(sh)
        gate.set_bias(synth.gate_bias(sh.E, 0.3, [9, sh.E]))
        Tm = max(ROUTER_T)
        x = torch.empty((Tm, sh.H), dtype=torch.bfloat16, device="cuda")
        synth.fill_bf16_device(x.data_ptr(), Tm * sh.H, seed=synth.x_seed(800), tensor=synth.T_X,
                               slab_elems=Tm * sh.H, sigma=1.0, stream=stream.cuda_stream)
        ids = torch.empty((Tm, sh.k), dtype=torch.int32, device="cuda")
        w = torch.empty((Tm, sh.k), dtype=torch.float32, device="cuda")
        ws = torch.empty(damoe.router_workspace_size(sh.E, sh.H, Tm), dtype=torch.uint8, device="cuda")
        for T in ROUTER_T:
            for _ in range(args.warmup):
                damoe.router(x, gate.wg, gate.bias, T, sh.H, sh.E, sh.k, None, ids, w, ws)
            pairs = []
            for _ in range(args.steps):
                torch.cuda._sleep(spin)
                e0, e1 = ev(), ev()
                e0.record(stream)
                damoe.router(x, gate.wg, gate.bias, T, sh.H, sh.E, sh.k, None, ids, w, ws)
                e1.record(stream)
                pairs.append((e0, e1))
            torch.cuda.synchronize()
            us = float(np.median([a.elapsed_time(b) for a, b in pairs])) * 1e3
            byts = router_bytes(sh, T)
            flops = 2.0 * T * sh.H * sh.E
            t_hbm, t_mfma = byts / (HBM_PEAK_GBS * 1e3), flops / (MFMA_BF16_PEAK_TFS * 1e6)  # us
            rows[f"{sh.name}_T{T}"] = {"us": round(us, 2), "GBs": round(byts / us / 1e3, 1),
                                       "TFs": round(flops / us / 1e6, 1),
                                       "frac": round(max(t_hbm, t_mfma) / us, 4),
                                       "bound": "hbm" if t_hbm >= t_mfma else "mfma"}
            log(f"router {sh.name} T={T}: {rows[f'{sh.name}_T{T}']}")
        del gate, x
        torch.cuda.empty_cache()
    big = rows[f"{synth.DS.name}_T{max(ROUTER_T)}"]
    out = {
        "metric": "router latency (gating logits + top-k + softmax gates), DeepSeek-V3 gate at T=8192",
        "value": big["us"],
        "unit": "us",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(big["us"] / 1e3, 4),
        "higher_is_better": False,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": "router: E=256 / 384, top-8, H=7168, bf16 x and gate, fp32 bias, "
                               f"T in {list(ROUTER_T)}"},
        "roofline": {"bound": big["bound"], "kernel": "k_router_logits + k_router_topk",
                     "achieved": big["GBs"] if big["bound"] == "hbm" else big["TFs"],
                     "peak": HBM_PEAK_GBS if big["bound"] == "hbm" else MFMA_BF16_PEAK_TFS,
                     "unit": "GB/s" if big["bound"] == "hbm" else "TFLOP/s", "frac": big["frac"],
                     "traffic": None},
        "per_point": rows,
    }
    print(json.dumps(out), flush=True)


IMB_T = (32, 64, 128, 256)
IMB_F = (0, 10, 20, 50, 100)


def run_imbalance(args):
    """Routing-skew ablation (the analog of the paper's imbalance-factor table, Sec. V-E) on the
    DeepSeek-V3 decode shape: T in {32, 64, 128, 256} x f in {0, 10, 20, 50, 100}; groups of
    about f% of the tokens share one routing row (base skew Dirichlet alpha = 1), REPS routings
    per point.  For each routing, the fused-MoE latency (a6-a8, HIP events behind a GPU spin,
    median of --steps runs) of every variant; from these the kernel the exemplar match picks
    (DA-MoE), the kernel the Effective-Experts-only map picks (DA-eff), the bucket's NoDA
    kernel and the per-routing best.  Speedups over NoDA per point and geomean per f."""
    import torch
    from paper_2607_23099_amd import damoe, synth
    from paper_2607_23099_amd.moe import DeviceLayer, Path

    shape = synth.DS
    log(f"filling {shape.name} weights on the device ({shape.E} experts, bf16)")
    dl = DeviceLayer(shape)
    path = Path(dl, max(IMB_T))
    path.fill_x(max(IMB_T), 1)
    torch.cuda.synchronize()
    table, note = load_or_tune_table(dl, path.x, args.quick_tune)
    td = table.data(shape.E)
    stream = torch.cuda.current_stream()
    spin = gpu_spin(torch, stream, 100.0)
    ev = lambda: torch.cuda.Event(enable_timing=True)
    nv = damoe.num_variants()
    rows, t0 = {}, time.perf_counter()
    for T in IMB_T:
        noda = int(td.noda[bucket_of(td, T)])
        for f in IMB_F:
            acc = {"da": [], "eff": [], "noda": [], "best": []}
            picks, effs = [], []
            for rep in range(REPS):
                r = synth.routing_repeated(shape.E, shape.k, T, f, 1.0, synth.seed_imbalance(T, f, rep))
                path.set_routing(r)
                path.route_dispatch_effexp(table, T)
                torch.cuda.synchronize()
                v_eff = int(path.variant.item())
                path.route_dispatch(table, T)
                torch.cuda.synchronize()
                v_da = int(path.variant.item())
                nd_ = path.numden.cpu().numpy()
                effs.append(float(nd_[0]) / max(float(nd_[1]), 1.0))
                path.candidates = 0
                lat = []
                for v in range(nv):
                    if not damoe.variant_supports(v, dl.wdtype):  # fp8-only variants
                        lat.append(float("inf"))
                        continue
                    for _ in range(args.warmup):
                        path.fused(T, v)
                    pairs = []
                    for _ in range(args.steps):
                        torch.cuda._sleep(spin)
                        e0, e1 = ev(), ev()
                        e0.record(stream)
                        path.fused(T, v)
                        e1.record(stream)
                        pairs.append((e0, e1))
                    torch.cuda.synchronize()
                    lat.append(float(np.median([a.elapsed_time(b) for a, b in pairs])) * 1e3)
                acc["da"].append(lat[v_da])
                acc["eff"].append(lat[v_eff])
                acc["noda"].append(lat[noda])
                acc["best"].append(min(lat))
                picks.append((damoe.variant_name(v_da), damoe.variant_name(v_eff)))
            m = {k_: float(np.mean(v_)) for k_, v_ in acc.items()}
            row = {"da_us": round(m["da"], 1), "eff_us": round(m["eff"], 1), "noda_us": round(m["noda"], 1),
                   "best_us": round(m["best"], 1), "da_speedup": round(m["noda"] / m["da"], 4),
                   "eff_speedup": round(m["noda"] / m["eff"], 4), "best_speedup": round(m["noda"] / m["best"], 4),
                   "eff_experts": round(float(np.mean(effs)), 1), "picks_da_eff": picks}
            rows[f"T{T}_f{f}"] = row
            log(f"imbalance T={T} f={f}: {row}")
    wall = time.perf_counter() - t0
    per_f = {}
    for f in IMB_F:
        sel = [rows[f"T{T}_f{f}"] for T in IMB_T]
        per_f[f"f{f}"] = {k_: round(geomean([r_[k_] for r_ in sel]), 4)
                          for k_ in ("da_speedup", "eff_speedup", "best_speedup")}
        log(f"f={f}: geomean {per_f[f'f{f}']}")
    out = {
        "metric": "fused-MoE speedup of DA-MoE over NoDA, geomean over the DeepSeek-V3 imbalance sweep",
        "value": round(geomean([r_["da_speedup"] for r_ in rows.values()]), 4),
        "unit": "x",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(wall * 1e3 / max(len(rows) * REPS, 1), 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": "dsv3-imbalance: E=256 top-8 H=7168 I=2048 bf16, T in {32,64,128,256} x imbalance "
                               "f in {0,10,20,50,100} (repeated routing rows, base Dirichlet alpha = 1)",
                   "table": note},
        "eff_only_speedup": round(geomean([r_["eff_speedup"] for r_ in rows.values()]), 4),
        "best_speedup": round(geomean([r_["best_speedup"] for r_ in rows.values()]), 4),
        "per_f": per_f,
        "per_point": rows,
    }
    print(json.dumps(out), flush=True)


EP_DEGREES = (1, 2, 4, 8)
EP_T = (32, 64, 128, 256)


def run_ep(args):
    """Expert-parallel ranks on one GPU (the analog of the paper's EP ablation, Sec. V-F):
    DeepSeek-V3 at EP in {1, 2, 4, 8} and T in {32, 64, 128, 256} global tokens, routing
    Dirichlet(1) with no repetition.  Rank r holds experts [r E / EP, (r + 1) E / EP) as views
    into the full layer and runs the fused layer on the tokens with a local slot (remote slots
    masked), with its own table (tables/dsv3-ep{EP}.damoe; EP = 1 uses dsv3.damoe).  Every rank
    of every routing is timed for every variant (a6-a8, HIP events behind a GPU spin); the
    exemplar match's kernel (DA-MoE), the bucket's NoDA kernel and the per-rank best are
    compared.  Speedup = NoDA / DA-MoE of the mean per-rank latency, geomean over T."""
    import torch
    from paper_2607_23099_amd import damoe, synth
    from paper_2607_23099_amd.moe import DeviceLayer, Path, RankLayer

    shape = synth.DS
    log(f"filling {shape.name} weights on the device ({shape.E} experts, bf16)")
    dl = DeviceLayer(shape)
    stream = torch.cuda.current_stream()
    spin = gpu_spin(torch, stream, 100.0)
    ev = lambda: torch.cuda.Event(enable_timing=True)
    nv = damoe.num_variants()
    Tm = max(EP_T)
    rows, t0 = {}, time.perf_counter()
    for ep in EP_DEGREES:
        name = "dsv3.damoe" if ep == 1 else f"dsv3-ep{ep}.damoe"
        tpath = os.path.join(TABLE_DIR, name)
        if not os.path.exists(tpath):
            raise SystemExit(f"{tpath} is missing: python -m paper_2607_23099_amd.tune_tables "
                             f"dsv3-ep{ep} --max-T {Tm} --out {tpath}")
        table = damoe.Table.load(tpath)
        local = shape if ep == 1 else synth.DS_EP[ep]
        td = table.data(local.E)
        ranks = [dl if ep == 1 else RankLayer(dl, ep, r_, local) for r_ in range(ep)]
        paths = [Path(rl, Tm) for rl in ranks]
        for p_ in paths:
            p_.fill_x(Tm, 2)
        for T in EP_T:
            acc = {"da": [], "noda": [], "best": []}
            picks, locs = [], []
            for rep in range(REPS):
                r = synth.routing(shape.E, shape.k, T, 1.0, synth.seed_ep(T, rep))
                lat_da, lat_nd, lat_best = [], [], []
                for rank, path in enumerate(paths):
                    keep, ids, w = synth.ep_local(r, ep, rank)
                    tl = len(keep)
                    locs.append(tl)
                    if tl == 0:
                        continue
                    path.set_routing(synth.Routing(ids, w, None, local.E, shape.k, 1.0))
                    path.route_dispatch(table, tl)
                    torch.cuda.synchronize()
                    v_da = int(path.variant.item())
                    noda = int(td.noda[bucket_of(td, tl)])
                    path.candidates = 0
                    lat = []
                    for v in range(nv):
                        if not damoe.variant_supports(v, path.dl.wdtype):  # fp8-only variants
                            lat.append(float("inf"))
                            continue
                        for _ in range(args.warmup):
                            path.fused(tl, v)
                        pairs = []
                        for _ in range(args.steps):
                            torch.cuda._sleep(spin)
                            e0, e1 = ev(), ev()
                            e0.record(stream)
                            path.fused(tl, v)
                            e1.record(stream)
                            pairs.append((e0, e1))
                        torch.cuda.synchronize()
                        lat.append(float(np.median([a.elapsed_time(b) for a, b in pairs])) * 1e3)
                    lat_da.append(lat[v_da])
                    lat_nd.append(lat[noda])
                    lat_best.append(min(lat))
                    picks.append(damoe.variant_name(v_da))
                acc["da"].append(float(np.mean(lat_da)))
                acc["noda"].append(float(np.mean(lat_nd)))
                acc["best"].append(float(np.mean(lat_best)))
            m = {k_: float(np.mean(v_)) for k_, v_ in acc.items()}
            row = {"local_tokens_mean": round(float(np.mean(locs)), 1), "da_us": round(m["da"], 1),
                   "noda_us": round(m["noda"], 1), "best_us": round(m["best"], 1),
                   "da_speedup": round(m["noda"] / m["da"], 4), "best_speedup": round(m["noda"] / m["best"], 4),
                   "kernels_da": sorted(set(picks))}
            rows[f"ep{ep}_T{T}"] = row
            log(f"ep={ep} T={T}: {row}")
        del paths, ranks
        torch.cuda.empty_cache()
    wall = time.perf_counter() - t0
    per_ep = {f"ep{ep}": {k_: round(geomean([rows[f"ep{ep}_T{T}"][k_] for T in EP_T]), 4)
                          for k_ in ("da_speedup", "best_speedup")} for ep in EP_DEGREES}
    for k_, v_ in per_ep.items():
        log(f"{k_}: geomean {v_}")
    out = {
        "metric": "fused-MoE speedup of DA-MoE over NoDA per expert-parallel rank, DeepSeek-V3 at EP = 4 "
                  "(geomean over T in 32..256)",
        "value": per_ep["ep4"]["da_speedup"],
        "unit": "x",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(wall * 1e3 / max(len(rows) * REPS, 1), 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": "dsv3-ep: E=256 top-8 H=7168 I=2048 bf16, EP in {1,2,4,8} rank layers on one GPU, "
                               "T in {32,64,128,256} global tokens, Dirichlet(1) routing, remote slots masked"},
        "per_ep": per_ep,
        "per_point": rows,
    }
    print(json.dumps(out), flush=True)


# Prefill grid: (shape, token counts, alphas, hot experts).  Kimi-K2 routes by Dirichlet 0.05
# with 40% of the mass moved onto 4 hot experts; DeepSeek-V3 carries fp8 block-128 weights.
PREFILL_GRID = (("kimi-k2", (16, 256, 2048, 8192), (0.05,), 4),
                ("dsv3-fp8", (1024, 4096, 16384), (0.05, 0.3, 1.0, 10.0), 0))


def gemm1_alg_bytes(shape, U: int, T: int, wbytes: float) -> float:
    """Algorithmic HBM bytes of one GEMM1 + SwiGLU launch (the decode roofline unit): W1 and W3
    of the U touched experts at `wbytes` per weight (bf16 2, MXFP4 17/32 with its E8M0 scales),
    plus the T token rows of x."""
    return U * 2 * shape.I * shape.H * wbytes + T * shape.H * 2


def path_alg_bytes(shape, U: int, T: int, wbytes: float) -> float:
    """Algorithmic HBM bytes of one decode layer call (a2-a8): W1, W3 and W2 of the U touched
    experts at `wbytes` per weight, x read and y written (T H bf16 each), ids and gates (8 B
    per assignment).  Over 8 TB/s it is the path's roofline time."""
    return U * 3 * shape.I * shape.H * wbytes + 2 * T * shape.H * 2 + 8 * T * shape.k


def prefill_alg(shape, T: int, counts) -> tuple:
    """Algorithmic FLOPs and HBM bytes of one a6-a8 call: 6 H I per assignment; the weights of
    the touched experts (fp8: codes and block scales), x and y, ids and gates."""
    A = int(counts.sum())
    U = int((counts > 0).sum())
    if shape.wdtype == "fp8":
        w_e = 3 * shape.H * shape.I + 3 * (shape.H // 128) * (shape.I // 128) * 4
    else:
        w_e = 3 * shape.H * shape.I * 2
    return 6.0 * shape.H * shape.I * A, float(U * w_e + 2 * T * shape.H * 2 + 8 * T * shape.k), U


def run_prefill(args):
    """Per-variant times over the prefill grid (every variant the layer's weight type supports):
    Kimi-K2 bf16 at T = 16, 256, 2048, 8192 and DeepSeek-V3 fp8 at T = 1024, 4096, 16384 x alpha
    in {0.05, 0.3, 1, 10}.  Per (point, variant), medians of `--steps` timed calls after one
    untimed call: routing (no match), GEMM1, GEMM2, reduce, fused (a6-a8) and path (a2-a8);
    algorithmic and padded TFLOP/s; weight-stream GB/s; and roofline_frac = t_roof / t_fused with
    t_roof = max(B_alg / 8 TB/s, t_MFMA) with t_MFMA = F_GEMM1 / 2.5 PFLOP/s + F_GEMM2 / P2, the
    peaks of the MFMAs the variant issues: bf16 for GEMM1 (fp8 weights are scaled to bf16 in
    registers) and for GEMM2, except the fp8-MFMA big tile's GEMM2 (P2 = 5.0 PFLOP/s fp8); fp8
    points also give the fraction of the 5 PFLOP/s fp8 peak."""
    import torch
    from paper_2607_23099_amd import damoe, synth
    from paper_2607_23099_amd.moe import DeviceLayer, Path

    shapes = {"kimi-k2": synth.KIMI, "dsv3-fp8": synth.DS_FP8}
    rows, points, library = {}, {}, {}
    best = None
    bw, mfma = 8000.0, 2500.0  # GB/s, TFLOP/s
    keep = {tuple(p.split(":")) for p in args.points.split(",") if p}
    for name, Ts, alphas, hot in PREFILL_GRID:
        if keep:
            Ts = tuple(T for T in Ts if (name, str(T)) in keep)
            if not Ts:
                continue
        shape = shapes[name]
        log(f"filling {shape.name} weights")
        dl = DeviceLayer(shape)
        path = Path(dl, max(Ts))
        path.fill_x(max(Ts), 5)
        V = [int(v) for v in args.variants.split(",")] if args.variants else list(range(damoe.num_variants()))
        V = [v for v in V if damoe.variant_supports(v, dl.wdtype)]
        oracle_cases = {}
        for T in Ts:
            for a in alphas:
                r = synth.routing(shape.E, shape.k, T, a, synth.seed_prefill(T, a, 0) if not hot else
                                  synth.seed_kimi(T, 0), n_hot=hot)
                path.set_routing(r)
                oracle_cases[f"{shape.name}_T{T}_a{a}"] = (
                    r, 5, np.sort(np.random.default_rng([11, T]).choice(T, min(T, 16), replace=False)))
                A = T * shape.k
                counts = np.bincount(r.ids.ravel(), minlength=shape.E)
                f_alg, b_alg, U = prefill_alg(shape, T, counts)
                f1, f2 = 4.0 * A * shape.H * shape.I, 2.0 * A * shape.H * shape.I
                t_roof = max(b_alg / bw / 1e3, f_alg / mfma / 1e6)  # us
                pkey = f"{shape.name}_T{T}_a{a}"
                for v in V:
                    bm = damoe.variant_tile_m(v)
                    pad = float(np.sum(-(-counts // bm) * bm)) / A
                    # The peaks of the MFMAs the variant issues: bf16 for GEMM1 (every variant) and
                    # for GEMM2, except the fp8 x fp8 GEMM2 of the fp8-MFMA variants.
                    peak2 = 5000.0 if damoe.variant_name(v) in ("big8_bm256", "deep8_bm64") else mfma
                    t_mfma_v = (f_alg * 2 / 3 / mfma + f_alg / 3 / peak2) / 1e6  # us
                    t_roof_v = max(b_alg / bw / 1e3, t_mfma_v)
                    peak_v = f_alg / t_mfma_v / 1e6  # the effective MFMA peak of the call, TFLOP/s
                    t = []
                    for rep in range(args.steps + 1):
                        e = [torch.cuda.Event(enable_timing=True) for _ in range(5)]
                        e[0].record()
                        path.route(T)
                        e[1].record()
                        path.fused_stage(0, T, v)
                        e[2].record()
                        path.fused_stage(1, T, v)
                        e[3].record()
                        path.fused_stage(2, T, v)
                        e[4].record()
                        torch.cuda.synchronize()
                        if rep:
                            t.append([e[i].elapsed_time(e[i + 1]) * 1e3 for i in range(4)])
                    ta = np.array(t)
                    med = np.median(ta, axis=0)
                    fused = np.median(ta[:, 1:].sum(axis=1))
                    path_us = np.median(ta.sum(axis=1))
                    key = f"{pkey}_{damoe.variant_name(v)}"
                    rows[key] = {"route_us": round(float(med[0]), 1), "gemm1_us": round(float(med[1]), 1),
                                 "gemm2_us": round(float(med[2]), 1), "reduce_us": round(float(med[3]), 1),
                                 "fused_us": round(float(fused), 1), "path_us": round(float(path_us), 1),
                                 "fused_min_us": round(float(ta[:, 1:].sum(axis=1).min()), 1),
                                 "fused_max_us": round(float(ta[:, 1:].sum(axis=1).max()), 1),
                                 "gemm1_tflops": round(float(f1 / med[1]) / 1e6, 1),
                                 "gemm2_tflops": round(float(f2 / med[2]) / 1e6, 1),
                                 "padded_gemm1_tflops": round(float(f1 * pad / med[1]) / 1e6, 1),
                                 "fused_tflops": round(float(f_alg / fused) / 1e6, 1),
                                 "weight_gbs": round(float(b_alg / fused) / 1e3, 1),
                                 "mfma_peak_tflops": round(peak_v, 1),
                                 "roofline_frac": round(float(t_roof_v / fused), 4)}
                    if shape.wdtype == "fp8":
                        rows[key]["fp8_peak_frac"] = round(float(f_alg / fused) / 1e6 / 5000.0, 4)
                    log(f"{key}: {rows[key]}")
                    if shape is synth.KIMI and T == 8192 and (best is None or med[1] < best[1]):
                        best = (key, float(med[1]), f1)  # GEMM1 us
                mine = {k_: v_ for k_, v_ in rows.items() if k_.startswith(pkey + "_")}
                fastest = min(mine, key=lambda k_: mine[k_]["fused_us"])
                points[pkey] = {"touched_experts": U, "alg_gflop": round(f_alg / 1e9, 1),
                                "alg_gb": round(b_alg / 1e9, 3), "roofline_us": round(t_roof, 1),
                                "bound": "hbm" if b_alg / bw / 1e3 >= f_alg / mfma / 1e6 else "mfma",
                                "best_variant": fastest.split(pkey + "_")[1], **mine[fastest]}
                log(f"{pkey}: {points[pkey]}")
                if dl.wdtype == damoe.W_BF16 and T >= 2048:
                    g1best = min(v_["gemm1_us"] for v_ in mine.values())
                    lm = library_gemm1_ms(counts, shape.H, shape.I, args.steps)
                    dm = library_gemm1_ms(np.array([A]), shape.H, shape.I, args.steps)
                    library[pkey] = {"gemm1_us": round(lm * 1e3, 1), "gemm1_tflops": round(f1 / lm / 1e9, 1),
                                     "fused_best_speedup": round(lm * 1e3 / g1best, 3),
                                     "dense_gemm_us": round(dm * 1e3, 1), "dense_tflops": round(f1 / dm / 1e9, 1)}
                    log(f"{pkey} per-expert hipBLASLt GEMM1: {library[pkey]}")
        if not args.no_cpu_baseline:
            # The oracle beside every point: 16 token rows of its routing, timed, extrapolated
            # per assignment to the call.
            log(f"oracle on 16 rows of every {shape.name} point (host cores)")
            for pk, o in oracle_leg(shape, oracle_cases).items():
                points[pk]["oracle_us"] = o["us_call"]
                points[pk]["oracle_extrapolated"] = o["extrapolated"]
                points[pk]["speedup_over_oracle"] = round(o["us_call"] / points[pk]["fused_us"], 1)
        del dl, path
        torch.cuda.empty_cache()
    if best is None:  # a --points selection without Kimi-K2 T = 8192: the best GEMM1 among those run
        k_ = max(rows, key=lambda k2: rows[k2]["gemm1_tflops"])
        best = (k_, rows[k_]["gemm1_us"], rows[k_]["gemm1_tflops"] * rows[k_]["gemm1_us"] * 1e6)
    out = {
        "metric": "grouped GEMM1 + SwiGLU TFLOP/s, Kimi-K2 prefill T=8192 (best variant)",
        "value": round(best[2] / best[1] / 1e6, 1),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": 1,
        "ms_per_step": round(best[1] / 1e3, 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": "prefill grid: kimi-k2 E=384 top-8 H=7168 I=2048 bf16 T in {16, 256, 2048, 8192} "
                               "(alpha 0.05 + 4 hot experts); dsv3 fp8 block-128 T in {1024, 4096, 16384} x "
                               "alpha in {0.05, 0.3, 1, 10}; every supported variant", "best": best[0]},
        "roofline": {"bound": "mfma", "achieved": round(best[2] / best[1] / 1e6, 1), "peak": mfma,
                     "unit": "TFLOP/s", "frac": round(best[2] / best[1] / 1e6 / mfma, 4), "traffic": None},
        # Per point: the fastest variant's fused call and its roofline (bound, t_roof).
        "points": points,
        "per_variant": rows,
        # bf16 points from T = 2048: one hipBLASLt GEMM per touched expert on pre-gathered tokens,
        # against the fastest fused GEMM1 + SwiGLU variant of the same point; and one dense hipBLASLt
        # GEMM of the same FLOPs (T k x H times H x 2I), the practical MFMA ceiling of a plain GEMM.
        "library_gemm1_per_expert": library,
    }
    kp = "kimi-k2_T8192_a0.05"
    if kp in points and "oracle_us" in points[kp]:
        out["cpu_baseline"] = {
            "value": round(points[kp]["alg_gflop"] * 1e3 / points[kp]["oracle_us"], 6), "unit": "TFLOP/s",
            "cores": oracle_cores(), "kind": "oracle",
            "sample": "the Kimi-K2 T=8192 layer's algorithmic FLOPs over the fp64 oracle's time on 16 of its token "
                      "rows, extrapolated per assignment (weight generation excluded); every point carries its own "
                      "oracle_us the same way"}
    print(json.dumps(out), flush=True)


def library_gemm1_ms(counts, H: int, I: int, steps: int) -> float:
    """Library baseline for GEMM1 at one routing: one hipBLASLt GEMM (torch's F.linear) per
    touched expert, x_e [t_e, H] times [W1_e; W3_e]^T.  The tokens are already gathered per
    expert and there is no SwiGLU epilogue, both in the library's favour.  Median over `steps`
    timed passes after one untimed pass, in ms."""
    import torch
    import torch.nn.functional as F
    rows = [int(c) for c in counts if c > 0]
    g = torch.Generator(device="cuda")
    g.manual_seed(11)
    xs = [torch.randn(c, H, device="cuda", dtype=torch.bfloat16, generator=g) for c in rows]
    ws = [torch.randn(2 * I, H, device="cuda", dtype=torch.bfloat16, generator=g) for _ in rows]
    t = []
    for rep in range(steps + 1):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for x, w in zip(xs, ws):
            F.linear(x, w)
        e1.record()
        torch.cuda.synchronize()
        if rep:
            t.append(e0.elapsed_time(e1))
    del xs, ws
    torch.cuda.empty_cache()
    return float(np.median(t))


def run_copy(args):
    """A plain device copy of known size (4 GiB read + 4 GiB written per call), the reference
    for scaling the FETCH_SIZE / WRITE_SIZE counters."""
    import torch
    n = 4 << 30
    src = torch.empty(n, dtype=torch.uint8, device="cuda")
    dst = torch.empty_like(src)
    src.fill_(1)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        dst.copy_(src)
    torch.cuda.synchronize()
    dt = (time.perf_counter() - t0) / args.steps
    print(json.dumps({"metric": "device copy bandwidth (counter calibration)", "value": round(2 * n / dt / 1e9, 1),
                      "unit": "GB/s", "n_gpus": 1, "steps": args.steps, "warmup": 0,
                      "ms_per_step": round(dt * 1e3, 3), "higher_is_better": True, "scaling": "weak",
                      "vs_baseline": None, "dtype": "u8", "data": "synthetic",
                      "config": {"workload": "torch copy_ of 4 GiB", "bytes_read_per_call": n,
                                 "bytes_written_per_call": n}}), flush=True)


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--quick-tune", action="store_true", help="ignore a committed table")
    ap.add_argument("--force-variant", type=int, default=-1, help="time one variant instead of dispatch")
    ap.add_argument("--workload", choices=["decode-sweep", "trace", "dispatch", "prefill", "copy", "e2e", "router", "imbalance", "ep"],
                    default="decode-sweep")
    ap.add_argument("--variants", default="", help="prefill: comma-separated variant ids")
    ap.add_argument("--points", default="", help="prefill: comma-separated points to run, e.g. kimi-k2:8192,dsv3-fp8:16384; "
                    "decode sweep: e.g. T128_a0.05,T128_a1.0")
    ap.add_argument("--wdtype", choices=["bf16", "mxfp4"], default="bf16",
                    help="decode sweep: expert weight format (activations and MFMA stay bf16)")
    ap.add_argument("--dispatch-reps", type=int, default=200)
    ap.add_argument("--trace-steps", type=int, default=1000)
    ap.add_argument("--trace-reps", type=int, default=3)
    ap.add_argument("--bench-trace-steps", type=int, default=100,
                    help="decode sweep: steps of the paired Kimi-K2 dispatch trace reported beside it (0 = none)")
    ap.add_argument("--summarize-trace", default="", metavar="DB_GLOB",
                    help="print the per-kernel table of rocprofv3 --kernel-trace SQLite output and exit")
    ap.add_argument("--summarize-traffic", default="", metavar="PMC_DIR",
                    help="write the GEMM1 traffic summary from rocprofv3 --pmc runs (no GPU needed)")
    args = ap.parse_args()
    if args.summarize_traffic:
        return summarize_traffic(args.summarize_traffic, args.wdtype)
    if args.summarize_trace:
        return summarize_trace(args.summarize_trace)

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU only: this build has no multi-GPU path "
              f"(asked for --gpus {args.gpus}, WORLD_SIZE={world})", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2607_23099_amd import damoe, synth
    from paper_2607_23099_amd.moe import DeviceLayer, Path

    if not torch.cuda.is_available():
        raise SystemExit("bench.py needs a ROCm GPU")
    damoe.lib()  # fails loudly if the HIP library is not built
    if args.workload == "trace":
        return run_trace(args)
    if args.workload == "dispatch":
        return run_dispatch(args)
    if args.workload == "prefill":
        return run_prefill(args)
    if args.workload == "copy":
        return run_copy(args)
    if args.workload == "e2e":
        return run_e2e(args)
    if args.workload == "router":
        return run_router(args)
    if args.workload == "imbalance":
        return run_imbalance(args)
    if args.workload == "ep":
        return run_ep(args)

    shape = synth.DS_MXFP4 if args.wdtype == "mxfp4" else synth.DS
    log(f"filling {shape.name} weights on the device ({shape.E} experts, {args.wdtype})")
    dl = DeviceLayer(shape)
    path = Path(dl, max(DECODE_T))
    points = [(T, a) for T in DECODE_T for a in DECODE_ALPHA]
    if args.points:  # e.g. --points T128_a0.05,T128_a1.0 (counter passes of chosen points)
        keep = set(args.points.split(","))
        points = [(T, a) for (T, a) in points if f"T{T}_a{a}" in keep]
        if not points:
            raise SystemExit(f"no decode point among {args.points}")
    # HBM bytes of one weight element: bf16 2; MXFP4 half a byte of code + 1/32 of a scale byte.
    wbytes = 17.0 / 32.0 if args.wdtype == "mxfp4" else 2.0
    dev = "cuda"
    ids_d, w_d, U = {}, {}, {}
    for (T, a) in points:
        for rep in range(REPS):
            r = synth.routing(shape.E, shape.k, T, a, synth.seed_decode(T, a, rep))
            ids_d[T, a, rep] = torch.from_numpy(r.ids.ravel().copy()).to(dev)
            w_d[T, a, rep] = torch.from_numpy(r.w.ravel().copy()).to(dev)
            U[T, a, rep] = touched_experts(r.ids)
    path.fill_x(max(DECODE_T), 1)
    torch.cuda.synchronize()

    table, table_note = load_or_tune_table(dl, path.x, args.quick_tune)
    log(f"dispatch table: {table_note}")

    stream = torch.cuda.current_stream()
    ev = lambda: torch.cuda.Event(enable_timing=True)
    force = args.force_variant

    def run_point(T, a, rep, events=None, clean=None):
        """One layer call.  `clean` = (start, end) events around the whole call, made as a caller
        would make it (route + dispatch, then one fused call); `events` = 5 events between the
        kernels of the instrumented form (route, GEMM1, GEMM2, reduce as separate calls)."""
        ids, w = ids_d[T, a, rep], w_d[T, a, rep]
        if clean:
            clean[0].record(stream)
            if force < 0:
                path.route_dispatch(table, T, ids=ids)
            else:
                path.route(T, ids=ids)
            path.fused(T, force, w=w)
            clean[1].record(stream)
            return
        if events:
            events[0].record(stream)
        if force < 0:
            path.route_dispatch(table, T, ids=ids)
        else:
            path.route(T, ids=ids)
        if events:
            events[1].record(stream)
        path.fused_stage(0, T, force, w=w)
        if events:
            events[2].record(stream)
        path.fused_stage(1, T, force, w=w)
        if events:
            events[3].record(stream)
        path.fused_stage(2, T, force, w=w)
        if events:
            events[4].record(stream)

    # Each step starts behind a ~1 ms spin, so the host has queued the step's first points
    # before the GPU reaches them and events time the GPU, not the host's launch pace.  Steps
    # alternate between the clean form (path latency: two events per call) and the instrumented
    # form (per-kernel times and the GEMM1 roofline: an event between every two kernels, which
    # adds about 3 us of gap per event to the path, so the path is never taken from it).
    spin = gpu_spin(torch, stream, 1000.0)
    for s in range(args.warmup):
        torch.cuda._sleep(spin)
        for (T, a) in points:
            run_point(T, a, s % REPS)
    torch.cuda.synchronize()

    rec = {p: [] for p in points}
    clean_rec = {p: [] for p in points}
    all_events, all_clean = [], []
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for s in range(args.steps):
        rep = (s // 2 + args.warmup) % REPS  # both forms of a step pair on the same routings
        torch.cuda._sleep(spin)
        for (T, a) in points:
            if s % 2 == 0:
                c = [ev(), ev()]
                run_point(T, a, rep, clean=c)
                all_clean.append(((T, a, rep), c))
            else:
                e = [ev() for _ in range(5)]
                run_point(T, a, rep, e)
                all_events.append(((T, a, rep), e))
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0

    g1_bytes, g1_ms = 0.0, 0.0
    for (T, a, rep), e in all_events:
        g1 = e[1].elapsed_time(e[2])
        g2 = e[2].elapsed_time(e[3])
        rec[T, a].append((e[0].elapsed_time(e[4]), g1, g2, e[0].elapsed_time(e[1]), e[3].elapsed_time(e[4])))
        g1_bytes += gemm1_alg_bytes(shape, U[T, a, rep], T, wbytes)
        g1_ms += g1
    for (T, a, rep), c in all_clean:
        clean_rec[T, a].append(c[0].elapsed_time(c[1]))

    # Per point: medians over the timed steps (a stall of the host between two launches lands
    # inside one step's events), and the path's mean beside its median.
    per_point = {}
    for (T, a), v in rec.items():
        arr = np.array(v)
        med = np.median(arr, axis=0) * 1e3
        cl = np.array(clean_rec[T, a]) * 1e3
        # Path roofline: the mean over the point's routings of its algorithmic bytes / 8 TB/s.
        t_roof = float(np.mean([path_alg_bytes(shape, U[T, a, r], T, wbytes) for r in range(REPS)])) \
            / HBM_PEAK_GBS / 1e3
        per_point[f"T{T}_a{a}"] = {
            "path_us": round(float(np.median(cl)), 1),
            "roofline_us": round(t_roof, 1),
            "roofline_frac": round(t_roof / float(np.median(cl)), 4),
            "path_us_mean": round(float(cl.mean()), 1),
            "instrumented_path_us": round(float(med[0]), 1),
            "gemm1_us": round(float(med[1]), 1),
            "gemm2_us": round(float(med[2]), 1),
            "route_dispatch_us": round(float(med[3]), 1),
            "reduce_us": round(float(med[4]), 1),
        }
    value = geomean([per_point[f"T{T}_a{a}"]["path_us"] for (T, a) in points])
    achieved = g1_bytes / (g1_ms * 1e-3) / 1e9
    for k_, v in per_point.items():
        log(f"{k_:>12}: {v}")

    out = {
        "metric": "fused-MoE layer latency (geomean over the DeepSeek-V3 decode skew sweep)",
        "value": round(value, 2),
        "unit": "us",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(wall / args.steps * 1e3, 3),
        "higher_is_better": False,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": f"dsv3-decode-sweep: E=256 top-8 H=7168 I=2048 {args.wdtype} weights, T in "
                               "{1,8,32,128} x Dirichlet alpha in {0.05,0.3,1,10}, adaptive dispatch"
                               + ("" if force < 0 else f" (forced variant {damoe.variant_name(force)})"),
                   "points": len(points), "table": table_note},
        "roofline": {"bound": "hbm", "kernel": "k_gemm_fp4<GEMM1+SwiGLU>" if args.wdtype == "mxfp4"
                     else "GEMM1+SwiGLU stage: k_gemm, k_gemm_deep where dispatched", "achieved": round(achieved, 1),
                     "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4),
                     "traffic": measured_traffic(args.wdtype),
                     "algorithmic_bytes_per_launch": round(g1_bytes / max(len(all_events), 1)),
                     "launches": len(all_events)},
        "per_point": per_point,
    }
    if not args.no_cpu_baseline:
        log("oracle on every sweep point (host cores)")
        cases = {(T, a): (synth.routing(shape.E, shape.k, T, a, synth.seed_decode(T, a, 0)), 1, None)
                 for (T, a) in points}
        leg = oracle_leg(shape, cases)
        out["cpu_baseline"] = {
            "value": round(geomean([leg[p]["us_call"] for p in points]), 1), "unit": "us",
            "cores": oracle_cores(), "kind": "oracle",
            "sample": f"every one of the {len(points)} sweep points in full ({sum(leg[p]['A'] for p in points)} "
                      "assignments; each point's first routing and the benchmark's tokens), fp64, expert-major, "
                      "weight generation excluded; geomean over the points of the oracle's layer time, as value",
            "per_point_us": {f"T{T}_a{a}": leg[T, a]["us"] for (T, a) in points}}
    if args.bench_trace_steps > 0 and args.wdtype == "bf16" and force < 0:
        # The dispatch half of the metric: a paired Kimi-K2 trace (adaptive against the best
        # static bucket and the per-step best), on a layer of its own.
        del dl, path
        torch.cuda.empty_cache()
        log(f"filling {synth.KIMI.name} weights for the dispatch trace")
        kl = DeviceLayer(synth.KIMI)
        kpath = Path(kl, 8192)
        kpath.fill_x(8192, 4)
        torch.cuda.synchronize()
        ktable, knote = load_or_tune_table(kl, kpath.x, args.quick_tune, [2 ** i for i in range(14)])
        res = trace_measure(torch, kl, kpath, ktable, args.bench_trace_steps, args.trace_reps, 8192, log_every=25)
        steps_ = res.pop("_steps")
        res.pop("_adaptive_us")
        res["workload"] = (f"kimi-k2 dispatch trace: E=384 top-8 H=7168 I=2048 bf16, {len(steps_)} steps, T "
                           "log-uniform in [1,8192], Dirichlet alpha log-uniform in [0.03,10]; table: " + knote)
        if not args.no_cpu_baseline:
            res["cpu_baseline"] = trace_oracle(synth.KIMI, steps_)
        out["dispatch_trace"] = res
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
