"""Offline auto-tuning of dispatch tables (Sec. IV-A) for the named layer shapes.

    python -m paper_2607_23099_amd.tune_tables dsv3 --max-T 128 --out tables/dsv3.damoe
    python -m paper_2607_23099_amd.tune_tables merge low.damoe high.damoe --out tables/x.damoe

The dsv3-ep{2,4,8} shapes are one expert-parallel rank's layer (256 / EP experts); they are
tuned on the rank's share of routings over the whole pool (remote slots masked), and their
tables serve the rank layers of the expert-parallel workload.

For each power-of-two token bucket up to --max-T, each ddist:X skew of the
grid (the paper's {1.1 ... 4.0} extended to 32) and S routing samples, every
variant is timed by the library's tuner, each timed run behind a 1 GiB write that
evicts the caches (as the benchmark's runs are); the table maps each skew's exemplar
to its fastest variant, plus the uniform-routing (NoDA) choice per bucket.
"""
from __future__ import annotations

import argparse
import os
import sys
import time

PAPER_SKEWS = [1.1, 1.3, 1.5, 1.7, 2.0, 2.5, 4.0]
EXTENDED_SKEWS = PAPER_SKEWS + [6.0, 8.0, 12.0, 16.0, 24.0, 32.0]
# Repeated-row exemplars (percent of a batch sharing one routing row).  Tuned with them by
# default: the DeepSeek-V3 decode layers, whose tables serve the repeated-row sweep, and the
# tiny test layer; the others (the Kimi-K2 trace is Dirichlet; expert-parallel ranks cannot
# take them) use the ddist:X skews only unless --repeat is given.
REPEAT_F = [10, 20, 50, 100]
REPEAT_BY_DEFAULT = ("dsv3", "dsv3-fp8", "tiny")
HERE = os.path.dirname(os.path.abspath(__file__))


def bucket_grid(max_T: int, grid: str = "octave") -> list:
    """Tuned token counts up to max_T: the powers of two ("octave"), or also 3 * 2^(i - 1) between
    them ("half": 1, 2, 3, 4, 6, 8, 12, ...).  A batch of T tokens takes the smallest tuned bucket
    >= T, so on the half grid every T is within 1.5x of the count its bucket was tuned at (2x on
    the octave grid)."""
    if grid not in ("octave", "half"):
        raise ValueError(f"unknown bucket grid {grid!r}")
    out, t = [], 1
    while t <= max_T:
        out.append(t)
        if grid == "half" and t >= 2 and 3 * t // 2 <= max_T:
            out.append(3 * t // 2)
        t *= 2
    return out


def merge_tables(paths, out: str) -> None:
    """Concatenate the token buckets of tables tuned for one layer shape over disjoint token
    ranges (in increasing order) into one table.  The files may come from libraries with more
    or fewer variants: variants are only ever appended, so every file's variant set must be a
    prefix of the largest one, whose header the merged table keeps."""
    sigs, shape, blocks = [], None, []
    for path in paths:
        lines = open(path).read().splitlines()
        if not lines or not lines[0].startswith("damoe-table 1 "):
            raise ValueError(f"{path}: not a damoe table")
        sigs.append(lines[0].split(" ", 2)[2].split(",")[1:])
        fields = lines[1].split()
        if shape is not None and fields[:5] != shape:
            raise ValueError(f"{path}: another layer shape ({fields[:5]} vs {shape})")
        shape = fields[:5]
        i = 2
        for _ in range(int(fields[5])):
            head = lines[i].split()
            if head[0] != "bucket":
                raise ValueError(f"{path}: malformed bucket line {lines[i]!r}")
            n_ex = int(head[2])
            blocks.append((int(head[1]), lines[i:i + 1 + n_ex]))
            i += 1 + n_ex
    Ts = [T for T, _ in blocks]
    if Ts != sorted(set(Ts)):
        raise ValueError(f"bucket token counts must increase across the files: {Ts}")
    names = max(sigs, key=len)
    if any(s_ != names[:len(s_)] for s_ in sigs):
        raise ValueError("the files' variant sets are not prefixes of one another")
    with open(out, "w") as f:
        f.write(f"damoe-table 1 {len(names)}," + ",".join(names) + "\n" + " ".join(shape + [str(len(blocks))]) + "\n")
        for _, b in blocks:
            f.write("\n".join(b) + "\n")


def tune_shape(shape_name: str, max_T: int, samples: int, reps: int, seed: int, verbose: bool = True,
               dl=None, repeat_f=None, flush_mib: int = 1024, grid: str = "octave", min_T: int = 1):
    import torch
    from . import damoe, synth
    from .moe import DeviceLayer
    shapes = {"dsv3": synth.DS, "dsv3-fp8": synth.DS_FP8, "dsv3-mxfp4": synth.DS_MXFP4, "kimi-k2": synth.KIMI,
              "tiny": synth.TINY,
              **{f"dsv3-ep{ep}": sh for ep, sh in synth.DS_EP.items()}}
    shape = shapes[shape_name]
    if dl is None:
        dl = DeviceLayer(shape)
    buckets = [t for t in bucket_grid(max_T, grid) if t >= min_T]
    x = torch.empty((max_T, shape.H), dtype=torch.bfloat16, device="cuda")
    synth.fill_bf16_device(x.data_ptr(), x.numel(), seed=synth.x_seed(999), tensor=synth.T_X,
                           slab_elems=x.numel(), sigma=1.0, stream=torch.cuda.current_stream().cuda_stream)
    t0 = time.perf_counter()
    ep = int(shape_name.split("-ep")[1]) if "-ep" in shape_name else 1
    if repeat_f is None:
        repeat_f = REPEAT_F if shape_name in REPEAT_BY_DEFAULT else []
    table = damoe.tune(dl.layer, buckets, EXTENDED_SKEWS, x, samples=samples, reps=reps, seed=seed,
                       verbose=verbose, ep=ep, repeat_f=repeat_f, flush_mib=flush_mib)
    return table, time.perf_counter() - t0, buckets, dl


def main():
    if len(sys.argv) > 1 and sys.argv[1] == "merge":
        # python -m paper_2607_23099_amd.tune_tables merge A.damoe B.damoe ... --out C.damoe
        ap = argparse.ArgumentParser(prog="tune_tables merge")
        ap.add_argument("tables", nargs="+")
        ap.add_argument("--out", required=True)
        args = ap.parse_args(sys.argv[2:])
        merge_tables(args.tables, args.out)
        return
    ap = argparse.ArgumentParser()
    ap.add_argument("shape", choices=["dsv3", "dsv3-fp8", "dsv3-mxfp4", "kimi-k2", "tiny", "dsv3-ep2", "dsv3-ep4",
                                      "dsv3-ep8"])
    ap.add_argument("--max-T", type=int, default=128)
    ap.add_argument("--samples", type=int, default=10)
    ap.add_argument("--reps", type=int, default=5)
    ap.add_argument("--seed", type=int, default=0x7AB1E)
    ap.add_argument("--out", required=True)
    ap.add_argument("--min-T", type=int, default=1, help="tune only the buckets from this token count on")
    ap.add_argument("--grid", choices=["octave", "half"], default="octave",
                    help="tuned token counts: powers of two, or also 3 * 2^(i - 1) between them")
    ap.add_argument("--flush-mib", type=int, default=1024,
                    help="MiB written before every timed run (evicts the caches, as in the benchmark)")
    rep = ap.add_mutually_exclusive_group()
    rep.add_argument("--no-repeat", action="store_true", help="ddist:X skews only")
    rep.add_argument("--repeat", action="store_true", help="add the repeated-row exemplars")
    args = ap.parse_args()
    table, secs, buckets, _ = tune_shape(args.shape, args.max_T, args.samples, args.reps, args.seed,
                                         repeat_f=[] if args.no_repeat else REPEAT_F if args.repeat else None,
                                         flush_mib=args.flush_mib, grid=args.grid, min_T=args.min_T)
    table.save(args.out)
    print(f"tuned {args.shape}: buckets {buckets}, {len(EXTENDED_SKEWS)} skews, S={args.samples}, "
          f"reps={args.reps} in {secs:.1f} s -> {args.out}", file=sys.stderr, flush=True)


if __name__ == "__main__":
    main()
