"""Host arithmetic of bench.py's roofline figures (no GPU): the algorithmic work per call."""
import importlib.util
import os

import numpy as np

from paper_2607_23099_amd import synth

_HERE = os.path.dirname(os.path.abspath(__file__))


def _bench():
    spec = importlib.util.spec_from_file_location("bench", os.path.join(_HERE, "..", "bench.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


def test_prefill_algorithmic_work_per_expert():
    # Per touched expert: 3 H I weights, 88,080,384 B in bf16 and 44,050,944 B in fp8 with its
    # 2688 fp32 block scales (H = 7168, I = 2048); 6 H I FLOPs per assignment.
    b = _bench()
    for shape, w_e in ((synth.KIMI, 88_080_384), (synth.DS_FP8, 44_050_944)):
        T = 64
        counts = np.zeros(shape.E, np.int64)
        counts[:3] = [T * shape.k - 10, 7, 3]  # three touched experts
        f, by, U = b.prefill_alg(shape, T, counts)
        assert U == 3
        assert f == 6.0 * shape.H * shape.I * T * shape.k
        assert by == 3 * w_e + 2 * T * shape.H * 2 + 8 * T * shape.k


def test_decode_gemm1_algorithmic_bytes():
    # W1 + W3 of one DeepSeek-V3 expert: 58,720,256 B in bf16; MXFP4 codes and scales 17/32 of
    # a byte per weight: 15,597,568 B.  Plus the token rows, T H 2 B.
    b = _bench()
    sh = synth.DS
    assert b.gemm1_alg_bytes(sh, 1, 0, 2.0) == 58_720_256
    assert b.gemm1_alg_bytes(sh, 1, 0, 17.0 / 32.0) == 15_597_568
    assert b.gemm1_alg_bytes(sh, 54, 8, 2.0) == 54 * 58_720_256 + 8 * 7168 * 2


def test_decode_path_algorithmic_bytes():
    # All three matrices of one DeepSeek-V3 expert: 88,080,384 B in bf16; T = 1 touches 8 experts
    # (704,643,072 B, 88.1 us at 8 TB/s) and moves x and y (2 x 14,336 B) and 64 B of ids and gates.
    b = _bench()
    sh = synth.DS
    assert b.path_alg_bytes(sh, 1, 0, 2.0) == 88_080_384
    assert b.path_alg_bytes(sh, 8, 1, 2.0) == 8 * 88_080_384 + 2 * 14_336 + 64
    assert abs(b.path_alg_bytes(sh, 8, 1, 2.0) / 8e12 * 1e6 - 88.1) < 0.05


def test_oracle_leg_measures_and_extrapolates():
    # Every row taken: the call's time is the measured one.  A sample of rows: scaled by the
    # call's assignments over the sample's, and marked as extrapolated.
    b = _bench()
    sh = synth.TINY
    r = synth.routing(sh.E, sh.k, 40, 1.0, [3])
    leg = b.oracle_leg(sh, {"full": (r, 0, None), "sample": (r, 0, np.array([1, 7, 30]))})
    assert leg["full"]["A"] == leg["full"]["assignments"] == 80 and not leg["full"]["extrapolated"]
    assert leg["full"]["us_call"] == leg["full"]["us"] > 0
    s = leg["sample"]
    assert s["assignments"] == 6 and s["A"] == 80 and s["extrapolated"]
    assert abs(s["us_call"] - s["us"] * 80 / 6) <= 0.05 * 80 / 6 + 0.05  # both rounded to 0.1 us


def test_bootstrap_interval_brackets_the_geomean():
    b = _bench()
    rng = np.random.default_rng(0)
    r = np.exp(rng.normal(0.05, 0.02, 400))
    lo, hi = b.bootstrap_ci(r)
    g = float(np.exp(np.mean(np.log(r))))
    assert lo < g < hi and hi - lo < 0.01
    assert b.bootstrap_ci(np.full(50, 1.25)) == [1.25, 1.25]
