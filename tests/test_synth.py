"""The seeded input generator: published known answers and distribution checks."""
import math

import numpy as np
import pytest

from paper_2607_23099_amd import synth


@pytest.fixture(scope="module", autouse=True)
def _built():
    import os
    from paper_2607_23099_amd import build
    if not os.path.exists(synth.LIB_PATH):
        build.build_synth()


def test_philox_known_answers():
    # Known-answer vectors published with the Random123 library for philox4x32-10.
    cases = [
        ([0, 0, 0, 0], [0, 0], [0x6627E8D5, 0xE169C58D, 0xBC57AC4C, 0x9B00DBD8]),
        ([0xFFFFFFFF] * 4, [0xFFFFFFFF] * 2, [0x408F276D, 0x41C83B0E, 0xA20BC7C6, 0x6D5451FD]),
        ([0x243F6A88, 0x85A308D3, 0x13198A2E, 0x03707344], [0xA4093822, 0x299F31D0],
         [0xD16CFE09, 0x94FDCCEB, 0x5001E420, 0x24126EA1]),
    ]
    for ctr, key, want in cases:
        assert list(synth.philox4x32_10(ctr, key)) == want


def test_bf16_fill_distribution_and_slicing():
    n = 1 << 20
    v = synth.fill_bf16_host(n, seed=11, tensor=synth.T_W1, sigma=0.02)
    f = synth.bf16_to_f64(v)
    assert abs(f.mean()) < 1e-4
    assert abs(f.std() / 0.02 - 1) < 0.01
    assert np.max(np.abs(f)) < 0.02 * 4.95
    # Irwin-Hall(8) kurtosis is 3 - 1.2/8 = 2.85.
    kurt = np.mean((f - f.mean()) ** 4) / f.var() ** 2
    assert abs(kurt - 2.85) < 0.03
    # A window of the stream equals the same window of the full fill.
    w = synth.fill_bf16_host(1000, seed=11, tensor=synth.T_W1, start=5000, slab_elems=n, sigma=0.02)
    np.testing.assert_array_equal(w, v[5000:6000])
    # Slabs and tensors are independent streams.
    a = synth.fill_bf16_host(4096, seed=11, tensor=synth.T_W1, slab0=1, slab_elems=4096, sigma=0.02)
    b = synth.fill_bf16_host(4096, seed=11, tensor=synth.T_W3, slab0=1, slab_elems=4096, sigma=0.02)
    assert np.mean(a == v[:4096]) < 0.1 and np.mean(a == b) < 0.1
    # Crossing a slab boundary restarts the element index in the next slab.
    two = synth.fill_bf16_host(8192, seed=11, tensor=synth.T_W1, slab0=0, slab_elems=4096, sigma=0.02)
    np.testing.assert_array_equal(two[4096:], a)


def test_fp8_fill_block_quantisation():
    q, s = synth.fill_fp8_host(256, 384, 2, seed=3, tensor=synth.T_W2, sigma=0.02)
    assert q.shape == (2, 256, 384) and s.shape == (2, 2, 3)
    # Every block's largest magnitude maps to +-448 (code 0x7E / 0xFE).
    for sl in range(2):
        for rb in range(2):
            for cb in range(3):
                blk = q[sl, rb * 128:(rb + 1) * 128, cb * 128:(cb + 1) * 128]
                assert np.any((blk & 0x7F) == 0x7E)
                assert not np.any((blk & 0x7F) == 0x7F)
    # Dequantised values are within half an e4m3 step (relative 2^-4) of the bf16 source.
    src = synth.bf16_to_f64(synth.fill_bf16_host(256 * 384, seed=3, tensor=synth.T_W2, slab0=1,
                                                 slab_elems=256 * 384, sigma=0.02)).reshape(256, 384)
    code = q[1].astype(np.int64)
    ex, man, sg = (code >> 3) & 15, code & 7, np.where(code >> 7, -1.0, 1.0)
    val = sg * np.where(ex == 0, man * 2.0 ** -9, (1 + man / 8) * 2.0 ** (ex - 7))
    deq = val * np.kron(s[1], np.ones((128, 128)))
    big = np.abs(src) > 0.02 * 448 / 4.9 / 64  # normal e4m3 range after scaling
    rel = np.abs(deq - src)[big] / np.abs(src)[big]
    assert rel.max() <= 2.0 ** -4 + 1e-9


@pytest.mark.parametrize("E,k,T,alpha,hot", [(8, 2, 64, 1.0, 0), (256, 8, 128, 0.05, 0),
                                             (384, 8, 256, 0.05, 4), (256, 8, 3, None, 0),
                                             (384, 8, 1000, 0.03, 0)])
def test_routing_invariants(E, k, T, alpha, hot):
    r = synth.routing(E, k, T, alpha, [1, T], n_hot=hot)
    assert r.ids.shape == (T, k) and r.ids.dtype == np.int32
    assert r.ids.min() >= 0 and r.ids.max() < E
    assert all(len(set(row)) == k for row in r.ids.tolist())
    assert np.all(r.w > 0) and np.allclose(r.w.sum(1), 1.0, atol=1e-6)
    assert np.all(np.isfinite(r.logp)) and abs(np.logaddexp.reduce(r.logp)) < 1e-12
    if hot:
        assert np.sum(np.exp(r.logp) >= 0.1 - 1e-12) >= hot


def test_routing_is_seeded_and_skew_follows_alpha():
    a = synth.routing(256, 8, 64, 0.3, [1, 2, 3])
    b = synth.routing(256, 8, 64, 0.3, [1, 2, 3])
    np.testing.assert_array_equal(a.ids, b.ids)
    np.testing.assert_array_equal(a.w, b.w)
    # Smaller alpha concentrates p (Sec. II-D): compare mean sum p^2 over draws.
    m = {al: np.mean([np.exp(2 * synth.routing(256, 8, 0, al, [s]).logp).sum() for s in range(200)])
         for al in (0.05, 1.0, 10.0)}
    for al, v in m.items():
        assert abs(v / ((al + 1) / (256 * al + 1)) - 1) < 0.15
    assert m[0.05] > m[1.0] > m[10.0]


def test_trace_params_ranges():
    ts, als = zip(*[synth.trace_step_params(s) for s in range(2000)])
    assert min(ts) >= 1 and max(ts) <= 8192
    assert min(als) >= 0.03 and max(als) <= 10.0
    # log-uniform: median of log T near ln(8192)/2.
    assert abs(np.median(np.log(ts)) - math.log(8192) / 2) < 0.3


def test_routing_repeated_groups():
    for T, f in [(32, 0), (32, 10), (64, 20), (128, 50), (256, 100), (7, 50), (0, 10)]:
        r = synth.routing_repeated(64, 8, T, f, 1.0, [5, T, f])
        assert r.ids.shape == (T, 8) and r.w.shape == (T, 8)
        if T == 0:
            continue
        g = 1 if f == 0 else max(1, round(f * T / 100))
        distinct = {tuple(row) for row in r.ids}
        assert len(distinct) <= -(-T // g)
        for t in range(T):  # tokens of one group share the row, ids and gates
            np.testing.assert_array_equal(r.ids[t], r.ids[(t // g) * g])
            np.testing.assert_array_equal(r.w[t], r.w[(t // g) * g])
        assert np.all(np.sort(r.ids, axis=1)[:, 1:] != np.sort(r.ids, axis=1)[:, :-1])
    # More repetition, fewer Effective Experts (the histogram concentrates).
    import oracle
    oracle.build()
    eff = [oracle.effexp(oracle.histogram(synth.routing_repeated(256, 8, 256, f, 1.0, [5, 256, f, 0]).ids,
                                          256))[2] for f in (0, 10, 50, 100)]
    assert eff[0] > eff[1] > eff[2] > eff[3] == 8.0


def test_mxfp4_quantizer():
    # Scale: X = 2^(floor(log2 amax) - 2); codes: round-to-nearest-even onto the e2m1 grid
    # (ties to an even mantissa bit), saturating at 6; the even element in the low nibble.
    import oracle
    oracle.build()
    grid = np.array([0, 0.5, 1, 1.5, 2, 3, 4, 6])
    w = np.zeros(32, np.float32)
    w[0] = 7.9         # amax: floor(log2 7.9) = 2 -> X = 1, 7.9 saturates to 6
    w[1:8] = [0.25, 0.75, 1.25, 1.75, 2.5, 3.5, 5.0]   # ties -> 0, 1, 1, 2, 2, 4, 4
    w[8:12] = [-0.26, -0.74, 1.26, -5.01]              # just past ties -> -0.5, -0.5, 1.5, -6
    q, s = synth.mxfp4_quantize(w)
    assert s[0] == 127
    codes = np.stack([q & 15, q >> 4], axis=1).ravel()
    dec = np.array([oracle.mxfp4_value(int(c), int(s[0])) for c in codes])
    np.testing.assert_array_equal(dec[:12], [6, 0, 1, 1, 2, 2, 4, 4, -0.5, -0.5, 1.5, -6])
    # A block scaled by 2^-9 gets X 2^-9 smaller and the same codes; an all-zero block X = 1.
    q2, s2 = synth.mxfp4_quantize(w * np.float32(2.0 ** -9))
    assert s2[0] == 127 - 9 and np.array_equal(q2, q)
    q3, s3 = synth.mxfp4_quantize(np.zeros(32, np.float32))
    assert s3[0] == 127 and not q3.any()
    # Round trip on generator values: within half a grid step (at most X) unless the value
    # saturates (amax < 8 X, so at most 2 X), and so within half the block's amax.
    rng = np.random.default_rng(9)
    v = rng.normal(0, 0.02, 32 * 50).astype(np.float32)
    q, s = synth.mxfp4_quantize(v)
    codes = np.stack([q & 15, q >> 4], axis=1).ravel()
    dec = np.array([oracle.mxfp4_value(int(c), int(s[i // 32])) for i, c in enumerate(codes)])
    X = 2.0 ** (s.astype(np.float64) - 127)
    err = np.abs(dec - v)
    sat = np.abs(v) > 6 * np.repeat(X, 32)
    assert np.all(err[~sat] <= np.repeat(X, 32)[~sat] + 1e-12)
    assert np.all(err <= 2 * np.repeat(X, 32) + 1e-12)
    assert np.all(err <= np.repeat(np.abs(v.reshape(-1, 32)).max(axis=1), 32) * 0.5 + 1e-12)
