"""Pins of the CPU oracle against what the paper and the mathematics fix.

None of these re-types an oracle formula: each compares the oracle with a
closed form, an invariant, a special case that reduces to a library routine
(numpy bincount / stable argsort / matmul), or brute force on tiny inputs.
"""
import math
from fractions import Fraction

import numpy as np
import pytest

import oracle
from paper_2607_23099_amd import synth
from tests.brute import moe_per_token, silu


@pytest.fixture(scope="module", autouse=True)
def _built():
    oracle.build()
    from paper_2607_23099_amd import build
    if not __import__("os").path.exists(synth.LIB_PATH):
        build.build_synth()


# ---------------------------------------------------------------- histogram (a2)

@pytest.mark.parametrize("E,k,T,alpha", [(8, 2, 64, 1.0), (256, 8, 128, 0.05), (384, 8, 2048, 10.0),
                                         (256, 8, 1, 0.3), (8, 8, 5, 1.0)])
def test_histogram_is_bincount(E, k, T, alpha):
    r = synth.routing(E, k, T, alpha, [9, T])
    c = oracle.histogram(r.ids, E)
    np.testing.assert_array_equal(c, np.bincount(r.ids.ravel(), minlength=E))
    assert c.sum() == T * k
    assert c.max() <= T  # k distinct experts per token


def test_histogram_skips_out_of_range():
    ids = np.array([0, 3, -1, 4, 2, 3], np.int32)
    c = oracle.histogram(ids, 4)
    np.testing.assert_array_equal(c, [1, 0, 1, 2])


# ---------------------------------------------------------------- Effective Experts (a3)

def test_effexp_closed_forms():
    # Uniform routing gives E exactly; one-hot gives 1 (Sec. III-A).
    for E, c in [(8, 1), (256, 5), (384, 1000)]:
        num, den, eff = oracle.effexp([c] * E)
        assert (num, den) == (E * E * c * c, E * c * c)
        assert eff == float(E)
    num, den, eff = oracle.effexp([0, 0, 9, 0, 0])
    assert num == den == 81 and eff == 1.0
    # Hand-computed: (3+1)^2 / (9+1) = 16/10.
    assert oracle.effexp([3, 1])[:2] == (16, 10)
    # No tokens.
    assert oracle.effexp([0] * 7) == (0, 0, 0.0)


def test_effexp_scale_invariant_and_bounded():
    rng = np.random.default_rng(1)
    for _ in range(50):
        E = int(rng.integers(1, 64))
        c = rng.integers(0, 50, E)
        if c.sum() == 0:
            continue
        n1, d1, e1 = oracle.effexp(c)
        n2, d2, _ = oracle.effexp(c * 7)
        assert Fraction(n1, d1) == Fraction(n2, d2)
        assert 1.0 <= e1 <= E + 1e-12
        assert Fraction(n1, d1) == Fraction(int(c.sum()) ** 2, int((c * c).sum()))


@pytest.mark.parametrize("E,k,T,alpha", [(256, 8, 32, 0.05), (384, 8, 256, 0.03), (256, 8, 8, 10.0)])
def test_effexp_topk_bounds(E, k, T, alpha):
    # k distinct experts per token: t_e <= T, so k <= eff_exp <= min(E, T*k).
    r = synth.routing(E, k, T, alpha, [5, T])
    _, _, eff = oracle.effexp(oracle.histogram(r.ids, E))
    assert k - 1e-9 <= eff <= min(E, T * k) + 1e-9


def test_effexp_balanced_routing_reaches_E():
    E, k, T = 16, 4, 12  # E divides T*k
    ids = np.array([[(t * k + j) % E for j in range(k)] for t in range(T)], np.int32)
    num, den, eff = oracle.effexp(oracle.histogram(ids, E))
    assert Fraction(num, den) == E


def _bucket_brute(counts, E):
    s, s2 = int(sum(counts)), int(sum(int(c) * int(c) for c in counts))
    if s2 == 0:
        return -1
    eff = Fraction(s * s, s2)
    return sum(1 for n, d in oracle.EFFEXP_X if eff <= Fraction(E) / Fraction(n, d))


def test_effexp_bucket_brute_force_and_boundaries():
    rng = np.random.default_rng(2)
    for _ in range(300):
        E = int(rng.choice([8, 64, 256, 384]))
        c = rng.integers(0, 30, E) * (rng.random(E) < rng.random())
        n, d, _ = oracle.effexp(c)
        assert oracle.effexp_bucket(n, d, E) == _bucket_brute(c, E)
    # eff = 4 exactly at E = 8 is on the X = 2 boundary: X in {1.1,1.3,1.5,1.7,2} qualify.
    n, d, _ = oracle.effexp([1, 1, 1, 1, 0, 0, 0, 0])
    assert oracle.effexp_bucket(n, d, 8) == 5
    # Uniform: eff = E > E/1.1 -> bucket 0.  One-hot at E = 256: 1 <= 256/32 -> 13.
    n, d, _ = oracle.effexp([3] * 256)
    assert oracle.effexp_bucket(n, d, 256) == 0
    n, d, _ = oracle.effexp([0] * 255 + [5])
    assert oracle.effexp_bucket(n, d, 256) == 13
    assert oracle.effexp_bucket(0, 0, 256) == -1


# ---------------------------------------------------------------- permutation (a4)

@pytest.mark.parametrize("E,k,T,alpha", [(8, 2, 64, 1.0), (256, 8, 128, 0.05), (384, 8, 1000, 0.3),
                                         (256, 8, 0, 1.0)])
def test_permutation_is_stable_argsort(E, k, T, alpha):
    r = synth.routing(E, k, T, alpha, [6, T])
    offsets, perm, inv = oracle.permute(r.ids, E)
    flat = r.ids.ravel()
    np.testing.assert_array_equal(perm, np.argsort(flat, kind="stable"))
    np.testing.assert_array_equal(offsets, np.concatenate([[0], np.cumsum(np.bincount(flat, minlength=E))]))
    np.testing.assert_array_equal(perm[inv], np.arange(flat.size))
    for e in range(E):
        seg = perm[offsets[e]:offsets[e + 1]]
        assert np.all(flat[seg] == e) and np.all(np.diff(seg) > 0)


def test_permutation_marks_out_of_range():
    offsets, perm, inv = oracle.permute(np.array([1, 5, 0, -2, 1], np.int32), 3)
    np.testing.assert_array_equal(offsets, [0, 1, 3, 3])
    np.testing.assert_array_equal(perm, [2, 0, 4])
    np.testing.assert_array_equal(inv, [1, -1, 0, -1, 2])


# ---------------------------------------------------------------- dispatch (a5)

def test_select_bucket_power_of_two_is_ceil_log2():
    buckets = [2 ** i for i in range(15)]
    for T in list(range(1, 70)) + [127, 128, 129, 5000, 16384, 16385, 10 ** 6]:
        want = min(14, math.ceil(math.log2(T)))
        assert oracle.select_bucket(buckets, T) == want
    # Paper grid {32..512}: T below 32 goes to the first bucket, above 512 to the last.
    grid = [32, 64, 128, 256, 512]
    assert [oracle.select_bucket(grid, t) for t in (1, 32, 33, 512, 600)] == [0, 0, 1, 4, 4]


def test_match_brute_force():
    rng = np.random.default_rng(3)
    for _ in range(200):
        E = int(rng.integers(1, 40))
        n_ex = int(rng.integers(1, 8))
        Q = rng.integers(0, 5, (n_ex, E)).astype(np.int32)
        c = rng.integers(0, 6, E)
        s = sorted((int(v) for v in c), reverse=True)
        scores = [sum(a * int(b) for a, b in zip(s, Q[i])) for i in range(n_ex)]
        best = scores.index(max(scores))
        i, sc = oracle.match(c, Q)
        assert i == best and list(sc) == scores


def test_match_planted_exemplar_and_ties():
    E = 64
    shapes = [np.ones(E), np.r_[np.ones(8) * 8, np.ones(56)], np.r_[100.0, np.zeros(63)],
              np.geomspace(50, 1, E)]
    Q = np.array([np.rint(v / np.linalg.norm(v) * 2 ** 15) for v in shapes], np.int32)
    rng = np.random.default_rng(4)
    for i, v in enumerate(shapes):
        counts = np.rint(v * 10).astype(np.int64)
        rng.shuffle(counts)  # expert identity must not matter
        assert oracle.match(counts, Q)[0] == i
    # Duplicate exemplars tie: the lower index wins.
    Qd = np.stack([Q[1], Q[2], Q[2], Q[1]])
    assert oracle.match(np.rint(shapes[2] * 10), Qd)[0] == 1
    assert oracle.match(np.rint(shapes[1] * 10), Qd)[0] == 0


def test_match_uniform_exemplar_score_is_effexp():
    # eff_exp = E cos^2(t, 1): the score against the unit uniform exemplar u = 1/sqrt(E)
    # is sum(t)/sqrt(E) * 2^15, so (score / 2^15 / ||t||)^2 * E = eff_exp.
    E = 256
    u = 1.0 / math.sqrt(E)
    Q = np.full((1, E), round(u * 2 ** 15), np.int32)  # 2048, exact
    r = synth.routing(E, 8, 64, 0.3, 11)
    c = oracle.histogram(r.ids, E)
    _, sc = oracle.match(c, Q)
    _, _, eff = oracle.effexp(c)
    cos = sc[0] / 2 ** 15 / np.linalg.norm(c)
    assert abs(cos * cos * E - eff) < 1e-9 * eff


def test_tiles_python_loop():
    rng = np.random.default_rng(5)
    for BM in (16, 32, 64, 128, 256):
        c = rng.integers(0, 300, 40) * (rng.random(40) < 0.6)
        want, p = [], 0
        for e, n in enumerate(c):
            j = 0
            while j * BM < n:
                want.append((p + j * BM, e, min(BM, n - j * BM)))
                j += 1
            p += n
        got = oracle.tiles(c, BM)
        assert [tuple(x) for x in got] == want


# ---------------------------------------------------------------- table construction

def test_exemplar_single_uniform_sample():
    E = 256
    Q = oracle.exemplar(np.full((1, E), 3))
    assert np.all(Q == 2048)  # 2^15 / sqrt(256)


def test_exemplar_invariances_and_norm():
    rng = np.random.default_rng(6)
    E, S = 128, 10
    C = np.stack([oracle.histogram(synth.routing(E, 8, 64, 0.1, [7, s]).ids, E) for s in range(S)])
    Q = oracle.exemplar(C)
    # Sorting removes expert identity; power-of-two scaling is exact under normalisation.
    Cp = np.stack([rng.permutation(row) for row in C])
    np.testing.assert_array_equal(oracle.exemplar(Cp), Q)
    np.testing.assert_array_equal(oracle.exemplar(C * 4), Q)
    # Sample order does not matter up to rounding of the centroid sum.
    assert np.max(np.abs(oracle.exemplar(C[::-1]) - Q)) <= 1
    # Unit norm up to quantisation, descending order.
    u = Q / 2 ** 15
    assert abs(np.linalg.norm(u) - 1.0) < E * 0.5 / 2 ** 15
    assert np.all(np.diff(Q) <= 0)
    # Centroid of identical samples equals the sample itself.
    np.testing.assert_array_equal(oracle.exemplar(np.stack([C[0]] * 5)), oracle.exemplar(C[:1]))
    # Direct computation for one sample.
    s = np.sort(C[0])[::-1].astype(float)
    np.testing.assert_array_equal(oracle.exemplar(C[:1]), np.rint(s / np.linalg.norm(s) * 2 ** 15))


def test_fastest_mean():
    lat = np.array([[3.0, 2.0, 2.5], [3.0, 4.0, 2.5]])
    assert oracle.fastest_mean(lat) == 2  # means 3.0, 3.0, 2.5
    lat = np.array([[3.0, 2.0, 2.5], [3.0, 3.0, 3.5]])
    assert oracle.fastest_mean(lat) == 1  # means 3.0, 2.5, 3.0
    assert oracle.fastest_mean(np.array([[1.0, 1.0]])) == 0  # tie: lower index
    assert oracle.fastest_mean(np.array([[2.0, 1.0, 1.0], [2.0, 3.0, 3.0]])) == 0  # 2.0, 2.0, 2.0


# ---------------------------------------------------------------- Dirichlet model and Alg. 1

def test_dirichlet_sample_moments():
    # Dir(alpha 1_E): E[p_i] = 1/E, Var[p_i] = (E-1)/(E^2 (E alpha + 1)), E[sum p^2] = (alpha+1)/(E alpha+1).
    for E, a in [(16, 0.5), (64, 0.05), (8, 3.0)]:
        P = np.exp(np.array([oracle.dirichlet_logp(E, a, s, 3) for s in range(3000)]))
        assert np.allclose(P.sum(1), 1.0, atol=1e-12)
        assert abs(P.mean() - 1 / E) < 1e-12
        var = (E - 1) / (E * E * (E * a + 1))
        assert abs(P.var(0).mean() / var - 1) < 0.06
        m2 = (a + 1) / (E * a + 1)
        assert abs((P ** 2).sum(1).mean() / m2 - 1) < 0.05


def test_dirichlet_small_alpha_no_underflow():
    lp = oracle.dirichlet_logp(384, 0.03, 0, 1)
    assert np.all(np.isfinite(lp))
    assert abs(np.logaddexp.reduce(lp)) < 1e-12


def test_alpha_search_closed_form():
    # Jensen: E[1/sum p^2] >= (E a + 1)/(a + 1), tight for large E a, so the alpha Alg. 1
    # returns for target m lies at or just below a* = (m - 1)/(E - m).
    E = 256
    for m in (232.0, 128.0, 60.0):
        a = oracle.alpha_search(E, m)
        a_star = (m - 1) / (E - m)
        assert 0.85 * a_star < a <= a_star * 1.02, (m, a, a_star)
        # The returned alpha reaches the target mean.
        assert abs(oracle.mean_effexp(E, a) / m - 1) < 1e-6


def test_alpha_search_monotone():
    E = 256
    targets = [8.0, 13.0, 20.0, 40.0, 64.0, 128.0, 200.0, 240.0]
    alphas = [oracle.alpha_search(E, m, S=16, iters=50) for m in targets]
    assert all(b > a for a, b in zip(alphas, alphas[1:]))
    vals = [oracle.mean_effexp(E, a, S=16) for a in (0.01, 0.03, 0.1, 0.3, 1, 3, 10, 100)]
    assert all(b > a for a, b in zip(vals, vals[1:]))
    assert vals[0] >= 1.0 and vals[-1] <= E


# ---------------------------------------------------------------- the MoE layer (a6-a8)

def _f64_weights_of(shape):
    return lambda e: tuple(synth.bf16_to_f64(m) for m in synth.expert_weights_host(shape, e))


def _oracle_y(ids, w, x_u16, shape, rows=None):
    T = ids.shape[0]
    rows = np.arange(T) if rows is None else np.asarray(rows)
    experts = np.unique(ids[rows][ids[rows] >= 0])
    return oracle.moe_rows(ids, w, shape.k, rows, x_u16[rows], shape.H, shape.I, experts,
                           lambda e: synth.expert_weights_host(shape, e))


def test_moe_matches_per_token_brute_force_tiny():
    sh = synth.TINY
    r = synth.routing(sh.E, sh.k, 64, 1.0, 0)
    x = synth.activations_host(64, sh.H, 0)
    y = _oracle_y(r.ids, r.w, x, sh)
    yb = moe_per_token(r.ids, r.w, synth.bf16_to_f64(x), _f64_weights_of(sh))
    assert np.max(np.abs(y - yb)) <= 1e-12 * np.max(np.abs(yb))


def test_moe_row_subset_equals_full_rows():
    sh = synth.TINY
    r = synth.routing(sh.E, sh.k, 40, 0.3, 1)
    x = synth.activations_host(40, sh.H, 1)
    y = _oracle_y(r.ids, r.w, x, sh)
    rows = [39, 0, 17, 17, 5]
    ys = _oracle_y(r.ids, r.w, x, sh, rows)
    np.testing.assert_allclose(ys, y[rows], rtol=0, atol=1e-14 * np.abs(y).max())


def test_moe_dense_special_case():
    # E = 1, k = 1, w = 1: a dense SwiGLU FFN, W2 (silu(W1 x) * (W3 x)), by numpy matmuls.
    rng = np.random.default_rng(8)
    T, H, I = 6, 64, 96
    bits = lambda a: synth.f32_to_bf16_bits(a)
    W1, W3, W2 = bits(rng.normal(0, 0.1, (I, H))), bits(rng.normal(0, 0.1, (I, H))), bits(rng.normal(0, 0.1, (H, I)))
    x = bits(rng.normal(0, 1, (T, H)))
    ids = np.zeros((T, 1), np.int32)
    w = np.ones((T, 1), np.float32)
    y = oracle.moe_rows(ids, w, 1, np.arange(T), x, H, I, [0], lambda e: (W1, W3, W2))
    X, A1, A3, A2 = (synth.bf16_to_f64(v) for v in (x, W1, W3, W2))
    G, U = X @ A1.T, X @ A3.T
    want = (silu(G) * U) @ A2.T
    np.testing.assert_allclose(y, want, rtol=1e-12, atol=1e-12)


def test_moe_permutation_matrix_closed_form():
    # With H = I and W1 = c P1, W3 = P3, W2 = P2 for permutation matrices (row i of P has its 1
    # in column pi[i]), one expert gives y[i] = sum_j w_j silu(c x[pi1[pi2[i]]]) x[pi3[pi2[i]]].
    # A transposed weight would use the inverse permutation and fail this.
    rng = np.random.default_rng(9)
    H = I = 32
    E, k, T = 3, 2, 5
    pis = {e: [rng.permutation(H) for _ in range(3)] for e in range(E)}
    c = 0.5

    def P(pi, scale=1.0):
        m = np.zeros((H, H), np.float32)
        m[np.arange(H), pi] = scale
        return synth.f32_to_bf16_bits(m)

    weights = {e: (P(pis[e][0], c), P(pis[e][1]), P(pis[e][2])) for e in range(E)}
    x = synth.f32_to_bf16_bits(rng.normal(0, 1, (T, H)))
    ids = np.array([[0, 1], [2, 0], [1, 2], [0, 2], [1, 0]], np.int32)
    w = np.array([[0.25, 0.75], [0.5, 0.5], [0.125, 0.875], [1.0, 0.0], [0.375, 0.625]], np.float32)
    y = oracle.moe_rows(ids, w, k, np.arange(T), x, H, I, range(E), lambda e: weights[e])
    xf = synth.bf16_to_f64(x)
    want = np.zeros((T, H))
    for t in range(T):
        for j in range(k):
            p1, p3, p2 = pis[int(ids[t, j])]
            for i in range(H):
                z = c * xf[t, p1[p2[i]]]
                want[t, i] += float(w[t, j]) * (z / (1 + math.exp(-z))) * xf[t, p3[p2[i]]]
    np.testing.assert_allclose(y, want, rtol=1e-13, atol=1e-13)


def test_moe_invariances():
    sh = synth.TINY
    T = 24
    r = synth.routing(sh.E, sh.k, T, 0.5, 2)
    x = synth.activations_host(T, sh.H, 2)
    wts = {e: synth.expert_weights_host(sh, e) for e in range(sh.E)}
    run = lambda ids, w, x, wof: oracle.moe_rows(ids, w, sh.k, np.arange(ids.shape[0]), x, sh.H, sh.I,
                                                 range(sh.E), wof)
    y = run(r.ids, r.w, x, lambda e: wts[e])
    scale = np.abs(y).max()
    # Linear in the gates.
    w2 = np.random.default_rng(1).random(r.w.shape).astype(np.float32)
    ya = run(r.ids, w2, x, lambda e: wts[e])
    yb = run(r.ids, (r.w + w2).astype(np.float32), x, lambda e: wts[e])
    wsum = (r.w + w2).astype(np.float32)  # float32 sum is what the oracle sees
    assert np.allclose(run(r.ids, wsum, x, lambda e: wts[e]), yb)
    assert np.max(np.abs(yb - (y + ya))) < 1e-5 * scale  # gate rounding in fp32 only
    # One-hot gate isolates a single expert; a zero gate removes it.
    w1h = np.zeros_like(r.w)
    w1h[:, 0] = 1
    y1 = run(r.ids, w1h, x, lambda e: wts[e])
    ids_only = r.ids.copy()
    ids_only[:, 1:] = ids_only[:, :1]  # all slots -> slot 0's expert, gates one-hot keep value
    assert np.allclose(run(ids_only, w1h, x, lambda e: wts[e]), y1)
    # Relabelling experts (permuting slabs and remapping ids) leaves y unchanged.
    perm = np.random.default_rng(2).permutation(sh.E)
    ids_r = perm[r.ids].astype(np.int32)
    inv = np.argsort(perm)
    yr = run(ids_r, r.w, x, lambda e: wts[int(inv[e])])
    np.testing.assert_allclose(yr, y, rtol=0, atol=1e-14 * scale)
    # Token permutation permutes y; duplicated rows give duplicated outputs.
    tp = np.random.default_rng(3).permutation(T)
    yt = run(r.ids[tp], r.w[tp], x[tp], lambda e: wts[e])
    np.testing.assert_allclose(yt, y[tp], rtol=0, atol=1e-14 * scale)
    dup = np.r_[np.arange(T), [3, 3]]
    yd = run(r.ids[dup], r.w[dup], x[dup], lambda e: wts[e])
    np.testing.assert_array_equal(yd[T], yd[3])
    np.testing.assert_array_equal(yd[T + 1], yd[3])


def test_e4m3_decode_table():
    # OCP e4m3fn reference values.
    q = np.arange(256, dtype=np.uint8).reshape(1, 1, 256)
    # Decode via the fp8 oracle path: one expert, H = I = 128 is the smallest block; take
    # a weight row that is the code sequence and x = unit vectors.
    known = {0x00: 0.0, 0x01: 2.0 ** -9, 0x07: 7 * 2.0 ** -9, 0x08: 2.0 ** -6, 0x38: 1.0, 0x40: 2.0,
             0x7E: 448.0, 0x80: -0.0, 0xB8: -1.0, 0xFE: -448.0, 0x3C: 1.5, 0x52: 10.0}
    H = I = 128
    for code, val in known.items():
        q1 = np.zeros((I, H), np.uint8)
        q1[0, 0] = code
        q3 = np.zeros((I, H), np.uint8)
        q3[0, 0] = 0x38  # 1.0
        q2 = np.zeros((H, I), np.uint8)
        q2[0, 0] = 0x38
        s = np.ones((1, 1), np.float32)
        x = np.zeros((1, H), np.uint16)
        x[0, 0] = synth.f32_to_bf16_bits(np.array([1.0], np.float32))[0]
        y = oracle.moe_rows(np.zeros((1, 1), np.int32), np.ones((1, 1), np.float32), 1, [0], x, H, I,
                            [0], lambda e: ((q1, s), (q3, s), (q2, s)))
        # y[0] = silu(v * 1) * (1 * 1) * 1
        assert y[0, 0] == pytest.approx(val / (1 + math.exp(-val)), rel=1e-15, abs=0)


def test_fp8_path_equals_bf16_path_when_values_coincide():
    # Codes whose values times a power-of-two scale are exact in bf16 give identical outputs.
    rng = np.random.default_rng(10)
    H = I = 256
    codes = rng.integers(0, 0x7F, (3, 256, 256)).astype(np.uint8)
    codes[codes == 0x7F] = 0
    codes |= (rng.random(codes.shape) < 0.5).astype(np.uint8) << 7
    scales = (2.0 ** rng.integers(-12, -4, (3, 2, 2))).astype(np.float32)
    val = np.vectorize(lambda c: (-1.0) ** (int(c) >> 7) * (
        (int(c) & 7) * 2.0 ** -9 if ((int(c) >> 3) & 15) == 0
        else (1 + (int(c) & 7) / 8) * 2.0 ** (((int(c) >> 3) & 15) - 7)))
    deq = [val(codes[m]) * np.kron(scales[m], np.ones((128, 128))) for m in range(3)]
    bf = [synth.f32_to_bf16_bits(d.astype(np.float32)) for d in deq]
    assert all(np.array_equal(synth.bf16_to_f64(b), d) for b, d in zip(bf, deq))
    x = synth.f32_to_bf16_bits(rng.normal(0, 1, (4, H)))
    ids = np.zeros((4, 1), np.int32)
    w = np.full((4, 1), 0.5, np.float32)
    y8 = oracle.moe_rows(ids, w, 1, np.arange(4), x, H, I, [0],
                         lambda e: ((codes[0], scales[0]), (codes[1], scales[1]), (codes[2], scales[2])))
    yb = oracle.moe_rows(ids, w, 1, np.arange(4), x, H, I, [0], lambda e: tuple(bf))
    np.testing.assert_array_equal(y8, yb)


def test_exemplar_normalises_each_sample_before_the_centroid():
    # One hot expert with 100 tokens and a uniform sample with 1 token each: unit vectors
    # (1,0,0,0) and (1/2,1/2,1/2,1/2), centroid (3/4,1/4,1/4,1/4), norm sqrt(3)/2.
    Q = oracle.exemplar(np.array([[0, 100, 0, 0], [1, 1, 1, 1]]))
    u = np.array([3, 1, 1, 1]) / 4 / (math.sqrt(3) / 2)
    np.testing.assert_array_equal(Q, np.rint(u * 2 ** 15))
    assert list(Q) == [28378, 9459, 9459, 9459]


# ---------------------------------------------------------------- router (the gate in front of a1)

def _router_inputs(T, H, E, seed, sigma_w=None):
    rng = np.random.default_rng(seed)
    x = synth.f32_to_bf16_bits(rng.normal(0, 1, (T, H)))
    wg = synth.f32_to_bf16_bits(rng.normal(0, sigma_w or 1 / math.sqrt(H), (E, H)))
    return x, wg


def test_router_logits_are_the_matmul():
    x, wg = _router_inputs(9, 96, 12, 30)
    bias = np.random.default_rng(31).normal(0, 1, 12).astype(np.float32)
    logits, _, _ = oracle.router(x, wg, 3, bias)
    want = synth.bf16_to_f64(x) @ synth.bf16_to_f64(wg).T + bias.astype(np.float64)
    np.testing.assert_allclose(logits, want, rtol=1e-13, atol=1e-13)


@pytest.mark.parametrize("T,H,E,k", [(17, 64, 8, 2), (5, 128, 256, 8), (3, 32, 5, 5), (4, 64, 9, 1)])
def test_router_topk_is_stable_argsort(T, H, E, k):
    x, wg = _router_inputs(T, H, E, T * E)
    logits, ids, _ = oracle.router(x, wg, k)
    want = np.argsort(-logits, axis=1, kind="stable")[:, :k]
    np.testing.assert_array_equal(ids, want)


def test_router_brute_force_subsets_and_gates():
    # The chosen set maximises the sum of logits over all k-subsets (distinct logits), and
    # the gate of a slot is exp(l) over the sum of exp over the set.
    import itertools
    x, wg = _router_inputs(6, 64, 7, 33)
    for k in (1, 2, 3):
        logits, ids, w = oracle.router(x, wg, k)
        for t in range(6):
            best = max(itertools.combinations(range(7), k), key=lambda s: sum(logits[t, list(s)]))
            assert set(ids[t].tolist()) == set(best)
            z = sum(math.exp(logits[t, e]) for e in best)
            for j in range(k):
                assert w[t, j] == pytest.approx(math.exp(logits[t, ids[t, j]]) / z, rel=1e-12)
            assert all(logits[t, ids[t, j]] >= logits[t, ids[t, j + 1]] for j in range(k - 1))


def test_router_gates_closed_forms_and_shift_invariance():
    x, wg = _router_inputs(8, 64, 16, 34)
    logits, ids, w = oracle.router(x, wg, 1)
    assert np.all(w == 1.0)
    logits, ids, w = oracle.router(x, wg, 2)
    d = logits[np.arange(8), ids[:, 0]] - logits[np.arange(8), ids[:, 1]]
    np.testing.assert_allclose(w[:, 0], 1 / (1 + np.exp(-d)), rtol=1e-13)
    np.testing.assert_allclose(w.sum(axis=1), 1.0, rtol=1e-14)
    # A common bias moves every logit alike: same slots, same gates.
    _, ids2, w2 = oracle.router(x, wg, 2, np.full(16, 5.0, np.float32))
    np.testing.assert_array_equal(ids2, ids)
    np.testing.assert_allclose(w2, w, rtol=1e-12)
    # A large bias on one expert puts it first in every row.
    b = np.zeros(16, np.float32)
    b[11] = 1000.0
    _, ids3, _ = oracle.router(x, wg, 2, b)
    assert np.all(ids3[:, 0] == 11)


def test_router_ties_go_to_the_lower_id():
    # Experts 2, 5, 6 share one gate row, and all-zero tokens tie every expert.
    x, wg = _router_inputs(4, 64, 8, 35)
    wg[5] = wg[2]
    wg[6] = wg[2]
    x[3] = 0
    b = np.zeros(8, np.float32)
    b[[2, 5, 6]] = 100.0
    _, ids, w = oracle.router(x, wg, 3, b)
    np.testing.assert_array_equal(ids[:3], [[2, 5, 6]] * 3)
    np.testing.assert_allclose(w[:3], 1 / 3, rtol=1e-14)
    _, ids, w = oracle.router(x[3:], wg, 4)
    np.testing.assert_array_equal(ids, [[0, 1, 2, 3]])
    np.testing.assert_allclose(w, 0.25, rtol=1e-14)


def test_topk_softmax_on_given_logits():
    # Selection on given values (as the GPU checks feed it fp32 logits): heavy ties from a
    # coarse grid, against numpy's stable argsort; gates against scipy's softmax.
    from scipy.special import softmax
    rng = np.random.default_rng(36)
    l = rng.integers(-3, 4, (50, 20)).astype(np.float32) / 4
    for k in (1, 4, 20):
        ids, w = oracle.topk_softmax(l, k)
        np.testing.assert_array_equal(ids, np.argsort(-l.astype(np.float64), axis=1, kind="stable")[:, :k])
        want = softmax(np.take_along_axis(l.astype(np.float64), ids, axis=1), axis=1)
        np.testing.assert_allclose(w, want, rtol=1e-13)


# ---------------------------------------------------------------- Effective-Experts-only dispatch (f4)

def test_effexp_map_hand_worked():
    # E = 64: the uniform exemplar has Effective Experts 64 (bucket 0), an exemplar with 16
    # equal entries 16 (X <= 4 pass: bucket 7), a one-hot exemplar 1 (bucket 13).  Empty
    # buckets take the nearest populated one, the lower on a tie (bucket 10 is 3 from 7 and
    # from 13); bucket -1 is the NoDA kernel.
    E = 64
    uni = np.full(E, 4096)
    m16 = np.r_[np.full(16, 8192), np.zeros(E - 16)]
    one = np.r_[32768, np.zeros(E - 1)]
    Q = np.stack([uni, m16, one]).astype(np.int32)
    got = oracle.effexp_map(Q, [3, 5, 1], noda=7)
    want = [7] + [3] * 4 + [5] * 7 + [1] * 3
    np.testing.assert_array_equal(got, want)
    # A second exemplar in a bucket loses to the first; scaling an exemplar changes nothing.
    got = oracle.effexp_map(np.stack([uni, m16, m16 * 2, one]).astype(np.int32), [3, 5, 6, 1], noda=7)
    np.testing.assert_array_equal(got, want)
    got = oracle.effexp_map(np.stack([one, uni // 2]).astype(np.int32), [2, 4], noda=0)
    np.testing.assert_array_equal(got, [0] + [4] * 7 + [2] * 7)


def test_effexp_map_brute_force_fractions():
    # The bucket of each exemplar from exact fractions, then the nearest-populated rule.
    rng = np.random.default_rng(37)
    X = [Fraction(11, 10), Fraction(13, 10), Fraction(3, 2), Fraction(17, 10), Fraction(2), Fraction(5, 2),
         Fraction(4), Fraction(6), Fraction(8), Fraction(12), Fraction(16), Fraction(24), Fraction(32)]
    for _ in range(60):
        E = int(rng.integers(2, 80))
        n_ex = int(rng.integers(1, 9))
        Q = -np.sort(-rng.integers(0, 30000, (n_ex, E)) * (rng.random((n_ex, E)) < rng.random()), axis=1)
        Q[:, 0] = np.maximum(Q[:, 0], 1)
        kid = rng.integers(0, 8, n_ex)
        first = {}
        for x in range(n_ex):
            eff = Fraction(int(Q[x].sum()) ** 2, int((Q[x].astype(object) ** 2).sum()))
            b = sum(1 for xx in X if eff <= Fraction(E) / xx)
            first.setdefault(b, x)
        want = [5]
        for b in range(14):
            pops = sorted(first, key=lambda p: (abs(p - b), p))
            want.append(int(kid[first[pops[0]]]))
        np.testing.assert_array_equal(oracle.effexp_map(Q.astype(np.int32), kid, noda=5), want)


def test_moe_masked_slots_equal_zero_gates():
    # Expert parallelism: a masked slot (negative id) contributes nothing, exactly like a slot
    # that names any expert with gate 0.
    sh = synth.TINY
    r = synth.routing(sh.E, sh.k, 24, 0.3, 13)
    x = synth.activations_host(24, sh.H, 13)
    ids_m = r.ids.copy()
    ids_m[::3, 1] = -1
    ids_m[5] = -1
    ids_z, w_z = r.ids.copy(), r.w.copy()
    w_z[ids_m < 0] = 0.0
    y_m = _oracle_y(ids_m, r.w, x, sh)
    y_z = _oracle_y(ids_z, w_z, x, sh)
    np.testing.assert_array_equal(y_m, y_z)
    assert np.all(y_m[5] == 0.0)


# ---------------------------------------------------------------- MXFP4 weights (NEXT row f3)

def test_mxfp4_decode_table():
    # OCP MX FP4 (e2m1): the 16 codes in order, and E8M0 scales 2^(s - 127) (255 is NaN).
    want = [0.0, 0.5, 1.0, 1.5, 2.0, 3.0, 4.0, 6.0, -0.0, -0.5, -1.0, -1.5, -2.0, -3.0, -4.0, -6.0]
    got = [oracle.mxfp4_value(c, 127) for c in range(16)]
    assert got == want
    assert oracle.mxfp4_value(2, 0) == 2.0 ** -127 and oracle.mxfp4_value(2, 254) == 2.0 ** 127
    assert oracle.mxfp4_value(7, 120) == 6.0 * 2.0 ** -7
    assert math.isnan(oracle.mxfp4_value(2, 255))


def test_mxfp4_layer_equals_bf16_layer_on_decoded_values():
    # Random codes and scales; the bf16 weights hold the decoded values (exact in bf16), so
    # both layers must agree bit for bit.  A swapped nibble order, a scale indexed by column
    # block of the wrong width or a transposed scale array would break the equality.
    rng = np.random.default_rng(40)
    T, H, I, E, k = 5, 64, 96, 3, 2
    codes = {m: rng.integers(0, 16, (E, r, c)).astype(np.uint8) for m, (r, c) in
             {"w1": (I, H), "w3": (I, H), "w2": (H, I)}.items()}
    scales = {m: rng.integers(118, 131, (E, r, c // 32)).astype(np.uint8) for m, (r, c) in
              {"w1": (I, H), "w3": (I, H), "w2": (H, I)}.items()}
    table = np.array([0.0, 0.5, 1.0, 1.5, 2.0, 3.0, 4.0, 6.0, -0.0, -0.5, -1.0, -1.5, -2.0, -3.0, -4.0, -6.0])

    def packed(m, e):
        c = codes[m][e]
        return (c[:, 0::2] | (c[:, 1::2] << 4)).astype(np.uint8)

    def decoded_bf16(m, e):
        c, s = codes[m][e], scales[m][e]
        v = table[c] * np.repeat(2.0 ** (s.astype(np.float64) - 127), 32, axis=1)
        return synth.f32_to_bf16_bits(v.astype(np.float32))

    r = synth.routing(E, k, T, 1.0, 41)
    x = synth.f32_to_bf16_bits(rng.normal(0, 1, (T, H)))
    y4 = oracle.moe_rows(r.ids, r.w, k, np.arange(T), x, H, I, range(E),
                         lambda e: tuple((packed(m, e), scales[m][e]) for m in ("w1", "w3", "w2")))
    yb = oracle.moe_rows(r.ids, r.w, k, np.arange(T), x, H, I, range(E),
                         lambda e: tuple(decoded_bf16(m, e) for m in ("w1", "w3", "w2")))
    np.testing.assert_array_equal(y4, yb)
    assert np.abs(y4).max() > 0
