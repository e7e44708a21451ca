"""C-ABI checks that need no GPU: exports, argument validation, layout, host-side math."""
import ctypes
import os
import re

import numpy as np
import pytest

import oracle
from paper_2607_23099_amd import damoe

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module", autouse=True)
def _built():
    if not os.path.exists(damoe.LIB_PATH):
        from paper_2607_23099_amd import build
        build.build_damoe()
    oracle.build()


def _declared():
    src = open(os.path.join(ROOT, "include", "damoe.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(damoe_[a-z0-9_]+)\s*\(", src)))


def test_every_declared_symbol_is_exported():
    names = _declared()
    assert len(names) >= 18
    L = ctypes.CDLL(damoe.LIB_PATH)
    for n in names:
        assert hasattr(L, n), n
    assert set(names) == set(damoe.EXPORTED)


def test_status_strings_and_registry():
    L = damoe.lib()
    for code in damoe.STATUS:
        assert L.damoe_status_string(code)
    nv = damoe.num_variants()
    assert nv >= 3
    names = [damoe.variant_name(v) for v in range(nv)]
    assert len(set(names)) == nv and all(names)
    assert damoe.variant_name(nv) == "" and damoe.variant_tile_m(-1) == 0
    assert all(damoe.variant_tile_m(v) in (16, 32, 64, 128, 256) for v in range(nv))
    # Every variant runs fp8 weights.
    assert all(damoe.variant_supports(v, damoe.W_FP8_B128) for v in range(nv))
    # The fp8-MFMA variants (GEMM2 on fp8 codes of h) run fp8 weights only.
    fp8_only = [names.index("big8_bm256"), names.index("deep8_bm64")]
    assert [v for v in range(nv) if not damoe.variant_supports(v, damoe.W_BF16)] == fp8_only
    assert not any(damoe.variant_supports(v, damoe.W_MXFP4) for v in fp8_only)
    assert not damoe.variant_supports(0, 7)


def test_table_signature_prefix(tmp_path):
    """A table saved by a library with fewer variants (the first n of this one's, same names)
    loads; a header naming another variant, or more variants than the library has, does not."""
    nv = damoe.num_variants()
    names = [damoe.variant_name(v) for v in range(nv)]
    src = os.path.join(ROOT, "paper_2607_23099_amd", "tables", "dsv3.damoe")
    body = open(src).read().split("\n", 1)[1]
    for n, sig_names, ok in [(nv - 1, names[:-1], True), (nv, names, True), (2, names[:2], True),
                             (nv - 1, names[:-2] + ["bogus"], False), (nv + 1, names + ["next"], False)]:
        f = tmp_path / f"t{n}_{ok}.damoe"
        f.write_text(f"damoe-table 1 {n},{','.join(sig_names)}\n" + body)
        if ok:
            damoe.Table.load(str(f))
        else:
            with pytest.raises(RuntimeError):
                damoe.Table.load(str(f))


def test_workspace_layout():
    for (E, k, H, I, T) in [(8, 2, 256, 512, 64), (256, 8, 7168, 2048, 128), (384, 8, 7168, 2048, 8192),
                            (256, 8, 7168, 2048, 0), (1024, 16, 256, 128, 3000), (37, 5, 64, 64, 1639)]:
        lo = damoe.workspace_layout(E, k, H, I, T)
        A = T * k
        nbp = (-(-A // 2048) + 3) // 4 * 4  # 2048-assignment blocks, rows padded to a multiple of 4
        # Per-block counts and offsets, and the tile starts of each size, at many tokens.
        route = (2 * nbp + damoe.N_TILE_SIZES) * E * 4 if A >= 8192 else 0
        regions = [(lo["ctrl"], 256)] + [(o, 8 + 8 * lo["tiles_cap"]) for o in lo["tiles"]] + \
                  [(lo["route"], route), (lo["h"], A * I * 2), (lo["out"], A * H * 2)]
        assert lo["route"] + route <= lo["h"]  # the routing calls need the workspace up to h
        for off, size in regions:
            assert off % 256 == 0 and off + size <= lo["total"]
        ends = sorted(regions)
        assert all(a[0] + a[1] <= b[0] for a, b in zip(ends, ends[1:]))
        # Enough tile slots for the worst case of every tile size.
        assert lo["tiles_cap"] >= A // 16 + min(E, A)
    L = damoe.lib()
    bad = damoe.WsLayout()
    assert L.damoe_workspace_layout(0, 1, 128, 128, 4, ctypes.byref(bad)) == -1
    # At most 2^20 tokens per call (the largest layout still fits the 32-bit positions).
    assert L.damoe_workspace_layout(1024, 16, 128, 128, 1 << 20, ctypes.byref(bad)) == 0
    assert L.damoe_workspace_layout(1024, 16, 128, 128, (1 << 20) + 1, ctypes.byref(bad)) == -1
    assert L.damoe_workspace_layout(8, 9, 128, 128, 4, ctypes.byref(bad)) == -1
    assert L.damoe_workspace_layout(2048, 8, 128, 128, 4, ctypes.byref(bad)) == -1
    assert L.damoe_workspace_layout(8, 2, 128, 128, -1, ctypes.byref(bad)) == -1


def test_tile_lists_of_two_token_counts_do_not_line_up():
    # The tile lists sit at offsets that depend on T (their capacity grows with T k), so a fused
    # call with another T than its routing call would read another list's entries or memory no
    # routing call wrote: the reason the routing call stamps each list with T k and the GEMM
    # kernels read only lists stamped with their own.
    for (E, k, T1, T2) in [(256, 8, 128, 64), (8, 2, 200, 150), (384, 8, 8192, 2048)]:
        a = damoe.workspace_layout(E, k, 7168, 2048, T1)
        b = damoe.workspace_layout(E, k, 7168, 2048, T2)
        assert a["tiles_cap"] != b["tiles_cap"]
        assert a["tiles"][0] == b["tiles"][0]  # the first list starts at the same offset
        assert all(x != y for x, y in zip(a["tiles"][1:], b["tiles"][1:]))
        assert a["h"] != b["h"] and a["out"] != b["out"]


def _fake_layer(**kw):
    d = dict(E=8, k=2, H=256, I=512, wdtype=0, layout=0, w1=0x1000, w3=0x2000, w2=0x3000, s1=0, s3=0, s2=0)
    d.update(kw)
    return damoe.Layer(d["E"], d["k"], d["H"], d["I"], d["wdtype"], d["layout"], d["w1"], d["w3"], d["w2"],
                       d["s1"], d["s3"], d["s2"])


def test_validation_before_launch():
    L = damoe.lib()
    P = 0x10000  # never dereferenced: every call below must fail validation first
    ws_ok = 1 << 30
    # route_histogram
    assert L.damoe_route_histogram(P, 4, 3, 2, P, P, P, P, P, P, P, ws_ok, None) == -1  # k > E
    assert L.damoe_route_histogram(P, -1, 2, 8, P, P, P, P, P, P, P, ws_ok, None) == -1
    assert L.damoe_route_histogram(P, 4, 2, 8, None, P, P, P, P, P, P, ws_ok, None) == -1
    assert L.damoe_route_histogram(None, 4, 2, 8, P, P, P, P, P, P, P, ws_ok, None) == -1
    assert L.damoe_route_histogram(P, 4, 2, 8, P, P, P, P, P, P, P, 16, None) == -3
    assert L.damoe_route_histogram(P, 4, 2, 4096, P, P, P, P, P, P, P, ws_ok, None) == -1
    # fused_moe
    fm = L.damoe_fused_moe
    lay = _fake_layer()
    assert fm(None, P, P, 4, P, P, P, -1, 0, P, P, ws_ok, None) == -1
    assert fm(ctypes.byref(_fake_layer(H=200)), P, P, 4, P, P, P, -1, 0, P, P, ws_ok, None) == -2
    assert fm(ctypes.byref(_fake_layer(w2=0)), P, P, 4, P, P, P, -1, 0, P, P, ws_ok, None) == -1
    assert fm(ctypes.byref(_fake_layer(wdtype=1)), P, P, 4, P, P, P, -1, 0, P, P, ws_ok, None) == -1  # no scales
    assert fm(ctypes.byref(_fake_layer(wdtype=1, s1=P, s3=P, s2=P)), P, P, 4, P, P, P, -1, 0, P, P, ws_ok,
              None) == -2  # fp8 needs H, I multiples of 512
    assert fm(ctypes.byref(_fake_layer(wdtype=5)), P, P, 4, P, P, P, -1, 0, P, P, ws_ok, None) == -2
    assert fm(ctypes.byref(_fake_layer(layout=2)), P, P, 4, P, P, P, -1, 0, P, P, ws_ok, None) == -2
    # pack_weights: the source must be row-major and the destinations must not overlap it
    pk = L.damoe_pack_weights
    assert pk(ctypes.byref(_fake_layer(layout=1)), P, P, P, None) == -1
    assert pk(ctypes.byref(_fake_layer()), 0x1000, 0x900000, 0xA00000, None) == -1  # w1 dst == w1 src
    assert pk(ctypes.byref(_fake_layer()), None, P, P, None) == -1
    far = 1 << 40
    assert pk(ctypes.byref(_fake_layer()), far, far + (1 << 20), far + (1 << 30), None) == -1  # w1, w3 dsts overlap
    # MXFP4: row-major needs scales; packed carries them (so the 512-multiple check is reached
    # first); destinations (E rows cols 17 / 32 bytes) must not overlap the scale sources either
    fp4 = dict(wdtype=2, H=512, I=512)
    assert fm(ctypes.byref(_fake_layer(**dict(fp4, H=256))), P, P, 4, P, P, P, -1, 0, P, P, ws_ok, None) == -1
    assert fm(ctypes.byref(_fake_layer(**dict(fp4, H=256), layout=1)), P, P, 4, P, P, P, -1, 0, P, P, ws_ok,
              None) == -2
    s1 = far + (1 << 34)
    lay4 = _fake_layer(**fp4, s1=s1, s3=s1 + (1 << 30), s2=s1 + (2 << 30))
    n = 8 * 512 * 512
    assert pk(ctypes.byref(lay4), s1 - n // 32 * 17 + 1, far, far + (1 << 30), None) == -1
    assert pk(ctypes.byref(lay4), far, far + (1 << 31), s1 + (1 << 30) - 100, None) == -1  # w2 dst over s3
    assert fm(ctypes.byref(lay), P, P, 4, P, P, P, damoe.num_variants(), 0, P, P, ws_ok, None) == -1
    assert fm(ctypes.byref(lay), P, P, 4, P, P, None, -1, 0, P, P, ws_ok, None) == -1  # no variant id
    assert fm(ctypes.byref(lay), P, P, 4, P, P, P, -1, 0, P, P, 1024, None) == -3
    assert fm(ctypes.byref(lay), P, P, -2, P, P, P, -1, 0, P, P, ws_ok, None) == -1
    assert fm(ctypes.byref(lay), None, None, 0, None, None, None, 0, 0, None, None, 0, None) == 0  # T = 0 no-op
    # candidates: bits beyond the registry are rejected; T * H * 2 must fit 31 bits
    nv = damoe.num_variants()
    assert fm(ctypes.byref(lay), P, P, 4, P, P, P, -1, 1 << nv, P, P, ws_ok, None) == -1
    assert fm(ctypes.byref(_fake_layer(H=7168)), P, P, 150000, P, P, P, -1, 0, P, P, 1 << 50, None) == -2
    # dispatch
    assert L.damoe_dispatch(None, P, 4, P, P, ws_ok, None) == -1
    # workspace size of an invalid layer is 0
    assert damoe.workspace_size(_fake_layer(k=0), 4) == 0
    assert damoe.workspace_size(_fake_layer(), 64) == damoe.workspace_layout(8, 2, 256, 512, 64)["total"]


def test_alpha_search_matches_oracle_and_closed_form():
    # Both sides solve Alg. 1's equation over the same counter-based random numbers, with
    # different root finders (the library bisects log alpha, the oracle alpha itself): they
    # must land on the same root, and the mean there must equal the target.
    for E, m in [(256, 128.0), (256, 13.0), (384, 200.0), (8, 4.0), (256, 8.4), (384, 380.0)]:
        a_lib = damoe.alpha_search(E, m, 32, 60, 5)
        a_or = oracle.alpha_search(E, m, S=32, iters=60, seed=5)
        assert a_lib == pytest.approx(a_or, rel=1e-7)
        assert oracle.mean_effexp(E, a_lib, S=32, seed=5) == pytest.approx(m, rel=1e-6)
    # Fewer halvings stop early but stay bracketed around the same root.
    a10 = damoe.alpha_search(256, 128.0, 32, 10, 5)
    assert 0.1 < a10 / oracle.alpha_search(256, 128.0, S=32, iters=60, seed=5) < 10
    a = damoe.alpha_search(256, 128.0, 64, 60, 0)
    assert a == pytest.approx(127.0 / 128.0, rel=0.05)


def test_table_roundtrip_host(tmp_path):
    rng = np.random.default_rng(0)
    E = 16
    nv = damoe.num_variants()
    td = damoe.TableData(E=E, k=2, H=256, I=512, wdtype=0, bucket_T=np.array([1, 4, 16]),
                         n_ex=np.array([2, 3, 1]), Q=rng.integers(0, 32768, (6, E)),
                         kid=rng.integers(0, nv, 6), noda=np.array([0, 1, 2]) % nv)
    t = damoe.Table.create(td)
    got = t.data(E)
    np.testing.assert_array_equal(got.bucket_T, td.bucket_T)
    np.testing.assert_array_equal(got.n_ex, td.n_ex)
    np.testing.assert_array_equal(got.Q, td.Q)
    np.testing.assert_array_equal(got.kid, td.kid)
    np.testing.assert_array_equal(got.noda, td.noda)
    p = str(tmp_path / "t.damoe")
    t.save(p)
    t2 = damoe.Table.load(p)
    g2 = t2.data(E)
    np.testing.assert_array_equal(g2.Q, td.Q)
    np.testing.assert_array_equal(g2.kid, td.kid)
    # A file written for another variant set is rejected.
    txt = open(p).read().split("\n")
    txt[0] = "damoe-table 1 2,other,set"
    open(p, "w").write("\n".join(txt))
    with pytest.raises(damoe.DamoeError) as ei:
        damoe.Table.load(p)
    assert ei.value.code == -4
    with pytest.raises(damoe.DamoeError) as ei:
        damoe.Table.load(str(tmp_path / "missing"))
    assert ei.value.code == -7
    # Invalid descriptions.
    for bad in (dict(bucket_T=np.array([4, 1, 16])), dict(n_ex=np.array([0, 3, 3])),
                dict(kid=np.full(6, nv)), dict(noda=np.array([0, 0, -1]))):
        d = damoe.TableData(**{**td.__dict__, **bad})
        with pytest.raises(damoe.DamoeError):
            damoe.Table.create(d)


def test_committed_tables_match_the_variant_registry():
    # bench.py loads these; a table written for another variant set would be rejected and
    # silently replaced by a quick start-up tune.
    tdir = os.path.join(ROOT, "paper_2607_23099_amd", "tables")
    names = sorted(f for f in os.listdir(tdir) if f.endswith(".damoe"))
    assert {"dsv3.damoe", "kimi-k2.damoe"} <= set(names)
    nv = damoe.num_variants()
    for f in names:
        t = damoe.Table.load(os.path.join(tdir, f))
        E = 384 if f.startswith("kimi") else 256 // (int(f.split("-ep")[1].split(".")[0]) if "-ep" in f else 1)
        td = t.data(E)
        assert td.kid.min() >= 0 and td.kid.max() < nv and td.noda.max() < nv
        assert np.all(np.diff(td.bucket_T) > 0)
        # every bucket's candidate mask holds exactly its kernels, plus its noda kernel when
        # it names several
        for b, T in enumerate(td.bucket_T):
            want = 0
            for v in td.kid[td.bucket_rows(b)]:
                want |= 1 << int(v)
            if bin(want).count("1") > 1:
                want |= 1 << int(td.noda[b])
            assert t.candidates(int(T)) == want


def test_router_validation_and_workspace_bound():
    L = damoe.lib()
    P = 0x10000  # never dereferenced: every call below stops in validation
    big = 1 << 40
    r = L.damoe_router
    assert r(P, P, None, 4, 256, 8, 9, None, P, P, P, big, None) == -1      # k > E
    assert r(P, P, None, 4, 256, 2048, 8, None, P, P, P, big, None) == -1   # E beyond the limit
    assert r(P, P, None, 4, 256, 8, 0, None, P, P, P, big, None) == -1      # k = 0
    assert r(P, P, None, -1, 256, 8, 2, None, P, P, P, big, None) == -1
    assert r(P, P, None, 4, 0, 8, 2, None, P, P, P, big, None) == -1
    assert r(P, P, None, 4, 100, 8, 2, None, P, P, P, big, None) == -2      # H not a multiple of 64
    assert r(P, P, None, 150000, 7168, 8, 2, None, P, P, P, big, None) == -2  # T*H*2 >= 2^31
    assert r(None, None, None, 0, 256, 8, 2, None, None, None, None, 0, None) == 0  # T = 0: no-op
    assert r(P, P, None, 4, 256, 8, 2, None, P, P, P, 0, None) == -3
    assert r(P, P, None, 4, 256, 8, 2, None, None, P, P, big, None) == -1    # no ids
    assert r(P, P, None, 4, 256, 8, 2, None, P, P, None, big, None) == -1    # no workspace
    assert damoe.router_workspace_size(0, 256, 4) == 0
    assert damoe.router_workspace_size(8, 100, 4) == 0
    # The size for T_max covers every T <= T_max (the split count, and with it S * T, is not
    # monotone in T): a call with that many bytes passes the workspace check and stops at the
    # missing activations instead.
    rng = np.random.default_rng(0)
    for E, H, T_max in [(8, 256, 600), (256, 7168, 4096), (384, 7168, 3000), (1000, 64, 300)]:
        ws = damoe.router_workspace_size(E, H, T_max)
        assert ws >= T_max * E * 4
        for T in np.unique(np.r_[1, T_max, rng.integers(1, T_max + 1, 300), np.arange(1, min(T_max, 300))]):
            assert r(None, P, None, int(T), H, E, 1, None, P, P, P, ws, None) == -1, (E, H, T)
            assert r(None, P, None, int(T), H, E, 1, None, P, P, P, 16, None) == -3


def test_effexp_map_matches_oracle():
    # The library derives each bucket's Effective-Experts map when a table is created; the
    # oracle derives it from the same exemplars independently.
    tdir = os.path.join(ROOT, "paper_2607_23099_amd", "tables")
    for f in ("dsv3.damoe", "kimi-k2.damoe"):
        t = damoe.Table.load(os.path.join(tdir, f))
        E = 256 if f.startswith("dsv3") else 384
        td = t.data(E)
        for b, T in enumerate(td.bucket_T):
            want = oracle.effexp_map(td.Q[td.bucket_rows(b)], td.kid[td.bucket_rows(b)], int(td.noda[b]))
            np.testing.assert_array_equal(t.effexp_map(int(T)), want)
            assert t.effexp_candidates(int(T)) == int(np.bitwise_or.reduce(1 << want.astype(np.int64)))
    rng = np.random.default_rng(3)
    nv = damoe.num_variants()
    for _ in range(20):
        E = int(rng.integers(2, 300))
        n_ex = rng.integers(1, 9, 3)
        Q = -np.sort(-(rng.integers(0, 32769, (int(n_ex.sum()), E)) * (rng.random((int(n_ex.sum()), E)) <
                                                                      rng.random())), axis=1)
        td = damoe.TableData(E=E, k=1, H=256, I=512, wdtype=0, bucket_T=np.array([4, 16, 64]), n_ex=n_ex,
                             Q=Q, kid=rng.integers(0, nv, int(n_ex.sum())), noda=rng.integers(0, nv, 3))
        t = damoe.Table.create(td)
        for b, T in enumerate((1, 16, 1000)):
            rows = td.bucket_rows(b)
            np.testing.assert_array_equal(t.effexp_map(T), oracle.effexp_map(Q[rows], td.kid[rows], int(td.noda[b])))


def test_effexp_dispatch_validation():
    L = damoe.lib()
    P = 0x10000
    E = 8
    td = damoe.TableData(E=E, k=2, H=256, I=512, wdtype=0, bucket_T=np.array([8]), n_ex=np.array([1]),
                         Q=np.full((1, E), 1000), kid=np.array([1]), noda=np.array([0]))
    for bad in (np.full((1, E), -1), np.full((1, E), 65537)):
        with pytest.raises(damoe.DamoeError):
            damoe.Table.create(damoe.TableData(**{**td.__dict__, "Q": bad}))
    t = damoe.Table.create(td)
    rd = L.damoe_route_dispatch_effexp
    assert rd(None, P, 4, 2, E, P, P, P, P, P, P, P, P, 1 << 30, None) == -1
    assert rd(t.handle, P, 4, 2, E, P, P, P, P, P, P, None, P, 1 << 30, None) == -1
    assert rd(t.handle, P, 4, 3, E, P, P, P, P, P, P, P, P, 1 << 30, None) == -4
    assert L.damoe_table_effexp_map(None, 4, P) == -1
    assert L.damoe_table_effexp_candidates(None, 4) == 0


def test_tune_rejects_bad_repeat_config():
    # Validated before any device work: repeat fractions outside 1..100, a missing array, too
    # many, or combined with expert parallelism.
    L = damoe.lib()
    lay = _fake_layer()
    bT = np.array([1, 4], np.int32)
    sx = np.array([1.1, 2.0], np.float64)

    def cfg(n_repeat, rf, ep=1):
        arr = np.asarray(rf, np.int32)
        c = damoe.TuneConfig(2, bT.ctypes.data, 2, sx.ctypes.data, 1, 1, 4, 4, 0, 0x10000, 0, ep, n_repeat,
                             arr.ctypes.data if len(arr) else None)
        return c, arr

    for n, rf, ep in [(1, [0], 1), (1, [101], 1), (2, [50, -3], 1), (1, [], 1), (65, [50] * 65, 1),
                      (-1, [], 1), (1, [50], 2)]:
        c, keep = cfg(n, rf, ep)
        h = ctypes.c_void_p()
        assert L.damoe_tune(ctypes.byref(lay), ctypes.byref(c), ctypes.byref(h), None) == -1, (n, rf, ep)
    for bad_flush in (-1, 16385):  # the cache-evicting write: 0 .. 16 GiB
        c, keep = cfg(0, [])
        c.flush_mib = bad_flush
        assert L.damoe_tune(ctypes.byref(lay), ctypes.byref(c), ctypes.byref(h), None) == -1, bad_flush
