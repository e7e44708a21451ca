"""GPU parity of a6-a8: the fused MoE layer of every variant against the CPU oracle."""
import numpy as np
import pytest

from paper_2607_23099_amd import damoe, synth
from tests.gpu_common import (TOL, Reference, bf16_rows, log, oracle_rows, row_err, tile_rows, torch_cuda,
                               variants_agree)

pytestmark = pytest.mark.gpu


def _variants(wdtype=damoe.W_BF16):
    """The variants that run a layer with these weights (every one for fp8; all but the
    fp8-MFMA big tile for bf16)."""
    return [v for v in range(damoe.num_variants()) if damoe.variant_supports(v, wdtype)]


def _run(path, r, x_tag, variant=None, table=None):
    """One layer call: route (+ dispatch when a table is given) and the fused computation."""
    torch = torch_cuda()
    path.set_routing(r)
    path.fill_x(r.T, x_tag)
    path.y.fill_(float("nan"))
    if table is not None:
        path.route_dispatch(table, r.T)
        path.fused(r.T, -1)
    else:
        path.route(r.T)
        path.fused(r.T, variant)
    torch.cuda.synchronize()


@pytest.fixture(scope="module", params=[False, True], ids=["rowmajor", "packed"])
def tiny(request):
    torch = torch_cuda()
    from paper_2607_23099_amd.moe import DeviceLayer, Path
    dl = DeviceLayer(synth.TINY, packed=request.param)
    yield dl, Path(dl, 256)
    torch.cuda.empty_cache()


@pytest.mark.parametrize("T,alpha,seed", [(64, 1.0, 0), (1, 1.0, 1), (37, 0.05, 2), (200, 10.0, 3)])
def test_tiny_every_variant(tiny, T, alpha, seed):
    dl, path = tiny
    sh = dl.shape
    r = synth.routing(sh.E, sh.k, T, alpha, [seed] if seed else 0)
    ref = oracle_rows(sh, r, seed, np.arange(T))
    for v in _variants():
        log(f"tiny T={T} alpha={alpha} variant={damoe.variant_name(v)}")
        _run(path, r, seed, v)
        err = row_err(bf16_rows(path.y, np.arange(T)), ref)
        assert err <= TOL["bf16"], (v, err)
        assert path.ctrl()[4] == v


@pytest.mark.parametrize("noda_same", [False, True], ids=["noda-other", "noda-same"])
def test_tiny_adaptive_uses_device_variant(tiny, noda_same):
    # A one-kernel bucket: its candidate mask is that kernel alone, whatever noda is, and
    # the launch runs it directly; the device-side id still records it.
    torch = torch_cuda()
    dl, path = tiny
    sh = dl.shape
    r = synth.routing(sh.E, sh.k, 64, 1.0, 0)
    for target in _variants():
        q = np.full((1, sh.E), int(round(2 ** 15 / np.sqrt(sh.E))), np.int32)
        noda = target if noda_same else 0
        td = damoe.TableData(E=sh.E, k=sh.k, H=sh.H, I=sh.I, wdtype=0, bucket_T=np.array([1 << 20]),
                             n_ex=np.array([1]), Q=q, kid=np.array([target]), noda=np.array([noda]))
        table = damoe.Table.create(td)
        assert table.candidates(64) == 1 << target  # one exemplar: one kernel, no noda
        _run(path, r, 0, table=table)
        assert int(path.variant.item()) == target and path.ctrl()[4] == target
        y_adaptive = path.y[:64].clone()
        _run(path, r, 0, variant=target)
        assert torch.equal(y_adaptive, path.y[:64])
    assert damoe.read_device_error(path.ws) == 0


def test_tiny_dispatch_outside_candidates_is_flagged(tiny):
    # A dispatched id that the caller's candidate mask does not hold runs no expert GEMM and
    # sets the sticky device error, whichever kernel class holds it (y is then unspecified).
    torch = torch_cuda()
    dl, path = tiny
    sh = dl.shape
    r = synth.routing(sh.E, sh.k, 64, 1.0, 0)
    big = [damoe.variant_name(v) for v in range(damoe.num_variants())].index("big_bm256")
    # masks of two variants, so the launches still read the device-side id
    for target, cand in [(3, 0b11), (big, 0b11), (0, (1 << big) | (1 << (big - 1)))]:
        q = np.full((1, sh.E), 1000, np.int32)
        td = damoe.TableData(E=sh.E, k=sh.k, H=sh.H, I=sh.I, wdtype=0, bucket_T=np.array([1 << 20]),
                             n_ex=np.array([1]), Q=q, kid=np.array([target]), noda=np.array([target]))
        table = damoe.Table.create(td)
        path.set_routing(r)
        path.fill_x(64, 0)
        path.y.fill_(float("nan"))
        path.route_dispatch(table, 64)
        path.candidates = cand
        path.fused(64, -1)
        torch.cuda.synchronize()
        assert int(path.variant.item()) == target
        assert damoe.read_device_error(path.ws) == damoe.DEVERR_VARIANT


SMALL_FP8 = synth.Shape("small-fp8", E=8, k=2, H=512, I=1024, shape_id=5, wdtype="fp8")


def test_tiny_large_tile_calls_repeat_after_one_route(tiny):
    # The tiled and big-tile kernels take their items from work queues whose counters live in
    # the workspace: each launch returns them to zero, so fused calls repeated after one routing
    # call (as a tuner or a graph replay makes them) compute the same layer, bit for bit.
    torch = torch_cuda()
    dl, path = tiny
    sh = dl.shape
    r = synth.routing(sh.E, sh.k, 250, 0.3, [77])
    rows = np.arange(0, 250, 37)
    ref = oracle_rows(sh, r, 77, rows)
    big = [v for v in _variants() if damoe.variant_tile_m(v) >= 128]
    assert big
    _run(path, r, 77, big[0])
    for v in big:
        outs = []
        for rep in range(3):
            path.y.fill_(float("nan"))
            path.fused(r.T, v)
            torch.cuda.synchronize()
            outs.append(path.y[:r.T].clone())
        log(f"tiny repeated calls variant={damoe.variant_name(v)}")
        assert row_err(bf16_rows(outs[0], rows), ref) <= TOL["bf16"]
        for o in outs[1:]:
            assert torch.equal(o.view(torch.int16), outs[0].view(torch.int16))
    assert damoe.read_device_error(path.ws) == 0


@pytest.fixture(scope="module", params=[False, True], ids=["rowmajor", "packed"])
def small_fp8(request):
    torch = torch_cuda()
    from paper_2607_23099_amd.moe import DeviceLayer, Path
    dl = DeviceLayer(SMALL_FP8, packed=request.param)
    yield dl, Path(dl, 512), synth.ExpertWeightSource(SMALL_FP8)
    torch.cuda.empty_cache()


@pytest.mark.parametrize("T,alpha,seed", [(64, 1.0, 4), (300, 0.05, 5), (3, 10.0, 6)])
def test_small_fp8_every_variant(small_fp8, T, alpha, seed):
    # fp8 block-128 weights in both layouts, tiles of every size incl. two 256-token tiles.
    dl, path, src = small_fp8
    sh = dl.shape
    r = synth.routing(sh.E, sh.k, T, alpha, [seed])
    rows = np.arange(T) if T <= 64 else np.sort(np.random.default_rng(T).choice(T, 48, replace=False))
    ref = oracle_rows(sh, r, seed, rows, src)
    for v in _variants(damoe.W_FP8_B128):
        log(f"small fp8 T={T} alpha={alpha} variant={damoe.variant_name(v)}")
        _run(path, r, seed, v)
        err = row_err(bf16_rows(path.y, rows), ref)
        assert err <= TOL["fp8"], (v, err)


def test_fused_reads_no_tile_list_of_another_T(tiny):
    # The routing call stamps its tile lists with T k.  A fused call with another T (whose
    # layout puts the lists elsewhere) reads none of them: every kernel class skips its items
    # and sets DAMOE_DEVERR_TILES.  The same T afterwards runs cleanly.
    torch = torch_cuda()
    dl, path = tiny
    sh = dl.shape
    r = synth.routing(sh.E, sh.k, 200, 1.0, [31])
    path.set_routing(r)
    path.fill_x(200, 31)
    path.route(200)
    assert damoe.read_device_error(path.ws) == 0
    for v in _variants():
        for T2 in (64, 150):
            log(f"stale tile lists: routed T=200, fused T={T2}, variant={damoe.variant_name(v)}")
            path.fused(T2, v)
            torch.cuda.synchronize()
            assert damoe.read_device_error(path.ws) == damoe.DEVERR_TILES, (v, T2)
    rows = np.arange(0, 200, 9)
    ref = oracle_rows(sh, r, 31, rows)
    for v in _variants():
        _run(path, r, 31, v)
        assert row_err(bf16_rows(path.y, rows), ref) <= TOL["bf16"]
    assert damoe.read_device_error(path.ws) == 0


def test_dispatch_rejects_counts_that_are_no_histogram(tiny):
    # damoe_dispatch takes its counts from the caller: a negative count, or counts summing past
    # T k, write the bucket's noda variant and set DAMOE_DEVERR_COUNTS.
    torch = torch_cuda()
    dl, path = tiny
    sh = dl.shape
    table = damoe.Table.create(damoe.TableData(
        E=sh.E, k=sh.k, H=sh.H, I=sh.I, wdtype=0, bucket_T=np.array([1 << 20]), n_ex=np.array([2]),
        Q=np.array([[30000] + [0] * (sh.E - 1), [11585] * sh.E], np.int32), kid=np.array([1, 2]),
        noda=np.array([5])))
    T = 64
    good = np.full(sh.E, T * sh.k // sh.E, np.int32)
    for counts, want_v, want_err in [
            (good, 2, 0),                                                     # uniform: exemplar 1
            (np.r_[T * sh.k, np.zeros(sh.E - 1, np.int32)], 1, 0),           # one expert: exemplar 0
            (np.r_[-1, good[1:]], 5, damoe.DEVERR_COUNTS),                    # a negative count
            (good + 1, 5, damoe.DEVERR_COUNTS),                               # sum above T k
            (np.r_[2 ** 31 - 1, 2 ** 31 - 1, good[2:]], 5, damoe.DEVERR_COUNTS)]:  # no int overflow
        path.counts.copy_(torch.from_numpy(np.asarray(counts, np.int32)))
        path.variant.fill_(-9)
        damoe.dispatch(table, path.counts, T, path.variant, path.ws)
        torch.cuda.synchronize()
        assert int(path.variant.item()) == want_v, counts
        assert damoe.read_device_error(path.ws) == want_err, counts


def test_tiny_zero_tokens_is_noop(tiny):
    torch = torch_cuda()
    dl, path = tiny
    path.y.fill_(3.0)
    r = synth.routing(dl.shape.E, dl.shape.k, 0, 1.0, 0)
    path.route(0)
    path.fused(0, 0)
    torch.cuda.synchronize()
    assert bool((path.y == 3.0).all())


def test_cold_experts_are_never_read():
    # Experts without tokens hold NaN weights; the output must not see them.
    torch = torch_cuda()
    from paper_2607_23099_amd.moe import DeviceLayer, Path
    sh = synth.Shape("tiny-cold", E=16, k=2, H=256, I=512, shape_id=0)
    dl = DeviceLayer(sh)
    path = Path(dl, 64)
    r = synth.routing(sh.E, sh.k, 64, 0.05, [21])
    cold = sorted(set(range(sh.E)) - set(np.unique(r.ids).tolist()))
    assert cold, "routing should leave some experts cold"
    for name in ("w1", "w3", "w2"):
        dl.w[name][cold] = float("nan")
    ref = oracle_rows(sh, r, 21, np.arange(64))
    for v in _variants():
        _run(path, r, 21, v)
        y = bf16_rows(path.y, np.arange(64))
        assert np.all(np.isfinite(y))
        assert row_err(y, ref) <= TOL["bf16"]


# Full-size cases: every point the benchmarks time, on their routing seeds and tokens.  Each
# case compares at least 64 token rows chosen from the oracle's tile lists (tile_rows: the
# ends of the first, last and first full tile of every tile size, the hottest expert's ragged
# last tile, token blocks 4..7 of a 256-row tile, a one-token expert) with the oracle, and
# every row of every variant with the first variant's output.
DS_POINTS = [(T, a) for T in (1, 8, 32, 128) for a in (0.05, 0.3, 1.0, 10.0)]
PREFILL_POINTS = [(T, a) for T in (1024, 4096, 16384) for a in (0.05, 0.3, 1.0, 10.0)]
KIMI_POINTS = [16, 256, 2048, 8192]
DECODE_X, PREFILL_X = 1, 5  # activation tags of the decode sweep and of the prefill grid


def _check_variants(path, r, x_tag, rows, ref, tol, variants, what):
    """Every variant on one routing: the chosen rows against the oracle, all rows against the
    first variant's output."""
    torch = torch_cuda()
    first = None
    for v in variants:
        log(f"{what} variant={damoe.variant_name(v)} ({len(rows)} oracle rows)")
        _run(path, r, x_tag, v)
        err = row_err(bf16_rows(path.y, rows), ref)
        assert err <= tol, (v, err)
        if first is None:
            first = path.y[:r.T].clone()
        else:
            agree = variants_agree(path.y, first, r.T)
            assert agree <= tol, (v, agree)
    assert damoe.read_device_error(path.ws) == 0
    del first
    torch.cuda.empty_cache()


def _cases(sh, points, routing_of, x_tag):
    cases = {}
    for p in points:
        r = routing_of(p)
        rows = tile_rows(r, sh.E, seed=r.T)
        cases[p] = (r, synth.activations_host(r.T, sh.H, x_tag, rows), rows)
    return cases


@pytest.fixture(scope="module")
def ds():
    torch = torch_cuda()
    from paper_2607_23099_amd.moe import DeviceLayer, Path
    log("filling DeepSeek-V3-shaped bf16 layer (22.5 GB)")
    dl = DeviceLayer(synth.DS)
    torch.cuda.synchronize()
    sh = dl.shape
    cases = _cases(sh, DS_POINTS, lambda p: synth.routing(sh.E, sh.k, p[0], p[1], synth.seed_decode(p[0], p[1], 0)),
                   DECODE_X)
    ref = Reference(sh, cases)
    yield dl, Path(dl, 128), cases, ref
    del dl
    torch.cuda.empty_cache()


@pytest.mark.parametrize("T,alpha", DS_POINTS)
def test_ds_decode_every_variant(ds, T, alpha):
    dl, path, cases, ref = ds
    r, _, rows = cases[T, alpha]
    _check_variants(path, r, DECODE_X, rows, ref.y[T, alpha], TOL["bf16"], _variants(),
                    f"ds decode T={T} alpha={alpha}")


@pytest.fixture(scope="module")
def kimi():
    torch = torch_cuda()
    from paper_2607_23099_amd.moe import DeviceLayer, Path
    log("filling Kimi-K2-shaped bf16 layer (33.8 GB)")
    dl = DeviceLayer(synth.KIMI)
    torch.cuda.synchronize()
    sh = dl.shape
    cases = _cases(sh, KIMI_POINTS, lambda T: synth.routing(sh.E, sh.k, T, 0.05, synth.seed_kimi(T, 0), n_hot=4),
                   PREFILL_X)
    ref = Reference(sh, cases)
    yield dl, Path(dl, 8192), cases, ref
    del dl
    torch.cuda.empty_cache()


@pytest.mark.parametrize("T", KIMI_POINTS)
def test_kimi_hot_experts(kimi, T):
    dl, path, cases, ref = kimi
    r, _, rows = cases[T]
    _check_variants(path, r, PREFILL_X, rows, ref.y[T], TOL["bf16"], _variants(), f"kimi T={T}")


@pytest.fixture(scope="module")
def ds_fp8():
    torch = torch_cuda()
    from paper_2607_23099_amd.moe import DeviceLayer, Path
    log("filling DeepSeek-V3-shaped fp8 block-128 layer")
    dl = DeviceLayer(synth.DS_FP8)
    torch.cuda.synchronize()
    sh = dl.shape
    cases = _cases(sh, PREFILL_POINTS,
                   lambda p: synth.routing(sh.E, sh.k, p[0], p[1], synth.seed_prefill(p[0], p[1], 0)), PREFILL_X)
    ref = Reference(sh, cases)
    yield dl, Path(dl, 16384), cases, ref
    del dl
    torch.cuda.empty_cache()


@pytest.mark.parametrize("T,alpha", PREFILL_POINTS)
def test_ds_prefill_fp8(ds_fp8, T, alpha):
    dl, path, cases, ref = ds_fp8
    r, _, rows = cases[T, alpha]
    _check_variants(path, r, PREFILL_X, rows, ref.y[T, alpha], TOL["fp8"], _variants(damoe.W_FP8_B128),
                    f"ds fp8 prefill T={T} alpha={alpha}")


SMALL_MXFP4 = synth.Shape("small-mxfp4", E=8, k=2, H=512, I=1024, shape_id=6, wdtype="mxfp4")


def _stream_variants(wdtype):
    return [v for v in range(damoe.num_variants()) if damoe.variant_supports(v, wdtype)]


@pytest.fixture(scope="module")
def small_mxfp4():
    torch = torch_cuda()
    from paper_2607_23099_amd.moe import DeviceLayer, Path
    dl = DeviceLayer(SMALL_MXFP4, packed=True)
    yield dl, Path(dl, 512), synth.ExpertWeightSource(SMALL_MXFP4)
    torch.cuda.empty_cache()


def test_mxfp4_device_fill_equals_host_fill(small_mxfp4):
    # The row-major fill before packing: regenerate one expert on the device and on the host.
    torch = torch_cuda()
    sh = SMALL_MXFP4
    for name in ("w1", "w2"):
        tid, r, c = synth.weight_dims(sh, name)
        q = torch.empty((2, r, c // 2), dtype=torch.uint8, device="cuda")
        s = torch.empty((2, r, c // 32), dtype=torch.uint8, device="cuda")
        synth.fill_mxfp4_device(q.data_ptr(), s.data_ptr(), r, c, 2, seed=sh.weight_seed, tensor=tid, slab0=3,
                                sigma=sh.w_sigma, stream=torch.cuda.current_stream().cuda_stream)
        torch.cuda.synchronize()
        qh, sh_ = synth.fill_mxfp4_host(r, c, 2, seed=sh.weight_seed, tensor=tid, slab0=3, sigma=sh.w_sigma)
        np.testing.assert_array_equal(q.cpu().numpy(), qh)
        np.testing.assert_array_equal(s.cpu().numpy(), sh_)


@pytest.mark.parametrize("T,alpha,seed", [(64, 1.0, 7), (300, 0.05, 8), (3, 10.0, 9), (1, 1.0, 10)])
def test_small_mxfp4_every_stream_variant(small_mxfp4, T, alpha, seed):
    dl, path, src = small_mxfp4
    sh = dl.shape
    r = synth.routing(sh.E, sh.k, T, alpha, [seed])
    rows = np.arange(T) if T <= 64 else np.sort(np.random.default_rng(T).choice(T, 48, replace=False))
    ref = oracle_rows(sh, r, seed, rows, src)
    variants = _stream_variants(damoe.W_MXFP4)
    assert len(variants) >= 4 and not damoe.variant_supports(damoe.num_variants() - 1, damoe.W_MXFP4)
    for v in variants:
        log(f"small mxfp4 T={T} alpha={alpha} variant={damoe.variant_name(v)}")
        _run(path, r, seed, v)
        err = row_err(bf16_rows(path.y, rows), ref)
        assert err <= TOL["bf16"], (v, err)


def test_mxfp4_reads_no_tile_list_of_another_T(small_mxfp4):
    torch = torch_cuda()
    dl, path, _ = small_mxfp4
    sh = dl.shape
    r = synth.routing(sh.E, sh.k, 100, 1.0, [12])
    path.set_routing(r)
    path.fill_x(100, 12)
    path.route(100)
    assert damoe.read_device_error(path.ws) == 0
    for v in _stream_variants(damoe.W_MXFP4):
        path.fused(40, v)
        torch.cuda.synchronize()
        assert damoe.read_device_error(path.ws) == damoe.DEVERR_TILES, v


def test_mxfp4_rejects_other_kernel_classes(small_mxfp4):
    # Host: a forced tiled or big variant is unsupported.  Device: a dispatched id of another
    # class runs nothing and sets the sticky error.
    torch = torch_cuda()
    dl, path, _ = small_mxfp4
    sh = dl.shape
    r = synth.routing(sh.E, sh.k, 64, 1.0, [11])
    path.set_routing(r)
    path.fill_x(64, 11)
    path.route(64)
    for v in range(damoe.num_variants()):
        if not damoe.variant_supports(v, damoe.W_MXFP4):
            with pytest.raises(damoe.DamoeError) as ei:
                path.fused(64, v)
            assert ei.value.code == -2
    q = np.full((1, sh.E), 1000, np.int32)
    td = damoe.TableData(E=sh.E, k=sh.k, H=sh.H, I=sh.I, wdtype=damoe.W_MXFP4, bucket_T=np.array([1 << 20]),
                         n_ex=np.array([1]), Q=q, kid=np.array([6]), noda=np.array([0]))
    table = damoe.Table.create(td)
    path.route_dispatch(table, 64)
    path.candidates = 0b1100001  # the tiled id plus two stream variants
    path.fused(64, -1)
    torch.cuda.synchronize()
    assert int(path.variant.item()) == 6
    assert damoe.read_device_error(path.ws) == damoe.DEVERR_VARIANT


@pytest.fixture(scope="module")
def ds_mxfp4():
    torch = torch_cuda()
    from paper_2607_23099_amd.moe import DeviceLayer, Path
    log("filling DeepSeek-V3-shaped MXFP4 layer (5.9 GB)")
    dl = DeviceLayer(synth.DS_MXFP4)
    torch.cuda.synchronize()
    sh = dl.shape
    cases = _cases(sh, DS_POINTS, lambda p: synth.routing(sh.E, sh.k, p[0], p[1], synth.seed_decode(p[0], p[1], 0)),
                   DECODE_X)
    ref = Reference(sh, cases)
    yield dl, Path(dl, 128), cases, ref
    del dl
    torch.cuda.empty_cache()


@pytest.mark.parametrize("T,alpha", DS_POINTS)
def test_ds_mxfp4_decode(ds_mxfp4, T, alpha):
    dl, path, cases, ref = ds_mxfp4
    r, _, rows = cases[T, alpha]
    _check_variants(path, r, DECODE_X, rows, ref.y[T, alpha], TOL["bf16"], _stream_variants(damoe.W_MXFP4),
                    f"ds mxfp4 T={T} alpha={alpha}")
