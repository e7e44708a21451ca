"""GPU parity of a2-a5: histogram, Effective Experts, permutation, token tiles, dispatch.

Every integer output is compared bit-exactly with the CPU oracle.
"""
import numpy as np
import pytest

import oracle
from paper_2607_23099_amd import damoe, synth
from tests.gpu_common import log, tiles_expected, torch_cuda

pytestmark = pytest.mark.gpu

ROUTE_CASES = (
    [("tiny", 8, 2, 64, 1.0, 0, [0])] +
    [("ds-decode", 256, 8, T, a, 0, synth.seed_decode(T, a, 0)) for T in (1, 8, 32, 128)
     for a in (0.05, 0.3, 1.0, 10.0)] +
    [("ds-prefill", 256, 8, T, a, 0, synth.seed_prefill(T, a, 0)) for T in (1024, 4096, 16384)
     for a in (0.05, 10.0)] +
    [("kimi", 384, 8, T, 0.05, 4, synth.seed_kimi(T, 0)) for T in (16, 256, 2048, 8192)] +
    [("e1k1", 1, 1, 100, 1.0, 0, [7]), ("emax", 1024, 16, 3000, 0.3, 0, [8]),
     ("odd", 37, 5, 777, 0.2, 0, [9])] +
    # Many assignments (blocks of 2048): 5 blocks, the last one 3 ids long; a single expert.
    [("odd-blocks", 37, 5, 1639, 0.2, 0, [10]), ("e1k1-blocks", 1, 1, 9001, 1.0, 0, [11])]
)


class RouteBufs:
    def __init__(self, torch, E, k, T):
        A = max(T * k, 1)
        dev = "cuda"
        self.ids = torch.zeros(A, dtype=torch.int32, device=dev)
        self.counts = torch.full((E,), -7, dtype=torch.int32, device=dev)
        self.offsets = torch.full((E + 1,), -7, dtype=torch.int32, device=dev)
        self.perm = torch.full((A,), -7, dtype=torch.int32, device=dev)
        self.inv = torch.full((A,), -7, dtype=torch.int32, device=dev)
        self.nd = torch.zeros(2, dtype=torch.int64, device=dev)
        self.bucket = torch.zeros(1, dtype=torch.int32, device=dev)
        self.lo = damoe.workspace_layout(E, k, 128, 128, T)
        self.ws = torch.zeros(self.lo["h"], dtype=torch.uint8, device=dev)
        self.E, self.k, self.T = E, k, T

    def run(self, ids_np):
        torch = torch_cuda()
        if self.T:
            self.ids.copy_(torch.from_numpy(np.ascontiguousarray(ids_np.ravel(), np.int32)))
        damoe.route_histogram(self.ids, self.T, self.k, self.E, self.counts, self.offsets, self.perm,
                              self.inv, self.nd, self.bucket, self.ws)
        torch.cuda.synchronize()

    def tiles(self, cls):
        import torch
        off = self.lo["tiles"][cls]
        n = int(self.ws[off:off + 4].view(torch.int32).item())
        return self.ws[off + 8: off + 8 + 8 * n].view(torch.int32).cpu().numpy().reshape(n, 2).astype(np.int64)


def _check_route(b: RouteBufs, ids_np):
    E, A = b.E, b.T * b.k
    counts = oracle.histogram(ids_np, E)
    np.testing.assert_array_equal(b.counts.cpu().numpy(), counts)
    offsets, perm, inv = oracle.permute(ids_np, E)
    np.testing.assert_array_equal(b.offsets.cpu().numpy(), offsets)
    n_valid = int(offsets[E])
    if A:
        np.testing.assert_array_equal(b.perm.cpu().numpy()[:n_valid], perm)
        np.testing.assert_array_equal(b.inv.cpu().numpy()[:A], inv)
    num, den, _ = oracle.effexp(counts)
    nd = b.nd.cpu().numpy().view(np.uint64)
    assert (int(nd[0]), int(nd[1])) == (num, den)
    assert int(b.bucket.item()) == oracle.effexp_bucket(num, den, E)
    for cls in range(damoe.N_TILE_SIZES):
        np.testing.assert_array_equal(b.tiles(cls), tiles_expected(counts, 16 << cls))


@pytest.mark.parametrize("case", ROUTE_CASES, ids=lambda c: f"{c[0]}-E{c[1]}-k{c[2]}-T{c[3]}-a{c[4]}")
def test_route_matches_oracle(case):
    torch = torch_cuda()
    name, E, k, T, alpha, hot, seed = case
    log(f"route {name} E={E} k={k} T={T} alpha={alpha}")
    r = synth.routing(E, k, T, alpha, seed, n_hot=hot)
    b = RouteBufs(torch, E, k, T)
    b.run(r.ids)
    _check_route(b, r.ids)
    # Deterministic: a second run gives identical bits.
    first = (b.perm.clone(), b.inv.clone())
    b.run(r.ids)
    assert torch.equal(first[0], b.perm) and torch.equal(first[1], b.inv)


def test_route_edge_cases():
    torch = torch_cuda()
    # T = 0: empty histogram, bucket -1.
    b = RouteBufs(torch, 64, 4, 0)
    b.run(np.zeros((0, 4), np.int32))
    assert b.counts.cpu().numpy().tolist() == [0] * 64
    assert int(b.bucket.item()) == -1 and b.nd.cpu().numpy().tolist() == [0, 0]
    for cls in range(damoe.N_TILE_SIZES):
        assert len(b.tiles(cls)) == 0
    # Every token on the same k experts (eff_exp = k), and a one-expert layer (eff_exp = 1).
    for E, k, T in [(256, 8, 600), (1, 1, 50), (8, 1, 1)]:
        ids = np.tile(np.arange(k, dtype=np.int32)[::-1], (T, 1))
        b = RouteBufs(torch, E, k, T)
        b.run(ids)
        _check_route(b, ids)
        nd = b.nd.cpu().numpy()
        assert nd[0] == k * nd[1]  # num / den == k


# (E, k, T): one workgroup, and T * k = 20000 assignments over ten blocks with a ragged last one.
@pytest.mark.parametrize("E,k,T", [(16, 2, 40), (64, 8, 2500)])
def test_route_drops_invalid_ids_and_flags_them(E, k, T):
    torch = torch_cuda()
    r = synth.routing(E, k, T, 1.0, [11])
    ids = r.ids.copy()
    bad = [(3, 0, -1), (7, 1, E), (20, 0, 1000), (T - 1, k - 1, -7)]
    for t, j, v in bad:
        ids[t, j] = v
    b = RouteBufs(torch, E, k, T)
    b.run(ids)
    _check_route(b, ids)
    inv = b.inv.cpu().numpy()
    assert all(inv[t * k + j] == -1 for t, j, _ in bad)
    assert damoe.read_device_error(b.ws) == 1
    assert damoe.read_device_error(b.ws) == 0  # read clears it


@pytest.mark.parametrize("T", [300, 3000])
def test_route_masked_slots_are_not_errors(T):
    # Expert parallelism: negative ids are slots whose expert lives on another rank; they are
    # dropped like invalid ids but raise no device error, also when whole tokens are masked.
    torch = torch_cuda()
    E, k = 64, 8
    r = synth.routing(256, k, T, 1.0, [12])
    ids = np.where(r.ids < E, r.ids, -1).astype(np.int32)  # rank 0 of four
    ids[5] = -1
    b = RouteBufs(torch, E, k, T)
    b.run(ids)
    _check_route(b, ids)
    assert np.all(b.inv.cpu().numpy()[ids.ravel() < 0] == -1)
    assert damoe.read_device_error(b.ws) == 0


def test_route_at_the_largest_sizes():
    # The largest call the header admits: T = 2^20 tokens, k = 16, E = 1024, i.e. 2^24
    # assignments over 8192 blocks of 2048.  Each token takes 16 distinct experts 64 apart
    # from a base skewed towards low ids, so the first experts hold tens of thousands of tiles.
    torch = torch_cuda()
    E, k, T = 1024, 16, 1 << 20
    rng = np.random.default_rng(21)
    base = (E * rng.random(T) ** 3).astype(np.int64)
    ids = ((base[:, None] + 64 * np.arange(k)[None, :]) % E).astype(np.int32)
    log(f"route at the largest sizes: E={E} k={k} T={T}")
    b = RouteBufs(torch, E, k, T)
    b.run(ids)
    _check_route(b, ids)
    assert damoe.read_device_error(b.ws) == 0


def _random_table(rng, E, buckets, nv):
    n_ex = rng.integers(1, 14, len(buckets))
    Q = []
    for b, T in enumerate(buckets):
        for i in range(int(n_ex[b])):
            alpha = float(np.exp(rng.uniform(np.log(0.03), np.log(10))))
            C = np.stack([oracle.histogram(synth.routing(E, 8, min(T, 512), alpha, [77, b, i, s]).ids, E)
                          for s in range(3)])
            Q.append(oracle.exemplar(C))
    Q = np.array(Q, np.int32)
    return damoe.TableData(E=E, k=8, H=7168, I=2048, wdtype=0, bucket_T=np.array(buckets, np.int32),
                           n_ex=n_ex.astype(np.int32), Q=Q, kid=rng.integers(0, nv, len(Q)).astype(np.int32),
                           noda=rng.integers(0, nv, len(buckets)).astype(np.int32))


@pytest.mark.parametrize("E", [256, 384])
def test_dispatch_matches_oracle(E):
    torch = torch_cuda()
    rng = np.random.default_rng(E)
    nv = damoe.num_variants()
    buckets = [2 ** i for i in range(14)]
    td = _random_table(rng, E, buckets, nv)
    table = damoe.Table.create(td)
    counts = torch.zeros(E, dtype=torch.int32, device="cuda")
    vid = torch.full((1,), -9, dtype=torch.int32, device="cuda")
    ws = torch.zeros(4096, dtype=torch.uint8, device="cuda")
    for step in range(60):
        T = int(np.floor(np.exp(rng.uniform(0, np.log(8192)))))
        alpha = float(np.exp(rng.uniform(np.log(0.03), np.log(10))))
        c = oracle.histogram(synth.routing(E, 8, T, alpha, [78, step]).ids, E)
        counts.copy_(torch.from_numpy(c.astype(np.int32)))
        damoe.dispatch(table, counts, T, vid, ws)
        torch.cuda.synchronize()
        b = oracle.select_bucket(td.bucket_T, T)
        rows = td.bucket_rows(b)
        i, scores = oracle.match(c, td.Q[rows])
        assert int(vid.item()) == int(td.kid[rows][i]), (step, T)
        ctrl = ws[:16].view(torch.int32).cpu().numpy()
        assert ctrl[1] == i
        assert int(np.array(ctrl[2:4], np.int32).view(np.int64)[0]) == scores[i]
    # The fused route + dispatch call gives the same histogram, permutation and choice.
    for step in range(20):
        T = int(np.floor(np.exp(rng.uniform(0, np.log(4096)))))
        alpha = float(np.exp(rng.uniform(np.log(0.03), np.log(10))))
        r = synth.routing(E, 8, T, alpha, [79, step])
        b = RouteBufs(torch, E, 8, T)
        b.ids.copy_(torch.from_numpy(r.ids.ravel().copy()))
        vid2 = torch.full((1,), -9, dtype=torch.int32, device="cuda")
        damoe.route_dispatch(table, b.ids, T, 8, E, b.counts, b.offsets, b.perm, b.inv, b.nd, b.bucket, vid2,
                             b.ws)
        torch.cuda.synchronize()
        _check_route(b, r.ids)
        c = oracle.histogram(r.ids, E)
        rows = td.bucket_rows(oracle.select_bucket(td.bucket_T, T))
        i, scores = oracle.match(c, td.Q[rows])
        assert int(vid2.item()) == int(td.kid[rows][i]), (step, T)
        ctrl = b.ws[:16].view(torch.int32).cpu().numpy()
        if np.all(td.kid[rows] == td.kid[rows][0]):
            assert ctrl[1] == -2  # single-variant bucket: written without scoring
        else:
            assert ctrl[1] == i and int(np.array(ctrl[2:4], np.int32).view(np.int64)[0]) == scores[i]
    # No tokens -> the bucket's noda variant.
    counts.zero_()
    damoe.dispatch(table, counts, 0, vid, ws)
    torch.cuda.synchronize()
    assert int(vid.item()) == int(td.noda[0])


def test_dispatch_ties_pick_lowest_index():
    torch = torch_cuda()
    E = 64
    q = np.rint(np.geomspace(9, 1, E) / np.linalg.norm(np.geomspace(9, 1, E)) * 2 ** 15).astype(np.int32)
    other = np.zeros(E, np.int32)
    other[0] = 2 ** 15
    td = damoe.TableData(E=E, k=8, H=256, I=256, wdtype=0, bucket_T=np.array([1 << 20], np.int32),
                         n_ex=np.array([4], np.int32), Q=np.stack([other, q, q, other]),
                         kid=np.array([0, 2, 1, 0], np.int32) % damoe.num_variants(),
                         noda=np.array([0], np.int32))
    table = damoe.Table.create(td)
    c = np.rint(np.geomspace(90, 10, E)).astype(np.int32)
    counts = torch.from_numpy(c).cuda()
    vid = torch.zeros(1, dtype=torch.int32, device="cuda")
    ws = torch.zeros(4096, dtype=torch.uint8, device="cuda")
    T = -(-int(c.sum()) // 8)  # the fewest tokens whose k = 8 slots hold these counts
    damoe.dispatch(table, counts, T, vid, ws)
    torch.cuda.synchronize()
    assert ws[:16].view(torch.int32).cpu().numpy()[0] == 0
    assert ws[:16].view(torch.int32).cpu().numpy()[1] == 1
    assert int(vid.item()) == td.kid[1]


def test_device_fill_equals_host_fill():
    torch = torch_cuda()
    sh = synth.DS
    n = sh.I * sh.H
    t = torch.empty(3 * n, dtype=torch.int16, device="cuda")
    synth.fill_bf16_device(t.data_ptr(), 3 * n, seed=sh.weight_seed, tensor=synth.T_W1, slab0=5,
                           slab_elems=n, sigma=sh.w_sigma)
    got = t.cpu().numpy().view(np.uint16)
    for i in (0, 2):
        want = synth.fill_bf16_host(n, seed=sh.weight_seed, tensor=synth.T_W1, slab0=5 + i, slab_elems=n,
                                    sigma=sh.w_sigma)
        np.testing.assert_array_equal(got[i * n:(i + 1) * n], want)
    q = torch.empty((2, 256, 384), dtype=torch.uint8, device="cuda")
    s = torch.empty((2, 2, 3), dtype=torch.float32, device="cuda")
    synth.fill_fp8_device(q.data_ptr(), s.data_ptr(), 256, 384, 2, seed=9, tensor=synth.T_W2, slab0=3)
    qh, sh_ = synth.fill_fp8_host(256, 384, 2, seed=9, tensor=synth.T_W2, slab0=3)
    np.testing.assert_array_equal(q.cpu().numpy(), qh)
    np.testing.assert_array_equal(s.cpu().numpy(), sh_)


def test_route_dispatch_single_variant_bucket():
    torch = torch_cuda()
    E, k, T = 64, 8, 40
    nv = damoe.num_variants()
    rng = np.random.default_rng(5)
    Q = rng.integers(0, 20000, (3, E)).astype(np.int32)
    td = damoe.TableData(E=E, k=k, H=256, I=256, wdtype=0, bucket_T=np.array([16, 64], np.int32),
                         n_ex=np.array([1, 2], np.int32), Q=Q, kid=np.array([0, 2, 2], np.int32) % nv,
                         noda=np.array([1, 1], np.int32) % nv)
    table = damoe.Table.create(td)
    r = synth.routing(E, k, T, 0.5, [80])
    b = RouteBufs(torch, E, k, T)
    b.ids.copy_(torch.from_numpy(r.ids.ravel().copy()))
    vid = torch.full((1,), -9, dtype=torch.int32, device="cuda")
    damoe.route_dispatch(table, b.ids, T, k, E, b.counts, b.offsets, b.perm, b.inv, b.nd, b.bucket, vid, b.ws)
    torch.cuda.synchronize()
    _check_route(b, r.ids)
    assert int(vid.item()) == 2 % nv and b.ws[:16].view(torch.int32).cpu().numpy()[1] == -2
    # No tokens: the bucket's noda variant.
    b0 = RouteBufs(torch, E, k, 0)
    damoe.route_dispatch(table, b0.ids, 0, k, E, b0.counts, b0.offsets, b0.perm, b0.inv, b0.nd, b0.bucket,
                         vid, b0.ws)
    torch.cuda.synchronize()
    assert int(vid.item()) == 1 % nv


@pytest.mark.parametrize("E", [16, 256, 384])
def test_effexp_dispatch_matches_oracle(E):
    # a2-a5 with the Effective-Experts-only matcher: the same histogram, permutation and tiles
    # as route_histogram, and the variant of the oracle's map at the oracle's bucket.  The
    # skews sweep the whole bucket range; T = 0 takes the NoDA kernel.
    torch = torch_cuda()
    rng = np.random.default_rng(100 + E)
    nv = damoe.num_variants()
    td = _random_table(rng, E, [2 ** i for i in range(14)], nv)
    table = damoe.Table.create(td)
    seen = set()
    for step in range(40):
        T = int(np.floor(np.exp(rng.uniform(0, np.log(4096)))))
        alpha = float(np.exp(rng.uniform(np.log(0.01), np.log(10))))
        r = synth.routing(E, min(8, E), T, alpha, [80, step])
        b = RouteBufs(torch, E, min(8, E), T)
        b.ids.copy_(torch.from_numpy(r.ids.ravel().copy()))
        vid = torch.full((1,), -9, dtype=torch.int32, device="cuda")
        damoe.route_dispatch_effexp(table, b.ids, T, b.k, E, b.counts, b.offsets, b.perm, b.inv, b.nd, b.bucket,
                                    vid, b.ws)
        torch.cuda.synchronize()
        _check_route(b, r.ids)
        c = oracle.histogram(r.ids, E)
        num, den, _ = oracle.effexp(c)
        eb = oracle.effexp_bucket(num, den, E)
        bt = oracle.select_bucket(td.bucket_T, T)
        rows = td.bucket_rows(bt)
        want = oracle.effexp_map(td.Q[rows], td.kid[rows], int(td.noda[bt]))[eb + 1]
        assert int(vid.item()) == int(want), (step, T, eb)
        assert b.ws[:16].view(torch.int32).cpu().numpy()[1] == -3
        seen.add(eb)
    log(f"E={E}: Effective Experts buckets seen {sorted(seen)}")
    assert len(seen) >= 4
    b = RouteBufs(torch, E, min(8, E), 0)
    vid = torch.full((1,), -9, dtype=torch.int32, device="cuda")
    damoe.route_dispatch_effexp(table, b.ids, 0, b.k, E, b.counts, b.offsets, b.perm, b.inv, b.nd, b.bucket, vid,
                                b.ws)
    torch.cuda.synchronize()
    assert int(vid.item()) == int(td.noda[0])
